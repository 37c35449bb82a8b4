"""GPU parity of every step of the hot path against the fp64 oracle.

Calls go through the C ABI (the ctypes binding of libe2f.so).  Bars:
radius graph bit-exact; float32 layer max relative error <= 1e-4 per output
irrep block; bf16 channel mixing <= 1e-2.
"""
import numpy as np
import pytest
import torch

import oracle as o
import e2f_synth as syn
from cases import TOL_BF16, TOL_F32, case, sample_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def e2f():
    import paper_2501_19216_amd as e
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return e


@pytest.fixture(scope="module")
def ctx(e2f):
    c = e2f.e2f_create(6, 0)
    yield c
    c.close()


def gpu(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def run_both(e2f, ctx, inp, rp, ci, alpha, L, H, cutoff, mix=None, mix_bf16=False, tile_side=0.0):
    pos, feat = gpu(inp.pos), gpu(inp.feat)
    row_ptr, col = gpu(rp), gpu(ci)
    al = gpu(alpha)
    gid = None if inp.graph_id is None else gpu(inp.graph_id)
    mw = None
    if mix is not None:
        mw = gpu(mix).to(torch.bfloat16) if mix_bf16 else gpu(mix)
    y6 = e2f.e2f_wigner6j_conv_forward(ctx, pos, feat, row_ptr, col, al, L, H, cutoff, mix_w=mw, graph_id=gid,
                                       tile_side=tile_side)
    ye = e2f.e2f_edge_tp_conv_forward(ctx, pos, feat, row_ptr, col, al, L, H, cutoff, mix_w=mw, graph_id=gid)
    torch.cuda.synchronize()
    return y6.cpu().numpy(), ye.cpu().numpy()


# ------------------------------------------------------------ radius graph
@pytest.mark.parametrize("name", ["cluster32_L2", "molecules256x30_L3", "water2000_L4", "protein20k_L4"])
def test_neighbor_list_bit_exact(e2f, ctx, name):
    inp, rp, ci, _ = case(name)
    wl = inp.workload
    gid = None if inp.graph_id is None else gpu(inp.graph_id)
    g_rp, g_ci = e2f.e2f_neighbor_list(ctx, gpu(inp.pos), wl.cutoff, gid)
    assert torch.equal(g_rp.cpu(), torch.from_numpy(rp))
    assert torch.equal(g_ci.cpu(), torch.from_numpy(ci))


def test_neighbor_list_edge_cases(e2f, ctx):
    # strict inequality on the grid, a single atom, isolated atoms
    pts = np.array([[0, 0, 0], [0, 0, 3.0], [0, 3.0 - 2.0 ** -16, 0], [50, 50, 50]], dtype=np.float32)
    rp, ci = e2f.e2f_neighbor_list(ctx, gpu(pts), 3.0)
    orp, oci = o.neighbor_list(pts, 3.0)
    assert np.array_equal(rp.cpu().numpy(), orp) and np.array_equal(ci.cpu().numpy(), oci)
    rp, ci = e2f.e2f_neighbor_list(ctx, gpu(pts[:1]), 3.0)
    assert rp.cpu().tolist() == [0, 0] and ci.numel() == 0
    with pytest.raises(e2f.E2FError):
        bad = pts.copy()
        bad[1, 2] = np.nan
        e2f.e2f_neighbor_list(ctx, gpu(bad), 3.0)


# ------------------------------------------------------------ per-node steps
def test_solid_harmonics(e2f, ctx):
    rng = np.random.default_rng(3)
    pos = syn.quantize(rng.uniform(-20, 20, size=(300, 3)))
    origins = syn.quantize(rng.uniform(-5, 5, size=(4, 3)))
    oid = rng.integers(0, 4, size=300).astype(np.int32)
    for L in [0, 1, 2, 4, 6]:
        got = e2f.e2f_solid_harmonics(ctx, gpu(pos), L, gpu(origins), gpu(oid)).cpu().numpy()
        ref = o.solid_harmonics(L, pos.astype(np.float64) - origins[oid].astype(np.float64))
        for l in range(L + 1):
            s = slice(l * l, (l + 1) ** 2)
            assert np.max(np.abs(got[:, s] - ref[:, s])) <= 1e-6 * np.max(np.abs(ref[:, s]))


def node_tp_reference(L, pos, feat):
    """[h^(a) (x) R^(b)(p)]^(d) over the blocks used by the factorised layer
    (some u <= L-b and o <= L can reach them), ordered (a, b, d, delta)."""
    tri = lambda a, b, c: abs(a - b) <= c <= a + b
    R = o.solid_harmonics(L, pos.astype(np.float64))
    rows = []
    for a in range(L + 1):
        for b in range(L + 1):
            for d in range(abs(a - b), a + b + 1):
                if not any(tri(a, b + u, oo) and tri(u, d, oo) for u in range(L - b + 1) for oo in range(L + 1)):
                    continue
                c = o.cg_real(a, b, d)
                rows.append(np.einsum("xyz,nxc,ny->nzc", c, feat[:, a * a:(a + 1) ** 2, :].astype(np.float64),
                                      R[:, b * b:(b + 1) ** 2]))
    return np.concatenate(rows, axis=1)


@pytest.mark.parametrize("L,C", [(2, 16), (3, 64), (4, 128), (6, 8)])
def test_node_tp(e2f, ctx, L, C):
    rng = np.random.default_rng(L)
    pos = syn.quantize(rng.uniform(-6, 6, size=(37, 3)))
    feat = rng.standard_normal((37, (L + 1) ** 2, C)).astype(np.float32)
    got = e2f.e2f_node_tp(ctx, gpu(pos), gpu(feat), L).cpu().numpy()
    ref = node_tp_reference(L, pos, feat)
    assert got.shape == ref.shape == (37, e2f.e2f_node_tp_dim(L), C)
    assert np.max(np.abs(got - ref)) <= 1e-5 * np.max(np.abs(ref))


# ------------------------------------------------------------ the layer
@pytest.mark.parametrize("name,rows", [("cluster32_L2", None), ("molecules256x30_L3", 512), ("water2000_L4", 96)])
def test_conv_parity(e2f, ctx, name, rows):
    inp, rp, ci, alpha = case(name)
    wl = inp.workload
    y6, ye = run_both(e2f, ctx, inp, rp, ci, alpha, wl.lmax, wl.heads, wl.cutoff, mix=inp.mix_w)
    r = sample_rows(inp.pos.shape[0], rows or inp.pos.shape[0])
    ref = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, inp.mix_w, rows=r)
    e6 = o.max_rel_err(y6[r], ref, wl.lmax)
    ee = o.max_rel_err(ye[r], ref, wl.lmax)
    print("%s: 6j err %.3e  edge err %.3e" % (name, e6, ee))
    assert e6 <= TOL_F32 and ee <= TOL_F32


def test_conv_parity_protein_fp32_and_bf16(e2f, ctx):
    inp, rp, ci, alpha = case("protein20k_L4")
    wl = inp.workload
    r = sample_rows(inp.pos.shape[0], 48, seed=1)
    y = o.conv_edge(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, rows=r)
    ref = o.mix(wl.lmax, y, inp.mix_w)
    y6, ye = run_both(e2f, ctx, inp, rp, ci, alpha, wl.lmax, wl.heads, wl.cutoff, mix=inp.mix_w)
    e6, ee = o.max_rel_err(y6[r], ref, wl.lmax), o.max_rel_err(ye[r], ref, wl.lmax)
    print("protein fp32: 6j err %.3e  edge err %.3e" % (e6, ee))
    assert e6 <= TOL_F32 and ee <= TOL_F32
    y6, ye = run_both(e2f, ctx, inp, rp, ci, alpha, wl.lmax, wl.heads, wl.cutoff, mix=inp.mix_w, mix_bf16=True)
    e6, ee = o.max_rel_err(y6[r], ref, wl.lmax), o.max_rel_err(ye[r], ref, wl.lmax)
    print("protein bf16 mix: 6j err %.3e  edge err %.3e" % (e6, ee))
    assert e6 <= TOL_BF16 and ee <= TOL_BF16


def test_conv_parity_bf16_mix_c64(e2f, ctx):
    # bf16 channel mixing at 64 channels (MFMA bf16 path, 4 channel blocks)
    inp, rp, ci, alpha = case("molecules256x30_L3")
    wl = inp.workload
    r = sample_rows(inp.pos.shape[0], 256, seed=3)
    ref = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, inp.mix_w, rows=r)
    y6, ye = run_both(e2f, ctx, inp, rp, ci, alpha, wl.lmax, wl.heads, wl.cutoff, mix=inp.mix_w, mix_bf16=True)
    e6, ee = o.max_rel_err(y6[r], ref, wl.lmax), o.max_rel_err(ye[r], ref, wl.lmax)
    print("molecules bf16 mix: 6j err %.3e  edge err %.3e" % (e6, ee))
    assert e6 <= TOL_BF16 and ee <= TOL_BF16


def test_conv_edge_cases(e2f, ctx):
    rng = np.random.default_rng(12)
    # ragged sizes, L = 0, isolated atoms, explicit path weights, no alpha
    for L, n, C, H in [(0, 13, 4, 1), (1, 29, 12, 3), (3, 57, 8, 2)]:
        pos = syn.quantize(rng.uniform(0, 9, size=(n, 3)))
        pos[-1] = [60.0, 60.0, 60.0]  # isolated
        rp, ci = o.neighbor_list(pos, 4.0)
        feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
        w = rng.uniform(0.2, 1.0, size=(L + 1) ** 3)
        ones = np.ones((len(ci), H), dtype=np.float32)
        ref = o.conv_edge(L, H, pos, feat, rp, ci, ones, w)
        for fn in (e2f.e2f_wigner6j_conv_forward, e2f.e2f_edge_tp_conv_forward):
            got = fn(ctx, gpu(pos), gpu(feat), gpu(rp), gpu(ci), None, L, H, 4.0, path_w=w).cpu().numpy()
            assert o.max_rel_err(got, ref, L) <= TOL_F32
            assert np.all(got[-1] == 0)
    # no edges at all
    pos = np.array([[0, 0, 0], [10, 0, 0]], dtype=np.float32)
    feat = rng.standard_normal((2, 4, 4)).astype(np.float32)
    rp = np.zeros(3, dtype=np.int64)
    ci = np.zeros(0, dtype=np.int32)
    for fn in (e2f.e2f_wigner6j_conv_forward, e2f.e2f_edge_tp_conv_forward):
        got = fn(ctx, gpu(pos), gpu(feat), gpu(rp), gpu(ci), None, 1, 1, 4.0).cpu().numpy()
        assert np.all(got == 0)


@pytest.mark.parametrize("copies", [1, 2])
def test_conv_graph_ids_sparse_and_interleaved(e2f, ctx, copies):
    # the receiver order's keys with graph ids near 2^31, not contiguous in
    # the atom order: one copy of the 256 molecules (7,680 atoms, the plan of
    # one workgroup, whose sort then runs over the id's digits) and two
    # copies side by side (15,360 atoms, the plan's large path)
    base, _, _, _ = case("molecules256x30_L3")
    wl = base.workload
    n0 = base.pos.shape[0]
    pos = np.concatenate([base.pos + np.float32(40.0 * c) for c in range(copies)])
    old = np.concatenate([base.graph_id + 256 * c for c in range(copies)]).astype(np.int64)
    gid = (2_147_000_000 - old * 4_000_001).astype(np.int32)
    feat = np.concatenate([base.feat] * copies)
    species = np.concatenate([base.species] * copies)
    perm = np.random.default_rng(77).permutation(n0 * copies)
    pos, gid, feat, species = pos[perm], gid[perm], feat[perm], species[perm]
    rp, ci = o.neighbor_list(pos, wl.cutoff, gid)
    alpha = syn.attention_weights(pos, species, rp, ci, wl.heads, wl.cutoff, wl.species, wl.seed)
    r = sample_rows(pos.shape[0], 128, seed=copies)
    ref = o.conv_edge(wl.lmax, wl.heads, pos, feat, rp, ci, alpha, base.path_w, rows=r)
    got = e2f.e2f_wigner6j_conv_forward(ctx, gpu(pos), gpu(feat), gpu(rp), gpu(ci), gpu(alpha), wl.lmax, wl.heads,
                                        wl.cutoff, path_w=base.path_w, graph_id=gpu(gid)).cpu().numpy()
    err = o.max_rel_err(got[r], ref, wl.lmax)
    print("sparse graph ids, %d atoms: err %.3e" % (pos.shape[0], err))
    assert err <= TOL_F32


@pytest.mark.parametrize("n", [2, 3, 511, 512, 8192, 8193])
def test_conv_plan_sizes(e2f, ctx, n):
    # the forward's plan at the sizes that change its shape: the one-workgroup
    # plan (up to 8,192 atoms; 64 threads below 512 atoms, 1,024 at 8,192) and
    # the multi-kernel plan above it, on random positions at 0.1 per A^3
    rng = np.random.default_rng(500 + n)
    L, C, H, cut = 2, 16, 2, 4.5
    box = max((n / 0.1) ** (1.0 / 3.0), 3.0)
    pos = syn.quantize(rng.uniform(0, box, size=(n, 3)))
    rp, ci = o.neighbor_list(pos, cut)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.05, 1.0, size=(len(ci), H)).astype(np.float32)
    w = rng.uniform(0.2, 1.0, size=(L + 1) ** 3)
    r = sample_rows(n, 64, seed=n)
    ref = o.conv_edge(L, H, pos, feat, rp, ci, alpha, w, rows=r)
    got = e2f.e2f_wigner6j_conv_forward(ctx, gpu(pos), gpu(feat), gpu(rp), gpu(ci), gpu(alpha), L, H, cut,
                                        path_w=w).cpu().numpy()
    scale = max(float(np.max(np.abs(ref))), 1e-30)
    err = o.max_rel_err(got[r], ref, L) if len(ci) else float(np.max(np.abs(got))) / scale
    print("plan sizes: n %d edges %d err %.3e" % (n, len(ci), err))
    assert err <= TOL_F32


@pytest.mark.parametrize("C,H", [(12, 3), (48, 4), (256, 8)])
def test_mixing_channel_counts(e2f, ctx, C, H):
    # channel mixing on both kernels: MFMA (C a multiple of 16 up to 128) and
    # the VALU fallback (other C), fp32 and bf16 weights
    rng = np.random.default_rng(C)
    L, n = 2, 61
    pos = syn.quantize(rng.uniform(0, 10, size=(n, 3)))
    rp, ci = o.neighbor_list(pos, 4.5)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.0, 1.0, size=(len(ci), H)).astype(np.float32)
    mix = (rng.standard_normal((L + 1, C, C)) / np.sqrt(C)).astype(np.float32)
    w = rng.uniform(0.2, 1.0, size=(L + 1) ** 3)
    ref = o.layer(L, H, pos, feat, rp, ci, alpha, w, mix)
    for bf16, tol in ((False, TOL_F32), (True, TOL_BF16)):
        mw = gpu(mix).to(torch.bfloat16) if bf16 else gpu(mix)
        for fn in (e2f.e2f_wigner6j_conv_forward, e2f.e2f_edge_tp_conv_forward):
            got = fn(ctx, gpu(pos), gpu(feat), gpu(rp), gpu(ci), gpu(alpha), L, H, 4.5, path_w=w,
                     mix_w=mw).cpu().numpy()
            err = o.max_rel_err(got, ref, L)
            assert err <= tol, (C, bf16, fn.__name__, err)


def test_determinism_and_translation(e2f, ctx):
    inp, rp, ci, alpha = case("water2000_L4")
    wl = inp.workload
    a1, b1 = run_both(e2f, ctx, inp, rp, ci, alpha, wl.lmax, wl.heads, wl.cutoff)
    a2, b2 = run_both(e2f, ctx, inp, rp, ci, alpha, wl.lmax, wl.heads, wl.cutoff)
    assert np.array_equal(a1, a2) and np.array_equal(b1, b2)
    shifted = type(inp)(inp.pos + np.float32(37.5), inp.graph_id, inp.species, inp.feat, inp.mix_w, inp.path_w, wl)
    a3, b3 = run_both(e2f, ctx, shifted, rp, ci, alpha, wl.lmax, wl.heads, wl.cutoff)
    assert o.max_rel_err(a3, a1, wl.lmax) <= TOL_F32 and o.max_rel_err(b3, b1, wl.lmax) <= TOL_F32


@pytest.mark.parametrize("L,C,H,cut,n,box", [(2, 32, 4, 5.0, 300, 12.0), (4, 128, 1, 5.0, 300, 12.0),
                                              (6, 64, 2, 5.0, 200, 10.0), (2, 16, 2, 30.0, 700, 10.0)])
def test_conv_wide_heads_and_long_rows(e2f, ctx, L, C, H, cut, n, box):
    # heads wider than the aggregation's tile (128 channels in one head at
    # L = 4, 32 per head at L = 6) are split into channel groups sharing the
    # head's weights; the last case is a complete graph of 700 atoms (rows of
    # 699 edges, several staging chunks per receiver)
    rng = np.random.default_rng(100 + L + n)
    pos = syn.quantize(rng.uniform(0, box, size=(n, 3)))
    rp, ci = o.neighbor_list(pos, cut)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.05, 1.0, size=(len(ci), H)).astype(np.float32)
    w = rng.uniform(0.2, 1.0, size=(L + 1) ** 3) * cut ** -np.arange(L + 1)[None, :, None].repeat(L + 1, 0).repeat(
        L + 1, 2).reshape(-1)
    r = sample_rows(n, 64, seed=L)
    ref = o.conv_edge(L, H, pos, feat, rp, ci, alpha, w, rows=r)
    print("wide heads / long rows: L %d C %d H %d n %d max degree %d" % (L, C, H, n, int(np.diff(rp).max())),
          flush=True)
    got = e2f.e2f_wigner6j_conv_forward(ctx, gpu(pos), gpu(feat), gpu(rp), gpu(ci), gpu(alpha), L, H, cut,
                                        path_w=w).cpu().numpy()
    err = o.max_rel_err(got[r], ref, L)
    print("wide heads / long rows: err %.3e" % err)
    assert err <= TOL_F32


def test_conv_workspace_slices(e2f, ctx):
    # the smallest workspace the forward accepts: receivers are aggregated and
    # recoupled in slices of 256, in the same order as in one pass, so the
    # output is bitwise that of the one-pass workspace
    inp, rp, ci, alpha = case("water2000_L4")
    wl = inp.workload
    n, E = inp.pos.shape[0], len(ci)
    r = sample_rows(n, 64, seed=3)
    ref = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, inp.mix_w, rows=r)
    args = (gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha), wl.lmax, wl.heads, wl.cutoff)
    full = e2f.e2f_wigner6j_conv_forward(ctx, *args, mix_w=gpu(inp.mix_w)).cpu().numpy()
    assert e2f.e2f_last_slices(ctx) == 1
    wmin = e2f.e2f_wigner6j_workspace_size(ctx, n, E, wl.lmax, wl.channels, wl.heads, wl.cutoff,
                                           mix_w=gpu(inp.mix_w), minimum=True)
    wfull = e2f.e2f_wigner6j_workspace_size(ctx, n, E, wl.lmax, wl.channels, wl.heads, wl.cutoff,
                                            mix_w=gpu(inp.mix_w))
    assert wmin < wfull
    ws = torch.empty(wmin, dtype=torch.uint8, device=DEV)
    sliced = e2f.e2f_wigner6j_conv_forward(ctx, *args, mix_w=gpu(inp.mix_w), workspace=ws).cpu().numpy()
    assert e2f.e2f_last_slices(ctx) == (n + 255) // 256
    assert np.array_equal(sliced, full)
    err = o.max_rel_err(sliced[r], ref, wl.lmax)
    print("water2000 in slices of 256 receivers: err %.3e" % err)
    assert err <= TOL_F32
    # one byte less than the minimum is refused before any device work
    with pytest.raises(e2f.E2FError) as ei:
        e2f.e2f_wigner6j_conv_forward(ctx, *args, mix_w=gpu(inp.mix_w),
                                      workspace=torch.empty(wmin - 1, dtype=torch.uint8, device=DEV))
    assert ei.value.status == e2f.E2F_ECAPACITY


def test_conv_stress_200k_sampled(e2f, ctx):
    # 200,000 atoms, cutoff 8 A, L = 6, C = 64: the factorised path only, checked
    # on sampled receiver rows (the definition is separable per row)
    inp, rp, ci, alpha = case("stress200k_L6")
    wl = inp.workload
    pos, feat = gpu(inp.pos), gpu(inp.feat)
    g_rp, g_ci = e2f.e2f_neighbor_list(ctx, pos, wl.cutoff)
    assert torch.equal(g_rp.cpu(), torch.from_numpy(rp)) and torch.equal(g_ci.cpu(), torch.from_numpy(ci))
    out = e2f.e2f_wigner6j_conv_forward(ctx, pos, feat, g_rp, g_ci, gpu(alpha), wl.lmax, wl.heads, wl.cutoff,
                                        mix_w=gpu(inp.mix_w))
    torch.cuda.synchronize()
    r = sample_rows(inp.pos.shape[0], 256, seed=5)
    ref = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, inp.mix_w, rows=r)
    err = o.max_rel_err(out.cpu().numpy()[r], ref, wl.lmax)
    print("stress200k: %d edges, err %.3e" % (len(ci), err))
    assert err <= TOL_F32


def test_stress_crop_both_paths(e2f, ctx):
    # the central 58.48 A crop of the 200,000-atom system (about 20k atoms,
    # 3.6 M edges, L = 6, C = 64): the factorised path and the per-edge
    # baseline against the definition on sampled rows
    inp, rp, ci, alpha = case("stress200k_L6")
    wl = inp.workload
    lo, hi = inp.pos.min(0), inp.pos.max(0)
    keep = np.nonzero(np.all(np.abs(inp.pos - (lo + hi) / 2) < syn._cube_side(20000) / 2, axis=1))[0]
    pos, feat = np.ascontiguousarray(inp.pos[keep]), np.ascontiguousarray(inp.feat[keep])
    crp, cci = o.neighbor_list(pos, wl.cutoff)
    calpha = syn.attention_weights(pos, inp.species[keep], crp, cci, wl.heads, wl.cutoff, wl.species, wl.seed)
    n = pos.shape[0]
    print("stress crop: %d atoms, %d edges" % (n, len(cci)), flush=True)
    y6, ye = run_both(e2f, ctx, type(inp)(pos, None, inp.species[keep], feat, inp.mix_w, inp.path_w, wl), crp, cci,
                      calpha, wl.lmax, wl.heads, wl.cutoff, mix=inp.mix_w)
    r = sample_rows(n, 256, seed=9)
    ref = o.layer(wl.lmax, wl.heads, pos, feat, crp, cci, calpha, inp.path_w, inp.mix_w, rows=r)
    e6, ee = o.max_rel_err(y6[r], ref, wl.lmax), o.max_rel_err(ye[r], ref, wl.lmax)
    print("stress crop: 6j err %.3e, edge-TP err %.3e" % (e6, ee))
    assert e6 <= TOL_F32 and ee <= TOL_F32
