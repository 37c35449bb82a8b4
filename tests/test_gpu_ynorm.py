"""Alg. 1's per-degree attention weights alpha / D^f (Y-based filters, the
y_norm flag): both forms of the layer on the GPU against the oracle's
definition of the variant.  The factorised forward weights the terms of
filter degree b + u = f by alpha / D^f: the two-kernel form aggregates once
per degree and recouples those terms from S^(f); the fused form stacks
degrees in the K rows of one pass (one pass below L = 4, two at L = 4).

Run with -m gpu."""
import numpy as np
import pytest
import torch

import e2f_synth as syn
import oracle as o
from cases import TOL_F32, case, sample_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def e2f():
    import paper_2501_19216_amd as m
    return m


@pytest.fixture(scope="module")
def ctx(e2f):
    c = e2f.e2f_create(6, 0)
    yield c
    c.close()


def gpu(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def both(e2f, ctx, inp, rp, ci, alpha, wl, mix, tile_side=0.0):
    pos, feat, row_ptr, col, al = gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha)
    gid = gpu(inp.graph_id)
    mw = gpu(mix)
    y6 = e2f.e2f_wigner6j_conv_forward(ctx, pos, feat, row_ptr, col, al, wl.lmax, wl.heads, wl.cutoff, mix_w=mw,
                                       graph_id=gid, tile_side=tile_side, y_norm=True)
    ye = e2f.e2f_edge_tp_conv_forward(ctx, pos, feat, row_ptr, col, al, wl.lmax, wl.heads, wl.cutoff, mix_w=mw,
                                      graph_id=gid, y_norm=True)
    return y6.cpu().numpy(), ye.cpu().numpy()


@pytest.mark.parametrize("name,rows,mix", [("cluster32_L2", None, False), ("molecules256x30_L3", 512, True),
                                            ("water2000_L4", 96, True), ("protein20k_L4", 128, False)])
def test_y_norm_workloads(e2f, ctx, name, rows, mix):
    inp, rp, ci, alpha = case(name)
    wl = inp.workload
    n = inp.pos.shape[0]
    r = np.arange(n, dtype=np.int32) if rows is None else sample_rows(n, rows, seed=11)
    mw = inp.mix_w if mix else None
    ref = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, mw, rows=r, y_norm=True)
    print("%s y_norm: case" % name, flush=True)
    y6, ye = both(e2f, ctx, inp, rp, ci, alpha, wl, mw)
    e6, ee = o.max_rel_err(y6[r], ref, wl.lmax), o.max_rel_err(ye[r], ref, wl.lmax)
    print("%s y_norm: 6j %.3e edge %.3e" % (name, e6, ee))
    assert e6 <= TOL_F32 and ee <= TOL_F32
    # the variant differs from the plain layer (the flag reaches both kernels)
    plain = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, mw, rows=r[:8])
    assert o.max_rel_err(ref[:8], plain, wl.lmax) > 1e-2


@pytest.mark.parametrize("form", ["split", "fused"])
def test_y_norm_both_forms(e2f, ctx, form):
    # alpha / D^f in both forms of the aggregation: the two-kernel form (S^(f)
    # per degree, recoupled by its terms b + u = f) and the fused form (two
    # passes at L = 4, each with the terms of the degrees its K rows stack)
    inp, rp, ci, alpha = case("water2000_L4")
    wl = inp.workload
    r = sample_rows(inp.pos.shape[0], 64, seed=21)
    ref = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, rows=r, y_norm=True)
    got = e2f.e2f_wigner6j_conv_forward(ctx, gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha), wl.lmax,
                                        wl.heads, wl.cutoff, path_w=inp.path_w, y_norm=True,
                                        form=form).cpu().numpy()
    err = o.max_rel_err(got[r], ref, wl.lmax)
    print("water2000 y_norm %s: err %.3e" % (form, err))
    assert err <= TOL_F32


@pytest.mark.parametrize("L", [1, 2, 3])
def test_y_norm_fused_below_l4(e2f, ctx, L):
    # below L = 4 the fused form runs alpha / D^f in one pass whose K rows
    # stack every filter degree (L, .., 0; 5, 14 and 30 rows at L = 1, 2, 3);
    # heads of 16 channels, random positions (contacts down to about 0.1 A),
    # rows of up to about 250 edges (two staging chunks); both forms against
    # the oracle
    rng = np.random.default_rng(70 + L)
    C, H, cutoff = 32, 2, 5.0
    pos = syn.quantize(rng.uniform(0.0, 11.0, size=(600, 3)))  # about half the rows longer than 128
    n = pos.shape[0]
    rp, ci = o.neighbor_list(pos, cutoff)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.1, 1.0, size=(len(ci), H)).astype(np.float32)
    w = rng.uniform(0.5, 1.5, size=(L + 1) ** 3)
    r = sample_rows(n, 48, seed=L)
    ref = o.layer(L, H, pos, feat, rp, ci, alpha, w, rows=r, y_norm=True)
    print("L%d y_norm: %d atoms, %d edges, longest row %d" % (L, n, len(ci), np.diff(rp).max()), flush=True)
    for form in ("fused", "split"):
        got = e2f.e2f_wigner6j_conv_forward(ctx, gpu(pos), gpu(feat), gpu(rp), gpu(ci), gpu(alpha), L, H, cutoff,
                                            path_w=w, y_norm=True, form=form).cpu().numpy()
        err = o.max_rel_err(got[r], ref, L)
        print("L%d y_norm %s: err %.3e" % (L, form, err), flush=True)
        assert err <= TOL_F32


def test_y_norm_short_contacts_and_slices(e2f, ctx):
    # L = 6 on uniform random positions (no minimum distance: the closest
    # pairs are about 0.1 A apart), where the weights 1/D^f of the short edges
    # amplify the rounding of the binomial expansion unless the local origins
    # are close enough (the tile side follows the shortest edge); then
    # water2000 through the smallest workspace (slices of 256 receivers)
    rng = np.random.default_rng(61)
    L, C, H, cutoff = 6, 8, 2, 5.0
    pos = syn.quantize(rng.uniform(0.0, 10.0, size=(343, 3)))
    n = pos.shape[0]
    rp, ci = o.neighbor_list(pos, cutoff)
    d = np.linalg.norm(pos[np.repeat(np.arange(n), np.diff(rp))].astype(np.float64) - pos[ci], axis=1)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.1, 1.0, size=(len(ci), H)).astype(np.float32)
    w = rng.uniform(0.5, 1.5, size=(L + 1) ** 3)
    r = sample_rows(n, 40, seed=2)
    near = np.unique(np.repeat(np.arange(n), np.diff(rp))[d < 0.5])
    r = np.unique(np.concatenate([r, near])).astype(np.int32)  # every receiver of a contact below 0.5 A
    ref = o.layer(L, H, pos, feat, rp, ci, alpha, w, rows=r, y_norm=True)
    print("L6 y_norm short contacts: shortest edge %.3f A, %d rows" % (d.min(), len(r)), flush=True)
    got = e2f.e2f_wigner6j_conv_forward(ctx, gpu(pos), gpu(feat), gpu(rp), gpu(ci), gpu(alpha), L, H, cutoff,
                                        path_w=w, y_norm=True).cpu().numpy()
    err = o.max_rel_err(got[r], ref, L)
    print("L6 y_norm short contacts: err %.3e" % err)
    assert err <= TOL_F32
    inp, rp, ci, alpha = case("water2000_L4")
    wl = inp.workload
    n, E = inp.pos.shape[0], len(ci)
    r = sample_rows(n, 48, seed=4)
    ref = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, rows=r, y_norm=True)
    wmin = e2f.e2f_wigner6j_workspace_size(ctx, n, E, wl.lmax, wl.channels, wl.heads, wl.cutoff, y_norm=True,
                                           minimum=True)
    print("water2000 y_norm slices: case", flush=True)
    got = e2f.e2f_wigner6j_conv_forward(ctx, gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha), wl.lmax,
                                        wl.heads, wl.cutoff, y_norm=True,
                                        workspace=torch.empty(wmin, dtype=torch.uint8, device=DEV)).cpu().numpy()
    assert e2f.e2f_last_slices(ctx) == (n + 255) // 256
    err = o.max_rel_err(got[r], ref, wl.lmax)
    print("water2000 y_norm in slices: err %.3e" % err)
    assert err <= TOL_F32


def test_y_norm_unit_lattice_equals_plain(e2f, ctx):
    # every edge of length 1: the variant is the plain layer
    import itertools
    g = np.array(list(itertools.product(range(6), repeat=3)), dtype=np.float32)
    L, C, H = 4, 16, 4
    rp, ci = o.neighbor_list(g, 1.2)
    rng = np.random.default_rng(8)
    feat = rng.standard_normal((len(g), (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.1, 1.0, size=(len(ci), H)).astype(np.float32)
    args = (gpu(g), gpu(feat), gpu(rp), gpu(ci), gpu(alpha), L, H, 1.2)
    a = e2f.e2f_wigner6j_conv_forward(ctx, *args, y_norm=True).cpu().numpy()
    b = e2f.e2f_wigner6j_conv_forward(ctx, *args).cpu().numpy()
    assert o.max_rel_err(a, b.astype(np.float64), L) <= TOL_F32


def test_y_norm_stress_200k_sampled(e2f, ctx):
    # the 200,000-atom L = 6 system, factorised path, 256 sampled receiver rows
    inp, rp, ci, alpha = case("stress200k_L6")
    wl = inp.workload
    r = sample_rows(inp.pos.shape[0], 256, seed=5)
    ref = o.layer(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, rows=r, y_norm=True)
    print("stress200k y_norm: case", flush=True)
    got = e2f.e2f_wigner6j_conv_forward(ctx, gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha), wl.lmax,
                                        wl.heads, wl.cutoff, path_w=inp.path_w, y_norm=True).cpu().numpy()
    err = o.max_rel_err(got[r], ref, wl.lmax)
    print("stress200k y_norm: err %.3e" % err)
    assert err <= TOL_F32
