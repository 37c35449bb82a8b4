"""GPU parity of the forward whose aggregation applies the i-side recouple
itself (L <= 4, heads of a multiple of 16 channels): against the fp64 oracle's
definition of the layer and against the two-kernel form (S written, then
recoupled), selected with the form argument ("fused", "split"; the default
"auto" picks the fused form at L = 4 once S would exceed 256 MiB).

Calls go through the C ABI.  Bar: float32 max relative error <= 1e-4 per
output irrep block.
"""
import numpy as np
import pytest
import torch

import oracle as o
import e2f_synth as syn
from cases import TOL_F32, case, sample_rows

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


def gpu(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


# L, C, H, atoms, box side, cutoff, with attention weights: every degree up to
# 4, one head of 16, several heads, a head of 32 and 64 channels (split into
# groups of 16 that share the head's weight), ragged atom counts, and rows
# longer than one staging chunk of 128 edges (the 9.5 A cutoff)
CASES = [(0, 16, 1, 37, 7.0, 4.0, True), (1, 32, 2, 53, 8.0, 4.0, False), (2, 16, 1, 91, 9.0, 4.5, True),
         (3, 64, 4, 150, 10.0, 5.0, True), (3, 32, 1, 77, 9.0, 4.5, True), (4, 48, 3, 120, 10.0, 5.0, True),
         (4, 64, 1, 101, 9.0, 4.5, False), (4, 32, 2, 260, 12.0, 9.5, True)]


@pytest.mark.parametrize("L,C,H,n,box,cut,with_alpha", CASES)
def test_fused_forward(e2f, ctx, L, C, H, n, box, cut, with_alpha):
    rng = np.random.default_rng(1000 + 10 * L + C + n)
    pos = syn.quantize(rng.uniform(0, box, size=(n, 3)))
    pos[-1] = [80.0, 80.0, 80.0]  # an isolated receiver
    rp, ci = o.neighbor_list(pos, cut)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.05, 1.0, size=(len(ci), H)).astype(np.float32)
    w = rng.uniform(0.2, 1.0, size=(L + 1) ** 3) * np.repeat(
        np.repeat((cut ** -np.arange(L + 1.0))[None, :, None], L + 1, 0), L + 1, 2).reshape(-1)
    r = sample_rows(n, 48, seed=L)
    a_ref = alpha if with_alpha else np.ones_like(alpha)
    ref = o.conv_edge(L, H, pos, feat, rp, ci, a_ref, w, rows=r)
    print("fused L %d C %d H %d n %d edges %d max degree %d" % (L, C, H, n, len(ci), int(np.diff(rp).max())),
          flush=True)
    args = (gpu(pos), gpu(feat), gpu(rp), gpu(ci), gpu(alpha) if with_alpha else None, L, H, cut)
    fused = e2f.e2f_wigner6j_conv_forward(ctx, *args, path_w=w, form="fused").cpu().numpy()
    split = e2f.e2f_wigner6j_conv_forward(ctx, *args, path_w=w, form="split").cpu().numpy()
    ef, es = o.max_rel_err(fused[r], ref, L), o.max_rel_err(split[r], ref, L)
    print("  fused err %.3e  two-kernel err %.3e" % (ef, es))
    assert ef <= TOL_F32 and es <= TOL_F32
    assert np.all(fused[-1] == 0)
    # both forms compute the same layer; they differ only in rounding order
    assert o.max_rel_err(fused, split, L) <= TOL_F32


def test_fused_protein_rows_and_workspace_sizes(e2f, ctx):
    # 20,000 atoms, L = 4, C = 128, H = 8 (the fused form): 256 sampled rows
    # against the definition, the two-kernel form on the same rows, and the
    # fused form in slices of the smallest workspace, bitwise equal to one pass
    inp, rp, ci, alpha = case("protein20k_L4")
    wl = inp.workload
    n, E = inp.pos.shape[0], len(ci)
    r = sample_rows(n, 256, seed=11)
    ref = o.conv_edge(wl.lmax, wl.heads, inp.pos, inp.feat, rp, ci, alpha, inp.path_w, rows=r)
    args = (gpu(inp.pos), gpu(inp.feat), gpu(rp), gpu(ci), gpu(alpha), wl.lmax, wl.heads, wl.cutoff)
    fused = e2f.e2f_wigner6j_conv_forward(ctx, *args).cpu().numpy()  # the automatic choice: fused (S 4.65 GB)
    assert e2f.e2f_last_slices(ctx) == 1
    assert np.array_equal(fused, e2f.e2f_wigner6j_conv_forward(ctx, *args, form="fused").cpu().numpy())
    split = e2f.e2f_wigner6j_conv_forward(ctx, *args, form="split").cpu().numpy()
    ef, es = o.max_rel_err(fused[r], ref, wl.lmax), o.max_rel_err(split[r], ref, wl.lmax)
    print("protein20k: fused err %.3e  two-kernel err %.3e on %d rows" % (ef, es, len(r)))
    assert ef <= TOL_F32 and es <= TOL_F32
    wmin = e2f.e2f_wigner6j_workspace_size(ctx, n, E, wl.lmax, wl.channels, wl.heads, wl.cutoff, minimum=True)
    wsplit = e2f.e2f_wigner6j_workspace_size(ctx, n, E, wl.lmax, wl.channels, wl.heads, wl.cutoff,
                                             form="split")
    wfull = e2f.e2f_wigner6j_workspace_size(ctx, n, E, wl.lmax, wl.channels, wl.heads, wl.cutoff)
    assert wmin < wfull < wsplit  # F_i (70 KB a receiver) instead of S_i (232 KB)
    ws = torch.empty(wmin, dtype=torch.uint8, device=DEV)
    sliced = e2f.e2f_wigner6j_conv_forward(ctx, *args, workspace=ws).cpu().numpy()
    assert e2f.e2f_last_slices(ctx) == (n + 255) // 256
    assert np.array_equal(sliced, fused)


@pytest.mark.parametrize("scale_exp", [-40, 40])
def test_fused_power_of_two_scaling_is_exact(e2f, ctx, scale_exp):
    # the forward is linear in h, and a power of two commutes with every step
    # of the fused form (the three-part bf16 split of the features, the exact
    # bf16 products, float sums, F_i G_i): scaling h by 2^k scales y bit for
    # bit, far from the float range's ends (values here stay within 2^-70 ..
    # 2^60)
    L, C, H, n = 4, 32, 2, 120
    rng = np.random.default_rng(77)
    pos = syn.quantize(rng.uniform(0, 10.0, size=(n, 3)))
    rp, ci = o.neighbor_list(pos, 5.0)
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.05, 1.0, size=(len(ci), H)).astype(np.float32)
    args = (gpu(rp), gpu(ci), gpu(alpha), L, H, 5.0)
    y1 = e2f.e2f_wigner6j_conv_forward(ctx, gpu(pos), gpu(feat), *args, form="fused").cpu().numpy()
    fs = np.ldexp(feat, scale_exp).astype(np.float32)
    y2 = e2f.e2f_wigner6j_conv_forward(ctx, gpu(pos), gpu(fs), *args, form="fused").cpu().numpy()
    assert np.array_equal(np.ldexp(y1, scale_exp).astype(np.float32), y2)
