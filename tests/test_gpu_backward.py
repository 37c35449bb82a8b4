"""GPU backward of the Wigner-6j convolution (vector-Jacobian products with
respect to the features, the attention weights and the positions) against
the oracle's products by the definition of the layer.  Run with -m gpu."""
import itertools

import numpy as np
import pytest
import torch

import e2f_synth as syn
import oracle as o
from cases import TOL_BF16, TOL_F32

pytestmark = pytest.mark.gpu


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
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def default_w(L, cutoff):
    w = np.zeros((L + 1) ** 3)
    for a, f, oo in itertools.product(range(L + 1), repeat=3):
        if abs(a - f) <= oo <= a + f:
            w[(a * (L + 1) + f) * (L + 1) + oo] = cutoff ** (-f)
    return w


def head_err(got, ref):
    return float(np.max(np.abs(got - ref).max(axis=0) / np.maximum(np.abs(ref).max(axis=0), 1e-30)))


def check(e2f, ctx, pos, rp, ci, L, C, H, cutoff, seed, mix=None, bf16=False, gid=None, tol=TOL_F32):
    rng = np.random.default_rng(seed)
    n = pos.shape[0]
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    alpha = rng.uniform(0.05, 1.0, size=(len(ci), H)).astype(np.float32)
    gout = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    w = default_w(L, cutoff)
    gy = gout.astype(np.float64)
    mw = None
    if mix is not None:
        m = mix
        if bf16:
            m = torch.from_numpy(mix).to(torch.bfloat16).float().numpy()  # the weights as the kernel sees them
        gy = o.mix(L, gy, np.transpose(m, (0, 2, 1)))
        mw = gpu(mix).to(torch.bfloat16) if bf16 else gpu(mix)
    gf_ref, ga_ref = o.conv_edge_vjp(L, H, pos, feat, gy, rp, ci, alpha, w)
    atoms = np.linspace(0, n - 1, min(n, 48)).astype(np.int32)
    gp_ref = o.conv_edge_grad_pos(L, H, pos, feat, gy, rp, ci, alpha, w, atoms=atoms)
    print("n %d L %d C %d H %d rc %g: case" % (n, L, C, H, cutoff), flush=True)
    gf, ga, gp = e2f.e2f_wigner6j_conv_backward(ctx, gpu(pos), gpu(feat), gpu(gout), gpu(rp), gpu(ci), gpu(alpha), L,
                                                H, cutoff, mix_w=mw, graph_id=gpu(gid), want_pos=True)
    ef = o.max_rel_err(gf.cpu().numpy(), gf_ref, L)
    ea = head_err(ga.cpu().numpy(), ga_ref)
    gp = gp.cpu().numpy()
    ep = float(np.abs(gp[atoms] - gp_ref).max() / np.abs(gp_ref).max())
    print("n %d L %d C %d mix %s bf16 %s: grad_feat %.3e grad_alpha %.3e grad_pos %.3e"
          % (n, L, C, mix is not None, bf16, ef, ea, ep))
    assert ef <= tol and ea <= tol and ep <= tol
    # the layer depends on differences of positions: the gradient sums to zero
    assert np.abs(gp.astype(np.float64).sum(0)).max() <= 1e-4 * np.abs(gp).max() * np.sqrt(n)
    return feat, alpha, gout, w, gf_ref, ga_ref


# head widths 4 and 8 take the per-edge kernels, multiples of 16 the per-receiver
# MFMA product (L=6 runs its filter rows in several passes; the 7 A cutoff
# gives receivers of more than 128 edges, several edge chunks)
@pytest.mark.parametrize("L,C,H,mix,rc", [(2, 16, 4, False, 5.0), (3, 32, 4, True, 5.0), (4, 64, 8, False, 5.0),
                                          (6, 16, 4, False, 5.0), (4, 128, 8, False, 5.0), (2, 64, 2, True, 5.0),
                                          (3, 64, 1, False, 5.0), (6, 32, 2, False, 5.0), (4, 32, 2, False, 7.0)])
def test_backward_radius_graph(e2f, ctx, L, C, H, mix, rc):
    rng = np.random.default_rng(L)
    pos = syn.quantize(rng.uniform(0, 14, size=(400, 3)))
    rp, ci = o.neighbor_list(pos, rc)
    m = (rng.standard_normal((L + 1, C, C)) / np.sqrt(C)).astype(np.float32) if mix else None
    check(e2f, ctx, pos, rp, ci, L, C, H, rc, 10 + L, mix=m)


def test_backward_bf16_mixing(e2f, ctx):
    rng = np.random.default_rng(8)
    pos = syn.quantize(rng.uniform(0, 12, size=(300, 3)))
    rp, ci = o.neighbor_list(pos, 5.0)
    m = (rng.standard_normal((4, 64, 64)) / 8.0).astype(np.float32)
    check(e2f, ctx, pos, rp, ci, 3, 64, 8, 5.0, 21, mix=m, bf16=True, tol=TOL_BF16)


def test_backward_knn_graph_is_transposed(e2f, ctx):
    # a kNN graph is not symmetric: the feature gradient needs the transposed graph
    rng = np.random.default_rng(3)
    pos = syn.quantize(rng.uniform(0, 16, size=(500, 3)))
    rp, ci = o.knn_graph(pos, 24)
    d = np.linalg.norm(pos[np.repeat(np.arange(500), np.diff(rp))] - pos[ci], axis=1)
    check(e2f, ctx, pos, rp, ci, 3, 32, 4, float(d.max()) * 1.001, 5)


@pytest.mark.parametrize("H", [8, 2])
def test_backward_graphs_and_single_outputs(e2f, ctx, H):
    inp = syn.make_inputs(syn.WORKLOADS["molecules256x30_L3"], n_atoms=40 * 30)
    rp, ci = o.neighbor_list(inp.pos, 5.0, inp.graph_id)
    feat, alpha, gout, w, gf_ref, ga_ref = check(e2f, ctx, inp.pos, rp, ci, 3, 32, H, 5.0, 6, gid=inp.graph_id)
    args = (gpu(inp.pos), gpu(feat), gpu(gout), gpu(rp), gpu(ci), gpu(alpha), 3, H, 5.0)
    gf, ga, _ = e2f.e2f_wigner6j_conv_backward(ctx, *args, graph_id=gpu(inp.graph_id), want_alpha=False)
    assert ga is None and o.max_rel_err(gf.cpu().numpy(), gf_ref, 3) <= TOL_F32
    gf, ga, _ = e2f.e2f_wigner6j_conv_backward(ctx, *args, graph_id=gpu(inp.graph_id), want_feat=False)
    assert gf is None and head_err(ga.cpu().numpy(), ga_ref) <= TOL_F32
    gf, ga, gp = e2f.e2f_wigner6j_conv_backward(ctx, *args, graph_id=gpu(inp.graph_id), want_feat=False,
                                                want_alpha=False, want_pos=True)
    at = np.arange(0, 1200, 37, dtype=np.int32)
    gp_ref = o.conv_edge_grad_pos(3, H, inp.pos, feat, gout.astype(np.float64), rp, ci, alpha, w, atoms=at)
    assert gf is None and ga is None
    assert np.abs(gp.cpu().numpy()[at] - gp_ref).max() <= TOL_F32 * np.abs(gp_ref).max()


def test_backward_protein_sampled(e2f, ctx):
    # the 20k-atom workload: grad_alpha on the edges of sampled rows, grad_feat on sampled senders
    from cases import case, sample_rows
    inp, rp, ci, alpha = case("protein20k_L4")
    wl = inp.workload
    rng = np.random.default_rng(2)
    gout = rng.standard_normal(inp.feat.shape).astype(np.float32)
    gf, ga, gp = e2f.e2f_wigner6j_conv_backward(ctx, gpu(inp.pos), gpu(inp.feat), gpu(gout), gpu(rp), gpu(ci),
                                                gpu(alpha), wl.lmax, wl.heads, wl.cutoff, want_pos=True)
    gf, ga, gp = gf.cpu().numpy(), ga.cpu().numpy(), gp.cpu().numpy()
    r = sample_rows(inp.pos.shape[0], 24, seed=4)
    gf_ref, ga_ref = o.conv_edge_vjp(wl.lmax, wl.heads, inp.pos, inp.feat, gout.astype(np.float64), rp, ci, alpha,
                                     inp.path_w, alpha_rows=r, feat_rows=r)
    ef = o.max_rel_err(gf[r], gf_ref[r], wl.lmax)
    ee = np.concatenate([np.arange(rp[i], rp[i + 1]) for i in r])
    ea = head_err(ga[ee], ga_ref[ee])
    rq = r[:12]
    gp_ref = o.conv_edge_grad_pos(wl.lmax, wl.heads, inp.pos, inp.feat, gout.astype(np.float64), rp, ci, alpha,
                                  inp.path_w, atoms=rq)
    ep = float(np.abs(gp[rq] - gp_ref).max() / np.abs(gp_ref).max())
    print("protein: grad_feat %.3e grad_alpha %.3e grad_pos %.3e" % (ef, ea, ep))
    assert ef <= TOL_F32 and ea <= TOL_F32 and ep <= TOL_F32


@pytest.mark.parametrize("L,C,H", [(4, 32, 2), (3, 16, 4)])
def test_backward_uniform_alpha_and_isolated_atoms(e2f, ctx, L, C, H):
    # alpha = NULL (uniform weights); atoms without neighbours give empty rows
    rng = np.random.default_rng(30 + L)
    lone = 60.0 + 20.0 * np.arange(5)[:, None] * np.ones((1, 3))
    pos = syn.quantize(np.concatenate([rng.uniform(0, 11, size=(200, 3)), lone]))
    rp, ci = o.neighbor_list(pos, 5.0)
    n = pos.shape[0]
    assert (np.diff(rp)[200:] == 0).all()
    feat = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    gout = rng.standard_normal((n, (L + 1) ** 2, C)).astype(np.float32)
    w = default_w(L, 5.0)
    ones = np.ones((len(ci), H))
    gf_ref, ga_ref = o.conv_edge_vjp(L, H, pos, feat, gout.astype(np.float64), rp, ci, ones, w)
    atoms = np.r_[np.arange(0, 200, 9), np.arange(200, n)].astype(np.int32)
    gp_ref = o.conv_edge_grad_pos(L, H, pos, feat, gout.astype(np.float64), rp, ci, ones, w, atoms=atoms)
    print("uniform alpha, isolated atoms: L %d C %d H %d" % (L, C, H), flush=True)
    gf, ga, gp = e2f.e2f_wigner6j_conv_backward(ctx, gpu(pos), gpu(feat), gpu(gout), gpu(rp), gpu(ci), None, L, H, 5.0,
                                                want_pos=True)
    gf, ga, gp = gf.cpu().numpy(), ga.cpu().numpy(), gp.cpu().numpy()
    assert o.max_rel_err(gf, gf_ref, L) <= TOL_F32 and head_err(ga, ga_ref) <= TOL_F32
    assert np.abs(gp[atoms] - gp_ref).max() <= TOL_F32 * np.abs(gp_ref).max()
    assert (gp[200:] == 0).all() and (gf[200:] == 0).all()


def test_backward_without_edges(e2f, ctx):
    pos = syn.quantize(10.0 * np.arange(12)[:, None] * np.ones((1, 3)))
    rp, ci = o.neighbor_list(pos, 5.0)
    assert len(ci) == 0
    rng = np.random.default_rng(1)
    feat = rng.standard_normal((12, 16, 16)).astype(np.float32)
    gout = rng.standard_normal((12, 16, 16)).astype(np.float32)
    gf, ga, gp = e2f.e2f_wigner6j_conv_backward(ctx, gpu(pos), gpu(feat), gpu(gout), gpu(rp), gpu(ci),
                                                gpu(np.zeros((0, 4), np.float32)), 3, 4, 5.0, want_pos=True)
    assert ga.shape == (0, 4) and (gf.cpu().numpy() == 0).all() and (gp.cpu().numpy() == 0).all()


def test_backward_forces_without_gradient_table(e2f, ctx, monkeypatch):
    # the per-edge kernel evaluates the harmonic gradients itself when the
    # per-edge table would exceed its memory cap; force that path here
    monkeypatch.setenv("E2F_GEOM_GT", "0")
    rng = np.random.default_rng(41)
    pos = syn.quantize(rng.uniform(0, 14, size=(400, 3)))
    rp, ci = o.neighbor_list(pos, 5.0)
    check(e2f, ctx, pos, rp, ci, 4, 32, 2, 5.0, 42)
    check(e2f, ctx, pos, rp, ci, 6, 16, 4, 5.0, 43)
