"""GPU parity of the standalone aggregation (Alg. 1's einsum over the graph's
edges with stored node tensors) against the fp64 oracle's edge loop.

Calls go through the C ABI.  Bar: max |err| <= 1e-5 max |ref| (float32 sums
of at most a few hundred products).
"""
import numpy as np
import pytest
import torch

import oracle as o
import e2f_synth as syn
from cases import case, sample_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-5


@pytest.fixture(scope="module")
def e2f():
    import paper_2501_19216_amd as e
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return e


@pytest.fixture(scope="module")
def ctx(e2f):
    c = e2f.e2f_create(4, 0)
    yield c
    c.close()


def gpu(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def rel_err(got, ref):
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))


def cell_order(pos, cell=4.0):
    # receivers sorted by a Morton key of 4 A cells (close atoms together)
    q = np.floor((pos - pos.min(0)) / cell).astype(np.int64)
    key = np.zeros(len(pos), dtype=np.int64)
    for b in range(10):
        for a in range(3):
            key |= ((q[:, a] >> b) & 1) << (3 * b + a)
    return np.argsort(key, kind="stable").astype(np.int32)


@pytest.mark.parametrize("n,box,cut,H,K,dh,with_alpha,order", [(301, 12.0, 5.0, 4, 9, 8, True, None),
                                                                (301, 12.0, 5.0, 4, 9, 8, True, "cells"),
                                                                (301, 12.0, 5.0, 4, 9, 8, False, "random"),
                                                                (77, 8.0, 4.0, 1, 3, 4, False, None),
                                                                (700, 10.0, 30.0, 2, 5, 4, True, "random")])
def test_aggregate_small(e2f, ctx, n, box, cut, H, K, dh, with_alpha, order):
    # a radius graph with an isolated atom, receivers in index, cell or random
    # order; the last case is a complete graph of 700 atoms (blocks of 16
    # receivers hold 11k edges: the per-receiver path)
    rng = np.random.default_rng(n + H)
    pos = syn.quantize(rng.uniform(0, box, size=(n, 3)))
    pos[-1] = [90.0, 90.0, 90.0]
    rp, ci = o.neighbor_list(pos, cut)
    T = rng.standard_normal((n, H, K, dh)).astype(np.float32)
    alpha = rng.uniform(0.0, 1.0, size=(len(ci), H)).astype(np.float32) if with_alpha else None
    print("aggregate: n %d edges %d max degree %d" % (n, len(ci), int(np.diff(rp).max())), flush=True)
    perm = None if order is None else (cell_order(pos) if order == "cells" else rng.permutation(n).astype(np.int32))
    S = e2f.e2f_aggregate(ctx, gpu(T), gpu(rp), gpu(ci), None if alpha is None else gpu(alpha),
                          order=None if perm is None else gpu(perm)).cpu().numpy()
    ref = o.aggregate(T, rp, ci, alpha)
    err = rel_err(S, ref)
    print("  err %.3e" % err)
    assert err <= TOL
    assert np.all(S[-1] == 0)


def test_aggregate_water2000_rows_of_T(e2f, ctx):
    # 2,000 atoms, 143k edges, T rows of the layer's width at L = 4, C = 128,
    # H = 8 (454 rows of 16 channels per head): sampled receivers
    inp, rp, ci, alpha = case("water2000_L4")
    n = inp.pos.shape[0]
    rng = np.random.default_rng(5)
    T = rng.standard_normal((n, 8, e2f.e2f_node_tp_dim(4), 16)).astype(np.float32)
    S = e2f.e2f_aggregate(ctx, gpu(T), gpu(rp), gpu(ci), gpu(alpha))
    r = sample_rows(n, 64, seed=2)
    ref = o.aggregate(T, rp, ci, alpha, rows=r)
    err = rel_err(S.cpu().numpy()[r], ref)
    print("water2000 aggregate: err %.3e" % err)
    assert err <= TOL


def test_aggregate_errors(e2f, ctx):
    rng = np.random.default_rng(3)
    n = 40
    pos = syn.quantize(rng.uniform(0, 6, size=(n, 3)))
    rp, ci = o.neighbor_list(pos, 3.5)
    T = gpu(rng.standard_normal((n, 2, 3, 4)).astype(np.float32))
    # a row whose senders are not ascending, and a sender out of range
    i = int(np.argmax(np.diff(rp)))
    bad = ci.copy()
    bad[rp[i]], bad[rp[i] + 1] = ci[rp[i] + 1], ci[rp[i]]
    with pytest.raises(e2f.E2FError) as ei:
        e2f.e2f_aggregate(ctx, T, gpu(rp), gpu(bad), None)
    assert ei.value.status == e2f.E2F_EINVAL and "16" in str(ei.value)
    bad = ci.copy()
    bad[0] = n
    with pytest.raises(e2f.E2FError) as ei:
        e2f.e2f_aggregate(ctx, T, gpu(rp), gpu(bad), None)
    assert ei.value.status == e2f.E2F_EINVAL
    # an order that is not a permutation (a repeated receiver, one out of range)
    for o_bad in (np.r_[np.arange(n - 1), 0], np.r_[np.arange(n - 1), n]):
        with pytest.raises(e2f.E2FError) as ei:
            e2f.e2f_aggregate(ctx, T, gpu(rp), gpu(ci), None, order=gpu(o_bad.astype(np.int32)))
        assert ei.value.status == e2f.E2F_EINVAL and "32" in str(ei.value)
    # a workspace below the size query
    need = e2f.lib.e2f_aggregate_workspace_size
    import ctypes
    b = ctypes.c_size_t(0)
    assert need(ctx.handle, n, len(ci), 2, ctypes.byref(b)) == e2f.E2F_OK
    with pytest.raises(e2f.E2FError) as ei:
        e2f.e2f_aggregate(ctx, T, gpu(rp), gpu(ci), None,
                          workspace=torch.empty(b.value - 256, dtype=torch.uint8, device=DEV))
    assert ei.value.status == e2f.E2F_ECAPACITY
    # no edges at all: zeros
    S = e2f.e2f_aggregate(ctx, T, gpu(np.zeros(n + 1, dtype=np.int64)), gpu(np.zeros(0, dtype=np.int32)), None)
    assert torch.count_nonzero(S).item() == 0
