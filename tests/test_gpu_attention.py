"""GPU attention weights (App. E; the alpha input of Alg. 1) against the
oracle.  Run with -m gpu."""
import numpy as np
import pytest
import torch

import e2f_synth as syn
import oracle as o
from cases import case

pytestmark = pytest.mark.gpu
TOL_ATT = 1e-5  # fp32 logits, exp and cos against fp64: max |d| / max |alpha| per head


@pytest.fixture(scope="module")
def e2f():
    import paper_2501_19216_amd as m
    return m


@pytest.fixture(scope="module")
def ctx(e2f):
    c = e2f.e2f_create(2, 0)
    yield c
    c.close()


def gpu(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def att_err(got, ref):
    return float(np.max(np.abs(got - ref).max(axis=0) / np.maximum(np.abs(ref).max(axis=0), 1e-30)))


def run(e2f, ctx, pos, rp, ci, rc, H, dk, R, seed):
    rng = np.random.default_rng(seed)
    n = pos.shape[0]
    q = rng.standard_normal((n, H, dk)).astype(np.float32) if dk else None
    k = rng.standard_normal((n, H, dk)).astype(np.float32) / max(dk, 1) ** 0.5 if dk else None
    w = rng.standard_normal((H, R)).astype(np.float32) if R else None
    ref = o.attention_weights(pos, q if dk else np.zeros((n, H, 0), np.float32),
                              k if dk else np.zeros((n, H, 0), np.float32),
                              w if R else np.zeros((H, 0), np.float32), rc, rp, ci)
    got = e2f.e2f_attention_weights(ctx, gpu(pos), gpu(rp), gpu(ci), rc, gpu(q), gpu(k), gpu(w), heads=H)
    return got, ref


def test_attention_protein_graph(e2f, ctx):
    inp, rp, ci, _ = case("protein20k_L4")
    wl = inp.workload
    got, ref = run(e2f, ctx, inp.pos, rp, ci, wl.cutoff, 8, 16, 8, 1)
    err = att_err(got.cpu().numpy(), ref)
    print("protein: %d edges, err %.3e" % (len(ci), err))
    assert err <= TOL_ATT
    got2, _ = run(e2f, ctx, inp.pos, rp, ci, wl.cutoff, 8, 16, 8, 1)
    assert torch.equal(got, got2)  # deterministic


@pytest.mark.parametrize("H,dk,R", [(1, 0, 2), (3, 1, 8), (8, 4, 0), (64, 2, 32), (5, 16, 5)])
def test_attention_shapes(e2f, ctx, H, dk, R):
    inp, rp, ci, _ = case("water2000_L4")
    got, ref = run(e2f, ctx, inp.pos, rp, ci, 6.0, H, dk, R, H + dk + R)
    err = att_err(got.cpu().numpy(), ref)
    print("H %d dk %d R %d: err %.3e" % (H, dk, R, err))
    assert err <= TOL_ATT


def test_attention_beyond_cutoff_and_empty_rows(e2f, ctx):
    rng = np.random.default_rng(4)
    pos = syn.quantize(rng.uniform(0, 15, size=(300, 3)))
    pos[-1] = [90.0, 90.0, 90.0]
    rp, ci = o.knn_graph(pos[:-1], 12)
    rp = np.append(rp, rp[-1])  # the far atom: an empty row
    got, ref = run(e2f, ctx, pos, rp, ci, 2.5, 4, 8, 6, 2)  # many kNN edges longer than the cutoff
    got = got.cpu().numpy()
    assert np.any(ref == 0) and np.all(got[ref == 0] == 0)
    assert att_err(got, ref) <= TOL_ATT
