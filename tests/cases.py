"""Seeded test cases shared by the GPU parity tests and the smoke check.

Inputs come from e2f_synth; the CSR and every expected value come from the
oracle only (never from the HIP path).
"""
from __future__ import annotations

import functools

import numpy as np

import e2f_synth as syn
import oracle as o

# float32 parity bar of the layer (max over output irreps of max|err|/max|ref|)
TOL_F32 = 1e-4
# bf16 channel mixing (bf16 inputs, fp32 accumulation)
TOL_BF16 = 1e-2


@functools.lru_cache(maxsize=None)
def case(name: str, n_atoms: int | None = None):
    wl = syn.WORKLOADS[name]
    inp = syn.make_inputs(wl, n_atoms)
    rp, ci = o.neighbor_list(inp.pos, wl.cutoff, inp.graph_id)
    alpha = syn.attention_weights(inp.pos, inp.species, rp, ci, wl.heads, wl.cutoff, wl.species, wl.seed)
    return inp, rp, ci, alpha


def sample_rows(n: int, k: int, seed: int = 0) -> np.ndarray:
    """k receiver rows: the first, the last and a seeded sample between."""
    if k >= n:
        return np.arange(n, dtype=np.int32)
    rng = np.random.default_rng(seed)
    mid = rng.choice(np.arange(1, n - 1), size=k - 2, replace=False)
    return np.sort(np.concatenate([[0, n - 1], mid])).astype(np.int32)
