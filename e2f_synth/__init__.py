"""Seeded synthetic inputs for the Wigner-6j convolution and its checks.

This module is shared by the fp64 oracle, the tests and the benchmark.  It
holds none of the layer's arithmetic: it only draws positions, species,
irrep features, attention weights and mixing weights with fixed seeds, in
the shapes of the paper's synthetic scaling study (Sec. 4.1: random graphs
of N atoms at several maximum degrees L) and of the five benchmark
workloads listed in ``WORKLOADS``.

Conventions shared with both implementations:
  * positions are float32 on a 2^-16 Angstrom grid, so that squared
    distances are exact integers on that grid;
  * features are [N, (L+1)^2, C] float32, irrep-major (index l*l+l+m);
  * channel c belongs to head c // (C // H);
  * attention weights are [E, H] float32 in CSR order (rows = receivers i,
    columns = senders j ascending);
  * mixing weights are [(L+1), C, C] float32, W[o][c_out][c_in].
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

GRID = 65536.0  # positions live on a 2^-16 Angstrom grid


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_atoms: int          # total atoms
    geometry: str         # "cube" or "molecules"
    side: float           # cube side (A) or molecule ball radius (A)
    n_graphs: int         # molecules (1 for a single cluster)
    min_dist: float
    cutoff: float
    lmax: int
    channels: int
    heads: int
    species: int
    seed: int


def _cube_side(n: int, density: float = 0.1) -> float:
    return (n / density) ** (1.0 / 3.0)


# The five benchmark workloads (sizes, densities and cutoffs of the layer's
# intended regimes: a small cluster, a batch of molecules, a liquid-density
# cluster, a protein-scale system and a scaling stress case).
WORKLOADS = {
    "cluster32_L2": Workload("cluster32_L2", 32, "cube", 6.0, 1, 0.8, 5.0, 2, 16, 4, 5, 1),
    "molecules256x30_L3": Workload("molecules256x30_L3", 256 * 30, "molecules", 7.0, 256, 0.9, 5.0, 3, 64, 8, 10, 2),
    "water2000_L4": Workload("water2000_L4", 2000, "cube", _cube_side(2000), 1, 0.9, 6.0, 4, 128, 8, 10, 3),
    "protein20k_L4": Workload("protein20k_L4", 20000, "cube", _cube_side(20000), 1, 0.9, 6.0, 4, 128, 8, 10, 4),
    "stress200k_L6": Workload("stress200k_L6", 200000, "cube", _cube_side(200000), 1, 0.9, 8.0, 6, 64, 8, 10, 5),
}


def quantize(x: np.ndarray) -> np.ndarray:
    """Round coordinates to the 2^-16 A grid (exact in float32 below 256 A)."""
    return (np.rint(np.asarray(x, dtype=np.float64) * GRID) / GRID).astype(np.float32)


def _rsa(rng: np.random.Generator, n: int, draw, min_dist: float) -> np.ndarray:
    """Greedy random sequential addition: candidates are drawn in order and
    kept unless an earlier kept candidate lies closer than min_dist."""
    from scipy.spatial import cKDTree

    kept = np.zeros((0, 3), dtype=np.float32)
    while kept.shape[0] < n:
        need = n - kept.shape[0]
        cand = quantize(draw(int(need * 1.3) + 16))
        allpts = np.concatenate([kept, cand]).astype(np.float64)
        tree = cKDTree(allpts)
        pairs = tree.query_pairs(min_dist, output_type="ndarray")
        k0 = kept.shape[0]
        alive = np.ones(allpts.shape[0], dtype=bool)
        if pairs.size:
            # exact check on the grid values (query_pairs uses <=)
            d2 = np.sum((allpts[pairs[:, 0]] - allpts[pairs[:, 1]]) ** 2, axis=1)
            pairs = pairs[d2 < min_dist * min_dist]
            lo = np.minimum(pairs[:, 0], pairs[:, 1])
            hi = np.maximum(pairs[:, 0], pairs[:, 1])
            order = np.lexsort((lo, hi))
            lo, hi = lo[order], hi[order]
            # visit candidates in order; a candidate dies if any earlier alive
            # point conflicts with it
            conflicts: dict[int, list[int]] = {}
            for a, b in zip(lo.tolist(), hi.tolist()):
                conflicts.setdefault(b, []).append(a)
            for b in sorted(conflicts):
                if b < k0:
                    continue
                if any(alive[a] for a in conflicts[b]):
                    alive[b] = False
        new = allpts[k0:][alive[k0:]].astype(np.float32)
        kept = np.concatenate([kept, new[:need]])
    return kept[:n]


def positions_cube(n: int, side: float, min_dist: float, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return _rsa(rng, n, lambda k: rng.uniform(0.0, side, size=(k, 3)), min_dist)


def positions_ball(n: int, radius: float, min_dist: float, rng: np.random.Generator) -> np.ndarray:
    def draw(k):
        v = rng.normal(size=(k, 3))
        v /= np.linalg.norm(v, axis=1, keepdims=True)
        r = radius * rng.uniform(0.0, 1.0, size=(k, 1)) ** (1.0 / 3.0)
        return v * r
    return _rsa(rng, n, draw, min_dist)


@dataclasses.dataclass
class Inputs:
    pos: np.ndarray            # [N,3] float32 on the grid
    graph_id: np.ndarray | None  # [N] int32 or None
    species: np.ndarray        # [N] int32
    feat: np.ndarray           # [N,(L+1)^2,C] float32
    mix_w: np.ndarray          # [(L+1),C,C] float32
    path_w: np.ndarray         # [(L+1)^3] float64, [a][f][o]
    workload: Workload


def default_path_weights(lmax: int, cutoff: float) -> np.ndarray:
    """w[a,f,o] = cutoff^-f on triangle-valid (a,f,o), zero elsewhere."""
    w = np.zeros((lmax + 1,) * 3, dtype=np.float64)
    for a in range(lmax + 1):
        for f in range(lmax + 1):
            for o in range(abs(a - f), min(a + f, lmax) + 1):
                w[a, f, o] = float(cutoff) ** (-f)
    return w.reshape(-1)


def make_inputs(wl: Workload, n_atoms: int | None = None) -> Inputs:
    """Draw the seeded inputs of a workload (optionally with fewer atoms)."""
    rng = np.random.default_rng(0xE2F00000 + wl.seed)
    n = wl.n_atoms if n_atoms is None else n_atoms
    if wl.geometry == "cube":
        side = wl.side if n_atoms is None else _cube_side(n) if wl.n_atoms > 64 else wl.side
        pos = positions_cube(n, side, wl.min_dist, 0xE2F00000 + wl.seed)
        graph_id = None
    else:
        per = wl.n_atoms // wl.n_graphs
        n_g = max(1, n // per)
        parts = [positions_ball(per, wl.side, wl.min_dist, rng) for _ in range(n_g)]
        pos = np.concatenate(parts)
        graph_id = np.repeat(np.arange(n_g, dtype=np.int32), per)
        n = pos.shape[0]
    species = rng.integers(0, wl.species, size=n).astype(np.int32)
    nk = (wl.lmax + 1) ** 2
    feat = rng.standard_normal((n, nk, wl.channels), dtype=np.float32)
    mix_w = (rng.standard_normal((wl.lmax + 1, wl.channels, wl.channels)) / math.sqrt(wl.channels)).astype(np.float32)
    return Inputs(pos, graph_id, species, feat, mix_w, default_path_weights(wl.lmax, wl.cutoff), wl)


def _attention_tables(heads: int, cutoff: float, n_species: int, seed: int):
    """The seeded species embedding, radial mixing weights and radial centres
    of the synthetic attention weights (shared by both generators below)."""
    rng = np.random.default_rng(0xA1FA0000 + seed)
    emb = rng.standard_normal((n_species, heads))
    rho = rng.standard_normal((heads, 8)) / math.sqrt(8.0)
    mu = np.arange(8) * cutoff / 7.0
    return emb, rho, mu, cutoff / 7.0


def attention_weights_device(pos, species, row_ptr, col_idx, heads: int, cutoff: float, n_species: int, seed: int,
                             device):
    """The same synthetic attention weights as attention_weights, computed
    with torch in float64 on `device` (for inputs too large for the host
    generator) and rounded to float32: [E, H].  Row sums are taken in another
    order than on the host, so values may differ from attention_weights in
    the last bit."""
    import torch
    emb, rho, mu, sigma = _attention_tables(heads, cutoff, n_species, seed)
    rp = torch.as_tensor(np.asarray(row_ptr, dtype=np.int64), device=device)
    ci = torch.as_tensor(np.asarray(col_idx, dtype=np.int64), device=device)
    n = rp.numel() - 1
    E = int(rp[-1].item())
    if E == 0:
        return torch.empty(0, heads, dtype=torch.float32, device=device)
    recv = torch.repeat_interleave(torch.arange(n, device=device), rp[1:] - rp[:-1])
    p64 = torch.as_tensor(np.asarray(pos, dtype=np.float64), device=device)
    sp = torch.as_tensor(np.asarray(species, dtype=np.int64), device=device)
    emb_t = torch.as_tensor(emb, device=device)
    rho_t = torch.as_tensor(rho, device=device)
    mu_t = torch.as_tensor(mu, device=device)
    logits = torch.empty(E, heads, dtype=torch.float64, device=device)
    env = torch.empty(E, dtype=torch.float64, device=device)
    chunk = 1 << 22
    for s in range(0, E, chunk):
        i, j = recv[s:s + chunk], ci[s:s + chunk]
        d = torch.linalg.norm(p64[i] - p64[j], dim=1)
        rbf = torch.exp(-(((d[:, None] - mu_t[None, :]) / sigma) ** 2))
        logits[s:s + chunk] = emb_t[sp[i]] * emb_t[sp[j]] + rbf @ rho_t.T
        env[s:s + chunk] = 0.5 * (torch.cos(math.pi * d / cutoff) + 1.0)
    idx = recv[:, None].expand(-1, heads)
    rmax = torch.zeros(n, heads, dtype=torch.float64, device=device).scatter_reduce_(0, idx, logits, "amax",
                                                                                      include_self=False)
    ex = torch.exp(logits - rmax[recv])
    den = torch.zeros(n, heads, dtype=torch.float64, device=device).index_add_(0, recv, ex)
    return (env[:, None] * ex / den[recv]).to(torch.float32)


def attention_weights(pos: np.ndarray, species: np.ndarray, row_ptr: np.ndarray, col_idx: np.ndarray,
                      heads: int, cutoff: float, n_species: int, seed: int) -> np.ndarray:
    """Synthetic per-edge, per-head attention weights [E, H] float32.

    logit_ijh = E_h[s_i] E_h[s_j] + sum_k rho_hk exp(-((d_ij - mu_k)/sigma)^2),
    alpha_ijh = (cos(pi d_ij / cutoff) + 1)/2 * softmax over j in N(i).
    Depends only on distances and species, so it is rotation and translation
    invariant.  Computed in float64, rounded to float32.
    """
    emb, rho, mu, sigma = _attention_tables(heads, cutoff, n_species, seed)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    n = row_ptr.shape[0] - 1
    E = int(row_ptr[-1])
    out = np.empty((E, heads), dtype=np.float32)
    if E == 0:
        return out
    recv = np.repeat(np.arange(n, dtype=np.int64), np.diff(row_ptr))
    chunk = 1 << 21
    p64 = pos.astype(np.float64)
    logits = np.empty((E, heads), dtype=np.float64)
    env = np.empty(E, dtype=np.float64)
    for s in range(0, E, chunk):
        i = recv[s:s + chunk]
        j = col_idx[s:s + chunk]
        d = np.linalg.norm(p64[i] - p64[j], axis=1)
        rbf = np.exp(-(((d[:, None] - mu[None, :]) / sigma) ** 2))
        logits[s:s + chunk] = emb[species[i]] * emb[species[j]] + rbf @ rho.T
        env[s:s + chunk] = 0.5 * (np.cos(np.pi * d / cutoff) + 1.0)
    # segmented softmax per receiver row (rows are contiguous in CSR order)
    deg = np.diff(row_ptr)
    nz = np.nonzero(deg)[0]
    starts = row_ptr[nz]
    rmax = np.zeros((n, heads))
    rmax[nz] = np.maximum.reduceat(logits, starts, axis=0)
    ex = np.exp(logits - rmax[recv])
    den = np.ones((n, heads))
    den[nz] = np.add.reduceat(ex, starts, axis=0)
    out[:] = (env[:, None] * ex / den[recv]).astype(np.float32)
    return out
