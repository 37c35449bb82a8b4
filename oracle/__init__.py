"""fp64 CPU oracle of the Wigner-6j convolution (E2Former, arXiv 2501.19216).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
baseline leg of the benchmark may import this package; the product library
never does.  The arithmetic lives in ``e2fo.c`` (plain C, fp64); this file
marshals numpy arrays and adds the Wigner D-matrices used by the
equivariance checks.  See ``e2fo.c`` for the passage of the paper each
function follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "e2fo.c")
_LIB = os.path.join(_HERE, "libe2fo.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle (gcc, -O2, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB):
                build(force=True)
            L = ctypes.CDLL(_LIB)
            d, i, i64, p = ctypes.c_double, ctypes.c_int, ctypes.c_int64, ctypes.c_void_p
            L.e2fo_wigner3j.restype = d
            L.e2fo_wigner3j.argtypes = [i] * 6
            L.e2fo_cg_complex.restype = d
            L.e2fo_cg_complex.argtypes = [i] * 6
            L.e2fo_cg_real.restype = i
            L.e2fo_cg_real.argtypes = [i, i, i, p]
            L.e2fo_wigner6j.restype = d
            L.e2fo_wigner6j.argtypes = [i] * 6
            L.e2fo_recoupling_x.restype = d
            L.e2fo_recoupling_x.argtypes = [i] * 5
            L.e2fo_solid_harmonics.restype = None
            L.e2fo_solid_harmonics.argtypes = [i, p, p]
            L.e2fo_solid_harmonics_grad.restype = None
            L.e2fo_solid_harmonics_grad.argtypes = [i, p, p]
            L.e2fo_conv_edge_grad_pos.restype = i
            L.e2fo_conv_edge_grad_pos.argtypes = [i, i, i, p, p, p, i, p, p, p, p, p, i, p]
            L.e2fo_neighbor_list.restype = i64
            L.e2fo_neighbor_list.argtypes = [p, p, i, ctypes.c_float, p, p, i64]
            L.e2fo_neighbor_list_cells.restype = i64
            L.e2fo_neighbor_list_cells.argtypes = [p, p, i, ctypes.c_float, p, p, i64]
            L.e2fo_knn_graph.restype = i64
            L.e2fo_knn_graph.argtypes = [p, p, i, i, p, p, i64]
            L.e2fo_conv_edge_vjp.restype = i
            L.e2fo_conv_edge_vjp.argtypes = [i, i, i, p, p, p, i, p, p, p, p, p, i, p, i, p, p]
            L.e2fo_attention_weights.restype = None
            L.e2fo_attention_weights.argtypes = [p, p, p, i, i, i, p, i, ctypes.c_float, p, p, p]
            L.e2fo_conv_edge.restype = i
            L.e2fo_conv_edge.argtypes = [i, i, i, p, p, i, p, p, p, p, p, i, i, p]
            L.e2fo_conv_factorised.restype = i
            L.e2fo_conv_factorised.argtypes = [i, i, i, p, p, i, p, p, p, p, p, p]
            L.e2fo_conv_global.restype = i
            L.e2fo_conv_global.argtypes = [i, i, p, p, i, p, p, p, i, p]
            L.e2fo_mix.restype = None
            L.e2fo_mix.argtypes = [i, i, i, p, p, p]
            L.e2fo_aggregate.restype = i
            L.e2fo_aggregate.argtypes = [i, i, i64, p, p, p, p, p, i, p]
            _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


# ---------------------------------------------------------------- algebra
def wigner3j(j1, j2, j3, m1, m2, m3) -> float:
    return lib().e2fo_wigner3j(j1, j2, j3, m1, m2, m3)


def cg_complex(l1, m1, l2, m2, l3, m3) -> float:
    return lib().e2fo_cg_complex(l1, m1, l2, m2, l3, m3)


def cg_real(l1, l2, l3) -> np.ndarray:
    """Real-basis CG tensor [2l1+1, 2l2+1, 2l3+1]."""
    out = np.zeros((2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1))
    rc = lib().e2fo_cg_real(l1, l2, l3, _ptr(out))
    if rc == 1:
        raise ArithmeticError("real CG (%d,%d,%d) is neither real nor imaginary" % (l1, l2, l3))
    return out


def wigner6j(j1, j2, j3, j4, j5, j6) -> float:
    return lib().e2fo_wigner6j(j1, j2, j3, j4, j5, j6)


def recoupling_x(a, b, u, o, d) -> float:
    return lib().e2fo_recoupling_x(a, b, u, o, d)


def solid_harmonics(lmax: int, v) -> np.ndarray:
    """R^(l)_m(v) for l <= lmax; v: [..., 3] -> [..., (lmax+1)^2] (float64)."""
    v = np.asarray(v, dtype=np.float64)
    flat = v.reshape(-1, 3)
    out = np.zeros((flat.shape[0], (lmax + 1) ** 2))
    L = lib()
    row = np.zeros((lmax + 1) ** 2)
    for k in range(flat.shape[0]):
        vk = np.ascontiguousarray(flat[k])
        L.e2fo_solid_harmonics(lmax, _ptr(vk), _ptr(row))
        out[k] = row
    return out.reshape(v.shape[:-1] + ((lmax + 1) ** 2,))


# ---------------------------------------------------------------- graph
def solid_harmonics_grad(lmax: int, v) -> np.ndarray:
    """dR^(l)_m / dv_x for l <= lmax; v: [3] -> [3, (lmax+1)^2] (float64)."""
    v = np.ascontiguousarray(v, dtype=np.float64)
    out = np.zeros((3, (lmax + 1) ** 2))
    lib().e2fo_solid_harmonics_grad(lmax, _ptr(v), _ptr(out))
    return out


def neighbor_list(pos, cutoff: float, graph_id=None, method: str = "auto"):
    """Radius graph as CSR (row_ptr int64 [N+1], col_idx int32 [E])."""
    pos = _c(pos, np.float32)
    gid = _c(graph_id, np.int32)
    n = pos.shape[0]
    fn = lib().e2fo_neighbor_list if (method == "brute" or (method == "auto" and n <= 4096)) else lib().e2fo_neighbor_list_cells
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    E = fn(_ptr(pos), _ptr(gid), n, float(cutoff), _ptr(row_ptr), None, 0)
    col = np.zeros(max(E, 1), dtype=np.int32)
    E2 = fn(_ptr(pos), _ptr(gid), n, float(cutoff), _ptr(row_ptr), _ptr(col), E)
    assert E2 == E
    return row_ptr, col[:E]


def knn_graph(pos, k: int, graph_id=None):
    """k-nearest-neighbour graph as CSR (Sec. 4.1 sparse graphs): row i holds
    the min(k, n_g - 1) atoms of i's graph first in (grid distance, index)
    order, by ascending index."""
    pos = _c(pos, np.float32)
    gid = _c(graph_id, np.int32)
    n = pos.shape[0]
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    E = lib().e2fo_knn_graph(_ptr(pos), _ptr(gid), n, int(k), _ptr(row_ptr), None, 0)
    col = np.zeros(max(E, 1), dtype=np.int32)
    E2 = lib().e2fo_knn_graph(_ptr(pos), _ptr(gid), n, int(k), _ptr(row_ptr), _ptr(col), E)
    assert E2 == E
    return row_ptr, col[:E]


def attention_weights(pos, q, k, rbf_w, cutoff: float, row_ptr, col_idx) -> np.ndarray:
    """Attention weights [E, H] float32 (App. E): q.k logits [N,H,dk] plus the
    radial basis with weights rbf_w [H,R], softmax over each row, cosine
    envelope."""
    pos = _c(pos, np.float32)
    q = _c(q, np.float32)
    k = _c(k, np.float32)
    rbf_w = _c(rbf_w, np.float32)
    row_ptr = _c(row_ptr, np.int64)
    col_idx = _c(col_idx, np.int32)
    n, heads, dk = q.shape
    out = np.zeros((col_idx.shape[0], heads), dtype=np.float32)
    lib().e2fo_attention_weights(_ptr(pos), _ptr(q), _ptr(k), n, heads, dk, _ptr(rbf_w), rbf_w.shape[1],
                                 float(cutoff), _ptr(row_ptr), _ptr(col_idx), _ptr(out))
    return out


# ---------------------------------------------------------------- the layer
def conv_edge(lmax, heads, pos, feat, row_ptr, col_idx, alpha, path_w, rows=None, y_norm=False) -> np.ndarray:
    """The layer by its definition; returns y [n_rows, (L+1)^2, C] float64.
    y_norm: attention weights alpha / D^f per filter degree f (Alg. 1)."""
    pos = _c(pos, np.float32)
    feat = _c(feat, np.float32)
    row_ptr = _c(row_ptr, np.int64)
    col_idx = _c(col_idx, np.int32)
    alpha = _c(alpha, np.float32)
    path_w = _c(path_w, np.float64)
    n, nk, C = feat.shape
    rows = np.arange(n, dtype=np.int32) if rows is None else _c(rows, np.int32)
    out = np.zeros((rows.shape[0], nk, C))
    rc = lib().e2fo_conv_edge(lmax, C, heads, _ptr(pos), _ptr(feat), n, _ptr(row_ptr), _ptr(col_idx),
                              _ptr(alpha), _ptr(path_w), _ptr(rows), rows.shape[0], int(bool(y_norm)), _ptr(out))
    if rc:
        raise ValueError("e2fo_conv_edge rejected its arguments")
    return out


def conv_edge_vjp(lmax, heads, pos, feat, gy, row_ptr, col_idx, alpha, path_w, want_feat=True, want_alpha=True,
                  alpha_rows=None, feat_rows=None):
    """Vector-Jacobian products of the layer (by its definition) for the
    output gradient gy [n, (L+1)^2, C]: (gfeat [n, (L+1)^2, C], galpha [E, H]),
    float64; either may be skipped (None).  alpha_rows: receivers whose edges
    get galpha; feat_rows: senders that get gfeat (default all; others 0)."""
    arows = _c(alpha_rows, np.int32)
    frows = _c(feat_rows, np.int32)
    pos = _c(pos, np.float32)
    feat = _c(feat, np.float32)
    gy = _c(gy, np.float64)
    row_ptr = _c(row_ptr, np.int64)
    col_idx = _c(col_idx, np.int32)
    alpha = _c(alpha, np.float32)
    path_w = _c(path_w, np.float64)
    n, nk, C = feat.shape
    gf = np.zeros((n, nk, C)) if want_feat else None
    ga = np.zeros((col_idx.shape[0], heads)) if want_alpha else None
    rc = lib().e2fo_conv_edge_vjp(lmax, C, heads, _ptr(pos), _ptr(feat), _ptr(gy), n, _ptr(row_ptr), _ptr(col_idx),
                                  _ptr(alpha), _ptr(path_w), _ptr(arows), 0 if arows is None else len(arows),
                                  _ptr(frows), 0 if frows is None else len(frows), _ptr(gf), _ptr(ga))
    if rc:
        raise ValueError("e2fo_conv_edge_vjp rejected its arguments")
    return gf, ga


def conv_edge_grad_pos(lmax, heads, pos, feat, gy, row_ptr, col_idx, alpha, path_w, atoms=None) -> np.ndarray:
    """Gradient of sum(gy * layer) with respect to the positions (the graph
    and alpha held fixed), by the definition: [n or len(atoms), 3] float64."""
    at = _c(atoms, np.int32)
    pos = _c(pos, np.float32)
    feat = _c(feat, np.float32)
    n, nk, C = feat.shape
    out = np.zeros((n if at is None else len(at), 3))
    rc = lib().e2fo_conv_edge_grad_pos(lmax, C, heads, _ptr(pos), _ptr(feat), _ptr(_c(gy, np.float64)), n,
                                       _ptr(_c(row_ptr, np.int64)), _ptr(_c(col_idx, np.int32)),
                                       _ptr(_c(alpha, np.float32)), _ptr(_c(path_w, np.float64)), _ptr(at),
                                       0 if at is None else len(at), _ptr(out))
    if rc:
        raise ValueError("e2fo_conv_edge_grad_pos rejected its arguments")
    return out


def conv_factorised(lmax, heads, pos, feat, row_ptr, col_idx, alpha, path_w, origin) -> np.ndarray:
    """The layer by node factorisation (tiny graphs); y [N, (L+1)^2, C] float64."""
    pos = _c(pos, np.float32)
    feat = _c(feat, np.float32)
    n, nk, C = feat.shape
    out = np.zeros((n, nk, C))
    org = np.ascontiguousarray(origin, dtype=np.float64)
    rc = lib().e2fo_conv_factorised(lmax, C, heads, _ptr(pos), _ptr(feat), n, _ptr(_c(row_ptr, np.int64)),
                                    _ptr(_c(col_idx, np.int32)), _ptr(_c(alpha, np.float32)),
                                    _ptr(_c(path_w, np.float64)), _ptr(org), _ptr(out))
    if rc:
        raise ValueError("e2fo_conv_factorised failed (%d)" % rc)
    return out


def conv_global(lmax, pos, feat, path_w, origin, rows=None) -> np.ndarray:
    """Uniform attention over the whole graph (alpha = 1 for every pair, self
    included) in the global-moment form of App. G; y [N or len(rows), (L+1)^2, C]
    float64."""
    pos = _c(pos, np.float32)
    feat = _c(feat, np.float32)
    n, nk, C = feat.shape
    r = None if rows is None else _c(rows, np.int32)
    out = np.zeros((n if r is None else len(r), nk, C))
    org = np.ascontiguousarray(origin, dtype=np.float64)
    rc = lib().e2fo_conv_global(lmax, C, _ptr(pos), _ptr(feat), n, _ptr(_c(path_w, np.float64)), _ptr(org),
                                None if r is None else _ptr(r), 0 if r is None else len(r), _ptr(out))
    if rc:
        raise ValueError("e2fo_conv_global failed (%d)" % rc)
    return out


def mix(lmax, y, W) -> np.ndarray:
    y = _c(y, np.float64)
    W = _c(W, np.float32)
    out = np.zeros_like(y)
    lib().e2fo_mix(lmax, y.shape[2], y.shape[0], _ptr(y), _ptr(W), _ptr(out))
    return out


def aggregate(T, row_ptr, col_idx, alpha=None, rows=None) -> np.ndarray:
    """S[i][h] = sum over row i's edges e = (i, j) of alpha[e][h] T[j][h]
    (Alg. 1's einsum "ijh,jhds->ihds" over the graph's edges), float64, for
    T [n, H, ...] float32 and alpha [E, H] or None (ones); rows: receivers
    (default all)."""
    T = _c(T, np.float32)
    n, H = T.shape[0], T.shape[1]
    W = int(np.prod(T.shape[2:]))
    row_ptr = _c(row_ptr, np.int64)
    col_idx = _c(col_idx, np.int32)
    a = None if alpha is None else _c(alpha, np.float32)
    r = None if rows is None else _c(rows, np.int32)
    nr = n if r is None else r.shape[0]
    out = np.zeros((nr,) + T.shape[1:])
    rc = lib().e2fo_aggregate(n, H, W, _ptr(T), _ptr(row_ptr), _ptr(col_idx), None if a is None else _ptr(a),
                              None if r is None else _ptr(r), nr, _ptr(out))
    if rc:
        raise ValueError("aggregate: an index is out of range")
    return out


def layer(lmax, heads, pos, feat, row_ptr, col_idx, alpha, path_w, mix_w=None, rows=None, y_norm=False) -> np.ndarray:
    """Definition plus optional per-irrep mixing: the full forward output."""
    y = conv_edge(lmax, heads, pos, feat, row_ptr, col_idx, alpha, path_w, rows, y_norm)
    return y if mix_w is None else mix(lmax, y, mix_w)


# ---------------------------------------------------------------- rotations
def wigner_d(lmax: int, Q: np.ndarray, n_probe: int = 64, seed: int = 7) -> list:
    """Real Wigner D^(l)(Q) for l <= lmax, from R^(l)(Q v) = D^(l) R^(l)(v)
    solved by least squares over random probe vectors (no Euler angles)."""
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((n_probe, 3))
    Rv = solid_harmonics(lmax, v)
    RQv = solid_harmonics(lmax, v @ Q.T)
    Ds = []
    for l in range(lmax + 1):
        s = slice(l * l, (l + 1) * (l + 1))
        A, B = Rv[:, s], RQv[:, s]
        Dt, *_ = np.linalg.lstsq(A, B, rcond=None)
        Ds.append(Dt.T)
    return Ds


def random_rotation(seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    q, r = np.linalg.qr(rng.standard_normal((3, 3)))
    q = q @ np.diag(np.sign(np.diag(r)))
    if np.linalg.det(q) < 0:
        q[:, 0] = -q[:, 0]
    return q


def max_rel_err(got: np.ndarray, ref: np.ndarray, lmax: int) -> float:
    """max over output irreps o of max|got-ref| / max|ref| on block o."""
    worst = 0.0
    for o in range(lmax + 1):
        s = slice(o * o, (o + 1) * (o + 1))
        den = float(np.max(np.abs(ref[:, s, :]))) if ref.size else 0.0
        num = float(np.max(np.abs(got[:, s, :] - ref[:, s, :]))) if ref.size else 0.0
        if den > 0:
            worst = max(worst, num / den)
        elif num > 0:
            worst = float("inf")
    return worst
