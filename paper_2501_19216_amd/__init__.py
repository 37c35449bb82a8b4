"""Python binding of libe2f, the MI355X Wigner-6j convolution (E2Former,
arXiv 2501.19216).

Argument marshalling only: every step of the layer runs in the HIP kernels
of ``libe2f.so`` through its C ABI (``include/e2f.h``); torch tensors are
used for device memory and the current stream.  The functions carry the
names of the C entry points.  If the library is not built, importing this
package raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libe2f.so")

E2F_OK, E2F_EINVAL, E2F_ECAPACITY, E2F_ENOMEM, E2F_EDEVICE, E2F_EUNSUPPORTED = range(6)
E2F_F32, E2F_BF16 = 0, 1
E2F_FORM_AUTO, E2F_FORM_SPLIT, E2F_FORM_FUSED = 0, 1, 2
_FORMS = {"auto": E2F_FORM_AUTO, "split": E2F_FORM_SPLIT, "fused": E2F_FORM_FUSED}
_STATUS = {0: "E2F_OK", 1: "E2F_EINVAL", 2: "E2F_ECAPACITY", 3: "E2F_ENOMEM", 4: "E2F_EDEVICE", 5: "E2F_EUNSUPPORTED"}

# every function declared in include/e2f.h
EXPORTED = ["e2f_create", "e2f_destroy", "e2f_last_error", "e2f_node_tp_dim", "e2f_real_cg", "e2f_knn_graph",
            "e2f_attention_weights", "e2f_recoupling_weight", "e2f_neighbor_list", "e2f_solid_harmonics",
            "e2f_node_tp", "e2f_aggregate_workspace_size", "e2f_aggregate", "e2f_wigner6j_workspace_size", "e2f_wigner6j_workspace_min", "e2f_wigner6j_prepare",
            "e2f_wigner6j_conv_forward", "e2f_wigner6j_conv_forward_noalloc", "e2f_validate_graph", "e2f_wigner6j_conv_forward_dense",
            "e2f_wigner6j_conv_forward_global", "e2f_wigner6j_conv_backward", "e2f_edge_tp_conv_forward",
            "e2f_profile", "e2f_profile_read", "e2f_last_slices"]


class E2FError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__("%s: %s (%s)" % (where, _STATUS.get(status, status), msg))
        self.status = status


class ConvParams(ctypes.Structure):
    _fields_ = [("lmax", ctypes.c_int), ("channels", ctypes.c_int32), ("heads", ctypes.c_int32),
                ("cutoff", ctypes.c_float), ("path_w", ctypes.c_void_p), ("mix_w", ctypes.c_void_p),
                ("mix_dtype", ctypes.c_int), ("tile_side", ctypes.c_float), ("y_norm", ctypes.c_int32),
                ("form", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libe2f.so is not built; run `python paper_2501_19216_amd/build_lib.py` "
                          "(or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    i, i32, i64, p, f = ctypes.c_int, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_float
    L.e2f_create.argtypes = [i, i, ctypes.POINTER(p)]
    L.e2f_create.restype = i
    L.e2f_destroy.argtypes = [p]
    L.e2f_destroy.restype = None
    L.e2f_last_error.argtypes = []
    L.e2f_last_error.restype = ctypes.c_char_p
    L.e2f_node_tp_dim.argtypes = [i]
    L.e2f_node_tp_dim.restype = i64
    L.e2f_real_cg.argtypes = [i, i, i, p]
    L.e2f_real_cg.restype = i
    L.e2f_recoupling_weight.argtypes = [i, i, i, i, i]
    L.e2f_recoupling_weight.restype = ctypes.c_double
    L.e2f_neighbor_list.argtypes = [p, p, p, i32, f, p, p, i64, ctypes.POINTER(i64), p]
    L.e2f_neighbor_list.restype = i
    L.e2f_knn_graph.argtypes = [p, p, p, i32, i32, p, p, i64, ctypes.POINTER(i64), p]
    L.e2f_knn_graph.restype = i
    L.e2f_attention_weights.argtypes = [p, p, p, p, i32, i32, i32, p, i32, f, p, p, i64, p, p]
    L.e2f_attention_weights.restype = i
    L.e2f_solid_harmonics.argtypes = [p, p, p, p, i32, i, p, p]
    L.e2f_solid_harmonics.restype = i
    L.e2f_node_tp.argtypes = [p, p, p, p, p, i32, i32, i, p, p]
    L.e2f_node_tp.restype = i
    L.e2f_aggregate_workspace_size.argtypes = [p, i32, i64, i32, ctypes.POINTER(ctypes.c_size_t)]
    L.e2f_aggregate_workspace_size.restype = i
    L.e2f_aggregate.argtypes = [p, p, i32, i32, i32, i32, p, p, i64, p, p, p, p, ctypes.c_size_t, p]
    L.e2f_aggregate.restype = i
    L.e2f_last_slices.argtypes = [p, ctypes.POINTER(i64)]
    L.e2f_last_slices.restype = i
    for name in ("e2f_wigner6j_workspace_size", "e2f_wigner6j_workspace_min"):
        fn = getattr(L, name)
        fn.argtypes = [p, ctypes.POINTER(ConvParams), i32, i64, ctypes.POINTER(ctypes.c_size_t)]
        fn.restype = i
    L.e2f_wigner6j_prepare.argtypes = [p, ctypes.POINTER(ConvParams)]
    L.e2f_wigner6j_prepare.restype = i
    L.e2f_validate_graph.argtypes = [p, i32, p, p, i64, ctypes.POINTER(i32), p]
    L.e2f_validate_graph.restype = i
    L.e2f_profile.argtypes = [p, i]
    L.e2f_profile.restype = i
    L.e2f_profile_read.argtypes = [p, ctypes.c_char_p, ctypes.c_size_t]
    L.e2f_profile_read.restype = i
    L.e2f_wigner6j_conv_forward.argtypes = [p, ctypes.POINTER(ConvParams), p, p, p, i32, p, p, i64, p, p, p,
                                            ctypes.c_size_t, p]
    L.e2f_wigner6j_conv_forward.restype = i
    L.e2f_wigner6j_conv_forward_noalloc.argtypes = [p, ctypes.POINTER(ConvParams), p, p, p, i32, p, p, i64, p, p,
                                                    p]
    L.e2f_wigner6j_conv_forward_noalloc.restype = i
    L.e2f_edge_tp_conv_forward.argtypes = [p, ctypes.POINTER(ConvParams), p, p, p, i32, p, p, i64, p, p, p]
    L.e2f_edge_tp_conv_forward.restype = i
    L.e2f_wigner6j_conv_forward_dense.argtypes = [p, ctypes.POINTER(ConvParams), p, p, i32, p, p, p]
    L.e2f_wigner6j_conv_forward_dense.restype = i
    L.e2f_wigner6j_conv_forward_global.argtypes = [p, ctypes.POINTER(ConvParams), p, p, i32, p, p]
    L.e2f_wigner6j_conv_forward_global.restype = i
    L.e2f_wigner6j_conv_backward.argtypes = [p, ctypes.POINTER(ConvParams), p, p, p, p, i32, p, p, i64, p, p, p, p, p]
    L.e2f_wigner6j_conv_backward.restype = i
    return L


lib = _load()


def _check(st: int, where: str, allow=()):
    if st != E2F_OK and st not in allow:
        raise E2FError(st, where, lib.e2f_last_error().decode())
    return st


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device=None):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dev(t, dtype, name):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype != dtype or not t.is_contiguous():
        raise ValueError("%s must be a contiguous %s tensor" % (name, dtype))
    return t


class Context:
    """Owns an e2f_ctx (coefficient tables) on one device, and the device
    workspace tensor the binding passes to the Wigner-6j forward."""

    def __init__(self, lmax_max: int = 6, device: int | None = 0):
        h = ctypes.c_void_p()
        dev = -1 if device is None else int(device)
        _check(lib.e2f_create(lmax_max, dev, ctypes.byref(h)), "e2f_create")
        self.handle = h
        self.device = dev
        self.lmax_max = lmax_max
        self.workspace = None

    def workspace_for(self, nbytes: int, device) -> torch.Tensor:
        """A device buffer of at least nbytes, kept for later calls."""
        if self.workspace is None or self.workspace.numel() < nbytes:
            self.workspace = None
            self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        return self.workspace

    def close(self):
        if self.handle:
            self.workspace = None
            lib.e2f_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def e2f_create(lmax_max: int = 6, device: int | None = 0) -> Context:
    return Context(lmax_max, device)


def e2f_destroy(ctx: Context) -> None:
    ctx.close()


def e2f_node_tp_dim(lmax: int) -> int:
    return int(lib.e2f_node_tp_dim(lmax))


def e2f_real_cg(l1: int, l2: int, l3: int):
    import numpy as np
    out = np.zeros((2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1))
    _check(lib.e2f_real_cg(l1, l2, l3, out.ctypes.data_as(ctypes.c_void_p)), "e2f_real_cg")
    return out


def e2f_recoupling_weight(a: int, b: int, u: int, o: int, d: int) -> float:
    return float(lib.e2f_recoupling_weight(a, b, u, o, d))


def e2f_neighbor_list(ctx: Context, pos: torch.Tensor, cutoff: float, graph_id: torch.Tensor | None = None,
                      row_ptr: torch.Tensor | None = None, col_idx: torch.Tensor | None = None):
    """Radius graph as device CSR (row_ptr int64 [N+1], col_idx int32 [E]).

    With preallocated row_ptr/col_idx large enough, one library call; else a
    size query first."""
    _dev(pos, torch.float32, "pos")
    _dev(graph_id, torch.int32, "graph_id")
    n = pos.shape[0]
    E = ctypes.c_int64(0)
    if row_ptr is not None and col_idx is not None:
        _dev(row_ptr, torch.int64, "row_ptr")
        _dev(col_idx, torch.int32, "col_idx")
        st = _check(lib.e2f_neighbor_list(ctx.handle, _ptr(pos), _ptr(graph_id), n, cutoff, _ptr(row_ptr),
                                          _ptr(col_idx), col_idx.numel(), ctypes.byref(E), _stream(pos.device)),
                    "e2f_neighbor_list", allow=(E2F_ECAPACITY,))
        if st == E2F_OK:
            return row_ptr, col_idx[:E.value]
    row_ptr = torch.empty(n + 1, dtype=torch.int64, device=pos.device)
    _check(lib.e2f_neighbor_list(ctx.handle, _ptr(pos), _ptr(graph_id), n, cutoff, _ptr(row_ptr), None, 0,
                                 ctypes.byref(E), _stream(pos.device)), "e2f_neighbor_list", allow=(E2F_ECAPACITY,))
    col = torch.empty(max(E.value, 1), dtype=torch.int32, device=pos.device)
    _check(lib.e2f_neighbor_list(ctx.handle, _ptr(pos), _ptr(graph_id), n, cutoff, _ptr(row_ptr), _ptr(col),
                                 col.numel(), ctypes.byref(E), _stream(pos.device)), "e2f_neighbor_list")
    return row_ptr, col[:E.value]


def e2f_knn_graph(ctx: Context, pos: torch.Tensor, k: int, graph_id: torch.Tensor | None = None):
    """k-nearest-neighbour graph as device CSR (row_ptr int64 [N+1], col_idx int32 [E])."""
    _dev(pos, torch.float32, "pos")
    _dev(graph_id, torch.int32, "graph_id")
    n = pos.shape[0]
    E = ctypes.c_int64(0)
    row_ptr = torch.empty(n + 1, dtype=torch.int64, device=pos.device)
    _check(lib.e2f_knn_graph(ctx.handle, _ptr(pos), _ptr(graph_id), n, k, _ptr(row_ptr), None, 0, ctypes.byref(E),
                             _stream(pos.device)), "e2f_knn_graph", allow=(E2F_ECAPACITY,))
    col = torch.empty(max(E.value, 1), dtype=torch.int32, device=pos.device)
    _check(lib.e2f_knn_graph(ctx.handle, _ptr(pos), _ptr(graph_id), n, k, _ptr(row_ptr), _ptr(col), col.numel(),
                             ctypes.byref(E), _stream(pos.device)), "e2f_knn_graph")
    return row_ptr, col[:E.value]


def e2f_attention_weights(ctx: Context, pos, row_ptr, col_idx, cutoff: float, q=None, k=None, rbf_w=None,
                          heads: int | None = None, out=None):
    """Attention weights [E, heads] float32: q, k [N, heads, dk] (or None),
    rbf_w [heads, R] (or None)."""
    for t, name in ((pos, "pos"), (q, "q"), (k, "k"), (rbf_w, "rbf_w")):
        _dev(t, torch.float32, name)
    _dev(row_ptr, torch.int64, "row_ptr")
    _dev(col_idx, torch.int32, "col_idx")
    n = pos.shape[0]
    H = heads if heads is not None else (q.shape[1] if q is not None else rbf_w.shape[0])
    dk = 0 if q is None else q.shape[2]
    R = 0 if rbf_w is None else rbf_w.shape[1]
    E = col_idx.numel()
    if out is None:
        out = torch.empty(E, H, dtype=torch.float32, device=pos.device)
    _dev(out, torch.float32, "out")
    _check(lib.e2f_attention_weights(ctx.handle, _ptr(pos), _ptr(q), _ptr(k), n, H, dk, _ptr(rbf_w), R, cutoff,
                                     _ptr(row_ptr), _ptr(col_idx), E, _ptr(out), _stream(pos.device)),
           "e2f_attention_weights")
    return out


def e2f_solid_harmonics(ctx: Context, pos: torch.Tensor, lmax: int, origins: torch.Tensor | None = None,
                        origin_id: torch.Tensor | None = None) -> torch.Tensor:
    _dev(pos, torch.float32, "pos")
    _dev(origins, torch.float32, "origins")
    _dev(origin_id, torch.int32, "origin_id")
    out = torch.empty(pos.shape[0], (lmax + 1) ** 2, dtype=torch.float32, device=pos.device)
    _check(lib.e2f_solid_harmonics(ctx.handle, _ptr(pos), _ptr(origins), _ptr(origin_id), pos.shape[0], lmax,
                                   _ptr(out), _stream(pos.device)), "e2f_solid_harmonics")
    return out


def e2f_node_tp(ctx: Context, pos: torch.Tensor, feat: torch.Tensor, lmax: int, origins: torch.Tensor | None = None,
                origin_id: torch.Tensor | None = None) -> torch.Tensor:
    _dev(pos, torch.float32, "pos")
    _dev(feat, torch.float32, "feat")
    _dev(origins, torch.float32, "origins")
    _dev(origin_id, torch.int32, "origin_id")
    n, nk, C = feat.shape
    out = torch.empty(n, e2f_node_tp_dim(lmax), C, dtype=torch.float32, device=feat.device)
    _check(lib.e2f_node_tp(ctx.handle, _ptr(pos), _ptr(origins), _ptr(origin_id), _ptr(feat), n, C, lmax, _ptr(out),
                           _stream(feat.device)), "e2f_node_tp")
    return out


def e2f_aggregate(ctx: Context, T: torch.Tensor, row_ptr: torch.Tensor, col_idx: torch.Tensor,
                  alpha: torch.Tensor | None, out: torch.Tensor | None = None,
                  workspace: torch.Tensor | None = None, order: torch.Tensor | None = None) -> torch.Tensor:
    """The aggregation alone: S[i][h] = sum over row i's edges e = (i, j) of
    alpha[e][h] T[j][h] for T [n, heads, rows, C/heads] float32 (head-major);
    alpha [E, heads] or None (ones); order: int32 [n], the permutation whose
    consecutive receivers form the blocks (None: index order).  Returns S of
    T's shape.  (sync)"""
    _dev(T, torch.float32, "T")
    _dev(row_ptr, torch.int64, "row_ptr")
    _dev(col_idx, torch.int32, "col_idx")
    _dev(alpha, torch.float32, "alpha")
    _dev(order, torch.int32, "order")
    if T.dim() != 4:
        raise ValueError("T must be [n, heads, rows, C/heads]")
    n, H, K, dh = T.shape
    E = col_idx.numel()
    if out is None:
        out = torch.empty_like(T)
    _dev(out, torch.float32, "out")
    if workspace is None:
        b = ctypes.c_size_t(0)
        _check(lib.e2f_aggregate_workspace_size(ctx.handle, n, E, H, ctypes.byref(b)), "e2f_aggregate_workspace_size")
        workspace = ctx.workspace_for(b.value, T.device)
    elif not workspace.is_cuda or workspace.dtype != torch.uint8 or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 device tensor")
    _check(lib.e2f_aggregate(ctx.handle, _ptr(T), n, K, H * dh, H, _ptr(row_ptr), _ptr(col_idx), E, _ptr(alpha),
                             _ptr(order), _ptr(out), _ptr(workspace), workspace.numel(), _stream(T.device)),
           "e2f_aggregate")
    return out


def _params(lmax, channels, heads, cutoff, path_w, mix_w, tile_side, y_norm=False, form="auto"):
    import numpy as np
    keep = None
    pw = None
    if path_w is not None:
        keep = np.ascontiguousarray(path_w, dtype=np.float64)
        if keep.size != (lmax + 1) ** 3:
            raise ValueError("path_w must have (lmax+1)^3 entries")
        pw = keep.ctypes.data_as(ctypes.c_void_p)
    mix_dtype = E2F_F32
    if mix_w is not None:
        if mix_w.dtype == torch.bfloat16:
            mix_dtype = E2F_BF16
        else:
            _dev(mix_w, torch.float32, "mix_w")
        if not mix_w.is_cuda or not mix_w.is_contiguous():
            raise ValueError("mix_w must be a contiguous device tensor")
    prm = ConvParams(lmax, channels, heads, cutoff, pw, None if mix_w is None else mix_w.data_ptr(), mix_dtype,
                     float(tile_side), int(bool(y_norm)), _FORMS[form] if isinstance(form, str) else int(form))
    return prm, keep


def _conv_args(pos, feat, row_ptr, col_idx, alpha, graph_id, out):
    _dev(pos, torch.float32, "pos")
    _dev(feat, torch.float32, "feat")
    _dev(row_ptr, torch.int64, "row_ptr")
    _dev(col_idx, torch.int32, "col_idx")
    _dev(alpha, torch.float32, "alpha")
    _dev(graph_id, torch.int32, "graph_id")
    if out is None:
        out = torch.empty_like(feat)
    _dev(out, torch.float32, "out")
    return out


def e2f_wigner6j_workspace_size(ctx, n, n_edges, lmax, channels, heads, cutoff, path_w=None, mix_w=None,
                                tile_side=0.0, y_norm=False, minimum=False, form="auto") -> int:
    """Workspace bytes of the forward (the one-pass size, or with minimum=True
    the smallest size it accepts)."""
    prm, keep = _params(lmax, channels, heads, cutoff, path_w, mix_w, tile_side, y_norm, form)
    b = ctypes.c_size_t(0)
    fn = lib.e2f_wigner6j_workspace_min if minimum else lib.e2f_wigner6j_workspace_size
    _check(fn(ctx.handle, ctypes.byref(prm), n, n_edges, ctypes.byref(b)),
           "e2f_wigner6j_workspace_min" if minimum else "e2f_wigner6j_workspace_size")
    del keep
    return b.value


def e2f_wigner6j_prepare(ctx, lmax, channels, heads, cutoff, path_w=None, mix_w=None, tile_side=0.0,
                         y_norm=False, form="auto") -> None:
    """Upload the coefficient set and coupling schedule these parameters use."""
    prm, keep = _params(lmax, channels, heads, cutoff, path_w, mix_w, tile_side, y_norm, form)
    _check(lib.e2f_wigner6j_prepare(ctx.handle, ctypes.byref(prm)), "e2f_wigner6j_prepare")
    del keep


def e2f_wigner6j_conv_forward(ctx, pos, feat, row_ptr, col_idx, alpha, lmax, heads, cutoff, path_w=None, mix_w=None,
                              graph_id=None, tile_side=0.0, out=None, y_norm=False, workspace=None,
                              form="auto"):
    """Wigner-6j convolution forward; returns out [N,(L+1)^2,C] float32.
    y_norm: attention weights alpha / |r_i - r_j|^f per filter degree f.
    workspace: a uint8 device tensor (any size from the minimum up); None
    uses the context's own, grown to the one-pass size.
    form: "auto", "split" (S written, then recoupled by a second kernel) or
    "fused" (the aggregation applies the recouple itself where it can)."""
    out = _conv_args(pos, feat, row_ptr, col_idx, alpha, graph_id, out)
    n, nk, C = feat.shape
    E = col_idx.numel()
    prm, keep = _params(lmax, C, heads, cutoff, path_w, mix_w, tile_side, y_norm, form)
    if workspace is None:
        b = ctypes.c_size_t(0)
        _check(lib.e2f_wigner6j_workspace_size(ctx.handle, ctypes.byref(prm), n, E, ctypes.byref(b)),
               "e2f_wigner6j_workspace_size")
        workspace = ctx.workspace_for(b.value, feat.device)
    elif not workspace.is_cuda or workspace.dtype != torch.uint8 or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 device tensor")
    st = lib.e2f_wigner6j_conv_forward(ctx.handle, ctypes.byref(prm), _ptr(pos), _ptr(graph_id), _ptr(feat), n,
                                       _ptr(row_ptr), _ptr(col_idx), E, _ptr(alpha), _ptr(out), _ptr(workspace),
                                       workspace.numel(), _stream(feat.device))
    del keep
    _check(st, "e2f_wigner6j_conv_forward")
    return out


def e2f_wigner6j_conv_forward_noalloc(ctx, pos, feat, row_ptr, col_idx, alpha, lmax, heads, cutoff, path_w=None,
                                      mix_w=None, graph_id=None, tile_side=0.0, out=None, y_norm=False,
                                      form="auto"):
    """The forward in the library's per-GPU scratch memory (no allocation;
    the parameters must have been prepared).  out must be given by callers
    that cannot allocate: with out=None the binding allocates it."""
    out = _conv_args(pos, feat, row_ptr, col_idx, alpha, graph_id, out)
    n, nk, C = feat.shape
    prm, keep = _params(lmax, C, heads, cutoff, path_w, mix_w, tile_side, y_norm, form)
    st = lib.e2f_wigner6j_conv_forward_noalloc(ctx.handle, ctypes.byref(prm), _ptr(pos), _ptr(graph_id), _ptr(feat),
                                               n, _ptr(row_ptr), _ptr(col_idx), col_idx.numel(), _ptr(alpha),
                                               _ptr(out), _stream(feat.device))
    del keep
    _check(st, "e2f_wigner6j_conv_forward_noalloc")
    return out


def e2f_edge_tp_conv_forward(ctx, pos, feat, row_ptr, col_idx, alpha, lmax, heads, cutoff, path_w=None, mix_w=None,
                             graph_id=None, tile_side=0.0, out=None, y_norm=False):
    """Per-edge SO(3) convolution baseline; same output as the 6j forward."""
    out = _conv_args(pos, feat, row_ptr, col_idx, alpha, graph_id, out)
    n, nk, C = feat.shape
    prm, keep = _params(lmax, C, heads, cutoff, path_w, mix_w, tile_side, y_norm)
    st = lib.e2f_edge_tp_conv_forward(ctx.handle, ctypes.byref(prm), _ptr(pos), _ptr(graph_id), _ptr(feat), n,
                                      _ptr(row_ptr), _ptr(col_idx), col_idx.numel(), _ptr(alpha), _ptr(out),
                                      _stream(feat.device))
    del keep
    _check(st, "e2f_edge_tp_conv_forward")
    return out


def e2f_validate_graph(ctx, n, row_ptr, col_idx) -> int:
    """0 if the device CSR is well formed, else the error bits of e2f.h."""
    _dev(row_ptr, torch.int64, "row_ptr")
    _dev(col_idx, torch.int32, "col_idx")
    bad = ctypes.c_int32(0)
    _check(lib.e2f_validate_graph(ctx.handle, n, _ptr(row_ptr), _ptr(col_idx), col_idx.numel(), ctypes.byref(bad),
                                  _stream(row_ptr.device)), "e2f_validate_graph")
    return bad.value


def e2f_wigner6j_conv_forward_dense(ctx, pos, feat, alpha, lmax, heads, cutoff, path_w=None, mix_w=None, out=None):
    """Dense-graph forward (every atom attends to every other): alpha [N,N,H]
    float32 (receiver, sender, head) or None; returns out [N,(L+1)^2,C]."""
    _dev(pos, torch.float32, "pos")
    _dev(feat, torch.float32, "feat")
    _dev(alpha, torch.float32, "alpha")
    n, nk, C = feat.shape
    if alpha is not None and tuple(alpha.shape) != (n, n, heads):
        raise ValueError("alpha must be [N, N, heads]")
    if out is None:
        out = torch.empty_like(feat)
    _dev(out, torch.float32, "out")
    prm, keep = _params(lmax, C, heads, cutoff, path_w, mix_w, 0.0)
    st = lib.e2f_wigner6j_conv_forward_dense(ctx.handle, ctypes.byref(prm), _ptr(pos), _ptr(feat), n, _ptr(alpha),
                                             _ptr(out), _stream(feat.device))
    del keep
    _check(st, "e2f_wigner6j_conv_forward_dense")
    return out


def e2f_wigner6j_conv_forward_global(ctx, pos, feat, lmax, heads, cutoff, path_w=None, mix_w=None, out=None):
    """Uniform attention over the whole graph (alpha = 1 for every pair, self
    included), in O(N) through the global moments; returns out [N,(L+1)^2,C]."""
    _dev(pos, torch.float32, "pos")
    _dev(feat, torch.float32, "feat")
    n, nk, C = feat.shape
    if out is None:
        out = torch.empty_like(feat)
    _dev(out, torch.float32, "out")
    prm, keep = _params(lmax, C, heads, cutoff, path_w, mix_w, 0.0)
    st = lib.e2f_wigner6j_conv_forward_global(ctx.handle, ctypes.byref(prm), _ptr(pos), _ptr(feat), n, _ptr(out),
                                              _stream(feat.device))
    del keep
    _check(st, "e2f_wigner6j_conv_forward_global")
    return out


def e2f_wigner6j_conv_backward(ctx, pos, feat, grad_out, row_ptr, col_idx, alpha, lmax, heads, cutoff, path_w=None,
                               mix_w=None, graph_id=None, tile_side=0.0, want_feat=True, want_alpha=True,
                               want_pos=False):
    """Vector-Jacobian products of the forward: (grad_feat [N,(L+1)^2,C],
    grad_alpha [E,H], grad_pos [N,3]), each None unless requested."""
    for t, name in ((pos, "pos"), (feat, "feat"), (grad_out, "grad_out"), (alpha, "alpha")):
        _dev(t, torch.float32, name)
    _dev(row_ptr, torch.int64, "row_ptr")
    _dev(col_idx, torch.int32, "col_idx")
    _dev(graph_id, torch.int32, "graph_id")
    n, nk, C = grad_out.shape
    E = col_idx.numel()
    gf = torch.empty_like(grad_out) if want_feat else None
    ga = torch.empty(E, heads, dtype=torch.float32, device=grad_out.device) if want_alpha else None
    gp = torch.empty(n, 3, dtype=torch.float32, device=grad_out.device) if want_pos else None
    prm, keep = _params(lmax, C, heads, cutoff, path_w, mix_w, tile_side)
    st = lib.e2f_wigner6j_conv_backward(ctx.handle, ctypes.byref(prm), _ptr(pos), _ptr(graph_id), _ptr(feat),
                                        _ptr(grad_out), n, _ptr(row_ptr), _ptr(col_idx), E, _ptr(alpha), _ptr(gf),
                                        _ptr(ga), _ptr(gp), _stream(grad_out.device))
    del keep
    _check(st, "e2f_wigner6j_conv_backward")
    return gf, ga, gp


def e2f_profile(ctx: Context, enable: bool) -> None:
    """Start (clearing earlier records) or stop event timing of every launch group."""
    _check(lib.e2f_profile(ctx.handle, 1 if enable else 0), "e2f_profile")


def e2f_profile_read(ctx: Context) -> dict:
    """{step name: (launch groups, total ms)} recorded since e2f_profile(ctx, True)."""
    buf = ctypes.create_string_buffer(1 << 16)
    _check(lib.e2f_profile_read(ctx.handle, buf, len(buf)), "e2f_profile_read")
    out = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.split()
        out[name] = (int(cnt), float(ms))
    return out


def e2f_last_slices(ctx: Context) -> int:
    """Receiver slices of the last factorised forward on this context."""
    v = ctypes.c_int64(0)
    _check(lib.e2f_last_slices(ctx.handle, ctypes.byref(v)), "e2f_last_slices")
    return v.value
