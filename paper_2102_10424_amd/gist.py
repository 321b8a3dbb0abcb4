"""ctypes binding of ``libgist.so`` (the C ABI declared in ``include/gist.h``).

Argument marshalling only: every function here forwards to the entry point
of the same name.  Device buffers are torch tensors (PyTorch supplies device
memory and the current HIP stream); host buffers are NumPy arrays.  Errors
raise :class:`GistError` carrying the library's status and message.

The library must be built (``python -m paper_2102_10424_amd.build``); if it
is missing this module raises on import rather than falling back to any
other implementation.
"""

import ctypes as C
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgist.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"libgist.so not found at {LIB_PATH}: build it with "
        "`python -m paper_2102_10424_amd.build` (hipcc, gfx950)")

# Device memory and streams come from PyTorch, so the library must run on
# PyTorch's HIP runtime: importing torch first makes the dynamic loader bind
# libgist's libamdhip64.so.7 to that already-loaded copy instead of loading a
# second runtime that owns none of torch's allocations.
import torch  # noqa: E402,F401  (load order matters, see above)

_lib = C.CDLL(LIB_PATH)

# ---- enums / flags (mirror include/gist.h) ---------------------------------
GIST_OK = 0
GIST_E_INVAL = -1
GIST_E_NOMEM = -2
GIST_E_DEVICE = -3
GIST_E_UNSUPPORTED = -4
GIST_E_NONFINITE = -5

GIST_PART_CATEGORICAL = 1
GIST_NORM_GCN_SYM, GIST_NORM_SAGE_MEAN, GIST_NORM_THEORY = 0, 1, 2
GIST_LAYER_GCN, GIST_LAYER_SAGE_MEAN = 0, 1
GIST_ACT_NONE, GIST_ACT_RELU = 0, 1
GIST_DTYPE_F32, GIST_DTYPE_BF16_IN = 0, 1
GIST_ORDER_AUTO, GIST_ORDER_AGG_FIRST, GIST_ORDER_XFORM_FIRST = 0, 1, 2
GIST_SUBAGG_CHECK_FINITE = 1
GIST_ADAM_FRESH = 1
GIST_NOALLOC_LOSS_MAX_ROWS = 4194304
GIST_LAYER_SHARED_INPUT, GIST_LAYER_GROUP_MAJOR_OUT, GIST_LAYER_CLUSTERED = 1, 2, 4
GIST_LAYER_DZ_IN, GIST_LAYER_MASK_DH = 8, 16

NORM_BY_NAME = {"gcn": GIST_NORM_GCN_SYM, "sage": GIST_NORM_SAGE_MEAN,
                "theory": GIST_NORM_THEORY}

# Every symbol include/gist.h declares.
EXPORTED = (
    "gist_last_error", "gist_status_str", "gist_create", "gist_destroy",
    "gist_set_stream", "gist_partition", "gist_build_minibatch_csr", "gist_ladies_sample",
    "gist_layer_workspace_size", "gist_gcn_layer_fwd", "gist_gcn_layer_bwd",
    "gist_gcn_layer_bwd_sgd",
    "gist_gat_workspace_size", "gist_gat_layer_fwd", "gist_gat_layer_bwd", "gist_gat_scores",
    "gist_softmax_xent_workspace", "gist_softmax_xent", "gist_softmax_xent_padded",
    "gist_softmax_xent_noalloc",
    "gist_gather_slice",
    "gist_sgd_update", "gist_adam_update", "gist_adam_coefficients", "gist_adam_update_dev",
    "gist_subagg", "gist_partition_inverse",
    "gist_subagg_gather", "gist_subagg_mean",
    "gist_profile_begin", "gist_profile_read", "gist_profile_end",
    "gist_capture_begin", "gist_capture_end", "gist_replay_launch", "gist_replay_destroy",
    "gist_copy",
    "gist_event_create", "gist_event_synchronize", "gist_event_destroy",
)


class GistError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{status_str(status)}: {msg}")
        self.status = status


# ---- structures --------------------------------------------------------------
class gist_graph(C.Structure):
    _fields_ = [("n", C.c_int64), ("rowptr", C.c_void_p), ("col", C.c_void_p),
                ("n_clusters", C.c_int32), ("cluster_ptr", C.c_void_p),
                ("cluster_nodes", C.c_void_p)]


class gist_csr(C.Structure):
    _fields_ = [("n", C.c_int64), ("nnz", C.c_int64), ("cap_n", C.c_int64),
                ("cap_nnz", C.c_int64), ("rowptr", C.c_void_p), ("col", C.c_void_p),
                ("val", C.c_void_p), ("node_map", C.c_void_p),
                ("t_rowptr", C.c_void_p), ("t_col", C.c_void_p), ("t_val", C.c_void_p)]


class gist_csr_dev(C.Structure):
    _fields_ = [("n", C.c_int64), ("nnz", C.c_int64), ("rowptr", C.c_void_p),
                ("col", C.c_void_p), ("val", C.c_void_p)]


class gist_layer_desc(C.Structure):
    _fields_ = [("kind", C.c_int32), ("act", C.c_int32), ("dtype", C.c_int32),
                ("order", C.c_int32), ("n", C.c_int64), ("s_in", C.c_int32),
                ("s_out", C.c_int32), ("groups", C.c_int32), ("flags", C.c_uint32),
                ("n_in", C.c_int64)]


class gist_ladies_layer(C.Structure):
    _fields_ = [("n_out", C.c_int64), ("n_in", C.c_int64), ("nnz", C.c_int64),
                ("cap_n", C.c_int64), ("cap_nnz", C.c_int64), ("nodes", C.c_void_p),
                ("rowptr", C.c_void_p), ("col", C.c_void_p), ("val", C.c_void_p),
                ("t_rowptr", C.c_void_p), ("t_col", C.c_void_p), ("t_val", C.c_void_p)]


class gist_gat_desc(C.Structure):
    _fields_ = [("n", C.c_int64), ("nnz", C.c_int64), ("s_in", C.c_int32), ("s_out", C.c_int32),
                ("act", C.c_int32), ("dtype", C.c_int32), ("slope", C.c_float),
                ("flags", C.c_uint32)]


class gist_slice_set(C.Structure):
    _fields_ = [("row_rank", C.c_void_p), ("row_offs", C.c_void_p), ("col_rank", C.c_void_p),
                ("col_offs", C.c_void_p), ("slices", C.c_void_p), ("ld", C.c_int64)]


class gist_prof_entry(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("launches", C.c_int64), ("ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


_P = C.c_void_p
_sigs = {
    "gist_profile_begin": (C.c_int, [_P, C.c_int64]),
    "gist_profile_read": (C.c_int, [_P, C.POINTER(gist_prof_entry), C.c_int32,
                                    C.POINTER(C.c_int32), C.POINTER(C.c_int64)]),
    "gist_profile_end": (C.c_int, [_P]),
    "gist_partition_inverse": (C.c_int, [C.c_int64, C.c_int32, _P, _P, _P]),
    "gist_adam_update": (C.c_int, [_P, _P, _P, _P, _P, C.c_int64, C.c_float, C.c_float, C.c_float,
                                   C.c_float, C.c_int64, C.c_uint32]),
    "gist_adam_coefficients": (C.c_int, [C.c_float, C.c_float, C.c_float, C.c_float, C.c_int64,
                                         C.c_uint32, _P]),
    "gist_adam_update_dev": (C.c_int, [_P, _P, _P, _P, _P, C.c_int64, C.c_float, C.c_float,
                                       C.c_float, _P]),
    "gist_subagg_gather": (C.c_int, [_P, _P, C.c_int64, C.c_int64, C.c_int64, C.c_int32,
                                     C.POINTER(gist_slice_set), C.POINTER(gist_slice_set)]),
    "gist_subagg_mean": (C.c_int, [_P, _P, C.c_int64, C.c_int64, C.c_int64, C.c_int32, _P,
                                   C.c_int64]),
    "gist_gat_workspace_size": (C.c_int, [C.POINTER(gist_gat_desc), C.POINTER(C.c_size_t),
                                          C.POINTER(C.c_size_t)]),
    "gist_gat_layer_fwd": (C.c_int, [_P, C.POINTER(gist_gat_desc), C.POINTER(gist_csr_dev)] +
                           [_P] * 8 + [C.c_size_t]),
    "gist_gat_layer_bwd": (C.c_int, [_P, C.POINTER(gist_gat_desc), C.POINTER(gist_csr_dev)] +
                           [_P] * 13 + [C.c_size_t]),
    "gist_gat_scores": (C.c_int, [_P, C.c_int64, C.c_int32, _P, C.c_int64, _P, _P, _P, _P]),
    "gist_last_error": (C.c_char_p, []),
    "gist_status_str": (C.c_char_p, [C.c_int]),
    "gist_create": (C.c_int, [C.c_int, _P, C.POINTER(_P)]),
    "gist_destroy": (C.c_int, [_P]),
    "gist_set_stream": (C.c_int, [_P, _P]),
    "gist_partition": (C.c_int, [C.c_int64, C.c_int32, C.c_uint64, C.c_uint32, _P, _P]),
    "gist_build_minibatch_csr": (C.c_int, [C.POINTER(gist_graph), _P, C.c_int32, C.c_int,
                                           C.POINTER(gist_csr)]),
    "gist_ladies_sample": (C.c_int, [C.POINTER(gist_csr), _P, C.c_int64, C.c_int32, C.c_int32,
                                     C.c_uint64, C.POINTER(gist_ladies_layer)]),
    "gist_layer_workspace_size": (C.c_int, [C.POINTER(gist_layer_desc),
                                            C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "gist_gcn_layer_fwd": (C.c_int, [_P, C.POINTER(gist_layer_desc), C.POINTER(gist_csr_dev),
                                     _P, _P, _P, _P, _P, C.c_size_t]),
    "gist_gcn_layer_bwd": (C.c_int, [_P, C.POINTER(gist_layer_desc), C.POINTER(gist_csr_dev),
                                     C.POINTER(gist_csr_dev), _P, _P, _P, _P, _P, _P, _P, _P,
                                     C.c_size_t]),
    "gist_gcn_layer_bwd_sgd": (C.c_int, [_P, C.POINTER(gist_layer_desc),
                                         C.POINTER(gist_csr_dev), C.POINTER(gist_csr_dev),
                                         _P, _P, _P, _P, _P, C.c_float, _P, _P, C.c_size_t]),
    "gist_softmax_xent_workspace": (C.c_size_t, [C.c_int64]),
    "gist_softmax_xent": (C.c_int, [_P, C.c_int64, C.c_int32, _P, _P, _P, _P, _P, C.c_size_t]),
    "gist_softmax_xent_padded": (C.c_int, [_P, C.c_int64, C.c_int32, _P, _P, _P, _P, _P, _P,
                                           C.c_size_t]),
    "gist_softmax_xent_noalloc": (C.c_int, [_P, C.c_int64, C.c_int32, _P, _P, _P, _P]),
    "gist_gather_slice": (C.c_int, [_P, _P, C.c_int64, _P, C.c_int32, _P, C.c_int32, _P,
                                    C.c_int64]),
    "gist_sgd_update": (C.c_int, [_P, _P, _P, C.c_int64, C.c_float]),
    "gist_subagg": (C.c_int, [_P, _P, C.c_int64, _P, C.c_int32, _P, C.c_int32, _P, C.c_int64,
                              C.c_uint32]),
    "gist_capture_begin": (C.c_int, [_P]),
    "gist_capture_end": (C.c_int, [_P, C.POINTER(_P)]),
    "gist_replay_launch": (C.c_int, [_P, _P, _P, _P, C.c_size_t, _P]),
    "gist_replay_destroy": (C.c_int, [_P]),
    "gist_copy": (C.c_int, [_P, _P, _P, C.c_size_t, _P]),
    "gist_event_create": (C.c_int, [C.POINTER(_P)]),
    "gist_event_synchronize": (C.c_int, [_P]),
    "gist_event_destroy": (C.c_int, [_P]),
}
for _name, (_res, _args) in _sigs.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def status_str(s):
    return _lib.gist_status_str(int(s)).decode()


def _check(status):
    if status != GIST_OK:
        raise GistError(status, _lib.gist_last_error().decode())


def _ptr(x):
    """Address of a torch tensor / NumPy array (None -> NULL)."""
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError("host array must be C-contiguous")
        return x.ctypes.data
    return x.data_ptr()


# ---- context -----------------------------------------------------------------
class Context:
    """A ``gist_ctx`` bound to a device and (by default) torch's current stream."""

    def __init__(self, device=0, stream=None):
        import torch
        if stream is None:
            stream = torch.cuda.current_stream(device).cuda_stream
        h = _P()
        _check(_lib.gist_create(int(device), _P(stream), C.byref(h)))
        self.handle = h
        self.device = device

    def set_stream(self, stream):
        _check(_lib.gist_set_stream(self.handle, _P(stream)))

    def close(self):
        if self.handle:
            _lib.gist_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---- host calls ----------------------------------------------------------------
def gist_partition(d, m, seed, flags=0):
    """Returns (idx int32[d], offs int64[m+1])."""
    idx = np.empty(max(int(d), 1), dtype=np.int32)
    offs = np.empty(max(int(m), 0) + 1, dtype=np.int64)
    _check(_lib.gist_partition(int(d), int(m), int(seed) & (2**64 - 1), int(flags),
                               _ptr(idx), _ptr(offs)))
    return idx[:int(d)], offs


def gist_partition_inverse(idx, offs):
    """rank int32[d] with rank[idx[k]] = k."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    offs = np.ascontiguousarray(offs, dtype=np.int64)
    d, m = idx.shape[0], offs.shape[0] - 1
    rank = np.empty(d, dtype=np.int32)
    _check(_lib.gist_partition_inverse(d, m, _ptr(idx), _ptr(offs), _ptr(rank)))
    return rank


def _graph_struct(graph):
    keep = dict(rowptr=np.ascontiguousarray(graph.rowptr, dtype=np.int64),
                col=np.ascontiguousarray(graph.col, dtype=np.int32),
                cptr=np.ascontiguousarray(graph.cluster_ptr, dtype=np.int64),
                cnodes=np.ascontiguousarray(graph.cluster_nodes, dtype=np.int32))
    g = gist_graph(int(graph.n), _ptr(keep["rowptr"]), _ptr(keep["col"]),
                   int(keep["cptr"].shape[0] - 1), _ptr(keep["cptr"]), _ptr(keep["cnodes"]))
    return g, keep


def gist_build_minibatch_csr(graph, clusters, norm):
    """Mini-batch CSR of the union of ``clusters`` (None: full graph) as NumPy arrays."""
    norm_id = NORM_BY_NAME[norm] if isinstance(norm, str) else int(norm)
    g, keep = _graph_struct(graph)
    if clusters is None:
        sel, nsel = None, -1
    else:
        sel = np.ascontiguousarray(clusters, dtype=np.int32)
        nsel = int(sel.shape[0])
    q = gist_csr()
    _check(_lib.gist_build_minibatch_csr(C.byref(g), _ptr(sel), nsel, norm_id, C.byref(q)))
    n, nnz = int(q.n), int(q.nnz)
    out = dict(n=n, nnz=nnz,
               rowptr=np.empty(n + 1, dtype=np.int32), col=np.empty(max(nnz, 1), dtype=np.int32),
               val=np.empty(max(nnz, 1), dtype=np.float32),
               node_map=np.empty(max(n, 1), dtype=np.int32))
    sage = norm_id == GIST_NORM_SAGE_MEAN
    if sage:
        out.update(t_rowptr=np.empty(n + 1, dtype=np.int32),
                   t_col=np.empty(max(nnz, 1), dtype=np.int32),
                   t_val=np.empty(max(nnz, 1), dtype=np.float32))
    q.cap_n, q.cap_nnz = n, nnz
    q.rowptr, q.col, q.val = _ptr(out["rowptr"]), _ptr(out["col"]), _ptr(out["val"])
    q.node_map = _ptr(out["node_map"])
    if sage:
        q.t_rowptr, q.t_col, q.t_val = (_ptr(out["t_rowptr"]), _ptr(out["t_col"]),
                                        _ptr(out["t_val"]))
    _check(_lib.gist_build_minibatch_csr(C.byref(g), _ptr(sel), nsel, norm_id, C.byref(q)))
    for k in ("col", "val", "t_col", "t_val"):
        if k in out:
            out[k] = out[k][:nnz]
    out["node_map"] = out["node_map"][:n]
    return out


class CsrHandle:
    """A host ``gist_csr`` over NumPy arrays kept alive with it (the full-graph
    matrix that ``gist_ladies_sample`` samples from)."""

    def __init__(self, csr):
        self._keep = dict(rowptr=np.ascontiguousarray(csr["rowptr"], dtype=np.int32),
                          col=np.ascontiguousarray(csr["col"], dtype=np.int32),
                          val=np.ascontiguousarray(csr["val"], dtype=np.float32))
        n, nnz = int(csr["n"]), int(csr["nnz"])
        self.struct = gist_csr(n, nnz, n, nnz, _ptr(self._keep["rowptr"]), _ptr(self._keep["col"]),
                               _ptr(self._keep["val"]), None, None, None, None)
        self.n, self.nnz = n, nnz


_LADIES_ARRAYS = (("nodes", np.int32, "n"), ("rowptr", np.int32, "n1"), ("col", np.int32, "z"),
                  ("val", np.float32, "z"), ("t_rowptr", np.int32, "n1"),
                  ("t_col", np.int32, "z"), ("t_val", np.float32, "z"))


def ladies_layers(L, caps=None):
    """An array of L ``gist_ladies_layer`` s; with ``caps`` = [(cap_n, cap_nnz)] * L
    each gets NumPy buffers of those capacities (returned alongside)."""
    arr = (gist_ladies_layer * L)()
    bufs = []
    for l in range(L):
        if caps is None:
            bufs.append(None)
            continue
        cn, cz = int(caps[l][0]), int(caps[l][1])
        size = dict(n=max(cn, 1), n1=cn + 1, z=max(cz, 1))
        b = {k: np.empty(size[w], dtype=t) for k, t, w in _LADIES_ARRAYS}
        arr[l].cap_n, arr[l].cap_nnz = cn, cz
        for k, _, _ in _LADIES_ARRAYS:
            setattr(arr[l], k, _ptr(b[k]))
        bufs.append(b)
    return arr, bufs


def ladies_sample_into(A_handle, batch, L, s, seed, arr):
    """``gist_ladies_sample`` into the layer descriptors ``arr`` (host buffers)."""
    batch = np.ascontiguousarray(batch, dtype=np.int32)
    _check(_lib.gist_ladies_sample(C.byref(A_handle.struct), _ptr(batch), int(batch.shape[0]),
                                   int(L), int(s), int(seed) & (2**64 - 1), arr))
    return arr


def gist_ladies_sample(A, batch, L, s, seed):
    """LADIES mini-batch as NumPy arrays: dict(nodes=[V_0..V_L], layers=[dict per layer]).

    ``A``: the full-graph GCN CSR (dict or :class:`CsrHandle`)."""
    h = A if isinstance(A, CsrHandle) else CsrHandle(A)
    q, _ = ladies_layers(L)
    ladies_sample_into(h, batch, L, s, seed, q)      # size query
    arr, bufs = ladies_layers(L, [(q[l].n_in, q[l].nnz) for l in range(L)])
    ladies_sample_into(h, batch, L, s, seed, arr)
    layers, nodes = [], []
    for l in range(L):
        d, b = arr[l], bufs[l]
        n_out, n_in, nnz = int(d.n_out), int(d.n_in), int(d.nnz)
        layers.append(dict(n=n_out, n_in=n_in, nnz=nnz, rowptr=b["rowptr"][:n_out + 1],
                           col=b["col"][:nnz], val=b["val"][:nnz],
                           t_rowptr=b["t_rowptr"][:n_in + 1], t_col=b["t_col"][:nnz],
                           t_val=b["t_val"][:nnz]))
        nodes.append(b["nodes"][:n_in])
    nodes.append(np.ascontiguousarray(batch, dtype=np.int32))
    return dict(nodes=nodes, layers=layers)


class GraphHandle:
    """A ``gist_graph`` over NumPy arrays kept alive with it (build once, reuse)."""

    def __init__(self, graph):
        self.struct, self._keep = _graph_struct(graph)


def build_minibatch_into(graph_handle, clusters, norm, q):
    """``gist_build_minibatch_csr`` into caller-provided buffers described by ``q``."""
    norm_id = NORM_BY_NAME[norm] if isinstance(norm, str) else int(norm)
    if clusters is None:
        sel, nsel = None, -1
    else:
        sel = np.ascontiguousarray(clusters, dtype=np.int32)
        nsel = int(sel.shape[0])
    _check(_lib.gist_build_minibatch_csr(C.byref(graph_handle.struct), _ptr(sel), nsel,
                                         norm_id, C.byref(q)))
    return q


# ---- device calls --------------------------------------------------------------
def csr_dev(n, nnz, rowptr, col, val):
    """A ``gist_csr_dev`` over torch device tensors (the tensors must outlive it)."""
    return gist_csr_dev(int(n), int(nnz), _ptr(rowptr), _ptr(col), _ptr(val))


def layer_desc(kind, act, n, s_in, s_out, dtype=GIST_DTYPE_F32, order=GIST_ORDER_AUTO,
               groups=1, flags=0, n_in=0):
    """``n_in``: input rows of a rectangular (layer-sampled) GCN layer; 0 means n."""
    return gist_layer_desc(int(kind), int(act), int(dtype), int(order), int(n), int(s_in),
                           int(s_out), int(groups), int(flags), int(n_in))


def gist_layer_workspace_size(desc):
    f, b = C.c_size_t(), C.c_size_t()
    _check(_lib.gist_layer_workspace_size(C.byref(desc), C.byref(f), C.byref(b)))
    return int(f.value), int(b.value)


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def gist_gcn_layer_fwd(ctx, desc, A, H, W, agg_save, H_out, ws):
    _check(_lib.gist_gcn_layer_fwd(ctx.handle, C.byref(desc), C.byref(A), _ptr(H), _ptr(W),
                                   _ptr(agg_save), _ptr(H_out), _ptr(ws), _nbytes(ws)))


def gist_gcn_layer_bwd(ctx, desc, A, A_T, H, agg_save, H_out, W, dH_out, dW, dH, ws):
    _check(_lib.gist_gcn_layer_bwd(ctx.handle, C.byref(desc), C.byref(A),
                                   C.byref(A_T) if A_T is not None else None, _ptr(H),
                                   _ptr(agg_save), _ptr(H_out), _ptr(W), _ptr(dH_out),
                                   _ptr(dW), _ptr(dH), _ptr(ws), _nbytes(ws)))


def gist_gcn_layer_bwd_sgd(ctx, desc, A, A_T, H, agg_save, H_out, W, dH_out, lr, dH, ws):
    """Backward pass with the SGD step fused: W <- W - lr dW in place, no dW."""
    _check(_lib.gist_gcn_layer_bwd_sgd(ctx.handle, C.byref(desc), C.byref(A),
                                       C.byref(A_T) if A_T is not None else None, _ptr(H),
                                       _ptr(agg_save), _ptr(H_out), _ptr(W), _ptr(dH_out),
                                       float(lr), _ptr(dH), _ptr(ws), _nbytes(ws)))


def gist_softmax_xent_workspace(n):
    return int(_lib.gist_softmax_xent_workspace(int(n)))


def gist_softmax_xent(ctx, n, C_, logits, labels, loss_dev, dlogits, ws):
    _check(_lib.gist_softmax_xent(ctx.handle, int(n), int(C_), _ptr(logits), _ptr(labels),
                                  _ptr(loss_dev), _ptr(dlogits), _ptr(ws), _nbytes(ws)))


def gist_softmax_xent_padded(ctx, n, C_, logits, labels, n_valid_dev, loss_dev, dlogits, ws):
    """Loss over a batch padded to n rows; the real row count is the device int32
    ``n_valid_dev``."""
    _check(_lib.gist_softmax_xent_padded(ctx.handle, int(n), int(C_), _ptr(logits), _ptr(labels),
                                         _ptr(n_valid_dev), _ptr(loss_dev), _ptr(dlogits),
                                         _ptr(ws), _nbytes(ws)))


def gist_softmax_xent_noalloc(ctx, n, C_, logits, labels, loss_dev, dlogits):
    _check(_lib.gist_softmax_xent_noalloc(ctx.handle, int(n), int(C_), _ptr(logits), _ptr(labels),
                                          _ptr(loss_dev), _ptr(dlogits)))


def gist_gather_slice(ctx, Wg, ldg, rows, nr, cols, nc, Ws, lds):
    _check(_lib.gist_gather_slice(ctx.handle, _ptr(Wg), int(ldg), _ptr(rows), int(nr),
                                  _ptr(cols), int(nc), _ptr(Ws), int(lds)))


def gist_sgd_update(ctx, W, dW, n, lr):
    _check(_lib.gist_sgd_update(ctx.handle, _ptr(W), _ptr(dW), int(n), float(lr)))


def gist_adam_update(ctx, W, dW, m, v, n, lr, step, beta1=0.9, beta2=0.999, eps=1e-8,
                     flags=0):
    _check(_lib.gist_adam_update(ctx.handle, _ptr(W), _ptr(dW), _ptr(m), _ptr(v), int(n),
                                 float(lr), float(beta1), float(beta2), float(eps), int(step),
                                 int(flags)))


def gist_adam_coefficients(lr, step, beta1=0.9, beta2=0.999, eps=1e-8, flags=0):
    """float32[3] {lr / (1 - beta1^k), 1 / sqrt(1 - beta2^k), fresh} for gist_adam_update_dev."""
    out = np.empty(3, dtype=np.float32)
    _check(_lib.gist_adam_coefficients(float(lr), float(beta1), float(beta2), float(eps),
                                       int(step), int(flags), _ptr(out)))
    return out


def gist_adam_update_dev(ctx, W, dW, m, v, n, coef_dev, beta1=0.9, beta2=0.999, eps=1e-8):
    _check(_lib.gist_adam_update_dev(ctx.handle, _ptr(W), _ptr(dW), _ptr(m), _ptr(v), int(n),
                                     float(beta1), float(beta2), float(eps), _ptr(coef_dev)))


GIST_GAT_MIRROR_IN_WS = 1


def gat_desc(n, nnz, s_in, s_out, act, dtype=GIST_DTYPE_F32, slope=0.2, flags=0):
    """``flags``: GIST_GAT_MIRROR_IN_WS (the backward workspace holds A's mirror map)."""
    return gist_gat_desc(int(n), int(nnz), int(s_in), int(s_out), int(act), int(dtype),
                         float(slope), int(flags))


def gist_gat_workspace_size(desc):
    f, b = C.c_size_t(), C.c_size_t()
    _check(_lib.gist_gat_workspace_size(C.byref(desc), C.byref(f), C.byref(b)))
    return int(f.value), int(b.value)


def gist_gat_layer_fwd(ctx, desc, A, H, W, a_src, a_dst, P_save, alpha_save, H_out, ws):
    _check(_lib.gist_gat_layer_fwd(ctx.handle, C.byref(desc), C.byref(A), _ptr(H), _ptr(W),
                                   _ptr(a_src), _ptr(a_dst), _ptr(P_save), _ptr(alpha_save),
                                   _ptr(H_out), _ptr(ws), 0 if ws is None else ws.numel()))


def gist_gat_layer_bwd(ctx, desc, A, H, P_save, alpha_save, H_out, W, a_src, a_dst, dH_out, dW,
                       da_src, da_dst, dH, ws):
    _check(_lib.gist_gat_layer_bwd(ctx.handle, C.byref(desc), C.byref(A), _ptr(H), _ptr(P_save),
                                   _ptr(alpha_save), _ptr(H_out), _ptr(W), _ptr(a_src),
                                   _ptr(a_dst), _ptr(dH_out), _ptr(dW), _ptr(da_src),
                                   _ptr(da_dst), _ptr(dH), _ptr(ws),
                                   0 if ws is None else ws.numel()))


def gist_gat_scores(ctx, n, s, P, ldp, a_src, a_dst, u, v):
    _check(_lib.gist_gat_scores(ctx.handle, int(n), int(s), _ptr(P), int(ldp), _ptr(a_src),
                                _ptr(a_dst), _ptr(u), _ptr(v)))


def slice_set(row_rank, row_offs, col_rank, col_offs, slice_ptrs, ld):
    """A ``gist_slice_set`` over device tensors (ranks int32, offsets int64, pointer table int64)."""
    return gist_slice_set(_ptr(row_rank), _ptr(row_offs), _ptr(col_rank), _ptr(col_offs),
                          _ptr(slice_ptrs), int(ld))


def gist_subagg_gather(ctx, Wg, rows, cols, ldg, m, done, next_):
    _check(_lib.gist_subagg_gather(ctx.handle, _ptr(Wg), int(rows), int(cols), int(ldg), int(m),
                                   C.byref(done) if done is not None else None,
                                   C.byref(next_) if next_ is not None else None))


def gist_subagg_mean(ctx, Wg, rows, cols, ldg, m, slice_ptrs, lds):
    """Wg = mean of the m slices; ``slice_ptrs`` is a device int64 tensor of their addresses."""
    _check(_lib.gist_subagg_mean(ctx.handle, _ptr(Wg), int(rows), int(cols), int(ldg), int(m),
                                 _ptr(slice_ptrs), int(lds)))


def gist_subagg(ctx, Wg, ldg, rows, nr, cols, nc, Ws, lds, flags=0):
    _check(_lib.gist_subagg(ctx.handle, _ptr(Wg), int(ldg), _ptr(rows), int(nr), _ptr(cols),
                            int(nc), _ptr(Ws), int(lds), int(flags)))


# ---- replays ---------------------------------------------------------------------
class Replay:
    """A captured sequence of library calls (``gist_capture_end``), freed with it."""

    def __init__(self, handle):
        self.handle = handle

    def close(self):
        if self.handle:
            _lib.gist_replay_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Event:
    """A ``gist_event``: recorded by ``gist_replay_launch``, waited on by ``synchronize``."""

    def __init__(self):
        h = _P()
        _check(_lib.gist_event_create(C.byref(h)))
        self.handle = h

    def synchronize(self):
        _check(_lib.gist_event_synchronize(self.handle))

    def __del__(self):
        try:
            if self.handle:
                _lib.gist_event_destroy(self.handle)
                self.handle = None
        except Exception:
            pass


def gist_capture_begin(ctx):
    _check(_lib.gist_capture_begin(ctx.handle))


def gist_capture_end(ctx):
    h = _P()
    _check(_lib.gist_capture_end(ctx.handle, C.byref(h)))
    return Replay(h)


def gist_replay_launch(ctx, replay, dst=None, src=None, nbytes=0, copied=None):
    """Copy ``nbytes`` from host ``src`` to device ``dst`` (tensors or addresses), record
    ``copied``, launch ``replay`` -- all on the stream of ``ctx``."""
    d = dst if isinstance(dst, int) or dst is None else _ptr(dst)
    s_ = src if isinstance(src, int) or src is None else _ptr(src)
    _check(_lib.gist_replay_launch(ctx.handle, replay.handle, d, s_, int(nbytes),
                                   copied.handle if copied is not None else None))


def gist_copy(ctx, dst, src, nbytes, copied=None):
    """``nbytes`` from ``src`` (device or pinned host) to device ``dst``, by a kernel on
    the stream of ``ctx``; then record ``copied``."""
    d = dst if isinstance(dst, int) else _ptr(dst)
    s_ = src if isinstance(src, int) else _ptr(src)
    _check(_lib.gist_copy(ctx.handle, d, s_, int(nbytes),
                          copied.handle if copied is not None else None))


# ---- instrumentation ------------------------------------------------------------
def gist_profile_begin(ctx, cap=65536):
    _check(_lib.gist_profile_begin(ctx.handle, int(cap)))


def gist_profile_read(ctx):
    """Synchronise and return {variant: dict(launches, ms, flops, bytes)}, plus dropped."""
    buf = (gist_prof_entry * 256)()
    n = C.c_int32()
    dropped = C.c_int64()
    _check(_lib.gist_profile_read(ctx.handle, buf, 256, C.byref(n), C.byref(dropped)))
    out = {}
    for i in range(n.value):
        e = buf[i]
        out[e.name.decode()] = dict(launches=int(e.launches), ms=float(e.ms),
                                    flops=float(e.flops), bytes=float(e.bytes))
    return out, int(dropped.value)


def gist_profile_end(ctx):
    _check(_lib.gist_profile_end(ctx.handle))
