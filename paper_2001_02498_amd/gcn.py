"""ctypes binding of libgcnact.so (the C ABI of include/gcn_act.h).

Argument marshalling only: every computation runs in the library (host C++
for graph preprocessing, HIP kernels for the training step). Device buffers
are torch tensors, passed by data pointer; streams are torch streams,
passed by handle. If the library has not been built this module raises on
import; there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libgcnact.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with "
                      "`python -m paper_2001_02498_amd.build`")
# One HIP runtime per process: torch's. torch's libraries name their bundled
# runtime `libamdhip64.so` while the library names `libamdhip64.so.7`; with
# torch loaded first the library's dependency resolves to torch's copy (same
# soname), but loaded first itself it maps the system copy and torch then
# maps a second runtime, which cannot open the GPU the first holds (and
# torch's stream handles would belong to the other runtime).
try:
    import torch  # noqa: F401
except ImportError:
    pass
_lib = C.CDLL(LIB_PATH)

OK = 0
E_INVALID_ARG = -1
E_HIP = -2
E_OOM = -3
E_UNSUPPORTED = -4
E_NONFINITE = -7
E_WORKSPACE = -5
E_INTERNAL = -6
MAX_ROUNDS = 64
MAX_LAYERS = 8
LOSS_SOFTMAX_CE = 0
LOSS_SIGMOID_BCE = 1
PREC_FP32 = 0
PREC_BF16 = 1
PIPE_PINNED = 1
PIPE_DEVICE_REDUCE = 2
ORDER_PAPER = 0
ORDER_NARROW = 1
OPT_SGD = 0
OPT_MOMENTUM = 1
OPT_ADAM = 2
AGG_MEAN = 0
AGG_TRANSPOSED = 1
ABI_VERSION = 7
BIN_GROUPS = 16

_i32, _i64, _f32 = C.c_int32, C.c_int64, C.c_float
_vp, _sz = C.c_void_p, C.c_size_t
_pi32 = C.POINTER(C.c_int32)
_pi64 = C.POINTER(C.c_int64)
_pf32 = C.POINTER(C.c_float)


class GcnError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class RrParams(C.Structure):
    _fields_ = [("theta", _i32), ("max_rounds", _i32), ("max_aux", _i64),
                ("num_threads", _i32), ("reserved", _i32)]


class RrRound(C.Structure):
    _fields_ = [("matched", _i64), ("weight_sum", _i64), ("nnz", _i64),
                ("num_add", _i64)]


class DGraph(C.Structure):
    _fields_ = [("n", _i32), ("naux", _i32), ("rounds", _i32), ("seg_len", _i32),
                ("nseg", _i32), ("nbins", _i32), ("nmulti", _i32), ("nhub", _i32),
                ("max_row", _i32), ("reserved", _i32),
                ("nnz", _i64), ("exp_nnz", _i64),
                ("rowptr", _vp), ("col", _vp), ("pairs", _vp), ("inv_deg", _vp),
                ("seg", _vp), ("bins", _vp), ("exp_col", _vp), ("exp_seg", _vp),
                ("round_offsets", _i32 * (MAX_ROUNDS + 1))]


class ModelDesc(C.Structure):
    _fields_ = [("L", _i32), ("f_in", _i32), ("h", _i32), ("C", _i32),
                ("loss", _i32), ("precision", _i32), ("has_bias", _i32),
                ("order", _i32), ("ld_x", _i64)]


class Params(C.Structure):
    _fields_ = [("W_self", _vp * MAX_LAYERS), ("W_neigh", _vp * MAX_LAYERS),
                ("b", _vp * MAX_LAYERS), ("W_cls", _vp), ("b_cls", _vp)]


class WsLayout(C.Structure):
    _fields_ = [("AH", _i64 * MAX_LAYERS), ("H", _i64 * MAX_LAYERS),
                ("ld_AH", _i64 * MAX_LAYERS), ("ld_H", _i64),
                ("logits", _i64), ("dlogits", _i64), ("ld_C", _i64),
                ("G", _i64 * MAX_LAYERS),
                ("scratch", _i64), ("scratch_bytes", _i64), ("total_bytes", _i64),
                ("ah_bytes", _i64), ("H16", _i64 * MAX_LAYERS), ("G16", _i64 * MAX_LAYERS),
                ("status", _i64)]


def _proto(name, args, res=C.c_int):
    f = getattr(_lib, name)
    f.argtypes = args
    f.restype = res
    return f


_last_error = _proto("gcn_last_error", [], C.c_char_p)
_abi_version = _proto("gcn_abi_version", [])
_subgraph_build = _proto("gcn_subgraph_build", [_i64, _vp, _vp, _i64, _vp, _i64, C.POINTER(_vp)])
_graph_info = _proto("gcn_graph_info", [_vp, _pi32, _pi64, C.POINTER(_pi32), C.POINTER(_pi32)])
_graph_free = _proto("gcn_graph_free", [_vp], None)
_sample_frontier = _proto("gcn_sample_frontier", [_vp, _i32, _i32, C.c_uint64, _i64, _vp,
                                                  _pi32, _pi64])
_subgraph_induce = _proto("gcn_subgraph_induce", [_vp, _vp, _i32, C.POINTER(_vp)])
_gather_rows = _proto("gcn_gather_rows", [_vp, _i64, _i64, _vp, _i32, _i64, _vp, _i64, _vp])
_reduce = _proto("gcn_redundancy_reduce", [_vp, C.POINTER(RrParams), C.POINTER(_vp)])
_reduce_dev_bytes = _proto("gcn_redundancy_reduce_device_bytes",
                           [_vp, C.POINTER(RrParams), C.POINTER(_sz)])
_reduce_dev = _proto("gcn_redundancy_reduce_device",
                     [_vp, C.POINTER(RrParams), _vp, _sz, _vp, C.POINTER(_vp)])
_reduced_info = _proto("gcn_reduced_info", [_vp, _pi32, _pi32, _pi32, _pi64,
                                            C.POINTER(_pi32), C.POINTER(_pi32), C.POINTER(_pi32),
                                            C.POINTER(_pi32), C.POINTER(C.POINTER(RrRound)),
                                            C.POINTER(_pi32)])
_reduced_free = _proto("gcn_reduced_free", [_vp], None)
_image_bytes = _proto("gcn_graph_image_bytes", [_vp, _i32, C.POINTER(_sz)])
_pack = _proto("gcn_graph_pack", [_vp, _i32, _vp, _sz])
_upload = _proto("gcn_graph_upload", [_vp, _sz, _vp, C.POINTER(DGraph), _vp])
_describe = _proto("gcn_graph_describe", [_vp, _sz, _vp, C.POINTER(DGraph)])
_scratch_bytes = _proto("gcn_scratch_bytes", [C.POINTER(DGraph), _i32, _i32, C.POINTER(_sz)])
_aggregate_noalloc = _proto("gcn_aggregate_noalloc", [C.POINTER(DGraph), _i32, _i32, _vp, _i64,
                                                      _vp, _i64, _vp])
AGG_NOALLOC_SCRATCH_BYTES = 64 << 20
_aggregate = _proto("gcn_aggregate", [C.POINTER(DGraph), _i32, _i32, _vp, _i64, _vp, _i64,
                                      _vp, _sz, _vp])
_layer_fwd = _proto("gcn_layer_fwd", [C.POINTER(DGraph), _i32, _i32, _vp, _i64, _vp, _vp, _vp,
                                      _vp, _i64, _vp, _i64, _i32, _vp, _sz, _vp])
_classifier_fwd = _proto("gcn_classifier_fwd", [_i32, _i32, _i32, _vp, _i64, _vp, _vp, _vp,
                                                _i64, _i32, _vp, _sz, _vp])
_loss = _proto("gcn_loss", [_i32, _i32, _i32, _vp, _i64, _vp, _vp, _i64, _vp, _vp, _sz, _vp])
_classifier_bwd = _proto("gcn_classifier_bwd", [_i32, _i32, _i32, _vp, _i64, _vp, _i64, _vp,
                                                _vp, _f32, _vp, _i64, _vp, _vp, _i32, _vp,
                                                _sz, _vp])
_layer_bwd = _proto("gcn_layer_bwd", [C.POINTER(DGraph), _i32, _i32, _vp, _i64, _vp, _i64, _vp,
                                      _i64, _vp, _vp, _vp, _f32, _vp, _i64, _vp, _vp, _vp,
                                      _i32, _vp, _sz, _vp])
_ws_layout = _proto("gcn_workspace_layout", [C.POINTER(DGraph), C.POINTER(ModelDesc),
                                             C.POINTER(WsLayout)])
_ws_bytes = _proto("gcn_workspace_bytes", [C.POINTER(DGraph), C.POINTER(ModelDesc),
                                           C.POINTER(_sz)])
_train_step = _proto("gcn_train_step", [C.POINTER(DGraph), C.POINTER(ModelDesc),
                                        C.POINTER(Params), _vp, _vp, _f32, _vp,
                                        C.POINTER(Params), _vp, _sz, _vp])


class Optim(C.Structure):
    _fields_ = [("kind", _i32), ("step", _i32), ("lr", _f32), ("momentum", _f32),
                ("beta1", _f32), ("beta2", _f32), ("eps", _f32), ("reserved", _f32)]


_infer = _proto("gcn_infer", [C.POINTER(DGraph), C.POINTER(ModelDesc), C.POINTER(Params), _vp,
                              _vp, _i64, _vp, _sz, _vp])
_train_step_optim = _proto("gcn_train_step_optim",
                           [C.POINTER(DGraph), C.POINTER(ModelDesc), C.POINTER(Params), _vp,
                            _vp, C.POINTER(Optim), C.POINTER(Params), C.POINTER(Params), _vp,
                            C.POINTER(Params), _vp, _sz, _vp])

class ProfileEntry(C.Structure):
    _fields_ = [("kind", _i32), ("launches", _i32), ("name", C.c_char_p),
                ("total_ms", C.c_double), ("min_ms", C.c_double), ("max_ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


_prof_enable = _proto("gcn_profile_enable", [_i32])
_prof_disable = _proto("gcn_profile_disable", [])
_prof_read = _proto("gcn_profile_read", [C.POINTER(ProfileEntry), _i32, _pi32, _i32])
_read_probe = _proto("gcn_read_probe", [_vp, _sz, _vp, _vp])
_status_check = _proto("gcn_status_check", [_vp, _vp])
READ_PROBE_SINK = 16384

class PipelineInfo(C.Structure):
    _fields_ = [("n", _i32), ("naux", _i32), ("rounds", _i32), ("reserved", _i32),
                ("nnz", _i64), ("nnz_direct", _i64), ("build_ms", C.c_double),
                ("reduce_ms", C.c_double), ("pack_ms", C.c_double),
                ("sample_ms", C.c_double), ("image_bytes", _i64),
                ("vertices_offset", _i64), ("steps", _i64)]


_pipe_create = _proto("gcn_pipeline_create", [C.POINTER(RrParams), _i32, _i32, _i32, _i32,
                                              _vp, _sz, C.POINTER(_vp)])
_pipe_create_mixed = _proto("gcn_pipeline_create_mixed", [C.POINTER(RrParams), _i32, _i32, _i32,
                                                          _i32, _i32, _vp, _sz, C.POINTER(_vp)])
_pipe_submit = _proto("gcn_pipeline_submit", [_vp, _i64, _vp, _vp, _i64, _vp, _i64,
                                              C.POINTER(_i64)])
_pipe_submit_sample = _proto("gcn_pipeline_submit_sample", [_vp, _vp, _i32, _i32, C.c_uint64,
                                                            _i64, C.POINTER(_i64)])
_pipe_next = _proto("gcn_pipeline_next", [_vp, C.POINTER(_i64), C.POINTER(_vp), C.POINTER(_sz),
                                          C.POINTER(PipelineInfo)])
_pipe_release = _proto("gcn_pipeline_release", [_vp, _i64])
_pipe_destroy = _proto("gcn_pipeline_destroy", [_vp], None)

EXPORTS = [
    "gcn_last_error", "gcn_abi_version", "gcn_subgraph_build", "gcn_graph_info",
    "gcn_graph_free", "gcn_sample_frontier", "gcn_subgraph_induce", "gcn_gather_rows",
    "gcn_redundancy_reduce", "gcn_reduced_info", "gcn_reduced_free",
    "gcn_redundancy_reduce_device_bytes", "gcn_redundancy_reduce_device",
    "gcn_graph_image_bytes", "gcn_graph_pack", "gcn_graph_upload", "gcn_graph_describe",
    "gcn_scratch_bytes", "gcn_aggregate", "gcn_layer_fwd", "gcn_classifier_fwd",
    "gcn_loss", "gcn_classifier_bwd", "gcn_layer_bwd", "gcn_workspace_layout",
    "gcn_workspace_bytes", "gcn_train_step", "gcn_train_step_optim", "gcn_infer", "gcn_profile_enable",
    "gcn_profile_disable",
    "gcn_profile_read", "gcn_pipeline_create", "gcn_pipeline_submit", "gcn_pipeline_next",
    "gcn_pipeline_release", "gcn_pipeline_destroy", "gcn_pipeline_submit_sample",
    "gcn_pipeline_create_mixed", "gcn_read_probe", "gcn_aggregate_noalloc",
    "gcn_status_check",
]


def last_error() -> str:
    return _last_error().decode()


def _check(rc):
    if rc != OK:
        raise GcnError(rc, last_error())


def abi_version() -> int:
    return _abi_version()


# ------------------------------------------------------------------ host side

def _np_ptr(a):
    return a.ctypes.data_as(_vp) if a is not None and a.size else None


class Graph:
    """Undirected simple subgraph in CSR form (owned by the library)."""

    def __init__(self, handle):
        self._h = _vp(handle)

    def __del__(self, _free=_graph_free, _null=_vp):
        # the free function is bound as a default: at interpreter teardown
        # the module's globals may already be gone
        if getattr(self, "_h", None) and self._h.value:
            _free(self._h)
            self._h = _null()

    def _info(self):
        n, nnz = _i32(), _i64()
        rp, cl = _pi32(), _pi32()
        _check(_graph_info(self._h, C.byref(n), C.byref(nnz), C.byref(rp), C.byref(cl)))
        return n.value, nnz.value, rp, cl

    @property
    def n(self):
        return self._info()[0]

    @property
    def nnz(self):
        return self._info()[1]

    def csr(self):
        n, nnz, rp, cl = self._info()
        rowptr = np.ctypeslib.as_array(rp, shape=(n + 1,)).copy()
        col = np.ctypeslib.as_array(cl, shape=(nnz,)).copy() if nnz else np.zeros(0, np.int32)
        return rowptr, col


def subgraph_build(n_full, src, dst, vertices=None) -> Graph:
    src = np.ascontiguousarray(src, dtype=np.int64)
    dst = np.ascontiguousarray(dst, dtype=np.int64)
    if src.shape != dst.shape:
        raise ValueError("src and dst differ in length")
    v = None if vertices is None else np.ascontiguousarray(vertices, dtype=np.int64)
    # an empty subset still passes a pointer (NULL means every vertex)
    vp = None if v is None else (_np_ptr(v) if v.size else np.zeros(1, np.int64).ctypes.data_as(_vp))
    out = _vp()
    _check(_subgraph_build(int(n_full), _np_ptr(src), _np_ptr(dst), src.size, vp,
                           0 if v is None else v.size, C.byref(out)))
    return Graph(out.value)


def sample_frontier(full: Graph, m, budget, seed, max_steps):
    """Frontier sampling of a minibatch's vertex set from `full`.
    Returns (vertices int32 ascending, steps taken)."""
    out = np.empty(max(int(budget), 0), dtype=np.int32)
    cnt, steps = _i32(), _i64()
    _check(_sample_frontier(full._h, int(m), int(budget), int(seed) & (2 ** 64 - 1),
                            int(max_steps), _np_ptr(out), C.byref(cnt), C.byref(steps)))
    return out[:cnt.value].copy(), steps.value


def subgraph_induce(full: Graph, vertices) -> Graph:
    """Subgraph of `full` induced on `vertices` (vertex vertices[k] becomes k)."""
    v = np.ascontiguousarray(vertices, dtype=np.int32)
    out = _vp()
    _check(_subgraph_induce(full._h, _np_ptr(v), v.size, C.byref(out)))
    return Graph(out.value)


def gather_rows(src, idx, dst, n_src=None, stream=None):
    """dst[k] = src[idx[k]] on the device for 2-D tensors (rows may be
    strided views; row widths equal), or 1-D tensors of 4-byte elements."""
    if src.dim() == 1:
        src, dst = src.view(-1, 1), dst.view(-1, 1)
    if src.dtype != dst.dtype or src.shape[1] != dst.shape[1]:
        raise ValueError("src and dst rows differ")
    if src.stride(1) != 1 or dst.stride(1) != 1 or idx.dtype.itemsize != 4:
        raise ValueError("rows must be contiguous and idx int32")
    es = src.element_size()
    n = idx.numel()
    if dst.shape[0] < n:
        raise ValueError("dst has fewer rows than idx")
    _check(_gather_rows(_ptr(src), src.stride(0) * es, src.shape[0] if n_src is None else n_src,
                        _ptr(idx), n, src.shape[1] * es, _ptr(dst), dst.stride(0) * es,
                        _stream(stream)))


class Reduced:
    """Output of the redundancy reduction (owned by the library)."""

    def __init__(self, handle):
        self._h = _vp(handle)

    def __del__(self, _free=_reduced_free, _null=_vp):
        if getattr(self, "_h", None) and self._h.value:
            _free(self._h)
            self._h = _null()

    def info(self):
        n, naux, rounds, nnz = _i32(), _i32(), _i32(), _i64()
        rp, cl, pr, ro, dg = _pi32(), _pi32(), _pi32(), _pi32(), _pi32()
        st = C.POINTER(RrRound)()
        _check(_reduced_info(self._h, C.byref(n), C.byref(naux), C.byref(rounds),
                             C.byref(nnz), C.byref(rp), C.byref(cl), C.byref(pr),
                             C.byref(ro), C.byref(st), C.byref(dg)))
        n, naux, rounds, nnz = n.value, naux.value, rounds.value, nnz.value

        def arr(p, k):
            return np.ctypeslib.as_array(p, shape=(k,)).copy() if k else np.zeros(0, np.int32)
        stats = [(st[i].matched, st[i].weight_sum, st[i].nnz, st[i].num_add)
                 for i in range(rounds)]
        return dict(n=n, naux=naux, rounds=rounds, nnz=nnz,
                    rowptr=arr(rp, n + 1), col=arr(cl, nnz),
                    pairs=arr(pr, 2 * naux).reshape(-1, 2),
                    round_offsets=arr(ro, rounds + 1), stats=stats, deg=arr(dg, n))


def redundancy_reduce(g: Graph, theta=2, max_rounds=5, max_aux=-1, num_threads=0) -> Reduced:
    p = RrParams(int(theta), int(max_rounds), int(max_aux), int(num_threads), 0)
    out = _vp()
    _check(_reduce(g._h, C.byref(p), C.byref(out)))
    return Reduced(out.value)


def redundancy_reduce_device_bytes(g: Graph, theta=2, max_rounds=5, max_aux=-1) -> int:
    p = RrParams(int(theta), int(max_rounds), int(max_aux), 0, 0)
    b = _sz()
    _check(_reduce_dev_bytes(g._h, C.byref(p), C.byref(b)))
    return b.value


def device_reduce_bytes(graphs, workers=1, theta=2, max_rounds=5, max_aux=-1) -> int:
    """Device workspace for `workers` GPU-reducing pipeline workers that can
    each reduce any of `graphs`: workers x the largest
    gcn_redundancy_reduce_device_bytes, in 256-byte-aligned shares."""
    need = max([redundancy_reduce_device_bytes(g, theta, max_rounds, max_aux) for g in graphs]
               + [256])
    return int(workers) * ((need + 255) // 256 * 256)


def redundancy_reduce_device(g: Graph, ws, theta=2, max_rounds=5, max_aux=-1,
                             stream=None) -> Reduced:
    """The rounds of Algorithms 1-3 on the GPU (synchronous); `ws` is a
    device workspace of redundancy_reduce_device_bytes() bytes."""
    p = RrParams(int(theta), int(max_rounds), int(max_aux), 0, 0)
    out = _vp()
    _check(_reduce_dev(g._h, C.byref(p), _ptr(ws), ws.numel(), _stream(stream), C.byref(out)))
    return Reduced(out.value)


def image_bytes(r: Reduced, seg_len=0) -> int:
    b = _sz()
    _check(_image_bytes(r._h, int(seg_len), C.byref(b)))
    return b.value


def pack(r: Reduced, buf_ptr: int, nbytes: int, seg_len=0):
    _check(_pack(r._h, int(seg_len), _vp(buf_ptr), nbytes))


def describe(host_ptr: int, nbytes: int, dev_ptr: int) -> DGraph:
    d = DGraph()
    _check(_describe(_vp(host_ptr), nbytes, _vp(dev_ptr), C.byref(d)))
    return d


# ---------------------------------------------------------------- device side

def _torch():
    import torch
    return torch


def _stream(stream):
    if stream is None:
        return _vp(_torch().cuda.current_stream().cuda_stream)
    return _vp(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _ptr(t):
    return None if t is None else _vp(t.data_ptr())


def _ld(t):
    if t is None:
        return 0
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("matrix must be 2-D with unit column stride")
    return t.stride(0)


class DeviceGraph:
    """A reduced graph resident in device memory (torch-owned buffer)."""

    def __init__(self, reduced: Reduced, seg_len=0, stream=None, device="cuda"):
        torch = _torch()
        nbytes = image_bytes(reduced, seg_len)
        self.host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
        pack(reduced, self.host.data_ptr(), nbytes, seg_len)
        self.dev = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        off = (-self.dev.data_ptr()) % 256
        self.dev_view = self.dev[off:off + nbytes]
        self.nbytes = nbytes
        self.desc = DGraph()
        _check(_upload(_vp(self.host.data_ptr()), nbytes, _vp(self.dev_view.data_ptr()),
                       C.byref(self.desc), _stream(stream)))

    @property
    def n(self):
        return self.desc.n


def alloc_ws(nbytes, device="cuda"):
    """256-byte-aligned device workspace as a uint8 tensor view."""
    torch = _torch()
    raw = torch.empty(int(nbytes) + 256, dtype=torch.uint8, device=device)
    off = (-raw.data_ptr()) % 256
    view = raw[off:off + int(nbytes)]
    view._raw = raw
    return view


def scratch_bytes(dg: DeviceGraph | None, max_width: int, n: int = 0) -> int:
    b = _sz()
    _check(_scratch_bytes(C.byref(dg.desc) if dg is not None else None, n, int(max_width),
                          C.byref(b)))
    return b.value


def aggregate(dg, mode, X, Y, ws, stream=None):
    _check(_aggregate(C.byref(dg.desc), mode, X.shape[1], _ptr(X), _ld(X), _ptr(Y), _ld(Y),
                      _ptr(ws), ws.numel(), _stream(stream)))


def aggregate_noalloc(dg, mode, X, Y, stream=None):
    """gcn_aggregate_noalloc: the aggregation on the library's fixed
    per-device scratch (no workspace; calls on one device must not
    overlap)."""
    _check(_aggregate_noalloc(C.byref(dg.desc), mode, X.shape[1], _ptr(X), _ld(X), _ptr(Y),
                              _ld(Y), _stream(stream)))


def layer_fwd(dg, H_in, W_self, W_neigh, bias, AH, H_out, ws, precision=PREC_FP32,
              stream=None):
    F, h = W_self.shape
    _check(_layer_fwd(C.byref(dg.desc), F, h, _ptr(H_in), _ld(H_in), _ptr(W_self),
                      _ptr(W_neigh), _ptr(bias), _ptr(AH), _ld(AH), _ptr(H_out),
                      _ld(H_out), precision, _ptr(ws), ws.numel(), _stream(stream)))


def classifier_fwd(H, K, W_cls, b_cls, logits, ws, precision=PREC_FP32, stream=None):
    n = H.shape[0]
    Cn = W_cls.shape[1]
    _check(_classifier_fwd(n, K, Cn, _ptr(H), _ld(H), _ptr(W_cls), _ptr(b_cls),
                           _ptr(logits), _ld(logits), precision, _ptr(ws), ws.numel(),
                           _stream(stream)))


def loss(kind, logits, C_, labels, dlogits, loss_out, ws, stream=None):
    n = logits.shape[0]
    _check(_loss(n, C_, kind, _ptr(logits), _ld(logits), _ptr(labels), _ptr(dlogits),
                 _ld(dlogits), _ptr(loss_out), _ptr(ws), ws.numel(), _stream(stream)))


def classifier_bwd(dZ, C_, H, K, W_cls, b_cls, lr, G_out, dW_out, db_out, ws,
                   precision=PREC_FP32, stream=None):
    n = dZ.shape[0]
    _check(_classifier_bwd(n, K, C_, _ptr(dZ), _ld(dZ), _ptr(H), _ld(H), _ptr(W_cls),
                           _ptr(b_cls), float(lr), _ptr(G_out), _ld(G_out), _ptr(dW_out),
                           _ptr(db_out), precision, _ptr(ws), ws.numel(), _stream(stream)))


def layer_bwd(dg, G, H_in, AH, W_self, W_neigh, bias, lr, G_in, dW_self, dW_neigh, db, ws,
              precision=PREC_FP32, stream=None):
    F, h = W_self.shape
    _check(_layer_bwd(C.byref(dg.desc), F, h, _ptr(G), _ld(G), _ptr(H_in), _ld(H_in),
                      _ptr(AH), _ld(AH), _ptr(W_self), _ptr(W_neigh), _ptr(bias),
                      float(lr), _ptr(G_in), _ld(G_in), _ptr(dW_self), _ptr(dW_neigh),
                      _ptr(db), precision, _ptr(ws), ws.numel(), _stream(stream)))


def model_desc(L, f_in, h, C_, loss_kind, ld_x, precision=PREC_FP32, has_bias=False,
               order=ORDER_PAPER):
    return ModelDesc(L, f_in, h, C_, loss_kind, precision, 1 if has_bias else 0, order, ld_x)


def make_params(W_self, W_neigh, W_cls, b=None, b_cls=None):
    p = Params()
    for l, (ws_, wn_) in enumerate(zip(W_self, W_neigh)):
        p.W_self[l] = None if ws_ is None else ws_.data_ptr()
        p.W_neigh[l] = None if wn_ is None else wn_.data_ptr()
        if b is not None and b[l] is not None:
            p.b[l] = b[l].data_ptr()
    p.W_cls = None if W_cls is None else W_cls.data_ptr()
    p.b_cls = None if b_cls is None else b_cls.data_ptr()
    return p


def workspace_layout(dg, desc) -> WsLayout:
    out = WsLayout()
    _check(_ws_layout(C.byref(dg.desc), C.byref(desc), C.byref(out)))
    return out


def workspace_bytes(dg, desc) -> int:
    b = _sz()
    _check(_ws_bytes(C.byref(dg.desc), C.byref(desc), C.byref(b)))
    return b.value


def train_step(dg, desc, params, X, labels, lr, loss_out, ws, grads=None, stream=None):
    _check(_train_step(C.byref(dg.desc), C.byref(desc), C.byref(params), _ptr(X),
                       _ptr(labels), float(lr), _ptr(loss_out),
                       C.byref(grads) if grads is not None else None, _ptr(ws), ws.numel(),
                       _stream(stream)))


def infer(dg, desc, params, X, logits, ws, stream=None):
    """Forward pass and classifier logits of the whole (reduced) graph."""
    _check(_infer(C.byref(dg.desc), C.byref(desc), C.byref(params), _ptr(X), _ptr(logits),
                  _ld(logits), _ptr(ws), ws.numel(), _stream(stream)))


def optim(kind, lr, step=1, momentum=0.9, beta1=0.9, beta2=0.999, eps=1e-8) -> Optim:
    return Optim(kind, step, lr, momentum, beta1, beta2, eps, 0.0)


def train_step_optim(dg, desc, params, X, labels, opt, loss_out, ws, state1=None, state2=None,
                     grads=None, stream=None):
    _check(_train_step_optim(C.byref(dg.desc), C.byref(desc), C.byref(params), _ptr(X),
                             _ptr(labels), C.byref(opt),
                             C.byref(state1) if state1 is not None else None,
                             C.byref(state2) if state2 is not None else None, _ptr(loss_out),
                             C.byref(grads) if grads is not None else None, _ptr(ws),
                             ws.numel(), _stream(stream)))


# ------------------------------------------------------------ launch timing

def profile_enable(capacity=4096):
    _check(_prof_enable(int(capacity)))


def profile_disable():
    _check(_prof_disable())


def profile_read(reset=True):
    """Per kernel class: dict(launches, total_ms, min_ms, max_ms, flops, bytes)."""
    buf = (ProfileEntry * 32)()
    cnt = _i32()
    _check(_prof_read(buf, 32, C.byref(cnt), 1 if reset else 0))
    return {buf[i].name.decode(): dict(launches=buf[i].launches, total_ms=buf[i].total_ms,
                                       min_ms=buf[i].min_ms, max_ms=buf[i].max_ms,
                                       flops=buf[i].flops, bytes=buf[i].bytes)
            for i in range(min(cnt.value, 32))}


def status_check(ws, offset=0, stream=None):
    """gcn_status_check on the status word at byte `offset` of the device
    buffer `ws` (0 for gcn_loss's ws; layout.status for a training step's):
    raises GcnError (E_INVALID_ARG: an invalid label; E_NONFINITE: the loss
    was not finite) after waiting for the stream."""
    _check(_status_check(_vp(ws.data_ptr() + int(offset)), _stream(stream)))


def read_probe(buf, sink, stream=None):
    """One streaming read of every byte of the device tensor `buf`
    (gcn_read_probe); `sink`: device float32 tensor of READ_PROBE_SINK."""
    torch = _torch()
    if not (buf.is_cuda and sink.is_cuda and sink.dtype == torch.float32
            and sink.numel() >= READ_PROBE_SINK and buf.is_contiguous()):
        raise ValueError("read_probe: contiguous device buffer and a float32 device sink "
                         f"of {READ_PROBE_SINK} needed")
    _check(_read_probe(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink),
                       _stream(stream)))


# ------------------------------------------------------ preparation pipeline

class Pipeline:
    """Host worker pool preparing graph images in submission order."""

    def __init__(self, theta=2, max_rounds=5, max_aux=-1, seg_len=0, workers=4, depth=8,
                 pinned=True, num_threads=1, device_reduce=False, device_workers=None,
                 device_ws=None):
        """`workers` threads reducing on the host (on the GPU with
        device_reduce); device_workers > 0 adds that many GPU-reducing
        workers beside `workers` host ones. GPU-reducing workers share
        `device_ws` (a 256-byte-aligned device uint8 tensor, e.g. from
        alloc_ws, kept alive by the pipeline), split evenly between them:
        size it with device_reduce_bytes()."""
        p = RrParams(int(theta), int(max_rounds), int(max_aux), int(num_threads), 0)
        self._h = _vp()
        self._borrowed = {}   # job id -> full graph a sampled job reads
        self._dev_ws = device_ws
        ws_ptr = _ptr(device_ws) if device_ws is not None else None
        ws_bytes = device_ws.numel() if device_ws is not None else 0
        if device_workers is not None:
            _check(_pipe_create_mixed(C.byref(p), int(seg_len), int(workers), int(device_workers),
                                      int(depth), PIPE_PINNED if pinned else 0, ws_ptr, ws_bytes,
                                      C.byref(self._h)))
            return
        flags = (PIPE_PINNED if pinned else 0) | (PIPE_DEVICE_REDUCE if device_reduce else 0)
        _check(_pipe_create(C.byref(p), int(seg_len), int(workers), int(depth), flags, ws_ptr,
                            ws_bytes, C.byref(self._h)))

    def submit(self, n_full, src, dst, vertices=None):
        src = np.ascontiguousarray(src, dtype=np.int64)
        dst = np.ascontiguousarray(dst, dtype=np.int64)
        v = None if vertices is None else np.ascontiguousarray(vertices, dtype=np.int64)
        jid = _i64()
        _check(_pipe_submit(self._h, int(n_full), _np_ptr(src), _np_ptr(dst), src.size,
                            _np_ptr(v) if v is not None else None, 0 if v is None else v.size,
                            C.byref(jid)))
        return jid.value

    def submit_sample(self, full: Graph, m, budget, seed, max_steps):
        """Queue a job that samples its subgraph from `full` (kept alive by
        the caller until the job is taken)."""
        jid = _i64()
        _check(_pipe_submit_sample(self._h, full._h, int(m), int(budget),
                                   int(seed) & (2 ** 64 - 1), int(max_steps), C.byref(jid)))
        self._borrowed[jid.value] = full   # freed only once the job is taken
        return jid.value

    def next(self):
        """(job_id, host_ptr, nbytes, info) of the oldest job not yet taken."""
        jid, ptr, nb, info = _i64(), _vp(), _sz(), PipelineInfo()
        rc = _pipe_next(self._h, C.byref(jid), C.byref(ptr), C.byref(nb), C.byref(info))
        self._borrowed.pop(jid.value, None)
        if rc != OK:
            raise GcnError(rc, last_error())
        return jid.value, ptr.value, nb.value, info

    def release(self, job_id):
        _check(_pipe_release(self._h, int(job_id)))

    def close(self, _destroy=_pipe_destroy, _null=_vp):
        # (the library functions are bound as defaults: __del__ may run
        # while the interpreter tears this module's globals down)
        if getattr(self, "_h", None) and self._h.value:
            _destroy(self._h)   # joins the workers: no job reads a graph after this
            self._h = _null()
        self._borrowed = {}
        self._dev_ws = None

    def __del__(self):
        self.close()


def upload_image(host_ptr, nbytes, dev_view, stream=None) -> DGraph:
    """Copy a packed image into a 256-byte-aligned device uint8 view."""
    d = DGraph()
    _check(_upload(_vp(host_ptr), nbytes, _vp(dev_view.data_ptr()), C.byref(d), _stream(stream)))
    return d
