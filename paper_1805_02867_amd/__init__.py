"""Python binding of libosoftmax (online-normalizer softmax and fused softmax +
top-k on MI355X).  Argument marshalling only: every step of the computation
runs in the library's HIP kernels, reached through its C ABI
(``include/osoftmax.h``).  PyTorch supplies device memory and the current
stream.  There is no fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libosoftmax.so")

F32, BF16 = 0, 1
NAIVE, SAFE, ONLINE, RESIDENT = 0, 1, 2, 3
RESIDENT_MAX_VEC = 16384
KERNEL_AUTO, KERNEL_ROWS, KERNEL_SPLIT = 0, 1, 2
OK, EINVAL, EUNSUPPORTED, EHIP, ENOMEM, ESCRATCH = 0, 1, 2, 3, 4, 5
NOALLOC_SCRATCH_BYTES = 1 << 20
TOPK_KMAX = 64
PROJ_KMAX = 16
TOPK_ONLINE_FUSED, TOPK_SAFE_FUSED, TOPK_SAFE_UNFUSED, TOPK_ONLINE_UNFUSED, TOPK_VALUES = range(5)
TOPK_ALGOS = {"online_fused": TOPK_ONLINE_FUSED, "safe_fused": TOPK_SAFE_FUSED,
              "safe_unfused": TOPK_SAFE_UNFUSED, "online_unfused": TOPK_ONLINE_UNFUSED,
              "values": TOPK_VALUES}
UNFUSED = (TOPK_SAFE_UNFUSED, TOPK_ONLINE_UNFUSED)

MODES = {"naive": NAIVE, "safe": SAFE, "online": ONLINE, "resident": RESIDENT}
_DTYPES = {torch.float32: F32, torch.bfloat16: BF16}

_lib = None


class OsmError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


def lib() -> ctypes.CDLL:
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                           "(or python paper_1805_02867_amd/build.py)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    L.softmax_fwd.argtypes = [vp, vp, i64, i64, i32, i32, vp]
    L.softmax_fwd.restype = i32
    L.softmax_fwd_ex.argtypes = [vp, vp, i64, i64, i32, i32, i32, i64, vp]
    L.softmax_fwd_ex.restype = i32
    L.softmax_topk.argtypes = [vp, vp, vp, i64, i64, i32, vp]
    L.softmax_topk.restype = i32
    L.softmax_topk_dt.argtypes = [vp, vp, vp, i64, i64, i32, i32, vp]
    L.softmax_topk_dt.restype = i32
    L.softmax_topk_ex.argtypes = [vp, vp, vp, i64, i64, i32, i32, i32, i64, vp]
    L.softmax_topk_ex.restype = i32
    L.softmax_topk_ex_noalloc.argtypes = [vp, vp, vp, i64, i64, i32, i32, i32, i64, vp]
    L.softmax_topk_ex_noalloc.restype = i32
    L.softmax_topk_algo.argtypes = [vp, vp, vp, vp, i64, i64, i32, i32, i32, i32, i64, vp]
    L.softmax_topk_algo.restype = i32
    L.topk_fwd.argtypes = [vp, vp, vp, i64, i64, i32, i32, vp]
    L.topk_fwd.restype = i32
    L.osm_topk_plan.argtypes = [i64, i64, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i64)]
    L.osm_topk_plan.restype = i32
    L.proj_fwd.argtypes = [vp, vp, vp, i64, i64, i64, vp]
    L.proj_fwd.restype = i32
    L.proj_softmax_topk.argtypes = [vp, vp, vp, vp, i64, i64, i64, i32, vp]
    L.proj_softmax_topk.restype = i32
    L.osm_plan.argtypes = [i64, i64, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i64)]
    L.osm_plan.restype = i32
    L.osm_stream_release.argtypes = [vp]
    L.osm_stream_release.restype = i32
    L.osm_ref_stream.argtypes = [i32, vp, vp, i64, vp]
    L.osm_ref_stream.restype = i32
    L.osm_status_string.argtypes = [i32]
    L.osm_status_string.restype = ctypes.c_char_p
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().osm_status_string(int(status)).decode()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _batch(x: torch.Tensor, name: str = "x"):
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if x.dtype not in _DTYPES:
        raise ValueError(f"{name} must be float32 or bfloat16, got {x.dtype}")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if x.dim() == 1:
        return 1, x.shape[0]
    if x.dim() != 2:
        raise ValueError(f"{name} must be 1-D or 2-D (N x V)")
    return x.shape[0], x.shape[1]


def _mode(mode) -> int:
    if isinstance(mode, str):
        if mode not in MODES:
            raise ValueError(f"mode must be one of {sorted(MODES)}")
        return MODES[mode]
    return int(mode)


def softmax_fwd(x: torch.Tensor, y: torch.Tensor | None = None, mode="online",
                stream=None, kernel: int = KERNEL_AUTO, param: int = 0) -> torch.Tensor:
    """y = Softmax(x) per row via ``softmax_fwd`` / ``softmax_fwd_ex``."""
    N, V = _batch(x)
    if y is None:
        y = torch.empty_like(x)
    else:
        Ny, Vy = _batch(y, "y")
        if (Ny, Vy) != (N, V) or y.dtype != x.dtype or y.device != x.device:
            raise ValueError("y must match x in shape, dtype and device")
    dt = _DTYPES[x.dtype]
    if kernel == KERNEL_AUTO:
        rc = lib().softmax_fwd(x.data_ptr(), y.data_ptr(), N, V, dt, _mode(mode),
                               _stream(stream))
    else:
        rc = lib().softmax_fwd_ex(x.data_ptr(), y.data_ptr(), N, V, dt, _mode(mode),
                                  int(kernel), int(param), _stream(stream))
    if rc != OK:
        raise OsmError(rc, "softmax_fwd")
    return y


def _topk_outputs(x, N, K, vals, idx):
    if vals is None:
        vals = torch.empty((N, K), dtype=torch.float32, device=x.device)
    if idx is None:
        idx = torch.empty((N, K), dtype=torch.int32, device=x.device)
    for t, dt, nm in ((vals, torch.float32, "vals"), (idx, torch.int32, "idx")):
        if (t.dtype != dt or not t.is_contiguous() or t.numel() != N * K
                or t.device != x.device):
            raise ValueError(f"{nm} must be a contiguous {dt} tensor of N*K elements on x's device")
    return vals, idx


def _algo(algo) -> int:
    if isinstance(algo, str):
        if algo not in TOPK_ALGOS:
            raise ValueError(f"algo must be one of {sorted(TOPK_ALGOS)}")
        return TOPK_ALGOS[algo]
    return int(algo)


def softmax_topk(x: torch.Tensor, K: int, vals: torch.Tensor | None = None,
                 idx: torch.Tensor | None = None, stream=None, kernel: int = KERNEL_AUTO,
                 param: int = 0, algo="online_fused", y: torch.Tensor | None = None):
    """(vals, idx) = softmax + top-k per row.

    The default (Alg. 4, one pass) goes through ``softmax_topk`` (binary32
    rows), ``softmax_topk_dt`` (bfloat16 rows) or, with an explicit kernel,
    ``softmax_topk_ex``.  Another ``algo`` (see ``TOPK_ALGOS``) goes through
    ``softmax_topk_algo``; the unfused ones write the softmax into ``y``
    (allocated here when not given)."""
    N, V = _batch(x)
    vals, idx = _topk_outputs(x, N, K, vals, idx)
    a = _algo(algo)
    dt = _DTYPES[x.dtype]
    if a != TOPK_ONLINE_FUSED:
        if a in UNFUSED:
            if y is None:
                y = torch.empty_like(x)
            elif (_batch(y, "y") != (N, V) or y.dtype != x.dtype or y.device != x.device):
                raise ValueError("y must match x in shape, dtype and device")
        yp = y.data_ptr() if (a in UNFUSED) else None
        rc = lib().softmax_topk_algo(x.data_ptr(), yp, vals.data_ptr(), idx.data_ptr(), N, V,
                                     int(K), dt, a, int(kernel), int(param), _stream(stream))
    elif kernel != KERNEL_AUTO:
        rc = lib().softmax_topk_ex(x.data_ptr(), vals.data_ptr(), idx.data_ptr(), N, V,
                                   int(K), dt, int(kernel), int(param), _stream(stream))
    elif x.dtype == torch.float32:
        rc = lib().softmax_topk(x.data_ptr(), vals.data_ptr(), idx.data_ptr(), N, V, int(K),
                                _stream(stream))
    else:
        rc = lib().softmax_topk_dt(x.data_ptr(), vals.data_ptr(), idx.data_ptr(), N, V,
                                   int(K), dt, _stream(stream))
    if rc != OK:
        raise OsmError(rc, "softmax_topk")
    return vals, idx


softmax_topk_dt = softmax_topk


def softmax_topk_noalloc(x: torch.Tensor, K: int, vals: torch.Tensor | None = None,
                         idx: torch.Tensor | None = None, stream=None,
                         kernel: int = KERNEL_AUTO, param: int = 0):
    """(vals, idx) as softmax_topk, through ``softmax_topk_ex_noalloc``: the
    library allocates nothing (split partials in its fixed per-device scratch
    array).  Calls that can overlap on one device race on that array."""
    N, V = _batch(x)
    vals, idx = _topk_outputs(x, N, K, vals, idx)
    rc = lib().softmax_topk_ex_noalloc(x.data_ptr(), vals.data_ptr(), idx.data_ptr(), N, V,
                                       int(K), _DTYPES[x.dtype], int(kernel), int(param),
                                       _stream(stream))
    if rc != OK:
        raise OsmError(rc, "softmax_topk_ex_noalloc")
    return vals, idx


def topk(x: torch.Tensor, K: int, vals: torch.Tensor | None = None,
         idx: torch.Tensor | None = None, stream=None):
    """(vals, idx) = the K largest elements of each row and their indices
    (``topk_fwd``); larger first, equal values in increasing index order."""
    N, V = _batch(x)
    vals, idx = _topk_outputs(x, N, K, vals, idx)
    rc = lib().topk_fwd(x.data_ptr(), vals.data_ptr(), idx.data_ptr(), N, V, int(K),
                        _DTYPES[x.dtype], _stream(stream))
    if rc != OK:
        raise OsmError(rc, "topk_fwd")
    return vals, idx


def stream_release(stream=None) -> None:
    """Frees the scratch the library keeps for `stream` (``osm_stream_release``),
    in stream order; call before destroying a stream that used the library."""
    rc = lib().osm_stream_release(_stream(stream))
    if rc != OK:
        raise OsmError(rc, "osm_stream_release")


def topk_plan(N: int, V: int, K: int, dtype=torch.float32):
    """(kernel, param) that the top-k entry points use for this shape."""
    k = ctypes.c_int()
    p = ctypes.c_int64()
    dt = _DTYPES[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    rc = lib().osm_topk_plan(int(N), int(V), dt, int(K), ctypes.byref(k), ctypes.byref(p))
    if rc != OK:
        raise OsmError(rc, "osm_topk_plan")
    return k.value, p.value


def plan(N: int, V: int, dtype=torch.float32, mode="online"):
    """(kernel, param) that softmax_fwd uses for this shape (``osm_plan``)."""
    k = ctypes.c_int()
    p = ctypes.c_int64()
    dt = _DTYPES[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    rc = lib().osm_plan(int(N), int(V), dt, _mode(mode), ctypes.byref(k), ctypes.byref(p))
    if rc != OK:
        raise OsmError(rc, "osm_plan")
    return k.value, p.value


def _proj_inputs(h: torch.Tensor, w: torch.Tensor):
    for t, nm in ((h, "h"), (w, "w")):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.bfloat16:
            raise ValueError(f"{nm} must be a bfloat16 CUDA (HIP) tensor")
        if t.dim() != 2 or not t.is_contiguous():
            raise ValueError(f"{nm} must be a contiguous 2-D tensor")
    if h.shape[1] != w.shape[1]:
        raise ValueError("h (N x H) and w (V x H) must have the same H")
    return h.shape[0], h.shape[1], w.shape[0]


def ref_stream(op: str, x: torch.Tensor, y: torch.Tensor, stream=None) -> None:
    """Reference streaming kernel for measurement (``osm_ref_stream``):
    op "read" reads all of x (y: a sink of at least 1 KB), "copy" copies x
    to y (same size).  Nothing of the method; the plain rates the other
    kernels are judged against."""
    if op not in ("read", "copy"):
        raise ValueError("op must be 'read' or 'copy'")
    n = x.numel() * x.element_size()
    if op == "copy" and y.numel() * y.element_size() < n:
        raise ValueError("y is smaller than x")
    rc = lib().osm_ref_stream(0 if op == "read" else 1, x.data_ptr(), y.data_ptr(), n,
                              _stream(stream))
    if rc != OK:
        raise OsmError(rc, "osm_ref_stream")


def proj(h: torch.Tensor, w: torch.Tensor, out: torch.Tensor | None = None, stream=None):
    """logits = h . w^T (``proj_fwd``): h N x H and w V x H bfloat16, binary32 out."""
    N, H, V = _proj_inputs(h, w)
    if out is None:
        out = torch.empty((N, V), dtype=torch.float32, device=h.device)
    elif (out.dtype != torch.float32 or not out.is_contiguous() or out.numel() != N * V):
        raise ValueError("out must be a contiguous float32 tensor of N*V elements")
    rc = lib().proj_fwd(h.data_ptr(), w.data_ptr(), out.data_ptr(), N, H, V, _stream(stream))
    if rc != OK:
        raise OsmError(rc, "proj_fwd")
    return out


def proj_softmax_topk(h: torch.Tensor, w: torch.Tensor, K: int, vals: torch.Tensor | None = None,
                      idx: torch.Tensor | None = None, stream=None):
    """(vals, idx) = top-k of softmax(h . w^T) per row without writing the
    logits (``proj_softmax_topk``)."""
    N, H, V = _proj_inputs(h, w)
    vals, idx = _topk_outputs(h, N, K, vals, idx)
    rc = lib().proj_softmax_topk(h.data_ptr(), w.data_ptr(), vals.data_ptr(), idx.data_ptr(),
                                 N, H, V, int(K), _stream(stream))
    if rc != OK:
        raise OsmError(rc, "proj_softmax_topk")
    return vals, idx
