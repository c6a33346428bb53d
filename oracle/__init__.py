"""Reference oracle for row-wise softmax and softmax+top-k, in binary64 on the CPU.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are its only users.  It shares no code with the HIP library
and the library never calls it.  The arithmetic lives in ``oracle.c`` (plain C,
binary64, libm ``exp``); this module only marshals numpy arrays into it.

Functions (all take row-major ``N x V`` numpy arrays: float32, float64, or
bfloat16 given as raw ``uint16`` bit patterns with ``dtype="bf16"``):

* :func:`softmax`        -- the safe formula, Eq. 2 (Section 2).
* :func:`softmax_naive`  -- the unprotected formula, Eq. 1 / Alg. 1.
* :func:`md_direct`      -- (m, d) by Theorem 1's closed form.
* :func:`md_online`      -- (m, d) by the online recurrence of Alg. 3.
* :func:`md_combine`     -- the merge operator of Eq. 4 (Section 3.1).
* :func:`topk`           -- Eq. 5 by a full sort, ties to the lower index.
* :func:`topk_select`    -- Eq. 5 by K selection passes, with the online
  normalizer of Alg. 3 (a second route to :func:`topk`, used to pin it).
* :func:`bf16_round`     -- binary64 -> bfloat16, round to nearest even.
* :func:`bf16_to_f64`    -- bfloat16 patterns -> binary64, exactly.
* :func:`proj`           -- the projection ahead of the softmax (Section 1):
  logits = h . w^T in binary64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

F32, BF16, F64 = 0, 1, 2
_DT = {"f32": F32, "bf16": BF16, "f64": F64}


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile ``oracle.c`` (or another copy of it) with gcc into a shared
    library: IEEE binary64, no fast-math, no FMA contraction."""
    tmp = out + ".tmp"
    subprocess.check_call([
        "gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
        "-Wall", "-Wextra", "-shared", "-fPIC", src, "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


class Oracle:
    """ctypes view of one build of ``oracle.c``."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        for name in ("orc_softmax", "orc_softmax_naive"):
            getattr(lib, name).argtypes = [vp, i32, i64, i64, vp]
            getattr(lib, name).restype = i32
        for name in ("orc_md_direct", "orc_md_online"):
            getattr(lib, name).argtypes = [vp, i32, i64, i64, vp, vp]
            getattr(lib, name).restype = i32
        for name in ("orc_topk", "orc_topk_select"):
            getattr(lib, name).argtypes = [vp, i32, i64, i64, i32, vp, vp]
            getattr(lib, name).restype = i32
        lib.orc_proj.argtypes = [vp, i32, vp, i32, i64, i64, i64, vp]
        lib.orc_proj.restype = i32
        lib.orc_md_combine.argtypes = [ctypes.c_double] * 4 + [vp, vp]
        lib.orc_md_combine.restype = None
        lib.orc_bf16_round.argtypes = [vp, i64, vp]
        lib.orc_bf16_round.restype = None
        lib.orc_bf16_widen.argtypes = [vp, i64, vp]
        lib.orc_bf16_widen.restype = None
        lib.orc_set_threads.argtypes = [i32]
        lib.orc_set_threads.restype = None
        lib.orc_get_threads.argtypes = []
        lib.orc_get_threads.restype = i32
        self.lib = lib
        self.path = path

    def set_threads(self, n: int) -> None:
        """Number of OpenMP threads per call (0 = OpenMP default)."""
        self.lib.orc_set_threads(int(n))

    def threads(self) -> int:
        """Threads the oracle's parallel regions use."""
        return int(self.lib.orc_get_threads())

    def softmax(self, x: np.ndarray, dtype: str | None = None) -> np.ndarray:
        """Eq. 2: y_i = e^{x_i - max x} / sum_j e^{x_j - max x}, binary64."""
        x, dt, n, v = _prep(x, dtype)
        y = np.empty((n, v), np.float64)
        _check(self.lib.orc_softmax(_ptr(x), dt, n, v, _ptr(y)), "softmax")
        return y

    def softmax_naive(self, x: np.ndarray, dtype: str | None = None) -> np.ndarray:
        """Eq. 1 as Alg. 1: y_i = e^{x_i} / sum_j e^{x_j}, binary64 (can overflow)."""
        x, dt, n, v = _prep(x, dtype)
        y = np.empty((n, v), np.float64)
        _check(self.lib.orc_softmax_naive(_ptr(x), dt, n, v, _ptr(y)), "softmax_naive")
        return y

    def md_direct(self, x: np.ndarray, dtype: str | None = None):
        """Theorem 1's closed form: m = max x, d = sum e^{x - m}; per row."""
        x, dt, n, v = _prep(x, dtype)
        m = np.empty(n, np.float64)
        d = np.empty(n, np.float64)
        _check(self.lib.orc_md_direct(_ptr(x), dt, n, v, _ptr(m), _ptr(d)), "md_direct")
        return m, d

    def md_online(self, x: np.ndarray, dtype: str | None = None):
        """Alg. 3's online recurrence, element by element; per row."""
        x, dt, n, v = _prep(x, dtype)
        m = np.empty(n, np.float64)
        d = np.empty(n, np.float64)
        _check(self.lib.orc_md_online(_ptr(x), dt, n, v, _ptr(m), _ptr(d)), "md_online")
        return m, d

    def md_combine(self, a, b):
        """Eq. 4: (m_i, d_i) (+) (m_j, d_j), with (-inf, 0) as identity."""
        m = ctypes.c_double()
        d = ctypes.c_double()
        self.lib.orc_md_combine(float(a[0]), float(a[1]), float(b[0]), float(b[1]),
                                ctypes.byref(m), ctypes.byref(d))
        return (m.value, d.value)

    def topk(self, x: np.ndarray, k: int, dtype: str | None = None):
        """Eq. 5 by full sort under (x desc, index asc); returns (v, z) with
        v float64 [N, K] = softmax values at z, z int32 [N, K], 0-based."""
        x, dt, n, v = _prep(x, dtype)
        vals = np.empty((n, k), np.float64)
        idx = np.empty((n, k), np.int32)
        _check(self.lib.orc_topk(_ptr(x), dt, n, v, int(k), _ptr(vals), _ptr(idx)), "topk")
        return vals, idx

    def topk_select(self, x: np.ndarray, k: int, dtype: str | None = None):
        """Eq. 5 by K selection passes (each the first element, under (x desc,
        index asc), ranked after the previous pick), values from the online
        pair of Alg. 3; returns (v, z) like :meth:`topk`."""
        x, dt, n, v = _prep(x, dtype)
        vals = np.empty((n, k), np.float64)
        idx = np.empty((n, k), np.int32)
        _check(self.lib.orc_topk_select(_ptr(x), dt, n, v, int(k), _ptr(vals), _ptr(idx)),
               "topk_select")
        return vals, idx

    def proj(self, h: np.ndarray, w: np.ndarray, hdtype: str | None = None,
             wdtype: str | None = None) -> np.ndarray:
        """logits[n][v] = sum_k h[n][k] w[v][k] in binary64 (h: N x H,
        w: V x H; each float32, float64 or bfloat16 patterns)."""
        h, hdt, n, hh = _prep(h, hdtype)
        w, wdt, v, hw = _prep(w, wdtype)
        if hh != hw:
            raise ValueError("h and w must have the same number of columns")
        out = np.empty((n, v), np.float64)
        _check(self.lib.orc_proj(_ptr(h), hdt, _ptr(w), wdt, n, hh, v, _ptr(out)), "proj")
        return out

    def bf16_round(self, y: np.ndarray) -> np.ndarray:
        """binary64 -> bfloat16 bit patterns (uint16), round to nearest, ties to
        even, in a single rounding step."""
        y = np.ascontiguousarray(y, dtype=np.float64)
        out = np.empty(y.shape, np.uint16)
        self.lib.orc_bf16_round(_ptr(y), y.size, _ptr(out))
        return out

    def bf16_to_f64(self, bits: np.ndarray) -> np.ndarray:
        """bfloat16 bit patterns (uint16) -> binary64, exactly (the widening
        of every bfloat16 input of the oracle)."""
        b = np.ascontiguousarray(bits, dtype=np.uint16)
        out = np.empty(b.shape, np.float64)
        self.lib.orc_bf16_widen(_ptr(b), b.size, _ptr(out))
        return out


_default: Oracle | None = None


def _get() -> Oracle:
    global _default
    if _default is None:
        if not os.path.exists(_LIB_PATH):
            build()
        _default = Oracle(_LIB_PATH)
    return _default


def load(path: str) -> Oracle:
    """An :class:`Oracle` over another build of ``oracle.c``."""
    return Oracle(path)


def _prep(x: np.ndarray, dtype: str | None):
    if x.ndim == 1:
        x = x[None, :]
    if x.ndim != 2:
        raise ValueError("x must be 1-D or 2-D")
    if dtype is None:
        if x.dtype == np.float32:
            dtype = "f32"
        elif x.dtype == np.float64:
            dtype = "f64"
        else:
            raise ValueError("pass dtype='bf16' for uint16 bfloat16 patterns")
    want = {"f32": np.float32, "f64": np.float64, "bf16": np.uint16}[dtype]
    if x.dtype != want:
        raise ValueError(f"dtype {dtype} needs a {np.dtype(want)} array, got {x.dtype}")
    x = np.ascontiguousarray(x)
    n, v = x.shape
    if v < 1:
        raise ValueError("V must be >= 1")
    return x, _DT[dtype], n, v


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with status {rc}")


def set_threads(n: int) -> None:
    _get().set_threads(n)


def threads() -> int:
    return _get().threads()


def softmax(x, dtype=None):
    return _get().softmax(x, dtype)


def softmax_naive(x, dtype=None):
    return _get().softmax_naive(x, dtype)


def md_direct(x, dtype=None):
    return _get().md_direct(x, dtype)


def md_online(x, dtype=None):
    return _get().md_online(x, dtype)


def md_combine(a, b):
    return _get().md_combine(a, b)


def topk(x, k, dtype=None):
    return _get().topk(x, k, dtype)


def topk_select(x, k, dtype=None):
    return _get().topk_select(x, k, dtype)


def bf16_round(y):
    return _get().bf16_round(y)


def proj(h, w, hdtype=None, wdtype=None):
    return _get().proj(h, w, hdtype, wdtype)


def bf16_to_f64(bits):
    return _get().bf16_to_f64(bits)
