"""ctypes front end of the C oracle (libsolref.so).  Test infrastructure only.

Arrays of bf16 values travel as numpy uint16 bit patterns, contiguous
[B, H, N, D] (the same layout the HIP library uses, so both sides read the
same bytes).
"""
import ctypes
import os

import numpy as np

from . import build as _build

# Head-dim split of the 3D rotary embedding across (t, h, w) and its base,
# as the workload fixes them for head dim 128.
DEFAULT_SPLIT = (32, 48, 48)
ROPE_BASE = 10000.0


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _u16(a):
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 tensors are passed as uint16 bit patterns, got %s" % a.dtype)
    return a


class Oracle:
    """One loaded copy of the C oracle (the tests also load mutated copies)."""

    def __init__(self, path):
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        lib.solref_round_bf16.argtypes = [P, P, i64]
        lib.solref_round_bf16.restype = None
        lib.solref_rope3d_f64.argtypes = [P, P, i64, i32, i32, i32, i32, i32, i32, i32, i32, f64]
        lib.solref_rope3d_f64.restype = None
        lib.solref_rope3d.argtypes = [P, P, i64, i32, i32, i32, i32, i32, i32, i32, i32, f64]
        lib.solref_rope3d.restype = None
        lib.solref_attn_rows.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32,
                                         i32, i32, i32, f64, i32, i32, P, i64, P, i32]
        lib.solref_attn_rows.restype = ctypes.c_int
        lib.solref_num_threads.argtypes = []
        lib.solref_num_threads.restype = ctypes.c_int
        self.lib = lib
        self.path = path

    def num_threads(self) -> int:
        """CPUs in this process's affinity mask (the oracle's default thread count)."""
        return self.lib.solref_num_threads()

    def round_bf16(self, x) -> np.ndarray:
        """float64 -> bf16 bit patterns, round to nearest even, from the double directly."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        y = np.empty(x.shape, dtype=np.uint16)
        self.lib.solref_round_bf16(_ptr(x), _ptr(y), x.size)
        return y

    def rope3d_f64(self, x, T, Hl, Wl, split=DEFAULT_SPLIT, base=ROPE_BASE) -> np.ndarray:
        """Exact-arithmetic (double) 3D rotary embedding of x[..., N, D] (float64)."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        N, D = x.shape[-2], x.shape[-1]
        y = np.empty_like(x)
        self.lib.solref_rope3d_f64(_ptr(x), _ptr(y), x.size // D, N, D, T, Hl, Wl,
                                   split[0], split[1], split[2], base)
        return y

    def rope3d_bf16(self, x_bits, T, Hl, Wl, split=DEFAULT_SPLIT, base=ROPE_BASE) -> np.ndarray:
        """Contract-mode rotation of bf16 bits x[..., N, D]: rotate in double, round once."""
        x = _u16(x_bits)
        N, D = x.shape[-2], x.shape[-1]
        y = np.empty_like(x)
        self.lib.solref_rope3d(_ptr(x), _ptr(y), x.size // D, N, D, T, Hl, Wl,
                               split[0], split[1], split[2], base)
        return y

    def attn_rows(self, q, k, v, T, Hl, Wl, rows=None, rope=True, contract=True,
                  split=DEFAULT_SPLIT, base=ROPE_BASE, threads=0) -> np.ndarray:
        """Attention output (float32) for selected global query rows.

        q, k, v : uint16 bf16 bits, [B, H, N, D]
        rows    : int64 global row ids (b*H + h)*N + i; None = every row
        returns : float32 [len(rows), D] (or [B, H, N, D] when rows is None)
        """
        q, k, v = _u16(q), _u16(k), _u16(v)
        if q.ndim != 4 or q.shape != k.shape or q.shape != v.shape:
            raise ValueError("q, k, v must share one [B, H, N, D] shape")
        B, H, N, D = q.shape
        full = rows is None
        if full:
            rows = np.arange(B * H * N, dtype=np.int64)
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        out = np.empty((rows.size, D), dtype=np.float32)
        rc = self.lib.solref_attn_rows(_ptr(q), _ptr(k), _ptr(v), B, H, N, D, T, Hl, Wl,
                                       split[0], split[1], split[2], base, int(bool(rope)),
                                       int(bool(contract)), _ptr(rows), rows.size, _ptr(out),
                                       threads)
        if rc != 0:
            raise ValueError("oracle rejected the arguments (rc=%d)" % rc)
        return out.reshape(B, H, N, D) if full else out


_default = None


def default() -> Oracle:
    """The oracle built from oracle/solref.c (compiled on first use if needed)."""
    global _default
    if _default is None:
        path = _build.LIB
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
            _build.build()
        _default = Oracle(path)
    return _default


def num_threads():
    return default().num_threads()


def round_bf16(x):
    return default().round_bf16(x)


def rope3d_f64(x, T, Hl, Wl, split=DEFAULT_SPLIT, base=ROPE_BASE):
    return default().rope3d_f64(x, T, Hl, Wl, split, base)


def rope3d_bf16(x_bits, T, Hl, Wl, split=DEFAULT_SPLIT, base=ROPE_BASE):
    return default().rope3d_bf16(x_bits, T, Hl, Wl, split, base)


def attn_rows(q, k, v, T, Hl, Wl, rows=None, rope=True, contract=True,
              split=DEFAULT_SPLIT, base=ROPE_BASE, threads=0):
    return default().attn_rows(q, k, v, T, Hl, Wl, rows, rope, contract, split, base, threads)
