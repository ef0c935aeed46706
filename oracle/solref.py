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
        lib.solref_round_e4m3.argtypes = [P, P, i64]
        lib.solref_round_e4m3.restype = None
        lib.solref_rope3d_f64.argtypes = [P, P, i64, i32, i32, i32, i32, i32, i32, i32, i32, f64]
        lib.solref_rope3d_f64.restype = None
        lib.solref_rope3d.argtypes = [P, P, i64, i32, i32, i32, i32, i32, i32, i32, i32, f64]
        lib.solref_rope3d.restype = None
        lib.solref_attn_rows.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32,
                                         i32, i32, i32, f64, i32, i32, P, i64, P, i32]
        lib.solref_attn_rows.restype = ctypes.c_int
        lib.solref_attn_rows_ex.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32, i32,
                                            i32, i32, i32, i32, i32, i32, f64, i32, i32, i32,
                                            P, P, f64, P, i64, P, i32]
        lib.solref_attn_rows_ex.restype = ctypes.c_int
        lib.solref_attn_rows_sparse.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32, i32,
                                                i32, i32, i32, i32, i32, i32, f64, i32, i32, i32,
                                                P, P, f64, P, i32, i32, P, i64, P, i32]
        lib.solref_attn_rows_sparse.restype = ctypes.c_int
        lib.solref_sparse_route.argtypes = [P, P, i32, i32, i32, i32, i32, i32, i32, i32, i32, f64,
                                            i32, i32, P, P, f64, i32, i32, f64, P, P, P]
        lib.solref_sparse_route.restype = ctypes.c_int
        lib.solref_qknorm_rope3d.argtypes = [P, P, P, i64, i32, i32, i32, i32, i32, i32, i32,
                                             i32, f64, i32, P, f64, i32]
        lib.solref_qknorm_rope3d.restype = None
        lib.solref_encode_qkv.argtypes = [P, P, P, i32, i32, i32, i32, P]
        lib.solref_encode_qkv.restype = ctypes.c_int
        lib.solref_decode_qkv.argtypes = [P, i32, i32, i32, i32, P, P, P]
        lib.solref_decode_qkv.restype = ctypes.c_int
        lib.solref_encode_out_records.argtypes = [P, i64, P]
        lib.solref_encode_out_records.restype = None
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

    def round_e4m3(self, x) -> np.ndarray:
        """float64 -> FP8 E4M3 codes (uint8): round to nearest even, saturating at +-448."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        y = np.empty(x.shape, dtype=np.uint8)
        self.lib.solref_round_e4m3(_ptr(x), _ptr(y), x.size)
        return y

    def encode_qkv(self, q, k, v) -> np.ndarray:
        """Block-INT8 QKV records of bf16 bits q, k, v [B, H, N, 128] (q and k
        as attention consumes them): uint8 [B, N, H, 400]."""
        q, k, v = _u16(q), _u16(k), _u16(v)
        if q.ndim != 4 or q.shape != k.shape or q.shape != v.shape:
            raise ValueError("q, k, v must share one [B, H, N, D] shape")
        B, H, N, D = q.shape
        rec = np.empty((B, N, H, 400), dtype=np.uint8)
        if self.lib.solref_encode_qkv(_ptr(q), _ptr(k), _ptr(v), B, H, N, D, _ptr(rec)) != 0:
            raise ValueError("oracle rejected the arguments")
        return rec

    def encode_out_records(self, x) -> np.ndarray:
        """Block-INT8 output records of float64 rows x [..., 128]: uint8 [..., 144]
        (128 codes, four UE5M3 scales, twelve zero bytes)."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        if x.shape[-1] != 128:
            raise ValueError("rows of 128 values")
        rec = np.empty(x.shape[:-1] + (144,), dtype=np.uint8)
        self.lib.solref_encode_out_records(_ptr(x), x.size // 128, _ptr(rec))
        return rec

    def decode_qkv(self, rec):
        """uint8 records [B, N, H, 400] -> (q, k, v) bf16 bits [B, H, N, 128]."""
        rec = np.ascontiguousarray(rec)
        if rec.dtype != np.uint8 or rec.ndim != 4 or rec.shape[3] != 400:
            raise ValueError("records must be uint8 [B, N, H, 400]")
        B, N, H = rec.shape[:3]
        q, k, v = (np.empty((B, H, N, 128), dtype=np.uint16) for _ in range(3))
        if self.lib.solref_decode_qkv(_ptr(rec), B, H, N, 128, _ptr(q), _ptr(k), _ptr(v)) != 0:
            raise ValueError("oracle rejected the arguments")
        return q, k, v

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

    def qknorm_rope3d(self, x_bits, T, Hl, Wl, gamma, eps, rope=True, contract=True,
                      split=DEFAULT_SPLIT, base=ROPE_BASE) -> np.ndarray:
        """RMS normalisation with weights gamma[D] and eps, then (if rope) the
        3D rotation, of bf16 bits x[..., N, D], all in double.  contract: round
        once to bf16 (uint16 bits out); else float64 out."""
        x = _u16(x_bits)
        N, D = x.shape[-2], x.shape[-1]
        g = np.ascontiguousarray(gamma, dtype=np.float64)
        if g.shape != (D,):
            raise ValueError("gamma must hold D = %d weights" % D)
        if contract:
            y, yf = np.empty_like(x), None
        else:
            y, yf = None, np.empty(x.shape, dtype=np.float64)
        self.lib.solref_qknorm_rope3d(_ptr(x), None if y is None else _ptr(y),
                                      None if yf is None else _ptr(yf), x.size // D, N, D, T, Hl,
                                      Wl, split[0], split[1], split[2], base, int(bool(rope)),
                                      _ptr(g), float(eps), int(bool(contract)))
        return y if contract else yf

    def sparse_route(self, q, k, T, Hl, Wl, tau, qblk=256, kblk=128, rope=True, contract=True,
                     q_gamma=None, k_gamma=None, eps=0.0, split=DEFAULT_SPLIT, base=ROPE_BASE):
        """Block routing of the block-sparse attention for the self-attention of
        q, k [B, H, N, D] (bf16 bits).  Returns (mask uint8 [B, H, nqb, nkb],
        scores float64 [B, H, nqb, nkb], thresholds float64 [B, H, nqb])."""
        q, k = _u16(q), _u16(k)
        if q.ndim != 4 or q.shape != k.shape:
            raise ValueError("q, k must share one [B, H, N, D] shape")
        B, H, N, D = q.shape
        nqb, nkb = -(-N // qblk), -(-N // kblk)
        gq, gk = (None if g is None else np.ascontiguousarray(g, dtype=np.float64)
                  for g in (q_gamma, k_gamma))
        mask = np.empty((B, H, nqb, nkb), dtype=np.uint8)
        scores = np.empty((B, H, nqb, nkb), dtype=np.float64)
        thr = np.empty((B, H, nqb), dtype=np.float64)
        rc = self.lib.solref_sparse_route(
            _ptr(q), _ptr(k), B * H, N, D, T, Hl, Wl, split[0], split[1], split[2], base,
            int(bool(rope)), int(bool(contract)), None if gq is None else _ptr(gq),
            None if gk is None else _ptr(gk), float(eps), qblk, kblk, float(tau), _ptr(mask),
            _ptr(scores), _ptr(thr))
        if rc != 0:
            raise ValueError("oracle rejected the arguments (rc=%d)" % rc)
        return mask, scores, thr

    def attn_rows(self, q, k, v, T, Hl, Wl, rows=None, rope=True, contract=True,
                  split=DEFAULT_SPLIT, base=ROPE_BASE, threads=0, q_gamma=None, k_gamma=None,
                  eps=0.0, kv_grid=None, rope_k=None, block_mask=None, qblk=256,
                  kblk=128) -> np.ndarray:
        """Attention output (float32) for selected global query rows.

        q       : uint16 bf16 bits, [B, H, Nq, D]; k, v: [B, H, Nkv, D]
        T, Hl, Wl : latent grid of the queries (and of the keys unless kv_grid)
        rows    : int64 global row ids (b*H + h)*Nq + i; None = every row
        q_gamma, k_gamma : RMS-normalisation weights [D] of the queries / keys
                  (None: not normalised); eps under the root
        kv_grid : (T, Hl, Wl) of the keys when it differs from the queries'
        rope_k  : rotate the keys (default: as rope)
        block_mask : uint8 [B, H, ceil(Nq/qblk), ceil(Nkv/kblk)]: query i attends
                  only to the keys of the key blocks its query block keeps
        returns : float32 [len(rows), D] (or [B, H, Nq, D] when rows is None)
        """
        q, k, v = _u16(q), _u16(k), _u16(v)
        if q.ndim != 4 or k.ndim != 4 or k.shape != v.shape or q.shape[:2] != k.shape[:2] \
                or q.shape[3] != k.shape[3]:
            raise ValueError("q must be [B, H, Nq, D] and k, v one [B, H, Nkv, D] shape")
        B, H, Nq, D = q.shape
        Nkv = k.shape[2]
        Tk, Hlk, Wlk = kv_grid if kv_grid is not None else (T, Hl, Wl)
        rope_k = rope if rope_k is None else rope_k
        gam = []
        for g in (q_gamma, k_gamma):
            if g is None:
                gam.append(None)
                continue
            g = np.ascontiguousarray(g, dtype=np.float64)
            if g.shape != (D,):
                raise ValueError("gamma must hold D = %d weights" % D)
            gam.append(g)
        full = rows is None
        if full:
            rows = np.arange(B * H * Nq, dtype=np.int64)
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        out = np.empty((rows.size, D), dtype=np.float32)
        common = (_ptr(q), _ptr(k), _ptr(v), B, H, Nq, Nkv, D, T, Hl, Wl, Tk, Hlk, Wlk,
                  split[0], split[1], split[2], base, int(bool(rope)), int(bool(rope_k)),
                  int(bool(contract)), None if gam[0] is None else _ptr(gam[0]),
                  None if gam[1] is None else _ptr(gam[1]), float(eps))
        if block_mask is None:
            rc = self.lib.solref_attn_rows_ex(*common, _ptr(rows), rows.size, _ptr(out), threads)
        else:
            bm = np.ascontiguousarray(block_mask, dtype=np.uint8)
            if bm.shape != (B, H, -(-Nq // qblk), -(-Nkv // kblk)):
                raise ValueError("block_mask must be [B, H, ceil(Nq/qblk), ceil(Nkv/kblk)]")
            rc = self.lib.solref_attn_rows_sparse(*common, _ptr(bm), qblk, kblk, _ptr(rows),
                                                  rows.size, _ptr(out), threads)
        if rc != 0:
            raise ValueError("oracle rejected the arguments (rc=%d)" % rc)
        return out.reshape(B, H, Nq, D) if full else out


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


def round_e4m3(x):
    return default().round_e4m3(x)


def encode_qkv(q, k, v):
    return default().encode_qkv(q, k, v)


def decode_qkv(rec):
    return default().decode_qkv(rec)


def encode_out_records(x):
    return default().encode_out_records(x)


def rope3d_f64(x, T, Hl, Wl, split=DEFAULT_SPLIT, base=ROPE_BASE):
    return default().rope3d_f64(x, T, Hl, Wl, split, base)


def rope3d_bf16(x_bits, T, Hl, Wl, split=DEFAULT_SPLIT, base=ROPE_BASE):
    return default().rope3d_bf16(x_bits, T, Hl, Wl, split, base)


def qknorm_rope3d(x_bits, T, Hl, Wl, gamma, eps, rope=True, contract=True,
                  split=DEFAULT_SPLIT, base=ROPE_BASE):
    return default().qknorm_rope3d(x_bits, T, Hl, Wl, gamma, eps, rope, contract, split, base)


def sparse_route(q, k, T, Hl, Wl, tau, **kw):
    return default().sparse_route(q, k, T, Hl, Wl, tau, **kw)


def attn_rows(q, k, v, T, Hl, Wl, rows=None, rope=True, contract=True,
              split=DEFAULT_SPLIT, base=ROPE_BASE, threads=0, **kw):
    return default().attn_rows(q, k, v, T, Hl, Wl, rows, rope, contract, split, base, threads,
                               **kw)
