"""Python binding of libsol.so (include/sol.h): argument marshalling only.

The ``sol_*`` functions mirror the C ABI one to one (device pointers and
streams as integers).  The other functions (``rope3d_table``, ``rope3d``,
``qknorm_rope3d``, ``attn_fwd``, ``prepare_kv[_ex]``, ``attn_fwd_prepared[_ex]``,
``qkv_encode``, ``attn_fwd_records`` ...) take torch tensors and pass their device pointers and the current HIP
stream.  Every
step of the computation runs in the HIP library; there is no fallback: if
libsol.so is missing or fails to load, every call raises.
"""
import ctypes
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsol.so")

SOL_OK = 0
SOL_ERR_INVALID_ARG = -1
SOL_ERR_UNSUPPORTED = -2
SOL_ERR_HIP = -3
SOL_RANGE_Q = 1
SOL_RANGE_K = 2
SOL_RANGE_V = 4
SOL_RANGE_OUT = 8
SOL_OUT_BF16 = 0
SOL_OUT_FP8_E4M3 = 1
SOL_OUT_INT8_RECORDS = 2
OUT_RECORD_BYTES = 144
HEAD_DIM = 128
ROPE_BASE = 10000.0

_lib = None


class SolError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(msg)
        self.status = status


def lib():
    """Load libsol.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libsol.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, i32, sz, f64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_double
        L.sol_rope3d_table_floats.argtypes = [i32, i32, i32, i32]
        L.sol_rope3d_table_floats.restype = sz
        L.sol_rope3d_table.argtypes = [P, sz, i32, i32, i32, i32, f64]
        L.sol_rope3d_table.restype = i32
        L.sol_rope3d_table_floats_ex.argtypes = [i32] * 7
        L.sol_rope3d_table_floats_ex.restype = sz
        L.sol_rope3d_table_ex.argtypes = [P, sz] + [i32] * 7 + [f64]
        L.sol_rope3d_table_ex.restype = i32
        L.sol_rope3d.argtypes = [P, P, i32, i32, i32, i32, i32, i32, i32, P, P]
        L.sol_rope3d.restype = i32
        L.sol_attn_fwd.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, i32, P, P]
        L.sol_attn_fwd.restype = i32
        L.sol_attn_fwd_plan.argtypes = [i32, i32, i32, i32]
        L.sol_attn_fwd_plan.restype = i32
        L.sol_prepare_kv.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, i32, P, P]
        L.sol_prepare_kv.restype = i32
        L.sol_attn_fwd_prepared.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, i32, P, P]
        L.sol_attn_fwd_prepared.restype = i32
        L.sol_prepared_kv_bytes.argtypes = [i32, i32, i32, i32]
        L.sol_prepared_kv_bytes.restype = sz
        L.sol_attn_workspace_bytes.argtypes = [i32, i32, i32, i32]
        L.sol_attn_workspace_bytes.restype = sz
        L.sol_attn_fwd_ws.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, i32, P, P, sz, P]
        L.sol_attn_fwd_ws.restype = i32
        L.sol_attn_fwd_noalloc.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, i32, P, P]
        L.sol_attn_fwd_noalloc.restype = i32
        f32 = ctypes.c_float
        L.sol_qknorm_rope3d.argtypes = [P, P] + [i32] * 10 + [P, P, f32, P]
        L.sol_qknorm_rope3d.restype = i32
        L.sol_prepare_kv_ex.argtypes = [P, P, P, P] + [i32] * 12 + [P, P, f32, P]
        L.sol_prepare_kv_ex.restype = i32
        L.sol_attn_fwd_prepared_ex.argtypes = [P, P, P, P] + [i32] * 11 + [P, P, f32, i32, P]
        L.sol_attn_fwd_prepared_ex.restype = i32
        L.sol_sparse_workspace_bytes.argtypes = [i32, i32, i32, i32]
        L.sol_sparse_workspace_bytes.restype = sz
        L.sol_sparse_route.argtypes = [P, P] + [i32] * 10 + [P, P, f32, f32, P, sz, P]
        L.sol_sparse_route.restype = i32
        L.sol_attn_fwd_sparse.argtypes = [P, P, P, P] + [i32] * 10 + [P, P, f32, P, sz, i32, P]
        L.sol_attn_fwd_sparse.restype = i32
        L.sol_qkv_record_bytes.argtypes = [i32, i32, i32]
        L.sol_qkv_record_bytes.restype = sz
        L.sol_qkv_encode.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, i32, P, P, P, f32, P]
        L.sol_qkv_encode.restype = i32
        i64 = ctypes.c_int64
        L.sol_qkv_encode_strided.argtypes = [P, P, P, i64, i64, i64, P, i32, i32, i32, i32, i32, i32,
                                             i32, P, P, P, f32, P]
        L.sol_qkv_encode_strided.restype = i32
        L.sol_qkv_decode.argtypes = [P, P, P, P, i32, i32, i32, i32, P]
        L.sol_qkv_decode.restype = i32
        L.sol_prepare_kv_records.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, P]
        L.sol_prepare_kv_records.restype = i32
        L.sol_attn_fwd_records.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, i32, P]
        L.sol_attn_fwd_records.restype = i32
        L.sol_mfma_probe.argtypes = [P, P, i32, i32, P]
        L.sol_mfma_probe.restype = i32
        L.sol_range_status.argtypes = [ctypes.POINTER(ctypes.c_uint), i32]
        L.sol_range_status.restype = i32
        L.sol_status_string.argtypes = [i32]
        L.sol_status_string.restype = ctypes.c_char_p
        L.sol_last_error.argtypes = []
        L.sol_last_error.restype = ctypes.c_char_p
        L.sol_version.argtypes = []
        L.sol_version.restype = i32
        _lib = L
    return _lib


# ---------------------------------------------------------------- raw C ABI

def sol_rope3d_table_floats(D, T, Hl, Wl):
    return lib().sol_rope3d_table_floats(D, T, Hl, Wl)


def sol_rope3d_table(host_tab, n_floats, D, T, Hl, Wl, base):
    return lib().sol_rope3d_table(host_tab, n_floats, D, T, Hl, Wl, base)


def sol_rope3d_table_floats_ex(D, T, Hl, Wl, dt, dh, dw):
    return lib().sol_rope3d_table_floats_ex(D, T, Hl, Wl, dt, dh, dw)


def sol_rope3d_table_ex(host_tab, n_floats, D, T, Hl, Wl, dt, dh, dw, base):
    return lib().sol_rope3d_table_ex(host_tab, n_floats, D, T, Hl, Wl, dt, dh, dw, base)


def sol_rope3d(x, y, B, H, N, D, T, Hl, Wl, rope_tab, stream):
    return lib().sol_rope3d(x, y, B, H, N, D, T, Hl, Wl, rope_tab, stream)


def sol_qknorm_rope3d(x, y, B, H, N, D, T, Hl, Wl, dt, dh, dw, rope_tab, gamma, eps, stream):
    return lib().sol_qknorm_rope3d(x, y, B, H, N, D, T, Hl, Wl, dt, dh, dw, rope_tab, gamma, eps,
                                   stream)


def sol_prepare_kv_ex(k, v, k_prep, v_prep, B, H, N, key0, n_kv, D, T, Hl, Wl, dt, dh, dw, rope_tab,
                      gamma, eps, stream):
    return lib().sol_prepare_kv_ex(k, v, k_prep, v_prep, B, H, N, key0, n_kv, D, T, Hl, Wl, dt, dh,
                                   dw, rope_tab, gamma, eps, stream)


def sol_attn_fwd_prepared_ex(q, k_prep, v_prep, out, B, H, N, n_kv, D, T, Hl, Wl, dt, dh, dw,
                             rope_tab, gamma, eps, out_format, stream):
    return lib().sol_attn_fwd_prepared_ex(q, k_prep, v_prep, out, B, H, N, n_kv, D, T, Hl, Wl, dt,
                                          dh, dw, rope_tab, gamma, eps, out_format, stream)


def sol_sparse_workspace_bytes(B, H, N, D):
    return lib().sol_sparse_workspace_bytes(B, H, N, D)


def sol_sparse_route(q, k_prep, B, H, N, D, T, Hl, Wl, dt, dh, dw, rope_tab, gamma, eps, tau,
                     workspace, workspace_bytes, stream):
    return lib().sol_sparse_route(q, k_prep, B, H, N, D, T, Hl, Wl, dt, dh, dw, rope_tab, gamma, eps,
                                  tau, workspace, workspace_bytes, stream)


def sol_attn_fwd_sparse(q, k_prep, v_prep, out, B, H, N, D, T, Hl, Wl, dt, dh, dw, rope_tab, gamma,
                        eps, workspace, workspace_bytes, out_format, stream):
    return lib().sol_attn_fwd_sparse(q, k_prep, v_prep, out, B, H, N, D, T, Hl, Wl, dt, dh, dw,
                                     rope_tab, gamma, eps, workspace, workspace_bytes, out_format,
                                     stream)


def sol_attn_fwd(q, k, v, out, B, H, N, D, T, Hl, Wl, rope_tab, stream):
    return lib().sol_attn_fwd(q, k, v, out, B, H, N, D, T, Hl, Wl, rope_tab, stream)


def sol_attn_fwd_plan(B, H, N, D):
    return lib().sol_attn_fwd_plan(B, H, N, D)


def sol_prepare_kv(k, v, k_prep, v_prep, B, H, N, D, T, Hl, Wl, rope_tab, stream):
    return lib().sol_prepare_kv(k, v, k_prep, v_prep, B, H, N, D, T, Hl, Wl, rope_tab, stream)


def sol_prepared_kv_bytes(B, H, N, D):
    return lib().sol_prepared_kv_bytes(B, H, N, D)


def sol_attn_fwd_prepared(q, k_prep, v_prep, out, B, H, N, D, T, Hl, Wl, rope_tab, stream):
    return lib().sol_attn_fwd_prepared(q, k_prep, v_prep, out, B, H, N, D, T, Hl, Wl, rope_tab, stream)


def sol_attn_workspace_bytes(B, H, N, D):
    return lib().sol_attn_workspace_bytes(B, H, N, D)


def sol_attn_fwd_ws(q, k, v, out, B, H, N, D, T, Hl, Wl, rope_tab, workspace, workspace_bytes, stream):
    return lib().sol_attn_fwd_ws(q, k, v, out, B, H, N, D, T, Hl, Wl, rope_tab, workspace,
                                 workspace_bytes, stream)


def sol_attn_fwd_noalloc(q, k, v, out, B, H, N, D, T, Hl, Wl, rope_tab, stream):
    return lib().sol_attn_fwd_noalloc(q, k, v, out, B, H, N, D, T, Hl, Wl, rope_tab, stream)


def sol_qkv_record_bytes(B, H, N):
    return lib().sol_qkv_record_bytes(B, H, N)


def sol_qkv_encode(q, k, v, rec, B, H, N, D, T, Hl, Wl, rope_tab, q_gamma, k_gamma, eps, stream):
    return lib().sol_qkv_encode(q, k, v, rec, B, H, N, D, T, Hl, Wl, rope_tab, q_gamma, k_gamma, eps,
                                stream)


def sol_qkv_encode_strided(q, k, v, stride_b, stride_h, stride_n, rec, B, H, N, D, T, Hl, Wl,
                           rope_tab, q_gamma, k_gamma, eps, stream):
    return lib().sol_qkv_encode_strided(q, k, v, stride_b, stride_h, stride_n, rec, B, H, N, D, T, Hl,
                                        Wl, rope_tab, q_gamma, k_gamma, eps, stream)


def sol_qkv_decode(rec, q, k, v, B, H, N, D, stream):
    return lib().sol_qkv_decode(rec, q, k, v, B, H, N, D, stream)


def sol_prepare_kv_records(rec, k_prep, v_prep, B, H, N, key0, n_kv, D, stream):
    return lib().sol_prepare_kv_records(rec, k_prep, v_prep, B, H, N, key0, n_kv, D, stream)


def sol_attn_fwd_records(rec, k_prep, v_prep, out, B, H, N, n_kv, D, out_format, stream):
    return lib().sol_attn_fwd_records(rec, k_prep, v_prep, out, B, H, N, n_kv, D, out_format, stream)


def sol_mfma_probe(operands, out, workgroups, iters, stream):
    return lib().sol_mfma_probe(operands, out, workgroups, iters, stream)


def sol_range_status(flags, clear):
    return lib().sol_range_status(flags, clear)


def sol_status_string(status):
    return lib().sol_status_string(status).decode()


def sol_last_error():
    return lib().sol_last_error().decode()


def sol_version():
    return lib().sol_version()


def check(status):
    """Raise SolError for a non-zero status, with the library's message."""
    if status != SOL_OK:
        raise SolError(status, "%s: %s" % (sol_status_string(status), sol_last_error()))


# ------------------------------------------------------- torch marshalling

DEFAULT_SPLIT = (HEAD_DIM // 4, 3 * HEAD_DIM // 8, 3 * HEAD_DIM // 8)


def _split(split):
    """(dt, dh, dw): the head dims turned by t, h, w (None: the default 32/48/48)."""
    if split is None:
        return DEFAULT_SPLIT
    dt, dh, dw = (int(x) for x in split)
    return dt, dh, dw


def rope3d_table_host(T, Hl, Wl, D=HEAD_DIM, base=ROPE_BASE, split=None) -> np.ndarray:
    """The rotary table of grid T x Hl x Wl and split (dt, dh, dw) as a host
    float32 array (built by the library)."""
    dt, dh, dw = _split(split)
    n = sol_rope3d_table_floats_ex(D, T, Hl, Wl, dt, dh, dw)
    tab = np.zeros(max(n, 4), dtype=np.float32)
    check(sol_rope3d_table_ex(tab.ctypes.data_as(ctypes.c_void_p), n, D, T, Hl, Wl, dt, dh, dw, base))
    return tab


def rope3d_table(T, Hl, Wl, D=HEAD_DIM, base=ROPE_BASE, device="cuda", split=None) -> torch.Tensor:
    """The rotary table, copied to `device` (float32)."""
    return torch.from_numpy(rope3d_table_host(T, Hl, Wl, D, base, split)).to(device)


def _stream(t):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _check_tensor(name, t, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != torch.bfloat16:
        raise TypeError("%s must be bfloat16, got %s" % (name, t.dtype))
    if not t.is_cuda:
        raise ValueError("%s must be on a HIP device" % name)
    if t.dim() != 4 or not t.is_contiguous():
        raise ValueError("%s must be a contiguous [B, H, N, D] tensor" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))


def _table_ptr(table, dev, D, T, Hl, Wl, split=None):
    """The device pointer of a rotary table, checked against the size the
    grid and split give it (the C ABI takes a bare pointer and finds the
    table's second plane half-way along it, so a table built for another grid
    or split would be read in the wrong places)."""
    if table is None:
        return None
    if table.dtype != torch.float32 or table.device != dev or not table.is_contiguous():
        raise ValueError("rope table must be a contiguous float32 tensor on %s" % dev)
    need = sol_rope3d_table_floats_ex(D, T, Hl, Wl, *_split(split))
    if T * Hl * Wl > 0 and table.numel() != need:
        raise ValueError("rope table holds %d floats; grid %dx%dx%d and split %s need %d"
                         % (table.numel(), T, Hl, Wl, _split(split), need))
    return ctypes.c_void_p(table.data_ptr())


def rope3d(x, T, Hl, Wl, table, out=None):
    """out = bf16(R(pos) x) for x [B, H, N, D] bf16 (out may be x)."""
    _check_tensor("x", x)
    B, H, N, D = x.shape
    if out is None:
        out = torch.empty_like(x)
    _check_tensor("out", out, x.shape)
    check(sol_rope3d(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(out.data_ptr()), B, H, N, D,
                     T, Hl, Wl, _table_ptr(table, x.device, D, T, Hl, Wl, None), _stream(x)))
    return out


def _gamma_ptr(gamma, dev):
    if gamma is None:
        return None
    if (not isinstance(gamma, torch.Tensor) or gamma.dtype != torch.float32 or gamma.device != dev
            or not gamma.is_contiguous() or gamma.shape != (HEAD_DIM,)):
        raise ValueError("gamma must be a contiguous float32 tensor of %d weights on %s"
                         % (HEAD_DIM, dev))
    return ctypes.c_void_p(gamma.data_ptr())


def qknorm_rope3d(x, T, Hl, Wl, table, gamma, eps=1e-6, out=None, split=None):
    """out = bf16(R(pos) rms_norm(x; gamma, eps)) for x [B, H, N, D] bf16."""
    _check_tensor("x", x)
    B, H, N, D = x.shape
    if out is None:
        out = torch.empty_like(x)
    _check_tensor("out", out, x.shape)
    check(sol_qknorm_rope3d(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(out.data_ptr()), B, H,
                            N, D, T, Hl, Wl, *_split(split), _table_ptr(table, x.device, D, T, Hl, Wl, split),
                            _gamma_ptr(gamma, x.device), float(eps), _stream(x)))
    return out


def attn_fwd(q, k, v, T, Hl, Wl, table=None, out=None):
    """softmax(q^ k^T / sqrt(D)) v with the 3D rotary embedding fused (table=None: none)."""
    _check_tensor("q", q)
    _check_tensor("k", k, q.shape)
    _check_tensor("v", v, q.shape)
    B, H, N, D = q.shape
    if out is None:
        out = torch.empty_like(q)
    _check_tensor("out", out, q.shape)
    check(sol_attn_fwd(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                       ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(out.data_ptr()), B, H, N, D,
                       T, Hl, Wl, _table_ptr(table, q.device, D, T, Hl, Wl, None), _stream(q)))
    return out


def attn_workspace(q):
    """A device workspace of the size attn_fwd_ws needs for q's shape (uint8)."""
    B, H, N, D = q.shape
    return torch.empty(sol_attn_workspace_bytes(B, H, N, D), dtype=torch.uint8, device=q.device)


def attn_fwd_ws(q, k, v, T, Hl, Wl, table=None, workspace=None, out=None):
    """attn_fwd through the workspace path (K rotated and V converted in one
    pass, then tile copies); bitwise the same result."""
    _check_tensor("q", q)
    _check_tensor("k", k, q.shape)
    _check_tensor("v", v, q.shape)
    B, H, N, D = q.shape
    if out is None:
        out = torch.empty_like(q)
    _check_tensor("out", out, q.shape)
    if workspace is None:
        workspace = attn_workspace(q)
    if not workspace.is_cuda or workspace.device != q.device or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous tensor on %s" % q.device)
    nbytes = workspace.numel() * workspace.element_size()
    check(sol_attn_fwd_ws(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                          ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(out.data_ptr()), B, H, N,
                          D, T, Hl, Wl, _table_ptr(table, q.device, D, T, Hl, Wl, None),
                          ctypes.c_void_p(workspace.data_ptr()), nbytes, _stream(q)))
    return out


def attn_fwd_noalloc(q, k, v, T, Hl, Wl, table=None, out=None):
    """attn_fwd_ws on the library's own static workspace (no device allocation
    by the library; out is allocated here when not given)."""
    _check_tensor("q", q)
    _check_tensor("k", k, q.shape)
    _check_tensor("v", v, q.shape)
    B, H, N, D = q.shape
    if out is None:
        out = torch.empty_like(q)
    _check_tensor("out", out, q.shape)
    check(sol_attn_fwd_noalloc(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                               ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(out.data_ptr()), B, H, N,
                               D, T, Hl, Wl, _table_ptr(table, q.device, D, T, Hl, Wl, None), _stream(q)))
    return out


def _check_prepared(name, t, nbytes, device):
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float16:
        raise TypeError("%s must be a float16 tensor" % name)
    if not t.is_cuda or t.device != device or not t.is_contiguous() or t.numel() * 2 < nbytes:
        raise ValueError("%s must be a contiguous float16 tensor on %s of at least %d bytes"
                         % (name, device, nbytes))


def prepare_kv(k, v, T, Hl, Wl, table=None, k_prep=None, v_prep=None):
    """(k_prep, v_prep): K rotated (rounded to bf16 like every rotation, then
    fp16) and V in fp16, in the prepared path's tile layout (flat float16
    tensors of sol_prepared_kv_bytes bytes each)."""
    _check_tensor("k", k)
    _check_tensor("v", v, k.shape)
    B, H, N, D = k.shape
    nbytes = sol_prepared_kv_bytes(B, H, N, D)
    if k_prep is None:
        k_prep = torch.empty(nbytes // 2, dtype=torch.float16, device=k.device)
    if v_prep is None:
        v_prep = torch.empty(nbytes // 2, dtype=torch.float16, device=k.device)
    _check_prepared("k_prep", k_prep, nbytes, k.device)
    _check_prepared("v_prep", v_prep, nbytes, k.device)
    check(sol_prepare_kv(ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(v.data_ptr()),
                         ctypes.c_void_p(k_prep.data_ptr()), ctypes.c_void_p(v_prep.data_ptr()),
                         B, H, N, D, T, Hl, Wl, _table_ptr(table, k.device, D, T, Hl, Wl, None), _stream(k)))
    return k_prep, v_prep


def attn_fwd_prepared(q, k_prep, v_prep, T, Hl, Wl, table=None, out=None):
    """Attention on prepare_kv's outputs; q rotated in the tile load."""
    _check_tensor("q", q)
    B, H, N, D = q.shape
    nbytes = sol_prepared_kv_bytes(B, H, N, D)
    _check_prepared("k_prep", k_prep, nbytes, q.device)
    _check_prepared("v_prep", v_prep, nbytes, q.device)
    if out is None:
        out = torch.empty_like(q)
    _check_tensor("out", out, q.shape)
    check(sol_attn_fwd_prepared(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k_prep.data_ptr()),
                                ctypes.c_void_p(v_prep.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                B, H, N, D, T, Hl, Wl, _table_ptr(table, q.device, D, T, Hl, Wl, None), _stream(q)))
    return out


def prepared_kv_buffers(B, H, n_kv, device):
    """Two zero-initialised float16 buffers for a prepared sequence of n_kv keys."""
    n = sol_prepared_kv_bytes(B, H, n_kv, HEAD_DIM) // 2
    return (torch.zeros(n, dtype=torch.float16, device=device),
            torch.zeros(n, dtype=torch.float16, device=device))


def prepare_kv_ex(k, v, T, Hl, Wl, table, k_prep, v_prep, key0=0, n_kv=None, gamma=None, eps=1e-6,
                  split=None):
    """Write k, v [B, H, N, D] (rotated with grid T x Hl x Wl, normalised with
    gamma if given) as keys key0 .. key0 + N - 1 of the prepared sequence of
    n_kv keys held by k_prep, v_prep."""
    _check_tensor("k", k)
    _check_tensor("v", v, k.shape)
    B, H, N, D = k.shape
    n_kv = N if n_kv is None else n_kv
    nbytes = sol_prepared_kv_bytes(B, H, n_kv, D)
    _check_prepared("k_prep", k_prep, nbytes, k.device)
    _check_prepared("v_prep", v_prep, nbytes, k.device)
    check(sol_prepare_kv_ex(ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(v.data_ptr()),
                            ctypes.c_void_p(k_prep.data_ptr()), ctypes.c_void_p(v_prep.data_ptr()),
                            B, H, N, key0, n_kv, D, T, Hl, Wl, *_split(split), _table_ptr(table, k.device, D, T, Hl, Wl, split),
                            _gamma_ptr(gamma, k.device), float(eps), _stream(k)))
    return k_prep, v_prep


def _out_tensor(out, B, H, N, device, fp8, int8_records):
    """The output tensor of an attention call in its format: bf16 [B, H, N, D],
    E4M3 codes uint8 [B, H, N, D], or block-INT8 records uint8 [B, N, H, 144]."""
    if fp8 and int8_records:
        raise ValueError("one output format at a time")
    if not fp8 and not int8_records:
        if out is None:
            out = torch.empty((B, H, N, HEAD_DIM), dtype=torch.bfloat16, device=device)
        _check_tensor("out", out, (B, H, N, HEAD_DIM))
        return out, SOL_OUT_BF16
    shape = (B, N, H, OUT_RECORD_BYTES) if int8_records else (B, H, N, HEAD_DIM)
    if out is None:
        out = torch.empty(shape, dtype=torch.uint8, device=device)
    if (out.dtype != torch.uint8 or tuple(out.shape) != shape or not out.is_contiguous()
            or out.device != device):
        raise ValueError("out must be a contiguous uint8 tensor of shape %s on %s" % (shape, device))
    return out, SOL_OUT_INT8_RECORDS if int8_records else SOL_OUT_FP8_E4M3


def attn_fwd_prepared_ex(q, k_prep, v_prep, n_kv, T, Hl, Wl, table=None, gamma=None, eps=1e-6,
                         out=None, fp8=False, int8_records=False, split=None):
    """q [B, H, N, D] (rotated with grid T x Hl x Wl, normalised with gamma if
    given) against the n_kv prepared keys of k_prep, v_prep.  fp8: the output
    is FP8 E4M3 codes (uint8 [B, H, N, D], unit scale) instead of bf16;
    int8_records: block-INT8 output records (uint8 [B, N, H, 144])."""
    _check_tensor("q", q)
    B, H, N, D = q.shape
    nbytes = sol_prepared_kv_bytes(B, H, n_kv, D)
    _check_prepared("k_prep", k_prep, nbytes, q.device)
    _check_prepared("v_prep", v_prep, nbytes, q.device)
    out, fmt = _out_tensor(out, B, H, N, q.device, fp8, int8_records)
    check(sol_attn_fwd_prepared_ex(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k_prep.data_ptr()),
                                   ctypes.c_void_p(v_prep.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                   B, H, N, n_kv, D, T, Hl, Wl, *_split(split), _table_ptr(table, q.device, D, T, Hl, Wl, split),
                                   _gamma_ptr(gamma, q.device), float(eps), fmt, _stream(q)))
    return out


# ------------------------------------------------------- block-sparse attention

SPARSE_QUERY_BLOCK = 256
SPARSE_KEY_BLOCK = 128


def sparse_workspace(q):
    """A device workspace for the block-sparse routing of q's shape (uint8)."""
    B, H, N, D = q.shape
    n = sol_sparse_workspace_bytes(B, H, N, D)
    if n == 0:
        raise ValueError("block-sparse attention does not take this shape")
    return torch.empty(n, dtype=torch.uint8, device=q.device)


def _check_workspace(ws, nbytes, device):
    if (not isinstance(ws, torch.Tensor) or not ws.is_cuda or ws.device != device
            or not ws.is_contiguous() or ws.numel() * ws.element_size() < nbytes):
        raise ValueError("workspace must be a contiguous device tensor of at least %d bytes on %s"
                         % (nbytes, device))


def sparse_route(q, k_prep, T, Hl, Wl, table, tau, workspace=None, gamma=None, eps=1e-6, split=None):
    """Route every 256-row query block of q [B, H, N, D] over the 128-key
    blocks of the prepared keys (threshold mean + tau * std, prefix sink).
    Returns the workspace holding the routing."""
    _check_tensor("q", q)
    B, H, N, D = q.shape
    _check_prepared("k_prep", k_prep, sol_prepared_kv_bytes(B, H, N, D), q.device)
    if workspace is None:
        workspace = sparse_workspace(q)
    nbytes = sol_sparse_workspace_bytes(B, H, N, D)
    _check_workspace(workspace, nbytes, q.device)
    check(sol_sparse_route(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k_prep.data_ptr()), B, H,
                           N, D, T, Hl, Wl, *_split(split), _table_ptr(table, q.device, D, T, Hl, Wl, split), _gamma_ptr(gamma, q.device),
                           float(eps), float(tau), ctypes.c_void_p(workspace.data_ptr()),
                           workspace.numel() * workspace.element_size(), _stream(q)))
    return workspace


def sparse_routing(workspace, B, H, N):
    """(counts int32 [B, H, nqb], blocks int16 [B, H, nqb, nkb]) views of the
    routing a sparse_route call left in the workspace (uint16 block indices
    read as int16: they are below 2^13)."""
    nqb = -(-N // SPARSE_QUERY_BLOCK)
    nkb = -(-N // SPARSE_KEY_BLOCK)
    n_counts = B * H * nqb
    off = (4 * n_counts + 255) // 256 * 256
    counts = workspace[: 4 * n_counts].view(torch.int32).view(B, H, nqb)
    blocks = workspace[off: off + 2 * n_counts * nkb].view(torch.int16).view(B, H, nqb, nkb)
    return counts, blocks


def attn_fwd_sparse(q, k_prep, v_prep, T, Hl, Wl, table, workspace, gamma=None, eps=1e-6, out=None,
                    fp8=False, int8_records=False, split=None):
    """Block-sparse attention under the routing held by the workspace."""
    _check_tensor("q", q)
    B, H, N, D = q.shape
    nbytes = sol_prepared_kv_bytes(B, H, N, D)
    _check_prepared("k_prep", k_prep, nbytes, q.device)
    _check_prepared("v_prep", v_prep, nbytes, q.device)
    _check_workspace(workspace, sol_sparse_workspace_bytes(B, H, N, D), q.device)
    out, fmt = _out_tensor(out, B, H, N, q.device, fp8, int8_records)
    check(sol_attn_fwd_sparse(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k_prep.data_ptr()),
                              ctypes.c_void_p(v_prep.data_ptr()), ctypes.c_void_p(out.data_ptr()), B, H,
                              N, D, T, Hl, Wl, *_split(split), _table_ptr(table, q.device, D, T, Hl, Wl, split),
                              _gamma_ptr(gamma, q.device),
                              float(eps), ctypes.c_void_p(workspace.data_ptr()),
                              workspace.numel() * workspace.element_size(), fmt, _stream(q)))
    return out


# ------------------------------------------------------ block-INT8 QKV records

QKV_RECORD_BYTES = 400


def _check_records(rec, B, H, N, device):
    if (not isinstance(rec, torch.Tensor) or rec.dtype != torch.uint8 or not rec.is_cuda
            or rec.device != device or not rec.is_contiguous()
            or tuple(rec.shape) != (B, N, H, QKV_RECORD_BYTES)):
        raise ValueError("records must be a contiguous uint8 [B, N, H, 400] tensor on %s" % device)


def qkv_encode(q, k, v, T=0, Hl=0, Wl=0, table=None, q_gamma=None, k_gamma=None, eps=1e-6,
               rec=None):
    """Block-INT8 QKV records (uint8 [B, N, H, 400]) of q, k, v [B, H, N, D]
    bf16: q and k normalised (gammas) and rotated (table, grid T x Hl x Wl)
    first, then every group of 32 values quantised to int8 codes and a UE5M3
    scale."""
    _check_tensor("q", q)
    _check_tensor("k", k, q.shape)
    _check_tensor("v", v, q.shape)
    B, H, N, D = q.shape
    if rec is None:
        rec = torch.empty((B, N, H, QKV_RECORD_BYTES), dtype=torch.uint8, device=q.device)
    _check_records(rec, B, H, N, q.device)
    check(sol_qkv_encode(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                         ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(rec.data_ptr()), B, H, N, D,
                         T, Hl, Wl, _table_ptr(table, q.device, D, T, Hl, Wl, None), _gamma_ptr(q_gamma, q.device),
                         _gamma_ptr(k_gamma, q.device), float(eps), _stream(q)))
    return rec


def qkv_encode_packed(qkv, T=0, Hl=0, Wl=0, table=None, q_gamma=None, k_gamma=None, eps=1e-6,
                      rec=None):
    """Records of a packed QKV buffer qkv [B, N, 3, H, D] bf16 (as a fused QKV
    projection writes it), read in place through its strides."""
    if (not isinstance(qkv, torch.Tensor) or qkv.dtype != torch.bfloat16 or not qkv.is_cuda
            or qkv.dim() != 5 or qkv.shape[2] != 3 or qkv.shape[4] != HEAD_DIM or not qkv.is_contiguous()):
        raise ValueError("qkv must be a contiguous bf16 [B, N, 3, H, %d] device tensor" % HEAD_DIM)
    B, N, _, H, D = qkv.shape
    if rec is None:
        rec = torch.empty((B, N, H, QKV_RECORD_BYTES), dtype=torch.uint8, device=qkv.device)
    _check_records(rec, B, H, N, qkv.device)
    base, el = qkv.data_ptr(), qkv.element_size()
    check(sol_qkv_encode_strided(ctypes.c_void_p(base), ctypes.c_void_p(base + H * D * el),
                                 ctypes.c_void_p(base + 2 * H * D * el), N * 3 * H * D, D, 3 * H * D,
                                 ctypes.c_void_p(rec.data_ptr()), B, H, N, D, T, Hl, Wl,
                                 _table_ptr(table, qkv.device, D, T, Hl, Wl, None), _gamma_ptr(q_gamma, qkv.device),
                                 _gamma_ptr(k_gamma, qkv.device), float(eps), _stream(qkv)))
    return rec


def qkv_decode(rec):
    """(q, k, v) bf16 [B, H, N, D] decoded from records [B, N, H, 400]."""
    B, N, H = rec.shape[:3]
    _check_records(rec, B, H, N, rec.device)
    q, k, v = (torch.empty((B, H, N, HEAD_DIM), dtype=torch.bfloat16, device=rec.device)
               for _ in range(3))
    check(sol_qkv_decode(ctypes.c_void_p(rec.data_ptr()), ctypes.c_void_p(q.data_ptr()),
                         ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(v.data_ptr()), B, H, N,
                         HEAD_DIM, _stream(rec)))
    return q, k, v


def prepare_kv_records(rec, k_prep, v_prep, key0=0, n_kv=None):
    """Write the k and v of records [B, N, H, 400] as keys key0 .. key0 + N - 1
    of the prepared sequence of n_kv keys held by k_prep, v_prep."""
    B, N, H = rec.shape[:3]
    _check_records(rec, B, H, N, rec.device)
    n_kv = N if n_kv is None else n_kv
    nbytes = sol_prepared_kv_bytes(B, H, n_kv, HEAD_DIM)
    _check_prepared("k_prep", k_prep, nbytes, rec.device)
    _check_prepared("v_prep", v_prep, nbytes, rec.device)
    check(sol_prepare_kv_records(ctypes.c_void_p(rec.data_ptr()), ctypes.c_void_p(k_prep.data_ptr()),
                                 ctypes.c_void_p(v_prep.data_ptr()), B, H, N, key0, n_kv, HEAD_DIM,
                                 _stream(rec)))
    return k_prep, v_prep


def attn_fwd_records(rec, k_prep, v_prep, n_kv=None, out=None, fp8=False, int8_records=False):
    """The queries of records [B, N, H, 400] against n_kv prepared keys; out
    bf16 [B, H, N, D] (E4M3 codes with fp8, block-INT8 output records
    [B, N, H, 144] with int8_records)."""
    B, N, H = rec.shape[:3]
    _check_records(rec, B, H, N, rec.device)
    n_kv = N if n_kv is None else n_kv
    nbytes = sol_prepared_kv_bytes(B, H, n_kv, HEAD_DIM)
    _check_prepared("k_prep", k_prep, nbytes, rec.device)
    _check_prepared("v_prep", v_prep, nbytes, rec.device)
    out, fmt = _out_tensor(out, B, H, N, rec.device, fp8, int8_records)
    check(sol_attn_fwd_records(ctypes.c_void_p(rec.data_ptr()), ctypes.c_void_p(k_prep.data_ptr()),
                               ctypes.c_void_p(v_prep.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                               B, H, N, n_kv, HEAD_DIM, fmt, _stream(rec)))
    return out


# ------------------------------------------------------------ measurement aid

def mfma_probe_flops(workgroups, iters):
    """Flops of one sol_mfma_probe launch."""
    return float(workgroups) * 4 * iters * 16 * 32768


def mfma_probe(operands, workgroups, iters, out=None):
    """Launch the dense fp16 MFMA probe on the current stream; operands: a
    float16 device tensor of 8192 values.  Returns `out` (per-thread sums)."""
    if (operands.dtype != torch.float16 or operands.numel() != 8192 or not operands.is_cuda
            or not operands.is_contiguous()):
        raise ValueError("operands must be a contiguous float16 device tensor of 8192 values")
    if out is None:
        out = torch.empty(workgroups * 256, dtype=torch.float32, device=operands.device)
    check(sol_mfma_probe(ctypes.c_void_p(operands.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                         workgroups, iters, _stream(operands)))
    return out


def range_status(clear=True):
    """The current device's SOL_RANGE_* bits raised since the last clear (waits
    for all work on the device); clears them unless clear=False."""
    flags = ctypes.c_uint(0)
    check(sol_range_status(ctypes.byref(flags), 1 if clear else 0))
    return flags.value
