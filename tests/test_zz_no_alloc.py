"""sol_attn_fwd_noalloc (the prepared path on the library's static per-GPU
workspace, for callers that cannot allocate) against sol_attn_fwd_ws (the same
kernels on a caller workspace), through the C ABI: bit for bit, on two calls
in a row, the second with a smaller input (the array keeps the first call's
contents), and the size limit rejected before any launch."""
import ctypes
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_35110_amd import sol
from paper_2609_35110_amd import workloads as W

from parity import assert_parity, compare

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def _case(w):
    q, k, v = W.make_inputs(w)
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV) if w.n_video else None
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    want = sol.attn_fwd_ws(qd, kd, vd, w.T, w.Hl, w.Wl, tab)
    got = torch.full_like(qd, float("nan"))
    st = sol.sol_attn_fwd_noalloc(ctypes.c_void_p(qd.data_ptr()), ctypes.c_void_p(kd.data_ptr()),
                                  ctypes.c_void_p(vd.data_ptr()), ctypes.c_void_p(got.data_ptr()),
                                  w.B, w.H, w.N, w.D, w.T, w.Hl, w.Wl,
                                  None if tab is None else ctypes.c_void_p(tab.data_ptr()),
                                  sol._stream(qd))
    assert st == 0, sol.sol_last_error()
    torch.cuda.synchronize()
    return q, k, v, got.cpu(), want.cpu()


def test_noalloc_equals_workspace_path_twice_second_smaller():
    assert torch.cuda.is_available()
    first = W.custom(1, 4, 4, 16, 20, n_text=77, seed_index=1404)   # N = 1357
    second = W.custom(1, 2, 2, 5, 7, n_text=9, seed_index=1401)     # N = 79: smaller
    for w in (first, second):
        q, k, v, got, want = _case(w)
        _log("noalloc %s: equal=%s" % (w.describe(), torch.equal(got, want)))
        assert torch.equal(got.view(torch.int16), want.view(torch.int16)), w.describe()
        ref = oracle.attn_rows(W.as_bits(q), W.as_bits(k), W.as_bits(v), w.T, w.Hl, w.Wl)
        R = w.B * w.H * w.N
        st = compare(W.as_bits(got).reshape(R, w.D), ref.reshape(R, w.D), np.repeat(np.arange(w.B * w.H), w.N))
        assert_parity(st, "noalloc " + w.describe())


def test_noalloc_rejects_sizes_beyond_its_workspace():
    # 40 heads of 111,600 tokens need 2.29 GB of workspace: rejected before any launch
    B, H, N, D = 1, 40, 111600, 128
    assert sol.sol_attn_workspace_bytes(B, H, N, D) > (256 << 20)
    q = torch.zeros((1, 1, 1, D), dtype=torch.bfloat16, device=DEV)
    p = ctypes.c_void_p(q.data_ptr())
    st = sol.sol_attn_fwd_noalloc(p, p, p, p, B, H, N, D, 0, 0, 0, None, None)
    assert st == -2 and "256 MiB" in sol.sol_last_error()
    # the largest accepted size: exactly the array
    n_ok = ((256 << 20) // (2 * 2 * 128 * 32)) * 32  # one head: 524,288 keys
    assert sol.sol_attn_workspace_bytes(1, 1, n_ok, D) == (256 << 20)
    assert sol.sol_attn_workspace_bytes(1, 1, n_ok + 1, D) > (256 << 20)
