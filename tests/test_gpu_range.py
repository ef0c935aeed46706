"""Fail-closed fp16 range, through the C ABI: the prepared path multiplies in
fp16, so operands beyond fp16's range cannot be represented.  Such inputs
must give a defined outcome -- SOL_RANGE_* bits in the device's sticky range
status (sol_range_status) and non-finite outputs where the bad operand takes
part -- never a silent inf/NaN or a finite wrong value.  In-range inputs up to
the largest bf16 below fp16's maximum (65280) are exact and raise nothing.
"""
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
Q, K, V, OUT = sol.SOL_RANGE_Q, sol.SOL_RANGE_K, sol.SOL_RANGE_V, sol.SOL_RANGE_OUT


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(autouse=True)
def _clear():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    sol.range_status(clear=True)
    yield
    sol.range_status(clear=True)


def _bits(t):
    return W.as_bits(t.cpu())


def _case(seed):
    w = W.custom(1, 2, 3, 8, 8, n_text=16, seed_index=seed)  # N = 208
    q, k, v = W.make_inputs(w)
    return w, q, k, v


def _paths(w, q, k, v):
    """{path: (output, flags)} for the fused and the prepared path, each with
    the range status it raised."""
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    res = {}
    for path, fn in [("fused", sol.attn_fwd), ("prepared", sol.attn_fwd_ws)]:
        sol.range_status(clear=True)
        out = fn(qd, kd, vd, w.T, w.Hl, w.Wl, tab)
        res[path] = (out.cpu(), sol.range_status(clear=True))
    return res


def _parity(w, q, k, v, out, label):
    ref = oracle.attn_rows(_bits(q), _bits(k), _bits(v), w.T, w.Hl, w.Wl)
    R = w.B * w.H * w.N
    st = compare(_bits(out).reshape(R, w.D), ref.reshape(R, w.D), np.repeat(np.arange(w.B * w.H), w.N))
    _log("%s: %s" % (label, st))
    assert_parity(st, label)


def test_in_range_inputs_raise_nothing():
    w, q, k, v = _case(1600)
    for path, (out, flags) in _paths(w, q, k, v).items():
        assert flags == 0, (path, flags)
        _parity(w, q, k, v, out, "in range " + path)


def test_values_at_the_largest_bf16_below_fp16_max_are_exact():
    """v = +-65280 (bf16 0x477F; fp16 holds it exactly) on a few keys: no bit,
    the oracle's result."""
    w, q, k, v = _case(1601)
    v[:, :, 17, :] = 65280.0
    v[:, :, 150, 3::7] = -65280.0
    for path, (out, flags) in _paths(w, q, k, v).items():
        assert flags == 0, (path, flags)
        _parity(w, q, k, v, out, "v at 65280 " + path)


def test_values_above_fp16_range_are_reported():
    """v = 65536 (bf16 0x4780, the next value up) on one key: fp16 cannot hold
    it.  The prepared path raises SOL_RANGE_V and SOL_RANGE_OUT, the fused one
    SOL_RANGE_OUT; the dimension the key carries is not finite in every output
    row (every row attends to that key), the other dims are untouched."""
    w, q, k, v = _case(1602)
    v[:, :, 40, 9] = 65536.0
    res = _paths(w, q, k, v)
    assert res["prepared"][1] == V | OUT, res["prepared"][1]
    assert res["fused"][1] == OUT, res["fused"][1]
    for path, (out, _) in res.items():
        o = out.float()
        assert not torch.isfinite(o[..., 9]).any(), path
        assert torch.isfinite(o[..., :9]).all() and torch.isfinite(o[..., 10:]).all(), path


def test_keys_above_fp16_range_are_reported():
    w, q, k, v = _case(1603)
    k[:, :, 100, 70] = 131072.0  # a prefix token? no: token 100 >= 16 is video; rotation keeps |k^| huge
    res = _paths(w, q, k, v)
    assert res["prepared"][1] & K, res["prepared"][1]
    assert not torch.isfinite(res["prepared"][0].float()).all()
    # bf16 scores: the fused path takes such keys (one key dominates the rows it aligns with)
    assert res["fused"][1] == 0, res["fused"][1]
    _parity(w, q, k, v, res["fused"][0], "large key fused")


def test_large_queries_are_reported_on_the_prepared_path():
    """q^ = 2^19 in one element of one row: q^ log2(e)/sqrt(128) = 66,846 >
    65504.  The prepared path raises SOL_RANGE_Q and that row is not finite
    (the others are exact); the fused path (bf16 scores) gives the oracle's
    result."""
    # (a seed whose correctly rounded bf16 output is itself inside the gate:
    # at this size the rounding floor alone reaches 0.0246 for seed 1604)
    w, q, k, v = _case(1607)
    row = 7  # a prefix row: not rotated, so q^ keeps the value
    q[0, 1, row, 11] = 524288.0
    res = _paths(w, q, k, v)
    out, flags = res["prepared"]
    assert flags & Q and flags & OUT, flags
    o = out.float()
    assert not torch.isfinite(o[0, 1, row]).all()
    keep = torch.ones(w.N, dtype=torch.bool)
    keep[row] = False
    assert torch.isfinite(o[0, 1, keep]).all() and torch.isfinite(o[0, 0]).all()
    assert res["fused"][1] == 0
    _parity(w, q, k, v, res["fused"][0], "large query fused")


def test_nan_inputs_are_reported():
    w, q, k, v = _case(1605)
    v[0, 0, 33, 0] = float("nan")
    res = _paths(w, q, k, v)
    assert res["prepared"][1] == V | OUT, res["prepared"][1]
    assert res["fused"][1] == OUT, res["fused"][1]


def test_status_is_sticky_until_cleared():
    w, q, k, v = _case(1606)
    v[0, 0, 5, 5] = 65536.0
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV)
    sol.attn_fwd_ws(q.to(DEV), k.to(DEV), v.to(DEV), w.T, w.Hl, w.Wl, tab)
    v[0, 0, 5, 5] = 1.0
    sol.attn_fwd_ws(q.to(DEV), k.to(DEV), v.to(DEV), w.T, w.Hl, w.Wl, tab)  # in range: adds nothing
    assert sol.range_status(clear=False) == V | OUT
    assert sol.range_status(clear=True) == V | OUT
    assert sol.range_status(clear=True) == 0
