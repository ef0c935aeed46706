"""GPU parity of partial RoPE (Sec. 3.5, fusion group 2: "QK normalization
with partial RoPE"), through the C ABI: rotary splits dt/dh/dw whose dims past
dt + dh + dw pass through unrotated, on every entry point that takes a split
-- the standalone normalisation + rotation, the prepared K/V, the prepared
attention and the block-sparse path -- against the oracle rotating with the
same split.  The default split 32/48/48 given explicitly reproduces the
split-less entry points bit for bit.
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
EPS = W.QK_NORM_EPS
SPLITS = [(16, 24, 24), (0, 64, 64), (32, 0, 48), (8, 8, 8)]


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    sol.lib()
    yield
    torch.cuda.synchronize()


def _bits(t):
    return W.as_bits(t.cpu())


def _ulps(got, want):
    got, want = got.astype(np.int32), want.astype(np.int32)
    same_sign = (got & 0x8000) == (want & 0x8000)
    return np.where(same_sign, np.abs(got - want), np.abs((got & 0x7FFF) + (want & 0x7FFF)))


@pytest.mark.parametrize("split", SPLITS, ids=[str(s) for s in SPLITS])
@pytest.mark.parametrize("norm", [False, True], ids=["rope", "qknorm+rope"])
def test_partial_rotation_matches_oracle(split, norm):
    """Standalone rotation (and normalisation) under a split.  Rotation
    alone: bit-identical to the oracle (exact rotation, one rounding), the
    pass-through dims the input's bits.  With normalisation (fp32 against the
    oracle's double): within one bf16 ulp, >= 99 % bit-exact."""
    w = W.custom(1, 3, 3, 11, 13, n_text=37, seed_index=1500 + sum(split), qk_norm=True)
    q, _, _ = W.make_inputs(w)
    gq, _ = W.norm_weights(w)
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV, split=split)
    y = sol.qknorm_rope3d(q.to(DEV), w.T, w.Hl, w.Wl, tab, gq.to(DEV) if norm else None, EPS, split=split)
    torch.cuda.synchronize()
    got = _bits(y)
    if norm:
        want = oracle.qknorm_rope3d(_bits(q), w.T, w.Hl, w.Wl, gq.numpy(), EPS, split=split)
    else:
        want = oracle.rope3d_bf16(_bits(q), w.T, w.Hl, w.Wl, split=split)
        tot = sum(split)
        assert np.array_equal(got[..., tot:], _bits(q)[..., tot:]), "pass-through dims changed"
    ulp = _ulps(got, want)
    _log("partial rope %s norm=%s: max ulp %d, exact %.5f" % (split, norm, ulp.max(), (ulp == 0).mean()))
    assert ulp.max() <= 1 and (ulp == 0).mean() >= (0.99 if norm else 1.0)


SHAPES = [
    # (B, H, T, Hl, Wl, n_text)
    (1, 2, 3, 11, 13, 37),   # N = 466: ragged row and key tiles, a text prefix
    (2, 1, 4, 8, 9, 0),      # B = 2
]


@pytest.mark.parametrize("split", SPLITS, ids=[str(s) for s in SPLITS])
@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_partial_rope_attention_matches_oracle(shape, split):
    """The prepared path (K rotated in sol_prepare_kv_ex, Q in the attention
    kernel's tile load) under a split, with QK normalisation, on full
    tensors against the oracle."""
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=1520 + sum(shape) + sum(split), qk_norm=True)
    q, k, v = W.make_inputs(w)
    gq, gk = W.norm_weights(w)
    tab = sol.rope3d_table(T, Hl, Wl, device=DEV, split=split)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    k_prep, v_prep = sol.prepared_kv_buffers(B, H, w.N, DEV)
    sol.prepare_kv_ex(kd, vd, T, Hl, Wl, tab, k_prep, v_prep, gamma=gk.to(DEV), eps=EPS, split=split)
    out = sol.attn_fwd_prepared_ex(qd, k_prep, v_prep, w.N, T, Hl, Wl, tab, gamma=gq.to(DEV), eps=EPS,
                                   split=split)
    torch.cuda.synchronize()
    ref = oracle.attn_rows(_bits(q), _bits(k), _bits(v), T, Hl, Wl, split=split, q_gamma=gq.numpy(),
                           k_gamma=gk.numpy(), eps=EPS)
    R = B * H * w.N
    st = compare(_bits(out).reshape(R, w.D), ref.reshape(R, w.D), np.repeat(np.arange(B * H), w.N))
    _log("partial rope attention %s %s: %s" % (shape, split, st))
    assert_parity(st, "partial rope %s %s" % (shape, split))


def test_partial_rope_differs_from_full_rope():
    """A split that leaves dims unrotated changes the result (the split is not
    silently replaced by the default)."""
    w = W.custom(1, 1, 3, 11, 13, n_text=0, seed_index=1540)
    q, k, v = W.make_inputs(w)
    outs = []
    for split in [(32, 48, 48), (16, 24, 24)]:
        tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV, split=split)
        k_prep, v_prep = sol.prepared_kv_buffers(1, 1, w.N, DEV)
        sol.prepare_kv_ex(k.to(DEV), v.to(DEV), w.T, w.Hl, w.Wl, tab, k_prep, v_prep, split=split)
        outs.append(sol.attn_fwd_prepared_ex(q.to(DEV), k_prep, v_prep, w.N, w.T, w.Hl, w.Wl, tab,
                                             split=split).cpu())
    assert not torch.equal(outs[0], outs[1])


def test_default_split_given_explicitly_is_bit_identical():
    """32/48/48 passed to the split-taking entry points gives the bits of the
    split-less ones (sol_attn_fwd_ws, sol_rope3d)."""
    w = W.custom(1, 2, 3, 11, 13, n_text=37, seed_index=1541)
    q, k, v = W.make_inputs(w)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV)
    tab_ex = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV, split=(32, 48, 48))
    a = sol.attn_fwd_ws(qd, kd, vd, w.T, w.Hl, w.Wl, tab)
    k_prep, v_prep = sol.prepared_kv_buffers(1, 2, w.N, DEV)
    sol.prepare_kv_ex(kd, vd, w.T, w.Hl, w.Wl, tab_ex, k_prep, v_prep, split=(32, 48, 48))
    b = sol.attn_fwd_prepared_ex(qd, k_prep, v_prep, w.N, w.T, w.Hl, w.Wl, tab_ex, split=(32, 48, 48))
    r1 = sol.rope3d(qd, w.T, w.Hl, w.Wl, tab)
    r2 = sol.qknorm_rope3d(qd, w.T, w.Hl, w.Wl, tab_ex, None, split=(32, 48, 48))
    torch.cuda.synchronize()
    assert torch.equal(tab, tab_ex)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(r1.view(torch.int16), r2.view(torch.int16))


@pytest.mark.parametrize("split", [(16, 24, 24), (0, 64, 64)], ids=str)
def test_partial_rope_block_sparse(split):
    """The block-sparse path under a split: tau -> -inf (every block kept) is
    the dense prepared kernel bit for bit, and tau = 1 matches the oracle's
    attention under the kernel's own routing, whose mask agrees with the
    oracle's away from the threshold."""
    from parity import sparse_mask
    w = W.custom(1, 2, 4, 16, 20, n_text=64, seed_index=1550 + sum(split), shared_dir=1.0)  # N = 1344
    q, k, v = W.make_inputs(w)
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV, split=split)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    k_prep, v_prep = sol.prepared_kv_buffers(1, 2, w.N, DEV)
    sol.prepare_kv_ex(kd, vd, w.T, w.Hl, w.Wl, tab, k_prep, v_prep, split=split)
    dense = sol.attn_fwd_prepared_ex(qd, k_prep, v_prep, w.N, w.T, w.Hl, w.Wl, tab, split=split)
    ws = sol.sparse_route(qd, k_prep, w.T, w.Hl, w.Wl, tab, -1e30, split=split)
    all_kept = sol.attn_fwd_sparse(qd, k_prep, v_prep, w.T, w.Hl, w.Wl, tab, ws, split=split)
    torch.cuda.synchronize()
    assert torch.equal(dense.view(torch.int16), all_kept.view(torch.int16))
    ws = sol.sparse_route(qd, k_prep, w.T, w.Hl, w.Wl, tab, 1.0, split=split)
    out = sol.attn_fwd_sparse(qd, k_prep, v_prep, w.T, w.Hl, w.Wl, tab, ws, split=split)
    torch.cuda.synchronize()
    mask = sparse_mask(ws, 1, 2, w.N)
    want_mask, scores, thr = oracle.sparse_route(_bits(q), _bits(k), w.T, w.Hl, w.Wl, 1.0, split=split)
    # decisions may differ only at rounding distance of the threshold or of the best score
    scale = np.abs(scores).max(axis=(2, 3), keepdims=True)
    near = ((np.abs(scores - thr[..., None]) <= 1e-4 * scale)
            | (np.abs(scores - scores.max(axis=3, keepdims=True)) <= 1e-4 * scale))
    assert np.all((mask == want_mask) | near)
    ref = oracle.attn_rows(_bits(q), _bits(k), _bits(v), w.T, w.Hl, w.Wl, split=split, block_mask=mask)
    R = 2 * w.N
    # local attention (shared q/k direction): row magnitudes spread too far for
    # one scale per slab, so errors are normalised per row
    st = compare(_bits(out).reshape(R, w.D), ref.reshape(R, w.D), np.arange(R))
    _log("partial rope sparse %s: %s" % (split, st))
    assert_parity(st, "partial rope sparse %s" % (split,))
