"""GPU parity of the two generalisations of the prepared path, through the C ABI:

* QK normalization ahead of the rotation (Sec. 3.5, fusion group 2): the
  standalone sol_qknorm_rope3d, and the normalisation fused into
  sol_prepare_kv_ex (keys) and sol_attn_fwd_prepared_ex (queries);
* queries and keys of different lengths, with a prepared key sequence filled
  from several sources -- the reference-KV cache of Sec. 5 (cached reference
  keys and values, then the current step's own tokens).

Each case is compared with the oracle (oracle/), which normalises and rotates
in double and rounds once to bf16, at sizes it finishes in seconds (several
tiles, ragged tails, tiles shared by two sources) and on sampled rows at the
full 720p sizes.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_35110_amd import sol
from paper_2609_35110_amd import workloads as W

from parity import assert_parity, bits_to_f32, compare

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
EPS = W.QK_NORM_EPS


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


def _table(T, Hl, Wl):
    return sol.rope3d_table(T, Hl, Wl, device=DEV) if T * Hl * Wl else None


# --------------------------------------------------------- QK normalization

NORM_SHAPES = [
    # (B, H, T, Hl, Wl, n_text)
    (1, 2, 3, 8, 8, 0),
    (1, 3, 3, 11, 13, 37),     # N=466: ragged row and key tiles, text prefix
    (2, 1, 5, 7, 9, 64),       # B=2
    (1, 2, 0, 0, 0, 100),      # no latent grid: normalisation only
]


@pytest.mark.parametrize("shape", NORM_SHAPES, ids=[str(s) for s in NORM_SHAPES])
def test_qknorm_rope3d_matches_oracle(shape):
    """Standalone normalisation + rotation vs the oracle (double, one
    rounding): within one bf16 ulp everywhere (fp32 against double) and
    bit-identical for >= 99 % of the elements."""
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=700 + sum(shape), qk_norm=True)
    q, _, _ = W.make_inputs(w)
    gq, _ = W.norm_weights(w)
    y = sol.qknorm_rope3d(q.to(DEV), T, Hl, Wl, _table(T, Hl, Wl), gq.to(DEV), EPS)
    torch.cuda.synchronize()
    got = _bits(y).astype(np.int32)
    want = oracle.qknorm_rope3d(_bits(q), T, Hl, Wl, gq.numpy(), EPS).astype(np.int32)
    # bf16 bit patterns of equal sign are ordered like their values
    same_sign = (got & 0x8000) == (want & 0x8000)
    ulp = np.where(same_sign, np.abs(got - want), np.abs((got & 0x7FFF) + (want & 0x7FFF)))
    exact = float((ulp == 0).mean())
    _log("qknorm_rope3d %s: max ulp %d, exact %.5f" % (shape, ulp.max(), exact))
    assert ulp.max() <= 1 and exact >= 0.99


def test_qknorm_without_weights_is_rope3d():
    """gamma = NULL is exactly sol_rope3d."""
    w = W.custom(1, 2, 2, 6, 6, n_text=5, seed_index=710)
    q, _, _ = W.make_inputs(w)
    tab = _table(w.T, w.Hl, w.Wl)
    a = sol.qknorm_rope3d(q.to(DEV), w.T, w.Hl, w.Wl, tab, None)
    b = sol.rope3d(q.to(DEV), w.T, w.Hl, w.Wl, tab)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def _norm_attn(w, q, k, v, gq, gk):
    """The fused normalisation path: K normalised + rotated in sol_prepare_kv_ex,
    Q in the attention kernel's tile load."""
    tab = _table(w.T, w.Hl, w.Wl)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    kp, vp = sol.prepared_kv_buffers(w.B, w.H, w.N, DEV)
    sol.prepare_kv_ex(kd, vd, w.T, w.Hl, w.Wl, tab, kp, vp, gamma=gk.to(DEV), eps=EPS)
    return sol.attn_fwd_prepared_ex(qd, kp, vp, w.N, w.T, w.Hl, w.Wl, tab, gamma=gq.to(DEV), eps=EPS)


@pytest.mark.parametrize("shape", NORM_SHAPES, ids=[str(s) for s in NORM_SHAPES])
def test_qknorm_attention_full_parity(shape):
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=720 + sum(shape), qk_norm=True)
    q, k, v = W.make_inputs(w)
    gq, gk = W.norm_weights(w)
    out = _norm_attn(w, q, k, v, gq, gk)
    torch.cuda.synchronize()
    ref = oracle.attn_rows(_bits(q), _bits(k), _bits(v), T, Hl, Wl, q_gamma=gq.numpy(),
                           k_gamma=gk.numpy(), eps=EPS)
    R = w.B * w.H * w.N
    st = compare(_bits(out).reshape(R, w.D), ref.reshape(R, w.D), np.repeat(np.arange(B * H), w.N))
    _log("qknorm attention %s: %s" % (w.describe(), st))
    assert_parity(st, "qknorm attention")


@pytest.mark.parametrize("shape", NORM_SHAPES[:3], ids=[str(s) for s in NORM_SHAPES[:3]])
def test_qknorm_fused_equals_standalone(shape):
    """Normalising + rotating q and k with sol_qknorm_rope3d, then attending
    with neither, is bit-identical to the fused path: the kernels normalise a
    row to the same bits whichever lanes hold it."""
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=740 + sum(shape), qk_norm=True)
    q, k, v = W.make_inputs(w)
    gq, gk = W.norm_weights(w)
    fused = _norm_attn(w, q, k, v, gq, gk)
    tab = _table(T, Hl, Wl)
    qh = sol.qknorm_rope3d(q.to(DEV), T, Hl, Wl, tab, gq.to(DEV), EPS)
    kh = sol.qknorm_rope3d(k.to(DEV), T, Hl, Wl, tab, gk.to(DEV), EPS)
    kp, vp = sol.prepared_kv_buffers(w.B, w.H, w.N, DEV)
    sol.prepare_kv_ex(kh, v.to(DEV), 0, 0, 0, None, kp, vp)
    pre = sol.attn_fwd_prepared_ex(qh, kp, vp, w.N, 0, 0, 0, None)
    torch.cuda.synchronize()
    assert torch.equal(fused, pre)


def test_qknorm_p720_sampled_parity():
    """Full 720p size (B=1, H=40, N=111,600), pre-normalisation inputs at
    scales 2^-4 .. 2^4, in the launch configuration the benchmark times."""
    w = W.WORKLOADS["p720n"]
    _log("generating %s" % w.describe())
    q, k, v = W.make_inputs(w)
    gq, gk = W.norm_weights(w)
    out = _norm_attn(w, q, k, v, gq, gk)
    torch.cuda.synchronize()
    rows = W.sample_rows(w, per_slab=8, head=32, tail=80).numpy()
    _log("oracle on %d rows" % len(rows))
    ref = oracle.attn_rows(_bits(q), _bits(k), _bits(v), w.T, w.Hl, w.Wl, rows=rows,
                           q_gamma=gq.numpy(), k_gamma=gk.numpy(), eps=EPS)
    got = _bits(out).reshape(-1, w.D)[rows]
    st = compare(got, ref, rows // w.N)
    _log("p720n: %s" % st)
    assert_parity(st, "p720n")


# ------------------------------------------------ keys from several sources

def _segments_oracle(q, Tq, Hlq, Wlq, segs, gq=None, gk=None):
    """Oracle output of queries q against the concatenation of segments
    [(k, v, (T, Hl, Wl))], each normalised (gk) and rotated with its own grid
    by the oracle's own rotation, in the order given."""
    kh = [oracle.qknorm_rope3d(_bits(k), *g, gk.numpy(), EPS) if gk is not None
          else oracle.rope3d_bf16(_bits(k), *g) for k, _, g in segs]
    vs = [_bits(v) for _, v, _ in segs]
    return oracle.attn_rows(_bits(q), np.concatenate(kh, 2), np.concatenate(vs, 2), Tq, Hlq, Wlq,
                            rope_k=False, q_gamma=None if gq is None else gq.numpy(), eps=EPS)


def _segments_gpu(q, Tq, Hlq, Wlq, segs, order, gq=None, gk=None, fill=None):
    """Prepare the segments (calls in `order`) into one key sequence and attend."""
    B, H, _, _ = q.shape
    n_kv = sum(k.shape[2] for k, _, _ in segs)
    kp, vp = sol.prepared_kv_buffers(B, H, n_kv, DEV)
    if fill is not None:
        kp.view(torch.int16).fill_(fill)
        vp.view(torch.int16).fill_(fill)
    starts = np.cumsum([0] + [k.shape[2] for k, _, _ in segs])
    for i in order:
        k, v, (T, Hl, Wl) = segs[i]
        sol.prepare_kv_ex(k.to(DEV), v.to(DEV), T, Hl, Wl, _table(T, Hl, Wl), kp, vp,
                          key0=int(starts[i]), n_kv=n_kv,
                          gamma=None if gk is None else gk.to(DEV), eps=EPS)
    out = sol.attn_fwd_prepared_ex(q.to(DEV), kp, vp, n_kv, Tq, Hlq, Wlq, _table(Tq, Hlq, Wlq),
                                   gamma=None if gq is None else gq.to(DEV), eps=EPS)
    return out, kp, vp


def _seg(B, H, T, Hl, Wl, nt, seed_index):
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=seed_index)
    _, k, v = W.make_inputs(w)
    return k, v, (T, Hl, Wl)


SEG_CASES = [
    # queries (B, H, T, Hl, Wl, n_text); segments [(T, Hl, Wl, n_text)]
    ((1, 2, 3, 8, 8, 0), [(2, 4, 5, 3), (3, 8, 8, 0)]),          # 43 + 192 keys: shared tile
    ((1, 3, 2, 5, 7, 9), [(1, 6, 6, 0), (2, 5, 7, 9), (1, 1, 1, 0)]),  # 36 + 79 + 1
    ((2, 1, 1, 4, 4, 0), [(4, 8, 10, 7)]),                       # Nq = 16 < Nkv = 327
    ((1, 2, 4, 8, 8, 1), [(0, 0, 0, 5)]),                        # Nq = 257 > Nkv = 5
]


@pytest.mark.parametrize("case", SEG_CASES, ids=[str(c) for c in SEG_CASES])
def test_key_segments_full_parity(case):
    (B, H, T, Hl, Wl, nt), segdefs = case
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=800 + sum(case[0]))
    q, _, _ = W.make_inputs(w)
    segs = [_seg(B, H, *sd, seed_index=810 + 7 * i + sum(sd)) for i, sd in enumerate(segdefs)]
    out, _, _ = _segments_gpu(q, T, Hl, Wl, segs, order=range(len(segs)))
    torch.cuda.synchronize()
    ref = _segments_oracle(q, T, Hl, Wl, segs)
    R = B * H * w.N
    st = compare(_bits(out).reshape(R, w.D), ref.reshape(R, w.D), np.repeat(np.arange(B * H), w.N))
    _log("segments %s -> Nkv=%d: %s" % (w.describe(), sum(s[0].shape[2] for s in segs), st))
    assert_parity(st, "key segments")


def test_key_segments_with_qknorm():
    w = W.custom(1, 2, 3, 8, 8, n_text=3, seed_index=830, qk_norm=True)
    q, _, _ = W.make_inputs(w)
    gq, gk = W.norm_weights(w)
    segs = [_seg(1, 2, 2, 4, 5, 3, 831), _seg(1, 2, 3, 8, 8, 3, 832)]
    out, _, _ = _segments_gpu(q, w.T, w.Hl, w.Wl, segs, order=[1, 0], gq=gq, gk=gk)
    torch.cuda.synchronize()
    ref = _segments_oracle(q, w.T, w.Hl, w.Wl, segs, gq=gq, gk=gk)
    R = w.B * w.H * w.N
    st = compare(_bits(out).reshape(R, w.D), ref.reshape(R, w.D), np.repeat(np.arange(2), w.N))
    _log("segments + qknorm: %s" % st)
    assert_parity(st, "key segments + qknorm")


def test_key_segments_write_only_their_keys():
    """Two sources sharing a tile (43 + 100 keys): each call writes only its own
    keys (sentinels elsewhere survive), the two calls in either order leave the
    same bytes, and one segment prepared alone equals a whole-sequence
    preparation of the same keys."""
    segs = [_seg(1, 2, 2, 4, 5, 3, 840), _seg(1, 2, 1, 10, 10, 0, 841)]
    n0, n_kv = 43, 143
    k0, v0, g0 = segs[0]
    kp, vp = sol.prepared_kv_buffers(1, 2, n_kv, DEV)
    kp.view(torch.int16).fill_(0x7777)
    vp.view(torch.int16).fill_(0x7777)
    sol.prepare_kv_ex(k0.to(DEV), v0.to(DEV), *g0, _table(*g0), kp, vp, key0=0, n_kv=n_kv)
    alone_k, alone_v = sol.prepare_kv(k0.to(DEV), v0.to(DEV), *g0, _table(*g0))
    torch.cuda.synchronize()
    # tile 1 holds keys 32..63: 32..42 belong to segment 0, 43..63 to segment 1
    per_tile = 32 * 128
    kt = kp[per_tile: 2 * per_tile].view(8, 2, 32, 8)       # [kk][hh][key][8]
    assert (kt[:, :, 11:].view(torch.int16) == 0x7777).all(), "segment 0 wrote keys it does not own"
    assert torch.equal(kt[:, :, :11], alone_k[per_tile: 2 * per_tile].view(8, 2, 32, 8)[:, :, :11])
    assert torch.equal(kp[:per_tile], alone_k[:per_tile]) and torch.equal(vp[:per_tile], alone_v[:per_tile])
    # V: key 16s + 8(i//4) + 4h + i%4 of the tile sits at [s][c][h][l][i]
    vt = vp[per_tile: 2 * per_tile].view(2, 4, 2, 32, 8)
    s_, h_, i_ = np.meshgrid(np.arange(2), np.arange(2), np.arange(8), indexing="ij")
    key = 16 * s_ + 8 * (i_ // 4) + 4 * h_ + i_ % 4
    for s in range(2):
        for h in range(2):
            for i in range(8):
                col = vt[s, :, h, :, i].view(torch.int16)
                if key[s, h, i] >= 11:
                    assert (col == 0x7777).all()
    # either order: identical bytes
    _, ka, va = _segments_gpu(torch.zeros(1, 2, 1, 128, dtype=torch.bfloat16), 0, 0, 0, segs, order=[0, 1])
    _, kb, vb = _segments_gpu(torch.zeros(1, 2, 1, 128, dtype=torch.bfloat16), 0, 0, 0, segs, order=[1, 0],
                              fill=0x5555)
    torch.cuda.synchronize()
    assert torch.equal(ka, kb) and torch.equal(va, vb)
    # padding past n_kv is zero
    pad = (n_kv + 31) // 32 * 32 - n_kv
    assert pad > 0
    last_k = ka.view(2, -1, 8, 2, 32, 8)[:, -1]
    assert (last_k[:, :, :, 32 - pad:] == 0).all()


def test_reference_cache_sampled_parity():
    """The reference-KV cache at 720p: queries 512 text + 31x45x80, keys = a
    cached 8x45x80 reference video prepared once, then the step's own
    tokens; sampled rows against the oracle."""
    w = W.WORKLOADS["ref720"]
    _log("generating %s" % w.describe())
    q, k, v = W.make_inputs(w)
    kr, vr = W.make_ref_inputs(w)
    segs = [(kr, vr, w.ref_grid), (k, v, (w.T, w.Hl, w.Wl))]
    out, _, _ = _segments_gpu(q, w.T, w.Hl, w.Wl, segs, order=[0, 1])
    torch.cuda.synchronize()
    rows = W.sample_rows(w, per_slab=8, head=32, tail=80).numpy()
    _log("oracle on %d rows" % len(rows))
    kh = np.concatenate([oracle.rope3d_bf16(_bits(kr), *w.ref_grid),
                         oracle.rope3d_bf16(_bits(k), w.T, w.Hl, w.Wl)], 2)
    ref = oracle.attn_rows(_bits(q), kh, np.concatenate([_bits(vr), _bits(v)], 2), w.T, w.Hl, w.Wl,
                           rows=rows, rope_k=False)
    got = _bits(out).reshape(-1, w.D)[rows]
    st = compare(got, ref, rows // w.N)
    _log("ref720: %s" % st)
    assert_parity(st, "ref720")
