"""GPU parity of the block-INT8 QKV records (Sec. 3.2, "Quantized
communication"), through the C ABI, against the oracle:

* sol_qkv_encode (the sender: QK normalisation and rotation fused ahead of
  the quantisation) and sol_qkv_decode: byte and bit work, compared exactly;
* sol_prepare_kv_records + sol_attn_fwd_records (the receiver: records
  decoded in the prepare pass and in the attention kernel's query tile load):
  within the attention tolerance of the oracle, which encodes with its own
  rotation, decodes and attends in double; and bit for bit equal to the
  prepared path on the decoded tensors.
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


def _spread(x, seed):
    """Rows scaled by 2^e, e in [-12, 12] (exact), a few all-zero rows and
    32-value groups, and rows scaled by 2^23, too large for any scale code:
    inputs whose groups span every kind of scale (subnormal, normal,
    saturated)."""
    gen = torch.Generator().manual_seed(seed)
    B, H, N, D = x.shape
    e = torch.randint(-12, 13, (B, H, N, 1), generator=gen).to(torch.float32)
    e[:, :, 3::11] = 23
    y = (x.to(torch.float32) * torch.exp2(e)).to(torch.bfloat16)
    y[:, :, ::7] = 0
    y[:, :, 1::5, 32:64] = 0
    return y


def _oracle_records(q, k, v, T, Hl, Wl, gq=None, gk=None):
    """The oracle's own records: rotation (and normalisation) in double,
    rounded to bf16, then its encoder."""
    if gq is not None:
        qh = oracle.qknorm_rope3d(_bits(q), T, Hl, Wl, gq.numpy(), EPS, rope=T * Hl * Wl > 0)
        kh = oracle.qknorm_rope3d(_bits(k), T, Hl, Wl, gk.numpy(), EPS, rope=T * Hl * Wl > 0)
    elif T * Hl * Wl:
        qh, kh = oracle.rope3d_bf16(_bits(q), T, Hl, Wl), oracle.rope3d_bf16(_bits(k), T, Hl, Wl)
    else:
        qh, kh = _bits(q), _bits(k)
    return oracle.encode_qkv(qh, kh, _bits(v))


def _oracle_attention(rec, rows=None, k_rec=None):
    """Oracle attention on decoded records (the queries' records; keys and
    values from k_rec when given)."""
    dq, dk, dv = oracle.decode_qkv(rec)
    if k_rec is not None:
        _, dk, dv = oracle.decode_qkv(k_rec)
    return oracle.attn_rows(dq, dk, dv, 0, 0, 0, rows=rows, rope=False)


def _gpu_attention(rec, fp8=False):
    B, N, H = rec.shape[:3]
    kp, vp = sol.prepared_kv_buffers(B, H, N, DEV)
    sol.prepare_kv_records(rec, kp, vp)
    return sol.attn_fwd_records(rec, kp, vp, fp8=fp8)


ENC_SHAPES = [
    # (B, H, T, Hl, Wl, n_text)
    (1, 3, 3, 5, 5, 2),      # N = 77: a ragged workgroup of records
    (2, 2, 2, 10, 15, 0),    # N = 300, B = 2
    (1, 1, 1, 1, 1, 0),      # one record
]


@pytest.mark.parametrize("shape", ENC_SHAPES, ids=[str(s) for s in ENC_SHAPES])
def test_encode_equals_oracle_bytes(shape):
    """Without rotation or normalisation the records are integer decisions on
    the same bf16 inputs: byte for byte the oracle's."""
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=1200 + sum(shape))
    q, k, v = (_spread(x, 1200 + i) for i, x in enumerate(W.make_inputs(w)))
    rec = sol.qkv_encode(q.to(DEV), k.to(DEV), v.to(DEV))
    torch.cuda.synchronize()
    want = oracle.encode_qkv(_bits(q), _bits(k), _bits(v))
    got = rec.cpu().numpy()
    assert got.shape == want.shape
    assert np.array_equal(got, want), "%d of %d bytes differ" % ((got != want).sum(), got.size)


def test_encode_fused_equals_normalise_rotate_then_encode():
    """The encoder's fused normalisation and rotation give the bits of
    sol_qknorm_rope3d: encoding its output without either is byte-identical."""
    w = W.custom(1, 2, 3, 11, 13, n_text=37, seed_index=1210, qk_norm=True)
    q, k, v = W.make_inputs(w)
    gq, gk = W.norm_weights(w)
    tab = _table(w.T, w.Hl, w.Wl)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    for gqd, gkd in ((gq.to(DEV), gk.to(DEV)), (None, None)):
        fused = sol.qkv_encode(qd, kd, vd, w.T, w.Hl, w.Wl, tab, gqd, gkd, EPS)
        if gqd is None:
            qh, kh = sol.rope3d(qd, w.T, w.Hl, w.Wl, tab), sol.rope3d(kd, w.T, w.Hl, w.Wl, tab)
        else:
            qh = sol.qknorm_rope3d(qd, w.T, w.Hl, w.Wl, tab, gqd, EPS)
            kh = sol.qknorm_rope3d(kd, w.T, w.Hl, w.Wl, tab, gkd, EPS)
        plain = sol.qkv_encode(qh, kh, vd)
        torch.cuda.synchronize()
        assert torch.equal(fused, plain)


def test_encode_packed_qkv_in_place():
    """The stride-aware encoder on a packed [B, N, 3, H, D] buffer (read where
    it lies) writes the records of the contiguous q, k, v, byte for byte, with
    the rotation and the normalisation fused."""
    w = W.custom(2, 3, 3, 7, 9, n_text=11, seed_index=1225, qk_norm=True)
    q, k, v = W.make_inputs(w)
    gq, gk = W.norm_weights(w)
    tab = _table(w.T, w.Hl, w.Wl)
    packed = torch.stack([q, k, v], 2).permute(0, 3, 2, 1, 4).contiguous().to(DEV)  # [B, N, 3, H, D]
    got = sol.qkv_encode_packed(packed, w.T, w.Hl, w.Wl, tab, gq.to(DEV), gk.to(DEV), EPS)
    want = sol.qkv_encode(q.to(DEV), k.to(DEV), v.to(DEV), w.T, w.Hl, w.Wl, tab, gq.to(DEV), gk.to(DEV), EPS)
    torch.cuda.synchronize()
    assert torch.equal(got, want)


def test_encode_with_rotation_equals_oracle_bytes():
    """With the rotation: the encoder turns q and k correctly rounded (fp64
    with the two-plane table, one rounding to bf16), as the oracle does from
    double trig, so every byte of every record is the oracle's -- codes,
    scale codes and the zero padding -- on 2,048 records of a grid with a
    text prefix and ragged frames."""
    w = W.custom(1, 2, 4, 12, 20, n_text=64, seed_index=1220)
    q, k, v = W.make_inputs(w)
    rec = sol.qkv_encode(q.to(DEV), k.to(DEV), v.to(DEV), w.T, w.Hl, w.Wl, _table(w.T, w.Hl, w.Wl))
    torch.cuda.synchronize()
    got, want = rec.cpu().numpy(), _oracle_records(q, k, v, w.T, w.Hl, w.Wl)
    codes = float((got[..., :384] == want[..., :384]).mean())
    scales = float((got[..., 384:396] == want[..., 384:396]).mean())
    _log("rotated encode: codes %.5f, scales %.5f equal" % (codes, scales))
    assert np.array_equal(got, want), "%d of %d bytes differ" % ((got != want).sum(), got.size)


def test_decode_equals_oracle_bits():
    rec = W.random_records(2, 3, 257, seed=1230)
    q, k, v = sol.qkv_decode(rec.to(DEV))
    torch.cuda.synchronize()
    for got, want in zip((q, k, v), oracle.decode_qkv(rec.numpy())):
        assert np.array_equal(_bits(got), want)


ATTN_SHAPES = [
    # (B, H, T, Hl, Wl, n_text, qk_norm)
    (1, 2, 3, 8, 8, 0, False),
    (1, 3, 3, 11, 13, 37, False),   # N = 466: ragged row and key tiles, text prefix
    (2, 1, 5, 7, 9, 64, True),      # B = 2, QK normalisation at the encoder
    (1, 2, 0, 0, 0, 300, False),    # no latent grid
]


@pytest.mark.parametrize("shape", ATTN_SHAPES, ids=[str(s) for s in ATTN_SHAPES])
def test_records_attention_parity(shape):
    B, H, T, Hl, Wl, nt, norm = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=1240 + sum(shape[:6]), qk_norm=norm)
    q, k, v = W.make_inputs(w)
    gq, gk = W.norm_weights(w) if norm else (None, None)
    rec = sol.qkv_encode(q.to(DEV), k.to(DEV), v.to(DEV), T, Hl, Wl, _table(T, Hl, Wl),
                         None if gq is None else gq.to(DEV), None if gk is None else gk.to(DEV), EPS)
    out = _gpu_attention(rec)
    torch.cuda.synchronize()
    ref = _oracle_attention(_oracle_records(q, k, v, T, Hl, Wl, gq, gk))
    R = B * H * w.N
    slabs = np.repeat(np.arange(B * H), w.N)
    st = compare(_bits(out).reshape(R, w.D), ref.reshape(R, w.D), slabs)
    # how far the int8 wire format moves the layer from unquantised attention
    exact = oracle.attn_rows(_bits(q), _bits(k), _bits(v), T, Hl, Wl,
                             q_gamma=None if gq is None else gq.numpy(),
                             k_gamma=None if gk is None else gk.numpy(), eps=EPS)
    qerr = compare(_bits(out).reshape(R, w.D), exact.reshape(R, w.D), slabs)
    _log("records attention %s: %s; against unquantised attention: max %.4f mean %.5f"
         % (w.describe(), st, qerr["max_abs"], qerr["mean_abs"]))
    assert_parity(st, "records attention")


@pytest.mark.parametrize("fp8", [False, True])
def test_records_attention_equals_prepared_on_decoded(fp8):
    """Decoding in the prepare pass and in the query tile load gives the bits
    of the prepared path run on the decoded tensors (no rotation)."""
    w = W.custom(2, 3, 3, 9, 11, n_text=20, seed_index=1260)
    q, k, v = W.make_inputs(w)
    rec = sol.qkv_encode(q.to(DEV), k.to(DEV), v.to(DEV), w.T, w.Hl, w.Wl, _table(w.T, w.Hl, w.Wl))
    out = _gpu_attention(rec, fp8=fp8)
    qd, kd, vd = sol.qkv_decode(rec)
    kp, vp = sol.prepared_kv_buffers(w.B, w.H, w.N, DEV)
    sol.prepare_kv_ex(kd, vd, 0, 0, 0, None, kp, vp)
    want = sol.attn_fwd_prepared_ex(qd, kp, vp, w.N, 0, 0, 0, None, fp8=fp8)
    torch.cuda.synchronize()
    assert torch.equal(out, want)


def test_records_key_segments():
    """The reference-KV cache from records: cached reference records prepared
    as keys 0 .. 299, the step's own records after them (tile 9 shared by the
    two), in either order; the step's queries attend to all 300 + 466 keys."""
    B, H = 1, 2
    wr = W.custom(B, H, 2, 10, 15, seed_index=1270)           # reference: 300 tokens
    wq = W.custom(B, H, 3, 11, 13, n_text=37, seed_index=1271)  # own tokens: 466
    qr, kr, vr = W.make_inputs(wr)
    q, k, v = W.make_inputs(wq)
    rec_r = sol.qkv_encode(qr.to(DEV), kr.to(DEV), vr.to(DEV), wr.T, wr.Hl, wr.Wl,
                           _table(wr.T, wr.Hl, wr.Wl))
    rec = sol.qkv_encode(q.to(DEV), k.to(DEV), v.to(DEV), wq.T, wq.Hl, wq.Wl,
                         _table(wq.T, wq.Hl, wq.Wl))
    n_kv = wr.N + wq.N
    outs = []
    for order in ((0, 1), (1, 0)):
        kp, vp = sol.prepared_kv_buffers(B, H, n_kv, DEV)
        kp.view(torch.int16).fill_(0x7E00)  # NaN in fp16: any key left unwritten would show
        vp.view(torch.int16).fill_(0x7E00)
        for i in order:
            sol.prepare_kv_records(rec_r if i == 0 else rec, kp, vp, key0=0 if i == 0 else wr.N,
                                   n_kv=n_kv)
        outs.append(sol.attn_fwd_records(rec, kp, vp, n_kv=n_kv))
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    orec_r = _oracle_records(qr, kr, vr, wr.T, wr.Hl, wr.Wl)
    orec = _oracle_records(q, k, v, wq.T, wq.Hl, wq.Wl)
    dq, dk, dv = oracle.decode_qkv(orec)
    _, dkr, dvr = oracle.decode_qkv(orec_r)
    ref = oracle.attn_rows(dq, np.concatenate([dkr, dk], 2), np.concatenate([dvr, dv], 2), 0, 0, 0,
                           rope=False)
    R = B * H * wq.N
    st = compare(_bits(outs[0]).reshape(R, 128), ref.reshape(R, 128), np.repeat(np.arange(B * H), wq.N))
    _log("records key segments: %s" % st)
    assert_parity(st, "records key segments")


def test_records_p720_sampled_parity():
    """Full 720p size (B=1, H=40, N=111,600) as the benchmark runs it: the
    encoder with the rotation fused, then the receiver's prepare pass and
    attention; sampled rows of the first and last heads against the oracle
    (which encodes only those heads: a record depends on its own token and
    head alone)."""
    w = W.WORKLOADS["p720"]
    _log("generating %s" % w.describe())
    q, k, v = W.make_inputs(w)
    rec = sol.qkv_encode(q.to(DEV), k.to(DEV), v.to(DEV), w.T, w.Hl, w.Wl, _table(w.T, w.Hl, w.Wl))
    out = _gpu_attention(rec)
    torch.cuda.synchronize()
    rows_all = W.sample_rows(w, per_slab=16, head=32, tail=80).numpy()
    for h in (0, w.H - 1):
        rows = rows_all[rows_all // w.N == h] - h * w.N
        sl = slice(h, h + 1)
        orec = _oracle_records(q[:, sl], k[:, sl], v[:, sl], w.T, w.Hl, w.Wl)
        ref = _oracle_attention(orec, rows=rows)
        got = _bits(out[:, sl]).reshape(-1, w.D)[rows]
        st = compare(got, ref, np.zeros(len(rows), np.int64))
        _log("p720 records, head %d: %s" % (h, st))
        assert_parity(st, "p720 records head %d" % h)
