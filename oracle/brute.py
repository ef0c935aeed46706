"""Brute-force numpy twin of the oracle, float64, for tiny inputs.  Test infrastructure.

Written independently of solref.c: the rotary embedding is complex
multiplication by exp(j*phi) over explicit per-token positions, attention
materialises the full score matrix and normalises it with scipy's softmax.
"""
import numpy as np
from scipy.special import softmax


def grid_positions(N, T, Hl, Wl):
    """Per-token (t, h, w) positions, int64 [N, 3]; -1 marks prefix (text) tokens.

    Packing is text first, then the video latent in t-major raster order
    (Sec. 3.4 "Safety rails": prefix tokens precede the target video).
    """
    nv = T * Hl * Wl
    nt = N - nv
    if nt < 0:
        raise ValueError("grid larger than the sequence")
    pos = -np.ones((N, 3), dtype=np.int64)
    tt, hh, ww = np.meshgrid(np.arange(T), np.arange(Hl), np.arange(Wl), indexing="ij")
    pos[nt:, 0] = tt.reshape(-1)
    pos[nt:, 1] = hh.reshape(-1)
    pos[nt:, 2] = ww.reshape(-1)
    return pos


def rope_angles(pos, D=128, split=(32, 48, 48), base=10000.0):
    """Rotation angle of every interleaved pair, float64 [N, D/2].

    Pair i of the chunk owned by axis a (width d_a) turns by
    pos_a * base**(-2 i / d_a); prefix tokens (pos < 0) and pairs beyond the
    three chunks do not turn.
    """
    N = pos.shape[0]
    ang = np.zeros((N, D // 2), dtype=np.float64)
    off = 0
    for a, d in enumerate(split):
        freq = base ** (-2.0 * np.arange(d // 2) / d)
        p = np.where(pos[:, a] >= 0, pos[:, a], 0).astype(np.float64)
        ang[:, off // 2: off // 2 + d // 2] = p[:, None] * freq[None, :]
        off += d
    return ang


def rope_np(x, ang):
    """Rotate x[..., N, D] (float64): (x_2i + j x_2i+1) * exp(j ang_i)."""
    z = x[..., 0::2] + 1j * x[..., 1::2]
    z = z * np.exp(1j * ang)
    y = np.empty_like(x, dtype=np.float64)
    y[..., 0::2] = z.real
    y[..., 1::2] = z.imag
    return y


def bf16_bits_to_f64(bits):
    """uint16 bf16 bit patterns -> float64 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def nearest_bf16(x):
    """Round float64 to the nearest bf16 (ties to even mantissa) by comparing the
    two bf16 neighbours, found by truncating the float32 bit pattern.  Finite,
    in-range inputs only.  Returns float64 values."""
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)  # may round; fix below with exact neighbour search
    bits = f.view(np.uint32) & np.uint32(0xFFFF0000)
    lo = bits.view(np.float32).astype(np.float64)
    # neighbours of the truncated value one bf16 step either side
    up = (bits + np.uint32(0x10000)).view(np.float32).astype(np.float64)
    dn = (bits - np.uint32(0x10000)).view(np.float32).astype(np.float64)
    cands = np.stack([dn, lo, up], axis=-1)
    dist = np.abs(cands - x[..., None])
    best = dist.min(axis=-1, keepdims=True)
    tie = dist == best
    cbits = np.stack([bits - np.uint32(0x10000), bits, bits + np.uint32(0x10000)], axis=-1)
    even = ((cbits >> np.uint32(16)) & np.uint32(1)) == 0
    pick = np.where(tie.sum(-1, keepdims=True) > 1, tie & even, tie)
    idx = np.argmax(pick, axis=-1)
    return np.take_along_axis(cands, idx[..., None], axis=-1)[..., 0]


def rms_norm_np(x, gamma, eps):
    """x / sqrt(mean(x^2) + eps) * gamma over the last axis (the head's D
    entries), float64: the QK normalization of Sec. 3.5's fusion group 2."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(np.square(x), axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gamma, dtype=np.float64)


def attention_np(qh, kh, v):
    """softmax(qh kh^T / sqrt(D)) v over the last two axes, float64, materialised."""
    D = qh.shape[-1]
    s = np.matmul(qh, np.swapaxes(kh, -1, -2)) / np.sqrt(D)
    p = softmax(s, axis=-1)
    return np.matmul(p, v), p


def prepare_np(x_bits, T, Hl, Wl, gamma=None, eps=0.0, rope=True, contract=True,
               split=(32, 48, 48), base=10000.0):
    """One side (queries or keys) of the path on bf16 bits [..., N, D]: optional
    RMS normalisation, then the rotation, then (contract) one bf16 rounding of
    every row that was changed.  float64 out."""
    x = bf16_bits_to_f64(x_bits)
    N, D = x.shape[-2], x.shape[-1]
    changed = np.zeros(N, dtype=bool)
    if gamma is not None:
        x = rms_norm_np(x, gamma, eps)
        changed[:] = True
    if rope:
        pos = grid_positions(N, T, Hl, Wl)
        x = rope_np(x, rope_angles(pos, D, split, base))
        changed |= pos[:, 0] >= 0
    if contract:
        x = np.where(changed[:, None], nearest_bf16(x), x)
    return x


def fused_reference(q_bits, k_bits, v_bits, T, Hl, Wl, contract=True,
                    split=(32, 48, 48), base=10000.0, q_gamma=None, k_gamma=None, eps=0.0,
                    kv_grid=None, rope_k=True):
    """The whole path on bf16 bits q [B, H, Nq, D], k, v [B, H, Nkv, D]:
    normalise (when a gamma is given) and rotate q and k (rounding once to bf16
    in contract mode), then exact attention.  The keys use kv_grid when given,
    else the queries' grid.  Returns (out, probs)."""
    v = bf16_bits_to_f64(v_bits)
    Tk, Hlk, Wlk = kv_grid if kv_grid is not None else (T, Hl, Wl)
    qh = prepare_np(q_bits, T, Hl, Wl, q_gamma, eps, True, contract, split, base)
    kh = prepare_np(k_bits, Tk, Hlk, Wlk, k_gamma, eps, rope_k, contract, split, base)
    return attention_np(qh, kh, v)


def e4m3_values():
    """The value of every FP8 E4M3 code 0..255 (OCP E4M3FN: bias 7, 3 mantissa
    bits, no infinities, 0x7F and 0xFF NaN), float64 [256], from the format's
    definition."""
    vals = np.empty(256, dtype=np.float64)
    for c in range(256):
        s = -1.0 if c & 0x80 else 1.0
        e = (c >> 3) & 0xF
        m = c & 7
        if e == 0xF and m == 7:
            vals[c] = np.nan
        elif e == 0:
            vals[c] = s * m * 2.0 ** -9
        else:
            vals[c] = s * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return vals


def nearest_e4m3(x):
    """Round float64 to the nearest finite E4M3 code by searching all of them
    (ties to the even code, saturating at +-448); finite inputs.  uint8 codes."""
    # beyond 448 the nearest finite code is +-448; clipping first keeps the
    # distances below exact for huge inputs
    x = np.clip(np.asarray(x, dtype=np.float64), -512.0, 512.0)
    vals = e4m3_values()
    codes = np.array([c for c in range(256) if np.isfinite(vals[c]) and c != 0x80], dtype=np.int64)
    cv = vals[codes]
    dist = np.abs(x[..., None] - cv)
    best = dist.min(axis=-1, keepdims=True)
    tie = dist == best
    even = (codes & 1) == 0
    pick = np.where(tie.sum(-1, keepdims=True) > 1, tie & even, tie)
    c = codes[np.argmax(pick, axis=-1)]
    # signed zero: keep the sign of x (code 0x80 is -0)
    c = np.where((cv[np.argmax(pick, axis=-1)] == 0) & np.signbit(x), 0x80, c)
    return c.astype(np.uint8)


def sparse_route_np(qh, kh, n_prefix, tau, qblk, kblk):
    """Block routing on the prepared rows qh, kh [..., N, D] (float64): mean-pooled
    blocks, scaled dot products, threshold mean + tau * std (numpy's population
    std), plus the prefix key blocks, the first best block, and every key block
    for query blocks holding a prefix row.  Returns (mask bool [..., nqb, nkb], scores)."""
    N, D = qh.shape[-2], qh.shape[-1]
    nqb, nkb = -(-N // qblk), -(-N // kblk)
    qbar = np.stack([qh[..., I * qblk:(I + 1) * qblk, :].mean(-2) for I in range(nqb)], -2)
    kbar = np.stack([kh[..., J * kblk:(J + 1) * kblk, :].mean(-2) for J in range(nkb)], -2)
    s = np.matmul(qbar, np.swapaxes(kbar, -1, -2)) / np.sqrt(D)
    thr = s.mean(-1, keepdims=True) + tau * s.std(-1, keepdims=True)
    mask = s > thr
    best = np.argmax(s, axis=-1)
    np.put_along_axis(mask, best[..., None], True, axis=-1)
    mask[..., :, (np.arange(nkb) * kblk) < n_prefix] = True
    mask[..., (np.arange(nqb) * qblk) < n_prefix, :] = True
    return mask, s


def sparse_attention_np(qh, kh, v, mask, qblk, kblk):
    """Exact attention where query i sees only the keys of the key blocks
    mask[i // qblk] keeps: the full score matrix with -inf elsewhere, scipy softmax."""
    N, D = qh.shape[-2], qh.shape[-1]
    s = np.matmul(qh, np.swapaxes(kh, -1, -2)) / np.sqrt(D)
    keys = np.repeat(np.repeat(mask, qblk, axis=-2), kblk, axis=-1)[..., :N, :kh.shape[-2]]
    s = np.where(keys, s, -np.inf)
    return np.matmul(softmax(s, axis=-1), v)


def ue5m3_values():
    """The value of every UE5M3 scale code 0..255 (unsigned, 5 exponent bits of
    bias 15, 3 mantissa bits; exponent 31 infinity or NaN), float64 [256], from
    the format's definition."""
    vals = np.empty(256, dtype=np.float64)
    for c in range(256):
        e, m = c >> 3, c & 7
        if e == 31:
            vals[c] = np.inf if m == 0 else np.nan
        elif e == 0:
            vals[c] = m * 2.0 ** -17
        else:
            vals[c] = (1.0 + m / 8.0) * 2.0 ** (e - 15)
    return vals


def encode_records_np(qh_bits, kh_bits, v_bits):
    """Block-INT8 QKV records (uint8 [B, N, H, 400]) of bf16 bits [B, H, N, 128],
    vectorised: per 32-value group the smallest finite positive UE5M3 scale s
    with 127 s >= max |x|, codes round(x / s) (numpy rounds half to even)
    clipped to +-127; scales after the 384 code bytes, then 4 zero bytes."""
    vals = ue5m3_values()
    fin = vals[1:0xF8]                                       # codes 1..0xF7, increasing
    parts = [bf16_bits_to_f64(x) for x in (qh_bits, kh_bits, v_bits)]
    B, H, N, D = parts[0].shape
    codes, scales = [], []
    for x in parts:
        g = x.reshape(B, H, N, D // 32, 32)
        amax = np.abs(g).max(-1)
        sc = 1 + np.searchsorted(127.0 * fin, amax, side="left")  # first with 127 s >= amax
        sc = np.minimum(sc, 0xF7)
        s = vals[sc][..., None]
        c = np.clip(np.rint(g / s), -127, 127).astype(np.int8).reshape(B, H, N, D)
        codes.append(c.view(np.uint8))
        scales.append(sc.astype(np.uint8))
    rec = np.zeros((B, N, H, 400), dtype=np.uint8)
    for p in range(3):
        rec[..., 128 * p:128 * (p + 1)] = np.transpose(codes[p], (0, 2, 1, 3))
        rec[..., 384 + 4 * p:388 + 4 * p] = np.transpose(scales[p], (0, 2, 1, 3))
    return rec


def decode_records_np(rec):
    """uint8 records [B, N, H, 400] -> float64 (q, k, v) [B, H, N, 128]: code
    times its group's scale, before any rounding."""
    vals = ue5m3_values()
    out = []
    for p in range(3):
        c = rec[..., 128 * p:128 * (p + 1)].view(np.int8).astype(np.float64)
        s = np.repeat(vals[rec[..., 384 + 4 * p:388 + 4 * p]], 32, axis=-1)
        out.append(np.transpose(c * s, (0, 2, 1, 3)))
    return tuple(out)
