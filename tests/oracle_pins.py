"""Pins of the CPU oracle against things other than itself.

Each ``pin_*`` takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with a closed form, an invariant, a library routine
(torch SDPA, torch's float->bf16 conversion, scipy rotations) or the
independent numpy brute force.  ``test_oracle.py`` runs them on the real
oracle and on deliberately broken copies of it (each copy must fail one).

Nothing the paper prints pins these values numerically: it gives no worked
example of the rotary embedding or of attention.  The paper fixes *what* is
computed (3D rotary embedding on q and k, then exact softmax attention, with
the text prefix unrotated); the pins below check that meaning.
"""
import math
import os

import numpy as np
import torch
from scipy.spatial.transform import Rotation

from oracle import brute

SPLIT = (32, 48, 48)
BASE = 10000.0
D = 128


def _bits(x):
    """float array -> bf16 bit patterns via torch's own conversion."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _rand_bits(rng, shape, std=1.0):
    return _bits(rng.standard_normal(shape) * std)


def _f(bits):
    return brute.bf16_bits_to_f64(bits)


# --------------------------------------------------------------- bf16 rounding

def pin_round_bf16_vs_torch(o):
    """RNE to bf16 equals torch's float32->bfloat16 conversion (library routine),
    including exact ties, subnormals, zeros and overflow to infinity."""
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(20000) * np.exp2(rng.integers(-140, 120, 20000))).astype(np.float32)
    # exact ties: a bf16 value plus half of its quantum
    base = _f(_bits(rng.standard_normal(2000)))
    quantum = np.exp2(np.floor(np.log2(np.abs(base))) - 7)
    ties = (base + 0.5 * quantum * np.sign(base)).astype(np.float32)
    specials = np.array([0.0, -0.0, 1e-45, -1e-45, 3.0e38, -3.4e38, 1.0, 1.00390625,
                         1.01171875, 2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -134], dtype=np.float32)
    for xs in (x, ties, specials):
        got = o.round_bf16(xs.astype(np.float64))
        want = torch.from_numpy(xs).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(got, want), "bf16 rounding differs from torch"


def pin_round_bf16_double_nearest(o):
    """For doubles that float32 cannot hold, the result is the nearest bf16
    (ties to even), found by brute-force neighbour comparison."""
    rng = np.random.default_rng(2)
    x = rng.standard_normal(20000) * np.exp2(rng.integers(-30, 30, 20000))
    got = _f(o.round_bf16(x))
    want = brute.nearest_bf16(x)
    assert np.array_equal(got, want), "bf16 rounding of doubles is not nearest-even"


# ----------------------------------------------------------- rotary embedding

def _extract_angles(o, N, T, Hl, Wl):
    """Rotate the unit vectors e_0 and e_1 of every pair at every token; return
    the per-pair 2x2 matrices [N, D/2, 2, 2] (columns = images of e_0, e_1)."""
    e0 = np.zeros((N, D))
    e0[:, 0::2] = 1.0
    e1 = np.zeros((N, D))
    e1[:, 1::2] = 1.0
    y0 = o.rope3d_f64(e0, T, Hl, Wl, SPLIT, BASE)
    y1 = o.rope3d_f64(e1, T, Hl, Wl, SPLIT, BASE)
    M = np.empty((N, D // 2, 2, 2))
    M[..., 0, 0] = y0[:, 0::2]
    M[..., 1, 0] = y0[:, 1::2]
    M[..., 0, 1] = y1[:, 0::2]
    M[..., 1, 1] = y1[:, 1::2]
    return M


def pin_rope_pairs_are_rotations(o):
    """Every interleaved pair is turned by a proper, counter-clockwise planar
    rotation (scipy's z-axis rotation by the extracted angle), and the map is
    linear in the input."""
    T, Hl, Wl = 2, 3, 4
    N = T * Hl * Wl + 3
    M = _extract_angles(o, N, T, Hl, Wl)
    phi = np.arctan2(M[..., 1, 0], M[..., 0, 0])
    R = Rotation.from_rotvec(np.stack([np.zeros(phi.size), np.zeros(phi.size), phi.ravel()], -1))
    want = R.as_matrix()[:, :2, :2].reshape(M.shape)
    assert np.allclose(M, want, atol=1e-13), "a pair is not rotated by a proper rotation"
    rng = np.random.default_rng(3)
    a, b = rng.standard_normal((2, N, D))
    lhs = o.rope3d_f64(2.0 * a - 3.0 * b, T, Hl, Wl, SPLIT, BASE)
    rhs = 2.0 * o.rope3d_f64(a, T, Hl, Wl, SPLIT, BASE) - 3.0 * o.rope3d_f64(b, T, Hl, Wl, SPLIT, BASE)
    assert np.allclose(lhs, rhs, atol=1e-12), "rotation is not linear"


def pin_rope_axis_chunks(o):
    """A grid that varies along one axis only changes only that axis's head dims:
    t -> [0,32), h -> [32,80), w -> [80,128)."""
    rng = np.random.default_rng(4)
    chunks = {0: (0, 32), 1: (32, 80), 2: (80, 128)}
    for axis in range(3):
        dims = [1, 1, 1]
        dims[axis] = 5
        N = 5
        x = rng.standard_normal((N, D))
        y = o.rope3d_f64(x, *dims, SPLIT, BASE)
        lo, hi = chunks[axis]
        keep = np.ones(D, bool)
        keep[lo:hi] = False
        assert np.array_equal(y[:, keep], x[:, keep]), "dims outside the axis chunk changed"
        assert np.abs(y[1:, lo:hi] - x[1:, lo:hi]).max() > 1e-3, "axis chunk did not rotate"


def pin_rope_frequency_schedule(o):
    """At position 1 along an axis of width d, pair i turns by theta_i with
    theta_0 = 1 rad and theta_{i+1}/theta_i = base^(-2/d) (a geometric
    progression with the stated base over the axis's own width)."""
    for axis, (lo, d) in enumerate([(0, 32), (32, 48), (80, 48)]):
        dims = [1, 1, 1]
        dims[axis] = 2
        M = _extract_angles(o, 2, *dims)
        phi = np.arctan2(M[1, :, 1, 0], M[1, :, 0, 0])
        sect = phi[lo // 2: (lo + d) // 2]
        assert abs(sect[0] - 1.0) < 1e-14, "lowest pair must turn by pos * 1 rad"
        ratio = sect[1:] / sect[:-1]
        assert np.allclose(ratio, BASE ** (-2.0 / d), rtol=1e-12), "frequencies not geometric in base^(-2/d)"
        others = np.ones(D // 2, bool)
        others[lo // 2: (lo + d) // 2] = False
        assert np.all(phi[others] == 0.0)


def pin_rope_token_order(o):
    """Tokens are a text prefix (unrotated) then the latent in t-major raster
    order; read back through the lowest pair of each axis, which turns by
    exactly the position (positions < pi, no wrap)."""
    T, Hl, Wl, nt = 2, 3, 3, 4
    N = nt + T * Hl * Wl
    M = _extract_angles(o, N, T, Hl, Wl)
    got = np.stack([np.arctan2(M[:, c, 1, 0], M[:, c, 0, 0]) for c in (0, 16, 40)], -1)
    want = np.zeros((N, 3))
    n = 0
    for t in range(T):
        for h in range(Hl):
            for w in range(Wl):
                want[nt + n] = (t, h, w)
                n += 1
    assert np.allclose(got, want, atol=1e-13), "token -> (t, h, w) order is not t-major raster"


def pin_rope_prefix_identity_and_origin(o):
    """Prefix tokens and the latent at (0, 0, 0) come back bit-identical."""
    rng = np.random.default_rng(5)
    T, Hl, Wl, nt = 2, 2, 2, 3
    x_bits = _rand_bits(rng, (1, 2, nt + T * Hl * Wl, D))
    y_bits = o.rope3d_bf16(x_bits, T, Hl, Wl, SPLIT, BASE)
    assert np.array_equal(y_bits[..., : nt + 1, :], x_bits[..., : nt + 1, :])
    assert not np.array_equal(y_bits[..., nt + 1:, :], x_bits[..., nt + 1:, :])


def pin_rope_group_law(o):
    """R(p1) R(p2) = R(p1 + p2) and norms of pairs are preserved, using tokens
    of one grid whose positions add up."""
    rng = np.random.default_rng(6)
    T, Hl, Wl = 4, 4, 4
    N = T * Hl * Wl

    def tok(t, h, w):
        return (t * Hl + h) * Wl + w

    x = rng.standard_normal(D)
    for p1, p2 in [((1, 0, 2), (2, 3, 1)), ((0, 1, 1), (3, 2, 2)), ((1, 1, 1), (1, 1, 1))]:
        p3 = tuple(a + b for a, b in zip(p1, p2))
        buf = np.zeros((N, D))
        buf[tok(*p1)] = x
        y = o.rope3d_f64(buf, T, Hl, Wl, SPLIT, BASE)[tok(*p1)]
        buf[:] = 0
        buf[tok(*p2)] = y
        y2 = o.rope3d_f64(buf, T, Hl, Wl, SPLIT, BASE)[tok(*p2)]
        buf[:] = 0
        buf[tok(*p3)] = x
        y3 = o.rope3d_f64(buf, T, Hl, Wl, SPLIT, BASE)[tok(*p3)]
        assert np.allclose(y2, y3, atol=1e-12), "rotations do not compose additively"
        assert np.allclose(np.hypot(y[0::2], y[1::2]), np.hypot(x[0::2], x[1::2]), atol=1e-13)


def pin_rope_relative_position(o):
    """<R(p) q, R(p') k> depends on p - p' only: shifting both tokens by the
    same offset along any axis leaves the score unchanged."""
    rng = np.random.default_rng(7)
    T, Hl, Wl = 5, 5, 5
    N = T * Hl * Wl

    def tok(t, h, w):
        return (t * Hl + h) * Wl + w

    q, k = rng.standard_normal((2, D))
    qs = np.broadcast_to(q, (N, D))
    ks = np.broadcast_to(k, (N, D))
    rq = o.rope3d_f64(qs, T, Hl, Wl, SPLIT, BASE)
    rk = o.rope3d_f64(ks, T, Hl, Wl, SPLIT, BASE)
    ref = rq[tok(1, 0, 2)] @ rk[tok(0, 2, 1)]
    for c in [(1, 0, 0), (0, 2, 0), (0, 0, 2), (3, 2, 1)]:
        a = tok(1 + c[0], 0 + c[1], 2 + c[2])
        b = tok(0 + c[0], 2 + c[1], 1 + c[2])
        assert abs(rq[a] @ rk[b] - ref) < 1e-10, "score is not a function of relative position"


def pin_rope_numpy_twin(o):
    """The C rotation equals the numpy complex-multiplication twin (with a prefix)."""
    rng = np.random.default_rng(8)
    T, Hl, Wl, nt = 3, 4, 5, 7
    N = nt + T * Hl * Wl
    x = rng.standard_normal((2, 3, N, D))
    ang = brute.rope_angles(brute.grid_positions(N, T, Hl, Wl), D, SPLIT, BASE)
    assert np.allclose(o.rope3d_f64(x, T, Hl, Wl, SPLIT, BASE), brute.rope_np(x, ang), atol=1e-12)


def pin_rope_partial_split(o):
    """Partial RoPE under a split (dt, dh, dw) with dt + dh + dw < D: the dims
    past dt + dh + dw pass through bit for bit, every other pair is a
    rotation, and at position 1 along axis a the pairs of that axis's section
    turn by a geometric progression starting at 1 rad with ratio
    base^(-2/d_a), d_a the split's own width (not the default one)."""
    rng = np.random.default_rng(10)
    for split in [(16, 24, 24), (0, 64, 64), (8, 0, 40)]:
        tot = sum(split)
        T, Hl, Wl = 3, 4, 5
        N = T * Hl * Wl
        x = rng.standard_normal((N, D))
        y = o.rope3d_f64(x, T, Hl, Wl, split, BASE)
        assert np.array_equal(y[:, tot:], x[:, tot:]), "pass-through dims changed under %s" % (split,)
        assert np.allclose(np.hypot(y[:, 0::2], y[:, 1::2]), np.hypot(x[:, 0::2], x[:, 1::2]), atol=1e-12)
        off = 0
        for axis, d in enumerate(split):
            if d:
                dims = [1, 1, 1]
                dims[axis] = 2
                u = np.zeros((2, D))
                u[:, 0::2] = 1.0  # every pair starts at angle 0
                r = o.rope3d_f64(u, *dims, split, BASE)  # token 1 sits at position 1 on `axis`
                ang = np.arctan2(r[1, off + 1:off + d:2], r[1, off:off + d:2])
                want = BASE ** (-2.0 * np.arange(d // 2) / d)
                assert np.allclose(ang, want, atol=1e-12), "axis %d of split %s" % (axis, split)
            off += d


def pin_rope_contract_rounding(o):
    """Contract mode is exactly: rotate in double, round once to nearest bf16."""
    rng = np.random.default_rng(9)
    T, Hl, Wl = 3, 8, 8
    x_bits = _rand_bits(rng, (1, 2, T * Hl * Wl, D))
    got = _f(o.rope3d_bf16(x_bits, T, Hl, Wl, SPLIT, BASE))
    want = brute.nearest_bf16(o.rope3d_f64(_f(x_bits), T, Hl, Wl, SPLIT, BASE))
    assert np.array_equal(got, want)


# ------------------------------------------------------------------ attention

def _sdpa64(q, k, v):
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v)).numpy()


def pin_attention_vs_torch_sdpa(o):
    """Without rotation the oracle is torch's scaled_dot_product_attention
    (float64, default 1/sqrt(D) scale) on the same values."""
    rng = np.random.default_rng(10)
    for N, std in [(37, 1.0), (130, 3.0), (1, 1.0)]:
        q, k, v = (_rand_bits(rng, (1, 3, N, D), std) for _ in range(3))
        got = o.attn_rows(q, k, v, 0, 0, 0, rope=False)
        want = _sdpa64(_f(q), _f(k), _f(v))
        assert np.allclose(got, want, atol=2e-6, rtol=1e-6), "plain attention differs from SDPA"


def pin_attention_unit_grid_is_sdpa(o):
    """A 1x1x1 grid (the lone latent token sits at the origin) plus a text
    prefix rotates nothing, so the RoPE path also equals SDPA."""
    rng = np.random.default_rng(11)
    N = 9
    q, k, v = (_rand_bits(rng, (2, 2, N, D)) for _ in range(3))
    got = o.attn_rows(q, k, v, 1, 1, 1, rope=True)
    assert np.allclose(got, _sdpa64(_f(q), _f(k), _f(v)), atol=2e-6, rtol=1e-6)


def pin_attention_vs_brute(o):
    """Rotated attention equals the numpy brute force (materialised scores,
    scipy softmax) on tiny grids, with and without a text prefix, in contract
    and pure-double modes."""
    rng = np.random.default_rng(12)
    for (T, Hl, Wl, nt) in [(2, 2, 3, 0), (2, 2, 3, 5), (3, 8, 8, 0)]:
        N = nt + T * Hl * Wl
        q, k, v = (_rand_bits(rng, (1, 2, N, D)) for _ in range(3))
        for contract in (True, False):
            got = o.attn_rows(q, k, v, T, Hl, Wl, contract=contract)
            want, _ = brute.fused_reference(q, k, v, T, Hl, Wl, contract=contract)
            assert np.allclose(got, want, atol=2e-6, rtol=1e-6), "rotated attention differs from brute force"


def pin_attention_weights_sum_to_one(o):
    """With one value column all ones the output in that column is the softmax
    row sum, 1."""
    rng = np.random.default_rng(13)
    T, Hl, Wl = 2, 3, 4
    N = T * Hl * Wl
    q, k, v = (_rand_bits(rng, (1, 2, N, D), 2.0) for _ in range(3))
    v = v.copy()
    v[..., 5] = _bits(np.ones(1))[0]
    out = o.attn_rows(q, k, v, T, Hl, Wl)
    assert np.allclose(out[..., 5], 1.0, atol=1e-6)


def pin_attention_constant_v(o):
    """Every v_j = c gives o_i = c exactly (up to float32 output rounding)."""
    rng = np.random.default_rng(14)
    T, Hl, Wl = 2, 3, 4
    N = T * Hl * Wl + 2
    q, k = (_rand_bits(rng, (1, 2, N, D), 3.0) for _ in range(2))
    c = _bits(rng.standard_normal(D))
    v = np.broadcast_to(c, (1, 2, N, D)).copy()
    out = o.attn_rows(q, k, v, T, Hl, Wl)
    assert np.allclose(out, np.broadcast_to(_f(c), out.shape), atol=1e-6, rtol=1e-6)


def pin_attention_joint_permutation(o):
    """Permuting the (rotated key, value) pairs together leaves every output
    unchanged; the fused call equals rotate-then-attend."""
    rng = np.random.default_rng(15)
    T, Hl, Wl, nt = 2, 3, 4, 3
    N = nt + T * Hl * Wl
    q, k, v = (_rand_bits(rng, (1, 2, N, D)) for _ in range(3))
    ref = o.attn_rows(q, k, v, T, Hl, Wl)
    qh = o.rope3d_bf16(q, T, Hl, Wl, SPLIT, BASE)
    kh = o.rope3d_bf16(k, T, Hl, Wl, SPLIT, BASE)
    perm = rng.permutation(N)
    out = o.attn_rows(qh, np.ascontiguousarray(kh[:, :, perm]), np.ascontiguousarray(v[:, :, perm]),
                      0, 0, 0, rope=False)
    assert np.allclose(out, ref, atol=1e-6, rtol=1e-6)


def pin_attention_one_hot(o):
    """A key aligned with the query and a logit gap >= 40 takes all the weight:
    o_i = v_{j*}."""
    rng = np.random.default_rng(16)
    N = 50
    q = _rand_bits(rng, (1, 1, N, D), 0.05)
    k = _rand_bits(rng, (1, 1, N, D), 0.05)
    v = _rand_bits(rng, (1, 1, N, D))
    i, j = 7, 31
    q[0, 0, i] = _bits(np.full(D, 2.0))
    k[0, 0, j] = _bits(np.full(D, 2.0))  # logit 4*128/sqrt(128) = 45 against ~0
    out = o.attn_rows(q, k, v, 0, 0, 0, rope=False)
    assert np.allclose(out[0, 0, i], _f(v[0, 0, j]), atol=1e-12 + 1e-12)


def pin_attention_zero_query(o):
    """q = 0 gives uniform weights: o_i = mean_j v_j."""
    rng = np.random.default_rng(17)
    T, Hl, Wl = 2, 2, 5
    N = T * Hl * Wl
    k, v = (_rand_bits(rng, (1, 2, N, D)) for _ in range(2))
    q = np.zeros_like(k)
    out = o.attn_rows(q, k, v, T, Hl, Wl)
    want = _f(v).mean(axis=2, keepdims=True)
    assert np.allclose(out, np.broadcast_to(want, out.shape), atol=1e-6)


def pin_attention_two_key_closed_form(o):
    """Two keys with logits a and 0 weigh their values by e^a : 1."""
    q = np.zeros((1, 1, 2, D), np.uint16)
    k = np.zeros((1, 1, 2, D), np.uint16)
    v = np.zeros((1, 1, 2, D), np.uint16)
    q[0, 0, :, 0] = _bits([1.5, 1.5])
    k[0, 0, 0, 0] = _bits([3.0])[0]
    v[0, 0, 0, 1] = _bits([1.0])[0]
    v[0, 0, 1, 2] = _bits([1.0])[0]
    a = 1.5 * 3.0 / math.sqrt(D)
    out = o.attn_rows(q, k, v, 0, 0, 0, rope=False)
    w = math.exp(a) / (math.exp(a) + 1.0)
    assert abs(out[0, 0, 0, 1] - w) < 1e-7 and abs(out[0, 0, 0, 2] - (1 - w)) < 1e-7


def pin_attention_rows_and_threads(o):
    """A row subset (any order) reproduces the full computation bit for bit,
    for one thread and many."""
    rng = np.random.default_rng(18)
    T, Hl, Wl = 2, 3, 5
    N = T * Hl * Wl
    q, k, v = (_rand_bits(rng, (2, 2, N, D)) for _ in range(3))
    full = o.attn_rows(q, k, v, T, Hl, Wl, threads=1)
    rows = rng.permutation(2 * 2 * N)[:17]
    sub = o.attn_rows(q, k, v, T, Hl, Wl, rows=rows, threads=4)
    assert np.array_equal(sub, full.reshape(-1, D)[rows])


# ------------------------------------------------- QK normalization (RMSNorm)

def _gamma(rng, spread=0.3):
    """Non-uniform per-dimension weights (bf16-exact values, as model weights)."""
    return _f(_bits(1.0 + spread * rng.standard_normal(D)))


def pin_qknorm_vs_torch_rms_norm(o):
    """Without rotation the normalisation is torch's rms_norm over the head's D
    entries (float64, weight gamma, eps under the root): in double, and after
    the one bf16 rounding."""
    rng = np.random.default_rng(30)
    for std, eps in [(1.0, 1e-6), (7.0, 0.0), (0.01, 1e-3)]:
        x = _rand_bits(rng, (2, 3, 21, D), std)
        g = _gamma(rng)
        want = torch.nn.functional.rms_norm(torch.from_numpy(_f(x)), (D,),
                                            weight=torch.from_numpy(g), eps=eps).numpy()
        got64 = o.qknorm_rope3d(x, 0, 0, 0, g, eps, rope=False, contract=False)
        assert np.allclose(got64, want, rtol=1e-14, atol=0), "normalisation differs from rms_norm"
        got = _f(o.qknorm_rope3d(x, 0, 0, 0, g, eps, rope=False))
        assert np.array_equal(got, brute.nearest_bf16(want)), "normalised rows not rounded once"


def pin_qknorm_unit_rms_rows_unchanged(o):
    """Rows whose root mean square is exactly 1 (entries +-1), unit weights and
    eps = 0: normalisation is the identity, so the result is the plain
    rotation (latent tokens) or the input itself (prefix tokens)."""
    rng = np.random.default_rng(31)
    T, Hl, Wl, nt = 2, 3, 4, 5
    N = nt + T * Hl * Wl
    x = _bits(rng.choice([-1.0, 1.0], size=(1, 2, N, D)))
    got = o.qknorm_rope3d(x, T, Hl, Wl, np.ones(D), 0.0)
    assert np.array_equal(got, o.rope3d_bf16(x, T, Hl, Wl, SPLIT, BASE))
    assert np.array_equal(got[:, :, :nt], x[:, :, :nt])


def pin_qknorm_gamma_closed_form(o):
    """A row of ones has mean square 1, so its normalised value is
    gamma / sqrt(1 + eps), dimension by dimension (prefix token: no rotation)."""
    rng = np.random.default_rng(32)
    g = _gamma(rng, 0.8)
    x = _bits(np.ones((1, 1, 3, D)))
    for eps in (0.0, 0.25, 3.0):
        got = o.qknorm_rope3d(x, 0, 0, 0, g, eps, contract=False)
        assert np.allclose(got, np.broadcast_to(g / math.sqrt(1.0 + eps), got.shape),
                           rtol=1e-15, atol=0)


def pin_qknorm_scale_invariance(o):
    """With eps = 0 the normalisation removes any positive scale of a row: rows
    scaled by powers of two (exact in bf16) give the same bits."""
    rng = np.random.default_rng(33)
    T, Hl, Wl = 2, 3, 4
    N = 3 + T * Hl * Wl
    x = _rand_bits(rng, (1, 2, N, D))
    g = _gamma(rng)
    scale = np.exp2(rng.integers(-6, 7, size=(1, 2, N, 1))).astype(np.float64)
    xs = _bits(_f(x) * scale)
    assert np.array_equal(o.qknorm_rope3d(x, T, Hl, Wl, g, 0.0), o.qknorm_rope3d(xs, T, Hl, Wl, g, 0.0))


def pin_qknorm_numpy_twin(o):
    """Normalise-then-rotate in C equals the numpy twin (rms_norm_np, then the
    complex rotation), with non-uniform weights that make the order matter."""
    rng = np.random.default_rng(34)
    T, Hl, Wl, nt = 3, 4, 5, 6
    N = nt + T * Hl * Wl
    x = _rand_bits(rng, (2, 2, N, D), 2.0)
    g = _gamma(rng, 0.5)
    got = o.qknorm_rope3d(x, T, Hl, Wl, g, 1e-6, contract=False)
    want = brute.prepare_np(x, T, Hl, Wl, g, 1e-6, contract=False)
    assert np.allclose(got, want, rtol=0, atol=1e-12)
    assert np.array_equal(_f(o.qknorm_rope3d(x, T, Hl, Wl, g, 1e-6)), brute.nearest_bf16(want))


def pin_attention_qknorm_vs_brute(o):
    """Attention with normalised and rotated q and k equals the numpy twin."""
    rng = np.random.default_rng(35)
    T, Hl, Wl, nt = 2, 3, 4, 4
    N = nt + T * Hl * Wl
    q, k, v = (_rand_bits(rng, (1, 2, N, D), 3.0) for _ in range(3))
    gq, gk = _gamma(rng, 0.5), _gamma(rng, 0.5)
    got = o.attn_rows(q, k, v, T, Hl, Wl, q_gamma=gq, k_gamma=gk, eps=1e-6)
    want, _ = brute.fused_reference(q, k, v, T, Hl, Wl, q_gamma=gq, k_gamma=gk, eps=1e-6)
    assert np.allclose(got, want, atol=2e-6, rtol=1e-6)


def pin_attention_qknorm_ignores_row_scale(o):
    """With eps = 0, scaling any query or key row by a power of two changes
    nothing (both sides are normalised before the products)."""
    rng = np.random.default_rng(36)
    T, Hl, Wl = 2, 2, 5
    N = 3 + T * Hl * Wl
    q, k, v = (_rand_bits(rng, (1, 2, N, D)) for _ in range(3))
    gq, gk = _gamma(rng), _gamma(rng)
    sq = np.exp2(rng.integers(-5, 6, size=(1, 2, N, 1))).astype(np.float64)
    sk = np.exp2(rng.integers(-5, 6, size=(1, 2, N, 1))).astype(np.float64)
    a = o.attn_rows(q, k, v, T, Hl, Wl, q_gamma=gq, k_gamma=gk, eps=0.0)
    b = o.attn_rows(_bits(_f(q) * sq), _bits(_f(k) * sk), v, T, Hl, Wl, q_gamma=gq, k_gamma=gk,
                    eps=0.0)
    assert np.array_equal(a, b)


# ------------------------------------------- queries and keys of other lengths

def pin_attention_kv_lengths_vs_sdpa(o):
    """Nq queries against Nkv != Nq keys, nothing rotated: torch SDPA (float64)."""
    rng = np.random.default_rng(37)
    for nq, nkv in [(37, 130), (130, 5), (1, 64)]:
        q = _rand_bits(rng, (2, 2, nq, D))
        k, v = (_rand_bits(rng, (2, 2, nkv, D)) for _ in range(2))
        got = o.attn_rows(q, k, v, 0, 0, 0, rope=False)
        assert got.shape == (2, 2, nq, D)
        want = _sdpa64(_f(q), _f(k), _f(v))
        assert np.allclose(got, want, atol=2e-6, rtol=1e-6)


def pin_attention_prefix_queries_of_self_attention(o):
    """Queries that are the text prefix of a sequence (Nq = Nt, unrotated)
    against that whole sequence's keys give exactly the first Nt rows of the
    sequence's self-attention."""
    rng = np.random.default_rng(38)
    T, Hl, Wl, nt = 2, 3, 4, 9
    N = nt + T * Hl * Wl
    q, k, v = (_rand_bits(rng, (1, 2, N, D)) for _ in range(3))
    full = o.attn_rows(q, k, v, T, Hl, Wl)
    part = o.attn_rows(np.ascontiguousarray(q[:, :, :nt]), k, v, 0, 0, 0, kv_grid=(T, Hl, Wl))
    assert np.array_equal(part, full[:, :, :nt])


def pin_attention_kv_segments_commute(o):
    """Keys and values made of two segments, each rotated with its own grid
    and then given as prepared keys: the order of the segments does not
    matter, and the result equals the numpy twin."""
    rng = np.random.default_rng(39)
    Tq, Hlq, Wlq = 2, 3, 3
    nq = 4 + Tq * Hlq * Wlq
    q = _rand_bits(rng, (1, 2, nq, D))
    segs = [((1, 4, 5), 3), ((2, 2, 2), 0)]  # (grid, prefix tokens)
    kh, vs = [], []
    for (T, Hl, Wl), nt in segs:
        n = nt + T * Hl * Wl
        k = _rand_bits(rng, (1, 2, n, D))
        kh.append(o.rope3d_bf16(k, T, Hl, Wl, SPLIT, BASE))
        vs.append(_rand_bits(rng, (1, 2, n, D)))
    ab = o.attn_rows(q, np.concatenate(kh, 2), np.concatenate(vs, 2), Tq, Hlq, Wlq, rope_k=False)
    ba = o.attn_rows(q, np.concatenate(kh[::-1], 2), np.concatenate(vs[::-1], 2), Tq, Hlq, Wlq,
                     rope_k=False)
    assert np.allclose(ab, ba, atol=1e-7, rtol=0)
    want, _ = brute.fused_reference(q, np.concatenate(kh, 2), np.concatenate(vs, 2), Tq, Hlq, Wlq,
                                    rope_k=False)
    assert np.allclose(ab, want, atol=2e-6, rtol=1e-6)


# ------------------------------------------------------- FP8 E4M3 output codes

def _e4m3_torch_codes(x):
    t = torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).numpy()


def _e4m3_test_values(rng):
    """Random values over the whole range (subnormals included), every exact
    midpoint between neighbouring finite codes, and the codes themselves."""
    vals = brute.e4m3_values()
    fin = np.sort(np.unique(vals[np.isfinite(vals)]))
    mids = (fin[:-1] + fin[1:]) / 2
    x = rng.standard_normal(20000) * np.exp2(rng.uniform(-11, 9, 20000))
    return np.concatenate([x, mids, fin, -mids])


def pin_e4m3_decode_table_is_torch(o):
    """The format's definition (numpy twin) decodes every code as torch's
    float8_e4m3fn does (library routine)."""
    want = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = brute.e4m3_values()
    assert np.array_equal(np.isnan(got), np.isnan(want))
    assert np.array_equal(got[~np.isnan(got)], want[~np.isnan(want)])


def pin_e4m3_round_vs_torch(o):
    """Inside the finite range (|x| < 464, where rounding cannot pass 448) the
    oracle's codes are torch's float8_e4m3fn conversion (round to nearest
    even), midpoints and subnormals included."""
    rng = np.random.default_rng(50)
    x = _e4m3_test_values(rng)
    x = x[np.abs(x) < 464].astype(np.float32).astype(np.float64)  # float32-exact inputs
    assert np.array_equal(o.round_e4m3(x), _e4m3_torch_codes(x))


def pin_e4m3_round_vs_brute(o):
    """The oracle's codes are the nearest finite code found by search (ties to
    the even code), saturating at +-448, over the whole range."""
    rng = np.random.default_rng(51)
    x = np.concatenate([_e4m3_test_values(rng), [449.0, -500.0, 1e6, -3e38]])
    assert np.array_equal(o.round_e4m3(x), brute.nearest_e4m3(x))


def pin_e4m3_saturation_and_specials(o):
    """Beyond the largest finite value (448) every input saturates, infinities
    included; NaN stays NaN; every finite code round-trips."""
    got = o.round_e4m3(np.array([448.0, 464.0, 1e4, np.inf, -np.inf, -449.0, np.nan, 0.0, -0.0]))
    assert got.tolist() == [0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE, 0x7F, 0x00, 0x80]
    vals = brute.e4m3_values()
    codes = np.array([c for c in range(256) if np.isfinite(vals[c])])
    assert np.array_equal(o.round_e4m3(vals[codes]), codes.astype(np.uint8))


# ----------------------------------------------------- block-sparse attention

def pin_sparse_route_vs_numpy_twin(o):
    """The C routing (pooled blocks, scores, mean + tau std threshold, sinks)
    equals the numpy twin, with and without QK normalisation, ragged blocks."""
    rng = np.random.default_rng(60)
    T, Hl, Wl, nt = 2, 6, 10, 37
    N = nt + T * Hl * Wl
    q, k = (_rand_bits(rng, (1, 2, N, D)) for _ in range(2))
    for tau, gq, gk in [(1.0, None, None), (0.25, _gamma(rng), _gamma(rng))]:
        m, sc, _ = o.sparse_route(q, k, T, Hl, Wl, tau, qblk=32, kblk=16, q_gamma=gq, k_gamma=gk,
                                  eps=1e-6)
        qh = brute.prepare_np(q, T, Hl, Wl, gq, 1e-6)
        kh = brute.prepare_np(k, T, Hl, Wl, gk, 1e-6)
        mb, sb = brute.sparse_route_np(qh, kh, nt, tau, 32, 16)
        assert np.allclose(sc, sb, rtol=0, atol=1e-12)
        assert np.array_equal(m.astype(bool), mb)
        assert 0.1 < m[:, :, 2:].mean() < 0.9, "routing should drop and keep blocks here"


def pin_sparse_threshold_closed_form(o):
    """Unrotated rows on one direction e: query rows a e, key block J rows c_J e,
    so s_J = a c_J / sqrt(D); c = (1, 2, 3, 10): mean 4, population std
    sqrt(12.5) (units a / sqrt(D)).  tau = 0.5 keeps block 3 only; -0.5 keeps
    blocks 2, 3 (the sample std would also keep block 1); -1.1 keeps all.  With
    one block kept, every query sees 8 equal keys: out = mean of their v."""
    e = np.zeros(D)
    e[5] = 1.0
    c = [1.0, 2.0, 3.0, 10.0]
    q = _bits(np.tile(0.5 * e, (1, 1, 32, 1)))
    k = _bits(np.concatenate([np.tile(cj * e, (1, 1, 8, 1)) for cj in c], axis=2))
    rng = np.random.default_rng(61)
    v = _rand_bits(rng, (1, 1, 32, D))
    for tau, want in [(0.5, [0, 0, 0, 1]), (-0.5, [0, 0, 1, 1]), (-1.1, [1, 1, 1, 1])]:
        m, _, _ = o.sparse_route(q, k, 1, 1, 32, tau, qblk=32, kblk=8, rope=False)
        assert m.reshape(-1).tolist() == want, (tau, m.reshape(-1).tolist())
    m, _, _ = o.sparse_route(q, k, 1, 1, 32, 0.5, qblk=32, kblk=8, rope=False)
    out = o.attn_rows(q, k, v, 1, 1, 32, rope=False, block_mask=m, qblk=32, kblk=8)
    assert np.allclose(out[0, 0], _f(v)[0, 0, 24:].mean(0)[None, :], atol=1e-6)


def pin_sparse_dense_limit(o):
    """tau -> -inf keeps every block, and the sparse attention is then the
    dense one bit for bit."""
    rng = np.random.default_rng(62)
    T, Hl, Wl, nt = 2, 5, 7, 11
    N = nt + T * Hl * Wl
    q, k, v = (_rand_bits(rng, (1, 2, N, D)) for _ in range(3))
    m, _, _ = o.sparse_route(q, k, T, Hl, Wl, -1e30, qblk=16, kblk=8)
    assert m.all()
    a = o.attn_rows(q, k, v, T, Hl, Wl, block_mask=m, qblk=16, kblk=8)
    assert np.array_equal(a, o.attn_rows(q, k, v, T, Hl, Wl))


def pin_sparse_prefix_sink_and_prefix_queries(o):
    """tau -> +inf: a video query block keeps exactly the key blocks holding a
    prefix key plus its best block; a query block holding a prefix row keeps
    every key block."""
    rng = np.random.default_rng(63)
    T, Hl, Wl, nt = 2, 6, 8, 21
    N = nt + T * Hl * Wl
    q, k = (_rand_bits(rng, (1, 1, N, D)) for _ in range(2))
    m, sc, _ = o.sparse_route(q, k, T, Hl, Wl, 1e30, qblk=16, kblk=8)
    m = m[0, 0].astype(bool)
    sink = np.arange(m.shape[1]) * 8 < nt
    for I in range(m.shape[0]):
        if I * 16 < nt:
            assert m[I].all()
        else:
            want = sink.copy()
            want[np.argmax(sc[0, 0, I])] = True
            assert np.array_equal(m[I], want)


def pin_sparse_attention_vs_numpy_twin(o):
    """Attention restricted to the kept key blocks equals the numpy twin's
    masked softmax on the full score matrix."""
    rng = np.random.default_rng(64)
    T, Hl, Wl, nt = 2, 5, 8, 9
    N = nt + T * Hl * Wl
    q, k, v = (_rand_bits(rng, (1, 2, N, D)) for _ in range(3))
    m, _, _ = o.sparse_route(q, k, T, Hl, Wl, 0.5, qblk=16, kblk=8)
    got = o.attn_rows(q, k, v, T, Hl, Wl, block_mask=m, qblk=16, kblk=8)
    qh, kh = brute.prepare_np(q, T, Hl, Wl), brute.prepare_np(k, T, Hl, Wl)
    want = brute.sparse_attention_np(qh, kh, _f(v), m.astype(bool), 16, 8)
    assert np.allclose(got, want, atol=2e-6, rtol=1e-6)
    assert not np.allclose(got, o.attn_rows(q, k, v, T, Hl, Wl), atol=1e-3), "mask had no effect"


# ------------------------------------------------ block-INT8 QKV records

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _record_format():
    """The record sizes the paper prints (tests/golden/qkv_record_format.txt)."""
    out = {}
    for ln in open(os.path.join(GOLDEN, "qkv_record_format.txt")):
        ln = ln.split("#")[0].strip()
        if ln:
            key, val = (x.strip() for x in ln.split("="))
            out[key] = int(val)
    return out


def _float16_of_code(c):
    """UE5M3 code c read as the IEEE half-precision number with the same
    exponent field and the top three mantissa bits (numpy's float16)."""
    return np.array([int(c) << 7], dtype=np.uint16).view(np.float16).astype(np.float64)[0]


def _one_record(q, k, v):
    return [_bits(x).reshape(1, 1, 1, 128) for x in (q, k, v)]


def pin_records_sizes_are_the_papers(o):
    """Record of 400 bytes: 3 x 128 code bytes, twelve scale codes each
    covering 32 values (a value moved across a 32-dim boundary moves to the
    next scale), four zero bytes (the paper's printed sizes)."""
    fmt = _record_format()
    rng = np.random.default_rng(70)
    q, k, v = (_rand_bits(rng, (2, 3, 5, 128)) for _ in range(3))
    rec = o.encode_qkv(q, k, v)
    assert rec.shape == (2, 5, 3, fmt["record_bytes"])
    assert 3 * 128 == fmt["value_bytes"]
    assert fmt["value_bytes"] + fmt["scale_codes"] + fmt["padding_bytes"] == fmt["record_bytes"]
    assert (rec[..., fmt["record_bytes"] - fmt["padding_bytes"]:] == 0).all()
    sc = rec[..., fmt["value_bytes"]:fmt["value_bytes"] + fmt["scale_codes"]]
    assert ((sc >= 1) & (sc <= 0xF7)).all()  # finite positive codes only
    G = fmt["group_size"]
    base = o.encode_qkv(*_one_record(np.ones(128), np.ones(128), np.ones(128)))[0, 0, 0]
    for p in range(3):
        for d in (0, G - 1, G, 2 * G + 5, 4 * G - 1):
            xs = [np.ones(128), np.ones(128), np.ones(128)]
            xs[p][d] = 100.0
            r = o.encode_qkv(*_one_record(*xs))[0, 0, 0]
            changed = {i for i in range(fmt["scale_codes"]) if r[384 + i] != base[384 + i]}
            assert changed == {4 * p + d // G}, (p, d, changed)


def pin_records_scale_values_are_float16(o):
    """A scale code's value is the half-precision number with the same
    exponent field and leading mantissa bits (numpy float16, library): every
    finite positive code, read through the decoder with a unit code."""
    codes = np.arange(1, 0xF8)
    rec = np.zeros((1, codes.size, 1, 400), dtype=np.uint8)
    rec[0, :, 0, 0] = 1                 # q dim 0: code +1
    rec[0, :, 0, 128 + 40] = 0xFF       # k dim 40: code -1
    rec[0, :, 0, 384] = codes           # q group 0
    rec[0, :, 0, 384 + 5] = codes       # k group 1
    rec[0, :, 0, 384 + 8:384 + 12] = 0x78  # v groups: scale 1.0
    dq, dk, _ = o.decode_qkv(rec)
    want = np.array([_float16_of_code(c) for c in codes])
    assert np.array_equal(_f(dq[0, 0, :, 0]), want)
    assert np.array_equal(_f(dk[0, 0, :, 40]), -want)
    assert _float16_of_code(0xF7) == 61440.0 and _float16_of_code(1) == 2.0 ** -17


def pin_records_hand_worked_example(o):
    """One record worked by hand from the format's definition: scale = the
    smallest code value s with 127 s >= max|x|, code = round-half-even(x/s)
    clamped to +-127 -- including exact ties, a zero group, subnormal scales,
    a group too large for any scale, and 127 s equal to max|x|."""
    q, k, v = np.zeros(128), np.zeros(128), np.zeros(128)
    q[0:32] = 1.0        # 127 * 2^-7 < 1 <= 127 * 1.125 * 2^-7: scale 0x41, 1 / 0.00878... -> 114
    q[32:64] = -2.5      # 127 * 0.01953125 < 2.5 <= 127 * 0.021484375: 0x4B, -116.36 -> -116
    q[96:102] = [15.875, 0.1875, 0.3125, -0.4375, 0.0625, -0.0625]  # 127 * 0.125 = 15.875: 0x60
    k[0], k[1:32] = 999424.0, 1.0    # 127 * 7680 < 999424 <= 127 * 8192: 0xE0, 122 exactly
    k[32], k[33] = 1e8, -1e8         # beyond 127 * 61440: 0xF7, clamped to +-127
    k[64:96] = 2.0 ** -20            # smallest code 0x01 (2^-17); 0.125 -> 0
    k[96:128] = 2.0 ** -10           # subnormal 0x02 (2^-16); 64 exactly
    v[0:32] = np.arange(32) - 16.0   # 127 * 0.125 < 16 <= 127 * 0.140625: 0x61
    v[32:] = 3.0                     # 127 * 0.0234375 < 3 <= 127 * 0.025390625: 0x4D, 118.15 -> 118
    r = o.encode_qkv(*_one_record(q, k, v))[0, 0, 0]
    assert r[384:400].tolist() == [0x41, 0x4B, 0x01, 0x60, 0xE0, 0xF7, 0x01, 0x02,
                                   0x61, 0x4D, 0x4D, 0x4D, 0, 0, 0, 0]
    c = r[:384].view(np.int8).astype(int)
    assert (c[0:32] == 114).all() and (c[32:64] == -116).all() and (c[64:96] == 0).all()
    assert c[96:102].tolist() == [127, 2, 2, -4, 0, 0]  # 1.5 -> 2, 2.5 -> 2, -3.5 -> -4, +-0.5 -> 0
    assert c[128] == 122 and (c[129:160] == 0).all()
    assert c[160:164].tolist() == [127, -127, 0, 0]
    assert (c[192:224] == 0).all() and (c[224:256] == 64).all()
    assert c[256] == -114 and c[257] == -107 and c[272] == 0 and c[273] == 7 and c[287] == 107
    assert (c[288:384] == 118).all()
    # decoding: code times scale, rounded once to bf16
    dq, dk, dv = o.decode_qkv(r.reshape(1, 1, 1, 400))
    assert _f(dq[0, 0, 0, 0]) == float(torch.tensor(114 * 0.0087890625).to(torch.bfloat16))
    assert _f(dk[0, 0, 0, 0]) == 999424.0 and _f(dk[0, 0, 0, 96]) == 2.0 ** -10
    assert _f(dk[0, 0, 0, 32]) == 7798784.0  # 127 * 61440 = 7802880, rounded to 8 bits


def pin_records_round_trip_bounds(o):
    """Random groups over 40 binades: every code within +-127, each value
    within half a scale of code * scale (unsaturated groups), the scale the
    smallest that fits (127 s(c-1) < max|x| <= 127 s(c)), multiples of the
    scale reproduced exactly, and decoding = bf16(code * scale) (torch)."""
    rng = np.random.default_rng(71)
    B, H, N = 1, 2, 64
    mag = np.exp2(rng.uniform(-20, 20, (B, H, N, 4, 1)))
    xs = [_bits((rng.standard_normal((B, H, N, 4, 32)) * mag).reshape(B, H, N, 128)) for _ in range(3)]
    rec = o.encode_qkv(*xs)
    dec = o.decode_qkv(rec)
    h16 = np.array([_float16_of_code(c) for c in range(0xF8)])
    for p in range(3):
        x = _f(xs[p]).transpose(0, 2, 1, 3).reshape(B, N, H, 4, 32)
        sc = rec[..., 384 + 4 * p:388 + 4 * p]
        s = h16[sc][..., None]
        c = rec[..., 128 * p:128 * (p + 1)].view(np.int8).astype(np.float64).reshape(B, N, H, 4, 32)
        amax = np.abs(x).max(-1)
        assert (np.abs(c) <= 127).all()
        assert (amax <= 127 * s[..., 0]).all()
        assert ((sc == 1) | (127 * h16[np.maximum(sc, 1) - 1] < amax)).all()
        assert (np.abs(c * s - x) <= s / 2).all()
        want = torch.from_numpy((c * s).astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
        got = _f(dec[p]).transpose(0, 2, 1, 3).reshape(B, N, H, 4, 32)
        assert np.array_equal(got, want)
    # exact multiples of the scale survive the round trip
    s = 2.0 ** -5  # code 0x50
    ints = rng.integers(-127, 128, (1, 1, 8, 128)).astype(np.float64)
    ints[..., ::32] = 127  # every group's max is 127 s, so its scale is s
    x = _bits(ints * s)
    assert np.array_equal(_f(x), ints * s)  # bf16-exact inputs
    rec = o.encode_qkv(x, x, x)
    assert (rec[..., 384:396] == 0x50).all()
    assert np.array_equal(o.decode_qkv(rec)[1], x)


def pin_records_vs_numpy_twin(o):
    """Encoding and decoding equal the vectorised numpy twin, ties included."""
    rng = np.random.default_rng(72)
    B, H, N = 2, 3, 7
    xs = []
    for _ in range(3):
        x = rng.standard_normal((B, H, N, 128)) * np.exp2(rng.uniform(-18, 18, (B, H, N, 1)))
        x[..., 5] = rng.integers(-60, 60, (B, H, N)) + 0.5  # half-way cases where the scale allows
        xs.append(_bits(x))
    rec = o.encode_qkv(*xs)
    assert np.array_equal(rec, brute.encode_records_np(*xs))
    for got, want in zip(o.decode_qkv(rec), brute.decode_records_np(rec)):
        assert np.array_equal(got, _bits(want.astype(np.float32)))  # code * scale is float32-exact


def pin_out_records_sizes_are_the_papers(o):
    """Output records of 144 bytes: 128 code bytes and four scale codes (132),
    padded with zeros to the next multiple of 16 (the paper's printed sizes);
    one scale per 32 dims."""
    fmt = _record_format()
    assert fmt["out_value_bytes"] + fmt["out_scale_codes"] == fmt["out_unpadded_bytes"]
    assert fmt["out_record_bytes"] % 16 == 0 and fmt["out_record_bytes"] - fmt["out_unpadded_bytes"] < 16
    rng = np.random.default_rng(73)
    rec = o.encode_out_records(rng.standard_normal((2, 5, 128)) * 1e-3)
    assert rec.shape == (2, 5, fmt["out_record_bytes"])
    assert (rec[..., fmt["out_unpadded_bytes"]:] == 0).all()
    base = o.encode_out_records(np.ones(128))
    for d in (0, 31, 32, 70, 127):
        x = np.ones(128)
        x[d] = 100.0
        r = o.encode_out_records(x)
        changed = {i for i in range(4) if r[128 + i] != base[128 + i]}
        assert changed == {d // fmt["group_size"]}, (d, changed)


def pin_out_records_quantise_like_qkv_records(o):
    """The output records follow the QKV records' rule: on bf16 values their
    codes and scales equal those of a record's q part; on double values the
    round-trip bound |code s - x| <= s/2 and the scale's minimality hold."""
    rng = np.random.default_rng(74)
    xb = _bits(rng.standard_normal((1, 2, 9, 128)) * np.exp2(rng.uniform(-15, 15, (1, 2, 9, 1))))
    q_rec = o.encode_qkv(xb, xb, xb)                       # [1, 9, 2, 400]
    out = o.encode_out_records(_f(xb))                     # [1, 2, 9, 144]
    q_rec = np.transpose(q_rec, (0, 2, 1, 3))
    assert np.array_equal(out[..., :128], q_rec[..., :128])
    assert np.array_equal(out[..., 128:132], q_rec[..., 384:388])
    x = rng.standard_normal((64, 4, 32)) * np.exp2(rng.uniform(-30, 10, (64, 4, 1)))
    rec = o.encode_out_records(x.reshape(64, 128))
    h16 = np.array([_float16_of_code(c) for c in range(0xF8)])
    sc = rec[:, 128:132]
    s = h16[sc][..., None]
    c = rec[:, :128].view(np.int8).astype(np.float64).reshape(64, 4, 32)
    amax = np.abs(x).max(-1)
    assert (amax <= 127 * s[..., 0]).all() and ((sc == 1) | (127 * h16[np.maximum(sc, 1) - 1] < amax)).all()
    assert (np.abs(c * s - x) <= s / 2).all()


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
