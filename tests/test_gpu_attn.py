"""GPU parity of the HIP path (libsol.so, through the C ABI) against the oracle.

Full-tensor comparisons at sizes the oracle finishes in seconds (several row
and key tiles, ragged tails, text prefixes, degenerate N); seeded row samples
at the full workload sizes, in the launch configuration the benchmark times.
"""
import os
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


# The two attention paths: "fused" (sol_attn_fwd: K rotated in every tile
# load, bf16 score operands) and "prepared" (sol_attn_fwd_ws: K rotated and
# converted once, fp16 score operands, the kernel the benchmark times).
PATHS = ["fused", "prepared"]


def _attn(path, q, k, v, w, tab, out=None):
    if path == "fused":
        return sol.attn_fwd(q, k, v, w.T, w.Hl, w.Wl, tab, out=out)
    return sol.attn_fwd_ws(q, k, v, w.T, w.Hl, w.Wl, tab, out=out)


def _run(q, k, v, w, rope=True, path="fused"):
    """HIP path on device copies; returns the bf16 output on the CPU."""
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV) if rope and w.n_video else None
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    out = _attn(path, qd, kd, vd, w, tab)
    torch.cuda.synchronize()
    return out.cpu()


def _full_parity(w, q, k, v, label, rope=True):
    """Both paths against one oracle evaluation; returns {path: output}."""
    ref = oracle.attn_rows(_bits(q), _bits(k), _bits(v), w.T, w.Hl, w.Wl, rope=rope)
    R = w.B * w.H * w.N
    slab = np.repeat(np.arange(w.B * w.H), w.N)
    outs = {}
    for path in PATHS:
        out = _run(q, k, v, w, rope, path)
        st = compare(_bits(out).reshape(R, w.D), ref.reshape(R, w.D), slab)
        _log("%s %s %s: %s" % (label, path, w.describe(), st))
        assert_parity(st, "%s %s" % (label, path))
        outs[path] = out
    return outs


def test_library_is_the_in_tree_build():
    assert os.path.dirname(sol.lib()._name) == os.path.dirname(sol.__file__)
    assert sol.sol_version() == 200


def test_mfma_probe_runs_every_product():
    """The rate probe's per-thread sums: every MFMA of every wave happened
    (iters * 4 copies of a fixed product per chain, so the sums scale exactly
    with iters for power-of-two operands)."""
    ops = torch.full((8192,), 0.5, dtype=torch.float16, device="cuda:0")
    one = sol.mfma_probe(ops, 8, 1)
    four = sol.mfma_probe(ops, 8, 4)
    torch.cuda.synchronize()
    # each accumulator element gets 4 MFMAs per iteration of 16 products 0.25
    # per chain: 16 elements x 4 chains x 4 x 16 x 0.25 = 1024 per iteration
    assert torch.all(one == 1024.0) and torch.all(four == 4096.0)


def test_tiny_full_parity():
    w = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(w)
    _full_parity(w, q, k, v, "tiny")


EDGE = [
    # (B, H, T, Hl, Wl, n_text): ragged row and key tiles, prefixes, degenerate N
    (1, 3, 3, 11, 13, 37),    # N=466: 2 row tiles, 8 key tiles, ragged, text prefix
    (2, 2, 2, 5, 7, 0),       # N=70: fewer rows than one tile
    (1, 1, 1, 1, 1, 0),       # N=1: o = v
    (1, 1, 4, 8, 8, 0),       # N=256: exact row tile, exact key tiles
    (1, 2, 1, 1, 1, 256),     # N=257: one token past a tile
    (1, 2, 2, 16, 16, 1),     # N=513
    (2, 1, 5, 7, 9, 64),      # N=379, B=2
]


@pytest.mark.parametrize("shape", EDGE, ids=[str(s) for s in EDGE])
def test_edge_shapes_full_parity(shape):
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=200 + sum(shape))
    q, k, v = W.make_inputs(w)
    outs = _full_parity(w, q, k, v, "edge")
    if w.N == 1:
        for path, out in outs.items():
            assert torch.equal(out, v), "N=1 must return v exactly (%s)" % path


def test_text_only_no_rotation():
    """An empty latent grid: nothing is rotated (plain attention, table NULL)."""
    w = W.custom(1, 2, 0, 0, 0, n_text=300, seed_index=301)
    q, k, v = W.make_inputs(w)
    _full_parity(w, q, k, v, "text-only", rope=False)


@pytest.mark.parametrize("name", ["low", "p480", "p720", "share"])
def test_workload_sampled_parity(name):
    """Full workload sizes, both paths, in the benchmark's launch
    configuration: per (b, h) 1,024 seeded rows, the first 64, the last 512
    (two 256-row tiles, the ragged one included) and the text/video boundary,
    every row against all keys."""
    w = W.WORKLOADS[name]
    _log("generating %s" % w.describe())
    q, k, v = W.make_inputs(w)
    rows = W.sample_rows(w, per_slab=1024, head=64, tail=512).numpy()
    _log("oracle on %d rows" % len(rows))
    ref = oracle.attn_rows(_bits(q), _bits(k), _bits(v), w.T, w.Hl, w.Wl, rows=rows)
    for path in PATHS:
        out = _run(q, k, v, w, path=path)
        got = _bits(out).reshape(-1, w.D)[rows]
        st = compare(got, ref, rows // w.N)
        _log("%s %s: %s" % (name, path, st))
        assert_parity(st, "%s %s" % (name, path))


# ------------------------------------------------------------ rotary kernel

@pytest.mark.parametrize("shape", [(1, 2, 3, 8, 8, 0), (2, 3, 3, 11, 13, 37), (1, 2, 31, 45, 80, 512)])
def test_rope3d_matches_oracle(shape):
    """Standalone rotation vs the oracle's contract rotation (double, one
    rounding), bit for bit.  The kernel turns each pair in fp64 with cos and
    sin to 48 bits and rounds once (through round-to-odd fp32), so it can
    differ only where the exact value lies within about 2^-47 |pair| of a bf16
    rounding midpoint: about 1e-11 of the elements (0.3 M here at most), where
    the fp32 rotation it replaced differed in about 1e-4."""
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=400 + sum(shape))
    q, _, _ = W.make_inputs(w)
    tab = sol.rope3d_table(T, Hl, Wl, device=DEV)
    y = sol.rope3d(q.to(DEV), T, Hl, Wl, tab)
    torch.cuda.synchronize()
    got_bits, want_bits, x_bits = _bits(y), oracle.rope3d_bf16(_bits(q), T, Hl, Wl), _bits(q)
    diff = int((got_bits != want_bits).sum())
    _log("rope3d %s: %d of %d elements differ from the oracle" % (shape, diff, got_bits.size))
    assert diff == 0
    assert np.array_equal(got_bits[..., :nt, :], x_bits[..., :nt, :]), "prefix must be copied"


def test_rope3d_in_place():
    w = W.custom(1, 2, 2, 6, 6, n_text=5, seed_index=410)
    q, _, _ = W.make_inputs(w)
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV)
    a = sol.rope3d(q.to(DEV), w.T, w.Hl, w.Wl, tab)
    b = q.to(DEV)
    sol.rope3d(b, w.T, w.Hl, w.Wl, tab, out=b)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def _quarter_turn_table(T, Hl, Wl, seed):
    """A rotary table of the default split whose (cos, sin) entries are random
    quarter turns, (1, 0), (0, 1), (-1, 0) or (0, -1), exact in any precision
    (position-0 rows stay the identity, as every table's: prefix tokens turn
    by them), and a lo plane of zeros."""
    tab = sol.rope3d_table_host(T, Hl, Wl)
    hi = tab[: tab.size // 2].reshape(-1, 2)
    gen = np.random.default_rng(seed)
    turn = np.array([[1, 0], [0, 1], [-1, 0], [0, -1]], np.float32)[gen.integers(0, 4, len(hi))]
    row0 = np.zeros(len(hi), bool)
    off = 0
    for ext, pairs in ((T, 16), (Hl, 24), (Wl, 24)):
        row0[off: off + pairs] = True
        off += ext * pairs
    hi[:] = np.where(row0[:, None], np.float32([1, 0]), turn)
    tab[tab.size // 2:] = 0.0
    return torch.from_numpy(tab).to(DEV)


@pytest.mark.parametrize("shape", [(1, 2, 3, 8, 8, 0), (1, 3, 3, 11, 13, 37), (2, 1, 5, 7, 9, 64)])
def test_fused_rotation_equals_prerotated(shape):
    """The fused kernel's rotations (queries exact, key tiles in fp32 with the
    hi plane) against sol_rope3d then attention without rotation.  With a table
    of quarter turns every form is exact, so the two are bit-identical: every
    table index of both kernels agrees.  With the real table the queries still
    agree bit for bit and the key tiles within one ulp, which leaves the
    outputs within the parity gate of each other and nearly all equal."""
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=500 + sum(shape))
    q, k, v = (t.to(DEV) for t in W.make_inputs(w))
    for quarter in (True, False):
        tab = _quarter_turn_table(T, Hl, Wl, 500 + sum(shape)) if quarter else sol.rope3d_table(T, Hl, Wl, device=DEV)
        fused = sol.attn_fwd(q, k, v, T, Hl, Wl, tab)
        qh, kh = sol.rope3d(q, T, Hl, Wl, tab), sol.rope3d(k, T, Hl, Wl, tab)
        pre = sol.attn_fwd(qh, kh, v, T, Hl, Wl, None)
        torch.cuda.synchronize()
        if quarter:
            assert not torch.equal(qh, q), "the quarter-turn table must rotate something"
            assert torch.equal(fused, pre)
        else:
            R = B * H * w.N
            st = compare(_bits(fused).reshape(R, w.D), bits_to_f32(_bits(pre)).reshape(R, w.D),
                         np.repeat(np.arange(B * H), w.N))
            same = float((fused == pre).float().mean())
            _log("fused vs pre-rotated %s: %s, equal %.4f" % (shape, st, same))
            assert_parity(st, "fused vs pre-rotated")
            assert same >= 0.95


def _prepared_layout(k_hat, v):
    """The prepared-path tile layout, rebuilt with plain tensor indexing from
    the rotated keys k_hat (bf16) and the values v: per slab, 32-key tiles
    (zero past N); K tile [kk][h][key l][8 dims 16kk+8h..]; V tile
    [s][c][h][l][i] = v[key 16s + 8(i//4) + 4h + i%4][dim 32c + l]."""
    B, H, N, D = v.shape
    nt = (N + 31) // 32
    pad = nt * 32 - N
    kf = torch.nn.functional.pad(k_hat.to(torch.float16), (0, 0, 0, pad)).view(B * H, nt, 32, 8, 2, 8)
    k_ref = kf.permute(0, 1, 3, 4, 2, 5).reshape(-1)
    vf = torch.nn.functional.pad(v.to(torch.float16), (0, 0, 0, pad)).view(B * H, nt, 32, D)
    s_, h_, i_ = torch.meshgrid(torch.arange(2), torch.arange(2), torch.arange(8), indexing="ij")
    keys = (16 * s_ + 8 * (i_ // 4) + 4 * h_ + i_ % 4).to(v.device)      # [s][h][i]
    g = vf[:, :, keys, :]                                                # [bh][t][s][h][i][D]
    g = g.view(B * H, nt, 2, 2, 8, 4, 32)                               # D -> [c][l]
    v_ref = g.permute(0, 1, 2, 5, 3, 6, 4).reshape(-1)                   # [s][c][h][l][i]
    return k_ref, v_ref


@pytest.mark.parametrize("shape", [(1, 2, 3, 8, 8, 0), (1, 3, 3, 11, 13, 37), (2, 1, 5, 7, 9, 64),
                                   (1, 1, 1, 1, 1, 0), (1, 2, 0, 0, 0, 300)])
def test_workspace_path_is_the_two_prepared_calls(shape):
    """sol_attn_fwd_ws == sol_prepare_kv then sol_attn_fwd_prepared, bit for
    bit; the workspace (and prepare_kv) hold exactly the documented tile
    layout of K rotated by sol_rope3d and of V, both in fp16."""
    B, H, T, Hl, Wl, nt = shape
    w = W.custom(B, H, T, Hl, Wl, n_text=nt, seed_index=550 + sum(shape))
    q, k, v = (t.to(DEV) for t in W.make_inputs(w))
    tab = sol.rope3d_table(T, Hl, Wl, device=DEV) if w.n_video else None
    ws = sol.attn_workspace(q)
    ws.fill_(0xFF)  # contents on entry are ignored
    a = sol.attn_fwd_ws(q, k, v, T, Hl, Wl, tab, workspace=ws)
    k_prep, v_prep = sol.prepare_kv(k, v, T, Hl, Wl, tab)
    b = sol.attn_fwd_prepared(q, k_prep, v_prep, T, Hl, Wl, tab)
    k_hat = sol.rope3d(k, T, Hl, Wl, tab) if tab is not None else k
    k_ref, v_ref = _prepared_layout(k_hat, v)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    n = k_ref.numel()
    assert k_prep.numel() == n and v_prep.numel() == n
    assert torch.equal(k_prep, k_ref)
    assert torch.equal(v_prep, v_ref)
    assert torch.equal(ws[: 2 * n].view(torch.float16), k_ref)
    assert torch.equal(ws[2 * n: 4 * n].view(torch.float16), v_ref)


@pytest.mark.parametrize("growth", [24.0, 300.0])
def test_rising_scores_raise_the_reference_in_place(growth):
    """Scores that climb along the key sequence far above the first key
    tile's max (by ~growth binades): on the prepared path nearly every tile's
    fp16 probabilities would overflow against the reference max, which is
    raised in place (O and l rescaled) before they are used.  Text-only, one
    direction u for every token: logit_j = a_j |u|^2 / sqrt(D)."""
    w = W.custom(1, 2, 0, 0, 0, n_text=700, seed_index=603)
    q, k, v = W.make_inputs(w)
    g = torch.Generator().manual_seed(9)
    u = torch.randn(w.D, generator=g)
    u = u / u.norm() * 4.0                                   # |u|^2 = 16
    scale = growth / 1.4426950408889634 * (w.D ** 0.5) / 16.0  # a_N-1 |u|^2/sqrt(D) log2(e) = growth
    a = torch.linspace(0.0, 1.0, w.N) * scale
    k = (a[None, None, :, None] * u).expand(w.B, w.H, w.N, w.D).to(torch.bfloat16).contiguous()
    q = (u + 0.1 * q.float()).to(torch.bfloat16)
    _full_parity(w, q, k, v, "growth%g" % growth, rope=False)


# ------------------------------------------------------------ closed forms

@pytest.mark.parametrize("path", PATHS)
def test_constant_values_give_constant_output(path):
    w = W.custom(1, 2, 3, 11, 13, n_text=37, seed_index=600)
    q, k, _ = W.make_inputs(w)
    c = torch.randn(w.D, generator=torch.Generator().manual_seed(5)).to(torch.bfloat16)
    v = c.expand(w.B, w.H, w.N, w.D).contiguous()
    out = _run(q, k, v, w, path=path).float()
    err = (out - c.float()).abs() / c.float().abs().clamp_min(1e-3)
    assert err.max().item() <= 2.0 ** -7, "constant V must give V back within one bf16 ulp"


@pytest.mark.parametrize("path", PATHS)
def test_zero_query_gives_mean_of_values(path):
    w = W.custom(1, 2, 3, 11, 13, n_text=37, seed_index=601)
    _, k, v = W.make_inputs(w)
    q = torch.zeros_like(k)
    out = _run(q, k, v, w, path=path).float()
    want = v.float().mean(dim=2, keepdim=True).expand_as(out)
    rms = want.pow(2).mean().sqrt()
    assert ((out - want).abs() / rms).max().item() < 2e-2


@pytest.mark.parametrize("path", PATHS)
def test_one_hot_attention_returns_the_value(path):
    """A key equal to the (unrotated) query with a logit gap of ~45 takes all
    the weight: the output row is that value row, exactly."""
    w = W.custom(1, 1, 0, 0, 0, n_text=200, seed_index=602)
    q, k, v = W.make_inputs(w)
    q.mul_(0.05)
    k.mul_(0.05)
    i, j = 17, 133
    q[0, 0, i] = 2.0
    k[0, 0, j] = 2.0
    out = _run(q, k, v, w, rope=False, path=path)
    assert torch.equal(out[0, 0, i], v[0, 0, j])


# ------------------------------------------------------------ guards

@pytest.mark.parametrize("path", PATHS)
def test_no_out_of_bounds_reads_or_writes(path):
    """Inputs live inside NaN-filled buffers and the output inside a sentinel
    buffer: nothing past N may be read (NaN would leak) or written."""
    w = W.custom(1, 2, 3, 11, 13, n_text=37, seed_index=700)
    q, k, v = W.make_inputs(w)
    numel = q.numel()
    pad = 4096 * w.D

    def nan_padded(t):
        buf = torch.full((numel + pad,), float("nan"), dtype=torch.bfloat16, device=DEV)
        buf[:numel].copy_(t.reshape(-1))
        return buf[:numel].view(t.shape)

    qd, kd, vd = nan_padded(q), nan_padded(k), nan_padded(v)
    sentinel = torch.full((numel + pad,), 123.0, dtype=torch.bfloat16, device=DEV)
    out = sentinel[:numel].view(q.shape)
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV)
    _attn(path, qd, kd, vd, w, tab, out=out)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    assert (sentinel[numel:] == 123.0).all(), "write past the end of out"
    clean = _run(q, k, v, w, path=path)
    assert torch.equal(out.cpu(), clean)


@pytest.mark.parametrize("path", PATHS)
def test_repeated_runs_are_bitwise_identical(path):
    w = W.custom(1, 4, 4, 16, 24, n_text=11, seed_index=701)
    q, k, v = (t.to(DEV) for t in W.make_inputs(w))
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV)
    a = _attn(path, q, k, v, w, tab)
    b = _attn(path, q, k, v, w, tab)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("path", PATHS)
def test_heads_and_batches_are_independent(path):
    """A slab's result is a function of its own data (and, for sol_attn_fwd,
    of which of its two routes it took): every slab of a batched call equals
    the same slab computed alone by that route, bit for bit."""
    w = W.custom(2, 3, 3, 11, 13, n_text=5, seed_index=702)
    q, k, v = (t.to(DEV) for t in W.make_inputs(w))
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV)
    full = _attn(path, q, k, v, w, tab)
    chunked = sol.sol_attn_fwd_plan(w.B, w.H, w.N, w.D) if path == "fused" else 0
    for b in range(w.B):
        for h in range(w.H):
            alone = [x[b:b + 1, h:h + 1].contiguous() for x in (q, k, v)]
            # one slab alone: sol_attn_fwd has no room for a chunk and runs the fused kernel
            route = "prepared" if b * w.H + h < chunked else path
            one = _attn(route, *alone, w, tab)
            torch.cuda.synchronize()
            assert torch.equal(full[b:b + 1, h:h + 1], one), (b, h, route)


def test_attn_fwd_runs_chunks_in_place_then_the_fused_kernel():
    """sol_attn_fwd's schedule (prepared chunks whose K and V live in the out
    slabs not yet written, then the fused kernel for the slabs after them):
    the chunked slabs equal the prepared path bit for bit, the rest equal the
    fused kernel alone, sampled rows of every slab match the oracle, and
    nothing is written outside out (sentinels)."""
    w = W.custom(2, 40, 4, 31, 33, n_text=8, seed_index=705)  # N = 4,100: ragged tiles, 80 slabs
    plan = sol.sol_attn_fwd_plan(w.B, w.H, w.N, w.D)
    assert 0 < plan < w.B * w.H
    q, k, v = (t.to(DEV) for t in W.make_inputs(w))
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=DEV)
    numel = q.numel()
    buf = torch.full((numel + 4096,), 123.0, dtype=torch.bfloat16, device=DEV)
    out = buf[:numel].view(q.shape)
    sol.attn_fwd(q, k, v, w.T, w.Hl, w.Wl, tab, out=out)
    prepared = sol.attn_fwd_ws(q, k, v, w.T, w.Hl, w.Wl, tab)
    S = w.B * w.H
    flat = lambda x: x.reshape(1, S, w.N, w.D)
    tail_in = [flat(x)[:, plan:].contiguous() for x in (q, k, v)]
    assert sol.sol_attn_fwd_plan(1, S - plan, w.N, w.D) == 0  # alone, the tail runs the fused kernel
    tail = sol.attn_fwd(*tail_in, w.T, w.Hl, w.Wl, tab)
    torch.cuda.synchronize()
    assert (buf[numel:] == 123.0).all(), "write past the end of out"
    assert torch.equal(flat(out)[:, :plan], flat(prepared)[:, :plan])
    assert torch.equal(flat(out)[:, plan:], tail)
    rows = W.sample_rows(w, per_slab=24, head=8, tail=40).numpy()
    ref = oracle.attn_rows(_bits(q.cpu()), _bits(k.cpu()), _bits(v.cpu()), w.T, w.Hl, w.Wl, rows=rows)
    got = _bits(out.cpu()).reshape(-1, w.D)[rows]
    st = compare(got, ref, rows // w.N)
    _log("attn_fwd chunks %d + fused %d: %s" % (plan, S - plan, st))
    assert_parity(st, "attn_fwd schedule")


def test_offsets_beyond_2_pow_31_elements():
    """B=1, H=160 heads of the 111,600-token layer: 2.29e9 elements per tensor.
    Only the last two heads carry data; the rest are zero.  Both paths."""
    base = W.WORKLOADS["p720"]
    H = 160
    w1 = W.custom(1, 2, base.T, base.Hl, base.Wl, seed_index=800)
    qs, ks, vs = W.make_inputs(w1)
    shape = (1, H, base.N, base.D)
    assert np.prod(shape) > 2 ** 31
    q = torch.zeros(shape, dtype=torch.bfloat16, device=DEV)
    k = torch.zeros_like(q)
    v = torch.zeros_like(q)
    q[:, H - 2:].copy_(qs)
    k[:, H - 2:].copy_(ks)
    v[:, H - 2:].copy_(vs)
    tab = sol.rope3d_table(base.T, base.Hl, base.Wl, device=DEV)
    tails = {}
    for path in PATHS:
        out = _attn(path, q, k, v, base, tab)
        torch.cuda.synchronize()
        tails[path] = out[:, H - 2:].cpu()
        del out
        torch.cuda.empty_cache()
    del q, k, v
    torch.cuda.empty_cache()
    rows = W.sample_rows(w1, per_slab=16, head=8, tail=80).numpy()
    ref = oracle.attn_rows(_bits(qs), _bits(ks), _bits(vs), w1.T, w1.Hl, w1.Wl, rows=rows)
    for path, tail in tails.items():
        st = compare(_bits(tail).reshape(-1, w1.D)[rows], ref, rows // w1.N)
        _log("2^31 offsets %s: %s" % (path, st))
        assert_parity(st, "large offsets " + path)
