"""Seeded synthetic workloads for the fused 3D-RoPE attention path.

This module only draws input tensors; it holds none of the method's
arithmetic, so both the HIP path and the CPU oracle consume its bytes.

The shapes stand in for the paper's low- and high-resolution denoising stages
(Sec. 3.1 two-stage generation; Sec. 3.2 attention on a head-sharded layout;
Sec. 3.4 text-first packed sequences).  The paper measures attention on no
public dataset; every tensor here is synthetic:

* ``tiny``  : B=1, H=2,  grid 3x8x8   (N=192)
* ``low``   : B=1, H=24, grid 8x30x52 (N=12,480), values N(0,1)/sqrt(2)
* ``p480``  : B=1, H=40, grid 31x30x52 (N=48,360), N(0,1), 1% of key tokens x8
* ``p720``  : B=1, H=40, grid 31x45x80 (N=111,600), N(0,1)
* ``share`` : B=2, H=5,  grid 31x45x80 + 512 text tokens first (N=112,112);
              video N(0,1), text q N(0,1), text k/v N(0, 0.5^2)
* ``p720n`` : ``p720`` before QK normalization (Sec. 3.5, fusion group 2):
              every q and k row scaled by 2^e, e uniform in [-4, 4] per token,
              and per-dimension weights gamma_q, gamma_k
* ``p720s`` : ``p720`` for the block-sparse attention (Sec. 3.4): q and k rows
              share a per-head direction c (N(0,1) per head, added to every row
              before the bf16 cast), so the rotary embedding makes attention
              local in (t, h, w), as in a video DiT
* ``ref720``: the reference-KV cache of Sec. 5 at 720p: queries = 512 text
              tokens + grid 31x45x80 (Nq=112,112); keys = one cached
              reference video (grid 8x45x80, 28,800 tokens, its own positions
              from 0) followed by the queries' own tokens (Nkv=140,912)

Recipe: every (tensor, b, h) slab has its own torch CPU ``Generator``, seeded
with ``slab_seed(seed, tensor, b*H + h)`` where seed = 20260903 + config index
and tensor is 0/1/2 for q/k/v; it draws the text prefix rows (if any), then the
video rows, as float32 ``randn`` -> (times the std, in float32) -> bf16 round to
nearest even.  The boosted keys are ``randperm(N)[:N//100]`` from a generator
seeded with ``slab_seed(seed, 3, 0)``, the same tokens in every head, multiplied
by 8 after the bf16 cast (exact).  Slabs are independent, so they are drawn in
parallel and any single slab can be regenerated alone.

QK-normalisation workloads (``qk_norm``): the q and k rows are then multiplied
by 2^e (exact), e = ``randint(-4, 5)`` per token from generators seeded with
``slab_seed(seed, 4 or 5, b*H + h)``; the weights are bf16-exact float32
values 1 + 0.25 N(0,1) (``slab_seed(seed, 6 or 7, 0)``).  Reference segments
(``n_ref``): k and v of the cached tokens are drawn like the video rows, with
tensor ids 8 and 9.  Shared directions (``shared_dir`` = beta): c is drawn
from ``slab_seed(seed, 10, b*H + h)`` and beta * c is added, in float32, to
every q and k row of that slab before the bf16 cast.
"""
from concurrent.futures import ThreadPoolExecutor
import os
from dataclasses import dataclass

import torch

SEED_BASE = 20260903
HEAD_DIM = 128


@dataclass(frozen=True)
class Workload:
    name: str
    index: int
    B: int
    H: int
    T: int
    Hl: int
    Wl: int
    n_text: int = 0
    scale: float = 1.0          # multiplier on the N(0,1) video draws
    text_kv_std: float = 1.0    # std of the text-prefix k and v draws
    boost_frac: float = 0.0     # fraction of key tokens multiplied by boost
    boost: float = 1.0
    qk_norm: bool = False       # q, k rows drawn at random scales; norm weights given
    ref_grid: tuple = ()        # grid (T, Hl, Wl) of a cached reference segment
    shared_dir: float = 0.0     # weight of a per-head direction shared by all q, k rows
    D: int = HEAD_DIM

    @property
    def n_video(self) -> int:
        return self.T * self.Hl * self.Wl

    @property
    def N(self) -> int:
        return self.n_text + self.n_video

    @property
    def seed(self) -> int:
        return SEED_BASE + self.index

    @property
    def n_ref(self) -> int:
        """Tokens of the cached reference segment (0: none)."""
        if not self.ref_grid:
            return 0
        T, Hl, Wl = self.ref_grid
        return T * Hl * Wl

    @property
    def n_kv(self) -> int:
        """Keys per (b, h): the reference segment, then the N own tokens."""
        return self.n_ref + self.N

    @property
    def flops(self) -> float:
        """Algorithmic flops of one layer: 4 Nq Nkv D per (b, h)."""
        return 4.0 * self.N * self.n_kv * self.D * self.H * self.B

    def describe(self) -> str:
        s = "B=%d H=%d D=%d grid %dx%dx%d" % (self.B, self.H, self.D, self.T, self.Hl, self.Wl)
        if self.n_text:
            s += " + %d text" % self.n_text
        s += " (N=%d)" % self.N
        if self.n_ref:
            s += ", cached reference grid %dx%dx%d (Nkv=%d)" % (self.ref_grid + (self.n_kv,))
        if self.qk_norm:
            s += ", QK norm"
        return s


WORKLOADS = {
    "tiny": Workload("tiny", 0, 1, 2, 3, 8, 8),
    "low": Workload("low", 1, 1, 24, 8, 30, 52, scale=2.0 ** -0.5),
    "p480": Workload("p480", 2, 1, 40, 31, 30, 52, boost_frac=0.01, boost=8.0),
    "p720": Workload("p720", 3, 1, 40, 31, 45, 80),
    "share": Workload("share", 4, 2, 5, 31, 45, 80, n_text=512, text_kv_std=0.5),
    "p720n": Workload("p720n", 5, 1, 40, 31, 45, 80, qk_norm=True),
    "ref720": Workload("ref720", 6, 1, 40, 31, 45, 80, n_text=512, ref_grid=(8, 45, 80)),
    "p720s": Workload("p720s", 7, 1, 40, 31, 45, 80, shared_dir=1.0),
}

# threshold parameters of the paper's three refinement steps (Sec. 3.4)
SPARSE_TAUS = (1.0, 1.25, 1.5)

# eps under the root of the QK normalisation in the qk_norm workloads
QK_NORM_EPS = 1e-6


def custom(B, H, T, Hl, Wl, n_text=0, seed_index=100, **kw) -> Workload:
    """An ad-hoc workload (tests of edge shapes); seed = 20260903 + seed_index."""
    return Workload("custom", seed_index, B, H, T, Hl, Wl, n_text=n_text, **kw)


def slab_seed(seed: int, tensor: int, slab: int) -> int:
    """Seed of one (tensor, slab) stream; tensor 0/1/2 = q/k/v, 3 = boost indices."""
    return (seed * 1000003 + tensor * 7919 + slab * 104729) % (2 ** 63)


def _fill_slab(dst, seed, tensor, slab, w: Workload):
    gen = torch.Generator().manual_seed(slab_seed(seed, tensor, slab))
    shared = None
    if w.shared_dir and tensor in (0, 1):
        cgen = torch.Generator().manual_seed(slab_seed(seed, 10, slab))
        shared = torch.randn(w.D, generator=cgen, dtype=torch.float32) * w.shared_dir
    if w.n_text:
        std = 1.0 if tensor == 0 else w.text_kv_std
        x = torch.randn((w.n_text, w.D), generator=gen, dtype=torch.float32)
        if std != 1.0:
            x.mul_(torch.tensor(std, dtype=torch.float32))
        if shared is not None:
            x.add_(shared)
        dst[: w.n_text].copy_(x)
    x = torch.randn((w.n_video, w.D), generator=gen, dtype=torch.float32)
    if w.scale != 1.0:
        x.mul_(torch.tensor(w.scale, dtype=torch.float32))
    if shared is not None:
        x.add_(shared)
    dst[w.n_text:].copy_(x)  # float32 -> bf16, round to nearest even


def boosted_tokens(w: Workload, seed: int = None):
    """Token indices whose keys are boosted (empty when the workload has none)."""
    if w.boost_frac <= 0:
        return torch.zeros(0, dtype=torch.int64)
    gen = torch.Generator().manual_seed(slab_seed(w.seed if seed is None else seed, 3, 0))
    return torch.randperm(w.N, generator=gen)[: int(w.N * w.boost_frac)]


def make_slab(w: Workload, tensor: int, bh: int, seed: int = None, boosted=None):
    """One (tensor, b*H + h) slab of make_inputs, bf16 [N, D] (CPU): tensor
    0/1/2 = q/k/v.  The whole recipe for that slab (draw, boosted keys, QK-norm
    row scales), so any slab can be regenerated alone.  boosted: the boosted
    token indices when the caller already has them."""
    seed = w.seed if seed is None else seed
    x = torch.empty((w.N, w.D), dtype=torch.bfloat16)
    _fill_slab(x, seed, tensor, bh, w)
    if tensor == 1 and w.boost_frac > 0:
        idx = boosted_tokens(w, seed) if boosted is None else boosted
        x[idx, :] *= torch.tensor(w.boost, dtype=torch.bfloat16)  # x8: exact
    if w.qk_norm and tensor in (0, 1):
        gen = torch.Generator().manual_seed(slab_seed(seed, 4 + tensor, bh))
        e = torch.randint(-4, 5, (w.N, 1), generator=gen).to(torch.float32)
        x.mul_(torch.exp2(e).to(torch.bfloat16))  # powers of two: exact
    return x


def make_inputs(w: Workload, seed: int = None, threads: int = None):
    """Return (q, k, v): bf16 CPU tensors [B, H, N, D], contiguous."""
    seed = w.seed if seed is None else seed
    out = [torch.empty((w.B, w.H, w.N, w.D), dtype=torch.bfloat16) for _ in range(3)]
    jobs = [(t, bh) for t in range(3) for bh in range(w.B * w.H)]
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))
    boosted = boosted_tokens(w, seed)

    def run(job):
        t, bh = job
        out[t].view(w.B * w.H, w.N, w.D)[bh].copy_(make_slab(w, t, bh, seed, boosted))

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(run, jobs))
    return tuple(out)


def norm_weights(w: Workload, seed: int = None):
    """(gamma_q, gamma_k): float32 [D] QK-normalisation weights, bf16-exact
    values 1 + 0.25 N(0,1)."""
    seed = w.seed if seed is None else seed
    res = []
    for t in (6, 7):
        gen = torch.Generator().manual_seed(slab_seed(seed, t, 0))
        g = 1.0 + 0.25 * torch.randn(w.D, generator=gen, dtype=torch.float32)
        res.append(g.to(torch.bfloat16).to(torch.float32))
    return tuple(res)


def make_ref_slab(w: Workload, tensor: int, bh: int, seed: int = None):
    """One slab of make_ref_inputs, bf16 [n_ref, D]: tensor 0 = k, 1 = v of the
    cached reference segment, drawn like video rows (N(0,1) times the workload
    scale) from stream 8 + tensor."""
    seed = w.seed if seed is None else seed
    rw = Workload("ref", w.index, w.B, w.H, *w.ref_grid, scale=w.scale, D=w.D)
    x = torch.empty((w.n_ref, w.D), dtype=torch.bfloat16)
    _fill_slab(x, seed, 8 + tensor, bh, rw)
    return x


def make_ref_inputs(w: Workload, seed: int = None, threads: int = None):
    """(k_ref, v_ref): the cached reference segment's keys and values, bf16
    [B, H, n_ref, D]."""
    out = [torch.empty((w.B, w.H, w.n_ref, w.D), dtype=torch.bfloat16) for _ in range(2)]
    jobs = [(t, bh) for t in range(2) for bh in range(w.B * w.H)]
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))

    def run(job):
        t, bh = job
        out[t].view(w.B * w.H, w.n_ref, w.D)[bh].copy_(make_ref_slab(w, t, bh, seed))

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(run, jobs))
    return tuple(out)


def random_records(B: int, H: int, N: int, seed: int):
    """Random block-INT8 QKV records, uint8 [B, N, H, 400] (CPU): codes uniform
    in [-127, 127], scale codes uniform in 0x30..0x97 (2^-9 .. 7.5), the four
    trailing bytes zero -- wire records as an encoder could write them."""
    gen = torch.Generator().manual_seed(seed)
    rec = torch.zeros((B, N, H, 400), dtype=torch.uint8)
    codes = torch.randint(-127, 128, (B, N, H, 384), generator=gen, dtype=torch.int16)
    rec[..., :384] = (codes & 0xFF).to(torch.uint8)
    rec[..., 384:396] = torch.randint(0x30, 0x98, (B, N, H, 12), generator=gen).to(torch.uint8)
    return rec


def as_bits(t: torch.Tensor):
    """bf16 tensor -> numpy uint16 view of its bit patterns (CPU, no copy when possible)."""
    import numpy as np
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def sample_rows(w: Workload, per_slab: int, head: int = 64, tail: int = 512, seed: int = None):
    """Seeded query rows to check at full size, as global ids (b*H + h)*N + i.

    Per (b, h): the first ``head`` rows, the last ``tail`` rows (which hold the
    ragged row tile), the text/video boundary when there is a prefix, and
    ``per_slab`` uniformly drawn rows.
    """
    gen = torch.Generator().manual_seed((w.seed if seed is None else seed) + 7777)
    N = w.N
    fixed = set(range(min(head, N)))
    fixed.update(range(max(0, N - tail), N))
    if w.n_text:
        fixed.update({w.n_text - 1, w.n_text})
    rows = []
    for bh in range(w.B * w.H):
        extra = torch.randint(0, N, (per_slab,), generator=gen).tolist()
        sel = sorted(fixed.union(extra))
        rows.extend(bh * N + i for i in sel)
    return torch.tensor(rows, dtype=torch.int64)
