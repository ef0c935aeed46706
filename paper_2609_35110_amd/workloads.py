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

Recipe: every (tensor, b, h) slab has its own torch CPU ``Generator``, seeded
with ``slab_seed(seed, tensor, b*H + h)`` where seed = 20260903 + config index
and tensor is 0/1/2 for q/k/v; it draws the text prefix rows (if any), then the
video rows, as float32 ``randn`` -> (times the std, in float32) -> bf16 round to
nearest even.  The boosted keys are ``randperm(N)[:N//100]`` from a generator
seeded with ``slab_seed(seed, 3, 0)``, the same tokens in every head, multiplied
by 8 after the bf16 cast (exact).  Slabs are independent, so they are drawn in
parallel and any single slab can be regenerated alone.
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
    def flops(self) -> float:
        """Algorithmic flops of one layer: 4 N^2 D per (b, h)."""
        return 4.0 * self.N * self.N * self.D * self.H * self.B

    def describe(self) -> str:
        s = "B=%d H=%d D=%d grid %dx%dx%d" % (self.B, self.H, self.D, self.T, self.Hl, self.Wl)
        if self.n_text:
            s += " + %d text" % self.n_text
        return s + " (N=%d)" % self.N


WORKLOADS = {
    "tiny": Workload("tiny", 0, 1, 2, 3, 8, 8),
    "low": Workload("low", 1, 1, 24, 8, 30, 52, scale=2.0 ** -0.5),
    "p480": Workload("p480", 2, 1, 40, 31, 30, 52, boost_frac=0.01, boost=8.0),
    "p720": Workload("p720", 3, 1, 40, 31, 45, 80),
    "share": Workload("share", 4, 2, 5, 31, 45, 80, n_text=512, text_kv_std=0.5),
}


def custom(B, H, T, Hl, Wl, n_text=0, seed_index=100, **kw) -> Workload:
    """An ad-hoc workload (tests of edge shapes); seed = 20260903 + seed_index."""
    return Workload("custom", seed_index, B, H, T, Hl, Wl, n_text=n_text, **kw)


def slab_seed(seed: int, tensor: int, slab: int) -> int:
    """Seed of one (tensor, slab) stream; tensor 0/1/2 = q/k/v, 3 = boost indices."""
    return (seed * 1000003 + tensor * 7919 + slab * 104729) % (2 ** 63)


def _fill_slab(dst, seed, tensor, slab, w: Workload):
    gen = torch.Generator().manual_seed(slab_seed(seed, tensor, slab))
    if w.n_text:
        std = 1.0 if tensor == 0 else w.text_kv_std
        x = torch.randn((w.n_text, w.D), generator=gen, dtype=torch.float32)
        if std != 1.0:
            x.mul_(torch.tensor(std, dtype=torch.float32))
        dst[: w.n_text].copy_(x)
    x = torch.randn((w.n_video, w.D), generator=gen, dtype=torch.float32)
    if w.scale != 1.0:
        x.mul_(torch.tensor(w.scale, dtype=torch.float32))
    dst[w.n_text:].copy_(x)  # float32 -> bf16, round to nearest even


def boosted_tokens(w: Workload, seed: int = None):
    """Token indices whose keys are boosted (empty when the workload has none)."""
    if w.boost_frac <= 0:
        return torch.zeros(0, dtype=torch.int64)
    gen = torch.Generator().manual_seed(slab_seed(w.seed if seed is None else seed, 3, 0))
    return torch.randperm(w.N, generator=gen)[: int(w.N * w.boost_frac)]


def make_inputs(w: Workload, seed: int = None, threads: int = None):
    """Return (q, k, v): bf16 CPU tensors [B, H, N, D], contiguous."""
    seed = w.seed if seed is None else seed
    out = [torch.empty((w.B, w.H, w.N, w.D), dtype=torch.bfloat16) for _ in range(3)]
    jobs = [(t, bh) for t in range(3) for bh in range(w.B * w.H)]
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))

    def run(job):
        t, bh = job
        _fill_slab(out[t].view(w.B * w.H, w.N, w.D)[bh], seed, t, bh, w)

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(run, jobs))
    idx = boosted_tokens(w, seed)
    if idx.numel():
        out[1][:, :, idx, :] *= torch.tensor(w.boost, dtype=torch.bfloat16)
    return tuple(out)


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
