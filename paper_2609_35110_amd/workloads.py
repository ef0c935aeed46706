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

Recipe: a torch CPU ``Generator`` seeded with 20260903 + config index; draws in
the order q, k, v (video part), then text q, k, v, then the boosted-key
indices; float32 ``randn`` -> (scale in float32) -> bf16 round-to-nearest-even.
"""
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


def _draw(gen, shape, std):
    x = torch.randn(shape, generator=gen, dtype=torch.float32)
    if std != 1.0:
        x.mul_(torch.tensor(std, dtype=torch.float32))
    return x.to(torch.bfloat16)


def make_inputs(w: Workload, seed: int = None):
    """Return (q, k, v): bf16 CPU tensors [B, H, N, D], contiguous."""
    gen = torch.Generator().manual_seed(w.seed if seed is None else seed)
    shp_v = (w.B, w.H, w.n_video, w.D)
    qv = _draw(gen, shp_v, w.scale)
    kv = _draw(gen, shp_v, w.scale)
    vv = _draw(gen, shp_v, w.scale)
    if w.n_text:
        shp_t = (w.B, w.H, w.n_text, w.D)
        qt = _draw(gen, shp_t, 1.0)
        kt = _draw(gen, shp_t, w.text_kv_std)
        vt = _draw(gen, shp_t, w.text_kv_std)
        q = torch.cat([qt, qv], dim=2)
        k = torch.cat([kt, kv], dim=2)
        v = torch.cat([vt, vv], dim=2)
        del qt, kt, vt
    else:
        q, k, v = qv, kv, vv
    if w.boost_frac > 0:
        n_boost = int(w.N * w.boost_frac)
        idx = torch.randperm(w.N, generator=gen)[:n_boost]
        # exact in bf16: the boost is a power of two
        k[:, :, idx, :] *= torch.tensor(w.boost, dtype=torch.bfloat16)
    return q.contiguous(), k.contiguous(), v.contiguous()


def as_bits(t: torch.Tensor):
    """bf16 tensor -> numpy uint16 view of its bit patterns (CPU, no copy when possible)."""
    import numpy as np
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def sample_rows(w: Workload, per_slab: int, bm: int = 256, seed: int = None):
    """Seeded query rows to check at full size, as global ids (b*H + h)*N + i.

    Per (b, h): the first 64 rows, the last two row tiles of ``bm`` (the ragged
    one included), the text/video boundary when there is a prefix, and
    ``per_slab`` uniformly drawn rows.
    """
    gen = torch.Generator().manual_seed((w.seed if seed is None else seed) + 7777)
    N = w.N
    fixed = set(range(min(64, N)))
    fixed.update(range(max(0, N - (N % bm or bm) - bm), N))
    if w.n_text:
        fixed.update({w.n_text - 1, w.n_text})
    rows = []
    for bh in range(w.B * w.H):
        extra = torch.randint(0, N, (per_slab,), generator=gen).tolist()
        sel = sorted(fixed.union(extra))
        rows.extend(bh * N + i for i in sel)
    return torch.tensor(rows, dtype=torch.int64)
