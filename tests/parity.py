"""Parity metrics between the HIP path and the oracle.

Errors are normalised per (b, h) by the RMS of the oracle's output over the
compared rows ("outputs of unit scale"): raw attention outputs shrink like
1/sqrt(N), so unnormalised tolerances would pass a badly wrong kernel at
large N.  Gate: max |err| <= 2e-2 and mean |err| <= 2e-3.
"""
import numpy as np
import torch

TOL_MAX = 2e-2
TOL_MEAN = 2e-3


def bits_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16_bits(x):
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _ordered(bits):
    b = bits.astype(np.int32)
    return np.where(b & 0x8000, -(b & 0x7FFF), b & 0x7FFF)


def compare(got_bits, ref, slab):
    """got_bits: uint16 [R, D] (bf16 from the GPU); ref: float32 [R, D];
    slab: int [R], the (b, h) slab of each row.  Returns a dict of metrics.

    ``floor_*`` are the same errors for bf16(ref), the correctly rounded
    output: no bf16 result can do better, so they show how much of the error
    is output rounding and how much the kernel adds."""
    got = bits_to_f32(got_bits).astype(np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    slab = np.asarray(slab)
    ref_bits = f32_to_bf16_bits(ref)
    norm = np.empty(len(slab))
    for s in np.unique(slab):
        m = slab == s
        rms = np.sqrt(np.mean(ref[m] ** 2))
        norm[m] = rms if rms > 0 else 1.0
    nerr = np.abs(got - ref) / norm[:, None]
    nfloor = np.abs(bits_to_f32(ref_bits).astype(np.float64) - ref) / norm[:, None]
    ulp = np.abs(_ordered(got_bits) - _ordered(ref_bits))
    return {
        "max_abs": float(nerr.max()),
        "mean_abs": float(nerr.mean()),
        "floor_max_abs": float(nfloor.max()),
        "floor_mean_abs": float(nfloor.mean()),
        "frac_ulp0": float((ulp == 0).mean()),
        "frac_ulp_le1": float((ulp <= 1).mean()),
        "rows": int(len(slab)),
        "finite": bool(np.isfinite(got).all()),
    }


def passes(stats):
    return stats["finite"] and stats["max_abs"] <= TOL_MAX and stats["mean_abs"] <= TOL_MEAN


def assert_parity(stats, label=""):
    assert passes(stats), "parity failed %s: %s" % (label, stats)


def sparse_mask(ws, B, H, N):
    """The kept-block mask [B, H, nqb, nkb] (uint8) of the block-sparse routing
    a sol_sparse_route call left in the device workspace ws; checks that each
    query block's list is non-empty, strictly ascending and in range."""
    from paper_2609_35110_amd import sol

    counts, blocks = sol.sparse_routing(ws, B, H, N)
    counts, blocks = counts.cpu().numpy(), blocks.cpu().numpy().astype(np.int64)
    nqb, nkb = blocks.shape[2], blocks.shape[3]
    mask = np.zeros((B, H, nqb, nkb), dtype=np.uint8)
    for b in range(B):
        for h in range(H):
            for I in range(nqb):
                c = counts[b, h, I]
                assert 1 <= c <= nkb
                lst = blocks[b, h, I, :c]
                assert (np.diff(lst) > 0).all() and lst[0] >= 0 and lst[-1] < nkb
                mask[b, h, I, lst] = 1
    return mask
