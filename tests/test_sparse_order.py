"""The block-sparse walk's order of a slab's query tiles (CPU only).

``sparse_order_stride``, ``sparse_order_len`` and ``sparse_order_block`` in
``csrc/sol_internal.h`` define how the grid positions of a slab map to query
tiles (position o of R S is tile (o % R) S + o / R); the kernel and its
launcher both take them from there.  The
header is compiled by the host compiler (with UndefinedBehaviorSanitizer,
which aborts on a signed overflow or a division by zero) into a tiny shared
library, and on shapes of
every kind -- the paper's latent grids, text prefixes, ragged ends, tiny and
huge frames -- the checks are:

* every tile of the slab appears at exactly one position (the other
  positions name no tile), so each query row is computed once;
* the positions fit the grid bound the entry points check against INT32;
* consecutive positions of a column are S tiles apart, S the tiles of a
  frame rounded, so they start at nearly the same place of consecutive
  frames -- the locality the order exists for.
"""
import ctypes
import os
import random
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_35110_amd", "csrc")
BLK = 256

SRC = r'''
#include "sol_internal.h"
// the kernel's mapping, position o of a slab -> tile (-1: none)
extern "C" int order_positions(int nqb, int T, int hw, int nt) {
  return sol::sparse_order_len(nqb, sol::sparse_order_stride(hw));
}
extern "C" int order_block(int nqb, int T, int hw, int nt, int o) {
  return sol::sparse_order_block(o, nqb, sol::sparse_order_stride(hw));
}
extern "C" int order_stride(int hw) { return sol::sparse_order_stride(hw); }
extern "C" long long max_workgroups(int N, int BH) { return (long long)sol::attn_max_workgroups(N, BH); }
'''


@pytest.fixture(scope="module")
def lib(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.isdir("/opt/rocm/include"):
        pytest.skip("g++ or the HIP headers not available")
    d = tmp_path_factory.mktemp("order")
    src, so = str(d / "order.cpp"), str(d / "liborder.so")
    open(src, "w").write(SRC)
    res = subprocess.run([gxx, "-std=c++17", "-shared", "-fPIC", "-O1", "-fsanitize=undefined",
                          "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__",
                          "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", CSRC, src,
                          "-o", so], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    lib = ctypes.CDLL(so)
    lib.max_workgroups.restype = ctypes.c_longlong
    return lib


def shapes():
    out = [(111600, 31, 3600, 0), (48360, 31, 1560, 0), (12480, 8, 1560, 0), (112112, 31, 3600, 512),
           (1032192, 31, 33296, 0), (1344, 4, 320, 64), (300, 0, 0, 300), (5000, 1, 4096, 904),
           (1032192, 1, 1032192, 0), (257, 1, 257, 0), (1, 1, 1, 0), (140912, 39, 3600, 512)]
    rng = random.Random(20261202)
    while len(out) < 400:
        T, hw, nt = rng.randint(1, 80), rng.randint(1, 6000), rng.randint(0, 5000)
        if 1 <= nt + T * hw <= 1032192:
            out.append((nt + T * hw, T, hw, nt))
    return out


def test_every_tile_at_exactly_one_position(lib):
    for N, T, hw, nt in shapes():
        nqb = -(-N // BLK)
        n_pos = lib.order_positions(nqb, T, hw, nt)
        # the launcher's grid: 8 ceil(positions / 8) per slab, within the checked bound
        assert 8 * (-(-n_pos // 8)) <= lib.max_workgroups(N, 1), (N, T, hw, nt)
        got = [lib.order_block(nqb, T, hw, nt, o) for o in range(n_pos)]
        tiles = sorted(b for b in got if b >= 0)
        assert tiles == list(range(nqb)), (N, T, hw, nt)
        assert all(b == -1 for b in got if b < 0)


def test_columns_hold_one_place_in_consecutive_frames(lib):
    for N, T, hw, nt in shapes():
        nqb = -(-N // BLK)
        S = lib.order_stride(hw)
        if hw < 2 * BLK:
            # frames under two tiles, or no grid: the plain order
            assert S == 1
            assert [lib.order_block(nqb, T, hw, nt, o) for o in range(nqb)] == list(range(nqb))
            continue
        assert abs(S * BLK - hw) <= BLK // 2  # a frame's tiles, rounded
        R = -(-nqb // S)
        for o in range(lib.order_positions(nqb, T, hw, nt) - 1):
            a, b = lib.order_block(nqb, T, hw, nt, o), lib.order_block(nqb, T, hw, nt, o + 1)
            if a >= 0 and b >= 0 and (o + 1) % R:
                assert b - a == S, (N, T, hw, nt, o)
