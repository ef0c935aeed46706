"""CPU oracle for fused 3D-RoPE + softmax attention.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
and the benchmark's CPU-baseline leg may import this package.  It shares no
code with the HIP library (package ``paper_2609_35110_amd``) and imports
nothing from it.

Two independent implementations, both in IEEE double:

* ``solref`` (C, ``libsolref.so``): the plain two-pass definition of
  attention, per query row, with the 3D rotary embedding applied explicitly to
  every query and key (Sec. 3.2 "Optimized attention collectives": the SDPA
  term; Sec. 3.5, fusion group 2: the partial/3D rotary embedding that feeds
  it; Sec. 3.4 "Safety rails": text-first sequence packing).  Fast enough for
  sampled rows of the largest workloads.
* ``brute`` (numpy): materialised rotation as complex multiplication, the full
  N x N score matrix and a library softmax, for tiny inputs.  It pins the C
  code, and is itself pinned by library routines, closed forms and invariants
  in the test suite.
"""
from .solref import (  # noqa: F401
    Oracle, default,
    DEFAULT_SPLIT, ROPE_BASE, attn_rows, decode_qkv, encode_out_records, encode_qkv, num_threads,
    qknorm_rope3d, rope3d_bf16, rope3d_f64, round_bf16, round_e4m3, sparse_route,
)
from . import brute  # noqa: F401
