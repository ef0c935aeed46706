"""The LDS-poison debug build (GPU).

``libsol_poison.so`` is the library compiled with -DSOL_LDS_POISON: every
workgroup of the attention, prepare and routing kernels first fills its
value-holding LDS arrays with NaN bit patterns.  A read that came before the
write it depends on (a missing barrier, a copy not yet waited for) would then
put NaN into the output instead of plausible stale values, and fail parity.
This test runs the full-tensor parity cases of every path on that build, in a
child process (the binding loads one library per process), once.
"""
import os
import subprocess
import sys

import pytest

from paper_2609_35110_amd import build as pkg_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CASES = [
    "tests/test_gpu_attn.py::test_tiny_full_parity",
    "tests/test_gpu_attn.py::test_edge_shapes_full_parity",
    "tests/test_gpu_attn.py::test_rising_scores_raise_the_reference_in_place",
    "tests/test_gpu_attn.py::test_workspace_path_is_the_two_prepared_calls",
    "tests/test_gpu_attn.py::test_no_out_of_bounds_reads_or_writes",
    "tests/test_gpu_attn.py::test_attn_fwd_runs_chunks_in_place_then_the_fused_kernel",
    "tests/test_gpu_sparse.py::test_sparse_full_parity",
    "tests/test_gpu_sparse.py::test_sparse_with_qknorm",
    "tests/test_gpu_qknorm_refkv.py::test_key_segments_full_parity",
    "tests/test_gpu_partial_rope.py::test_partial_rope_attention_matches_oracle",
]


@pytest.mark.gpu
def test_parity_on_the_lds_poison_build():
    lib = pkg_build.POISON_LIB
    if not os.path.exists(lib):
        pytest.fail("libsol_poison.so is not built; run __graft_entry__.build()")
    code = (
        "import sys, pytest\n"
        "from paper_2609_35110_amd import sol\n"
        "sol.LIB_PATH = %r\n"
        "rc = pytest.main(%r + ['-q', '-x', '-p', 'no:cacheprovider', '-m', 'gpu',"
        " '--timeout', '300', '--timeout-method', 'thread'])\n"
        "assert sol.lib()._name == sol.LIB_PATH, sol.lib()._name\n"
        "print('library loaded:', sol.lib()._name)\n"
        "sys.exit(rc)\n" % (lib, CASES))
    print("poison build: %d case groups" % len(CASES), flush=True)
    res = subprocess.run([sys.executable, "-u", "-c", code], cwd=ROOT, capture_output=True, text=True,
                         timeout=900)
    out = res.stdout + res.stderr
    print(out[-3000:], flush=True)
    assert res.returncode == 0, "parity failed on the LDS-poison build:\n" + out[-6000:]
    assert "library loaded: " + lib in out
