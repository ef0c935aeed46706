"""Write workload_sha256.txt: SHA-256 fingerprints of the bytes the seeded
input generator (paper_2609_35110_amd/workloads.py) produces for every named
workload -- the first and last (b, h) slab of q, k and v, the reference
segment's k and v slabs, the boosted-key indices and the QK-norm weights --
so that a change of generator, library or machine that would change the
inputs is caught.  Run from the repository root:

    python tests/golden/make_workload_sha256.py

It calls the input generator only (no method arithmetic, no oracle, no HIP).
"""
import hashlib
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from paper_2609_35110_amd import workloads as W  # noqa: E402

OUT = os.path.join(HERE, "workload_sha256.txt")


def fingerprints():
    """[(workload, item, sha256 hex)] in a fixed order."""
    rows = []
    h = lambda t: hashlib.sha256(t.contiguous().numpy().tobytes() if t.dtype != W.torch.bfloat16
                                 else W.as_bits(t).tobytes()).hexdigest()
    for name, w in W.WORKLOADS.items():
        last = w.B * w.H - 1
        boosted = W.boosted_tokens(w)
        for t, tn in enumerate("qkv"):
            for bh in sorted({0, last}):
                rows.append((name, "%s/%d" % (tn, bh), h(W.make_slab(w, t, bh, boosted=boosted))))
        if w.n_ref:
            for t, tn in enumerate(("k_ref", "v_ref")):
                for bh in sorted({0, last}):
                    rows.append((name, "%s/%d" % (tn, bh), h(W.make_ref_slab(w, t, bh))))
        if boosted.numel():
            rows.append((name, "boosted", h(boosted)))
        if w.qk_norm:
            gq, gk = W.norm_weights(w)
            rows.append((name, "gamma_q", h(gq)))
            rows.append((name, "gamma_k", h(gk)))
    return rows


def main():
    with open(OUT, "w") as f:
        f.write("# SHA-256 of the seeded inputs (written by make_workload_sha256.py from the input\n"
                "# generator alone).  workload  item (tensor/slab b*H+h, or a side draw)  sha256\n")
        for r in fingerprints():
            f.write("%s %s %s\n" % r)
    print(OUT)


if __name__ == "__main__":
    main()
