"""Benchmark of the fused 3D-RoPE + softmax attention layer on one MI355X.

A step is one pass of the whole path over one layer (every batch and head):
by default the prepared path -- sol_prepare_kv_ex (k rotated, k and v
converted to fp16 tiles, one pass) then sol_attn_fwd_prepared_ex (q rotated in
its tile load, softmax(q^ k^T / sqrt(D)) v, bf16 out); --path fused times
sol_attn_fwd, the workspace-free signature (the prepared path chunk by
chunk with its K and V in the out slabs not yet written, then the fused
kernel -- q and k rotated in every tile load -- for the last slabs).  The p720n workload adds
the QK normalization ahead of the rotation; ref720 attends to a cached
reference segment prepared once, before the timed steps; --tau runs the
block-sparse attention, --records the block-INT8 QKV wire records (encoded,
then decoded in the prepare pass and the query tile load).  Inputs are
resident in HBM before the timed region starts.

Prints ONE JSON line: throughput in TFLOP/s (4 Nq Nkv D H B algorithmic flops
per layer), ms per layer, the fraction of the dense bf16 MFMA peak measured
with HIP events on the kernel's stream, the CPU oracle timed on a bounded
row sample of the same workload, and the parity of those rows.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

METRIC = "attention TFLOP/s + % of bf16 MFMA peak and ms/layer at 111,600 tokens"
# MI355X dense bf16 MFMA peak: 256 CUs x 4 SIMDs x 1024 flop/clk x 2.4 GHz.
PEAK_BF16_TFLOPS = 2516.6
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_fwd_traffic.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_35110_amd", "csrc", "sol_kernels.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash():
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(workload_name, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    runs, if they were taken on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    entry = rec.get("%s/%s" % (workload_name, kernel))
    if not entry or entry.get("kernel_sha") != kernel_source_hash():
        return None
    return entry.get("bytes_per_launch")


def cpu_baseline(w, q, k, v, out_gpu, rows_per_thread, ref_kv=None, records=False, block_mask=None):
    """Time the oracle on a bounded, seeded sample of query rows drawn from
    every (b, h) slab, against all keys; check those rows of the GPU output
    against it.  records: the sample comes from slab (0, 0), for which the
    oracle first rotates (and normalises) q and k, encodes the slab's
    block-INT8 records and decodes them, then attends without rotation.
    block_mask: the kernel's block-sparse routing, under which the oracle
    attends (each row to the keys of its query block's kept key blocks)."""
    import numpy as np
    import torch

    import oracle
    from parity import compare
    from paper_2609_35110_amd import workloads as W

    threads = oracle.num_threads()
    slabs = 1 if records else w.B * w.H
    n_rows = min(w.N * slabs, rows_per_thread * threads)
    gen = torch.Generator().manual_seed(w.seed + 31337)
    rows = np.sort(torch.randperm(w.N * slabs, generator=gen)[:n_rows].numpy()).astype(np.int64)
    if records:
        qb, kb, vb = (W.as_bits(t[:1, :1].contiguous()) for t in (q, k, v))
    else:
        qb, kb, vb = (W.as_bits(t) for t in (q, k, v))
    kw = {}
    if w.qk_norm:
        gq, gk = W.norm_weights(w)
        kw = dict(q_gamma=gq.numpy(), k_gamma=gk.numpy(), eps=W.QK_NORM_EPS)
    if block_mask is not None:
        kw["block_mask"] = block_mask
    t0 = time.perf_counter()
    if records:
        if w.qk_norm:
            qh = oracle.qknorm_rope3d(qb, w.T, w.Hl, w.Wl, kw["q_gamma"], kw["eps"])
            kh = oracle.qknorm_rope3d(kb, w.T, w.Hl, w.Wl, kw["k_gamma"], kw["eps"])
        else:
            qh, kh = oracle.rope3d_bf16(qb, w.T, w.Hl, w.Wl), oracle.rope3d_bf16(kb, w.T, w.Hl, w.Wl)
        qb, kb, vb = oracle.decode_qkv(oracle.encode_qkv(qh, kh, vb))
        kw = dict(rope=False)
    if ref_kv is not None:
        # keys: the cached reference segment (its own grid), then the own tokens
        krb, vrb = (W.as_bits(t) for t in ref_kv)
        kb = np.concatenate([oracle.rope3d_bf16(krb, *w.ref_grid),
                             oracle.rope3d_bf16(kb, w.T, w.Hl, w.Wl)], 2)
        vb = np.concatenate([vrb, vb], 2)
        kw["rope_k"] = False
    ref = oracle.attn_rows(qb, kb, vb, w.T, w.Hl, w.Wl, rows=rows, threads=threads, **kw)
    dt = time.perf_counter() - t0
    if block_mask is None:
        flops = 4.0 * w.n_kv * w.D * n_rows
    else:
        # each row attends to the keys of its query block's kept key blocks
        nkb = block_mask.shape[-1]
        keys_in = np.minimum(w.N - np.arange(nkb) * 128, 128)
        kept_keys = (block_mask.reshape(-1, nkb) * keys_in).sum(-1)  # per (slab, query block)
        flops = 4.0 * w.D * float(kept_keys[(rows // w.N) * block_mask.shape[2] + (rows % w.N) // 256].sum())
    got = W.as_bits(out_gpu.cpu()).reshape(-1, w.D)[rows]
    # errors in units of the head's output RMS; for local attention (shared
    # q/k direction) row magnitudes spread too far for one scale, so per row
    groups = np.arange(n_rows) if w.shared_dir else rows // w.N
    par = compare(got, ref, groups)
    where = "head (0,0)" if records else "all %d heads" % slabs
    cpu = {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "%d query rows (seeded) over %s, each against %s, fp64 C oracle, %.1f s; "
                  "full layer extrapolates to %.0f s" % (
                      n_rows, where,
                      "all %d keys" % w.n_kv if block_mask is None else "the keys of its kept blocks",
                      dt, dt * w.B * w.H * w.N / n_rows),
    }
    return cpu, par


def calibrate_copy(mib):
    """A plain copy of known size: each launch reads and writes mib MiB."""
    import torch
    n = mib * 1024 * 1024 // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": n * 4, "launches": 3}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="p720",
                    help="tiny | low | p480 | p720 | share | p720n (QK normalization) | "
                         "ref720 (cached reference keys)")
    ap.add_argument("--path", default="prepared", choices=["fused", "prepared"],
                    help="prepared: sol_prepare_kv (K rotated, V to fp16, one pass) then "
                         "sol_attn_fwd_prepared (q rotated in its tile load); fused: sol_attn_fwd "
                         "(no workspace: prepared chunks in the unwritten out slabs, the fused kernel "
                         "for the last slabs)")
    ap.add_argument("--tau", type=float, default=None,
                    help="block-sparse attention with this threshold parameter (the paper's "
                         "refinement steps use 1.0, 1.25, 1.5); the step is then sol_prepare_kv_ex + "
                         "sol_sparse_route + sol_attn_fwd_sparse")
    ap.add_argument("--records", action="store_true",
                    help="block-INT8 QKV records (the quantized exchange format): the step is "
                         "sol_qkv_encode (normalise, rotate, quantise) + sol_prepare_kv_records + "
                         "sol_attn_fwd_records (q decoded in the tile load)")
    ap.add_argument("--cpu-rows-per-thread", type=int, default=1536,
                    help="oracle rows per host thread for the CPU baseline (p720: about 14 s on 16 cores)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-path", action="store_true",
                    help="skip timing the other dense path (profiling runs: one path per trace)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (3 times), the "
                         "known-size reference for the FETCH_SIZE / WRITE_SIZE counters")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the attention layer would shard by heads, one GPU per head group). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_35110_amd import sol
    from paper_2609_35110_amd import workloads as W

    if not torch.cuda.is_available():
        print("no HIP device visible", file=sys.stderr)
        sys.exit(1)
    w = W.WORKLOADS[args.workload]
    dev = "cuda:0"
    log("workload %s: %s" % (w.name, w.describe()))
    t0 = time.perf_counter()
    q, k, v = W.make_inputs(w)
    log("inputs generated in %.1f s" % (time.perf_counter() - t0))
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    out = torch.empty_like(qd)
    tab = sol.rope3d_table(w.T, w.Hl, w.Wl, device=dev)
    torch.cuda.synchronize()

    k_prep, v_prep = sol.prepared_kv_buffers(w.B, w.H, w.n_kv, dev)
    gq = gk = None
    if w.qk_norm:
        gq, gk = (g.to(dev) for g in W.norm_weights(w))
    ref_kv = None
    if w.n_ref:
        # the cached reference keys and values: prepared once, outside the step
        ref_kv = W.make_ref_inputs(w)
        rtab = sol.rope3d_table(*w.ref_grid, device=dev)
        sol.prepare_kv_ex(ref_kv[0].to(dev), ref_kv[1].to(dev), *w.ref_grid, rtab, k_prep, v_prep,
                          key0=0, n_kv=w.n_kv)
        torch.cuda.synchronize()
    sparse = args.tau is not None
    records = args.records
    special = w.qk_norm or w.n_ref or sparse or records
    if records and (sparse or w.n_ref):
        print("--records runs the dense self-attention of one sequence", file=sys.stderr)
        sys.exit(2)
    if special and args.path == "fused":
        print("the fused path has neither QK normalization, nor a key cache, nor block sparsity",
              file=sys.stderr)
        sys.exit(2)
    if sparse and w.n_ref:
        print("block-sparse attention is the self-attention of one sequence (no key cache)",
              file=sys.stderr)
        sys.exit(2)
    sws = sol.sparse_workspace(qd) if sparse else None
    rec = (torch.empty((w.B, w.N, w.H, sol.QKV_RECORD_BYTES), dtype=torch.uint8, device=dev)
           if records else None)

    def launches(path):
        """The launches of one step, in order: [(name, fn)]."""
        if path == "prepared" and records:
            return [("qkv_encode", lambda: sol.qkv_encode(qd, kd, vd, w.T, w.Hl, w.Wl, tab, gq, gk,
                                                          W.QK_NORM_EPS, rec=rec)),
                    ("prepare_kv", lambda: sol.prepare_kv_records(rec, k_prep, v_prep)),
                    ("attn_fwd_records", lambda: sol.attn_fwd_records(rec, k_prep, v_prep, out=out))]
        if path == "prepared" and sparse:
            return [("prepare_kv", lambda: sol.prepare_kv_ex(kd, vd, w.T, w.Hl, w.Wl, tab, k_prep, v_prep,
                                                             gamma=gk, eps=W.QK_NORM_EPS)),
                    ("sparse_route", lambda: sol.sparse_route(qd, k_prep, w.T, w.Hl, w.Wl, tab, args.tau,
                                                              workspace=sws, gamma=gq, eps=W.QK_NORM_EPS)),
                    ("attn_fwd_sparse", lambda: sol.attn_fwd_sparse(qd, k_prep, v_prep, w.T, w.Hl, w.Wl, tab,
                                                                    sws, gamma=gq, eps=W.QK_NORM_EPS,
                                                                    out=out))]
        if path == "prepared":
            return [("prepare_kv", lambda: sol.prepare_kv_ex(kd, vd, w.T, w.Hl, w.Wl, tab, k_prep, v_prep,
                                                             key0=w.n_ref, n_kv=w.n_kv, gamma=gk,
                                                             eps=W.QK_NORM_EPS)),
                    ("attn_fwd_prepared", lambda: sol.attn_fwd_prepared_ex(qd, k_prep, v_prep, w.n_kv, w.T, w.Hl,
                                                                           w.Wl, tab, gamma=gq,
                                                                           eps=W.QK_NORM_EPS, out=out))]
        return [("attn_fwd", lambda: sol.attn_fwd(qd, kd, vd, w.T, w.Hl, w.Wl, tab, out=out))]

    def timed(path, steps, warmup):
        """HIP events around every launch on the launch stream: per-step ms and
        per-launch ms lists."""
        ls = launches(path)
        for _ in range(warmup):
            for _, fn in ls:
                fn()
        stream = torch.cuda.current_stream()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps * len(ls) + 1)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        e = 1
        for _ in range(steps):
            for _, fn in ls:
                fn()
                ev[e].record(stream)
                e += 1
        torch.cuda.synchronize()
        per = {name: [] for name, _ in ls}
        for i in range(steps):
            for j, (name, _) in enumerate(ls):
                a = i * len(ls) + j
                per[name].append(ev[a].elapsed_time(ev[a + 1]))
        total = ev[0].elapsed_time(ev[-1])
        return total / steps, per

    ms_step, per = timed(args.path, args.steps, args.warmup)
    main_kernel = ("attn_fwd" if args.path == "fused" else "attn_fwd_sparse" if sparse
                   else "attn_fwd_records" if records else "attn_fwd_prepared")
    kern = per[main_kernel]
    ms_launch = sum(kern) / len(kern)
    ks = sorted(kern)
    ms_median = ks[len(ks) // 2]
    tflops = w.flops / (ms_step * 1e-3) / 1e12
    achieved = w.flops / (ms_launch * 1e-3) / 1e12
    sparsity = None
    if sparse:
        # flops the sparse kernel executes: each query block's rows times the
        # keys of its kept blocks, 4 D per (query, key) pair
        counts, blocks = sol.sparse_routing(sws, w.B, w.H, w.N)
        counts = counts.cpu().to(torch.int64)
        blocks = blocks.cpu().to(torch.int64)
        nkb = blocks.shape[-1]
        keys_in = torch.clamp(w.N - torch.arange(nkb) * sol.SPARSE_KEY_BLOCK, max=sol.SPARSE_KEY_BLOCK)
        kept = torch.arange(nkb)[None, None, None, :] < counts[..., None]
        kept_keys = (keys_in[blocks.clamp(0, nkb - 1)] * kept).sum(-1)            # [B, H, nqb]
        nqb = counts.shape[-1]
        rows = torch.clamp(w.N - torch.arange(nqb) * sol.SPARSE_QUERY_BLOCK, max=sol.SPARSE_QUERY_BLOCK)
        pairs = float((kept_keys * rows).sum())
        exec_flops = 4.0 * w.D * pairs
        sparsity = {"tau": args.tau, "density": pairs / (w.B * w.H * float(w.N) ** 2),
                    "executed_flops": exec_flops,
                    "executed_tflops": exec_flops / (ms_launch * 1e-3) / 1e12}
        achieved = sparsity["executed_tflops"]
        # the step's throughput counts the flops it executes: the kept blocks'
        tflops = exec_flops / (ms_step * 1e-3) / 1e12
        log("block-sparse tau=%g: density %.4f, %.1f executed TFLOP/s in %s"
            % (args.tau, sparsity["density"], achieved, main_kernel))
    log("timed %d steps (%s): %.3f ms/step, %s %.3f ms avg (median %.3f) -> %.1f TFLOP/s"
        % (args.steps, args.path, ms_step, main_kernel, ms_launch, ms_median, tflops))
    other = "fused" if args.path == "prepared" else "prepared"
    ms_other = None
    if not special and not args.no_other_path:
        ms_other, _ = timed(other, min(3, args.steps), 1)
        log("other path (%s): %.3f ms/step" % (other, ms_other))

    # the dense fp16 MFMA rate this machine sustains at the attention kernels'
    # launch shape (one wave per SIMD), with seeded operands
    gen = torch.Generator().manual_seed(w.seed + 4242)
    ops = torch.randn(8192, generator=gen).to(torch.float16).to(dev)
    probe_wg, probe_iters = 2048, 25000
    sol.mfma_probe(ops, probe_wg, 1000)
    probe_ms = []
    for _ in range(3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        sol.mfma_probe(ops, probe_wg, probe_iters)
        e1.record()
        torch.cuda.synchronize()
        probe_ms.append(e0.elapsed_time(e1))
    probe_tflops = sol.mfma_probe_flops(probe_wg, probe_iters) / (min(probe_ms) * 1e-3) / 1e12
    log("mfma probe: %.1f TFLOP/s (%.2f GHz equivalent); the step reaches %.1f %% of it"
        % (probe_tflops, 2.4 * probe_tflops / PEAK_BF16_TFLOPS, 100.0 * tflops / probe_tflops))

    traffic = measured_traffic(w.name + ("@tau%g" % args.tau if sparse else ""), main_kernel)
    result = {
        "metric": METRIC,
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # MFMA operand type: the fused path multiplies bf16, the prepared path
        # fp16 (bf16 inputs and output, fp32 accumulation in both)
        "dtype": "bf16" if args.path == "fused" else "f16",
        "data": "synthetic (seeded N(0,1) bf16 q/k/v of the layer's shape)",
        "config": {
            "workload": "%s: %s" % (w.name, w.describe()),
            "B": w.B, "H": w.H, "N": w.N, "D": w.D, "grid": [w.T, w.Hl, w.Wl], "n_text": w.n_text,
            "n_kv": w.n_kv, "qk_norm": w.qk_norm,
            "rope": ("3d (32/48/48, base 1e4) fused into the q and k tile loads" if args.path == "fused"
                     else "3d (32/48/48, base 1e4): q in the tile load, k in a one-pass prologue"),
            "path": ("sol_attn_fwd" if args.path == "fused"
                     else "sol_qkv_encode + sol_prepare_kv_records + sol_attn_fwd_records" if records
                     else "sol_prepare_kv_ex + sol_sparse_route + sol_attn_fwd_sparse" if sparse
                     else "sol_prepare_kv_ex + sol_attn_fwd_prepared_ex"),
            "qkv_records": records,
        },
        "ms_per_layer": ms_step,
        "kernel_ms_median": ms_median,
        "pct_peak_bf16": 100.0 * tflops / PEAK_BF16_TFLOPS,
        "kernel_ms": {name: sum(v) / len(v) for name, v in per.items()},
        "block_sparse": sparsity,
        "mfma_probe": {
            "what": "fp16 32x32x16 MFMAs only, one wave per SIMD, seeded operands (sol_mfma_probe)",
            "tflops": probe_tflops,
            "ghz_equivalent": 2.4 * probe_tflops / PEAK_BF16_TFLOPS,
            "pct_of_probe": 100.0 * tflops / probe_tflops,
            "kernel_frac_of_probe": achieved / probe_tflops,
        },
        "other_path": None if ms_other is None else {
            "path": other, "ms_per_step": ms_other, "tflops": w.flops / (ms_other * 1e-3) / 1e12},
        "roofline": {
            "kernel": main_kernel,
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": traffic,
        },
    }
    if sparse:
        result["metric"] = METRIC + " (block-sparse: the flops of the kept blocks)"
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        mask = None
        if sparse:
            from parity import sparse_mask
            mask = sparse_mask(sws, w.B, w.H, w.N)
        cpu, par = cpu_baseline(w, q, k, v, out, args.cpu_rows_per_thread, ref_kv, records, mask)
        result["cpu_baseline"] = cpu
        result["parity"] = par
        from parity import passes
        if not passes(par):
            # fail closed: no throughput for a kernel that disagrees with the oracle
            result["value"] = None
            result["error"] = "parity failed on the sampled rows"
        log("cpu baseline: %s; parity %s" % (cpu, par))
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
