#!/usr/bin/env python3
"""Benchmark of one Set Block Decoding decode step on one MI355X.

One step = the whole hot path over one batch: the SBD block forward of the decoder
(all layers + LM head, fp32 logits for every block row) followed by one EB-Sampler
step on those logits.  Workload: Llama-3.1-8B shape with random-init bf16 weights,
batch 1, a 2048-token random prompt prefilled into the KV cache, block k = 16 (the last
committed token + 15 masks), gamma = 1.0.  Inputs are resident in HBM before timing.

Prints one JSON line: value = algorithmic HBM bytes of a step / step time (GB/s),
plus the block-forward ms, the EB-select microseconds, the spread of step times, the same
step with the EB statistics taken from the LM head (sbd_block_step), the measured
streaming ceiling of the device, a roofline entry for the dominant kernel (the per-XCD MLP layer kernel, the fused decode forward, or the gate/up
projection on the per-kernel path; timed live with HIP events on the library stream) and the CPU oracle timed on a bounded sample of the same workload.
"""
import argparse
import dataclasses
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SBD block-forward ms + HBM GB/s (8B shape, k=16); EB-select µs"
PEAK_HBM_GBS = 8000.0


def step_bytes(shape, lens, k, wbytes=2, kvbytes=2):
    """Algorithmic HBM bytes of one step: weights once (wbytes per element: 2 for bf16, 1 for
    e4m3), KV read once and staged K/V written (kvbytes per element, likewise), fp32 logits
    written, EB reads the masked rows' logits."""
    s = shape
    d, F, V = s.d_model, s.ffn_dim, s.vocab
    qd, kvd = s.n_q_heads * s.head_dim, s.n_kv_heads * s.head_dim
    per_layer = (qd + 2 * kvd) * d + d * qd + 2 * F * d + d * F
    weights = wbytes * (s.n_layers * per_layer + V * d)
    B = len(lens)
    M = B * k
    kv_read = sum(lens) * s.n_layers * kvd * 2 * kvbytes
    kv_write = M * s.n_layers * kvd * 2 * kvbytes
    logits = 4 * M * V
    eb = 4 * B * (k - 1) * V
    fwd = weights + kv_read + kv_write + logits
    return fwd, eb


def gate_up_bytes(shape, M):
    """Algorithmic bytes of one gate/up launch: both weight matrices, the bf16 input rows,
    the bf16 SwiGLU output rows."""
    return 2 * 2 * shape.ffn_dim * shape.d_model + 2 * M * shape.d_model + 2 * M * shape.ffn_dim


def layer_mlp_bytes(shape, M, wbytes=2):
    """Algorithmic bytes of one layer_mlp launch (gate/up + SwiGLU + down + residual): the three
    MLP weight matrices, plus the residual rows (int64 fixed point) read once and updated once."""
    d, F = shape.d_model, shape.ffn_dim
    return wbytes * 3 * F * d + 8 * M * d + 8 * M * d


KERNEL_SOURCES = {
    "fused": ("fused.hip", "attention_body.h", "qkv_epilogue.h", "sbd_device.h"),
    "gate_up": ("gemv.hip", "gemv_body.h", "qkv_epilogue.h", "sbd_device.h"),
    "layer_mlp": ("layer_xcd.hip", "gemv_body.h", "attention_body.h", "qkv_epilogue.h", "sbd_device.h"),
}


def source_hash(kind):
    """Hash of the sources of the kernel the counter file describes (stale counters are not used)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kind]:
        with open(os.path.join(ROOT, "paper_2509_04185_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def blas_threads():
    """Threads numpy's BLAS runs the oracle's matrix products on."""
    try:
        from threadpoolctl import threadpool_info
        n = [p["num_threads"] for p in threadpool_info() if p.get("user_api") == "blas"]
        if n:
            return max(n)
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


def cpu_baseline(wl, w_dev, lens, toks, gamma, min_seconds, kv_fp8=False):
    """Time the oracle (fp32, as it stands) on the host: the whole block forward (every layer
    and the LM head) plus the EB step on the same block, repeated until min_seconds have
    passed; returns the mean seconds per step.  kv_fp8: the cache in e4m3 (scale 1)."""
    import numpy as np
    import synth
    from oracle import sbd_oracle as O

    s = wl.shape
    host = synth.weights_to_host(w_dev)
    caches = []
    for b, L in enumerate(lens):
        kk, vv = synth.make_kv(s, wl.seed, b, L, device="cpu")
        c = O.SeqCache.from_arrays(synth.to_host_bits(kk), synth.to_host_bits(vv), np.float32)
        caches.append(c.to_e4m3(0) if kv_fp8 else c)
    model = O.Model(s, host, dtype=np.float32, cache_decoded=False, kv_fp8_exp=0 if kv_fp8 else None)
    is_mask = (toks == s.mask_id).astype(np.uint8)
    reps, total = 0, 0.0
    while total < min_seconds and reps < 8:
        t0 = time.perf_counter()
        res = model.block_forward(caches, toks, [1] * len(lens))
        O.eb_select(res.logits.astype(np.float32), is_mask, gamma, s.mask_id)
        total += time.perf_counter() - t0
        reps += 1
    return total / reps, {"reps": reps, "sample_s": total}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def copy_ceiling(torch, dev):
    """Measured streaming ceiling of the device (GB/s): the library's read probe
    (sbd_stream_probe: non-temporal 16-byte loads, 8 in flight per thread, 8 workgroups per
    CU) over 4 GiB, best of 5 runs.  Before it, a 256 MiB device copy: the calibration that
    counter runs scale FETCH_SIZE / WRITE_SIZE by."""
    from paper_2509_04185_amd.binding import stream_probe
    src = torch.empty(256 * 2**20, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    buf = torch.ones(2**30, dtype=torch.float32, device=dev)
    sink = torch.zeros(64, dtype=torch.int32, device=dev)
    best = 0.0
    for _ in range(5):
        e0.record()
        stream_probe(buf, sink)
        e1.record()
        torch.cuda.synchronize()
        best = max(best, buf.numel() * 4 / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del buf
    torch.cuda.empty_cache()
    return best


def speedup_table(args):
    """time(1), time(k), time(2k) of block forwards at the Llama-3.1-8B shape, and the wall-clock
    speedup model of the paper's Sec. 4.2, speedup(l, k) = k time(1) / (time(2k) + (l - 1) time(k))
    for a block of k tokens sampled in l forwards (NFE speedup k / l).

    time(1): one causal row per sequence (next-token prediction); time(k): k prediction rows;
    time(2k): the first forward of a block, the previous block's k tokens re-fed as causal rows
    plus k new mask rows.  Caches hold synthetic K/V installed with sbd_kv_import (the timing
    does not depend on their values).  Prints a markdown table on stderr and one JSON line.
    """
    import numpy as np
    import torch

    import synth
    from paper_2509_04185_amd import Sbd

    s = synth.LLAMA8B
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    k = 16
    batches = (1, 4, 8)
    lens = (2048, 16384)
    print("[bench] speedup table: generating weights", file=sys.stderr, flush=True)
    w = (synth.make_weights_fp8 if args.weights == "fp8" else synth.make_weights)(s, 1002, device=dev)
    lib = Sbd(s, w, max_batch=max(batches), max_seq_len=max(lens) + 2 * k + 64, max_block=2 * k,
              kv_format="fp8_e4m3" if args.kv == "fp8" else "bf16")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def fwd_ms(B, kk, nc):
        toks, msk = synth.block_rows(1002, s, B, kk, n_causal=nc)
        out = torch.empty((B, kk, s.vocab), dtype=torch.float32, device=dev)
        ids = list(range(B))
        ncs = [nc] * B
        for _ in range(3):
            lib.block_forward(ids, toks, is_mask=msk, n_causal=ncs, out=out)
        torch.cuda.synchronize()
        reps = []
        for _ in range(args.steps):
            e0.record()
            lib.block_forward(ids, toks, is_mask=msk, n_causal=ncs, out=out)
            e1.record()
            torch.cuda.synchronize()
            reps.append(e0.elapsed_time(e1))
        return float(np.median(reps))

    rows = []
    for L in lens:
        print(f"[bench] installing {max(batches)} caches of {L} tokens", file=sys.stderr, flush=True)
        for b in range(max(batches)):
            lib.reset(b)
            kk_, vv_ = synth.make_kv(s, 1002, b, L, device=dev)
            lib.kv_import(b, 0, kk_, vv_)
            del kk_, vv_
        for B in batches:
            t1, tk, t2k = fwd_ms(B, 1, 1), fwd_ms(B, k, 0), fwd_ms(B, 2 * k, k)
            sp = {nfe: k * t1 / (t2k + (k // nfe - 1) * tk) for nfe in (2, 4, 8)}
            rows.append({"cache_len": L, "batch": B, "time_1_ms": round(t1, 4), "time_k_ms": round(tk, 4),
                         "time_2k_ms": round(t2k, 4), "slowdown_k": round(tk / t1, 3),
                         "slowdown_2k": round(t2k / t1, 3),
                         "speedup": {f"nfe_{n}": round(v, 3) for n, v in sp.items()}})
            print(f"[bench] L {L} B {B}: time(1) {t1:.3f} time({k}) {tk:.3f} time({2 * k}) {t2k:.3f} ms",
                  file=sys.stderr, flush=True)
    print(f"\n| cache | batch | time(1) ms | time({k}) ms | time({2 * k}) ms | time({k})/time(1) | "
          f"time({2 * k})/time(1) | speedup, NFE 2 | NFE 4 | NFE 8 |", file=sys.stderr)
    print("|---|---|---|---|---|---|---|---|---|---|", file=sys.stderr)
    for r in rows:
        sp = r["speedup"]
        print(f"| {r['cache_len']} | {r['batch']} | {r['time_1_ms']} | {r['time_k_ms']} | {r['time_2k_ms']} | "
              f"{r['slowdown_k']} | {r['slowdown_2k']} | {sp['nfe_2']} | {sp['nfe_4']} | {sp['nfe_8']} |",
              file=sys.stderr)
    print(json.dumps({"metric": "SBD block-forward time(1), time(k), time(2k) and speedup(l, k)", "k": k,
                      "shape": s.name, "data": "synthetic (random-init weights, synthetic KV caches)",
                      "weights": args.weights, "kv": args.kv, "rows": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama8b_b1_l2048_k16")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="minimum time of the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the per-kernel event pass")
    ap.add_argument("--decode-path", default="auto", choices=["auto", "fused", "kernels", "layers"],
                    help="kernels of decode-sized forwards (sbd_set_decode_path)")
    ap.add_argument("--weights", default="bf16", choices=["bf16", "fp8"],
                    help="weight format: bf16, or e4m3 with a power-of-two scale per matrix (Sec. 4.1's FP8 weights)")
    ap.add_argument("--kv", default="bf16", choices=["bf16", "fp8"],
                    help="KV-cache format: bf16, or e4m3 with scale 1 (Sec. 4.1's 1-byte KV)")
    ap.add_argument("--speedup-table", action="store_true",
                    help="measure time(1), time(k), time(2k) and the paper's speedup(l, k) instead")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(batch sharding across GPUs is a design note only).", file=sys.stderr)
        sys.exit(2)
    if args.kv == "fp8" and args.decode_path == "fused":
        print("the fused decode path reads a bf16 KV cache only", file=sys.stderr)
        sys.exit(2)
    if args.speedup_table:
        return speedup_table(args)

    import numpy as np
    import torch

    import synth
    from paper_2509_04185_amd import Sbd

    wl = synth.WORKLOADS[args.workload]
    s = wl.shape
    gamma = wl.gammas[0]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lens = wl.cache_lens()
    B, k = wl.batch, wl.k
    print(f"[bench] {wl.name}: generating weights", file=sys.stderr, flush=True)
    fp8 = args.weights == "fp8"
    wbytes = 1 if fp8 else 2
    kv8 = args.kv == "fp8"
    kvbytes = 1 if kv8 else 2
    w = (synth.make_weights_fp8 if fp8 else synth.make_weights)(s, wl.seed, device=dev)
    lib = Sbd(s, w, max_batch=B, max_seq_len=max(lens) + k + 64, max_block=k,
              kv_format="fp8_e4m3" if kv8 else "bf16")
    lib.set_decode_path(args.decode_path)
    print(f"[bench] prefilling {B} x {lens[0]}..{lens[-1]} tokens", file=sys.stderr, flush=True)
    for b, L in enumerate(lens):
        lib.prefill(b, synth.make_tokens(wl.seed, L, s, stream=100 + b), want_logits=False)
    torch.cuda.synchronize()
    toks, is_mask = synth.block_rows(wl.seed, s, B, k, n_causal=1)
    seq_ids = list(range(B))
    logits = torch.empty((B, k, s.vocab), dtype=torch.float32, device=dev)

    def step():
        lib.block_forward(seq_ids, toks, is_mask=is_mask, out=logits)
        return lib.eb_select(logits, is_mask, gamma, s.mask_id, want_entropy=False)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # per-step events inside the timed region give the spread of step times
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    e0.record()
    marks[0].record()
    for i in range(args.steps):
        out = step()
        marks[i + 1].record()
    e1.record()
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    per_step = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)])
    n_acc = int(out[0][0])

    # block forward alone and EB select alone
    e0.record()
    for _ in range(args.steps):
        lib.block_forward(seq_ids, toks, is_mask=is_mask, out=logits)
    e1.record()
    torch.cuda.synchronize()
    ms_fwd = e0.elapsed_time(e1) / args.steps
    # EB select alone: each call is queued behind a block forward, so that its events time the
    # device (the mask upload and both kernels), not the host's Python call
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for ea, eb in evs:
        lib.block_forward(seq_ids, toks, is_mask=is_mask, out=logits)
        ea.record()
        lib.eb_select(logits, is_mask, gamma, s.mask_id, want_entropy=False)
        eb.record()
    torch.cuda.synchronize()
    us_eb = 1000.0 * sum(ea.elapsed_time(eb) for ea, eb in evs) / args.steps

    # the same step through sbd_block_step: the EB statistics come from the LM head's
    # epilogue and the logits are neither stored nor read back
    if B * k <= 512 and args.decode_path != "fused":
        for _ in range(3):
            lib.block_step(seq_ids, toks, "eb_entropy", gamma, is_mask=is_mask)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            lib.block_step(seq_ids, toks, "eb_entropy", gamma, is_mask=is_mask)
        e1.record()
        torch.cuda.synchronize()
        ms_fused_step = e0.elapsed_time(e1) / args.steps
    else:
        ms_fused_step = None

    fwd_bytes, eb_bytes = step_bytes(s, lens, k, wbytes, kvbytes)
    value = (fwd_bytes + eb_bytes) / (ms_step * 1e-3) / 1e9
    ceiling = copy_ceiling(torch, dev)

    # per-kernel durations, HIP events around each launch on the library stream
    kernels = {}
    fused_kernels = None
    roofline = None
    if not args.no_profile:
        lib.profile(True)
        lib.profile_read()
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        prof = lib.profile_read()
        lib.profile(False)
        kernels = {n: {"launches": c, "avg_us": 1000.0 * t / c if c else None}
                   for n, (c, t) in prof.items() if c}
        if ms_fused_step is not None:
            lib.profile(True)
            for _ in range(args.steps):
                lib.block_step(seq_ids, toks, "eb_entropy", gamma, is_mask=is_mask)
            torch.cuda.synchronize()
            fprof = lib.profile_read()
            lib.profile(False)
            fused_kernels = {n: {"launches": c, "avg_us": 1000.0 * t / c}
                             for n, (c, t) in fprof.items() if c and n in ("lm_head", "eb_partial", "eb_select")}
        if prof.get("fused", (0, 0.0))[0]:
            # one launch runs every layer and the LM head: its bytes are the block forward's
            kind, bpl = "fused", fwd_bytes
            label = "fused_forward_kernel<128> (all layers + LM head, M = 16)"
        elif prof.get("layer_mlp", (0, 0.0))[0]:
            kind, bpl = "layer_mlp", layer_mlp_bytes(s, B * k, wbytes)
            label = "layer_mlp_kernel (gate/up + SwiGLU + down + residual, per-XCD)"
        else:
            kind, bpl = "gate_up", gate_up_bytes(s, B * k)
            if B * k <= 16:
                label = "gemv_kernel<…, EPI_SWIGLU> (gate/up projection + SwiGLU, decode-sized GEMM)"
            else:
                label = f"gemm_kernel<…, EPI_SWIGLU> (gate/up projection + SwiGLU, M = {B * k})"
        c, t = prof[kind]
        avg_s = t / c * 1e-3
        achieved = bpl / avg_s / 1e9
        traffic = None
        traffic_file = os.path.join(ROOT, "profiles", f"{kind}_traffic_{wl.name}{'_fp8' if fp8 else ''}.json")
        if os.path.exists(traffic_file):
            with open(traffic_file) as f:
                tr = json.load(f)
            if tr.get("kernel_source") == source_hash(kind):
                traffic = tr.get("bytes_per_launch")
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
                    "kernel": label, "bytes_per_launch": bpl, "avg_launch_us": round(avg_s * 1e6, 2),
                    "launches": c}


    cpu = None
    if not args.no_cpu_baseline:
        print(f"[bench] oracle: full block forward + EB, at least {args.cpu_seconds:.0f} s", file=sys.stderr, flush=True)
        est, info = cpu_baseline(wl, w, lens, toks, gamma, args.cpu_seconds, kv8)
        cores = blas_threads()
        cpu = {"value": round((fwd_bytes + eb_bytes) / est / 1e9, 4), "unit": "GB/s", "cores": cores,
               "kind": "oracle", "ms_per_step": round(est * 1e3, 1), "cpu_model": cpu_model(),
               "sample": (f"fp32 numpy oracle: the whole block forward ({s.n_layers} layers + LM head) and the EB "
                          f"select on the same block, {info['reps']} runs, {info['sample_s']:.1f} s timed")}

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": (("fp8-e4m3" if fp8 else "bf16") + " weights, bf16 activations, " +
                  ("fp8-e4m3" if kv8 else "bf16") + " KV") if fp8 or kv8 else "bf16",
        "data": "synthetic (seeded random-init weights, uniform random prompt tokens)",
        "config": {"workload": wl.name, "shape": s.name, "batch": B, "cache_len": lens, "k": k,
                   "gamma": gamma, "n_causal": 1, "decode_path": args.decode_path, "weights": args.weights,
                   "kv": args.kv},
        "block_forward_ms": round(ms_fwd, 4),
        "block_forward_gbs": round(fwd_bytes / (ms_fwd * 1e-3) / 1e9, 1),
        "block_forward_frac_of_peak": round(fwd_bytes / (ms_fwd * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "eb_select_us": round(us_eb, 2),
        "step_ms_p10_p50_p90": [round(float(np.percentile(per_step, q)), 4) for q in (10, 50, 90)],
        "fused_step_ms": None if ms_fused_step is None else round(ms_fused_step, 4),
        "fused_step_kernels": fused_kernels,
        "copy_ceiling_gbs": round(ceiling, 1),
        "block_forward_frac_of_ceiling": round(fwd_bytes / (ms_fwd * 1e-3) / 1e9 / ceiling, 4),
        "step_bytes": fwd_bytes + eb_bytes, "eb_accepted": n_acc,
        "roofline": roofline, "cpu_baseline": cpu, "kernels": kernels,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
