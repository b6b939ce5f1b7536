"""Benchmark of the quantized-KV attention hot path on one MI355X.

Default workload: Llama-3-8B-shaped decode (batch 16, 32 q heads / 8 kv heads,
head_dim 128, context 4096, 2-bit K/V with partition 32, 4 K channels x10).
One step = one hack_decode_step launch: quantize-on-write of one new token per
(sequence, kv head) fused with decode attention over the whole compressed cache.
Ten replicas of the cache rotate so that the 256 MB Infinity Cache cannot hold the
working set.  Also measured: causal prefill (batch 1, 32/8 heads, 8192 tokens,
4-bit K/V, partition 64).  --workload selects another decode workload instead
(ragged paged 70B share, 128K append loop, or the bit-width/partition sweep).

Prints ONE JSON line.  `value` is compressed bytes moved per step / step time.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, 8 TB/s
INT8_PEAK_TOPS = 5000.0      # MI355X dense int8 MFMA, 5.0 POPS


def decode_bytes_per_seq_head(L: int, d: int, bits: int, pi: int, sum_bytes: int) -> int:
    """Compressed bytes one decode reads for one (sequence, kv head) of length L:
    per token K codes + (min, scale) + sums; per full V block codes + (min, scale) +
    sums for every channel; the fp16 open block."""
    P = d // pi
    F, T = L // pi, L % pi
    k = L * (d * bits // 8 + P * 4 + P * sum_bytes)
    v = F * d * (pi * bits // 8 + 4 + sum_bytes)
    return k + v + T * d * 2


def append_bytes(B: int, H: int, d: int, bits: int, pi: int, sum_bytes: int, T_after: int) -> int:
    """Bytes one append moves: fp16 k/v in, one token's K partitions and the fp16
    V value out, plus the block quantization when the open block fills."""
    P = d // pi
    per = 2 * d * 2 + (d * bits // 8 + P * (4 + sum_bytes)) + d * 2
    if T_after == 0:  # the block filled: read the fp16 block, write codes + meta + sums
        per += pi * d * 2 + d * (pi * bits // 8 + 4 + sum_bytes)
    return B * H * per


def quantize_bytes(B: int, H: int, L: int, d: int, bits: int, pi: int, sum_bytes: int) -> int:
    """Bytes one hack_quantize moves: fp16 K and V read once, the compressed cache
    (K rows, full V blocks, the fp16 open block) written once."""
    return B * H * (2 * L * d * 2 + decode_bytes_per_seq_head(L, d, bits, pi, sum_bytes))


def time_quantize(hk, lay, cache, k, v, lens, L, iters: int = 5):
    """Median duration (ms) of hack_quantize on the current stream, HIP events around each call."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ts = []
    for _ in range(iters):
        e0.record()
        hk.hack_quantize(lay, cache, k, v, lens, L)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def profiled_traffic(kernel_file: str, summary: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None when
    the kernel source has changed since the counters were taken."""
    import hashlib
    try:
        text = open(os.path.join(ROOT, "profiles", summary)).read()
        src = open(os.path.join(ROOT, "paper_2502_03589_amd", "csrc", kernel_file), "rb").read()
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines() if ": " in line and not line.startswith(" "))
    if fields.get("kernel_source_sha256", "").strip() != hashlib.sha256(src).hexdigest():
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


VALU_PEAK_LANE_OPS = 16 * 4 * 256 * 2.4e9  # 16 lanes x 4 SIMDs x 256 CUs x 2.4 GHz (unpacked fp32)


def profiled_field(kernel_file: str, summary: str, field: str, sha_field: str = "kernel_source_sha256"):
    """An integer field of a committed rocprofv3 summary, or None when the kernel source
    has changed since the summary was taken."""
    import hashlib
    try:
        text = open(os.path.join(ROOT, "profiles", summary)).read()
        src = open(os.path.join(ROOT, "paper_2502_03589_amd", "csrc", kernel_file), "rb").read()
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines() if ": " in line and not line.startswith(" "))
    if fields.get(sha_field, "").strip() != hashlib.sha256(src).hexdigest():
        return None
    try:
        return int(fields[field])
    except (KeyError, ValueError):
        return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--replicas", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--prefill-iters", type=int, default=10)
    ap.add_argument("--workload", choices=["decode_tiny_l256", "decode_70b_ragged", "decode_long_l131072",
                                           "sweep_bits_partition"],
                    default=None,
                    help="time another decode workload instead (one JSON line per configuration; "
                         "not the headline line)")
    ap.add_argument("--only", choices=["decode", "prefill", "copy"], default=None,
                    help="profiling aid: run one leg alone (copy = plain device copy of a known size, "
                         "the calibration for HBM byte counters)")
    return ap.parse_args()


def copy_calibration(mib: int = 512, iters: int = 5):
    """A plain device-to-device copy of `mib` MiB, `iters` times: a kernel whose HBM
    traffic is known exactly (mib MiB read + mib MiB written per launch)."""
    import torch
    src = torch.ones(mib << 18, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(iters):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_mib": mib, "launches": iters}), flush=True)


def copy_bandwidth(mib: int = 1024, iters: int = 10) -> float:
    """GB/s of a plain device-to-device copy (read + write bytes over the time): the
    bandwidth a streaming kernel reaches on this machine, beside the 8 TB/s datasheet peak."""
    import torch
    src = torch.ones(mib << 18, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(iters):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / iters
    del src, dst
    return 2 * (mib << 20) / (ms * 1e-3) / 1e9


def cpu_baseline_decode(wl, budget_s: float = 15.0):
    """The oracle timed on host cores over a bounded sample of the decode workload:
    whole (sequence, kv head) pairs at the full context, all G query heads each."""
    from threadpoolctl import threadpool_limits

    from oracle import hack_oracle as O
    from paper_2502_03589_amd import synth
    d, L, G = wl.head_dim, wl.context, wl.group
    ch = synth.outlier_channels(wl.seed, d, wl.outlier_channels)
    pairs, bytes_done, t_used = 0, 0, 0.0
    sb = O.sum_bytes(wl.kv_bits, wl.partition)
    while t_used < budget_s and pairs < wl.batch * wl.kv_heads:
        b, h = divmod(pairs, wl.kv_heads)
        k = synth.scale_channels_f16(synth.normal_f16(wl.seed, "k", (L, d), sub=1 + pairs), ch, 10.0)
        v = synth.normal_f16(wl.seed, "v", (L, d), sub=1 + pairs)
        q = synth.normal_f16(wl.seed, "q", (G, d), sub=1 + pairs)
        sq = O.quantize_sequence(k, v, wl.kv_bits, wl.partition)
        with threadpool_limits(1):  # numpy's BLAS on one thread, as reported in `cores`
            t0 = time.perf_counter()
            for g in range(G):
                O.decode_row(q[g], sq)
            t_used += time.perf_counter() - t0
        bytes_done += decode_bytes_per_seq_head(L, d, wl.kv_bits, wl.partition, sb) + G * d * (2 + 4)
        pairs += 1
    return {"value": round(bytes_done / t_used / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{pairs} of {wl.batch * wl.kv_heads} (sequence, kv head) pairs at context {L}, "
                      f"{G} query heads each; {t_used:.1f} s single-threaded numpy"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the decode path shards by "
              f"(sequence, kv head) with no communication, so N GPUs run N independent copies.",
              file=sys.stderr)
        sys.exit(2)
    if args.only == "copy":
        copy_calibration()
        return
    if args.workload is not None:
        bench_workload(args.workload, args.steps, args.warmup)
        return
    if args.only == "prefill":
        print(json.dumps({"prefill": bench_prefill(args.prefill_iters)}), flush=True)
        return
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = synth.WORKLOADS["decode_llama8b_l4096"]
    B, Hq, H, d, L0 = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.context
    bits, pi, R = wl.kv_bits, wl.partition, args.replicas
    total_steps = args.warmup + args.steps
    grow = (total_steps + R - 1) // R
    cap = ((L0 + grow + pi - 1) // pi) * pi
    lay = hk.hack_kv_layout_make(d, H, bits, pi, cap)

    # inputs: K with 4 outlier channels x10, V, the new tokens and the queries
    ch = synth.outlier_channels(wl.seed, d, wl.outlier_channels)
    k = torch.from_numpy(synth.scale_channels_f16(synth.normal_f16(wl.seed, "k", (B, H, L0, d)), ch, 10.0)).to(dev)
    v = torch.from_numpy(synth.normal_f16(wl.seed, "v", (B, H, L0, d))).to(dev)
    nk = torch.from_numpy(synth.scale_channels_f16(synth.normal_f16(wl.seed, "step_k", (8, B, H, d)), ch, 10.0)).to(dev)
    nv = torch.from_numpy(synth.normal_f16(wl.seed, "step_v", (8, B, H, d))).to(dev)
    qs = torch.from_numpy(synth.normal_f16(wl.seed, "q", (8, B, Hq, d))).to(dev)
    caches, lens = [], []
    for r in range(R):
        c = hk.KVCache(lay, B, B, None, dev)
        ln = torch.full((B,), L0, dtype=torch.int32, device=dev)
        if r == 0:
            hk.hack_quantize(lay, c, k, v, ln, L0)
        else:
            for name in hk.SECTIONS:
                c.buffers[name].copy_(caches[0].buffers[name])
        caches.append(c)
        lens.append(ln)
    sb = lay.sum_bytes
    # quantize-on-write of the whole prompt (the prefill side's output), same cache
    q_ms = time_quantize(hk, lay, caches[0], k, v, lens[0], L0)
    q_gbs = quantize_bytes(B, H, L0, d, bits, pi, sb) / (q_ms * 1e-3) / 1e9
    del k, v
    out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)

    # One step = append one token per (sequence, kv head) (quantize-on-write) + decode
    # attention, fused in one launch (hack_decode_step).  The calls are bound once
    # (arguments marshalled up front) so the host runs ahead of the GPU; the length
    # arrays of a replica alternate between input and output; max_len arguments are
    # upper bounds (the kernels read the true lengths from device memory).
    stream = torch.cuda.current_stream()
    lens2 = [torch.zeros_like(x) for x in lens]
    ws = hk.decode_workspace(lay, B, Hq, cap)
    step_calls = [[hk.bind_decode_step(lay, caches[r], nk[r % 8], nv[r % 8], qs[r % 8], src, dst, cap - 1,
                                       hk.TAIL_FP16, out, ws)
                   for src, dst in ((lens[r], lens2[r]), (lens2[r], lens[r]))] for r in range(R)]
    parity = [0] * R

    def step(i):
        r = i % R
        step_calls[r][parity[r]](stream)
        parity[r] ^= 1

    def step_bytes_at(i):
        """Algorithmic bytes of step i: the replica's cache grows by one token per step."""
        Lr = L0 + i // R + 1
        dec = B * H * decode_bytes_per_seq_head(Lr, d, bits, pi, sb) + B * Hq * d * (2 + 4)
        return dec + append_bytes(B, H, d, bits, pi, sb, Lr % pi)

    for i in range(args.warmup):
        step(i)
    nbytes = sum(step_bytes_at(args.warmup + j) for j in range(args.steps))
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for j in range(args.steps):
        step(args.warmup + j)
    ev1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    # the timed region holds nothing but the step launches: the events' span per step
    # is the step kernel's average duration (launches queue back to back)
    avg_kern_ms = ev0.elapsed_time(ev1) / args.steps
    step_bytes = nbytes / args.steps
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    achieved = step_bytes / (avg_kern_ms * 1e-3) / 1e9

    result = {
        "metric": "decode: compressed-KV GB/s (append + attend per step)",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "decode_llama8b_l4096", "batch": B, "q_heads": Hq, "kv_heads": H,
                   "head_dim": d, "context": L0, "kv_bits": bits, "partition": pi, "qp_bits": 8,
                   "outlier_k_channels": wl.outlier_channels, "cache_replicas": R,
                   "step": "append 1 token + decode attention (one launch)", "parallelism": "1 GPU"},
        "roofline": {"bound": "hbm", "kernel": "decode_kernel (hack_decode_step: append + attention + split-K merge)",
                     "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": profiled_traffic("kernels_decode.hip", "decode_llama8b_l4096_hbm_counters.txt"),
                     "avg_kernel_us": round(avg_kern_ms * 1e3, 3),
                     "bytes_per_launch": int(step_bytes)},
        "box_copy_GBs": round(copy_bandwidth(), 1),
        "quantize": {"workload": "decode_llama8b_l4096 prompt (hack_quantize of 16 x 8 x 4096 tokens)",
                     "ms": round(q_ms, 4), "GBs": round(q_gbs, 1), "frac_hbm": round(q_gbs / HBM_PEAK_GBS, 4)},
    }
    if not args.no_prefill and args.only is None:
        result["prefill"] = bench_prefill(args.prefill_iters)
        # the same workload with 4-bit Q/P codes (the literal reading of its 4-bit Q/K/V/P)
        result["prefill_qp4"] = bench_prefill(max(3, args.prefill_iters // 2), 4)
        # the paper's rounding: stochastic K/V, Q and P codes
        result["prefill_stochastic"] = bench_prefill(max(3, args.prefill_iters // 2), 8, 1)
    if not args.no_cpu_baseline and args.only is None:
        result["cpu_baseline"] = cpu_baseline_decode(wl)
    print(json.dumps(result), flush=True)


def bench_prefill(iters: int, qp_bits: int = 8, rounding: int = 0):
    """Causal prefill (batch 1, 32/8 heads, 8192 tokens, 4-bit K/V, partition 64, Q/P
    codes of qp_bits bits): quantize-on-write of the prompt's K/V then attention; int8
    ops of the causal triangle = 2 products x 32 heads x L(L+1)/2 x 128 x 2."""
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    wl = synth.WORKLOADS["prefill_l8192"]
    B, Hq, H, d, L = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.context
    dev = torch.device("cuda:0")
    lay = hk.hack_kv_layout_make(d, H, wl.kv_bits, wl.partition, L, qp_bits, rounding, wl.seed)
    c = hk.KVCache(lay, B, B, None, dev)
    k = torch.from_numpy(synth.normal_f16(wl.seed, "k", (B, H, L, d))).to(dev)
    v = torch.from_numpy(synth.normal_f16(wl.seed, "v", (B, H, L, d))).to(dev)
    q = torch.from_numpy(synth.normal_f16(wl.seed, "q", (B, Hq, L, d))).to(dev)
    ln = torch.full((B,), L, dtype=torch.int32, device=dev)
    out = torch.empty((B, Hq, L, d), dtype=torch.float32, device=dev)
    hk.hack_quantize(lay, c, k, v, ln, L)
    try:
        hk.hack_attend_prefill(lay, c, q, True, out)
    except hk.HackError as e:
        return {"status": f"unavailable: {e}"}
    torch.cuda.synchronize()
    ops = 2 * Hq * (L * (L + 1) // 2) * d * 2 * B
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    qt, at = [], []
    for _ in range(iters):
        e0.record()
        hk.hack_quantize(lay, c, k, v, ln, L)
        e1.record()
        hk.hack_attend_prefill(lay, c, q, True, out)
        e2.record()
        torch.cuda.synchronize()
        qt.append(e0.elapsed_time(e1))
        at.append(e1.elapsed_time(e2))
    a_ms = float(np.median(at))
    q_ms = float(np.median(qt))
    tops = ops / (a_ms * 1e-3) / 1e12
    q_gbs = quantize_bytes(B, H, L, d, wl.kv_bits, wl.partition, lay.sum_bytes) / (q_ms * 1e-3) / 1e9
    res = {"workload": "prefill_l8192", "qp_bits": qp_bits, "rounding": "stochastic" if rounding else "nearest",
           "int8_ops": ops, "attend_ms": round(a_ms, 4),
           "quantize_ms": round(q_ms, 4), "quantize_GBs": round(q_gbs, 1), "TOPS": round(tops, 2),
           "peak_TOPS": INT8_PEAK_TOPS, "frac": round(tops / INT8_PEAK_TOPS, 4)}
    if qp_bits == 8 and rounding == 0:
        # the path is bound by its VALU work: VALU lane-operations per second (profiled
        # instruction count x 64 lanes over the measured time) against the VALU peak
        n = profiled_field("kernels_prefill.hip", "prefill_l8192_valu_mfma_counters.txt", "prefill_valu_instructions_per_launch",
                           "prefill_kernel_source_sha256")
        if n is not None:
            ach = n * 64 / (a_ms * 1e-3) / 1e12
            res["alu_roofline"] = {"bound": "alu", "achieved": round(ach, 2), "peak": round(VALU_PEAK_LANE_OPS / 1e12, 1),
                                   "unit": "T VALU lane-ops/s", "frac": round(ach * 1e12 / VALU_PEAK_LANE_OPS, 4),
                                   "valu_instructions_per_launch": n}
    return res


def bench_workload(name: str, steps: int, warmup: int):
    """Decode throughput on the ragged paged workload (decode calls only) or on the
    128K-context loop (append + decode per step, 2/4 bits, both open-block modes)."""
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    dev = torch.device("cuda:0")
    wl = synth.WORKLOADS[name if name != "sweep_bits_partition" else "decode_llama8b_l4096"]
    B, Hq, H, d, pi = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.partition

    def timed(fn, n):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for i in range(n):
            ev[i][0].record()
            fn(i)
            ev[i][1].record()
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in ev]))

    if name == "sweep_bits_partition":
        # decode_llama8b_l4096's shapes and inputs for each code width and partition the
        # kernels support (attention only, over replicated caches)
        base = synth.WORKLOADS["decode_llama8b_l4096"]
        B, Hq, H, d, L = base.batch, base.q_heads, base.kv_heads, base.head_dim, base.context
        k = torch.from_numpy(synth.normal_f16(base.seed, "k", (B, H, L, d))).to(dev)
        v = torch.from_numpy(synth.normal_f16(base.seed, "v", (B, H, L, d))).to(dev)
        q = torch.from_numpy(synth.normal_f16(base.seed, "q", (B, Hq, d))).to(dev)
        ln = torch.full((B,), L, dtype=torch.int32, device=dev)
        R = 10
        for bits, part, se, rnd in ((2, 32, True, 0), (2, 64, True, 0), (4, 32, True, 0), (4, 64, True, 0),
                                    (2, 32, False, 0), (2, 64, False, 0), (4, 32, False, 0), (4, 64, False, 0),
                                    (2, 32, True, 1), (4, 64, True, 1),
                                    (2, 128, True, 0), (4, 128, True, 0), (2, 128, False, 0), (4, 128, False, 0),
                                    (2, 128, True, 1)):
            # se=False: summation elimination off, no cached sums (fewer bytes, sums rebuilt);
            # rnd=1: stochastic rounding of K/V, Q and P codes
            lay = hk.hack_kv_layout_make(d, H, bits, part, L, 8, rnd, base.seed, sums_cached=se)
            caches = [hk.KVCache(lay, B, B, None, dev) for _ in range(R)]
            for cache in caches:
                hk.hack_quantize(lay, cache, k, v, ln, L)
            ws = hk.decode_workspace(lay, B, Hq, L)
            out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)
            calls = [hk.bind_attend_decode(lay, cache, q, ln, L, hk.TAIL_FP16, out, ws) for cache in caches]
            for i in range(warmup):
                calls[i % R]()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(steps):
                calls[i % R]()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            nbytes = B * H * decode_bytes_per_seq_head(L, d, bits, part, lay.sum_bytes) + B * Hq * d * 6
            print(json.dumps({"workload": name, "kv_bits": bits, "partition": part, "sums_cached": se,
                              "rounding": "stochastic" if rnd else "nearest",
                              "metric": "decode GB/s",
                              "value": round(nbytes / ms / 1e6, 2), "unit": "GB/s", "us_per_call": round(ms * 1e3, 2),
                              "bytes_per_call": int(nbytes), "bytes_per_token_head": round(nbytes / (B * H * L), 2),
                              "frac_of_8TBs": round(nbytes / ms / 1e6 / HBM_PEAK_GBS, 4)}), flush=True)
            del caches, calls
        return
    if name == "decode_tiny_l256":
        # one decode call of batch 1, one q / kv head, 256 tokens: launch-latency sized, so
        # the figure is microseconds per call; 64 replicas keep the inputs out of the caches
        L, R = wl.context, 64
        lay = hk.hack_kv_layout_make(d, H, wl.kv_bits, pi, L)
        k = torch.from_numpy(synth.normal_f16(wl.seed, "k", (B, H, L, d))).to(dev)
        v = torch.from_numpy(synth.normal_f16(wl.seed, "v", (B, H, L, d))).to(dev)
        q = torch.from_numpy(synth.normal_f16(wl.seed, "q", (B, Hq, d))).to(dev)
        ln = torch.full((B,), L, dtype=torch.int32, device=dev)
        caches = [hk.KVCache(lay, B, B, None, dev) for _ in range(R)]
        for cache in caches:
            hk.hack_quantize(lay, cache, k, v, ln, L)
        ws = hk.decode_workspace(lay, B, Hq, L)
        out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)
        calls = [hk.bind_attend_decode(lay, cache, q, ln, L, hk.TAIL_FP16, out, ws) for cache in caches]
        for i in range(warmup):
            calls[i % R]()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(steps):
            calls[i % R]()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        nbytes = B * H * decode_bytes_per_seq_head(L, d, wl.kv_bits, pi, lay.sum_bytes) + B * Hq * d * 6
        print(json.dumps({"workload": name, "metric": "decode us per call", "value": round(ms * 1e3, 2),
                          "unit": "us", "GBs": round(nbytes / ms / 1e6, 2), "bytes_per_call": int(nbytes),
                          "note": "back-to-back calls; launch-latency bound, % of HBM peak not meaningful"}),
              flush=True)
        return
    if name == "decode_70b_ragged":
        lens = synth.uniform_lengths(wl.seed, B, *wl.len_range)
        table, pages = synth.page_table(wl.seed, lens, wl.page_tokens)
        lay = hk.hack_kv_layout_make(d, H, wl.kv_bits, pi, wl.page_tokens)
        cache = hk.KVCache(lay, pages, B, torch.from_numpy(table).to(dev), dev)
        lens_dev = torch.from_numpy(lens.copy()).to(dev)
        for b in range(B):
            L = int(lens[b])
            k = torch.from_numpy(synth.normal_f16(wl.seed, "k", (1, H, L, d), sub=1 + b)).to(dev)
            v = torch.from_numpy(synth.normal_f16(wl.seed, "v", (1, H, L, d), sub=1 + b)).to(dev)
            hk.hack_quantize(lay, cache.sequences(b, 1), k, v, lens_dev[b:b + 1], L)
        q = torch.from_numpy(synth.normal_f16(wl.seed, "q", (B, Hq, d))).to(dev)
        ws = hk.decode_workspace(lay, B, Hq, int(lens.max()))
        out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)
        call = hk.bind_attend_decode(lay, cache, q, lens_dev, int(lens.max()), hk.TAIL_FP16, out, ws)
        for _ in range(warmup):
            call()
        ms = timed(lambda i: call(), steps)
        sb = lay.sum_bytes
        nbytes = sum(H * decode_bytes_per_seq_head(int(L), d, wl.kv_bits, pi, sb) for L in lens) + B * Hq * d * 6
        print(json.dumps({"workload": name, "metric": "decode GB/s", "value": round(nbytes / ms / 1e6, 2),
                          "unit": "GB/s", "us_per_call": round(ms * 1e3, 2), "bytes_per_call": int(nbytes),
                          "frac_of_8TBs": round(nbytes / ms / 1e6 / HBM_PEAK_GBS, 4), "tokens": int(lens.sum())}),
              flush=True)
        return
    # decode_long_l131072: 64 steps of (append one token, decode) after quantizing 131072 tokens
    L0, nsteps = wl.context, wl.steps
    cap = L0 + nsteps
    k_all = torch.from_numpy(np.stack([synth.normal_f16(wl.seed, "k", (H, cap, d), sub=1 + b) for b in range(B)])).to(dev)
    v_all = torch.from_numpy(np.stack([synth.normal_f16(wl.seed, "v", (H, cap, d), sub=1 + b) for b in range(B)])).to(dev)
    qs = torch.from_numpy(np.stack([synth.normal_f16(wl.seed, "q", (B, Hq, d), sub=1 + i) for i in range(nsteps)])).to(dev)
    knew = [k_all[:, :, L0 + i].contiguous() for i in range(nsteps)]
    vnew = [v_all[:, :, L0 + i].contiguous() for i in range(nsteps)]
    for bits in (2, 4):
        for tail in (hk.TAIL_FP16, hk.TAIL_REQUANT, hk.TAIL_DEQUANT):
            lay = hk.hack_kv_layout_make(d, H, bits, pi, cap)
            cache = hk.KVCache(lay, B, B, None, dev)
            lens = torch.full((B,), L0, dtype=torch.int32, device=dev)
            k0, v0 = k_all[:, :, :L0].contiguous(), v_all[:, :, :L0].contiguous()
            ws = hk.decode_workspace(lay, B, Hq, cap)
            out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)
            lens2 = torch.zeros_like(lens)
            calls = [hk.bind_decode_step(lay, cache, knew[i], vnew[i], qs[i], *((lens, lens2) if i % 2 == 0 else (lens2, lens)),
                                         cap - 1, tail, out, ws) for i in range(nsteps)]
            # pass 0 warms the kernels up; both passes start from the same quantized prefix
            for timed_pass in (False, True):
                lens.fill_(L0)
                hk.hack_quantize(lay, cache, k0, v0, lens, L0)
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for i in range(nsteps):
                    calls[i]()
                torch.cuda.synchronize()
                step_ms = (time.perf_counter() - t0) * 1e3 / nsteps
            del k0, v0
            sb = lay.sum_bytes
            dbytes = np.mean([B * H * decode_bytes_per_seq_head(L0 + i + 1, d, bits, pi, sb) for i in range(nsteps)])
            dbytes += B * Hq * d * 6
            abytes = np.mean([append_bytes(B, H, d, bits, pi, sb, (L0 + i + 1) % pi) for i in range(nsteps)])
            print(json.dumps({"workload": name, "kv_bits": bits,
                              "tail_mode": {0: "fp16", 1: "requant", 2: "dequant_requant"}[tail],
                              "metric": "append+decode GB/s", "value": round((dbytes + abytes) / step_ms / 1e6, 2),
                              "unit": "GB/s", "ms_per_step": round(step_ms, 4), "decode_bytes": int(dbytes),
                              "frac_of_8TBs": round((dbytes + abytes) / step_ms / 1e6 / HBM_PEAK_GBS, 4)}),
                  flush=True)
            del cache, ws


if __name__ == "__main__":
    main()
