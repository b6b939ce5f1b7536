"""Benchmark of the quantized-KV attention hot path on one MI355X.

Headline workload: the 70B-shaped one-GPU decode share (batch 64, 64 q heads / 8 kv
heads, head_dim 128, per-request context uniform in [1024, 32768], 256-token pages,
2-bit K/V with partition 32).  One step = one hack_decode_step: quantize-on-write of
one new token per (sequence, kv head) fused with decode attention over the whole
compressed cache (0.88 GB, beyond the 256 MB Infinity Cache, so no replicas are
needed).  Also measured, each with its own roofline: the Llama-3-8B-shaped decode
(batch 16, 32/8 heads, context 4096, 4 K channels x10; ten cache replicas), the
128K-context append loop (batch 4, 32/8 heads, 2- and 4-bit), the single small decode
(launch-latency bound), causal prefill (batch 1, 32/8 heads, 8192 tokens, 4-bit K/V,
partition 64) and quantize-on-write of a prompt.  The oracle is timed on the host's
cores over a bounded sample of the headline workload, before the GPU is touched.

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


def time_quantize(hk, lay, cache, k, v, lens, L, iters: int = 5, calls: int = 10):
    """Per-call duration (ms) of hack_quantize: the median over `iters` groups of `calls`
    back-to-back calls on the current stream (HIP events around each group; every call
    rewrites the same cache), so one call's launch latency is not counted as its work."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    hk.hack_quantize(lay, cache, k, v, lens, L)
    ts = []
    for _ in range(iters):
        e0.record()
        for _ in range(calls):
            hk.hack_quantize(lay, cache, k, v, lens, L)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) / calls)
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
                                           "sweep_bits_partition", "sweep_prefill_partition"],
                    default=None,
                    help="time another decode workload instead (one JSON line per configuration; "
                         "not the headline line)")
    ap.add_argument("--only", choices=["decode", "llama8b", "long", "tiny", "prefill", "project", "copy", "cpu"],
                    default=None,
                    help="profiling aid: run one leg alone (decode = the headline 70B-share decode step; "
                         "copy = plain device copy of a known size, the calibration for HBM byte counters)")
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


# ---------------------------------------------------------------------------------
# Oracle baseline on the host cores (run before the GPU is initialised)
# ---------------------------------------------------------------------------------
def _oracle_worker(pairs, barrier, results, slot):
    """Times the oracle's decode attention (G query rows over L tokens) for each
    (sequence, kv head, L) of `pairs`, after building their quantized caches untimed.
    All workers start their timed section together (barrier)."""
    from threadpoolctl import threadpool_limits

    from oracle import hack_oracle as O
    from paper_2502_03589_amd import synth
    wl = synth.WORKLOADS["decode_70b_ragged"]
    d, G, H = wl.head_dim, wl.group, wl.kv_heads
    with threadpool_limits(1):
        prepared = []
        per_seq = {}
        for b, h, L in pairs:
            if b not in per_seq:
                per_seq = {b: (synth.normal_f16(wl.seed, "k", (1, H, L, d), sub=1 + b),
                               synth.normal_f16(wl.seed, "v", (1, H, L, d), sub=1 + b))}
            k, v = per_seq[b]
            sq = O.quantize_sequence(k[0, h], v[0, h], wl.kv_bits, wl.partition)
            q = synth.normal_f16(wl.seed, "q", (1, H * G, d))[0, h * G:(h + 1) * G]
            prepared.append((sq, q, L))
        per_seq = None
        if barrier is not None:
            barrier.wait()
        t0 = time.perf_counter()
        nbytes = 0
        sb = O.sum_bytes(wl.kv_bits, wl.partition)
        for sq, q, L in prepared:
            for g in range(G):
                O.decode_row(q[g], sq)
            nbytes += decode_bytes_per_seq_head(L, d, wl.kv_bits, wl.partition, sb) + G * d * (2 + 4)
        dt = time.perf_counter() - t0
    if results is not None:
        results[slot] = (nbytes, dt)
    return nbytes, dt


def cpu_baseline_decode(pairs_per_core: int = 10):
    """The oracle on every host core: one forked worker per core, each timing the
    decode attention of `pairs_per_core` whole (sequence, kv head) pairs of the headline
    workload (lengths from the same seeded draw); aggregate rate = all bytes / the
    slowest worker's timed span.  Also one worker alone on one core, as a second figure."""
    import multiprocessing as mp

    from paper_2502_03589_amd import synth
    wl = synth.WORKLOADS["decode_70b_ragged"]
    lens = synth.uniform_lengths(wl.seed, wl.batch, *wl.len_range)
    cores = len(os.sched_getaffinity(0))
    all_pairs = [(b, h, int(lens[b])) for b in range(wl.batch) for h in range(wl.kv_heads)]
    n = min(len(all_pairs), cores * pairs_per_core)
    ctx = mp.get_context("fork")  # no GPU state exists yet in this process
    one_b, one_t = _oracle_worker(all_pairs[:pairs_per_core], None, None, 0)
    barrier = ctx.Barrier(cores)
    results = ctx.Manager().dict()
    procs = [ctx.Process(target=_oracle_worker, args=(all_pairs[w:n:cores], barrier, results, w))
             for w in range(cores)]
    for pr in procs:
        pr.start()
    for pr in procs:
        pr.join()
    if any(pr.exitcode != 0 for pr in procs) or len(results) != cores:
        return {"status": "oracle workers failed"}
    tot_b = sum(v[0] for v in results.values())
    span = max(v[1] for v in results.values())
    lsum = sum(int(L) for _, _, L in all_pairs[:n])
    return {"value": round(tot_b / span / 1e9, 4), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": f"decode attention of {n} of {len(all_pairs)} (sequence, kv head) pairs of decode_70b_ragged "
                      f"({lsum} cached tokens, {wl.group} query rows each, inputs quantized untimed), "
                      f"{cores} forked workers of single-threaded numpy, {span:.1f} s wall",
            "single_core": {"value": round(one_b / one_t / 1e9, 4), "unit": "GB/s", "cores": 1,
                            "sample": f"first {pairs_per_core} pairs, {one_t:.1f} s"}}


# ---------------------------------------------------------------------------------
# GPU legs
# ---------------------------------------------------------------------------------
def roofline_hbm(kernel: str, step_bytes: float, avg_kern_ms: float, kernel_file: str, counters: str):
    achieved = step_bytes / (avg_kern_ms * 1e-3) / 1e9
    return {"bound": "hbm", "kernel": kernel, "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": profiled_traffic(kernel_file, counters),
            "avg_kernel_us": round(avg_kern_ms * 1e3, 3), "bytes_per_launch": int(step_bytes)}


def run_steps(step, step_bytes_at, warmup: int, steps: int, stream):
    """Warm up, then time `steps` steps: wall clock (host, synchronized on both sides)
    and HIP events recorded on the launch stream around the queued launches."""
    import torch
    for i in range(warmup):
        step(i)
    nbytes = sum(step_bytes_at(warmup + j) for j in range(steps))
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for j in range(steps):
        step(warmup + j)
    ev1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    return nbytes / steps, (t1 - t0) * 1e3 / steps, ev0.elapsed_time(ev1) / steps


def bench_ragged(steps: int, warmup: int):
    """Headline: decode steps (append one token + attend) on the 70B-shaped share."""
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    dev = torch.device("cuda:0")
    wl = synth.WORKLOADS["decode_70b_ragged"]
    B, Hq, H, d, pi, pt = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.partition, wl.page_tokens
    total = warmup + steps
    lens = synth.uniform_lengths(wl.seed, B, *wl.len_range)
    # each sequence gets pages for its prompt plus every token the steps append
    table, pages = synth.page_table(wl.seed, lens, pt, spare_pages=(total + pt - 1) // pt)
    lay = hk.hack_kv_layout_make(d, H, wl.kv_bits, pi, pt)
    cache = hk.KVCache(lay, pages, B, torch.from_numpy(table).to(dev), dev)
    lens_a = torch.from_numpy(lens.copy()).to(dev)
    for b in range(B):
        L = int(lens[b])
        k = torch.from_numpy(synth.normal_f16(wl.seed, "k", (1, H, L, d), sub=1 + b)).to(dev)
        v = torch.from_numpy(synth.normal_f16(wl.seed, "v", (1, H, L, d), sub=1 + b)).to(dev)
        hk.hack_quantize(lay, cache.sequences(b, 1), k, v, lens_a[b:b + 1], L)
    del k, v
    nk = torch.from_numpy(synth.normal_f16(wl.seed, "step_k", (8, B, H, d))).to(dev)
    nv = torch.from_numpy(synth.normal_f16(wl.seed, "step_v", (8, B, H, d))).to(dev)
    qs = torch.from_numpy(synth.normal_f16(wl.seed, "q", (8, B, Hq, d))).to(dev)
    lens_b = torch.zeros_like(lens_a)
    max_len = int(lens.max()) + total - 1  # bounds the lengths before any of the steps
    ws = hk.decode_workspace(lay, B, Hq, max_len + 1)
    out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)
    calls = [[hk.bind_decode_step(lay, cache, nk[r], nv[r], qs[r], src, dst, max_len, hk.TAIL_FP16, out, ws)
              for src, dst in ((lens_a, lens_b), (lens_b, lens_a))] for r in range(8)]
    stream = torch.cuda.current_stream()
    sb = lay.sum_bytes

    def step(i):
        calls[i % 8][i % 2](stream)

    def step_bytes_at(i):
        dec = sum(H * decode_bytes_per_seq_head(int(L) + i + 1, d, wl.kv_bits, pi, sb) for L in lens)
        app = sum(append_bytes(1, H, d, wl.kv_bits, pi, sb, (int(L) + i + 1) % pi) for L in lens)
        return dec + B * Hq * d * (2 + 4) + app

    step_bytes, ms, kern_ms = run_steps(step, step_bytes_at, warmup, steps, stream)
    cfg = {"workload": "decode_70b_ragged", "batch": B, "q_heads": Hq, "kv_heads": H, "head_dim": d,
           "context": f"uniform [{wl.len_range[0]}, {wl.len_range[1]}] per request ({int(lens.sum())} tokens)",
           "page_tokens": pt, "kv_bits": wl.kv_bits, "partition": pi, "qp_bits": 8,
           "step": "append 1 token per (sequence, kv head) + decode attention (one launch)",
           "parallelism": "1 GPU"}
    roof = roofline_hbm("decode_kernel (hack_decode_step: append + attention + split-K merge)", step_bytes,
                        kern_ms, "kernels_decode.hip", "decode_70b_ragged_hbm_counters.txt")
    return step_bytes, ms, cfg, roof


def bench_llama8b(steps: int, warmup: int, R: int):
    """Decode steps on the Llama-3-8B-shaped workload over R cache replicas."""
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    dev = torch.device("cuda:0")
    wl = synth.WORKLOADS["decode_llama8b_l4096"]
    B, Hq, H, d, L0 = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.context
    bits, pi = wl.kv_bits, wl.partition
    grow = (warmup + steps + R - 1) // R
    cap = ((L0 + grow + pi - 1) // pi) * pi
    lay = hk.hack_kv_layout_make(d, H, bits, pi, cap)
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
        Lr = L0 + i // R + 1
        dec = B * H * decode_bytes_per_seq_head(Lr, d, bits, pi, sb) + B * Hq * d * (2 + 4)
        return dec + append_bytes(B, H, d, bits, pi, sb, Lr % pi)

    step_bytes, ms, kern_ms = run_steps(step, step_bytes_at, warmup, steps, stream)
    res = {"workload": "decode_llama8b_l4096", "step": "append 1 token + decode attention (one launch)",
           "cache_replicas": R, "ms_per_step": round(ms, 5), "GBs": round(step_bytes / (ms * 1e-3) / 1e9, 2),
           "roofline": roofline_hbm("decode_kernel (hack_decode_step)", step_bytes, kern_ms,
                                    "kernels_decode.hip", "decode_llama8b_l4096_hbm_counters.txt")}
    quant = {"workload": "decode_llama8b_l4096 prompt (hack_quantize of 16 x 8 x 4096 tokens)",
             "ms": round(q_ms, 4), "GBs": round(q_gbs, 1), "frac_hbm": round(q_gbs / HBM_PEAK_GBS, 4)}
    return res, quant


def bench_long(bits_list=(2, 4)):
    """The 128K-context loop: after quantizing 131072 tokens per sequence, 64 steps of
    (append one token per (sequence, kv head), decode attention), fp16 open block."""
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    dev = torch.device("cuda:0")
    wl = synth.WORKLOADS["decode_long_l131072"]
    B, Hq, H, d, pi = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.partition
    L0, nsteps = wl.context, wl.steps
    cap = L0 + nsteps
    k_all = torch.from_numpy(np.stack([synth.normal_f16(wl.seed, "k", (H, cap, d), sub=1 + b) for b in range(B)])).to(dev)
    v_all = torch.from_numpy(np.stack([synth.normal_f16(wl.seed, "v", (H, cap, d), sub=1 + b) for b in range(B)])).to(dev)
    qs = torch.from_numpy(np.stack([synth.normal_f16(wl.seed, "q", (B, Hq, d), sub=1 + i) for i in range(nsteps)])).to(dev)
    knew = [k_all[:, :, L0 + i].contiguous() for i in range(nsteps)]
    vnew = [v_all[:, :, L0 + i].contiguous() for i in range(nsteps)]
    k0, v0 = k_all[:, :, :L0].contiguous(), v_all[:, :, :L0].contiguous()
    del k_all, v_all
    stream = torch.cuda.current_stream()
    res = {}
    for bits in bits_list:
        lay = hk.hack_kv_layout_make(d, H, bits, pi, cap)
        cache = hk.KVCache(lay, B, B, None, dev)
        lens = torch.full((B,), L0, dtype=torch.int32, device=dev)
        lens2 = torch.zeros_like(lens)
        ws = hk.decode_workspace(lay, B, Hq, cap)
        out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)
        calls = [hk.bind_decode_step(lay, cache, knew[i], vnew[i], qs[i], *((lens, lens2) if i % 2 == 0 else (lens2, lens)),
                                     cap - 1, hk.TAIL_FP16, out, ws) for i in range(nsteps)]
        sb = lay.sum_bytes

        def step_bytes_at(i):
            dec = B * H * decode_bytes_per_seq_head(L0 + i + 1, d, bits, pi, sb) + B * Hq * d * 6
            return dec + append_bytes(B, H, d, bits, pi, sb, (L0 + i + 1) % pi)

        # pass 0 warms the kernels up; both passes start from the same quantized prefix
        for timed_pass in (False, True):
            lens.fill_(L0)
            hk.hack_quantize(lay, cache, k0, v0, lens, L0)
            step_bytes, ms, kern_ms = run_steps(lambda i: calls[i](stream), step_bytes_at, 0, nsteps, stream)
        res[f"b{bits}"] = {"kv_bits": bits, "steps": nsteps, "tail_mode": "fp16", "ms_per_step": round(ms, 5),
                           "GBs": round(step_bytes / (ms * 1e-3) / 1e9, 2),
                           "roofline": roofline_hbm("decode_kernel (hack_decode_step)", step_bytes, kern_ms,
                                                    "kernels_decode.hip", f"decode_long_l131072_b{bits}_hbm_counters.txt")}
        del cache, ws
    return res


def bench_tiny(steps: int = 200, warmup: int = 20):
    """One decode call of batch 1, one q / kv head, 256 tokens: launch-latency sized."""
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    dev = torch.device("cuda:0")
    wl = synth.WORKLOADS["decode_tiny_l256"]
    B, Hq, H, d, pi, L, R = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.partition, wl.context, 64
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
    stream = torch.cuda.current_stream()
    nbytes = B * H * decode_bytes_per_seq_head(L, d, wl.kv_bits, pi, lay.sum_bytes) + B * Hq * d * 6
    _, ms, kern_ms = run_steps(lambda i: calls[i % R](stream), lambda i: nbytes, warmup, steps, stream)
    return {"workload": "decode_tiny_l256", "us_per_call": round(kern_ms * 1e3, 2), "bytes_per_call": int(nbytes),
            "note": "back-to-back calls; launch-latency bound, a fraction of HBM peak is not meaningful"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the decode path shards by "
              f"(sequence, kv head) with no communication, so N GPUs run N independent copies.",
              file=sys.stderr)
        sys.exit(2)
    # the oracle baseline forks worker processes: before anything initialises the GPU
    cpu = None
    if not args.no_cpu_baseline and args.only in (None, "cpu"):
        cpu = cpu_baseline_decode()
        print(f"[bench] oracle baseline: {cpu.get('value')} GB/s on {cpu.get('cores')} cores", file=sys.stderr, flush=True)
        if args.only == "cpu":
            print(json.dumps({"cpu_baseline": cpu}), flush=True)
            return
    if args.only == "copy":
        copy_calibration()
        return
    if args.workload == "sweep_prefill_partition":
        # the causal prefill workload's shapes for each code width and partition
        for bits in (4, 2):
            for part in (32, 64, 128):
                res = bench_prefill(max(3, args.prefill_iters // 2), 8, 0, bits, part)
                print(json.dumps({"workload": "sweep_prefill_partition", "kv_bits": bits, "partition": part,
                                  "attend_ms": res.get("attend_ms"), "TOPS": res.get("roofline", {}).get("achieved"),
                                  "frac_of_5POPS": res.get("roofline", {}).get("frac")}), flush=True)
        return
    if args.workload is not None:
        bench_workload(args.workload, args.steps, args.warmup)
        return
    if args.only == "prefill":
        print(json.dumps({"prefill": bench_prefill(args.prefill_iters)}), flush=True)
        return
    if args.only == "project":
        print(json.dumps({"prefill_from_embeddings": bench_prefill_embeddings(args.prefill_iters)}), flush=True)
        return
    if args.only == "llama8b":
        r, q = bench_llama8b(args.steps, args.warmup, args.replicas)
        print(json.dumps({"decode_llama8b_l4096": r, "quantize": q}), flush=True)
        return
    if args.only == "long":
        print(json.dumps({"decode_long_l131072": bench_long()}), flush=True)
        return
    if args.only == "tiny":
        print(json.dumps({"decode_tiny_l256": bench_tiny(args.steps, args.warmup)}), flush=True)
        return
    import torch
    torch.cuda.set_device(torch.device("cuda:0"))

    def progress(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    step_bytes, ms_per_step, cfg, roof = bench_ragged(args.steps, args.warmup)
    progress(f"decode_70b_ragged: {ms_per_step:.4f} ms per step")
    result = {
        "metric": "decode: compressed-KV GB/s (append + attend per step)",
        "value": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 2),
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
        "config": cfg,
        "roofline": roof,
    }
    if args.only is None:
        result["decode_llama8b_l4096"], result["quantize"] = bench_llama8b(args.steps, args.warmup, args.replicas)
        progress("decode_llama8b_l4096 done")
        result["decode_long_l131072"] = bench_long()
        progress("decode_long_l131072 done")
        result["decode_tiny_l256"] = bench_tiny()
        result["box_copy_GBs"] = round(copy_bandwidth(), 1)
        if not args.no_prefill:
            result["prefill"] = bench_prefill(args.prefill_iters)
            # the same workload with 4-bit Q/P codes (the literal reading of its 4-bit Q/K/V/P)
            result["prefill_qp4"] = bench_prefill(max(3, args.prefill_iters // 2), 4)
            # the paper's rounding: stochastic K/V, Q and P codes
            result["prefill_stochastic"] = bench_prefill(max(3, args.prefill_iters // 2), 8, 1)
            result["prefill_from_embeddings"] = bench_prefill_embeddings(max(3, args.prefill_iters // 2))
            progress("prefill done")
        if cpu is not None:
            result["cpu_baseline"] = cpu
    print(json.dumps(result), flush=True)


def bench_prefill(iters: int, qp_bits: int = 8, rounding: int = 0, kv_bits: int = 0, partition: int = 0):
    """Causal prefill (batch 1, 32/8 heads, 8192 tokens, 4-bit K/V, partition 64, Q/P
    codes of qp_bits bits; kv_bits / partition override the code width and partition):
    quantize-on-write of the prompt's K/V then attention; int8 ops of the causal
    triangle = 2 products x 32 heads x L(L+1)/2 x 128 x 2."""
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    wl = synth.WORKLOADS["prefill_l8192"]
    B, Hq, H, d, L = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.context
    dev = torch.device("cuda:0")
    kvb, part = kv_bits or wl.kv_bits, partition or wl.partition
    lay = hk.hack_kv_layout_make(d, H, kvb, part, L, qp_bits, rounding, wl.seed)
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
    stream = torch.cuda.current_stream()
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    qt, at = [], []
    for _ in range(iters):
        e0.record(stream)
        hk.hack_quantize(lay, c, k, v, ln, L)
        e1.record(stream)
        hk.hack_attend_prefill(lay, c, q, True, out)
        e2.record(stream)
        torch.cuda.synchronize()
        qt.append(e0.elapsed_time(e1))
        at.append(e1.elapsed_time(e2))
    a_ms = float(np.median(at))
    q_ms = float(np.median(qt))
    tops = ops / (a_ms * 1e-3) / 1e12
    q_gbs = quantize_bytes(B, H, L, d, kvb, part, lay.sum_bytes) / (q_ms * 1e-3) / 1e9
    return {"workload": "prefill_l8192", "qp_bits": qp_bits, "rounding": "stochastic" if rounding else "nearest",
            "int8_ops": ops, "attend_ms": round(a_ms, 4),
            "quantize_ms": round(q_ms, 4), "quantize_GBs": round(q_gbs, 1),
            "roofline": {"bound": "mfma", "kernel": "prefill_kernel", "achieved": round(tops, 2),
                         "peak": INT8_PEAK_TOPS, "unit": "TOPS (int8)", "frac": round(tops / INT8_PEAK_TOPS, 4),
                         "traffic": None}}


def bench_prefill_embeddings(iters: int):
    """The prefill from embeddings at the prefill workload's shapes with a
    Llama-3-8B-sized hidden dimension (batch 1, 8192 tokens, 32/8 heads, hidden 4096,
    4-bit K/V, partition 64): the fused QKV projection + quantize-on-write kernel, then
    the attention.  The projection's work is 2 x tokens x hidden x (H_q + 2 H_kv) x 128
    fp16 operations on the matrix cores."""
    import torch
    from paper_2502_03589_amd import hack as hk
    from paper_2502_03589_amd import synth
    wl = synth.WORKLOADS["prefill_l8192"]
    B, Hq, H, d, L, hidden = wl.batch, wl.q_heads, wl.kv_heads, wl.head_dim, wl.context, 4096
    N = (Hq + 2 * H) * d
    dev = torch.device("cuda:0")
    lay = hk.hack_kv_layout_make(d, H, wl.kv_bits, wl.partition, L, 8, 0, wl.seed)
    c = hk.KVCache(lay, B, B, None, dev)
    e = torch.from_numpy(synth.normal_f16(wl.seed, "misc", (B, L, hidden), sub=1)).to(dev)
    w = torch.from_numpy((synth.normal_f16(wl.seed, "misc", (N, hidden), sub=2).astype(np.float32)
                          / np.sqrt(hidden)).astype(np.float16)).to(dev)
    q = torch.empty((B, Hq, L, d), dtype=torch.float16, device=dev)
    out = torch.empty((B, Hq, L, d), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    hk.hack_prefill_from_embeddings(lay, c, e, w, Hq, True, q, out)
    torch.cuda.synchronize()
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    pt, at = [], []
    for _ in range(iters):
        e0.record(stream)
        hk.hack_project_qkv(lay, c, e, w, Hq, q)
        e1.record(stream)
        hk.hack_attend_prefill(lay, c, q, True, out)
        e2.record(stream)
        torch.cuda.synchronize()
        pt.append(e0.elapsed_time(e1))
        at.append(e1.elapsed_time(e2))
    p_ms, a_ms = float(np.median(pt)), float(np.median(at))
    flops = 2 * B * L * hidden * N
    tf = flops / (p_ms * 1e-3) / 1e12
    return {"workload": "prefill_l8192 from embeddings (hidden 4096)", "project_ms": round(p_ms, 4),
            "attend_ms": round(a_ms, 4), "total_ms": round(p_ms + a_ms, 4), "project_flops": flops,
            "roofline": {"bound": "mfma", "kernel": "project_kernel (QKV GEMM + quantize-on-write)",
                         "achieved": round(tf, 2), "peak": 2500.0, "unit": "TFLOP/s (fp16)",
                         "frac": round(tf / 2500.0, 4),
                         "traffic": profiled_traffic("kernels_project.hip", "project_l8192_h4096_hbm_counters.txt")}}


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
