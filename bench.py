#!/usr/bin/env python3
"""Benchmark of the sparse causal attention hot path on one MI355X.

One step = the whole hot path over the WAN-14B-shaped 480p chunk: append the
current chunk's K/V to the cache (c_0 and the previous chunk already cached),
then one sparse causal attention call of its 4680 queries over
1560 + 4680 + 4680 keys, 40 heads of width 128, bf16. Inputs are seeded
synthetic tensors of the latent shapes, resident in HBM before timing starts.

Prints ONE JSON line: throughput in TFLOP/s counting only unmasked
(query, key) pairs (4 * head_dim FLOPs each), the attention kernel's roofline
fraction against the bf16 dense MFMA peak (timed live with HIP events on the
launch stream), append and fused-producer bandwidth, ms per streamed chunk
(2 denoising steps x 40 layers of append + attention, measured on the
streaming loop), and the CPU oracle timed on a bounded sample of the same
workload.

Timing order: about 0.3 s of untimed attention launches (the GPU reaches its
steady clock), the attention kernel back to back, W warmup steps and K timed
steps, the append and the producer back to back, a cold launch after a cache
flush, the other workloads, the streaming loop and the CPU oracle.

    python bench.py [--gpus 1] [--steps 20] [--warmup 10]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X published dense bf16 MFMA peak
PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E
METRIC = "sparse-causal attn TFLOP/s (unmasked) & % bf16 MFMA peak; ms per chunk"

TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "attn_traffic.json")
ATTN_SOURCE = os.path.join(ROOT, "paper_2506_03099_amd", "csrc", "attn_fwd.hip")


def measured_traffic():
    """HBM bytes per attention launch (FETCH_SIZE + WRITE_SIZE from rocprofv3
    --pmc, scaled by the same counters read on a plain copy of known size), or
    None when the kernel source has changed since the counters were taken."""
    import hashlib
    try:
        with open(TRAFFIC_RECORD) as f:
            rec = json.load(f)
        with open(ATTN_SOURCE, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
    except OSError:
        return None
    return rec["bytes_per_launch"] if rec.get("kernel_source_sha256") == sha else None


def device_peak_tflops(torch):
    """Dense bf16 MFMA peak derived from the device: compute units x peak
    shader clock x 4096 bf16 FLOP per CU per clock (one 32x32x16 bf16 MFMA,
    32768 FLOP, per SIMD every 32 clocks, 4 SIMDs per CU); the roofline uses
    the published 2.5 PFLOP/s."""
    p = torch.cuda.get_device_properties(0)
    cus = getattr(p, "multi_processor_count", 0)
    try:  # peak clock in kHz from the HIP runtime
        import ctypes
        hip = ctypes.CDLL("libamdhip64.so")
        khz = ctypes.c_int(0)
        attr = 5  # hipDeviceAttributeClockRate, the sixth entry of hipDeviceAttribute_t
        if hip.hipDeviceGetAttribute(ctypes.byref(khz), attr, 0) != 0 or khz.value <= 0:
            return None
    except OSError:
        return None
    return {"cus": cus, "peak_clock_mhz": round(khz.value / 1e3, 1),
            "tflops": round(cus * khz.value * 1e3 * 4096 / 1e12, 1)}


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--stream-chunks", type=int, default=10,
                   help="chunks of the streaming loop measured for ms per chunk (0 = skip)")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="time budget of the CPU oracle sample (0 = skip)")
    p.add_argument("--other-workloads", type=int, default=1,
                   help="also time the 480p full sequence and the 720p two-stream chunk (0 = skip)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run one plain 512 MiB device copy (for counter calibration)")
    return p.parse_args()


def workload_desc(tm, w):
    return tm.make_desc(w.batch, w.heads, w.head_dim, w.tokens_per_frame, w.chunk_frames,
                        w.ref_frames, w.window, w.dtype)


def upload(torch, d):
    def dev(name):
        bits = np.ascontiguousarray(d[name + "_bits"]).view(np.int16)
        return torch.from_numpy(bits).view(torch.bfloat16).cuda()
    return dev("q"), dev("k"), dev("v")


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the hot path here is the single-GPU kernel "
              f"(it would shard by head across GPUs; no multi-GPU path is implemented); "
              f"--gpus {args.gpus} is not supported.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2506_03099_amd import tm
    from synth import WORKLOADS, draw_chunk

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    tm.lib()  # fails loudly if libtm.so is missing
    stream = torch.cuda.current_stream()

    # ---------------------------------------------------------------- 480p chunk step
    w = WORKLOADS["wan14b_480p_chunk"]
    desc = workload_desc(tm, w)
    cache = tm.KVCache(desc)
    chunks = [draw_chunk(w, t) for t in range(w.n_chunks + 1)]
    dev = [upload(torch, c) for c in chunks]
    for t in range(w.n_chunks):
        tm.tm_kv_append(cache, t, dev[t][1], dev[t][2])
    cur = w.n_chunks
    q, k, v = dev[cur]
    o = torch.empty_like(q)
    tm.tm_kv_append(cache, cur, k, v)
    pairs = tm.tm_allowed_pairs(desc, cur, cache)
    flops = 4.0 * w.head_dim * w.heads * w.batch * pairs
    append_bytes = 4.0 * q.shape[1] * w.heads * w.head_dim * w.batch * 2

    def step():
        tm.tm_kv_append(cache, cur, k, v)
        tm.tm_sparse_causal_attn_fwd(desc, q, cur, cache=cache, o=o)

    if args.copy_calibration:
        a = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # settle: the first tens of milliseconds of work after set-up run below the
    # GPU's steady clock, so about 0.3 s of untimed attention launches precede
    # every measurement
    for _ in range(300):
        tm.tm_sparse_causal_attn_fwd(desc, q, cur, cache=cache, o=o)
    torch.cuda.synchronize()

    # per-kernel average durations: each kernel launched back to back on the
    # same stream, bracketed by one pair of HIP events
    def timed(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(args.steps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / args.steps

    attn_ms = timed(lambda: tm.tm_sparse_causal_attn_fwd(desc, q, cur, cache=cache, o=o))

    # the step: W untimed warmup steps, then K timed steps
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / args.steps

    # the append and the fused producer, each back to back; after the step,
    # since a burst of HBM-bound launches lowers the clock of the MFMA-bound
    # launches that follow it for some milliseconds
    append_ms = timed(lambda: tm.tm_kv_append(cache, cur, k, v))
    # the fused producer on the same chunk: RMS-normalised q into q_out, the
    # normalised k and v into the cache (one pass over q, k, v; gains given)
    q_out = torch.empty_like(q)
    gain_q = torch.ones(w.heads, w.head_dim, dtype=torch.float32, device="cuda")
    gain_k = torch.ones_like(gain_q)
    producer_ms = timed(lambda: tm.tm_qkv_produce(cache, cur, q, k, v, q_gain=gain_q, k_gain=gain_k,
                                                  eps=1e-6, q_out=q_out))
    producer_bytes = 1.5 * append_bytes  # q, k, v read and q_out, K, V written once
    tm.tm_kv_append(cache, cur, k, v)  # the bench's keys stay the workload's as drawn

    value = flops / (ms_per_step * 1e-3) / 1e12
    attn_tflops = flops / (attn_ms * 1e-3) / 1e12
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) q/k/v, q and k RMS-normalised per token and head, "
                "rounded to bf16)",
        "config": {
            "workload": w.name,
            "batch": w.batch, "heads": w.heads, "head_dim": w.head_dim,
            "tokens_per_frame": w.tokens_per_frame, "chunk_frames": w.chunk_frames,
            "ref_frames": w.ref_frames, "window": w.window,
            "q_tokens": int(q.shape[1]), "kv_tokens": int(pairs // q.shape[1]),
            "step": "kv append of the current chunk + one attention call",
        },
        "pct_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "peak_bf16_device_tflops": device_peak_tflops(torch),
        "unmasked_tflop_per_step": round(flops / 1e12, 4),
        "attn_ms": round(attn_ms, 4),
        "attn_tflops": round(attn_tflops, 2),
        "append_us": round(append_ms * 1e3, 2),
        "append_gbps": round(append_bytes / (append_ms * 1e-3) / 1e9, 1),
        "producer_us": round(producer_ms * 1e3, 2),
        "producer_gbps": round(producer_bytes / (producer_ms * 1e-3) / 1e9, 1),
        "producer_frac_hbm": round(producer_bytes / (producer_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "timing": "warm: the chunk's K/V (224 MB) fit the 256 MB Infinity Cache",
        "roofline": {
            "kernel": "attn_fwd_bf16_kernel<128, true>",
            "bound": "mfma",
            "achieved": round(attn_tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic(),
        },
    }
    # cold: the attention launch after 1 GiB has been written, which evicts the
    # chunk's K/V from the Infinity Cache and the L2s
    flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    cold = []
    for _ in range(5):
        flush.fill_(1)
        a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a_.record(stream)
        tm.tm_sparse_causal_attn_fwd(desc, q, cur, cache=cache, o=o)
        b_.record(stream)
        torch.cuda.synchronize()
        cold.append(a_.elapsed_time(b_))
    del flush
    result["attn_cold_ms"] = round(float(np.median(cold)), 4)
    result["attn_cold_tflops"] = round(flops / (np.median(cold) * 1e-3) / 1e12, 2)
    del cache, dev, chunks
    torch.cuda.empty_cache()

    # ---------------------------------------------------------------- audio cross-attention
    result["audio_cross_attn"] = audio_cross_attn(torch, tm, stream, args.steps)

    # ---------------------------------------------------------------- other workloads
    if args.other_workloads:
        result["other_workloads"] = other_workloads(torch, tm, WORKLOADS, stream)

    # ---------------------------------------------------------------- streaming loop
    if args.stream_chunks > 0:
        result["ms_per_chunk"] = stream_loop(torch, tm, WORKLOADS["wan14b_480p_stream"],
                                             args.stream_chunks, stream)

    # ---------------------------------------------------------------- CPU oracle
    if args.cpu_seconds > 0:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
        result["cpu_baselines"] = cpu_baselines_other(WORKLOADS, result["cpu_baseline"])

    print(json.dumps(result), flush=True)


def audio_cross_attn(torch, tm, stream, steps):
    """The audio cross-attention of the 480p chunk (frames 4..6 of 21, one
    face of 14% of the tokens, 32 audio tokens per latent frame, five-frame
    window), launched back to back. HBM-bound: algorithmic bytes are every
    output row written, the queries of face rows read, the face ids and the
    audio keys and values of the chunk's windows read once."""
    from synth import AUDIO_WORKLOADS, draw_audio
    w = AUDIO_WORKLOADS["wan14b_480p_audio_chunk"]
    d = draw_audio(w)

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()

    q, ak, av = dev(d["q_bits"]), dev(d["ak_bits"]), dev(d["av_bits"])
    face = torch.from_numpy(d["face"]).cuda()
    o = torch.empty_like(q)
    desc = tm.make_audio_desc(w.batch, w.heads, w.head_dim, w.tokens_per_frame, w.audio_per_frame,
                              w.audio_frames, w.streams, w.half_window)
    call = lambda: tm.tm_audio_cross_attn_fwd(desc, q, w.first_frame, ak, av, face, o=o)
    # a launch takes about 20 us: 200 untimed launches bring the GPU to its
    # steady clock after the previous phase, and the figure averages 5 x 20
    for _ in range(200):
        call()
    torch.cuda.synchronize()
    reps = 5 * steps
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(reps):
        call()
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    row = w.heads * w.head_dim * 2
    face_rows = int((d["face"] >= 0).sum())
    lo = max(0, w.first_frame - w.half_window)
    hi = min(w.audio_frames - 1, w.first_frame + w.n_frames - 1 + w.half_window)
    audio_tok = (hi - lo + 1) * w.audio_per_frame * w.streams * w.batch
    nbytes = w.batch * w.n_tok * row + face_rows * row + d["face"].nbytes + 2 * audio_tok * row
    keys = [(min(w.audio_frames - 1, f + w.half_window) - max(0, f - w.half_window) + 1)
            * w.audio_per_frame for f in range(w.first_frame, w.first_frame + w.n_frames)]
    per_frame = d["face"][0].reshape(w.n_frames, -1) >= 0
    flop = sum(4.0 * w.head_dim * w.heads * int(per_frame[i].sum()) * keys[i]
               for i in range(w.n_frames)) * w.batch
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"workload": w.name, "kernel": "audio_attn_bf16_kernel<128>", "bound": "hbm",
            "us": round(ms * 1e3, 2), "algorithmic_mb": round(nbytes / 1e6, 2),
            "gbps": round(gbps, 1), "frac_hbm": round(gbps / PEAK_HBM_GBPS, 4),
            "face_fraction": round(face_rows / (w.batch * w.n_tok), 4),
            "keys_per_face_row": keys, "tflops": round(flop / (ms * 1e-3) / 1e12, 2)}


def timing_inputs(torch, shape, seed):
    """Seeded synthetic q, k, v of the given [B, L, H, D] shape drawn on the
    GPU (the same distribution as the parity inputs: N(0,1), q and k
    RMS-normalised per token and head, rounded to bf16); for timing only."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    out = []
    for i in range(3):
        x = torch.randn(shape, generator=g, device="cuda", dtype=torch.float32)
        if i < 2:
            x = x / x.pow(2).mean(-1, keepdim=True).sqrt()
        out.append(x.to(torch.bfloat16))
        del x
    return out


def other_workloads(torch, tm, workloads, stream, reps=10):
    """Attention TFLOP/s (unmasked pairs) of the 480p full sequence (21 latent
    frames, one call over all 32760 queries) and of its backward, of the 720p
    chunk with two streams and of the 512x512 chunk (attention over a cache of
    c_0 and the previous chunk)."""
    def time_call(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    out = {}
    w = workloads["wan14b_480p_full_sequence"]
    desc = workload_desc(tm, w)
    L = w.n_frames * w.tokens_per_frame
    q, k, v = timing_inputs(torch, (w.batch, L, w.heads, w.head_dim), 3)
    o = torch.empty_like(q)
    pairs = tm.tm_allowed_pairs(desc, -1, None, w.n_frames)
    flops = 4.0 * w.head_dim * w.heads * w.batch * pairs
    ms = time_call(lambda: tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v,
                                                        n_frames=w.n_frames, o=o))
    out[w.name] = {"queries": L, "keys": L, "allowed_pairs_per_head": int(pairs),
                   "density": round(pairs / float(L * L), 4), "ms": round(ms, 4),
                   "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
                   "dense_equivalent_tflops": round(4.0 * w.head_dim * w.heads * L * L /
                                                    (ms * 1e-3) / 1e12, 2)}
    # the backward of the same call (training): delta, dQ and dK/dV kernels;
    # 10 * head_dim FLOPs per allowed pair (S recomputed, dP, dV, dQ, dK)
    lse = torch.empty(w.batch, w.heads, L, dtype=torch.float32, device="cuda")
    tm.tm_sparse_causal_attn_fwd(desc, q, -1, k=k, v=v, n_frames=w.n_frames, o=o, lse=lse)
    dout = timing_inputs(torch, (w.batch, L, w.heads, w.head_dim), 4)[2]
    delta = torch.empty_like(lse)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ms_b = time_call(lambda: tm.tm_sparse_causal_attn_bwd(desc, w.n_frames, q, k, v, o, lse, dout,
                                                          delta=delta, dq=dq, dk=dk, dv=dv))
    out[w.name + "_backward"] = {"ms": round(ms_b, 4),
                                 "tflops": round(2.5 * flops / (ms_b * 1e-3) / 1e12, 2),
                                 "pct_bf16_peak": round(100 * 2.5 * flops / (ms_b * 1e-3) / 1e12 /
                                                        PEAK_BF16_TFLOPS, 2),
                                 "flop_count": "10 * head_dim per allowed pair"}
    del q, k, v, o, lse, dout, delta, dq, dk, dv
    torch.cuda.empty_cache()

    # chunks over a cache of c_0 and the previous chunk: the 720p chunk with two
    # streams, and the paper's deployed 512x512 resolution (1024 tokens/frame)
    for i, name in enumerate(("wan14b_720p_chunk_b2", "paper_512_chunk")):
        w = workloads[name]
        desc = workload_desc(tm, w)
        cache = tm.KVCache(desc)
        shape = lambda n: (w.batch, n, w.heads, w.head_dim)
        ref = timing_inputs(torch, shape(w.ref_frames * w.tokens_per_frame), 50 + 3 * i)
        prev = timing_inputs(torch, shape(w.chunk_frames * w.tokens_per_frame), 51 + 3 * i)
        q, k, v = timing_inputs(torch, shape(w.chunk_frames * w.tokens_per_frame), 52 + 3 * i)
        tm.tm_kv_append(cache, 0, ref[1], ref[2])
        tm.tm_kv_append(cache, 1, prev[1], prev[2])
        tm.tm_kv_append(cache, 2, k, v)
        o = torch.empty_like(q)
        pairs = tm.tm_allowed_pairs(desc, 2, cache)
        flops = 4.0 * w.head_dim * w.heads * w.batch * pairs
        ms = time_call(lambda: tm.tm_sparse_causal_attn_fwd(desc, q, 2, cache=cache, o=o))
        out[w.name] = {"batch": w.batch, "queries": int(q.shape[1]),
                       "keys": int(pairs // q.shape[1]), "ms": round(ms, 4),
                       "tflops": round(flops / (ms * 1e-3) / 1e12, 2)}
        del cache, ref, prev, q, k, v, o
        torch.cuda.empty_cache()
    return out


def stream_loop(torch, tm, w, n_chunks, stream):
    """Chunks 1..n of the streaming loop: per chunk, for each of 2 denoising
    steps and 40 layers, append the chunk's K/V to that (step, layer)'s cache
    and run its attention. Inputs cycle through a pool of 4 seeded chunks."""
    from synth import draw_chunk
    desc = workload_desc(tm, w)
    caches = [[tm.KVCache(desc) for _ in range(w.layers)] for _ in range(w.steps)]
    pool = [upload(torch, draw_chunk(w, 1 + i)) for i in range(4)]
    ref = upload(torch, draw_chunk(w, 0))
    o = torch.empty_like(pool[0][0])
    for s in range(w.steps):
        for l in range(w.layers):
            tm.tm_kv_append(caches[s][l], 0, ref[1], ref[2])
    torch.cuda.synchronize()
    events = [torch.cuda.Event(enable_timing=True) for _ in range(n_chunks + 1)]
    total_flops = 0.0
    events[0].record(stream)
    i = 0
    for t in range(1, n_chunks + 1):
        for s in range(w.steps):
            for l in range(w.layers):
                q, k, v = pool[i % 4]
                i += 1
                tm.tm_kv_append(caches[s][l], t, k, v)
                tm.tm_sparse_causal_attn_fwd(desc, q, t, cache=caches[s][l], o=o)
        total_flops += 4.0 * w.head_dim * w.heads * w.steps * w.layers * \
            tm.tm_allowed_pairs(desc, t, caches[0][0])
        events[t].record(stream)
    torch.cuda.synchronize()
    per = [events[t - 1].elapsed_time(events[t]) for t in range(1, n_chunks + 1)]
    total_ms = sum(per)
    out = {
        "workload": w.name,
        "calls_per_chunk": w.steps * w.layers,
        "first_chunk_ms": round(per[0], 3),
        "steady_ms": round(float(np.mean(per[1:])) if len(per) > 1 else per[0], 3),
        "chunks": n_chunks,
        "tflops": round(total_flops / (total_ms * 1e-3) / 1e12, 2),
    }
    del caches, pool, ref
    torch.cuda.empty_cache()
    return out


def cpu_baseline(w, budget_s):
    """The oracle, untouched, on whole heads of the same 480p chunk until the
    time budget is spent; scaled to TFLOP/s of unmasked pairs."""
    from oracle import ChunkGeometry, StreamHistory
    from synth import draw_chunk
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # threadpoolctl missing: report the core count
        threads = os.cpu_count()
    g = ChunkGeometry(w.tokens_per_frame, w.chunk_frames, w.ref_frames, w.window)
    hist = StreamHistory(g)
    chunks = [draw_chunk(w, t) for t in range(w.n_chunks + 1)]
    for t, c in enumerate(chunks):
        hist.append(t, c["k"], c["v"])
    q = chunks[-1]["q"]
    n_keys = sum(c["k"].shape[1] for c in chunks)
    heads = 0
    t0 = time.perf_counter()
    while heads < w.heads and (heads == 0 or time.perf_counter() - t0 < budget_s):
        hist.attend(q, w.n_chunks, heads=[heads])
        heads += 1
    dt = time.perf_counter() - t0
    flops = 4.0 * w.head_dim * heads * q.shape[1] * n_keys
    return {
        "value": round(flops / dt / 1e12, 5),
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"{heads} of {w.heads} heads of the 480p chunk ({q.shape[1]} queries x "
                  f"{n_keys} keys each), fp32 numpy, {dt:.1f} s",
        "host_cpus": os.cpu_count(),
        "note": "BLAS matmuls use all threads; numpy exp/where/max are single-threaded",
    }


def cpu_baselines_other(workloads, cfg2):
    """The oracle on the other workloads, on the host's cores: the tiny fp32
    workload in full; one head of the 480p full sequence (complete masked rows
    in blocks of 2048) and one (stream, head) of the 720p chunk, each
    extrapolated to all heads and streams (heads and streams are independent
    problems of the same shape); the streaming loop's steady chunk as 80 calls
    of the 480p chunk (from the timed cfg2 figure). Every extrapolation is
    labelled."""
    from oracle import ChunkGeometry, StreamHistory, full_sequence_attention
    from synth import draw_chunk, draw_qkv_sequence
    from synth.inputs import Workload
    out = {}

    def geom(w):
        return ChunkGeometry(w.tokens_per_frame, w.chunk_frames, w.ref_frames, w.window)

    # tiny fp32: 4 streamed chunks and the 9-frame sequence, all heads
    w = workloads["tiny_f32"]
    hist = StreamHistory(geom(w))
    chunks = [draw_chunk(w, t) for t in range(w.n_chunks + 1)]
    pairs = 0
    t0 = time.perf_counter()
    for t, c in enumerate(chunks):
        hist.append(t, c["k"], c["v"])
        hist.attend(c["q"], t)
    q = np.concatenate([c["q"] for c in chunks], axis=1)
    k = np.concatenate([c["k"] for c in chunks], axis=1)
    v = np.concatenate([c["v"] for c in chunks], axis=1)
    full_sequence_attention(q, k, v, geom(w))
    dt = time.perf_counter() - t0
    from oracle import allowed_pair_count
    L = w.n_frames * w.tokens_per_frame

    def stream_keys(t):  # c_0, then chunks max(1, t - W) .. t
        return chunks[0]["k"].shape[1] + sum(c["k"].shape[1] for c in chunks[max(1, t - w.window):t + 1])

    pairs = allowed_pair_count(L, geom(w)) + sum(c["q"].shape[1] * stream_keys(t)
                                                 for t, c in enumerate(chunks))
    out[w.name] = {"seconds": round(dt, 4), "kind": "oracle", "extrapolated": False,
                   "sample": "all: 4 streamed chunks + the 9-frame sequence, 2 heads",
                   "tflops": round(4.0 * w.head_dim * w.heads * pairs / dt / 1e12, 6)}

    # 480p full sequence: one head, extrapolated to 40
    w = workloads["wan14b_480p_full_sequence"]
    one = Workload(w.wid, w.name, w.dtype, w.batch, 1, w.head_dim, w.tokens_per_frame,
                   w.chunk_frames, w.ref_frames, w.window, n_frames=w.n_frames)
    d = draw_qkv_sequence(one)
    t0 = time.perf_counter()
    full_sequence_attention(d["q"], d["k"], d["v"], geom(w), row_block=2048)
    dt = time.perf_counter() - t0
    L = w.n_frames * w.tokens_per_frame
    pairs = allowed_pair_count(L, geom(w))
    out[w.name] = {"seconds_one_head": round(dt, 2), "kind": "oracle", "extrapolated": True,
                   "sample": f"1 of {w.heads} heads (32760 x 32760 masked rows in blocks of 2048); "
                             f"ms extrapolated x{w.heads}",
                   "ms_extrapolated": round(dt * w.heads * 1e3, 1),
                   "tflops": round(4.0 * w.head_dim * pairs / dt / 1e12, 5)}
    del d

    # 720p chunk: one (stream, head), extrapolated to 2 streams x 40 heads
    w = workloads["wan14b_720p_chunk_b2"]
    one = Workload(w.wid, w.name, w.dtype, 1, 1, w.head_dim, w.tokens_per_frame, w.chunk_frames,
                   w.ref_frames, w.window, n_chunks=w.n_chunks)
    hist = StreamHistory(geom(w))
    cs = [draw_chunk(one, t) for t in range(w.n_chunks + 1)]
    for t, c in enumerate(cs):
        hist.append(t, c["k"], c["v"])
    n_keys = sum(c["k"].shape[1] for c in cs)
    t0 = time.perf_counter()
    hist.attend(cs[-1]["q"], w.n_chunks)
    dt = time.perf_counter() - t0
    n_q = cs[-1]["q"].shape[1]
    out[w.name] = {"seconds_one_head": round(dt, 2), "kind": "oracle", "extrapolated": True,
                   "sample": f"1 of {w.batch * w.heads} (stream, head) pairs ({n_q} queries x "
                             f"{n_keys} keys); ms extrapolated x{w.batch * w.heads}",
                   "ms_extrapolated": round(dt * w.batch * w.heads * 1e3, 1),
                   "tflops": round(4.0 * w.head_dim * n_q * n_keys / dt / 1e12, 5)}

    # streaming loop: a steady chunk is 80 calls of the 480p chunk
    w = workloads["wan14b_480p_stream"]
    calls = w.steps * w.layers
    ms_call = 1.0466 / cfg2["value"]  # seconds per 480p-chunk call at the oracle's TFLOP/s
    out[w.name] = {"kind": "oracle", "extrapolated": True,
                   "sample": f"{calls} x the timed 480p-chunk oracle call (no separate run)",
                   "ms_per_steady_chunk_extrapolated": round(calls * ms_call * 1e3, 1)}
    return out


if __name__ == "__main__":
    main()
