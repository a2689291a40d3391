"""Benchmark: one decode step of TurboESM on the full ESM-2 650M cache shape.

Workload (default "esm2-650m-33layer-seq1024"): 33 layers x 20 heads x 64,
batch 1, 1024 cached tokens, fp16 I/O, synthetic seeded inputs. One step =
tq_decode_step over all 33 layers: append the new token (RoPE, rotation,
3-bit codes, QJL signs, packing) and attend over the 1025 cached tokens, in
one kernel launch (decode_kernel: each (layer, head) block reads its Pi
once, rotates the query, quantizes the new key and value, and attends).
Steps rotate over replicas of every per-step input (cache, Pi, query, new
token) totalling >= 1 GiB, so each step reads its data from HBM rather than
from the 256 MB Infinity Cache. The K timed steps are captured in one HIP
graph and replayed once between two synchronizations; HIP events on the
graph's stream give the average step duration for the roofline.

Besides the contract's keys ("value", "roofline", "cpu_baseline") the line
carries: the median, p10 and p90 step time over further replays of the
graph; the same step as 33 per-layer launches; a streaming read of the same
bytes (tq_read_probe) as the size's read ceiling; the ragged batch of 64
sequences and the ESM-2 3B shape ("configs": their own KV GB/s, roofline
fraction, steps/s and an oracle sample timed with all threads and one); the
GPU calibration time of the whole 650M model; the prefill, the
dequantize-then-attend path and plain fp16 attention for context.

Prints one JSON line.
    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline] [--no-extra]
    python bench.py --workload esm2-650m-ragged-b64     (one batched workload alone)
    python bench.py --only prefill|dequant|lengths --steps K     (eager launches, for counters)
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

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="esm2-650m-33layer-seq1024")
    ap.add_argument("--replica-bytes", type=float, default=1.1 * 2 ** 30)
    ap.add_argument("--replicas", type=int, default=0,
                    help="number of input replicas (default: enough for --replica-bytes)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-fp16-baseline", action="store_true",
                    help="skip the plain fp16 attention timing (PyTorch) printed for context")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--copy-probe", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--decode-only", action="store_true",
                    help="time K graph-captured decode launches only (for profiling)")
    ap.add_argument("--eager", action="store_true",
                    help="launch the K timed steps one by one instead of as one HIP graph "
                         "(for counter collection)")
    ap.add_argument("--only", choices=("prefill", "dequant", "lengths"), default=None,
                    help="run only K eager launches of the prefill quantizer or of the dequantize "
                         "baseline on the headline shape, or (lengths) of decode_attend and "
                         "decode_step over 1, 513 and 1025 tokens (for counter collection)")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the ragged-batch and ESM-2 3B decode lines")
    ap.add_argument("--replays", type=int, default=10,
                    help="graph replays of the K steps behind the median and p10/p90 step times")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(every (sequence, layer, head) unit is independent, so heads or sequences would shard across GPUs with no communication).",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2603_26110_amd as tq
    from paper_2603_26110_amd import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.copy_probe:
        # One elementwise kernel that reads n bytes and writes n bytes (int32
        # negation): the known traffic against which FETCH_SIZE and WRITE_SIZE
        # are scaled.
        n = args.copy_probe * 2 ** 20
        a = torch.ones(n // 4, dtype=torch.int32, device=dev)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        for _ in range(3):
            torch.neg(a, out=b)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n}))
        return

    wl = synth.WORKLOADS[args.workload]
    if wl.batch != 1 or wl.ragged is not None:
        # a batched workload on its own (the default line carries it as well)
        print(json.dumps(workload_line(torch, tq, synth, wl.name, args.replays, args.cpu_seconds,
                                       eager=args.eager, cpu=not args.no_cpu_baseline)))
        return
    L, H, T = wl.layers, wl.heads, wl.seq
    n_ctx = T + 1                     # tokens attended per step (prefill + the new one)
    slots = ((n_ctx + 63) // 64) * 64
    g = synth.rng(wl.seed)
    ch = synth.outlier_channels(g, L, H)
    io = torch.float16 if wl.io_dtype == "f16" else torch.float32
    k_all = synth.as_io(synth.keys(g, L, 1, n_ctx, H, ch), wl.io_dtype)
    v_all = synth.as_io(synth.values(g, L, 1, n_ctx, H), wl.io_dtype)
    q = synth.as_io(synth.queries(g, L, 1, H), wl.io_dtype)
    pi = synth.rotations(g, L, H)
    S = synth.qjl_matrix(g)
    lut = np.broadcast_to(synth.GAUSS_LEVELS_MAX1960, (L, H, 8)).copy()

    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    cs = tq.rope_table(slots + 64)
    params = tq.Params(L, H, cs, io_dtype=io, flags=tq.V_ROTATE)
    S_d, lut_d = t_(S), t_(lut)
    zero_i32, zero_i64 = t_(np.zeros(1, np.int32)), t_(np.zeros(1, np.int64))
    pos_new, slot_new = t_(np.array([T], np.int32)), t_(np.array([T], np.int64))
    qpos, slen = t_(np.array([n_ctx - 1], np.int32)), t_(np.array([n_ctx], np.int32))
    cached = t_(np.array([T], np.int32))           # tokens in the cache before a step

    # replica 0: prefill the cache with the first T tokens
    base_cache = tq.Cache(L, H, slots, device=dev)
    pi_d = t_(pi)
    tq.quantize_pack(params, base_cache, t_(k_all[:, :, :T]), t_(v_all[:, :, :T]), zero_i32, zero_i64,
                     pi_d, lut_d, lut_d, S_d)
    k_new, v_new = t_(k_all[:, :, T:T + 1]), t_(v_all[:, :, T:T + 1])
    q_d = t_(q)
    per_replica = (tq.cache_bytes(L, H, slots) + pi_d.numel() * 4 + 2 * q_d.numel() * q_d.element_size()
                   + 2 * k_new.numel() * k_new.element_size())
    R = args.replicas if args.replicas > 0 else max(2, math.ceil(args.replica_bytes / per_replica))
    reps = []
    for r in range(R):
        c = tq.Cache(L, H, slots, device=dev)
        c.k_codes.copy_(base_cache.k_codes)
        c.v_codes.copy_(base_cache.v_codes)
        c.scalars.copy_(base_cache.scalars)
        kr, vr = k_new.clone(), v_new.clone()
        reps.append(dict(cache=c, pi=pi_d.clone(), q=q_d.clone(), k=kr, v=vr, k1=kr[:, :, 0], v1=vr[:, :, 0],
                         out=torch.empty_like(q_d)))
    ws_bytes = tq.decode_workspace_bytes(params, 1, L, n_ctx)
    ws = torch.zeros(max(ws_bytes, 16), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    def append(r):
        d = reps[r]
        tq.quantize_pack(params, d["cache"], d["k"], d["v"], pos_new, slot_new, d["pi"], lut_d, lut_d, S_d)

    def attend(r):
        d = reps[r]
        tq.decode_attend(params, d["cache"], d["q"], qpos, zero_i64, slen, n_ctx, d["pi"], lut_d, lut_d,
                         S_d, out=d["out"], workspace=ws)

    def step(r):
        # append the token at position T (slot T) and attend over T + 1 tokens
        d = reps[r]
        tq.decode_step(params, d["cache"], d["q"], d["k1"], d["v1"], pos_new, zero_i64, cached, n_ctx,
                       d["pi"], lut_d, lut_d, S_d, out=d["out"], workspace=ws)

    def two_calls(r):
        append(r)
        attend(r)

    # warmup (eager), then check that a graph replay reproduces the eager output
    # and that the fused step gives what the two separate calls give
    for s in range(args.warmup):
        two_calls(s % R)
    torch.cuda.synchronize()
    two_call_out = reps[0]["out"].clone()
    for s in range(args.warmup):
        step(s % R)
    torch.cuda.synchronize()
    eager_out = reps[0]["out"].clone()
    assert torch.equal(eager_out, two_call_out), "decode_step differs from quantize_pack + decode_attend"

    K = args.steps
    if args.only:
        only_kernel(torch, tq, args.only, K, params, reps, base_cache, t_, k_all, v_all, T, n_ctx, L, H, slots,
                    pi_d, lut_d, S_d, zero_i32, zero_i64)
        return
    if args.eager:
        for s in range(K):
            (attend if args.decode_only else step)(s % R)
        torch.cuda.synchronize()
        print(json.dumps({"eager_steps": K, "decode_only": bool(args.decode_only)}))
        return
    stream = torch.cuda.Stream(device=dev)

    def capture(fn):
        g_ = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_, stream=stream):
            for s in range(K):
                fn(s % R)
        g_.replay()                                 # untimed warm replay
        torch.cuda.synchronize()
        return g_

    graph = capture(attend if args.decode_only else step)
    if not args.decode_only:
        assert torch.equal(reps[0]["out"], eager_out), "graph replay differs from eager decode"

    # timed region: exactly K steps; HIP events on the graph's stream give the
    # average step duration for the roofline
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        e0.record(stream)
        graph.replay()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / K
    step_ms = e0.elapsed_time(e1) / K
    # spread over further replays of the same graph (not the timed region)
    spread = replay_spread(torch, graph, stream, K, args.replays)

    # for comparison (not the headline): the same step as two calls, and the
    # attention call alone
    def graph_ms(fn):
        g_ = capture(fn)
        a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            a_.record(stream)
            g_.replay()
            b_.record(stream)
        torch.cuda.synchronize()
        return a_.elapsed_time(b_) / K

    two_call_ms = graph_ms(two_calls) if not args.decode_only else None
    # Context, not HBM: the same step without replica rotation, so the 60 MB
    # of one cache stay in the 256 MB Infinity Cache between steps (what a
    # serving loop over one resident cache of this size sees)
    warm_ms = graph_ms(lambda r: step(0)) if not args.decode_only else None
    attend_ms = graph_ms(attend) if not args.decode_only else step_ms

    units = L * H
    kv_bytes = units * n_ctx * 72
    pi_bytes = units * 64 * 64 * 4
    io_b = 2 if io == torch.float16 else 4
    # algorithmic bytes of one step: every cached token-head once (72 B), each
    # Pi once, S and the tables once, q, k, v in and out once, and the new
    # token-head written (72 B)
    alg_bytes = (kv_bytes + pi_bytes + 64 * 64 * 4 + units * 8 * 4 * 2 + units * 64 * io_b * 4
                 + units * 72)
    if args.decode_only:
        alg_bytes = kv_bytes + pi_bytes + 64 * 64 * 4 + units * 8 * 4 * 2 + units * 64 * io_b * 2
    achieved = alg_bytes / (step_ms * 1e-3) / 1e9
    value = kv_bytes / (ms_per_step * 1e-3) / 1e9
    traffic, traffic_src = (None, None) if args.decode_only else measured_traffic(wl.name)

    # prefill (not the headline): tq_quantize_pack of the T cached tokens of
    # every unit into a cache of its own, outside the timed region
    pf_cache = tq.Cache(L, H, slots, device=dev)
    k_pf, v_pf = t_(k_all[:, :, :T]), t_(v_all[:, :, :T])
    for _ in range(2):
        tq.quantize_pack(params, pf_cache, k_pf, v_pf, zero_i32, zero_i64, pi_d, lut_d, lut_d, S_d)
    pa, pb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    pa.record()
    for _ in range(5):
        tq.quantize_pack(params, pf_cache, k_pf, v_pf, zero_i32, zero_i64, pi_d, lut_d, lut_d, S_d)
    pb.record()
    torch.cuda.synchronize()
    pf_ms = pa.elapsed_time(pb) / 5
    pf_th = L * H * T
    pf_bytes = pf_th * (2 * 64 * io_b + 72)
    prefill = {"ms": round(pf_ms, 4), "token_heads": pf_th,
               "kernel": "quantize_tiles_kernel (rotations and S r on fp16 MFMA with hi/lo parts, quantizer steps on VALU)",
               "alg_bytes": pf_bytes, "gbs": round(pf_bytes / (pf_ms * 1e-3) / 1e9, 1),
               "rotation_tflops": round(2 * 2 * 64 * 64 * pf_th / (pf_ms * 1e-3) / 1e12, 2)}
    del pf_cache, k_pf, v_pf

    two_step = None
    if not args.decode_only and not args.no_fp16_baseline:
        attend(0)                                   # reps[0]["out"]: the fused output on replica 0
        torch.cuda.synchronize()
        two_step = two_step_baseline(torch, tq, params, reps, L, H, n_ctx, cs.view(-1, 32, 2),
                                     [d["pi"].view(L, H, 64, 64) for d in reps], lut_d, S_d, K, attend_ms)

    fp16_base = None if args.decode_only or args.no_fp16_baseline else fp16_attention_baseline(
        torch, L * H, n_ctx, args.replica_bytes, K)
    if fp16_base:
        fp16_base["decode_attend_speedup_vs_sdpa"] = round(fp16_base["sdpa_ms"] / attend_ms, 2)
        fp16_base["decode_step_speedup_vs_sdpa"] = round(fp16_base["sdpa_ms"] / step_ms, 2)

    per_layer = None
    if not args.decode_only:
        per_layer = per_layer_launches(torch, tq, params, reps, L, n_ctx, pos_new, zero_i64, cached, lut_d, S_d,
                                       K, stream, kv_bytes)
    probe = hbm_read_probe(torch, tq, alg_bytes, args.replica_bytes, K)
    probe["decode_step_frac_of_probe"] = round(achieved / probe["gbs"], 4)

    extra = {}
    if not args.decode_only and not args.no_extra:
        for name in ("esm2-650m-ragged-b64", "esm2-3b-36layer-b16-seq8192"):
            extra[name] = workload_line(torch, tq, synth, name, args.replays, args.cpu_seconds / 3,
                                        cpu=not args.no_cpu_baseline)
            torch.cuda.empty_cache()

    calibration = None
    if not args.decode_only:
        from paper_2603_26110_amd import quality
        calibration = quality.calibration_timing()
        calibration = {"heads": calibration["heads"], "calibration_vectors_per_head": calibration["ncal"],
                       "seconds": round(calibration["seconds"], 3),
                       "what": "head-wise SVD rotation and separate K and V tables of the 33 x 20 heads "
                               "of ESM-2 650M on the GPU (Sec. 3.2 quotes 2-5 min for its calibration)"}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(k_all, v_all, S, lut, pi, q, L, H, slots, n_ctx, args.cpu_seconds)

    line = {
        "metric": "fused 3-bit decode attention: KV GB/s (% HBM peak) and decode steps/s",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u4 codes, fp32 compute, fp16 I/O",
        "data": "synthetic (seeded; ESM-2-shaped keys with outlier channels, Student-t values)",
        "config": {"workload": wl.name, "layers": L, "heads": H, "head_dim": 64, "batch": 1,
                   "cached_tokens": n_ctx, "io": wl.io_dtype, "replicas": R,
                   "replica_bytes": int(R * per_replica)},
        "kv_pct_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "decode_steps_per_s": round(1e3 / ms_per_step, 1),
        "step_event_ms": round(step_ms, 5),
        "step_ms_median": spread["median"],
        "step_ms_p10": spread["p10"],
        "step_ms_p90": spread["p90"],
        "step_spread_replays": spread["replays"],
        "per_layer_launches": per_layer,
        "hbm_read_probe": probe,
        "two_call_step_ms": None if two_call_ms is None else round(two_call_ms, 5),
        "warm_infinity_cache_step_ms_not_hbm": None if warm_ms is None else round(warm_ms, 5),
        "decode_attend_ms": round(attend_ms, 5),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "traffic_source": traffic_src,
                     "kernel": ("decode_kernel<8, false> (one launch per tq_decode_attend call)"
                                if args.decode_only else
                                "decode_kernel<8, false> (one launch per tq_decode_step call)"),
                     "alg_bytes_per_launch": int(alg_bytes)},
        "cpu_baseline": cpu,
        "configs": extra or None,
        "calibration": calibration,
        "prefill_quantize": prefill,
        "two_step_baseline": two_step,
        "fp16_attention_baseline": fp16_base,
        "paper_context": {"memory_reduction": "7.1x (Table 4, fp32 baseline, 'CUDA')",
                          "kv_fetch_speedup": "1.96x Triton vs PyTorch fetch_unpacked, 143 tokens, "
                                              "NVIDIA GPU on Colab, model and precision unstated (Table 6)"},
    }
    print(json.dumps(line))


def replay_spread(torch, graph, stream, K, replays):
    """Per-step time of `replays` further replays of the K-step graph (HIP
    events on the graph's stream around each replay): median, p10, p90."""
    per = []
    for _ in range(max(1, replays)):
        a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            a_.record(stream)
            graph.replay()
            b_.record(stream)
        torch.cuda.synchronize()
        per.append(a_.elapsed_time(b_) / K)
    per = np.asarray(per)
    return {"median": round(float(np.median(per)), 5), "p10": round(float(np.percentile(per, 10)), 5),
            "p90": round(float(np.percentile(per, 90)), 5), "replays": len(per)}


def per_layer_launches(torch, tq, params, reps, L, n_ctx, pos_new, slot0, cached, lut_d, S_d, K, stream,
                       kv_bytes):
    """The same decode step as one tq_decode_step launch per layer (33 calls of
    20 units each, as a model that decodes layer by layer would make them),
    captured in one graph of K steps; each call's split-K workspace is
    preallocated and left zero by the kernel."""
    R = len(reps)
    p1 = params
    need = tq.decode_workspace_bytes(p1, 1, 1, n_ctx)
    ws = torch.zeros(max(need, 16), dtype=torch.uint8, device="cuda")

    def step(r):
        d = reps[r]
        for l in range(L):
            tq.decode_step(p1, d["cache"], d["q"][l:l + 1], d["k1"][l:l + 1], d["v1"][l:l + 1], pos_new, slot0,
                           cached, n_ctx, d["pi"], lut_d, lut_d, S_d, layer0=l, out=d["out"][l:l + 1], workspace=ws)

    for r in range(2):
        step(r % R)
    torch.cuda.synchronize()
    g_ = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_, stream=stream):
        for k in range(K):
            step(k % R)
    g_.replay()
    torch.cuda.synchronize()
    sp = replay_spread(torch, g_, stream, K, 5)
    del g_
    return {"launches_per_step": L, "units_per_launch": params.num_heads, "step_ms_median": sp["median"],
            "step_ms_p10": sp["p10"], "step_ms_p90": sp["p90"],
            "kv_gbs": round(kv_bytes / (sp["median"] * 1e-3) / 1e9, 1)}


def hbm_read_probe(torch, tq, nbytes, replica_bytes, K):
    """A plain streaming read of as many bytes as one decode step's algorithmic
    bytes, in the same run (the library's tq_read_probe: 16-byte loads, four
    in flight per thread), over rotating replicas so that every call reads
    HBM; the best of a few grid sizes. The ceiling a read of this size reaches
    on this GPU, next to which the fused step's rate is judged."""
    n = int(nbytes) // 16 * 16
    R = max(2, math.ceil(replica_bytes / n))
    bufs = [torch.ones(n // 4, dtype=torch.int32, device="cuda") for _ in range(R)]
    sink = torch.zeros(65536, dtype=torch.int32, device="cuda")
    out = {"bytes": n, "replicas": R, "calls": K}

    def timed(fn):
        for r in range(R):
            fn(bufs[r])
        torch.cuda.synchronize()
        best = None
        for rep in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for k in range(K):
                fn(bufs[k % R])
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / K
            best = ms if best is None else min(best, ms)
        return n / (best * 1e-3) / 1e9

    best = None
    for blocks in (512, 1024, 2048, 4096):
        gbs = timed(lambda x, b=blocks: tq.read_probe(x, b, sink))
        out[f"blocks_{blocks}_gbs"] = round(gbs, 1)
        if best is None or gbs > best[1]:
            best = (blocks, gbs)
    out["blocks"], out["gbs"] = best[0], round(best[1], 1)
    out["frac_of_peak"] = round(best[1] / HBM_PEAK_GBS, 4)
    del bufs
    torch.cuda.empty_cache()
    return out


def workload_line(torch, tq, synth, name, replays, cpu_seconds, eager=False, cpu=True):
    """Decode steps of a batched workload: the ragged batch of 64 ESM-2 650M
    sequences, or the ESM-2 3B shape (16 sequences of 8192 tokens, head-wise
    SVD rotations and calibrated tables). The cache is prefilled with
    tq_quantize_pack from keys and values drawn on the GPU; then K steps
    (each one tq_decode_step over every layer, sequence and head: append the
    sequence's next token and attend) are captured in one graph and replayed.
    The cache itself (1.7 GB and 13.7 GB) is far larger than the Infinity
    Cache, so no replicas are needed. Figures: KV GB/s and the roofline
    fraction of the step's algorithmic bytes, steps/s, and the oracle
    decoding a seeded sample of units from the GPU's cache bytes (timed with
    all threads and with one, and compared with the GPU's output)."""
    from oracle import oracle
    wl = synth.WORKLOADS[name]
    dev = torch.device("cuda:0")
    L, H, B = wl.layers, wl.heads, wl.batch
    K = wl.decode_steps if wl.decode_steps > 1 else 20
    g = synth.rng(wl.seed)
    ch = synth.outlier_channels(g, L, H)
    S = synth.qjl_matrix(g)
    lens = (synth.ragged_lengths(g, B, *wl.ragged) if wl.ragged else np.full(B, wl.seq, np.int64)).astype(np.int32)
    offs, slots = synth.tile_aligned_offsets(lens, extra=K)
    caps = np.diff(np.append(offs, slots))
    positions = int(lens.max()) + K + 64
    cs = tq.rope_table(positions)
    io = torch.float16
    t_ = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    S_d = t_(S)

    # rotations and tables
    t0 = time.perf_counter()
    if wl.rotation == "svd":
        pi_d = torch.empty((L, H, 64, 64), dtype=torch.float32, device=dev)
        lk_d = torch.empty((L, H, 8), dtype=torch.float32, device=dev)
        lv_d = torch.empty((L, H, 8), dtype=torch.float32, device=dev)
        for l in range(L):
            gen = synth.device_generator(wl.seed + 7919, l, dev)
            ck = synth.keys_on(gen, 1, wl.calib_vectors, H, ch[l], io, dev)[0].float()
            cv = synth.values_on(gen, 1, wl.calib_vectors, H, io, dev)[0].float()
            cpos = torch.randint(0, wl.seq, (wl.calib_vectors,), generator=gen, device=dev)
            c_, s_ = cs[cpos, :, 0].unsqueeze(1), cs[cpos, :, 1].unsqueeze(1)
            a_, b_ = ck[..., 0::2], ck[..., 1::2]
            kr = torch.empty_like(ck)
            kr[..., 0::2] = a_ * c_ - b_ * s_
            kr[..., 1::2] = a_ * s_ + b_ * c_
            xk = kr.transpose(0, 1).contiguous()
            p_, _ = tq.calibrate_rotation(xk)
            pi_d[l] = p_
            lk_d[l] = tq.calibrate_lut(xk, p_)
            lv_d[l] = tq.calibrate_lut(cv.transpose(0, 1).contiguous(), p_)
    else:
        pi_d = t_(synth.rotations(g, L, H))
        lk_d = lv_d = t_(np.broadcast_to(synth.GAUSS_LEVELS_MAX1960, (L, H, 8)).copy())
    torch.cuda.synchronize()
    calib_s = time.perf_counter() - t0

    # prefill, and the K steps' queries and new tokens
    params = tq.Params(L, H, cs, io_dtype=io, flags=tq.V_ROTATE)
    cache = tq.Cache(L, H, slots, device=dev)
    q_all = torch.empty((K, L, B, H, 64), dtype=io, device=dev)
    k_all = torch.empty_like(q_all)
    v_all = torch.empty_like(q_all)
    offs_d = t_(offs)
    tmax = int(lens.max())
    same = bool(np.all(lens == lens[0]))
    bidx = torch.arange(B, device=dev)
    lens_d = t_(lens.astype(np.int64))
    tokens_d = t_(lens.astype(np.int32))
    pf_ms = 0.0
    for l in range(L):
        gen = synth.device_generator(wl.seed, l, dev)
        kl = synth.keys_on(gen, B, tmax + K, H, ch[l], io, dev)
        vl = synth.values_on(gen, B, tmax + K, H, io, dev)
        for s in range(K):
            q_all[s, l] = synth.queries_on(gen, B, H, io, dev)
            k_all[s, l] = kl[bidx, lens_d + s]
            v_all[s, l] = vl[bidx, lens_d + s]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        # one call per layer; a ragged batch passes each sequence's length
        # (its rows past that length are padding, not read)
        kp, vp = kl[None, :, :tmax].contiguous(), vl[None, :, :tmax].contiguous()
        e0.record()
        tq.quantize_pack(params, cache, kp, vp, t_(np.zeros(B, np.int32)), offs_d, pi_d, lk_d, lv_d, S_d,
                         layer0=l, seq_tokens=None if same else tokens_d)
        e1.record()
        torch.cuda.synchronize()
        pf_ms += e0.elapsed_time(e1)
        del kl, vl
    torch.cuda.empty_cache()

    pos = [t_((lens + s).astype(np.int32)) for s in range(K)]
    outs = torch.empty((K, L, B, H, 64), dtype=io, device=dev)
    ws_need = tq.decode_workspace_bytes(params, B, L, tmax + K)
    ws = torch.zeros(max(ws_need, 16), dtype=torch.uint8, device=dev)

    def step(s):
        tq.decode_step(params, cache, q_all[s], k_all[s], v_all[s], pos[s], offs_d, pos[s], tmax + s + 1, pi_d,
                       lk_d, lv_d, S_d, out=outs[s], workspace=ws)

    for s in range(K):
        step(s)
    torch.cuda.synchronize()
    if eager:
        for s in range(K):
            step(s)
        torch.cuda.synchronize()
        return {"workload": name, "eager_steps": K}
    stream = torch.cuda.Stream(device=dev)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for s in range(K):
            step(s)
    graph.replay()
    torch.cuda.synchronize()
    sp = replay_spread(torch, graph, stream, K, replays)
    del graph

    units = L * B * H
    tok = float(np.sum(lens)) * L * H          # token-heads cached before the first step
    kv_bytes = (tok + units * (K + 1) / 2.0) * 72       # average over the K steps
    alg_bytes = kv_bytes + L * H * 64 * 64 * 4 + 64 * 64 * 4 + L * H * 8 * 4 * 2 + units * 64 * 2 * 4 + units * 72
    ms = sp["median"]
    line = {"workload": name, "layers": L, "heads": H, "batch": B,
            "cached_tokens": ({"min": int(lens.min()), "mean": round(float(lens.mean()), 1), "max": int(lens.max())}
                              if wl.ragged else int(lens[0])),
            "steps": K, "rotation": wl.rotation, "replays": sp["replays"],
            "step_ms_median": ms, "step_ms_p10": sp["p10"], "step_ms_p90": sp["p90"],
            "kv_gbs": round(kv_bytes / (ms * 1e-3) / 1e9, 1),
            "decode_steps_per_s": round(1e3 / ms, 1),
            "roofline": {"bound": "hbm", "achieved": round(alg_bytes / (ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(alg_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                         "alg_bytes_per_launch": int(alg_bytes),
                         "kernel": "decode_kernel<8, false> (one launch per tq_decode_step call)"},
            "calibration_s": round(calib_s, 3),
            "prefill_quantize_ms": round(pf_ms, 3),
            "prefill_token_heads": int(tok)}
    if cpu:
        line["cpu_baseline"] = oracle_sample(torch, oracle, cache, pi_d, lk_d, lv_d, S, q_all[K - 1], outs[K - 1],
                                             lens + K, offs, caps, L, H, B, positions, cpu_seconds, wl.seed)
    del cache, q_all, k_all, v_all, outs
    torch.cuda.empty_cache()
    return line


def oracle_sample(torch, oracle, cache, pi_d, lk_d, lv_d, S, q_last, out_last, n_att, offs, caps, L, H, B,
                  positions, seconds, seed):
    """The oracle's fp64 decode of a seeded sample of units, from the GPU
    cache's bytes after the timed steps (each sequence's units in a cache of
    their own): timed with all of the oracle's threads and with one, in KV
    GB/s, and compared with the GPU's output of the last step."""
    g = np.random.default_rng(seed + 17)
    seqs = sorted(set(int(x) for x in g.choice(B, size=min(2, B), replace=False)))
    per_seq = 16
    jobs = []
    cs = oracle.rope_table(positions)
    kc, vc, sc = cache.k_codes, cache.v_codes, cache.scalars
    slots = cache.slots
    for b in seqs:
        picks = sorted(set((int(g.integers(L)), int(g.integers(H))) for _ in range(per_seq)))
        cap = int(caps[b])
        oc = oracle.Cache(1, len(picks), cap)
        for i, (l, h) in enumerate(picks):
            base = (l * H + h) * slots + int(offs[b])
            oc.k[i * cap * 32:(i + 1) * cap * 32] = kc[base * 32:(base + cap) * 32].cpu().numpy()
            oc.v[i * cap * 32:(i + 1) * cap * 32] = vc[base * 32:(base + cap) * 32].cpu().numpy()
            oc.s[i * cap * 4:(i + 1) * cap * 4] = sc[base * 4:(base + cap) * 4].cpu().numpy().view(np.uint16)
        ls = [l for l, _ in picks]
        hs = [h for _, h in picks]
        q = q_last[ls, b, hs].float().cpu().numpy()[None, None]
        pi = pi_d[ls, hs].cpu().numpy()[None]
        lk = lk_d[ls, hs].cpu().numpy()[None]
        lv = lv_d[ls, hs].cpu().numpy()[None]
        ref_gpu = out_last[ls, b, hs].float().cpu().numpy()
        n = int(n_att[b])
        jobs.append((oc, q, pi, lk, lv, ref_gpu, n, len(picks)))

    def run_all():
        errs = []
        for oc, q, pi, lk, lv, ref_gpu, n, _ in jobs:
            o = oracle.decode(oc, oracle.V_ROTATE, cs, q, [n - 1], [0], [n], pi, lk, lv, S)
            errs.append(float(np.max(np.abs(o[0, 0] - ref_gpu))))
        return max(errs)

    kv = sum(cnt * n * 72 for _, _, _, _, _, _, n, cnt in jobs)
    res = {"kind": "oracle", "unit": "GB/s", "nproc": len(os.sched_getaffinity(0)),
           "sample": f"{sum(j[7] for j in jobs)} (layer, head) units of sequences {seqs} (seeded), "
                     f"fp64 decode of the GPU cache's bytes after the timed steps"}
    threads = oracle.max_threads()
    for label, nt in (("all", threads), ("one", 1)):
        oracle.set_threads(nt)
        runs, tt, err = 0, 0.0, 0.0
        while tt < seconds / 2 or runs == 0:
            t0 = time.perf_counter()
            err = run_all()
            tt += time.perf_counter() - t0
            runs += 1
        gbs = kv * runs / tt / 1e9
        if label == "all":
            res["value"], res["cores"] = round(gbs, 4), nt
        else:
            res["value_1thread"] = round(gbs, 4)
        res["max_abs_err_vs_gpu"] = round(err, 6)
        res["within_2e-3"] = bool(err <= 2e-3)
    oracle.set_threads(threads)
    return res


def only_kernel(torch, tq, which, K, params, reps, base_cache, t_, k_all, v_all, T, n_ctx, L, H, slots, pi_d,
                lut_d, S_d, zero_i32, zero_i64):
    """K eager launches of one kernel on the headline shape, for counter
    collection: the prefill quantizer (tq_quantize_pack of the T cached
    tokens of every unit), the dequantize baseline (tq_dequantize of the
    n_ctx tokens of every unit), or (lengths) the decode kernel over 1, 513
    and n_ctx tokens of every unit, first as attends (K launches per length)
    and then as steps (K per length; a step over n tokens appends token n - 1
    of replica 0's cache). The lengths separate a unit's fixed work (no
    tile: only the last token), one tile per wave (8 tiles) and two."""
    if which == "lengths":
        lens = [1, 513, n_ctx]
        times = {}
        d = reps[0]
        for mode in ("attend", "step"):
            for n in lens:
                qpos = torch.tensor([n - 1], dtype=torch.int32, device="cuda")
                slen = torch.tensor([n if mode == "attend" else n - 1], dtype=torch.int32, device="cuda")
                ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                for k in range(K + 1):
                    if k == 1:
                        ea.record()
                    if mode == "attend":
                        tq.decode_attend(params, d["cache"], d["q"], qpos, zero_i64, slen, n_ctx, d["pi"], lut_d,
                                         lut_d, S_d, out=d["out"])
                    else:
                        tq.decode_step(params, d["cache"], d["q"], d["k1"], d["v1"], qpos, zero_i64, slen, n_ctx,
                                       d["pi"], lut_d, lut_d, S_d, out=d["out"])
                eb.record()
                torch.cuda.synchronize()
                times[f"{mode}_{n}"] = round(ea.elapsed_time(eb) / max(K, 1), 5)
        print(json.dumps({"only": which, "launches_per_case": K + 1, "order": list(times),
                          "eager_ms_per_launch": times}))
        return
    if which == "prefill":
        pf_cache = tq.Cache(L, H, slots, device="cuda")
        k_pf, v_pf = t_(k_all[:, :, :T]), t_(v_all[:, :, :T])
        for _ in range(K):
            tq.quantize_pack(params, pf_cache, k_pf, v_pf, zero_i32, zero_i64, pi_d, lut_d, lut_d, S_d)
    else:
        shape = (L, 1, H, n_ctx, 64)
        ko = torch.empty(shape, dtype=torch.float16, device="cuda")
        vo = torch.empty(shape, dtype=torch.float16, device="cuda")
        sl = torch.tensor([n_ctx], dtype=torch.int32, device="cuda")
        for k in range(K):
            tq.dequantize(params, reps[k % len(reps)]["cache"], zero_i64, sl, n_ctx, lut_d, lut_d, S_d,
                          k_out=ko, v_out=vo)
    torch.cuda.synchronize()
    print(json.dumps({"only": which, "launches": K}))


def fp16_attention_baseline(torch, units, n_ctx, replica_bytes, K):
    """Plain decode attention over an unquantized fp16 cache of the same shape
    (one query per (layer, head) unit, n_ctx cached keys and values of 64
    fp16 each, 256 B per token-head against the packed cache's 72 B), with
    PyTorch on the same GPU: scaled_dot_product_attention, and an explicit
    matmul - softmax (fp32) - matmul. Replicas rotate as for the fused path so
    each call reads HBM. Context for the fused kernel, not part of the path."""
    import torch.nn.functional as F
    dev = torch.device("cuda:0")
    per = units * n_ctx * 64 * 2 * 2
    R = max(2, math.ceil(replica_bytes / per))
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    kv = [(torch.randn((1, units, n_ctx, 64), generator=g, device=dev, dtype=torch.float16),
           torch.randn((1, units, n_ctx, 64), generator=g, device=dev, dtype=torch.float16)) for _ in range(R)]
    q = torch.randn((1, units, 1, 64), generator=g, device=dev, dtype=torch.float16)

    def sdpa(r):
        return F.scaled_dot_product_attention(q, kv[r][0], kv[r][1])

    def explicit(r):
        k, v = kv[r]
        w = torch.softmax(torch.matmul(k[0], q[0].transpose(1, 2).contiguous()).float() * 0.125, dim=1)
        return torch.matmul(w.transpose(1, 2).to(torch.float16).contiguous(), v[0])

    out = {"units": units, "tokens": n_ctx, "kv_bytes_per_call": units * n_ctx * 256, "replicas": R}
    for name, fn in (("sdpa", sdpa), ("matmul_softmax", explicit)):
        for r in range(R):
            fn(r)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for s in range(K):
            fn(s % R)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / K
        out[name + "_ms"] = round(ms, 5)
        out[name + "_kv_gbs"] = round(units * n_ctx * 256 / (ms * 1e-3) / 1e9, 1)
    del kv
    torch.cuda.empty_cache()
    return out


def two_step_baseline(torch, tq, params, reps, L, H, n_ctx, cs, pi_list, lut_d, S_d, K, fused_ms):
    """The dequantize-then-attend path on the same packed caches (the analog of
    the paper's Table 6 comparison, fused kernel against unpacking first):
    tq_dequantize writes fp16 k~ and v~ rows of every cached token to HBM,
    then PyTorch rotates the query (RoPE, Pi q'), runs
    scaled_dot_product_attention over the rows and applies Pi^T. Context for
    the fused kernel, not part of the path."""
    import torch.nn.functional as F
    dev = torch.device("cuda:0")
    units = L * H
    shape = (L, 1, H, n_ctx, 64)
    ko = torch.empty(shape, dtype=torch.float16, device=dev)
    vo = torch.empty(shape, dtype=torch.float16, device=dev)
    s0 = torch.zeros(1, dtype=torch.int64, device=dev)
    sl = torch.tensor([n_ctx], dtype=torch.int32, device=dev)
    c, s = cs[n_ctx - 1, :, 0], cs[n_ctx - 1, :, 1]
    R = len(reps)

    def dequant(r):
        tq.dequantize(params, reps[r]["cache"], s0, sl, n_ctx, lut_d, lut_d, S_d, k_out=ko, v_out=vo)

    def attend(r):
        qf = reps[r]["q"].float()
        x0, x1 = qf[..., 0::2], qf[..., 1::2]
        qr = torch.stack((x0 * c - x1 * s, x0 * s + x1 * c), dim=-1).reshape(qf.shape)
        pi = pi_list[r]
        qh = torch.matmul(pi.unsqueeze(1), qr.unsqueeze(-1)).squeeze(-1)     # [L, 1, H, 64]
        oh = F.scaled_dot_product_attention(qh.half().reshape(1, units, 1, 64), ko.view(1, units, n_ctx, 64),
                                            vo.view(1, units, n_ctx, 64), scale=0.125)
        return torch.matmul(oh.float().reshape(L, 1, H, 1, 64), pi.unsqueeze(1)).reshape(L, 1, H, 64)

    def timed(fn):
        for r in range(3):
            fn(r % R)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for k in range(K):
            fn(k % R)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    dq_ms = timed(dequant)
    total_ms = timed(lambda r: (dequant(r), attend(r)))
    dequant(0)
    out = attend(0)
    torch.cuda.synchronize()
    th = units * n_ctx
    res = {"dequantize_ms": round(dq_ms, 5), "total_ms": round(total_ms, 5),
           "dequantize_gbs": round(th * (72 + 256) / (dq_ms * 1e-3) / 1e9, 1),
           "rows_bytes": th * 256,
           "fused_decode_attend_speedup": round(total_ms / fused_ms, 2),
           "max_abs_diff_vs_fused": round(float((out - reps[0]["out"].float()).abs().max()), 5)}
    del ko, vo
    torch.cuda.empty_cache()
    return res


def measured_traffic(workload):
    """HBM bytes per step of the decode-step kernels from the committed counter
    summary (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy's readings), or
    None when the kernel sources have changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"decode_step_traffic__{workload}.json")
    if not os.path.exists(path):
        return None, None
    with open(path) as f:
        rec = json.load(f)
    h = hashlib.sha256()
    for src in rec["sources"]:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    if h.hexdigest() != rec["sources_sha256"]:
        return None, None
    return int(rec["traffic_bytes_per_step"]), os.path.relpath(path, ROOT)


def cpu_baseline(k_all, v_all, S, lut, pi, q, L, H, slots, n_ctx, seconds):
    """The CPU oracle on the same workload, timed on the host: it quantizes
    the cached tokens into a cache of its own (untimed, like the GPU's
    prefill), then each timed run is one oracle step: append the new token of
    every (layer, head) and decode (fp64, OpenMP over units). If one run over
    all units would exceed `seconds`, the decode covers a leading subset of
    units; runs repeat until ~`seconds`. Value in KV GB/s like the GPU line."""
    from oracle import oracle
    T = n_ctx - 1
    oc = oracle.Cache(L, H, slots)
    cs = oracle.rope_table(slots + 64)
    oracle.quantize_pack(oc, 1, cs, k_all[:, :, :T], v_all[:, :, :T], [0], [0], pi, lut, lut, S)
    k_new, v_new = k_all[:, :, T:T + 1], v_all[:, :, T:T + 1]
    qf = np.asarray(q, np.float32)
    threads = oracle.max_threads()

    def run(units):
        oracle.quantize_pack(oc, 1, cs, k_new, v_new, [T], [T], pi, lut, lut, S)
        oracle.decode(oc, 1, cs, qf, [T], [0], [n_ctx], pi, lut, lut, S, units=units)

    runs, t_total = 0, 0.0
    units_per_run = L * H
    # one step over all units may be long; time a unit subset if so
    sample = None
    n_probe = min(32, L * H)
    t0 = time.perf_counter()
    run(np.arange(n_probe))
    probe = time.perf_counter() - t0
    if probe * (L * H) / n_probe > seconds:
        nu = max(1, int(seconds / probe * n_probe))
        sample = np.arange(min(nu, L * H))
        units_per_run = len(sample)
    while t_total < seconds:
        t0 = time.perf_counter()
        run(sample)
        t_total += time.perf_counter() - t0
        runs += 1
    kv = units_per_run * n_ctx * 72 * runs
    # the same step with one thread, over a leading subset of units (the
    # append is serial anyway)
    oracle.set_threads(1)
    one_units = np.arange(max(1, min(L * H, units_per_run // max(1, threads))))
    t1, runs1 = 0.0, 0
    while t1 < seconds / 3 or runs1 == 0:
        t0 = time.perf_counter()
        run(one_units)
        t1 += time.perf_counter() - t0
        runs1 += 1
    oracle.set_threads(threads)
    return {"value": round(kv / t_total / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "nproc": len(os.sched_getaffinity(0)), "os_cpu_count": os.cpu_count(),
            "value_1thread": round(len(one_units) * n_ctx * 72 * runs1 / t1 / 1e9, 4),
            "sample": f"{runs} oracle step(s): append of the new token to all {L * H} (layer, head) units, "
                      f"then fp64 decode of {units_per_run} of them over {n_ctx} tokens, {t_total:.1f} s "
                      f"({threads} threads); one thread: {runs1} step(s) decoding {len(one_units)} units, "
                      f"{t1:.1f} s"}


if __name__ == "__main__":
    main()
