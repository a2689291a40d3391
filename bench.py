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

Prints one JSON line (see the "value", "roofline" and "cpu_baseline" keys).
    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline]
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
    assert wl.batch == 1 and wl.ragged is None, "the bench drives the batch-1 decode workloads"
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
        "two_call_step_ms": None if two_call_ms is None else round(two_call_ms, 5),
        "decode_attend_ms": round(attend_ms, 5),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "traffic_source": traffic_src,
                     "kernel": ("decode_kernel<8, false> (one launch per tq_decode_attend call)"
                                if args.decode_only else
                                "decode_kernel<8, false> (one launch per tq_decode_step call)"),
                     "alg_bytes_per_launch": int(alg_bytes)},
        "cpu_baseline": cpu,
        "prefill_quantize": prefill,
        "two_step_baseline": two_step,
        "fp16_attention_baseline": fp16_base,
        "paper_context": {"memory_reduction": "7.1x (Table 4, fp32 baseline, 'CUDA')",
                          "kv_fetch_speedup": "1.96x Triton vs PyTorch fetch_unpacked, 143 tokens, "
                                              "NVIDIA GPU on Colab, model and precision unstated (Table 6)"},
    }
    print(json.dumps(line))


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
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))

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
    return {"value": round(kv / t_total / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{runs} oracle step(s): append of the new token to all {L * H} (layer, head) units, "
                      f"then fp64 decode of {units_per_run} of them over {n_ctx} tokens, {t_total:.1f} s"}


if __name__ == "__main__":
    main()
