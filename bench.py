"""Benchmark of the QEvict tiered decode step on one MI355X.

Workload: the Llama-3-8B-shaped layer at 32K context (batch 1, 32 query / 8 KV
heads, head_dim 128, windows of 32, 20% bf16 / 30% int4 group-32 / 50%
evicted, routing every step, drifting queries).  One step is the whole hot
path for one layer: append + tiered split-K attention + split merge and
window-score accumulation (decode_attend) followed by the re-rank and the
quantize / promote migrations (retier).

Sixteen independent caches of this shape (one per "layer" of one workspace,
each with its own seeds) are stepped round robin.  A cache is used again only
after the other fifteen, so the 16 x ~49 MB working set exceeds the 256 MB
Infinity Cache and every step streams its windows from HBM.  Inputs for all
timed steps are generated and copied to the GPU before timing.  By default the
routing work runs on the library's routing stream (QEVICT_FLAG_ASYNC_ROUTING),
overlapping the attention of the following layers; --routing sync keeps every
kernel on one stream.

Prints one JSON line.  `value` is microseconds per step (lower is better):
the GPU time of the K timed steps on the cache's stream (HIP events), taken
in steady state -- the routing requests the warm-up left queued run inside the
timed region, and those still queued when it closes are drained after it and
reported as `routing_tail_us` -- divided by K.  `roofline` reports
decode_attend's algorithmic bytes per call over its average duration (the
attention pass and the split merge), measured with HIP events on the cache's
stream around rounds of back-to-back decode_attend calls with no routing
running; `roofline.traffic` is the HBM traffic per call from the committed
FETCH_SIZE / WRITE_SIZE record over the same duration (null when the sources
of the attention path changed since it was taken, and on any run other than
the default one it covers).  Initial window scores come from the prompt's last
W queries attending to the prompt (qevict_prefill_scores); the latency of one
such call (host marshalling and its three launches, GPU otherwise idle) is
reported as `prefill_scores_call_us`.

`--workload` runs another synthetic shape instead (all sequences of its batch,
byte-budget capacities where it gives a budget, a routing event after every
R-th step of a cache at its routing interval R); such runs are context, not
the benchmark line.  The 32-layer batch-8 workload runs its 32 layers back to
back per decode step: `value` is then microseconds per decode step of the
whole model.
"""
from __future__ import annotations

import argparse
import json
from fractions import Fraction
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tiered decode-attention µs/step + achieved HBM GB/s (8B shape, 32k ctx, 1 GPU)"
HBM_PEAK_GBPS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=1024)
    p.add_argument("--warmup", type=int, default=160)
    p.add_argument("--instances", type=int, default=16, help="independent layer caches rotated")
    p.add_argument("--workload", default="c2")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle baseline time budget")
    p.add_argument("--no-cpu", action="store_true")
    p.add_argument("--splits", type=int, default=0, help="split-K factor (0 = library default)")
    p.add_argument("--routing", choices=("async", "queue", "device", "sync"), default="async",
                   help="async: a layer's routing runs on the library's routing stream, overlapping "
                        "the attention of the other layers, ordered after the cache stream as the "
                        "library chooses; queue / device: the same, always with the queue-level / "
                        "device-side wait; sync: everything on one stream")
    p.add_argument("--no-kernel-events", action="store_true",
                   help="do not time each kernel launch with HIP events (no roofline)")
    p.add_argument("--rope-base", type=float, default=0.0,
                   help="RoPE-aware Quantized tier with this base (0: off, the default workload)")
    p.add_argument("--prefill-scores", action="store_true",
                   help="time the initial-window-score kernels on the workload's prompt instead")
    p.add_argument("--init-scores", choices=("prompt", "synthetic"), default="prompt",
                   help="initial window scores: prompt attention of the last W prompt queries "
                        "(qevict_prefill_scores, the default), or the synthetic log-normal scores")
    p.add_argument("--calibrate-copy", type=float, default=0.0, metavar="MB",
                   help="only run 8 plain device-to-device copies of this many MB (hardware "
                        "counter calibration) and exit")
    return p.parse_args()


def calibrate_copy(mb):
    """Eight copies of a known size, for scaling the FETCH_SIZE / WRITE_SIZE
    counters.  The copies rotate over four source / destination pairs of 4x the
    last-level cache size in total, so no source line is still cached."""
    import torch
    n = int(mb * 1e6) // 4
    pairs = [(torch.ones(n, dtype=torch.float32, device="cuda"),
              torch.empty(n, dtype=torch.float32, device="cuda")) for _ in range(4)]
    torch.cuda.synchronize()
    for i in range(8):
        src, dst = pairs[i % 4]
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "copy", "bytes_read_per_copy": 4 * n, "bytes_written_per_copy": 4 * n,
                      "copies": 8}))
    return 0


def to_dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def workload_desc(wl):
    if wl.name == "c2":
        return ("Llama-3-8B-shaped layer, 32768-token context, batch 1, 32 query / 8 KV heads, "
                "head_dim 128, windows of 32, 20% bf16 / 30% int4 group 32 / 50% evicted, re-tier "
                "every step, drifting queries")
    bits = {4: "int4", 2: "int2", 42: "int4 / int2 by rank"}[wl.bits]
    tiers = (f"byte budget {wl.budget_frac} of the full cache, quantized share {wl.q_frac}"
             if wl.budget_frac else f"{wl.frac_full} bf16 / {wl.frac_quant} quantized")
    layers = f"{wl.layers} layers back to back per step, " if wl.layers > 1 else ""
    return (f"{layers}{wl.prompt_len}-token context, batch {wl.batch}, {wl.num_q_heads} query / "
            f"{wl.num_kv_heads} KV heads, head_dim {wl.head_dim}, windows of {wl.window}, {bits} "
            f"group {wl.group}, {tiers}, sink {wl.sink}, recent {wl.recent}, "
            + ("re-tier every step" if wl.retier_interval == 1 else f"re-tier every {wl.retier_interval} steps"))


def attend_bytes(wl, n_full, n_q4, n_q2, recent_tokens):
    """Algorithmic bytes of one attention pass of one sequence-layer.

    Live bf16 windows (K + V), live quantized codes with fp16 scale/zero,
    bf16 recent tokens, the bf16 query and output, and the window scores
    read and written.  Evicted windows and split partials are not counted.
    """
    h, d, w = wl.num_kv_heads, wl.head_dim, wl.window
    meta = h * (d * 4 + w * (d // wl.group) * 4)   # keys: one group per channel
    full = n_full * 2 * h * w * d * 2
    q4 = n_q4 * (2 * h * w * d * 4 // 8 + meta)
    q2 = n_q2 * (2 * h * w * d * 2 // 8 + meta)
    recent = recent_tokens * 2 * h * d * 2
    qo = 2 * wl.num_q_heads * d * 2
    scores = 2 * (n_full + n_q4 + n_q2 + 1) * 4
    return full + q4 + q2 + recent + qo + scores


COUNTERS = os.path.join(ROOT, "profiles", "decode_attend_8b_32k_hbm_counters.md")


# sources that build the decode-attention kernels, their launch and the layouts
# they read (the live list and split plan the re-rank kernel writes)
ATTEND_SOURCES = ("attend.hip", "retier.hip", "runtime.cpp", "qv_device.h", "qv_layout.h")


def kernel_source_hash():
    """sha256 over the sources of the decode-attention path (any edit of them changes it)."""
    import hashlib
    d = os.path.join(ROOT, "paper_2608_05326_amd", "csrc")
    h = hashlib.sha256()
    for f in ATTEND_SOURCES:
        h.update(f.encode())
        h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per decode_attend from the committed FETCH_SIZE / WRITE_SIZE
    counter record, or None when the kernels changed since it was taken."""
    try:
        lines = open(COUNTERS).read().splitlines()
    except OSError:
        return None
    for ln in lines:
        if ln.startswith("record: "):
            rec = json.loads(ln[len("record: "):])
            if rec.get("source_sha256") == kernel_source_hash():
                return rec
    return None


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return 1


def cpu_baseline(wl, seed, budget_s, units_per_step=1):
    """The float64 oracle stepping one sequence-layer of the same workload (append,
    attention and score accumulation every step, routing at the workload's
    interval).  A step of a workload with several sequences or layers is
    `units_per_step` such unit steps: the time of one is scaled by that count."""
    from oracle.qevict_oracle import OracleConfig, QEvictUnit
    import synthetic as syn
    cores = blas_threads()
    kf, kq = wl.capacity_full, wl.capacity_quant
    if wl.budget_frac:
        from oracle.qevict_oracle import tier_capacities
        full = 2 * wl.num_kv_heads * wl.head_dim * wl.prompt_len * 2
        kf, kq = tier_capacities(int(Fraction(wl.budget_frac) * full), int(Fraction(wl.q_frac) * 1000),
                                 wl.num_kv_heads, wl.head_dim, wl.window, wl.group, wl.bits,
                                 wl.sink, wl.recent)
    cfg = OracleConfig(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window, wl.group, wl.bits,
                       kf, kq, sink=wl.sink, recent=wl.recent)
    # decode steps beyond the workload's own count, so that the sample fills the budget
    n_max = max(wl.steps, 2048)
    u = QEvictUnit(cfg, wl.prompt_len + n_max)
    k, v = syn.prompt_kv(wl, seed, 0, 0)
    f = syn.bf16_bits_to_f32
    u.prefill(f(k).astype(np.float64), f(v).astype(np.float64), syn.init_scores(wl, seed, 0, 0))
    del k, v
    qs, ks, vs = syn.decode_inputs(wl, seed, 0, 0, n_max)
    n = 0
    t0 = time.perf_counter()
    while n < n_max and (n < 3 or time.perf_counter() - t0 < budget_s):
        u.step(f(qs[n]).astype(np.float64), f(ks[n]).astype(np.float64), f(vs[n]).astype(np.float64))
        if (n + 1) % wl.retier_interval == 0:
            u.route()
        n += 1
    dt = time.perf_counter() - t0
    per = dt / n * 1e6 * units_per_step
    sample = (f"{n} decode steps (attend + score + route every {wl.retier_interval}) of one "
              f"{wl.prompt_len}-token sequence-layer after prefill, float64 numpy, {dt:.1f} s")
    if units_per_step > 1:
        sample += f"; times {units_per_step} sequence-layers per step (extrapolated)"
    return {"value": round(per, 1), "unit": "us/step", "cores": cores, "kind": "oracle",
            "sample": sample}


def bench_prefill_scores(args):
    """Initial window scores of a prompt (qevict_prefill_scores): W observation
    queries attending causally to the whole prompt, per-window masses.  Eight
    prompts of the workload's shape are rotated so that their keys (64 MB each
    at 32K) do not stay in the Infinity Cache between calls; one call reads the
    keys once."""
    import torch
    import paper_2608_05326_amd as qv
    import synthetic as syn
    wl = syn.get_workload(args.workload)
    n_obs = wl.window
    NP = 8
    cfg = qv.Config(batch=wl.batch, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                    window_tokens=wl.window, group_size=wl.group, quant_bits=wl.bits,
                    max_context=wl.prompt_len + 64, capacity_full=wl.capacity_full,
                    capacity_quant=wl.capacity_quant, sink_tokens=wl.sink, recent_tokens=wl.recent)
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)
    cache = qv.Cache(cfg, stream=stream)
    Ks, Qs, hk, hq = [], [], None, None
    for i in range(NP):
        k = np.stack([syn.prompt_kv(wl, args.seed, b, i)[0] for b in range(wl.batch)])
        q = np.stack([syn.observation_queries(wl, args.seed, b, i, n_obs) for b in range(wl.batch)])
        if i == 0:
            hk, hq = k[0], q[0]
        Ks.append(to_dev(k))
        Qs.append(to_dev(q))
    n_w = -(-(wl.prompt_len - wl.sink) // wl.window)
    out = torch.empty((wl.batch, n_w), dtype=torch.float32, device="cuda")
    scratch = torch.empty(qv.qevict.prefill_scores_scratch_size(cfg, wl.prompt_len, n_obs),
                          dtype=torch.uint8, device="cuda")
    for i in range(max(args.warmup // 16, 2) * NP):
        cache.prefill_scores(Qs[i % NP], Ks[i % NP], out, scratch)
    steps = max(args.steps // 16, NP)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(steps):
        cache.prefill_scores(Qs[i % NP], Ks[i % NP], out, scratch)
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / steps
    B, Hkv, Hq, T, d = wl.batch, wl.num_kv_heads, wl.num_q_heads, wl.prompt_len, wl.head_dim
    min_bytes = B * (Hkv * T * d * 2 + Hq * n_obs * d * 2 + n_w * 4)
    flops = 2 * B * Hq * n_obs * T * d           # one QK^T over every (row, key) pair
    ach = min_bytes / (us * 1e-6) / 1e9
    res = {
        "metric": "initial window scores µs per prompt layer (observation-query attention masses)",
        "value": round(us, 3), "unit": "us/call", "n_gpus": 1, "steps": steps,
        "warmup": max(args.warmup // 16, 2) * NP, "ms_per_step": round(us / 1e3, 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16 (fp32 accumulate)", "data": "synthetic",
        "config": {"workload": f"{wl.prompt_len}-token prompt, batch {B}, {Hq} query / {Hkv} KV heads, "
                               f"head_dim {d}, windows of {wl.window}, {n_obs} observation queries",
                   "prompts_rotated": NP, "parallelism": "single GPU"},
        "tflops": round(flops / (us * 1e-6) / 1e12, 1),
        "roofline": {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(ach / HBM_PEAK_GBPS, 4), "traffic": None},
    }
    if not args.no_cpu:
        from oracle.qevict_oracle import prefill_window_scores
        f = syn.bf16_bits_to_f32
        t0 = time.perf_counter()
        prefill_window_scores(f(hq).astype(np.float64), f(hk).astype(np.float64), wl.sink, wl.window)
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": round(dt * 1e6 * B, 1), "unit": "us/call", "cores": blas_threads(),
                               "kind": "oracle",
                               "sample": f"one sequence's scores (float64 numpy, {dt:.1f} s), times {B}"}
    print(json.dumps(res))
    cache.close()
    return 0


def host_cpu():
    """Host CPU model name and logical CPU count."""
    model = None
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, os.cpu_count()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU; the decode path has no "
                                   "multi-GPU mode",
                          "n_gpus": args.gpus}))
        return 2
    if args.calibrate_copy > 0:
        return calibrate_copy(args.calibrate_copy)
    if args.prefill_scores:
        return bench_prefill_scores(args)
    import torch
    import paper_2608_05326_amd as qv
    import synthetic as syn

    wl = syn.get_workload(args.workload)
    # A workload of several layers (the 32-layer batch-8 one) runs all of them back
    # to back per decode step; a single-layer workload rotates `instances`
    # independent layer caches, one layer call per step.
    whole_model = wl.layers > 1
    NL = wl.layers if whole_model else args.instances
    LPS = NL if whole_model else 1                 # layer calls per step
    prof_rounds = 4                   # rounds of back-to-back decode_attend timing
    # routing timing and routing statistics each take two routing periods (R steps
    # of every layer cache, so that every cache routes at least twice)
    route_rounds = 2 * max(1, wl.retier_interval)
    per_layer = -(-((args.warmup + args.steps) * LPS) // NL) + prof_rounds + 2 * route_rounds + 1
    asyncr = args.routing in ("async", "queue", "device")
    R = wl.retier_interval            # routing event after every R-th step of a layer cache
    kf, kq = wl.capacity_full, wl.capacity_quant
    if wl.budget_frac:
        # byte budget: a fraction of the prompt's full bf16 cache, quantized share q
        full = 2 * wl.num_kv_heads * wl.head_dim * wl.prompt_len * 2
        probe = qv.Config(batch=wl.batch, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                          window_tokens=wl.window, group_size=wl.group, quant_bits=wl.bits,
                          max_context=wl.prompt_len + per_layer, capacity_full=0, capacity_quant=0,
                          sink_tokens=wl.sink, recent_tokens=wl.recent, retier_interval=R)
        kf, kq = qv.qevict.capacities_for_budget(probe, int(Fraction(wl.budget_frac) * full),
                                                 int(Fraction(wl.q_frac) * 1000))
    cfg = qv.Config(batch=wl.batch, num_layers=NL, num_q_heads=wl.num_q_heads,
                    num_kv_heads=wl.num_kv_heads, window_tokens=wl.window, group_size=wl.group,
                    quant_bits=wl.bits, max_context=wl.prompt_len + per_layer,
                    capacity_full=kf, capacity_quant=kq,
                    sink_tokens=wl.sink, recent_tokens=wl.recent, retier_interval=R,
                    num_splits=args.splits,
                    flags=(qv.FLAG_ASYNC_ROUTING if asyncr else 0) |
                          (qv.FLAG_ROUTING_QUEUE_WAIT if args.routing == "queue" else 0) |
                          (qv.FLAG_ROUTING_DEVICE_WAIT if args.routing == "device" else 0),
                    rope_base=args.rope_base)
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)
    cache = qv.Cache(cfg, stream=stream)
    order = cache.routing_order()
    print(f"[bench] workspace {cache.workspace.numel() / 1e6:.1f} MB for {NL} layer caches of "
          f"batch {wl.batch}", file=sys.stderr, flush=True)

    # ---- prefill every layer cache; initial window scores from the prompt's last
    # W queries attending to the prompt (qevict_prefill_scores), unless asked for
    # the synthetic scores ----
    observed = args.init_scores == "prompt"
    n_obs = wl.window

    def gen(layer):
        kv = [syn.prompt_kv(wl, args.seed, b, layer) for b in range(wl.batch)]
        if observed:
            init = np.stack([syn.observation_queries(wl, args.seed, b, layer, n_obs)
                             for b in range(wl.batch)])
        else:
            init = np.stack([syn.init_scores(wl, args.seed, b, layer) for b in range(wl.batch)])
        return layer, np.stack([x[0] for x in kv]), np.stack([x[1] for x in kv]), init

    t0 = time.time()
    ps_ms = []
    scratch = None
    with ThreadPoolExecutor(max_workers=8) as ex:
        for layer, k, v, init in ex.map(gen, range(NL)):
            K, V = to_dev(k), to_dev(v)                  # [B, H_kv, T, d]
            if observed:
                Qo = to_dev(init)                        # [B, H_q, n_obs, d]
                if scratch is None:
                    scratch = torch.empty(qv.qevict.prefill_scores_scratch_size(cfg, wl.prompt_len, n_obs),
                                          dtype=torch.uint8, device="cuda")
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                S = cache.prefill_scores(Qo, K, scratch=scratch)
                e1.record(stream)
                torch.cuda.synchronize()
                ps_ms.append(e0.elapsed_time(e1))
                del Qo
            else:
                S = torch.from_numpy(np.ascontiguousarray(init)).cuda()
            cache.prefill_assign(layer, K, V, S)
            torch.cuda.synchronize()
            del K, V, S
    del scratch
    print(f"[bench] prefilled {NL} layers in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)

    # ---- per-step inputs, resident on the GPU before timing ----
    dec = [[syn.decode_inputs(wl, args.seed, b, layer, per_layer) for b in range(wl.batch)]
           for layer in range(NL)]
    Q = [to_dev(np.stack([x[0] for x in d], axis=1)) for d in dec]     # [steps, B, H_q, d]
    KN = [to_dev(np.stack([x[1] for x in d], axis=1)) for d in dec]
    VN = [to_dev(np.stack([x[2] for x in d], axis=1)) for d in dec]
    del dec
    # the decode calls below pass raw pointers: check every extent on the host first
    for l in range(NL):
        assert tuple(Q[l].shape) == (per_layer, wl.batch, wl.num_q_heads, wl.head_dim), Q[l].shape
        for x in (KN[l], VN[l]):
            assert tuple(x.shape) == (per_layer, wl.batch, wl.num_kv_heads, wl.head_dim), x.shape
    out = torch.empty((wl.batch, wl.num_q_heads, wl.head_dim), dtype=torch.float32, device="cuda")

    import ctypes
    lib, h = cache.lib, cache.handle
    optr = ctypes.c_void_p(out.data_ptr())
    ptrs = [[(ctypes.c_void_p(Q[l][t].data_ptr()), ctypes.c_void_p(KN[l][t].data_ptr()),
              ctypes.c_void_p(VN[l][t].data_ptr())) for t in range(per_layer)] for l in range(NL)]
    counter = [0] * NL

    def attend(layer):
        t = counter[layer]
        counter[layer] += 1
        q, k, v = ptrs[layer][t]
        if lib.qevict_decode_attend(h, layer, q, k, v, optr):
            raise RuntimeError(lib.qevict_last_error().decode())

    def route(layer):
        if counter[layer] % R:        # not the end of a routing period
            return
        if lib.qevict_retier(h, layer, None):
            raise RuntimeError(lib.qevict_last_error().decode())

    # A layer call is one layer cache's decode_attend followed (before that cache is
    # used again) by its retier; layer calls cycle over the caches.  With
    # asynchronous routing the retier goes to the library's routing stream and the
    # next layer's attention proceeds; with synchronous routing the calls run in
    # rounds (the decode_attend of every cache, then the retier of each).
    def run_calls(first, count):
        i = first
        while i < first + count:
            layers = [(i + k) % NL for k in range(min(NL - i % NL, first + count - i))]
            if asyncr:
                for l in layers:
                    attend(l)
                    route(l)
            else:
                for l in layers:
                    attend(l)
                for l in layers:
                    route(l)
            i += len(layers)

    run_calls(0, args.warmup * LPS)
    torch.cuda.synchronize()
    st0 = [[cache.get_state(l, b) for b in range(wl.batch)] for l in range(NL)]

    # ---- timed region: K steps in steady state.  Routing requests still queued
    # when it closes (asynchronous routing) are drained after it and reported
    # apart; the requests queued by the warm-up run inside it. ----
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    t_wall = time.perf_counter()
    run_calls(args.warmup * LPS, args.steps * LPS)
    ev1.record(stream)
    wall = time.perf_counter() - t_wall
    torch.cuda.synchronize()
    gpu_ms = ev0.elapsed_time(ev1)
    ms_per_step = gpu_ms / args.steps
    d0, d1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    d0.record(stream)
    cache.join_routing()
    d1.record(stream)
    torch.cuda.synchronize()
    drain_us = d0.elapsed_time(d1) * 1e3
    done = (args.warmup + args.steps) * LPS

    # ---- decode_attend timing: rounds of NL back-to-back calls (one per layer
    # cache) bracketed by HIP events on the cache's stream, with no routing
    # running beside them (each round starts after the previous round's routing
    # and routes only after its attention) ----
    attn_events = []
    if not args.no_kernel_events:
        for _ in range(max(1, prof_rounds)):
            cache.join_routing()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for l in range(NL):
                attend(l)
            e1.record(stream)
            torch.cuda.synchronize()
            attn_events.append((e0.elapsed_time(e1), NL))
            for l in range(NL):
                route(l)
            done += NL
        cache.join_routing()
        torch.cuda.synchronize()
    # ---- routing kernels: HIP events around every re-rank and migration launch
    # (the library's profile counters, on the stream each runs on) over a few
    # more rounds, with nothing else on the GPU while they run (the attention of
    # a round finishes first), so that each duration is the routing latency and
    # not a wait for compute units held by other layers' attention; each such
    # duration also holds the launch's dispatch ----
    lp = None
    if not args.no_kernel_events:
        cache.profile_enable(True)
        for _ in range(route_rounds):
            for l in range(NL):
                attend(l)
            cache.join_routing()
            torch.cuda.synchronize()
            for l in range(NL):
                route(l)
            cache.join_routing()
            torch.cuda.synchronize()
            done += NL
        lp = {k: cache.profile_read(k) for k in (2, 3)}
        cache.profile_enable(False)

    # ---- routing activity: more (untimed) rounds with the retier stats read back ----
    promo = react = evict = 0
    n_ev = 0
    for _ in range(route_rounds):
        for l in range(NL):
            attend(l)
        for l in range(NL):
            if counter[l] % R == 0:
                s_ = cache.retier(l, stats=True)
                promo += s_["promotions"]
                react += s_["reactivations"]
                evict += s_["evictions"]
                n_ev += 1

    # ---- algorithmic bytes of the timed attention launches ----
    total_bytes = 0
    for i in range(args.warmup * LPS, (args.warmup + args.steps) * LPS):
        layer = i % NL
        T = wl.prompt_len + (i // NL) + 1
        recent = (T - wl.sink) - ((T - wl.sink) // wl.window) * wl.window
        recent = recent if recent else wl.window
        for st in st0[layer]:   # every sequence of the batch
            n_full = int(np.sum(st["tiers"] == qv.TIER_FULL))
            bits = st["bits"][st["tiers"] == qv.TIER_QUANT]
            total_bytes += attend_bytes(wl, n_full, int(np.sum(bits == 4)), int(np.sum(bits == 2)),
                                        recent)
    bytes_per_call = total_bytes / (args.steps * LPS)
    bytes_per_step = total_bytes / args.steps

    cpu_model, n_cpu = host_cpu()
    res = {
        "metric": METRIC,
        "value": round(ms_per_step * 1e3, 3),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16+" + {4: "int4", 2: "int2", 42: "int4/int2"}[wl.bits] + " (fp32 accumulate)",
        "data": "synthetic",
        "config": {"workload": workload_desc(wl),
                   "layer_caches": NL, "layer_calls_per_step": LPS, "global_batch": wl.batch,
                   "seq_len": wl.prompt_len, "routing": args.routing,
                   "routing_order": {0: "single stream", 1: "device-side gate", 2: "queue-level wait"}[order],
                   "routing_interval": R,
                   "init_scores": "prompt attention (qevict_prefill_scores, W observation queries)"
                   if observed else "synthetic", "rope_base": args.rope_base,
                   "parallelism": "single GPU"},
        "step_GBps": round(bytes_per_step / (ms_per_step * 1e-3) / 1e9, 1),
        "algorithmic_MB_per_step": round(bytes_per_step / 1e6, 3),
        "host_wall_us_per_step": round(wall / args.steps * 1e6, 2),
        "routing_tail_us": round(drain_us, 1),
        # moves per routing event of one sequence-layer (an event every R steps)
        "routing_per_event": {"promotions": round(promo / max(n_ev * wl.batch, 1), 2),
                              "reactivations": round(react / max(n_ev * wl.batch, 1), 2),
                              "evictions": round(evict / max(n_ev * wl.batch, 1), 2)},
    }
    if ps_ms:
        # latency of one initial-score call while the GPU is otherwise idle: HIP events
        # around the binding call, so its host-side marshalling and the three launches
        # are inside (kernel times: `bench.py --prefill-scores` and the profiles)
        res["prefill_scores_call_us"] = round(sum(ps_ms[1:] or ps_ms) / len(ps_ms[1:] or ps_ms) * 1e3, 1)
    if lp:
        per = {k: (lp[k][0] * 1e3 / lp[k][1] if lp[k][1] else None) for k in lp}
        if per[2] is not None:
            ev_us = per[2] + (per[3] or 0.0)
            # per layer routing event: event durations of the launches (each holds its
            # dispatch, about 2 us) over the layers they served (asynchronous routing
            # launches the events of a batch of layers together)
            res["routing_kernel_us"] = {"rerank": round(per[2], 2),
                                        "migrate": round(per[3], 2) if per[3] is not None else None}
            res["routing_us_per_event"] = round(ev_us, 2)
            # App. H cost model: routing cost per generated token = (T_rank + T_migrate) / R;
            # the scores are accumulated inside every step's attention (no separate pass)
            res["routing_us_per_token_amortized"] = round(ev_us / R, 3)
    if attn_events:
        attend_us = sum(ms for ms, _ in attn_events) * 1e3 / sum(n for _, n in attn_events)
        res["attend_us_per_launch"] = round(attend_us, 3)
        ach = bytes_per_call / (attend_us * 1e-6) / 1e9
        # the counter record was taken on the default run (8B / 32K workload, no RoPE,
        # library split count): other runs report no traffic
        default_run = args.workload == "c2" and args.rope_base == 0 and args.splits == 0
        rec = measured_traffic() if default_run else None
        traffic = None
        if rec:
            traffic = round(rec["hbm_bytes_per_launch"] / (attend_us * 1e-6) / 1e9, 1)
            res["traffic_MB_per_launch"] = round(rec["hbm_bytes_per_launch"] / 1e6, 3)
        res["roofline"] = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS,
                           "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4), "traffic": traffic}
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(wl, args.seed, args.cpu_seconds, LPS * wl.batch)
        res["cpu_baseline"]["host_cpus"] = n_cpu
        res["cpu_baseline"]["cpu_model"] = cpu_model
    print(json.dumps(res))
    cache.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
