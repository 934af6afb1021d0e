"""Benchmark: decode tokens/s of the DeepSeek-MoE-16B-shaped stack at a 50% expert cache.

The reported value: decode tokens/s of the DeepSeek-MoE-16B-shaped stack.
One step = one decode token (batch 1) through all 27 layers of the hot path:
attention surrogate, look-ahead prediction and speculative plan, gate + top-k +
precise plan, chunked high/low-priority copies from pinned host memory, expert
FFN over the cache slots in the route order, combine, residual.  Inputs (the
per-step hidden states) are resident in HBM before the timed region; expert
weights live where the method puts them: 32 of 64 experts per layer in the HBM
cache, all 64 in pinned host memory.

Speculative plans fill at most one slot each by default (--spec-fill-limit 1):
with the host link saturated, that is the configuration of the method that
measured fastest; the ablation leg reports the others, the unlimited fill of
the algorithm as written included.

Prints one JSON line.  The roofline entry is for the dominant kernel of that
workload (the decode FFN gate/up GEMV), with the down GEMV beside it; every
expert launch is timed by the start and end events the launch itself records
(hipExtLaunchKernelGGL), over the timed region.  The cpu_baseline entry times
the CPU oracle on a bounded sample of the same workload on this host.  Further
legs (in "detail"): every expert resident (the HBM-bound decode), the other
four workloads (Qwen1.5-MoE decode; Mixtral-8x7B and Qwen2-57B prefill and
decode at 4 bits over all their layers, and in bf16 over 16 of them), the
Qwen1.5-MoE prefill, the shared-expert MFMA GEMMs, the ablation, the cache-rate
and batch sweeps, 4-bit experts, offline predictor training, and the oracle
timed on each workload.  A compact summary line goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "decode & prefill tok/s at 50% expert cache; expert-FFN HBM GB/s, MFMA util"
KERNEL_CLASSES = ("gemv_gateup", "gemv_down", "gemm_gateup_routed", "gemm_down_routed", "gemm_gateup_shared",
                  "gemm_down_shared")
DEFAULT_LEGS = "decode,allres,prefill,configs,mfma,ablation,sweep,int4,predtrain,hbmsize,cpu"


def parse(argv=None):
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=128)
    p.add_argument("--warmup", type=int, default=8)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="bound on the headline oracle sample")
    p.add_argument("--cpu-config-seconds", type=float, default=6.0, help="bound on each other workload's sample")
    p.add_argument("--no-prefetch", action="store_true", help="reactive LRU (predictions ignored)")
    p.add_argument("--trained-predictor", action="store_true",
                   help="decode with look-ahead predictors trained offline on the model's own traces (other "
                        "inputs than the timed ones), as the paper trains its predictors; default: the "
                        "constructed skip predictor")
    p.add_argument("--spec-fill-limit", type=int, default=1,
                   help="slots a predicted plan may fill: 0 no limit, n>0 the first n, -1 none")
    p.add_argument("--copy-calib-mib", type=int, default=1024,
                   help="size of the plain device copy run after the timed region (counter calibration)")
    p.add_argument("--legs", default=DEFAULT_LEGS,
                   help="decode is always run (it is the reported value); the others: " + DEFAULT_LEGS)
    p.add_argument("--config-filter", default="", help="configs leg: run only the workloads whose name contains "
                                                         "this text (default: all)")
    p.add_argument("--prefill-steps", type=int, default=3)
    p.add_argument("--prefill-warmup", type=int, default=1)
    p.add_argument("--allres-steps", type=int, default=64)
    p.add_argument("--ablation-steps", type=int, default=32)
    p.add_argument("--sweep-steps", type=int, default=24)
    p.add_argument("--train-steps", type=int, default=64, help="predtrain leg: trace steps of 512 tokens")
    p.add_argument("--train-epochs", type=int, default=8)
    p.add_argument("--train-lr", type=float, default=3e-4)
    return p.parse_args(argv)


def read_traffic(kernel):
    """(HBM bytes per launch of `kernel`, those bytes over the algorithmic bytes of the same
    counter runs) from the committed counter summary, or (None, None) when the summary is
    missing or was taken on a different kernel source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_counters.txt")
    csrc = os.path.join(ROOT, "paper_2410_22134_amd", "csrc")
    if not os.path.exists(path):
        return None, None
    # the GEMV kernels' source and the device helpers they inline
    src = b"".join(open(os.path.join(csrc, f), "rb").read() for f in ("kernels_gemv.hip", "common.hpp"))
    digest = hashlib.sha256(src).hexdigest()[:16]
    for line in open(path):
        f = line.split()
        if len(f) >= 4 and f[0] == "traffic" and f[1] == kernel:
            if f[2] != digest:
                return None, None
            ratio = round(float(f[3]) / float(f[4]), 4) if len(f) >= 5 else None
            return int(float(f[3])), ratio
    return None, None


def traffic_here(ratio, cls):
    """HBM bytes per launch of this run: the counter runs' measured bytes over
    algorithmic bytes, applied to this run's algorithmic bytes per launch (the
    average launch differs between runs with the cache's hit pattern)."""
    if ratio is None or not cls.get("bytes_per_launch"):
        return None
    return int(round(ratio * cls["bytes_per_launch"]))


def prediction_metrics(s):
    """GoodPred = Accuracy x FetchRate (Sec. "A New Prediction Metric: GoodPred").
    Accuracy: predicted experts that the target layer routes (exact, device counters);
    FetchRate: of those, the ones whose bytes had all landed when the route ran;
    proactive coverage: fetched experts that a prediction brought in before the route."""
    acc = s["pred_correct"] / s["pred_n"] if s["pred_n"] else None
    fetch = s["pred_in_time"] / s["pred_correct"] if s["pred_correct"] else None
    fetched = s["spec_used"] + s["miss"]
    return {"accuracy": None if acc is None else round(acc, 4),
            "fetch_rate": None if fetch is None else round(fetch, 4),
            "goodpred": None if acc is None or fetch is None else round(acc * fetch, 4),
            "proactive_coverage": round(s["spec_used"] / fetched, 4) if fetched else None,
            "pred_n": s["pred_n"], "pred_correct": s["pred_correct"], "pred_in_time": s["pred_in_time"]}


def overlap_metrics(s, elapsed, h2d_gbs, deferred_issue=False):
    """Share of copy time hidden behind compute: H_time = 1 - stall / load, where stall is
    the compute stream's measured wait on copies and load = copied bytes at the link rate
    (the measured probe rate, or the rate this run itself achieved if that is higher);
    H_max = min(1, (elapsed - stall) / load) bounds it.  With deferred issue (no early
    preemption: a position's copies are issued only after the previous position's
    compute) a wait also covers copies that had not been issued when compute reached
    them, so stall is not a measure of hidden load: H_time is then reported as None."""
    copied = s["bytes_high"] + s["bytes_low"]
    rate = max(h2d_gbs or 0.0, copied / elapsed / 1e9 if elapsed > 0 else 0.0)
    load = copied / (rate * 1e9) if rate else 0.0
    stall = s["stall_ms"] * 1e-3
    if load <= 0:
        return None
    h_max = min(1.0, max(elapsed - stall, 0.0) / load)
    if deferred_issue:
        return {"load_s": round(load, 4), "stall_s": round(stall, 4), "H_time": None, "H_max": round(h_max, 4),
                "H_time_over_H_max": None, "note": "copies issued on access (no early preemption): undefined"}
    h_time = 1.0 - stall / load
    return {"load_s": round(load, 4), "stall_s": round(stall, 4), "H_time": round(h_time, 4),
            "H_max": round(h_max, 4), "H_time_over_H_max": round(h_time / h_max, 4) if h_max > 0 else None}


def kernel_classes(s):
    """Per kernel class: launches, average launch time (start/end events of each
    launch), algorithmic bytes and flops per launch, achieved GB/s and TFLOP/s, and
    the fraction of the nominal HBM or MFMA peak."""
    out = {}
    for i, nm in enumerate(KERNEL_CLASSES):
        n, ms, by, fl = s["k_launches"][i], s["k_ms"][i], s["k_bytes"][i], s["k_flops"][i]
        if n:
            gbs, tfs = by / (ms * 1e-3) / 1e9, fl / (ms * 1e-3) / 1e12
            out[nm] = {"launches": n, "avg_us": round(ms / n * 1e3, 3), "GBps": round(gbs, 1),
                       "TFLOPs": round(tfs, 1), "bytes_per_launch": round(by / n), "flops_per_launch": round(fl / n),
                       "frac_hbm": round(gbs / HBM_PEAK_GBPS, 4), "frac_mfma": round(tfs / MFMA_BF16_PEAK_TFLOPS, 4)}
    return out


def gemv_rate(s, classes=(0, 1)):
    """Achieved GB/s of the decode GEMVs over the given classes together (bytes over time)."""
    by = sum(s["k_bytes"][i] for i in classes)
    ms = sum(s["k_ms"][i] for i in classes)
    return by / (ms * 1e-3) / 1e9 if ms else 0.0


def h2d_probe(torch, mib=256, reps=5, pieces=8):
    """Pinned host -> device copy bandwidth (GB/s): `mib` MiB in `pieces` copies
    alternating over two streams, as the library's copy engine issues them
    (best of `reps`)."""
    n = mib << 20
    piece = n // pieces
    src = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    ss = (torch.cuda.Stream(), torch.cuda.Stream())
    best = 0.0
    for _ in range(reps):
        torch.cuda.synchronize()
        a, b, j = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        a.record(ss[0])
        ss[1].wait_event(a)
        for i in range(pieces):
            with torch.cuda.stream(ss[i % 2]):
                dst[i * piece:(i + 1) * piece].copy_(src[i * piece:(i + 1) * piece], non_blocking=True)
        j.record(ss[1])
        ss[0].wait_event(j)
        b.record(ss[0])
        b.synchronize()
        best = max(best, pieces * piece / (a.elapsed_time(b) * 1e-3) / 1e9)
    del src, dst
    return best


def measure_peaks(torch, hbm_gib=4, reps=5):
    """Achievable peaks of this GPU, measured with the library's probes: one
    streaming read of a buffer far larger than the 256 MB Infinity Cache (best of
    `reps`), and a register-only bf16 MFMA loop (two waves per SIMD)."""
    from paper_2410_22134_amd import _abi
    n = hbm_gib << 30
    buf = torch.zeros(n, dtype=torch.uint8, device="cuda")
    blocks = n // (32 << 10)            # 32 KiB contiguous per block
    sink = torch.empty(max(blocks, 1024 * 512), dtype=torch.float32, device="cuda")

    def timed(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) * 1e-3

    _abi.peak_hbm_read(buf, n, sink, blocks)
    t_hbm = min(timed(lambda: _abi.peak_hbm_read(buf, n, sink, blocks)) for _ in range(reps))
    del buf
    mblocks, iters = 1024, 2000
    flops = mblocks * 8 * iters * 32 * 16384.0
    _abi.peak_mfma_bf16(sink, mblocks, 100)
    t_mfma = min(timed(lambda: _abi.peak_mfma_bf16(sink, mblocks, iters)) for _ in range(3))
    torch.cuda.synchronize()
    return {"hbm_read_GBps": round(n / t_hbm / 1e9, 1), "hbm_read_bytes": n,
            "mfma_bf16_TFLOPs": round(flops / t_mfma / 1e12, 1),
            "how": "promoe_peak_hbm_read (16-byte non-temporal reads, 32 KiB contiguous per block, best of 5) and "
                   "promoe_peak_mfma_bf16 (32 independent 16x16x32 bf16 MFMAs per wave, 8 waves per block)"}


# ---------------------------------------------------------------- the oracle on the CPU
def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return len(os.sched_getaffinity(0))


def _oracle_step(cfg, model, lcs, h, t0, budget_s):
    """One step of T tokens (h [T, H] float64) through the oracle's layers, stopping
    after the layer that passes the budget; returns the layers done."""
    import numpy as np
    from oracle import bf16 as obf
    from oracle import ffn as offn
    from oracle import predictor as opred
    from oracle import quant as oquant
    from oracle import router as orouter
    from oracle import stack as ostack
    from synth import model as sm
    layers = 0
    for l in range(cfg.n_layers):
        if cfg.attn_surrogate:
            h = ostack.attn_surrogate(h, obf.decode(sm.attn(cfg, l)), cfg.dtype)
        x = ostack.moe_input(h, cfg.dtype)
        pred = model.np_pred[l]
        tgt = sm.predictor_target(cfg, l)
        if pred is not None and tgt is not None:
            q = opred.logits(x, obf.decode(pred[0]), None if pred[1] is None else obf.decode(pred[1]))
            Q, votes, _ = opred.vote(opred.per_token(q, cfg.top_k), cfg.n_experts, cfg.slots)
            lcs[tgt].spec_plan(Q, voted=np.nonzero(votes)[0].tolist())
        z = orouter.gate_logits(x, obf.decode(model.np_gate[l]), model.np_bias[l])
        ids, w, _ = orouter.route(z, cfg.top_k, bool(cfg.renorm))
        lcs[l].precise_plan(np.unique(ids).tolist())

        def expert_fn(e, l=l):
            if cfg.weight_format == "int4":
                return oquant.decode_expert(model.expert_host(l, e), cfg.inter, cfg.hidden)
            wg, wu, wd = sm.expert_from_bytes(cfg, model.expert_host(l, e))
            return obf.decode(wg), obf.decode(wu), obf.decode(wd)
        parts = [tuple(obf.decode(m) for m in p) for p in sm.shared_parts(cfg, l)]
        s = None
        if cfg.n_shared and cfg.shared_gate:
            s = orouter.shared_scale(x, obf.decode(model.np_sgate[l]))
        y = offn.round_out(offn.moe_forward(x, ids, w, expert_fn, cfg.dtype == "bf16", parts or None, s), cfg.dtype)
        h = h + y
        layers += 1
        if time.perf_counter() - t0 > budget_s:
            break
    return layers


def oracle_rate(cfg, model, T, budget_s, seed0=10_000, threads=None):
    """tok/s of the oracle on consecutive steps of T tokens (every layer of each) until
    the budget is spent, scaled to whole steps; the last step may stop part-way."""
    from oracle import cache as ocache
    from synth import model as sm
    lcs = [ocache.LayerCache(cfg.n_experts, cfg.slots) for _ in range(cfg.n_layers)]
    t0 = time.perf_counter()
    layers = steps = 0
    while time.perf_counter() - t0 <= budget_s:
        layers += _oracle_step(cfg, model, lcs, sm.stack_input(cfg, seed0 + steps, T).astype("float64"), t0, budget_s)
        steps += 1
    dt = time.perf_counter() - t0
    per_step = dt / layers * cfg.n_layers
    return {"value": round(T / per_step, 4), "unit": "tok/s", "cores": int(threads or _blas_threads()),
            "kind": "oracle", "sample": f"{layers} layers ({layers / cfg.n_layers:.2f} steps of {T} tokens over "
                                        f"{cfg.n_layers} layers), float64 NumPy, {dt:.1f} s, scaled to whole steps"}


def cpu_baseline(cfg, model, budget_s):
    """The oracle on the headline workload (decode tokens of batch 1), plus its
    single-thread rate on a shorter sample."""
    out = oracle_rate(cfg, model, 1, budget_s)
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            one = oracle_rate(cfg, model, 1, budget_s / 3, seed0=20_000, threads=1)
        out["single_thread_value"] = one["value"]
        out["single_thread_sample"] = one["sample"] + ", one BLAS thread"
    except Exception as e:  # threadpoolctl missing or unable to limit: report the main figure only
        out["single_thread_value"] = None
        out["single_thread_sample"] = f"not measured ({type(e).__name__})"
    return out


# ---------------------------------------------------------------- GPU legs
def run_steps(torch, model, st, inputs, warmup, steps):
    for i in range(warmup):
        st.step(inputs[i])
    model.ctx.sync()
    torch.cuda.synchronize()
    model.ctx.reset_stats()
    t0 = time.perf_counter()
    for i in range(steps):
        st.step(inputs[warmup + i])
    model.ctx.sync()
    torch.cuda.synchronize()
    return time.perf_counter() - t0, model.ctx.stats()


def _inputs(torch, cfg, seed0, n, T):
    import numpy as np
    from synth import model as sm
    return torch.from_numpy(np.stack([sm.stack_input(cfg, seed0 + i, T) for i in range(n)])).cuda()


def leg_allres(torch, args, model):
    """Every expert resident (64 of 64 slots per layer, nothing copied): the decode of
    the DeepSeek-MoE-16B shape is bound by HBM.  tok/s against the weight-streaming
    ceiling, and the decode GEMVs' rates at their largest launches (one gate/up
    launch of six experts and the shared expert per layer, and one down launch).
    `model` is the headline decode's model, re-opened with every slot."""
    from paper_2410_22134_amd import FLAG_PROFILE
    from paper_2410_22134_amd.stack import Stack
    model.max_tokens = 1
    cfg = model.cfg.with_(slots=model.cfg.n_experts)
    h = _inputs(torch, cfg, 8000, 8 + args.allres_steps, 1)
    # tok/s without launch timing (a launch that records its own start and end
    # events costs the host ~3x a plain one, and this step is bound by the
    # host's issue of small launches); then the same steps timed per launch
    runs = {}
    for flags in (0, FLAG_PROFILE):
        model.open(flags=flags, spec_fill_limit=args.spec_fill_limit, slots=cfg.n_experts)
        st = Stack(model, 1)
        runs[flags] = run_steps(torch, model, st, h, 8, args.allres_steps)
        del st
    (dt, _), (dt_p, s) = runs[0], runs[FLAG_PROFILE]
    per_token = (cfg.top_k * cfg.expert_bytes + 3 * cfg.shared_total * cfg.hidden * 2) * cfg.n_layers
    tok_s = args.allres_steps / dt
    ceiling = HBM_PEAK_GBPS * 1e9 / per_token
    return {"workload": "DeepSeek-MoE-16B-shaped decode, batch 1, 27 layers, all 64 experts per layer in HBM",
            "tok_s": round(tok_s, 2), "ms_per_step": round(dt / args.allres_steps * 1e3, 3),
            "tok_s_with_launch_timing": round(args.allres_steps / dt_p, 2),
            "expert_bytes_per_token": per_token, "hbm_ceiling_tok_s": round(ceiling, 1),
            "of_ceiling": round(tok_s / ceiling, 4),
            "copied_GB": round((s["bytes_high"] + s["bytes_low"]) / 1e9, 3), "miss": s["miss"],
            "lazy_routes": s["lazy_routes"],
            "gemv_GBps": round(gemv_rate(s), 1), "gemv_frac": round(gemv_rate(s) / HBM_PEAK_GBPS, 4),
            "kernels": kernel_classes(s)}


def leg_prefill(torch, args, flags, limit, model, cpu=False):
    """Qwen1.5-MoE-A2.7B shape, 24 layers, 512-token prompt, 30 of 60 experts cached
    (`model`: that shape with max_tokens >= 512)."""
    from paper_2410_22134_amd.stack import Stack
    T = 512
    model.open(flags=flags, spec_fill_limit=limit)
    cfg = model.cfg
    st = Stack(model, T)
    h = _inputs(torch, cfg, 1000, args.prefill_warmup + args.prefill_steps, T)
    dt, s = run_steps(torch, model, st, h, args.prefill_warmup, args.prefill_steps)
    out = {"workload": "Qwen1.5-MoE-A2.7B-shaped stack prefill: 24 layers, hidden 2048, 60 routed experts "
                       "(I=1408) top-4 + gated shared expert (I=5632), 512-token prompt, 30 of 60 experts "
                       "per layer cached, look-ahead 2",
           "tok_s": round(T * args.prefill_steps / dt, 1), "ms_per_step": round(dt / args.prefill_steps * 1e3, 2),
           "copied_GB": round((s["bytes_high"] + s["bytes_low"]) / 1e9, 3),
           "copy_GBps_over_timed_region": round((s["bytes_high"] + s["bytes_low"]) / dt / 1e9, 2),
           "hit": s["hit"], "miss": s["miss"], "kernels": kernel_classes(s)}
    if cpu and not args.no_cpu_baseline:
        out["cpu_oracle"] = oracle_rate(cfg, model, T, args.cpu_config_seconds, seed0=30_000)
    return out


def leg_ablation(torch, args, name, model, slots):
    """The paper's ablation steps and baselines (LRU; + prefetch, chunked prefetch,
    early preemption, reordered inference; static cache; reactive with every other
    technique on; the unlimited and limit-1 speculative fills) on one workload
    ("decode": DeepSeek-16B shape, batch 1; "prefill": Qwen1.5-MoE shape, 512
    tokens), one context per mode over the same weights, `slots` cached per layer."""
    from paper_2410_22134_amd import ABLATION, FLAG_FILL_BY_DEADLINE, FLAG_NO_PREFETCH
    from paper_2410_22134_amd.stack import Stack
    modes = [(k, f, 0) for k, f in ABLATION.items()] + [("+cer (no prefetch)", FLAG_NO_PREFETCH, 0),
                                                         ("+pcer fill limit 1", 0, 1),
                                                         ("+pcer fill by deadline", FLAG_FILL_BY_DEADLINE, 0)]
    T, warm, steps = (1, 4, args.ablation_steps) if name == "decode" else (512, 1, 2)
    cfg = model.cfg
    st = Stack(model, T)
    h = _inputs(torch, cfg, 3000, warm + steps, T)
    res = {}
    for mode, flags, lim in modes:
        model.open(flags=flags, spec_fill_limit=lim, slots=slots)
        dt, s = run_steps(torch, model, st, h, warm, steps)
        res[mode] = {"tok_s": round(T * steps / dt, 2),
                     "copied_GB": round((s["bytes_high"] + s["bytes_low"]) / 1e9, 3),
                     "hit": s["hit"], "miss": s["miss"], "spec_wasted": s["spec_wasted"]}
        print(f"[bench] ablation {name} {mode}: {res[mode]}", file=sys.stderr, flush=True)
    return res


def leg_sweep(torch, args, model):
    """Cache-rate sweep (25-90% of the experts cached, batch 1) and batch sweep
    (1-8 tokens per step at 50%) of the DeepSeek-MoE-16B-shaped decode, for the
    method (fill limit as configured) and reactive LRU, on the headline model."""
    from paper_2410_22134_amd import FLAG_FILL_BY_DEADLINE, FLAG_NO_PREFETCH, FLAG_PROFILE
    from paper_2410_22134_amd.stack import Stack
    cfg = model.cfg
    E, warm, steps = cfg.n_experts, 4, args.sweep_steps
    modes = (("method", 0, args.spec_fill_limit), ("deadline", FLAG_FILL_BY_DEADLINE, 0),
             ("reactive", FLAG_NO_PREFETCH, 0))
    model.max_tokens = 8
    out = {"cache_rate": [], "batch": []}

    def one(T, slots, flags, lim):
        model.open(flags=flags | FLAG_PROFILE, spec_fill_limit=lim, slots=slots)
        st = Stack(model, T)
        h = _inputs(torch, cfg, 4000, warm + steps, T)
        dt, s = run_steps(torch, model, st, h, warm, steps)
        copied = s["bytes_high"] + s["bytes_low"]
        return {"tok_s": round(T * steps / dt, 2), "copied_GB_per_step": round(copied / steps / 1e9, 3),
                "hit_rate": round(s["hit"] / max(1, s["prec_access"]), 4),
                "overlap": overlap_metrics(s, dt, 56.7), "prediction": prediction_metrics(s)}
    try:
        for frac in (0.25, 0.5, 0.75, 0.9):
            C = int(round(frac * E))
            row = {"cached": f"{C}/{E}"}
            for mode, flags, lim in modes:
                row[mode] = one(1, C, flags, lim)
            print(f"[bench] sweep cache {C}/{E}: method {row['method']['tok_s']}, deadline {row['deadline']['tok_s']}, "
                  f"reactive {row['reactive']['tok_s']} tok/s", file=sys.stderr, flush=True)
            out["cache_rate"].append(row)
        for T in (1, 2, 4, 8):
            row = {"batch": T}
            for mode, flags, lim in modes:
                row[mode] = one(T, E // 2, flags, lim)
            print(f"[bench] sweep batch {T}: method {row['method']['tok_s']}, deadline {row['deadline']['tok_s']}, "
                  f"reactive {row['reactive']['tok_s']} tok/s", file=sys.stderr, flush=True)
            out["batch"].append(row)
    finally:
        model.max_tokens = 1
    return out


def train_decode_predictors(torch, model, args, steps=64, T=512):
    """Train the decode model's look-ahead predictors offline (before the timed
    region): routing traces of `steps` x `T` tokens from the model's own forward
    pass with every expert resident (inputs from other seeds than the timed
    ones), then each layer's MLP fitted as in the predtrain leg."""
    import numpy as np
    from paper_2410_22134_amd import train_predictor as tp
    cfg = model.cfg
    t0 = time.perf_counter()
    keep = model.max_tokens
    model.max_tokens = T
    model.open(slots=cfg.n_experts)
    xs, ids = tp.collect_traces(model, steps, T)
    model.max_tokens = keep
    res = tp.train_all(model, xs, ids, cfg.lookahead, epochs=args.train_epochs, lr=args.train_lr)
    del xs, ids
    tp.install(model, res)
    a0 = float(np.mean([m["acc_start"] for _, _, m in res.values()]))
    a1 = float(np.mean([m["acc_trained"] for _, _, m in res.values()]))
    took = time.perf_counter() - t0
    print(f"[bench] decode predictors trained in {took:.1f} s: held-out accuracy {a0:.3f} -> {a1:.3f}",
          file=sys.stderr, flush=True)
    return {"trace_tokens": steps * T, "seconds": round(took, 1), "heldout_acc_constructed": round(a0, 4),
            "heldout_acc_trained": round(a1, 4)}


def leg_predtrain(torch, args, model):
    """Offline predictor training on synthetic traces (DeepSeek-MoE-16B shape, the
    headline model): traces from the library's forward pass with every expert
    resident, 9:1 split, look-ahead 1 and 2; then the decode workload (50% cached)
    with the trained look-ahead-1 predictors against the constructed ones (the
    constructed ones are put back afterwards)."""
    import numpy as np
    from paper_2410_22134_amd import FLAG_PROFILE
    from paper_2410_22134_amd import train_predictor as tp
    from paper_2410_22134_amd.stack import Stack
    T = 512
    model.max_tokens = T
    model.open(slots=model.cfg.n_experts)
    cfg = model.cfg
    keep = (list(model.d_pred), list(model.np_pred))
    out = {"trace_tokens": args.train_steps * T, "epochs": args.train_epochs}
    try:
        t0 = time.perf_counter()
        xs, ids = tp.collect_traces(model, args.train_steps, T)
        out["trace_s"] = round(time.perf_counter() - t0, 1)
        trained = {}
        for d in (1, 2):
            t0 = time.perf_counter()
            res = tp.train_all(model, xs, ids, d, epochs=args.train_epochs, lr=args.train_lr)
            a0 = [m["acc_start"] for _, _, m in res.values()]
            a1 = [m["acc_trained"] for _, _, m in res.values()]
            out[f"lookahead_{d}"] = {
                "layers": len(res), "train_s": round(time.perf_counter() - t0, 1),
                "heldout_acc_constructed": {"mean": round(float(np.mean(a0)), 4), "min": round(float(np.min(a0)), 4),
                                            "max": round(float(np.max(a0)), 4)},
                "heldout_acc_trained": {"mean": round(float(np.mean(a1)), 4), "min": round(float(np.min(a1)), 4),
                                        "max": round(float(np.max(a1)), 4)},
                "train_split_acc_trained_mean": round(float(np.mean([m["acc_train"] for _, _, m in res.values()])), 4),
                "per_layer_trained": [round(x, 3) for x in a1]}
            print(f"[bench] predtrain d={d}: held-out accuracy {np.mean(a0):.3f} -> {np.mean(a1):.3f} (train split "
                  f"{out[f'lookahead_{d}']['train_split_acc_trained_mean']:.3f})",
                  file=sys.stderr, flush=True)
            trained[d] = res
        del xs, ids
        # runtime: decode at 50% cached, constructed vs trained look-ahead-1 predictors
        st = Stack(model, 1)
        n = 4 + args.sweep_steps * 2
        h = _inputs(torch, cfg, 6000, n, 1)
        runtime = {}
        for name in ("constructed", "trained"):
            if name == "trained":
                tp.install(model, trained[1])
            model.open(flags=FLAG_PROFILE, spec_fill_limit=args.spec_fill_limit, slots=cfg.n_experts // 2)
            dt, s = run_steps(torch, model, st, h, 4, n - 4)
            runtime[name] = {"tok_s": round((n - 4) / dt, 2), "hit_rate": round(s["hit"] / max(1, s["prec_access"]), 4),
                             "prediction": prediction_metrics(s)}
            print(f"[bench] predtrain runtime {name}: {runtime[name]['tok_s']} tok/s, accuracy "
                  f"{runtime[name]['prediction']['accuracy']}, GoodPred {runtime[name]['prediction']['goodpred']}",
                  file=sys.stderr, flush=True)
        out["decode_50pct_fill_limit"] = args.spec_fill_limit
        out["decode_50pct"] = runtime
    finally:
        model.d_pred, model.np_pred = keep
        model.max_tokens = 1
    return out


# The other workloads: (name, config, layers run, weight format, oracle timed,
# runs).  Runs are (kind, tokens per step, warm-up steps, timed steps); decode
# follows the prefill on the cache it left, as in serving.  A process may pin at
# most 64 GiB of host memory on these machines: 4-bit experts (the paper's
# precision for the Mixtral and Qwen2-57B models) fit at full depth (23 and 26
# GB), bf16 ones (90 and 99 GB) only over 16 layers.
CONFIG_PLAN = (
    ("Qwen1.5-MoE-A2.7B", "C3", None, "dense", True, (("decode", 1, 4, 24),)),
    ("Mixtral-8x7B int4", "C4", None, "int4", True, (("prefill", 256, 1, 2), ("decode", 1, 2, 8))),
    ("Qwen2-57B-A14B int4", "C5", None, "int4", True, (("prefill", 1024, 1, 2), ("decode", 1, 2, 8),
                                                        ("decode", 8, 2, 8))),
    ("Mixtral-8x7B bf16 (16 layers)", "C4", 16, "dense", False, (("prefill", 256, 1, 2), ("decode", 1, 2, 6))),
    ("Qwen2-57B-A14B bf16 (16 layers)", "C5", 16, "dense", False, (("prefill", 1024, 1, 2), ("decode", 1, 2, 6),
                                                                   ("decode", 8, 2, 6))),
)


def leg_configs(torch, args, h2d_gbs, cpu=False):
    """The other workloads at their real per-layer sizes (see CONFIG_PLAN).  Per run:
    tok/s, host-to-device GB per step, hit rate, overlap, the link bound (tokens per
    step over bytes per step at the measured copy rate) and the expert kernels'
    rates; with `cpu`, the oracle timed on a bounded sample of each workload."""
    from synth import configs
    from paper_2410_22134_amd import FLAG_PROFILE
    from paper_2410_22134_amd.model import SyntheticModel
    from paper_2410_22134_amd.stack import Stack
    out = {}
    for name, key, n_layers, fmt, timed_oracle, runs in CONFIG_PLAN:
        if args.config_filter and args.config_filter not in name:
            continue
        full = getattr(configs, key)
        cfg = full.with_(n_layers=n_layers or full.n_layers, weight_format=fmt)
        t0 = time.perf_counter()
        model = SyntheticModel(cfg, max_tokens=max(T for _, T, _, _ in runs), gen_threads=8,
                               flags=FLAG_PROFILE, spec_fill_limit=args.spec_fill_limit)
        setup = time.perf_counter() - t0
        print(f"[bench] configs {name}: weights generated in {setup:.1f} s", file=sys.stderr, flush=True)
        rows = []
        try:
            for kind, T, warm, steps in runs:
                st = Stack(model, T)
                h = _inputs(torch, cfg, 6000, warm + steps, T)
                dt, s = run_steps(torch, model, st, h, warm, steps)
                copied = (s["bytes_high"] + s["bytes_low"]) / steps
                row = {"workload": kind, "tokens_per_step": T, "steps": steps, "tok_s": round(T * steps / dt, 2),
                       "ms_per_step": round(dt / steps * 1e3, 2), "copied_GB_per_step": round(copied / 1e9, 3),
                       "copy_GBps": round(copied * steps / dt / 1e9, 2),
                       "link_bound_tok_s": round(T / (copied / (h2d_gbs * 1e9)), 2) if copied else None,
                       "hit_rate": round(s["hit"] / max(1, s["prec_access"]), 4),
                       "overlap": overlap_metrics(s, dt, h2d_gbs), "prediction": prediction_metrics(s),
                       "kernels": kernel_classes(s)}
                if cpu and timed_oracle and not args.no_cpu_baseline:
                    row["cpu_oracle"] = oracle_rate(cfg, model, T, args.cpu_config_seconds, seed0=30_000)
                rows.append(row)
                print(f"[bench] configs {name} {kind} T={T}: {row['tok_s']} tok/s over {cfg.n_layers} layers "
                      f"(link bound {row['link_bound_tok_s']})", file=sys.stderr, flush=True)
                del st, h
        finally:
            model.close()
        out[name] = {"layers_run": cfg.n_layers, "layers_full": full.n_layers, "weights": fmt,
                     "experts": cfg.n_experts, "top_k": cfg.top_k, "cached_per_layer": cfg.slots,
                     "expert_MB": round(cfg.expert_bytes / 1e6, 2), "setup_s": round(setup, 1), "runs": rows}
    return out


def leg_int4(torch, args):
    """4-bit routed experts (the paper's bits-per-weight study): decode of the
    DeepSeek-MoE-16B shape (50% cached) and 512-token prefill of the
    Qwen1.5-MoE shape, under the LRU baseline, the method (unlimited fills and
    fill limit 1) and reactive; plus the dequantising GEMV's rate."""
    from synth import configs
    from paper_2410_22134_amd import ABLATION, FLAG_FILL_BY_DEADLINE, FLAG_NO_PREEMPT, FLAG_NO_PREFETCH, FLAG_PROFILE
    from paper_2410_22134_amd.model import SyntheticModel
    from paper_2410_22134_amd.stack import Stack
    modes = (("lru", ABLATION["lru"], 0), ("+pcer", 0, 0), ("+pcer fill limit 1", 0, 1),
             ("+pcer fill by deadline", FLAG_FILL_BY_DEADLINE, 0), ("+cer (no prefetch)", FLAG_NO_PREFETCH, 0))
    out = {}
    for name, base, T, warm, steps in (("decode", configs.C2, 1, 4, args.ablation_steps * 2),
                                       ("prefill", configs.C3, 512, 1, 2)):
        cfg = base.with_(weight_format="int4")
        model = SyntheticModel(cfg, max_tokens=T, gen_threads=8)
        try:
            st = Stack(model, T)
            h = _inputs(torch, cfg, 7000, warm + steps, T)
            res = {"expert_MB": round(cfg.expert_bytes / 1e6, 3)}
            for mode, flags, lim in modes:
                model.open(flags=flags | FLAG_PROFILE, spec_fill_limit=lim)
                dt, s = run_steps(torch, model, st, h, warm, steps)
                r = {"tok_s": round(T * steps / dt, 2),
                     "copied_GB": round((s["bytes_high"] + s["bytes_low"]) / 1e9, 3),
                     "hit": s["hit"], "miss": s["miss"],
                     "overlap": overlap_metrics(s, dt, 56.7, deferred_issue=bool(flags & FLAG_NO_PREEMPT))}
                if name == "decode":
                    r["kernels"] = kernel_classes(s)
                res[mode] = r
                print(f"[bench] int4 {name} {mode}: {r['tok_s']} tok/s, {r['copied_GB']} GB", file=sys.stderr,
                      flush=True)
            out[name] = res
        finally:
            model.close()
    return out


def leg_mfma(torch, args):
    """Shared-expert GEMMs at the Qwen2-57B-A14B shape (hidden 3584, shared I = 20480),
    1024-token prefill, two layers with every expert resident (compute only)."""
    from synth import configs
    from paper_2410_22134_amd import FLAG_PROFILE
    from paper_2410_22134_amd.model import SyntheticModel
    from paper_2410_22134_amd.stack import Stack
    base = configs.C5
    cfg = base.with_(n_layers=2, slots=base.n_experts)
    T = 1024
    model = SyntheticModel(cfg, max_tokens=T, flags=FLAG_PROFILE, gen_threads=8)
    try:
        st = Stack(model, T)
        h = _inputs(torch, cfg, 2000, 4, T)
        dt, s = run_steps(torch, model, st, h, 1, 3)
        cls = kernel_classes(s)
        fl = s["k_flops"][4] + s["k_flops"][5]
        ms = s["k_ms"][4] + s["k_ms"][5]
        tf = fl / (ms * 1e-3) / 1e12 if ms else 0.0
        return {"bound": "mfma", "kernel": "k_gemm_ffn (shared expert, gate/up + down)",
                "achieved": round(tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
                "workload": "Qwen2-57B-A14B shape: M = 1024 tokens, hidden 3584, shared I = 20480, bf16",
                "timing": "kernel start and end events recorded by each launch", "kernels": cls}
    finally:
        model.close()


def leg_hbm_sizes(torch, reps=20):
    """The library's streaming-read probe (contiguous 32 KiB per block) at the byte
    counts of single decode GEMV launches: what a kernel that only streams
    reaches at each launch size.  Each size runs `reps` launches over fresh parts
    of a 4 GiB buffer (no cache reuse), queued behind two full reads of the
    buffer so that they run back to back; the batch is timed with events (per
    launch: the kernel and the gap to the next one).  Kernel-only durations come
    from a rocprofv3 kernel trace of the same run."""
    from paper_2410_22134_amd import _abi
    G = 4 << 30
    buf = torch.empty(G, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.empty(G // (32 << 10), dtype=torch.float32, device="cuda")
    out = []
    off = 0
    for mb in (11.5, 23.1, 34.6, 46.1, 69.2, 92.3, 138.4, 276.8, 1024.0):
        n = int(mb * 1e6) // 4096 * 4096
        blocks = max(1, n // (32 << 10))
        offs = []
        for _ in range(reps):
            if off + n > G:
                off = 0
            offs.append(off)
            off += n
        _abi.peak_hbm_read(buf.data_ptr() + offs[0], n, sink, blocks)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        for _ in range(2):  # ~1.2 ms of queued work while the host enqueues the batch
            _abi.peak_hbm_read(buf, G, sink, G // (32 << 10))
        a.record()
        for o in offs:
            _abi.peak_hbm_read(buf.data_ptr() + o, n, sink, blocks)
        b.record()
        b.synchronize()
        us = a.elapsed_time(b) * 1e3 / reps
        out.append({"MB": mb, "blocks": blocks, "us_per_launch_back_to_back": round(us, 2),
                    "GBps": round(n / (us * 1e-6) / 1e9, 1), "frac": round(n / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)})
    del buf, sink
    return out


def summary_line(out):
    """One compact line of the secondary figures (stderr)."""
    d = out["detail"]
    r = out["roofline"]
    parts = [f"decode {out['value']} tok/s", f"GEMV gateup {r['frac']:.3f} down {r['down']['frac']:.3f} of HBM"]
    ov, pr = d.get("overlap") or {}, d.get("prediction") or {}
    if ov.get("H_time_over_H_max") is not None:
        parts.append(f"H_time/H_max {ov['H_time_over_H_max']:.2f}")
    if pr.get("goodpred") is not None:
        parts.append(f"GoodPred {pr['goodpred']:.3f} (acc {pr['accuracy']:.3f})")
    if "allres" in d:
        a = d["allres"]
        k = a["kernels"]
        parts.append(f"all-resident {a['tok_s']} tok/s ({a['of_ceiling']:.2f} of HBM ceiling), GEMV gateup "
                     f"{k.get('gemv_gateup', {}).get('frac_hbm', 0):.3f} down "
                     f"{k.get('gemv_down', {}).get('frac_hbm', 0):.3f}")
    if "prefill" in d:
        parts.append(f"QW1.5 prefill {d['prefill']['tok_s']} tok/s")
    if "roofline_prefill_gemm" in out:
        parts.append(f"shared GEMM {out['roofline_prefill_gemm']['frac']:.3f} of MFMA")
    for name, c in d.get("configs", {}).items():
        runs = ", ".join(f"{x['workload']}{'' if x['workload'] == 'prefill' else ' b' + str(x['tokens_per_step'])} "
                         f"{x['tok_s']}" for x in c["runs"])
        parts.append(f"{name}: {runs}")
    if "predictor_training" in d and "lookahead_1" in d["predictor_training"]:
        p = d["predictor_training"]
        parts.append(f"trained predictor held-out acc d1 {p['lookahead_1']['heldout_acc_trained']['mean']:.3f} "
                     f"d2 {p['lookahead_2']['heldout_acc_trained']['mean']:.3f}")
    if "cpu_baseline" in out:
        parts.append(f"oracle {out['cpu_baseline']['value']} tok/s")
    return "[bench] summary: " + "; ".join(parts)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (expert-parallel sharding "
              "is a design note); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    from synth import configs
    from paper_2410_22134_amd import FLAG_NO_PREFETCH, FLAG_PROFILE
    from paper_2410_22134_amd.model import SyntheticModel
    from paper_2410_22134_amd.stack import Stack

    legs = set(args.legs.split(","))
    torch.cuda.set_device(0)
    cfg = configs.C2
    flags = FLAG_PROFILE | (FLAG_NO_PREFETCH if args.no_prefetch else 0)
    t_setup = time.perf_counter()
    model = SyntheticModel(cfg, max_tokens=1, flags=flags, gen_threads=8, spec_fill_limit=args.spec_fill_limit)
    train_info = None
    if args.trained_predictor:
        train_info = train_decode_predictors(torch, model, args)
        model.open(flags=flags, spec_fill_limit=args.spec_fill_limit, slots=configs.C2.slots)
    st = Stack(model, 1)
    h_in = _inputs(torch, cfg, 0, args.warmup + args.steps, 1)
    setup_s = time.perf_counter() - t_setup
    print(f"[bench] decode: setup {setup_s:.1f}s; {args.warmup} warm-up + {args.steps} timed steps",
          file=sys.stderr, flush=True)
    elapsed, s = run_steps(torch, model, st, h_in, args.warmup, args.steps)
    tok_s = args.steps / elapsed

    cls = kernel_classes(s)
    gu, dn = cls.get("gemv_gateup", {}), cls.get("gemv_down", {})
    copy_bytes = s["bytes_high"] + s["bytes_low"]
    h2d_gbs = h2d_probe(torch)
    # the link moved at least what this run moved: never price the load below it
    h2d_eff = max(h2d_gbs, copy_bytes / elapsed / 1e9)
    peaks = measure_peaks(torch)
    load_s = s["bytes_high"] / (h2d_eff * 1e9) if h2d_eff else 0.0
    traffic, traffic_ratio = read_traffic("k_ffn_gateup")
    traffic_d, traffic_ratio_d = read_traffic("k_ffn_down")
    hbm_meas = peaks["hbm_read_GBps"]

    def roof(c):
        return {"achieved": c.get("GBps", 0.0), "frac": c.get("frac_hbm", 0.0),
                "frac_of_measured": round(c.get("GBps", 0.0) / hbm_meas, 4) if hbm_meas else None,
                "avg_launch_us": c.get("avg_us", 0.0), "bytes_per_launch": c.get("bytes_per_launch", 0),
                "launches": c.get("launches", 0)}

    both = gemv_rate(s)
    out = {
        "metric": METRIC,
        "value": round(tok_s, 3),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) hidden states)",
        "config": {"workload": "DeepSeek-MoE-16B-shaped stack decode, batch 1: 27 layers, hidden 2048, 64 routed "
                               "experts (I=1408) top-6 + 2 shared, 32 of 64 experts per layer cached in HBM, "
                               "the rest in pinned host memory, look-ahead 1, 2-layer MLP predictor",
                   "global_batch": 1, "seq_len": 1, "parallelism": "none (1 GPU)",
                   "prefetch": not args.no_prefetch, "spec_fill_limit": args.spec_fill_limit,
                   "predictor": "trained offline on the model's traces" if args.trained_predictor else
                                "constructed skip predictor"},
        "roofline": {"bound": "hbm", "kernel": "k_ffn_gateup<bf16,1,4,1>", **roof(gu),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "traffic": traffic_here(traffic_ratio, gu),
                     "traffic_over_algorithmic": traffic_ratio, "traffic_in_counter_runs": traffic,
                     "peak_measured": hbm_meas,
                     "down": {"kernel": "k_ffn_down<bf16,1,3,2>", **roof(dn),
                              "traffic": traffic_here(traffic_ratio_d, dn),
                              "traffic_over_algorithmic": traffic_ratio_d, "traffic_in_counter_runs": traffic_d},
                     "gateup_and_down": {"achieved": round(both, 1), "frac": round(both / HBM_PEAK_GBPS, 4)},
                     "timing": "kernel start and end events recorded by each launch (hipExtLaunchKernelGGL), "
                               "averaged over every launch of the timed region"},
        "detail": {
            "decode_kernels": cls,
            "h2d_copy_GBps_measured_256MiB": round(h2d_gbs, 2),
            "h2d_GBps_for_overlap": round(h2d_eff, 2),
            "measured_peaks": peaks,
            "copied_GB": round(copy_bytes / 1e9, 3),
            "copy_GBps_over_timed_region": round(copy_bytes / elapsed / 1e9, 2),
            "hit": s["hit"], "miss": s["miss"], "prec_access": s["prec_access"],
            "spec_issued": s["spec_issued"], "spec_used": s["spec_used"], "spec_wasted": s["spec_wasted"],
            "low_purged_subcopies": s["low_purged"],
            "prediction": prediction_metrics(s),
            "overlap": overlap_metrics(s, elapsed, h2d_eff),
            "stall_s": round(s["stall_ms"] * 1e-3, 4), "miss_load_s_at_measured_h2d": round(load_s, 4),
            "setup_s": round(setup_s, 1),
        },
    }
    if train_info is not None:
        out["detail"]["predictor_training"] = train_info
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(cfg, model, args.cpu_seconds)
    del st, h_in
    # plain device copy of known size (FETCH_SIZE / WRITE_SIZE calibration under rocprofv3 --pmc)
    n = args.copy_calib_mib << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    del a, b
    # legs over the headline model's weights (DeepSeek-16B shape), re-opened per policy
    try:
        if "allres" in legs:
            print("[bench] all-resident decode leg", file=sys.stderr, flush=True)
            out["detail"]["allres"] = leg_allres(torch, args, model)
        if "sweep" in legs:
            print("[bench] sweep leg", file=sys.stderr, flush=True)
            out["detail"]["sweep"] = leg_sweep(torch, args, model)
        if "ablation" in legs:
            print("[bench] ablation leg (decode)", file=sys.stderr, flush=True)
            out["detail"]["ablation"] = {"decode": leg_ablation(torch, args, "decode", model, cfg.slots)}
        if "predtrain" in legs:
            print("[bench] predictor training leg", file=sys.stderr, flush=True)
            out["detail"]["predictor_training"] = leg_predtrain(torch, args, model)
    finally:
        model.close()
    del model
    # legs over the Qwen1.5-MoE shape's weights
    if "prefill" in legs or "ablation" in legs:
        model3 = SyntheticModel(configs.C3, max_tokens=512, flags=flags, gen_threads=8,
                                spec_fill_limit=args.spec_fill_limit)
        try:
            if "prefill" in legs:
                print("[bench] prefill leg", file=sys.stderr, flush=True)
                out["detail"]["prefill"] = leg_prefill(torch, args, flags, args.spec_fill_limit, model3,
                                                       cpu="cpu" in legs)
            if "ablation" in legs:
                print("[bench] ablation leg (prefill)", file=sys.stderr, flush=True)
                out["detail"]["ablation"]["prefill"] = leg_ablation(torch, args, "prefill", model3, configs.C3.slots)
        finally:
            model3.close()
        del model3
    if "mfma" in legs:
        print("[bench] shared-expert MFMA leg", file=sys.stderr, flush=True)
        g = leg_mfma(torch, args)
        g["peak_measured"] = peaks["mfma_bf16_TFLOPs"]
        g["frac_of_measured"] = round(g["achieved"] / peaks["mfma_bf16_TFLOPs"], 4) if peaks["mfma_bf16_TFLOPs"] else None
        out["roofline_prefill_gemm"] = g
    if "hbmsize" in legs:
        print("[bench] streaming-read probe at GEMV launch sizes", file=sys.stderr, flush=True)
        out["detail"]["hbm_read_by_launch_size"] = leg_hbm_sizes(torch)
    if "int4" in legs:
        print("[bench] 4-bit experts leg", file=sys.stderr, flush=True)
        out["detail"]["int4"] = leg_int4(torch, args)
    if "configs" in legs:
        print("[bench] other workloads leg", file=sys.stderr, flush=True)
        out["detail"]["configs"] = leg_configs(torch, args, h2d_gbs, cpu="cpu" in legs)
    torch.cuda.synchronize()
    print(summary_line(out), file=sys.stderr, flush=True)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
