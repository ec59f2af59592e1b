#!/usr/bin/env python3
"""Benchmark of the BiCache shared-prefix denoising step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--depth d]

Workload (one "step" = one bc_step_forward call, the whole hot path):
  32-layer random-init transformer of the LLaDA-8B layer shape (hidden 4096,
  32 x 128 heads, SwiGLU 12288, RMSNorm, RoPE), bf16 weights and operands,
  fp32 residual; B = 16 requests sharing a cached 1536-token prefix, each with
  512 suffix tokens (shared-prefix ratio 0.75), reuse depth d (default 8):
  layers 0..d-1 project only the suffix rows and attend over the cached prefix
  K/V; layers d..31 recompute the prefix with full bidirectional attention.
  Inputs are seeded synthetic Gaussians already resident in HBM.

Prints ONE JSON line: request-denoise-steps/s of that step (value), the
roofline of its dominant kernel (the gate/up + SwiGLU GEMM) measured live with
HIP events inside the timed region, the fp64 CPU oracle timed on a bounded
sample (rank 0), plus the per-depth step times, the deep-layer reuse steps of
Eq. 5 (refresh, reuse, and their mix at refresh interval 16), the profiling
pass of Eq. 3 (KV similarity of every request and layer), a batch over four
prefixes of different lengths, the shared-prefix attention throughput of the
attention-only workloads, and the full step at the Dream-7B shape (GQA).
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "request-denoise-steps/s + shared-prefix attn TFLOP/s (% MFMA peak), LLaDA-8B shape"
PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def step_flops(cfg, B, m, n_s, d):
    """Algorithmic FLOPs of one step: linear layers 2*(rows)*(params) and
    attention 4*n_q*n_k*dh per (request, head), no causal halving."""
    h, F, L = cfg["hidden"], cfg["ffn"], cfg["n_layers"]
    Hq, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    lin_qkv = 2 * h * (Hq + 2 * Hkv) * dh
    lin = lin_qkv + 2 * (Hq * dh * h + 3 * h * F)
    N = m + n_s
    shallow = B * n_s * lin + 4 * B * Hq * n_s * N * dh
    deep = B * N * lin + 4 * B * Hq * N * N * dh
    if d >= L:
        return L * shallow
    # the last layer's prefix rows only supply K/V: their attention, O
    # projection and FFN outputs are never read, and are not computed
    last = B * N * lin_qkv + B * n_s * (lin - lin_qkv) + 4 * B * Hq * n_s * N * dh
    return d * shallow + (L - d - 1) * deep + last


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gate_up_swiglu_c3_step_d8_traffic.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2606_07571_amd", "csrc", "gemm.hip")


def measured_traffic(d):
    """HBM bytes per gate_up launch from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by the copy calibration), or None
    when there is none for this depth or the GEMM source changed since."""
    import hashlib
    try:
        txt = open(TRAFFIC_PROFILE).read()
        fields = dict(line.split(":", 1) for line in txt.splitlines() if line.startswith(("bytes_per_launch:", "gemm_source_sha256:", "depth:")))
        sha = hashlib.sha256(open(GEMM_SOURCE, "rb").read()).hexdigest()
        if fields.get("gemm_source_sha256", "").strip() != sha or int(fields.get("depth", "-1")) != d:
            return None
        return int(float(fields["bytes_per_launch"]))
    except (OSError, KeyError, ValueError):
        return None


def gate_up_flops(cfg, rows):
    return 2.0 * rows * 2 * cfg["ffn"] * cfg["hidden"]


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[1])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--depth", type=int, default=8)
    ap.add_argument("--depth-steps", type=int, default=3, help="timed steps per extra depth")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-step", action="store_true",
                    help="run the warmup and timed steps at --depth plus a 512 MiB copy (counter calibration) "
                         "and exit; the command profiled under rocprofv3")
    ap.add_argument("--profile-attention", action="store_true",
                    help="run only the attention configurations, exactly as the bench times them (5 warm-up "
                         "and 3 x 20 timed launches each), log their figures and exit; the command profiled "
                         "under rocprofv3")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures the single-GPU path only (asked for --gpus {args.gpus}, "
              f"WORLD_SIZE={world}); the step shards by request across GPUs, which is not implemented here.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_07571_amd as bc
    from paper_2606_07571_amd import synth

    bc.lib()                                   # fails loudly if the library is not built
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log = lambda *a: print(*a, file=sys.stderr, flush=True)

    # ---------------------------------------------------------------- attention configs
    # Measured first, on their own inputs, before the long full-step runs heat
    # the card: 5 warm-up launches, then the median of 3 repetitions of 20.
    attention = {}
    for cid in (() if args.profile_step else (0, 1, 2, 4)):
        s = synth.ATTN_CONFIGS[cid]
        ins = synth.attention_inputs(s, 1000 * cid, device=dev)
        o = torch.empty((s.B, s.Hq, s.n_s, s.dh), dtype=torch.float32, device=dev)
        for _ in range(5):
            bc.shared_prefix_attention(*ins, out=o)
        torch.cuda.synchronize()
        n, reps = 20, []
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(n):
                bc.shared_prefix_attention(*ins, out=o)
            e1.record()
            torch.cuda.synchronize()
            reps.append(e0.elapsed_time(e1) / n)
        t = sorted(reps)[1]
        fl = 4.0 * s.B * s.Hq * s.n_s * (s.m + s.n_s) * s.dh
        attention[f"C{cid}"] = {"ms": round(t, 4), "tflops": round(fl / (t / 1e3) / 1e12, 1),
                                "frac_of_peak": round(fl / (t / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                                "ms_range": [round(min(reps), 4), round(max(reps), 4)]}
        if args.profile_attention:
            log(f"profiled C{cid}: 5 warm-up + 3 x {n} timed launches, {json.dumps(attention[f'C{cid}'])}")
        del ins, o
    torch.cuda.empty_cache()
    if args.profile_attention:
        return

    # ---------------------------------------------------------------- C3 setup
    cfg = synth.model_config()
    sc = synth.STEP_CONFIG
    B, m, n_s, d = sc["B"], sc["m"], sc["n_s"], args.depth
    L = cfg["n_layers"]
    log(f"bench: generating 32-layer weights on the device ({cfg})")
    weights = synth.model_weights(cfg, 3000, device=dev)
    xp, xs = synth.step_inputs(cfg, B, m, n_s, 3500, device=dev)
    model = bc.Model(cfg, weights, cache_capacity=4)
    key = bc.prefix_key(range(m))
    model.populate(key, xp, L)
    torch.cuda.synchronize()
    out = torch.empty((B, n_s, cfg["hidden"]), dtype=torch.float32, device=dev)

    if args.profile_step:
        # the bench's warmup and timed steps, back to back, for the profiler
        for _ in range(args.warmup + args.steps):
            model.step(key, xs, d, out=out)
        # plain copy of known size: 512 MiB read + 512 MiB written, the
        # reference that scales the HBM byte counters
        src = torch.empty(256 * 2 ** 20, dtype=torch.float16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: profile step done (d={d}; calibration copy {src.numel() * 2} bytes)")
        model.close()
        return

    # populate timing (prefix-only forward of all 32 layers, m = 1536)
    populate = {"m1536_L32": time_populate(model, key, xp, L, cfg, torch)}

    # ---------------------------------------------------------------- timed steps
    log(f"bench: warmup {args.warmup}, timed {args.steps} steps at d={d}")
    for _ in range(args.warmup):
        model.step(key, xs, d, out=out)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    model.profile_begin(["gate_up_swiglu"])    # HIP events around the dominant kernel only
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        model.step(key, xs, d, out=out)
    ev1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - w0) * 1e3
    prof = model.profile_end()
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    value = B / (ms_per_step / 1e3)

    gu_ms, gu_n = prof["gate_up_swiglu"]
    # gate_up rows: suffix rows in the shallow layers and the last one, all rows between
    rows_per_step = (L * B * n_s if d >= L else (d + 1) * B * n_s + (L - d - 1) * B * (m + n_s))
    gu_flops = gate_up_flops(cfg, rows_per_step) * args.steps
    gu_tflops = gu_flops / (gu_ms / 1e3) / 1e12
    roofline = {"bound": "mfma", "kernel": "gate_up_swiglu GEMM (bf16 MFMA)",
                "achieved": round(gu_tflops, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(gu_tflops / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic(d),
                "launches": gu_n, "avg_launch_ms": round(gu_ms / gu_n, 4)}

    # per-kernel breakdown of one extra profiled step (all classes)
    model.profile_begin()
    model.step(key, xs, d, out=out)
    prof = model.profile_end()
    breakdown = {k: round(v[0], 3) for k, v in prof.items()}
    # HBM-bound paths of the same step against the 8 TB/s peak, algorithmic
    # bytes only: RMSNorm reads the fp32 residual and writes the bf16 operand
    # (two norms per layer over B*n_s rows below d, B*(m+n_s) rows from d on,
    # except the last layer's second norm, over the suffix rows only); the
    # transition writes the full residual of every request and reads the
    # suffix rows and the cached prefix residual once
    h = cfg["hidden"]
    norm_rows = (2 * L * B * n_s if d >= L else
                 2 * d * B * n_s + 2 * (L - d - 1) * B * (m + n_s) + B * (m + n_s) + B * n_s)
    norm_bytes = norm_rows * h * (4 + 2)
    trans_bytes = (B * (m + n_s) + B * n_s + m) * h * 4 if d < L else 0
    hbm = {}
    for name, nbytes in (("rmsnorm", norm_bytes), ("transition", trans_bytes)):
        if name in prof and nbytes:
            t_ms = prof[name][0]
            hbm[name] = {"ms": round(t_ms, 3), "launches": prof[name][1], "bytes": nbytes,
                         "gbs": round(nbytes / (t_ms / 1e3) / 1e9, 1),
                         "frac": round(nbytes / (t_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4)}

    # ---------------------------------------------------------------- other depths
    per_depth = {}
    for dd in sorted(set([0, 4, 8, 16, d])):
        model.step(key, xs, dd, out=out)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.depth_steps):
            model.step(key, xs, dd, out=out)
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / args.depth_steps
        per_depth[dd] = {"ms": round(t, 3), "request_steps_per_s": round(B / (t / 1e3), 2),
                         "tflops": round(step_flops(cfg, B, m, n_s, dd) / (t / 1e3) / 1e12, 1)}
    base = per_depth[0]["ms"]
    f0 = step_flops(cfg, B, m, n_s, 0)
    for dd, r in per_depth.items():
        r["speedup_vs_d0"] = round(base / r["ms"], 3)
        r["ideal_speedup"] = round(f0 / step_flops(cfg, B, m, n_s, dd), 3)

    # ------------------------------------------------ deep-layer reuse (Eq. 5)
    # refresh steps write the deep layers' K/V into a per-batch store; the
    # steps in between run every layer on the suffix rows only.  Amortized over
    # a refresh interval of 16 (one refresh, 15 reuse steps).
    def timed(fn, n):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    delta = 16
    deep_reuse = {}
    for dd in sorted(set([0, d])):
        if dd >= L:
            continue
        store = model.new_deep_store(key, B, n_s, dd, device=dev)
        t_ref = timed(lambda: model.step(key, xs, dd, out=out, deep="refresh", deep_store=store),
                      args.depth_steps)
        t_reu = timed(lambda: model.step(key, xs, dd, out=out, deep="reuse", deep_store=store),
                      args.depth_steps)
        amort = (t_ref + (delta - 1) * t_reu) / delta
        deep_reuse[dd] = {"refresh_ms": round(t_ref, 3), "reuse_ms": round(t_reu, 3),
                          "reuse_tflops": round(step_flops(cfg, B, m, n_s, L) / (t_reu / 1e3) / 1e12, 1),
                          "delta": delta, "amortized_ms": round(amort, 3),
                          "request_steps_per_s": round(B / (amort / 1e3), 2),
                          "speedup_vs_d0": round(per_depth[0]["ms"] / amort, 3),
                          "store_gib": round(store.numel() / 2 ** 30, 2)}
        del store
        torch.cuda.empty_cache()

    # ------------------------------------------------ profiling (Eq. 3, Sec. 5.1)
    # sim_{l,1} of the 16 requests at every layer: the un-cached step storing
    # every layer's K/V, then the HBM-bound similarity reduction (one call
    # covers every layer)
    sims = model.profile_similarity(key, xs)
    torch.cuda.synchronize()
    t_prof = timed(lambda: model.profile_similarity(key, xs, sims=sims), args.depth_steps)
    model.profile_begin(["kv_similarity"])
    model.profile_similarity(key, xs, sims=sims)
    sim_ms, sim_n = model.profile_end()["kv_similarity"]
    Hkv, dh = cfg["n_kv_heads"], cfg["head_dim"]
    kv_layer_bytes = 2 * Hkv * m * dh * 2
    sim_bytes = L * (kv_layer_bytes + B * kv_layer_bytes)   # KV$ once, each request's KV^ref once
    profiling = {"requests": B, "layers": L, "profile_ms": round(t_prof, 3),
                 "similarity_ms": round(sim_ms, 4), "similarity_calls": sim_n,
                 "similarity_bytes": sim_bytes,
                 "similarity_gbs": round(sim_bytes / (sim_ms / 1e3) / 1e9, 1),
                 "similarity_frac_of_hbm": round(sim_bytes / (sim_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4),
                 "sim_layer_mean_min": [round(float(x), 6) for x in (sims.mean().item(), sims.min().item())]}
    hbm["kv_similarity"] = {"ms": profiling["similarity_ms"], "launches": sim_n, "bytes": sim_bytes,
                            "gbs": profiling["similarity_gbs"], "frac": profiling["similarity_frac_of_hbm"]}
    del sims
    torch.cuda.empty_cache()

    # ------------------------------------------------ several prefixes (Sec. 6.5)
    # four tenants' prefixes of different lengths, four requests each, in one
    # batch, against the same groups stepped one after another
    mt_m = (1536, 1024, 2048, 512)
    mt_keys = [key]
    for i, mm in enumerate(mt_m[1:]):
        k_i = bc.prefix_key([10 ** 6 * (i + 1) + t for t in range(mm)])
        model.populate(k_i, synth.gaussian((mm, cfg["hidden"]), 4200 + i, device=dev), L)
        mt_keys.append(k_i)
    mt_counts = [B // 4] * 4
    t_multi = timed(lambda: model.step_multi(mt_keys, mt_counts, xs, d, out=out), args.depth_steps)
    xs_parts = [xs[i * (B // 4):(i + 1) * (B // 4)].contiguous() for i in range(4)]

    def separate():
        for k_i, x_i in zip(mt_keys, xs_parts):
            model.step(k_i, x_i, d)
    t_sep = timed(separate, args.depth_steps)
    mt_flops = sum(step_flops(cfg, B // 4, mm, n_s, d) for mm in mt_m)
    multi_prefix = {"prefixes": list(mt_m), "requests_per_prefix": B // 4, "depth": d,
                    "batched_ms": round(t_multi, 3), "separate_ms": round(t_sep, 3),
                    "request_steps_per_s": round(B / (t_multi / 1e3), 2),
                    "tflops": round(mt_flops / (t_multi / 1e3) / 1e12, 1),
                    "speedup_vs_separate": round(t_sep / t_multi, 3)}
    for k_i in mt_keys[1:]:
        model.invalidate(k_i)
    del xs_parts
    torch.cuda.empty_cache()

    # C4 populate: 8 layers of the same shape over an 8192-token prefix
    xp4 = synth.gaussian((8192, cfg["hidden"]), 4100, device=dev)
    key4 = bc.prefix_key(range(8192))
    model.populate(key4, xp4, 8)
    populate["m8192_L8"] = time_populate(model, key4, xp4, 8, cfg, torch)
    model.invalidate(key4)
    del xp4
    torch.cuda.empty_cache()

    # ---------------------------------------------------------------- CPU oracle baseline
    # the fp64 oracle's full step on requests 0 and 15 at d, on the host,
    # against the GPU rows of the same requests from the timed step's output
    cpu = None
    if not args.no_cpu_baseline:
        model.step(key, xs, d, out=out)
        torch.cuda.synchronize()
        cpu = cpu_baseline(cfg, weights, xp, xs, out, d, log)
    model.close()
    del weights, model
    torch.cuda.empty_cache()

    # ---------------------------------------------------------------- Dream-7B-shaped full step
    # 28 layers, GQA 28/4 x 128, hidden 3584, SwiGLU 18944, Q/K/V bias; the GQA
    # workload's sizes: 64 requests, shared prefix 1024, suffix 384
    dcfg = synth.dream_config()
    ds = synth.DREAM_STEP
    dB, dm, dn = ds["B"], ds["m"], ds["n_s"]
    log(f"bench: Dream-7B-shaped step ({dcfg})")
    dweights = synth.model_weights(dcfg, 8000, device=dev)
    dxp, dxs = synth.step_inputs(dcfg, dB, dm, dn, 8500, device=dev)
    dmodel = bc.Model(dcfg, dweights, cache_capacity=1)
    dkey = bc.prefix_key(range(dm))
    dmodel.populate(dkey, dxp, dcfg["n_layers"])
    dout = torch.empty((dB, dn, dcfg["hidden"]), dtype=torch.float32, device=dev)
    dream = {"model": "Dream-7B shape (28 layers, 28/4 x 128 heads, h 3584, F 18944, QKV bias)",
             "B": dB, "prefix": dm, "suffix": dn}
    d0_ms = None
    for dd in (0, 8):
        t = timed(lambda: dmodel.step(dkey, dxs, dd, out=dout), args.depth_steps)
        fl = step_flops(dcfg, dB, dm, dn, dd)
        if dd == 0:
            d0_ms = t
        dream[f"d{dd}"] = {"ms": round(t, 3), "request_steps_per_s": round(dB / (t / 1e3), 2),
                           "tflops": round(fl / (t / 1e3) / 1e12, 1),
                           "speedup_vs_d0": round(d0_ms / t, 3),
                           "ideal_speedup": round(step_flops(dcfg, dB, dm, dn, 0) / fl, 3)}
    dmodel.close()
    del dweights, dmodel, dxp, dxs, dout
    torch.cuda.empty_cache()

    line = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "request-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "wall_ms_per_step": round(wall_ms / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Gaussian inputs, random-init weights)",
        "config": {"workload": f"full 32-layer denoising step, LLaDA-8B layer shape (h=4096, 32x128 heads, "
                               f"SwiGLU 12288), B={B} requests, shared prefix {m} + suffix {n_s} tokens, "
                               f"reuse depth d={d}",
                   "global_batch": B, "seq_len": m + n_s, "prefix": m, "suffix": n_s, "depth": d,
                   "parallelism": "single GPU"},
        "step_tflops": round(step_flops(cfg, B, m, n_s, d) / (ms_per_step / 1e3) / 1e12, 1),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "per_depth": per_depth,
        "deep_reuse": deep_reuse,
        "multi_prefix": multi_prefix,
        "profiling": profiling,
        "kernel_ms_one_step": breakdown,
        "hbm": hbm,
        "attention": attention,
        "dream_step": dream,
        "populate": populate,
    }
    print(json.dumps(line), flush=True)


class _HostLayersF64:
    """Per-layer host fp64 copies of device weights, widened exactly on first
    use (the oracle's inputs are the very bf16 values the GPU reads)."""

    def __init__(self, layers):
        self._dev, self._host = layers, {}

    def __len__(self):
        return len(self._dev)

    def __getitem__(self, l):
        if l not in self._host:
            self._host[l] = {k: (None if v is None else v.detach().to("cpu").float().double().numpy())
                             for k, v in self._dev[l].items()}
        return self._host[l]


def cpu_baseline(cfg, weights, xp, xs, out, d, log, requests=(0, 15)):
    """The fp64 oracle (NumPy, host threads) on a bounded sample of the timed
    workload: the full step at depth d of `requests` of the batch, each timed
    on its own.  The oracle first runs its own prefix-only forward over the d
    layers the step reuses (its cache; not timed: it is the once-per-prefix
    populate, not the step).  The oracle's rows are compared with the GPU's
    rows of the same requests (parity on exactly the sampled requests)."""
    import numpy as np
    from oracle import transformer as OT
    from paper_2606_07571_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    W = _HostLayersF64(weights)
    log(f"bench: oracle populate of {d} layers (fp64, host)")
    t0 = time.perf_counter()
    cache = OT.populate(synth.to_f64(xp), W, cfg, d)
    t_pop = time.perf_counter() - t0
    for l in range(len(W)):     # widen every layer before the timed steps
        W[l]
    times, errs = [], []
    for b in requests:
        log(f"bench: oracle step d={d} request {b}")
        xb = synth.to_f64(xs[b:b + 1])
        t0 = time.perf_counter()
        ref = OT.step(cache, xb, d, W, cfg)[0]
        times.append(time.perf_counter() - t0)
        err = np.abs(out[b].double().cpu().numpy() - ref)
        errs.append((float(err.max()), float(err.mean())))
    t_req = sum(times) / len(times)
    return {"value": round(1.0 / t_req, 6), "unit": "request-steps/s", "cores": threads,
            "kind": "oracle",
            "sample": f"full {cfg['n_layers']}-layer step at d={d} of requests {list(requests)} of the "
                      f"timed batch of {xs.shape[0]}, each timed alone (mean {t_req:.2f} s per "
                      f"request-step); the oracle's own {d}-layer populate ({t_pop:.1f} s) not timed",
            "sample_seconds": round(sum(times), 2),
            "parity_vs_gpu": {"requests": list(requests),
                              "max_abs": round(max(e[0] for e in errs), 6),
                              "mean_abs": round(max(e[1] for e in errs), 7)}}


def time_populate(model, key, xp, Lc, cfg, torch, reps=3):
    """Populate of `key` (already cached once, so warm) timed with HIP events on
    the launch stream, median of `reps`; its algorithmic FLOPs (prefix-only
    forward of Lc layers) and the cache bytes it writes (KV$ bf16 + H$ fp32)."""
    m = xp.shape[0]
    ts = []
    for _ in range(reps):
        model.invalidate(key)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        model.populate(key, xp, Lc)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    t = sorted(ts)[len(ts) // 2]
    h, F, L = cfg["hidden"], cfg["ffn"], cfg["n_layers"]
    Hq, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    lin_qkv = 2 * h * (Hq + 2 * Hkv) * dh
    lin = lin_qkv + 2 * (Hq * dh * h + 3 * h * F)
    flops = Lc * (m * lin + 4 * Hq * m * m * dh)
    if Lc == L:   # the last layer's output residual has no H$ slot: only its K/V are computed
        flops -= m * (lin - lin_qkv) + 4 * Hq * m * m * dh
    kv_bytes = Lc * 2 * Hkv * m * dh * 2
    h_bytes = min(Lc + 1, L) * m * h * 4
    return {"ms": round(t, 3), "tflops": round(flops / (t / 1e3) / 1e12, 1),
            "kv_cache_bytes": kv_bytes, "h_cache_bytes": h_bytes,
            "cache_write_gbs": round((kv_bytes + h_bytes) / (t / 1e3) / 1e9, 1)}


if __name__ == "__main__":
    main()
