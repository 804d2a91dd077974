"""Decode-step benchmark of the grouped-cache runtime on one MI355X.

A step is one pass of the decode hot path over every layer of the workload:
for each layer, append the new token to every unit and attend with the
layer's query (one ``hwkv_append_decode_attn`` call per layer).  The cache is
materialised once before timing (``hwkv_prefill_write`` per layer); inputs
are resident in HBM before the timed region starts.

Default workload: 16 residual global layers at a 112K context (114,688
tokens), batch 1, 24 query / 4 KV heads, head_dim 256, bf16 K/V, 4 sinks,
per-unit levels over {2048, 8192, 32768, full} drawn at a 45-50% residency
budget, 128 decode steps after a 114,560-token prompt.

Prints ONE JSON line: resident-KV GB/s (``value``), microseconds per step,
the roofline of the dominant kernel and the oracle's CPU baseline.

``--workload calib128k`` times the calibration replay of one traced layer:
a 131,072-token trace, 256 query positions from its final quarter, candidate
windows {2048, 8192, 32768} and full; a step is one ``hwkv_calib_replay``
(every candidate's outputs, the scores and the per-head means).  The
algorithmic FLOP count sums every candidate's retained pairs; the one-pass
kernel forms each product once for all of them.

``--workload prefill128k`` instead times the long-prefill path: a step is a
131,072-token prompt processed in 8,192-token chunks, each chunk's sink +
window causal attention (``hwkv_prefill_attn``, bf16 MFMA) followed by its
materialisation (``hwkv_prefill_write``), over KV heads with windows
{2048, 8192, 32768, full}; ``value`` is algorithmic attention TFLOP/s.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn µs/step + resident-KV HBM GB/s (% of peak) at 112K ctx, 1 GPU"
CALIB_METRIC = "calibration replay TFLOP/s (128K trace, 256 rows, 3 windows + full, 1 GPU)"
PREFILL_METRIC = "prefill-attn TFLOP/s (128K prompt in 8K chunks, sink+window causal, 1 GPU)"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="suite",
                    choices=["suite", "ctx112k", "ctx32k", "batch16", "pr1", "prefill128k",
                             "calib128k", "probe"],
                    help="suite (default): the 112K headline (--steps/--warmup) plus every "
                         "other configuration in one line; or one workload alone")
    ap.add_argument("--intervals", type=int, default=3,
                    help="decode workloads: the timed steps are cut into this many consecutive "
                         "intervals; us/step is their median")
    ap.add_argument("--kv-format", default="bf16", choices=["bf16", "f16", "fp8"],
                    help="cache format of the decode workloads (fp8: E4M3 with the "
                         "workload's per-unit scales)")
    ap.add_argument("--paged", action="store_true",
                    help="page the full units (pages of 256 rows from a pool sized to the "
                         "workload's final lengths) instead of reserving max_ctx rows")
    ap.add_argument("--replicas", type=int, default=1,
                    help="decode workloads: R independent caches of the workload (own seeded "
                         "data), steps cycling through them, so that a cache smaller than the "
                         "256 MB Infinity Cache is read cold from HBM (ctx32k: 16 replicas)")
    ap.add_argument("--unfused", action="store_true",
                    help="time hwkv_append + hwkv_decode_attn instead of the fused call")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time budget of the oracle sample")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="first run a plain device copy of MIB MiB three times, so that "
                         "a counter run (rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE) sees a "
                         "kernel of known traffic beside the decode kernels")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the grouped-cache runtime is built and "
              "timed on a single MI355X (no sharding, no collectives). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads as W
    from paper_2609_02029_amd import hwkv

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.workload == "prefill128k":
        print(json.dumps(prefill_run(args, dev)), flush=True)
        return
    if args.workload == "calib128k":
        calib_main(args, dev)
        return
    if args.workload == "probe":
        probe_main(args, dev)
        return
    if args.workload == "suite":
        print(json.dumps(suite(args, dev)), flush=True)
        return
    print(json.dumps(decode_run(args, dev)), flush=True)


def decode_run(args, dev, one_core=True):
    """One decode workload (``args.workload``, ``kv_format``, ``paged``,
    ``replicas``, ``steps``, ``warmup``, ...): the result dict of its line."""
    import numpy as np
    import torch

    import workloads as W
    from paper_2609_02029_amd import hwkv

    cfg = W.CONFIGS[args.workload]
    L, B = cfg["n_layers"], cfg["batch"]
    Hq, Hkv, D, S = cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"], cfg["n_sinks"]
    levels = W.levels(cfg)
    windows = W.windows_of(cfg, levels)
    # warmup, the timed region, then the kernel-timing region (same length);
    # with replicas, step s decodes replica s mod R, for its (s // R)-th time
    R = max(1, args.replicas)
    total_steps = args.warmup + 2 * args.steps
    rep_steps = (total_steps + R - 1) // R
    prompts = W.prompts(cfg)
    max_ctx = cfg["max_ctx"]
    if rep_steps > cfg["steps"]:
        # keep the final context at max_ctx: start from a shorter prompt
        extra = rep_steps - cfg["steps"]
        prompts = [max(1, p - extra) for p in prompts]
    scale = 1.0 / math.sqrt(D)

    pol = hwkv.policy_set(L, Hkv, Hq, D, S, cfg["level_windows"], levels)
    fmt = args.kv_format
    eb = hwkv.KV_FORMATS[fmt][1]                  # bytes per stored element
    scales = W.fp8_scales(cfg) if fmt == "fp8" else None
    n_pages = None
    if args.paged:
        # every full unit of every layer holds ceil(n_b / 256) pages at the
        # final length n_b = prompt_b + rep_steps
        full = sum(1 for l in range(L) for h in range(Hkv)
                   if windows[l][h] == 0 or S + windows[l][h] >= max_ctx)
        n_pages = full * sum((p + rep_steps + hwkv.PAGE_TOKENS - 1) // hwkv.PAGE_TOKENS
                             for p in prompts)
    caches = [hwkv.cache_alloc(pol, B, max_ctx, kv_format=fmt, k_scale=scales, v_scale=scales,
                               n_pages=n_pages) for _ in range(R)]
    cache = caches[0]
    cache_bytes = hwkv.cache_bytes(pol, B, max_ctx, fmt, n_pages=n_pages)
    reserved_bytes = hwkv.cache_bytes(pol, B, max_ctx, fmt)
    ws = torch.zeros(hwkv.decode_workspace_bytes(cache), dtype=torch.uint8, device=dev)
    caps = [[hwkv.cache_unit_info(cache, l, h)[0] for h in range(Hkv)] for l in range(L)]
    outl = W.outlier_channels(cfg)
    osc = cfg.get("outlier_scale", 1.0)

    t0 = time.time()
    for r, c in enumerate(caches):                # replica r: its own seeded streams
        for l in range(L):
            for b in range(B):
                k = W.normal_bf16_device((prompts[b], Hkv, D), cfg["seed"], l, W.K, b + 4096 * r,
                                         device=dev, scale_channels=outl, scale=osc)
                v = W.normal_bf16_device((prompts[b], Hkv, D), cfg["seed"], l, W.V, b + 4096 * r,
                                         device=dev, scale_channels=outl, scale=osc)
                hwkv.prefill_write(c, l, b, 0, k, v)
                del k, v
    torch.cuda.synchronize()
    prefill_s = time.time() - t0

    # per-step inputs, resident on the device before timing
    def dev_bf16(a):
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    qs = torch.stack([torch.stack([dev_bf16(W.normal_bf16((B, Hq, D), cfg["seed"], l, W.Q, s))
                                   for l in range(L)]) for s in range(total_steps)]).to(dev)
    kn = torch.stack([torch.stack([dev_bf16(W.normal_bf16((B, Hkv, D), cfg["seed"], l, W.K_NEW, s,
                                                          scale_channels=outl, scale=osc))
                                   for l in range(L)]) for s in range(total_steps)]).to(dev)
    vn = torch.stack([torch.stack([dev_bf16(W.normal_bf16((B, Hkv, D), cfg["seed"], l, W.V_NEW, s,
                                                          scale_channels=outl, scale=osc))
                                   for l in range(L)]) for s in range(total_steps)]).to(dev)
    out = torch.empty((L, B, Hq, D), dtype=torch.float32, device=dev)

    def kv_bytes(step_idx):
        """Algorithmic resident-KV bytes of step ``step_idx`` (per layer)."""
        per_layer = []
        for l in range(L):
            tot = 0
            for b in range(B):
                n = prompts[b] + step_idx // R + 1
                for h in range(Hkv):
                    tot += min(n, caps[l][h]) * D * 2 * eb
            per_layer.append(tot)
        return per_layer

    # the fused calls of the timed steps go through the raw-address entry of
    # the binding (the tensors are checked once, by the first warmup step,
    # which uses the checked call): the Python checks of every call would
    # otherwise take about as long as a layer's kernels
    stream = torch.cuda.current_stream().cuda_stream
    kv_stride = B * Hkv * D * 2
    q_stride = B * Hq * D * 2
    o_stride = B * Hq * D * 4
    kn_p, vn_p, q_p, o_p = kn.data_ptr(), vn.data_ptr(), qs.data_ptr(), out.data_ptr()
    ws_p, ws_n = ws.data_ptr(), ws.numel()

    def run_step(s, checked=False):
        c = caches[s % R]
        for l in range(L):
            if args.unfused:
                hwkv.append(c, l, kn[s, l], vn[s, l])
                hwkv.decode_attn(c, l, qs[s, l], scale, out[l], ws)
            elif checked:
                hwkv.append_decode_attn(c, l, kn[s, l], vn[s, l], qs[s, l], scale, out[l], ws)
            else:
                i = s * L + l
                hwkv.append_decode_attn_ptr(c, l, kn_p + i * kv_stride, vn_p + i * kv_stride,
                                            q_p + i * q_stride, scale, o_p + l * o_stride,
                                            ws_p, ws_n, stream)

    for s in range(args.warmup):
        run_step(s, checked=(s == 0))
    torch.cuda.synchronize()

    # the timed region: K steps, bracketed by events on the stream the
    # kernels are launched on (torch's current stream), cut into consecutive
    # intervals by events between them; us/step is the median interval's
    n_int = max(1, min(args.intervals, args.steps))
    cuts = [args.steps * i // n_int for i in range(n_int + 1)]
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_int + 1)]
    torch.cuda.synchronize()
    evs[0].record()
    for k in range(n_int):
        for i in range(cuts[k], cuts[k + 1]):
            run_step(args.warmup + i)
        evs[k + 1].record()
    torch.cuda.synchronize()
    total_ms = evs[0].elapsed_time(evs[-1])
    int_ms = [evs[k].elapsed_time(evs[k + 1]) / (cuts[k + 1] - cuts[k]) for k in range(n_int)]
    ms_per_step = float(np.median(int_ms))

    bytes_steps = [sum(kv_bytes(args.warmup + i)) for i in range(args.steps)]
    bytes_per_step = sum(bytes_steps) / args.steps
    gbs = bytes_per_step / (ms_per_step * 1e-3) / 1e9

    # Kernel-timing region: the next K steps again, with the library
    # launching each decode call's split kernel (the dominant kernel: it
    # streams every resident K/V byte) and its merge kernel with start and
    # stop HIP events on the same stream, which take the kernels' own start
    # and end times.
    for c in caches:
        hwkv.decode_timing(c, True)
    for i in range(args.steps):
        run_step(args.warmup + args.steps + i)
    split_ms = merge_ms = 0.0
    launches = 0
    for c in caches:
        sp, mg, n = hwkv.decode_timing_read(c)
        hwkv.decode_timing(c, False)
        split_ms, merge_ms, launches = split_ms + sp, merge_ms + mg, launches + n
    bytes_t = [sum(kv_bytes(args.warmup + args.steps + i)) for i in range(args.steps)]
    split_avg_ms = split_ms / launches
    merge_avg_ms = merge_ms / launches
    launch_bytes = sum(bytes_t) / launches
    achieved = launch_bytes / (split_avg_ms * 1e-3) / 1e9

    rate = hwkv.policy_rate(pol, max_ctx)
    traffic, traffic_detail = measured_traffic(args)
    result = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "us_per_step": round(ms_per_step * 1e3, 1),
        "us_per_step_intervals": [round(x * 1e3, 1) for x in int_ms],
        "us_per_step_mean": round(total_ms / args.steps * 1e3, 1),
        "step_decomposition_us": {
            "decode_split": round(split_avg_ms * 1e3 * launches / args.steps, 1),
            "decode_combine": round(merge_avg_ms * 1e3 * launches / args.steps, 1),
            "between_kernels": round(ms_per_step * 1e3 - (split_avg_ms + merge_avg_ms) * 1e3
                                     * launches / args.steps, 1),
            "launches_per_step": launches // args.steps,
            "note": ("kernel times from start/stop events the library passes to each launch "
                     "(a separate run of the same steps); between_kernels = median us/step "
                     "minus both"),
        },
        "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16 (fp32 accumulate)",
                  "f16": "f16 K/V, bf16 q (fp32 accumulate)",
                  "fp8": "fp8-e4m3 K/V, bf16 q (fp32 accumulate)"}[fmt],
        "data": "synthetic",
        "config": {
            "kv_format": fmt,
            "paged": bool(args.paged),
            "replicas": R,
            "cache_bytes": int(cache_bytes),
            "cache_bytes_reserved_layout": int(reserved_bytes),
            "workload": (f"{cfg['name']}: {L} residual global layers, batch {B}, "
                         f"{Hq} q / {Hkv} kv heads, head_dim {D}, {S} sinks, levels "
                         f"{cfg['level_windows']} (0 = full), R={rate:.4f} at {max_ctx} tokens, "
                         f"prompt {prompts[0] if B == 1 else 'ragged'}, "
                         f"{'append+decode' if args.unfused else 'fused append+decode'} per layer"),
            "max_ctx": max_ctx,
            "resident_kv_bytes_per_step": int(bytes_per_step),
            "prefill_write_s": round(prefill_s, 3),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": ("decode_mfma (split-K attention over one layer's resident fp8 K/V, "
                       "products on the matrix cores)" if args.kv_format == "fp8" else
                       "decode_split (split-K attention over one layer's resident K/V)"),
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "traffic_detail": traffic_detail,
            "launch_us_mean": round(split_avg_ms * 1e3, 2),
            "merge_us_mean": round(merge_avg_ms * 1e3, 2),
            "kv_bytes_per_launch": int(launch_bytes),
            "launches_timed": int(launches),
        },
    }

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(args, cfg, prompts, windows, caps, scale, outl, osc,
                                              dev, ms_per_step, bytes_per_step, eb, scales,
                                              one_core=one_core)
    for c in caches:
        c.free()
    del ws
    return result


def suite(args, dev):
    """The default run: the 112K-context headline (``--steps``, ``--warmup``,
    ``--cpu-seconds``) and, under ``configs``, every other configuration of
    the workload set -- the PR1 reference, 32K warm and cold (16 replicas),
    the batch-16 serving mix reserved and paged, the 112K workload in the
    fp8 and binary16 cache formats, and the 128K prefill -- each with its own
    roofline and, where noted, its own oracle baseline on a bounded sample."""
    import copy

    def opts(**kw):
        o = copy.copy(args)
        o.kv_format, o.paged, o.replicas, o.unfused = "bf16", False, 1, False
        for k, v in kw.items():
            setattr(o, k, v)
        return o

    head = decode_run(opts(workload="ctx112k"), dev)
    keep = ("metric", "value", "unit", "steps", "warmup", "ms_per_step", "us_per_step",
            "us_per_step_intervals", "frac_of_hbm_peak", "step_decomposition_us", "dtype",
            "roofline", "cpu_baseline", "config")
    configs = {}

    def add(name, fn):
        t0 = time.time()
        try:
            r = fn()
        except Exception as e:          # a refused call is reported, not fatal
            r = {"error": f"{type(e).__name__}: {e}"}
        r = {k: v for k, v in r.items() if k in keep or k == "error"}
        r["bench_seconds"] = round(time.time() - t0, 1)
        configs[name] = r
        print(f"[bench] {name}: {r.get('us_per_step', r.get('ms_per_step'))} "
              f"({r['bench_seconds']} s)", file=sys.stderr, flush=True)

    add("pr1", lambda: decode_run(opts(workload="pr1", steps=6, warmup=2, cpu_seconds=2.0), dev))
    add("ctx32k", lambda: decode_run(opts(workload="ctx32k", steps=60, warmup=8,
                                          cpu_seconds=2.0), dev, one_core=False))
    add("ctx32k_cold16", lambda: decode_run(opts(workload="ctx32k", steps=60, warmup=8,
                                                 replicas=16, no_cpu_baseline=True), dev))
    add("batch16", lambda: decode_run(opts(workload="batch16", steps=30, warmup=2,
                                           cpu_seconds=2.0), dev, one_core=False))
    add("batch16_paged", lambda: decode_run(opts(workload="batch16", steps=30, warmup=2,
                                                 paged=True, no_cpu_baseline=True), dev))
    # the headline's steps and warmup: with fewer, the first of the three
    # intervals has not reached the steady state and the median shows it
    add("ctx112k_fp8", lambda: decode_run(opts(workload="ctx112k", kv_format="fp8", steps=60,
                                               warmup=8, no_cpu_baseline=True), dev))
    add("ctx112k_f16", lambda: decode_run(opts(workload="ctx112k", kv_format="f16", steps=60,
                                               warmup=8, no_cpu_baseline=True), dev))
    add("prefill128k", lambda: prefill_run(opts(workload="prefill128k", steps=3, warmup=1,
                                                cpu_seconds=8.0), dev))
    head["configs"] = configs
    return head


def measured_traffic(args):
    """HBM bytes per split launch (decode_split, or decode_mfma for fp8) from
    the committed counter record
    (FETCH_SIZE + WRITE_SIZE, copy-calibrated), if it was taken on the current
    kernel source and on this workload; otherwise None."""
    if args.workload != "ctx112k" or args.unfused or args.paged:
        return None, None
    from paper_2609_02029_amd import profiling
    name = ("decode_split_ctx112k_traffic.json" if args.kv_format == "bf16"
            else f"decode_split_ctx112k_{args.kv_format}_traffic.json")
    path = os.path.join(ROOT, "profiles", name)
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None, None
    if rec.get("kernel_source_sha256_16") != profiling.kernel_source_hash(rec["kernel"]):
        return None, "counter record is stale: decode kernel source changed"
    from paper_2609_02029_amd import hwkv
    code = hwkv.KV_FORMATS[args.kv_format][0]
    kern = rec.get("kernel", "")
    ok = (kern.startswith("decode_mfma<") if args.kv_format == "fp8"
          else kern.startswith("decode_split<") and kern.endswith(f", {code}>"))
    if not ok:
        return None, "counter record is for another cache format"
    total = rec["fetch_bytes"] + rec["write_bytes"]
    return round(total), {"fetch_bytes": round(rec["fetch_bytes"]),
                          "write_bytes": round(rec["write_bytes"]),
                          "source": "profiles/" + name}


def cpu_baseline(args, cfg, prompts, windows, caps, scale, outl, osc, dev, gpu_ms, step_bytes,
                 eb=2, scales=None, one_core=True):
    """The fp64 oracle timed on the host cores on a bounded sample of the same
    step: whole layers of decode step 0 (every sequence and query head),
    regenerated from the same seeds, until about ``--cpu-seconds`` of oracle
    time; scaled to a full step by the sampled layers' share of the step's
    resident bytes.  For the f16 and fp8 formats the oracle attends over the
    stored values (encoded before the timed call)."""
    import numpy as np
    import torch

    import oracle
    import workloads as W
    from oracle import kvformat as KF
    fmt = args.kv_format

    L, B = cfg["n_layers"], cfg["batch"]
    Hq, Hkv, D = cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    threads = max(1, min(16, os.cpu_count() or 1))
    done_bytes, spent, layers = 0, 0.0, 0
    first = None                   # layer 0's inputs, timed again on one core
    step = args.warmup  # the first timed step
    for l in range(L):
        kh, vh, t = [], [], []
        for b in range(B):
            P = prompts[b]
            k = W.normal_bf16_device((P, Hkv, D), cfg["seed"], l, W.K, b, device=dev,
                                     scale_channels=outl, scale=osc)
            v = W.normal_bf16_device((P, Hkv, D), cfg["seed"], l, W.V, b, device=dev,
                                     scale_channels=outl, scale=osc)
            hk = np.empty((P + step + 1, Hkv, D), dtype=np.uint16)
            hv = np.empty_like(hk)
            hk[:P] = k.view(torch.int16).cpu().numpy().view(np.uint16)
            hv[:P] = v.view(torch.int16).cpu().numpy().view(np.uint16)
            del k, v
            for s in range(step + 1):
                hk[P + s] = W.normal_bf16((B, Hkv, D), cfg["seed"], l, W.K_NEW, s,
                                          scale_channels=outl, scale=osc)[b]
                hv[P + s] = W.normal_bf16((B, Hkv, D), cfg["seed"], l, W.V_NEW, s,
                                          scale_channels=outl, scale=osc)[b]
            kh.append(hk)
            vh.append(hv)
            t.append(P + step)
        q = W.normal_bf16((B, Hq, D), cfg["seed"], l, W.Q, step)
        if fmt == "bf16":
            t0 = time.perf_counter()
            oracle.decode_layer(q, kh, vh, t, cfg["n_sinks"], windows[l], scale,
                                n_threads=threads)
            if first is None:
                first = (q, kh, vh, t, l)
        else:
            sc = scales[l] if scales is not None else np.ones(Hkv, dtype=np.float32)
            kv = [np.stack([KF.values(KF.store(x[:, h], fmt, sc[h]), fmt, sc[h])
                            for h in range(Hkv)], axis=1) for x in kh]
            vv = [np.stack([KF.values(KF.store(x[:, h], fmt, sc[h]), fmt, sc[h])
                            for h in range(Hkv)], axis=1) for x in vh]
            t0 = time.perf_counter()
            KF.attend_values(KF.bf16_values(q), kv, vv, t, cfg["n_sinks"], windows[l], scale)
            del kv, vv
        spent += time.perf_counter() - t0
        layers += 1
        for b in range(B):
            for h in range(Hkv):
                done_bytes += min(prompts[b] + step + 1, caps[l][h]) * D * 2 * eb
        del kh, vh
        if spent >= args.cpu_seconds:
            break
    us_per_step = spent / done_bytes * step_bytes * 1e6
    one_core_rec = None
    if first is not None and one_core:
        q, kh, vh, t, l = first
        t0 = time.perf_counter()
        oracle.decode_layer(q, kh, vh, t, cfg["n_sinks"], windows[l], scale, n_threads=1)
        s1 = time.perf_counter() - t0
        b1 = sum(min(prompts[b] + step + 1, caps[l][h]) * D * 2 * eb
                 for b in range(B) for h in range(Hkv))
        one_core_rec = {"value": round(s1 / b1 * step_bytes * 1e6, 1), "unit": "us/step",
                    "gbs": round(b1 / s1 / 1e9, 3), "sample": f"layer {l} of step {step}",
                    "seconds": round(s1, 2)}
        del first
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {
        "value": round(us_per_step, 1),
        "unit": "us/step",
        "gbs": round(done_bytes / spent / 1e9, 3),
        "cores": threads,
        "hardware_concurrency": os.cpu_count(),
        "cpu": model,
        "kind": "oracle",
        "one_core": one_core_rec,
        "sample": (f"decode step {step} (first timed step), layers 0..{layers - 1} of {L}, every "
                   f"sequence and query head; fp64 masked-full-history oracle"
                   f"{'' if fmt == 'bf16' else ' over the stored ' + fmt + ' values'}, "
                   f"{spent:.1f} s of CPU time; scaled to the whole step by resident bytes"),
        "gpu_speedup": round(us_per_step / (gpu_ms * 1e3), 1),
    }


def prefill_pairs(N, p0, p1, S, w):
    """Sum over query tokens t in [p0, p1) of |R(t + 1) restricted to [0, t]|:
    t + 1 keys while t + 1 <= S + w (always for a full unit), S + w after."""
    def upto(n):   # sum over t < n
        if w == 0 or n <= S + w:
            return n * (n + 1) // 2
        c = S + w
        return c * (c + 1) // 2 + (n - c) * c
    return upto(p1) - upto(p0)


def prefill_run(args, dev):
    import numpy as np
    import torch

    import workloads as W
    from paper_2609_02029_amd import hwkv

    cfg = W.CONFIGS["prefill128k"]
    Hq, Hkv, D, S = cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"], cfg["n_sinks"]
    G = Hq // Hkv
    N, C = cfg["prompt"][0], cfg["chunk"]
    windows = W.windows_of(cfg)[0]
    scale = 1.0 / math.sqrt(D)
    cuts = list(range(0, N, C)) + [N]
    chunk_flop = [sum(G * prefill_pairs(N, a, b, S, w) * 4 * D for w in windows)
                  for a, b in zip(cuts[:-1], cuts[1:])]
    step_flop = sum(chunk_flop)
    steps, warmup = max(1, args.steps), max(0, args.warmup)
    if steps > 5:        # a step is a whole 128K prefill: keep the run short
        steps = 3
    if warmup > 2:
        warmup = 1

    pol = hwkv.policy_set(1, Hkv, Hq, D, S, cfg["level_windows"], cfg["levels"])
    q = W.normal_bf16_device((N, Hq, D), cfg["seed"], 0, W.Q_PROMPT, 0, device=dev)
    k = W.normal_bf16_device((N, Hkv, D), cfg["seed"], 0, W.K, 0, device=dev)
    v = W.normal_bf16_device((N, Hkv, D), cfg["seed"], 0, W.V, 0, device=dev)
    out = torch.empty((N, Hq, D), dtype=torch.float32, device=dev)
    # one fresh cache per step (prefill fills it), allocated before timing;
    # --paged: the full units take pages of 256 rows as the prompt grows
    n_pages = None
    if args.paged:
        full = sum(1 for w in windows if w == 0 or S + w >= cfg["max_ctx"])
        n_pages = full * ((cfg["max_ctx"] + hwkv.PAGE_TOKENS - 1) // hwkv.PAGE_TOKENS)
    caches = [hwkv.cache_alloc(pol, 1, cfg["max_ctx"], n_pages=n_pages)
              for _ in range(warmup + 2 * steps)]
    torch.cuda.synchronize()

    def run_step(cache, events=None):
        for i, (a, b) in enumerate(zip(cuts[:-1], cuts[1:])):
            if events is not None:
                events[i][0].record()
            hwkv.prefill_attn(cache, 0, 0, a, q[a:b], k[a:b], v[a:b], scale, out[a:b])
            if events is not None:
                events[i][1].record()
            hwkv.prefill_write(cache, 0, 0, a, k[a:b], v[a:b])

    for s in range(warmup):
        run_step(caches[s])
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for s in range(steps):
        run_step(caches[warmup + s])
    end.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(end) / steps

    # kernel-timing region: events around every attention launch
    n_chunks = len(cuts) - 1
    attn_ms = np.zeros(n_chunks)
    for s in range(steps):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(n_chunks)]
        run_step(caches[warmup + steps + s], ev)
        torch.cuda.synchronize()
        attn_ms += np.array([a.elapsed_time(b) for a, b in ev])
    attn_ms /= steps
    attn_total_ms = float(attn_ms.sum())
    achieved = step_flop / (attn_total_ms * 1e-3) / 1e12
    tfs = step_flop / (ms_per_step * 1e-3) / 1e12

    result = {
        "metric": PREFILL_METRIC,
        "value": round(tfs, 1),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 (fp32 accumulate)",
        "data": "synthetic",
        "config": {
            "workload": (f"prefill128k: {N}-token prompt in {C}-token chunks, 1 layer, batch 1, "
                         f"{Hq} q / {Hkv} kv heads, head_dim {D}, {S} sinks, kv head windows "
                         f"{windows} (0 = full); per chunk prefill_attn then prefill_write"),
            "paged": bool(args.paged),
            "algorithmic_flop_per_step": step_flop,
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "prefill_attn (bf16 MFMA sink+window causal attention of one chunk)",
            "achieved": round(achieved, 1),
            "peak": MFMA_BF16_PEAK_TFS,
            "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_BF16_PEAK_TFS, 4),
            "traffic": prefill_traffic(n_chunks),
            "launch_ms_mean": round(attn_total_ms / n_chunks, 3),
            "launch_ms_per_chunk": [round(x, 3) for x in attn_ms],
            "flop_per_launch_mean": step_flop / n_chunks,
            "launches_timed": n_chunks * steps,
        },
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = prefill_cpu_baseline(args, cfg, q, k, v, windows, scale,
                                                      step_flop, ms_per_step)
    for c in caches:
        c.free()
    return result


def prefill_traffic(n_chunks):
    """HBM bytes per prefill_attn launch (mean over the chunks) from the
    committed counter record, if it was taken on the current kernel source."""
    from paper_2609_02029_amd import profiling
    path = os.path.join(ROOT, "profiles", "prefill_attn_prefill128k_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256_16") != profiling.kernel_source_hash(rec["kernel"]):
        return None
    return round(rec["fetch_bytes"] + rec["write_bytes"])


def probe_main(args, dev):
    """The practical read ceiling beside the decode roofline: passes of 16
    launches of the read probe (``_lib/libhwkv_probe.so``, measurement
    tooling beside the library), each over its own region of the ctx112k
    mean layer size (213.5 MB), as the 16 decode_split launches of a step
    read theirs; the flat grid-stride sweep at 2, 4 and 8 wavefronts per
    SIMD, and the split kernel's own walk without its arithmetic."""
    import ctypes

    import torch

    from paper_2609_02029_amd import build

    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.hwkv_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    lib.hwkv_read_probe.restype = ctypes.c_int
    stream = torch.cuda.current_stream().cuda_stream

    L, per = 16, 3416322048 // 16 // 65536 * 65536
    buf = torch.empty(L * per, dtype=torch.uint8, device=dev)
    buf.fill_(1)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    reps = max(1, min(args.steps, 20))
    out = {}
    for name, pattern, wps in [("flat, 2 waves/SIMD, 4 loads in flight", 0, 2),
                               ("flat, 4 waves/SIMD, 2 loads in flight", 0, 4),
                               ("flat, 8 waves/SIMD, 1 load in flight", 0, 8),
                               ("decode_split walk without arithmetic, 4 loads in flight "
                                "(the kernel's)", 1, 4),
                               ("decode_split walk, 2 loads in flight", 1, 2),
                               ("decode_split walk, 8 loads in flight", 1, 8)]:
        def one_pass():
            for l in range(L):
                rc = lib.hwkv_read_probe(buf.data_ptr() + l * per, per, pattern, wps,
                                         sink.data_ptr(), stream)
                if rc != 0:
                    raise RuntimeError(f"hwkv_read_probe returned {rc}")
        for _ in range(3):
            one_pass()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            one_pass()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b)
        out[name] = {"gbs": round(L * per * reps / (ms * 1e-3) / 1e9, 1),
                     "us_per_launch": round(ms * 1e3 / (reps * L), 2)}
    best = max(v["gbs"] for k, v in out.items() if k.startswith("flat"))
    result = {
        "metric": "read-probe GB/s (16 launches of 213.5 MB, the 112K decode step's reads)",
        "value": best,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": reps,
        "warmup": 3,
        "frac_of_hbm_peak": round(best / HBM_PEAK_GBS, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8 (loads only)",
        "data": "synthetic",
        "config": {"workload": f"probe: {L} regions of {per} bytes, one launch each per pass",
                   "patterns": out},
    }
    print(json.dumps(result), flush=True)


def calib_main(args, dev):
    import numpy as np
    import torch

    import workloads as W
    from paper_2609_02029_amd import hwkv

    cfg = W.CONFIGS["calib128k"]
    N, Hq, Hkv, D, S = cfg["prompt"][0], cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"], \
        cfg["n_sinks"]
    G = Hq // Hkv
    windows = [w for w in cfg["level_windows"] if w]
    rows = W.calib_rows(cfg)
    R = len(rows)
    scale = 1.0 / math.sqrt(D)
    k = W.normal_bf16_device((N, Hkv, D), cfg["seed"], 0, W.K, 0, device=dev)
    v = W.normal_bf16_device((N, Hkv, D), cfg["seed"], 0, W.V, 0, device=dev)
    q = W.normal_bf16_device((R, Hq, D), cfg["seed"], 0, W.Q_PROMPT, 0, device=dev)
    K = len(windows)
    outs = torch.empty((K + 1, R, Hq, D), dtype=torch.float32, device=dev)
    scores = torch.empty((K, R, Hq), dtype=torch.float32, device=dev)
    means = torch.empty((K, Hkv), dtype=torch.float32, device=dev)
    fmt = args.kv_format
    if fmt not in ("bf16", "fp8"):
        raise SystemExit("calib128k replays bf16 or fp8 caches (binary16 values are not bf16)")
    # fp8: every candidate over the trace as an fp8 cache stores it, with
    # the decode workloads' scale recipe per kv head
    scales = W.fp8_scales(cfg)[0] if fmt == "fp8" else None
    ws = torch.zeros(hwkv.calib_workspace_bytes(Hq, D, S, k.shape[0], R, n_kv_heads=Hkv,
                                                kv_format=fmt),
                     dtype=torch.uint8, device=dev)
    # algorithmic FLOP: every candidate of every row and q head, 4d per
    # retained key
    pairs = 0
    for w in windows + [0]:
        for t in rows:
            pairs += (t + 1) if w == 0 else min(t + 1, S + w)
    flop = pairs * Hq * 4 * D
    # the one-pass replay forms each (row, key) product once for every
    # candidate: the full candidate's pairs (edge tiles add a little)
    flop_once = sum(t + 1 for t in rows) * Hq * 4 * D
    steps, warmup = min(max(1, args.steps), 10), min(max(0, args.warmup), 3)

    def run():
        hwkv.calib_replay(k, v, rows, q, windows, S, scale, outs, scores, means, ws,
                          kv_format=fmt, k_scale=scales, v_scale=scales)

    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    ms = []
    for _ in range(steps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        run()
        b.record()
        torch.cuda.synchronize()
        ms.append(a.elapsed_time(b))
    ms_step = sum(ms) / len(ms)
    tfs = flop / (ms_step * 1e-3) / 1e12
    result = {
        "metric": CALIB_METRIC,
        "value": round(tfs, 1),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("bf16 (fp32 accumulate)" if fmt == "bf16"
                  else "fp8-e4m3 trace values, bf16 q (fp32 accumulate)"),
        "data": "synthetic",
        "config": {
            "workload": (f"calib128k: one traced layer of {N} tokens, {R} query rows from the "
                         f"final quarter, {Hq} q / {Hkv} kv heads, head_dim {D}, {S} sinks, "
                         f"candidates {windows} + full; outputs, scores and per-head means"),
            "kv_format": fmt,
            "algorithmic_flop_per_step": flop,
            "computed_flop_per_step": flop_once,
            "means": [[round(float(x), 5) for x in row] for row in means.cpu().numpy()],
        },
        "roofline": {
            "bound": "mfma",
            "kernel": ("replay_attn (one pass over the trace for every candidate) + merge + "
                       "scores + means; achieved = every candidate's algorithmic FLOP / time"),
            "achieved": round(tfs, 1),
            "peak": MFMA_BF16_PEAK_TFS,
            "unit": "TFLOP/s",
            "frac": round(tfs / MFMA_BF16_PEAK_TFS, 4),
            "traffic": None,
        },
    }
    if not args.no_cpu_baseline:
        import oracle
        bits = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        kh, vh, qh = bits(k), bits(v), bits(q)
        threads = max(1, min(16, os.cpu_count() or 1))
        spent, done_pairs, done = 0.0, 0, 0
        for i in range(R):
            t0 = time.perf_counter()
            oracle.replay_outputs(qh[i:i + 1], kh, vh, [rows[i]], S, windows + [0], scale,
                                  n_threads=threads)
            spent += time.perf_counter() - t0
            done_pairs += sum((rows[i] + 1) if w == 0 else min(rows[i] + 1, S + w)
                              for w in windows + [0])
            done += 1
            if spent >= args.cpu_seconds:
                break
        result["cpu_baseline"] = {
            "value": round(done_pairs * Hq * 4 * D / spent / 1e9, 3),
            "unit": "GFLOP/s",
            "ms_per_step": round(spent / done_pairs * pairs * 1e3, 1),
            "cores": threads,
            "kind": "oracle",
            "sample": (f"{done} of the {R} rows (all {Hq} q heads, every candidate), fp64 "
                       f"masked-full-history oracle, {spent:.1f} s; scaled by retained pairs"
                       + ("" if fmt == "bf16" else "; over the bf16 trace (the C oracle's "
                          "cost does not depend on the values)")),
        }
    print(json.dumps(result), flush=True)


def prefill_cpu_baseline(args, cfg, q, k, v, windows, scale, step_flop, gpu_ms):
    """The fp64 oracle on the host cores over the parity sample rows of the
    same workload (in order, until about ``--cpu-seconds``), scaled to the
    whole prefill by the sampled rows' share of the algorithmic FLOP."""
    import numpy as np
    import torch

    import oracle
    import workloads as W

    Hq, Hkv, D, S = cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"], cfg["n_sinks"]
    G = Hq // Hkv
    threads = max(1, min(16, os.cpu_count() or 1))
    rows = W.prefill_sample_rows(cfg)
    kh = k.view(torch.int16).cpu().numpy().view(np.uint16)
    vh = v.view(torch.int16).cpu().numpy().view(np.uint16)
    spent, flop, done = 0.0, 0, 0
    batch = 16
    for i in range(0, len(rows), batch):
        rr = np.asarray(rows[i:i + batch], dtype=np.int64)
        qr = q[torch.from_numpy(rr).to(q.device)].view(torch.int16).cpu().numpy().view(np.uint16)
        t0 = time.perf_counter()
        oracle.decode_layer(qr, [kh] * len(rr), [vh] * len(rr), rr, S, windows, scale,
                            n_threads=threads)
        spent += time.perf_counter() - t0
        for t in rr:
            flop += sum(G * prefill_pairs(0, int(t), int(t) + 1, S, w) * 4 * D for w in windows)
        done += len(rr)
        if spent >= args.cpu_seconds:
            break
    ms = spent / flop * step_flop * 1e3
    return {
        "value": round(flop / spent / 1e9, 3),
        "unit": "GFLOP/s",
        "ms_per_step": round(ms, 1),
        "cores": threads,
        "kind": "oracle",
        "sample": (f"{done} query rows (all {Hq} heads) of the parity sample of the 128K prefill, "
                   f"fp64 masked-full-history oracle, {spent:.1f} s of CPU time; "
                   f"scaled to the whole prefill by algorithmic FLOP"),
        "gpu_speedup": round(ms / gpu_ms, 1),
    }


if __name__ == "__main__":
    main()
