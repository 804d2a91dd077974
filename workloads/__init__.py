"""Seeded synthetic inputs shared by the tests and the benchmark.

This module holds no part of the method's arithmetic: it only draws seeded
normal values, rounds them to bf16, and describes the workload shapes.  The
budget-constrained level matrices of the 112K and batched workloads are read
from ``policies.json``, written by ``make_policies.py`` with the oracle's rate
function (they are inputs, fixed once and committed).

Recipe (per tensor): ``numpy.random.default_rng(SeedSequence([cfg_seed,
layer, kind, step]))`` draws fp32 standard normals which are rounded to bf16
(round to nearest, ties to even).  Large tensors are drawn on the device with
a ``torch.Generator`` seeded from the same SeedSequence; either way both the
HIP path and the oracle receive the same bf16 bit patterns.
"""
import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))

# kinds of seeded tensors (Q_PROMPT: queries of the prompt tokens, for
# prefill attention)
Q, K, V, K_NEW, V_NEW, LEVELS, PROMPTS, OUTLIERS, SAMPLE, Q_PROMPT = range(10)

FULL = 0  # window encoding: 0 = full history

# Workload shapes.  "K" = 1024 tokens.
CONFIGS = {
    # 1 global layer, 8 q / 2 kv heads, d=64, 2048-token prompt, 16 steps;
    # kv head 0 keeps 4 sinks + 256 recent tokens, kv head 1 full history.
    "pr1": dict(name="pr1", seed=1, n_layers=1, batch=1, n_q_heads=8,
                n_kv_heads=2, head_dim=64, n_sinks=4,
                level_windows=[256, FULL], levels=[[0, 1]],
                prompt=[2048], steps=16, max_ctx=2048 + 16),
    # 1 residual global layer at 32K: 24 q / 4 kv, d=256, 2 outlier channels
    # per kv head scaled x8; windows drawn per head over 4 levels.
    "ctx32k": dict(name="ctx32k", seed=2, n_layers=1, batch=1, n_q_heads=24,
                   n_kv_heads=4, head_dim=256, n_sinks=4,
                   level_windows=[1024, 4096, 16384, FULL], levels=None,
                   prompt=[32768 - 256], steps=256, max_ctx=32768,
                   outlier_channels=2, outlier_scale=8.0),
    # 112K context through 16 stacked residual global layers, 50% budget.
    "ctx112k": dict(name="ctx112k", seed=3, n_layers=16, batch=1,
                    n_q_heads=24, n_kv_heads=4, head_dim=256, n_sinks=4,
                    level_windows=[2048, 8192, 32768, FULL], levels=None,
                    prompt=[114688 - 128], steps=128, max_ctx=114688,
                    budget=(0.45, 0.50), rate_ctx=114688),
    # batched serving: 16 sequences, prompts U[16K, 64K], 8 layers, 25% budget.
    "batch16": dict(name="batch16", seed=4, n_layers=8, batch=16,
                    n_q_heads=24, n_kv_heads=4, head_dim=256, n_sinks=4,
                    level_windows=[1024, 4096, 16384, FULL], levels=None,
                    prompt=None, prompt_range=(16384, 65536), steps=64,
                    max_ctx=65536 + 64, budget=(0.20, 0.25), rate_ctx=65536),
    # calibration replay of one traced layer: a 128K-token trace, 256 query
    # positions sampled from its final quarter, candidates {2K, 8K, 32K, full}.
    "calib128k": dict(name="calib128k", seed=6, n_layers=1, batch=1, n_q_heads=24,
                      n_kv_heads=4, head_dim=256, n_sinks=4,
                      level_windows=[2048, 8192, 32768, FULL], levels=[[3, 3, 3, 3]],
                      prompt=[131072], n_rows=256, steps=0, max_ctx=131072),
    # long prefill: 128K prompt in 8K chunks; kv head h gets level h.
    "prefill128k": dict(name="prefill128k", seed=5, n_layers=1, batch=1,
                        n_q_heads=24, n_kv_heads=4, head_dim=256, n_sinks=4,
                        level_windows=[2048, 8192, 32768, FULL],
                        levels=[[0, 1, 2, 3]], prompt=[131072], chunk=8192,
                        steps=0, max_ctx=131072),
}


def seed_seq(*words):
    return np.random.SeedSequence([int(w) for w in words])


def rng(*words):
    return np.random.default_rng(seed_seq(*words))


def torch_seed(*words):
    """A 63-bit torch seed derived from the same SeedSequence words."""
    return int(seed_seq(*words).generate_state(2, dtype=np.uint64)[0] >> np.uint64(1))


def f32_to_bf16_bits(x):
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + (((u >> np.uint64(16)) & np.uint64(1)) + np.uint64(0x7FFF)))
         >> np.uint64(16)).astype(np.uint16)
    r[np.isnan(x)] = np.uint16(0x7FC0)
    return r


def bf16_bits_to_f32(b):
    """Exact widening of bf16 bits to fp32 (input preparation / display only)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(shape, *words, scale_channels=None, scale=1.0):
    """Seeded N(0,1) values rounded to bf16, as uint16 bits, on the host.

    ``scale_channels``: optional ``{kv_head: [channels]}`` whose values are
    multiplied by ``scale`` before rounding (last two axes are [head, d])."""
    x = rng(*words).standard_normal(size=shape, dtype=np.float32)
    if scale_channels:
        for h, chans in scale_channels.items():
            for c in chans:
                x[..., h, c] *= np.float32(scale)
    return f32_to_bf16_bits(x)


def normal_bf16_device(shape, *words, device="cuda", scale_channels=None,
                       scale=1.0):
    """Seeded N(0,1) bf16 tensor drawn on ``device`` (torch.bfloat16)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(torch_seed(*words))
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if scale_channels:
        for h, chans in scale_channels.items():
            for c in chans:
                x[..., h, c] *= scale
    return x.to(torch.bfloat16)


def outlier_channels(cfg):
    """Per kv head, the distinct channels scaled up (``None`` if the workload
    has none)."""
    n = cfg.get("outlier_channels", 0)
    if not n:
        return None
    r = rng(cfg["seed"], 0, OUTLIERS, 0)
    return {h: sorted(int(c) for c in r.choice(cfg["head_dim"], size=n, replace=False))
            for h in range(cfg["n_kv_heads"])}


def fp8_scales(cfg, sigmas=8.0):
    """fp8 scales of every (layer, kv head), for K and for V alike: the
    synthetic keys and values are unit normal (outlier channels scaled by
    ``outlier_scale``), and ``sigmas`` standard deviations of the largest
    channel map to the largest E4M3 magnitude, 448."""
    s = sigmas * max(1.0, float(cfg.get("outlier_scale", 1.0))) / 448.0
    return np.full((cfg["n_layers"], cfg["n_kv_heads"]), s, dtype=np.float32)


def _stored_policies():
    path = os.path.join(HERE, "policies.json")
    with open(path) as f:
        return json.load(f)


def levels(cfg):
    """``[n_layers][n_kv_heads]`` level indices of a workload."""
    if cfg.get("levels") is not None:
        return [list(row) for row in cfg["levels"]]
    if cfg.get("budget") is not None:
        return _stored_policies()[cfg["name"]]["levels"]
    r = rng(cfg["seed"], 0, LEVELS, 0)
    m = r.integers(0, len(cfg["level_windows"]), size=(cfg["n_layers"], cfg["n_kv_heads"]))
    return m.tolist()


def prompts(cfg):
    """Prompt length of every sequence."""
    if cfg.get("prompt") is not None:
        return list(cfg["prompt"])
    lo, hi = cfg["prompt_range"]
    r = rng(cfg["seed"], 0, PROMPTS, 0)
    return [int(x) for x in r.integers(lo, hi, size=cfg["batch"], endpoint=True)]


def prefill_sample_rows(cfg, n_rows=512):
    """Query rows of the long-prefill workload checked against the oracle:
    boundary rows (each chunk's first and last token; S - 1, S, S + w - 1,
    S + w and S + w + 1 for every finite window) and, to make up ``n_rows``,
    rows drawn uniformly without replacement from the rest of [0, N)."""
    N = cfg["prompt"][0]
    S = cfg["n_sinks"]
    edge = set()
    for p0 in range(0, N, cfg["chunk"]):
        edge.update((p0, min(p0 + cfg["chunk"], N) - 1))
    for w in cfg["level_windows"]:
        if w:
            edge.update(t for t in (S - 1, S, S + w - 1, S + w, S + w + 1) if 0 <= t < N)
    edge = sorted(edge)
    rest = np.setdiff1d(np.arange(N), np.asarray(edge))
    r = rng(cfg["seed"], 0, SAMPLE, 0)
    extra = r.choice(rest, size=max(0, n_rows - len(edge)), replace=False)
    return sorted(edge + [int(x) for x in extra])


def calib_rows(cfg):
    """The calibration workload's query positions: ``n_rows`` distinct
    positions drawn uniformly from the final quarter of the trace, ascending
    (the paper samples 256 unique positions from the final quarter)."""
    N = cfg["prompt"][0]
    r = rng(cfg["seed"], 0, SAMPLE, 1)
    return sorted(int(x) for x in r.choice(np.arange(N - N // 4, N), size=cfg["n_rows"],
                                           replace=False))


def windows_of(cfg, lv=None):
    """``[n_layers][n_kv_heads]`` windows (0 = full)."""
    lv = levels(cfg) if lv is None else lv
    return [[int(cfg["level_windows"][k]) for k in row] for row in lv]


def small(cfg_name, **over):
    """A copy of a workload with some fields replaced (for reduced tests)."""
    c = dict(CONFIGS[cfg_name])
    c.update(over)
    return c
