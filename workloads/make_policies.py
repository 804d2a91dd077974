"""Write ``policies.json``: the budget-constrained level matrices.

For each workload with a residency budget (lo, hi), draw whole
``[n_layers][n_kv_heads]`` matrices of level indices, iid uniform over the
codebook, from ``numpy.random.default_rng(SeedSequence([seed, 0, LEVELS, 0]))``
and keep the first one whose normalized rate (Eq. normalized-rate, evaluated
by the oracle at the workload's reference context, with sinks counted in the
retained tokens) lies in [lo, hi].  The accepted matrix, its rate and the
number of draws are stored.  Only the oracle is called.

Run:  python -m workloads.make_policies
"""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workloads as W  # noqa: E402


def draw(cfg, max_draws=1_000_000):
    lo, hi = cfg["budget"]
    lw = np.array(cfg["level_windows"], dtype=np.int64)
    r = W.rng(cfg["seed"], 0, W.LEVELS, 0)
    for i in range(1, max_draws + 1):
        m = r.integers(0, len(lw), size=(cfg["n_layers"], cfg["n_kv_heads"]))
        rate = oracle.rate(cfg["rate_ctx"], cfg["n_sinks"], lw[m].ravel())
        if lo <= rate <= hi:
            return m.tolist(), rate, i
    raise RuntimeError("no matrix met the budget")


def main():
    out = {}
    for name, cfg in W.CONFIGS.items():
        if cfg.get("budget") is None:
            continue
        m, rate, n = draw(cfg)
        out[name] = {"levels": m, "rate": rate, "draws": n,
                     "rate_ctx": cfg["rate_ctx"], "budget": list(cfg["budget"]),
                     "seed": cfg["seed"], "level_windows": cfg["level_windows"]}
        print(f"{name}: R={rate:.6f} after {n} draws")
    path = os.path.join(W.HERE, "policies.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
