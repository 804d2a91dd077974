"""Summaries of rocprofv3 results databases for the hwkv kernels.

``python -m paper_2609_02029_amd.profiling kernels DB``     per-kernel durations
``python -m paper_2609_02029_amd.profiling traffic DB_FETCH DB_WRITE MIB``
    HBM traffic per dispatch of each kernel from a FETCH_SIZE run and a
    WRITE_SIZE run, each scaled by what the counter reads for the plain copy
    of MIB MiB that ``bench.py --copy-calibration MIB`` performs first
    (expected: MIB MiB read and MIB MiB written per copy).
``python -m paper_2609_02029_amd.profiling record DB_FETCH DB_WRITE MIB [KERNEL]``
    the head_dim-256 line of one kernel in the traffic table as JSON
    (``decode_split`` by default, ``decode_mfma`` or ``prefill_attn``), with the hash of the
    kernel source it was measured on
``python -m paper_2609_02029_amd.profiling mfma DB``
    MFMA busy fraction and bf16 MFMA FLOP per dispatch of every kernel that
    issued MFMA, from a run with SQ_VALU_MFMA_BUSY_CYCLES,
    SQ_INSTS_VALU_MFMA_MOPS_BF16 and GRBM_GUI_ACTIVE (busy cycles summed over
    the 1024 SIMDs over the GPU's active cycles; one MOP = 512 FLOP)
``python -m paper_2609_02029_amd.profiling lds DB``
    LDS bank-conflict and LDS-active cycles per dispatch (SQ_LDS_BANK_CONFLICT,
    SQ_LDS_IDX_ACTIVE, GRBM_GUI_ACTIVE), as fractions of CU cycles
``python -m paper_2609_02029_amd.profiling stalls DB``
    per kernel, summed over its dispatches: where its wavefronts' cycles go
    (SQ_WAIT_ANY, SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_VALU / _VMEM / _LDS over
    SQ_WAVE_CYCLES) and its VALU instructions per wavefront (SQ_INSTS_VALU
    over SQ_WAVES)
"""
import collections
import hashlib
import json
import os
import re
import sqlite3
import statistics
import sys

KERNELS = (r"(decode_split<[^>]*>|decode_mfma<[^>]*>|decode_combine<[^>]*>|prefill_write<[^>]*>"
           r"|append_token<[^>]*>|prefill_attn<[^>]*>)")
N_SIMD = 1024   # 256 CUs x 4 SIMDs
N_CU = 256
# GRBM_GUI_ACTIVE comes back as one value per dispatch that sums the active
# cycles of the 8 XCDs (an 8.9 ms dispatch reads 1.59e8 = 8 x 2.2 GHz x 8.9 ms)
N_XCD = 8


def short(name):
    m = re.search(KERNELS, name or "")
    if m:
        return m.group(1)
    if "copyBuffer" in (name or ""):  # the runtime's blit kernel (torch copy_)
        return "copy:" + (name or "")[:60]
    return (name or "")[:60]


def kernels(db):
    cur = sqlite3.connect(db).cursor()
    rows = list(cur.execute("select name, start, end from kernels order by start"))
    by = collections.defaultdict(list)
    for n, s, e in rows:
        by[short(n)].append((e - s) / 1000.0)
    out = []
    for k, v in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        out.append((k, len(v), statistics.mean(v), statistics.median(v), min(v), max(v), sum(v)))
    return out


def counter(db, name, reduce="sum"):
    """{dispatch id: (kernel, value reduced over the counter's instances)}."""
    cur = sqlite3.connect(db).cursor()
    vals = {}
    kern = {}
    for did, kn, cn, v in cur.execute(
            "select dispatch_id, kernel_name, counter_name, value from counters_collection"):
        if cn == name:
            if did not in vals:
                vals[did] = v
            elif reduce == "sum":
                vals[did] += v
            else:
                vals[did] = max(vals[did], v)
            kern[did] = short(kn)
    return {d: (kern[d], vals[d]) for d in vals}


def mfma(db):
    busy = counter(db, "SQ_VALU_MFMA_BUSY_CYCLES")
    mops = counter(db, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
    act = counter(db, "GRBM_GUI_ACTIVE", reduce="max")
    rows = []
    for d in sorted(busy):
        k, b = busy[d]
        if b <= 0 or d not in act:
            continue
        cyc = act[d][1] / N_XCD
        rows.append((d, k, b / (cyc * N_SIMD), mops.get(d, (k, 0.0))[1] * 512, cyc))
    return rows


def lds(db):
    conf = counter(db, "SQ_LDS_BANK_CONFLICT")
    idx = counter(db, "SQ_LDS_IDX_ACTIVE")
    act = counter(db, "GRBM_GUI_ACTIVE", reduce="max")
    rows = []
    for d in sorted(idx):
        k, a = idx[d]
        if a <= 0 or d not in act:
            continue
        cyc = act[d][1] / N_XCD * N_CU
        rows.append((d, k, a / cyc, conf.get(d, (k, 0.0))[1] / cyc))
    return rows


def traffic(db_fetch, db_write, mib):
    f = counter(db_fetch, "FETCH_SIZE")
    w = counter(db_write, "WRITE_SIZE")
    copies_f = [v for k, v in f.values() if k.startswith("copy:") and v > 0]
    copies_w = [v for k, v in w.values() if k.startswith("copy:") and v > 0]
    known_kib = mib * 1024.0
    scale_f = known_kib / statistics.median(copies_f) if copies_f else None
    scale_w = known_kib / statistics.median(copies_w) if copies_w else None
    per = {}
    for name, table, scale in (("fetch", f, scale_f), ("write", w, scale_w)):
        acc = collections.defaultdict(list)
        for k, v in table.values():
            acc[k].append(v)
        per[name] = {k: (statistics.mean(v), len(v)) for k, v in acc.items()}
    return scale_f, scale_w, per


# source files of each profiled kernel (the split kernel's template and the
# format helpers it inlines)
SOURCES = {"decode_split<": ["decode_split.h", "kv_format.h"],
           "decode_mfma<": ["decode_mfma.h", "decode_split.h", "kv_format.h"],
           "prefill_attn<": ["prefill_attn_kernels.hip"]}


def kernel_source_hash(kernel="decode_split<256, 6, 0>"):
    """Hash of a kernel's source files: a traffic record is current only while
    the kernel it was measured on is unchanged."""
    files = next(f for k, f in SOURCES.items() if kernel.startswith(k))
    h = hashlib.sha256()
    for src in files:
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", src)
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_record(db_fetch, db_write, mib, kernel="decode_split<256, 6, 0>"):
    sf, sw, per = traffic(db_fetch, db_write, mib)
    fv, fn = per["fetch"][kernel]
    wv, _ = per["write"].get(kernel, (0.0, 0))
    return {"kernel": kernel, "dispatches": fn, "fetch_bytes": fv * sf * 1024,
            "write_bytes": wv * sw * 1024, "fetch_scale": sf, "write_scale": sw,
            "copy_mib": mib, "kernel_source_sha256_16": kernel_source_hash(kernel)}


STALL_COUNTERS = ("SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_VALU",
                  "SQ_ACTIVE_INST_VMEM", "SQ_ACTIVE_INST_LDS")


def stalls(db):
    """{kernel: (dispatches, {counter: fraction of SQ_WAVE_CYCLES}, VALU
    instructions per wavefront)}."""
    per = {}
    for name in ("SQ_WAVE_CYCLES", "SQ_WAVES", "SQ_INSTS_VALU") + STALL_COUNTERS:
        per[name] = counter(db, name)
    out = {}
    for k in sorted({v[0] for v in per["SQ_WAVE_CYCLES"].values()}):
        ds = [d for d, (kk, _) in per["SQ_WAVE_CYCLES"].items() if kk == k]
        tot = lambda name: sum(per[name].get(d, (k, 0.0))[1] for d in ds)
        cyc = tot("SQ_WAVE_CYCLES")
        if cyc <= 0:
            continue
        waves = tot("SQ_WAVES")
        out[k] = (len(ds), {n: tot(n) / cyc for n in STALL_COUNTERS},
                  tot("SQ_INSTS_VALU") / waves if waves else float("nan"))
    return out


def main(argv):
    if argv[0] == "kernels":
        print("| kernel | calls | mean us | median us | min us | max us | total us |")
        print("|---|---|---|---|---|---|---|")
        for k, n, mean, med, mn, mx, tot in kernels(argv[1]):
            print(f"| {k} | {n} | {mean:.2f} | {med:.2f} | {mn:.2f} | {mx:.2f} | {tot:.1f} |")
    elif argv[0] == "traffic":
        sf, sw, per = traffic(argv[1], argv[2], float(argv[3]))
        print(f"copy calibration: FETCH_SIZE scale {sf}, WRITE_SIZE scale {sw} "
              f"(known KiB / counted KiB for a {argv[3]} MiB copy)")
        print("| kernel | dispatches | FETCH_SIZE KiB/dispatch | scaled fetch MB | "
              "WRITE_SIZE KiB/dispatch | scaled write MB |")
        print("|---|---|---|---|---|---|")
        for k in sorted(set(per["fetch"]) | set(per["write"])):
            fv, fn = per["fetch"].get(k, (0.0, 0))
            wv, _ = per["write"].get(k, (0.0, 0))
            fs = fv * (sf or 0) * 1024 / 1e6
            ws = wv * (sw or 0) * 1024 / 1e6
            print(f"| {k} | {fn} | {fv:.0f} | {fs:.2f} | {wv:.0f} | {ws:.2f} |")
    elif argv[0] == "record":
        prefix = argv[4] + "<" if len(argv) > 4 else "decode_split<"
        _, _, per = traffic(argv[1], argv[2], float(argv[3]))
        kernel = next(k for k in per["fetch"] if k.startswith(prefix + "256"))
        print(json.dumps(traffic_record(argv[1], argv[2], float(argv[3]), kernel), indent=1))
    elif argv[0] == "mfma":
        rows = mfma(argv[1])
        print("| dispatch | kernel | MFMA busy (of SIMD cycles) | bf16 MFMA TFLOP | GPU cycles |")
        print("|---|---|---|---|---|")
        for d, k, u, fl, a in rows:
            print(f"| {d} | {k} | {u:.3f} | {fl / 1e12:.3f} | {a:.0f} |")
        by = collections.defaultdict(list)
        for d, k, u, fl, a in rows:
            by[k].append((u, fl, a))
        for k, v in by.items():
            tot_a = sum(x[2] for x in v)
            print(f"\n{k}: {len(v)} dispatches, cycle-weighted MFMA busy "
                  f"{sum(x[0] * x[2] for x in v) / tot_a:.3f}, bf16 MFMA FLOP "
                  f"{sum(x[1] for x in v) / 1e12:.2f} T")
    elif argv[0] == "lds":
        print("| dispatch | kernel | LDS active (of CU cycles) | bank conflict (of CU cycles) |")
        print("|---|---|---|---|")
        for d, k, a, c in lds(argv[1]):
            print(f"| {d} | {k} | {a:.3f} | {c:.4f} |")
    elif argv[0] == "stalls":
        print("| kernel | dispatches | " + " | ".join(STALL_COUNTERS) +
              " | VALU instructions per wavefront |")
        print("|---|---|" + "---|" * len(STALL_COUNTERS) + "---|")
        for k, (n, f, vpw) in stalls(argv[1]).items():
            print(f"| {k} | {n} | " + " | ".join(f"{f[c]:.3f}" for c in STALL_COUNTERS) +
                  f" | {vpw:.0f} |")
    else:
        raise SystemExit(__doc__)


if __name__ == "__main__":
    main(sys.argv[1:])
