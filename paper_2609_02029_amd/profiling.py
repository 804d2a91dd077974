"""Summaries of rocprofv3 results databases for the decode kernels.

``python -m paper_2609_02029_amd.profiling kernels DB``     per-kernel durations
``python -m paper_2609_02029_amd.profiling traffic DB_FETCH DB_WRITE MIB``
``python -m paper_2609_02029_amd.profiling record DB_FETCH DB_WRITE MIB``
    the decode_split line of the traffic table as JSON, with the hash of the
    kernel source it was measured on
    HBM traffic per dispatch of each kernel from a FETCH_SIZE run and a
    WRITE_SIZE run, each scaled by what the counter reads for the plain copy
    of MIB MiB that ``bench.py --copy-calibration MIB`` performs first
    (expected: MIB MiB read and MIB MiB written per copy).
"""
import collections
import hashlib
import json
import os
import re
import sqlite3
import statistics
import sys

KERNELS = r"(decode_split<[^>]*>|decode_combine<[^>]*>|prefill_write<[^>]*>|append_token<[^>]*>)"


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


def counter(db, name):
    """{dispatch id: (kernel, value summed over the counter's instances)}."""
    cur = sqlite3.connect(db).cursor()
    vals = collections.defaultdict(float)
    kern = {}
    for did, kn, cn, v in cur.execute(
            "select dispatch_id, kernel_name, counter_name, value from counters_collection"):
        if cn == name:
            vals[did] += v
            kern[did] = short(kn)
    return {d: (kern[d], vals[d]) for d in vals}


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


def kernel_source_hash():
    """Hash of the decode kernel source: a traffic record is current only
    while the kernel it was measured on is unchanged."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc",
                        "decode_kernels.hip")
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_record(db_fetch, db_write, mib, kernel="decode_split<256, 6>"):
    sf, sw, per = traffic(db_fetch, db_write, mib)
    fv, fn = per["fetch"][kernel]
    wv, _ = per["write"].get(kernel, (0.0, 0))
    return {"kernel": kernel, "dispatches": fn, "fetch_bytes": fv * sf * 1024,
            "write_bytes": wv * sw * 1024, "fetch_scale": sf, "write_scale": sw,
            "copy_mib": mib, "kernel_source_sha256_16": kernel_source_hash()}


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
        print(json.dumps(traffic_record(argv[1], argv[2], float(argv[3])), indent=1))
    else:
        raise SystemExit(__doc__)


if __name__ == "__main__":
    main(sys.argv[1:])
