"""Summaries of rocprofv3 output for profiles/.

    python -m paper_2609_30950_amd.pmc_summary --workload decode \\
        --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR --copy-mib 512
    python -m paper_2609_30950_amd.pmc_summary --trace DIR --last N
    python -m paper_2609_30950_amd.pmc_summary --sq DIR

Traffic: each DIR holds a run_counter_collection.csv.  The kda kernels'
FETCH_SIZE and WRITE_SIZE per dispatch are scaled by the bytes-per-count
factor of a plain copy kernel of known size (pmc_copy.py) measured the same
way, and written to profiles/traffic.json.
Trace: per kernel, the mean/median/min/max duration of the last N dispatches
of a --kernel-trace run (the timed steps of a benchmark run; warm-up
dispatches come first).
SQ: per kernel, the median per dispatch of every counter of a --pmc run.
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import statistics

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


# device-kernel sources that the counter summaries describe
KERNEL_SOURCES = ("kda_alloc.hpp", "kda_chunked.hip", "kda_device.hpp", "kda_kernels.hip",
                  "kda_kernels.hpp", "kda_record.hpp", "kda_recur.hpp", "kda_requant.hpp")


def source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(HERE, "csrc")
    for f in KERNEL_SOURCES:
            h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def per_kernel(d, counter):
    vals = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return vals


def short(name):
    for k in ("k_chunk_prep", "k_chunk_apply", "k_chunk_rates"):
        if "kda::" + k in name:
            return k[8:]
    for k in ("k_requant", "k_chunk", "k_alloc", "k_step32", "k_pack", "k_unpack"):
        if "kda::" + k in name:
            return {"k_chunk": "stats", "k_requant": "requant", "k_alloc": "alloc"}.get(k, k[2:])
    return None


def trace_summary(d, last):
    """{kernel: (n, mean_us, median_us, min_us, max_us)} over the last dispatches."""
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            rows.append((int(r["Start_Timestamp"]), r["Kernel_Name"],
                         (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0))
    rows.sort()
    by = {}
    for _, name, us in rows:
        by.setdefault(name, []).append(us)
    out = {}
    for name, v in by.items():
        v = v[-last:]
        out[name] = (len(v), statistics.mean(v), statistics.median(v), min(v), max(v))
    return out


def sq_summary(d):
    out = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            out.setdefault(r["Kernel_Name"], {}).setdefault(r["Counter_Name"], []).append(
                float(r["Counter_Value"]))
    return {k: {c: statistics.median(v) for c, v in cs.items()} for k, cs in out.items()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace")
    ap.add_argument("--last", type=int, default=120)
    ap.add_argument("--sq")
    ap.add_argument("--workload")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--copy-mib", type=int)
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "traffic.json"))
    a = ap.parse_args()
    if a.trace:
        for name, (n, mean, med, lo, hi) in sorted(trace_summary(a.trace, a.last).items(),
                                                   key=lambda kv: -kv[1][1]):
            print(f"| `{name[:60]}` | {n} | {mean:.1f} | {med:.1f} | {lo:.1f} | {hi:.1f} |")
        return
    if a.sq:
        print(json.dumps(sq_summary(a.sq), indent=1))
        return
    nbytes = a.copy_mib * 1024 * 1024
    factors = {}
    for cnt, d in (("FETCH_SIZE", a.copy_fetch), ("WRITE_SIZE", a.copy_write)):
        v = [x for k, xs in per_kernel(d, cnt).items() if "copy" in k.lower() for x in xs]
        factors[cnt] = nbytes / statistics.median(v)
    out = json.load(open(a.out)) if os.path.exists(a.out) else {}
    res = {}
    fetch = per_kernel(a.fetch, "FETCH_SIZE")
    write = per_kernel(a.write, "WRITE_SIZE")
    for name, fv in fetch.items():
        s = short(name)
        if s is None or name not in write:
            continue
        fb = statistics.median(fv) * factors["FETCH_SIZE"]
        wb = statistics.median(write[name]) * factors["WRITE_SIZE"]
        res[s] = dict(fetch_bytes_per_launch=fb, write_bytes_per_launch=wb,
                      hbm_bytes_per_launch=fb + wb, source_hash=source_hash(),
                      bytes_per_count=factors)
    out[a.workload] = res
    json.dump(out, open(a.out, "w"), indent=1, sort_keys=True)
    print(json.dumps(res, indent=1))


if __name__ == "__main__":
    main()
