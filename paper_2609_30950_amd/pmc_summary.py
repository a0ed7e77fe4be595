"""Turn rocprofv3 --pmc CSVs into per-launch HBM bytes for profiles/traffic.json.

    python -m paper_2609_30950_amd.pmc_summary --workload decode \\
        --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR --copy-mib 512

Each DIR holds a run_counter_collection.csv.  The kda kernels' FETCH_SIZE and
WRITE_SIZE per dispatch are scaled by the bytes-per-count factor of a plain
copy kernel of known size (pmc_copy.py) measured the same way.
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


KERNEL_SOURCES = ("kda_alloc.hpp", "kda_device.hpp", "kda_kernels.hip", "kda_kernels.hpp")


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
    for k in ("k_requant", "k_chunk", "k_alloc", "k_step32", "k_pack", "k_unpack"):
        if "kda::" + k in name:
            return {"k_chunk": "stats", "k_requant": "requant", "k_alloc": "alloc"}.get(k, k[2:])
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", required=True)
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--copy-fetch", required=True)
    ap.add_argument("--copy-write", required=True)
    ap.add_argument("--copy-mib", type=int, required=True)
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "traffic.json"))
    a = ap.parse_args()
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
