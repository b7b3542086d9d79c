"""Records the attention kernel's HBM traffic per launch for bench.py.

Input: the counter CSVs of two rocprofv3 runs of

    python bench.py --steps 2 --warmup 1 --sets 1 --no-cpu-baseline --copy-calibration-mib 1024

one with ``--pmc FETCH_SIZE`` and one with ``--pmc WRITE_SIZE`` (both with
``--kernel-include-regex "bsattn|copy"``).  FETCH_SIZE and WRITE_SIZE are
read in KiB per dispatch.  Each counter is scaled by the factor that makes
it read the known size on the device copy of the calibration buffer (the
copy reads and writes that many bytes), then averaged over the attention
kernel's dispatches.

Output: measured_traffic.json beside this file, holding the bytes per launch
together with the SHA-256 of the kernel source; bench.py reports the figure
only while the source still matches.

    python -m paper_2609_32420_amd.traffic_record --fetch F.csv --write W.csv \\
        --copy-mib 1024 --head-dim 128 --block 128
"""
import argparse
import csv
import hashlib
import json
import os
import statistics

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "measured_traffic.json")
SOURCE = os.path.join(HERE, "csrc", "attn_kernels.hip")


def _per_dispatch(path, counter, name_part):
    vals = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter or name_part not in r["Kernel_Name"]:
                continue
            key = r.get("Dispatch_Id") or r.get("Correlation_Id") or str(len(vals))
            vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
    return list(vals.values())


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--copy-mib", type=int, required=True)
    ap.add_argument("--head-dim", type=int, required=True)
    ap.add_argument("--block", type=int, required=True)
    ap.add_argument("--kernel", default="bsattn_kernel")
    ap.add_argument("--copy-kernel", default="copyBuffer")
    a = ap.parse_args()
    copy_kib = a.copy_mib * 1024.0
    cf = _per_dispatch(a.fetch, "FETCH_SIZE", a.copy_kernel)
    cw = _per_dispatch(a.write, "WRITE_SIZE", a.copy_kernel)
    # the calibration copy is the largest copy dispatch of each run
    f_fetch = copy_kib / max(cf)
    f_write = copy_kib / max(cw)
    kf = _per_dispatch(a.fetch, "FETCH_SIZE", a.kernel)
    kw = _per_dispatch(a.write, "WRITE_SIZE", a.kernel)
    fetch_b = statistics.mean(kf) * f_fetch * 1024.0
    write_b = statistics.mean(kw) * f_write * 1024.0
    rec = {
        "kernel": "%s<%d, %d, false>" % (a.kernel, a.head_dim, a.block),
        "head_dim": a.head_dim,
        "block": a.block,
        "source_sha256": hashlib.sha256(open(SOURCE, "rb").read()).hexdigest(),
        "dispatches": [len(kf), len(kw)],
        "fetch_kib_raw": statistics.mean(kf),
        "write_kib_raw": statistics.mean(kw),
        "copy_factor_fetch": f_fetch,
        "copy_factor_write": f_write,
        "fetch_bytes_per_launch": fetch_b,
        "write_bytes_per_launch": write_b,
        "bytes_per_launch": fetch_b + write_b,
    }
    with open(OUT, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec, indent=1))


if __name__ == "__main__":
    main()
