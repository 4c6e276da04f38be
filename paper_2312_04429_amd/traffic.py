"""HBM bytes per kernel launch from two rocprofv3 --pmc passes.

Pass 1 collects FETCH_SIZE, pass 2 WRITE_SIZE (KiB per dispatch).  Each is
scaled by what the same counter reads for the calibration dispatch of the
benchmark (`bench.py --calib-copy`: one elementwise kernel that reads and
writes exactly 1 GiB), then averaged per launch of a kernel family.

Usage: python paper_2312_04429_amd/traffic.py FETCH_CSV WRITE_CSV OUT_DIR --cmd "..."
Writes OUT_DIR/traffic_<family>.json for the conv, linear, attention and scan
families, tagged with the hash of the kernel source they were taken on.
"""
import argparse
import csv
import hashlib
import json
import os

HERE = os.path.dirname(os.path.abspath(__file__))
FAMS = {"conv3x3_igemm": (("gemm_f16<1", "gemm_s<1"), ["gemm.hip", "gemm.h"]),
        "linear_gemm": (("gemm_f16<0", "gemm_s<0"), ["gemm.hip", "gemm.h"]),
        "attention": (("attn_f16",), ["attention.hip"]),
        "cache_scan": (("lk_scan",), ["lookup.hip"])}
CALIB_BYTES = float(1 << 30)


def sha(files):
    h = hashlib.sha256()
    for f in files:
        h.update(open(os.path.join(HERE, "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def per_dispatch(path, counter):
    vals = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        key = (r["Dispatch_Id"], r["Kernel_Name"])
        vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
    return vals


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("fetch_csv")
    ap.add_argument("write_csv")
    ap.add_argument("out_dir")
    ap.add_argument("--cmd", default="")
    a = ap.parse_args()
    fetch = per_dispatch(a.fetch_csv, "FETCH_SIZE")
    write = per_dispatch(a.write_csv, "WRITE_SIZE")
    cf = [v for (d, n), v in fetch.items() if "elementwise" in n]
    cw = [v for (d, n), v in write.items() if "elementwise" in n]
    if not cf or not cw:
        raise SystemExit("calibration dispatch not found")
    kib_f = max(cf) * 1024.0 / CALIB_BYTES   # counter bytes per true byte
    kib_w = max(cw) * 1024.0 / CALIB_BYTES
    for fam, (keys, files) in FAMS.items():
        f = [v for (d, n), v in fetch.items() if any(k in n for k in keys)]
        w = [v for (d, n), v in write.items() if any(k in n for k in keys)]
        if not f or not w:
            continue
        fb = sum(f) / len(f) * 1024.0 / kib_f
        wb = sum(w) / len(w) * 1024.0 / kib_w
        rec = {"family": fam, "kernel_source_sha": sha(files), "launches_fetch": len(f),
               "launches_write": len(w), "fetch_bytes_per_launch": fb,
               "write_bytes_per_launch": wb, "hbm_bytes_per_launch": fb + wb,
               "calibration": {"fetch_counter_bytes_per_byte": kib_f,
                               "write_counter_bytes_per_byte": kib_w,
                               "dispatch": "elementwise x*2 over 2^28 float32 (1 GiB in, 1 GiB out)"},
               "command": a.cmd}
        with open(os.path.join(a.out_dir, f"traffic_{fam}.json"), "w") as fh:
            json.dump(rec, fh, indent=1)
        print(fam, f"{fb / 1e6:.2f} MB fetch + {wb / 1e6:.2f} MB write per launch")


if __name__ == "__main__":
    main()
