"""Summarise a rocprofv3 kernel trace (rocpd SQLite output) per kernel and per
kernel family (the families the library's launch tracer uses).

Usage: python paper_2312_04429_amd/profsum.py RESULTS_DB [UNITS] [--title T] [--cmd C]
UNITS divides totals (e.g. the number of UNet evaluations in the trace).
"""
import argparse
import sqlite3

FAMILIES = [("conv3x3_igemm", "gemm_f16<1"), ("linear_gemm", "gemm_f16<0"),
            ("conv3x3_igemm", "gemm_s<1"), ("linear_gemm", "gemm_s<0"),
            ("attention", "attn_f16"), ("cache_scan", "lk_scan"), ("splitk_reduce", "splitk_reduce"),
            ("groupnorm", "gn_"), ("layernorm", "layernorm"), ("other", "")]


def family(name):
    for fam, key in FAMILIES:
        if key in name:
            return fam
    return "other"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("db")
    ap.add_argument("units", nargs="?", type=float, default=1.0)
    ap.add_argument("--title", default="")
    ap.add_argument("--cmd", default="")
    a = ap.parse_args()
    cur = sqlite3.connect(a.db).cursor()
    rows = cur.execute("select name, count(*), sum(end-start), avg(end-start), min(end-start), "
                       "max(end-start) from kernels group by name order by sum(end-start) desc"
                       ).fetchall()
    tot = sum(r[2] for r in rows)
    if a.title:
        print(f"# {a.title}\n")
    if a.cmd:
        print(f"command: `{a.cmd}`\n")
    print(f"total kernel time {tot / 1e6:.3f} ms; per unit ({a.units:g} units) "
          f"{tot / 1e6 / a.units:.3f} ms\n")
    print("| family | launches/unit | ms/unit | avg us/launch |")
    print("|---|---:|---:|---:|")
    fam = {}
    for r in rows:
        f = family(r[0])
        c, t = fam.get(f, (0, 0))
        fam[f] = (c + r[1], t + r[2])
    for f, (c, t) in sorted(fam.items(), key=lambda x: -x[1][1]):
        print(f"| {f} | {c / a.units:.1f} | {t / 1e6 / a.units:.3f} | {t / c / 1e3:.2f} |")
    print("\n| kernel | calls | total ms | avg us | min us | max us |")
    print("|---|---:|---:|---:|---:|---:|")
    for r in rows[:25]:
        print(f"| `{r[0][:90]}` | {r[1]} | {r[2] / 1e6:.3f} | {r[3] / 1e3:.2f} | {r[4] / 1e3:.2f} | "
              f"{r[5] / 1e3:.2f} |")


if __name__ == "__main__":
    main()
