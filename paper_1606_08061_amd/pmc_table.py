"""Per-kernel averages of a rocprofv3 counter-collection CSV (any counters).

    python -m paper_1606_08061_amd.pmc_table COUNTERS.csv [--kernels PREFIX ...]

Prints one markdown row per kernel: the number of dispatches and, per counter, the
average value per dispatch.
"""
from __future__ import annotations

import argparse
import collections
import csv


def _short(name: str) -> str:
    return name.replace("lst::(anonymous namespace)::", "").replace("void ", "").split("(")[0]


def table(path: str, prefixes=None):
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(path)):
        k = _short(r["Kernel_Name"])
        if prefixes and not any(k.startswith(p) for p in prefixes):
            continue
        vals[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return vals


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("csv")
    ap.add_argument("--kernels", nargs="*")
    a = ap.parse_args()
    vals = table(a.csv, a.kernels)
    names = sorted({c for v in vals.values() for c in v})
    print("| kernel | dispatches | " + " | ".join(names) + " |")
    print("|---|---|" + "---|" * len(names))
    for k in sorted(vals):
        n = max(len(x) for x in vals[k].values())
        cells = []
        for c in names:
            x = vals[k].get(c)
            cells.append(f"{sum(x) / len(x):.4g}" if x else "-")
        print(f"| `{k}` | {n} | " + " | ".join(cells) + " |")


if __name__ == "__main__":
    main()
