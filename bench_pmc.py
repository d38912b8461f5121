"""Hardware-counter summaries of the step's kernels from rocprofv3 counter-collection CSVs.

    python bench_pmc.py table COUNTERS.csv [--kernels PREFIX ...]
        one markdown row per kernel: dispatches and, per counter, the average per dispatch
    python bench_pmc.py traffic FETCH.csv WRITE.csv --calib-mib 256 --out SUMMARY.md
        per-launch HBM bytes of each phase from a FETCH_SIZE pass and a WRITE_SIZE pass
        over `bench.py --no-cpu --no-naive --no-secondary --copy-calib 256`
    python bench_pmc.py stats KERNEL_STATS.csv [--kernels PREFIX ...]
        one markdown row per kernel of a `rocprofv3 --kernel-trace --stats` summary

Both counters read KiB per dispatch; the bench's plain device copy of a known size (the
largest __amd_rocclr_copyBuffer dispatch) gives the factor that turns each into bytes.
The traffic summary ends with a JSON block (per phase: kernel, source files and their
SHA-256, average fetched and written bytes per launch) that bench.py reads, reporting
the traffic only while the kernel's sources are unchanged.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re

ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_1606_08061_amd", "csrc")

# kernel name prefix -> (phase, source files that define the kernel's code)
KERNELS = [
    ("step_contract_kernel", "contract", "fused.hip+gemm_tiles.h"),
    ("step_gather_kernel", "gather", "fused.hip+gemm_tiles.h"),
    ("step_zgrad_kernel", "zgrad", "fused.hip+gemm_tiles.h"),
    ("step_mid_kernel", "mid", "fused.hip+gemm_tiles.h"),
    ("step_update_kernel", "update", "fused.hip+gemm_tiles.h+scatter.h"),
    ("online_step_kernel", "online", "online.hip"),
    ("restore_kernel", "restore", "stabilize.hip"),
    ("fix_v_kernel", "fix_v", "stabilize.hip"),
]


def source_sha(names: str) -> str:
    """SHA-256 of the named sources ("a+b": their bytes in that order)."""
    h = hashlib.sha256()
    for n in names.split("+"):
        with open(os.path.join(CSRC, n), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _short(name: str) -> str:
    return name.replace("lst::(anonymous namespace)::", "").replace("void ", "").split("(")[0]


def _rows(path):
    with open(path) as fh:
        return list(csv.DictReader(fh))


def table(path: str, prefixes=None) -> str:
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in _rows(path):
        k = _short(r["Kernel_Name"])
        if prefixes and not any(k.startswith(p) for p in prefixes):
            continue
        vals[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    counters = sorted({c for v in vals.values() for c in v})
    out = ["| kernel | dispatches | " + " | ".join(counters) + " |",
           "|---|---|" + "---|" * len(counters)]
    for k, v in vals.items():
        n = max(len(x) for x in v.values())
        out.append(f"| `{k}` | {n} | " +
                   " | ".join(f"{sum(v[c]) / len(v[c]):.4g}" if c in v else "-" for c in counters) +
                   " |")
    return "\n".join(out)


def stats(path: str, prefixes=None) -> str:
    out = ["| kernel | calls | average us | min us | max us | share of GPU time |",
           "|---|---|---|---|---|---|"]
    for r in _rows(path):
        k = _short(r["Name"])
        if prefixes and not any(k.startswith(p) for p in prefixes):
            continue
        out.append(f"| `{k}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.3f} | "
                   f"{float(r['MinNs']) / 1e3:.3f} | {float(r['MaxNs']) / 1e3:.3f} | "
                   f"{float(r['Percentage']):.2f} % |")
    return "\n".join(out)


def _per_kernel(path, counter):
    acc = collections.defaultdict(list)
    for r in _rows(path):
        if r["Counter_Name"] == counter:
            acc[_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return acc


def traffic(fetch_csv, write_csv, calib_mib):
    """{phase: {kernel, launches, fetch_bytes, write_bytes, source, source_sha256}} and the
    two scale factors (bytes per KiB of FETCH_SIZE and of WRITE_SIZE)."""
    fetch, write = _per_kernel(fetch_csv, "FETCH_SIZE"), _per_kernel(write_csv, "WRITE_SIZE")
    copy_bytes = calib_mib * 1 << 20
    cf = copy_bytes / (max(fetch["__amd_rocclr_copyBuffer"]) * 1024.0)
    cw = copy_bytes / (max(write["__amd_rocclr_copyBuffer"]) * 1024.0)
    out = {}
    for prefix, phase, src in KERNELS:
        ks = [k for k in fetch if k.startswith(prefix)]
        if not ks:
            continue
        k = max(ks, key=lambda x: len(fetch[x]))
        f, w = fetch[k], write.get(k, [0.0])
        out[phase] = {"kernel": k, "launches": len(f),
                      "fetch_bytes": int(sum(f) / len(f) * 1024 * cf),
                      "write_bytes": int(sum(w) / len(w) * 1024 * cw),
                      "source": src, "source_sha256": source_sha(src)}
    return out, cf, cw


def read_traffic_block(md_path: str) -> dict:
    """The per-phase JSON block of a traffic summary written by `traffic`."""
    with open(md_path) as fh:
        text = fh.read()
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    return json.loads(m.group(1))["phases"] if m else {}


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("table")
    t.add_argument("csv")
    t.add_argument("--kernels", nargs="*")
    st = sub.add_parser("stats")
    st.add_argument("csv")
    st.add_argument("--kernels", nargs="*")
    tr = sub.add_parser("traffic")
    tr.add_argument("fetch_csv")
    tr.add_argument("write_csv")
    tr.add_argument("--calib-mib", type=int, required=True)
    tr.add_argument("--out", required=True)
    tr.add_argument("--header", default="", help="markdown placed before the table")
    a = ap.parse_args()
    if a.cmd == "table":
        print(table(a.csv, a.kernels))
        return
    if a.cmd == "stats":
        print(stats(a.csv, a.kernels))
        return
    ph, cf, cw = traffic(a.fetch_csv, a.write_csv, a.calib_mib)
    lines = [a.header.rstrip(), "",
             f"Calibration: a plain device copy of {a.calib_mib} MiB; fetched bytes = FETCH_SIZE x "
             f"1024 x {cf:.4f}, written bytes = WRITE_SIZE x 1024 x {cw:.4f}.", "",
             "| phase | kernel | launches | fetched MB | written MB | total MB |",
             "|---|---|---|---|---|---|"]
    for p, r in ph.items():
        lines.append(f"| {p} | `{r['kernel']}` | {r['launches']} | {r['fetch_bytes'] / 1e6:.3f} | "
                     f"{r['write_bytes'] / 1e6:.3f} | {(r['fetch_bytes'] + r['write_bytes']) / 1e6:.3f} |")
    lines += ["", "```json", json.dumps({"phases": ph}, indent=1), "```", ""]
    with open(a.out, "w") as fh:
        fh.write("\n".join(lines))
    print(a.out)


if __name__ == "__main__":
    main()
