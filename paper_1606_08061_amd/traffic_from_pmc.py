"""Per-launch HBM traffic of the factored step's kernels from two rocprofv3 counter passes.

    python -m paper_1606_08061_amd.traffic_from_pmc FETCH.csv WRITE.csv --calib-mib 256

FETCH.csv and WRITE.csv are the counter_collection files of
`rocprofv3 --pmc FETCH_SIZE` and `rocprofv3 --pmc WRITE_SIZE` over
`bench.py --no-cpu --no-naive --copy-calib 256` (the step's kernels and, from the
bench's stabilisation leg, the pristine restore and the fix-singular-value pass
over V).  Both counters read KiB per
dispatch; the bench's plain device copy of a known size (the largest
__amd_rocclr_copyBuffer dispatch) gives the factor that turns each counter into
bytes.  Writes traffic.json next to this file: per phase, the kernel, the source
file and its SHA-256 (bench.py reports the traffic only while the source is
unchanged), and the average fetched and written bytes per launch.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")

# kernel name prefix -> (phase, source files that define the kernel's code)
KERNELS = [
    ("gemm16_plan_kernel<0>", "gram", "gemm.hip"),
    ("gemm16_plan_kernel<1>", "contract", "gemm.hip"),
    ("gemm16_plan_kernel<2>", "zgrad", "gemm.hip"),
    ("gemm_plan_kernel<0,", "gram", "gemm.hip"),
    ("gemm_plan_kernel<1,", "contract", "gemm.hip"),
    ("gemm_plan_kernel<2,", "zgrad", "gemm.hip"),
    ("gemm_plan_kernel<3,", "mid", "gemm.hip"),
    ("gemm_plan_kernel<4,", "update", "gemm.hip"),
    ("gather_reg_kernel", "gather", "step_kernels.hip"),
    ("gather_kernel", "gather", "step_kernels.hip"),
    ("mblock_kernel", "mblock", "step_kernels.hip"),
    ("woodbury_blocked_kernel", "woodbury", "step_kernels.hip+woodbury_gj.h"),
    ("scatter_kernel", "scatter", "step_kernels.hip+scatter.h"),
    ("update_scatter_kernel", "update", "gemm.hip+scatter.h"),
    ("restore_kernel", "restore", "stabilize.hip"),
    ("fix_v_kernel", "fix_v", "stabilize.hip"),
]


def source_sha(names: str) -> str:
    """SHA-256 of the named sources ("a+b": their bytes in that order)."""
    h = hashlib.sha256()
    for n in names.split("+"):
        h.update(open(os.path.join(CSRC, n), "rb").read())
    return h.hexdigest()


def _short(name: str) -> str:
    return name.replace("lst::(anonymous namespace)::", "").replace("void ", "").split("(")[0]


def load(path: str):
    rows = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        rows[_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("fetch_csv")
    ap.add_argument("write_csv")
    ap.add_argument("--calib-mib", type=int, required=True)
    ap.add_argument("--out", default=os.path.join(PKG, "traffic.json"))
    a = ap.parse_args()
    fetch, write = load(a.fetch_csv), load(a.write_csv)
    calib = a.calib_mib << 20
    f_cal = max(fetch["__amd_rocclr_copyBuffer"])
    w_cal = max(write["__amd_rocclr_copyBuffer"])
    f_scale, w_scale = calib / (f_cal * 1024.0), calib / (w_cal * 1024.0)
    out = {"calibration": {"copy_bytes": calib, "fetch_KiB": f_cal, "write_KiB": w_cal,
                           "fetch_factor": round(f_scale, 4), "write_factor": round(w_scale, 4)},
           "phases": {}}
    for prefix, phase, src in KERNELS:
        names = [n for n in fetch if n.replace(" ", "").startswith(prefix.replace(" ", ""))]
        if not names or phase in out["phases"]:
            continue
        fv = [v for n in names for v in fetch[n]]
        wv = [v for n in names for v in write.get(n, [])]
        out["phases"][phase] = {
            "kernel": names[0], "source": src, "source_sha256": source_sha(src),
            "launches": len(fv),
            "fetch_bytes": round(sum(fv) / len(fv) * 1024.0 * f_scale),
            "write_bytes": round(sum(wv) / max(len(wv), 1) * 1024.0 * w_scale),
        }
    json.dump(out, open(a.out, "w"), indent=1)
    print(json.dumps(out, indent=1))


if __name__ == "__main__":
    main()
