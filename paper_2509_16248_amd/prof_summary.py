"""Turn two rocprofv3 counter runs (FETCH_SIZE, then WRITE_SIZE) of the
benchmark into the HBM traffic record of the GEMM kernel that bench.py
reports as ``roofline.traffic``.

    python -m paper_2509_16248_amd.prof_summary FETCH_DIR WRITE_DIR OUT.json

Only the launches of the whole-batch shapes are counted: bench.py's
roofline is measured on its eager per-kernel profile, which runs the whole
batch per launch (the graph splits the batch into concurrent parts).

Calibration: both runs contain the runtime's copy kernel moving the token
embedding (vocab x d_model x 2 bytes) into library memory; the largest such
dispatch gives the bytes each counter unit stands for (FETCH_SIZE of a copy
reads counts half its bytes on this GPU, WRITE_SIZE all of them).  The
record carries the SHA-256 of gm_gemm.hip so that a stale measurement is
not reported after the kernel changes.  Prints a markdown table as well.
"""
from __future__ import annotations

import collections
import csv
import glob
import hashlib
import json
import os
import sys

KERNEL = "void gm::k_gemm_x<unsigned short, 128, 128, 2, 4, 2>"
COPY = "__amd_rocclr_copyBuffer"
SHAPES = {  # grid size (threads) of each GEMM of the 12-layer d 768 model at 8 x 512 tokens
    294912: "QKV 4096x2304x768",
    98304: "O/down 4096x768",
    393216: "up 4096x3072x768",
    6438912: "head 4096x50257x768",
}
EMB_BYTES = 50257 * 768 * 2


def _rows(d, counter):
    path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not path:
        raise SystemExit(f"no counter_collection.csv under {d}")
    out = []
    for r in csv.DictReader(open(path[0])):
        if r["Counter_Name"] == counter:
            out.append((r["Kernel_Name"], int(r["Grid_Size"]), float(r["Counter_Value"])))
    return out


def summarize(fetch_dir, write_dir, src):
    f, w = _rows(fetch_dir, "FETCH_SIZE"), _rows(write_dir, "WRITE_SIZE")
    fscale = EMB_BYTES / (max(v for k, _, v in f if k.startswith(COPY)) * 1024)
    wscale = EMB_BYTES / (max(v for k, _, v in w if k.startswith(COPY)) * 1024)
    per = collections.OrderedDict()
    tot_f = tot_w = n = 0
    for rows, key in ((f, "fetch"), (w, "write")):
        for k, g, v in rows:
            # the whole-batch launches (the eager per-kernel profile that
            # bench.py's roofline is measured on); the graph's batch-part
            # launches have other grids
            if not k.startswith(KERNEL) or g not in SHAPES:
                continue
            name = SHAPES[g]
            e = per.setdefault(name, {"dispatches": 0, "fetch_kib": [], "write_kib": []})
            e[key + "_kib"].append(v)
    for name, e in per.items():
        e["dispatches"] = len(e["fetch_kib"])
        fk = sum(e["fetch_kib"]) / max(1, len(e["fetch_kib"]))
        wk = sum(e["write_kib"]) / max(1, len(e["write_kib"]))
        e["traffic_mb_scaled"] = round((fk * fscale + wk * wscale) * 1024 / 1e6, 1)
        tot_f += sum(e["fetch_kib"]) * fscale * 1024
        tot_w += sum(e["write_kib"]) * wscale * 1024
        n += e["dispatches"]
        e["fetch_kib_raw"] = round(fk, 1)
        e["write_kib_raw"] = round(wk, 1)
        del e["fetch_kib"], e["write_kib"]
    return {"kernel": "k_gemm_x<bf16,128,128,2,4,2>",
            "gm_gemm_hip_sha256": hashlib.sha256(open(src, "rb").read()).hexdigest(),
            "fetch_scale": round(fscale, 3), "write_scale": round(wscale, 3),
            "traffic_bytes_per_launch": int((tot_f + tot_w) / n),
            "fetch_bytes_per_launch": int(tot_f / n), "write_bytes_per_launch": int(tot_w / n),
            "per_shape": per}


def main(argv):
    if len(argv) != 3:
        raise SystemExit(__doc__)
    src = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "gm_gemm.hip")
    rec = summarize(argv[0], argv[1], src)
    with open(argv[2], "w") as fh:
        json.dump(rec, fh, indent=1)
    print(f"fetch scale {rec['fetch_scale']}, write scale {rec['write_scale']}")
    print("| launches | dispatches | FETCH_SIZE KiB (raw, avg) | WRITE_SIZE KiB (raw, avg) | scaled MB per launch |")
    print("|---|---|---|---|---|")
    for name, e in rec["per_shape"].items():
        print(f"| {name} | {e['dispatches']} | {e['fetch_kib_raw']} | {e['write_kib_raw']} | "
              f"{e['traffic_mb_scaled']} |")
    print(f"average over all GEMM launches: {rec['traffic_bytes_per_launch'] / 1e6:.1f} MB")


if __name__ == "__main__":
    main(sys.argv[1:])
