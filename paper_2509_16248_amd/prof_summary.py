"""Turn two rocprofv3 counter runs of the benchmark (FETCH_SIZE, then
WRITE_SIZE) into the HBM traffic record of the GEMM kernels that bench.py
reports as ``roofline.traffic``.

    python -m paper_2509_16248_amd.prof_summary WORKLOAD FETCH_DIR WRITE_DIR OUT.json

WORKLOAD is decoder_4096 (the headline: every GEMM launch of its forward,
whose eager profiled forwards run the same launches as its graph) or
causal_lm_768 (the whole-batch launches of its eager profiled forwards).

Calibration: both runs contain the runtime's copy kernel moving a weight of
known size into library memory (the token embedding: vocab x d_model x 2
bytes); the largest such dispatch gives the bytes each counter unit stands
for (FETCH_SIZE of a copy counts half its bytes on this GPU, WRITE_SIZE all
of them).  The record carries the SHA-256 of gm_gemm.hip so that a stale
measurement is not reported after the kernel changes.  Prints a markdown
table as well.
"""
from __future__ import annotations

import collections
import csv
import glob
import hashlib
import json
import os
import sys

COPY = "__amd_rocclr_copyBuffer"
WORKLOADS = {
    "decoder_4096": {
        "kernels": ("void gm::k_gemm_big<", "void gm::k_gemm_x<"),
        # grid size (threads) -> the launch it is, at 1 x 2048 tokens
        "shapes": {262144: "QKV 2048x12288x4096 (128x384 tiles, BK 64 x 2)",
                   131072: "O 2048x4096x4096 / down 2048x4096x11008 (128x256 tiles)",
                   352256: "gate|up 2048x22016x4096 (256x256 tiles, BK 64 x 2)",
                   512000: "head 2048x32000x4096 (256x256 tiles, BK 64 x 2)"},
        "copy_bytes": 32000 * 4096 * 2,
        "algorithmic": {   # operands read once + output written once (+ residual read)
            262144: 2 * (2048 * 4096 + 12288 * 4096 + 2048 * 12288),
            131072: None,  # O and down differ; averaged from the two below
            352256: 2 * (2048 * 4096 + 22016 * 4096 + 2048 * 11008),
            512000: 2 * (2048 * 4096 + 32000 * 4096 + 2048 * 32000)},
        "o_down": (2 * (2048 * 4096 + 4096 * 4096 + 2 * 2048 * 4096),
                   2 * (2048 * 11008 + 4096 * 11008 + 2 * 2048 * 4096)),
    },
    "causal_lm_768": {
        "kernels": ("void gm::k_gemm_x<unsigned short, 128, 128, 2, 4, 2>",),
        "shapes": {294912: "QKV 4096x2304x768", 98304: "O/down 4096x768",
                   393216: "up 4096x3072x768", 6438912: "head 4096x50257x768"},
        "copy_bytes": 50257 * 768 * 2,
    },
}


def _rows(d, counter):
    path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not path:
        raise SystemExit(f"no counter_collection.csv under {d}")
    out = []
    for r in csv.DictReader(open(path[0])):
        if r["Counter_Name"] == counter:
            out.append((r["Kernel_Name"], int(r["Grid_Size"]), float(r["Counter_Value"])))
    return out


def summarize(workload, fetch_dir, write_dir, src):
    wl = WORKLOADS[workload]
    f, w = _rows(fetch_dir, "FETCH_SIZE"), _rows(write_dir, "WRITE_SIZE")
    copies_f = [v for k, _, v in f if k.startswith(COPY)]
    copies_w = [v for k, _, v in w if k.startswith(COPY)]
    fscale = wl["copy_bytes"] / (max(copies_f) * 1024)
    wscale = wl["copy_bytes"] / (max(copies_w) * 1024)
    per = collections.OrderedDict()
    for rows, key in ((f, "fetch"), (w, "write")):
        for k, g, v in rows:
            if not k.startswith(wl["kernels"]) or g not in wl["shapes"]:
                continue
            e = per.setdefault(wl["shapes"][g], {"grid": g, "fetch_kib": [], "write_kib": []})
            e[key + "_kib"].append(v)
    tot_f = tot_w = n = 0
    for name, e in per.items():
        e["dispatches"] = len(e["fetch_kib"])
        fk = sum(e["fetch_kib"]) / max(1, len(e["fetch_kib"]))
        wk = sum(e["write_kib"]) / max(1, len(e["write_kib"]))
        e["traffic_mb_scaled"] = round((fk * fscale + wk * wscale) * 1024 / 1e6, 1)
        alg = wl.get("algorithmic", {}).get(e["grid"])
        if e["grid"] == 131072 and "o_down" in wl:
            alg = sum(wl["o_down"]) / 2
        if alg:
            e["algorithmic_mb"] = round(alg / 1e6, 1)
        tot_f += sum(e["fetch_kib"]) * fscale * 1024
        tot_w += sum(e["write_kib"]) * wscale * 1024
        n += e["dispatches"]
        e["fetch_kib_raw"] = round(fk, 1)
        e["write_kib_raw"] = round(wk, 1)
        del e["fetch_kib"], e["write_kib"]
    return {"workload": workload, "kernels": list(wl["kernels"]),
            "gm_gemm_hip_sha256": hashlib.sha256(open(src, "rb").read()).hexdigest(),
            "fetch_scale": round(fscale, 3), "write_scale": round(wscale, 3),
            "traffic_bytes_per_launch": int((tot_f + tot_w) / n),
            "fetch_bytes_per_launch": int(tot_f / n), "write_bytes_per_launch": int(tot_w / n),
            "per_shape": per}


def main(argv):
    if len(argv) != 4 or argv[0] not in WORKLOADS:
        raise SystemExit(__doc__)
    src = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "gm_gemm.hip")
    rec = summarize(argv[0], argv[1], argv[2], src)
    with open(argv[3], "w") as fh:
        json.dump(rec, fh, indent=1)
    print(f"fetch scale {rec['fetch_scale']}, write scale {rec['write_scale']}")
    print("| launches | grid | dispatches | FETCH_SIZE KiB (raw, avg) | WRITE_SIZE KiB (raw, avg) "
          "| scaled MB per launch | algorithmic MB |")
    print("|---|---|---|---|---|---|---|")
    for name, e in rec["per_shape"].items():
        print(f"| {name} | {e['grid']} | {e['dispatches']} | {e['fetch_kib_raw']} | "
              f"{e['write_kib_raw']} | {e['traffic_mb_scaled']} | {e.get('algorithmic_mb', '')} |")
    print(f"average over all GEMM launches: {rec['traffic_bytes_per_launch'] / 1e6:.1f} MB")


if __name__ == "__main__":
    main(sys.argv[1:])
