"""HBM traffic record of the decode step from rocprofv3 counter runs.

Usage (after the counter runs listed in the summary it writes):

    python -m paper_2604_09752_amd.profile_record --config 7b \\
        --fetch OUT/prof_7b_FETCH_SIZE --write OUT/prof_7b_WRITE_SIZE \\
        --cfetch OUT/prof_copy_FETCH_SIZE --cwrite OUT/prof_copy_WRITE_SIZE \\
        [--reqs OUT/prof_7b_REQ --creqs OUT/prof_copy_REQ]

Each directory holds one rocprofv3 ``--pmc`` run (``*_counter_collection.csv``).
FETCH_SIZE and WRITE_SIZE are per-dispatch KiB; each is scaled by what the
same counter reads for a plain device-to-device copy of a known size (the
copy reads and writes the same number of bytes), and the per-launch traffic
of the step kernel is the median over its dispatches (the few launches that
also write timing records do not move the median).  The optional request
runs count the memory read requests by size (TCC_EA0_RDREQ_32B, _64B,
_128B and all of them), which gives the read bytes without a calibration
factor.

The record names the SHA-256 of the step kernel's device sources; bench.py
reports ``traffic`` only while they are unchanged.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DEVICE_SOURCES = ["paper_2604_09752_amd/csrc/step_kernel.hip",
                  "paper_2604_09752_amd/csrc/step_kernel.h",
                  "paper_2604_09752_amd/csrc/common.h"]
# workload names of the records (bench --config -> profile name)
WORKLOADS = {"1b": "1b_2k", "7b": "7b_2k", "7b_32k": "7b_32k", "7b_int8": "7b_int8_2k"}


def record_path(config: str) -> str:
    return os.path.join(ROOT, "profiles", "k_step_%s_traffic.json" % WORKLOADS[config])


def sources_sha256() -> str:
    h = hashlib.sha256()
    for f in DEVICE_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def per_dispatch(run_dir: str, kernel: str) -> dict:
    """{counter: [value per dispatch of kernels whose name contains `kernel`]}
    (the counter's rows of one dispatch summed)."""
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError("no counter_collection.csv under " + run_dir)
    sums: dict = {}
    names: dict = {}
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if kernel not in r["Kernel_Name"]:
                    continue
                key = (r["Counter_Name"], r["Dispatch_Id"])
                sums[key] = sums.get(key, 0.0) + float(r["Counter_Value"])
                names[r["Dispatch_Id"]] = r["Kernel_Name"]
    out: dict = {}
    for (c, d), v in sorted(sums.items(), key=lambda kv: int(kv[0][1])):
        out.setdefault(c, []).append(v)
    out["_kernel"] = sorted(set(names.values()))
    return out


def stats(v) -> dict:
    a = np.asarray(v, dtype=np.float64)
    return {"n": int(a.size), "median": float(np.median(a)), "min": float(a.min()),
            "max": float(a.max())}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--config", required=True, choices=sorted(WORKLOADS))
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--cfetch", required=True)
    ap.add_argument("--cwrite", required=True)
    ap.add_argument("--reqs")
    ap.add_argument("--creqs")
    ap.add_argument("--copy-bytes", type=int, default=1 << 30)
    args = ap.parse_args()

    import synth
    from paper_2604_09752_amd import traffic
    cfg = synth.CONFIGS[args.config]
    P = cfg.prompt_len

    f = per_dispatch(args.fetch, "k_step")
    w = per_dispatch(args.write, "k_step")
    cf = per_dispatch(args.cfetch, "copyBuffer")
    cw = per_dispatch(args.cwrite, "copyBuffer")
    fs, ws = stats(f["FETCH_SIZE"]), stats(w["WRITE_SIZE"])
    cfs, cws = stats(cf["FETCH_SIZE"]), stats(cw["WRITE_SIZE"])
    copy_kib = args.copy_bytes / 1024.0
    ff, wf = copy_kib / cfs["median"], copy_kib / cws["median"]
    read_b = fs["median"] * 1024.0 * ff
    write_b = ws["median"] * 1024.0 * wf
    algo = traffic.step_bytes(cfg, P)
    rec = {
        "kernel": f["_kernel"],
        "workload": "%s @ %d positions, %s weights" % (args.config, P, cfg.wfmt),
        "device_sources": DEVICE_SOURCES,
        "sources_sha256": sources_sha256(),
        "dispatches": fs["n"],
        "fetch_size_kib": fs,
        "write_size_kib": ws,
        "copy_fetch_size_kib": cfs,
        "copy_write_size_kib": cws,
        "fetch_factor": round(ff, 5),
        "write_factor": round(wf, 5),
        "read_bytes_per_launch": int(read_b),
        "write_bytes_per_launch": int(write_b),
        "traffic_bytes_per_launch": int(read_b + write_b),
        "algorithmic_bytes_per_launch": int(algo),
        "traffic_over_algorithmic": round((read_b + write_b) / algo, 4),
    }
    if args.reqs:
        rq = per_dispatch(args.reqs, "k_step")
        r = {c: stats(rq[c])["median"] for c in rq if c.startswith("TCC_EA0_RDREQ")}
        b = 32 * r.get("TCC_EA0_RDREQ_32B", 0) + 64 * r.get("TCC_EA0_RDREQ_64B", 0) + \
            128 * r.get("TCC_EA0_RDREQ_128B", 0)
        rec["read_requests"] = r
        rec["read_bytes_from_request_sizes"] = int(b)
        if args.creqs:
            cq = per_dispatch(args.creqs, "copyBuffer")
            c = {k: stats(cq[k])["median"] for k in cq if k.startswith("TCC_EA0_RDREQ")}
            cb = 32 * c.get("TCC_EA0_RDREQ_32B", 0) + 64 * c.get("TCC_EA0_RDREQ_64B", 0) + \
                128 * c.get("TCC_EA0_RDREQ_128B", 0)
            rec["copy_read_requests"] = c
            rec["copy_read_bytes_from_request_sizes"] = int(cb)
    os.makedirs(os.path.dirname(record_path(args.config)), exist_ok=True)
    with open(record_path(args.config), "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
