"""Turn rocprofv3 FETCH_SIZE / WRITE_SIZE counter runs into HBM bytes per call.

Inputs are the ``*_counter_collection.csv`` files of four runs: the bench
command and the calibration copy (``hbm_copy``), each once with FETCH_SIZE
and once with WRITE_SIZE.  The copy moves a known number of bytes per
dispatch in each direction, which fixes the counter scale; the decode
kernels' per-dispatch counters are scaled by it and summed over the two
launches of one decode call (attend_kernel + merge_kernel of the IPPD path).

Usage: python -m paper_2609_05707_amd.traffic --fetch F.csv --write W.csv
           --copy-fetch CF.csv --copy-write CW.csv --copy-mib 256
           --workload 2 --command "..." --out profiles/traffic_decode_step_wl2.json
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


KERNEL_SOURCES = ("decode_step.hip", "tile_attend.h", "ippd_device.h", "ippd_internal.h", "ippd_api.hip")


def code_only(text: str) -> str:
    """Source text without comments, blank lines or layout: what a counter
    record's fingerprint covers (a comment or layout edit leaves the kernels,
    and so their counters, as they were).  String and character literals are
    kept whole, so a "//" or "/*" inside one is code."""
    out = []
    i, n = 0, len(text)
    while i < n:
        ch = text[i]
        if ch in "\"'":
            j = i + 1
            while j < n and text[j] != ch:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            while i < n and text[i] != "\n":
                i += 1
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(ch)
            i += 1
    lines = (" ".join(line.split()) for line in "".join(out).splitlines())
    return "\n".join(line for line in lines if line)


def kernel_source_hash(csrc: str = os.path.join(ROOT, "paper_2609_05707_amd", "csrc")) -> str:
    """Fingerprint of the decode kernels' code, stored with each counter
    record; bench.py uses a record only while the sources still match it."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def per_dispatch(path: str, counter: str):
    """Mean counter value per dispatch, by kernel name prefix."""
    vals = defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            fused = re.search(r"attend_kernel<[^>]*\btrue\b", name) is not None
            key = "attend" if fused else \
                  "merge" if "merge_kernel" in name else \
                  "copy" if "copyBuffer" in name else name
            vals[key].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in vals.items()}


def main() -> None:
    ap = argparse.ArgumentParser(description=__doc__)
    for a in ("--fetch", "--write", "--copy-fetch", "--copy-write", "--command", "--out"):
        ap.add_argument(a, required=True)
    ap.add_argument("--copy-mib", type=int, default=256)
    ap.add_argument("--workload", type=int, required=True)
    args = ap.parse_args()
    nbytes = args.copy_mib << 20
    cf = per_dispatch(args.copy_fetch, "FETCH_SIZE").get("copy")
    cw = per_dispatch(args.copy_write, "WRITE_SIZE").get("copy")
    f = per_dispatch(args.fetch, "FETCH_SIZE")
    w = per_dispatch(args.write, "WRITE_SIZE")
    fs, ws = nbytes / cf, nbytes / cw
    rec = {
        "workload": args.workload,
        "kernel_source_hash": kernel_source_hash(),
        "command": args.command,
        "copy_calibration": {"mib": args.copy_mib, "fetch_counter_per_dispatch": cf,
                             "write_counter_per_dispatch": cw,
                             "bytes_per_fetch_unit": fs, "bytes_per_write_unit": ws},
        "attend_fetch_bytes": f.get("attend", 0.0) * fs, "attend_write_bytes": w.get("attend", 0.0) * ws,
        "merge_fetch_bytes": f.get("merge", 0.0) * fs, "merge_write_bytes": w.get("merge", 0.0) * ws,
    }
    rec["hbm_bytes_per_launch"] = int(rec["attend_fetch_bytes"] + rec["attend_write_bytes"] +
                                      rec["merge_fetch_bytes"] + rec["merge_write_bytes"])
    with open(args.out, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


if __name__ == "__main__":
    main()
