"""HBM traffic per kernel launch from two rocprofv3 counter runs.

    python -m paper_2607_02501_amd.traffic <FETCH_SIZE csv> <WRITE_SIZE csv> \
        <workload> <kernel label> <kernel symbol substring> <calibration bytes> [out.json] [a:b]

Both runs execute `bench.py --calibrate-copy <bytes>`, which starts with one
plain device-to-device copy of known size.  Each counter is scaled by
(bytes copied) / (counter value of that copy dispatch), so the reported
traffic is in true bytes whatever unit the counter reports in.  The record
is stamped with a hash of the kernel sources; bench.py ignores it once the
sources change.  The optional a:b keeps only the a-th to (b-1)-th dispatches of
the symbol, in launch order (when one kernel symbol serves launches of
different sizes, e.g. a fused launch of a whole pass and of one kernel group).
"""
import csv
import json
import sys

from paper_2607_02501_amd.srchash import family, kernel_sources_sha


def per_dispatch(path, symbol, pick=None):
    vals, copy = [], []
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
    for r in rows:
        v = float(r["Counter_Value"]) * 1024.0  # counters are reported in KiB
        if "copyBuffer" in r["Kernel_Name"]:
            copy.append(v)
        elif symbol in r["Kernel_Name"]:
            vals.append(v)
    if pick:
        a, b = (int(t) for t in pick.split(":"))
        vals = vals[a:b]
    return vals, max(copy) if copy else None


def main():
    fcsv, wcsv, workload, label, symbol, calib = sys.argv[1:7]
    out = sys.argv[7] if len(sys.argv) > 7 else "profiles/traffic.json"
    pick = sys.argv[8] if len(sys.argv) > 8 else None
    calib = float(calib)
    fv, fc = per_dispatch(fcsv, symbol, pick)
    wv, wc = per_dispatch(wcsv, symbol, pick)
    fscale, wscale = calib / fc, calib / wc
    fetch = sum(fv) / len(fv) * fscale
    write = sum(wv) / len(wv) * wscale
    try:
        db = json.load(open(out))
    except (OSError, ValueError):
        db = {}
    db.setdefault(workload, {})[label] = {
        "kernel_symbol": symbol, "dispatches": len(fv), "dispatch_range": pick,
        "fetch_bytes_per_launch": round(fetch), "write_bytes_per_launch": round(write),
        "hbm_bytes_per_launch": round(fetch + write),
        "fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4),
        "calibration_copy_bytes": int(calib),
        "kernel_sources_sha": kernel_sources_sha(family(symbol)),
    }
    json.dump(db, open(out, "w"), indent=1, sort_keys=True)
    print(json.dumps(db[workload][label]))


if __name__ == "__main__":
    main()
