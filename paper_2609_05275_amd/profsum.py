"""Summaries of rocprofv3 results for the repository's profiles folder.

  python -m paper_2609_05275_amd.profsum trace DB TITLE COMMAND > summary.md
      top kernels of a --kernel-trace --stats run (rocpd database)

  python -m paper_2609_05275_amd.profsum traffic FETCH_DB WRITE_DB KERNEL SOURCE COMMAND > summary.md
      HBM traffic per dispatch of KERNEL from two counter passes (FETCH_SIZE,
      then WRITE_SIZE, each in KiB per dispatch), each scaled by what the same
      counter reads for the calibration copy that bench.py --copy-calib-mib
      runs (an elementwise y = 1 * x over float32 tensors of known size).
      SOURCE lists the files the kernel is built from ('+'-separated); their
      SHA-256 goes into the summary so that a reader can tell when the kernel
      has changed since the counters were taken.

Reads only rocprofv3 output; runs nothing on a GPU.
"""
from __future__ import annotations

import hashlib
import json
import os
import re
import sqlite3
import sys

TRAFFIC_TAG = "traffic-json:"
CALIB_KERNEL = "mul"  # name fragment of the calibration kernel (torch elementwise multiply)
CALIB_DISPATCHES = 3  # bench.py runs it 3 times before any other GPU work


def short(name: str) -> str:
    n = re.sub(r"\(anonymous namespace\)::", "", name)
    m = re.search(r"(ld_[a-z0-9_]+(<[^>]*>)?)", n)
    if m:
        return m.group(1).replace(" ", "")
    return n[:70]


def source_hash(paths: str, root: str = "") -> str:
    """SHA-256 over the files of a '+'-separated list (relative to root)."""
    h = hashlib.sha256()
    for p in paths.split("+"):
        with open(os.path.join(root, p), "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    return h.hexdigest()


def trace(db: str, title: str, cmd: str) -> str:
    con = sqlite3.connect(db)
    rows = list(con.execute(
        "select name, total_calls, total_duration, average, percentage from top_kernels"))
    out = [f"# {title}", "", "Command:", "", f"    {cmd}", "",
           "rocprofv3 top_kernels (durations in microseconds):", "",
           "| kernel | calls | total us | avg us | % |", "|---|---|---|---|---|"]
    for n, c, t, a, p in rows:
        if p < 0.05:
            continue
        out.append(f"| {short(n)} | {c} | {t:.0f} | {a:.1f} | {p:.2f} |")
    return "\n".join(out) + "\n"


def _per_dispatch(db: str, counter: str) -> list[tuple[int, str, float]]:
    """(dispatch id, kernel name, value) of every dispatch, in dispatch order."""
    con = sqlite3.connect(db)
    rows = [(int(d), name, float(val)) for d, name, cn, val in con.execute(
        "select dispatch_id, kernel_name, counter_name, value from counters_collection")
        if cn == counter]
    return sorted(rows)


def _calibration(rows: list[tuple[int, str, float]]) -> list[float]:
    """The first CALIB_DISPATCHES multiply dispatches: the calibration copy."""
    vals = [v for _, n, v in rows if CALIB_KERNEL in n.lower() and "ld_" not in n]
    return vals[:CALIB_DISPATCHES]


def traffic(fetch_db: str, write_db: str, kernel: str, source: str, cmd: str) -> str:
    fetch = _per_dispatch(fetch_db, "FETCH_SIZE")
    write = _per_dispatch(write_db, "WRITE_SIZE")
    kf = [v for _, n, v in fetch if short(n) == kernel]
    kw = [v for _, n, v in write if short(n) == kernel]
    cf = _calibration(fetch)
    cw = _calibration(write)
    if not kf or not kw or len(cf) < CALIB_DISPATCHES or len(cw) < CALIB_DISPATCHES:
        raise SystemExit(f"missing dispatches: kernel fetch {len(kf)} write {len(kw)}, "
                         f"calibration fetch {len(cf)} write {len(cw)}")
    calib_kib = float(re.search(r"--copy-calib-mib (\d+)", cmd).group(1)) * 1024.0
    f_fac = (sum(cf) / len(cf)) / calib_kib
    w_fac = (sum(cw) / len(cw)) / calib_kib
    fk = sum(kf) / len(kf)
    wk = sum(kw) / len(kw)
    bytes_per_launch = (fk / f_fac + wk / w_fac) * 1024.0
    rec = {"kernel": kernel, "source": source, "source_sha256": source_hash(source),
           "dispatches": len(kf), "fetch_kib": round(fk, 1), "write_kib": round(wk, 1),
           "fetch_factor": round(f_fac, 4), "write_factor": round(w_fac, 4),
           "hbm_bytes_per_launch": round(bytes_per_launch)}
    wm = re.search(r"--workload (\S+)", cmd)
    workload = wm.group(1) if wm else "1b"
    rec["workload"] = workload
    out = [f"# HBM traffic per dispatch: {kernel}, stack step of workload {workload}", "",
           "Commands (one counter pass each):", "", f"    {cmd}", "",
           f"- {kernel}: {len(kf)} dispatches, FETCH_SIZE {fk:.1f} KiB and WRITE_SIZE "
           f"{wk:.1f} KiB per dispatch (mean)",
           f"- calibration (elementwise y = 1 * x, float32, {calib_kib:.0f} KiB read and "
           f"{calib_kib:.0f} KiB written): FETCH_SIZE reads {f_fac:.4f} x and WRITE_SIZE "
           f"{w_fac:.4f} x the known bytes",
           f"- scaled HBM traffic per {kernel} dispatch: {bytes_per_launch / 2**20:.1f} MiB", "",
           f"{TRAFFIC_TAG} {json.dumps(rec)}", ""]
    return "\n".join(out)


def read_traffic(md_path: str) -> dict | None:
    """The record a traffic summary carries, or None if there is none."""
    try:
        with open(md_path) as f:
            for line in f:
                if line.startswith(TRAFFIC_TAG):
                    return json.loads(line[len(TRAFFIC_TAG):])
    except OSError:
        return None
    return None


def main(argv: list[str]) -> None:
    if len(argv) >= 4 and argv[0] == "trace":
        sys.stdout.write(trace(argv[1], argv[2], argv[3]))
    elif len(argv) >= 6 and argv[0] == "traffic":
        sys.stdout.write(traffic(argv[1], argv[2], argv[3], argv[4], argv[5]))
    else:
        raise SystemExit(__doc__)


if __name__ == "__main__":
    main(sys.argv[1:])
