"""Summaries of rocprofv3 results for the repository's profiles folder.

  python -m paper_2609_05275_amd.profsum trace DB TITLE COMMAND > summary.md
      top kernels of a --kernel-trace --stats run (rocpd database)

  python -m paper_2609_05275_amd.profsum counters TRACE_DB MFMA_DB FETCH_DB WRITE_DB TITLE COMMAND > summary.md
      per-kernel counters of one command run four times: a --kernel-trace
      --stats pass (durations), an MFMA pass (SQ_VALU_MFMA_BUSY_CYCLES,
      GRBM_GUI_ACTIVE, SQ_INSTS_VALU_MFMA_MOPS_BF16) and the FETCH_SIZE and
      WRITE_SIZE passes; MFMA busy fraction, shader clock and executed bf16
      MFMA rate for the matrix kernels, counter-measured HBM bytes and GB/s
      (scaled by the calibration copy as below) for every kernel.  The
      command must include --copy-calib-mib.

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


COUNTERS_TAG = "counters-json:"
# rocprofv3 reports GRBM_GUI_ACTIVE summed over the chip's XCDs; the MFMA
# busy cycles are per SIMD (4 per CU)
N_XCD = 8
N_SIMD = 256 * 4
MFMA_FLOP_PER_MOP = 512          # SQ_INSTS_VALU_MFMA_MOPS_* count 512-FLOP units
KERNEL_FILES = {"ld_gemm": "k_gemm.hip", "ld_splitk": "k_gemm.hip", "ld_attn": "k_attn.hip",
                "ld_mask": "k_rows.hip", "ld_rmsnorm": "k_rows.hip", "ld_gather": "k_rows.hip",
                "ld_scatter": "k_rows.hip", "ld_swiglu": "k_rows.hip", "ld_relu2": "k_rows.hip",
                "ld_zero": "k_rows.hip"}


def kernel_source(kernel: str) -> str | None:
    """The sources a kernel is built from ('+'-separated, repository paths)."""
    for prefix, f in KERNEL_FILES.items():
        if kernel.startswith(prefix):
            return f"paper_2609_05275_amd/csrc/{f}+paper_2609_05275_amd/csrc/ld_internal.h"
    return None


def _durations(db: str) -> dict[str, tuple[int, float]]:
    """(calls, total microseconds) per kernel of a --kernel-trace --stats run."""
    con = sqlite3.connect(db)
    out: dict[str, tuple[int, float]] = {}
    for n, c, t in con.execute("select name, total_calls, total_duration from top_kernels"):
        k = short(n)
        c0, t0 = out.get(k, (0, 0.0))
        out[k] = (c0 + int(c), t0 + float(t))   # top_kernels durations are in microseconds
    return out


def _means(db: str, counter: str) -> dict[str, tuple[int, float]]:
    acc: dict[str, list[float]] = {}
    for _, n, v in _per_dispatch(db, counter):
        if n.startswith("ld_") or "ld_" in n:
            acc.setdefault(short(n), []).append(v)
    return {k: (len(v), sum(v) / len(v)) for k, v in acc.items()}


def counters(trace_db: str, mfma_db: str, fetch_db: str, write_db: str, title: str, cmd: str) -> str:
    dur = _durations(trace_db)
    busy = _means(mfma_db, "SQ_VALU_MFMA_BUSY_CYCLES")
    grbm = _means(mfma_db, "GRBM_GUI_ACTIVE")
    mops = _means(mfma_db, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
    fetch_rows = _per_dispatch(fetch_db, "FETCH_SIZE")
    write_rows = _per_dispatch(write_db, "WRITE_SIZE")
    cf, cw = _calibration(fetch_rows), _calibration(write_rows)
    if len(cf) < CALIB_DISPATCHES or len(cw) < CALIB_DISPATCHES:
        raise SystemExit("calibration dispatches missing")
    calib_kib = float(re.search(r"--copy-calib-mib (\d+)", cmd).group(1)) * 1024.0
    f_fac = (sum(cf) / len(cf)) / calib_kib
    w_fac = (sum(cw) / len(cw)) / calib_kib
    fetch = _means(fetch_db, "FETCH_SIZE")
    write = _means(write_db, "WRITE_SIZE")
    recs = {}
    for k in sorted(dur, key=lambda k: -dur[k][1]):
        calls, tot_us = dur[k]
        if not k.startswith("ld_") or calls == 0:
            continue
        avg_us = tot_us / calls
        r = {"calls": calls, "avg_us": round(avg_us, 2)}
        if k in grbm and grbm[k][1] > 0:
            cyc = grbm[k][1] / N_XCD
            r["clock_ghz"] = round(cyc / (avg_us * 1e3), 3)
            if k in busy:
                r["mfma_busy"] = round(busy[k][1] / (cyc * N_SIMD), 4)
            if k in mops and mops[k][1] > 0:
                r["mfma_tflops"] = round(mops[k][1] * MFMA_FLOP_PER_MOP / (avg_us * 1e-6) / 1e12, 1)
        if k in fetch and k in write:
            b = (fetch[k][1] / f_fac + write[k][1] / w_fac) * 1024.0
            r["hbm_bytes"] = round(b)
            r["hbm_gbs"] = round(b / (avg_us * 1e-6) / 1e9, 1)
        src = kernel_source(k)
        if src:
            r["source"] = src
            r["source_sha256"] = source_hash(src)
        recs[k] = r
    out = [f"# {title}", "", "Commands (the same command under each pass):", "", f"    {cmd}", "",
           "Passes: `--kernel-trace --stats` (durations); `--pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
           "SQ_INSTS_VALU_MFMA_MOPS_BF16`; `--pmc FETCH_SIZE`; `--pmc WRITE_SIZE`.", "",
           f"Calibration copy (elementwise y = 1 * x over float32, {calib_kib:.0f} KiB read and written): "
           f"FETCH_SIZE reads {f_fac:.4f} x and WRITE_SIZE {w_fac:.4f} x the known bytes; HBM bytes below "
           "are the counters divided by these factors.  MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / "
           f"(GRBM_GUI_ACTIVE / {N_XCD} XCDs x {N_SIMD} SIMDs); clock = GRBM_GUI_ACTIVE / {N_XCD} / duration; "
           f"MFMA TFLOP/s = SQ_INSTS_VALU_MFMA_MOPS_BF16 x {MFMA_FLOP_PER_MOP} / duration (executed, "
           "including padding).", "",
           "| kernel | calls | avg us | clock GHz | MFMA busy | MFMA TFLOP/s | HBM MiB/launch | HBM GB/s |",
           "|---|---|---|---|---|---|---|---|"]
    for k, r in recs.items():
        def g(key, fmt):
            return fmt.format(r[key]) if key in r else "-"
        mib = f"{r['hbm_bytes'] / 2**20:.1f}" if "hbm_bytes" in r else "-"
        out.append(f"| {k} | {r['calls']} | {r['avg_us']:.1f} | {g('clock_ghz', '{:.2f}')} | "
                   f"{g('mfma_busy', '{:.3f}')} | {g('mfma_tflops', '{:.0f}')} | {mib} | {g('hbm_gbs', '{:.0f}')} |")
    out += ["", f"{COUNTERS_TAG} {json.dumps(recs)}", ""]
    return "\n".join(out)


def read_counters(md_path: str) -> dict | None:
    """The per-kernel records a counters summary carries, or None."""
    try:
        with open(md_path) as f:
            for line in f:
                if line.startswith(COUNTERS_TAG):
                    return json.loads(line[len(COUNTERS_TAG):])
    except OSError:
        return None
    return None


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
    elif len(argv) >= 7 and argv[0] == "counters":
        sys.stdout.write(counters(argv[1], argv[2], argv[3], argv[4], argv[5], argv[6]))
    elif len(argv) >= 6 and argv[0] == "traffic":
        sys.stdout.write(traffic(argv[1], argv[2], argv[3], argv[4], argv[5]))
    else:
        raise SystemExit(__doc__)


if __name__ == "__main__":
    main(sys.argv[1:])
