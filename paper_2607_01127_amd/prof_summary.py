"""Summaries of rocprofv3 output for the profiles/ folder.

kernel-stats: python -m paper_2607_01127_amd.prof_summary stats STATS_CSV CMD > profiles/X.md
trace:        python -m paper_2607_01127_amd.prof_summary trace TRACE_CSV CMD > profiles/X.md
counters:     python -m paper_2607_01127_amd.prof_summary counters PMC_CSV KERNEL_SUBSTR CMD > X.md
mfma:         python -m paper_2607_01127_amd.prof_summary mfma PMC_CSV CUS XCDS CMD KERNEL... > X.md
pass-traffic: python -m paper_2607_01127_amd.prof_summary pass_traffic FETCH_CSV COPY_FETCH_CSV \
                  COPY_BYTES LAUNCHES_PER_PASS ALGO_BYTES CMD > profiles/X.md
traffic:      python -m paper_2607_01127_amd.prof_summary traffic KERNEL_SUBSTR FETCH_CSV WRITE_CSV \
                  COPY_FETCH_CSV COPY_WRITE_CSV COPY_BYTES CMD > profiles/X.md

The traffic summary scales the per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of the kernel by
copy_bytes / (what the same counter reads for a plain device copy of copy_bytes bytes), and
records the sha256 of the GEMV's device source so that bench.py reports the figure only while
that source is unchanged (and only for the kernel instance the profile names).
"""
import csv
import hashlib
import os
import statistics
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCE = os.path.join(HERE, "csrc", "logbq_kernels.hip")


GEMV_BEGIN = "// ------------------------------------------------------------------ shared device helpers"
GEMV_END = "// ------------------------------------------------------------------ GPTQ calibration"


def source_hash() -> str:
    """sha256 (16 hex digits) of the GEMV's device source: the shared device helpers and the
    GEMV kernel, the part of the kernel file that decides the traffic of a GEMV launch."""
    text = open(KERNEL_SOURCE, encoding="utf-8").read()
    i, j = text.index(GEMV_BEGIN), text.index(GEMV_END)
    return hashlib.sha256(text[i:j].encode("utf-8")).hexdigest()[:16]


def _short(name: str) -> str:
    name = name.replace("void ", "").replace("(anonymous namespace)::", "")
    return name.split("(")[0][:60]


def stats(path, cmd):
    rows = list(csv.DictReader(open(path)))
    print("# rocprofv3 kernel statistics\n")
    print(f"Command: `{cmd}`\n")
    print("| kernel | calls | average (us) | min (us) | max (us) | total % |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        name = _short(r["Name"])
        if "at::native" in r["Name"] or "rocclr" in r["Name"]:
            continue
        avg = float(r["AverageNs"]) / 1e3
        print(f"| `{name}` | {r['Calls']} | {avg:.2f} | {float(r['MinNs'])/1e3:.2f} | "
              f"{float(r['MaxNs'])/1e3:.2f} | {float(r['Percentage']):.1f} |")


def _pct(vals, q):
    v = sorted(vals)
    if not v:
        return float("nan")
    i = min(len(v) - 1, max(0, int(round(q * (len(v) - 1)))))
    return v[i]


def trace(path, cmd):
    """Per-kernel dispatch-duration distribution from a rocprofv3 kernel trace."""
    durs = {}
    for r in csv.DictReader(open(path)):
        name = r["Kernel_Name"]
        if "at::native" in name or "rocclr" in name:
            continue
        d = (float(r["End_Timestamp"]) - float(r["Start_Timestamp"])) / 1e3
        durs.setdefault(_short(name), []).append(d)
    print("# rocprofv3 kernel trace: dispatch durations\n")
    print(f"Command: `{cmd}`\n")
    print("| kernel | dispatches | mean (us) | p10 (us) | median (us) | p90 (us) | total (ms) |")
    print("|---|---|---|---|---|---|---|")
    for name, v in sorted(durs.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{name}` | {len(v)} | {statistics.fmean(v):.2f} | {_pct(v, 0.1):.2f} | "
              f"{_pct(v, 0.5):.2f} | {_pct(v, 0.9):.2f} | {sum(v) / 1e3:.2f} |")


def counters(path, substr, cmd):
    """Median per-dispatch value of every counter collected for kernels matching substr."""
    vals = {}
    for r in csv.DictReader(open(path)):
        if substr in r["Kernel_Name"]:
            vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    print("# rocprofv3 counters per dispatch\n")
    print(f"Command: `{cmd}`\n")
    print(f"kernel: `{substr}`\n")
    for name, v in sorted(vals.items()):
        print(f"- {name}: median {statistics.median(v):.6g} over {len(v)} dispatches")


def mfma(path, cus, xcds, cmd, kernels):
    """MFMA-pipe busy fraction per kernel from SQ_VALU_MFMA_BUSY_CYCLES (summed over every SIMD
    of the chip; a v_mfma_f32_16x16x32_f16 adds 16 cycles, its issue time at the dense peak
    rate), GRBM_GUI_ACTIVE (the GPU clock counter summed over the XCDs) and SQ_BUSY_CU_CYCLES.
    busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x CUs x GRBM_GUI_ACTIVE / XCDs)."""
    cus, xcds = int(cus), int(xcds)
    print("# MFMA utilisation per dispatch (rocprofv3 --pmc)\n")
    print(f"Command: `{cmd}`\n")
    print(f"Normalisation: busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x {cus} CUs x "
          f"GRBM_GUI_ACTIVE / {xcds} XCDs); SQ_VALU_MFMA_BUSY_CYCLES is summed over every SIMD "
          f"(16 cycles per v_mfma_f32_16x16x32_f16), GRBM_GUI_ACTIVE over the {xcds} XCDs. "
          f"Medians over the dispatches of each kernel.\n")
    print("| kernel | dispatches | GRBM_GUI_ACTIVE | SQ_BUSY_CU_CYCLES | SQ_VALU_MFMA_BUSY_CYCLES "
          "| cycles per XCD | MFMA busy |")
    print("|---|---|---|---|---|---|---|")
    for k in kernels:
        vals = {}
        for r in csv.DictReader(open(path)):
            if _short(r["Kernel_Name"]).startswith(k):
                vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
        g = statistics.median(vals.get("GRBM_GUI_ACTIVE", [float("nan")]))
        b = statistics.median(vals.get("SQ_BUSY_CU_CYCLES", [float("nan")]))
        mf = statistics.median(vals.get("SQ_VALU_MFMA_BUSY_CYCLES", [float("nan")]))
        n = len(vals.get("GRBM_GUI_ACTIVE", []))
        per_xcd = g / xcds
        busy = mf / (4 * cus * per_xcd)
        print(f"| `{k}` | {n} | {g:.6g} | {b:.6g} | {mf:.6g} | {per_xcd:.6g} | {busy:.3f} |")


def _counter(path, substr, counter):
    vals = []
    for r in csv.DictReader(open(path)):
        if substr in r["Kernel_Name"] and r["Counter_Name"] == counter:
            vals.append(float(r["Counter_Value"]))
    return vals


def pass_traffic(fetch, cfetch, copy_bytes, per_pass, algo, cmd):
    """HBM bytes fetched per decode pass: FETCH_SIZE of the library's GEMV and split-K launches
    in dispatch order, in consecutive groups of `per_pass` launches (one pass each), scaled by
    the copy calibration; reports the median pass."""
    rows = []
    for r in csv.DictReader(open(fetch)):
        name = r["Kernel_Name"]
        if r["Counter_Name"] == "FETCH_SIZE" and ("k_gemv" in name or "k_mfma" in name):
            rows.append((int(r.get("Dispatch_Id", 0) or 0), float(r["Counter_Value"])))
    rows.sort()
    cf = _counter(cfetch, "copy", "FETCH_SIZE") or _counter(cfetch, "Copy", "FETCH_SIZE")
    kf = float(copy_bytes) / (statistics.median(cf) * 1024.0)
    per_pass, algo = int(per_pass), float(algo)
    passes = [sum(v for _, v in rows[i:i + per_pass]) * 1024.0 * kf
              for i in range(0, len(rows) - per_pass + 1, per_pass)]
    print("# HBM bytes per decode pass (rocprofv3 --pmc FETCH_SIZE)\n")
    print(f"Command: `{cmd}`\n")
    print(f"- launches per pass: {per_pass}; passes counted: {len(passes)}")
    print(f"- copy calibration factor {kf:.4f}")
    print(f"- fetched bytes per pass (median): {statistics.median(passes):.0f}")
    print(f"- packed code bytes per pass (algorithmic): {algo:.0f}")
    print(f"- ratio fetched / algorithmic: {statistics.median(passes) / algo:.4f}")


def traffic(substr, fetch, write, cfetch, cwrite, copy_bytes, cmd):
    f = _counter(fetch, substr, "FETCH_SIZE")
    w = _counter(write, substr, "WRITE_SIZE")
    cf = _counter(cfetch, "copy", "FETCH_SIZE") or _counter(cfetch, "Copy", "FETCH_SIZE")
    cw = _counter(cwrite, "copy", "WRITE_SIZE") or _counter(cwrite, "Copy", "WRITE_SIZE")
    copy_bytes = float(copy_bytes)
    kf = copy_bytes / (statistics.median(cf) * 1024.0)
    kw = copy_bytes / (statistics.median(cw) * 1024.0)
    fb = statistics.median(f) * 1024.0 * kf
    wb = statistics.median(w) * 1024.0 * kw
    print("# HBM traffic per launch (rocprofv3 --pmc)\n")
    print(f"Command: `{cmd}`\n")
    print(f"kernel: `{substr}`, dispatches: {len(f)}\n")
    print(f"- FETCH_SIZE median {statistics.median(f):.1f} KiB, copy calibration factor {kf:.4f}")
    print(f"- WRITE_SIZE median {statistics.median(w):.1f} KiB, copy calibration factor {kw:.4f}")
    print(f"- fetch_bytes: {fb:.0f}")
    print(f"- write_bytes: {wb:.0f}")
    print(f"- traffic_bytes: {fb + wb:.0f}")
    print(f"- gemv_source_sha256_16: {source_hash()}")


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(sys.argv[2], sys.argv[3])
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:9])
    elif sys.argv[1] == "trace":
        trace(sys.argv[2], sys.argv[3])
    elif sys.argv[1] == "counters":
        counters(sys.argv[2], sys.argv[3], sys.argv[4])
    elif sys.argv[1] == "pass_traffic":
        pass_traffic(*sys.argv[2:8])
    elif sys.argv[1] == "mfma":
        mfma(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5], sys.argv[6:])
