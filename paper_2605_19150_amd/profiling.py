"""Summaries of rocprofv3 output for profiles/ (text files), and the reader
bench.py uses to attach counter-measured HBM traffic to its roofline object.

    # per-kernel durations (rocprofv3 --kernel-trace --stats ... -o run --output-format csv)
    python -m paper_2605_19150_amd.profiling stats DIR --title T --command "CMD" > profiles/X.md

    # HBM bytes per launch from two counter runs of a kernel and two of the
    # 1 GiB device copy of `bench.py --copy-calibration` (the scale factors)
    python -m paper_2605_19150_amd.profiling traffic --kernel k_fwd_fused --workload NAME \\
        --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR --command "..." > profiles/Y.md

A traffic summary records a hash of the kernel's sources (KERNEL_SOURCES);
read_traffic_summary returns None once they differ from the ones the counters
were taken on.
"""
import argparse
import collections
import csv
import glob
import hashlib
import os
import re
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
COPY_BYTES = 1 << 30  # bench.py --copy-calibration copies 1 GiB (reads 1 GiB, writes 1 GiB)


def _code_only(text):
    """Source text without comments and blank space, so that documentation
    edits do not count as kernel changes."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


# The device code of each measured kernel: its translation unit and the
# headers it includes.  A traffic summary stays valid while these are
# unchanged (comments aside).
KERNEL_SOURCES = {
    "k_fwd_fused": ["pdssm_fused.hip", "pdssm_fused.h", "pdssm_device.h", "pdssm_io.h"],
    "k_bwd_fused": ["pdssm_fused.hip", "pdssm_fused.h", "pdssm_device.h", "pdssm_io.h"],
    "k_bwd_fused_ste": ["pdssm_fused.hip", "pdssm_fused.h", "pdssm_device.h", "pdssm_io.h"],
    "k_fwd_fused_bf16": ["pdssm_fused.hip", "pdssm_fused.h", "pdssm_device.h", "pdssm_io.h"],
    "k_bwd_fused_bf16": ["pdssm_fused.hip", "pdssm_fused.h", "pdssm_device.h", "pdssm_io.h"],
    "k_fwd_fused_real": ["pdssm_fused.hip", "pdssm_fused.h", "pdssm_device.h", "pdssm_io.h"],
    "k_bwd_fused_real": ["pdssm_fused.hip", "pdssm_fused.h", "pdssm_device.h", "pdssm_io.h"],
    "k_ste_gemm": ["pdssm_ste.hip", "pdssm_internal.h", "pdssm_device.h", "pdssm_io.h"],
}


def source_hash(kernel=None):
    """Hash of the code (comments and layout ignored) of the source files the
    kernel is built from (every library source when the kernel is not
    listed in KERNEL_SOURCES)."""
    h = hashlib.sha256()
    if kernel in KERNEL_SOURCES:
        files = [os.path.join(PKG, "csrc", f) for f in KERNEL_SOURCES[kernel]]
    else:
        files = sorted(glob.glob(os.path.join(PKG, "csrc", "*"))) + [os.path.join(ROOT, "include", "pdssm.h")]
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def _rows(d, name):
    paths = glob.glob(os.path.join(d, "**", name), recursive=True)
    if not paths:
        raise FileNotFoundError("no %s under %s" % (name, d))
    with open(paths[0], newline="") as fh:
        return list(csv.DictReader(fh))


def stats_markdown(d, title, command):
    rows = _rows(d, "*kernel_stats.csv")
    out = ["# %s" % title, "", "Command (from the repository root, one MI355X):", "", "    " + command, "",
           "| kernel | calls | total (us) | average (us) | min (us) | max (us) | % |",
           "|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append("| %s | %s | %.1f | %.2f | %.2f | %.2f | %.1f |" % (
            r["Name"], r["Calls"], float(r["TotalDurationNs"]) / 1e3, float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    return "\n".join(out) + "\n"


def _counter_mean(d, counter, kernel_substr):
    """Mean per-dispatch value (KiB for FETCH_SIZE / WRITE_SIZE) of a counter
    over the dispatches whose kernel name contains kernel_substr."""
    vals = collections.defaultdict(float)
    for r in _rows(d, "*counter_collection.csv"):
        if r["Counter_Name"] == counter and kernel_substr in r["Kernel_Name"]:
            vals[r["Dispatch_Id"]] += float(r["Counter_Value"])
    if not vals:
        raise ValueError("no %s samples for %s in %s" % (counter, kernel_substr, d))
    return sum(vals.values()) / len(vals), len(vals)


def traffic_markdown(kernel, workload, fetch, write, copy_fetch, copy_write, command, match=None):
    """`kernel` names the summary (what read_traffic_summary looks up);
    `match` (default: kernel) selects the dispatches by a substring of their
    demangled name."""
    match = match or kernel
    # several dispatches per call (e.g. an aggregate pass and the scan):
    # substrings separated by ";;", their per-dispatch means add up
    f_kib = w_kib = 0.0
    nf = nw = 0
    for m in match.split(";;"):
        fk, n1 = _counter_mean(fetch, "FETCH_SIZE", m)
        wk, n2 = _counter_mean(write, "WRITE_SIZE", m)
        f_kib += fk
        w_kib += wk
        nf, nw = max(nf, n1), max(nw, n2)
    cf_kib, _ = _counter_mean(copy_fetch, "FETCH_SIZE", "copyBuffer")
    cw_kib, _ = _counter_mean(copy_write, "WRITE_SIZE", "copyBuffer")
    sf = COPY_BYTES / (cf_kib * 1024.0)
    sw = COPY_BYTES / (cw_kib * 1024.0)
    fetch_b = f_kib * 1024.0 * sf
    write_b = w_kib * 1024.0 * sw
    lines = [
        "# HBM traffic per launch: %s, workload %s" % (kernel, workload),
        "",
        "kernel: %s" % kernel,
        "dispatches: %s" % match,
        "workload: %s" % workload,
        "source-hash: %s" % source_hash(kernel),
        "fetch-bytes-per-launch: %.0f" % fetch_b,
        "write-bytes-per-launch: %.0f" % write_b,
        "traffic-bytes-per-launch: %.0f" % (fetch_b + write_b),
        "",
        "FETCH_SIZE %.1f KiB/dispatch (%d dispatches) x scale %.4f; WRITE_SIZE %.1f KiB/dispatch "
        "(%d dispatches) x scale %.4f." % (f_kib, nf, sf, w_kib, nw, sw),
        "Scales: a 1 GiB device copy (bench.py --copy-calibration) reads 1 GiB and writes 1 GiB; "
        "its counters read FETCH_SIZE %.1f KiB and WRITE_SIZE %.1f KiB per dispatch." % (cf_kib, cw_kib),
        "",
        "Commands (from the repository root, one MI355X, one counter per run):",
        "",
    ] + ["    " + c for c in command.split(" ;; ")]
    return "\n".join(lines) + "\n"


def _counter_means(d, kernel_substr):
    """Mean per-dispatch value of every counter of the dispatches whose
    kernel name contains kernel_substr: {counter: (mean, dispatches)}."""
    vals = collections.defaultdict(lambda: collections.defaultdict(float))
    for r in _rows(d, "*counter_collection.csv"):
        if kernel_substr in r["Kernel_Name"]:
            vals[r["Counter_Name"]][r["Dispatch_Id"]] += float(r["Counter_Value"])
    return {k: (sum(v.values()) / len(v), len(v)) for k, v in vals.items()}


# Counters the occupancy / LDS / VALU summaries explain.
COUNTER_NOTES = {
    "LDSBankConflict": "% of GPU time the LDS is stalled by bank conflicts (100 SQ_LDS_BANK_CONFLICT / GRBM_GUI_ACTIVE / CUs)",
    "VALUBusy": "% of GPU time the vector ALUs process instructions (100 SQ_ACTIVE_INST_VALU / CUs / GRBM_GUI_ACTIVE)",
    "OccupancyPercent": "waves resident as % of the maximum (400 SQ_WAVE_CYCLES / GRBM_GUI_ACTIVE / CUs / 32)",
    "SQ_INSTS_LDS": "LDS instructions issued",
    "SQ_INSTS_VALU": "VALU instructions issued",
    "SQ_LDS_IDX_ACTIVE": "cycles the LDS serves indexed accesses",
    "SQ_LDS_BANK_CONFLICT": "cycles the LDS is stalled by bank conflicts",
    "SQ_WAVES": "waves launched",
    "SQ_WAIT_INST_LDS": "wave-cycles (x4) waiting to issue an LDS instruction",
    "SQ_ACTIVE_INST_LDS": "wave-cycles (x4) spent on LDS instructions",
    "SQ_WAIT_ANY": "wave-cycles (x4) waiting for anything",
    "SQ_ACTIVE_INST_ANY": "wave-cycles (x4) spent on any instruction",
    "SQ_BUSY_CYCLES": "cycles with active waves in a shader engine",
    "GRBM_GUI_ACTIVE": "GPU busy cycles",
}


def counters_markdown(kernel, workload, dirs, command, match=None, state_updates=None):
    """Summary of counter runs (one directory per pass) of one kernel: mean
    per dispatch of every counter, per state update for the instruction
    counts when state_updates is given."""
    match = match or kernel
    rows = []
    for d in dirs:
        for name, (mean, n) in sorted(_counter_means(d, match).items()):
            rows.append((name, mean, n))
    out = ["# Occupancy, LDS and VALU counters: %s, workload %s" % (kernel, workload), "",
           "kernel: %s" % kernel, "dispatches: %s" % match, "workload: %s" % workload,
           "source-hash: %s" % source_hash(kernel), "",
           "Instruction counts are wave instructions (one per 64 lanes); the per-state-update column",
           "divides them by the launch's B*L*H*N state updates.", "",
           "| counter | mean per dispatch | per state update | dispatches | meaning |", "|---|---|---|---|---|"]
    for name, mean, n in rows:
        per = ("%.2f" % (mean / state_updates)) if state_updates and name.startswith("SQ_INSTS") else ""
        out.append("| %s | %.6g | %s | %d | %s |" % (name, mean, per, n, COUNTER_NOTES.get(name, "")))
    out += ["", "Commands (from the repository root, one MI355X, one pass per run):", ""]
    out += ["    " + c for c in command.split(" ;; ")]
    return "\n".join(out) + "\n"


def read_traffic_summary(profiles_dir, kernel, workload):
    """traffic-bytes-per-launch of the matching summary in profiles_dir, or
    None (no summary, or taken on other kernel sources)."""
    want = source_hash(kernel)
    for path in sorted(glob.glob(os.path.join(profiles_dir, "*.md"))):
        kv = {}
        with open(path) as fh:
            for line in fh:
                if ": " in line and not line.startswith(("#", " ", "|")):
                    k, v = line.rstrip("\n").split(": ", 1)
                    kv[k.strip()] = v.strip()
        # traffic summaries only (counter summaries name the same kernel)
        if "traffic-bytes-per-launch" not in kv:
            continue
        if kv.get("kernel") == kernel and kv.get("workload") == workload:
            if kv.get("source-hash") != want:
                return None
            return float(kv["traffic-bytes-per-launch"])
    return None


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    t = sub.add_parser("traffic")
    for k in ("kernel", "workload", "fetch", "write", "copy_fetch", "copy_write", "command"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    t.add_argument("--match", default=None, help="substring of the dispatches' kernel name (default: --kernel)")
    c = sub.add_parser("counters")
    for k in ("kernel", "workload", "command"):
        c.add_argument("--" + k, dest=k, required=True)
    c.add_argument("--dirs", nargs="+", required=True)
    c.add_argument("--match", default=None)
    c.add_argument("--state-updates", dest="state_updates", type=float, default=None)
    sub.add_parser("hash")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        sys.stdout.write(stats_markdown(a.dir, a.title, a.command))
    elif a.cmd == "counters":
        sys.stdout.write(counters_markdown(a.kernel, a.workload, a.dirs, a.command, a.match, a.state_updates))
    elif a.cmd == "traffic":
        sys.stdout.write(traffic_markdown(a.kernel, a.workload, a.fetch, a.write, a.copy_fetch,
                                          a.copy_write, a.command, a.match))
    else:
        for k in sorted(KERNEL_SOURCES):
            print(k, source_hash(k))


if __name__ == "__main__":
    main()
