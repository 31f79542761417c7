#!/usr/bin/env python3
"""Summaries of rocprofv3 output for the profiles/ folder.

    python profiles/summarize.py trace  <kernel_trace results.db> <title> <command>
    python profiles/summarize.py traffic <FETCH_SIZE results.db> <WRITE_SIZE results.db> <title> <command>

`trace` prints per-kernel dispatch counts and durations.  `traffic` prints,
per kernel, the FETCH_SIZE / WRITE_SIZE counters (KiB per dispatch) and the
same figures scaled by what the counters read for the run's plain device copy
(bench.py copies COPY_CAL_BYTES once before timing): bytes = counter *
(copy bytes / counter of the copy).
"""
import sqlite3
import statistics
import sys

COPY_BYTES = 256 << 20
COPY_KERNEL = "__amd_rocclr_copyBuffer"


def short(name, n=72):
    return name if len(name) <= n else name[:n - 3] + "..."


def trace(db, title, cmd):
    con = sqlite3.connect(db)
    rows = con.execute("select name, start, end from kernels").fetchall()
    agg = {}
    for name, s, e in rows:
        agg.setdefault(name, []).append((e - s) / 1000.0)
    tot = sum(sum(v) for v in agg.values())
    print("# %s\n\ncommand: `%s`\n" % (title, cmd))
    print("| kernel | calls | total us | avg us | min us | max us | % |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        print("| %s | %d | %.1f | %.2f | %.2f | %.2f | %.1f |" % (short(k), len(v), sum(v), statistics.mean(v),
                                                            min(v), max(v), 100 * sum(v) / tot))


def counters(db):
    con = sqlite3.connect(db)
    out = {}
    for name, val in con.execute("select name, counter_value from pmc_events"):
        out.setdefault(name, []).append(val)
    return out


def traffic(fdb, wdb, title, cmd):
    f, w = counters(fdb), counters(wdb)
    # the calibration copy is the largest copyBuffer dispatch
    fc, wc = max(f.get(COPY_KERNEL, [0])), max(w.get(COPY_KERNEL, [0]))
    ff = COPY_BYTES / 1024.0 / fc if fc else float("nan")
    wf = COPY_BYTES / 1024.0 / wc if wc else float("nan")
    print("# %s\n\ncommand (one run per counter): `%s`\n" % (title, cmd))
    print("calibration copy of %d MiB: FETCH_SIZE %.0f KiB (scale %.3f), WRITE_SIZE %.0f KiB (scale %.3f)\n"
          % (COPY_BYTES >> 20, fc, ff, wc, wf))
    print("| kernel | dispatches | FETCH KiB/dispatch | WRITE KiB/dispatch | scaled read MB | scaled write MB | scaled total MB |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for k in sorted(set(f) | set(w), key=lambda k: -statistics.mean(f.get(k, [0]))):
        if k == COPY_KERNEL:
            continue
        fv, wv = statistics.mean(f.get(k, [0])), statistics.mean(w.get(k, [0]))
        r, wr = fv * 1024 * ff / 1e6, wv * 1024 * wf / 1e6
        print("| %s | %d | %.0f | %.0f | %.1f | %.1f | %.1f |" % (short(k), len(f.get(k, [])), fv, wv, r, wr, r + wr))


if __name__ == "__main__":
    if sys.argv[1] == "trace":
        trace(sys.argv[2], sys.argv[3], sys.argv[4])
    else:
        traffic(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5])


def source_hash(root):
    """sha256 over the HIP sources of the library (the kernels a traffic
    figure was measured on)."""
    import glob
    import hashlib
    import os
    hs = hashlib.sha256()
    for fn in sorted(glob.glob(os.path.join(root, "paper_2402_09900_amd", "csrc", "*"))):
        hs.update(os.path.basename(fn).encode())
        hs.update(open(fn, "rb").read())
    return hs.hexdigest()


# kernels making up each library call, by name prefix
CALL_KERNELS = {
    "fwd": ("memoroid::ws_init_kernel", "void memoroid::diag_fwd_kernel"),
    "bwd": ("memoroid::ws_init_kernel", "void memoroid::diag_bwd_kernel", "memoroid::colsum_kernel"),
    "linattn": ("memoroid::ws_init_kernel", "void memoroid::diag_fwd_kernel", "memoroid::linattn_",
                "memoroid::fill_f32_kernel", "memoroid::ep_"),
}


def call_traffic(fdb, wdb, call, ndispatch_per_call):
    """Scaled bytes of one library call: the per-dispatch traffic of every
    kernel the call launches, times how often the call launches it."""
    f, w = counters(fdb), counters(wdb)
    ff = COPY_BYTES / 1024.0 / max(f[COPY_KERNEL])
    wf = COPY_BYTES / 1024.0 / max(w[COPY_KERNEL])
    total = 0.0
    for k in set(f) | set(w):
        if k.startswith(CALL_KERNELS[call]):
            n = ndispatch_per_call.get(k.split("(")[0].split("<")[0].replace("void ", ""), 1)
            total += n * (statistics.mean(f.get(k, [0])) * 1024 * ff + statistics.mean(w.get(k, [0])) * 1024 * wf)
    return total
