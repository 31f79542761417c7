#!/usr/bin/env python3
"""Summaries of rocprofv3 output for the profiles/ folder.

    python profsum.py trace  <kernel_trace results.db> <title> <command>
    python profsum.py traffic <FETCH_SIZE results.db> <WRITE_SIZE results.db> <title> <command>
    python profsum.py json <out.json> <command> <workload>=<FETCH db>,<WRITE db> ...
    python profsum.py mfma <SQ counter db> <kernel trace db> <title> <command> <kernel>=<wavefronts> ...

`trace` prints per-kernel dispatch counts and durations.  `traffic` prints,
per kernel, the FETCH_SIZE / WRITE_SIZE counters (KiB per dispatch) and the
same figures scaled by what the counters read for the run's plain device copy
(bench.py copies COPY_CAL_BYTES once before timing): bytes = counter *
(copy bytes / counter of the copy).  `json` writes the scaled bytes of every
library call bench.py times (the sum over the kernels the call launches,
CALLS below), with the hash of the HIP sources they were measured on.
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
    notes = []
    if any(k.startswith("memoroid::ws_init_kernel") for k in agg):
        notes.append("`ws_init_kernel`: the preparation of the prepared workspaces "
                     "(memoroid_workspace_prepare) before the timed steps, and the workspace fills of the "
                     "self-initialising steps bench.py times after them.")
    if COPY_KERNEL in agg:
        notes.append("`%s`: input uploads and the byte-counter calibration copy, before the timed steps."
                     % COPY_KERNEL)
    torch_kernels = [k for k in agg if not k.startswith(("memoroid::", "void memoroid::")) and k != COPY_KERNEL]
    if torch_kernels:
        notes.append("other kernels (%s): bench.py's own buffer fills and its copy-bandwidth probe (a 1 GiB "
                     "elementwise negation), outside the timed steps." % ", ".join("`%s`" % short(k, 40)
                                                                                   for k in torch_kernels))
    if notes:
        print()
        for n in notes:
            print("- " + n)


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




# kernels each timed library call launches (name after "memoroid::"), per
# workload, once per call
_DIAG = {"fwd": ["diag_fwd_kernel"], "bwd": ["diag_bwd_kernel"]}
_LIN_FWD = ["linattn_summary_kernel", "diag_fwd_kernel", "linattn_output_kernel"]
CALLS = {
    2: _DIAG,
    4: {"fwd": ["diag_fwd_kernel"]},
    5: _DIAG,
    6: {"return": ["disc_kernel<4, false>"], "gae": ["disc_kernel<4, true>"]},
    7: {"fwd": ["diag_fwd_kernel"], "bwd": ["diag_bwd_kernel", "ffm_bwd_finish_kernel"]},
    8: {"insert": ["tbb_begins_kernel"],
        "sample": ["tbb_rows_kernel", "tbb_gather_kernel"]},
    3: {"linattn_fwd": _LIN_FWD},
    9: {"linattn_fwd": _LIN_FWD,
        "linattn_bwd": ["linattn_summary_kernel", "diag_fwd_kernel", "linattn_bwd_summary_kernel", "diag_bwd_kernel",
                        "linattn_bwd_grad_kernel"]},
}


MFMA_FLOPS = 2 * 16 * 16 * 4      # one v_mfma_f32_16x16x4_f32
FP32_MFMA_PEAK = 157.3e12


def mfma(pmc_db, trace_db, waves_per_kernel, title, cmd):
    """MFMA use of the linear-attention kernels from SQ counters.  The SQ
    block samples one shader engine, so the counters give MFMA instructions
    per wavefront (SQ_INSTS_VALU_MFMA_F32 / SQ_WAVES); flops issued = that x
    the launch's wavefronts x 2048, over the kernel's mean traced duration
    and the fp32 MFMA peak."""
    c = {}
    con = sqlite3.connect(pmc_db)
    for k, name, v in con.execute("select name, counter_name, counter_value from pmc_events"):
        c.setdefault(k, {}).setdefault(name, []).append(v)
    con = sqlite3.connect(trace_db)
    dur = {}
    for k, s0, e0 in con.execute("select name, start, end from kernels"):
        dur.setdefault(k, []).append((e0 - s0) * 1e-9)
    print("# %s\n\ncommand: `%s`\n" % (title, cmd))
    print("| kernel | wavefronts / launch | MFMA instr / wavefront | flops issued / launch | mean duration us "
          "| issued TFLOP/s | % of fp32 MFMA peak |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for k, nw in waves_per_kernel:
        full = [kk for kk in c if kk.startswith(k) or kk.startswith("void " + k)]
        if not full:
            continue
        d = c[full[0]]
        per_wave = sum(d["SQ_INSTS_VALU_MFMA_F32"]) / max(sum(d["SQ_WAVES"]), 1)
        flops = per_wave * nw * MFMA_FLOPS
        t = statistics.mean(next(v for kk, v in dur.items() if kk.startswith(k) or kk.startswith("void " + k)))
        print("| %s | %d | %.1f | %.3g | %.1f | %.1f | %.1f |" % (short(full[0]), nw, per_wave, flops, t * 1e6,
                                                                 flops / t / 1e12, 100 * flops / t / FP32_MFMA_PEAK))


def per_dispatch_bytes(fdb, wdb):
    """Scaled bytes per dispatch of every kernel in a pair of counter runs."""
    f, w = counters(fdb), counters(wdb)
    ff = COPY_BYTES / 1024.0 / max(f[COPY_KERNEL])
    wf = COPY_BYTES / 1024.0 / max(w[COPY_KERNEL])
    out = {}
    for k in set(f) | set(w):
        if k == COPY_KERNEL:
            continue
        out[k] = statistics.mean(f.get(k, [0])) * 1024 * ff + statistics.mean(w.get(k, [0])) * 1024 * wf
    return out


def call_bytes(key, fdb, wdb):
    per = per_dispatch_bytes(fdb, wdb)
    res = {}
    for call, kernels in CALLS[key].items():
        total = 0.0
        for kname in kernels:
            hits = [v for k, v in per.items() if ("memoroid::" + kname) in k]
            if len(hits) != 1:
                raise SystemExit("workload %d call %s: kernel %s matched %d entries" % (key, call, kname, len(hits)))
            total += hits[0]
        res[call] = int(round(total))
    return res


def write_json(out, cmd, specs):
    import json
    import os
    root = os.path.dirname(os.path.abspath(__file__))
    rec = {"source_sha256": source_hash(root),
           "note": "bytes per library call: FETCH_SIZE + WRITE_SIZE of every kernel the call launches, "
                   "scaled by what the counters read for a 256 MiB device copy",
           "command": cmd, "workloads": {}}
    for spec in specs:
        key, dbs = spec.split("=")
        fdb, wdb = dbs.split(",")
        rec["workloads"][key] = call_bytes(int(key), fdb, wdb)
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")


if __name__ == "__main__":
    if sys.argv[1] == "trace":
        trace(sys.argv[2], sys.argv[3], sys.argv[4])
    elif sys.argv[1] == "mfma":
        # mfma <pmc db> <trace db> <title> <command> <kernel>=<wavefronts per launch> ...
        specs = [(a.split("=")[0], int(a.split("=")[1])) for a in sys.argv[6:]]
        mfma(sys.argv[2], sys.argv[3], specs, sys.argv[4], sys.argv[5])
    elif sys.argv[1] == "traffic":
        traffic(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5])
    else:
        write_json(sys.argv[2], sys.argv[3], sys.argv[4:])
