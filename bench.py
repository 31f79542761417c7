#!/usr/bin/env python3
"""Throughput of the resettable memoroid scan on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload N]

A step is one pass of the whole hot path over one synthetic tape already
resident in HBM: for the diagonal workloads the forward scan (with episode
indices) and, where the workload has one, the reverse (gradient) scan; for the
linear-attention workload the chunked forward readout; for the RL-target
workload the discounted return and the advantage estimate.  Prints ONE JSON line.

Workloads (seeded, synthetic; laws in paper_2402_09900_amd.tapes):
  1  diag real f32, T=1024, d=32, 8 episodes, forward
  2  diag complex64 (LRU-style, time-invariant a), T=65536, d=256, Geometric(200)
     episodes, forward + reverse
  3  linear-transformer memoroid, T=32768, 4 heads x 64, Geometric(500), chunk 64
  4  diag real, 64 tapes x T=16384, d=512, bf16 in / fp32 state / bf16 out
  5  diag real f32, T=1048576, d=256, lognormal(5, 1.5) episodes, forward + reverse
     (the largest single-GPU configuration)                        [default]
  6  discounted return + generalized advantage estimate, one tape of 2^24 steps,
     U{1..1000} episodes, gamma 0.99, lambda 0.95
  7  FFM aggregator, T=262144, m=32 x c=8 complex state, Geometric(200) episodes,
     forward + gradient (x, alpha, omega)
  8  tape-based batching: begin indices of a 2^24-transition buffer (64-byte
     rows, U{1..1000} episodes) and a sampled batch of 2^20 rows
  9  workload 3 with the gradient of the readout (dq, dk, dv)

Every buffer exists in several copies (at least 1 GiB cycled, at least 3) and
step i uses copy i mod n, so inputs are read from HBM rather than from the
256 MB last-level cache left warm by the previous step.

value = tape timesteps x features per second of the whole step (B*T*d, or
T*H*dv for linear attention), from the wall time of the K timed steps.  The
timed calls are the *_prepared entry points on workspaces prepared once
before timing (one kernel per call); config.self_init_ms_per_step is the
same step through the self-initialising entry points (which add a fill of
each call's workspace header, counters and first descriptor bank).
roofline: the dominant call's algorithmic bytes (or flops) per launch over
its average launch time, measured in the timed steps with HIP events on the
launch stream.  The dominant call is the slowest one in the warmup steps,
which carry events on every call; in the timed steps only it does (an event
pair costs the GPU a few microseconds of idle time between calls), and the
other calls' times in config.ms_per_call come from as many steps again after
the timed ones.  roofline.step_frac puts the whole step's algorithmic bytes
(or flops) over the step time.

cpu_baseline: the fp64 oracle, unchanged, timed on this host on the very
input arrays the GPU steps read (the whole workload; the flags' SHA-256 is in
config), median of 3 runs, on one thread and on N threads.  The N-thread
figure runs the same oracle functions on N independent slices of the
problem at once (feature blocks or tapes of a diagonal scan, heads of linear
attention, trace rows of FFM), through ctypes, which releases the GIL for
each call; N is this process's CPU share, at most 16.  Input decoding to
fp64 and slicing happen before timing.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tape timesteps×features/sec for resettable scan; % of HBM peak (diag)"
UNIT = "timestep-features/s"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix
COPY_CAL_BYTES = 256 << 20     # size of the counter-calibration copy


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", type=int, default=5, choices=[1, 2, 3, 4, 5, 6, 7, 8, 9])
    p.add_argument("--no-cpu-baseline", action="store_true")
    return p.parse_args()


HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


class TimingEvent:
    """A timing-only HIP event, created with hipEventDisableSystemFence.  A
    default event (torch.cuda.Event) performs a system-scope release when it
    is recorded, writing back and invalidating the caches: on this GPU that
    left about 6 us of idle time around each record and started the next
    kernel cold, inflating both the per-call and the per-step times.  The
    HIP runtime is the one torch has loaded (same soname)."""
    _hip = None

    @classmethod
    def hip(cls):
        if cls._hip is None:
            L = ctypes.CDLL("libamdhip64.so.7")
            L.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            L.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            L.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            L.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = L
        return cls._hip

    def __init__(self):
        self.h = ctypes.c_void_p()
        st = self.hip().hipEventCreateWithFlags(ctypes.byref(self.h), HIP_EVENT_DISABLE_SYSTEM_FENCE)
        if st != 0:
            raise RuntimeError("hipEventCreateWithFlags failed: %d" % st)

    def record(self, stream):
        st = self.hip().hipEventRecord(self.h, ctypes.c_void_p(stream))
        if st != 0:
            raise RuntimeError("hipEventRecord failed: %d" % st)

    def elapsed_time(self, other):
        ms = ctypes.c_float()
        st = self.hip().hipEventElapsedTime(ctypes.byref(ms), self.h, other.h)
        if st != 0:
            raise RuntimeError("hipEventElapsedTime failed: %d" % st)
        return float(ms.value)

    def __del__(self):
        if self._hip is not None and self.h:
            self._hip.hipEventDestroy(self.h)


class Timer:
    """Timing-only HIP events on the launch stream around one library call."""

    def __init__(self, torch):
        self.torch = torch
        self.pairs = []

    def __call__(self, fn):
        stream = self.torch.cuda.current_stream().cuda_stream
        e0, e1 = TimingEvent(), TimingEvent()
        e0.record(stream)
        fn()
        e1.record(stream)
        self.pairs.append((e0, e1))

    def times_ms(self):
        return [a.elapsed_time(b) for a, b in self.pairs]

    def mean_ms(self):
        return float(np.mean(self.times_ms())) if self.pairs else 0.0

    def median_ms(self):
        return float(np.median(self.times_ms())) if self.pairs else 0.0

    def percentiles_ms(self, qs=(10, 50, 90)):
        v = self.times_ms()
        return [round(float(np.percentile(v, q)), 4) for q in qs] if v else None


COPY_PROBE_BYTES = 1 << 30     # plain read + write kernel, larger than the 256 MB last-level cache


def copy_probe_gbps(torch, reps=5):
    """Bandwidth of a plain device copy kernel (a torch elementwise negation
    of a 1 GiB float32 buffer: read 1 GiB, write 1 GiB), median of `reps`
    event-timed runs; the attainable ceiling the scans are compared with."""
    src = torch.empty(COPY_PROBE_BYTES // 4, dtype=torch.float32, device="cuda")
    src.fill_(1.0)
    dst = torch.empty_like(src)
    tm = Timer(torch)
    torch.neg(src, out=dst)
    for _ in range(reps):
        tm(lambda: torch.neg(src, out=dst))
    torch.cuda.synchronize()
    ms = tm.median_ms()
    del src, dst
    return 2 * COPY_PROBE_BYTES / (ms * 1e-3) / 1e9


def dev_tensor(torch, arr, kind):
    arr = np.ascontiguousarray(arr)
    if kind == "bf16":
        return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(arr).cuda()


def n_sets(set_bytes):
    """Copies of every buffer to rotate through, so that a step does not find
    its inputs in the 256 MB last-level cache (MALL) from an earlier step:
    enough copies to cycle over at least 1 GiB, at least 3, at most 16."""
    need = -(-(1 << 30) // max(int(set_bytes), 1))
    return int(min(16, max(3, need)))


PREPARED = []
SUFFIX = ["_prepared"]      # "" switches every call to the self-initialising entry points


def entry(mb, name):
    """The entry point `name` of the current mode (prepared or self-initialising)."""
    return getattr(mb, name + SUFFIX[0])


def prepared_ws(torch, mb, nbytes):
    """Workspace of a prepared entry point: allocated and prepared once;
    every timed call then finds it ready (one kernel per call).  Its status
    is checked after the timed region."""
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")
    st = mb.memoroid_workspace_prepare(ws.data_ptr(), ws.numel(), torch.cuda.current_stream().cuda_stream)
    assert st == 0, mb.status_string(st)
    PREPARED.append(ws)
    return ws


def setup_diag(torch, mb, tapes, key):
    w = tapes.make_diag(key)
    kind = w.dtype
    code = {"f32": mb.F32, "bf16": mb.BF16, "c64": mb.C64}
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "c64": torch.complex64}
    ebytes = {"f32": 4, "bf16": 2, "c64": 8}
    B, T, d = w.B, w.T, w.d
    n = B * T * d
    stride = 0 if w.a_invariant else d
    a_bytes = (d if w.a_invariant else n) * ebytes[kind]
    nb = mb.memoroid_scan_diag_workspace_bytes(B, T, d, code[kind], code[w.out_dtype])
    nbb = mb.memoroid_scan_diag_bwd_workspace_bytes(B, T, d, code[kind], stride) if w.g is not None else 0
    da_bytes = (d if w.a_invariant else n) * ebytes[kind]
    set_bytes = a_bytes + n * ebytes[kind] + n * ebytes[w.out_dtype] + B * T * 5 + nb
    if w.g is not None:
        set_bytes += 2 * n * ebytes[kind] + da_bytes + nbb
    stream = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731
    sets = []
    for _ in range(n_sets(set_bytes)):
        a, x, s = dev_tensor(torch, w.a, kind), dev_tensor(torch, w.x, kind), dev_tensor(torch, w.start, "u8")
        h = torch.empty((B, T, d), dtype=tdt[w.out_dtype], device="cuda")
        idx = torch.empty((B, T), dtype=torch.int32, device="cuda")
        ws = prepared_ws(torch, mb, nb)
        calls = {}

        def fwd(a=a, x=x, s=s, h=h, idx=idx, ws=ws):
            st = entry(mb, "memoroid_scan_diag")(a.data_ptr(), stride, x.data_ptr(), s.data_ptr(), h.data_ptr(),
                                       idx.data_ptr(), B, T, d, code[kind], code[w.out_dtype], ws.data_ptr(),
                                       ws.numel(), stream())
            assert st == 0, mb.status_string(st)
        calls["fwd"] = fwd
        if w.g is not None:
            g = dev_tensor(torch, w.g, kind)
            hb = h if w.out_dtype == kind else h.to(tdt[kind])
            gx = torch.empty_like(g)
            ga = torch.empty((d,) if w.a_invariant else (B, T, d), dtype=tdt[kind], device="cuda")
            wsb = prepared_ws(torch, mb, nbb)

            def bwd(a=a, s=s, hb=hb, g=g, gx=gx, ga=ga, wsb=wsb):
                st = entry(mb, "memoroid_scan_diag_bwd")(a.data_ptr(), stride, s.data_ptr(), hb.data_ptr(), g.data_ptr(),
                                               gx.data_ptr(), ga.data_ptr(), B, T, d, code[kind], wsb.data_ptr(),
                                               wsb.numel(), stream())
                assert st == 0, mb.status_string(st)
            calls["bwd"] = bwd
        sets.append(calls)
    bytes_per = {"fwd": a_bytes + n * ebytes[kind] + n * ebytes[w.out_dtype] + B * T * (1 + 4)}
    if w.g is not None:
        # read a_{t+1}, g, h_{t-1}; write dx, da (da per step, or [d])
        bytes_per["bwd"] = a_bytes + 3 * n * ebytes[kind] + da_bytes + B * T
    return w, sets, bytes_per, n


def setup_linattn(torch, mb, tapes, key=3):
    wl = tapes.WORKLOADS[key]
    la = tapes.make_linattn(key)
    n = la.T * la.H * la.dv
    nb = mb.memoroid_scan_linattn_workspace_bytes(la.T, la.H, 64, 64, 64)
    nbb = mb.memoroid_scan_linattn_bwd_workspace_bytes(la.T, la.H, 64, 64, 64) if wl.backward else 0
    g_host = np.random.Generator(np.random.PCG64(key + 100)).standard_normal(la.v.shape, dtype=np.float32)
    la.g_host = g_host
    stream = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731
    sets = []
    for _ in range(n_sets((4 + (5 if wl.backward else 0)) * n * 4 + la.T * 5 + nb + nbb)):
        q, k, v = (dev_tensor(torch, t, "f32") for t in (la.q, la.k, la.v))
        s = dev_tensor(torch, la.start, "u8")
        out = torch.empty_like(v)
        idx = torch.empty((la.T,), dtype=torch.int32, device="cuda")
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")

        def fwd(q=q, k=k, v=v, s=s, out=out, idx=idx, ws=ws):
            st = mb.memoroid_scan_linattn(q.data_ptr(), k.data_ptr(), v.data_ptr(), s.data_ptr(), out.data_ptr(),
                                          idx.data_ptr(), la.T, la.H, 64, 64, 64, ws.data_ptr(), ws.numel(),
                                          stream())
            assert st == 0, mb.status_string(st)
        calls = {"fwd": fwd}
        if wl.backward:
            g = dev_tensor(torch, g_host, "f32")
            gq, gk, gv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
            wsb = torch.empty(nbb, dtype=torch.uint8, device="cuda")

            def bwd(q=q, k=k, v=v, s=s, out=out, g=g, gq=gq, gk=gk, gv=gv, wsb=wsb):
                st = mb.memoroid_scan_linattn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), s.data_ptr(),
                                                  out.data_ptr(), g.data_ptr(), gq.data_ptr(), gk.data_ptr(),
                                                  gv.data_ptr(), la.T, la.H, 64, 64, 64, wsb.data_ptr(), wsb.numel(),
                                                  stream())
                assert st == 0, mb.status_string(st)
            calls["bwd"] = bwd
        sets.append(calls)
    # algorithmic: q, k, v read and out written once (4 B each), flags, idx;
    # backward: q, k, v, out, grad read and dq, dk, dv written once
    bytes_per = {"fwd": 4 * n * 4 + la.T * 5, "bwd": 8 * n * 4 + la.T}
    # chunked-dense flops per (chunk, head), 2*64^3 each: forward 4
    # contractions (QK^T, A V, Q S_in, the chunk summary); backward 10 (the
    # forward chunk summary, A, dP = dnum V^T, two for dq, two for dk, two
    # for dv, and the reverse chunk summary)
    unit = 2 * 64 ** 3 * (la.T // 64) * la.H
    flops = {"fwd": 4 * unit, "bwd": 10 * unit}
    return la, sets, bytes_per, n, flops


def setup_discount(torch, mb, tapes, key):
    tp = tapes.make_discount(key)
    B, T = tp.B, tp.T
    n = B * T
    nb = mb.memoroid_discount_workspace_bytes(B, T)
    stream = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731
    sets = []
    for _ in range(n_sets(n * (4 * 6 + 2) + 4 * nb)):
        r, v, vn = dev_tensor(torch, tp.r, "f32"), dev_tensor(torch, tp.v, "f32"), dev_tensor(torch, tp.vn, "f32")
        s, done = dev_tensor(torch, tp.start, "u8"), dev_tensor(torch, tp.done, "u8")
        G, adv, tg = (torch.empty((B, T), dtype=torch.float32, device="cuda") for _ in range(3))
        ws = prepared_ws(torch, mb, nb)       # the return and the advantage bind one workspace each
        wsg = prepared_ws(torch, mb, nb)

        def ret(r=r, s=s, G=G, ws=ws):
            st = entry(mb, "memoroid_discounted_return")(r.data_ptr(), s.data_ptr(), tp.gamma, G.data_ptr(), B, T,
                                               ws.data_ptr(), ws.numel(), stream())
            assert st == 0, mb.status_string(st)

        def gae(r=r, v=v, vn=vn, done=done, s=s, adv=adv, tg=tg, wsg=wsg):
            st = entry(mb, "memoroid_gae")(r.data_ptr(), v.data_ptr(), vn.data_ptr(), done.data_ptr(), s.data_ptr(),
                                 tp.gamma, tp.lam, adv.data_ptr(), tg.data_ptr(), B, T, wsg.data_ptr(), wsg.numel(),
                                 stream())
            assert st == 0, mb.status_string(st)
        sets.append({"return": ret, "gae": gae})
    # return: read r, flags; write G.  gae: read r, V, V', done, flags; write adv, target
    bytes_per = {"return": n * (4 + 1 + 4), "gae": n * (3 * 4 + 2 + 2 * 4)}
    return tp, sets, bytes_per, n


def setup_ffm(torch, mb, tapes, key):
    wl = tapes.WORKLOADS[key]
    f = tapes.make_ffm(key)
    B, T, m, c = f.B, f.T, f.m, f.c
    n = B * T * m * c
    nb = mb.memoroid_scan_ffm_workspace_bytes(B, T, m, c)
    nbb = mb.memoroid_scan_ffm_bwd_workspace_bytes(B, T, m, c) if wl.backward else 0
    g_host = None
    if wl.backward:
        rng = np.random.Generator(np.random.PCG64(key + 100))
        g_host = (rng.standard_normal((B, T, m, c), dtype=np.float32)
                  + 1j * rng.standard_normal((B, T, m, c), dtype=np.float32)).astype(np.complex64)
    f.g_host = g_host
    stream = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731
    sets = []
    for _ in range(n_sets(n * (16 if wl.backward else 8) + B * T * (m * 8 + 5) + nb + nbb)):
        al, om, x, s = (dev_tensor(torch, a, k) for a, k in ((f.alpha, "f32"), (f.omega, "f32"), (f.x, "f32"),
                                                              (f.start, "u8")))
        S = torch.empty((B, T, m, c), dtype=torch.complex64, device="cuda")
        idx = torch.empty((B, T), dtype=torch.int32, device="cuda")
        ws = prepared_ws(torch, mb, nb)

        def fwd(al=al, om=om, x=x, s=s, S=S, idx=idx, ws=ws):
            st = entry(mb, "memoroid_scan_ffm")(al.data_ptr(), om.data_ptr(), x.data_ptr(), s.data_ptr(), S.data_ptr(),
                                      idx.data_ptr(), B, T, m, c, ws.data_ptr(), ws.numel(), stream())
            assert st == 0, mb.status_string(st)
        calls = {"fwd": fwd}
        if wl.backward:
            G = dev_tensor(torch, g_host, "c64")
            gx = torch.empty((B, T, m), dtype=torch.float32, device="cuda")
            ga = torch.empty(m, dtype=torch.float32, device="cuda")
            gw = torch.empty(c, dtype=torch.float32, device="cuda")
            wsb = prepared_ws(torch, mb, nbb)

            def bwd(al=al, om=om, s=s, S=S, G=G, gx=gx, ga=ga, gw=gw, wsb=wsb):
                st = entry(mb, "memoroid_scan_ffm_bwd")(al.data_ptr(), om.data_ptr(), s.data_ptr(), S.data_ptr(), G.data_ptr(),
                                              gx.data_ptr(), ga.data_ptr(), gw.data_ptr(), B, T, m, c,
                                              wsb.data_ptr(), wsb.numel(), stream())
                assert st == 0, mb.status_string(st)
            calls["bwd"] = bwd
        sets.append(calls)
    # fwd: read x (real, m per step) and flags; write S (complex, m*c per
    # step) and idx.  bwd: read dL/dS and S_{t-1}, flags; write dx (real, m per
    # step); the parameter gradients are a reduction to m + c values
    bytes_per = {"fwd": B * T * (m * 4 + 1 + 4) + n * 8, "bwd": n * 16 + B * T * (1 + m * 4)}
    return f, sets, bytes_per, n


def setup_tbb(torch, mb, tapes, key):
    tb = tapes.make_tbb(key)
    n, row = tb.D.shape
    K = tb.draws.size
    nbi = mb.memoroid_tbb_begin_indices_workspace_bytes(n)
    nbs = mb.memoroid_tbb_sample_workspace_bytes(K, tb.batch)
    stream = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731
    row_bytes = row * 4
    sets = []
    set_bytes = n * (row_bytes + 1 + 8) + tb.batch * (row_bytes + 9) + K * 8 * 2 + nbi + nbs
    for _ in range(n_sets(set_bytes)):
        D, s, I, draws = dev_tensor(torch, tb.D, "f32"), dev_tensor(torch, tb.start, "u8"), \
            dev_tensor(torch, tb.begins, "i64"), dev_tensor(torch, tb.draws, "i64")
        idx = torch.empty(n, dtype=torch.int64, device="cuda")
        cnt = torch.empty(1, dtype=torch.int64, device="cuda")
        out = torch.empty((tb.batch, row), dtype=torch.float32, device="cuda")
        ost = torch.empty(tb.batch, dtype=torch.uint8, device="cuda")
        osrc = torch.empty(tb.batch, dtype=torch.int64, device="cuda")
        filled = torch.empty(1, dtype=torch.int64, device="cuda")
        wsi = prepared_ws(torch, mb, nbi)
        wss = prepared_ws(torch, mb, nbs)

        def insert(s=s, idx=idx, cnt=cnt, wsi=wsi):
            st = entry(mb, "memoroid_tbb_begin_indices")(s.data_ptr(), n, 0, idx.data_ptr(), cnt.data_ptr(), wsi.data_ptr(),
                                               wsi.numel(), stream())
            assert st == 0, mb.status_string(st)

        def sample(D=D, I=I, draws=draws, out=out, ost=ost, osrc=osrc, filled=filled, wss=wss):
            st = entry(mb, "memoroid_tbb_sample")(D.data_ptr(), n, row_bytes, I.data_ptr(), I.numel(), draws.data_ptr(), K,
                                        tb.batch, out.data_ptr(), ost.data_ptr(), osrc.data_ptr(), filled.data_ptr(),
                                        wss.data_ptr(), wss.numel(), stream())
            assert st == 0, mb.status_string(st)
        sets.append({"insert": insert, "sample": sample})
    n_I = tb.begins.size
    # insert: read the flags, write the begin indices.  sample: read the draws
    # and their I entries, read and write the batch rows, write flags and
    # source rows
    bytes_per = {"insert": n + 8 * n_I, "sample": K * (8 + 16) + tb.batch * (2 * row_bytes + 1 + 8)}
    return tb, sets, bytes_per, tb.batch


def kernel_source_hash():
    """sha256 over the library's HIP sources (same recipe as
    profsum.py), to tell whether recorded counters still apply."""
    import glob
    import hashlib
    hs = hashlib.sha256()
    for fn in sorted(glob.glob(os.path.join(ROOT, "paper_2402_09900_amd", "csrc", "*"))):
        hs.update(os.path.basename(fn).encode())
        hs.update(open(fn, "rb").read())
    return hs.hexdigest()


def recorded_traffic(key, call):
    """HBM bytes per call from the committed counter runs, or None when the
    kernels changed since they were taken."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != kernel_source_hash():
        return None
    return rec.get("workloads", {}).get(str(key), {}).get(call)


def _cpu_share():
    """CPU model of this host and the threads this process may use (at most
    16: the CPU share of one GPU on the boxes this runs on)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return model, max(1, min(avail, 16))


def _median_seconds(fn, reps=3):
    ts = []
    for _ in range(reps):
        t0 = time.perf_counter()
        fn()
        ts.append(time.perf_counter() - t0)
    return float(np.median(ts))


def _run_parallel(jobs, threads):
    """Run the oracle calls in `jobs` on `threads` threads (each a ctypes
    call into the oracle, which runs without the GIL)."""
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(lambda job: job(), jobs))


def _bounds(n, parts):
    parts = max(1, min(parts, n))
    edges = [n * i // parts for i in range(parts + 1)]
    return [(edges[i], edges[i + 1]) for i in range(parts) if edges[i + 1] > edges[i]]


def cpu_baseline(key, tapes, w):
    """The oracle as it stands, on the workload's own inputs (the arrays the
    GPU steps were built from), on 1 thread and on N threads over independent
    slices; the figure reported as value is the N-thread one."""
    import oracle
    wl = tapes.WORKLOADS[key]
    model, threads = _cpu_share()
    one, jobs, units, what, lanes = None, [], 0, "", ""
    if wl.kind == "tbb":
        units = w.batch
        one = lambda: oracle.tbb_sample(w.D, oracle.tbb_begin_indices(w.start), w.draws, w.batch)  # noqa: E731
        what = "begin indices of %d flags and a batch of %d rows" % (w.start.size, w.batch)
        lanes = None
    elif wl.kind == "ffm":
        al, om, x = w.alpha.astype(np.float64), w.omega.astype(np.float64), w.x.astype(np.float64)
        G = w.g_host.astype(np.complex128) if wl.backward else None
        units = w.B * w.T * w.m * w.c

        def one():
            S, _ = oracle.ffm(al, om, x, w.start)
            if G is not None:
                oracle.ffm_bwd(al, om, w.start, S, G)
        for j0, j1 in _bounds(w.m, threads):
            xs = np.ascontiguousarray(x[:, :, j0:j1])
            Gs = np.ascontiguousarray(G[:, :, j0:j1]) if G is not None else None

            def job(j0=j0, j1=j1, xs=xs, Gs=Gs):
                S, _ = oracle.ffm(al[j0:j1], om, xs, w.start)
                if Gs is not None:
                    oracle.ffm_bwd(al[j0:j1], om, w.start, S, Gs)
            jobs.append(job)
        what = ("forward + gradient" if wl.backward else "forward") + ", fp64"
        lanes = "trace rows j of the m x c state"
    elif wl.kind == "discount":
        r, v, vn = (a.astype(np.float64) for a in (w.r, w.v, w.vn))
        g32, l32 = float(np.float32(w.gamma)), float(np.float32(w.lam))
        units = w.B * w.T

        def one():
            oracle.discounted_return(r, w.start, g32)
            oracle.gae(r, v, w.start, g32, l32, vn=vn, done=w.done)
        for b0, b1 in _bounds(w.B, threads):
            def job(b0=b0, b1=b1):
                oracle.discounted_return(r[b0:b1], w.start[b0:b1], g32)
                oracle.gae(r[b0:b1], v[b0:b1], w.start[b0:b1], g32, l32, vn=vn[b0:b1], done=w.done[b0:b1])
            jobs.append(job)
        what = "return + advantage, fp64"
        lanes = "tapes"
    elif wl.kind == "linattn":
        q, k, v = w.q.astype(np.float64), w.k.astype(np.float64), w.v.astype(np.float64)
        g = w.g_host.astype(np.float64) if wl.backward else None
        units = w.T * w.H * w.dv

        def one():
            oracle.linattn(q, k, v, w.start)
            if g is not None:
                oracle.linattn_bwd(q, k, v, w.start, g)
        for h0, h1 in _bounds(w.H, threads):
            sl = [np.ascontiguousarray(t[:, h0:h1]) for t in (q, k, v)]
            gs = np.ascontiguousarray(g[:, h0:h1]) if g is not None else None

            def job(sl=sl, gs=gs):
                oracle.linattn(*sl, w.start)
                if gs is not None:
                    oracle.linattn_bwd(*sl, w.start, gs)
            jobs.append(job)
        what = ("forward readout and its gradient" if wl.backward else "forward readout") + ", fp64"
        lanes = "heads"
    else:
        a, x = w.decoded("a"), w.decoded("x")
        g = w.decoded("g") if wl.backward else None
        units = w.B * w.T * w.d

        def one():
            h, _ = oracle.diag_fwd(a, x, w.start)
            if g is not None:
                oracle.diag_bwd(a, w.start, h, g)
        if w.B >= threads:
            for b0, b1 in _bounds(w.B, threads):
                sl = (a if w.a_invariant else a[b0:b1], x[b0:b1], w.start[b0:b1], None if g is None else g[b0:b1])
                jobs.append(sl)
            lanes = "tapes"
        else:
            for j0, j1 in _bounds(w.d, threads):
                sl = (np.ascontiguousarray(a[j0:j1] if w.a_invariant else a[:, :, j0:j1]),
                      np.ascontiguousarray(x[:, :, j0:j1]), w.start,
                      None if g is None else np.ascontiguousarray(g[:, :, j0:j1]))
                jobs.append(sl)
            lanes = "feature blocks"

        def make(sl):
            def job():
                h, _ = oracle.diag_fwd(sl[0], sl[1], sl[2])
                if sl[3] is not None:
                    oracle.diag_bwd(sl[0], sl[2], h, sl[3])
            return job
        jobs = [make(sl) for sl in jobs]
        what = ("forward + reverse" if wl.backward else "forward") + ", fp64"
    t1 = _median_seconds(one)
    res = {"unit": UNIT, "kind": "oracle", "cpu_model": model, "cpu_share": threads,
           "one_thread": {"value": units / t1, "cores": 1, "seconds": round(t1, 4)}}
    split = "no independent slices to split over"
    if len(jobs) > 1:
        tn = _median_seconds(lambda: _run_parallel(jobs, threads))
        res["n_threads"] = {"value": units / tn, "cores": len(jobs), "seconds": round(tn, 4)}
        split = "the %d-thread run splits it over independent %s" % (len(jobs), lanes)
    best = max((res["one_thread"], res.get("n_threads")), key=lambda v: v["value"] if v else -1.0)
    res["value"], res["cores"] = best["value"], best["cores"]
    res["sample"] = ("the whole workload on the GPU steps' own input arrays (%s), median of 3 runs on 1 thread and "
                     "on up to %d; %s; value is the faster" % (what, threads, split))
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the scan is measured at one GPU's share of the tape; "
              "--gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2402_09900_amd import binding as mb
    from paper_2402_09900_amd import tapes

    key = args.workload
    wl = tapes.WORKLOADS[key]
    flops = None
    if wl.kind == "linattn":
        w, sets, bytes_per, n, flops = setup_linattn(torch, mb, tapes, key)
    elif wl.kind == "discount":
        w, sets, bytes_per, n = setup_discount(torch, mb, tapes, key)
    elif wl.kind == "ffm":
        w, sets, bytes_per, n = setup_ffm(torch, mb, tapes, key)
    elif wl.kind == "tbb":
        w, sets, bytes_per, n = setup_tbb(torch, mb, tapes, key)
    else:
        w, sets, bytes_per, n = setup_diag(torch, mb, tapes, key)
    calls = sets[0]
    # the warmup steps carry HIP events on every call; the slowest call is
    # the dominant one, and in the timed steps only it carries events (each
    # event pair left the GPU idle for a few microseconds between calls)
    warm = {name: Timer(torch) for name in calls}
    timers = {name: Timer(torch) for name in calls}

    # calibration anchor for hardware byte counters: one plain device copy of
    # a known size (outside the timed region)
    cal_src = torch.empty(COPY_CAL_BYTES, dtype=torch.uint8, device="cuda")
    cal_dst = torch.empty_like(cal_src)
    cal_dst.copy_(cal_src)
    torch.cuda.synchronize()
    del cal_src, cal_dst

    def step(i, tm, which):
        for name, fn in sets[i % len(sets)].items():
            if name in which:
                tm[name](fn)
            else:
                fn()

    for i in range(max(args.warmup, 1)):      # with no warmup, one untimed step picks the dominant call
        step(i, warm, calls)
    torch.cuda.synchronize()
    dom = max(calls, key=lambda k: warm[k].median_ms())   # the median ignores a slow first call
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, timers, (dom,))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # the other calls' durations, from as many steps again after the timed
    # region, with events on every call
    for i in range(args.steps):
        step(args.warmup + args.steps + i, timers, tuple(k for k in calls if k != dom))
    torch.cuda.synchronize()
    ms_per_step = wall * 1e3 / max(args.steps, 1)
    value = n / (ms_per_step * 1e-3)
    # every call on a prepared workspace ran (no mismatch) and no wait gave up
    for ws in PREPARED:
        st = mb.memoroid_workspace_status(ws.data_ptr(), ws.numel(), torch.cuda.current_stream().cuda_stream)
        if st != 0:
            print("bench.py: workspace status %s" % mb.status_string(st), file=sys.stderr)
            sys.exit(1)

    # the same step through the self-initialising entry points (a fill of
    # each call's workspace header, counters and first bank, then the
    # kernels); the prepared workspaces are rebound by this, so their status
    # was checked above
    SUFFIX[0] = ""
    for i in range(max(args.warmup, 1)):
        step(i, warm, ())
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, timers, ())
    torch.cuda.synchronize()
    self_init_ms = (time.perf_counter() - t0) * 1e3 / max(args.steps, 1)
    SUFFIX[0] = "_prepared"

    per_call_ms = {name: timers[name].mean_ms() for name in calls}
    if flops is not None:
        achieved = flops[dom] / (per_call_ms[dom] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": FP32_MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": None}
    else:
        achieved = bytes_per[dom] / (per_call_ms[dom] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None}
    roof["traffic"] = recorded_traffic(key, ("linattn_" + dom) if wl.kind == "linattn" else dom)
    roof["traffic_unit"] = "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
    roof["kernel"] = {"fwd": {"diag": "memoroid_scan_diag", "linattn": "memoroid_scan_linattn",
                              "ffm": "memoroid_scan_ffm"}.get(wl.kind),
                      "bwd": {"linattn": "memoroid_scan_linattn_bwd", "ffm": "memoroid_scan_ffm_bwd"}.get(
                          wl.kind, "memoroid_scan_diag_bwd"), "return": "memoroid_discounted_return",
                      "gae": "memoroid_gae", "insert": "memoroid_tbb_begin_indices",
                      "sample": "memoroid_tbb_sample"}[dom]
    roof["ms_per_launch"] = round(per_call_ms[dom], 4)
    roof["ms_per_launch_p10_p50_p90"] = timers[dom].percentiles_ms()
    if flops is None:
        # the fraction of what a plain copy kernel reaches on this GPU, from
        # the same harness (after the timed steps)
        cgbps = copy_probe_gbps(torch)
        roof["copy_probe_GBps"] = round(cgbps, 1)
        roof["frac_of_copy_probe"] = round(achieved / cgbps, 4)
    roof["algorithmic_bytes_per_launch"] = int(bytes_per[dom])
    if flops is not None:
        roof["algorithmic_flops_per_launch"] = int(flops[dom])
        # the recurrent form's own count (no chunking, no masked work), the
        # O(dk) normaliser terms left out: per step and head the forward adds
        # phi(k) v^T to the state and reads phi(q)^T S (2 dk dv each); the
        # gradient rebuilds the state, reads dq from it, accumulates the
        # state's gradient and reads dk and dv from that (2 dk dv each)
        dkdv = wl.dk * wl.dv * wl.T * wl.d
        rec = {"fwd": 4 * dkdv, "bwd": 10 * dkdv}[dom]
        roof["recurrent_flops_per_launch"] = int(rec)
        roof["frac_recurrent"] = round(rec / (per_call_ms[dom] * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4)
        roof["step_frac"] = round(sum(flops.get(k, 0) for k in calls) / (ms_per_step * 1e-3) / 1e12
                                  / FP32_MFMA_PEAK_TFLOPS, 4)
    else:
        roof["step_frac"] = round(sum(bytes_per[k] for k in calls) / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)

    result = {
        "metric": METRIC,
        "value": value,
        "unit": UNIT,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"f32": "f32", "bf16": "bf16 in / f32 state", "c64": "c64"}[wl.dtype],
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "T": wl.T,
                   ("heads" if wl.kind == "linattn" else "d"): wl.d,
                   **({"m": wl.dk, "c": wl.dv} if wl.kind == "ffm" else {}),
                   **({"gamma": wl.gamma, "lambda": wl.lam} if wl.kind == "discount" else {}),
                   "passes": list(calls.keys()),
                   "flags_sha256": tapes.flags_sha256(w.start),
                   "entry_points": "*_prepared (workspaces prepared once before timing)",
                   "self_init_ms_per_step": round(self_init_ms, 4),
                   "buffer_sets": len(sets),
                   "ms_per_call": {k: round(v, 4) for k, v in per_call_ms.items()},
                   "GBps_per_call": {k: round(bytes_per[k] / (per_call_ms[k] * 1e-3) / 1e9, 1)
                                     for k in calls}},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(key, tapes, w)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
