"""Seeded synthetic tapes shaped like the paper's RL rollouts.

This module only draws random numbers and stores them in the dtypes the
library consumes; it contains none of the scan's arithmetic, so both the HIP
path and the CPU oracle can be fed from it.

A tape is a run of episodes laid end to end (Tape-Based Batching, Section 4.1
and Fig. 2): per-step begin flags ``start[B][T]`` (uint8, nonzero = an episode
begins here; Section 2.1) and per-step data ``[B][T][d]`` with features
contiguous.  Episode lengths are drawn from a per-workload law until they cover
T; the last episode is cut at the tape end, the way Alg. 2 truncates a sampled
batch to exactly its size.

Generator: ``numpy.random.Generator(PCG64(seed))``; draw order is episode
lengths, then a, then x (or q, k, v), then the upstream gradient g.  Floating
values are drawn in float32 (complex: two float32 parts) and bf16 inputs are
rounded from those float32 draws to nearest-even.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Callable, Dict, Optional

import numpy as np

# ----------------------------------------------------------------- bf16 codec


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); returns the
    uint16 bit patterns.  NaN stays NaN (quiet bit forced)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    chunk = 1 << 24
    flat_u, flat_o = u.reshape(-1), out.reshape(-1)
    for i in range(0, flat_u.size, chunk):
        v = flat_u[i:i + chunk]
        lsb = (v >> 16) & np.uint32(1)
        r = ((v + np.uint32(0x7FFF) + lsb) >> 16).astype(np.uint16)
        nan = (v & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
        if nan.any():
            r[nan] = ((v[nan] >> 16) | np.uint32(0x0040)).astype(np.uint16)
        flat_o[i:i + chunk] = r
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact decode of bfloat16 bit patterns to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


# ------------------------------------------------------------ episode flags


def flags_from_lengths(lengths, T: int) -> np.ndarray:
    """Begin flags for episodes of the given lengths laid end to end, cut at T."""
    flags = np.zeros(T, dtype=np.uint8)
    pos = 0
    for n in lengths:
        if pos >= T:
            break
        flags[pos] = 1
        pos += int(n)
    flags[0] = 1
    return flags


def _flags_from_sampler(rng: np.random.Generator, T: int,
                        draw: Callable[[np.random.Generator, int], np.ndarray]) -> np.ndarray:
    """Draw episode lengths (in batches) until they cover T steps."""
    lengths = []
    covered = 0
    while covered < T:
        n = draw(rng, 1024)
        n = np.maximum(n.astype(np.int64), 1)
        lengths.append(n)
        covered += int(n.sum())
    lens = np.concatenate(lengths)
    ends = np.cumsum(lens)
    starts = np.concatenate([[0], ends[:-1]])
    starts = starts[starts < T]
    flags = np.zeros(T, dtype=np.uint8)
    flags[starts] = 1
    return flags


def _uniform_boundaries(n_episodes: int):
    def make(rng: np.random.Generator, T: int) -> np.ndarray:
        flags = np.zeros(T, dtype=np.uint8)
        flags[0] = 1
        k = min(n_episodes - 1, T - 1)
        if k > 0:
            cut = rng.choice(np.arange(1, T), size=k, replace=False)
            flags[cut] = 1
        return flags
    return make


def _geometric(mean: float):
    def make(rng, T):
        return _flags_from_sampler(rng, T, lambda r, n: r.geometric(1.0 / mean, size=n))
    return make


def _uniform_int(lo: int, hi: int):
    def make(rng, T):
        return _flags_from_sampler(rng, T, lambda r, n: r.integers(lo, hi + 1, size=n))
    return make


def _lognormal(mu: float, sigma: float):
    def make(rng, T):
        return _flags_from_sampler(
            rng, T, lambda r, n: np.maximum(1, np.rint(r.lognormal(mu, sigma, size=n))))
    return make


# ------------------------------------------------------------------ values


def _uniform_f32(rng, lo, hi, shape):
    return (np.float32(lo) + np.float32(hi - lo) * rng.random(shape, dtype=np.float32)).astype(np.float32)


def _normal_f32(rng, shape):
    return rng.standard_normal(shape, dtype=np.float32)


def _cnormal_c64(rng, shape):
    """Standard complex normal: real and imaginary parts ~ N(0, 1/2)."""
    out = np.empty(shape, dtype=np.complex64)
    v = out.view(np.float32).reshape(shape + (2,))
    v[...] = rng.standard_normal(shape + (2,), dtype=np.float32)
    v *= np.float32(math.sqrt(0.5))
    return out


# ------------------------------------------------------------------ configs


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: shape, dtypes and the laws it is drawn from."""
    key: int
    name: str
    kind: str                 # "diag", "linattn", "discount", "ffm" or "tbb"
    B: int
    T: int
    d: int                    # features (diag) or heads (linattn)
    dtype: str                # storage dtype of a, x: "f32", "bf16", "c64"
    out_dtype: str
    a_invariant: bool
    a_range: tuple            # |a| ~ U(lo, hi)
    episodes: Callable        # (rng, T) -> uint8 flags[T]
    backward: bool
    dk: int = 0
    dv: int = 0
    chunk: int = 0
    gamma: float = 0.0        # discount (returns / advantages)
    lam: float = 0.0          # GAE lambda

    def describe(self) -> str:
        return self.name


WORKLOADS: Dict[int, Workload] = {
    1: Workload(1, "diag_real_f32_T1024_d32_8ep_fwd", "diag", 1, 1024, 32, "f32", "f32",
                False, (0.5, 0.99), _uniform_boundaries(8), False),
    2: Workload(2, "diag_complex_c64_T65536_d256_geom200_fwd_bwd", "diag", 1, 65536, 256, "c64", "c64",
                True, (0.9, 0.999), _geometric(200.0), True),
    3: Workload(3, "linattn_f32_T32768_H4_dk64_dv64_geom500_chunk64", "linattn", 1, 32768, 4, "f32", "f32",
                False, (0.0, 0.0), _geometric(500.0), False, dk=64, dv=64, chunk=64),
    4: Workload(4, "diag_real_bf16_B64_T16384_d512_unif10_1000_fwd", "diag", 64, 16384, 512, "bf16", "bf16",
                False, (0.8, 0.999), _uniform_int(10, 1000), False),
    5: Workload(5, "diag_real_f32_T1048576_d256_lognormal5_1.5_fwd_bwd", "diag", 1, 1 << 20, 256, "f32", "f32",
                False, (0.5, 0.99), _lognormal(5.0, 1.5), True),
    6: Workload(6, "return_gae_f32_T16777216_unif1_1000_g0.99_l0.95", "discount", 1, 1 << 24, 1, "f32", "f32",
                False, (0.0, 0.0), _uniform_int(1, 1000), False, gamma=0.99, lam=0.95),
    7: Workload(7, "ffm_c64_T262144_m32_c8_geom200_fwd_bwd", "ffm", 1, 1 << 18, 32, "c64", "c64",
                True, (0.5, 0.995), _geometric(200.0), True, dk=32, dv=8),
    8: Workload(8, "tbb_D16777216_row64B_batch1048576_unif1_1000", "tbb", 1, 1 << 24, 16, "f32", "f32",
                False, (0.0, 0.0), _uniform_int(1, 1000), False, chunk=1 << 20),
    9: Workload(9, "linattn_f32_T32768_H4_dk64_dv64_geom500_chunk64_fwd_bwd", "linattn", 1, 32768, 4, "f32", "f32",
                False, (0.0, 0.0), _geometric(500.0), True, dk=64, dv=64, chunk=64),
}


@dataclasses.dataclass
class DiagTape:
    """Inputs of a diagonal-recurrence workload, in storage dtypes.

    a: float32 / complex64 / uint16 (bf16 bits); [B,T,d] or [d] if invariant.
    x, g: same dtype as a, [B,T,d] (g is None for forward-only workloads).
    start: uint8 [B,T]."""
    a: np.ndarray
    x: np.ndarray
    start: np.ndarray
    g: Optional[np.ndarray]
    dtype: str
    out_dtype: str
    B: int
    T: int
    d: int
    a_invariant: bool

    def decoded(self, name: str) -> np.ndarray:
        """float64 / complex128 copy of an input, decoded exactly."""
        v = getattr(self, name)
        if self.dtype == "bf16":
            return bf16_bits_to_f32(v).astype(np.float64)
        if self.dtype == "c64":
            return v.astype(np.complex128)
        return v.astype(np.float64)


@dataclasses.dataclass
class LinAttnTape:
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    start: np.ndarray
    T: int
    H: int
    dk: int
    dv: int
    chunk: int


def make_diag(key: int, seed: Optional[int] = None, B: Optional[int] = None,
              T: Optional[int] = None, d: Optional[int] = None,
              with_grad: Optional[bool] = None, flag_bytes: bool = False) -> DiagTape:
    """Draw a diagonal-recurrence tape for workload ``key``; sizes may be
    overridden (same laws) for reduced-size parity cases.

    flag_bytes: write random nonzero bytes (1..255) instead of 1 at begin steps."""
    w = WORKLOADS[key]
    assert w.kind == "diag"
    B = w.B if B is None else B
    T = w.T if T is None else T
    d = w.d if d is None else d
    with_grad = w.backward if with_grad is None else with_grad
    rng = np.random.Generator(np.random.PCG64(key if seed is None else seed))
    start = np.stack([w.episodes(rng, T) for _ in range(B)]) if T > 0 else np.zeros((B, 0), np.uint8)
    start = start.reshape(B, T).astype(np.uint8)
    if flag_bytes and start.size:
        nz = start != 0
        start[nz] = rng.integers(1, 256, size=int(nz.sum()), dtype=np.uint16).astype(np.uint8)
    lo, hi = w.a_range
    if w.dtype == "c64":
        shape_a = (d,) if w.a_invariant else (B, T, d)
        mag = _uniform_f32(rng, lo, hi, shape_a).astype(np.float64)
        theta = 2.0 * math.pi * rng.random(shape_a)
        a = (mag * np.exp(1j * theta)).astype(np.complex64)
        x = _cnormal_c64(rng, (B, T, d))
        g = _cnormal_c64(rng, (B, T, d)) if with_grad else None
    else:
        shape_a = (d,) if w.a_invariant else (B, T, d)
        a = _uniform_f32(rng, lo, hi, shape_a)
        x = _normal_f32(rng, (B, T, d))
        g = _normal_f32(rng, (B, T, d)) if with_grad else None
        if w.dtype == "bf16":
            a = f32_to_bf16_bits(a)
            x = f32_to_bf16_bits(x)
            g = f32_to_bf16_bits(g) if g is not None else None
    return DiagTape(a=a, x=x, start=start, g=g, dtype=w.dtype, out_dtype=w.out_dtype,
                    B=B, T=T, d=d, a_invariant=w.a_invariant)


def make_linattn(key: int = 3, seed: Optional[int] = None, T: Optional[int] = None,
                 H: Optional[int] = None, dk: Optional[int] = None,
                 dv: Optional[int] = None) -> LinAttnTape:
    w = WORKLOADS[key]
    assert w.kind == "linattn"
    T = w.T if T is None else T
    H = w.d if H is None else H
    dk = w.dk if dk is None else dk
    dv = w.dv if dv is None else dv
    rng = np.random.Generator(np.random.PCG64(key if seed is None else seed))
    start = w.episodes(rng, T) if T > 0 else np.zeros(0, np.uint8)
    q = _normal_f32(rng, (T, H, dk))
    k = _normal_f32(rng, (T, H, dk))
    v = _normal_f32(rng, (T, H, dv))
    return LinAttnTape(q=q, k=k, v=v, start=start.astype(np.uint8), T=T, H=H, dk=dk, dv=dv,
                       chunk=w.chunk)


def flags_sha256(start: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(start, dtype=np.uint8).tobytes()).hexdigest()


def make_custom_diag(dtype: str, B: int, T: int, d: int, a_invariant: bool, seed: int,
                     a_range=(0.5, 0.99), mean_episode: float = 50.0, with_grad: bool = True,
                     out_dtype: Optional[str] = None) -> DiagTape:
    """A diagonal tape of any shape and dtype for edge-case tests: Geometric
    episode lengths of the given mean, |a| ~ U(a_range) (uniform phase for
    complex), x and g standard normal."""
    rng = np.random.Generator(np.random.PCG64(seed))
    start = np.stack([_geometric(mean_episode)(rng, T) for _ in range(B)]) if T > 0 else np.zeros((B, 0), np.uint8)
    start = start.reshape(B, T).astype(np.uint8)
    shape_a = (d,) if a_invariant else (B, T, d)
    lo, hi = a_range
    if dtype == "c64":
        mag = _uniform_f32(rng, lo, hi, shape_a).astype(np.float64)
        a = (mag * np.exp(2j * math.pi * rng.random(shape_a))).astype(np.complex64)
        x = _cnormal_c64(rng, (B, T, d))
        g = _cnormal_c64(rng, (B, T, d)) if with_grad else None
    else:
        a = _uniform_f32(rng, lo, hi, shape_a)
        x = _normal_f32(rng, (B, T, d))
        g = _normal_f32(rng, (B, T, d)) if with_grad else None
        if dtype == "bf16":
            a, x = f32_to_bf16_bits(a), f32_to_bf16_bits(x)
            g = None
    return DiagTape(a=a, x=x, start=start, g=g, dtype=dtype, out_dtype=out_dtype or dtype,
                    B=B, T=T, d=d, a_invariant=a_invariant)


@dataclasses.dataclass
class DiscountTape:
    """Transitions of an RL tape for the return / advantage workloads.

    r, v, vn: float32 [B,T] (reward, V(s_t), V(s'_t)); done, start: uint8 [B,T]."""
    r: np.ndarray
    v: np.ndarray
    vn: np.ndarray
    done: np.ndarray
    start: np.ndarray
    gamma: float
    lam: float
    B: int
    T: int


def make_discount(key: int = 6, seed: Optional[int] = None, B: Optional[int] = None, T: Optional[int] = None,
                  episodes: Optional[Callable] = None, done_rate: float = 0.5) -> DiscountTape:
    """Rewards and values of a tape of episodes.  Draw order: episode lengths
    (per tape), rewards ~ N(0,1), values V(s_t) ~ N(0,1), the value of each
    episode's final next state ~ N(0,1), then each episode end is terminal
    with probability done_rate (except at the tape end, where the episode is
    cut off, not finished).  Inside an episode V(s'_t) = V(s_{t+1})."""
    w = WORKLOADS[key]
    assert w.kind == "discount"
    B = w.B if B is None else B
    T = w.T if T is None else T
    law = w.episodes if episodes is None else episodes
    rng = np.random.Generator(np.random.PCG64(key if seed is None else seed))
    start = (np.stack([law(rng, T) for _ in range(B)]) if T > 0 else np.zeros((B, 0), np.uint8))
    start = start.reshape(B, T).astype(np.uint8)
    r = _normal_f32(rng, (B, T))
    v = _normal_f32(rng, (B, T))
    boot = _normal_f32(rng, (B, T))
    coin = rng.random((B, T)) < done_rate
    ends = np.zeros((B, T), dtype=bool)
    if T > 0:
        ends[:, :-1] = start[:, 1:] != 0
    vn = np.empty((B, T), dtype=np.float32)
    if T > 0:
        vn[:, :-1] = v[:, 1:]
        vn[:, -1] = boot[:, -1]
    vn[ends] = boot[ends]
    done = (ends & coin).astype(np.uint8)
    return DiscountTape(r=r, v=v, vn=vn, done=done, start=start, gamma=w.gamma, lam=w.lam, B=B, T=T)


@dataclasses.dataclass
class FfmTape:
    """Inputs of the FFM aggregator: alpha [m], omega [c], x [B,T,m] float32,
    start [B,T] uint8."""
    alpha: np.ndarray
    omega: np.ndarray
    x: np.ndarray
    start: np.ndarray
    B: int
    T: int
    m: int
    c: int


def make_ffm(key: int = 7, seed: Optional[int] = None, B: Optional[int] = None, T: Optional[int] = None,
             m: Optional[int] = None, c: Optional[int] = None, episodes: Optional[Callable] = None) -> FfmTape:
    """FFM inputs.  |gamma_j| = exp(-|alpha_j|) is spread log-uniformly in
    decay time between the workload's |a| bounds (signs of alpha random),
    omega_k evenly spaced in [0, pi), x ~ N(0, 1).  Draw order: episode
    lengths (per tape), alpha signs, x."""
    w = WORKLOADS[key]
    assert w.kind == "ffm"
    B = w.B if B is None else B
    T = w.T if T is None else T
    m = w.dk if m is None else m
    c = w.dv if c is None else c
    law = w.episodes if episodes is None else episodes
    rng = np.random.Generator(np.random.PCG64(key if seed is None else seed))
    start = (np.stack([law(rng, T) for _ in range(B)]) if T > 0 else np.zeros((B, 0), np.uint8))
    start = start.reshape(B, T).astype(np.uint8)
    lo, hi = w.a_range
    tau = np.exp(np.linspace(np.log(-1.0 / np.log(lo)), np.log(-1.0 / np.log(hi)), m))  # decay times
    sign = np.where(rng.random(m) < 0.5, -1.0, 1.0)
    alpha = (sign / tau).astype(np.float32)
    omega = (np.pi * np.arange(c) / max(c, 1)).astype(np.float32)
    x = _normal_f32(rng, (B, T, m))
    return FfmTape(alpha=alpha, omega=omega, x=x, start=start, B=B, T=T, m=m, c=c)


@dataclasses.dataclass
class TbbBuffer:
    """A replay buffer D of n_D transitions (rows of `row` float32 values),
    the begin flags it was filled with, the begin positions used to place
    them (as the generator laid the episodes out), and uniform draws of
    positions in that list (Alg. 2 samples them from U(0, card(I) - 1))."""
    D: np.ndarray
    start: np.ndarray
    begins: np.ndarray
    draws: np.ndarray
    batch: int


def make_tbb(key: int = 8, seed: Optional[int] = None, n: Optional[int] = None, row: Optional[int] = None,
             batch: Optional[int] = None, n_draws: Optional[int] = None,
             episodes: Optional[Callable] = None) -> TbbBuffer:
    """Draw order: episode lengths, D ~ N(0, 1), draws."""
    w = WORKLOADS[key]
    assert w.kind == "tbb"
    n = w.T if n is None else n
    row = w.d if row is None else row
    batch = w.chunk if batch is None else batch
    law = w.episodes if episodes is None else episodes
    rng = np.random.Generator(np.random.PCG64(key if seed is None else seed))
    start = law(rng, n) if n > 0 else np.zeros(0, np.uint8)
    begins = np.flatnonzero(start).astype(np.int64)        # where the generator placed each episode
    D = _normal_f32(rng, (n, row))
    nd = batch if n_draws is None else n_draws
    draws = rng.integers(0, max(begins.size, 1), size=nd).astype(np.int64)
    return TbbBuffer(D=D, start=start.astype(np.uint8), begins=begins, draws=draws, batch=batch)
