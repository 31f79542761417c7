"""The cross-tile protocol of the single-pass scans under randomised
interleavings, on the CPU (tests/lookback_model/lookback_model.cpp, built
here with g++ and ThreadSanitizer).

The GPU runs the protocol in the dispatcher's natural order only; the model
runs its state machine with worker threads delayed at random points: tickets
from wrapping per-chain counters (epoch parity) or, as in the FFM forward,
from one counter per (chain, group of workgroups) over a padded grid, two banks of self-validating
descriptor words cleared for the next call by their owners, the look-back,
the episode-index counts, the workspace signature (binding, poisoning,
standing down), and the discounted return's index-ordered tiles with per-tile
epoch words and the fallback that computes an awaited tile from its inputs.
Every call is compared with the fp64 oracle on the same seeded inputs (the
reset theorem of Section 4 applied to the diagonal monoid and to the return
monoid of App. D).  Each mutation alters one step of the protocol and must be
caught.  Any data race ThreadSanitizer sees fails the run."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2402_09900_amd import tapes

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lookback_model", "lookback_model.cpp")

MUTATIONS_DIAG = {1: "no idle-bank clear", 2: "one bank", 3: "counter wraps every call", 4: "signature ignored",
                  5: "no poison", 6: "NaN not canonicalised", 9: "own count published as inclusive"}
MUTATIONS_RETURN = {1: "no idle-bank clear", 2: "one bank", 7: "epoch word not stored",
                    8: "fallback folds the wrong tile"}


@pytest.fixture(scope="module")
def model(tmp_path_factory):
    d = tmp_path_factory.mktemp("lookback_model")
    exe = str(d / "lookback_model")
    subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-pthread", "-fsanitize=thread", "-Wall", "-Werror",
                    "-o", exe, SRC], check=True)
    _write_problems(str(d))
    return exe, str(d)


def _write_problems(d):
    """Three diagonal problems and three return problems of one shape each
    (consecutive calls on one workspace cycle through them), with NaN inputs
    in one of them, and the oracle's results and companions."""
    for k in range(3):
        rng = np.random.Generator(np.random.PCG64(900 + k))
        B, T, dd = 2, 90, 5
        start = np.stack([tapes.flags_from_lengths(rng.integers(1, 30 if k != 2 else 4, size=T), T)
                          for _ in range(B)]).astype(np.uint8)
        a = rng.uniform(0.3, 1.0, size=(B, T, dd)).astype(np.float32)
        x = rng.standard_normal((B, T, dd)).astype(np.float32)
        if k == 1:
            # a NaN whose bits are all ones, the pattern of an unpublished
            # descriptor word: it stays in its episode, and every word it
            # reaches must be published canonicalised
            x.view(np.uint32)[0, 40, 2] = 0xFFFFFFFF
        ref, mag = oracle.diag_fwd(a.astype(np.float64), x.astype(np.float64), start)
        idx = oracle.episode_idx(start).astype(np.int32)
        base = os.path.join(d, "diag%d" % k)
        open(base + ".shape", "w").write("%d %d %d\n" % (B, T, dd))
        for ext, arr in ((".a", a), (".x", x), (".start", start), (".ref", ref), (".mag", mag), (".idx", idx)):
            np.ascontiguousarray(arr).tofile(base + ext)
    for k in range(3):
        rng = np.random.Generator(np.random.PCG64(950 + k))
        B, T, gamma = 2, 120, np.float32(0.9)
        start = np.stack([tapes.flags_from_lengths(rng.integers(1, 60, size=T), T) for _ in range(B)])
        start = start.astype(np.uint8)
        r = rng.standard_normal((B, T)).astype(np.float32)
        ref, mag = oracle.discounted_return(r.astype(np.float64), start, float(gamma))
        base = os.path.join(d, "ret%d" % k)
        open(base + ".shape", "w").write("%d %d %.9g\n" % (B, T, float(gamma)))
        for ext, arr in ((".r", r), (".start", start), (".ref", ref), (".mag", mag)):
            np.ascontiguousarray(arr).tofile(base + ext)


TSAN_EXIT = 66


def _run(model, what, schedules, mutation):
    exe, d = model
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 exitcode=%d report_signal_unsafe=0" % TSAN_EXIT)
    return subprocess.run([exe, d, what, str(schedules), str(mutation)], capture_output=True, text=True, env=env,
                          timeout=600)


def _clean(res):
    assert "ThreadSanitizer" not in res.stderr, res.stderr[-3000:]
    assert res.returncode == 0, res.stdout + res.stderr[-2000:]
    assert "failures 0" in res.stdout


def _caught(res, name):
    """A mutation is caught by a wrong result, a missed stand-down or a wait
    that gives up (the model exits 0 having seen it), or by a data race."""
    raced = res.returncode == TSAN_EXIT and "ThreadSanitizer" in res.stderr
    assert raced or res.returncode == 0, "not caught: " + name + "\n" + res.stdout + res.stderr[-1500:]


def test_diag_protocol_under_random_schedules(model):
    _clean(_run(model, "diag", 3000, 0))


def test_grouped_counters_under_random_schedules(model):
    """One counter per (chain, group): a workgroup's predecessor position
    belongs to another counter, claimed by a workgroup earlier in the grid;
    with as few workers as the model draws, every wait still ends."""
    _clean(_run(model, "diag_grouped", 2000, 0))


@pytest.mark.parametrize("mutation", [2, 3], ids=["one_bank", "counter_wraps_every_call"])
def test_grouped_counters_mutation_is_caught(model, mutation):
    _caught(_run(model, "diag_grouped", 400, mutation), MUTATIONS_DIAG[mutation])


def test_return_protocol_and_fallback_under_random_schedules(model):
    _clean(_run(model, "return", 7000, 0))


@pytest.mark.parametrize("mutation", sorted(MUTATIONS_DIAG), ids=lambda m: MUTATIONS_DIAG[m].replace(" ", "_"))
def test_diag_protocol_mutation_is_caught(model, mutation):
    _caught(_run(model, "diag", 400, mutation), MUTATIONS_DIAG[mutation])


@pytest.mark.parametrize("mutation", sorted(MUTATIONS_RETURN), ids=lambda m: MUTATIONS_RETURN[m].replace(" ", "_"))
def test_return_protocol_mutation_is_caught(model, mutation):
    _caught(_run(model, "return", 600, mutation), MUTATIONS_RETURN[mutation])
