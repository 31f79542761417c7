"""Parity of the discounted-return and advantage kernels (through the C ABI)
with the fp64 oracle.

Inputs come from paper_2402_09900_amd.tapes; outputs are compared element by
element with the conditioned relative error (|y - r| / max(|r|, m), m the
oracle's magnitude companion), at most 1e-4 (fp32 arithmetic).  The full
workload (one tape of 2^24 steps) is compared whole: the oracle's loop is
linear in T.
"""
import numpy as np
import pytest

import oracle
from conftest import announce, cond_err, forced_fallback
from paper_2402_09900_amd import tapes

torch = pytest.importorskip("torch")
from paper_2402_09900_amd import binding as mb  # noqa: E402

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-4


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def run_return(r, start, gamma, ws=None):
    G = mb.discounted_return(dev(r), dev(start), gamma, workspace=ws)
    torch.cuda.synchronize()
    return G.cpu().numpy()


def run_gae(tp, gamma, lam, with_vn=True, with_done=True, target=True):
    adv, tg = mb.gae(dev(tp.r), dev(tp.v), dev(tp.start), gamma, lam,
                     value_next=dev(tp.vn) if with_vn else None,
                     done=dev(tp.done) if with_done else None, target=target)
    torch.cuda.synchronize()
    return adv.cpu().numpy(), (tg.cpu().numpy() if tg is not None else None)


def ref_gae(tp, gamma, lam, with_vn=True, with_done=True):
    g32, l32 = float(np.float32(gamma)), float(np.float32(lam))
    return oracle.gae(tp.r.astype(np.float64), tp.v.astype(np.float64), tp.start, g32, l32,
                      vn=tp.vn.astype(np.float64) if with_vn else None,
                      done=tp.done if with_done else None)


def check_return(tp, gamma, label):
    announce("return %s B=%d T=%d gamma=%g" % (label, tp.B, tp.T, gamma))
    G = run_return(tp.r, tp.start, gamma)
    ref, m = oracle.discounted_return(tp.r.astype(np.float64), tp.start, float(np.float32(gamma)))
    e = cond_err(G, ref, m)
    assert e <= TOL, (label, e)


def check_gae(tp, gamma, lam, label, with_vn=True, with_done=True, target=True):
    announce("gae %s B=%d T=%d gamma=%g lam=%g vn=%s done=%s target=%s"
             % (label, tp.B, tp.T, gamma, lam, with_vn, with_done, target))
    adv, tg = run_gae(tp, gamma, lam, with_vn, with_done, target)
    ra, rt, ma, mt = ref_gae(tp, gamma, lam, with_vn, with_done)
    e = cond_err(adv, ra, ma)
    assert e <= TOL, (label, "adv", e)
    if target:
        e = cond_err(tg, rt, mt)
        assert e <= TOL, (label, "target", e)
    else:
        assert tg is None


@pytest.fixture(scope="module")
def w6():
    return tapes.make_discount(6)


def test_workload6_full_return(w6):
    check_return(w6, w6.gamma, "workload6")


def test_workload6_full_gae(w6):
    check_gae(w6, w6.gamma, w6.lam, "workload6")


# T around the tiles (8192 steps for the return, 4096 for the advantage),
# the wavefront runs (2048 / 1024 steps), the lanes' runs (32 / 16 steps) and
# the 4-step vector: ragged tails, one-tile tapes, T % 4 != 0 (scalar kernel)
SHAPES = [(1, 1), (1, 3), (1, 4), (2, 5), (1, 15), (2, 16), (1, 17), (1, 31), (2, 32), (2, 33), (3, 63),
          (1, 64), (2, 65), (1, 1023), (2, 1024), (1, 1025), (1, 2047), (2, 2048), (2, 2049), (1, 4095),
          (2, 4096), (3, 4097), (1, 8191), (2, 8192), (3, 8193), (2, 2 * 8192 + 1), (2, 3 * 4096 + 36),
          (5, 3 * 4096 + 37), (4, 20000), (7, 9 * 4096 + 2)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dT%d" % s)
def test_shapes_return_and_gae(shape):
    B, T = shape
    tp = tapes.make_discount(6, seed=100 + B * 7 + T, B=B, T=T, episodes=tapes._geometric(300.0))
    check_return(tp, 0.99, "shape")
    check_gae(tp, 0.99, 0.95, "shape")


@pytest.mark.parametrize("with_vn", [False, True])
@pytest.mark.parametrize("with_done", [False, True])
@pytest.mark.parametrize("target", [False, True])
def test_gae_optional_inputs(with_vn, with_done, target):
    tp = tapes.make_discount(6, seed=31, B=3, T=50000, episodes=tapes._uniform_int(1, 1000))
    check_gae(tp, 0.99, 0.95, "optional", with_vn, with_done, target)


@pytest.mark.parametrize("gamma,lam", [(0.0, 0.95), (1.0, 1.0), (0.99, 0.0), (0.5, 1.0), (1.0, 0.3)])
def test_discount_limits(gamma, lam):
    tp = tapes.make_discount(6, seed=41, B=2, T=30000, episodes=tapes._uniform_int(1, 1000))
    check_return(tp, gamma, "limits")
    check_gae(tp, gamma, lam, "limits")


def _flags(kind, B, T, rng):
    s = np.zeros((B, T), np.uint8)
    if kind == "all_begins":
        s[:] = 1
    elif kind == "single_episode":
        pass
    elif kind == "tile_boundaries":
        s[:, ::4096] = 1
    elif kind == "after_tile_boundaries":
        s[:, 1::4096] = 1
    elif kind == "last_step":
        s[:, -1] = 1
    elif kind == "flag_bytes":
        s = (rng.random((B, T)) < 0.01).astype(np.uint8) * rng.integers(1, 256, size=(B, T)).astype(np.uint8)
    return s


@pytest.mark.parametrize("kind", ["all_begins", "single_episode", "tile_boundaries", "after_tile_boundaries",
                                  "last_step", "flag_bytes"])
def test_flag_patterns(kind):
    rng = np.random.default_rng(51)
    B, T = 2, 40 * 4096
    tp = tapes.make_discount(6, seed=52, B=B, T=T)
    tp.start = _flags(kind, B, T, rng)
    tp.done = np.zeros((B, T), np.uint8)
    check_return(tp, 0.999, kind)
    check_return(tp, 1.0, kind)
    check_gae(tp, 0.99, 0.95, kind, with_vn=False, with_done=False)


def test_long_single_episode_undiscounted():
    """gamma = 1 over one episode of 2^22 steps: every tile's value depends on
    every tile to its right (the longest look-back chains)."""
    rng = np.random.default_rng(61)
    T = 1 << 22
    r = rng.standard_normal((1, T)).astype(np.float32)
    s = np.zeros((1, T), np.uint8)
    announce("return single episode T=%d gamma=1" % T)
    G = run_return(r, s, 1.0)
    ref, m = oracle.discounted_return(r.astype(np.float64), s, 1.0)
    assert cond_err(G, ref, m) <= TOL


def test_misaligned_rows_take_scalar_kernel():
    """Tensors starting 4 bytes into an allocation are not 16-byte aligned:
    the scalar kernel must give the same results."""
    tp = tapes.make_discount(6, seed=71, B=2, T=12288)
    announce("return/gae misaligned B=2 T=12288")
    n = tp.B * tp.T
    big_r = torch.zeros(n + 1, dtype=torch.float32, device=DEV)
    big_r[1:] = dev(tp.r.reshape(-1))
    r_mis = big_r[1:].view(tp.B, tp.T)
    G = mb.discounted_return(r_mis, dev(tp.start), 0.99)
    ref, m = oracle.discounted_return(tp.r.astype(np.float64), tp.start, float(np.float32(0.99)))
    assert cond_err(G.cpu().numpy(), ref, m) <= TOL
    big_v = torch.zeros(n + 1, dtype=torch.float32, device=DEV)
    big_v[1:] = dev(tp.v.reshape(-1))
    adv, tg = mb.gae(r_mis, big_v[1:].view(tp.B, tp.T), dev(tp.start), 0.99, 0.95,
                     value_next=dev(tp.vn), done=dev(tp.done))
    ra, rt, ma, mt = ref_gae(tp, 0.99, 0.95)
    assert cond_err(adv.cpu().numpy(), ra, ma) <= TOL
    assert cond_err(tg.cpu().numpy(), rt, mt) <= TOL


def test_nan_stays_in_its_episode():
    tp = tapes.make_discount(6, seed=81, B=1, T=5 * 4096)
    s = np.zeros((1, tp.T), np.uint8)
    s[0, [0, 5000, 9000, 15000]] = 1
    tp.start = s
    r = tp.r.copy()
    r[0, 7000] = np.nan
    announce("return nan T=%d" % tp.T)
    G = run_return(r, s, 0.99)
    ref, m = oracle.discounted_return(r.astype(np.float64), s, float(np.float32(0.99)))
    assert np.all(np.isnan(G[0, 5000:7001]))
    ok = ~np.isnan(ref)
    assert not np.any(np.isnan(G[ok]))
    assert cond_err(G[ok], ref[ok], m[ok]) <= TOL


def test_repeated_calls_share_a_workspace():
    tp = tapes.make_discount(6, seed=91, B=3, T=100000)
    ws = torch.empty(mb.memoroid_discount_workspace_bytes(3, 100000), dtype=torch.uint8, device=DEV)
    announce("return repeated B=3 T=100000")
    ref, m = oracle.discounted_return(tp.r.astype(np.float64), tp.start, float(np.float32(0.97)))
    for _ in range(3):
        G = run_return(tp.r, tp.start, 0.97, ws=ws)
        assert mb.workspace_status(ws) == mb.OK
        assert cond_err(G, ref, m) <= TOL


def test_lookback_fallback_computes_awaited_tiles():
    """With the fallback threshold at 0 polls, a look-back that finds its
    nearest tile unpublished computes that tile's aggregate from the inputs at
    once; results must not change."""
    with forced_fallback():
        for T, law in ((64 * 4096 + 12, tapes._uniform_int(1000, 30000)), (40 * 4096, tapes._uniform_int(1, 1000))):
            tp = tapes.make_discount(6, seed=93, B=2, T=T, episodes=law)
            check_return(tp, 0.999, "fallback")
            check_gae(tp, 0.99, 0.95, "fallback", with_vn=False)
        tp = tapes.make_discount(6, seed=94, B=1, T=32 * 4096 + 3)        # scalar kernel
        tp.start[:] = 0
        check_return(tp, 1.0, "fallback scalar")
        check_gae(tp, 0.99, 0.95, "fallback scalar")
