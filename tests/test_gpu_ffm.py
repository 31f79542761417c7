"""Parity of the FFM aggregator kernel (through the C ABI) with the fp64
oracle: conditioned relative error (|y - r| / max(|r|, m), m the oracle's
magnitude companion) at most 1e-4 (fp32 arithmetic), episode indices
bit-exact.  The full workload is compared on every element."""
import numpy as np
import pytest

import oracle
from conftest import announce, cond_err
from paper_2402_09900_amd import tapes

torch = pytest.importorskip("torch")
from paper_2402_09900_amd import binding as mb  # noqa: E402

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-4


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def check(f, label, x_override=None):
    announce("ffm %s B=%d T=%d m=%d c=%d" % (label, f.B, f.T, f.m, f.c))
    x = f.x if x_override is None else x_override
    S, idx = mb.scan_ffm(dev(f.alpha), dev(f.omega), dev(x), dev(f.start), episode_idx=True)
    torch.cuda.synchronize()
    ref, m = oracle.ffm(f.alpha.astype(np.float64), f.omega.astype(np.float64), x.astype(np.float64), f.start)
    got = S.cpu().numpy()
    e = cond_err(got, ref, m)
    assert e <= TOL, (label, e)
    np.testing.assert_array_equal(idx.cpu().numpy(), oracle.episode_idx(f.start))
    return got, ref


def test_workload7_full():
    check(tapes.make_ffm(7), "workload7")


# odd c -> one feature per lane (384-step tiles), even c -> two (768-step
# tiles); c = 1; m = 1; ragged T around one and several tiles; tile counts
# per chain below, at and past one group of 8 positions (the forward's grid
# is padded to whole groups)
SHAPES = [(1, 1, 1, 1), (1, 5, 1, 3), (2, 513, 3, 5), (1, 1000, 32, 8), (3, 2049, 7, 2), (2, 4096, 1, 16),
          (1, 777, 16, 1), (4, 3000, 5, 4), (1, 767, 8, 4), (2, 769, 4, 2), (1, 1537, 6, 3), (1, 385, 2, 1),
          (2, 6144, 4, 4), (1, 6913, 2, 8), (1, 12289, 3, 3)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "B%dT%dm%dc%d" % s)
def test_shapes(shape):
    B, T, m, c = shape
    check(tapes.make_ffm(7, seed=200 + T + m * c, B=B, T=T, m=m, c=c, episodes=tapes._geometric(150.0)), "shape")


def test_misaligned_output_takes_scalar_kernel():
    f = tapes.make_ffm(7, seed=211, B=2, T=1500, m=4, c=4)
    announce("ffm misaligned output")
    n = f.B * f.T * f.m * f.c
    big = torch.empty(n + 1, dtype=torch.complex64, device=DEV)
    ws = torch.empty(mb.memoroid_scan_ffm_workspace_bytes(f.B, f.T, f.m, f.c), dtype=torch.uint8, device=DEV)
    assert mb.memoroid_workspace_prepare(ws.data_ptr(), ws.numel(), torch.cuda.current_stream().cuda_stream) == mb.OK
    S = big[1:]
    al, om, x, s = dev(f.alpha), dev(f.omega), dev(f.x), dev(f.start)     # held until the kernel has run
    st = mb.memoroid_scan_ffm_prepared(al.data_ptr(), om.data_ptr(), x.data_ptr(), s.data_ptr(), S.data_ptr(), None,
                              f.B, f.T, f.m, f.c, ws.data_ptr(), ws.numel(), torch.cuda.current_stream().cuda_stream)
    assert st == mb.OK
    torch.cuda.synchronize()
    ref, m = oracle.ffm(f.alpha.astype(np.float64), f.omega.astype(np.float64), f.x.astype(np.float64), f.start)
    assert cond_err(S.cpu().numpy().reshape(ref.shape), ref, m) <= TOL


def test_nan_stays_in_its_episode():
    f = tapes.make_ffm(7, seed=212, B=1, T=3000, m=4, c=2)
    s = np.zeros((1, f.T), np.uint8)
    s[0, [0, 1000, 1700, 2500]] = 1
    f.start = s
    x = f.x.copy()
    x[0, 1200, 1] = np.nan
    announce("ffm nan")
    S = mb.scan_ffm(dev(f.alpha), dev(f.omega), dev(x), dev(s)).cpu().numpy()
    ref, m = oracle.ffm(f.alpha.astype(np.float64), f.omega.astype(np.float64), x.astype(np.float64), s)
    bad = np.isnan(ref)
    assert np.array_equal(np.isnan(S), bad)
    assert bad[0, 1200:1700, 1].all() and not bad[0, 1700:].any()
    assert cond_err(S[~bad], ref[~bad], m[~bad]) <= TOL


# ----------------------------------------------------------------- gradient

GTOL = 1e-4


def check_grad(f, label, seed=3):
    announce("ffm bwd %s B=%d T=%d m=%d c=%d" % (label, f.B, f.T, f.m, f.c))
    rng = np.random.Generator(np.random.PCG64(seed))
    G = (rng.standard_normal((f.B, f.T, f.m, f.c), dtype=np.float32)
         + 1j * rng.standard_normal((f.B, f.T, f.m, f.c), dtype=np.float32)).astype(np.complex64)
    al, om, x, s = dev(f.alpha), dev(f.omega), dev(f.x), dev(f.start)
    S = mb.scan_ffm(al, om, x, s)
    gx, ga, gw = mb.scan_ffm_bwd(al, om, s, S, dev(G))
    torch.cuda.synchronize()
    rdx, rda, rdw, mdx, mda, mdw = oracle.ffm_bwd(f.alpha.astype(np.float64), f.omega.astype(np.float64), f.start,
                                                  S.cpu().numpy().astype(np.complex128), G.astype(np.complex128))
    assert cond_err(gx.cpu().numpy(), rdx, mdx) <= GTOL, label
    assert cond_err(ga.cpu().numpy(), rda, mda) <= GTOL, label
    assert cond_err(gw.cpu().numpy(), rdw, mdw) <= GTOL, label


def test_grad_workload7_full():
    check_grad(tapes.make_ffm(7), "workload7")


# m up to 32: the finish kernel gathers rows in LDS; 33 and 40: the direct copy
@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (2, 513, 3, 4), (1, 1000, 32, 8), (3, 2049, 7, 2), (2, 4096, 1, 16),
                                   (1, 777, 16, 1), (4, 3000, 5, 4), (2, 300, 33, 4), (1, 700, 40, 2)],
                         ids=lambda s: "B%dT%dm%dc%d" % s)
def test_grad_shapes(shape):
    B, T, m, c = shape
    check_grad(tapes.make_ffm(7, seed=400 + T + m * c, B=B, T=T, m=m, c=c, episodes=tapes._geometric(150.0)),
               "shape")


def test_grad_nonfinite_adjoint_at_a_begin():
    """A non-finite upstream gradient at a begin step reaches that step's
    input gradient only: the step before ends an episode, and begin steps
    take no term of dalpha, domega (at 704 a lane's first step, at 1500
    inside a lane)."""
    f = tapes.make_ffm(7, seed=402, B=1, T=3000, m=4, c=4)
    s = np.zeros((1, f.T), np.uint8)
    s[0, [0, 704, 1500, 2200]] = 1
    f.start = s
    rng = np.random.Generator(np.random.PCG64(10))
    G = (rng.standard_normal((1, f.T, 4, 4), dtype=np.float32)
         + 1j * rng.standard_normal((1, f.T, 4, 4), dtype=np.float32)).astype(np.complex64)
    G[0, 704, 1, 2] = np.nan
    G[0, 1500, 3, 0] = np.nan
    announce("ffm bwd NaN adjoint at begins")
    al, om, x, sd = dev(f.alpha), dev(f.omega), dev(f.x), dev(s)
    S = mb.scan_ffm(al, om, x, sd)
    gx, ga, gw = mb.scan_ffm_bwd(al, om, sd, S, dev(G))
    gx, ga, gw = gx.cpu().numpy(), ga.cpu().numpy(), gw.cpu().numpy()
    rdx, rda, rdw, mdx, mda, mdw = oracle.ffm_bwd(f.alpha.astype(np.float64), f.omega.astype(np.float64), s,
                                                  S.cpu().numpy().astype(np.complex128), G.astype(np.complex128))
    bad = np.isnan(rdx)
    assert bad[0, 704, 1] and bad[0, 1500, 3] and bad.sum() == 2
    assert np.array_equal(np.isnan(gx), bad)
    assert cond_err(gx[~bad], rdx[~bad], mdx[~bad]) <= GTOL
    assert np.isfinite(ga).all() and np.isfinite(gw).all()
    assert cond_err(ga, rda, mda) <= GTOL
    assert cond_err(gw, rdw, mdw) <= GTOL


def test_grad_without_parameter_gradients():
    f = tapes.make_ffm(7, seed=401, B=2, T=2000, m=8, c=4)
    announce("ffm bwd x only")
    rng = np.random.Generator(np.random.PCG64(9))
    G = (rng.standard_normal((2, 2000, 8, 4), dtype=np.float32)
         + 1j * rng.standard_normal((2, 2000, 8, 4), dtype=np.float32)).astype(np.complex64)
    gx, ga, gw = mb.scan_ffm_bwd(dev(f.alpha), dev(f.omega), dev(f.start), None, dev(G), params=False)
    assert ga is None and gw is None
    S = np.zeros((2, 2000, 8, 4), np.complex128)          # unused by the input gradient
    rdx, _, _, mdx, _, _ = oracle.ffm_bwd(f.alpha.astype(np.float64), f.omega.astype(np.float64), f.start, S,
                                          G.astype(np.complex128))
    assert cond_err(gx.cpu().numpy(), rdx, mdx) <= GTOL
