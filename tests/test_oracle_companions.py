"""Pins of the oracle's magnitude companions from above.

Every GPU parity test divides its error by max(|r|, m), where r is the
oracle's result and m its magnitude companion: the same computation with
every term replaced by its absolute value.  The companion is therefore an
upper bound m >= |r| that equals |r| wherever the terms cannot cancel.  A
companion that is too large would silently widen every tolerance, so each
one is pinned here against something other than itself:

  * the oracle's own (independently pinned) primary output on inputs made
    non-negative, where the absolute-value computation *is* the plain one
    (e.g. the companion of the complex scan equals the real scan of |a|, |x|);
  * equality m == |r| on inputs whose terms all share one sign;
  * for the linear-attention gradients, the term-by-term absolute sum of the
    attention-matrix form of the readout (App. G.1), written out here in
    numpy.

A companion inflated by any factor, or missing a decay factor, fails at least
one of these (checked by tests/test_oracle_mutants.py).
"""
import numpy as np
import pytest

import oracle
from paper_2402_09900_amd import tapes

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

RTOL = 1e-13


def _flags(rng, B, T, max_len=40):
    return np.stack([tapes.flags_from_lengths(rng.integers(1, max_len, size=T), T) for _ in range(B)])


def _cnormal(rng, shape):
    return rng.standard_normal(shape) + 1j * rng.standard_normal(shape)


def _close(x, ref, rtol=RTOL):
    np.testing.assert_allclose(x, ref, rtol=rtol, atol=0)


# ------------------------------------------------------------ diagonal scan


@pytest.mark.parametrize("invariant", [False, True])
def test_complex_scan_companion_is_the_scan_of_magnitudes(invariant):
    """Complex forward scan (LRU, App. G.3): its companion equals the real
    scan of |a| and |x| (the oracle's primary output, pinned elsewhere)."""
    rng = np.random.default_rng(101)
    B, T, d = 2, 300, 5
    flags = _flags(rng, B, T)
    a = _cnormal(rng, (d,) if invariant else (B, T, d)) * 0.6
    x = _cnormal(rng, (B, T, d))
    h, m = oracle.diag_fwd(a, x, flags)
    hr, _ = oracle.diag_fwd(np.abs(a), np.abs(x), flags)
    _close(m, hr)
    assert np.all(m >= np.abs(h) * (1 - 1e-15))


@pytest.mark.parametrize("invariant", [False, True])
def test_complex_scan_companion_equals_result_on_positive_axis(invariant):
    rng = np.random.default_rng(102)
    B, T, d = 2, 300, 4
    flags = _flags(rng, B, T)
    a = rng.uniform(0.05, 0.99, size=(d,) if invariant else (B, T, d)) + 0j
    x = rng.uniform(0.0, 2.0, size=(B, T, d)) + 0j
    h, m = oracle.diag_fwd(a, x, flags)
    assert np.all(h.imag == 0)
    _close(m, h.real)


def test_real_scan_companion_is_the_scan_of_magnitudes():
    rng = np.random.default_rng(103)
    B, T, d = 2, 300, 5
    flags = _flags(rng, B, T)
    a = rng.uniform(-1.0, 1.0, size=(B, T, d))
    x = rng.standard_normal((B, T, d))
    _, m = oracle.diag_fwd(a, x, flags)
    hr, _ = oracle.diag_fwd(np.abs(a), np.abs(x), flags)
    _close(m, hr)


@pytest.mark.parametrize("cplx", [False, True])
@pytest.mark.parametrize("invariant", [False, True])
def test_reverse_scan_companions_are_reverse_scans_of_magnitudes(cplx, invariant):
    """m_dx is the real reverse scan of |a|, |g|; m_da is that scan's da with
    |h| as the saved state (time-invariant a: summed over tapes and steps)."""
    rng = np.random.default_rng(104 + 2 * cplx + invariant)
    B, T, d = 2, 257, 6
    flags = _flags(rng, B, T)
    ashape = (d,) if invariant else (B, T, d)
    if cplx:
        a = _cnormal(rng, ashape) * 0.6
        h, g = _cnormal(rng, (B, T, d)), _cnormal(rng, (B, T, d))
    else:
        a = rng.uniform(-1.0, 1.0, size=ashape)
        h, g = rng.standard_normal((B, T, d)), rng.standard_normal((B, T, d))
    dx, da, m_dx, m_da = oracle.diag_bwd(a, flags, h, g)
    dxr, dar, _, _ = oracle.diag_bwd(np.abs(a), flags, np.abs(h), np.abs(g))
    _close(m_dx, dxr)
    _close(m_da, dar)
    assert np.all(m_dx >= np.abs(dx) * (1 - 1e-15))
    assert np.all(m_da >= np.abs(da) * (1 - 1e-13))


@pytest.mark.parametrize("cplx", [False, True])
@pytest.mark.parametrize("invariant", [False, True])
def test_reverse_scan_companions_equal_results_on_positive_inputs(cplx, invariant):
    """a in (0, 1), g > 0, h > 0: nothing cancels, so m_dx = dx and m_da = da."""
    rng = np.random.default_rng(108 + 2 * cplx + invariant)
    B, T, d = 2, 257, 6
    flags = _flags(rng, B, T)
    a = rng.uniform(0.05, 0.99, size=(d,) if invariant else (B, T, d))
    h = rng.uniform(0.1, 2.0, size=(B, T, d))
    g = rng.uniform(0.1, 2.0, size=(B, T, d))
    if cplx:
        a, h, g = a + 0j, h + 0j, g + 0j
    dx, da, m_dx, m_da = oracle.diag_bwd(a, flags, h, g)
    _close(m_dx, np.real(dx))
    _close(m_da, np.real(da))


# -------------------------------------------------------- linear attention


def _phi(u):
    return np.where(u > 0, u + 1.0, np.exp(np.minimum(u, 0.0)))


def _dphi(u):
    return np.where(u > 0, 1.0, np.exp(np.minimum(u, 0.0)))


def _episode_mask(flags):
    """M[t, s] = [s <= t and s, t in the same episode] (App. G.1 with resets)."""
    ep = oracle.episode_idx(flags)
    T = len(flags)
    idx = np.arange(T)
    return (idx[None, :] <= idx[:, None]) & (ep[None, :] == ep[:, None])


def _linattn_case(seed, T=96, H=2, dk=5, dv=7):
    rng = np.random.default_rng(seed)
    flags = tapes.flags_from_lengths(rng.integers(1, 30, size=T), T)
    q = rng.standard_normal((T, H, dk))
    k = rng.standard_normal((T, H, dk))
    v = rng.standard_normal((T, H, dv))
    g = rng.standard_normal((T, H, dv))
    return flags, q, k, v, g


def test_linattn_companion_is_the_readout_of_magnitudes():
    """m(q, k, v) = out(q, k, |v|): the weights phi(q).phi(k) are positive."""
    flags, q, k, v, _ = _linattn_case(111)
    out, m = oracle.linattn(q, k, v, flags)
    out_abs, _ = oracle.linattn(q, k, np.abs(v), flags)
    _close(m, out_abs)
    v_pos = np.abs(v) + 0.1
    out_p, m_p = oracle.linattn(q, k, v_pos, flags)
    _close(m_p, out_p)
    assert np.all(m >= np.abs(out) * (1 - 1e-13))


def _linattn_grad_abs_terms(flags, q, k, v, g):
    """Term-by-term absolute sums of the readout gradient in its
    attention-matrix form, per head.  With Q = phi(q), K = phi(k),
    W_ts = M_ts Q_t.K_s, den_t = sum_s W_ts, z_t = sum_s M_ts K_s and
    C_ts = sum_j |g_tj| |v_sj|:
        dq_ti = phi'(q_ti) [sum_s M_ts K_si (sum_j g_tj v_sj) / den_t
                            - z_ti sum_s W_ts (sum_j g_tj v_sj) / den_t^2]
        dk_ti = phi'(k_ti) sum_s M_st Q_si [(sum_j g_sj v_tj) / den_s + dden_s]
        dv_tj = sum_s W_st g_sj / den_s
    and the companions replace every product by its absolute value."""
    T, H, dk = q.shape
    M = _episode_mask(flags).astype(np.float64)
    mq, mk, mv = np.empty_like(q), np.empty_like(k), np.empty_like(v)
    for h in range(H):
        Q, K = _phi(q[:, h]), _phi(k[:, h])
        W = (Q @ K.T) * M
        den = W.sum(axis=1)
        z = M @ K
        C = np.abs(g[:, h]) @ np.abs(v[:, h]).T
        mdden = (W * C).sum(axis=1) / den ** 2
        mq[:, h] = _dphi(q[:, h]) * (((M * C) @ K) / den[:, None] + z * mdden[:, None])
        mk[:, h] = _dphi(k[:, h]) * ((M * C).T @ (Q / den[:, None]) + M.T @ (Q * mdden[:, None]))
        mv[:, h] = W.T @ (np.abs(g[:, h]) / den[:, None])
    return mq, mk, mv


@pytest.mark.parametrize("dk,dv", [(5, 7), (8, 3)])
def test_linattn_grad_companions_are_absolute_term_sums(dk, dv):
    flags, q, k, v, g = _linattn_case(112 + dk, dk=dk, dv=dv)
    dq, dkk, dvv, m_dq, m_dk, m_dv = oracle.linattn_bwd(q, k, v, flags, g)
    mq, mk, mv = _linattn_grad_abs_terms(flags, q, k, v, g)
    _close(m_dq, mq, 1e-12)
    _close(m_dk, mk, 1e-12)
    _close(m_dv, mv, 1e-12)
    assert np.all(m_dq >= np.abs(dq) * (1 - 1e-12))
    assert np.all(m_dk >= np.abs(dkk) * (1 - 1e-12))
    assert np.all(m_dv >= np.abs(dvv) * (1 - 1e-12))


def test_linattn_grad_value_companion_equals_result_for_positive_upstream():
    """dv does not depend on v, and with g > 0 nothing cancels: m_dv = dv;
    for any g, m_dv(g) = dv(|g|)."""
    flags, q, k, v, g = _linattn_case(115)
    _, _, dvv, _, _, m_dv = oracle.linattn_bwd(q, k, v, flags, np.abs(g) + 0.05)
    _close(m_dv, dvv)
    _, _, dv_abs, _, _, _ = oracle.linattn_bwd(q, k, v, flags, np.abs(g))
    _, _, _, _, _, m_dv_g = oracle.linattn_bwd(q, k, v, flags, g)
    _close(m_dv_g, dv_abs)


# ------------------------------------------------------ return and advantage


def test_return_companion_is_the_return_of_magnitudes():
    rng = np.random.default_rng(121)
    B, T = 3, 400
    flags = _flags(rng, B, T, 80)
    r = rng.standard_normal((B, T))
    G, m = oracle.discounted_return(r, flags, 0.97)
    Gabs, _ = oracle.discounted_return(np.abs(r), flags, 0.97)
    _close(m, Gabs)
    assert np.all(m >= np.abs(G) * (1 - 1e-13))


def _next_in_episode(v, flags):
    """V(s_{t+1}) inside an episode, 0 at its last step (the default V(s'))."""
    B, T = v.shape
    out = np.zeros_like(v)
    for b in range(B):
        for t in range(T - 1):
            if flags[b, t + 1] == 0:
                out[b, t] = v[b, t + 1]
    return out


@pytest.mark.parametrize("with_vn", [False, True])
@pytest.mark.parametrize("with_done", [False, True])
def test_gae_companions_are_advantages_of_magnitudes(with_vn, with_done):
    """The TD error's companion is |r| + gamma [not done] |V(s')| + |V(s)|:
    the advantage of (|r|, -|V(s)|, |V(s')|), whose terms are all >= 0."""
    rng = np.random.default_rng(122 + 2 * with_vn + with_done)
    B, T = 2, 300
    flags = _flags(rng, B, T, 60)
    flags[:, 0] = 1
    r, v = rng.standard_normal((B, T)), rng.standard_normal((B, T))
    vn = rng.standard_normal((B, T)) if with_vn else None
    done = (rng.random((B, T)) < 0.2).astype(np.uint8) if with_done else None
    adv, target, m_adv, m_target = oracle.gae(r, v, flags, 0.99, 0.95, vn=vn, done=done)
    vn_abs = np.abs(vn) if with_vn else np.abs(_next_in_episode(v, flags))
    ref, _, _, _ = oracle.gae(np.abs(r), -np.abs(v), flags, 0.99, 0.95, vn=vn_abs, done=done)
    _close(m_adv, ref)
    _close(m_target - np.abs(v), ref)
    assert np.all(m_adv >= np.abs(adv) * (1 - 1e-13))
    assert np.all(m_target >= np.abs(target) * (1 - 1e-13))


@pytest.mark.parametrize("with_vn", [False, True])
def test_gae_companions_equal_results_without_cancellation(with_vn):
    """V(s) = 0 and r, V(s') >= 0: every TD error is a sum of non-negative
    terms, so m_adv = adv and m_target = target."""
    rng = np.random.default_rng(126 + with_vn)
    B, T = 2, 300
    flags = _flags(rng, B, T, 60)
    r = rng.uniform(0.0, 2.0, size=(B, T))
    v = np.zeros((B, T))
    vn = rng.uniform(0.0, 2.0, size=(B, T)) if with_vn else None
    done = (rng.random((B, T)) < 0.2).astype(np.uint8)
    adv, target, m_adv, m_target = oracle.gae(r, v, flags, 0.99, 0.95, vn=vn, done=done)
    _close(m_adv, adv)
    _close(m_target, target)


# ------------------------------------------------------------------- FFM


def _ffm_case(seed, B=2, T=200, m=3, c=4):
    rng = np.random.default_rng(seed)
    flags = _flags(rng, B, T, 50)
    alpha = rng.uniform(0.01, 0.7, size=m) * rng.choice([-1.0, 1.0], size=m)
    omega = rng.uniform(-np.pi, np.pi, size=c)
    x = rng.standard_normal((B, T, m))
    return flags, alpha, omega, x


def _ffm_as_real_scan(alpha, c, x):
    """The FFM magnitudes as a real diagonal scan over d = m c features:
    a_jk = exp(-|alpha_j|) = |gamma_jk|, input |x_j| broadcast over k."""
    a = np.repeat(np.exp(-np.abs(alpha)), c)
    B, T, m = x.shape
    xr = np.repeat(np.abs(x), c, axis=2).reshape(B, T, m * c)
    return a, xr


def test_ffm_companion_is_the_real_scan_of_magnitudes():
    """|gamma| = exp(-|alpha|) for every column (App. G.4), so the companion
    is the real diagonal scan of (exp(-|alpha|), |x|)."""
    flags, alpha, omega, x = _ffm_case(131)
    c = len(omega)
    S, m = oracle.ffm(alpha, omega, x, flags)
    a, xr = _ffm_as_real_scan(alpha, c, x)
    hr, _ = oracle.diag_fwd(a, xr, flags)
    _close(m.reshape(hr.shape), hr)
    assert np.all(m >= np.abs(S) * (1 - 1e-13))


def test_ffm_companion_equals_result_without_rotation():
    flags, alpha, omega, x = _ffm_case(132)
    S, m = oracle.ffm(alpha, np.zeros_like(omega), np.abs(x), flags)
    assert np.all(S.imag == 0)
    _close(m, S.real)


def test_ffm_grad_companions_are_reverse_scans_of_magnitudes():
    """m_dx sums over k the real reverse scan of (|gamma|, |G|); the
    parameter companions weight that scan's da (with |S| as the saved
    state) by |gamma|: m_dalpha_j = sum_k |gamma_jk| da_jk, m_domega_k =
    sum_j |gamma_jk| da_jk."""
    flags, alpha, omega, x = _ffm_case(133)
    rng = np.random.default_rng(134)
    B, T, m = x.shape
    c = len(omega)
    S, _ = oracle.ffm(alpha, omega, x, flags)
    G = _cnormal(rng, S.shape)
    dx, dal, dom, m_dx, m_dal, m_dom = oracle.ffm_bwd(alpha, omega, flags, S, G)
    a = np.repeat(np.exp(-np.abs(alpha)), c)
    dxr, dar, _, _ = oracle.diag_bwd(a, flags, np.abs(S).reshape(B, T, m * c), np.abs(G).reshape(B, T, m * c))
    _close(m_dx, dxr.reshape(B, T, m, c).sum(axis=3))
    w = (a * dar).reshape(m, c)
    _close(m_dal, w.sum(axis=1))
    _close(m_dom, w.sum(axis=0))
    assert np.all(m_dx >= np.abs(dx) * (1 - 1e-13))
    assert np.all(m_dal >= np.abs(dal) * (1 - 1e-13))
    assert np.all(m_dom >= np.abs(dom) * (1 - 1e-13))


def test_ffm_grad_companions_equal_results_without_cancellation():
    """omega = 0, x > 0 (so S > 0), alpha > 0: with a real positive G every
    term of dx and of -dalpha is positive; with G = i |G| every term of
    domega is."""
    flags, alpha, omega, x = _ffm_case(135)
    alpha, omega, x = np.abs(alpha), np.zeros_like(omega), np.abs(x) + 0.05
    S, _ = oracle.ffm(alpha, omega, x, flags)
    rng = np.random.default_rng(136)
    G = rng.uniform(0.1, 1.0, size=S.shape) + 0j
    dx, dal, _, m_dx, m_dal, _ = oracle.ffm_bwd(alpha, omega, flags, S, G)
    _close(m_dx, dx)
    _close(m_dal, -dal)
    _, _, dom, _, _, m_dom = oracle.ffm_bwd(alpha, omega, flags, S, 1j * G.real)
    _close(m_dom, dom)
