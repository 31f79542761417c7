"""The oracle's pins must fail on a wrong oracle.

Each case below plants one plausible mistake in a copy of oracle.c (a
dropped term, a wrong sign, index or flag, a missing conjugate or absolute
value, a transposed operand, an inflated or undamped magnitude companion),
compiles the copy with gcc, routes the oracle wrappers through it and runs
every pin of tests/test_oracle_pins.py and tests/test_oracle_companions.py
until one fails.  A case passes when some pin fails: a mistake that no pin
notices would fail it.  Everything here runs on the CPU against the oracle
only.

Each planted pattern is matched against the current oracle.c with its exact
number of occurrences, so an edit of the oracle that moves a pattern makes
the case error out instead of silently testing nothing.
"""
import inspect
import itertools

import pytest

import oracle
import test_oracle_companions as companions
import test_oracle_pins as pins

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

# (id, pattern, replacement, occurrences of the pattern, which occurrence to alter)
MUTANTS = [
    # ---------------------------------------------------- primary outputs
    ("episode_idx_starts_at_one", "int32_t c = -1;", "int32_t c = 0;", 1, 0),
    ("step0_not_forced_begin", "return t == 0 || start[b * T + t] != 0;", "return start[b * T + t] != 0;", 1, 0),
    ("fwd_real_sign_of_x", "h[row + j] = at[j] * h[row - d + j] + x[row + j];",
     "h[row + j] = at[j] * h[row - d + j] - x[row + j];", 2, 0),
    ("fwd_real_dropped_a", "h[row + j] = at[j] * h[row - d + j] + x[row + j];",
     "h[row + j] = h[row - d + j] + x[row + j];", 2, 0),
    ("fwd_complex_dropped_a", "h[row + j] = at[j] * h[row - d + j] + x[row + j];",
     "h[row + j] = h[row - d + j] + x[row + j];", 2, 1),
    ("fwd_complex_conj_a", "h[row + j] = at[j] * h[row - d + j] + x[row + j];",
     "h[row + j] = conj(at[j]) * h[row - d + j] + x[row + j];", 2, 1),
    ("bwd_complex_missing_conj", "lam[j] = g[row + j] + (flows ? conj(anext[j]) * lam[j] : 0.0);",
     "lam[j] = g[row + j] + (flows ? anext[j] * lam[j] : 0.0);", 1, 0),
    ("bwd_real_a_of_step_t", "lam[j] = g[row + j] + (flows ? anext[j] * lam[j] : 0.0);",
     "lam[j] = g[row + j] + (flows ? (a_stride_t ? a + row : a)[j] * lam[j] : 0.0);", 1, 0),
    ("bwd_real_reset_off_by_one", "const int flows = (t + 1 < T) && !is_begin(start, T, b, t + 1);",
     "const int flows = (t + 1 < T) && !is_begin(start, T, b, t);", 2, 0),
    ("bwd_complex_reset_off_by_one", "const int flows = (t + 1 < T) && !is_begin(start, T, b, t + 1);",
     "const int flows = (t + 1 < T) && !is_begin(start, T, b, t);", 2, 1),
    ("bwd_real_da_uses_h_t", "const double dat = begin ? 0.0 : lam[j] * h[row - d + j];",
     "const double dat = begin ? 0.0 : lam[j] * h[row + j];", 1, 0),
    ("bwd_complex_da_missing_conj", "const double complex dat = begin ? 0.0 : lam[j] * conj(h[row - d + j]);",
     "const double complex dat = begin ? 0.0 : lam[j] * h[row - d + j];", 1, 0),
    ("phi_without_one", "double oracle_phi(double u) { return u > 0.0 ? u + 1.0 : exp(u); }",
     "double oracle_phi(double u) { return u > 0.0 ? u : exp(u); }", 1, 0),
    ("linattn_den_uses_k", "for (int64_t i = 0; i < dk; ++i) den += qf[i] * z[i];",
     "for (int64_t i = 0; i < dk; ++i) den += kf[i] * z[i];", 1, 0),
    ("linattn_readout_transposed", "num += qf[i] * S[i * dv + j];", "num += qf[i] * S[j * dk + i];", 1, 0),
    ("linattn_z_not_reset", "memset(z, 0, (size_t)dk * sizeof(double));", "(void)0;", 1, 0),
    ("linattn_state_uses_phi_q", "S[i * dv + j] += kf[i] * vt[j];", "S[i * dv + j] += qf[i] * vt[j];", 1, 0),
    ("linattn_grad_phi_prime_one", "static double phi_prime(double u) { return u > 0.0 ? 1.0 : exp(u); }",
     "static double phi_prime(double u) { return u > 0.0 ? 1.0 : 1.0; }", 1, 0),
    ("linattn_grad_dden_sign", "dden[t] = -go / den;", "dden[t] = go / den;", 1, 0),
    ("linattn_grad_reverse_reset_off_by_one", "const int last = (t == T - 1) || is_begin(start, T, 0, t + 1);",
     "const int last = (t == T - 1) || is_begin(start, T, 0, t);", 1, 0),
    ("linattn_grad_dq_dropped_state_term", "a += S[i * dv + j] * dnum[t * dv + j];", "(void)0;", 1, 0),
    ("linattn_grad_dk_uses_k", "a += U[i * dv + j] * vt[j];", "a += U[i * dv + j] * vt[j] * Kf[i];", 1, 0),
    ("linattn_grad_dv_uses_q", "a += U[i * dv + j] * Kf[i];", "a += U[i * dv + j] * Qf[i];", 1, 0),
    ("linattn_grad_w_dropped", "w[i] += dden[t] * Qf[i];", "(void)0;", 1, 0),
    ("return_dropped_gamma", "g = last ? rb[t] : rb[t] + gamma * g;", "g = last ? rb[t] : rb[t] + g;", 1, 0),
    ("return_episode_end_off_by_one", "const int last = (t == T - 1) || is_begin(start, T, b, t + 1);",
     "const int last = (t == T - 1) || is_begin(start, T, b, t);", 2, 0),
    ("gae_episode_end_off_by_one", "const int last = (t == T - 1) || is_begin(start, T, b, t + 1);",
     "const int last = (t == T - 1) || is_begin(start, T, b, t);", 2, 1),
    ("gae_done_ignored", "const double delta = r[i] + gamma * keep * next_v - v[i];",
     "const double delta = r[i] + gamma * next_v - v[i];", 1, 0),
    ("gae_td_without_gamma", "const double delta = r[i] + gamma * keep * next_v - v[i];",
     "const double delta = r[i] + keep * next_v - v[i];", 1, 0),
    ("gae_decay_gamma_only", "A = last ? delta : delta + gl * A;", "A = last ? delta : delta + gamma * A;", 1, 0),
    ("gae_target_sign", "if (target) target[i] = A + v[i];", "if (target) target[i] = A - v[i];", 1, 0),
    ("ffm_rotation_sign", "const double complex g = mag * cexp(I * omega[k]);",
     "const double complex g = mag * cexp(-I * omega[k]);", 2, 0),
    ("ffm_decay_without_abs", "const double mag = exp(-fabs(alpha[j]));", "const double mag = exp(-alpha[j]);", 2, 0),
    ("ffm_grad_rotation_sign", "const double complex g = mag * cexp(I * omega[k]);",
     "const double complex g = mag * cexp(-I * omega[k]);", 2, 1),
    ("ffm_grad_decay_without_abs", "const double mag = exp(-fabs(alpha[j]));", "const double mag = exp(-alpha[j]);",
     2, 1),
    ("ffm_grad_missing_conj", "lam = cont ? gt + conj(g) * lam : gt;", "lam = cont ? gt + g * lam : gt;", 1, 0),
    ("ffm_grad_dalpha_sign", "if (dalpha) dalpha[j] += -sgn * creal(w);", "if (dalpha) dalpha[j] += sgn * creal(w);",
     1, 0),
    ("ffm_grad_domega_sign", "if (domega) domega[k] += cimag(w);", "if (domega) domega[k] += -cimag(w);", 1, 0),
    ("ffm_grad_param_missing_conj", "const double complex w = conj(g) * da;", "const double complex w = g * da;", 1, 0),
    ("ffm_grad_da_missing_conj", "da += lam * conj(sp);", "da += lam * sp;", 1, 0),
    ("ffm_grad_dx_imaginary", "dx[(b * T + t) * m + j] += creal(lam);", "dx[(b * T + t) * m + j] += cimag(lam);",
     1, 0),
    ("tbb_offset_dropped", "if (start[t] != 0) out[k++] = offset + t;", "if (start[t] != 0) out[k++] = t;", 1, 0),
    ("tbb_episode_one_short", "const int64_t hi = i + 1 < n_I ? begins[i + 1] : n_D;",
     "const int64_t hi = i + 1 < n_I ? begins[i + 1] - 1 : n_D;", 1, 0),
    ("tbb_begin_flag_at_last_row", "out_start[len] = r == lo ? 1 : 0;", "out_start[len] = r == hi - 1 ? 1 : 0;", 1, 0),
    # ------------------------------------------ magnitude companions
    ("m_fwd_real_x2", "m[row + j] = fabs(at[j]) * m[row - d + j] + fabs(x[row + j]);",
     "m[row + j] = 2.0 * (fabs(at[j]) * m[row - d + j] + fabs(x[row + j]));", 1, 0),
    ("m_fwd_real_no_decay", "m[row + j] = fabs(at[j]) * m[row - d + j] + fabs(x[row + j]);",
     "m[row + j] = m[row - d + j] + fabs(x[row + j]);", 1, 0),
    ("m_fwd_complex_x2", "m[row + j] = cabs(at[j]) * m[row - d + j] + cabs(x[row + j]);",
     "m[row + j] = 2.0 * (cabs(at[j]) * m[row - d + j] + cabs(x[row + j]));", 1, 0),
    ("m_fwd_complex_no_decay", "m[row + j] = cabs(at[j]) * m[row - d + j] + cabs(x[row + j]);",
     "m[row + j] = m[row - d + j] + cabs(x[row + j]);", 1, 0),
    ("m_dx_real_x2", "mlam[j] = fabs(g[row + j]) + (flows ? fabs(anext[j]) * mlam[j] : 0.0);",
     "mlam[j] = 2.0 * (fabs(g[row + j]) + (flows ? fabs(anext[j]) * mlam[j] : 0.0));", 1, 0),
    ("m_dx_real_no_decay", "mlam[j] = fabs(g[row + j]) + (flows ? fabs(anext[j]) * mlam[j] : 0.0);",
     "mlam[j] = fabs(g[row + j]) + (flows ? mlam[j] : 0.0);", 1, 0),
    ("m_da_real_x2", "const double mdat = begin ? 0.0 : mlam[j] * fabs(h[row - d + j]);",
     "const double mdat = begin ? 0.0 : 2.0 * mlam[j] * fabs(h[row - d + j]);", 1, 0),
    ("m_dx_complex_x2", "mlam[j] = cabs(g[row + j]) + (flows ? cabs(anext[j]) * mlam[j] : 0.0);",
     "mlam[j] = 2.0 * (cabs(g[row + j]) + (flows ? cabs(anext[j]) * mlam[j] : 0.0));", 1, 0),
    ("m_dx_complex_no_decay", "mlam[j] = cabs(g[row + j]) + (flows ? cabs(anext[j]) * mlam[j] : 0.0);",
     "mlam[j] = cabs(g[row + j]) + (flows ? mlam[j] : 0.0);", 1, 0),
    ("m_da_complex_x2", "const double mdat = begin ? 0.0 : mlam[j] * cabs(h[row - d + j]);",
     "const double mdat = begin ? 0.0 : 2.0 * mlam[j] * cabs(h[row - d + j]);", 1, 0),
    ("m_linattn_x2", "if (mt) mt[j] = numabs / den;", "if (mt) mt[j] = 2.0 * numabs / den;", 1, 0),
    ("m_linattn_missing_abs", "Sabs[i * dv + j] += kf[i] * fabs(vt[j]);", "Sabs[i * dv + j] += kf[i] * vt[j];", 1, 0),
    ("m_dq_x2", "if (m_dq) m_dq[(t * H + hh) * dk + i] = am * d;", "if (m_dq) m_dq[(t * H + hh) * dk + i] = 2.0 * am * d;",
     1, 0),
    ("m_dk_x2", "if (m_dk) m_dk[(t * H + hh) * dk + i] = am * d;", "if (m_dk) m_dk[(t * H + hh) * dk + i] = 2.0 * am * d;",
     1, 0),
    ("m_dv_x2", "if (m_dv) m_dv[(t * H + hh) * dv + j] = am;", "if (m_dv) m_dv[(t * H + hh) * dv + j] = 2.0 * am;",
     1, 0),
    ("m_dden_x2", "mdden[t] = gm / den;", "mdden[t] = 2.0 * gm / den;", 1, 0),
    ("m_dnum_x2", "mdnum[t * dv + j] = fabs(gt[j]) / den;", "mdnum[t * dv + j] = 2.0 * fabs(gt[j]) / den;", 1, 0),
    ("m_dk_w_x2", "wa[i] += mdden[t] * Qf[i];", "wa[i] += 2.0 * mdden[t] * Qf[i];", 1, 0),
    ("m_dk_missing_abs_v", "am += Ua[i * dv + j] * fabs(vt[j]);", "am += Ua[i * dv + j] * vt[j];", 1, 0),
    ("m_return_x2", "ga = last ? fabs(rb[t]) : fabs(rb[t]) + gamma * ga;",
     "ga = 2.0 * (last ? fabs(rb[t]) : fabs(rb[t]) + gamma * ga);", 1, 0),
    ("m_return_no_decay", "ga = last ? fabs(rb[t]) : fabs(rb[t]) + gamma * ga;",
     "ga = last ? fabs(rb[t]) : fabs(rb[t]) + ga;", 1, 0),
    ("m_adv_x2", "Am = last ? dmag : dmag + gl * Am;", "Am = 2.0 * (last ? dmag : dmag + gl * Am);", 1, 0),
    ("m_adv_no_decay", "Am = last ? dmag : dmag + gl * Am;", "Am = last ? dmag : dmag + Am;", 1, 0),
    ("m_target_x2", "if (m_target) m_target[i] = Am + fabs(v[i]);",
     "if (m_target) m_target[i] = 2.0 * (Am + fabs(v[i]));", 1, 0),
    ("m_td_error_dropped_value", "const double dmag = fabs(r[i]) + gamma * keep * fabs(next_v) + fabs(v[i]);",
     "const double dmag = fabs(r[i]) + gamma * keep * fabs(next_v);", 1, 0),
    ("m_ffm_x2", "sm = sm * mag + fabs(xv);", "sm = 2.0 * (sm * mag + fabs(xv));", 1, 0),
    ("m_ffm_no_decay", "sm = sm * mag + fabs(xv);", "sm = sm + fabs(xv);", 1, 0),
    ("m_ffm_dx_x2", "ml = cont ? cabs(gt) + mag * ml : cabs(gt);", "ml = 2.0 * (cont ? cabs(gt) + mag * ml : cabs(gt));",
     1, 0),
    ("m_ffm_dx_no_decay", "ml = cont ? cabs(gt) + mag * ml : cabs(gt);", "ml = cont ? cabs(gt) + ml : cabs(gt);", 1, 0),
    ("m_ffm_dx_sum_x2", "if (m_dx) m_dx[(b * T + t) * m + j] += ml;", "if (m_dx) m_dx[(b * T + t) * m + j] += 2.0 * ml;",
     1, 0),
    ("m_dalpha_x2", "if (m_dalpha) m_dalpha[j] += mag * mda;", "if (m_dalpha) m_dalpha[j] += 2.0 * mag * mda;", 1, 0),
    ("m_dalpha_no_decay", "if (m_dalpha) m_dalpha[j] += mag * mda;", "if (m_dalpha) m_dalpha[j] += mda;", 1, 0),
    ("m_domega_x2", "if (m_domega) m_domega[k] += mag * mda;", "if (m_domega) m_domega[k] += 2.0 * mag * mda;", 1, 0),
    ("m_domega_no_decay", "if (m_domega) m_domega[k] += mag * mda;", "if (m_domega) m_domega[k] += mda;", 1, 0),
    ("m_ffm_da_x2", "mda += ml * cabs(sp);", "mda += 2.0 * ml * cabs(sp);", 1, 0),
]


def _expand(fn):
    """Every parameter combination of a pytest test function, as kwargs."""
    grids = []
    for mark in getattr(fn, "pytestmark", []):
        if mark.name != "parametrize":
            continue
        names, values = mark.args[0], mark.args[1]
        names = [n.strip() for n in names.split(",")] if isinstance(names, str) else list(names)
        rows = [v if len(names) > 1 else (v,) for v in values]
        grids.append([dict(zip(names, row)) for row in rows])
    if not grids:
        return [{}]
    out = []
    for combo in itertools.product(*grids):
        kw = {}
        for part in combo:
            kw.update(part)
        out.append(kw)
    return out


def _pins():
    cases = []
    for mod in (companions, pins):
        for name, fn in inspect.getmembers(mod, inspect.isfunction):
            if name.startswith("test_") and fn.__module__ == mod.__name__:
                for kw in _expand(fn):
                    cases.append(("%s.%s%s" % (mod.__name__, name, kw or ""), fn, kw))
    return cases


def _plant(src, pattern, replacement, count, which):
    found = src.count(pattern)
    assert found == count, "pattern occurs %d times in oracle.c, expected %d: %r" % (found, count, pattern)
    pos = -1
    for _ in range(which + 1):
        pos = src.index(pattern, pos + 1)
    return src[:pos] + replacement + src[pos + len(pattern):]


@pytest.mark.parametrize("mid,pattern,replacement,count,which", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_fail_on_planted_mistake(mid, pattern, replacement, count, which, tmp_path):
    src = _plant(oracle.source(), pattern, replacement, count, which)
    with oracle.variant(src, str(tmp_path)):
        for label, fn, kw in _pins():
            try:
                fn(**kw)
            except AssertionError:
                return                  # a pin noticed the mistake
    pytest.fail("no pin fails when oracle.c has the mistake %r" % mid)


def test_unaltered_oracle_passes_every_pin(tmp_path):
    """The harness itself: the unaltered source, compiled the same way,
    passes every pin (so a failure above is the planted mistake's)."""
    with oracle.variant(oracle.source(), str(tmp_path)):
        for label, fn, kw in _pins():
            fn(**kw)
