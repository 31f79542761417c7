/*
 * oracle.c -- fp64 sequential reference for the resettable memoroid scan.
 * TEST INFRASTRUCTURE ONLY: see oracle.h.  Built with gcc as a plain shared
 * object; no code here is shared with the HIP library.
 *
 * Every loop runs the recurrence step by step in tape order, exactly as the
 * memoroid definition of Section 4 states it (h_t = e_I . f(P_0) . ... . f(P_t)),
 * with the resettable transform of the Section 4 reset theorem taking the form
 * "at a begin step the state restarts from the identity".
 */
#include "oracle.h"

#include <complex.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

/* t = 0 of every tape is a begin step: the scan starts from g_I = (e_I, 0). */
static int is_begin(const uint8_t* start, int64_t T, int64_t b, int64_t t) {
    return t == 0 || start[b * T + t] != 0;
}

void oracle_episode_idx(const uint8_t* start, int64_t B, int64_t T, int32_t* idx) {
    for (int64_t b = 0; b < B; ++b) {
        int32_t c = -1;
        for (int64_t t = 0; t < T; ++t) {
            if (is_begin(start, T, b, t)) c += 1;
            idx[b * T + t] = c;
        }
    }
}

/* ---------------------------------------------------------------- diag fwd */

void oracle_diag_fwd(const double* a, int64_t a_stride_t, const double* x,
                     const uint8_t* start, int64_t B, int64_t T, int64_t d,
                     double* h, double* m) {
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t t = 0; t < T; ++t) {
            const int64_t row = (b * T + t) * d;
            const double* at = a_stride_t ? a + row : a;
            const int begin = is_begin(start, T, b, t);
            for (int64_t j = 0; j < d; ++j) {
                if (begin) {
                    h[row + j] = x[row + j];
                    if (m) m[row + j] = fabs(x[row + j]);
                } else {
                    h[row + j] = at[j] * h[row - d + j] + x[row + j];
                    if (m) m[row + j] = fabs(at[j]) * m[row - d + j] + fabs(x[row + j]);
                }
            }
        }
    }
}

void oracle_diag_fwd_c(const double* a_, int64_t a_stride_t, const double* x_,
                       const uint8_t* start, int64_t B, int64_t T, int64_t d,
                       double* h_, double* m) {
    const double complex* a = (const double complex*)a_;
    const double complex* x = (const double complex*)x_;
    double complex* h = (double complex*)h_;
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t t = 0; t < T; ++t) {
            const int64_t row = (b * T + t) * d;
            const double complex* at = a_stride_t ? a + row : a;
            const int begin = is_begin(start, T, b, t);
            for (int64_t j = 0; j < d; ++j) {
                if (begin) {
                    h[row + j] = x[row + j];
                    if (m) m[row + j] = cabs(x[row + j]);
                } else {
                    h[row + j] = at[j] * h[row - d + j] + x[row + j];
                    if (m) m[row + j] = cabs(at[j]) * m[row - d + j] + cabs(x[row + j]);
                }
            }
        }
    }
}

/* ---------------------------------------------------------------- diag bwd */

void oracle_diag_bwd(const double* a, int64_t a_stride_t, const uint8_t* start,
                     const double* h, const double* g,
                     int64_t B, int64_t T, int64_t d,
                     double* dx, double* da, double* m_dx, double* m_da) {
    double* lam = (double*)calloc((size_t)(d > 0 ? d : 1), sizeof(double));
    double* mlam = (double*)calloc((size_t)(d > 0 ? d : 1), sizeof(double));
    if (da && !a_stride_t) memset(da, 0, (size_t)d * sizeof(double));
    if (m_da && !a_stride_t) memset(m_da, 0, (size_t)d * sizeof(double));
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t t = T - 1; t >= 0; --t) {
            const int64_t row = (b * T + t) * d;
            /* the state of step t flows into step t+1 unless t+1 begins a new
               episode or lies past the end of the tape */
            const int flows = (t + 1 < T) && !is_begin(start, T, b, t + 1);
            const double* anext = flows ? (a_stride_t ? a + row + d : a) : NULL;
            const int begin = is_begin(start, T, b, t);
            for (int64_t j = 0; j < d; ++j) {
                lam[j] = g[row + j] + (flows ? anext[j] * lam[j] : 0.0);
                mlam[j] = fabs(g[row + j]) + (flows ? fabs(anext[j]) * mlam[j] : 0.0);
                dx[row + j] = lam[j];
                if (m_dx) m_dx[row + j] = mlam[j];
                const double dat = begin ? 0.0 : lam[j] * h[row - d + j];
                const double mdat = begin ? 0.0 : mlam[j] * fabs(h[row - d + j]);
                if (da) {
                    if (a_stride_t) da[row + j] = dat; else da[j] += dat;
                }
                if (m_da) {
                    if (a_stride_t) m_da[row + j] = mdat; else m_da[j] += mdat;
                }
            }
        }
    }
    free(lam);
    free(mlam);
}

void oracle_diag_bwd_c(const double* a_, int64_t a_stride_t, const uint8_t* start,
                       const double* h_, const double* g_,
                       int64_t B, int64_t T, int64_t d,
                       double* dx_, double* da_, double* m_dx, double* m_da) {
    const double complex* a = (const double complex*)a_;
    const double complex* h = (const double complex*)h_;
    const double complex* g = (const double complex*)g_;
    double complex* dx = (double complex*)dx_;
    double complex* da = (double complex*)da_;
    double complex* lam = (double complex*)calloc((size_t)(d > 0 ? d : 1), sizeof(double complex));
    double* mlam = (double*)calloc((size_t)(d > 0 ? d : 1), sizeof(double));
    if (da && !a_stride_t) memset(da, 0, (size_t)d * sizeof(double complex));
    if (m_da && !a_stride_t) memset(m_da, 0, (size_t)d * sizeof(double));
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t t = T - 1; t >= 0; --t) {
            const int64_t row = (b * T + t) * d;
            const int flows = (t + 1 < T) && !is_begin(start, T, b, t + 1);
            const double complex* anext = flows ? (a_stride_t ? a + row + d : a) : NULL;
            const int begin = is_begin(start, T, b, t);
            for (int64_t j = 0; j < d; ++j) {
                lam[j] = g[row + j] + (flows ? conj(anext[j]) * lam[j] : 0.0);
                mlam[j] = cabs(g[row + j]) + (flows ? cabs(anext[j]) * mlam[j] : 0.0);
                dx[row + j] = lam[j];
                if (m_dx) m_dx[row + j] = mlam[j];
                const double complex dat = begin ? 0.0 : lam[j] * conj(h[row - d + j]);
                const double mdat = begin ? 0.0 : mlam[j] * cabs(h[row - d + j]);
                if (da) {
                    if (a_stride_t) da[row + j] = dat; else da[j] += dat;
                }
                if (m_da) {
                    if (a_stride_t) m_da[row + j] = mdat; else m_da[j] += mdat;
                }
            }
        }
    }
    free(lam);
    free(mlam);
}

/* ----------------------------------------------------------- linear attn */

double oracle_phi(double u) { return u > 0.0 ? u + 1.0 : exp(u); }

void oracle_linattn(const double* q, const double* k, const double* v,
                    const uint8_t* start, int64_t T, int64_t H, int64_t dk, int64_t dv,
                    double* out, double* m) {
    double* S = (double*)malloc((size_t)(dk * dv > 0 ? dk * dv : 1) * sizeof(double));
    double* Sabs = (double*)malloc((size_t)(dk * dv > 0 ? dk * dv : 1) * sizeof(double));
    double* z = (double*)malloc((size_t)(dk > 0 ? dk : 1) * sizeof(double));
    double* kf = (double*)malloc((size_t)(dk > 0 ? dk : 1) * sizeof(double));
    double* qf = (double*)malloc((size_t)(dk > 0 ? dk : 1) * sizeof(double));
    for (int64_t hh = 0; hh < H; ++hh) {
        for (int64_t t = 0; t < T; ++t) {
            if (is_begin(start, T, 0, t)) {
                memset(S, 0, (size_t)(dk * dv) * sizeof(double));
                memset(Sabs, 0, (size_t)(dk * dv) * sizeof(double));
                memset(z, 0, (size_t)dk * sizeof(double));
            }
            const double* qt = q + (t * H + hh) * dk;
            const double* kt = k + (t * H + hh) * dk;
            const double* vt = v + (t * H + hh) * dv;
            for (int64_t i = 0; i < dk; ++i) {
                kf[i] = oracle_phi(kt[i]);
                qf[i] = oracle_phi(qt[i]);
            }
            /* X_n = X_{n-1} + phi(k) v^T ;  x_n = x_{n-1} + phi(k) */
            for (int64_t i = 0; i < dk; ++i) {
                z[i] += kf[i];
                for (int64_t j = 0; j < dv; ++j) {
                    S[i * dv + j] += kf[i] * vt[j];
                    Sabs[i * dv + j] += kf[i] * fabs(vt[j]);
                }
            }
            /* readout phi(q)^T S / (phi(q)^T z) */
            double den = 0.0;
            for (int64_t i = 0; i < dk; ++i) den += qf[i] * z[i];
            double* ot = out + (t * H + hh) * dv;
            double* mt = m ? m + (t * H + hh) * dv : NULL;
            for (int64_t j = 0; j < dv; ++j) {
                double num = 0.0, numabs = 0.0;
                for (int64_t i = 0; i < dk; ++i) {
                    num += qf[i] * S[i * dv + j];
                    numabs += qf[i] * Sabs[i * dv + j];
                }
                ot[j] = num / den;
                if (mt) mt[j] = numabs / den;
            }
        }
    }
    free(S);
    free(Sabs);
    free(z);
    free(kf);
    free(qf);
}

/* ----------------------------------------------- linear attention, grad */

static double phi_prime(double u) { return u > 0.0 ? 1.0 : exp(u); }

void oracle_linattn_bwd(const double* q, const double* k, const double* v, const uint8_t* start,
                        const double* g, int64_t T, int64_t H, int64_t dk, int64_t dv,
                        double* dq, double* dk_out, double* dv_out,
                        double* m_dq, double* m_dk, double* m_dv) {
    const size_t nS = (size_t)(dk * dv > 0 ? dk * dv : 1);
    const size_t nk = (size_t)(dk > 0 ? dk : 1), nv = (size_t)(dv > 0 ? dv : 1);
    double* S = (double*)malloc(nS * sizeof(double));
    double* Sa = (double*)malloc(nS * sizeof(double));
    double* z = (double*)malloc(nk * sizeof(double));
    double* U = (double*)malloc(nS * sizeof(double));
    double* Ua = (double*)malloc(nS * sizeof(double));
    double* w = (double*)malloc(nk * sizeof(double));
    double* wa = (double*)malloc(nk * sizeof(double));
    double* Qf = (double*)malloc(nk * sizeof(double));
    double* Kf = (double*)malloc(nk * sizeof(double));
    const size_t steps = (size_t)(T > 0 ? T : 1);
    /* per step of one head: dnum (dv), dden, and their companions */
    double* dnum = (double*)malloc(steps * nv * sizeof(double));
    double* mdnum = (double*)malloc(steps * nv * sizeof(double));
    double* dden = (double*)malloc(steps * sizeof(double));
    double* mdden = (double*)malloc(steps * sizeof(double));
    for (int64_t hh = 0; hh < H; ++hh) {
        /* forward in time: the states (S, z), the readout, dnum, dden, dq */
        for (int64_t t = 0; t < T; ++t) {
            if (is_begin(start, T, 0, t)) {
                memset(S, 0, nS * sizeof(double));
                memset(Sa, 0, nS * sizeof(double));
                memset(z, 0, nk * sizeof(double));
            }
            const double* qt = q + (t * H + hh) * dk;
            const double* kt = k + (t * H + hh) * dk;
            const double* vt = v + (t * H + hh) * dv;
            const double* gt = g + (t * H + hh) * dv;
            for (int64_t i = 0; i < dk; ++i) {
                Qf[i] = oracle_phi(qt[i]);
                Kf[i] = oracle_phi(kt[i]);
            }
            for (int64_t i = 0; i < dk; ++i) {
                z[i] += Kf[i];
                for (int64_t j = 0; j < dv; ++j) {
                    S[i * dv + j] += Kf[i] * vt[j];
                    Sa[i * dv + j] += Kf[i] * fabs(vt[j]);
                }
            }
            double den = 0.0;
            for (int64_t i = 0; i < dk; ++i) den += Qf[i] * z[i];
            double go = 0.0, gm = 0.0;
            for (int64_t j = 0; j < dv; ++j) {
                double num = 0.0, numa = 0.0;
                for (int64_t i = 0; i < dk; ++i) {
                    num += Qf[i] * S[i * dv + j];
                    numa += Qf[i] * Sa[i * dv + j];
                }
                go += gt[j] * (num / den);
                gm += fabs(gt[j]) * (numa / den);
                dnum[t * dv + j] = gt[j] / den;
                mdnum[t * dv + j] = fabs(gt[j]) / den;
            }
            dden[t] = -go / den;
            mdden[t] = gm / den;
            for (int64_t i = 0; i < dk; ++i) {
                double a = dden[t] * z[i], am = mdden[t] * z[i];
                for (int64_t j = 0; j < dv; ++j) {
                    a += S[i * dv + j] * dnum[t * dv + j];
                    am += Sa[i * dv + j] * mdnum[t * dv + j];
                }
                const double d = phi_prime(qt[i]);
                dq[(t * H + hh) * dk + i] = a * d;
                if (m_dq) m_dq[(t * H + hh) * dk + i] = am * d;
            }
        }
        /* backward in time: the reverse states (U, w), dk and dv */
        for (int64_t t = T - 1; t >= 0; --t) {
            const int last = (t == T - 1) || is_begin(start, T, 0, t + 1);
            if (last) {
                memset(U, 0, nS * sizeof(double));
                memset(Ua, 0, nS * sizeof(double));
                memset(w, 0, nk * sizeof(double));
                memset(wa, 0, nk * sizeof(double));
            }
            const double* qt = q + (t * H + hh) * dk;
            const double* kt = k + (t * H + hh) * dk;
            const double* vt = v + (t * H + hh) * dv;
            for (int64_t i = 0; i < dk; ++i) {
                Qf[i] = oracle_phi(qt[i]);
                Kf[i] = oracle_phi(kt[i]);
                w[i] += dden[t] * Qf[i];
                wa[i] += mdden[t] * Qf[i];
                for (int64_t j = 0; j < dv; ++j) {
                    U[i * dv + j] += Qf[i] * dnum[t * dv + j];
                    Ua[i * dv + j] += Qf[i] * mdnum[t * dv + j];
                }
            }
            for (int64_t i = 0; i < dk; ++i) {
                double a = w[i], am = wa[i];
                for (int64_t j = 0; j < dv; ++j) {
                    a += U[i * dv + j] * vt[j];
                    am += Ua[i * dv + j] * fabs(vt[j]);
                }
                const double d = phi_prime(kt[i]);
                dk_out[(t * H + hh) * dk + i] = a * d;
                if (m_dk) m_dk[(t * H + hh) * dk + i] = am * d;
            }
            for (int64_t j = 0; j < dv; ++j) {
                double a = 0.0, am = 0.0;
                for (int64_t i = 0; i < dk; ++i) {
                    a += U[i * dv + j] * Kf[i];
                    am += Ua[i * dv + j] * Kf[i];
                }
                dv_out[(t * H + hh) * dv + j] = a;
                if (m_dv) m_dv[(t * H + hh) * dv + j] = am;
            }
        }
    }
    free(S); free(Sa); free(z); free(U); free(Ua); free(w); free(wa); free(Qf); free(Kf);
    free(dnum); free(mdnum); free(dden); free(mdden);
}

/* ------------------------------------------------------ returns and GAE */

void oracle_discounted_return(const double* r, const uint8_t* start, double gamma,
                              int64_t B, int64_t T, double* G, double* m) {
    for (int64_t b = 0; b < B; ++b) {
        const double* rb = r + b * T;
        /* walk backwards: G_t = r_t + gamma * G_{t+1} inside an episode, and
         * G_e = r_e at its last step (the sum above, evaluated by Horner) */
        double g = 0.0, ga = 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const int last = (t == T - 1) || is_begin(start, T, b, t + 1);
            g = last ? rb[t] : rb[t] + gamma * g;
            ga = last ? fabs(rb[t]) : fabs(rb[t]) + gamma * ga;
            G[b * T + t] = g;
            if (m) m[b * T + t] = ga;
        }
    }
}

void oracle_gae(const double* r, const double* v, const double* vn, const uint8_t* done,
                const uint8_t* start, double gamma, double lambda, int64_t B, int64_t T,
                double* adv, double* target, double* m_adv, double* m_target) {
    const double gl = gamma * lambda;
    for (int64_t b = 0; b < B; ++b) {
        double A = 0.0, Am = 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const int64_t i = b * T + t;
            const int last = (t == T - 1) || is_begin(start, T, b, t + 1);
            double next_v;
            if (vn) next_v = vn[i];
            else next_v = last ? 0.0 : v[i + 1];
            const double keep = (done && done[i]) ? 0.0 : 1.0;
            const double delta = r[i] + gamma * keep * next_v - v[i];
            const double dmag = fabs(r[i]) + gamma * keep * fabs(next_v) + fabs(v[i]);
            A = last ? delta : delta + gl * A;
            Am = last ? dmag : dmag + gl * Am;
            adv[i] = A;
            if (target) target[i] = A + v[i];
            if (m_adv) m_adv[i] = Am;
            if (m_target) m_target[i] = Am + fabs(v[i]);
        }
    }
}

/* ---------------------------------------------------------------- FFM */

void oracle_ffm(const double* alpha, const double* omega, const double* x, const uint8_t* start,
                int64_t B, int64_t T, int64_t m, int64_t c, double* S, double* m_out) {
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t j = 0; j < m; ++j) {
            const double mag = exp(-fabs(alpha[j]));
            for (int64_t k = 0; k < c; ++k) {
                const double complex g = mag * cexp(I * omega[k]);
                double complex s = 0.0;
                double sm = 0.0;
                for (int64_t t = 0; t < T; ++t) {
                    const double xv = x[(b * T + t) * m + j];
                    if (is_begin(start, T, b, t)) {
                        s = xv;
                        sm = fabs(xv);
                    } else {
                        s = s * g + xv;
                        sm = sm * mag + fabs(xv);
                    }
                    const int64_t o = ((b * T + t) * m + j) * c + k;
                    S[2 * o] = creal(s);
                    S[2 * o + 1] = cimag(s);
                    if (m_out) m_out[o] = sm;
                }
            }
        }
    }
}

/* ------------------------------------------------- tape-based batching */

int64_t oracle_tbb_begin_indices(const uint8_t* start, int64_t n, int64_t offset, int64_t* out) {
    int64_t k = 0;
    for (int64_t t = 0; t < n; ++t)
        if (start[t] != 0) out[k++] = offset + t;
    return k;
}

int64_t oracle_tbb_sample(const uint8_t* D, int64_t n_D, int64_t row_bytes, const int64_t* begins, int64_t n_I,
                          const int64_t* draws, int64_t n_draws, int64_t batch,
                          uint8_t* out, uint8_t* out_start, int64_t* out_src) {
    int64_t len = 0;                       /* rows in the batch so far */
    for (int64_t k = 0; k < n_draws && len < batch; ++k) {
        const int64_t i = draws[k];
        const int64_t lo = begins[i];
        const int64_t hi = i + 1 < n_I ? begins[i + 1] : n_D;
        for (int64_t r = lo; r < hi && len < batch; ++r) {
            memcpy(out + len * row_bytes, D + r * row_bytes, (size_t)row_bytes);
            out_start[len] = r == lo ? 1 : 0;
            out_src[len] = r;
            len += 1;
        }
    }
    for (int64_t t = len; t < batch; ++t) {
        memset(out + t * row_bytes, 0, (size_t)row_bytes);
        out_start[t] = 0;
        out_src[t] = -1;
    }
    return len;
}

void oracle_ffm_bwd(const double* alpha, const double* omega, const uint8_t* start, const double* S,
                    const double* G, int64_t B, int64_t T, int64_t m, int64_t c,
                    double* dx, double* dalpha, double* domega,
                    double* m_dx, double* m_dalpha, double* m_domega) {
    memset(dx, 0, (size_t)(B * T * m) * sizeof(double));
    if (m_dx) memset(m_dx, 0, (size_t)(B * T * m) * sizeof(double));
    for (int64_t j = 0; j < m; ++j) {
        if (dalpha) dalpha[j] = 0.0;
        if (m_dalpha) m_dalpha[j] = 0.0;
    }
    for (int64_t k = 0; k < c; ++k) {
        if (domega) domega[k] = 0.0;
        if (m_domega) m_domega[k] = 0.0;
    }
    for (int64_t j = 0; j < m; ++j) {
        const double mag = exp(-fabs(alpha[j]));
        const double sgn = alpha[j] > 0.0 ? 1.0 : (alpha[j] < 0.0 ? -1.0 : 0.0);
        for (int64_t k = 0; k < c; ++k) {
            const double complex g = mag * cexp(I * omega[k]);
            double complex da = 0.0;
            double mda = 0.0;
            for (int64_t b = 0; b < B; ++b) {
                double complex lam = 0.0;
                double ml = 0.0;
                for (int64_t t = T - 1; t >= 0; --t) {
                    const int64_t o = ((b * T + t) * m + j) * c + k;
                    const double complex gt = G[2 * o] + I * G[2 * o + 1];
                    const int cont = (t + 1 < T) && !is_begin(start, T, b, t + 1);
                    lam = cont ? gt + conj(g) * lam : gt;
                    ml = cont ? cabs(gt) + mag * ml : cabs(gt);
                    dx[(b * T + t) * m + j] += creal(lam);
                    if (m_dx) m_dx[(b * T + t) * m + j] += ml;
                    if (!is_begin(start, T, b, t)) {
                        const int64_t p = ((b * T + t - 1) * m + j) * c + k;
                        const double complex sp = S[2 * p] + I * S[2 * p + 1];
                        da += lam * conj(sp);
                        mda += ml * cabs(sp);
                    }
                }
            }
            const double complex w = conj(g) * da;
            if (dalpha) dalpha[j] += -sgn * creal(w);
            if (domega) domega[k] += cimag(w);
            if (m_dalpha) m_dalpha[j] += mag * mda;
            if (m_domega) m_domega[k] += mag * mda;
        }
    }
}
