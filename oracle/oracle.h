/*
 * oracle.h -- plain, slow, obviously correct CPU reference for the resettable
 * memoroid scan ("Recurrent Reinforcement Learning with Memoroids",
 * arXiv 2402.09900).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes
 * or calls this code; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark use it.  It shares no header, helper or constant with the
 * HIP path.
 *
 * Every routine is the sequential definition written out in fp64:
 *   - the memoroid recurrence  h_t = e_I . f(P_0) . ... . f(P_t)      (Def. of
 *     a memoroid, Section 4 "Approach");
 *   - with the resettable monoid transform of Section 4 "Inline Recurrent
 *     State Resets" (resettable-monoid theorem): within an episode the
 *     transformed operator equals the original one, and no information crosses
 *     an episode boundary.  A begin flag b_t = 1 marks the first step of an
 *     episode (Section 2.1), so the state at a begin step holds that step's
 *     input and nothing older.
 *
 * Conventions shared by all routines (readings of the paper, see the design
 * notes of the repository):
 *   - start[b*T + t] != 0 means "an episode begins at step t of tape b"; any
 *     nonzero byte counts, and t = 0 of every tape is a begin step whatever the
 *     byte says (the pre-tape state is the identity g_I = (e_I, 0)).
 *   - data is row-major [B][T][d], features contiguous.
 *   - complex arrays are interleaved (re, im) doubles, i.e. C99 double complex.
 *   - the reset is a select, not the arithmetic A*(1-b') + e_I*b' form, so that
 *     a NaN/Inf in one episode never reaches the next (0*Inf = NaN would).
 *   - "magnitude companion" outputs (m, m_*) are the same recurrence run on
 *     absolute values; they bound the size of the rounding error any
 *     reordering of the sums can make, and the tests divide errors by
 *     max(|r|, m).  Pass NULL to skip them.
 *
 * Parity status: every routine here is pinned by CPU tests (brute force over
 * bracketings, closed forms, autograd, quadratic forms, worked examples of
 * Fig. 1 and Fig. 2).  No routine is "parity unpinned".
 */
#ifndef MEMOROID_ORACLE_H
#define MEMOROID_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Episode index of every step: the number of begin steps at or before t in
 * the same tape, minus one (Fig. 2; Alg. 1 stores I = where(b)).  idx[B][T]. */
void oracle_episode_idx(const uint8_t* start, int64_t B, int64_t T, int32_t* idx);

/* Diagonal linear memoroid, forward (S5 / LRU memoroids of App. G.2-G.3 with a
 * diagonal transition): h_t = x_t if step t begins an episode, else
 * a_t * h_{t-1} + x_t.
 *   a: a_stride_t == d -> per-step a[B][T][d];  a_stride_t == 0 -> a[d] shared
 *      by every tape and step (time-invariant transition).
 *   m: optional magnitude companion [B][T][d]:  m_t = |x_t| (+ |a_t| m_{t-1}). */
void oracle_diag_fwd(const double* a, int64_t a_stride_t, const double* x,
                     const uint8_t* start, int64_t B, int64_t T, int64_t d,
                     double* h, double* m);

/* Complex version (LRU memoroid of App. G.3).  a, x, h interleaved complex. */
void oracle_diag_fwd_c(const double* a, int64_t a_stride_t, const double* x,
                       const uint8_t* start, int64_t B, int64_t T, int64_t d,
                       double* h, double* m);

/* Reverse (gradient) scan of the diagonal memoroid.  The paper obtains it by
 * automatic differentiation; written out with the conjugate convention of
 * complex autograd (grad = dL/d conj(z)):
 *   lam_t = g_t + [step t+1 exists in the tape and is not a begin step] * conj(a_{t+1}) * lam_{t+1}
 *   dx_t  = lam_t
 *   da_t  = [t is not a begin step] * lam_t * conj(h_{t-1})
 * h is the forward output (an input here), g = dL/dh.
 *   da: [B][T][d] when a_stride_t == d;  [d] (summed over tapes and steps)
 *       when a_stride_t == 0.  NULL skips it.
 *   m_dx (optional, [B][T][d]): companion of lam on |a|, |g|.
 *   m_da (optional, shape of da): sum/element of m_dx,t * |h_{t-1}|. */
void oracle_diag_bwd(const double* a, int64_t a_stride_t, const uint8_t* start,
                     const double* h, const double* g,
                     int64_t B, int64_t T, int64_t d,
                     double* dx, double* da, double* m_dx, double* m_da);

void oracle_diag_bwd_c(const double* a, int64_t a_stride_t, const uint8_t* start,
                       const double* h, const double* g,
                       int64_t B, int64_t T, int64_t d,
                       double* dx, double* da, double* m_dx, double* m_da);

/* phi(u) = 1 + ELU(u) with alpha = 1 (App. G.1), evaluated as u + 1 for u > 0
 * and exp(u) otherwise, which is the same function without the 1 + (e^u - 1)
 * cancellation. */
double oracle_phi(double u);

/* Linear-transformer memoroid (App. G.1) over one tape with H independent
 * heads.  Per head, with S (dk x dv) and z (dk) reset to zero at every begin
 * step:
 *   S_t = S_{t-1} + phi(k_t) v_t^T,  z_t = z_{t-1} + phi(k_t),
 *   out_t = phi(q_t)^T S_t / (phi(q_t)^T z_t).
 * q, k: [T][H][dk]; v, out: [T][H][dv] (raw, pre-phi q and k).
 * m (optional, [T][H][dv]): phi(q)^T S_abs / (phi(q)^T z) with S_abs built
 * from |v|. */
void oracle_linattn(const double* q, const double* k, const double* v,
                    const uint8_t* start, int64_t T, int64_t H, int64_t dk, int64_t dv,
                    double* out, double* m);

/* Gradient of the linear-transformer memoroid readout (App. G.1; the paper
 * differentiates it automatically, Alg. 3 trains through it).  With
 * Q = phi(q), K = phi(k), the state (S, z) of the forward routine, num_t =
 * Q_t^T S_t, den_t = Q_t^T z_t, out_t = num_t / den_t and g = dL/dout:
 *   dnum_t = g_t / den_t,  dden_t = -(g_t . out_t) / den_t,
 *   dQ_t   = S_t dnum_t + dden_t z_t,
 *   U_t    = sum over steps s >= t of t's episode of Q_s dnum_s^T   (dk x dv),
 *   w_t    = sum over the same steps of dden_s Q_s,
 *   dK_t   = U_t v_t + w_t,  dV_t = U_t^T K_t,
 *   dq = dQ (.) phi'(q), dk = dK (.) phi'(k), phi'(u) = 1 (u > 0) or exp(u).
 * q, k, dq, dk: [T][H][dk]; v, g, dv: [T][H][dv].
 * m_dq, m_dk, m_dv (optional): magnitude companions, the same sums over
 * |v|, |g| and the companion of out. */
void oracle_linattn_bwd(const double* q, const double* k, const double* v, const uint8_t* start,
                        const double* g, int64_t T, int64_t H, int64_t dk, int64_t dv,
                        double* dq, double* dk_out, double* dv_out,
                        double* m_dq, double* m_dk, double* m_dv);

/* Fast-and-forgetful-memory aggregator (App. G.4, FFM memoroid): per step a
 * complex m x c state
 *   S_t = x_t 1_c^T                          at a begin step,
 *   S_t = S_{t-1} (.) gamma + x_t 1_c^T      otherwise,
 * with gamma[j][k] = exp(-|alpha_j| + i omega_k) (the outer sum of the paper's
 * memoroid, one step of its time count).  x: [B][T][m] real; S: [B][T][m][c]
 * interleaved complex; alpha[m], omega[c].
 * m_out (optional, [B][T][m][c]): magnitude companion, the same recurrence on
 * |gamma| = exp(-|alpha_j|) and |x|. */
void oracle_ffm(const double* alpha, const double* omega, const double* x, const uint8_t* start,
                int64_t B, int64_t T, int64_t m, int64_t c, double* S, double* m_out);

/* Tape-Based Batching insertion (Alg. 1): the begin indices of a rollout,
 * I = offset + where(b).  Every step whose flag byte is nonzero is listed,
 * in order; step 0 is NOT forced (a rollout may continue the episode in
 * flight).  out has room for n entries; returns the count. */
int64_t oracle_tbb_begin_indices(const uint8_t* start, int64_t n, int64_t offset, int64_t* out);

/* Tape-Based Batching sampling (Alg. 2): concatenate the episodes
 * D[I[i] : I[i+1]] (I = begins, I[n_I] standing for n_D) for i = draws[0], draws[1], ...
 * until the batch holds `batch` transitions, then cut it to exactly `batch`.
 * D holds n_D rows of row_bytes bytes.  Outputs per batch row: the row
 * (out), 1 at the first row of every appended episode (out_start), and the
 * source row in D (out_src).  If the draws run out first, the remaining rows
 * are zero, with out_start 0 and out_src -1.  Returns the rows filled. */
int64_t oracle_tbb_sample(const uint8_t* D, int64_t n_D, int64_t row_bytes, const int64_t* begins, int64_t n_I,
                          const int64_t* draws, int64_t n_draws, int64_t batch,
                          uint8_t* out, uint8_t* out_start, int64_t* out_src);

/* Gradient of the FFM aggregator (App. G.4) with the conjugate convention
 * of complex autograd.  G = dL/dS [B][T][m][c] (complex), S the forward
 * output.  Per feature (j, k), with gamma as in oracle_ffm:
 *   lam_t = G_t + [step t+1 exists and is not a begin step] conj(gamma) lam_{t+1}
 *   dx[b][t][j] = sum_k Re(lam_t[j][k])                       (x is real)
 *   da[j][k]    = sum over b, t not a begin step of lam_t conj(S_{t-1})
 *   dalpha[j]   = -sign(alpha_j) sum_k Re(conj(gamma_jk) da_jk)
 *   domega[k]   = sum_j Im(conj(gamma_jk) da_jk)
 * dx: [B][T][m]; dalpha: [m]; domega: [c] (NULL skips the parameter grads).
 * m_dx, m_dalpha, m_domega (optional): magnitude companions (|gamma|, |G|, |S|). */
void oracle_ffm_bwd(const double* alpha, const double* omega, const uint8_t* start, const double* S,
                    const double* G, int64_t B, int64_t T, int64_t m, int64_t c,
                    double* dx, double* dalpha, double* domega,
                    double* m_dx, double* m_dalpha, double* m_domega);

/* Discounted return over a tape (App. D, discounted-return memoroid; the
 * done-flag convention of Section 2): for every step, the discounted sum of
 * the rewards from that step to the end of its episode,
 *   G_t = sum_{i=t}^{e} gamma^(i-t) r_i,
 * where e is the last step of t's episode: the step before the next begin
 * step of the tape, or T-1.  Nothing beyond an episode's last step enters
 * (the episode is complete).  r, G: [B][T].
 * m (optional, [B][T]): the same sum over |r_i|. */
void oracle_discounted_return(const double* r, const uint8_t* start, double gamma,
                              int64_t B, int64_t T, double* G, double* m);

/* Generalized advantage estimate over a tape (App. E, GAE memoroid), with the
 * terminal (done) flag of Section 2:
 *   delta_t = r_t + gamma * [done_t == 0] * vn_t - v_t,
 *   A_t     = sum_{l=0}^{e-t} (gamma*lambda)^l delta_{t+l},
 * e as for the return.  vn_t is the value of the step's next state: vn[t] if
 * vn is given, otherwise v[t+1] when step t+1 is in t's episode and 0 at the
 * episode's last step.  done NULL means no step is terminal.
 *   r, v, vn, adv, target: [B][T]; done, start: [B][T] bytes.
 *   target (optional): A_t + v_t.
 *   m_adv (optional): the same sums over |r_t| + gamma |vn_t| + |v_t|;
 *   m_target (optional): m_adv + |v_t|. */
void oracle_gae(const double* r, const double* v, const double* vn, const uint8_t* done,
                const uint8_t* start, double gamma, double lambda, int64_t B, int64_t T,
                double* adv, double* target, double* m_adv, double* m_target);

#ifdef __cplusplus
}
#endif

#endif
