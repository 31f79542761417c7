/*
 * memoroid.h -- C ABI of libmemoroid.so: resettable memoroid scans on AMD
 * MI355X (gfx950).
 *
 * The library computes the hot path of "Recurrent Reinforcement Learning with
 * Memoroids" (arXiv 2402.09900): the inclusive scan of a memoroid over a tape
 * of episodes laid end to end (Tape-Based Batching, Section 4.1), where the
 * resettable monoid transform (Section 4, "Inline Recurrent State Resets")
 * stops all information flow at every episode boundary, and the reverse scan
 * that back-propagates through it.
 *
 * Conventions common to every entry point
 * ---------------------------------------
 *  - Every data pointer is a DEVICE pointer (hipMalloc / torch CUDA memory),
 *    owned by the caller.  The library allocates nothing on the call path and
 *    keeps no state between calls.
 *  - Calls are asynchronous: they validate the arguments, enqueue kernels on
 *    `stream` (a hipStream_t passed as void*, NULL = the null stream) and
 *    return.  Faults inside a kernel surface at the caller's next
 *    synchronisation.
 *  - Return value: MEMOROID_OK (0) or a negative memoroid_status.  Argument
 *    errors are detected before any HIP call, so nothing is enqueued when a
 *    call fails validation.  No C++ exception crosses this boundary.
 *  - A tape is row-major [B][T][d] with the d features of a step contiguous;
 *    start[B][T] holds one byte per step, nonzero meaning "an episode begins
 *    at this step" (the begin flag b of Section 2.1).  Step 0 of every tape is
 *    treated as a begin step whatever its byte is: the scan starts from the
 *    identity g_I = (e_I, 0) of the resettable monoid.
 *  - Resets are selects: the state after a begin step holds that step's input
 *    and nothing older, so a NaN or Inf never crosses an episode boundary.
 *  - An empty problem (B, T or d equal to 0) returns MEMOROID_OK and enqueues
 *    nothing.
 *  - Outputs must not alias inputs (MEMOROID_EINVAL if the same pointer is
 *    passed for both).
 *  - Every pointer must be aligned to its element size (4 bytes for f32, 2 for
 *    bf16, 8 for complex64, 4 for int32).  Rows whose pointers are 16-byte
 *    aligned and whose d is a multiple of the vector width (4 f32, 4 bf16,
 *    2 complex64) take the vectorised kernels; other shapes take a scalar
 *    kernel with identical results.
 *  - The workspace is caller-allocated device memory of at least the size the
 *    matching *_workspace_bytes query (or memoroid_workspace_bytes) returns
 *    for the same arguments, 16-byte aligned (256 for linear attention).
 *    Concurrent calls must use distinct workspaces.  Two kinds of call:
 *      * SELF-INITIALISING -- every entry point without the _prepared
 *        suffix.  The workspace contents are undefined on entry and on exit;
 *        the call initialises what it needs on `stream` (one fill kernel of
 *        the workspace's header, counters and first descriptor bank, then
 *        the computation).  Any workspace of sufficient size works, whatever
 *        it held before.
 *      * PREPARED -- the *_prepared variants of the diagonal scans, FFM and
 *        its gradient, return, GAE and the TBB operations, for callers that
 *        repeat a call with the same sizes and want no fill kernel: the call
 *        initialises nothing (sampling runs two kernels, the others one).
 *        The workspace must have been prepared with
 *        memoroid_workspace_prepare() (on a stream ordered before the call)
 *        and then used only by calls of this library.  The first call binds
 *        it to that entry point and those sizes; every later call with the
 *        same entry point, sizes and flags finds it ready again, with no
 *        preparation in between.  The binding also covers: the dtypes;
 *        whether the vectorised kernels run (pointer alignment, d); a
 *        time-invariant a; whether grad_a / the FFM parameter gradients are
 *        asked for.  A call that differs in any of these returns MEMOROID_OK
 *        but computes nothing and leaves its outputs as they were:
 *        memoroid_workspace_status() then reports MEMOROID_EMISMATCH, and the
 *        workspace must be prepared again before any further use.  Prepare
 *        it again as well after MEMOROID_ETIMEOUT, and after any other writes
 *        to its memory (a self-initialising call included).
  */
#ifndef MEMOROID_H
#define MEMOROID_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MEMOROID_ABI_VERSION 4

typedef enum {
    MEMOROID_OK = 0,
    MEMOROID_EINVAL = -1,       /* bad pointer, extent, stride, alignment or aliasing */
    MEMOROID_EUNSUPPORTED = -2, /* valid but unsupported dtype pair or shape */
    MEMOROID_EWORKSPACE = -3,   /* workspace NULL or smaller than the query's size */
    MEMOROID_EHIP = -4,         /* a HIP runtime call or kernel launch failed */
    MEMOROID_ETIMEOUT = -5,     /* memoroid_workspace_status: a cross-tile wait gave up */
    MEMOROID_EMISMATCH = -6     /* memoroid_workspace_status: the workspace was bound to
                                   another call (or not prepared); prepare it again */
} memoroid_status;

typedef enum {
    MEMOROID_F32 = 0,   /* float */
    MEMOROID_BF16 = 1,  /* bfloat16, stored as uint16 bit patterns */
    MEMOROID_C64 = 2    /* complex float, interleaved (re, im) */
} memoroid_dtype;

/* Entry points, for the generic workspace query. */
typedef enum {
    MEMOROID_OP_DIAG = 0,              /* memoroid_scan_diag[_prepared]:      (B, T, d_or_H = d) */
    MEMOROID_OP_DIAG_BWD = 1,          /* memoroid_scan_diag_bwd[_prepared]:  (B, T, d_or_H = d) */
    MEMOROID_OP_LINATTN = 2,           /* memoroid_scan_linattn:      (T, d_or_H = H, dk, dv, chunk) */
    MEMOROID_OP_LINATTN_BWD = 3,       /* memoroid_scan_linattn_bwd:  (T, d_or_H = H, dk, dv, chunk) */
    MEMOROID_OP_FFM = 4,               /* memoroid_scan_ffm[_prepared]:       (B, T, d_or_H = m, dk = c) */
    MEMOROID_OP_FFM_BWD = 5,           /* memoroid_scan_ffm_bwd[_prepared]:   (B, T, d_or_H = m, dk = c) */
    MEMOROID_OP_RETURN = 6,            /* memoroid_discounted_return[_prepared]: (B, T) */
    MEMOROID_OP_GAE = 7,               /* memoroid_gae[_prepared]:            (B, T) */
    MEMOROID_OP_TBB_BEGIN_INDICES = 8, /* memoroid_tbb_begin_indices[_prepared]: (T = n) */
    MEMOROID_OP_TBB_SAMPLE = 9         /* memoroid_tbb_sample[_prepared]:     (B = n_draws, T = batch) */
} memoroid_op;

/* Version of this header the library was built from (MEMOROID_ABI_VERSION). */
int memoroid_abi_version(void);

/* Static, human-readable text for a memoroid_status value. */
const char* memoroid_status_string(int status);

/* ------------------------------------------------------------------------
 * Workspace size of any entry point: enough for every dtype and flag
 * combination the entry point accepts at these sizes (the per-entry queries
 * below give the exact size for one combination).  Arguments an operation
 * does not use are ignored; the comments of memoroid_op say which ones each
 * operation reads (B is ignored by the linear-attention operations, which
 * take one tape).  Returns 0 for an empty problem, for sizes or shapes the
 * operation rejects (negative extents, linear attention with dk, dv or chunk
 * other than 64), and for an unknown op.
 * ------------------------------------------------------------------------ */
size_t memoroid_workspace_bytes(memoroid_op op, int64_t B, int64_t T, int64_t d_or_H,
                                int64_t dk, int64_t dv, int64_t chunk);

/* ------------------------------------------------------------------------
 * Diagonal linear memoroid, forward.
 *
 * The S5 and LRU memoroids (App. G.2, G.3) with a diagonal transition, whose
 * monoid is (X, x) . (X', x') = (X'X, X'x + x') with e_I = (1, 0), give under
 * the reset transform the recurrence
 *     h_t = x_t                       if step t begins an episode,
 *     h_t = a_t * h_{t-1} + x_t       otherwise,
 * element-wise over the d features (complex multiply for MEMOROID_C64).  The
 * FFM memoroid (App. G.4) is the complex case with a time-invariant a.
 *
 *   a          per-step a[B][T][d] when a_stride_t == d, or one a[d] shared by
 *              every tape and step when a_stride_t == 0 (the time-invariant
 *              transition of S5 / LRU / FFM).  Any other stride: EINVAL.
 *   x          x[B][T][d], the lifted inputs f(o_t) computed by the caller.
 *   start      start[B][T] begin flags.
 *   h          out h[B][T][d].
 *   episode_idx  optional out int32[B][T]: number of begin steps at or before
 *              t in the same tape, minus one (the episode index of Fig. 2).
 *              NULL skips it.
 *   in_dtype / out_dtype: (F32,F32), (BF16,BF16), (BF16,F32), (C64,C64).
 *              bf16 inputs are decoded exactly and the state is carried in
 *              fp32; bf16 outputs are rounded to nearest even.  Other pairs:
 *              EUNSUPPORTED.
 *   Workspace: memoroid_scan_diag_workspace_bytes(B, T, d, in_dtype, out_dtype) bytes;
 *   memoroid_scan_diag initialises it, memoroid_scan_diag_prepared takes a
 *   prepared one (same arguments otherwise).
 * ------------------------------------------------------------------------ */
size_t memoroid_scan_diag_workspace_bytes(int64_t B, int64_t T, int64_t d,
                                          int in_dtype, int out_dtype);

int memoroid_scan_diag(const void* a, int64_t a_stride_t,
                       const void* x, const uint8_t* start,
                       void* h, int32_t* episode_idx,
                       int64_t B, int64_t T, int64_t d,
                       int in_dtype, int out_dtype,
                       void* workspace, size_t workspace_bytes, void* stream);

int memoroid_scan_diag_prepared(const void* a, int64_t a_stride_t,
                                const void* x, const uint8_t* start,
                                void* h, int32_t* episode_idx,
                                int64_t B, int64_t T, int64_t d,
                                int in_dtype, int out_dtype,
                                void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * memoroid_scan_diag for callers that cannot allocate device memory or own
 * a workspace: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments and results as memoroid_scan_diag
 * without the workspace: the call uses a fixed scratch array of
 * MEMOROID_NOALLOC_SCRATCH_BYTES inside the library (device memory that each
 * GPU the library runs on holds from the library's load until the process
 * ends), initialises what it needs of it on `stream` (a fill kernel, no
 * memset), and calls no hipMalloc, hipFree or other allocating routine.  The
 * first call with a device current looks up that device's copy of the
 * array once.
 *
 * Limit: a call whose tiling needs more than MEMOROID_NOALLOC_SCRATCH_BYTES
 * of workspace returns MEMOROID_EWORKSPACE and enqueues nothing.  Every
 * problem for which memoroid_scan_diag_workspace_bytes(...) is at most that
 * size is accepted (2^20 steps x 256 fp32 features, for example).  The
 * vectorised kernels (16-byte aligned tensors, d a multiple of the vector
 * width) need a quarter of that query's size or less, so e.g. 64 tapes x
 * 16384 steps x 512 bf16 features fits on them too.
 *
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (on different streams, or from different threads) race and
 * must be serialised by the caller.  The array keeps the last call's
 * contents, which the next call re-initialises.
 * ------------------------------------------------------------------------ */
#define MEMOROID_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

int memoroid_scan_diag_noalloc(const void* a, int64_t a_stride_t,
                               const void* x, const uint8_t* start,
                               void* h, int32_t* episode_idx,
                               int64_t B, int64_t T, int64_t d,
                               int in_dtype, int out_dtype, void* stream);

/* ------------------------------------------------------------------------
 * Diagonal linear memoroid, reverse scan (gradients).
 *
 * The paper differentiates through the scan with automatic differentiation;
 * this is that derivative written out, with the conjugate convention of
 * complex autograd (a gradient is dL/d conj(z)):
 *     lam_t = g_t + [t+1 < T and t+1 is not a begin step] * conj(a_{t+1}) * lam_{t+1}
 *     grad_x_t = lam_t
 *     grad_a_t = [t is not a begin step] * lam_t * conj(h_{t-1})
 * i.e. the same resettable scan run from the end of the tape, with the
 * episode ends (the steps before begin steps, and the tape end) as resets.
 *
 *   a, a_stride_t  as in memoroid_scan_diag.
 *   start      start[B][T].
 *   h          the forward output h[B][T][d] (saved activation).
 *   grad_h     upstream gradient g = dL/dh, [B][T][d].
 *   grad_x     out [B][T][d].
 *   grad_a     out [B][T][d] when a_stride_t == d; out [d], summed over every
 *              tape and step, when a_stride_t == 0.  NULL skips it.
 *   dtype      MEMOROID_F32 or MEMOROID_C64 (all tensors of that dtype).
 *   Workspace: memoroid_scan_diag_bwd_workspace_bytes(B, T, d, dtype, a_stride_t)
 *   bytes; self-initialising, or prepared for memoroid_scan_diag_bwd_prepared.
 * ------------------------------------------------------------------------ */
size_t memoroid_scan_diag_bwd_workspace_bytes(int64_t B, int64_t T, int64_t d,
                                              int dtype, int64_t a_stride_t);

int memoroid_scan_diag_bwd(const void* a, int64_t a_stride_t,
                           const uint8_t* start, const void* h, const void* grad_h,
                           void* grad_x, void* grad_a,
                           int64_t B, int64_t T, int64_t d, int dtype,
                           void* workspace, size_t workspace_bytes, void* stream);

int memoroid_scan_diag_bwd_prepared(const void* a, int64_t a_stride_t,
                                    const uint8_t* start, const void* h, const void* grad_h,
                                    void* grad_x, void* grad_a,
                                    int64_t B, int64_t T, int64_t d, int dtype,
                                    void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * FFM aggregator (App. G.4, the fast-and-forgetful-memory memoroid): a
 * complex m x c state per step,
 *     S_t = x_t 1_c^T                          at a begin step,
 *     S_t = S_{t-1} (.) gamma + x_t 1_c^T      otherwise,
 * gamma[j][k] = exp(-|alpha_j| + i omega_k), i.e. the paper's time-count
 * monoid (X, t) . (X', t') = (X (.) exp(t' (-|alpha| (+) i omega)) + X', t + t')
 * advanced one step at a time.  gamma is generated in the kernel (fp32
 * exp/sincos); the input gate x = (W1 o + b1) (.) sigma(W2 o + b2) and the
 * readout g are left to the caller.
 *
 *   alpha      [m] fp32;  omega: [c] fp32.
 *   x          [B][T][m] fp32, real; broadcast over the c columns.
 *   start      start[B][T] (as above).
 *   S          out [B][T][m][c] complex64, interleaved (re, im).
 *   episode_idx  optional out int32[B][T]; NULL skips it.
 *   Vectorised when m * c is even and S is 16-byte aligned.
 *   Workspace: memoroid_scan_ffm_workspace_bytes(B, T, m, c) bytes;
 *   self-initialising, or prepared for memoroid_scan_ffm_prepared.
 * ------------------------------------------------------------------------ */
size_t memoroid_scan_ffm_workspace_bytes(int64_t B, int64_t T, int64_t m, int64_t c);

int memoroid_scan_ffm(const float* alpha, const float* omega, const float* x,
                      const uint8_t* start, void* S, int32_t* episode_idx,
                      int64_t B, int64_t T, int64_t m, int64_t c,
                      void* workspace, size_t workspace_bytes, void* stream);

int memoroid_scan_ffm_prepared(const float* alpha, const float* omega, const float* x,
                               const uint8_t* start, void* S, int32_t* episode_idx,
                               int64_t B, int64_t T, int64_t m, int64_t c,
                               void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Gradient of the FFM aggregator (App. G.4), conjugate (PyTorch) convention
 * for the complex upstream gradient.  Per feature (j, k):
 *     lam_t = G_t + [step t+1 is not a begin step] conj(gamma_jk) lam_{t+1}
 *     grad_x[b][t][j] = sum_k Re(lam_t[j][k])
 *     da_jk = sum over tapes and non-begin steps of lam_t conj(S_{t-1})
 *     grad_alpha[j] = -sign(alpha_j) sum_k Re(conj(gamma_jk) da_jk)
 *     grad_omega[k] = sum_j Im(conj(gamma_jk) da_jk)
 *
 *   alpha, omega, start  as for memoroid_scan_ffm.
 *   S          the forward output [B][T][m][c] complex64 (needed only for the
 *              parameter gradients; may be NULL when both are NULL).
 *   grad_S     dL/dS [B][T][m][c] complex64.
 *   grad_x     out [B][T][m] fp32.
 *   grad_alpha optional out [m] fp32;  grad_omega: optional out [c] fp32.
 *   c must be a power of two no larger than 16 (MEMOROID_EUNSUPPORTED
 *   otherwise): the input gradient is reduced over c inside the kernel.
 *   Workspace: memoroid_scan_ffm_bwd_workspace_bytes(B, T, m, c) bytes;
 *   self-initialising, or prepared for memoroid_scan_ffm_bwd_prepared.
 * ------------------------------------------------------------------------ */
size_t memoroid_scan_ffm_bwd_workspace_bytes(int64_t B, int64_t T, int64_t m, int64_t c);

int memoroid_scan_ffm_bwd(const float* alpha, const float* omega, const uint8_t* start,
                          const void* S, const void* grad_S, float* grad_x,
                          float* grad_alpha, float* grad_omega,
                          int64_t B, int64_t T, int64_t m, int64_t c,
                          void* workspace, size_t workspace_bytes, void* stream);

int memoroid_scan_ffm_bwd_prepared(const float* alpha, const float* omega, const uint8_t* start,
                                   const void* S, const void* grad_S, float* grad_x,
                                   float* grad_alpha, float* grad_omega,
                                   int64_t B, int64_t T, int64_t m, int64_t c,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Linear-transformer memoroid (App. G.1), forward readout, one tape of T
 * steps with H independent heads.  Per head, with S (dk x dv) and z (dk)
 * reset to zero at every begin step:
 *     S_t = S_{t-1} + phi(k_t) v_t^T,   z_t = z_{t-1} + phi(k_t),
 *     out_t = phi(q_t)^T S_t / (phi(q_t)^T z_t),   phi(u) = 1 + ELU(u).
 * The MLP and residual of the paper's readout g are left to the caller.
 *
 *   q, k       raw (pre-phi) [T][H][dk] fp32;  v: [T][H][dv] fp32.
 *   start      start[T].
 *   out        out [T][H][dv] fp32.
 *   episode_idx  optional out int32[T] (as above); NULL skips it.
 *   dk, dv, chunk: this version supports dk == dv == 64 and chunk == 64
 *              (EUNSUPPORTED otherwise).
 *   Workspace (self-initialising): memoroid_scan_linattn_workspace_bytes(T, H, dk, dv, chunk).
 * ------------------------------------------------------------------------ */
size_t memoroid_scan_linattn_workspace_bytes(int64_t T, int64_t H, int64_t dk,
                                             int64_t dv, int64_t chunk);

int memoroid_scan_linattn(const float* q, const float* k, const float* v,
                          const uint8_t* start, float* out, int32_t* episode_idx,
                          int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t chunk,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Gradient of the linear-transformer memoroid readout (App. G.1; Alg. 3
 * trains through it).  With Q = phi(q), K = phi(k) and g = dL/dout:
 *     dnum_t = g_t / den_t,  dden_t = -(g_t . out_t) / den_t,
 *     dQ_t = S_t dnum_t + dden_t z_t,
 *     dK_t = U_t v_t + w_t,  dV_t = U_t^T K_t,
 * where (S, z) are the forward states and U_t, w_t sum Q_s dnum_s^T and
 * dden_s Q_s over the steps s >= t of t's episode; dq = dQ (.) phi'(q),
 * dk = dK (.) phi'(k).  Chunked like the forward pass (chunk states are
 * recomputed, so only the forward output is needed).
 *
 *   q, k, v, start  as for memoroid_scan_linattn.
 *   out        the forward output [T][H][dv] for the same inputs.
 *   grad_out   dL/dout [T][H][dv].
 *   grad_q, grad_k, grad_v  out [T][H][64] fp32, distinct from every input.
 *   dk == dv == chunk == 64 (MEMOROID_EUNSUPPORTED otherwise); 16-byte
 *   aligned fp32 arrays.
 *   Workspace (self-initialising): memoroid_scan_linattn_bwd_workspace_bytes(T, H, dk, dv, chunk).
 * ------------------------------------------------------------------------ */
size_t memoroid_scan_linattn_bwd_workspace_bytes(int64_t T, int64_t H, int64_t dk,
                                                 int64_t dv, int64_t chunk);

int memoroid_scan_linattn_bwd(const float* q, const float* k, const float* v,
                              const uint8_t* start, const float* out, const float* grad_out,
                              float* grad_q, float* grad_k, float* grad_v,
                              int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t chunk,
                              void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Discounted return over a tape (App. D, the discounted-return memoroid
 * (a, r) . (a', r') = (a a', a r' + r) with f(r) = (gamma, r)), restarted at
 * every episode: for each step, the sum of gamma^(i-t) r_i over the steps i
 * from t to the last step of t's episode, which is the step before the next
 * begin step or the tape's last step (episodes are complete: nothing is
 * bootstrapped after them).
 *
 *   r          rewards [B][T] fp32.
 *   start      start[B][T] begin flags (as above).
 *   gamma      discount, 0 <= gamma <= 1 (MEMOROID_EINVAL otherwise, NaN too).
 *   G          out [B][T] fp32; must not alias r or start.
 *   Rows with T % 4 == 0 and 16-byte aligned r and G (4-byte aligned start)
 *   take the vectorised kernel, other shapes a scalar one.
 *   Workspace: memoroid_discount_workspace_bytes(B, T) bytes; self-initialising,
 *   or prepared for memoroid_discounted_return_prepared.
 * ------------------------------------------------------------------------ */
size_t memoroid_discount_workspace_bytes(int64_t B, int64_t T);

int memoroid_discounted_return(const float* r, const uint8_t* start, float gamma, float* G,
                               int64_t B, int64_t T,
                               void* workspace, size_t workspace_bytes, void* stream);

int memoroid_discounted_return_prepared(const float* r, const uint8_t* start, float gamma, float* G,
                                        int64_t B, int64_t T,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Generalized advantage estimate over a tape (App. E, the GAE memoroid:
 * the return's monoid with gamma*lambda as the discount and the TD error as
 * the reward), restarted at every episode, with the terminal (done) flag of
 * Section 2 removing the bootstrap value of a terminal transition:
 *     delta_t = r_t + gamma * [done_t == 0] * vn_t - value_t
 *     adv_t   = sum_{l=0}^{e-t} (gamma*lambda)^l delta_{t+l},  e = last step of t's episode
 *     target_t = adv_t + value_t
 *
 *   r, value   [B][T] fp32: reward of the transition, V(s_t).
 *   value_next optional [B][T] fp32: V(s'_t), the value of the transition's
 *              next state (used at every step, episode ends included).  NULL:
 *              vn_t = value_{t+1} when step t+1 is in t's episode, 0 at the
 *              episode's last step.
 *   done       optional [B][T] bytes, nonzero = the transition ends in a
 *              terminal state; NULL = no terminal steps.
 *   start      start[B][T] begin flags (as above).
 *   gamma, lambda  in [0, 1] (MEMOROID_EINVAL otherwise).  The recurrence
 *              runs with the fp32 product gamma*lambda.
 *   adv        out [B][T] fp32;  target: optional out [B][T] fp32 (NULL skips).
 *              Outputs must not alias any input or each other.
 *   Vectorised when T % 4 == 0, every fp32 pointer is 16-byte aligned and
 *   the flag pointers 4-byte aligned.
 *   Workspace: memoroid_discount_workspace_bytes(B, T) bytes; self-initialising,
 *   or prepared for memoroid_gae_prepared.
 * ------------------------------------------------------------------------ */
int memoroid_gae(const float* r, const float* value, const float* value_next, const uint8_t* done,
                 const uint8_t* start, float gamma, float lambda, float* adv, float* target,
                 int64_t B, int64_t T,
                 void* workspace, size_t workspace_bytes, void* stream);

int memoroid_gae_prepared(const float* r, const float* value, const float* value_next, const uint8_t* done,
                          const uint8_t* start, float gamma, float lambda, float* adv, float* target,
                          int64_t B, int64_t T,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Tape-Based Batching, insertion (Alg. 1): the begin indices of a rollout,
 *     indices[0 .. count) = offset + where(start[0 .. n) != 0),
 * in increasing order.  Step 0 is NOT treated as a begin here: a rollout
 * may continue the episode that the previous one left unfinished, and only
 * its flag byte decides.
 *
 *   start      [n] flag bytes.
 *   offset     added to every index (card(D) before the rollout is appended).
 *   indices    out, room for n int64 values (only count are written).
 *   count      out, one int64 in device memory.
 *   n < 2^31 (MEMOROID_EUNSUPPORTED otherwise); n == 0 writes count = 0.
 *   Workspace: memoroid_tbb_begin_indices_workspace_bytes(n) bytes;
 *   self-initialising, or prepared for memoroid_tbb_begin_indices_prepared.
 * ------------------------------------------------------------------------ */
size_t memoroid_tbb_begin_indices_workspace_bytes(int64_t n);

int memoroid_tbb_begin_indices(const uint8_t* start, int64_t n, int64_t offset,
                               int64_t* indices, int64_t* count,
                               void* workspace, size_t workspace_bytes, void* stream);

int memoroid_tbb_begin_indices_prepared(const uint8_t* start, int64_t n, int64_t offset,
                                        int64_t* indices, int64_t* count,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Tape-Based Batching, sampling (Alg. 2): the batch is the concatenation of
 * the episodes D[I[i] : I[i+1]] for i = draws[0], draws[1], ... (I[n_I]
 * standing for n_D), cut to exactly `batch` rows.  The random positions are
 * drawn by the caller (Alg. 2 draws them uniformly from 0 .. n_I - 1).
 *
 *   D          [n_D][row_bytes] transitions (any payload).
 *   I          [n_I] int64 begin indices, increasing, in [0, n_D]; values
 *              outside that range are clamped (an episode never reads past D).
 *   draws      [n_draws] int64 positions in I, clamped to [0, n_I).
 *   out        out [batch][row_bytes].
 *   out_start  out [batch] bytes: 1 at the first row of every appended
 *              episode (the begin flags of the batch as a tape), else 0.
 *   out_src    optional out [batch] int64: source row in D, -1 if unfilled.
 *   filled     optional out int64 (device): rows filled, min(batch, total
 *              length of the drawn episodes).  Rows past it are zero, with
 *              out_start 0.  Since every episode has at least one row,
 *              n_draws >= batch always fills the batch.
 *   n_draws <= 2^24, row_bytes <= 2^24, batch < 2^47 and n_D < 2^47
 *   (MEMOROID_EUNSUPPORTED otherwise).  Rows move in 16-byte units when
 *   row_bytes % 16 == 0 and D, out are 16-byte aligned.
 *   Workspace: memoroid_tbb_sample_workspace_bytes(n_draws, batch) bytes,
 *   self-initialising, or prepared for memoroid_tbb_sample_prepared (bound to
 *   n_draws and batch); not used when n_draws or batch is 0.  It holds, per call, where each draw starts in
 *   the batch and which draw holds the first row of each group of 256
 *   output rows.  A prepared call that finds it bound to other sizes writes
 *   no output (memoroid_workspace_status reports MEMOROID_EMISMATCH).
 * ------------------------------------------------------------------------ */
size_t memoroid_tbb_sample_workspace_bytes(int64_t n_draws, int64_t batch);

int memoroid_tbb_sample(const void* D, int64_t n_D, int64_t row_bytes,
                        const int64_t* I, int64_t n_I, const int64_t* draws, int64_t n_draws,
                        int64_t batch, void* out, uint8_t* out_start, int64_t* out_src,
                        int64_t* filled, void* workspace, size_t workspace_bytes, void* stream);

int memoroid_tbb_sample_prepared(const void* D, int64_t n_D, int64_t row_bytes,
                                 const int64_t* I, int64_t n_I, const int64_t* draws, int64_t n_draws,
                                 int64_t batch, void* out, uint8_t* out_start, int64_t* out_src,
                                 int64_t* filled, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Prepare a workspace for the PREPARED calls (the *_prepared variants, see
 * the conventions above):
 * enqueues on `stream` one kernel that fills the first workspace_bytes
 * (rounded down to a multiple of 16) with all-ones bytes: an unbound
 * workspace, with no tile counted and no descriptor published.  workspace
 * must be 16-byte aligned and at least 256 bytes (MEMOROID_EINVAL
 * otherwise).  Not needed by the self-initialising calls.  The caller keeps
 * ownership; nothing is allocated.
 * ------------------------------------------------------------------------ */
int memoroid_workspace_prepare(void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Health of the calls that used `workspace` since it was prepared (for a
 * SELF-INITIALISING call: of the last call): synchronises `stream`, then
 * returns MEMOROID_OK; MEMOROID_EMISMATCH if a call found the workspace
 * bound to another call (that call's outputs are invalid); MEMOROID_ETIMEOUT
 * if a kernel's bounded wait for a predecessor tile gave up (its outputs are
 * then invalid); MEMOROID_EHIP if the copy failed.  Intended for tests and
 * debugging.
 * ------------------------------------------------------------------------ */
int memoroid_workspace_status(const void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MEMOROID_H */
