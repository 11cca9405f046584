/*
 * rlcs: RL credit-assignment scans for AMD Instinct MI355X (gfx950).
 *
 * Seven estimators share one first-order linear recurrence, evaluated independently over every
 * row of a [N, T] rollout buffer (Section 1, Eq. 1):
 *     backward:  A_t = alpha_t + beta_t * A_{t+1}      (GAE, V-Trace, Retrace, TD(lambda),
 *                                                       discounted returns)
 *     forward:   A_t = alpha_t + beta_t * A_{t-1}      (eligibility traces, episodic prefix sums)
 * Each entry point builds the per-step coefficients of Table 1 on chip from the raw rollout
 * tensors, scans them with the associative combine of Eq. 2, and writes its outputs once.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers   All array pointers are DEVICE pointers. Arrays are [N, T] row-major and
 *            contiguous (element (n, t) at n*T + t) unless stated otherwise; per-row arrays
 *            are [N]. Data inputs are `const void*` holding `dtype` elements (RLCS_F32: float,
 *            RLCS_BF16: bfloat16 bit patterns). Outputs are always float32.
 * Flags      `term` / `trunc` are uint8 [N, T]: nonzero = the episode terminated / was
 *            truncated after step t (Table 1 caption; d = term OR trunc). A step with both
 *            set counts as terminated. NULL means no step carries that flag.
 * bv         Continuation value V(s_{t+1}) of a truncated step (Section 3.2), [N, T], read
 *            only where trunc is set. Required (non-NULL) exactly when trunc is non-NULL.
 * boot       Value of the state just past the window, V(s_T) (Section 3.2, window edge), [N];
 *            NULL means 0 (no bootstrap).
 * Outputs    Must not overlap any input or each other. An output documented as optional may
 *            be NULL, in which case it is not written.
 * Alignment  Every pointer must be aligned to its element size. 16-byte aligned data pointers
 *            (and flag pointers aligned to 4 bytes for float32, 8 for bfloat16) take the
 *            vectorised path; others a slower one.
 * Sizes      N >= 0, 0 <= T <= 2^30, N*T representable. N == 0 or T == 0 is a no-op returning
 *            RLCS_OK.
 * Params     Discount gamma and trace parameter lambda must lie in [0, 1]; clipping
 *            thresholds rho_bar, c_bar must be > 0 (+infinity allowed). NaN is rejected.
 * Numerics   Arithmetic is float32 (bfloat16 inputs are widened exactly); the scan may
 *            associate differently from a sequential loop (Proposition 1), so results differ
 *            from one only by rounding. Results are bitwise reproducible run to run for a
 *            given shape and variant. Inputs must be finite.
 * Stream     `stream` is a hipStream_t (NULL = the default stream). Every call only enqueues
 *            work and returns; outputs are valid once the stream has reached that point.
 * Workspace  `ws` (optional) is device memory of at least rlcs_workspace_size(N, T) bytes.
 *            With it, calls of few long rows (under 256 rows longer than 4096 fp32 or 8192
 *            bf16 steps, T a multiple of 4 or 8) split each row into tiles over several
 *            workgroups that pass carries to each other through `ws`, which fills the GPU
 *            when N is small. `ws` must be zero-filled once before its first use; every call
 *            leaves it ready for the next one. Calls sharing one `ws` must be ordered on one
 *            stream. With ws == NULL (or ws_bytes too small) the library processes each row
 *            within one workgroup: same results up to rounding, less parallel.
 * Memory     The library allocates nothing and keeps no state between calls; it is safe to
 *            call from several threads.
 * Errors     Every argument is checked on the host before any HIP call; an error returns a
 *            status and enqueues nothing. RLCS_ERR_LAUNCH reports a failed kernel launch.
 */
#ifndef RLCS_H
#define RLCS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RLCS_OK = 0,
    RLCS_ERR_INVALID_ARG = 1, /* bad size, NULL required pointer, bad parameter or enum */
    RLCS_ERR_DTYPE = 2,       /* unknown dtype */
    RLCS_ERR_WORKSPACE = 3,   /* workspace required by the forced variant is missing/too small */
    RLCS_ERR_LAUNCH = 4       /* the HIP kernel launch failed */
} rlcs_status;

typedef enum { RLCS_F32 = 0, RLCS_BF16 = 1 } rlcs_dtype;

/* Episodic prefix sum boundary convention (Section 3.3.6). */
typedef enum {
    RLCS_ENDS_AT = 0,  /* a flag at t-1 ends the running sum: beta_t = 1 - d_{t-1} */
    RLCS_STARTS_AT = 1 /* a flag at t starts a new running sum: beta_t = 1 - d_t */
} rlcs_boundary;

typedef enum { RLCS_BACKWARD = 0, RLCS_FORWARD = 1 } rlcs_direction;

/* hipStream_t, passed as an opaque pointer so that this header needs no HIP headers. */
typedef void* rlcs_stream_t;

/* Generalized Advantage Estimation (Table 1; Section 3.3.1):
 *   alpha_t = r_t + gamma * succ(V)_t - V_t,   beta_t = gamma * lambda * (1 - d_t),   A_T = 0,
 * where succ(V)_t is V_{t+1} inside an episode, bv_t after a truncation, 0 after a termination
 * and boot[n] at the last step (Section 3.2).
 *   r, v     [N, T] rewards and values V(s_t), dtype
 *   adv      [N, T] float32 out: advantages A_t
 *   ret      [N, T] float32 out, optional: value targets A_t + V_t                            */
rlcs_status rlcs_gae(const void* r, const void* v, const uint8_t* term, const uint8_t* trunc,
                     const void* bv, const void* boot, float* adv, float* ret,
                     int64_t N, int64_t T, float gamma, float lambda, rlcs_dtype dtype,
                     void* ws, size_t ws_bytes, rlcs_stream_t stream);

/* V-Trace (Table 1; Section 3.3.2), with rho_t = min(rho_bar, exp(log_rho_t)),
 * c_t = min(c_bar, exp(log_rho_t)):
 *   alpha_t = rho_t (r_t + gamma succ(V)_t - V_t),  beta_t = gamma c_t (1 - d_t),  Delta_T = 0.
 *   log_rho  [N, T] log(pi(a_t|s_t) / mu(a_t|s_t)), dtype
 *   vs       [N, T] float32 out: value targets vs_t = V_t + Delta_t
 *   pg       [N, T] float32 out, optional: policy-gradient advantages
 *            rho_t (r_t + gamma succ(vs)_t - V_t), where succ(vs) is vs_{t+1} inside an
 *            episode and otherwise follows the succ(V) rule above.                            */
rlcs_status rlcs_vtrace(const void* r, const void* v, const void* log_rho, const uint8_t* term,
                        const uint8_t* trunc, const void* bv, const void* boot, float* vs,
                        float* pg, int64_t N, int64_t T, float gamma, float rho_bar, float c_bar,
                        rlcs_dtype dtype, void* ws, size_t ws_bytes, rlcs_stream_t stream);

/* Retrace(lambda) (Table 1; Section 3.3.3), with c_t = lambda * min(c_bar, exp(log_rho_t)) and
 * c_T = 0:
 *   alpha_t = r_t + gamma succ(E_pi Q)_t - Q(s_t, a_t),  beta_t = gamma c_{t+1} (1 - d_t),
 *   Delta_T = 0.
 *   q        [N, T] Q(s_t, a_t) of the taken action, dtype
 *   eq       [N, T] E_{a ~ pi} Q(s_t, a), dtype; boot[n] is E_pi Q(s_T, .) and bv_t is
 *            E_pi Q of the true successor of a truncated step
 *   log_rho  [N, T] log(pi(a_t|s_t) / mu(a_t|s_t)), dtype
 *   delta    [N, T] float32 out: corrections Delta_t
 *   q_ret    [N, T] float32 out, optional: Retrace targets Q(s_t, a_t) + Delta_t              */
rlcs_status rlcs_retrace(const void* r, const void* q, const void* eq, const void* log_rho,
                         const uint8_t* term, const uint8_t* trunc, const void* bv,
                         const void* boot, float* delta, float* q_ret, int64_t N, int64_t T,
                         float gamma, float lambda, float c_bar, rlcs_dtype dtype, void* ws,
                         size_t ws_bytes, rlcs_stream_t stream);

/* Retrace(lambda) in its full form (Section 3.3.3; the [N, T, A] inputs of Section 7.3): the
 * per-step terms are computed in the kernel from the action axis,
 *   E_pi Q(s_t) = sum_a pi(a|s_t) Q(s_t, a),  Q(s_t, a_t),  rho_t = pi(a_t|s_t) / mu_t,
 *   c_t = lambda * min(c_bar, rho_t),  c_T = 0,
 * and then scanned exactly as rlcs_retrace does.
 *   q, pi    [N, T, A] Q-values and target-policy probabilities, dtype, contiguous
 *   actions  [N, T] int32 taken actions. An action outside [0, A) is a caller error the
 *            kernel cannot return: that step takes Q(s_t, a_t) = pi(a_t|s_t) = 0 (so rho_t = 0),
 *            and if `ws` is given the call sets its error word (below) to 2
 *   mu       [N, T] behaviour-policy probability of the taken action, dtype (nonzero)
 *   bv, boot E_pi Q of the true successor of a truncated step / of s_T, as for rlcs_retrace
 *   delta, q_ret  as for rlcs_retrace
 *   A        number of actions, A >= 1. Each workgroup stages its chunk's [steps, A] slices
 *            of q and pi in LDS: whole for A <= 28, in slices of the action axis otherwise
 *            (32 actions at a time: one 128-byte line of float32, half a line of bfloat16).
 *   ws       optional, at least 64 bytes, 64-byte aligned, zero-filled by the caller: the int32
 *            at byte 8 becomes 2 when a call meets an out-of-range action, and stays so until
 *            the caller clears it. Unused otherwise; NULL = no report.
 * Rows are never split across workgroups for this entry point.                             */
rlcs_status rlcs_retrace_full(const void* r, const void* q, const void* pi,
                              const int32_t* actions, const void* mu, const uint8_t* term,
                              const uint8_t* trunc, const void* bv, const void* boot,
                              float* delta, float* q_ret, int64_t N, int64_t T, int64_t A,
                              float gamma, float lambda, float c_bar, rlcs_dtype dtype,
                              void* ws, size_t ws_bytes, rlcs_stream_t stream);

/* TD(lambda) returns (Table 1; Section 3.3.4):
 *   alpha_t = r_t + gamma (1 - lambda) succ(V)_t,  beta_t = gamma lambda (1 - d_t),  G_T = boot,
 * except that a truncated step continues with the full discount: alpha_t = r_t + gamma bv_t.
 *   ret      [N, T] float32 out: lambda-returns G_t                                         */
rlcs_status rlcs_td_lambda(const void* r, const void* v, const uint8_t* term,
                           const uint8_t* trunc, const void* bv, const void* boot, float* ret,
                           int64_t N, int64_t T, float gamma, float lambda, rlcs_dtype dtype,
                           void* ws, size_t ws_bytes, rlcs_stream_t stream);

/* Discounted returns (Table 1; Section 3.3.4):
 *   alpha_t = r_t (+ gamma bv_t at a truncated step),  beta_t = gamma (1 - d_t),  G_T = boot.
 *   ret      [N, T] float32 out: returns G_t                                                */
rlcs_status rlcs_discounted(const void* r, const uint8_t* term, const uint8_t* trunc,
                            const void* bv, const void* boot, float* ret, int64_t N, int64_t T,
                            float gamma, rlcs_dtype dtype, void* ws, size_t ws_bytes,
                            rlcs_stream_t stream);

/* Eligibility traces, forward (Table 1; Section 3.3.5), one scalar per step:
 *   z_t = gamma lambda (1 - d_{t-1}) z_{t-1} + x_t,  d_{-1} = 0,  z_{-1} = 0.
 *   x        [N, T] per-step gradient / feature values, dtype
 *   z        [N, T] float32 out: traces z_t                                                 */
rlcs_status rlcs_elig_trace(const void* x, const uint8_t* term, const uint8_t* trunc, float* z,
                            int64_t N, int64_t T, float gamma, float lambda, rlcs_dtype dtype,
                            void* ws, size_t ws_bytes, rlcs_stream_t stream);

/* Episodic prefix sum, forward (Table 1; Section 3.3.6):
 *   RLCS_ENDS_AT:   C_t = x_t + (1 - d_{t-1}) C_{t-1};  RLCS_STARTS_AT: C_t = x_t + (1 - d_t) C_{t-1};
 *   C_{-1} = 0.
 *   c        [N, T] float32 out: running sums C_t                                            */
rlcs_status rlcs_episodic_prefix(const void* x, const uint8_t* term, const uint8_t* trunc,
                                 float* c, int64_t N, int64_t T, rlcs_boundary boundary,
                                 rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                 rlcs_stream_t stream);

/* The bare recurrence with caller-supplied coefficients (the generic scan of Section 4.1):
 *   RLCS_BACKWARD: out_t = alpha_t + beta_t out_{t+1}, out_T = carry[n];
 *   RLCS_FORWARD:  out_t = alpha_t + beta_t out_{t-1}, out_{-1} = carry[n].
 *   alpha, beta [N, T] dtype; carry [N] dtype, optional (NULL = 0); out [N, T] float32.     */
rlcs_status rlcs_affine_scan(const void* alpha, const void* beta, const void* carry, float* out,
                             int64_t N, int64_t T, rlcs_direction direction, rlcs_dtype dtype,
                             void* ws, size_t ws_bytes, rlcs_stream_t stream);

/* Bytes of workspace that let any entry point above split rows of an [N, T] call over
 * several workgroups: a fixed 65600-byte part plus 16 bytes per row per 1024 steps, rounded up
 * (0 if the size overflows). Every entry point of this header lays the workspace out the same
 * way, so one workspace at least as large as each call needs serves calls of every kind and
 * shape, row-major and time-major alike, as long as they are ordered on one stream. */
size_t rlcs_workspace_size(int64_t N, int64_t T);

/* GAE with observation-skip masking, for multi-turn and tool-use trajectories (the extension
 * planned in Section 9.3: the recurrence is carried across masked tokens, beta_t = 1), with
 * optional whitening of the advantages.
 *   mask     [N, T] uint8: nonzero = the step takes part (an action token); zero = it is
 *            skipped (an observation token). NULL = every step takes part (plain GAE).
 * A skipped step passes on the advantage of the step after it and the value the step before
 * it sees as its successor: an unmasked step t has
 *   A_t = r_t + gamma W_t - V_t + gamma lambda A_{t+1} (the continuation term only without
 *   a flag at t),
 * with W_t the value of the next unmasked step, or 0 / bv / boot[n] if a termination /
 * truncation / the window edge comes first; a skipped step has A_t = A_{t+1}, or 0 if it
 * carries a flag. Flags cut where they occur, on skipped steps too (a truncated skipped step
 * hands its bv to the step before it).
 *   adv      [N, T] float32 out: A_t at every step (skipped steps carry the advantage)
 *   ret      [N, T] float32 out, optional: A_t + V_t (from the advantage before whitening)
 *   normalize  0: adv as above; 1: adv is whitened, (A_t - mean) / sqrt(var + eps), mean and
 *            unbiased variance over the steps that take part (var 0 with fewer than two),
 *            applied to every step. eps >= 0, finite.
 *   ws       required when normalize = 1: rlcs_workspace_size_masked(N, T) bytes, 64-byte
 *            aligned, zero-filled once before its first use (every call leaves it ready for
 *            the next); calls sharing it must be ordered on one stream. After the call its
 *            first 16 bytes hold the mean and 1/sqrt(var + eps) as two doubles. Unused when
 *            normalize = 0.
 * Rows are never split across workgroups for this entry point. A whitened call whose rows fit
 * in one workgroup's chunk (T <= 4096 float32 / 8192 bfloat16 steps) and whose workgroups
 * are all resident on the GPU at once runs as one kernel that reads and writes every array
 * once; otherwise a second kernel rewrites the advantages.                                  */
rlcs_status rlcs_gae_masked(const void* r, const void* v, const uint8_t* mask,
                            const uint8_t* term, const uint8_t* trunc, const void* bv,
                            const void* boot, float* adv, float* ret, int64_t N, int64_t T,
                            float gamma, float lambda, int normalize, float eps,
                            rlcs_dtype dtype, void* ws, size_t ws_bytes, rlcs_stream_t stream);

/* Workspace bytes that rlcs_gae_masked needs for whitening an [N, T] call (0 for negative
 * sizes). */
size_t rlcs_workspace_size_masked(int64_t N, int64_t T);

/* rlcs_gae_masked without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc). Same
 * arguments, results and kernels as rlcs_gae_masked; whitening (normalize = 1) uses a
 * workspace built into the library instead of `ws`: a static device array of 2.2 MiB per
 * GPU, held until the process ends, enough for N <= 65536 rows. The call itself allocates nothing
 * (no hipMalloc, no allocating library routine).
 *   N > 65536  RLCS_ERR_WORKSPACE, checked first (also with normalize = 0), before any HIP
 *              call; the other checks are rlcs_gae_masked's.
 *   The array's device address is looked up on the first call on each device (that device
 *   current); if the lookup fails the call returns RLCS_ERR_LAUNCH and enqueues nothing.
 * Every call on one GPU shares that GPU's array, which starts zero-filled when the library is
 * loaded on that device; every call leaves it ready for the next, so nothing needs clearing.
 * Calls that can overlap on one GPU (other streams, other threads, other graph replays
 * running at the same time) race on the array and must not whiten at once; calls ordered on
 * one stream are safe. The mean and 1/sqrt(var + eps) of the last call are not returned (use
 * rlcs_gae_masked with a workspace for them). */
rlcs_status rlcs_gae_masked_noalloc(const void* r, const void* v, const uint8_t* mask,
                                    const uint8_t* term, const uint8_t* trunc, const void* bv,
                                    const void* boot, float* adv, float* ret, int64_t N, int64_t T,
                                    float gamma, float lambda, int normalize, float eps,
                                    rlcs_dtype dtype, rlcs_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Strided layouts. The entry points below compute exactly what their row-major namesakes
 * compute, for [N, T] arrays laid out with element (n, t) at n * stride_n + t * stride_t:
 *   - time-major buffers ([T, ld] storage, step t of environment n at t * ld + n):
 *     stride_n = 1, stride_t = ld (>= N);
 *   - strided rows ([N, ld] storage, e.g. a view of the first T steps of wider rows):
 *     stride_n = ld (>= T), stride_t = 1;
 *   - dense row-major (stride_n = T, stride_t = 1) runs the row-major entry point itself.
 * Both strides are >= 1, counted in elements, and one dimension must nest inside the other
 * (stride_n >= T * stride_t or stride_t >= N * stride_n), so that distinct (n, t) are distinct
 * elements. All [N, T] arrays of a call (data, flags, bv and outputs) share the strides; boot
 * stays [N], contiguous. Elements outside the (n, t) grid are neither read nor written.
 * Sizes: N >= 0, 0 <= T <= 2^30, the largest element offset representable.
 * Workspace: at least rlcs_workspace_size_columns(N, T) bytes, zero-filled once, lets few
 * environments (N below about 64K) be split along T over several workgroups; without it each
 * group of 64 environments is scanned by one workgroup (the dense layout takes
 * rlcs_workspace_size(N, T) instead; Retrace splits below about 16K environments); calls of
 * fewer than 64 environments, or that split into
 * fewer than 256 tiles of 64 columns by 64 steps, split groups of 16 float32 (32 bfloat16)
 * columns instead. Calls of at most 256 steps over 4096 to 8192
 * float32 (8192 to 16384 bfloat16) environments use none: each workgroup scans 16 (32) whole
 * columns.
 * Every other convention is the row-major one.                                             */
rlcs_status rlcs_gae_strided(const void* r, const void* v, const uint8_t* term,
                             const uint8_t* trunc, const void* bv, const void* boot, float* adv,
                             float* ret, int64_t N, int64_t T, int64_t stride_n, int64_t stride_t,
                             float gamma, float lambda, rlcs_dtype dtype, void* ws,
                             size_t ws_bytes, rlcs_stream_t stream);
rlcs_status rlcs_vtrace_strided(const void* r, const void* v, const void* log_rho,
                                const uint8_t* term, const uint8_t* trunc, const void* bv,
                                const void* boot, float* vs, float* pg, int64_t N, int64_t T,
                                int64_t stride_n, int64_t stride_t, float gamma, float rho_bar,
                                float c_bar, rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                rlcs_stream_t stream);
rlcs_status rlcs_retrace_strided(const void* r, const void* q, const void* eq, const void* log_rho,
                                 const uint8_t* term, const uint8_t* trunc, const void* bv,
                                 const void* boot, float* delta, float* q_ret, int64_t N,
                                 int64_t T, int64_t stride_n, int64_t stride_t, float gamma,
                                 float lambda, float c_bar, rlcs_dtype dtype, void* ws,
                                 size_t ws_bytes, rlcs_stream_t stream);
rlcs_status rlcs_td_lambda_strided(const void* r, const void* v, const uint8_t* term,
                                   const uint8_t* trunc, const void* bv, const void* boot,
                                   float* ret, int64_t N, int64_t T, int64_t stride_n,
                                   int64_t stride_t, float gamma, float lambda, rlcs_dtype dtype,
                                   void* ws, size_t ws_bytes, rlcs_stream_t stream);
rlcs_status rlcs_discounted_strided(const void* r, const uint8_t* term, const uint8_t* trunc,
                                    const void* bv, const void* boot, float* ret, int64_t N,
                                    int64_t T, int64_t stride_n, int64_t stride_t, float gamma,
                                    rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                    rlcs_stream_t stream);
rlcs_status rlcs_elig_trace_strided(const void* x, const uint8_t* term, const uint8_t* trunc,
                                    float* z, int64_t N, int64_t T, int64_t stride_n,
                                    int64_t stride_t, float gamma, float lambda, rlcs_dtype dtype,
                                    void* ws, size_t ws_bytes, rlcs_stream_t stream);
rlcs_status rlcs_episodic_prefix_strided(const void* x, const uint8_t* term, const uint8_t* trunc,
                                         float* c, int64_t N, int64_t T, int64_t stride_n,
                                         int64_t stride_t, rlcs_boundary boundary,
                                         rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                         rlcs_stream_t stream);

/* Eligibility traces of feature vectors (Section 3.3.5: the trace of the gradient, or of the
 * feature vector under linear function approximation), forward:
 *   z_t = gamma lambda (1 - d_{t-1}) z_{t-1} + x_t,  d_{-1} = 0,  z_{-1} = 0,
 * with x_t, z_t in R^F and one scalar coefficient per step shared by all F features (the
 * paper's scalar-beta restriction; per-feature beta is not supported).
 *   x        [N, T, F] feature values, dtype, row-major (features innermost)
 *   term, trunc  [N, T] as above (one flag per step, for every feature)
 *   z        [N, T, F] float32 out: traces
 * Sizes: N, F >= 0, 0 <= T <= 2^30, N*T*F representable; any of them 0 is a no-op.
 * Calls whose F is a multiple of the 16-byte vector width (4 float32 or 8 bfloat16 features)
 * with a power-of-two number of vectors up to 64, short enough rows (F = 16 float32: up to 512
 * steps) and enough of them for 256 workgroups run along rows, x and z 16-byte aligned; the
 * others scan the N*F feature columns. Workspace: rlcs_workspace_size_columns(N * F, T) bytes,
 * as for the strided calls (used by the column scans when N*F is below about 64K).        */
rlcs_status rlcs_elig_trace_vec(const void* x, const uint8_t* term, const uint8_t* trunc,
                                float* z, int64_t N, int64_t T, int64_t F, float gamma,
                                float lambda, rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                rlcs_stream_t stream);

/* Workspace bytes for the strided calls (columns = N) and rlcs_elig_trace_vec
 * (columns = N * F) over T steps: the fixed 65600-byte part plus 16 bytes per column per 32
 * steps (rounded up); 0 for negative sizes or a size that overflows. */
size_t rlcs_workspace_size_columns(int64_t columns, int64_t T);

/* Static description of a status code. Never NULL. */
const char* rlcs_status_string(rlcs_status status);

/* Library version as major * 10000 + minor * 100 + patch. */
int rlcs_version(void);


#ifdef __cplusplus
}
#endif

#endif /* RLCS_H */
