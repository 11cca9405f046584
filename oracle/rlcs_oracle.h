/*
 * Sequential fp64 CPU oracle for the seven credit-assignment recurrences.
 *
 * TEST INFRASTRUCTURE ONLY. This library is the correctness reference that the GPU path is
 * compared against. It shares no code with the GPU library and must never be linked into it,
 * and nothing on the product path may call it.
 *
 * Every function evaluates the recurrence A_t = alpha_t + beta_t * A_{t+1} (or its forward
 * mirror, Section 1, Eq. 1) one step at a time, in fp64, exactly as the estimator's definition
 * reads (Table 1 and Sections 3.2-3.3). Inputs are host arrays:
 *   - data arrays are double, [N, T] row-major (callers widen float32 or bfloat16 exactly);
 *   - term / trunc are uint8 [N, T], nonzero = flag set, NULL = all clear;
 *   - bv is double [N, T], the continuation value read only at truncated steps; it must be
 *     non-NULL when trunc is non-NULL;
 *   - boot is double [N], the value of the state just past the window, NULL = 0.
 * Outputs are double [N, T] and must not alias inputs. N, T >= 0; nothing happens if either
 * is zero.
 */
#ifndef RLCS_ORACLE_H
#define RLCS_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

void oracle_gae(const double* r, const double* v, const uint8_t* term, const uint8_t* trunc,
                const double* bv, const double* boot, double* adv, double* ret,
                int64_t N, int64_t T, double gamma, double lambda);

void oracle_td_lambda(const double* r, const double* v, const uint8_t* term,
                      const uint8_t* trunc, const double* bv, const double* boot, double* ret,
                      int64_t N, int64_t T, double gamma, double lambda);

void oracle_discounted(const double* r, const uint8_t* term, const uint8_t* trunc,
                       const double* bv, const double* boot, double* ret,
                       int64_t N, int64_t T, double gamma);

void oracle_vtrace(const double* r, const double* v, const double* log_rho,
                   const uint8_t* term, const uint8_t* trunc, const double* bv,
                   const double* boot, double* vs, double* pg,
                   int64_t N, int64_t T, double gamma, double rho_bar, double c_bar);

void oracle_retrace(const double* r, const double* q, const double* eq, const double* log_rho,
                    const uint8_t* term, const uint8_t* trunc, const double* bv,
                    const double* boot, double* delta, double* q_ret,
                    int64_t N, int64_t T, double gamma, double lambda, double c_bar);

/* Full-form Retrace: Q(s_t, .) and pi(.|s_t) as [N, T, A], the taken actions (int32, [N, T])
 * and the behaviour probability mu(a_t|s_t) ([N, T]) replace the per-step inputs above:
 * E_pi Q(s_t) = sum_a pi(a|s_t) Q(s_t, a), Q(s_t, a_t) and rho_t = pi(a_t|s_t) / mu(a_t|s_t).
 * An action outside [0, A) selects nothing (its Q and pi are taken as 0). bv and boot are
 * expected values E_pi Q of the true successor / of s_T, as above. */
void oracle_retrace_full(const double* r, const double* q, const double* pi,
                         const int32_t* actions, const double* mu, const uint8_t* term,
                         const uint8_t* trunc, const double* bv, const double* boot,
                         double* delta, double* q_ret, int64_t N, int64_t T, int64_t A,
                         double gamma, double lambda, double c_bar);

void oracle_elig_trace(const double* x, const uint8_t* term, const uint8_t* trunc, double* z,
                       int64_t N, int64_t T, double gamma, double lambda);

/* GAE with observation-skip masking: mask uint8 [N, T], nonzero = the step takes part, NULL =
 * every step does. Masked steps carry the advantage and the successor value through; flags cut
 * where they occur. adv, ret as oracle_gae (ret = adv + v at every step). */
void oracle_gae_masked(const double* r, const double* v, const uint8_t* mask,
                       const uint8_t* term, const uint8_t* trunc, const double* bv,
                       const double* boot, double* adv, double* ret, int64_t N, int64_t T,
                       double gamma, double lambda);

/* Eligibility traces of F-vectors: x and z are double [N, T, F] (features innermost), the
 * flags [N, T]; the scalar coefficient gamma * lambda * (1 - d_{t-1}) of a step applies to
 * every feature. */
void oracle_elig_trace_vec(const double* x, const uint8_t* term, const uint8_t* trunc, double* z,
                           int64_t N, int64_t T, int64_t F, double gamma, double lambda);

/* starts_at = 0: a set flag at t-1 ends the running sum before t ("ends_at");
 * starts_at = 1: a set flag at t starts a new running sum at t. */
void oracle_episodic_prefix(const double* x, const uint8_t* term, const uint8_t* trunc,
                            double* c, int64_t N, int64_t T, int starts_at);

/* Plain affine recurrence with given coefficients. reverse = 1: A_t = alpha_t + beta_t A_{t+1},
 * A_T = carry[n]; reverse = 0: A_t = alpha_t + beta_t A_{t-1}, A_{-1} = carry[n].
 * carry NULL = 0. */
void oracle_affine_scan(const double* alpha, const double* beta, const double* carry,
                        double* out, int64_t N, int64_t T, int reverse);

#ifdef __cplusplus
}
#endif

#endif /* RLCS_ORACLE_H */
