/*
 * Sequential fp64 CPU oracle for the seven credit-assignment recurrences.
 *
 * TEST INFRASTRUCTURE ONLY: the reference the GPU path is checked against. It shares no code,
 * header or constant with the GPU library; only tests, the smoke check and the CPU-baseline
 * leg of the benchmark may load it.
 *
 * Each function walks every row one step at a time in the direction of its recurrence
 * (Section 1, Eq. 1), with the per-step terms of Table 1 and the boundary rules of
 * Section 3.2. No scan, no blocking, no reordering: the parallel scan reaches the same
 * result up to rounding because the combine of Eq. 2 is associative (Proposition 1).
 *
 * Readings taken where the paper is silent (also listed with the design notes):
 *   - a step with both flags set is treated as terminated (successor value 0, carry cut);
 *   - at a truncated step the continuation value bv_t enters with the full discount gamma
 *     for every backward estimator (Section 3.2; TD(lambda) as stated in Section 3.3.4,
 *     discounted returns by the same argument);
 *   - V-Trace's policy-gradient advantage uses the successor of the corrected value target:
 *     v-trace target at t+1 inside the episode, bv_t after a truncation, 0 after a
 *     termination, the window bootstrap at the last step (Section 3.3.2);
 *   - Retrace's trace coefficient is c_t = lambda * min(c_bar, rho_t) with c_T = 0
 *     (Section 3.3.3); its outputs are the correction Delta_t and Q_ret = Q(s_t, a_t) + Delta_t;
 *   - the forward scans use d = term OR trunc and no bootstrap (Section 3.2).
 */
#include "rlcs_oracle.h"

#include <math.h>
#include <stddef.h>
#include <stdlib.h>

/* Flag helpers: a NULL flag array means every flag is clear. */
static int flag_at(const uint8_t* f, int64_t i) { return f != NULL && f[i] != 0; }

/* Successor value u(s_{t+1}) as seen from step t of one row (Section 3.2):
 *   terminated          -> 0 (no successor value),
 *   truncated, not term -> bv_t (caller-supplied continuation),
 *   last step of window -> the row's bootstrap B,
 *   otherwise           -> u_{t+1}.                                                        */
static double successor(const double* u_row, const uint8_t* term_row, const uint8_t* trunc_row,
                        const double* bv_row, double B, int64_t t, int64_t T) {
    if (flag_at(term_row, t)) return 0.0;
    if (flag_at(trunc_row, t)) return bv_row[t];
    if (t == T - 1) return B;
    return u_row[t + 1];
}

static const uint8_t* row_of_flags(const uint8_t* f, int64_t n, int64_t T) {
    return f == NULL ? NULL : f + n * T;
}

static const double* row_of(const double* a, int64_t n, int64_t T) {
    return a == NULL ? NULL : a + n * T;
}

/* GAE, Table 1 and Section 3.3.1:
 *   delta_t = r_t + gamma * succ(V)_t - V_t,
 *   A_t     = delta_t + gamma * lambda * (1 - d_t) * A_{t+1},  A_T = 0,
 *   R_t     = A_t + V_t (the value target).                                                 */
void oracle_gae(const double* r, const double* v, const uint8_t* term, const uint8_t* trunc,
                const double* bv, const double* boot, double* adv, double* ret,
                int64_t N, int64_t T, double gamma, double lambda) {
    for (int64_t n = 0; n < N; ++n) {
        const double* rr = r + n * T;
        const double* vv = v + n * T;
        const uint8_t* te = row_of_flags(term, n, T);
        const uint8_t* tr = row_of_flags(trunc, n, T);
        const double* bb = row_of(bv, n, T);
        const double B = boot ? boot[n] : 0.0;
        double A_next = 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const double d = (flag_at(te, t) || flag_at(tr, t)) ? 1.0 : 0.0;
            const double delta = rr[t] + gamma * successor(vv, te, tr, bb, B, t, T) - vv[t];
            const double A = delta + gamma * lambda * (1.0 - d) * A_next;
            adv[n * T + t] = A;
            ret[n * T + t] = A + vv[t];
            A_next = A;
        }
    }
}

/* GAE with observation-skip masking (the planned extension of Section 9.3: the recurrence is
 * carried across masked tokens, beta_t = 1). mask[t] != 0 marks a step that takes part (an
 * action token); masked steps (observations) are skipped: the advantage passes through them
 * unchanged, and so does the value a preceding step sees as its successor, which is the value
 * of the next unmasked step. A flag cuts where it occurs, masked step or not: a terminated
 * masked step passes on advantage 0 and successor value 0, a truncated one advantage 0 and its
 * continuation bv_t. Walking backward with the running advantage A and the running successor
 * value W (A = 0 and W = boot past the window):
 *   unmasked: A_t = r_t + gamma * s - V_t + gamma * lambda * (cont ? A : 0),  W <- V_t
 *   masked:   A_t = cont ? A : 0,                                             W <- s
 * where s = 0 after a termination, bv_t after a truncation, else W, and cont = no flag at t.
 * Outputs: adv_t = A_t and ret_t = A_t + V_t at every step. mask NULL = every step takes part. */
void oracle_gae_masked(const double* r, const double* v, const uint8_t* mask,
                       const uint8_t* term, const uint8_t* trunc, const double* bv,
                       const double* boot, double* adv, double* ret, int64_t N, int64_t T,
                       double gamma, double lambda) {
    for (int64_t n = 0; n < N; ++n) {
        const double* rr = r + n * T;
        const double* vv = v + n * T;
        const uint8_t* mk = row_of_flags(mask, n, T);
        const uint8_t* te = row_of_flags(term, n, T);
        const uint8_t* tr = row_of_flags(trunc, n, T);
        const double* bb = row_of(bv, n, T);
        double A = 0.0;
        double W = boot ? boot[n] : 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const int is_term = flag_at(te, t);
            const int is_trunc = !is_term && flag_at(tr, t);
            const int cont = !is_term && !is_trunc;
            const double s = is_term ? 0.0 : (is_trunc ? bb[t] : W);
            const int in = mk == NULL || mk[t] != 0;
            double At;
            if (in) {
                At = rr[t] + gamma * s - vv[t] + gamma * lambda * (cont ? A : 0.0);
                W = vv[t];
            } else {
                At = cont ? A : 0.0;
                W = s;
            }
            adv[n * T + t] = At;
            ret[n * T + t] = At + vv[t];
            A = At;
        }
    }
}

/* TD(lambda) returns, Table 1 and Section 3.3.4:
 *   G_t = r_t + gamma * [(1 - lambda) V(s_{t+1}) + lambda G_{t+1}] inside an episode,
 *   with the successor value given by Section 3.2; a truncated step takes the continuation
 *   with the full gamma; a terminated step has no successor; the window carry is G_T = B, so
 *   the last step receives gamma (1 - lambda) B + gamma lambda B = gamma B.                 */
void oracle_td_lambda(const double* r, const double* v, const uint8_t* term,
                      const uint8_t* trunc, const double* bv, const double* boot, double* ret,
                      int64_t N, int64_t T, double gamma, double lambda) {
    for (int64_t n = 0; n < N; ++n) {
        const double* rr = r + n * T;
        const double* vv = v + n * T;
        const uint8_t* te = row_of_flags(term, n, T);
        const uint8_t* tr = row_of_flags(trunc, n, T);
        const double* bb = row_of(bv, n, T);
        const double B = boot ? boot[n] : 0.0;
        double G_next = B;
        for (int64_t t = T - 1; t >= 0; --t) {
            const int is_term = flag_at(te, t);
            const int is_trunc = flag_at(tr, t) && !is_term;
            const double d = (is_term || flag_at(tr, t)) ? 1.0 : 0.0;
            const double w = is_trunc ? 1.0 : (1.0 - lambda);
            const double G = rr[t] + gamma * w * successor(vv, te, tr, bb, B, t, T)
                           + gamma * lambda * (1.0 - d) * G_next;
            ret[n * T + t] = G;
            G_next = G;
        }
    }
}

/* Discounted returns, Table 1 and Section 3.3.4 (lambda = 1 with no value function):
 *   G_t = r_t + gamma * (1 - d_t) * G_{t+1},  G_T = B,
 *   plus gamma * bv_t at a truncated step, where the carry is cut.                          */
void oracle_discounted(const double* r, const uint8_t* term, const uint8_t* trunc,
                       const double* bv, const double* boot, double* ret,
                       int64_t N, int64_t T, double gamma) {
    for (int64_t n = 0; n < N; ++n) {
        const double* rr = r + n * T;
        const uint8_t* te = row_of_flags(term, n, T);
        const uint8_t* tr = row_of_flags(trunc, n, T);
        const double* bb = row_of(bv, n, T);
        const double B = boot ? boot[n] : 0.0;
        double G_next = B;
        for (int64_t t = T - 1; t >= 0; --t) {
            const int is_term = flag_at(te, t);
            const int is_trunc = flag_at(tr, t) && !is_term;
            const double d = (is_term || flag_at(tr, t)) ? 1.0 : 0.0;
            const double cont = is_trunc ? bb[t] : 0.0;
            const double G = rr[t] + gamma * cont + gamma * (1.0 - d) * G_next;
            ret[n * T + t] = G;
            G_next = G;
        }
    }
}

/* V-Trace, Table 1 and Section 3.3.2:
 *   rho_t = min(rho_bar, exp(log_rho_t)),  c_t = min(c_bar, exp(log_rho_t)),
 *   Delta_t = rho_t (r_t + gamma succ(V)_t - V_t) + gamma c_t (1 - d_t) Delta_{t+1}, Delta_T = 0,
 *   vs_t = Delta_t + V_t,
 *   pg_t = rho_t (r_t + gamma succ(vs)_t - V_t).                                            */
void oracle_vtrace(const double* r, const double* v, const double* log_rho,
                   const uint8_t* term, const uint8_t* trunc, const double* bv,
                   const double* boot, double* vs, double* pg,
                   int64_t N, int64_t T, double gamma, double rho_bar, double c_bar) {
    for (int64_t n = 0; n < N; ++n) {
        const double* rr = r + n * T;
        const double* vv = v + n * T;
        const double* lr = log_rho + n * T;
        const uint8_t* te = row_of_flags(term, n, T);
        const uint8_t* tr = row_of_flags(trunc, n, T);
        const double* bb = row_of(bv, n, T);
        const double B = boot ? boot[n] : 0.0;
        double* vs_row = vs + n * T;
        double Delta_next = 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            const double ratio = exp(lr[t]);
            const double rho = fmin(rho_bar, ratio);
            const double c = fmin(c_bar, ratio);
            const double d = (flag_at(te, t) || flag_at(tr, t)) ? 1.0 : 0.0;
            const double dv = rho * (rr[t] + gamma * successor(vv, te, tr, bb, B, t, T) - vv[t]);
            const double Delta = dv + gamma * c * (1.0 - d) * Delta_next;
            vs_row[t] = Delta + vv[t];
            Delta_next = Delta;
        }
        for (int64_t t = 0; t < T; ++t) {
            const double rho = fmin(rho_bar, exp(lr[t]));
            pg[n * T + t] = rho * (rr[t] + gamma * successor(vs_row, te, tr, bb, B, t, T) - vv[t]);
        }
    }
}

/* The Retrace(lambda) recurrence of one row given its per-step terms (Table 1 and
 * Section 3.3.3): with c_T = 0,
 *   delta_t = r_t + gamma succ(E_pi Q)_t - Q(s_t, a_t),
 *   Delta_t = delta_t + gamma c_{t+1} (1 - d_t) Delta_{t+1},  Delta_T = 0,
 *   Q_ret_t = Q(s_t, a_t) + Delta_t.                                                          */
static void retrace_row(const double* rr, const double* qq, const double* ee, const double* cc,
                        const uint8_t* te, const uint8_t* tr, const double* bb, double B,
                        double* delta, double* q_ret, int64_t T, double gamma) {
    double Delta_next = 0.0;
    double c_next = 0.0; /* c_T = 0 */
    for (int64_t t = T - 1; t >= 0; --t) {
        const double d = (flag_at(te, t) || flag_at(tr, t)) ? 1.0 : 0.0;
        const double td = rr[t] + gamma * successor(ee, te, tr, bb, B, t, T) - qq[t];
        const double Delta = td + gamma * c_next * (1.0 - d) * Delta_next;
        delta[t] = Delta;
        q_ret[t] = qq[t] + Delta;
        Delta_next = Delta;
        c_next = cc[t];
    }
}

/* Retrace(lambda), Table 1 and Section 3.3.3, with c_t = lambda * min(c_bar, exp(log_rho_t)).
 * The row bootstrap is E_pi Q(s_T, .).                                                      */
void oracle_retrace(const double* r, const double* q, const double* eq, const double* log_rho,
                    const uint8_t* term, const uint8_t* trunc, const double* bv,
                    const double* boot, double* delta, double* q_ret,
                    int64_t N, int64_t T, double gamma, double lambda, double c_bar) {
    double* c = (double*)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
    if (!c) return;
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t t = 0; t < T; ++t) c[t] = lambda * fmin(c_bar, exp(log_rho[n * T + t]));
        retrace_row(r + n * T, q + n * T, eq + n * T, c, row_of_flags(term, n, T),
                    row_of_flags(trunc, n, T), row_of(bv, n, T), boot ? boot[n] : 0.0,
                    delta + n * T, q_ret + n * T, T, gamma);
    }
    free(c);
}

/* Full-form Retrace (Sections 3.3.3 and 7.3): the per-step terms come from the [N, T, A]
 * Q-values and target-policy probabilities, the taken actions and the behaviour
 * probabilities of the taken actions:
 *   E_pi Q(s_t) = sum_a pi(a|s_t) Q(s_t, a),  Q(s_t, a_t),
 *   rho_t = pi(a_t|s_t) / mu(a_t|s_t),  c_t = lambda * min(c_bar, rho_t).                    */
void oracle_retrace_full(const double* r, const double* q, const double* pi,
                         const int32_t* actions, const double* mu, const uint8_t* term,
                         const uint8_t* trunc, const double* bv, const double* boot,
                         double* delta, double* q_ret, int64_t N, int64_t T, int64_t A,
                         double gamma, double lambda, double c_bar) {
    const size_t n_t = (size_t)(T > 0 ? T : 1);
    double* c = (double*)malloc(sizeof(double) * n_t);
    double* qa = (double*)malloc(sizeof(double) * n_t);
    double* eq = (double*)malloc(sizeof(double) * n_t);
    if (!c || !qa || !eq) { free(c); free(qa); free(eq); return; }
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t t = 0; t < T; ++t) {
            const double* qs = q + (n * T + t) * A;
            const double* ps = pi + (n * T + t) * A;
            const int32_t a = actions[n * T + t];
            double e = 0.0;
            for (int64_t k = 0; k < A; ++k) e += ps[k] * qs[k];
            const int in_range = a >= 0 && a < A;
            const double q_taken = in_range ? qs[a] : 0.0;
            const double pi_taken = in_range ? ps[a] : 0.0;
            eq[t] = e;
            qa[t] = q_taken;
            c[t] = lambda * fmin(c_bar, pi_taken / mu[n * T + t]);
        }
        retrace_row(r + n * T, qa, eq, c, row_of_flags(term, n, T), row_of_flags(trunc, n, T),
                    row_of(bv, n, T), boot ? boot[n] : 0.0, delta + n * T, q_ret + n * T, T,
                    gamma);
    }
    free(c); free(qa); free(eq);
}

/* Eligibility traces (forward), Table 1 and Section 3.3.5:
 *   z_t = gamma * lambda * (1 - d_{t-1}) * z_{t-1} + x_t,  d_{-1} = 0, z_{-1} = 0.           */
void oracle_elig_trace(const double* x, const uint8_t* term, const uint8_t* trunc, double* z,
                       int64_t N, int64_t T, double gamma, double lambda) {
    for (int64_t n = 0; n < N; ++n) {
        const double* xx = x + n * T;
        const uint8_t* te = row_of_flags(term, n, T);
        const uint8_t* tr = row_of_flags(trunc, n, T);
        double z_prev = 0.0;
        double d_prev = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            const double zt = gamma * lambda * (1.0 - d_prev) * z_prev + xx[t];
            z[n * T + t] = zt;
            z_prev = zt;
            d_prev = (flag_at(te, t) || flag_at(tr, t)) ? 1.0 : 0.0;
        }
    }
}

/* Vector eligibility traces (forward), Section 3.3.5 with a feature vector per step:
 *   z_t = gamma * lambda * (1 - d_{t-1}) * z_{t-1} + x_t,  z_{-1} = 0,  d_{-1} = 0,
 * where x_t and z_t are F-vectors ([N, T, F], features innermost) and the scalar coefficient
 * of a step (flags [N, T]) multiplies every feature alike. Features are walked one at a time. */
void oracle_elig_trace_vec(const double* x, const uint8_t* term, const uint8_t* trunc, double* z,
                           int64_t N, int64_t T, int64_t F, double gamma, double lambda) {
    for (int64_t n = 0; n < N; ++n) {
        const uint8_t* te = row_of_flags(term, n, T);
        const uint8_t* tr = row_of_flags(trunc, n, T);
        for (int64_t f = 0; f < F; ++f) {
            double z_prev = 0.0;
            double d_prev = 0.0;
            for (int64_t t = 0; t < T; ++t) {
                const int64_t i = (n * T + t) * F + f;
                const double zt = gamma * lambda * (1.0 - d_prev) * z_prev + x[i];
                z[i] = zt;
                z_prev = zt;
                d_prev = (flag_at(te, t) || flag_at(tr, t)) ? 1.0 : 0.0;
            }
        }
    }
}

/* Episodic prefix sum (forward), Table 1 and Section 3.3.6:
 *   ends_at:   C_t = x_t + (1 - d_{t-1}) C_{t-1},  d_{-1} = 0,
 *   starts_at: C_t = x_t + (1 - d_t) C_{t-1},
 *   C_{-1} = 0.                                                                             */
void oracle_episodic_prefix(const double* x, const uint8_t* term, const uint8_t* trunc,
                            double* c, int64_t N, int64_t T, int starts_at) {
    for (int64_t n = 0; n < N; ++n) {
        const double* xx = x + n * T;
        const uint8_t* te = row_of_flags(term, n, T);
        const uint8_t* tr = row_of_flags(trunc, n, T);
        double C_prev = 0.0;
        double d_prev = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            const double d_t = (flag_at(te, t) || flag_at(tr, t)) ? 1.0 : 0.0;
            const double keep = starts_at ? (1.0 - d_t) : (1.0 - d_prev);
            const double C = xx[t] + keep * C_prev;
            c[n * T + t] = C;
            C_prev = C;
            d_prev = d_t;
        }
    }
}

/* The bare recurrence of Eq. 1 with supplied coefficients (the generic scan of Section 4.1). */
void oracle_affine_scan(const double* alpha, const double* beta, const double* carry,
                        double* out, int64_t N, int64_t T, int reverse) {
    for (int64_t n = 0; n < N; ++n) {
        const double* a = alpha + n * T;
        const double* b = beta + n * T;
        double A = carry ? carry[n] : 0.0;
        if (reverse) {
            for (int64_t t = T - 1; t >= 0; --t) {
                A = a[t] + b[t] * A;
                out[n * T + t] = A;
            }
        } else {
            for (int64_t t = 0; t < T; ++t) {
                A = a[t] + b[t] * A;
                out[n * T + t] = A;
            }
        }
    }
}
