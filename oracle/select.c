/*
 * CPU oracle: runtime server-expert selection of one MoE layer.
 * TEST INFRASTRUCTURE ONLY -- used by tests/, the smoke check and the CPU
 * baseline of the benchmark; never by the library's product path.
 *
 * Follows Section V of the paper for a single layer l:
 *   - location s (eq 36) enters as loc_in, accumulated loss Qhat as qhat_in;
 *   - feasible execution set V_{l,r} = {r} U R_{l,r} (eq 7-8), where R_{l,r}
 *     holds the experts k != r of r's similarity group with Sim(r,k) >= theta;
 *   - substitution loss Q(r,k) = (1 - Sim(r,k)) / 2 with phi = identity (eq 18);
 *   - budget-feasible candidate set A (eq 40): x[m][k] = 1, k in V, and
 *     Qhat + Q(r,k) <= Qbar;
 *   - selection (eq 43): argmin over A of J = S[s][m][k] + (omega_Q/Qbar) * Q,
 *     where S[s][m][k] already holds omega_T * d(m,k | s) / d_ref plus the
 *     look-ahead cost-to-go (eq 37-38, 42) in fp32;
 *   - update (eq 44): s <- m*, Qhat <- Qhat + Q(r, k*).
 *
 * Readings for top-k layers (the paper is top-1): every rank slot of a token
 * is one decision, taken in rank order, sharing the token's budget; the token
 * resides on slot 0's execution server after the layer.  Ties in J are broken
 * by (Q, exact before substitute, k, local before remote, m).  With
 * pin_local_exact a target deployed on the token's own server is kept there
 * without a search.  With allow_sub = 0 or Qbar = 0 only exact execution is a
 * candidate.
 *
 * All decision arithmetic is fp32 with an explicit fmaf for J, the same
 * operations the paper's formulas name, so that results do not depend on
 * compiler contraction (built with -ffp-contract=off).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

enum { CLS_LOCAL_EXACT = 0, CLS_LOCAL_SUB = 1, CLS_REMOTE_EXACT = 2, CLS_REMOTE_SUB = 3 };

typedef struct {
    float J, q;
    int sub, k, remote, m;
} cand_t;

/* lexicographic order of eq 43's argmin with the tie-break reading above */
static int cand_less(const cand_t* a, const cand_t* b) {
    if (a->J != b->J) return a->J < b->J;
    if (a->q != b->q) return a->q < b->q;
    if (a->sub != b->sub) return a->sub < b->sub;
    if (a->k != b->k) return a->k < b->k;
    if (a->remote != b->remote) return a->remote < b->remote;
    return a->m < b->m;
}

/* Returns 0 on success, -1 if some slot has an empty candidate set (a
 * deployment violating eq 2), -2 on bad arguments. */
int orc_select(int64_t T, int32_t k, int32_t E, int32_t M,
               const int32_t* idx,      /* [T][k] routed targets in rank order */
               const uint8_t* x,        /* [M][E] deployment x_{m,l,j} */
               const float* sim,        /* [E][E] Sim_l (fp32) */
               const int32_t* group_of, /* [E] similarity group id */
               float theta,             /* theta_l */
               const float* S,          /* [M][M][E] static cost, fp32 */
               float Qbar, float omega_Q,
               int32_t pin_local_exact, int32_t allow_sub,
               const uint8_t* loc_in,   /* [T] s_{q,l} */
               const float* qhat_in,    /* [T] Qhat_{q,l} */
               int32_t* exec_k,         /* [T][k] */
               uint8_t* exec_m,         /* [T][k] */
               uint8_t* cls,            /* [T][k] */
               float* qhat_out,         /* [T] */
               uint8_t* loc_out)        /* [T] */
{
    if (T < 0 || k <= 0 || E <= 0 || M <= 0 || M > 255) return -2;
    const float cq = (Qbar > 0.0f) ? omega_Q / Qbar : 0.0f;
    const int subs_on = allow_sub && Qbar > 0.0f;
    int bad = 0;

#pragma omp parallel for schedule(static) reduction(| : bad)
    for (int64_t t = 0; t < T; ++t) {
        const int s = loc_in[t];
        float qhat = qhat_in[t];
        int first_m = s;
        for (int slot = 0; slot < k; ++slot) {
            const int r = idx[t * k + slot];
            cand_t best;
            int have = 0;
            if (pin_local_exact && x[(int64_t)s * E + r]) {
                best.J = 0.0f; best.q = 0.0f; best.sub = 0; best.k = r; best.remote = 0; best.m = s;
                have = 1;
            } else {
                for (int kk = 0; kk < E; ++kk) {
                    const int is_sub = (kk != r);
                    float q = 0.0f;
                    if (is_sub) {
                        if (!subs_on) continue;
                        if (group_of[kk] != group_of[r]) continue;
                        if (!(sim[(int64_t)r * E + kk] >= theta)) continue;
                        q = (1.0f - sim[(int64_t)r * E + kk]) * 0.5f;
                        if (!(qhat + q <= Qbar)) continue;
                    }
                    for (int m = 0; m < M; ++m) {
                        if (!x[(int64_t)m * E + kk]) continue;
                        if (is_sub && allow_sub == 2 && m != s) continue;   /* local substitutes only */
                        cand_t c;
                        c.J = fmaf(cq, q, S[((int64_t)s * M + m) * E + kk]);
                        c.q = q; c.sub = is_sub; c.k = kk; c.remote = (m != s); c.m = m;
                        if (!have || cand_less(&c, &best)) { best = c; have = 1; }
                    }
                }
            }
            if (!have) {
                bad = 1;
                exec_k[t * k + slot] = -1; exec_m[t * k + slot] = 255; cls[t * k + slot] = 255;
                continue;
            }
            exec_k[t * k + slot] = best.k;
            exec_m[t * k + slot] = (uint8_t)best.m;
            cls[t * k + slot] = (uint8_t)((best.remote ? 2 : 0) | (best.sub ? 1 : 0));
            qhat = qhat + best.q;
            if (slot == 0) first_m = best.m;
        }
        qhat_out[t] = qhat;
        loc_out[t] = (uint8_t)first_m;
    }
    return bad ? -1 : 0;
}
