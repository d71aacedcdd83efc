// Host-side parts of OrderMoE: layer-aware grouping (eq 24-28), importance-
// aware deployment (Algorithm 1, eq 29-35), per-layer decision tables
// (eq 6-8, 18, 37-38) and the look-ahead cost-to-go (eq 41-42).
//
// All of this is offline, small (E <= 256, M <= 32) and integer or double
// arithmetic, so it runs on the CPU; the results are uploaded once and read by
// the route/select kernel.

#include <algorithm>
#include <cmath>
#include <limits>
#include <numeric>
#include <string>
#include <vector>

#include "common.hpp"

using namespace ordermoe;

extern "C" int ordermoe_group_experts(int32_t E, const float* sim, const int64_t* counts,
                                      float theta, double alpha_f, int32_t* group_of,
                                      int32_t* centres, int32_t* num_groups,
                                      double* importance) {
    if (E < 1 || E > ORDERMOE_MAX_EXPERTS) return fail(ORDERMOE_EINVAL, "group_experts: E out of range");
    if (!sim || !counts || !group_of || !centres || !num_groups || !importance)
        return fail(ORDERMOE_EINVAL, "group_experts: null pointer");
    if (!(alpha_f >= 0.0 && alpha_f <= 1.0))
        return fail(ORDERMOE_EINVAL, "group_experts: alpha_f must lie in [0, 1]");

    // visiting order: decreasing activation count, ties to the lower index (eq 5 ordering)
    std::vector<int> order(E);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return counts[a] > counts[b]; });

    std::vector<int> dom;  // dominant experts in creation order
    std::vector<int> g(E, -1);
    for (int j : order) {
        int best = -1;
        float best_s = 0.f;
        for (int c = 0; c < (int)dom.size(); ++c) {
            float s = sim[(size_t)j * E + dom[c]];
            if (best < 0 || s > best_s) { best = c; best_s = s; }
        }
        if (best < 0 || best_s < theta) {  // eq 24: strictly below the threshold
            dom.push_back(j);
            g[j] = (int)dom.size() - 1;
        } else {
            g[j] = best;                   // eq 25
        }
    }

    int64_t tot = 0;
    for (int j = 0; j < E; ++j) tot += counts[j];
    std::vector<int> gsize(dom.size(), 0);
    for (int j = 0; j < E; ++j) gsize[g[j]]++;
    for (int j = 0; j < E; ++j) {
        double acc = 0.0;
        for (int kk = 0; kk < E; ++kk)
            if (g[kk] == g[j]) acc += (double)sim[(size_t)j * E + kk];
        double rho = acc / gsize[g[j]];                              // eq 27
        double f = tot > 0 ? (double)counts[j] / (double)tot : 0.0;  // eq 5
        importance[j] = alpha_f * f + (1.0 - alpha_f) * rho;         // eq 28
        group_of[j] = g[j];
    }
    for (int c = 0; c < E; ++c) centres[c] = c < (int)dom.size() ? dom[c] : -1;
    *num_groups = (int32_t)dom.size();
    clear_error();
    return ORDERMOE_OK;
}

extern "C" int ordermoe_place(int32_t N, const int32_t* E_l, int32_t M, const int32_t* group_of,
                              const double* importance, const double* p, const double* C,
                              const double* pi, double lambda1, int32_t redundancy,
                              uint8_t* x_out, double* used_out) {
    if (N < 1 || M < 1 || M > ORDERMOE_MAX_SERVERS) return fail(ORDERMOE_EINVAL, "place: N or M out of range");
    if (!E_l || !group_of || !importance || !p || !C || !pi || !x_out || !used_out)
        return fail(ORDERMOE_EINVAL, "place: null pointer");
    if (redundancy < 0 || redundancy > 2) return fail(ORDERMOE_EINVAL, "place: redundancy must be 0, 1 or 2");
    std::vector<size_t> base(N + 1, 0);
    for (int l = 0; l < N; ++l) {
        if (E_l[l] < 1 || E_l[l] > ORDERMOE_MAX_EXPERTS) return fail(ORDERMOE_EINVAL, "place: E_l out of range");
        base[l + 1] = base[l] + (size_t)E_l[l];
    }
    double need = 0.0, have = 0.0;
    for (size_t i = 0; i < base[N]; ++i) {
        if (!(p[i] > 0.0)) return fail(ORDERMOE_EINVAL, "place: memory demand p must be positive");
        need += p[i];
    }
    for (int m = 0; m < M; ++m) {
        if (!(C[m] > 0.0)) return fail(ORDERMOE_EINVAL, "place: capacity C must be positive");
        have += C[m];
    }
    if (need > have) return fail(ORDERMOE_ECAPACITY, "place: total expert memory exceeds total capacity");

    const double lambda2 = 1.0 - lambda1;
    std::vector<double> b(M, 0.0);
    // x[l] is [M][E_l] at offset M * base[l]
    std::vector<uint8_t> x((size_t)M * base[N], 0);
    auto X = [&](int l, int m, int j) -> uint8_t& { return x[(size_t)M * base[l] + (size_t)m * E_l[l] + j]; };

    for (int l = 0; l < N; ++l) {
        const int E = E_l[l];
        const int32_t* g = group_of + base[l];
        const double* pl = p + base[l];
        std::vector<int> order(E);
        std::iota(order.begin(), order.end(), 0);
        std::stable_sort(order.begin(), order.end(), [&](int a, int c) { return pl[a] > pl[c]; });
        std::vector<int> waiting;
        // eta[m][group] = experts of that group already on m in this layer
        int G = 0;
        for (int j = 0; j < E; ++j) G = std::max(G, g[j] + 1);
        std::vector<int> eta((size_t)M * G, 0);
        for (int j : order) {
            int best = -1;
            double best_score = 0.0;
            for (int m = 0; m < M; ++m) {
                if (!(b[m] + pl[j] <= C[m])) continue;                              // eq 29
                double score = lambda1 * b[m] / C[m] + lambda2 * eta[(size_t)m * G + g[j]];  // eq 30
                if (best < 0 || score < best_score) { best = m; best_score = score; }       // eq 31
            }
            if (best < 0) { waiting.push_back(j); continue; }
            X(l, best, j) = 1;
            b[best] += pl[j];
            eta[(size_t)best * G + g[j]]++;
        }
        for (int j : waiting) {
            int best = 0;
            for (int m = 1; m < M; ++m)
                if (C[m] - b[m] > C[best] - b[best]) best = m;
            X(l, best, j) = 1;
            b[best] += pl[j];
            eta[(size_t)best * G + g[j]]++;
        }
    }

    if (redundancy) {
        for (;;) {
            double bestB = 0.0;
            int bl = -1, bm = -1, bj = -1;
            for (int l = 0; l < N; ++l) {
                const int E = E_l[l];
                const int32_t* g = group_of + base[l];
                int G = 0;
                for (int j = 0; j < E; ++j) G = std::max(G, g[j] + 1);
                for (int m = 0; m < M; ++m) {
                    std::vector<uint8_t> y(G, 0);                                     // eq 32
                    for (int j = 0; j < E; ++j)
                        if (X(l, m, j)) y[g[j]] = 1;
                    for (int j = 0; j < E; ++j) {
                        const double pj = p[base[l] + j];
                        if (X(l, m, j) || !(b[m] + pj <= C[m])) continue;             // eq 35
                        // eq 33; redundancy = 2 drops the group-coverage factor (popularity replication)
                        double B = redundancy == 2 ? pi[m] * importance[base[l] + j] / pj
                                                   : pi[m] * importance[base[l] + j] * (1 - y[g[j]]) / pj;
                        if (!(B > 0.0)) continue;
                        if (bl < 0 || B > bestB) { bestB = B; bl = l; bm = m; bj = j; }
                    }
                }
            }
            if (bl < 0) break;
            X(bl, bm, bj) = 1;
            b[bm] += p[base[bl] + bj];
        }
    }
    std::copy(x.begin(), x.end(), x_out);
    for (int m = 0; m < M; ++m) used_out[m] = b[m];
    clear_error();
    return ORDERMOE_OK;
}

static double step_delay(int s, int m, int k, int M, double z_bits, const double* B,
                         const double* tau, const double* c, const double* F) {
    // eq 37: transfer only when the execution server differs from the location
    double trans = (s != m) ? (z_bits / B[(size_t)s * M + m] + tau[(size_t)s * M + m]) : 0.0;
    return trans + c[k] / F[m];
}

extern "C" int ordermoe_build_tables(int32_t E, int32_t M, const float* sim,
                                     const int32_t* group_of, float theta, const uint8_t* x,
                                     const double* B, const double* tau, const double* F,
                                     double z_bits, const double* c, double d_ref,
                                     double omega_T, const double* phi, int32_t gmax,
                                     int32_t* t1_k, float* t1_q, int32_t* t1_n,
                                     uint32_t* srvmask, float* S) {
    if (E < 1 || E > ORDERMOE_MAX_EXPERTS || M < 1 || M > ORDERMOE_MAX_SERVERS)
        return fail(ORDERMOE_EINVAL, "build_tables: E or M out of range");
    if (gmax < 1 || gmax > ORDERMOE_MAX_SUBS) return fail(ORDERMOE_EINVAL, "build_tables: gmax out of range");
    if (!sim || !group_of || !x || !B || !tau || !F || !c || !t1_k || !t1_q || !t1_n || !srvmask || !S)
        return fail(ORDERMOE_EINVAL, "build_tables: null pointer");
    if (!(d_ref > 0.0)) return fail(ORDERMOE_EINVAL, "build_tables: d_ref must be positive");
    for (int m = 0; m < M; ++m)
        if (!(F[m] > 0.0)) return fail(ORDERMOE_EINVAL, "build_tables: F must be positive");

    std::vector<uint32_t> mask(E, 0);
    for (int j = 0; j < E; ++j) {
        for (int m = 0; m < M; ++m)
            if (x[(size_t)m * E + j]) mask[j] |= (1u << m);
        if (!mask[j])
            return fail(ORDERMOE_EINVAL, "build_tables: expert " + std::to_string(j) +
                                             " is deployed on no server (eq 2)");
    }
    std::vector<int32_t> tk((size_t)E * gmax, -1);
    std::vector<float> tq((size_t)E * gmax, std::numeric_limits<float>::infinity());
    std::vector<int32_t> tn(E, 0);
    for (int r = 0; r < E; ++r) {
        std::vector<std::pair<float, int>> subs;
        for (int k = 0; k < E; ++k) {
            if (k == r || group_of[k] != group_of[r]) continue;
            const float s = sim[(size_t)r * E + k];
            if (!(s >= theta)) continue;                               // eq 7
            subs.push_back({(1.0f - s) * 0.5f, k});                    // eq 18
        }
        std::sort(subs.begin(), subs.end());
        if ((int)subs.size() > gmax)
            return fail(ORDERMOE_EINVAL, "build_tables: target " + std::to_string(r) + " has " +
                                             std::to_string(subs.size()) + " substitutes > gmax");
        tn[r] = (int32_t)subs.size();
        for (size_t i = 0; i < subs.size(); ++i) {
            tk[(size_t)r * gmax + i] = subs[i].second;
            tq[(size_t)r * gmax + i] = subs[i].first;
        }
    }
    for (int s = 0; s < M; ++s)
        for (int m = 0; m < M; ++m)
            for (int k = 0; k < E; ++k) {
                double v = omega_T * step_delay(s, m, k, M, z_bits, B, tau, c, F) / d_ref;  // eq 38
                if (phi) v = v + phi[(size_t)m * E + k];
                S[((size_t)s * M + m) * E + k] = (float)v;
            }
    std::copy(tk.begin(), tk.end(), t1_k);
    std::copy(tq.begin(), tq.end(), t1_q);
    std::copy(tn.begin(), tn.end(), t1_n);
    std::copy(mask.begin(), mask.end(), srvmask);
    clear_error();
    return ORDERMOE_OK;
}

extern "C" int ordermoe_build_lookahead(int32_t N, int32_t E, int32_t M, int32_t H,
                                        const double* P, const uint8_t* x, const float* sim,
                                        const int32_t* group_of, const float* theta,
                                        const double* z_bits, const double* c,
                                        const double* d_ref, const double* B,
                                        const double* tau, const double* F, double omega_T,
                                        double omega_Q, float Qbar, int32_t pin_local_exact,
                                        int32_t allow_sub, double* phi_out) {
    if (N < 1 || E < 1 || E > ORDERMOE_MAX_EXPERTS || M < 1 || M > ORDERMOE_MAX_SERVERS || H < 1)
        return fail(ORDERMOE_EINVAL, "build_lookahead: size out of range");
    if ((N > 1 && !P) || !x || !sim || !group_of || !theta || !z_bits || !c || !d_ref || !B || !tau ||
        !F || !phi_out)
        return fail(ORDERMOE_EINVAL, "build_lookahead: null pointer");
    if (allow_sub < 0 || allow_sub > 2) return fail(ORDERMOE_EINVAL, "build_lookahead: allow_sub must be 0, 1 or 2");
    const size_t ME = (size_t)M * E;
    // cost of the best next-layer candidate of target r1 at layer l1 from source s,
    // plus that candidate's own cost-to-go (eq 42's inner minimum)
    auto best_next = [&](int l1, int s, int r1, const std::vector<double>& nxt) {
        const uint8_t* xl = x + (size_t)l1 * ME;
        const float* sl = sim + (size_t)l1 * E * E;
        const int32_t* gl = group_of + (size_t)l1 * E;
        const double* cl = c + (size_t)l1 * E;
        auto g_of = [&](int m1, int k1) {
            double q = 0.0;
            if (k1 != r1) q = (double)((1.0f - sl[(size_t)r1 * E + k1]) * 0.5f);
            double v = omega_T * step_delay(s, m1, k1, M, z_bits[l1], B, tau, cl, F) / d_ref[l1];
            if (Qbar > 0.0f) v += omega_Q * q / (double)Qbar;
            return v + nxt[(size_t)m1 * E + k1];
        };
        if (pin_local_exact && xl[(size_t)s * E + r1]) return g_of(s, r1);
        bool have = false;
        double best = 0.0;
        for (int k1 = 0; k1 < E; ++k1) {
            if (k1 != r1) {
                if (!(allow_sub && Qbar > 0.0f)) continue;
                if (gl[k1] != gl[r1] || !(sl[(size_t)r1 * E + k1] >= theta[l1])) continue;
            }
            for (int m1 = 0; m1 < M; ++m1) {
                if (!xl[(size_t)m1 * E + k1]) continue;
                if (allow_sub == 2 && k1 != r1 && m1 != s) continue;   // local substitutes only
                double v = g_of(m1, k1);
                if (!have || v < best) { best = v; have = true; }
            }
        }
        return have ? best : 0.0;
    };
    // phi[h][l] for h = 0..H-1, computed bottom-up over h
    std::vector<std::vector<double>> prev(N, std::vector<double>(ME, 0.0)), cur;
    for (int h = 1; h <= H - 1; ++h) {
        cur.assign(N, std::vector<double>(ME, 0.0));
        for (int l = 0; l + 1 < N; ++l) {
            std::vector<double> V(ME, 0.0);
            for (int m = 0; m < M; ++m)
                for (int r1 = 0; r1 < E; ++r1) V[(size_t)m * E + r1] = best_next(l + 1, m, r1, prev[l + 1]);
            const double* Pl = P + (size_t)l * E * E;
            for (int m = 0; m < M; ++m)
                for (int k = 0; k < E; ++k) {
                    double acc = 0.0;
                    for (int r1 = 0; r1 < E; ++r1) acc += Pl[(size_t)k * E + r1] * V[(size_t)m * E + r1];
                    cur[l][(size_t)m * E + k] = acc;
                }
        }
        prev.swap(cur);
    }
    for (int l = 0; l < N; ++l) std::copy(prev[l].begin(), prev[l].end(), phi_out + (size_t)l * ME);
    clear_error();
    return ORDERMOE_OK;
}

extern "C" int ordermoe_estimate_transitions(int32_t N, int32_t E, int64_t T_cal,
                                             const int32_t* top1, double* P_out) {
    if (N < 1 || E < 1 || E > ORDERMOE_MAX_EXPERTS || T_cal < 0)
        return fail(ORDERMOE_EINVAL, "estimate_transitions: size out of range");
    if (N == 1) { clear_error(); return ORDERMOE_OK; }
    if (!top1 || !P_out) return fail(ORDERMOE_EINVAL, "estimate_transitions: null pointer");
    for (int64_t i = 0; i < (int64_t)N * T_cal; ++i)
        if (top1[i] < 0 || top1[i] >= E) return fail(ORDERMOE_EINVAL, "estimate_transitions: expert id out of range");
    const size_t EE = (size_t)E * E;
    std::vector<int64_t> n(EE);
    for (int l = 0; l + 1 < N; ++l) {
        std::fill(n.begin(), n.end(), 0);
        const int32_t* a = top1 + (size_t)l * T_cal;
        const int32_t* b = a + T_cal;
        for (int64_t t = 0; t < T_cal; ++t) ++n[(size_t)a[t] * E + b[t]];
        double* P = P_out + (size_t)l * EE;
        for (int k = 0; k < E; ++k) {
            int64_t tot = 0;
            for (int k1 = 0; k1 < E; ++k1) tot += n[(size_t)k * E + k1];
            for (int k1 = 0; k1 < E; ++k1)
                P[(size_t)k * E + k1] = tot > 0 ? (double)n[(size_t)k * E + k1] / (double)tot : 0.0;
        }
    }
    clear_error();
    return ORDERMOE_OK;
}

extern "C" int ordermoe_theta_layer(int32_t l, int32_t N, double theta_min, double theta_max,
                                    float* theta_out) {
    if (N < 1 || l < 1 || l > N || !(theta_min <= theta_max) || !theta_out)
        return fail(ORDERMOE_EINVAL, "theta_layer: need 1 <= l <= N and theta_min <= theta_max");
    const double lo = theta_min, hi = theta_max;
    *theta_out = N == 1 ? (float)(0.5 * (lo + hi))
                        : (float)(lo + (hi - lo) * (double)(N - l) / (double)(N - 1));
    clear_error();
    return ORDERMOE_OK;
}

extern "C" int ordermoe_adapt_weights(double omega_Q, double kappa, double T_bar, double Q_bar,
                                      double* omega_Q_out, double* omega_T_out) {
    if (!omega_Q_out || !omega_T_out || !(omega_Q >= 0.0 && omega_Q <= 1.0) || !(kappa >= 0.0) ||
        !std::isfinite(kappa) || !(T_bar >= 0.0) || !std::isfinite(T_bar) || !(Q_bar >= 0.0) ||
        !std::isfinite(Q_bar))
        return fail(ORDERMOE_EINVAL, "adapt_weights: need omega_Q in [0,1], kappa >= 0, finite T_bar, Q_bar >= 0");
    // eq 45: a projected step on omega_Q towards the objective that is further behind
    double w = omega_Q + kappa * (Q_bar - T_bar);
    w = w < 0.0 ? 0.0 : (w > 1.0 ? 1.0 : w);
    *omega_Q_out = w;
    *omega_T_out = 1.0 - w;
    clear_error();
    return ORDERMOE_OK;
}

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): the state advances by the
// golden-ratio constant, the output is a two-multiply mix of the state.
namespace {
struct SplitMix64 {
    uint64_t state;
    uint64_t next() {
        uint64_t z = (state += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    uint64_t below(uint64_t n) { return next() % n; }
};
}  // namespace

extern "C" int ordermoe_place_random(int32_t N, const int32_t* E_l, int32_t M, const double* p, const double* C,
                                     uint64_t seed, int32_t redundancy, uint8_t* x_out, double* used_out) {
    if (N < 1 || M < 1 || M > ORDERMOE_MAX_SERVERS) return fail(ORDERMOE_EINVAL, "place_random: N or M out of range");
    if (!E_l || !p || !C || !x_out || !used_out) return fail(ORDERMOE_EINVAL, "place_random: null pointer");
    std::vector<size_t> base(N + 1, 0);
    for (int l = 0; l < N; ++l) {
        if (E_l[l] < 1 || E_l[l] > ORDERMOE_MAX_EXPERTS) return fail(ORDERMOE_EINVAL, "place_random: E_l out of range");
        base[l + 1] = base[l] + (size_t)E_l[l];
    }
    double need = 0.0, have = 0.0;
    for (size_t i = 0; i < base[N]; ++i) {
        if (!(p[i] > 0.0)) return fail(ORDERMOE_EINVAL, "place_random: memory demand p must be positive");
        need += p[i];
    }
    for (int m = 0; m < M; ++m) {
        if (!(C[m] > 0.0)) return fail(ORDERMOE_EINVAL, "place_random: capacity C must be positive");
        have += C[m];
    }
    if (need > have) return fail(ORDERMOE_ECAPACITY, "place_random: total expert memory exceeds total capacity");
    SplitMix64 rng{seed};
    std::vector<double> b(M, 0.0);
    std::vector<uint8_t> x((size_t)M * base[N], 0);
    auto X = [&](int l, int m, int j) -> uint8_t& { return x[(size_t)M * base[l] + (size_t)m * E_l[l] + j]; };
    // every expert once, on a uniformly drawn memory-feasible server (none: the
    // server with the most remaining memory, ties to the lower index)
    std::vector<int> feas;
    for (int l = 0; l < N; ++l)
        for (int j = 0; j < E_l[l]; ++j) {
            const double pj = p[base[l] + j];
            feas.clear();
            for (int m = 0; m < M; ++m)
                if (b[m] + pj <= C[m]) feas.push_back(m);
            int m;
            if (!feas.empty()) {
                m = feas[(size_t)rng.below(feas.size())];
            } else {
                m = 0;
                for (int q = 1; q < M; ++q)
                    if (C[q] - b[q] > C[m] - b[m]) m = q;
            }
            X(l, m, j) = 1;
            b[m] += pj;
        }
    // replicas: every (layer, server, expert) without a copy, in an order shuffled
    // by Fisher-Yates, each placed if it fits
    if (redundancy) {
        std::vector<uint64_t> cand;
        for (int l = 0; l < N; ++l)
            for (int m = 0; m < M; ++m)
                for (int j = 0; j < E_l[l]; ++j)
                    if (!X(l, m, j)) cand.push_back(((uint64_t)l << 40) | ((uint64_t)m << 20) | (uint64_t)j);
        for (size_t i = cand.size(); i > 1; --i) std::swap(cand[i - 1], cand[(size_t)rng.below(i)]);
        for (uint64_t c : cand) {
            const int l = (int)(c >> 40), m = (int)((c >> 20) & 0xFFFFF), j = (int)(c & 0xFFFFF);
            const double pj = p[base[l] + j];
            if (b[m] + pj <= C[m]) { X(l, m, j) = 1; b[m] += pj; }
        }
    }
    std::copy(x.begin(), x.end(), x_out);
    std::copy(b.begin(), b.end(), used_out);
    clear_error();
    return ORDERMOE_OK;
}

// Delay, workload and traffic of realized decisions (eq 13-17, eq 22), one
// layer at a time: each token's delay grows by its executed slots' transfer
// (from the location it entered the layer with) and compute terms, then the
// token moves to slot 0's server.
extern "C" int ordermoe_simulate_delay(int32_t N, int64_t T, int32_t k, int32_t M, const int32_t* E_l,
                                       const uint8_t* loc0, const uint8_t* exec_m, const int32_t* exec_k,
                                       const double* c, const double* z_bits, const double* B,
                                       const double* tau, const double* F, double* delay_out,
                                       double* work_out, double* stats_out, uint8_t* loc_out) {
    if (N < 1 || T < 0 || k < 1 || k > ORDERMOE_MAX_TOPK || M < 1 || M > ORDERMOE_MAX_SERVERS)
        return fail(ORDERMOE_EINVAL, "simulate_delay: N, T, k or M out of range");
    if (!E_l || !c || !z_bits || !B || !tau || !F || !delay_out || !work_out || !stats_out ||
        (T > 0 && (!loc0 || !exec_m || !exec_k)))
        return fail(ORDERMOE_EINVAL, "simulate_delay: null pointer");
    std::vector<size_t> cbase(N + 1, 0);
    for (int l = 0; l < N; ++l) {
        if (E_l[l] < 1 || E_l[l] > ORDERMOE_MAX_EXPERTS) return fail(ORDERMOE_EINVAL, "simulate_delay: E_l out of range");
        cbase[l + 1] = cbase[l] + (size_t)E_l[l];
    }
    for (int m = 0; m < M; ++m)
        if (!(F[m] > 0.0)) return fail(ORDERMOE_EINVAL, "simulate_delay: F must be positive");
    // validate every executed slot before writing anything
    {
        std::vector<uint8_t> at(loc0, loc0 + T);
        for (int l = 0; l < N; ++l)
            for (int64_t t = 0; t < T; ++t) {
                if (at[t] >= M) continue;
                const size_t o = ((size_t)l * T + t) * k;
                for (int j = 0; j < k; ++j) {
                    const int m = exec_m[o + j];
                    if (m >= M) continue;
                    if (exec_k[o + j] < 0 || exec_k[o + j] >= E_l[l])
                        return fail(ORDERMOE_EINVAL, "simulate_delay: executed expert out of range");
                    if (m != at[t] && !(B[(size_t)at[t] * M + m] > 0.0))
                        return fail(ORDERMOE_EINVAL, "simulate_delay: B must be positive between servers");
                }
                if (exec_m[o] < M) at[t] = exec_m[o];
            }
    }
    std::vector<uint8_t> at(loc0, loc0 + T);
    std::vector<double> delay(T, 0.0), work(M, 0.0);
    double transfers = 0.0, traffic = 0.0, remote = 0.0, slots = 0.0;
    for (int l = 0; l < N; ++l) {
        const double z = z_bits[l];
        const double* cl = c + cbase[l];
        for (int64_t t = 0; t < T; ++t) {
            if (loc_out) loc_out[(size_t)l * T + t] = at[t];
            const int s = at[t];
            if (s >= M) continue;
            const size_t o = ((size_t)l * T + t) * k;
            uint32_t dest = 0;
            for (int j = 0; j < k; ++j) {
                const int m = exec_m[o + j];
                if (m >= M) continue;
                if (m != s) {
                    delay[t] += z / B[(size_t)s * M + m] + tau[(size_t)s * M + m];   // eq 13 / 14
                    dest |= 1u << m;
                    remote += 1.0;
                }
                delay[t] += cl[exec_k[o + j]] / F[m];                                 // eq 15
                work[m] += cl[exec_k[o + j]];                                         // eq 22
                slots += 1.0;
            }
            const int nd = __builtin_popcount(dest);
            transfers += nd;
            traffic += nd * (z / 8.0);
            if (exec_m[o] < M) at[t] = exec_m[o];                   // resides on slot 0's server
        }
    }
    std::copy(delay.begin(), delay.end(), delay_out);
    std::copy(work.begin(), work.end(), work_out);
    stats_out[0] = transfers;
    stats_out[1] = traffic;
    stats_out[2] = remote;
    stats_out[3] = slots;
    clear_error();
    return ORDERMOE_OK;
}
