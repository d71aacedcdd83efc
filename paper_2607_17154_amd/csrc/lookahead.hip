// Transition statistics (eq 41) and the look-ahead cost-to-go Phi (eq 42) on
// the device, for every layer of a stack.  The results equal the host
// library's ordermoe_estimate_transitions and ordermoe_build_lookahead bit for
// bit: counts are integers (atomic increments commute), each probability is
// one fp64 division of a count by its row total, every candidate cost is
// formed with the same fp64 operations in the same order (no contraction), a
// minimum of doubles does not depend on the order it is taken in, and each
// Phi entry is a dot product summed in target order.
//
//   fill_f64 / fill_u32        zero the buffers (a kernel, not a memset, so
//                              that the calls can be captured in a graph)
//   transition_count_kernel    one thread per (layer pair, calibration token)
//   transition_norm_kernel     one thread per (layer, row): P = n / total
//   lookahead_next_kernel      V[l][s][r'] = min over the next layer's
//                              candidates of target r' from source s of
//                              g_{l+1}(m', k' | s) + Phi^(h-1)_{l+1}(m', k')
//   lookahead_phi_kernel       Phi^(h)_l[m][k] = sum_r' P_l[k][r'] V[l][m][r']
#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.hpp"

namespace ordermoe {
namespace {

constexpr int LA_THREADS = 256;

__global__ void __launch_bounds__(LA_THREADS) fill_f64(double* p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * LA_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * LA_THREADS)
        p[i] = 0.0;
}

__global__ void __launch_bounds__(LA_THREADS) fill_u32(uint32_t* p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * LA_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * LA_THREADS)
        p[i] = 0u;
}

// ids outside [0, E) are not counted
__global__ void __launch_bounds__(LA_THREADS) transition_count_kernel(const int32_t* top1, int32_t N, int32_t E,
                                                                      int64_t T_cal, uint32_t* cnt) {
    const int64_t n = (int64_t)(N - 1) * T_cal;
    for (int64_t i = (int64_t)blockIdx.x * LA_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * LA_THREADS) {
        const int64_t l = i / T_cal, t = i - l * T_cal;
        const int32_t a = top1[l * T_cal + t], b = top1[(l + 1) * T_cal + t];
        if (a >= 0 && a < E && b >= 0 && b < E) atomicAdd(&cnt[(l * E + a) * E + b], 1u);
    }
}

__global__ void __launch_bounds__(LA_THREADS) transition_norm_kernel(const uint32_t* cnt, int32_t N, int32_t E,
                                                                     double* P) {
    const int64_t rows = (int64_t)(N - 1) * E;
    for (int64_t row = (int64_t)blockIdx.x * LA_THREADS + threadIdx.x; row < rows;
         row += (int64_t)gridDim.x * LA_THREADS) {
        const uint32_t* c = cnt + row * E;
        double* p = P + row * E;
        int64_t tot = 0;
        for (int k = 0; k < E; ++k) tot += c[k];
        for (int k = 0; k < E; ++k) p[k] = tot > 0 ? (double)c[k] / (double)tot : 0.0;
    }
}

struct LookArgs {
    int32_t N, E, M;
    const double* P;          // [N-1][E][E]
    const uint8_t* x;         // [N][M][E]
    const float* sim;         // [N][E][E]
    const int32_t* group_of;  // [N][E]
    const float* theta;       // [N]
    const double* z_bits;     // [N]
    const double* c;          // [N][E]
    const double* d_ref;      // [N]
    const double* B;          // [M][M]
    const double* tau;        // [M][M]
    const double* F;          // [M]
    double omega_T, omega_Q;
    float Qbar;
    int32_t pin, allow_sub;
};

// eq 37's per-step delay of (m, k) from source s
__device__ inline double step_delay_dev(const LookArgs& a, int s, int m, int k, double z, const double* cl) {
    const double trans = (s != m) ? (z / a.B[(size_t)s * a.M + m] + a.tau[(size_t)s * a.M + m]) : 0.0;
    return trans + cl[k] / a.F[m];
}

// one thread per (l, s, r'), l = 0 .. N-2: the candidates of target r' at layer l + 1
__global__ void __launch_bounds__(LA_THREADS) lookahead_next_kernel(const LookArgs a, const double* prev,
                                                                    double* V) {
    const int E = a.E, M = a.M;
    const int64_t ME = (int64_t)M * E;
    const int64_t n = (int64_t)(a.N - 1) * ME;
    for (int64_t i = (int64_t)blockIdx.x * LA_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * LA_THREADS) {
        const int l = (int)(i / ME);
        const int s = (int)((i - l * ME) / E);
        const int r1 = (int)(i - l * ME - (int64_t)s * E);
        const int l1 = l + 1;
        const uint8_t* xl = a.x + (size_t)l1 * ME;
        const float* sl = a.sim + (size_t)l1 * E * E;
        const int32_t* gl = a.group_of + (size_t)l1 * E;
        const double* cl = a.c + (size_t)l1 * E;
        const double* nxt = prev + (size_t)l1 * ME;
        const double z = a.z_bits[l1], dref = a.d_ref[l1];
        auto g_of = [&](int m1, int k1) {
            double q = 0.0;
            if (k1 != r1) q = (double)((1.0f - sl[(size_t)r1 * E + k1]) * 0.5f);     // eq 18
            double v = a.omega_T * step_delay_dev(a, s, m1, k1, z, cl) / dref;          // eq 38
            if (a.Qbar > 0.0f) v += a.omega_Q * q / (double)a.Qbar;
            return v + nxt[(size_t)m1 * E + k1];
        };
        double best = 0.0;
        if (a.pin && xl[(size_t)s * E + r1]) {
            best = g_of(s, r1);                                // a local target is kept
        } else {
            bool have = false;
            const bool subs = a.allow_sub && a.Qbar > 0.0f;
            const float th = a.theta[l1];
            const int32_t gr = gl[r1];
            for (int k1 = 0; k1 < E; ++k1) {
                // the target and its feasible substitutes (eq 7-8), budget-free
                if (k1 != r1 && !(subs && gl[k1] == gr && sl[(size_t)r1 * E + k1] >= th)) continue;
                for (int m1 = 0; m1 < M; ++m1) {
                    if (!xl[(size_t)m1 * E + k1]) continue;
                    if (a.allow_sub == 2 && k1 != r1 && m1 != s) continue;   // local substitutes only
                    const double v = g_of(m1, k1);
                    if (!have || v < best) { best = v; have = true; }
                }
            }
        }
        V[i] = best;
    }
}

// one thread per (l, m, k), l = 0 .. N-2
__global__ void __launch_bounds__(LA_THREADS) lookahead_phi_kernel(const LookArgs a, const double* V, double* cur) {
    const int E = a.E, M = a.M;
    const int64_t ME = (int64_t)M * E;
    const int64_t n = (int64_t)(a.N - 1) * ME;
    for (int64_t i = (int64_t)blockIdx.x * LA_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * LA_THREADS) {
        const int l = (int)(i / ME);
        const int m = (int)((i - l * ME) / E);
        const int k = (int)(i - l * ME - (int64_t)m * E);
        const double* Pl = a.P + (size_t)l * E * E + (size_t)k * E;
        const double* Vl = V + (size_t)l * ME + (size_t)m * E;
        double acc = 0.0;
        for (int r1 = 0; r1 < E; ++r1) acc += Pl[r1] * Vl[r1];                  // eq 42
        cur[i] = acc;
    }
}

unsigned blocks_for(int64_t n) {
    const int64_t b = (n + LA_THREADS - 1) / LA_THREADS;
    return (unsigned)(b < 1 ? 1 : (b > 65535 ? 65535 : b));
}

}  // namespace

size_t transitions_device_workspace(int32_t N, int32_t E) {
    return N > 1 ? (size_t)(N - 1) * E * E * sizeof(uint32_t) : 0;
}

size_t lookahead_device_workspace(int32_t N, int32_t E, int32_t M) {
    // the second Phi buffer of the ping-pong and the V table
    return (size_t)2 * N * M * E * sizeof(double);
}

int launch_transitions_device(int32_t N, int32_t E, int64_t T_cal, const int32_t* top1, double* P, void* ws,
                              void* stream) {
    hipStream_t st = (hipStream_t)stream;
    if (N < 2) return 0;
    uint32_t* cnt = (uint32_t*)ws;
    const int64_t nc = (int64_t)(N - 1) * E * E;
    fill_u32<<<blocks_for(nc), LA_THREADS, 0, st>>>(cnt, nc);
    if (T_cal > 0) {
        const int64_t n = (int64_t)(N - 1) * T_cal;
        transition_count_kernel<<<blocks_for(n), LA_THREADS, 0, st>>>(top1, N, E, T_cal, cnt);
    }
    transition_norm_kernel<<<blocks_for((int64_t)(N - 1) * E), LA_THREADS, 0, st>>>(cnt, N, E, P);
    return (int)hipGetLastError();
}

int launch_lookahead_device(const LookaheadDeviceArgs& d, void* stream) {
    hipStream_t st = (hipStream_t)stream;
    const int64_t ME = (int64_t)d.M * d.E, NME = (int64_t)d.N * ME;
    double* other = (double*)d.ws;                 // [N][M][E]
    double* V = other + NME;                       // [N-1][M][E]
    fill_f64<<<blocks_for(NME), LA_THREADS, 0, st>>>(d.phi, NME);
    if (d.H > 1 && d.N > 1) {
        fill_f64<<<blocks_for(NME), LA_THREADS, 0, st>>>(other, NME);
        LookArgs a;
        a.N = d.N; a.E = d.E; a.M = d.M; a.P = d.P; a.x = d.x; a.sim = d.sim; a.group_of = d.group_of;
        a.theta = d.theta; a.z_bits = d.z_bits; a.c = d.c; a.d_ref = d.d_ref; a.B = d.B; a.tau = d.tau;
        a.F = d.F; a.omega_T = d.omega_T; a.omega_Q = d.omega_Q; a.Qbar = d.Qbar; a.pin = d.pin;
        a.allow_sub = d.allow_sub;
        const int64_t n = (int64_t)(d.N - 1) * ME;
        // depth h writes the buffer that the last depth (H - 1) leaves in phi;
        // both start at zero, and the last layer of either is never written
        for (int h = 1; h <= d.H - 1; ++h) {
            double* cur = ((d.H - 1 - h) % 2 == 0) ? d.phi : other;
            const double* prev = cur == d.phi ? other : d.phi;
            lookahead_next_kernel<<<blocks_for(n), LA_THREADS, 0, st>>>(a, prev, V);
            lookahead_phi_kernel<<<blocks_for(n), LA_THREADS, 0, st>>>(a, V, cur);
        }
    }
    return (int)hipGetLastError();
}

}  // namespace ordermoe
