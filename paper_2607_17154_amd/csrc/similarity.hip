// Expert similarity model on gfx950 (eq 3-5): for chunks of calibration
// tokens, the routing-logit tile H = W_r X_chunk^T is formed on chip and used
// twice before it is dropped -- for the activation counts (top-k per token) and
// for the Gram matrix H H^T -- so H never reaches HBM.
//
//   sim_partial_kernel   persistent over chunks of SIM_TC tokens:
//                          bf16: H tile by v_mfma_f32_16x16x32_bf16 (2 x 2 waves,
//                                each 64 experts x 64 tokens), fp32 accumulate;
//                          fp32: fp64 dot products rounded to fp32;
//                        H tile -> LDS; per-token top-k -> block histogram;
//                        Gram += H H^T with an 8 x 8 register tile per thread;
//                        per-block partial Gram and counts to the workspace
//   sim_finalize_kernel  fixed-order fp64 sum of the partials, cosine (eq 4)
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "common.hpp"

namespace ordermoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int SIM_TC = 128;        // tokens per chunk
constexpr int SIM_EMAX = 128;      // experts supported by the fused kernel
constexpr int SIM_LDH = SIM_TC + 4;

__global__ void __launch_bounds__(256) sim_partial_kernel(const SimArgs a) {
    __shared__ float s_H[SIM_EMAX][SIM_LDH];
    __shared__ int s_cnt[SIM_EMAX];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int E = a.E, d = a.d;
    const int nchunks = (int)((a.T_cal + SIM_TC - 1) / SIM_TC);
    for (int i = tid; i < SIM_EMAX; i += 256) s_cnt[i] = 0;

    // Gram register tile: rows ti + 16 u, columns tj + 16 v (u, v < 8)
    const int ti = tid >> 4, tj = tid & 15;
    float gacc[8][8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int v = 0; v < 8; ++v) gacc[u][v] = 0.f;

    for (int ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
        const int64_t t0 = (int64_t)ch * SIM_TC;
        if (a.dtype == ORDERMOE_BF16) {
            const __bf16* X = (const __bf16*)a.x_cal;
            const __bf16* W = (const __bf16*)a.w_router;
            const int wm = wave >> 1, wn = wave & 1;       // 64 experts x 64 tokens per wave
            const int r16 = lane & 15, kg = (lane >> 4) * 8;
            const bf16x8 zero8 = {};
            const __bf16* wp[4];
            bool wok[4];
            const __bf16* xp[4];
            bool xok[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int e = wm * 64 + i * 16 + r16;
                wok[i] = e < E;
                wp[i] = W + (int64_t)(wok[i] ? e : 0) * d + kg;
                const int64_t t = t0 + wn * 64 + i * 16 + r16;
                xok[i] = t < a.T_cal;
                xp[i] = X + (xok[i] ? t : 0) * (int64_t)d + kg;
            }
            f32x4 acc[4][4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
            // U K-steps of loads are issued before they are multiplied, so each
            // wave keeps 8 * U loads of 16 bytes in flight (d % 64 == 0)
            constexpr int U = 4;
            int kk = 0;
            for (; kk + 32 * U <= d; kk += 32 * U) {
                bf16x8 av[U][4], bv[U][4];
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        av[u][i] = wok[i] ? *(const bf16x8*)(wp[i] + kk + 32 * u) : zero8;
                        bv[u][i] = xok[i] ? *(const bf16x8*)(xp[i] + kk + 32 * u) : zero8;
                    }
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[u][i], bv[u][j], acc[i][j], 0, 0, 0);
            }
            for (; kk < d; kk += 32) {
                bf16x8 av[4], bv[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    av[i] = wok[i] ? *(const bf16x8*)(wp[i] + kk) : zero8;
                    bv[i] = xok[i] ? *(const bf16x8*)(xp[i] + kk) : zero8;
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
            }
            // acc[i][j][q]: expert wm*64 + i*16 + (lane/16)*4 + q, token wn*64 + j*16 + lane%16
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        s_H[wm * 64 + i * 16 + (lane >> 4) * 4 + q][wn * 64 + j * 16 + r16] = acc[i][j][q];
        } else {
            const float* X = (const float*)a.x_cal;
            const float* W = (const float*)a.w_router;
            for (int p = tid; p < SIM_EMAX * SIM_TC; p += 256) {
                const int e = p / SIM_TC, tt = p % SIM_TC;
                const int64_t t = t0 + tt;
                float v = 0.f;
                if (e < E && t < a.T_cal) {
                    const float* xr = X + t * (int64_t)d;
                    const float* wr = W + (int64_t)e * d;
                    double s = 0.0;
                    for (int i = 0; i < d; ++i) s = fma((double)xr[i], (double)wr[i], s);
                    v = (float)s;
                }
                s_H[e][tt] = v;
            }
        }
        __syncthreads();

        // activation counts: top-k of each token's logits, ties to the lower
        // index; 16 lanes per token, each holding experts lane%16 + 16 i, a
        // 64-bit (logit, -index) key max-reduced over the lanes per rank
        {
            const int g16 = lane >> 4, j16 = lane & 15;
            for (int tb = wave * 4; tb < SIM_TC; tb += 16) {
                const int tt = tb + g16;
                const bool tok = t0 + tt < a.T_cal;
                uint32_t removed = 0;
                for (int r = 0; r < a.k; ++r) {
                    uint64_t best = 0;
                    for (int i = 0, e = j16; e < E; ++i, e += 16) {
                        if (removed & (1u << i)) continue;
                        const uint32_t u = __float_as_uint(s_H[e][tt]);
                        const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
                        const uint64_t key = ((uint64_t)o << 32) | (uint32_t)(0xFFFFu - (uint32_t)e);
                        best = key > best ? key : best;
                    }
#pragma unroll
                    for (int off = 8; off >= 1; off >>= 1) {
                        uint32_t lo = (uint32_t)best, hi = (uint32_t)(best >> 32);
                        lo = __shfl_xor(lo, off, 16);
                        hi = __shfl_xor(hi, off, 16);
                        const uint64_t o = ((uint64_t)hi << 32) | lo;
                        best = o > best ? o : best;
                    }
                    const int e = (int)(0xFFFFu - (uint32_t)(best & 0xFFFFu));
                    if (r == 0 && j16 == 0 && tok && a.top1) a.top1[t0 + tt] = e;
                    if ((e & 15) == j16) {
                        removed |= 1u << (e >> 4);
                        if (tok) atomicAdd(&s_cnt[e], 1);
                    }
                }
            }
        }
        // Gram of this chunk; rows/columns beyond E hold zeros from the MFMA padding
        const int tmax = (int)((a.T_cal - t0) < SIM_TC ? (a.T_cal - t0) : SIM_TC);
        for (int t = 0; t < tmax; ++t) {
            float hu[8], hv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) { hu[u] = s_H[ti + 16 * u][t]; hv[u] = s_H[tj + 16 * u][t]; }
#pragma unroll
            for (int u = 0; u < 8; ++u)
#pragma unroll
                for (int v = 0; v < 8; ++v) gacc[u][v] = fmaf(hu[u], hv[v], gacc[u][v]);
        }
        __syncthreads();
    }
    float* gp = a.gram_part + (int64_t)blockIdx.x * SIM_EMAX * SIM_EMAX;
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int v = 0; v < 8; ++v) gp[(ti + 16 * u) * SIM_EMAX + tj + 16 * v] = gacc[u][v];
    __syncthreads();
    for (int i = tid; i < SIM_EMAX; i += 256) a.count_part[(int64_t)blockIdx.x * SIM_EMAX + i] = s_cnt[i];
}

// Fixed-order fp64 sum of the per-block partial Gram matrices and counts;
// one thread per (i, j) entry, consecutive threads on consecutive columns.
__global__ void __launch_bounds__(256) sim_reduce_kernel(const SimArgs a, int nparts, double* gram) {
    const int p = blockIdx.x * 256 + threadIdx.x;
    if (p >= SIM_EMAX * SIM_EMAX) return;
    const int i = p / SIM_EMAX, j = p % SIM_EMAX;
    if (i >= a.E || j >= a.E) return;
    // 8 interleaved partial sums (fixed order) keep 8 loads in flight
    double s8[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const float* src = a.gram_part + p;
    int b = 0;
    for (; b + 8 <= nparts; b += 8) {
#pragma unroll
        for (int q = 0; q < 8; ++q) s8[q] += (double)src[(int64_t)(b + q) * SIM_EMAX * SIM_EMAX];
    }
    for (int q = 0; b < nparts; ++b, ++q) s8[q] += (double)src[(int64_t)b * SIM_EMAX * SIM_EMAX];
    double s = 0.0;
#pragma unroll
    for (int q = 0; q < 8; ++q) s += s8[q];
    gram[p] = s;
    if (i == 0) {
        int64_t c = 0;
        for (int b = 0; b < nparts; ++b) c += (int64_t)a.count_part[(int64_t)b * SIM_EMAX + j];
        a.counts[j] = c;
    }
}

// cosine of eq 4 from the reduced Gram matrix; a zero norm gives 0 off the
// diagonal, every diagonal entry is 1
__global__ void __launch_bounds__(256) sim_normalise_kernel(const SimArgs a, const double* gram) {
    const int p = blockIdx.x * 256 + threadIdx.x;
    const int E = a.E;
    if (p >= E * E) return;
    const int i = p / E, j = p % E;
    float out = 1.0f;
    if (i != j) {
        const double den = sqrt(gram[i * SIM_EMAX + i]) * sqrt(gram[j * SIM_EMAX + j]);
        out = den > 0.0 ? (float)(gram[i * SIM_EMAX + j] / den) : 0.0f;
    }
    a.sim[p] = out;
}

__global__ void pack_gate_up_kernel(int esz, int64_t n, int f, int d, const char* g, const char* u,
                                    char* out) {
    // one block per packed row; rows [64b, 64b+32) <- gate [32b, 32b+32), [64b+32, 64b+64) <- up
    const int64_t prow = blockIdx.x;                  // over n * 2f rows
    const int64_t ex = prow / (2 * f);
    const int pr = (int)(prow % (2 * f));
    const int blk = pr / 64, within = pr % 64;
    const int src_row = blk * 32 + (within & 31);
    const char* src = (within < 32 ? g : u) + ((ex * f + src_row) * (int64_t)d) * esz;
    char* dst = out + prow * (int64_t)d * esz;
    const int64_t nbytes = (int64_t)d * esz;
    for (int64_t i = threadIdx.x * 4; i < nbytes; i += blockDim.x * 4)
        *(uint32_t*)(dst + i) = *(const uint32_t*)(src + i);
}

}  // namespace

int64_t similarity_tokens_per_chunk(int) { return SIM_TC; }
int similarity_max_experts() { return SIM_EMAX; }

int launch_similarity(const SimArgs& a, void* stream) {
    hipStream_t st = (hipStream_t)stream;
    {
        KernelTimer kt_("sim_partial", st);
        hipLaunchKernelGGL(sim_partial_kernel, dim3(a.nchunk), dim3(256), 0, st, a);
        }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
    {
        KernelTimer kt_("sim_reduce", st);
        hipLaunchKernelGGL(sim_reduce_kernel, dim3(SIM_EMAX * SIM_EMAX / 256), dim3(256), 0, st, a,
                           a.nchunk, a.gram);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
    {
        KernelTimer kt_("sim_normalise", st);
        hipLaunchKernelGGL(sim_normalise_kernel, dim3((a.E * a.E + 255) / 256), dim3(256), 0, st, a,
                           (const double*)a.gram);
    }
    e = hipGetLastError();
    return (int)e;
}

int launch_pack_gate_up(int dtype, int n, int f, int d, const void* g, const void* u, void* out,
                        void* stream) {
    const int esz = dtype == ORDERMOE_BF16 ? 2 : 4;
    const int64_t rows = (int64_t)n * 2 * f;
    if (rows == 0) return 0;
    hipLaunchKernelGGL(pack_gate_up_kernel, dim3((unsigned)rows), dim3(256), 0, (hipStream_t)stream,
                       esz, (int64_t)n, f, d, (const char*)g, (const char*)u, (char*)out);
    return (int)hipGetLastError();
}

}  // namespace ordermoe
