// Routing and runtime server-expert selection of one MoE layer on gfx950.
//
// Kernel 1 (route_select_kernel), one block per RT_TB tokens:
//   * router logits l = x W_r^T (eq 3, one token at a time):
//       bf16: v_mfma_f32_16x16x32_bf16, the block's 16 tokens x all experts,
//             d split over the 4 waves, partial sums added in wave order;
//       fp32: fp64 dot products (exact products), rounded once to fp32;
//   * per token (16 lanes each): top-(k+1) by a 64-bit (logit, -index) key
//     max-reduced over the lanes, gates, margin and flag;
//   * per slot in rank order: the candidate search of eq (40)/(43) -- lane 0
//     takes the exact candidate, lane j the (j-1)-th substitute of the LDS-
//     staged table; each lane scans the servers holding its expert and keeps a
//     64-bit key (J, position, remote, server); a min-reduce over the 16 lanes
//     gives (m*, k*); the budget is updated as eq (44);
//   * per-block counters and per-destination remote-slot counts.
// Kernel 2 (dispatch_scan_kernel), one block: exclusive scans of the
//   per-block destination counts (one wave per destination), totals of the
//   counters.
// Kernel 3 (dispatch_scatter_kernel), one block per RT_TB tokens: stable
//   placement of the block's remote slots into the (destination, token, slot)
//   ordered dispatch list.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.hpp"

namespace ordermoe {
namespace {

constexpr int RT_TB = 16;        // tokens per block
constexpr int RT_THREADS = 512;  // 8 waves share the router's K loop; waves 0-3 then
                                 // run the token stage, 16 lanes per token
constexpr int RT_WAVES = RT_THREADS / 64;
constexpr int RT_SLOTS = 4;      // partial-sum slots of the two-round wave reduction

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// order-preserving map of fp32 onto uint32
__device__ inline uint32_t f2ord(float v) {
    uint32_t u = __float_as_uint(v);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ inline float ord2f(uint32_t o) {
    uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
    return __uint_as_float(u);
}

__device__ inline uint64_t shfl_xor64(uint64_t v, int mask) {
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    lo = __shfl_xor(lo, mask, 16);
    hi = __shfl_xor(hi, mask, 16);
    return ((uint64_t)hi << 32) | lo;
}

// Router partial logits of this block's 16 tokens over the K steps of 32 that
// belong to this wave (steps wave, wave + 8, ...): v_mfma_f32_16x16x32_bf16
// with the tokens as rows and 16 experts per block as columns.  U steps are
// loaded before they are multiplied so that each wave keeps U * (1 + NB)
// 16-byte loads in flight.
template <int NB, int U>
__device__ inline void router_k_loop(const RouteArgs& a, int wave, int lane, int64_t t0, f32x4* acc) {
    const __bf16* X = (const __bf16*)a.x;
    const __bf16* W = (const __bf16*)a.w_router;
    const int d = a.d, E = a.E;
    const int r16 = lane & 15, kg = (lane >> 4) * 8;
    const int64_t tok = t0 + r16;
    const bool tok_ok = tok < a.T;
    const __bf16* xrow = X + (tok_ok ? tok : 0) * (int64_t)d + kg;
    const __bf16* wrow[NB];
    bool wok[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int e = nb * 16 + r16;
        wok[nb] = e < E;
        wrow[nb] = W + (int64_t)(wok[nb] ? e : 0) * d + kg;
    }
    const bf16x8 zero8 = {};
    const int nsteps = d / 32;
    int s0 = wave;
    for (; s0 + (U - 1) * RT_WAVES < nsteps; s0 += U * RT_WAVES) {
        bf16x8 av[U], bv[U][NB];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = (s0 + u * RT_WAVES) * 32;
            av[u] = tok_ok ? *(const bf16x8*)(xrow + k) : zero8;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bv[u][nb] = wok[nb] ? *(const bf16x8*)(wrow[nb] + k) : zero8;
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[u], bv[u][nb], acc[nb], 0, 0, 0);
    }
    for (; s0 < nsteps; s0 += RT_WAVES) {
        const int k = s0 * 32;
        const bf16x8 x8 = tok_ok ? *(const bf16x8*)(xrow + k) : zero8;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const bf16x8 w8 = wok[nb] ? *(const bf16x8*)(wrow[nb] + k) : zero8;
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x8, w8, acc[nb], 0, 0, 0);
        }
    }
}

// global -> LDS copy of five arrays of 32-bit words by the block, as one
// index space with 8 reads in flight per thread before their stores
__device__ inline void stage_copy5(int32_t* const* dst, const int32_t* const* src, const int* len,
                                   int tid) {
    int end[5];
    int tot = 0;
#pragma unroll
    for (int q = 0; q < 5; ++q) { tot += len[q]; end[q] = tot; }
    auto locate = [&](int i, int& q, int& o) {
        q = 0;
        o = i;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (i >= end[c]) { q = c + 1; o = i - end[c]; }
    };
    for (int i0 = 0; i0 < tot; i0 += 8 * RT_THREADS) {
        int32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * RT_THREADS + tid;
            int q, o;
            locate(i, q, o);
            v[u] = i < tot ? src[q][o] : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * RT_THREADS + tid;
            int q, o;
            locate(i, q, o);
            if (i < tot) dst[q][o] = v[u];
        }
    }
}

// Small batches (at most RT_SPLIT_MAX_T tokens): the router GEMM alone on many
// waves.  Wave (token block, expert block, K slice) forms the 16 x 16 partial
// logits of its K slice with v_mfma_f32_16x16x32_bf16, its loads issued 16
// steps at a time; route_select_kernel adds the slices in slice order.
constexpr int64_t RT_SPLIT_MAX_T = 1024;
constexpr int RT_SPLIT_MAX_K = 16;

__global__ void __launch_bounds__(64) router_split_kernel(const RouteArgs a) {
    const __bf16* X = (const __bf16*)a.x;
    const __bf16* W = (const __bf16*)a.w_router;
    const int lane = threadIdx.x;
    const int r16 = lane & 15, kg = (lane >> 4) * 8;
    const int d = a.d, E = a.E;
    const int Epad = (E + 15) & ~15;
    const int64_t tok = (int64_t)blockIdx.x * 16 + r16;
    const int e = blockIdx.y * 16 + r16;
    const bool tok_ok = tok < a.T, e_ok = e < E;
    const int kc = d / a.ksplit;                          // a multiple of 32
    const __bf16* xrow = X + (tok_ok ? tok : 0) * (int64_t)d + blockIdx.z * kc + kg;
    const __bf16* wrow = W + (int64_t)(e_ok ? e : 0) * d + blockIdx.z * kc + kg;
    const bf16x8 zero8 = {};
    const int nsteps = kc / 32;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < nsteps; s0 += 16) {
        bf16x8 xv[16], wv[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const bool in = s0 + u < nsteps;
            xv[u] = tok_ok && in ? *(const bf16x8*)(xrow + (s0 + u) * 32) : zero8;
            wv[u] = e_ok && in ? *(const bf16x8*)(wrow + (s0 + u) * 32) : zero8;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv[u], wv[u], acc, 0, 0, 0);
    }
    // acc[i]: token (lane/16)*4 + i of the block, expert lane%16 of the block
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t t = (int64_t)blockIdx.x * 16 + (lane >> 4) * 4 + i;
        if (t < a.T) a.logit_part[((int64_t)blockIdx.z * a.T + t) * Epad + blockIdx.y * 16 + r16] = acc[i];
    }
}

template <int NBT>
__global__ void __launch_bounds__(RT_THREADS, 2)
route_select_kernel(const RouteArgs a) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t t0 = (int64_t)blockIdx.x * RT_TB;
    const int E = a.E, d = a.d, k = a.k, M = a.M;
    const int Epad = (E + 15) & ~15;

    extern __shared__ float smem[];
    float* s_part = smem;                               // [RT_SLOTS][RT_TB][Epad]
    float* s_logit = smem;                              // reuses slot 0 after the sum
    int32_t* s_t1k = (int32_t*)(smem + RT_SLOTS * RT_TB * Epad);   // [E][gmax]
    float* s_t1q = (float*)(s_t1k + E * a.gmax);                   // [E][gmax]
    int32_t* s_t1n = (int32_t*)(s_t1q + E * a.gmax);               // [E]
    uint32_t* s_mask = (uint32_t*)(s_t1n + E);                     // [E]
    int* s_cnt = (int*)(s_mask + E);                               // [8 + M]
    float* s_S = (float*)(s_cnt + 8 + M);                          // [M][M][E] if a.S_in_lds
    const float* Stab = a.S_in_lds ? s_S : a.S;

    // stage the candidate tables (small) and clear the block counters; the
    // copies issue several reads per thread before their LDS stores
    {
        const int32_t* src[5] = {a.t1_k, (const int32_t*)a.t1_q, a.t1_n, (const int32_t*)a.srvmask,
                                 (const int32_t*)a.S};
        int32_t* dst[5] = {s_t1k, (int32_t*)s_t1q, s_t1n, (int32_t*)s_mask, (int32_t*)s_S};
        const int len[5] = {E * a.gmax, E * a.gmax, E, E, a.S_in_lds ? M * M * E : 0};
        stage_copy5(dst, src, len, tid);
    }
    for (int i = tid; i < 8 + M; i += RT_THREADS) s_cnt[i] = 0;
    // this thread's token location and budget, read before the router loop so
    // that their latency is hidden behind it (lanes of waves 0-3 own tokens)
    int loc_pre = 0;
    float qhat_pre = 0.f;
    {
        const int64_t tp = t0 + (wave * 4 + (lane >> 4));
        if (wave < RT_TB / 4 && tp < a.T) { loc_pre = a.loc_in[tp]; qhat_pre = a.qhat_in[tp]; }
    }

    // ---------------- router logits ----------------
    if (a.ksplit > 0) {
        // split router: add the K slices in slice order (the reads of all
        // slices of an element are issued before the additions)
        for (int i = tid; i < RT_TB * Epad; i += RT_THREADS) {
            const int64_t tok = t0 + i / Epad;
            float pv[RT_SPLIT_MAX_K];
#pragma unroll
            for (int z = 0; z < RT_SPLIT_MAX_K; ++z)
                pv[z] = (z < a.ksplit && tok < a.T) ? a.logit_part[((int64_t)z * a.T + tok) * Epad + i % Epad] : 0.f;
            float v = 0.f;
#pragma unroll
            for (int z = 0; z < RT_SPLIT_MAX_K; ++z)
                if (z < a.ksplit) v += pv[z];
            s_logit[i] = v;
        }
    } else if (a.dtype == ORDERMOE_BF16) {
        const int nblk = Epad / 16;
        f32x4 acc[NBT];
#pragma unroll
        for (int i = 0; i < NBT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        // unroll depth: every wave keeps 9-16 loads of 16 bytes in flight, within
        // 128 registers so that two blocks share a CU
        if constexpr (NBT == 1) router_k_loop<1, 8>(a, wave, lane, t0, acc);
        else if constexpr (NBT == 2) router_k_loop<2, 4>(a, wave, lane, t0, acc);
        else if constexpr (NBT == 4) router_k_loop<4, 2>(a, wave, lane, t0, acc);
        else if constexpr (NBT == 8) router_k_loop<8, 1>(a, wave, lane, t0, acc);
        else router_k_loop<16, 1>(a, wave, lane, t0, acc);
        // acc[nb][i] = partial logit of token (lane/16)*4 + i, expert nb*16 + lane%16.
        // Two-round reduction over the 8 waves in a fixed order: waves 4-7 hand
        // their sums to waves 0-3, then the four slots are added.
        const int r16 = lane & 15;
        if (wave >= RT_SLOTS) {
#pragma unroll
            for (int nb = 0; nb < NBT; ++nb)
                if (nb < nblk)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        s_part[((wave - RT_SLOTS) * RT_TB + (lane >> 4) * 4 + i) * Epad + nb * 16 + r16] = acc[nb][i];
        }
        __syncthreads();
        if (wave < RT_SLOTS) {
#pragma unroll
            for (int nb = 0; nb < NBT; ++nb)
                if (nb < nblk)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float* sp = &s_part[(wave * RT_TB + (lane >> 4) * 4 + i) * Epad + nb * 16 + r16];
                        *sp = acc[nb][i] + *sp;
                    }
        }
        __syncthreads();
        for (int i = tid; i < RT_TB * Epad; i += RT_THREADS) {
            float v = s_part[i];
            for (int w = 1; w < RT_SLOTS; ++w) v += s_part[w * RT_TB * Epad + i];
            s_logit[i] = v;
        }
    } else {
        const float* X = (const float*)a.x;
        const float* W = (const float*)a.w_router;
        for (int p = tid; p < RT_TB * Epad; p += RT_THREADS) {
            const int tr = p / Epad, e = p % Epad;
            const int64_t tok = t0 + tr;
            float v = 0.f;
            if (tok < a.T && e < E) {
                const float* xr = X + tok * (int64_t)d;
                const float* wr = W + (int64_t)e * d;
                double s = 0.0;
                for (int i = 0; i < d; ++i) s = fma((double)xr[i], (double)wr[i], s);
                v = (float)s;
            }
            s_logit[p] = v;
        }
    }
    __syncthreads();

    // ---------------- per-token stage: 16 lanes per token, waves 0-3 ----------------
    if (wave < RT_TB / 4) {
    const int g = lane >> 4;                 // token within the wave
    const int j = lane & 15;                 // lane within the token group
    const int tr = wave * 4 + g;             // token within the block
    const int64_t t = t0 + tr;
    const bool valid = t < a.T;
    const float* lg = s_logit + tr * Epad;

    // top-(k+1) selection by (logit desc, index asc); this lane's logits (experts
    // j + 16 i) are read once and kept as order-preserving keys
    constexpr int PER_LANE = ORDERMOE_MAX_EXPERTS / 16;
    const int kk1 = (k + 1 < E) ? k + 1 : E;
    uint32_t okey[PER_LANE];
#pragma unroll
    for (int i = 0; i < PER_LANE; ++i) okey[i] = (j + 16 * i < E) ? f2ord(lg[j + 16 * i]) : 0u;
    uint32_t removed = 0;                    // bit i: local element j + 16 i taken
    int sel_e[ORDERMOE_MAX_TOPK + 1];
    float sel_v[ORDERMOE_MAX_TOPK + 1];
#pragma unroll
    for (int r = 0; r < ORDERMOE_MAX_TOPK + 1; ++r) {
        if (r < kk1) {
            uint64_t best = 0;
#pragma unroll
            for (int i = 0; i < PER_LANE; ++i) {
                const int e = j + 16 * i;
                if (e >= E || (removed & (1u << i))) continue;
                const uint64_t key = ((uint64_t)okey[i] << 32) | (uint32_t)(0xFFFFu - (uint32_t)e);
                best = key > best ? key : best;
            }
#pragma unroll
            for (int off = 8; off >= 1; off >>= 1) {
                uint64_t o = shfl_xor64(best, off);
                best = o > best ? o : best;
            }
            const int e = (int)(0xFFFFu - (uint32_t)(best & 0xFFFFu));
            sel_e[r] = e;
            sel_v[r] = ord2f((uint32_t)(best >> 32));
            if ((e & 15) == j) removed |= 1u << (e >> 4);
        }
    }
    float mg = __builtin_inff();
#pragma unroll
    for (int r = 0; r < ORDERMOE_MAX_TOPK; ++r) {
        if (r + 1 < kk1) {
            float gap = sel_v[r] - sel_v[r + 1];
            mg = gap < mg ? gap : mg;
        }
    }
    // gates: softmax renormalised over the top-k, or over all experts
    float den = 0.f;
    if (a.renorm) {
#pragma unroll
        for (int r = 0; r < ORDERMOE_MAX_TOPK; ++r)
            if (r < k) den += expf(sel_v[r] - sel_v[0]);
    } else {
        for (int e = j; e < E; e += 16) den += expf(lg[e] - sel_v[0]);
#pragma unroll
        for (int off = 8; off >= 1; off >>= 1) den += __shfl_xor(den, off, 16);
    }

    // server-expert selection, slots in rank order
    const int s_loc = loc_pre;
    const bool loc_ok = s_loc < M;
    float qhat = qhat_pre;
    const bool subs_on = a.allow_sub && a.Qbar > 0.f;
    const uint32_t mmask = M >= 32 ? 0xFFFFFFFFu : ((1u << M) - 1u);   // servers that exist
    int first_m = s_loc, ncls[4] = {0, 0, 0, 0}, nremote = 0;
    uint32_t dstmask = 0;
#pragma unroll
    for (int slot = 0; slot < ORDERMOE_MAX_TOPK; ++slot) {
        if (slot >= k) break;
        const int r = sel_e[slot];
        int km = r, mm = s_loc;
        float qsel = 0.f;
        const uint32_t rmask = s_mask[r];
        if (loc_ok && !(a.pin && ((rmask >> s_loc) & 1u))) {
            // lane j holds candidate expert: j = 0 exact, j >= 1 substitute j-1
            uint64_t key = ~0ull;
            int ke = -1;
            float qe = 0.f;
            if (j == 0) { ke = r; qe = 0.f; }
            else if (subs_on && j - 1 < s_t1n[r]) {
                ke = s_t1k[r * a.gmax + j - 1];
                qe = s_t1q[r * a.gmax + j - 1];
                if (!(qhat + qe <= a.Qbar)) ke = -1;        // eq 40 budget test
            }
            if (ke >= 0 && ke < E) {
                uint32_t ms = s_mask[ke] & mmask;
                while (ms) {
                    const int m = __builtin_ctz(ms);
                    ms &= ms - 1;
                    const float J = fmaf(a.cq, qe, Stab[((int64_t)s_loc * M + m) * E + ke]);
                    const uint64_t cand = ((uint64_t)__float_as_uint(J) << 32) |
                                          ((uint32_t)j << 6) | ((uint32_t)(m != s_loc) << 5) |
                                          (uint32_t)m;
                    key = cand < key ? cand : key;
                }
            }
#pragma unroll
            for (int off = 8; off >= 1; off >>= 1) {
                uint64_t o = shfl_xor64(key, off);
                key = o < key ? o : key;
            }
            const int pos = (int)((key >> 6) & 15u);
            mm = (int)(key & 31u);
            if (pos == 0) { km = r; qsel = 0.f; }
            else { km = s_t1k[r * a.gmax + pos - 1]; qsel = s_t1q[r * a.gmax + pos - 1]; }
        }
        const int remote = mm != s_loc;
        const int c = (remote << 1) | (km != r);
        qhat = qhat + qsel;
        if (slot == 0) first_m = mm;
        if (valid && j == 0) {
            const int64_t o = t * k + slot;
            a.out.idx[o] = r;
            a.out.w[o] = expf(sel_v[slot] - sel_v[0]) / den;
            if (loc_ok) {
                a.out.exec_k[o] = km;
                a.out.exec_m[o] = (uint8_t)mm;
                a.out.cls[o] = (uint8_t)c;
                ncls[c]++;
                if (remote) { nremote++; dstmask |= 1u << mm; atomicAdd(&s_cnt[8 + mm], 1); }
            } else {
                a.out.exec_k[o] = -1;
                a.out.exec_m[o] = 255;
                a.out.cls[o] = 255;
            }
        }
    }
    if (valid && j == 0) {
        a.out.margin[t] = mg;
        const int fl = mg < ORDERMOE_MARGIN_FLAG;
        a.out.flag[t] = (uint8_t)fl;
        a.out.qhat_out[t] = loc_ok ? qhat : a.qhat_in[t];
        a.out.loc_out[t] = loc_ok ? (uint8_t)first_m : a.loc_in[t];
        if (loc_ok) {
            for (int c = 0; c < 4; ++c) if (ncls[c]) atomicAdd(&s_cnt[c], ncls[c]);
            if (nremote) atomicAdd(&s_cnt[6], nremote);
            if (dstmask) atomicAdd(&s_cnt[5], __builtin_popcount(dstmask));
        } else {
            atomicAdd(&s_cnt[7], 1);
        }
        if (fl) atomicAdd(&s_cnt[4], 1);
    }
    }   // token stage
    __syncthreads();
    if (tid < 8) a.blk_cnt[(int64_t)blockIdx.x * 8 + tid] = s_cnt[tid];
    if (tid < M) a.blk_dst[(int64_t)blockIdx.x * M + tid] = s_cnt[8 + tid];
}

constexpr int SCAN_THREADS = 1024;
constexpr int SCAN_WAVES = SCAN_THREADS / 64;

// One block, every wave on its own (no block-wide barriers): waves 0-7 total
// the eight counters over the token blocks; wave w (and w + 16) scans the
// per-block counts of destination w over the blocks, giving each block's
// first position inside that destination's segment and the destination's
// total.  The segments follow in server order (dispatch_scatter_kernel adds
// the segment start).
__global__ void __launch_bounds__(SCAN_THREADS)
dispatch_scan_kernel(const int32_t* blk_dst, const int64_t* blk_cnt, int nblk, int M,
                     int32_t* dst_base, int32_t* dst_count, int64_t* counters) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (wave < 8) {
        int64_t v = 0;
        for (int b = lane; b < nblk; b += 64) v += blk_cnt[(int64_t)b * 8 + wave];
        for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
        if (lane == 0) counters[wave] = v;
    }
    for (int m = wave; m < M; m += SCAN_WAVES) {
        int32_t carry = 0;
        for (int b0 = 0; b0 < nblk; b0 += 64) {
            const int b = b0 + lane;
            const int32_t v = b < nblk ? blk_dst[(int64_t)b * M + m] : 0;
            int32_t inc = v;
            for (int off = 1; off < 64; off <<= 1) {
                const int32_t o = __shfl_up(inc, off);
                if (lane >= off) inc += o;
            }
            if (b < nblk) dst_base[(int64_t)b * M + m] = carry + inc - v;
            carry += __shfl(inc, 63);
        }
        if (lane == 0) dst_count[m] = carry;
    }
}

__global__ void __launch_bounds__(RT_THREADS)
dispatch_scatter_kernel(const uint8_t* exec_m, const uint8_t* loc_in, int64_t T, int k, int M,
                        const int32_t* dst_base, const int32_t* dst_count, int32_t* dispatch) {
    __shared__ int8_t s_dst[RT_TB * ORDERMOE_MAX_TOPK];
    const int tid = threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.x * RT_TB;
    const int n = RT_TB * k;
    if (tid < n) {
        const int64_t t = t0 + tid / k;
        int dst = -1;
        if (t < T) {
            const int s = loc_in[t];
            const int m = exec_m[t * k + tid % k];
            if (s < M && m != s) dst = m;
        }
        s_dst[tid] = (int8_t)dst;
    }
    __syncthreads();
    if (tid < n && s_dst[tid] >= 0) {
        const int dst = s_dst[tid];
        int rank = 0;
        for (int i = 0; i < tid; ++i) rank += (s_dst[i] == dst);
        int32_t start = 0;                        // the destination's segment
        for (int m = 0; m < dst; ++m) start += dst_count[m];
        const int32_t pos = start + dst_base[(int64_t)blockIdx.x * M + dst] + rank;
        dispatch[pos] = (int32_t)((t0 + tid / k) * k + tid % k);
    }
}

template <int NBT>
int launch_route_kernel(const RouteArgs& a, size_t smem, hipStream_t st) {
    if (smem > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)route_select_kernel<NBT>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return (int)e;
    }
    KernelTimer kt_("route_select", st);
    hipLaunchKernelGGL(route_select_kernel<NBT>, dim3(a.nblk), dim3(RT_THREADS), smem, st, a);
    return (int)hipGetLastError();
}

}  // namespace

int route_tokens_per_block() { return RT_TB; }

size_t route_smem_bytes(int E, int gmax, int M, bool S_in_lds) {
    const int Epad = (E + 15) & ~15;
    return sizeof(float) * (size_t)RT_SLOTS * RT_TB * Epad + (size_t)E * gmax * 8 + (size_t)E * 8 +
           sizeof(int) * (size_t)(8 + M) + (S_in_lds ? sizeof(float) * (size_t)M * M * E : 0);
}

// partial logits of the split router: at most 256 blocks of RT_TB tokens times
// the K slices (the launcher keeps slices * blocks <= 256), every expert count
size_t route_split_buffer_floats(int64_t T) {
    const int64_t rows = T * RT_SPLIT_MAX_K < 256 * RT_TB ? T * RT_SPLIT_MAX_K : 256 * RT_TB;
    return (size_t)(rows > 0 ? rows : 1) * ORDERMOE_MAX_EXPERTS;
}

// the cost table is staged in LDS when it is small enough to leave room for
// two blocks per CU, or, for batches of at most one block per CU, when it fits
static bool route_S_in_lds(int E, int gmax, int M, int nblk) {
    const size_t b = route_smem_bytes(E, gmax, M, true);
    return b <= 64 * 1024 || (nblk <= 256 && b <= 150 * 1024);
}

int launch_route_select(const RouteArgs& a, void* stream) {
    hipStream_t st = (hipStream_t)stream;
    if (a.nblk > 0) {
        RouteArgs b = a;
        b.S_in_lds = route_S_in_lds(a.E, a.gmax, a.M, a.nblk) ? 1 : 0;
        const size_t smem = route_smem_bytes(a.E, a.gmax, a.M, b.S_in_lds != 0);
        b.ksplit = 0;
        if (a.dtype == ORDERMOE_BF16 && a.T <= RT_SPLIT_MAX_T && a.logit_part) {
            // enough waves to cover the CUs, K slices a multiple of 32
            const int nbe = (a.E + 15) / 16;
            int ks = 256 / (a.nblk * nbe);
            ks = ks < 1 ? 1 : (ks > RT_SPLIT_MAX_K ? RT_SPLIT_MAX_K : ks);
            while (ks > 1 && a.d % (32 * ks) != 0) --ks;
            b.ksplit = ks;
            KernelTimer kt_("router_split", st);
            router_split_kernel<<<dim3((unsigned)a.nblk, (unsigned)nbe, (unsigned)ks), dim3(64), 0, st>>>(b);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return (int)e;
        }
        const int nb = (a.E + 15) / 16;
        const int nbt = nb <= 1 ? 1 : nb <= 2 ? 2 : nb <= 4 ? 4 : nb <= 8 ? 8 : 16;
        int e = 0;
        switch (nbt) {
            case 1: e = launch_route_kernel<1>(b, smem, st); break;
            case 2: e = launch_route_kernel<2>(b, smem, st); break;
            case 4: e = launch_route_kernel<4>(b, smem, st); break;
            case 8: e = launch_route_kernel<8>(b, smem, st); break;
            default: e = launch_route_kernel<16>(b, smem, st); break;
        }
        if (e) return e;
    }
    {
        KernelTimer kt_("dispatch_scan", st);
        hipLaunchKernelGGL(dispatch_scan_kernel, dim3(1), dim3(SCAN_THREADS), 0, st, a.blk_dst,
                       a.blk_cnt, a.nblk, a.M, a.dst_base, a.out.dst_count, a.out.counters);
        }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
    if (a.nblk > 0) {
        {
        KernelTimer kt_("dispatch_scatter", st);
        hipLaunchKernelGGL(dispatch_scatter_kernel, dim3(a.nblk), dim3(RT_THREADS), 0, st,
                           a.out.exec_m, a.loc_in, a.T, a.k, a.M, a.dst_base, a.out.dst_count,
                           a.out.dispatch);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return (int)e;
    }
    return 0;
}

}  // namespace ordermoe
