// Expert similarity model on gfx950 (eq 3-5): for tiles of calibration
// tokens, the routing-logit tile H = X_tile W_r^T is formed on chip and used
// twice before it is dropped -- for the activation counts (top-k per token) and
// for the Gram matrix H^T H -- so H never reaches HBM.
//
//   sim_tile_kernel      bf16, persistent over tiles of 256 tokens x 128
//                        experts by v_mfma_f32_32x32x16_bf16: the calibration
//                        tokens streamed from HBM once, straight into operand
//                        registers several K steps ahead, W_r through LDS; the
//                        fp32 H tile then parked in LDS for the per-token top-k
//                        counts (and top-1), then Gram += H^T H by bf16 MFMAs
//                        on a two-term bf16 split of H; per-workgroup partial
//                        Gram and counts to the workspace
//   sim_partial_kernel   fp32 storage: chunks of 128 tokens, fp64 dot products
//                        rounded to fp32, same partial outputs
//   sim_reduce_kernel    fixed-order fp64 sum of the partials: 16 slices of
//                        parts per entry, then the slices in order
//   sim_normalise_kernel cosine (eq 4)
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "common.hpp"

namespace ordermoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int SIM_TC = 128;        // tokens per chunk
constexpr int SIM_EMAX = 128;      // experts supported by the fused kernel
constexpr int SIM_LDH = SIM_TC + 4;

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int ST_BM = 256;                 // tokens per tile (32 per wave)
constexpr int ST_WAVES = 8;
constexpr int ST_THREADS = ST_WAVES * 64;
constexpr int ST_BK = 64, ST_LDK = ST_BK + 8;
constexpr int ST_STAGES = 4;               // K steps of reads in flight per wave
constexpr int ST_LDH = SIM_EMAX + 4;       // row stride of the parked H tile (floats)
constexpr int ST_LDT = ST_BM + 8;          // row stride of the h / l planes of H^T (bf16)
constexpr int ST_LDA = 144;                // bytes per staged token row (64 bf16 + 16)
constexpr size_t ST_LDS_A = (size_t)ST_BM * ST_LDA;      // token staging, 32 rows per wave
constexpr int ST_WCH = 2;                 // K steps per W chunk (one barrier per chunk)
constexpr size_t ST_LDS_KLOOP = (size_t)2 * ST_WCH * SIM_EMAX * ST_LDK * 2 + ST_LDS_A;
constexpr size_t ST_LDS_H = (size_t)ST_BM * ST_LDH * 4;
constexpr size_t ST_LDS_HL = (size_t)2 * SIM_EMAX * ST_LDT * 2;
constexpr size_t ST_LDS_MAX2 = ST_LDS_KLOOP > ST_LDS_H ? ST_LDS_KLOOP : ST_LDS_H;
constexpr size_t ST_LDS = ST_LDS_MAX2 > ST_LDS_HL ? ST_LDS_MAX2 : ST_LDS_HL;

__device__ inline bf16x8 st_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
    return __builtin_bit_cast(bf16x8, v);
}

// One workgroup per tile of 256 calibration tokens; wave w owns tokens
// 32w .. 32w+31 against all 128 experts (4 blocks of 32x32).  The tokens are
// streamed from HBM once: a wave reads its 32 token rows coalesced (an
// instruction covers 8 rows x 128 bytes, whole cache lines) into registers,
// then passes them through its own padded LDS rows into the MFMA operand
// layout (lane: token lane%32, K elements 8*(lane/32) .. +7 of each 16); the
// router rows W_r (L2 resident) go through a double-buffered LDS tile shared by
// the waves.  The reads of a K step are issued ST_STAGES steps ahead.  After the K loop the
// fp32 H tile is parked in LDS for the top-k counts, then replaced by the bf16
// h / l planes of H^T for the Gram update; the Gram partial of a workgroup
// lives in its workspace slot.
__global__ void __launch_bounds__(ST_THREADS, 1) sim_tile_kernel(const SimArgs a) {
    constexpr int BN = SIM_EMAX, BK = ST_BK, LDK = ST_LDK, S = ST_STAGES;
    constexpr int FN = BN / 32;                         // per wave: 32 tokens x 128 experts
    constexpr int BV = BN * BK / 8 / ST_THREADS;        // W loads per thread per K step
    extern __shared__ __attribute__((aligned(16))) char lds_raw[];
    __shared__ int s_cnt[SIM_EMAX];
    __bf16* sB = (__bf16*)lds_raw;                      // [2][ST_WCH][BN][LDK]
    float* sH = (float*)lds_raw;                        // [ST_BM][ST_LDH], after the K loop

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lrow = tid >> 3, lch = (tid & 7) * 8;     // W load slot: rows lrow + 64 v
    const int E = a.E, d = a.d;
    const int KT = d / BK;
    const int ntiles = (int)((a.T_cal + ST_BM - 1) / ST_BM);
    for (int i = tid; i < SIM_EMAX; i += ST_THREADS) s_cnt[i] = 0;
    const __amdgpu_buffer_rsrc_t rb_rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.w_router), (short)0, E * d * 2, 0x00020000);
    const uint32_t boff0 = ((uint32_t)lrow * (uint32_t)d + lch) * 2u;
    const uint32_t bstride = 128u * (uint32_t)d;        // 64 rows, in bytes
    const int brow_off = (lane & 31) * LDK + (lane >> 5) * 8;
    // this wave's token staging rows, after the W buffers
    char* astg = lds_raw + (size_t)2 * ST_WCH * BN * LDK * 2 + (size_t)wave * 32 * ST_LDA;
    char* adst = astg + (lane >> 3) * ST_LDA + (lane & 7) * 16;
    const char* afrag = astg + (lane & 31) * ST_LDA + (lane >> 5) * 16;   // row lane%32, chunk 2ks + h
    constexpr uint32_t OOR = 0x80000000u;
    float* gp = a.gram_part + (int64_t)blockIdx.x * SIM_EMAX * SIM_EMAX;
    bool first_tile = true;

    const int vid = (gridDim.x & 7) == 0 ? (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3)
                                         : (int)blockIdx.x;
    for (int tile = vid; tile < ntiles; tile += gridDim.x) {
        const int64_t t0 = (int64_t)tile * ST_BM;
        const int nt = (int)((a.T_cal - t0) < ST_BM ? (a.T_cal - t0) : ST_BM);
        // this tile's tokens only: rows past the end read zeros through the range check
        const __amdgpu_buffer_rsrc_t ra_rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<__bf16*>((const __bf16*)a.x_cal + t0 * d), (short)0, nt * d * 2, 0x00020000);
        // token reads: lane l takes row 8i + l/8 of the wave's 32, 16-byte chunk l%8 of the step
        const uint32_t aoff = ((uint32_t)(wave * 32 + (lane >> 3)) * (uint32_t)d + 8u * (lane & 7)) * 2u;
        const uint32_t astride8 = 16u * (uint32_t)d;    // 8 rows, in bytes

        f32x16 acc[FN];
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
        bf16x8 ax[S][4];                                // token operands of S K steps
        bf16x8 rb[S][BV], bfr[FN];                      // W rows of S K steps
        auto loadA = [&](int st, int step) {
            const uint32_t ok = step < KT ? 0u : OOR;    // past the end: zeros, never used
            const uint32_t k0 = (uint32_t)step * BK * 2u;
#pragma unroll
            for (int i = 0; i < 4; ++i) ax[st][i] = st_load16(ra_rs, (aoff + i * astride8) | ok, k0);
        };
        auto loadB = [&](int st, int step) {
            const uint32_t ok = step < KT ? 0u : OOR;
#pragma unroll
            for (int v = 0; v < BV; ++v)
                rb[st][v] = st_load16(rb_rs, (boff0 + v * bstride) | ok, (uint32_t)step * BK * 2u);
        };
        // W of one K step into sub-buffer `sub` of LDS buffer `buf`
        auto storeB = [&](int st, int buf, int sub) {
            __bf16* p = sB + (buf * ST_WCH + sub) * BN * LDK + lrow * LDK + lch;
#pragma unroll
            for (int v = 0; v < BV; ++v) *(bf16x8*)(p + v * 64 * LDK) = rb[st][v];
        };
        auto mma = [&](int st, int buf, int sub) {
            const __bf16* pb = sB + (buf * ST_WCH + sub) * BN * LDK + brow_off;
            // the wave's own token rows: stores, then fragment reads, in program order
#pragma unroll
            for (int i = 0; i < 4; ++i) *(bf16x8*)(adst + i * 8 * ST_LDA) = ax[st][i];
            bf16x8 af[4];
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) af[ks] = *(const bf16x8*)(afrag + ks * 32);
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
                for (int j = 0; j < FN; ++j) bfr[j] = *(const bf16x8*)(pb + j * 32 * LDK + ks * 16);
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks], bfr[j], acc[j], 0, 0, 0);
            }
        };
        // The reads of one K step (tokens, then W rows) form a batch issued S
        // steps before the step is multiplied.  The memory counter retires reads
        // in issue order, so waiting for the W rows of the next chunk (to put
        // them in LDS) never waits for the younger batches still in flight.
        // W goes to LDS in chunks of ST_WCH = 2 K steps, one barrier per chunk
        // (a barrier per step cost about a tenth of the stream rate).
        // prologue: batches 0 .. S-1, W of chunk 0 in LDS
        static_assert(S % ST_WCH == 0 && ST_WCH == 2, "whole chunks per unrolled pass");
#pragma unroll
        for (int st = 0; st < S; ++st) { loadA(st, st); loadB(st, st); }
        storeB(0, 0, 0);
        storeB(1, 0, 1);
        __syncthreads();
        // steady state, unrolled by S so that every register stage has a fixed name:
        // step kt multiplies stage kt % S from sub-buffer kt % 2 of LDS buffer
        // (kt / 2) & 1 and refills the stage with batch kt + S; after the second
        // step of a chunk, W of the next chunk (steps kt + 1, kt + 2) moves to
        // the other buffer (KT is a multiple of S: d % 256 == 0 for this kernel)
        for (int kt0 = 0; kt0 < KT; kt0 += S) {
#pragma unroll
            for (int u = 0; u < S; ++u) {
                const int kt = kt0 + u;
                mma(u, (kt >> 1) & 1, u & 1);
                __builtin_amdgcn_sched_barrier(0);
                loadA(u, kt + S);
                loadB(u, kt + S);
                __builtin_amdgcn_sched_barrier(0);
                if (u & 1) {
                    storeB((u + 1) % S, ((kt + 1) >> 1) & 1, 0);
                    storeB((u + 2) % S, ((kt + 1) >> 1) & 1, 1);
                    __syncthreads();
                }
            }
        }
        __syncthreads();   // every wave is done with the W buffers
        // park H: element e of a 32x32 block is token (e/4)*8 + (lane/32)*4 + e%4,
        // expert lane%32
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int tr = wave * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
                sH[tr * ST_LDH + j * 32 + (lane & 31)] = acc[j][e];
            }
        __syncthreads();

        // activation counts: top-k of each token's logits, ties to the lower
        // index.  Two threads per token: lanes l and l + 32 of wave w take token
        // 32 w + l % 32, the first scanning experts 0..63, the second 64..127.
        // A logit and its expert form one 64-bit key (order-preserving bits of
        // the logit, -0 as +0, then 0xFFFF - expert), so that a larger key is a
        // larger logit or, on equal logits, the lower index; -inf, NaN and the
        // padding past E get key 0 and are never counted.  Each thread keeps
        // its top eight keys sorted: every batch of eight logits is sorted by a
        // 19-comparator network and merged in (the elementwise larger of the
        // list and the reversed batch is bitonic and holds the top eight; three
        // half-cleaner stages sort it).  The two halves' lists merge the same
        // way.
        {
            constexpr int MK = ORDERMOE_MAX_TOPK;
            static_assert(MK == 8, "the sorting networks are for eight keys");
            // the lane index passes through an empty asm, so that the token's
            // addresses are formed here rather than held across the tile loop
            int lane_t = lane;
            asm volatile("" : "+v"(lane_t));
            const int tt = wave * 32 + (lane_t & 31);
            const int half = lane_t >> 5;
            auto cx = [](uint64_t& x, uint64_t& y) {          // x <- larger, y <- smaller
                const bool c = x < y;
                const uint64_t hi = c ? y : x, lo = c ? x : y;
                x = hi;
                y = lo;
            };
            auto sort8 = [&](uint64_t* s) {
                cx(s[0], s[1]); cx(s[2], s[3]); cx(s[4], s[5]); cx(s[6], s[7]);
                cx(s[0], s[2]); cx(s[1], s[3]); cx(s[4], s[6]); cx(s[5], s[7]);
                cx(s[1], s[2]); cx(s[5], s[6]);
                cx(s[0], s[4]); cx(s[1], s[5]); cx(s[2], s[6]); cx(s[3], s[7]);
                cx(s[2], s[4]); cx(s[3], s[5]);
                cx(s[1], s[2]); cx(s[3], s[4]); cx(s[5], s[6]);
            };
            // L <- top eight of L and S, both sorted in descending order
            auto merge8 = [&](uint64_t* L, const uint64_t* S) {
#pragma unroll
                for (int r = 0; r < 8; ++r) L[r] = L[r] > S[7 - r] ? L[r] : S[7 - r];
                cx(L[0], L[4]); cx(L[1], L[5]); cx(L[2], L[6]); cx(L[3], L[7]);
                cx(L[0], L[2]); cx(L[1], L[3]); cx(L[4], L[6]); cx(L[5], L[7]);
                cx(L[0], L[1]); cx(L[2], L[3]); cx(L[4], L[5]); cx(L[6], L[7]);
            };
            auto key = [&](float v, int e) -> uint64_t {
                const bool keep = e < E && v > -__builtin_inff();          // false for NaN too
                const uint32_t u = __float_as_uint(v == 0.f ? 0.f : v);
                const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
                return keep ? ((uint64_t)o << 32) | (uint32_t)(0xFFFF - e) : 0ull;
            };
            const float* row = sH + (tt < nt ? tt : 0) * ST_LDH + half * (SIM_EMAX / 2);
            const int e0 = half * (SIM_EMAX / 2);
            uint64_t L[8], S[8];
            auto batch = [&](int b) {
                const f32x4 v0 = *(const f32x4*)(row + 8 * b), v1 = *(const f32x4*)(row + 8 * b + 4);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    S[q] = key(v0[q], e0 + 8 * b + q);
                    S[4 + q] = key(v1[q], e0 + 8 * b + 4 + q);
                }
                sort8(S);
            };
            batch(0);
#pragma unroll
            for (int r = 0; r < 8; ++r) L[r] = S[r];
#pragma unroll 1
            for (int b = 1; b < SIM_EMAX / 2 / 8; ++b) {
                batch(b);
                merge8(L, S);
            }
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const uint32_t lo = (uint32_t)L[r], hi = (uint32_t)(L[r] >> 32);
                S[r] = ((uint64_t)(uint32_t)__shfl_xor((int)hi, 32) << 32) | (uint32_t)__shfl_xor((int)lo, 32);
            }
            merge8(L, S);
            if (half == 0 && tt < nt) {
                if (a.top1) a.top1[t0 + tt] = L[0] ? (int)(0xFFFFu - (uint32_t)(L[0] & 0xFFFFu)) : -1;
#pragma unroll
                for (int r = 0; r < MK; ++r)
                    if (r < a.k && L[r]) atomicAdd(&s_cnt[0xFFFFu - (uint32_t)(L[r] & 0xFFFFu)], 1);
            }
        }
        __syncthreads();   // the top-k is done with the fp32 H tile
        // Gram += H^T H over this tile's tokens by v_mfma_f32_32x32x16_bf16 on
        // a two-term bf16 split H = h + l (h = bf16(H), l = bf16(H - h)):
        // H_i H_j ~ h_i h_j + h_i l_j + l_i h_j, leaving out l_i l_j and the
        // rounding of l, each below 2^-17 |H_i H_j|; the products are exact in
        // the fp32 accumulators.  H^T goes to LDS as h and l planes [expert]
        // [token] straight from the K-loop accumulators (tokens past the tile
        // end are zero rows).  Wave w owns the 32 x 32 Gram blocks
        // (w / 2, 2 (w % 2)) and (w / 2, 2 (w % 2) + 1).
        {
            constexpr int LDT = ST_LDT;
            __bf16* sHh = (__bf16*)lds_raw;                 // [SIM_EMAX][LDT]
            __bf16* sHl = sHh + SIM_EMAX * LDT;
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int ex = j * 32 + (lane & 31);
                    const int tk = wave * 32 + g * 8 + (lane >> 5) * 4;
                    bf16x4 hv, lv;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float x = acc[j][4 * g + q];
                        const __bf16 h = (__bf16)x;
                        hv[q] = h;
                        lv[q] = (__bf16)(x - (float)h);
                    }
                    *(bf16x4*)(sHh + ex * LDT + tk) = hv;
                    *(bf16x4*)(sHl + ex * LDT + tk) = lv;
                }
            __syncthreads();
            const int bi = wave >> 1, bj0 = (wave & 1) * 2;
            f32x16 g0, g1;
            // element e of a block: row (e/4)*8 + (lane/32)*4 + e%4, column lane%32
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int gr = bi * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
                const int gc = lane & 31;
                g0[e] = first_tile ? 0.f : gp[gr * SIM_EMAX + bj0 * 32 + gc];
                g1[e] = first_tile ? 0.f : gp[gr * SIM_EMAX + (bj0 + 1) * 32 + gc];
            }
            // operand lane l: expert row l % 32 of the block, tokens t + 8 (l / 32) .. +7
            const int ro = (lane & 31) * LDT + (lane >> 5) * 8;
            const __bf16* pa = sHh + bi * 32 * LDT + ro;
            const __bf16* pb0 = sHh + bj0 * 32 * LDT + ro;
            const __bf16* pb1 = sHh + (bj0 + 1) * 32 * LDT + ro;
            constexpr int PL = SIM_EMAX * LDT;              // h plane -> l plane
#pragma unroll 4
            for (int t = 0; t < ST_BM; t += 16) {
                const bf16x8 ah = *(const bf16x8*)(pa + t), al = *(const bf16x8*)(pa + PL + t);
                const bf16x8 b0h = *(const bf16x8*)(pb0 + t), b0l = *(const bf16x8*)(pb0 + PL + t);
                const bf16x8 b1h = *(const bf16x8*)(pb1 + t), b1l = *(const bf16x8*)(pb1 + PL + t);
                g0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b0h, g0, 0, 0, 0);
                g1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b1h, g1, 0, 0, 0);
                g0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b0l, g0, 0, 0, 0);
                g1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b1l, g1, 0, 0, 0);
                g0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b0h, g0, 0, 0, 0);
                g1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b1h, g1, 0, 0, 0);
            }
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int gr = bi * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
                const int gc = lane & 31;
                gp[gr * SIM_EMAX + bj0 * 32 + gc] = g0[e];
                gp[gr * SIM_EMAX + (bj0 + 1) * 32 + gc] = g1[e];
            }
        }
        first_tile = false;
        __syncthreads();   // before the next tile's W overwrites H
    }
    if (first_tile)        // no tile for this workgroup: an empty partial
        for (int p = tid; p < SIM_EMAX * SIM_EMAX; p += ST_THREADS) gp[p] = 0.f;
    __syncthreads();
    for (int i = tid; i < SIM_EMAX; i += ST_THREADS) a.count_part[(int64_t)blockIdx.x * SIM_EMAX + i] = s_cnt[i];
}


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

// Fixed-order fp64 sum of the per-block partial Gram matrices and counts.
// A block of 1024 threads takes 64 consecutive entries; thread (s, c) adds the
// parts s, s + 16, ... of entry c (independent loads, coalesced over c), then
// the 16 slices are added in slice order.
constexpr int RED_SLICES = 16, RED_COLS = 64;

__global__ void __launch_bounds__(RED_SLICES * RED_COLS) sim_reduce_kernel(const SimArgs a, int nparts,
                                                                           double* gram) {
    __shared__ double s_g[RED_SLICES][RED_COLS];
    __shared__ int64_t s_c[RED_SLICES][RED_COLS];
    const int c = threadIdx.x % RED_COLS, sl = threadIdx.x / RED_COLS;
    const int p = blockIdx.x * RED_COLS + c;            // entry of the 128 x 128 Gram
    double g = 0.0;
    int64_t n = 0;
    const float* src = a.gram_part + p;
#pragma unroll 4
    for (int b = sl; b < nparts; b += RED_SLICES) g += (double)src[(int64_t)b * SIM_EMAX * SIM_EMAX];
    if (p < SIM_EMAX)
        for (int b = sl; b < nparts; b += RED_SLICES) n += a.count_part[(int64_t)b * SIM_EMAX + p];
    s_g[sl][c] = g;
    s_c[sl][c] = n;
    __syncthreads();
    if (sl == 0) {
        double t = 0.0;
        int64_t m = 0;
        for (int q = 0; q < RED_SLICES; ++q) { t += s_g[q][c]; m += s_c[q][c]; }
        gram[p] = t;
        if (p < a.E) a.counts[p] = m;
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

}  // namespace

int64_t similarity_tokens_per_chunk(int) { return SIM_TC; }
int similarity_max_experts() { return SIM_EMAX; }

int launch_similarity(const SimArgs& a, void* stream) {
    hipStream_t st = (hipStream_t)stream;
    int nparts = a.nchunk;
    hipError_t e;
    if (a.dtype == ORDERMOE_BF16 && a.d % (ST_BK * ST_STAGES) == 0) {
        static int lds_ok = -1;
        if (lds_ok < 0)
            lds_ok = (int)hipFuncSetAttribute((const void*)sim_tile_kernel,
                                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)ST_LDS);
        if (lds_ok) return lds_ok;
        // one workgroup per tile up to the partial slots the workspace holds
        const int64_t ntiles = (a.T_cal + ST_BM - 1) / ST_BM;
        nparts = (int)(ntiles < a.nchunk ? ntiles : a.nchunk);
        KernelTimer kt_("sim_partial", st);
        sim_tile_kernel<<<dim3(nparts), dim3(ST_THREADS), ST_LDS, st>>>(a);
    } else {
        KernelTimer kt_("sim_partial", st);
        hipLaunchKernelGGL(sim_partial_kernel, dim3(a.nchunk), dim3(256), 0, st, a);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
    {
        KernelTimer kt_("sim_reduce", st);
        hipLaunchKernelGGL(sim_reduce_kernel, dim3(SIM_EMAX * SIM_EMAX / RED_COLS), dim3(RED_SLICES * RED_COLS),
                           0, st, a, nparts, a.gram);
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

}  // namespace ordermoe
