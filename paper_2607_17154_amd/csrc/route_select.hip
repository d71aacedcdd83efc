// Routing and runtime server-expert selection of one MoE layer on gfx950.
//
// Kernel 1 (route_select_kernel), one block of 8 waves per TB tokens (TB = 16,
// or 32 for large batches of at most 64 experts), compiled for slot bounds of
// 2, 4, 6 and 8 (the smallest that holds k runs):
//   * the first words of the candidate tables are read into registers first,
//     so that their latency hides behind the router loop, and stored to LDS
//     after it together with the rest;
//   * router logits l = x W_r^T (eq 3, one token at a time):
//       bf16: v_mfma_f32_16x16x32_bf16 on 16-token row groups, the K steps of a
//             row group split over its waves, partial sums added in wave order;
//       fp32: fp64 dot products (exact products), rounded once to fp32;
//   * per token (16 lanes, one DPP row): top-(k+1) by a 64-bit (logit, -index)
//     key max-reduced over the row with DPP rotations, gates, margin and flag;
//   * per slot in rank order: the candidate search of eq (40)/(43) -- lane 0
//     takes the exact candidate, lane j the (j-1)-th substitute of the LDS-
//     staged table; each lane scans the servers holding its expert and keeps a
//     64-bit key (J, position, remote, server); a min-reduce over the row gives
//     (m*, k*); the budget is updated as eq (44);
//   * per-block counters and per-destination remote-slot counts.
// Kernel 2 (dispatch_kernel), one block per TB tokens: each block totals the
//   per-block destination counts of the blocks before it (the exclusive scan,
//   redone per block so that no separate scan kernel is needed), then places
//   its own remote slots, stably, into the (destination, token, slot) ordered
//   dispatch list; block 0 also writes the counter totals and the
//   per-destination counts.
// Batches of at most 1024 slots run kernel 2 as one single-block kernel
// (dispatch_small_kernel).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.hpp"

namespace ordermoe {
namespace {

constexpr int RT_TB = 16;        // tokens per block (RT_TB2 for large batches)
constexpr int RT_TB2 = 32;
constexpr int RT_THREADS = 512;  // 8 waves share the router's K loop, then run the
                                 // token stage, 16 lanes per token
constexpr int RT_WAVES = RT_THREADS / 64;
constexpr int RT_SLOTS = 4;      // partial-sum slots of the wave reduction

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

// Reductions over each row of 16 lanes (one token's lanes) with DPP row
// rotations by 8, 4, 2, 1: after the four steps every lane of the row holds
// the result.  Max and min are exact in any order; the float sum is used by
// lane 0 of the row only.
template <int CTRL>
__device__ inline uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ inline uint64_t dpp_u64(uint64_t v) {
    const uint32_t lo = dpp_u32<CTRL>((uint32_t)v), hi = dpp_u32<CTRL>((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}
constexpr int DPP_ROR8 = 0x128, DPP_ROR4 = 0x124, DPP_ROR2 = 0x122, DPP_ROR1 = 0x121;
__device__ inline uint64_t row_max_u64(uint64_t v) {
    uint64_t o;
    o = dpp_u64<DPP_ROR8>(v); v = o > v ? o : v;
    o = dpp_u64<DPP_ROR4>(v); v = o > v ? o : v;
    o = dpp_u64<DPP_ROR2>(v); v = o > v ? o : v;
    o = dpp_u64<DPP_ROR1>(v); v = o > v ? o : v;
    return v;
}
__device__ inline uint64_t row_min_u64(uint64_t v) {
    uint64_t o;
    o = dpp_u64<DPP_ROR8>(v); v = o < v ? o : v;
    o = dpp_u64<DPP_ROR4>(v); v = o < v ? o : v;
    o = dpp_u64<DPP_ROR2>(v); v = o < v ? o : v;
    o = dpp_u64<DPP_ROR1>(v); v = o < v ? o : v;
    return v;
}
__device__ inline float row_sum_f32(float v) {
    v += __uint_as_float(dpp_u32<DPP_ROR8>(__float_as_uint(v)));
    v += __uint_as_float(dpp_u32<DPP_ROR4>(__float_as_uint(v)));
    v += __uint_as_float(dpp_u32<DPP_ROR2>(__float_as_uint(v)));
    v += __uint_as_float(dpp_u32<DPP_ROR1>(__float_as_uint(v)));
    return v;
}

// Raw buffer loads: the hardware range check returns zeros for offsets at or
// past the resource's size, so rows and experts outside the batch need no
// branch (their offset is set to RT_OOR).
constexpr uint32_t RT_OOR = 0x80000000u;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ inline bf16x8 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0));
}

// Router partial logits of one 16-token row group (first token tr0) over the
// K steps of 32 that belong to wave kw of the KW waves sharing the row group
// (steps kw, kw + KW, ...): v_mfma_f32_16x16x32_bf16 with the tokens as rows
// and 16 experts per block as columns.  The steps go in groups of U with two
// register sets: the reads of the next group are in flight while the current
// group is multiplied.  Steps past the end read zeros and add nothing.
template <int NB, int U, int KW>
__device__ inline void router_k_loop(const RouteArgs& a, int kw, int lane, int64_t tr0, f32x4* acc) {
    const int d = a.d, E = a.E;
    const int r16 = lane & 15, kg = (lane >> 4) * 8;
    const int64_t left = a.T - tr0;
    const int nrows = left < 0 ? 0 : (left > 16 ? 16 : (int)left);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc((const __bf16*)a.x + (tr0 < a.T ? tr0 : 0) * (int64_t)d,
                                                (uint32_t)nrows * (uint32_t)d * 2u);
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w_router, (uint32_t)E * (uint32_t)d * 2u);
    const uint32_t xo = r16 < nrows ? ((uint32_t)r16 * (uint32_t)d + kg) * 2u : RT_OOR;
    uint32_t wo[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int e = nb * 16 + r16;
        wo[nb] = e < E ? ((uint32_t)e * (uint32_t)d + kg) * 2u : RT_OOR;
    }
    const int nsteps = d / 32;
    const int ns = (nsteps - kw + KW - 1) / KW;       // steps of this wave
    const int ngroups = (ns + U - 1) / U;
    bf16x8 av[2][U], bv[2][U][NB];
    auto load = [&](int buf, int grp) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = grp * U + u;
            const uint32_t past = i < ns ? 0u : RT_OOR;
            const uint32_t so = (uint32_t)(kw + KW * (i < ns ? i : 0)) * 64u;   // bytes
            av[buf][u] = buf_load16(rx, xo | past, so);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bv[buf][u][nb] = buf_load16(rw, wo[nb] | past, so);
        }
    };
    auto mma = [&](int buf) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[buf][u], bv[buf][u][nb], acc[nb], 0, 0, 0);
    };
    load(0, 0);
    for (int g = 0; g < ngroups; g += 2) {
        load(1, g + 1);
        __builtin_amdgcn_sched_barrier(0);
        mma(0);
        __builtin_amdgcn_sched_barrier(0);
        load(0, g + 2);
        __builtin_amdgcn_sched_barrier(0);
        mma(1);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Router partial logits of a 16-token block of at most 16 experts whose token
// rows fit in LDS (d % 512 == 0, d <= RT_XLDS_MAX_D): the block's 16 rows go
// from memory straight into LDS in whole 1 KB pieces, every piece of every wave
// issued at once beside the wave's router fragments (into registers), so that
// the block's whole share of the token stream is in flight together instead of
// two groups of steps per wave.  Row r sits at r (2d + RT_XPAD) bytes: the pad
// puts the 16 rows of one fragment read on distinct banks.  Then the wave's K
// steps (kw, kw + KW, ...) as in router_k_loop, token fragments read from LDS.
// Rows past the batch lie past the buffer resource and arrive as zeros.
constexpr int RT_XLDS_MAX_D = 4096;
constexpr int RT_XPAD = 16;                  // bytes

__host__ __device__ inline int route_xlds_bytes(int d) { return RT_TB * (2 * d + RT_XPAD); }

typedef __attribute__((address_space(3))) void* lds_ptr;

// The reads: the wave's router fragments into wv, its token pieces into LDS.
template <int KW>
__device__ inline void router_dma_issue(const RouteArgs& a, int kw, int lane, int64_t tr0, char* sx, bf16x8* wv) {
    constexpr int MAXS = RT_XLDS_MAX_D / (32 * KW);   // K steps (and pieces) per wave
    const int d = a.d, E = a.E;
    const int r16 = lane & 15, kg = (lane >> 4) * 8;
    const int64_t left = a.T - tr0;                   // >= 1: the block holds a token
    const int nrows = left > 16 ? 16 : (int)left;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc((const __bf16*)a.x + tr0 * (int64_t)d, (uint32_t)nrows * (uint32_t)d * 2u);
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w_router, (uint32_t)E * (uint32_t)d * 2u);
    const int ns = d / (32 * KW);
    const int cpr = d / 512;                          // 1 KB pieces per token row
    const uint32_t xs = 2u * (uint32_t)d + RT_XPAD;
    const uint32_t wo = r16 < E ? ((uint32_t)r16 * (uint32_t)d + kg) * 2u : RT_OOR;
#pragma unroll
    for (int i = 0; i < MAXS; ++i)
        if (i < ns) wv[i] = buf_load16(rw, wo, (uint32_t)(kw + KW * i) * 64u);
#pragma unroll
    for (int i = 0; i < MAXS; ++i)
        if (i < ns) {
            const int p = kw + KW * i;                // piece p: row p / cpr, chunk p % cpr
            const int row = p / cpr, ch = p - row * cpr;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr)(sx + row * xs + ch * 1024), 16, lane * 16,
                                                     (uint32_t)row * 2u * (uint32_t)d + (uint32_t)ch * 1024u, 0, 0);
        }
}

// The MFMAs, after every piece of the block has arrived.
template <int KW>
__device__ inline void router_dma_mma(const RouteArgs& a, int kw, int lane, f32x4* acc, const char* sx,
                                      const bf16x8* wv) {
    constexpr int MAXS = RT_XLDS_MAX_D / (32 * KW);
    const int d = a.d;
    const int r16 = lane & 15, kg = (lane >> 4) * 8;
    const int ns = d / (32 * KW);
    const uint32_t xs = 2u * (uint32_t)d + RT_XPAD;
    __syncthreads();                                  // waits for every piece (vmcnt 0), then the barrier
    const char* fr = sx + r16 * xs + kg * 2;
#pragma unroll
    for (int i = 0; i < MAXS; ++i)
        if (i < ns) {
            const bf16x8 av = *(const bf16x8*)(fr + (kw + KW * i) * 64);
            acc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, wv[i], acc[0], 0, 0, 0);
        }
}

// Router partial logits for 32-token blocks of more than 16 experts: the
// router rows are shared by both 16-token row groups through LDS.  The K axis
// goes in chunks of RT_CK = 128 (one 32-step per K wave of a row group); the
// block reads each chunk of W_r coalesced (a wave instruction covers 4 rows x
// 256 bytes) two chunks ahead into registers and stores it to one of two
// padded LDS buffers; token rows go from global memory straight into MFMA
// registers four chunks ahead.  One barrier per chunk.  Requires d % 512 == 0.
constexpr int RT_CK = 128;
constexpr int RT_WLD = RT_CK + 8;            // bf16 per LDS row of a W chunk
constexpr int RT_XD = 4;                     // token chunks in flight per wave

template <int NB>
__device__ inline void router_lds_loop(const RouteArgs& a, int kw, int lane, int tid, int64_t tr0,
                                       f32x4* acc, __bf16* sW) {
    constexpr int KW = 4;
    constexpr int TPR = RT_CK / 8;                   // threads per W row (16 bytes each)
    constexpr int RPR = RT_THREADS / TPR;            // W rows per block round
    constexpr int WR = NB * 16 / RPR;                // rounds per chunk (NB * 16 rows)
    static_assert(WR >= 1 && NB * 16 % RPR == 0, "whole rounds of W rows");
    const int d = a.d, E = a.E;
    const int r16 = lane & 15, kg = (lane >> 4) * 8;
    const int64_t left = a.T - tr0;
    const int nrows = left < 0 ? 0 : (left > 16 ? 16 : (int)left);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc((const __bf16*)a.x + (tr0 < a.T ? tr0 : 0) * (int64_t)d,
                                                (uint32_t)nrows * (uint32_t)d * 2u);
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w_router, (uint32_t)E * (uint32_t)d * 2u);
    const uint32_t xo = r16 < nrows ? ((uint32_t)r16 * (uint32_t)d + kg + 32 * kw) * 2u : RT_OOR;
    // W staging slot of this thread: row wrow + RPR * i, 8 elements at wcol of the chunk
    const int wrow = tid / TPR, wcol = (tid % TPR) * 8;
    uint32_t wo[WR];
#pragma unroll
    for (int i = 0; i < WR; ++i) {
        const int e = wrow + RPR * i;
        wo[i] = e < E ? ((uint32_t)e * (uint32_t)d + wcol) * 2u : RT_OOR;
    }
    const int NC = d / RT_CK;
    bf16x8 xr[RT_XD], wreg[2][WR];
    auto xload = [&](int slot, int c) {
        const uint32_t past = c < NC ? 0u : RT_OOR;
        xr[slot] = buf_load16(rx, xo | past, (uint32_t)(c < NC ? c : 0) * (RT_CK * 2u));
    };
    auto wload = [&](int set, int c) {
#pragma unroll
        for (int i = 0; i < WR; ++i) wreg[set][i] = buf_load16(rw, wo[i], (uint32_t)c * (RT_CK * 2u));
    };
    auto wstore = [&](int buf, int set) {
        __bf16* p = sW + buf * (NB * 16 * RT_WLD) + wrow * RT_WLD + wcol;
#pragma unroll
        for (int i = 0; i < WR; ++i) *(bf16x8*)(p + i * RPR * RT_WLD) = wreg[set][i];
    };
    const __bf16* frag = sW + r16 * RT_WLD + kw * 32 + kg;
    auto mma = [&](int buf, int slot) {
        bf16x8 bf[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) bf[nb] = *(const bf16x8*)(frag + buf * (NB * 16 * RT_WLD) + nb * 16 * RT_WLD);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xr[slot], bf[nb], acc[nb], 0, 0, 0);
    };
#pragma unroll
    for (int u = 0; u < RT_XD; ++u) xload(u, u);
    wload(0, 0);
    wload(1, 1);
    wstore(0, 0);
    __syncthreads();
    // chunk c: store chunk c+1 (read one chunk ago) to the other buffer, read
    // chunk c+2 into the freed register set, multiply chunk c, read token
    // chunk c + RT_XD into the freed slot; unrolled by RT_XD (NC % 4 == 0)
    for (int c0 = 0; c0 < NC; c0 += RT_XD) {
#pragma unroll
        for (int u = 0; u < RT_XD; ++u) {
            const int c = c0 + u;
            if (c + 1 < NC) wstore((u + 1) & 1, (u + 1) & 1);
            if (c + 2 < NC) wload(u & 1, c + 2);
            mma(u & 1, u);
            xload(u, c + RT_XD);
            __syncthreads();
        }
    }
}

// One candidate table (T1 experts, T1 losses, T1 lengths, server masks, or the
// cost table when it is staged) copied to LDS by the block in batches of whole
// block rounds: words [B * RT_THREADS, (B + P) * RT_THREADS) are read into P
// registers per thread (reads past the table re-read word 0 and are
// discarded, so no branch separates them) and stored later.  The first batch
// is read before the router loop, so that its latency hides behind the loop;
// the second batches of all tables are read together after it; whatever is
// left is copied by table_copy_from.
template <int B, int P>
__device__ inline void table_read(const int32_t* src, int n, int tid, int32_t* v) {
    if (n <= B * RT_THREADS) return;
#pragma unroll
    for (int u = 0; u < P; ++u) {
        const int i = (B + u) * RT_THREADS + tid;
        v[u] = src[i < n ? i : 0];
    }
}

template <int B, int P>
__device__ inline void table_write(int32_t* dst, int n, int tid, const int32_t* v) {
#pragma unroll
    for (int u = 0; u < P; ++u) {
        const int i = (B + u) * RT_THREADS + tid;
        if (i < n) dst[i] = v[u];
    }
}

template <int B>
__device__ inline void table_copy_from(const int32_t* src, int32_t* dst, int n, int tid) {
    for (int i0 = B * RT_THREADS + tid; i0 < n; i0 += 16 * RT_THREADS) {
        int32_t w[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) w[u] = src[i0 + u * RT_THREADS < n ? i0 + u * RT_THREADS : i0];
#pragma unroll
        for (int u = 0; u < 16; ++u)
            if (i0 + u * RT_THREADS < n) dst[i0 + u * RT_THREADS] = w[u];
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

// floats of the first LDS region: the partial-sum slots, or (32-token blocks of
// more than 16 experts) the two staged router-row buffers if larger
__host__ __device__ inline int route_region0_floats(int tb, int E, int xlds) {
    const int Epad = (E + 15) & ~15;
    const int part = RT_SLOTS * tb * Epad;
    // the staged loop keeps NBT * 16 rows per buffer (32 or 64), two buffers of bf16
    const int rows = Epad <= 32 ? 32 : 64;
    const int wbuf = (tb == RT_TB2 && Epad > 16 && Epad <= 64) ? rows * RT_WLD : 0;
    const int r = part > wbuf ? part : wbuf;
    return r > xlds / 4 ? r : xlds / 4;               // the LDS-staged token rows
}

// up to 64 experts: at most 128 VGPRs (4 waves per SIMD), so two blocks share a CU.
// KM: the slot arrays and loops of the token stage are sized for k <= KM (2, 4,
// 6 or 8), so that a top-2 layer does not carry the work of eight slots.
template <int NBT, int TB, int KM>
__global__ void __launch_bounds__(RT_THREADS) __attribute__((amdgpu_waves_per_eu(NBT <= 4 ? 4 : 2)))
route_select_kernel(const RouteArgs a) {
    static_assert(KM >= 1 && KM <= ORDERMOE_MAX_TOPK, "slots");
    constexpr int RG = TB / 16;                 // 16-token row groups of the router
    constexpr int KW = RT_WAVES / RG;           // waves sharing one row group's K loop
    static_assert(KW == 8 || KW == RT_SLOTS, "one or two reduction rounds");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t t0 = (int64_t)blockIdx.x * TB;
    const int E = a.E, d = a.d, k = a.k, M = a.M;
    const int Epad = (E + 15) & ~15;

    extern __shared__ float smem[];
    float* s_part = smem;                               // [RT_SLOTS][TB][Epad]
    float* s_logit = smem;                              // reuses slot 0 after the sum
    int32_t* s_t1k = (int32_t*)(smem + route_region0_floats(TB, E, a.x_lds));   // [E][gmax]
    float* s_t1q = (float*)(s_t1k + E * a.gmax);                   // [E][gmax]
    int32_t* s_t1n = (int32_t*)(s_t1q + E * a.gmax);               // [E]
    uint32_t* s_mask = (uint32_t*)(s_t1n + E);                     // [E]
    int* s_cnt = (int*)(s_mask + E);                               // [8 + M]
    float* s_S = (float*)(s_cnt + 8 + M);                          // [M][M][E] if a.S_in_lds
    const float* Stab = a.S_in_lds ? s_S : a.S;

    // the candidate tables: reads issued now, LDS stores after the router loop
    const int n1 = E * a.gmax, nS = a.S_in_lds ? M * M * E : 0;
    int32_t pk[2], pq[2], pn[1], pm[1], ps[2];
    table_read<0, 2>(a.t1_k, n1, tid, pk);
    table_read<0, 2>((const int32_t*)a.t1_q, n1, tid, pq);
    table_read<0, 1>(a.t1_n, E, tid, pn);
    table_read<0, 1>((const int32_t*)a.srvmask, E, tid, pm);
    table_read<0, 2>((const int32_t*)a.S, nS, tid, ps);
    for (int i = tid; i < 8 + M; i += RT_THREADS) s_cnt[i] = 0;
    // this thread's token location and budget, read before the router loop so
    // that their latency is hidden behind it (lanes of waves 0 .. TB/4-1 own tokens)
    int loc_pre = 0;
    float qhat_pre = 0.f;
    {
        const int64_t tp = t0 + (wave * 4 + (lane >> 4));
        if (wave < TB / 4 && tp < a.T) { loc_pre = a.loc_in[tp]; qhat_pre = a.qhat_in[tp]; }
    }

    // ---------------- router logits ----------------
    if (a.ksplit > 0) {
        // split router: add the K slices in slice order (the reads of all
        // slices of an element are issued before the additions)
        // PU elements per round: one round of 16-token blocks up to 128
        // experts (up to 64 with two, within the 128 registers of those
        // kernels); reads past the slices or the batch re-read the first
        // partial (discarded), so that no branch separates the reads
        constexpr int PU = NBT >= 8 ? 4 : 2;
        for (int i0 = tid; i0 < TB * Epad; i0 += PU * RT_THREADS) {
            float pv[PU][RT_SPLIT_MAX_K];
#pragma unroll
            for (int u = 0; u < PU; ++u) {
                const int i = i0 + u * RT_THREADS;
                const int64_t tok = t0 + i / Epad;
                const bool ok = i < TB * Epad && tok < a.T;
#pragma unroll
                for (int z = 0; z < RT_SPLIT_MAX_K; ++z)
                    pv[u][z] = a.logit_part[(z < a.ksplit && ok) ? ((int64_t)z * a.T + tok) * Epad + i % Epad : 0];
            }
#pragma unroll
            for (int u = 0; u < PU; ++u) {
                const int i = i0 + u * RT_THREADS;
                float v = 0.f;
#pragma unroll
                for (int z = 0; z < RT_SPLIT_MAX_K; ++z)
                    if (z < a.ksplit) v += pv[u][z];
                if (i < TB * Epad) s_logit[i] = (t0 + i / Epad < a.T) ? v : 0.f;
            }
        }
    } else if (a.dtype == ORDERMOE_BF16) {
        const int nblk = Epad / 16;
        const int rg = wave / KW, kw = __builtin_amdgcn_readfirstlane(wave % KW);
        f32x4 acc[NBT];
#pragma unroll
        for (int i = 0; i < NBT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        // group size: two groups of reads in flight per wave, within 128
        // registers so that two blocks share a CU
        if constexpr (NBT == 1 && TB == RT_TB) {
            if (a.x_lds) {
                bf16x8 wv[RT_XLDS_MAX_D / (32 * KW)];
                router_dma_issue<KW>(a, kw, lane, t0, (char*)smem, wv);
                // the first batch of the candidate tables (read at the start) goes
                // to LDS while the token rows arrive
                table_write<0, 2>(s_t1k, n1, tid, pk);
                table_write<0, 2>((int32_t*)s_t1q, n1, tid, pq);
                table_write<0, 1>(s_t1n, E, tid, pn);
                table_write<0, 1>((int32_t*)s_mask, E, tid, pm);
                table_write<0, 2>((int32_t*)s_S, nS, tid, ps);
                router_dma_mma<KW>(a, kw, lane, acc, (const char*)smem, wv);
            } else {
                router_k_loop<1, 4, KW>(a, kw, lane, t0, acc);
            }
        } else if constexpr (NBT == 1) router_k_loop<1, 4, KW>(a, kw, lane, t0 + rg * 16, acc);
        else if constexpr (TB == RT_TB2 && NBT == 2) router_lds_loop<2>(a, kw, lane, tid, t0 + rg * 16, acc, (__bf16*)smem);
        else if constexpr (TB == RT_TB2 && NBT == 4) router_lds_loop<4>(a, kw, lane, tid, t0 + rg * 16, acc, (__bf16*)smem);
        else if constexpr (NBT == 2) router_k_loop<2, 2, KW>(a, kw, lane, t0 + rg * 16, acc);
        else if constexpr (NBT == 4) router_k_loop<4, 2, KW>(a, kw, lane, t0 + rg * 16, acc);
        else if constexpr (NBT == 8) router_k_loop<8, 1, KW>(a, kw, lane, t0 + rg * 16, acc);
        else router_k_loop<16, 1, KW>(a, kw, lane, t0 + rg * 16, acc);
        // acc[nb][i] = partial logit of token rg*16 + (lane/16)*4 + i, expert
        // nb*16 + lane%16.  Slots are added in a fixed order: with 8 waves per
        // row group, waves 4-7 first hand their sums to waves 0-3.
        const int r16 = lane & 15;
        const int trow = rg * 16 + (lane >> 4) * 4;
        // the staged router rows and token rows share LDS with the partial-sum slots
        if constexpr (TB == RT_TB2 && (NBT == 2 || NBT == 4)) __syncthreads();
        if constexpr (NBT == 1 && TB == RT_TB)
            if (a.x_lds) __syncthreads();
        if (KW == 8 && wave >= RT_SLOTS) {
#pragma unroll
            for (int nb = 0; nb < NBT; ++nb)
                if (nb < nblk)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        s_part[((wave - RT_SLOTS) * TB + trow + i) * Epad + nb * 16 + r16] = acc[nb][i];
        }
        if (KW == 8) __syncthreads();
        if (KW == RT_SLOTS || wave < RT_SLOTS) {
            const int slot = KW == 8 ? wave : kw;
#pragma unroll
            for (int nb = 0; nb < NBT; ++nb)
                if (nb < nblk)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float* sp = &s_part[(slot * TB + trow + i) * Epad + nb * 16 + r16];
                        *sp = KW == 8 ? acc[nb][i] + *sp : acc[nb][i];
                    }
        }
        __syncthreads();
        for (int i = tid; i < TB * Epad; i += RT_THREADS) {
            float v = s_part[i];
            for (int w = 1; w < RT_SLOTS; ++w) v += s_part[w * TB * Epad + i];
            s_logit[i] = v;
        }
    } else {
        const float* X = (const float*)a.x;
        const float* W = (const float*)a.w_router;
        for (int p = tid; p < TB * Epad; p += RT_THREADS) {
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
    {
        // second batches of the larger tables, read together
        int32_t qk[2], qq[2], qs[14];
        table_read<2, 2>(a.t1_k, n1, tid, qk);
        table_read<2, 2>((const int32_t*)a.t1_q, n1, tid, qq);
        table_read<2, 14>((const int32_t*)a.S, nS, tid, qs);
        // (the LDS-staged router path wrote the first batch already)
        if (!(NBT == 1 && TB == RT_TB && a.x_lds && a.ksplit == 0 && a.dtype == ORDERMOE_BF16)) {
            table_write<0, 2>(s_t1k, n1, tid, pk);
            table_write<0, 2>((int32_t*)s_t1q, n1, tid, pq);
            table_write<0, 1>(s_t1n, E, tid, pn);
            table_write<0, 1>((int32_t*)s_mask, E, tid, pm);
            table_write<0, 2>((int32_t*)s_S, nS, tid, ps);
        }
        table_write<2, 2>(s_t1k, n1, tid, qk);
        table_write<2, 2>((int32_t*)s_t1q, n1, tid, qq);
        table_write<2, 14>((int32_t*)s_S, nS, tid, qs);
        table_copy_from<4>(a.t1_k, s_t1k, n1, tid);
        table_copy_from<4>((const int32_t*)a.t1_q, (int32_t*)s_t1q, n1, tid);
        table_copy_from<1>(a.t1_n, s_t1n, E, tid);
        table_copy_from<1>((const int32_t*)a.srvmask, (int32_t*)s_mask, E, tid);
        table_copy_from<16>((const int32_t*)a.S, (int32_t*)s_S, nS, tid);
    }
    __syncthreads();

    // ---------------- per-token stage: 16 lanes (one DPP row) per token ----------------
    if (wave < TB / 4) {
    const int g = lane >> 4;                 // token within the wave
    const int j = lane & 15;                 // lane within the token's row
    const int tr = wave * 4 + g;             // token within the block
    const int64_t t = t0 + tr;
    const bool valid = t < a.T;
    const float* lg = s_logit + tr * Epad;

    // top-(k+1) selection by (logit desc, index asc); this lane's logits (experts
    // j + 16 i) are read once and kept as order-preserving keys
    const int kk1 = (k + 1 < E) ? k + 1 : E;
    // (reads at clamped addresses and selects instead of branches, so that the
    // LDS reads issue together and no per-element branch splits the wave)
    uint32_t okey[NBT];
#pragma unroll
    for (int i = 0; i < NBT; ++i) {
        const int e = j + 16 * i;
        const float v = lg[e < E ? e : E - 1];
        okey[i] = e < E ? f2ord(v) : 0u;
    }
    uint32_t removed = 0;                    // bit i: local element j + 16 i taken
    int sel_e[KM + 1];
    float sel_v[KM + 1];
#pragma unroll
    for (int r = 0; r < KM + 1; ++r) {
        if (r < kk1) {
            uint64_t best = 0;
#pragma unroll
            for (int i = 0; i < NBT; ++i) {
                const int e = j + 16 * i;
                const bool live = e < E && !((removed >> i) & 1u);
                const uint64_t key = live ? (((uint64_t)okey[i] << 32) | (uint32_t)(0xFFFFu - (uint32_t)e)) : 0ull;
                best = key > best ? key : best;
            }
            best = row_max_u64(best);
            const int e = (int)(0xFFFFu - (uint32_t)(best & 0xFFFFu));
            sel_e[r] = e;
            sel_v[r] = ord2f((uint32_t)(best >> 32));
            if ((e & 15) == j) removed |= 1u << (e >> 4);
        }
    }
    float mg = __builtin_inff();
#pragma unroll
    for (int r = 0; r < KM; ++r) {
        if (r + 1 < kk1) {
            float gap = sel_v[r] - sel_v[r + 1];
            mg = gap < mg ? gap : mg;
        }
    }
    // gates: softmax renormalised over the top-k, or over all experts
    float den = 0.f;
    if (a.renorm) {
#pragma unroll
        for (int r = 0; r < KM; ++r)
            if (r < k) den += expf(sel_v[r] - sel_v[0]);
    } else {
        for (int e = j; e < E; e += 16) den += expf(lg[e] - sel_v[0]);
        den = row_sum_f32(den);
    }

    // server-expert selection.  Lane j holds candidate j of every slot: j = 0
    // the exact target, j >= 1 its (j-1)-th substitute in the LDS-staged table.
    // The search does not depend on the budget, so it runs for all slots at
    // once: each lane keeps, per slot, the smallest 64-bit key (J, position,
    // remote, server, expert) over the servers holding its expert.  Then the
    // slots are taken in rank order: the budget test of eq (40) masks the
    // substitutes, a min over the row picks (m*, k*) (eq 43) and the budget is
    // updated as eq (44).
    const int s_loc = loc_pre;
    const bool loc_ok = s_loc < M;
    float qhat = qhat_pre;
    const bool subs_on = a.allow_sub && a.Qbar > 0.f;
    const uint32_t mmask = M >= 32 ? 0xFFFFFFFFu : ((1u << M) - 1u);   // servers that exist
    const int jm1 = j >= 1 ? j - 1 : 0;
    int ke[KM];
    float qe[KM];
    uint32_t msv[KM];
    uint64_t key[KM];
    bool search[KM];
    // every slot's table reads are issued (slots past k read slot 0's entries,
    // discarded), then masked, so that no per-slot branch serialises them
#pragma unroll
    for (int slot = 0; slot < KM; ++slot) {
        const bool on = slot < k;
        const int r = sel_e[on ? slot : 0];
        const uint32_t rmask = s_mask[r];
        const int nsub = s_t1n[r];
        const int tk = s_t1k[r * a.gmax + jm1];
        const float tq = s_t1q[r * a.gmax + jm1];
        // uniform over the token's row: the reductions below read only lanes of the row
        search[slot] = on && loc_ok && !(a.pin && ((rmask >> s_loc) & 1u));
        const bool sub = j >= 1 && subs_on && j - 1 < nsub;
        int kc = j == 0 ? r : (sub ? tk : -1);
        if (!on || kc < 0 || kc >= E) kc = -1;
        ke[slot] = kc;
        qe[slot] = on && sub ? tq : 0.f;
        key[slot] = ~0ull;
    }
    // the servers holding each candidate (a substitute only on the token's
    // server in the Local Substitute Only mode)
    const uint32_t lmask = a.allow_sub == 2 && j >= 1 ? 1u << (s_loc & 31) : ~0u;
#pragma unroll
    for (int slot = 0; slot < KM; ++slot) {
        const uint32_t hm = s_mask[ke[slot] >= 0 ? ke[slot] : 0];
        msv[slot] = search[slot] && ke[slot] >= 0 ? hm & mmask & lmask : 0u;
    }
    // servers holding each candidate, one per round for every slot together
    for (;;) {
        uint32_t any = 0;
#pragma unroll
        for (int slot = 0; slot < KM; ++slot) any |= msv[slot];
        if (!__builtin_amdgcn_ballot_w64(any != 0)) break;
#pragma unroll
        for (int slot = 0; slot < KM; ++slot) {
            if (msv[slot]) {
                const int m = __builtin_ctz(msv[slot]);
                msv[slot] &= msv[slot] - 1;
                const float J = fmaf(a.cq, qe[slot], Stab[((int64_t)s_loc * M + m) * E + ke[slot]]);
                // J's order as a float (negative costs included; -0 counts as +0)
                const uint64_t cand = ((uint64_t)f2ord(J == 0.f ? 0.f : J) << 32) | ((uint32_t)j << 16) |
                                      ((uint32_t)(m != s_loc) << 15) | ((uint32_t)m << 8) |
                                      (uint32_t)ke[slot];
                key[slot] = cand < key[slot] ? cand : key[slot];
            }
        }
    }
    int first_m = s_loc, ncls[4] = {0, 0, 0, 0}, nremote = 0;
    uint32_t dstmask = 0;
#pragma unroll
    for (int slot = 0; slot < KM; ++slot) {
        if (slot >= k) break;
        const int r = sel_e[slot];
        int km = r, mm = s_loc;
        float qsel = 0.f;
        if (search[slot]) {
            // eq (40): a substitute must fit the remaining budget; the exact target always does
            uint64_t kk = (j == 0 || qhat + qe[slot] <= a.Qbar) ? key[slot] : ~0ull;
            kk = row_min_u64(kk);
            const int pos = (int)((kk >> 16) & 15u);
            mm = (int)((kk >> 8) & 31u);
            km = (int)(kk & 0xFFu);
            // the chosen candidate's loss, from its lane (a sum of one term: exact)
            qsel = row_sum_f32(j == pos ? qe[slot] : 0.f);
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

// The dispatch list, one block per routing block.  Each block first totals
// the routing blocks' per-destination counts on its own (a few thousand
// integers at most): its first position inside each destination's segment
// (the counts of the blocks before it) and every destination's total, from
// which the segment starts follow in server order; block 0 also writes the
// per-destination totals and the eight counters.  Then each remote slot of the
// block goes to segment start + block position + its rank among the block's
// earlier slots to the same destination (slot order), so the list is sorted by
// (destination, token, slot).
__global__ void __launch_bounds__(RT_THREADS)
dispatch_kernel(const int32_t* blk_dst, const int64_t* blk_cnt, int nblk, const uint8_t* exec_m,
                const uint8_t* loc_in, int64_t T, int k, int M, int tb, int32_t* dst_count, int64_t* counters,
                int32_t* dispatch) {
    __shared__ int8_t s_dst[RT_TB2 * ORDERMOE_MAX_TOPK];
    __shared__ int32_t s_base[ORDERMOE_MAX_SERVERS], s_tot[ORDERMOE_MAX_SERVERS], s_start[ORDERMOE_MAX_SERVERS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = (int)blockIdx.x;
    // this thread's slot, read first so that its latency overlaps the totals
    const int64_t t0 = (int64_t)b * tb;
    const int n = tb * k;
    int s_loc = M, s_m = 0;
    if (tid < n) {
        const int64_t t = t0 + tid / k;
        if (t < T) {
            s_loc = loc_in[t];
            s_m = exec_m[t * k + tid % k];
        }
    }
    for (int m = wave; m < M; m += RT_WAVES) {
        int32_t lo = 0, tot = 0;
        for (int i = lane; i < nblk; i += 64) {
            const int32_t v = blk_dst[(int64_t)i * M + m];
            tot += v;
            lo += i < b ? v : 0;
        }
        for (int off = 32; off >= 1; off >>= 1) {
            lo += __shfl_xor(lo, off);
            tot += __shfl_xor(tot, off);
        }
        if (lane == 0) { s_base[m] = lo; s_tot[m] = tot; }
    }
    if (b == 0 && wave < 8) {
        int64_t v = 0;
        for (int i = lane; i < nblk; i += 64) v += blk_cnt[(int64_t)i * 8 + wave];
        for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
        if (lane == 0) counters[wave] = v;
    }
    if (tid < n) s_dst[tid] = (int8_t)(s_loc < M && s_m != s_loc ? s_m : -1);
    __syncthreads();
    if (tid == 0) {
        int32_t acc = 0;
        for (int m = 0; m < M; ++m) { s_start[m] = acc; acc += s_tot[m]; }
    }
    if (b == 0 && tid < M) dst_count[tid] = s_tot[tid];
    __syncthreads();
    if (tid < n && s_dst[tid] >= 0) {
        const int dst = s_dst[tid];
        int rank = 0;
        for (int i = 0; i < tid; ++i) rank += (s_dst[i] == dst);
        dispatch[s_start[dst] + s_base[dst] + rank] = (int32_t)((t0 + tid / k) * k + tid % k);
    }
}

// Batches of at most DS_THREADS slots (decode): the dispatch list in one block,
// one slot per thread -- totals of the routing blocks' counters, each slot's
// rank among its wave's slots to the same destination (ballots), destination
// totals and segment starts, placement.  Replaces the scan and scatter kernels.
constexpr int DS_THREADS = 1024;
constexpr int DS_WAVES = DS_THREADS / 64;

__global__ void __launch_bounds__(DS_THREADS)
dispatch_small_kernel(const int64_t* blk_cnt, int nblk, const uint8_t* exec_m, const uint8_t* loc_in,
                      int64_t T, int k, int M, int32_t* dst_count, int64_t* counters, int32_t* dispatch) {
    __shared__ int32_t s_wcnt[DS_WAVES][ORDERMOE_MAX_SERVERS];
    __shared__ int32_t s_tot[ORDERMOE_MAX_SERVERS];
    __shared__ int32_t s_start[ORDERMOE_MAX_SERVERS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (wave < 8) {
        int64_t v = 0;
        for (int b = lane; b < nblk; b += 64) v += blk_cnt[(int64_t)b * 8 + wave];
        for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
        if (lane == 0) counters[wave] = v;
    }
    const int n = (int)(T * k);
    int dst = -1;
    if (tid < n) {
        const int s = loc_in[tid / k];
        const int m = exec_m[tid];
        if (s < M && m != s) dst = m;
    }
    int rank = 0;
    for (int m = 0; m < M; ++m) {
        const uint64_t bal = __ballot(dst == m);
        if (lane == 0) s_wcnt[wave][m] = __popcll(bal);
        if (dst == m) rank = __popcll(bal & ((1ull << lane) - 1ull));
    }
    __syncthreads();
    if (tid < M) {
        int32_t tot = 0;
        for (int w = 0; w < DS_WAVES; ++w) tot += s_wcnt[w][tid];
        s_tot[tid] = tot;
        dst_count[tid] = tot;
    }
    __syncthreads();
    if (tid == 0) {
        int32_t acc = 0;
        for (int m = 0; m < M; ++m) { s_start[m] = acc; acc += s_tot[m]; }
    }
    __syncthreads();
    if (dst >= 0) {
        int32_t pos = s_start[dst] + rank;
        for (int w = 0; w < wave; ++w) pos += s_wcnt[w][dst];
        dispatch[pos] = tid;                      // slot index token * k + slot
    }
}

template <int NBT, int TB, int KM>
int launch_route_kernel_k(const RouteArgs& a, size_t smem, hipStream_t st) {
    if (smem > 65536) {
        hipError_t e = hipFuncSetAttribute((const void*)route_select_kernel<NBT, TB, KM>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return (int)e;
    }
    KernelTimer kt_("route_select", st);
    hipLaunchKernelGGL((route_select_kernel<NBT, TB, KM>), dim3(a.nblk), dim3(RT_THREADS), smem, st, a);
    return (int)hipGetLastError();
}

// the kernel sized for the smallest slot bound (2, 4, 6, 8) that holds k
template <int NBT, int TB>
int launch_route_kernel(const RouteArgs& a, size_t smem, hipStream_t st) {
    if (a.k <= 2) return launch_route_kernel_k<NBT, TB, 2>(a, smem, st);
    if (a.k <= 4) return launch_route_kernel_k<NBT, TB, 4>(a, smem, st);
    if (a.k <= 6) return launch_route_kernel_k<NBT, TB, 6>(a, smem, st);
    return launch_route_kernel_k<NBT, TB, ORDERMOE_MAX_TOPK>(a, smem, st);
}

size_t route_smem(int tb, int E, int gmax, int M, bool S_in_lds, int xlds) {
    return sizeof(float) * (size_t)route_region0_floats(tb, E, xlds) + (size_t)E * gmax * 8 + (size_t)E * 8 +
           sizeof(int) * (size_t)(8 + M) + (S_in_lds ? sizeof(float) * (size_t)M * M * E : 0);
}

constexpr size_t RT_LDS_MAX = 160 * 1024;

// the cost table is staged in LDS when it is small enough to leave room for
// two blocks per CU, or, for batches of at most one block per CU, when it fits
bool route_S_in_lds(int tb, int E, int gmax, int M, int nblk, int xlds) {
    const size_t b = route_smem(tb, E, gmax, M, true, xlds);
    return b <= 64 * 1024 || (nblk <= 256 && b <= (xlds ? RT_LDS_MAX : 150 * 1024));
}

}  // namespace

// the workspace is sized for blocks of RT_TB tokens, the smallest block
int route_tokens_per_block() { return RT_TB; }


// partial logits of the split router: at most 256 blocks of RT_TB tokens times
// the K slices (the launcher keeps slices * blocks <= 256), every expert count
size_t route_split_buffer_floats(int64_t T) {
    const int64_t rows = T * RT_SPLIT_MAX_K < 256 * RT_TB ? T * RT_SPLIT_MAX_K : 256 * RT_TB;
    return (size_t)(rows > 0 ? rows : 1) * ORDERMOE_MAX_EXPERTS;
}

int launch_route_select(const RouteArgs& a, void* stream) {
    hipStream_t st = (hipStream_t)stream;
    const int nb = (a.E + 15) / 16;
    const int nbt = nb <= 1 ? 1 : nb <= 2 ? 2 : nb <= 4 ? 4 : nb <= 8 ? 8 : 16;
    const bool split = a.dtype == ORDERMOE_BF16 && a.T <= RT_SPLIT_MAX_T && a.logit_part;
    // Large bf16 batches take blocks of 32 tokens, so that all 8 waves run the
    // token stage: at most 16 experts from more than 512 blocks of 16 tokens,
    // 17..64 experts from 512 such blocks on (their router rows are then staged
    // in LDS and shared by the two row groups, which needs d % 512 == 0; the
    // 32-token kernels of 17..64 experts always take that loop).
    const int64_t nb16 = (a.T + RT_TB - 1) / RT_TB;
    const bool bf = a.dtype == ORDERMOE_BF16 && !split;
    const bool staged = bf && (nbt == 2 || nbt == 4) && a.d % 512 == 0 && nb16 >= 512;
    const int tb = staged || (bf && nbt == 1 && nb16 > 512) ? RT_TB2 : RT_TB;
    RouteArgs b = a;
    b.nblk = (int)((a.T + tb - 1) / tb);
    // batches of at most one 16-token block per CU stage their token rows in
    // LDS when the rows and the tables fit
    b.x_lds = 0;
    if (bf && nbt == 1 && tb == RT_TB && b.nblk <= 256 && a.d % 512 == 0 && a.d <= RT_XLDS_MAX_D &&
        route_smem(tb, a.E, a.gmax, a.M, false, route_xlds_bytes(a.d)) <= RT_LDS_MAX)
        b.x_lds = route_xlds_bytes(a.d);
    if (b.nblk > 0) {
        b.S_in_lds = route_S_in_lds(tb, a.E, a.gmax, a.M, b.nblk, b.x_lds) ? 1 : 0;
        const size_t smem = route_smem(tb, a.E, a.gmax, a.M, b.S_in_lds != 0, b.x_lds);
        b.ksplit = 0;
        if (split) {
            // enough waves to cover the CUs, K slices a multiple of 32
            int ks = 256 / (b.nblk * nb);
            ks = ks < 1 ? 1 : (ks > RT_SPLIT_MAX_K ? RT_SPLIT_MAX_K : ks);
            while (ks > 1 && a.d % (32 * ks) != 0) --ks;
            b.ksplit = ks;
            KernelTimer kt_("router_split", st);
            router_split_kernel<<<dim3((unsigned)b.nblk, (unsigned)nb, (unsigned)ks), dim3(64), 0, st>>>(b);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return (int)e;
        }
        int e = 0;
        if (tb == RT_TB2) {
            switch (nbt) {
                case 1: e = launch_route_kernel<1, RT_TB2>(b, smem, st); break;
                case 2: e = launch_route_kernel<2, RT_TB2>(b, smem, st); break;
                default: e = launch_route_kernel<4, RT_TB2>(b, smem, st); break;
            }
        } else {
            switch (nbt) {
                case 1: e = launch_route_kernel<1, RT_TB>(b, smem, st); break;
                case 2: e = launch_route_kernel<2, RT_TB>(b, smem, st); break;
                case 4: e = launch_route_kernel<4, RT_TB>(b, smem, st); break;
                case 8: e = launch_route_kernel<8, RT_TB>(b, smem, st); break;
                default: e = launch_route_kernel<16, RT_TB>(b, smem, st); break;
            }
        }
        if (e) return e;
    }
    if (b.T * b.k <= DS_THREADS) {
        KernelTimer kt_("dispatch_small", st);
        hipLaunchKernelGGL(dispatch_small_kernel, dim3(1), dim3(DS_THREADS), 0, st, b.blk_cnt, b.nblk,
                           b.out.exec_m, b.loc_in, b.T, b.k, b.M, b.out.dst_count, b.out.counters,
                           b.out.dispatch);
        return (int)hipGetLastError();
    }
    // here T k > DS_THREADS, so there is at least one routing block
    {
        KernelTimer kt_("dispatch", st);
        hipLaunchKernelGGL(dispatch_kernel, dim3(b.nblk), dim3(RT_THREADS), 0, st, b.blk_dst, b.blk_cnt, b.nblk,
                           b.out.exec_m, b.loc_in, b.T, b.k, b.M, tb, b.out.dst_count, b.out.counters,
                           b.out.dispatch);
    }
    return (int)hipGetLastError();
}

}  // namespace ordermoe
