// Local MoE execution of one server on gfx950: the (token, slot) pairs that
// the selection assigned to this server are turned into expert rows, run
// through a grouped SwiGLU FFN and combined per token.
//
//   rows_count_kernel    per-block row counts per group (local experts, then
//                        the shared pseudo-expert), duplicates of one token
//                        merged
//   rows_scatter_kernel  each block totals the count table itself (group
//                        offsets, its position in each group, tile counts of
//                        the two GEMMs), then places its rows stably (token
//                        order inside a group) with the merged gate weight
//                        and the token -> rows map
//   rows_small_kernel    both row kernels as one block (batches of at most
//                        1024 tokens)
//   ggemm_bf16<.., 0>    gate/up projection, X rows gathered through row_tok,
//                        packed [2f][d] weights, epilogue silu(g) * u -> bf16
//   ggemm_bf16<.., 1>    down projection of the activations, epilogue scales
//                        each row by its gate weight -> bf16 row outputs
//   combine_kernel       y[t] = sum of t's row outputs in slot order (fp32)
// The GEMMs are persistent: each workgroup walks the tile list, whose length
// is read from device memory, so no host synchronisation is needed.  Tiles of
// one expert are ordered m-fastest so consecutive tiles share a weight tile,
// and workgroup ids are remapped so that each XCD (and its L2) works on a
// contiguous range of tiles.  The bf16 GEMMs run whole rounds of tiles (one
// tile per workgroup per round); the tiles left over, fewer than the grid, are
// cut along K into pieces at the same positions in every tile when that keeps
// at least two workgroups per tile busy, and the last workgroup to finish a
// piece of a split tile adds the pieces in a fixed order and runs the
// epilogue.  A shared group with a K at least twice the routed K has its tiles
// cut into two K halves the same way, so that they no longer set the length of
// the launch.
#include <hip/hip_runtime.h>

#include <type_traits>

#include <cstdint>

#include "common.hpp"

namespace ordermoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int FT_TB = 256;        // tokens per block in the row kernels
constexpr int MAXG = ORDERMOE_MAX_LOCAL + 1;
constexpr int MAXR = ORDERMOE_MAX_TOPK + 1;   // rows per token (routed + shared)
// bf16 GEMM launches: at most SK_MAX_GRID workgroups.  Split tiles use one
// partial tile per workgroup (its slot) and one arrival counter per split
// tile, in one array of SK_MAX_GRID counters per GEMM (gate/up, down), zeroed
// by the row kernels before every forward.  A tile is cut into at most
// SK_SPLIT pieces (the last arrival reads them all).
constexpr int SK_MAX_GRID = 256;
constexpr int SK_SPLIT = 4;
constexpr int SK_MIN_PIECE_KT = 16;   // K tiles of 64 per piece, at least

struct RowsArgs {
    int64_t T;
    int k, E, n_local, has_shared, server;
    const float* w;
    const int32_t* exec_k;
    const uint8_t* exec_m;
    const uint8_t* loc_in;
    int32_t lidx[ORDERMOE_MAX_EXPERTS];   // expert -> local slot (kernel argument)
    int32_t* blk_rows;        // [nblk][G]
    int32_t* row_offsets;     // [n_local + 2]
    int32_t* row_tok;
    float* row_w;
    int32_t* tok_rows;        // [T][k+1]
    int32_t* tile_info;       // [4]
    int32_t* sk_cnt;          // [2][SK_MAX_GRID] split-tile arrival counters, zeroed here
    int nblk;
    // tile geometry for the tile counts
    int bm_gu, bn_gu, bm_dn, bn_dn;
    int n_gu_r, n_gu_s, n_dn;
};

// One token's slots as read from memory: executing server, expert and gate
// weight per slot, and the token's server.  The reads are issued together
// (unused slots re-read the last slot, in range, and are discarded, so no
// branch separates them); the placement kernels issue them first, so that
// their latency overlaps the reads of the count table.  The arrays are
// indexed only by unrolled constants so that they stay in registers.
struct TokSlots {
    int m[ORDERMOE_MAX_TOPK], ek[ORDERMOE_MAX_TOPK];
    float wv[ORDERMOE_MAX_TOPK];
    int loc;
};
__device__ inline void token_read(const RowsArgs& a, int64_t t, TokSlots& s) {
#pragma unroll
    for (int i = 0; i < ORDERMOE_MAX_TOPK; ++i) {
        const int64_t o = t * a.k + (i < a.k ? i : a.k - 1);
        s.m[i] = a.exec_m[o];
        s.ek[i] = a.exec_k[o];
        s.wv[i] = a.w[o];
    }
    s.loc = a.has_shared ? (int)a.loc_in[t] : -1;
}

// rows of one token: group ids (local slot, or n_local for the shared group)
// and merged gate weights, in slot order of first occurrence
__device__ inline int token_rows(const RowsArgs& a, const int32_t* s_lidx, const TokSlots& ts, int* grp,
                                 float* wsum) {
    int m[ORDERMOE_MAX_TOPK], ek[ORDERMOE_MAX_TOPK];
    float wv[ORDERMOE_MAX_TOPK];
#pragma unroll
    for (int s = 0; s < ORDERMOE_MAX_TOPK; ++s) {
        const bool used = s < a.k;
        m[s] = used ? ts.m[s] : -1;
        ek[s] = used ? ts.ek[s] : -1;
        wv[s] = used ? ts.wv[s] : 0.f;
    }
    const int loc = ts.loc;
#pragma unroll
    for (int q = 0; q < MAXR; ++q) { grp[q] = -1; wsum[q] = 0.f; }
    int n = 0;
#pragma unroll
    for (int s = 0; s < ORDERMOE_MAX_TOPK; ++s) {
        const int e = ek[s];
        const int ls = (m[s] == a.server && e >= 0 && e < a.E) ? s_lidx[e] : -1;
        if (ls >= 0) {
            bool found = false;
#pragma unroll
            for (int q = 0; q < MAXR; ++q)
                if (grp[q] == ls) { wsum[q] = wsum[q] + wv[s]; found = true; }
            if (!found) {
#pragma unroll
                for (int q = 0; q < MAXR; ++q)
                    if (q == n) { grp[q] = ls; wsum[q] = wv[s]; }
                ++n;
            }
        }
    }
    if (loc == a.server) {
#pragma unroll
        for (int q = 0; q < MAXR; ++q)
            if (q == n) { grp[q] = a.n_local; wsum[q] = 1.0f; }
        ++n;
    }
    return n;
}

// Ranks of a wave's rows inside their groups (token order): each lane ORs its
// bit into the 64-bit lane mask of every group it has a row in (LDS atomics),
// then a row's rank is the number of lower lanes in its group's mask.  The
// wave's LDS operations run in program order, so the reads see every OR.  Also
// writes the wave's row count of every group to wcnt[0 .. G).
__device__ inline void wave_group_ranks(unsigned long long* msk, int G, int lane, const int* grp, int n,
                                        int* rank, int32_t* wcnt) {
    for (int g = lane; g < G; g += 64) msk[g] = 0ull;
    const unsigned long long bit = 1ull << lane;
#pragma unroll
    for (int q = 0; q < MAXR; ++q)
        if (q < n) atomicOr(&msk[grp[q]], bit);
#pragma unroll
    for (int q = 0; q < MAXR; ++q) {
        rank[q] = 0;
        if (q < n) rank[q] = __popcll(msk[grp[q]] & (bit - 1ull));
    }
    for (int g = lane; g < G; g += 64) wcnt[g] = __popcll(msk[g]);
}

__global__ void __launch_bounds__(FT_TB) rows_count_kernel(const RowsArgs a) {
    __shared__ int32_t s_lidx[ORDERMOE_MAX_EXPERTS];
    __shared__ int32_t s_h[MAXG];
    const int G = a.n_local + a.has_shared;
    for (int i = threadIdx.x; i < a.E; i += FT_TB) s_lidx[i] = a.lidx[i];
    for (int i = threadIdx.x; i < G; i += FT_TB) s_h[i] = 0;
    __syncthreads();
    const int64_t t = (int64_t)blockIdx.x * FT_TB + threadIdx.x;
    if (t < a.T) {
        TokSlots ts;
        token_read(a, t, ts);
        int grp[MAXR];
        float ws[MAXR];
        const int n = token_rows(a, s_lidx, ts, grp, ws);
#pragma unroll
        for (int q = 0; q < MAXR; ++q)
            if (q < n) atomicAdd(&s_h[grp[q]], 1);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < G; i += FT_TB) a.blk_rows[(int64_t)blockIdx.x * G + i] = s_h[i];
}

constexpr int SCAN_THREADS = 1024;
constexpr int SCAN_WAVES = SCAN_THREADS / 64;

// One wave: the group offsets (exclusive scan of the group totals tot[0..G),
// local experts then the shared group) into first[], and, when `publish`, the
// row offsets and the tile counts of the two GEMMs into device memory.
__device__ inline void group_layout(const RowsArgs& a, const int32_t* tot, int32_t* first, int lane, bool publish) {
    const int G = a.n_local + a.has_shared;
    int32_t base = 0;
    int64_t tiles_gu = 0, tiles_dn = 0;
    for (int g0 = 0; g0 <= a.n_local; g0 += 64) {
        const int g = g0 + lane;
        const int32_t R = g < G ? tot[g] : 0;
        int32_t inc = R;
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t o = __shfl_up(inc, off);
            if (lane >= off) inc += o;
        }
        if (g <= a.n_local) {
            first[g] = base + inc - R;
            if (publish) a.row_offsets[g] = base + inc - R;
        }
        int64_t tg = 0, td = 0;
        if (g < G) {
            const bool sh = g == a.n_local;
            tg = (int64_t)((R + a.bm_gu - 1) / a.bm_gu) * ((sh ? a.n_gu_s : a.n_gu_r) / a.bn_gu);
            td = (int64_t)((R + a.bm_dn - 1) / a.bm_dn) * (a.n_dn / a.bn_dn);
        }
        for (int off = 32; off >= 1; off >>= 1) {
            tg += __shfl_xor(tg, off);
            td += __shfl_xor(td, off);
        }
        tiles_gu += tg;
        tiles_dn += td;
        base += __shfl(inc, 63);
    }
    if (publish && lane == 0) {
        a.row_offsets[a.n_local + 1] = base;
        a.tile_info[0] = (int32_t)tiles_gu;
        a.tile_info[1] = (int32_t)tiles_dn;
        a.tile_info[2] = base;
        a.tile_info[3] = 0;
    }
}

// Placement of every row, one block per block of rows_count_kernel.  Each
// block first totals the count table on its own (groups x blocks integers):
// its first row inside each group (the counts of the blocks before it) and the
// group totals, whose exclusive scan gives the group offsets; block 0 also
// publishes the row offsets and tile counts and clears the split-tile arrival
// counters of the GEMMs.  Then every row goes to its group offset + block
// position + its rank in token order.
__global__ void __launch_bounds__(FT_TB) rows_scatter_kernel(const RowsArgs a) {
    __shared__ int32_t s_lidx[ORDERMOE_MAX_EXPERTS];
    __shared__ int32_t s_wcnt[FT_TB / 64][MAXG];
    __shared__ unsigned long long s_msk[FT_TB / 64][MAXG];
    __shared__ int32_t s_lo[MAXG], s_tot[MAXG];
    __shared__ int32_t s_first[MAXG];        // first row of this block in each group
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int G = a.n_local + a.has_shared;
    const int b = (int)blockIdx.x;
    const int64_t t = (int64_t)b * FT_TB + tid;
    TokSlots ts;
    if (t < a.T) token_read(a, t, ts);
    for (int i = tid; i < a.E; i += FT_TB) s_lidx[i] = a.lidx[i];
    if (b == 0)
        for (int i = tid; i < 2 * SK_MAX_GRID; i += FT_TB) a.sk_cnt[i] = 0;
    for (int g = wave; g < G; g += FT_TB / 64) {
        int32_t lo = 0, tot = 0;
        for (int i = lane; i < a.nblk; i += 64) {
            const int32_t v = a.blk_rows[(int64_t)i * G + g];
            tot += v;
            lo += i < b ? v : 0;
        }
        for (int off = 32; off >= 1; off >>= 1) {
            lo += __shfl_xor(lo, off);
            tot += __shfl_xor(tot, off);
        }
        if (lane == 0) { s_lo[g] = lo; s_tot[g] = tot; }
    }
    __syncthreads();
    int grp[MAXR], rank[MAXR];
    float ws[MAXR];
    int n = 0;
    if (t < a.T) {
        n = token_rows(a, s_lidx, ts, grp, ws);
    } else {
#pragma unroll
        for (int q = 0; q < MAXR; ++q) { grp[q] = -1; ws[q] = 0.f; }
    }
    wave_group_ranks(s_msk[wave], G, lane, grp, n, rank, s_wcnt[wave]);
    if (wave == 0) {
        group_layout(a, s_tot, s_first, lane, b == 0);
        for (int g = lane; g < G; g += 64) s_first[g] += s_lo[g];
    }
    __syncthreads();
    if (t < a.T) {
        const int stride = a.k + 1;
#pragma unroll
        for (int q = 0; q < MAXR; ++q) {
            if (q < n) {
                const int g = grp[q];
                int32_t pos = s_first[g] + rank[q];
                for (int w = 0; w < wave; ++w) pos += s_wcnt[w][g];
                a.row_tok[pos] = (int32_t)t;
                a.row_w[pos] = ws[q];
                a.tok_rows[t * stride + q] = pos;
            } else if (q < stride) {
                a.tok_rows[t * stride + q] = -1;
            }
        }
    }
}

// Batches of at most SCAN_THREADS tokens (decode): the row kernels as one
// block, one token per thread -- group ranks by wave lane masks, group totals,
// row offsets and tile counts, then the placement (as rows_scatter_kernel).
__global__ void __launch_bounds__(SCAN_THREADS) rows_small_kernel(const RowsArgs a) {
    __shared__ int32_t s_lidx[ORDERMOE_MAX_EXPERTS];
    __shared__ int32_t s_wcnt[SCAN_WAVES][MAXG];
    __shared__ unsigned long long s_msk[SCAN_WAVES][MAXG];
    __shared__ int32_t s_first[MAXG], s_tot[MAXG];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int G = a.n_local + a.has_shared;
    const int64_t t = tid;
    TokSlots ts;
    if (t < a.T) token_read(a, t, ts);
    for (int i = tid; i < a.E; i += SCAN_THREADS) s_lidx[i] = a.lidx[i];
    for (int i = tid; i < 2 * SK_MAX_GRID; i += SCAN_THREADS) a.sk_cnt[i] = 0;
    __syncthreads();
    int grp[MAXR], rank[MAXR];
    float ws[MAXR];
    int n = 0;
    if (t < a.T) {
        n = token_rows(a, s_lidx, ts, grp, ws);
    } else {
#pragma unroll
        for (int q = 0; q < MAXR; ++q) { grp[q] = -1; ws[q] = 0.f; }
    }
    wave_group_ranks(s_msk[wave], G, lane, grp, n, rank, s_wcnt[wave]);
    __syncthreads();
    if (wave == 0) {
        for (int g = lane; g < G; g += 64) {
            int32_t R = 0;
            for (int w = 0; w < SCAN_WAVES; ++w) R += s_wcnt[w][g];
            s_tot[g] = R;
        }
        group_layout(a, s_tot, s_first, lane, true);
    }
    __syncthreads();
    if (t < a.T) {
        const int stride = a.k + 1;
#pragma unroll
        for (int q = 0; q < MAXR; ++q) {
            if (q < n) {
                const int g = grp[q];
                int32_t pos = s_first[g] + rank[q];
                for (int w = 0; w < wave; ++w) pos += s_wcnt[w][g];
                a.row_tok[pos] = (int32_t)t;
                a.row_w[pos] = ws[q];
                a.tok_rows[t * stride + q] = pos;
            } else if (q < stride) {
                a.tok_rows[t * stride + q] = -1;
            }
        }
    }
}

// ---------------------------------------------------------------- weights
// One-time packing (offline).  bf16 weights are stored tile-blocked: a matrix
// [N][K] (N % 256 == 0, K % 64 == 0) becomes [N/256][K/64][256][64], so that
// the 256 weight rows a GEMM tile reads in one 64-deep K step are one 32 KB
// block (and the 64 rows a thin-GEMM workgroup reads per K step 8 KB of it):
// the weight stream leaves DRAM in whole contiguous blocks instead of 128-byte
// slices of rows 8 or 28 KB apart.  fp32 weights keep the row layout.
constexpr int WB_ROWS = 256, WB_K = 64;
__host__ __device__ inline int64_t wblk_elem(int64_t n, int64_t k, int64_t K) {
    return ((n / WB_ROWS) * (K / WB_K) + k / WB_K) * (WB_ROWS * WB_K) + (n % WB_ROWS) * WB_K + k % WB_K;
}

// gate/up: one block per packed row p of the n 2f rows; rows [64b, 64b+32) of
// an expert <- gate rows [32b, 32b+32), rows [64b+32, 64b+64) <- the matching up
// rows; bf16 rows then go to their blocked places in 16-byte pieces
__global__ void pack_gate_up_kernel(int esz, int f, int d, const char* g, const char* u, char* out) {
    const int64_t prow = blockIdx.x;                  // over n * 2f rows
    const int64_t ex = prow / (2 * f);
    const int pr = (int)(prow % (2 * f));
    const int blk = pr / 64, within = pr % 64;
    const int src_row = blk * 32 + (within & 31);
    const char* src = (within < 32 ? g : u) + ((ex * f + src_row) * (int64_t)d) * esz;
    if (esz == 4) {
        char* dst = out + prow * (int64_t)d * esz;
        for (int64_t i = threadIdx.x * 4; i < (int64_t)d * esz; i += blockDim.x * 4)
            *(uint32_t*)(dst + i) = *(const uint32_t*)(src + i);
        return;
    }
    __bf16* dst = (__bf16*)out + ex * 2 * f * (int64_t)d;
    for (int k = threadIdx.x * 8; k < d; k += blockDim.x * 8)
        *(uint4*)(dst + wblk_elem(pr, k, d)) = *(const uint4*)((const __bf16*)src + k);
}

// down: one block per row p of the n d rows of [n][d][f]
__global__ void pack_down_kernel(int esz, int d, int f, const char* w, char* out) {
    const int64_t row = blockIdx.x;                   // over n * d rows
    const int64_t ex = row / d;
    const int r = (int)(row % d);
    const char* src = w + row * (int64_t)f * esz;
    if (esz == 4) {
        char* dst = out + row * (int64_t)f * esz;
        for (int64_t i = threadIdx.x * 4; i < (int64_t)f * esz; i += blockDim.x * 4)
            *(uint32_t*)(dst + i) = *(const uint32_t*)(src + i);
        return;
    }
    __bf16* dst = (__bf16*)out + ex * (int64_t)d * f;
    for (int k = threadIdx.x * 8; k < f; k += blockDim.x * 8)
        *(uint4*)(dst + wblk_elem(r, k, f)) = *(const uint4*)((const __bf16*)src + k);
}

// ---------------------------------------------------------------- GEMMs
struct GemmArgs {
    const int32_t* offsets;   // [G + 1] row offsets of the groups (device)
    const int32_t* ntiles;    // device: number of tiles
    int G, n_routed;          // groups; groups >= n_routed are the shared group
    int Nr, Kr, Ns, Ks;       // N, K of routed and shared groups
    const void* Wr;           // [n_routed][Nr][Kr]
    const void* Ws;           // [Ns][Ks]
    const void* X;            // mode 0: token rows [T][ldx]
    const int32_t* row_tok;   // mode 0
    int ldx;
    uint32_t x_bytes;         // mode 0: size of X in bytes
    const void* Ar;           // mode 1: routed activations [*][Kr]
    const void* As;           // mode 1: shared activations [*][Ks]
    void* Or;                 // mode 0: routed activations out; mode 1: row outputs [*][Nr]
    void* Os;                 // mode 0: shared activations out; mode 1: unused
    const float* row_w;       // mode 1
    float* sk_part;           // bf16: [SK_MAX_GRID][BM * BN] partial tiles of split tiles
    int32_t* sk_cnt;          // bf16: [2][SK_MAX_GRID] arrival counters (zero at launch)
};

struct TileLoc {
    int g, m0, n0, R, N, K, rowbase;
};

// Tile order: the shared group first (its down projection has the longest K,
// so its tiles start first and the shorter routed tiles fill in around them),
// then the routed groups; inside a group tiles are m-fastest.
template <int BM, int BN>
__device__ inline bool decode_tile(const GemmArgs& p, int tile, TileLoc& L) {
    int rem = tile;
    const bool has_sh = p.G > p.n_routed;
    for (int gi = 0; gi < p.G; ++gi) {
        const int g = has_sh ? (gi == 0 ? p.n_routed : gi - 1) : gi;
        const int off = p.offsets[g];
        const int R = p.offsets[g + 1] - off;
        const bool sh = g >= p.n_routed;
        const int N = sh ? p.Ns : p.Nr;
        const int mt = (R + BM - 1) / BM;
        const int cnt = mt * (N / BN);
        if (rem < cnt) {
            L.g = g; L.R = R; L.N = N; L.K = sh ? p.Ks : p.Kr; L.rowbase = off;
            L.m0 = (rem % mt) * BM;
            L.n0 = (rem / mt) * BN;
            return true;
        }
        rem -= cnt;
    }
    return false;
}

// Position of workgroup vid in round r of n work items (n <= grid): odd
// rounds mirrored (snake order); with `spread`, a partial round is shared
// evenly by the 8 XCDs (vid / (grid / 8) is the workgroup's XCD), so that no
// XCD sits idle while another runs a full share.  -1: no item for this
// workgroup.
__device__ inline int round_pos(int vid, int r, int n, int grid, bool spread) {
    const int v = (r & 1) ? grid - 1 - vid : vid;
    if (n >= grid || !spread) return v < n ? v : -1;
    const int g8 = grid >> 3, x = v / g8, j = v - x * g8;
    const int lo = x * n / 8, hi = (x + 1) * n / 8;
    return j < hi - lo ? lo + j : -1;
}

// silu(g) = g / (1 + e^-g), with the hardware reciprocal (1 ulp) instead of an
// IEEE divide: the result is rounded to bf16 right after
__device__ inline float silu_f(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

// s_waitcnt operand on gfx9-class GPUs: vmcnt (6 bits, split), expcnt (left at
// its maximum), lgkmcnt (4 bits)
constexpr int waitcnt_enc(int vm, int lgkm) { return (vm & 0xF) | ((vm >> 4) << 14) | (7 << 4) | ((lgkm & 0xF) << 8); }

// Workgroup barrier of the K loop.  __syncthreads() (and a workgroup fence on
// LDS alone) waits for every outstanding load into LDS (vmcnt 0), which would
// also drain the loads of a buffer that is read only a tile later; this one
// is the bare s_barrier, and the memory clobber keeps the compiler from moving
// memory accesses across it.  The caller first waits (s_waitcnt vmcnt) for its
// own loads into the buffers read after the barrier, and every LDS read of a
// buffer has returned its data (it fed an MFMA) before the barrier that
// precedes the next load into that buffer.
__device__ inline void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr;

constexpr int BUF_DWORD3 = 0x00020000;   // raw buffer resource word 3 on gfx9-class GPUs
constexpr int SC1 = 16;                  // buffer load/store cache bit sc1: coherent at agent scope

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, BUF_DWORD3);
}

__device__ inline bf16x8 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
    return __builtin_bit_cast(bf16x8, v);
}

// Scheduling pattern of one MFMA sub-step: NM MFMAs with NR LDS fragment
// reads and NX other memory instructions (mask XMASK) spread between them,
// reads after even-numbered MFMAs, the others after odd-numbered ones.
template <int Q, int NM, int NR, int NX, int XMASK>
__device__ inline void sched_interleave() {
    if constexpr (Q < NM) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        constexpr int r = ((Q + 1) * NR + NM - 1) / NM - (Q * NR + NM - 1) / NM;
        if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);   // LDS read
        constexpr int x = (Q + 1) * NX / NM - Q * NX / NM;
        if constexpr (x > 0) __builtin_amdgcn_sched_group_barrier(XMASK, x, 0);
        sched_interleave<Q + 1, NM, NR, NX, XMASK>();
    }
}

// bf16 grouped GEMM C = A B^T per tile of BM x BN, K step 64, 4 waves (2 x 2),
// each wave a (BM/2) x (BN/2) block of v_mfma_f32_32x32x16_bf16 tiles.
// Operands go from memory straight into LDS (buffer loads to LDS), two
// buffers; the layout is described at the K loop.  The K position travels in
// the buffer load's scalar offset, and rows past the end of a group read as
// zeros through the buffer range check (their offset is set past the buffer).
// Byte offsets inside one operand fit in 31 bits (checked by the host).
//
// Work: rounds of whole tiles while a round fills the grid; the tiles left
// over are cut along K into equal pieces when that puts at least two
// workgroups on each (split-K), else they run whole as a last, partial round.
// A piece stores its fp32 partial tile in its slot, and the workgroup whose
// arrival completes the tile's counter sums the tile's pieces in K order (so
// the result does not depend on who is last) and runs the epilogue.  No
// workgroup waits for another.
template <int BM, int BN, int MODE>
__global__ void __launch_bounds__(256, 1) ggemm_bf16(const GemmArgs p) {
    constexpr int BK = 64;
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 32, FN = WN / 32;
    constexpr int AV = BM / 32;                     // 8-row load instructions per wave and K tile
    constexpr int BV = BN / 32;
    static_assert(FN % 2 == 0, "gate/up pairs need an even number of 32-column blocks");
    static_assert(BM % 64 == 0 && BN % 64 == 0, "an even number of load instructions per wave");
    // two buffers of the A and B tiles, [rows][64] bf16 each
    // two buffers of the A tile and three of the B tile, [rows][64] bf16 each
    __shared__ __attribute__((aligned(16))) __bf16 sA0[BM * 64], sA1[BM * 64], sB0[BN * 64], sB1[BN * 64];
    __shared__ __attribute__((aligned(16))) __bf16 sB2[BN * 64];
    // the split-tile arrival flag lives in sB2, which is idle from the end of a
    // K loop until the first K tile of the next one (a prologue loads sA0, sA1,
    // sB0 and sB1 only), so that the buffers of 256 x 256 tiles fill the LDS
    int* const s_last = (int*)sB2;
    // down: the gate weights of the tile's rows, for the epilogue; 256-row tiles
    // keep them in sB2 too (past the flag), so that their buffers fill the LDS
    constexpr bool ROWW_IN_SB2 = MODE == 1 && (2 * BM + 3 * BN) * 64 * 2 + BM * 4 > 160 * 1024;
    static_assert(!ROWW_IN_SB2 || 256 + BM * 4 <= BN * 64 * 2, "flag and row weights fit sB2");
    float* s_roww;
    if constexpr (ROWW_IN_SB2) {
        s_roww = (float*)sB2 + 64;
    } else {
        __shared__ float s_roww_own[MODE == 1 ? BM : 1];
        s_roww = s_roww_own;
    }

    const int tid = threadIdx.x;
    const int total = *p.ntiles;
    const int grid = (int)gridDim.x;                // a multiple of 8, at most SK_MAX_GRID
    const int vid = (blockIdx.x & 7) * (grid >> 3) + (blockIdx.x >> 3);
    constexpr uint32_t OOR = 0x80000000u;           // offset past every buffer: reads zero
    // A shared group whose K is at least twice the routed K (the down
    // projection of several shared experts) has tiles that outlast the routed
    // ones several times over.  When the grid holds two pieces of each, every
    // shared tile is cut along K into two halves: work item i < 2 nsh is half
    // i / nsh of shared tile i mod nsh (the shared tiles come first in the
    // list), and the routed tiles follow as whole items, so that they fill in
    // around the halves.
    int nsh = 0;
    if (p.G > p.n_routed) {
        const int rsh = p.offsets[p.n_routed + 1] - p.offsets[p.n_routed];
        nsh = (rsh + BM - 1) / BM * (p.Ns / BN);
    }
    const bool sh_split = nsh > 0 && p.Ks >= 2 * p.Kr && p.Ks % (4 * BK) == 0 && 2 * nsh <= grid;
    const int items = sh_split ? total + nsh : total;
    const int rounds = items / grid, head = rounds * grid;

    // the tiles left after the whole rounds: when at least two workgroups per
    // tile are free, each tile is cut along K into `split` pieces at the same
    // positions in every tile (piece j of the tile at head + i goes to
    // position j * left + i of the round), so that the workgroups of an XCD
    // read the same K range of neighbouring tiles together, as in a whole
    // round.  Positions follow the snake order of the rounds.  Only when all
    // tiles have the same K: then every workgroup finishes its rounds at about
    // the same time (a shared group with a longer K keeps some workgroups busy
    // while the pieces would go out).
    const int left = items - head;
    int split = left > 0 ? grid / left : 0;
    if (split > SK_SPLIT) split = SK_SPLIT;
    if (split > p.Kr / (2 * BK)) split = p.Kr / (2 * BK);
    // a piece keeps at least SK_MIN_PIECE_KT K tiles: shorter pieces cost more
    // in partial-tile stores and fix-up reads than the idle workgroups they
    // fill, most of all when another batch's kernels can take those CUs
    if (split > p.Kr / BK / SK_MIN_PIECE_KT) split = p.Kr / BK / SK_MIN_PIECE_KT;
    if (p.G > p.n_routed && p.Ks != p.Kr) split = 1;
    // slots of the pieces of one split tile lie sstride apart
    const int sstride = sh_split ? nsh : left;
    // the last, partial round is spread over the XCDs when every tile has the
    // same K; otherwise the snake order gives it to the workgroups that just
    // ran short tiles
    const bool spread = !(p.G > p.n_routed && p.Ks != p.Kr);

    for (int r = 0; r <= rounds; ++r) {
        // the thread index passes through an empty asm once per tile, so that
        // the thread-dependent offsets below are recomputed per tile instead of
        // being held (and spilled to scratch) across the whole persistent loop
        int tid_r = tid;
        asm volatile("" : "+v"(tid_r));
        const int lane_r = tid_r & 63, wave_r = tid_r >> 6;
        const int wm_r = wave_r >> 1, wn_r = wave_r & 1;
        // the wave index as a scalar: the LDS destinations of the loads into LDS
        // (the M0 operand) are then scalar expressions, not VGPRs held per buffer
        const int wave_u = __builtin_amdgcn_readfirstlane(wave_r);
        TileLoc L;
        int kt_lo = 0, kt_hi = 0;       // K tiles of 64 of this piece
        int nseg = 1, ctr = 0, pslot = 0;
        if (r < rounds || split < 2) {
            // whole tiles (or shared halves) in rounds of `grid`, in snake
            // order (odd rounds reversed), so that the workgroups that took
            // the long tiles at the head of the list take the last tiles of
            // the next round; the last round may be partial
            const int pos = round_pos(vid, r, r < rounds ? grid : items - head, grid, spread);
            if (pos < 0) break;
            const int item = r * grid + pos;
            if (item >= items) break;
            if (sh_split && item < 2 * nsh) {
                const int j = item / nsh;
                ctr = item - j * nsh;
                pslot = item;
                if (!decode_tile<BM, BN>(p, ctr, L)) break;
                const int half = L.K / (2 * BK);          // even: K is a multiple of 4 BK
                kt_lo = j * half;
                kt_hi = kt_lo + half;
                nseg = 2;
            } else {
                if (!decode_tile<BM, BN>(p, sh_split ? item - nsh : item, L)) break;
                kt_hi = L.K / BK;
            }
        } else {
            const int pos = round_pos(vid, rounds, split * left, grid, spread);
            if (pos < 0) break;
            const int j = pos / left;
            ctr = pos - j * left;
            pslot = pos;
            if (!decode_tile<BM, BN>(p, head + ctr, L)) break;
            const int units = L.K / (2 * BK);
            kt_lo = 2 * (j * units / split);
            kt_hi = 2 * ((j + 1) * units / split);
            nseg = split;
        }
        const bool shared = L.g >= p.n_routed;
        const int K = L.K;
        const __bf16* Bw = shared ? (const __bf16*)p.Ws
                                  : (const __bf16*)p.Wr + (size_t)L.g * L.N * K;
        const __amdgpu_buffer_rsrc_t rb_rs = make_rsrc(Bw, (uint32_t)((size_t)L.N * K * 2));
        // LDS rows of 64 K values (128 bytes, unpadded); 16-byte chunk q of
        // row r holds the operand's chunk q ^ ((r >> 1) & 7), so that the 16
        // rows a fragment read serves per LDS cycle (16 lanes of 16 bytes over
        // the 64 banks) fall on distinct banks.  Load instruction v of wave_r w
        // covers rows (w AV + v) 8 .. +7 of the tile: lane_r l takes row + l / 8
        // and fetches the chunk that the direct-to-LDS load writes at position
        // l & 7 of that row, (l & 7) ^ ((r >> 1) & 7); with AV, BV even that is
        // gc0 for even v and gc1 for odd v.
        const int gc0 = (lane_r & 7) ^ (lane_r >> 4);
        const int gc1 = (lane_r & 7) ^ (4 | (lane_r >> 4));
        const int rsub = lane_r >> 3;
        // A: the gathered token rows of X (gate/up) or the group's activation rows (down)
        const __bf16* Ab = MODE == 0 ? (const __bf16*)p.X
                                     : (shared ? (const __bf16*)p.As : (const __bf16*)p.Ar + (size_t)L.rowbase * K);
        const __amdgpu_buffer_rsrc_t ra_rs =
            make_rsrc(Ab, MODE == 0 ? p.x_bytes : (uint32_t)((size_t)L.R * K * 2));
        // down: thread tid_r < BM reads the gate weight of tile row tid_r now (one
        // branch-free load, rows past the group read zero) and parks it in LDS
        // after the K loop, so that the epilogue waits for no global load
        float roww = 0.f;
        if constexpr (MODE == 1) {
            const __amdgpu_buffer_rsrc_t rw_rs = make_rsrc(p.row_w + L.rowbase, (uint32_t)L.R * 4u);
            const int rr = L.m0 + tid_r;
            roww = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                 rw_rs, tid_r < BM && rr < L.R ? rr * 4 : (int)OOR, 0, 0));
        }
        uint32_t aoff[AV];
#pragma unroll
        for (int v = 0; v < AV; ++v) {
            const int row = L.m0 + (wave_r * AV + v) * 8 + rsub;
            const uint32_t src = MODE == 0 ? (row < L.R ? (uint32_t)p.row_tok[L.rowbase + row] : 0u) : (uint32_t)row;
            aoff[v] = row < L.R ? (src * (uint32_t)(MODE == 0 ? p.ldx : K) + ((v & 1) ? gc1 : gc0) * 8) * 2u : OOR;
        }
        // B: the blocked weights (256-row blocks of 64-deep K steps, 128-byte
        // rows): load instruction v of wave_r w covers rows (w BV + v) 8 .. +7
        // of the tile's block, 1 KB in a row; the K step goes in the scalar offset
        static_assert(BN == WB_ROWS, "a tile's weight rows are one block");
        const uint32_t bblk = (uint32_t)(L.n0 / BN) * (uint32_t)(K / WB_K) * (uint32_t)(BN * WB_K * 2) +
                              (uint32_t)(wave_r * BV * 8 + rsub) * (WB_K * 2u);

        f32x16 acc[FM][FN];
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

        // the loads of a K tile go from memory straight into LDS buffer b
        auto dmaA = [&](__bf16* sa, int k0) {
#pragma unroll
            for (int v = 0; v < AV; ++v) {
                // (a local copy: the host pass drops the kernel when an array
                // element captured by reference is the builtin's operand)
                const uint32_t vo = aoff[v];
                __builtin_amdgcn_raw_ptr_buffer_load_lds(ra_rs, (lds_ptr)(sa + (wave_u * AV + v) * 8 * 64), 16, vo,
                                                         (uint32_t)k0 * 2u, 0, 0);
            }
        };
        auto dmaB = [&](__bf16* sb, int k0) {
#pragma unroll
            for (int v = 0; v < BV; ++v)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rb_rs, (lds_ptr)(sb + (wave_u * BV + v) * 8 * 64), 16,
                                                         bblk + v * 1024u + (uint32_t)((v & 1) ? gc1 : gc0) * 16u,
                                                         (uint32_t)k0 * (uint32_t)(BN * 2), 0, 0);
        };
        // fragment of row (lane_r & 31) of each 32-row block, K chunk 2 ks + lane_r / 32
        const int arow = (wm_r * WM + (lane_r & 31)) * 64;
        const int brow = (wn_r * WN + (lane_r & 31)) * 64;
        bf16x8 af[2][FM], bfm[2][FN];
        auto fload = [&](const __bf16* sa, const __bf16* sb, int ks, int slot) {
            const int pos = ((2 * ks + (lane_r >> 5)) ^ ((lane_r >> 1) & 7)) * 8;   // row & 31 = lane_r & 31
#pragma unroll
            for (int i = 0; i < FM; ++i) af[slot][i] = *(const bf16x8*)(sa + arow + i * 32 * 64 + pos);
#pragma unroll
            for (int j = 0; j < FN; ++j) bfm[slot][j] = *(const bf16x8*)(sb + brow + j * 32 * 64 + pos);
        };
        // the first sub-step's fragments after the barrier, in the order the
        // MFMAs consume them (A0 B0, then B1.., then A1..), each read fenced so
        // that the first MFMAs wait for their own operands only (the scheduler
        // had issued B0 and B1 last, so every K tile began by waiting for seven
        // of the eight reads)
        auto fload_first = [&](const __bf16* sa, const __bf16* sb) {
            const int pos = ((lane_r >> 5) ^ ((lane_r >> 1) & 7)) * 8;   // sub-step 0
            af[0][0] = *(const bf16x8*)(sa + arow + pos);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                bfm[0][j] = *(const bf16x8*)(sb + brow + j * 32 * 64 + pos);
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int i = 1; i < FM; ++i) {
                af[0][i] = *(const bf16x8*)(sa + arow + i * 32 * 64 + pos);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        auto mfmas = [&](int slot) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[slot][i], bfm[slot][j], acc[i][j], 0, 0, 0);
        };
        // Each K tile of 64 is four MFMA sub-steps of 16; every sub-step reads
        // the fragments of the next one.  The buffers are separate LDS arrays
        // and the loop is unrolled over a pass of six tiles (A cycles over two
        // buffers, B over three), so that every access names a fixed array and
        // the loads into one buffer are never taken to alias the reads of
        // another.  The barrier of K tile t sits before its last sub-step.
        // Sub-step 0 issues the B loads of tile t + 2 (into the buffer tile
        // t - 1 read, free since barrier t - 1); after sub-step 2 every fragment
        // of tile t has been read, so the wave waits for its own loads of tile
        // t + 1 (everything but the B loads just issued) and its reads, and the
        // barrier follows; sub-step 3's MFMAs then overlap the first fragment
        // reads of tile t + 1 and the A loads of tile t + 2 into the A buffer
        // tile t has just finished with.  The A loads keep a lead of four
        // sub-steps, the B loads of seven; no tile starts by waiting for its
        // first fragments.  Loads past the piece re-read its last K tile into
        // an idle buffer.
        constexpr int NM = FM * FN, NR = FM + FN;
        constexpr int VMEM_READ = 0x020;
        auto ktile = [&](__bf16* ca, __bf16* cb, __bf16* na, __bf16* nbn, __bf16* nbl, int kn2)
                         __attribute__((always_inline)) {
            dmaB(nbl, kn2);
            fload(ca, cb, 1, 1);
            mfmas(0);
            sched_interleave<0, NM, NR, BV, VMEM_READ>();
            __builtin_amdgcn_sched_barrier(0);
            fload(ca, cb, 2, 0);
            mfmas(1);
            sched_interleave<0, NM, NR, 0, VMEM_READ>();
            __builtin_amdgcn_sched_barrier(0);
            fload(ca, cb, 3, 1);
            mfmas(0);
            sched_interleave<0, NM, NR, 0, VMEM_READ>();
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_waitcnt(waitcnt_enc(BV, 0));
            lds_barrier();
            dmaA(ca, kn2);
            fload(na, nbn, 0, 0);
            mfmas(1);
            sched_interleave<0, NM, NR, AV, VMEM_READ>();
            __builtin_amdgcn_sched_barrier(0);
        };
        // the piece's K tiles [kt_lo, kt_hi): an even number (K units of 128)
        const int klast = kt_hi - 1;
        auto kc = [&](int k) { return (k < kt_hi ? k : klast) * BK; };
        // buffers of tile kt + u of a pass (compile-time u)
        auto bufA = [&](auto u) -> __bf16* { return decltype(u)::value % 2 == 0 ? sA0 : sA1; };
        auto bufB = [&](auto u) -> __bf16* {
            constexpr int j = decltype(u)::value % 3;
            if constexpr (j == 0) return sB0; else if constexpr (j == 1) return sB1; else return sB2;
        };
        // prologue: tiles kt_lo and kt_lo + 1 of both operands
        dmaA(sA0, kt_lo * BK);
        dmaB(sB0, kt_lo * BK);
        dmaB(sB1, kc(kt_lo + 1));
        dmaA(sA1, kc(kt_lo + 1));
        static_assert(AV + BV < 64, "vmcnt field");
        __builtin_amdgcn_s_waitcnt(waitcnt_enc(AV + BV, 15));   // tile kt_lo's loads are in LDS
        lds_barrier();
        fload_first(sA0, sB0);
        __builtin_amdgcn_sched_barrier(0);
        auto step = [&](auto u, int kt) __attribute__((always_inline)) {
            constexpr int U = decltype(u)::value;
            using N1 = std::integral_constant<int, U + 1>;
            using N2 = std::integral_constant<int, U + 2>;
            ktile(bufA(u), bufB(u), bufA(N1{}), bufB(N1{}), bufB(N2{}), kc(kt + U + 2));
        };
        using I0 = std::integral_constant<int, 0>;
        using I1 = std::integral_constant<int, 1>;
        using I2 = std::integral_constant<int, 2>;
        using I3 = std::integral_constant<int, 3>;
        using I4 = std::integral_constant<int, 4>;
        using I5 = std::integral_constant<int, 5>;
        int kt = kt_lo;
        for (; kt + 6 <= kt_hi; kt += 6) {
            step(I0{}, kt); step(I1{}, kt); step(I2{}, kt);
            step(I3{}, kt); step(I4{}, kt); step(I5{}, kt);
        }
        // the two or four tiles left start a pass
        if (kt < kt_hi) {
            step(I0{}, kt); step(I1{}, kt);
            if (kt + 2 < kt_hi) { step(I2{}, kt); step(I3{}, kt); }
        }
        // loads of the tiles after the last may still be in flight
        __builtin_amdgcn_s_waitcnt(0x0F70);

        if (nseg > 1) {
            // a piece of a split tile: its partial sums go to slot j sstride + ctr
            // (its position in the round), thread tid_r's 16-byte group h of
            // block (i, j) at byte (((i FN + j) 4 + h) 256 + tid_r) 16 of the slot
            // (each store instruction writes 4 KB in a row).  Buffer stores and loads keep the lane_r's offset in
            // one register and the slot and group in the scalar offset.  They
            // carry the sc1 cache bit (the bit of agent-scope atomic loads and
            // stores), so each location is coherent across the XCDs' L2 caches
            // without a whole-cache write-back or invalidate, which would also
            // evict the tiles of every other workgroup on the XCD.  The stores
            // complete (vmcnt 0) before the arrival is counted, and the last
            // arrival's loads are issued after the count is read.
            constexpr uint32_t TILE_BYTES = (uint32_t)BM * BN * 4u;
            const __amdgpu_buffer_rsrc_t rp = make_rsrc(p.sk_part, (uint32_t)SK_MAX_GRID * TILE_BYTES);
            const uint32_t lo = (uint32_t)tid_r * 16u;
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        const f32x4 v{acc[i][j][4 * h], acc[i][j][4 * h + 1], acc[i][j][4 * h + 2], acc[i][j][4 * h + 3]};
                        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rp, (int)lo,
                                                               (int)((uint32_t)pslot * TILE_BYTES +
                                                                     (uint32_t)((i * FN + j) * 4 + h) * 4096u), SC1);
                    }
            __builtin_amdgcn_s_waitcnt(0x0F70);          // vmcnt(0): this wave_r's stores are done
            __syncthreads();
            if (tid_r == 0) *s_last = atomicAdd(p.sk_cnt + MODE * SK_MAX_GRID + ctr, 1) == nseg - 1;
            __syncthreads();
            if (!*s_last) continue;
            // the last arrival: the tile is the sum of its pieces in K order
            // (piece j in slot j * sstride + ctr).  Every group reads SK_SPLIT
            // pieces without a branch, so that the loads of many groups are in
            // flight together: the pieces past nseg have a lane_r offset past the
            // buffer (the range check covers the lane_r offset) and read as
            // zeros, and adding them leaves the sum as it is (up to the sign of
            // a zero).
            uint32_t pbase[SK_SPLIT], plo[SK_SPLIT];
#pragma unroll
            for (int sg = 0; sg < SK_SPLIT; ++sg) {
                pbase[sg] = sg < nseg ? (uint32_t)(ctr + sg * sstride) * TILE_BYTES : 0u;
                plo[sg] = sg < nseg ? lo : OOR;
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        const uint32_t go = (uint32_t)((i * FN + j) * 4 + h) * 4096u;
                        f32x4 pv[SK_SPLIT];
#pragma unroll
                        for (int sg = 0; sg < SK_SPLIT; ++sg) {
                            const uint32_t vo = plo[sg];
                            pv[sg] = __builtin_bit_cast(
                                f32x4, __builtin_amdgcn_raw_buffer_load_b128(rp, (int)vo, (int)(pbase[sg] + go), SC1));
                        }
                        f32x4 v = pv[0];
#pragma unroll
                        for (int sg = 1; sg < SK_SPLIT; ++sg) v += pv[sg];
                        acc[i][j][4 * h] = v[0];
                        acc[i][j][4 * h + 1] = v[1];
                        acc[i][j][4 * h + 2] = v[2];
                        acc[i][j][4 * h + 3] = v[3];
                    }
        }

        // epilogue: element e of a 32x32 block is row (e/4)*8 + (lane_r/32)*4 + e%4,
        // column lane_r%32.  Down scales each row by its gate weight, parked in
        // LDS by the workgroup (the barrier also orders it after the previous
        // tile's reads, which precede this tile's K-loop barriers).
        if constexpr (MODE == 1) {
            // (in sB2: after every wave's last fragment reads of the K loop)
            if constexpr (ROWW_IN_SB2) lds_barrier();
            if (tid_r < BM) s_roww[tid_r] = roww;
            lds_barrier();
        }
        const int rbase = L.m0 + wm_r * WM + (lane_r >> 5) * 4;
        if constexpr (MODE == 0) {
            __bf16* out = shared ? (__bf16*)p.Os : (__bf16*)p.Or;
            const int ldo = L.N / 2;
            const int orow0 = shared ? 0 : L.rowbase;
            const int cbase = (L.n0 + wn_r * WN) / 2 + (lane_r & 31);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int row = rbase + i * 32 + (e >> 2) * 8 + (e & 3);
                    if (row < L.R) {
#pragma unroll
                        for (int q = 0; q < FN / 2; ++q) {
                            const float gv = acc[i][2 * q][e], uv = acc[i][2 * q + 1][e];
                            out[(size_t)(orow0 + row) * ldo + cbase + q * 32] = (__bf16)(silu_f(gv) * uv);
                        }
                    }
                }
        } else {
            __bf16* out = (__bf16*)p.Or;
            const int ldo = L.N;
            const int cbase = L.n0 + wn_r * WN + (lane_r & 31);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int row = rbase + i * 32 + (e >> 2) * 8 + (e & 3);
                    const float wr = s_roww[row - L.m0];
                    if (row < L.R) {
#pragma unroll
                        for (int j = 0; j < FN; ++j)
                            out[(size_t)(L.rowbase + row) * ldo + cbase + j * 32] = (__bf16)(acc[i][j][e] * wr);
                    }
                }
        }
    }
}

// Thin grouped GEMM for small batches (decode): a few rows per expert, so the
// time is the weight stream from HBM and the MFMA work is incidental.  A
// workgroup computes 32 rows x 64 weight rows (a gate/up granule pair, or 64
// output columns of the down projection) over the whole K.  Its 4 waves take
// interleaved K steps of 64 (wave w: steps w, w+4, ...), so the workgroup
// streams 512 contiguous bytes of each weight row per round.  The weight rows
// are read coalesced (a wave instruction covers 8 rows x 128 bytes, whole cache
// lines) into registers, passed through the wave's own LDS rows (padded by 16
// bytes) into the v_mfma_f32_32x32x16_bf16 layout (lane: row lane%32, K
// elements 8*(lane/32) .. +7 of each 16); the activation rows go from global
// memory straight into MFMA registers.  Two register sets keep the next step's
// reads in flight during the current step.  The waves' partial sums meet in LDS
// and are added in wave order, then the epilogue of ggemm_bf16 runs on the
// sums.
constexpr int TH_BM = 32, TH_BN = 64, TH_WAVES = 4;
constexpr int TH_LDK = 144;                        // bytes per staged weight row
constexpr int TH_LDS = TH_WAVES * TH_BN * TH_LDK;  // staging; reused for the partial sums

template <int MODE>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
ggemm_thin(const GemmArgs p) {
    __shared__ __attribute__((aligned(16))) char th_lds[TH_LDS];
    static_assert(sizeof(float) * TH_WAVES * 2 * 16 * 64 <= TH_LDS, "partial sums fit the staging rows");
    float (*red)[2][16][64] = (float (*)[2][16][64])th_lds;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: K offsets go in SGPRs
    const int c = lane & 31, h = lane >> 5;
    const int total = *p.ntiles;
    const int per_xcd = gridDim.x >> 3;
    const int vid = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    constexpr uint32_t OOR = 0x80000000u;

    // rounds of gridDim.x tiles; the last, partial round shared evenly by the
    // XCDs when every tile has the same K
    const bool spread = !(p.G > p.n_routed && p.Ks != p.Kr);
    for (int r = 0; r * (int)gridDim.x < total; ++r) {
        const int n = total - r * (int)gridDim.x;
        const int pos = round_pos(vid, 0, n, (int)gridDim.x, spread);
        if (pos < 0) break;
        const int tile = r * (int)gridDim.x + pos;
        TileLoc L;
        if (!decode_tile<TH_BM, TH_BN>(p, tile, L)) break;
        const bool shared = L.g >= p.n_routed;
        const int K = L.K;
        const __bf16* Bw = shared ? (const __bf16*)p.Ws
                                  : (const __bf16*)p.Wr + (size_t)L.g * L.N * K;
        const __amdgpu_buffer_rsrc_t rb_rs = make_rsrc(Bw, (uint32_t)((size_t)L.N * K * 2));
        // weight reads from the blocked layout: the tile's 64 rows of one K step
        // are 8 KB in a row; lane l takes row 8i + l/8, 16-byte chunk l%8 of
        // that row's 128 bytes, and the K step goes in the scalar offset
        const uint32_t wblk0 = (uint32_t)(L.n0 / WB_ROWS) * (uint32_t)(K / WB_K) * (uint32_t)(WB_ROWS * WB_K * 2) +
                               (uint32_t)((L.n0 % WB_ROWS) + (lane >> 3)) * (WB_K * 2u) + (uint32_t)(lane & 7) * 16u;
        char* stg = th_lds + wave * (TH_BN * TH_LDK);
        char* wdst = stg + (lane >> 3) * TH_LDK + (lane & 7) * 16;
        const char* frag = stg + c * TH_LDK + h * 16;                  // row c, chunk 2i + h
        const int row = L.m0 + c;
        __amdgpu_buffer_rsrc_t ra_rs;
        uint32_t aoff;
        if (MODE == 0) {
            ra_rs = make_rsrc(p.X, p.x_bytes);
            aoff = row < L.R ? ((uint32_t)p.row_tok[L.rowbase + row] * (uint32_t)p.ldx + 8u * h) * 2u : OOR;
        } else {
            const __bf16* Ab = shared ? (const __bf16*)p.As : (const __bf16*)p.Ar + (size_t)L.rowbase * K;
            ra_rs = make_rsrc(Ab, (uint32_t)((size_t)L.R * K * 2));
            aoff = row < L.R ? ((uint32_t)row * (uint32_t)K + 8u * h) * 2u : OOR;
        }
        const int KS = K / 64;
        const int nst = (KS - wave + TH_WAVES - 1) / TH_WAVES;   // steps of this wave

        f32x16 acc0, acc1;
#pragma unroll
        for (int e = 0; e < 16; ++e) { acc0[e] = 0.f; acc1[e] = 0.f; }
        bf16x8 w[2][8], a[2][4];
        auto load = [&](int buf, int it) {
            const int st = wave + it * TH_WAVES;
            // a step past the end reads zeros through the range check and adds nothing
            const uint32_t ok = it < nst ? 0u : OOR;
            const uint32_t k0 = (uint32_t)st * 128u;   // bytes into a token or activation row
            const uint32_t kb = (uint32_t)st * (uint32_t)(WB_ROWS * WB_K * 2);   // bytes into the weight blocks
#pragma unroll
            for (int i = 0; i < 8; ++i) w[buf][i] = buf_load16(rb_rs, (wblk0 + i * 1024u) | ok, kb);
#pragma unroll
            for (int i = 0; i < 4; ++i) a[buf][i] = buf_load16(ra_rs, aoff | ok, k0 + 32u * i);
        };
        auto mma = [&](int buf) {
            // the wave's own LDS rows: stores, then fragment reads, in program order
#pragma unroll
            for (int i = 0; i < 8; ++i) *(bf16x8*)(wdst + i * 8 * TH_LDK) = w[buf][i];
            bf16x8 b0[4], b1[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                b0[i] = *(const bf16x8*)(frag + i * 32);
                b1[i] = *(const bf16x8*)(frag + 32 * TH_LDK + i * 32);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[buf][i], b0[i], acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[buf][i], b1[i], acc1, 0, 0, 0);
            }
        };
        load(0, 0);
        for (int it = 0; it < nst; it += 2) {
            load(1, it + 1);
            __builtin_amdgcn_sched_barrier(0);
            mma(0);
            __builtin_amdgcn_sched_barrier(0);
            load(0, it + 2);
            __builtin_amdgcn_sched_barrier(0);
            mma(1);
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();     // every wave is done with its staging rows
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            red[wave][0][e][lane] = acc0[e];
            red[wave][1][e][lane] = acc1[e];
        }
        __syncthreads();
        // element e of lane l in a 32x32 block: row (e/4)*8 + (l/32)*4 + e%4, column l%32
        if (MODE == 0) {
            __bf16* out = shared ? (__bf16*)p.Os : (__bf16*)p.Or;
            const int ldo = L.N / 2;
            const int orow0 = shared ? 0 : L.rowbase;
            const int col = tid & 31, rg = tid >> 5;
            const int ln = col + 32 * (rg >> 2);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = rg + 8 * i;            // row inside the tile
                const int e = 4 * i + (rg & 3);
                float gv = 0.f, uv = 0.f;
#pragma unroll
                for (int w = 0; w < TH_WAVES; ++w) { gv += red[w][0][e][ln]; uv += red[w][1][e][ln]; }
                if (L.m0 + r < L.R)
                    out[(size_t)(orow0 + L.m0 + r) * ldo + L.n0 / 2 + col] = (__bf16)(silu_f(gv) * uv);
            }
        } else {
            __bf16* out = (__bf16*)p.Or;
            const int ldo = L.N;
            const int col = tid & 63, rg = tid >> 6;
            const int j = col >> 5, cl = col & 31;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int r = rg + 4 * i;
                const int e = 4 * (r >> 3) + (r & 3);
                const int ln = cl + 32 * ((r >> 2) & 1);
                float v = 0.f;
#pragma unroll
                for (int w = 0; w < TH_WAVES; ++w) v += red[w][j][e][ln];
                if (L.m0 + r < L.R) {
                    const float wr = p.row_w[L.rowbase + L.m0 + r];
                    out[(size_t)(L.rowbase + L.m0 + r) * ldo + L.n0 + col] = (__bf16)(v * wr);
                }
            }
        }
        __syncthreads();
    }
}

// fp32 storage: plain LDS-tiled FMA GEMM, 64 x 64 tiles, 4 x 4 outputs per thread
template <int MODE>
__global__ void __launch_bounds__(256) ggemm_f32(const GemmArgs p) {
    constexpr int BM = 64, BN = 64, BK = 16;
    __shared__ float sA[BK][BM + 4];
    __shared__ float sB[BK][BN + 4];
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int total = *p.ntiles;
    for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
        TileLoc L;
        if (!decode_tile<BM, BN>(p, tile, L)) break;
        const bool shared = L.g >= p.n_routed;
        const float* Bw = shared ? (const float*)p.Ws : (const float*)p.Wr + (int64_t)L.g * L.N * L.K;
        float acc[4][4] = {};
        for (int k0 = 0; k0 < L.K; k0 += BK) {
            // A tile: 64 rows x 16 k, B tile: 64 cols x 16 k (4 elements per thread each)
            for (int v = 0; v < 4; ++v) {
                const int id = v * 256 + tid, r = id >> 4, kk = id & 15;
                const int row = L.m0 + r;
                float av = 0.f;
                if (row < L.R) {
                    if (MODE == 0) {
                        const int tok = p.row_tok[L.rowbase + row];
                        av = ((const float*)p.X)[(int64_t)tok * p.ldx + k0 + kk];
                    } else {
                        const float* base = shared ? (const float*)p.As
                                                   : (const float*)p.Ar + (int64_t)L.rowbase * L.K;
                        av = base[(int64_t)row * L.K + k0 + kk];
                    }
                }
                sA[kk][r] = av;
                sB[kk][r] = Bw[(int64_t)(L.n0 + r) * L.K + k0 + kk];
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < BK; ++kk) {
                float a4[4], b4[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) { a4[i] = sA[kk][ty * 4 + i]; b4[i] = sB[kk][tx * 4 + i]; }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a4[i], b4[j], acc[i][j]);
            }
            __syncthreads();
        }
        if (MODE == 1) {
            float* out = (float*)p.Or;
            for (int i = 0; i < 4; ++i) {
                const int row = L.m0 + ty * 4 + i;
                if (row >= L.R) continue;
                const float wr = p.row_w[L.rowbase + row];
                for (int j = 0; j < 4; ++j)
                    out[(int64_t)(L.rowbase + row) * L.N + L.n0 + tx * 4 + j] = acc[i][j] * wr;
            }
        }
        if (MODE == 0) {
            // packed rows alternate 16 gate / 16 up columns: pair them up
            // through LDS, then write silu(g) * u
            __shared__ float sC[BM][BN + 1];
            for (int i = 0; i < 4; ++i)
                for (int j = 0; j < 4; ++j) sC[ty * 4 + i][tx * 4 + j] = acc[i][j];
            __syncthreads();
            float* out = shared ? (float*)p.Os : (float*)p.Or;
            const int ldo = L.N / 2;
            for (int idx = tid; idx < BM * (BN / 2); idx += 256) {
                const int r = idx / (BN / 2), c = idx % (BN / 2);   // activation column within tile
                const int row = L.m0 + r;
                if (row >= L.R) continue;
                const int blk = c >> 5, cc = c & 31;
                const float gv = sC[r][blk * 64 + cc], uv = sC[r][blk * 64 + 32 + cc];
                const int orow = (shared ? 0 : L.rowbase) + row;
                out[(int64_t)orow * ldo + L.n0 / 2 + c] = gv / (1.0f + __expf(-gv)) * uv;   // fp32: IEEE divide
            }
            __syncthreads();
        }
    }
}

struct CombineArgs {
    int64_t T;
    int d, stride, dtype;
    const int32_t* tok_rows;
    const void* obuf;
    void* y;
};

__global__ void __launch_bounds__(256) combine_kernel(const CombineArgs c) {
    const int64_t t = blockIdx.x;
    int rows[MAXR];
    int n = 0;
    for (int i = 0; i < c.stride; ++i) {
        const int r = c.tok_rows[t * c.stride + i];
        if (r >= 0) rows[n++] = r;
    }
    if (c.dtype == ORDERMOE_BF16) {
        const __bf16* O = (const __bf16*)c.obuf;
        __bf16* Y = (__bf16*)c.y + t * c.d;
        for (int col = threadIdx.x * 8; col < c.d; col += 256 * 8) {
            float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            for (int i = 0; i < n; ++i) {
                const bf16x8 v = *(const bf16x8*)(O + (int64_t)rows[i] * c.d + col);
#pragma unroll
                for (int q = 0; q < 8; ++q) s[q] += (float)v[q];
            }
            bf16x8 o;
#pragma unroll
            for (int q = 0; q < 8; ++q) o[q] = (__bf16)s[q];
            *(bf16x8*)(Y + col) = o;
        }
    } else {
        const float* O = (const float*)c.obuf;
        float* Y = (float*)c.y + t * c.d;
        for (int col = threadIdx.x; col < c.d; col += 256) {
            float s = 0.f;
            for (int i = 0; i < n; ++i) s += O[(int64_t)rows[i] * c.d + col];
            Y[col] = s;
        }
    }
}


constexpr int GU_BM = 256, GU_BN = 256, DN_BM = 192, DN_BN = 256;   // bf16 GEMM tiles
// Large batches take 256-row down tiles: when even 256-row tiles would fill
// the grid DN_TALL_ROUNDS times over by the host's upper bound on the rows,
// the taller tile's better operand reuse outweighs the rounding of the last
// tile of each group and the shorter last round; smaller batches keep 192
// rows, which spread a few thousand rows over more of the 256 CUs.
constexpr int DN_BM_TALL = 256;
constexpr int64_t DN_TALL_ROUNDS = 8;
constexpr int F32_BM = 64, F32_BN = 64;
// bf16 batches of at most THIN_MAX_T tokens (every expert then has at most that
// many rows) take the thin GEMM, THIN_PER_CU resident workgroups per CU
constexpr int64_t THIN_MAX_T = 128;
constexpr int THIN_PER_CU = 3;

int persistent_grid(int64_t upper_tiles, int per_cu) {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) cus = v;
    }
    int64_t g = (int64_t)cus * per_cu;
    if (upper_tiles < g) g = upper_tiles;
    g = (g + 7) & ~int64_t(7);
    return (int)(g < 8 ? 8 : g);
}

// grid of a bf16 GEMM launch: up to SK_SPLIT workgroups per tile (the split
// tiles are shared out over them), at most SK_MAX_GRID
int bf16_grid(int64_t upper_tiles) {
    const int g = persistent_grid((int64_t)SK_SPLIT * upper_tiles, 1);
    return g < SK_MAX_GRID ? g : SK_MAX_GRID;
}

}  // namespace

size_t forward_split_counters() { return 2 * SK_MAX_GRID; }

size_t forward_split_floats(int dtype, int64_t T) {
    if (dtype != ORDERMOE_BF16 || forward_uses_thin(dtype, T)) return 0;
    const size_t tile = (size_t)GU_BM * GU_BN > (size_t)DN_BM * DN_BN ? (size_t)GU_BM * GU_BN : (size_t)DN_BM * DN_BN;
    return (size_t)SK_MAX_GRID * tile;
}

int forward_tokens_per_block() { return FT_TB; }

bool forward_uses_thin(int dtype, int64_t T) { return dtype == ORDERMOE_BF16 && T <= THIN_MAX_T; }

void forward_tile_shape(int dtype, int64_t T, int* bm_gu, int* bn_gu, int* bm_dn, int* bn_dn) {
    if (forward_uses_thin(dtype, T)) { *bm_gu = *bm_dn = TH_BM; *bn_gu = *bn_dn = TH_BN; }
    else if (dtype == ORDERMOE_BF16) { *bm_gu = GU_BM; *bn_gu = GU_BN; *bm_dn = DN_BM; *bn_dn = DN_BN; }
    else { *bm_gu = F32_BM; *bn_gu = F32_BN; *bm_dn = F32_BM; *bn_dn = F32_BN; }
}

int launch_local_forward(const ForwardArgs& f, void* stream) {
    hipStream_t st = (hipStream_t)stream;
    const int has_sh = f.n_shared > 0 ? 1 : 0;
    const int G = f.n_local + has_sh;
    const bool thin = forward_uses_thin(f.dtype, f.T);
    int bm_gu, bn_gu, bm_dn, bn_dn;
    forward_tile_shape(f.dtype, f.T, &bm_gu, &bn_gu, &bm_dn, &bn_dn);
    const int64_t rows_r = f.rmax_routed, rows_s = has_sh ? f.T : 0;
    if (!thin && f.dtype == ORDERMOE_BF16 &&
        ((rows_r + rows_s + DN_BM_TALL - 1) / DN_BM_TALL + G) * (f.d / DN_BN) >= DN_TALL_ROUNDS * SK_MAX_GRID)
        bm_dn = DN_BM_TALL;

    RowsArgs r;
    r.T = f.T; r.k = f.k; r.E = f.E; r.n_local = f.n_local; r.has_shared = has_sh; r.server = f.server;
    r.w = f.w; r.exec_k = f.exec_k; r.exec_m = f.exec_m; r.loc_in = f.loc_in;
    for (int i = 0; i < ORDERMOE_MAX_EXPERTS; ++i) r.lidx[i] = f.lidx[i];
    r.blk_rows = f.blk_rows; r.row_offsets = f.row_offsets;
    r.row_tok = f.row_tok; r.row_w = f.row_w; r.tok_rows = f.tok_rows; r.tile_info = f.tile_info;
    r.sk_cnt = f.sk_cnt; r.nblk = f.nblk;
    r.bm_gu = bm_gu; r.bn_gu = bn_gu; r.bm_dn = bm_dn; r.bn_dn = bn_dn;
    r.n_gu_r = 2 * f.f; r.n_gu_s = 2 * f.n_shared * f.f; r.n_dn = f.d;

    hipError_t e;
    if (f.T <= SCAN_THREADS) {
        {
            KernelTimer kt_("rows_small", st);
            hipLaunchKernelGGL(rows_small_kernel, dim3(1), dim3(SCAN_THREADS), 0, st, r);
        }
        if ((e = hipGetLastError()) != hipSuccess) return (int)e;
        if (f.nblk == 0) return 0;
    } else {
        {
            KernelTimer kt_("rows_count", st);
            hipLaunchKernelGGL(rows_count_kernel, dim3(f.nblk), dim3(FT_TB), 0, st, r);
        }
        if ((e = hipGetLastError()) != hipSuccess) return (int)e;
        {
            KernelTimer kt_("rows_scatter", st);
            hipLaunchKernelGGL(rows_scatter_kernel, dim3(f.nblk), dim3(FT_TB), 0, st, r);
        }
        if ((e = hipGetLastError()) != hipSuccess) return (int)e;
    }

    GemmArgs g{};
    g.offsets = f.row_offsets; g.G = G; g.n_routed = f.n_local;
    g.X = f.x; g.row_tok = f.row_tok; g.ldx = f.d; g.row_w = f.row_w;
    g.x_bytes = (uint32_t)((size_t)f.T * f.d * (f.dtype == ORDERMOE_BF16 ? 2 : 4));
    g.sk_part = f.sk_part; g.sk_cnt = f.sk_cnt;

    // gate/up: [rows][d] x [2f][d]^T -> activations [rows][f]
    g.ntiles = f.tile_info + 0;
    g.Nr = 2 * f.f; g.Kr = f.d; g.Ns = 2 * f.n_shared * f.f; g.Ks = f.d;
    g.Wr = f.w_gu; g.Ws = f.w_sh_gu; g.Ar = nullptr; g.As = nullptr; g.Or = f.act_r; g.Os = f.act_s;
    int64_t ub_gu = ((rows_r + bm_gu - 1) / bm_gu + f.n_local) * (2 * f.f / bn_gu) +
                    (has_sh ? ((rows_s + bm_gu - 1) / bm_gu + 1) * (2 * f.n_shared * f.f / bn_gu) : 0);
    int64_t ub_dn = ((rows_r + rows_s + bm_dn - 1) / bm_dn + G) * (f.d / bn_dn);

    if (thin) {
        {
        KernelTimer kt_("gemm_gate_up", st);
        ggemm_thin<0><<<dim3(persistent_grid(ub_gu, THIN_PER_CU)), dim3(256), 0, st>>>(g);
        }
        if ((e = hipGetLastError()) != hipSuccess) return (int)e;
    } else if (f.dtype == ORDERMOE_BF16) {
        {
        KernelTimer kt_("gemm_gate_up", st);
        ggemm_bf16<GU_BM, GU_BN, 0><<<dim3(bf16_grid(ub_gu)), dim3(256), 0, st>>>(g);
        }
        if ((e = hipGetLastError()) != hipSuccess) return (int)e;
    } else {
        {
        KernelTimer kt_("gemm_gate_up", st);
        ggemm_f32<0><<<dim3(persistent_grid(ub_gu, 4)), dim3(256), 0, st>>>(g);
        }
        if ((e = hipGetLastError()) != hipSuccess) return (int)e;
    }

    // down: activations [rows][f] x [d][f]^T -> row outputs [rows][d], scaled by the gate
    g.ntiles = f.tile_info + 1;
    g.Nr = f.d; g.Kr = f.f; g.Ns = f.d; g.Ks = f.n_shared * f.f;
    g.Wr = f.w_dn; g.Ws = f.w_sh_dn; g.Ar = f.act_r; g.As = f.act_s; g.Or = f.obuf; g.Os = nullptr;
    if (thin) {
        {
        KernelTimer kt_("gemm_down", st);
        ggemm_thin<1><<<dim3(persistent_grid(ub_dn, THIN_PER_CU)), dim3(256), 0, st>>>(g);
        }
    } else if (f.dtype == ORDERMOE_BF16) {
        {
        KernelTimer kt_("gemm_down", st);
        if (bm_dn == DN_BM_TALL) ggemm_bf16<DN_BM_TALL, DN_BN, 1><<<dim3(bf16_grid(ub_dn)), dim3(256), 0, st>>>(g);
        else ggemm_bf16<DN_BM, DN_BN, 1><<<dim3(bf16_grid(ub_dn)), dim3(256), 0, st>>>(g);
        }
    } else {
        {
        KernelTimer kt_("gemm_down", st);
        ggemm_f32<1><<<dim3(persistent_grid(ub_dn, 4)), dim3(256), 0, st>>>(g);
        }
    }
    if ((e = hipGetLastError()) != hipSuccess) return (int)e;

    CombineArgs c;
    c.T = f.T; c.d = f.d; c.stride = f.k + 1; c.dtype = f.dtype; c.tok_rows = f.tok_rows;
    c.obuf = f.obuf; c.y = f.y;
    {
        KernelTimer kt_("combine", st);
        hipLaunchKernelGGL(combine_kernel, dim3((unsigned)f.T), dim3(256), 0, st, c);
        }
    if ((e = hipGetLastError()) != hipSuccess) return (int)e;
    return 0;
}

int launch_pack_gate_up(int dtype, int n, int f, int d, const void* g, const void* u, void* out,
                        void* stream) {
    const int esz = dtype == ORDERMOE_BF16 ? 2 : 4;
    const int64_t rows = (int64_t)n * 2 * f;
    if (rows == 0) return 0;
    hipLaunchKernelGGL(pack_gate_up_kernel, dim3((unsigned)rows), dim3(256), 0, (hipStream_t)stream,
                       esz, f, d, (const char*)g, (const char*)u, (char*)out);
    return (int)hipGetLastError();
}

int launch_pack_down(int dtype, int n, int d, int f, const void* w, void* out, void* stream) {
    const int esz = dtype == ORDERMOE_BF16 ? 2 : 4;
    const int64_t rows = (int64_t)n * d;
    if (rows == 0) return 0;
    hipLaunchKernelGGL(pack_down_kernel, dim3((unsigned)rows), dim3(256), 0, (hipStream_t)stream,
                       esz, d, f, (const char*)w, (char*)out);
    return (int)hipGetLastError();
}

}  // namespace ordermoe
