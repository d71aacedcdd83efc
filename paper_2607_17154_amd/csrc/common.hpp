// Internal declarations shared by the library's translation units.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/ordermoe.h"

namespace ordermoe {

// Thread-local error message behind ordermoe_last_error().
void set_error(const std::string& msg);
void clear_error();

// Returns `code` after recording `msg` (for `return fail(...)` in entry points).
int fail(int code, const std::string& msg);

// Workspace carving: aligned sub-buffers taken in order from one caller buffer.
struct Carver {
    char* base;
    size_t off = 0;
    explicit Carver(void* b) : base(static_cast<char*>(b)) {}
    template <typename T>
    T* take(size_t count) {
        off = (off + 255) & ~size_t(255);
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
    size_t size() const { return (off + 255) & ~size_t(255); }
};

// Brackets one kernel launch with timing events when timing is enabled.
class KernelTimer {
  public:
    KernelTimer(const char* name, void* stream);
    ~KernelTimer();
    KernelTimer(const KernelTimer&) = delete;
    KernelTimer& operator=(const KernelTimer&) = delete;

  private:
    const char* name_;
    void* stream_;
    void* start_ = nullptr;
};

// ---- kernel launchers (defined in the .hip files) ----------------------
// All return a hipError_t value as int (0 = success).

struct RouteArgs {
    int dtype, d, E, k, M, gmax, pin, allow_sub, renorm;
    float Qbar, cq;
    const void* w_router;
    const int32_t* t1_k;
    const float* t1_q;
    const int32_t* t1_n;
    const uint32_t* srvmask;
    const float* S;
    const void* x;
    int64_t T;
    const uint8_t* loc_in;
    const float* qhat_in;
    ordermoe_route_out out;
    // workspace
    int32_t* blk_dst;      // [nblk][M] remote slots per destination per block
    int64_t* blk_cnt;      // [nblk][8] per-block counters
    float* logit_part;     // [ksplit][T][Epad] router partial logits of small batches
    int nblk;
    int S_in_lds;          // set by the launcher: stage the cost table in LDS
    int ksplit;            // set by the launcher: K slices of the split router (0: fused)
    int x_lds;             // set by the launcher: bytes of the LDS-staged token rows (0: none)
};
int launch_route_select(const RouteArgs& a, void* stream);
int route_tokens_per_block();
size_t route_split_buffer_floats(int64_t T);

struct ForwardArgs {
    int dtype, d, f, E, n_local, n_shared, k;
    int32_t lidx[ORDERMOE_MAX_EXPERTS];  // expert id -> local slot, -1 if not held
    const void* w_gu;
    const void* w_dn;
    const void* w_sh_gu;
    const void* w_sh_dn;
    const void* x;
    int64_t T;
    const float* w;
    const int32_t* exec_k;
    const uint8_t* exec_m;
    const uint8_t* loc_in;
    int server;
    void* y;
    int32_t* row_offsets;
    // workspace
    int32_t* blk_rows;     // [nblk][G] rows per group per block (G = n_local + has_shared)
    int32_t* row_tok;      // [rmax] token of each row
    float* row_w;          // [rmax] merged gate weight of each row
    int32_t* tok_rows;     // [T][k + 1] rows of each token, -1 padded
    int32_t* tile_info;    // [4]: tiles of the gate/up GEMM, of the down GEMM, rows, 0
    void* act_r;           // [rmax_routed][f] routed activations
    void* act_s;           // [T][n_shared * f] shared activations
    void* obuf;            // [rmax][d] per-row outputs
    float* sk_part;        // bf16 GEMMs: partial tiles of split tiles
    int32_t* sk_cnt;       // [forward_split_counters()] arrival counters of split tiles
    int64_t rmax_routed;
    int nblk;
};
int launch_local_forward(const ForwardArgs& a, void* stream);
int forward_tokens_per_block();
bool forward_uses_thin(int dtype, int64_t T);
void forward_tile_shape(int dtype, int64_t T, int* bm_gu, int* bn_gu, int* bm_dn, int* bn_dn);
size_t forward_split_counters();
size_t forward_split_floats(int dtype, int64_t T);

struct SimArgs {
    int dtype, d, E, k;
    const void* x_cal;
    int64_t T_cal;
    const void* w_router;
    float* sim;            // [E][E]
    int64_t* counts;       // [E]
    int32_t* top1;         // [T_cal] top-1 expert of each token, or null
    float* gram_part;      // [nchunk][128][128] per-block partial Gram matrices
    int32_t* count_part;   // [nchunk][128] per-block activation counts
    double* gram;          // [128][128] reduced Gram matrix
    int nchunk;            // blocks of the partial kernel (= number of partials)
};
int launch_similarity(const SimArgs& a, void* stream);
int64_t similarity_tokens_per_chunk(int E);
int similarity_max_experts();

// transition statistics and look-ahead tables on the device (lookahead.hip)
struct LookaheadDeviceArgs {
    int32_t N, E, M, H;
    const double* P;
    const uint8_t* x;
    const float* sim;
    const int32_t* group_of;
    const float* theta;
    const double* z_bits;
    const double* c;
    const double* d_ref;
    const double* B;
    const double* tau;
    const double* F;
    double omega_T, omega_Q;
    float Qbar;
    int32_t pin, allow_sub;
    double* phi;
    void* ws;
};
size_t transitions_device_workspace(int32_t N, int32_t E);
size_t lookahead_device_workspace(int32_t N, int32_t E, int32_t M);
int launch_transitions_device(int32_t N, int32_t E, int64_t T_cal, const int32_t* top1, double* P, void* ws,
                              void* stream);
int launch_lookahead_device(const LookaheadDeviceArgs& d, void* stream);

int launch_pack_gate_up(int dtype, int n, int f, int d, const void* g, const void* u, void* out,
                        void* stream);
int launch_pack_down(int dtype, int n, int d, int f, const void* w, void* out, void* stream);

}  // namespace ordermoe
