// C ABI entry points of the device side: validation, workspace carving and
// kernel launches.  The host-only algorithms live in host_logic.cpp.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"

namespace ordermoe {

static thread_local std::string g_err;

void set_error(const std::string& msg) { g_err = msg; }
void clear_error() { g_err.clear(); }
int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

static int hip_fail(int e, const char* where) {
    return fail(ORDERMOE_EHIP, std::string(where) + ": " + hipGetErrorString((hipError_t)e));
}

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace ordermoe

using namespace ordermoe;

extern "C" const char* ordermoe_last_error(void) { return g_err.c_str(); }

// ------------------------------------------------------------ similarity
static int sim_parts(int64_t T_cal) {
    const int64_t tc = similarity_tokens_per_chunk(0);
    const int64_t chunks = (T_cal + tc - 1) / tc;
    return (int)std::min<int64_t>(chunks, 256);   // one partial per CU at most
}

static size_t sim_ws(int64_t T_cal, Carver& c, SimArgs* a) {
    const int parts = sim_parts(T_cal);
    const int emax = similarity_max_experts();
    float* g = c.take<float>((size_t)parts * emax * emax);
    int32_t* n = c.take<int32_t>((size_t)parts * emax);
    double* gr = c.take<double>((size_t)emax * emax);
    if (a) { a->gram_part = g; a->count_part = n; a->gram = gr; a->nchunk = parts; }
    return c.size();
}

extern "C" size_t ordermoe_similarity_workspace_size(int64_t T_cal, int32_t d, int32_t E) {
    (void)d; (void)E;
    if (T_cal < 1) return 0;
    Carver c(nullptr);
    return sim_ws(T_cal, c, nullptr);
}

extern "C" int ordermoe_build_similarity(const void* x_cal, int64_t T_cal, int32_t d,
                                         const void* w_router, int32_t E, int32_t dtype,
                                         int32_t topk, float theta, double alpha_f,
                                         float* sim_dev, int64_t* counts_dev, int32_t* top1_dev,
                                         float* sim_host,
                                         int64_t* counts_host, int32_t* group_of,
                                         int32_t* centres, int32_t* num_groups,
                                         double* importance, void* ws, size_t ws_bytes,
                                         void* stream) {
    if (dtype != ORDERMOE_F32 && dtype != ORDERMOE_BF16) return fail(ORDERMOE_EDTYPE, "build_similarity: dtype");
    if (T_cal < 1 || d < 64 || d % 64 != 0) return fail(ORDERMOE_EINVAL, "build_similarity: need T_cal >= 1 and d % 64 == 0");
    if (E < 1 || E > similarity_max_experts())
        return fail(ORDERMOE_EINVAL, "build_similarity: E must lie in [1, " + std::to_string(similarity_max_experts()) + "]");
    if (topk < 1 || topk > E || topk > ORDERMOE_MAX_TOPK) return fail(ORDERMOE_EINVAL, "build_similarity: topk out of range");
    if (!x_cal || !w_router || !sim_dev || !counts_dev || !group_of || !centres || !num_groups || !importance)
        return fail(ORDERMOE_EINVAL, "build_similarity: null pointer");
    if (!aligned16(x_cal) || !aligned16(w_router)) return fail(ORDERMOE_EINVAL, "build_similarity: inputs must be 16-byte aligned");
    if (!(alpha_f >= 0.0 && alpha_f <= 1.0)) return fail(ORDERMOE_EINVAL, "build_similarity: alpha_f must lie in [0, 1]");
    const size_t need = ordermoe_similarity_workspace_size(T_cal, d, E);
    if (!ws || ws_bytes < need)
        return fail(ORDERMOE_EWORKSPACE, "build_similarity: workspace needs " + std::to_string(need) + " bytes");

    SimArgs a{};
    a.dtype = dtype; a.d = d; a.E = E; a.k = topk; a.x_cal = x_cal; a.T_cal = T_cal;
    a.w_router = w_router; a.sim = sim_dev; a.counts = counts_dev; a.top1 = top1_dev;
    Carver c(ws);
    sim_ws(T_cal, c, &a);
    int e = launch_similarity(a, stream);
    if (e) return hip_fail(e, "build_similarity launch");

    std::vector<float> sim((size_t)E * E);
    std::vector<int64_t> cnt(E);
    hipStream_t st = (hipStream_t)stream;
    if ((e = (int)hipMemcpyAsync(sim.data(), sim_dev, sim.size() * 4, hipMemcpyDeviceToHost, st)))
        return hip_fail(e, "build_similarity copy");
    if ((e = (int)hipMemcpyAsync(cnt.data(), counts_dev, cnt.size() * 8, hipMemcpyDeviceToHost, st)))
        return hip_fail(e, "build_similarity copy");
    if ((e = (int)hipStreamSynchronize(st))) return hip_fail(e, "build_similarity sync");
    if (sim_host) std::copy(sim.begin(), sim.end(), sim_host);
    if (counts_host) std::copy(cnt.begin(), cnt.end(), counts_host);
    return ordermoe_group_experts(E, sim.data(), cnt.data(), theta, alpha_f, group_of, centres,
                                  num_groups, importance);
}

// ------------------------------------------------------------ route / select
static size_t route_ws(int64_t T, int32_t k, int32_t M, Carver& c, RouteArgs* a) {
    (void)k;
    const int tb = route_tokens_per_block();
    const int nblk = (int)((T + tb - 1) / tb);
    int32_t* bd = c.take<int32_t>((size_t)std::max(nblk, 1) * M);
    int64_t* bc = c.take<int64_t>((size_t)std::max(nblk, 1) * 8);
    // small batches split the router over K slices: room for their partial logits
    float* lp = c.take<float>(route_split_buffer_floats(T));
    if (a) { a->blk_dst = bd; a->blk_cnt = bc; a->logit_part = lp; a->nblk = nblk; }
    return c.size();
}

extern "C" size_t ordermoe_route_workspace_size(int64_t T, int32_t k, int32_t M) {
    if (T < 0 || M < 1) return 0;
    Carver c(nullptr);
    return route_ws(T, k, M, c, nullptr);
}

static int run_route(const ordermoe_layer* L, const void* x, int64_t T, const uint8_t* loc_in,
                     const float* qhat_in, const ordermoe_route_out* out, void* ws, void* stream,
                     const char* who);

static int check_route_args(const ordermoe_layer* L, const void* x, int64_t T, const uint8_t* loc_in,
                            const float* qhat_in, const ordermoe_route_out* out) {
    if (!L || !out) return fail(ORDERMOE_EINVAL, "route_select: null layer or output struct");
    if (L->dtype != ORDERMOE_F32 && L->dtype != ORDERMOE_BF16) return fail(ORDERMOE_EDTYPE, "route_select: dtype");
    if (L->d < 64 || L->d % 64 != 0) return fail(ORDERMOE_EINVAL, "route_select: d must be a positive multiple of 64");
    if (L->E < 1 || L->E > ORDERMOE_MAX_EXPERTS) return fail(ORDERMOE_EINVAL, "route_select: E out of range");
    if (L->k < 1 || L->k > L->E || L->k > ORDERMOE_MAX_TOPK) return fail(ORDERMOE_EINVAL, "route_select: k out of range");
    if (L->M < 1 || L->M > ORDERMOE_MAX_SERVERS) return fail(ORDERMOE_EINVAL, "route_select: M out of range");
    if (L->gmax < 1 || L->gmax > ORDERMOE_MAX_SUBS) return fail(ORDERMOE_EINVAL, "route_select: gmax out of range");
    if (!(L->Qbar >= 0.0f) || !(L->omega_Q >= 0.0f)) return fail(ORDERMOE_EINVAL, "route_select: Qbar and omega_Q must be >= 0");
    if (L->allow_sub < 0 || L->allow_sub > 2) return fail(ORDERMOE_EINVAL, "route_select: allow_sub must be 0, 1 or 2");
    if (T < 0) return fail(ORDERMOE_EINVAL, "route_select: T < 0");
    if (T > ((int64_t)1 << 31) / ORDERMOE_MAX_TOPK) return fail(ORDERMOE_EINVAL, "route_select: T too large");
    if (!L->w_router || !L->t1_k || !L->t1_q || !L->t1_n || !L->srvmask || !L->S)
        return fail(ORDERMOE_EINVAL, "route_select: null table pointer");
    if (!out->dst_count || !out->counters) return fail(ORDERMOE_EINVAL, "route_select: null output pointer");
    if (T > 0 && (!x || !loc_in || !qhat_in || !out->idx || !out->w || !out->margin || !out->flag ||
                  !out->exec_k || !out->exec_m || !out->cls || !out->qhat_out || !out->loc_out ||
                  !out->dispatch))
        return fail(ORDERMOE_EINVAL, "route_select: null pointer");
    if ((T > 0 && !aligned16(x)) || !aligned16(L->w_router))
        return fail(ORDERMOE_EINVAL, "route_select: x and w_router must be 16-byte aligned");
    return ORDERMOE_OK;
}

extern "C" int ordermoe_route_select(const ordermoe_layer* L, const void* x, int64_t T,
                                     const uint8_t* loc_in, const float* qhat_in,
                                     const ordermoe_route_out* out, void* ws, size_t ws_bytes,
                                     void* stream) {
    const int rc = check_route_args(L, x, T, loc_in, qhat_in, out);
    if (rc) return rc;
    const size_t need = ordermoe_route_workspace_size(T, L->k, L->M);
    if (!ws || ws_bytes < need)
        return fail(ORDERMOE_EWORKSPACE, "route_select: workspace needs " + std::to_string(need) + " bytes");
    return run_route(L, x, T, loc_in, qhat_in, out, ws, stream, "route_select launch");
}

// scratch of ordermoe_route_select_noalloc: one copy per GPU, held for the life
// of the process; host code addresses it only through the device address that
// hipGetSymbolAddress returns for the current device (never by this name)
static __device__ __align__(256) char scratch[ORDERMOE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_dev[kMaxDevices] = {};

// the current device's copy of `scratch`, looked up once per device
static int scratch_address(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail((int)e, "route_select_noalloc: hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(ORDERMOE_EINVAL, "route_select_noalloc: device id beyond " + std::to_string(kMaxDevices));
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail((int)e, "route_select_noalloc: hipGetSymbolAddress(scratch)");
        g_scratch_dev[dev] = p;
    }
    *ptr = g_scratch_dev[dev];
    return ORDERMOE_OK;
}

extern "C" int ordermoe_route_select_noalloc(const ordermoe_layer* L, const void* x, int64_t T,
                                             const uint8_t* loc_in, const float* qhat_in,
                                             const ordermoe_route_out* out, void* stream) {
    const int rc = check_route_args(L, x, T, loc_in, qhat_in, out);
    if (rc) return rc;
    const size_t need = ordermoe_route_workspace_size(T, L->k, L->M);
    if (need > (size_t)ORDERMOE_NOALLOC_SCRATCH_BYTES)
        return fail(ORDERMOE_EWORKSPACE, "route_select_noalloc: this batch needs " + std::to_string(need) +
                                            " bytes of scratch, above the fixed " +
                                            std::to_string((size_t)ORDERMOE_NOALLOC_SCRATCH_BYTES));
    void* ws = nullptr;
    const int r2 = scratch_address(&ws);
    if (r2) return r2;
    return run_route(L, x, T, loc_in, qhat_in, out, ws, stream, "route_select_noalloc launch");
}

static int run_route(const ordermoe_layer* L, const void* x, int64_t T, const uint8_t* loc_in,
                     const float* qhat_in, const ordermoe_route_out* out, void* ws, void* stream,
                     const char* who) {
    RouteArgs a{};
    a.dtype = L->dtype; a.d = L->d; a.E = L->E; a.k = L->k; a.M = L->M; a.gmax = L->gmax;
    a.pin = L->pin_local_exact; a.allow_sub = L->allow_sub; a.renorm = L->renorm;
    a.Qbar = L->Qbar;
    a.cq = L->Qbar > 0.0f ? L->omega_Q / L->Qbar : 0.0f;   // eq 38 weight of Q, fp32
    a.w_router = L->w_router; a.t1_k = L->t1_k; a.t1_q = L->t1_q; a.t1_n = L->t1_n;
    a.srvmask = L->srvmask; a.S = L->S;
    a.x = x; a.T = T; a.loc_in = loc_in; a.qhat_in = qhat_in; a.out = *out;
    Carver c(ws);
    route_ws(T, L->k, L->M, c, &a);
    int e = launch_route_select(a, stream);
    if (e) return hip_fail(e, who);
    clear_error();
    return ORDERMOE_OK;
}

// ------------------------------------------------------------ local forward
static int64_t fwd_rmax_routed(const ordermoe_experts* W, int64_t T, int32_t k) {
    return T * (int64_t)std::min(k, W->n_local);
}

static size_t fwd_ws(const ordermoe_experts* W, int64_t T, int32_t k, Carver& c, ForwardArgs* a) {
    const int tb = forward_tokens_per_block();
    const int nblk = (int)((T + tb - 1) / tb);
    const int has_sh = W->n_shared > 0;
    const int G = W->n_local + has_sh;
    const int64_t rr = fwd_rmax_routed(W, T, k);
    const int64_t rs = has_sh ? T : 0;
    const size_t esz = W->dtype == ORDERMOE_BF16 ? 2 : 4;
    int32_t* br = c.take<int32_t>((size_t)std::max(nblk, 1) * std::max(G, 1));
    int32_t* rt = c.take<int32_t>((size_t)std::max<int64_t>(rr + rs, 1));
    float* rw = c.take<float>((size_t)std::max<int64_t>(rr + rs, 1));
    int32_t* tr = c.take<int32_t>((size_t)std::max<int64_t>(T * (k + 1), 1));
    int32_t* ti = c.take<int32_t>(4);
    char* ar = c.take<char>((size_t)rr * W->f * esz);
    char* as = c.take<char>((size_t)rs * W->n_shared * W->f * esz);
    char* ob = c.take<char>((size_t)(rr + rs) * W->d * esz);
    int32_t* sc = c.take<int32_t>(forward_split_counters());
    float* sp = c.take<float>(forward_split_floats(W->dtype, T));
    if (a) {
        a->blk_rows = br; a->row_tok = rt; a->row_w = rw; a->tok_rows = tr;
        a->tile_info = ti; a->act_r = ar; a->act_s = as; a->obuf = ob; a->rmax_routed = rr;
        a->sk_cnt = sc; a->sk_part = sp;
        a->nblk = nblk;
    }
    return c.size();
}

static int check_experts(const ordermoe_experts* W) {
    if (!W) return fail(ORDERMOE_EINVAL, "experts: null");
    if (W->dtype != ORDERMOE_F32 && W->dtype != ORDERMOE_BF16) return fail(ORDERMOE_EDTYPE, "experts: dtype");
    const int dmul = W->dtype == ORDERMOE_BF16 ? 256 : 64;
    const int fmul = W->dtype == ORDERMOE_BF16 ? 128 : 32;
    if (W->d < dmul || W->d % dmul != 0)
        return fail(ORDERMOE_EINVAL, "experts: d must be a positive multiple of " + std::to_string(dmul));
    if (W->f < fmul || W->f % fmul != 0)
        return fail(ORDERMOE_EINVAL, "experts: f must be a positive multiple of " + std::to_string(fmul));
    if (W->E < 1 || W->E > ORDERMOE_MAX_EXPERTS) return fail(ORDERMOE_EINVAL, "experts: E out of range");
    if (W->n_local < 0 || W->n_local > ORDERMOE_MAX_LOCAL || W->n_local > W->E)
        return fail(ORDERMOE_EINVAL, "experts: n_local out of range");
    if (W->n_shared < 0 || W->n_shared > 16) return fail(ORDERMOE_EINVAL, "experts: n_shared out of range");
    if (W->n_local > 0 && (!W->local_experts || !W->w_gate_up || !W->w_down))
        return fail(ORDERMOE_EINVAL, "experts: null routed weights");
    if (W->n_shared > 0 && (!W->w_shared_gate_up || !W->w_shared_down))
        return fail(ORDERMOE_EINVAL, "experts: null shared weights");
    for (int i = 0; i < W->n_local; ++i) {
        const int e = W->local_experts[i];
        if (e < 0 || e >= W->E || (i > 0 && e <= W->local_experts[i - 1]))
            return fail(ORDERMOE_EINVAL, "experts: local_experts must be increasing ids below E");
    }
    if ((W->w_gate_up && !aligned16(W->w_gate_up)) || (W->w_down && !aligned16(W->w_down)) ||
        (W->w_shared_gate_up && !aligned16(W->w_shared_gate_up)) ||
        (W->w_shared_down && !aligned16(W->w_shared_down)))
        return fail(ORDERMOE_EINVAL, "experts: weights must be 16-byte aligned");
    return ORDERMOE_OK;
}

// The GEMMs address each operand through a buffer resource with 32-bit byte
// offsets and mark rows past a group's end with offset 2^31, so every operand
// they read must span fewer than 2^31 bytes: the token rows (T x d), one
// expert's packed gate/up weights (2f x d) and down weights (d x f), the shared
// experts' concatenated weights (2 n_shared f x d, d x n_shared f), and one
// group's activation rows (at most T rows of f, or of n_shared f).
static bool operands_fit_31_bits(const ordermoe_experts* W, int64_t T) {
    const int64_t lim = ((int64_t)1 << 31) - 1;
    const int64_t esz = W->dtype == ORDERMOE_BF16 ? 2 : 4;
    const int64_t ns = W->n_shared > 0 ? W->n_shared : 1;
    const int64_t d = W->d, f = W->f;
    return T * d * esz <= lim && 2 * f * d * esz <= lim && 2 * ns * f * d * esz <= lim &&
           T * ns * f * esz <= lim;
}

extern "C" size_t ordermoe_forward_workspace_size(const ordermoe_experts* W, int64_t T, int32_t k) {
    if (check_experts(W) != ORDERMOE_OK || T < 0 || k < 1 || k > ORDERMOE_MAX_TOPK) return 0;
    if (!operands_fit_31_bits(W, T)) return 0;
    Carver c(nullptr);
    return fwd_ws(W, T, k, c, nullptr);
}

extern "C" int ordermoe_local_moe_forward(const ordermoe_experts* W, const void* x, int64_t T,
                                          int32_t k, const float* w, const int32_t* exec_k,
                                          const uint8_t* exec_m, const uint8_t* loc_in,
                                          int32_t server, void* y, int32_t* row_offsets,
                                          void* ws, size_t ws_bytes, void* stream) {
    int rc = check_experts(W);
    if (rc) return rc;
    if (k < 1 || k > ORDERMOE_MAX_TOPK) return fail(ORDERMOE_EINVAL, "local_moe_forward: k out of range");
    if (T < 0 || T > ((int64_t)1 << 31) / (ORDERMOE_MAX_TOPK + 1))
        return fail(ORDERMOE_EINVAL, "local_moe_forward: T out of range");
    if (!operands_fit_31_bits(W, T))
        return fail(ORDERMOE_EINVAL, "local_moe_forward: T*d, 2*f*d, 2*n_shared*f*d and T*n_shared*f elements "
                                     "must each span fewer than 2^31 bytes");
    if (server < 0 || server >= ORDERMOE_MAX_SERVERS) return fail(ORDERMOE_EINVAL, "local_moe_forward: server out of range");
    if (!row_offsets) return fail(ORDERMOE_EINVAL, "local_moe_forward: null row_offsets");
    if (T > 0 && (!x || !w || !exec_k || !exec_m || !loc_in || !y))
        return fail(ORDERMOE_EINVAL, "local_moe_forward: null pointer");
    if (T > 0 && (!aligned16(x) || !aligned16(y)))
        return fail(ORDERMOE_EINVAL, "local_moe_forward: x and y must be 16-byte aligned");
    const size_t need = ordermoe_forward_workspace_size(W, T, k);
    if (!ws || ws_bytes < need)
        return fail(ORDERMOE_EWORKSPACE, "local_moe_forward: workspace needs " + std::to_string(need) + " bytes");

    ForwardArgs a{};
    a.dtype = W->dtype; a.d = W->d; a.f = W->f; a.E = W->E; a.n_local = W->n_local;
    a.n_shared = W->n_shared; a.k = k;
    for (int i = 0; i < ORDERMOE_MAX_EXPERTS; ++i) a.lidx[i] = -1;
    for (int i = 0; i < W->n_local; ++i) a.lidx[W->local_experts[i]] = i;
    a.w_gu = W->w_gate_up; a.w_dn = W->w_down; a.w_sh_gu = W->w_shared_gate_up;
    a.w_sh_dn = W->w_shared_down;
    a.x = x; a.T = T; a.w = w; a.exec_k = exec_k; a.exec_m = exec_m; a.loc_in = loc_in;
    a.server = server; a.y = y; a.row_offsets = row_offsets;
    Carver c(ws);
    fwd_ws(W, T, k, c, &a);
    const int e = launch_local_forward(a, stream);
    if (e) return hip_fail(e, "local_moe_forward launch");
    clear_error();
    return ORDERMOE_OK;
}

extern "C" int ordermoe_pack_gate_up(int32_t dtype, int32_t n, int32_t f, int32_t d,
                                     const void* w_gate, const void* w_up, void* out,
                                     void* stream) {
    if (dtype != ORDERMOE_F32 && dtype != ORDERMOE_BF16) return fail(ORDERMOE_EDTYPE, "pack_gate_up: dtype");
    if (n < 0 || f < 32 || f % 32 != 0 || d < 8 || d % 8 != 0)
        return fail(ORDERMOE_EINVAL, "pack_gate_up: need n >= 0, f % 32 == 0, d % 8 == 0");
    if (dtype == ORDERMOE_BF16 && (f % 128 != 0 || d % 64 != 0))
        return fail(ORDERMOE_EINVAL, "pack_gate_up: bf16 needs f % 128 == 0 and d % 64 == 0");
    if (n > 0 && (!w_gate || !w_up || !out)) return fail(ORDERMOE_EINVAL, "pack_gate_up: null pointer");
    if (n > 0 && (!aligned16(w_gate) || !aligned16(w_up) || !aligned16(out)))
        return fail(ORDERMOE_EINVAL, "pack_gate_up: pointers must be 16-byte aligned");
    const int e = launch_pack_gate_up(dtype, n, f, d, w_gate, w_up, out, stream);
    if (e) return hip_fail(e, "pack_gate_up launch");
    clear_error();
    return ORDERMOE_OK;
}

extern "C" int ordermoe_pack_down(int32_t dtype, int32_t n, int32_t d, int32_t f, const void* w_down,
                                  void* out, void* stream) {
    if (dtype != ORDERMOE_F32 && dtype != ORDERMOE_BF16) return fail(ORDERMOE_EDTYPE, "pack_down: dtype");
    if (n < 0 || d < 1 || f < 8 || f % 8 != 0) return fail(ORDERMOE_EINVAL, "pack_down: need n >= 0, d >= 1, f % 8 == 0");
    if (dtype == ORDERMOE_BF16 && (d % 256 != 0 || f % 64 != 0))
        return fail(ORDERMOE_EINVAL, "pack_down: bf16 needs d % 256 == 0 and f % 64 == 0");
    if (n > 0 && (!w_down || !out)) return fail(ORDERMOE_EINVAL, "pack_down: null pointer");
    if (n > 0 && (!aligned16(w_down) || !aligned16(out)))
        return fail(ORDERMOE_EINVAL, "pack_down: pointers must be 16-byte aligned");
    const int e = launch_pack_down(dtype, n, d, f, w_down, out, stream);
    if (e) return hip_fail(e, "pack_down launch");
    clear_error();
    return ORDERMOE_OK;
}

extern "C" size_t ordermoe_transitions_device_workspace_size(int32_t N, int32_t E) {
    if (N < 1 || E < 1 || E > ORDERMOE_MAX_EXPERTS) return 0;
    return transitions_device_workspace(N, E);
}

extern "C" int ordermoe_estimate_transitions_device(int32_t N, int32_t E, int64_t T_cal, const int32_t* top1,
                                                    double* P, void* ws, size_t ws_bytes, void* stream) {
    if (N < 1 || E < 1 || E > ORDERMOE_MAX_EXPERTS || T_cal < 0)
        return fail(ORDERMOE_EINVAL, "estimate_transitions_device: size out of range");
    if (N == 1) { clear_error(); return ORDERMOE_OK; }
    if (!P || !ws || (T_cal > 0 && !top1)) return fail(ORDERMOE_EINVAL, "estimate_transitions_device: null pointer");
    const size_t need = transitions_device_workspace(N, E);
    if (ws_bytes < need)
        return fail(ORDERMOE_EWORKSPACE, "estimate_transitions_device: workspace needs " + std::to_string(need) + " bytes");
    const int e = launch_transitions_device(N, E, T_cal, top1, P, ws, stream);
    if (e) return hip_fail(e, "estimate_transitions_device launch");
    clear_error();
    return ORDERMOE_OK;
}

extern "C" size_t ordermoe_lookahead_device_workspace_size(int32_t N, int32_t E, int32_t M) {
    if (N < 1 || E < 1 || E > ORDERMOE_MAX_EXPERTS || M < 1 || M > ORDERMOE_MAX_SERVERS) return 0;
    return lookahead_device_workspace(N, E, M);
}

extern "C" int ordermoe_build_lookahead_device(int32_t N, int32_t E, int32_t M, int32_t H, const double* P,
                                               const uint8_t* x, const float* sim, const int32_t* group_of,
                                               const float* theta, const double* z_bits, const double* c,
                                               const double* d_ref, const double* B, const double* tau,
                                               const double* F, double omega_T, double omega_Q, float Qbar,
                                               int32_t pin_local_exact, int32_t allow_sub, double* phi_out,
                                               void* ws, size_t ws_bytes, void* stream) {
    if (N < 1 || E < 1 || E > ORDERMOE_MAX_EXPERTS || M < 1 || M > ORDERMOE_MAX_SERVERS || H < 1)
        return fail(ORDERMOE_EINVAL, "build_lookahead_device: size out of range");
    if (allow_sub < 0 || allow_sub > 2) return fail(ORDERMOE_EINVAL, "build_lookahead_device: allow_sub must be 0, 1 or 2");
    if (!phi_out || !ws) return fail(ORDERMOE_EINVAL, "build_lookahead_device: null pointer");
    if (H > 1 && N > 1 && (!P || !x || !sim || !group_of || !theta || !z_bits || !c || !d_ref || !B || !tau || !F))
        return fail(ORDERMOE_EINVAL, "build_lookahead_device: null pointer");
    const size_t need = lookahead_device_workspace(N, E, M);
    if (ws_bytes < need)
        return fail(ORDERMOE_EWORKSPACE, "build_lookahead_device: workspace needs " + std::to_string(need) + " bytes");
    LookaheadDeviceArgs d;
    d.N = N; d.E = E; d.M = M; d.H = H; d.P = P; d.x = x; d.sim = sim; d.group_of = group_of; d.theta = theta;
    d.z_bits = z_bits; d.c = c; d.d_ref = d_ref; d.B = B; d.tau = tau; d.F = F; d.omega_T = omega_T;
    d.omega_Q = omega_Q; d.Qbar = Qbar; d.pin = pin_local_exact; d.allow_sub = allow_sub; d.phi = phi_out;
    d.ws = ws;
    const int e = launch_lookahead_device(d, stream);
    if (e) return hip_fail(e, "build_lookahead_device launch");
    clear_error();
    return ORDERMOE_OK;
}
