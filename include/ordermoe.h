/*
 * ordermoe.h -- C ABI of the OrderMoE layer library for AMD Instinct MI355X (gfx950).
 *
 * OrderMoE (arXiv 2607.17154) keeps MoE inference local on distributed edge
 * servers: experts of a layer are grouped by the similarity of their router
 * logits, similar experts are spread over servers, and at run time each token
 * either runs its routed ("target") expert, a feasible local substitute from
 * the target's similarity group, or is sent to another server.  This library
 * runs the data-parallel part of that method for one layer on the experts one
 * server holds:
 *
 *   ordermoe_build_similarity   Section III-B / IV-A, eq (3)-(5), (24)-(28)
 *   ordermoe_place              Section IV-B / IV-C, eq (29)-(35), Algorithm 1
 *   ordermoe_place_random       Section VI-A, the Random Deployment baseline
 *   ordermoe_simulate_delay     Section III-C/D/F, eq (13)-(17), (22)
 *   ordermoe_build_tables       eq (6)-(8), (18), (37)-(38) (+ eq (42) input)
 *   ordermoe_route_select       router + Section V, eq (36)-(44), Algorithm 2
 *   ordermoe_local_moe_forward  execution of the selected (server, expert)
 *                               pairs of one server (Algorithm 2, "execute
 *                               token q on S_m* by expert k*")
 *
 * Conventions
 *   - Every entry point returns ORDERMOE_OK (0) or a negative status code and
 *     never throws; ordermoe_last_error() returns a thread-local message for
 *     the last failure of the calling thread.
 *   - Arguments are validated before any device work is queued; on an error
 *     nothing has been launched and no output has been written.
 *   - The caller owns every buffer.  "dev" pointers are device memory on the
 *     current HIP device, "host" pointers are ordinary host memory.  The
 *     device entry points never allocate: scratch space comes from the
 *     caller's workspace, sized by the matching *_workspace_size function.
 *   - Device work is queued on the caller's stream (a hipStream_t passed as
 *     void*; NULL is the default stream).  ordermoe_route_select and
 *     ordermoe_local_moe_forward never wait for the device; their counters
 *     and row counts are written to device memory.  The library keeps no
 *     device state between calls (ordermoe_route_select_noalloc aside), so
 *     calls on different streams may run at the same time when no output or
 *     workspace of one is written or read by another: weights, tables and
 *     inputs are only read and may be shared.
 *   - Storage types: ORDERMOE_F32 (IEEE binary32) or ORDERMOE_BF16 (bfloat16).
 *     Matrices are row-major; weight matrices use the [out][in] layout of
 *     torch.nn.Linear.
 */
#ifndef ORDERMOE_H
#define ORDERMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define ORDERMOE_OK 0
#define ORDERMOE_EINVAL (-1)     /* bad argument: null pointer, size or range */
#define ORDERMOE_EDTYPE (-2)     /* unsupported storage type */
#define ORDERMOE_ECAPACITY (-3)  /* the servers cannot hold every expert once (eq 1-2) */
#define ORDERMOE_EHIP (-4)       /* a HIP runtime call failed */
#define ORDERMOE_EWORKSPACE (-5) /* workspace smaller than the required size */

/* storage types */
#define ORDERMOE_F32 0
#define ORDERMOE_BF16 1

/* execution classes of a (token, slot), as counted in Section VI-C */
#define ORDERMOE_LOCAL_EXACT 0
#define ORDERMOE_LOCAL_SUB 1
#define ORDERMOE_REMOTE_EXACT 2
#define ORDERMOE_REMOTE_SUB 3

/* limits */
#define ORDERMOE_MAX_SERVERS 32   /* M: one bit per server in a 32-bit mask */
#define ORDERMOE_MAX_EXPERTS 256  /* E per layer */
#define ORDERMOE_MAX_TOPK 8       /* k */
#define ORDERMOE_MAX_SUBS 15      /* substitutes per target kept in the table */
#define ORDERMOE_MAX_LOCAL 64     /* routed experts one server holds per layer */

/* a token whose smallest gap between adjacent sorted top-(k+1) router logits
 * is below this value is flagged: its routing is within rounding distance of
 * a tie */
#define ORDERMOE_MARGIN_FLAG 1.0e-4f

/* counters written by ordermoe_route_select (int64 each) */
#define ORDERMOE_CNT_LOCAL_EXACT 0
#define ORDERMOE_CNT_LOCAL_SUB 1
#define ORDERMOE_CNT_REMOTE_EXACT 2
#define ORDERMOE_CNT_REMOTE_SUB 3
#define ORDERMOE_CNT_FLAGGED 4     /* tokens with margin < ORDERMOE_MARGIN_FLAG */
#define ORDERMOE_CNT_TRANSFERS 5   /* distinct (token, destination server) pairs */
#define ORDERMOE_CNT_REMOTE_SLOTS 6
#define ORDERMOE_CNT_INVALID 7     /* tokens whose loc_in is not a server index */
#define ORDERMOE_NUM_COUNTERS 8

/* Message describing the calling thread's last failure ("" if none). */
const char* ordermoe_last_error(void);

/* ------------------------------------------------------------------------
 * Similarity model (Section III-B, IV-A; Algorithm 1, grouping part).
 *
 * Device part: H = W_r X_cal^T (eq 3) over the calibration tokens, the
 * expert-by-expert cosine similarity of the rows of H (eq 4), and the
 * activation counts n_j: the number of (calibration token, top-k slot) pairs
 * routed to expert j, top-k by logit with ties to the lower index (eq 5).
 * H is never stored: the Gram matrix H H^T is accumulated from it chunk by
 * chunk.  A row of zero norm has similarity 0 to the others and 1 to itself.
 * Host part: the greedy grouping of ordermoe_group_experts.
 *
 *   x_cal      dev  [T_cal][d] calibration tokens, storage `dtype`
 *   w_router   dev  [E][d] router weights W_r, storage `dtype`
 *   topk       k of the router (1 <= topk <= min(E, ORDERMOE_MAX_TOPK))
 *   theta      similarity threshold theta_l of the layer (eq 6)
 *   alpha_f    weight of the frequency in the importance (eq 28), alpha_r = 1 - alpha_f
 *   sim_dev    dev  [E][E] float, out: Sim_l
 *   counts_dev dev  [E] int64, out: n_j
 *   top1_dev   dev  [T_cal] int32, out (may be NULL): the top-1 expert of each
 *              calibration token under the same rule -- the input of the
 *              transition estimate of eq (41)
 *   sim_host, counts_host  host, out: copies of the two (may be NULL)
 *   group_of   host [E] int32, out: group index of each expert (groups are
 *              numbered in the order their dominant expert was chosen)
 *   centres    host [E] int32, out: dominant expert of each group, -1 padded
 *   num_groups host int32, out: K_l
 *   importance host [E] double, out: I_j (eq 28)
 * Requires d % 64 == 0, 1 <= E <= 128, T_cal >= 1.
 * Synchronises `stream` (the grouping runs on the host).
 */
size_t ordermoe_similarity_workspace_size(int64_t T_cal, int32_t d, int32_t E);
int ordermoe_build_similarity(const void* x_cal, int64_t T_cal, int32_t d, const void* w_router,
                              int32_t E, int32_t dtype, int32_t topk, float theta, double alpha_f,
                              float* sim_dev, int64_t* counts_dev, int32_t* top1_dev,
                              float* sim_host,
                              int64_t* counts_host, int32_t* group_of, int32_t* centres,
                              int32_t* num_groups, double* importance, void* ws, size_t ws_bytes,
                              void* stream);

/* Greedy representative cover and importance (eq 24-28), host only.
 * Experts are visited in decreasing count (ties: lower index); an expert whose
 * largest similarity to the existing dominant experts is below theta starts a
 * new group, otherwise it joins the most similar dominant expert (ties: the one
 * chosen first).  rho_j is the mean similarity of j to its group (j included),
 * I_j = alpha_f * n_j / sum(n) + (1 - alpha_f) * rho_j.
 *   sim host [E][E] float, counts host [E] int64; outputs as above. */
int ordermoe_group_experts(int32_t E, const float* sim, const int64_t* counts, float theta,
                           double alpha_f, int32_t* group_of, int32_t* centres,
                           int32_t* num_groups, double* importance);

/* ------------------------------------------------------------------------
 * Deployment (Section IV-B, IV-C; Algorithm 1, deployment parts), host only.
 *
 * Mandatory part per layer: experts in non-increasing memory demand (ties:
 * lower index) go to the memory-feasible server (eq 29) of least
 *   Score = lambda1 * b_m / C_m + (1 - lambda1) * eta_m        (eq 30-31)
 * (ties: lower server), eta_m being the expert's group-mates already on m.
 * Experts that fit nowhere wait and are placed after the layer on the server
 * with the most remaining memory (ties: lower server) -- this can exceed C_m
 * when memory is fragmented, exactly as the algorithm states; used_out shows it.
 * Redundant part (if `redundancy`), over all layers: repeatedly the replica
 * of largest positive benefit pi_m I_j (1 - y_{m,l,g(j)}) / p_j that fits
 * (eq 32-35; ties: lower (layer, server, expert)).  redundancy = 2 drops the
 * group-coverage factor, B = pi_m w_j / p_j with w the given per-expert
 * weights: with activation frequencies as w this is the paper's
 * Popularity-based Replication baseline (Section VI-A).
 *
 *   N layers; E_l host [N] experts per layer; M servers (<= ORDERMOE_MAX_SERVERS)
 *   group_of, importance, p   host, concatenated over layers (sum E_l entries)
 *   C host [M] capacities, pi host [M] trajectory shares pi_m
 *   x_out host uint8, concatenated over layers of [M][E_l]: x_{m,l,j}
 *   used_out host [M]: b_m after placement
 * Returns ORDERMOE_ECAPACITY if sum(p) > sum(C) (nothing written).
 */
int ordermoe_place(int32_t N, const int32_t* E_l, int32_t M, const int32_t* group_of,
                   const double* importance, const double* p, const double* C, const double* pi,
                   double lambda1, int32_t redundancy, uint8_t* x_out, double* used_out);

/* ------------------------------------------------------------------------
 * Decision tables of one layer (host only).
 *
 *   t1: for each target r the feasible substitutes R_{l,r} (eq 7): the
 *       experts k != r of r's group with Sim(r,k) >= theta (fp32 compare),
 *       with Q(r,k) = fp32((1 - Sim(r,k)) * 0.5) (eq 18, phi = identity),
 *       sorted by (Q, k); t1_n[r] entries are used, the rest are padded with
 *       k = -1, Q = +inf.
 *   srvmask[j]: bit m set iff x[m][j] = 1.
 *   S[s][m][k] = fp32( omega_T * d(m,k|s) / d_ref + phi[m][k] ) with
 *       d(m,k|s) = [s != m] (z_bits / B[s][m] + tau[s][m]) + c[k] / F[m]
 *       (eq 37-38, without the token-dependent quality term), evaluated in
 *       double in that order and rounded once.  phi may be NULL (no look-ahead).
 *   gmax: row length of t1 (1..ORDERMOE_MAX_SUBS).
 * Errors: EINVAL if an expert is deployed on no server (eq 2) or a target has
 * more than gmax substitutes.
 */
int ordermoe_build_tables(int32_t E, int32_t M, const float* sim, const int32_t* group_of,
                          float theta, const uint8_t* x, const double* B, const double* tau,
                          const double* F, double z_bits, const double* c, double d_ref,
                          double omega_T, const double* phi, int32_t gmax, int32_t* t1_k,
                          float* t1_q, int32_t* t1_n, uint32_t* srvmask, float* S);

/* Look-ahead cost-to-go Phi_l^{(H-1)} for every layer of a stack (eq 41-42),
 * host only, double precision.
 *   Phi_l^{(h)}(m,k) = sum_k' P_l[k][k'] * V_{l+1}^{(h)}(m, k'),
 *   V_{l+1}^{(h)}(m,k') = min over the candidates (m',k'') of target k' at
 *       layer l+1 of omega_T d_{l+1}(m',k''|m)/d_ref_{l+1}
 *       + omega_Q Q_{l+1}(k',k'')/Qbar + Phi_{l+1}^{(h-1)}(m',k'')
 * with Phi^{(0)} = 0 and 0 for the last layer.  The candidate sets drop the
 * budget test; with pin_local_exact a target deployed on m is kept on m;
 * allow_sub: 0 exact only, 1 substitutes on any server, 2 substitutes only on
 * the source server m.
 *   N layers of E experts each (same E for all layers), M servers.
 *   P host [N-1][E][E] transition probabilities (rows may be all zero),
 *   x host [N][M][E], sim host [N][E][E] float, group_of host [N][E],
 *   theta host [N], z_bits host [N], c host [N][E], d_ref host [N],
 *   B, tau host [M][M], F host [M]; phi_out host [N][M][E].
 */
int ordermoe_build_lookahead(int32_t N, int32_t E, int32_t M, int32_t H, const double* P,
                             const uint8_t* x, const float* sim, const int32_t* group_of,
                             const float* theta, const double* z_bits, const double* c,
                             const double* d_ref, const double* B, const double* tau,
                             const double* F, double omega_T, double omega_Q, float Qbar,
                             int32_t pin_local_exact, int32_t allow_sub, double* phi_out);

/* The same Phi on the device (eq 41-42): every array is device memory with
 * the layout of ordermoe_build_lookahead, and the result equals that host
 * routine's bit for bit (the candidate costs are formed in the same fp64
 * operations and order, each Phi entry is summed in target order).
 *   ws: device workspace of ordermoe_lookahead_device_workspace_size(N, E, M)
 *   bytes; phi_out and ws are written, all inputs are only read.  The work
 *   is ordered on `stream` (a hipStream_t); the call does not synchronise.
 *   EINVAL for bad sizes or null pointers, EWORKSPACE for a short workspace. */
size_t ordermoe_lookahead_device_workspace_size(int32_t N, int32_t E, int32_t M);
int ordermoe_build_lookahead_device(int32_t N, int32_t E, int32_t M, int32_t H, const double* P,
                                    const uint8_t* x, const float* sim, const int32_t* group_of,
                                    const float* theta, const double* z_bits, const double* c,
                                    const double* d_ref, const double* B, const double* tau,
                                    const double* F, double omega_T, double omega_Q, float Qbar,
                                    int32_t pin_local_exact, int32_t allow_sub, double* phi_out,
                                    void* ws, size_t ws_bytes, void* stream);

/* The paper's Random Deployment baseline (Section VI-A), host only: every
 * expert once, layer by layer in index order, on a server drawn uniformly
 * from the memory-feasible ones (none: the server with the most remaining
 * memory, ties to the lower index); then, if `redundancy`, every (layer,
 * server, expert) without a copy, in an order shuffled by Fisher-Yates, is
 * placed when it fits.  The draws come from SplitMix64 seeded with `seed`
 * (uniform integers below n as next() % n).  Same layouts as ordermoe_place;
 * ECAPACITY if sum(p) > sum(C), EINVAL for bad sizes or non-positive p, C. */
int ordermoe_place_random(int32_t N, const int32_t* E_l, int32_t M, const double* p, const double* C,
                          uint64_t seed, int32_t redundancy, uint8_t* x_out, double* used_out);

/* Transition probabilities between consecutive layers (eq 41), host only:
 * P_l[k][k'] = the share of the calibration tokens with top-1 expert k at
 * layer l whose top-1 expert at layer l+1 is k'; a row with no token is zero.
 *   N layers (>= 1) of E experts, T_cal tokens followed through the stack;
 *   top1 host [N][T_cal] int32 (from ordermoe_build_similarity's top1_dev of
 *   each layer; an entry outside [0, E) is an EINVAL error);
 *   P_out host [N-1][E][E] double (nothing is written when N = 1). */
int ordermoe_estimate_transitions(int32_t N, int32_t E, int64_t T_cal, const int32_t* top1,
                                  double* P_out);

/* The same transition probabilities on the device (eq 41): top1 device
 * [N][T_cal] int32 (entries outside [0, E) are not counted), P device
 * [N-1][E][E] double, equal to ordermoe_estimate_transitions' bit for bit
 * (integer counts, one fp64 division per entry).  ws: device workspace of
 * ordermoe_transitions_device_workspace_size(N, E) bytes.  Ordered on
 * `stream`; no synchronisation.  EINVAL for bad sizes or null pointers,
 * EWORKSPACE for a short workspace; nothing is written when N = 1. */
size_t ordermoe_transitions_device_workspace_size(int32_t N, int32_t E);
int ordermoe_estimate_transitions_device(int32_t N, int32_t E, int64_t T_cal, const int32_t* top1, double* P,
                                         void* ws, size_t ws_bytes, void* stream);

/* Similarity threshold of layer l (1-based) of an N-layer stack (eq 6):
 * theta_l = theta_min + (theta_max - theta_min) (N - l) / (N - 1), in double,
 * rounded to float.  N = 1, where eq 6 divides by zero, gives the midpoint.
 * EINVAL unless 1 <= l <= N and theta_min <= theta_max. */
int ordermoe_theta_layer(int32_t l, int32_t N, double theta_min, double theta_max, float* theta_out);

/* Weight adaptation of the runtime cost (Section V-D, eq 45), host only: one
 * update per observation window,
 *   omega_Q' = min(1, max(0, omega_Q + kappa (Q_bar - T_bar))),  omega_T' = 1 - omega_Q',
 * where T_bar is the window's average delay normalised by the delay of pure
 * exact execution on the same deployment and Q_bar its average budget
 * utilisation (accumulated loss over the per-token budget), both as in eq 23.
 *   omega_Q in [0, 1]; kappa >= 0 (the step size); T_bar, Q_bar >= 0, finite;
 *   omega_Q_out, omega_T_out host scalars.  EINVAL otherwise (nothing written). */
int ordermoe_adapt_weights(double omega_Q, double kappa, double T_bar, double Q_bar, double* omega_Q_out,
                           double* omega_T_out);

/* Delay, server workload and cross-server traffic of realized decisions
 * (Section III-C/D, eq 13-17; Section III-F, eq 22), host only.  The paper's
 * model has one execution server per token and layer; with top-k every
 * executed slot pays eq 15's compute c_k / F_m and, when its server m is not
 * the token's location s, the transfer z_l / B_{s,m} + tau_{s,m} of eq 13
 * (first layer, s = the access server) or eq 14.  After a layer the token
 * resides on slot 0's server (the return path is not modelled).  A token whose
 * location is >= M, or a slot whose server is >= M, executes nothing there.
 *   N layers, T tokens, k slots, M servers; E_l [N] experts per layer.
 *   loc0 [T] u8: access servers; exec_m [N][T][k] u8 and exec_k [N][T][k] i32:
 *   each layer's decisions (as ordermoe_route_select writes them);
 *   c [sum E_l] f64 FLOP per expert, layer-major; z_bits [N]; B, tau [M][M]
 *   row-major (bit/s, s); F [M] FLOP/s.
 *   Outputs (host, caller-owned): delay_out [T] seconds per token (eq 16-17:
 *   per-user delays are sums over the user's tokens); work_out [M] FLOP per
 *   server (eq 22); stats_out [4] = {transfers (distinct token-destination
 *   pairs per layer), traffic bytes (z_l / 8 per transfer), remote slots,
 *   executed slots}; loc_out [N][T] u8 (the location entering each layer) or
 *   null.  Sums run in the order layer, token, slot, in fp64.  EINVAL for
 *   bad sizes, an executed expert outside [0, E_l), F <= 0 or B <= 0 on a
 *   used link (nothing written). */
int ordermoe_simulate_delay(int32_t N, int64_t T, int32_t k, int32_t M, const int32_t* E_l,
                            const uint8_t* loc0, const uint8_t* exec_m, const int32_t* exec_k,
                            const double* c, const double* z_bits, const double* B, const double* tau,
                            const double* F, double* delay_out, double* work_out, double* stats_out,
                            uint8_t* loc_out);

/* ------------------------------------------------------------------------
 * Routing and server-expert selection of one layer (Section V, the per-layer
 * loop of Algorithm 2 for every token of a batch), on the device.
 *
 * Router: logits l = x W_r^T in fp32 (bf16 inputs: exact products, fp32
 * accumulation; fp32 inputs: fp64 accumulation rounded to fp32); top-k by
 * logit, ties to the lower index; gate weight = softmax probability
 * renormalised over the top-k (renorm = 1) or over all E (renorm = 0);
 * margin = smallest gap between adjacent sorted top-(k+1) logits (top-k when
 * k = E); flag = margin < ORDERMOE_MARGIN_FLAG.
 *
 * Selection, per token, slots in rank order, sharing the token's budget:
 *   r = routed target, s = loc_in[token], Qh = running accumulated loss;
 *   if pin_local_exact and r is deployed on s: (s, r), Q = 0;
 *   else argmin over the candidates of eq (40) -- (m, r) for every server m
 *   holding r, and (m, k) for k in t1[r] held by m with fp32 Qh + Q <= Qbar
 *   (only if allow_sub and Qbar > 0; allow_sub = 2 keeps only substitutes held by
 *   s, the paper's Local Substitute Only baseline) -- of J = fmaf(omega_Q/Qbar, Q, S[s][m][k])
 *   (eq 43), ties by (Q, exact first, k, local first, m); then Qh += Q (eq 44).
 *   The token resides after the layer on slot 0's execution server.
 * Dispatch list: every (token, slot) whose execution server differs from
 * loc_in, as token * k + slot, ordered by (destination, token, slot);
 * dst_count[m] entries go to server m.
 */
typedef struct {
    int32_t dtype;          /* storage of x and w_router */
    int32_t d, E, k, M;     /* hidden size, experts, top-k, servers */
    int32_t gmax;           /* row length of the t1 tables */
    int32_t pin_local_exact, allow_sub, renorm;
    float Qbar;             /* per-token budget (eq 39) */
    float omega_Q;          /* weight of the quality term (eq 38) */
    const void* w_router;   /* dev [E][d] */
    const int32_t* t1_k;    /* dev [E][gmax] */
    const float* t1_q;      /* dev [E][gmax] */
    const int32_t* t1_n;    /* dev [E] */
    const uint32_t* srvmask;/* dev [E] */
    const float* S;         /* dev [M][M][E] */
} ordermoe_layer;

typedef struct {
    int32_t* idx;        /* dev [T][k] routed targets in rank order */
    float* w;            /* dev [T][k] gate weights */
    float* margin;       /* dev [T] */
    uint8_t* flag;       /* dev [T] 1 if margin < ORDERMOE_MARGIN_FLAG */
    int32_t* exec_k;     /* dev [T][k] executed expert k* */
    uint8_t* exec_m;     /* dev [T][k] execution server m* */
    uint8_t* cls;        /* dev [T][k] ORDERMOE_LOCAL_EXACT .. ORDERMOE_REMOTE_SUB */
    float* qhat_out;     /* dev [T] accumulated loss after the layer */
    uint8_t* loc_out;    /* dev [T] location after the layer */
    int32_t* dispatch;   /* dev [T*k] (only the first counters[REMOTE_SLOTS] are written) */
    int32_t* dst_count;  /* dev [M] */
    int64_t* counters;   /* dev [ORDERMOE_NUM_COUNTERS] */
} ordermoe_route_out;

/* Requirements: d % 64 == 0; 1 <= E <= ORDERMOE_MAX_EXPERTS;
 * 1 <= k <= min(E, ORDERMOE_MAX_TOPK); 1 <= M <= ORDERMOE_MAX_SERVERS;
 * 1 <= gmax <= ORDERMOE_MAX_SUBS; T >= 0 (T = 0 writes zero counters only).
 * A token whose loc_in is not below M is not routed to any server: its slots
 * get exec_k = -1, exec_m = 255, cls = 255, it enters no list and is counted
 * in counters[ORDERMOE_CNT_INVALID].
 * Tables must come from ordermoe_build_tables for the same (E, M). */
size_t ordermoe_route_workspace_size(int64_t T, int32_t k, int32_t M);
int ordermoe_route_select(const ordermoe_layer* L, const void* x, int64_t T,
                          const uint8_t* loc_in, const float* qhat_in,
                          const ordermoe_route_out* out, void* ws, size_t ws_bytes, void* stream);

/* ordermoe_route_select for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results, with the workspace taken from a
 * fixed scratch array of ORDERMOE_NOALLOC_SCRATCH_BYTES in device memory that
 * the library holds on each GPU it runs on until the process ends.  The call
 * allocates and frees nothing.  Batches whose
 * ordermoe_route_workspace_size(T, k, M) exceeds the scratch return
 * ORDERMOE_EWORKSPACE before any launch.  Every call on one GPU uses that GPU's
 * one scratch array: calls whose device work overlaps (other streams, other
 * threads) race and must be ordered by the caller.  The scratch is rewritten
 * before it is read on every call, so nothing needs clearing between calls. */
#define ORDERMOE_NOALLOC_SCRATCH_BYTES (8u << 20)
int ordermoe_route_select_noalloc(const ordermoe_layer* L, const void* x, int64_t T,
                                  const uint8_t* loc_in, const float* qhat_in,
                                  const ordermoe_route_out* out, void* stream);

/* ------------------------------------------------------------------------
 * Local MoE execution on one server.
 *
 * For server `server`, every (token, slot) with exec_m == server is executed
 * by expert exec_k with its gate weight; slots of one token that selected the
 * same expert are merged into one row whose weight is the sum of their gate
 * weights (fp32, slot order).  Tokens residing on `server` (loc_in) also run
 * the always-local shared experts with weight 1; the shared experts are
 * executed as one FFN of width n_shared * f (their weights concatenated).
 *   y[t] = sum over t's rows of w_row * W_down (silu(W_gate x) * (W_up x))
 * with silu(a) = a / (1 + exp(-a)).  Tokens with no row get y = 0.
 * bf16: products exact, fp32 accumulation, the SwiGLU activation rounded to
 * bf16 before the down projection, each row's output rounded to bf16, rows
 * summed in fp32 and y rounded to bf16.  fp32: fp32 throughout.
 */
typedef struct {
    int32_t dtype;               /* storage of weights, x and y */
    int32_t d, f, E;             /* hidden size, FFN width, routed experts in the layer */
    int32_t n_local;             /* routed experts held by this server (0..ORDERMOE_MAX_LOCAL) */
    int32_t n_shared;            /* shared experts (0 = none) */
    const int32_t* local_experts;/* host [n_local] expert ids, strictly increasing */
    const void* w_gate_up;       /* dev [n_local][2f][d] packed by ordermoe_pack_gate_up */
    const void* w_down;          /* dev [n_local][d][f] packed by ordermoe_pack_down */
    const void* w_shared_gate_up;/* dev [2*n_shared*f][d] packed, or NULL if n_shared = 0 */
    const void* w_shared_down;   /* dev [d][n_shared*f] packed by ordermoe_pack_down (n = 1): the
                                    n_shared W_down side by side */
} ordermoe_experts;

/* Requirements: bf16 d % 256 == 0 and f % 128 == 0, fp32 d % 64 == 0 and
 * f % 32 == 0 (else ORDERMOE_EINVAL); weights, x and y 16-byte aligned;
 * T >= 0; 1 <= k <= ORDERMOE_MAX_TOPK.  Each operand the GEMMs read must span
 * fewer than 2^31 bytes (else ORDERMOE_EINVAL, and the workspace size is 0):
 * T*d, 2*f*d, 2*max(n_shared,1)*f*d and T*max(n_shared,1)*f elements times the
 * element size (bf16: T*d < 2^30 and T*f < 2^30, so at d = 4096 and
 * f = 14336 at most 74898 tokens per call).
 * w, exec_k, exec_m: dev [T][k] as written by ordermoe_route_select.
 * y: dev [T][d].  row_offsets: dev [n_local + 2] int32, out: start row of
 * each local expert, then of the shared rows, then the total row count.
 * ws: dev, at least ordermoe_forward_workspace_size(W, T, k) bytes (else
 * ORDERMOE_EWORKSPACE): row tables, the activations, the per-row outputs and,
 * for bf16 batches above 128 tokens, 64 MiB of fp32 partial tiles for GEMM
 * tiles split along K (summed in K order, so results are deterministic).  The
 * call uses it until the stream passes the call; calls in flight at the same
 * time need workspaces of their own. */
size_t ordermoe_forward_workspace_size(const ordermoe_experts* W, int64_t T, int32_t k);
int ordermoe_local_moe_forward(const ordermoe_experts* W, const void* x, int64_t T, int32_t k,
                               const float* w, const int32_t* exec_k, const uint8_t* exec_m,
                               const uint8_t* loc_in, int32_t server, void* y,
                               int32_t* row_offsets, void* ws, size_t ws_bytes, void* stream);

/* One-time weight packing for ordermoe_local_moe_forward (device, ordered on
 * `stream`; out must not overlap the inputs).  The FFN weights of eq (15)'s
 * experts in the torch Linear layout [out][in] go in; the forward reads only
 * the packed copies.
 *
 * ordermoe_pack_gate_up: w_gate, w_up: dev [n][f][d]; out: dev [n][2f][d]
 * holding, for every block b of 32 FFN columns, the gate rows [32b, 32b+32) as
 * rows [64b, 64b+32) and the matching up rows as rows [64b+32, 64b+64).
 * ordermoe_pack_down: w_down: dev [n][d][f]; out: dev [n][d][f].
 * fp32: the rows of each expert's matrix stay in row order.  bf16: each
 * expert's matrix [N][K] (gate/up N = 2f, K = d; down N = d, K = f) is stored
 * tile-blocked as [N/256][K/64][256][64], element (r, c) at
 * ((r/256) (K/64) + c/64) 16384 + (r%256) 64 + c%64: the 256 rows of one
 * 64-deep K step of a GEMM tile are one contiguous 32 KB block.
 * Requires gate/up f % 32 == 0 and d % 8 == 0 (bf16: f % 128 == 0 and
 * d % 64 == 0), down f % 8 == 0 (bf16: d % 256 == 0 and f % 64 == 0), and
 * 16-byte aligned pointers; else ORDERMOE_EINVAL. */
int ordermoe_pack_gate_up(int32_t dtype, int32_t n, int32_t f, int32_t d, const void* w_gate,
                          const void* w_up, void* out, void* stream);
int ordermoe_pack_down(int32_t dtype, int32_t n, int32_t d, int32_t f, const void* w_down, void* out,
                       void* stream);

/* ------------------------------------------------------------------------
 * Kernel timing (measurement support, off by default).
 *
 * While enabled, every kernel launched by the entry points above is bracketed
 * by two HIP events recorded on the caller's stream.  ordermoe_timing_read
 * waits for the recorded events, then reports for each kernel name the total
 * elapsed milliseconds and the number of launches since the last reset.
 *   names     host [max_entries][ORDERMOE_TIMING_NAME] char, NUL-terminated
 *   total_ms  host [max_entries], launches host [max_entries]
 *   n_entries host, out: number of kernel names recorded (may exceed max_entries)
 *   reset     non-zero: clear the totals after reading
 */
#define ORDERMOE_TIMING_NAME 64
int ordermoe_timing_enable(int32_t on);
int ordermoe_timing_read(int32_t max_entries, char* names, double* total_ms, int64_t* launches,
                         int32_t* n_entries, int32_t reset);

#ifdef __cplusplus
}
#endif

#endif /* ORDERMOE_H */
