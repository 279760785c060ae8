/*
 * ec_moe.h - C interface of the expert-choice (EC) mixture-of-experts layer
 * for AMD Instinct MI355X (gfx950).
 *
 * The layer (paper Section 2.2, "Expert-choice"; SwiGLU experts per Appendix E):
 *   S   = softmax(X Wg^T / tau) over the E experts, one row per token;
 *   T_gj = the k_g tokens of routing group g with the largest S[:, j]
 *          (equal scores: the lower token index wins), for every expert j;
 *   y_i = sum over experts j with i in T_gj of  S_ij * FFN_j(x_i),
 *   FFN_j(x) = W2_j (SiLU(W1_j x) * (W3_j x)),   y_i = 0 if no expert chose i.
 * A routing group is one sequence: every expert chooses from the tokens of the
 * same sequence (Section 5.2), and its capacity k_g may depend on the
 * sequence's mask ratio (Section 4.2): k_g = L_g c(t_g) / E, where c is the
 * average number of experts per token (Section 2.2 relates the two: E k = c L).
 *
 * Conventions for every entry point
 *  - Pointers are DEVICE pointers unless marked HOST.  Device buffers must be
 *    16-byte aligned.  All arrays are dense row-major with the shapes given.
 *  - Storage dtype (ec_problem.dtype) applies to X, Wg, W1, W3, W2, Y, dY, dX,
 *    dW1, dW3, dW2.  S, gates and dWg are always fp32; accumulation is fp32.
 *  - The caller owns every buffer (inputs, outputs, the saved activations and
 *    the workspace).  The library allocates no device memory and keeps no
 *    pointer to a caller's device buffer after returning.  Its only mutable
 *    state is per calling thread: the last error, and the host array of
 *    stage-timing events that ec_set_stage_events registers, which the library
 *    keeps (and records into on later calls) until ec_set_stage_events is
 *    called again on that thread; calls from different threads are independent.
 *  - Work is enqueued on `stream` and the call returns without waiting for it.
 *    Capacities and group offsets are HOST arrays so that planning needs no
 *    device synchronisation.
 *  - Every argument is validated before anything is enqueued; an invalid call
 *    returns a non-zero ec_status and enqueues nothing.  A failed launch
 *    returns EC_ERR_HIP.  ec_last_error() gives the detail of the most recent
 *    failure on the calling thread.  No function aborts or throws.
 *  - Results are deterministic: no floating-point atomics are used, so two
 *    calls with the same inputs give bitwise identical outputs.
 */
#ifndef EC_MOE_H
#define EC_MOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EC_OK = 0,
  EC_ERR_ARG = 1,        /* null pointer, bad enum, non-finite temperature      */
  EC_ERR_SHAPE = 2,      /* sizes out of range or inconsistent                  */
  EC_ERR_CAPACITY = 3,   /* some k_g < 0 or k_g > L_g                           */
  EC_ERR_DTYPE = 4,      /* unknown storage dtype                               */
  EC_ERR_ALIGN = 5,      /* a device pointer is not 16-byte aligned             */
  EC_ERR_WORKSPACE = 6,  /* workspace or saved buffer smaller than required     */
  EC_ERR_HIP = 7         /* a HIP launch or runtime call failed                 */
} ec_status;

typedef enum { EC_F32 = 0, EC_BF16 = 1 } ec_dtype;

/* Capacity schedulers s(r) of the paper's Table 1 (Appendix H for the
 * Gaussian, sigma = 0.22).  c(t) = clamp(c_min + (c_max - c_min) s(t), c_min, c_max). */
typedef enum {
  EC_SCHED_LINEAR = 0,        /* s(r) = r                    */
  EC_SCHED_LINEAR_REV = 1,    /* s(r) = 1 - r                */
  EC_SCHED_COSINE = 2,        /* s(r) = (1 - cos(pi r)) / 2  */
  EC_SCHED_COSINE_REV = 3,    /* s(r) = (1 + cos(pi r)) / 2  */
  EC_SCHED_GAUSSIAN = 4,      /* normalised Gaussian bump    */
  EC_SCHED_GAUSSIAN_REV = 5   /* 1 - normalised Gaussian     */
} ec_scheduler;

/* Problem description.  Limits: 1 <= E <= 256; d and h multiples of 64 with
 * 64 <= d, h <= 16384; 1 <= G; N = group_offsets[G] < 2^31; every expert
 * buffer within 2^31 elements: E * K_tot * 2 * max(d, h) < 2^31 (the backward's
 * [E, K_tot, 2h] buffer); E * N < 2^31; N * 2 * max(d, hs) < 2^31.            */
typedef struct {
  int64_t n_tokens;              /* N = sum of the group lengths                       */
  int32_t d_model;               /* d                                                  */
  int32_t n_experts;             /* E                                                  */
  int32_t d_ff;                  /* h, hidden width of each SwiGLU expert              */
  int32_t n_groups;              /* G routing groups (sequences)                       */
  const int32_t *group_offsets;  /* HOST [G+1]: group g = tokens [off[g], off[g+1]),
                                    off[0] = 0, non-decreasing, off[G] = N              */
  const int32_t *capacity;       /* HOST [G]: k_g tokens per expert in group g,
                                    0 <= k_g <= off[g+1] - off[g]                       */
  float inv_temperature;         /* 1/tau > 0; S = softmax(logits * inv_temperature)   */
  ec_dtype dtype;                /* storage dtype                                      */
  int32_t d_shared;              /* hidden width hs of the shared experts, 0 for none:
                                    n_s shared SwiGLU experts of width h_s are one
                                    SwiGLU of width hs = n_s h_s (hidden units side by
                                    side), applied to every token and added to y
                                    without a gate (Appendix D: shared experts process
                                    all tokens; Appendix E: 2 per layer).  0 or a
                                    multiple of 64 in [64, 16384].                      */
} ec_problem;

/* Byte offsets of the forward activations inside the `saved` buffer that
 * ec_moe_forward fills and ec_moe_backward reads (K = K_tot = sum_g k_g).
 * Expert j's rows of every [E, K, .] buffer are [j K, (j+1) K); inside them
 * group g's k_g tokens follow groups 0..g-1, in ascending token order.        */
typedef struct {
  size_t S;          /* fp32  [N, E]    router scores                          */
  size_t sel_token;  /* int32 [E, K]    selected token of each expert row       */
  size_t sel_gate;   /* fp32  [E, K]    its gate S[token, j]                    */
  size_t slot;       /* int32 [E, N]    [j, i]: row of token i in expert j's
                        buffer, or -1 if expert j did not select token i        */
  size_t Xe;         /* fp32 [E, K, d] gathered tokens (bf16: none, = total;
                        its products read the selected rows of X)               */
  size_t H1;         /* dtype [E, K, h] W1 projection                           */
  size_t H3;         /* dtype [E, K, h] W3 projection                           */
  size_t A;          /* dtype [E, K, h] gate * SiLU(H1) * H3                    */
  size_t O;          /* dtype [E, K, d] gate-weighted expert outputs A W2^T     */
  size_t Hs1;        /* dtype [N, hs]   shared experts' W1 projection           */
  size_t Hs3;        /* dtype [N, hs]   shared experts' W3 projection           */
  size_t As;         /* dtype [N, hs]   shared experts' SiLU(Hs1) * Hs3         */
  size_t total;      /* bytes of the whole buffer                               */
} ec_saved_layout;

/* Human-readable name of a status code (static string).                      */
const char *ec_status_string(int status);

/* Detail of the most recent failure on the calling thread ("" if none).      */
const char *ec_last_error(void);

/* K_tot = sum_g k_g after validating the problem; -1 on an invalid problem.  */
int64_t ec_total_capacity(const ec_problem *p);

/* Workspace bytes needed by
 *   mode 0: ec_route;
 *   mode 1: ec_moe_forward without a saved buffer (inference: the workspace
 *           then also holds the routing and expert activations);
 *   mode 2: ec_moe_backward;
 *   mode 3: ec_moe_forward with a saved buffer (training: the activations go
 *           to the saved buffer, so the workspace is much smaller).
 * 0 on an invalid problem or mode (see ec_last_error).                       */
size_t ec_workspace_size(const ec_problem *p, int mode);

/* Bytes of the saved buffer that ec_moe_forward fills for ec_moe_backward
 * (= ec_saved_layout.total).  0 on an invalid problem.                       */
size_t ec_saved_size(const ec_problem *p);

/* Layout of the saved buffer; returns an ec_status.                          */
int ec_saved_layout_of(const ec_problem *p, ec_saved_layout *out /* HOST */);

/* Capacity rule (Section 2.2 with Section 4.2's time-dependent capacity):
 *   k_g = clamp(rint(L_g * c_g / E), 0, L_g)  (rint: half to even, in double),
 *   c_g = c_fixed                                if t == NULL,
 *   c_g = clamp(c_min + (c_max - c_min) s(t_g), c_min, c_max) otherwise.
 * group_lengths, t and k_out are HOST arrays of length G.  Returns ec_status.  */
int ec_capacity(int32_t n_groups, const int32_t *group_lengths, int32_t n_experts,
                double c_fixed, const double *t, double c_min, double c_max,
                int scheduler, int32_t *k_out);

/* Routing only: the router GEMM + softmax and the per-(group, expert) column
 * top-k (Section 2.2; tie-break toward the lower token index; Section 5.2's
 * per-sequence pool).  Used for the retrofit's selection swap (Section 5).
 *   X  [N, d] dtype, Wg [E, d] dtype (row j = expert j's router vector)
 *   S  [N, E] fp32 out;  sel_token [E, K] int32 out;
 *   sel_gate [E, K] fp32 out, may be NULL (= S at the selected entries);
 *   slot [E, N] int32 out, may be NULL ([j, i] = row of token i in expert j's
 *   buffer, -1 if not selected).
 * ws: ec_workspace_size(p, 0) bytes.                                           */
int ec_route(const ec_problem *p, const void *X, const void *Wg, float *S,
             int32_t *sel_token, float *sel_gate, int32_t *slot,
             void *ws, size_t ws_bytes, hipStream_t stream);

/* Routing for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, outputs and errors as ec_route, without the workspace: its
 * scratch (the transposed scores, E N 4 bytes, and the slot map, another
 * E N 4 bytes, when slot is NULL) lives in a static device array of
 * EC_ROUTE_NOALLOC_MAX_BYTES that the library holds on every GPU it runs on
 * until the process ends; the call allocates nothing and enqueues no memset.
 * A problem needing more scratch than that returns EC_ERR_WORKSPACE before
 * anything is enqueued.  Every call on one GPU shares that GPU's array: calls
 * that overlap on one GPU (on different streams, or from different threads
 * without ordering) race and give undefined results; calls ordered on one
 * stream are safe.  The first call on a device looks up the array's address
 * (hipGetSymbolAddress) with that device current.                           */
#define EC_ROUTE_NOALLOC_MAX_BYTES ((size_t)16 << 20)
int ec_route_noalloc(const ec_problem *p, const void *X, const void *Wg, float *S,
                     int32_t *sel_token, float *sel_gate, int32_t *slot,
                     hipStream_t stream);

/* Token drop statistic (Appendix D: the fraction of tokens that no routed
 * expert chose, whose layer output is therefore zero).  Reads a slot map as
 * written by ec_route or kept in the saved buffer:
 *   slot [E, N] int32 ([j, i] = row of token i in expert j's buffer or -1);
 *   experts_per_token [N] int32 out: number of experts that chose token i;
 *   dropped [G] int32 out: number of tokens of group g that no expert chose.
 * Exact integer counts; no workspace.  slot and experts_per_token may be NULL
 * only when N = 0.                                                            */
int ec_token_coverage(const ec_problem *p, const int32_t *slot,
                      int32_t *experts_per_token, int32_t *dropped,
                      hipStream_t stream);

/* Layer forward: routing, gather, SwiGLU experts as a grouped GEMM, and the
 * gate-weighted combine (Section 2.2, Appendix E), plus the shared experts'
 * FFN of every token when p->d_shared > 0.
 *   W1, W3 [E, h, d] dtype;  W2 [E, d, h] dtype;
 *   Ws1, Ws3 [hs, d] dtype;  Ws2 [d, hs] dtype (NULL when d_shared = 0);
 *   Y [N, d] dtype out.
 * saved: NULL for inference, else ec_saved_size(p) bytes that receive the
 * activations the backward needs.  ws: ec_workspace_size(p, 1) bytes without a
 * saved buffer, ec_workspace_size(p, 3) with one.                              */
int ec_moe_forward(const ec_problem *p, const void *X, const void *Wg,
                   const void *W1, const void *W3, const void *W2,
                   const void *Ws1, const void *Ws3, const void *Ws2, void *Y,
                   void *saved, size_t saved_bytes,
                   void *ws, size_t ws_bytes, hipStream_t stream);

/* Layer backward: gradients of sum(Y * dY) with the selection held fixed (the
 * selection is an index set; gradient reaches the router through the gate
 * values S_ij of the selected pairs and the softmax).
 *   dY [N, d] dtype;  saved: filled by ec_moe_forward with the same inputs;
 *   dX [N, d] dtype out;  dWg [E, d] fp32 out;  dW1, dW3 [E, h, d] and
 *   dW2 [E, d, h] dtype out;  dWs1, dWs3 [hs, d] and dWs2 [d, hs] dtype out
 *   (NULL when d_shared = 0).  Outputs are overwritten, not accumulated.
 * ws: ec_workspace_size(p, 2) bytes.                                           */
int ec_moe_backward(const ec_problem *p, const void *X, const void *Wg,
                    const void *W1, const void *W3, const void *W2,
                    const void *Ws1, const void *Ws3, const void *Ws2,
                    const void *dY, const void *saved, size_t saved_bytes,
                    void *dX, float *dWg, void *dW1, void *dW3, void *dW2,
                    void *dWs1, void *dWs3, void *dWs2,
                    void *ws, size_t ws_bytes, hipStream_t stream);

/* ---- Token choice (Section 2.2), the policy expert choice is compared with,
 * on the same kernels.  Every token takes the top_k experts of its row of S
 * (equal scores: the lower expert index) with gates normalised over those k
 * experts, g_ij = S_ij / sum of the k chosen S_ij'; expert j keeps at most
 * p->capacity[g] of the tokens of group g that chose it, the lowest token
 * indices first; the other pairs are dropped (their gate weight is lost, not
 * renormalised).  Per-expert loads are data dependent: the kept pairs are
 * packed expert after expert, expert j's rows being
 * [expert_rows[j], expert_rows[j+1]), tokens ascending within each group.    */

/* TC capacity: cap_g = min(L_g, ceil(cf * top_k * L_g / E)); cf <= 0: no cap
 * (dropless, cap_g = L_g).  HOST arrays of length G.  Returns ec_status.      */
int ec_tc_capacity(int32_t n_groups, const int32_t *group_lengths, int32_t n_experts,
                   int32_t top_k, double cf, int32_t *cap_out);

/* Workspace bytes of ec_tc_route (mode 0) or ec_tc_forward (mode 1); 0 on an
 * invalid problem.                                                            */
size_t ec_tc_workspace_size(const ec_problem *p, int32_t top_k, int mode);

/* Token-choice routing: S [N, E] fp32 out; G [N, E] fp32 out, the gate of every
 * kept pair (0 for unchosen or dropped pairs); slot [E, N] int32 out, the
 * packed row of pair (j, i) or -1; expert_rows [E+1] int32 out;
 * sel_token [min(top_k N, E sum_g cap_g)] int32 out, the token of each packed
 * row (the first expert_rows[E] entries are written).  1 <= top_k <= E.      */
int ec_tc_route(const ec_problem *p, int32_t top_k, const void *X, const void *Wg,
                float *S, float *G, int32_t *slot, int32_t *expert_rows,
                int32_t *sel_token, void *ws, size_t ws_bytes, hipStream_t stream);

/* Token-choice layer forward (inference): y_i = sum over kept pairs of
 * g_ij FFN_j(x_i), plus the shared experts when p->d_shared > 0.  Weights as
 * for ec_moe_forward; expert_rows [E+1] int32 out, may be NULL.  The stage
 * events of ec_set_stage_events are those of ec_moe_forward.                */
int ec_tc_forward(const ec_problem *p, int32_t top_k, const void *X, const void *Wg,
                  const void *W1, const void *W3, const void *W2,
                  const void *Ws1, const void *Ws3, const void *Ws2, void *Y,
                  int32_t *expert_rows, void *ws, size_t ws_bytes, hipStream_t stream);

/* Stage timing for profiling.  After this call, every entry point called on
 * the same thread records events[0] on its stream before its first kernel and
 * events[s+1] after stage s, for s < n_events - 1, so that
 * hipEventElapsedTime(events[s], events[s+1]) is the duration of stage s.
 * The caller creates and owns the events; pass NULL / 0 to stop recording.
 * Stages of ec_moe_forward: 0 router+softmax, 1 top-k, 2 gather,
 *   3 W1/W3 grouped GEMM + SwiGLU, 4 W2 grouped GEMM, 5 shared W1/W3 + SwiGLU,
 *   6 shared W2, 7 combine (5 and 6 are empty without shared experts).
 * Stages of ec_moe_backward: 0 dY gather (empty for bf16: the dA product
 *   reads the selected rows itself), 1 dA grouped GEMM + SwiGLU backward + gate
 *   gradient partials, 2 dW2, 3 dXe, 4 dW1/dW3, 5 router dZ, 6 router dX,
 *   7 shared dA + SwiGLU backward, 8 shared dW2, 9 shared dX, 10 shared
 *   dW1/dW3 (7-10 empty without shared experts), 11 combine of dXe, 12 dWg.
 * Stages of ec_route: 0 router+softmax, 1 top-k.                              */
int ec_set_stage_events(hipEvent_t *events /* HOST array */, int n_events);

#ifdef __cplusplus
}
#endif

#endif /* EC_MOE_H */
