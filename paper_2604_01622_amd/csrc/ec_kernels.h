// Internal launchers of the expert-choice MoE kernels.  Each returns the
// hipError_t of its launch(es); all work goes on the given stream.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ec {

enum { DT_F32 = 0, DT_BF16 = 1 };

// Groups handled by one top-k launch (the table travels as a kernel argument).
constexpr int TOPK_MAX_GROUPS = 128;

struct GroupTable {
  int n;                            // groups in this launch
  int off[TOPK_MAX_GROUPS];         // first token of the group
  int len[TOPK_MAX_GROUPS];         // tokens in the group
  int k[TOPK_MAX_GROUPS];           // tokens each expert takes from the group
  int seg[TOPK_MAX_GROUPS];         // first row of the group's segment in an expert buffer
};

// S [N,E] and ST [E,N] fp32 from X [N,d] and Wg [E,d].
hipError_t launch_router_softmax(int dtype, const void* X, const void* Wg, float* S, float* ST,
                                 int N, int d, int E, float inv_tau, hipStream_t st);

// Column top-k of ST per (group, expert): sel_token/sel_gate [E,K], slotT [E,N].
hipError_t launch_topk(const float* ST, int N, int E, int K, const GroupTable& tab,
                       int32_t* sel_token, float* sel_gate, int32_t* slotT, hipStream_t st);

// Xe[r, :] = X[sel_token[r], :] for all rows (with rows_dev: for r < *rows_dev,
// rows being an upper bound).
hipError_t launch_gather(int dtype, const void* X, const int32_t* sel_token, void* Xe,
                         long rows, int d, int N, hipStream_t st,
                         const int32_t* rows_dev = nullptr);

// Y[i, :] = Xr[i, :] (if Xr) + sum_j S[i,j] O[j kstride + slotT[j,i], :] over experts j
// with 0 <= slotT[j,i] < K (Xr may alias Y); kstride < 0 means K (one buffer of K
// rows per expert), 0 means slot holds rows of one packed buffer.
hipError_t launch_combine(int dtype, const void* O, const float* S, const int32_t* slotT,
                          const void* Xr, void* Y, int N, int E, int K, int d, hipStream_t st,
                          long kstride = -1);

// Backward combine: dX[i,:] = Xr[i,:] + sum_j dXe[j, slotT[j,i], :]  (Xr may alias dX).
hipError_t launch_bwd_combine(int dtype, const void* dXe, const int32_t* slotT, const void* Xr,
                              void* dX, int N, int E, int K, int d, hipStream_t st);

// Router backward, part 1: dZ = S * (dS - <S, dS>) / tau  [N,E] fp32, from
// S_ij dS_ij = sum over q of dsp[(j K + slot_ij) nparts + q] on the selection
// (0 elsewhere); dZb (optional) is a bf16 copy [N, EP] with zero columns E..EP-1.
hipError_t launch_router_dz(const float* S, const float* dsp, int nparts, const int32_t* slotT,
                            float* dZ, uint16_t* dZb, int N, int E, int EP, int K, float inv_tau,
                            hipStream_t st);

// Router backward, part 2: dX = dZ Wg  (bf16: dZ is the padded bf16 copy).
hipError_t launch_router_dx(int dtype, const void* dZ, const void* Wg, void* dX, int N, int E,
                            int EP, int d, hipStream_t st);

// Router backward, part 3: dWg [E,d] fp32 = dZ^T X, split over the tokens into
// `splits` partial sums (part [splits,E,d] fp32) added in a fixed order.
hipError_t launch_router_dwg(int dtype, const void* dZ, const void* X, float* dWg, float* part,
                             int splits, int N, int E, int EP, int d, hipStream_t st);
int router_dwg_splits(int N, int E, int d);

// ---- grouped GEMMs over E experts (M = K rows per expert) ----

// H = Xe W1^T, Xe W3^T -> A = SiLU(H1) * H3 (and H1, H3 if non-null).
// `shared`: the same product for the shared experts (own kernel symbol).
// rows (bf16 routed experts, may be null): Xe is then X itself and row m of
// expert e reads X[rows[e M + m]] (the gather happens in the operand load).
// gate (may be null): [E, M] fp32, row m of expert e is written as
// A = gate[e M + m] SiLU(H1) H3 (H1, H3 themselves unscaled).
hipError_t launch_gemm_w13(int dtype, const void* Xe, const void* W1, const void* W3, void* A,
                           void* H1, void* H3, int E, int M, int d, int h, hipStream_t st,
                           bool shared = false, const int32_t* rows = nullptr,
                           const float* gate = nullptr);
// O = A W2^T.
hipError_t launch_gemm_w2(int dtype, const void* A, const void* W2, void* O, int E, int M, int d,
                          int h, hipStream_t st, bool shared = false);
// dA = g dO W2 and the SwiGLU backward: dH[:, 0:h] = dH1, dH[:, h:2h] = dH3
// ([E,M,2h]), g = gate[e M + m] per row (1 when gate is null); W2 is read
// K-major.  dsp (may be null):
// [E M, dsp_parts(dtype, h)] fp32, per row and column block the sum of dA * A
// (A = SiLU(H1) H3), whose row sum is the gate's gradient times the gate when
// dO holds the rows of dY.  rows (bf16, may be null): dO is then dY itself and
// row m of expert e reads dY[rows[e M + m]].
hipError_t launch_gemm_dA(int dtype, const void* dO, const void* W2, const void* H1,
                          const void* H3, void* dH, int E, int M, int d, int h, hipStream_t st,
                          bool shared = false, float* dsp = nullptr, const int32_t* rows = nullptr,
                          const float* gate = nullptr);
// gate-gradient partials per row of the dA product (blocks of 128 columns of
// d_ff in bf16, 64 in fp32)
int dsp_parts(int dtype, int h);
// dXe = dH1 W1 + dH3 W3  ([E,M,d]).
// shared: dXe += dH1 W1 + dH3 W3 (the shared experts' term added to dX).
// The weights are read K-major (bf16: h a multiple of 64).
hipError_t launch_gemm_dXe(int dtype, const void* dH, const void* W1, const void* W3, void* dXe,
                           int E, int M, int d, int h, hipStream_t st, bool shared = false);
// dW2 = dO^T A  ([E,d,h]).  rows (bf16, may be null): dO is then dY itself and
// row m of expert e reads dY[rows[e M + m]] (the gather happens in the loads).
hipError_t launch_gemm_dW2(int dtype, const void* dO, const void* A, void* dW2, int E, int M,
                           int d, int h, hipStream_t st, const int32_t* rows = nullptr);
// dW1 = dH1^T Xe, dW3 = dH3^T Xe  ([E,h,d] each).  rows (bf16, may be null): Xe
// is then X itself and row m of expert e reads X[rows[e M + m]].
hipError_t launch_gemm_dW13(int dtype, const void* dH, const void* Xe, void* dW1, void* dW3,
                            int E, int M, int d, int h, hipStream_t st,
                            const int32_t* rows = nullptr);

// Token drop statistic: cnt[i] = #{j : slotT[j, i] >= 0} for i < N, then
// dropped[g] = #{i in group g : cnt[i] == 0} for the tab.n groups of the table.
hipError_t launch_coverage_count(const int32_t* slotT, int N, int E, int32_t* cnt,
                                 hipStream_t st);
hipError_t launch_coverage_drop(const int32_t* cnt, const GroupTable& tab, int32_t* dropped,
                                hipStream_t st);

// Shared experts' weight gradients (one batch of N rows, K-major operands):
// dW2 = dY^T A ([d,h]) and [dW1; dW3] = dH^T X ([h,d] each), split over the
// rows into `splits` fp32 partials (part: splits * max(d*h, 2*h*d) floats)
// added in a fixed order.
int wgrad_splits(int M, int N, int K);
hipError_t launch_shared_dW2(int dtype, const void* dY, const void* A, void* dW2, int N, int d,
                             int h, float* part, int splits, hipStream_t st);
hipError_t launch_shared_dW13(int dtype, const void* dH, const void* X, void* dW1, void* dW3,
                              int N, int d, int h, float* part, int splits, hipStream_t st);

// ---- token choice (the comparison policy): packed, data-dependent expert loads ----

// Row block of the grouped GEMMs (the tile tables of the packed buffers count
// ceil(M_e / TC_BM) row blocks per expert) and their column blocks.
constexpr int TC_BM = 256;
int tc_col_blocks_w13(int h);
int tc_col_blocks_w2(int d);
// G [N,E]: normalised gates of each token's top-k experts; flagT [E,N]: 1 if chosen.
hipError_t launch_tc_topk(const float* S, int N, int E, int k, float* G, int32_t* flagT,
                          hipStream_t st);
// cnt[(g0+g) E + j] = min(tokens of group g that chose j, cap_g) for the table's groups.
hipError_t launch_tc_count(const int32_t* flagT, int N, int E, const GroupTable& tab, int g0,
                           int32_t* cnt, hipStream_t st);
// Packed row offsets rows [E+1], per-(group, expert) row offsets seg [G,E] and the
// tile offsets of the two grouped products (tiles13, tiles2 [E+1]).
hipError_t launch_tc_offsets(const int32_t* cnt, int G, int E, int bm, int nt13, int nt2,
                             int32_t* rows, int32_t* seg, int32_t* tiles13, int32_t* tiles2,
                             hipStream_t st);
// slotT: choice flags in, packed rows (-1: not kept) out; sel[row] = token; G zeroed
// on dropped pairs.
hipError_t launch_tc_place(int32_t* slotT, float* G, int N, int E, const GroupTable& tab, int g0,
                           const int32_t* seg, int32_t* sel, hipStream_t st);
// The forward products over packed rows: expert e owns rows [rows[e], rows[e+1]).
// sel (bf16, may be null): Xe is then X itself and packed row r reads X[sel[r]].
hipError_t launch_gemm_w13_var(int dtype, const void* Xe, const void* W1, const void* W3, void* A,
                               int E, const int32_t* rows, const int32_t* tiles, long max_rows,
                               int max_rows_per_expert, int d, int h, hipStream_t st,
                               const int32_t* sel = nullptr);
hipError_t launch_gemm_w2_var(int dtype, const void* A, const void* W2, void* O, int E,
                              const int32_t* rows, const int32_t* tiles, long max_rows,
                              int max_rows_per_expert, int d, int h, hipStream_t st);

// Fill n int32/fp32/bytes with zero (a kernel, not a memset node).
hipError_t launch_zero(void* p, size_t bytes, hipStream_t st);


}  // namespace ec
