// Token-choice routing (Section 2.2, the policy expert choice is compared
// with): every token takes the top_k experts of its row of S (equal scores:
// the lower expert index), with gates normalised over those k experts; expert
// j keeps at most cap_g of the tokens of routing group g that chose it, the
// lowest token indices first, and drops the others.  Per-expert loads are
// data dependent, so the kept pairs are packed expert after expert into one
// buffer and the grouped GEMMs read a per-expert (row, tile) offset table
// from device memory.
#include "ec_common.h"
#include "ec_kernels.h"

namespace ec {

namespace {

constexpr int TC_TOK = 16;   // tokens per workgroup of the row top-k (one per 16-lane group)

// Row top-k of S [N, E] (E <= 256).  Sixteen lanes per token (four tokens per
// wave, sixteen per workgroup, so that several waves per SIMD hide the
// latency of the selection's dependent steps): lane r of a token's group holds
// experts r, r + 16, ...,
// r + 16 (NQ - 1); k rounds of an arg-max (larger score, then lower index) over
// the group, the lanes exchanging candidates within their 16-lane DPP row.
// G[i, j] = S_ij / (sum of the chosen scores) for chosen j, 0 elsewhere;
// flagT[j, i] = 1 if token i chose expert j, else 0 (transposed through LDS so
// that every expert row is written contiguously).
template <int NQ>
__global__ __launch_bounds__(256) void tc_topk_kernel(const float* __restrict__ S, int N, int E,
                                                      int k, float* __restrict__ G,
                                                      int32_t* __restrict__ flagT) {
  __shared__ uint8_t sflag[TC_TOK][256];
  const int tid = threadIdx.x, r = tid & 15, grp = tid >> 4;   // 16 groups of 16 lanes
  const int i0 = blockIdx.x * TC_TOK;
  constexpr int TPG = TC_TOK / 16;                 // tokens per lane group
  // every token's scores are loaded before the first selection
  float v[TPG][NQ];
#pragma unroll
  for (int u = 0; u < TPG; ++u) {
    const int i = i0 + grp + 16 * u;
    const int ii = i < N ? i : N - 1;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int j = r + 16 * q;
      v[u][q] = (j < E) ? S[(size_t)ii * E + j] : -INFINITY;
    }
  }
#pragma unroll
  for (int u = 0; u < TPG; ++u) {
    const int t = grp + 16 * u;
    const int i = i0 + t;
    if (i >= N) break;                              // uniform over the group
    uint32_t taken = 0u;                            // bit q: expert r + 16 q chosen
    float sum = 0.f;
    for (int c = 0; c < k; ++c) {
      float bv = -INFINITY;
      int bj = 0x7fffffff;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int j = r + 16 * q;
        if (j < E && !((taken >> q) & 1u) && (v[u][q] > bv || (v[u][q] == bv && j < bj))) {
          bv = v[u][q];
          bj = j;
        }
      }
      // all-reduce over the 16-lane row by DPP: rotations by 8 and 4, then the
      // quad exchanges (the comparison is commutative and associative)
      auto better = [&](float ov, int oj) {
        if (ov > bv || (ov == bv && oj < bj)) {
          bv = ov;
          bj = oj;
        }
      };
      better(dpp_f32<0x128>(bv), (int)dpp_u32<0x128>((uint32_t)bj));
      better(dpp_f32<0x124>(bv), (int)dpp_u32<0x124>((uint32_t)bj));
      better(dpp_f32<0x4E>(bv), (int)dpp_u32<0x4E>((uint32_t)bj));
      better(dpp_f32<0xB1>(bv), (int)dpp_u32<0xB1>((uint32_t)bj));
      if ((bj & 15) == r) taken |= 1u << (bj >> 4);
      sum += bv;
    }
    const float inv = 1.0f / sum;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int j = r + 16 * q;
      if (j < E) {
        const bool ch = (taken >> q) & 1u;
        G[(size_t)i * E + j] = ch ? v[u][q] * inv : 0.f;
        sflag[t][j] = ch ? 1 : 0;
      }
    }
  }
  __syncthreads();
  for (int c = tid; c < E * TC_TOK; c += 256) {
    const int j = c / TC_TOK, t = c % TC_TOK;
    if (i0 + t < N) flagT[(size_t)j * N + i0 + t] = sflag[t][j];
  }
}

__device__ __forceinline__ int block_sum_256(int v, int* red) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const int s = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return s;
}

// Kept pairs per (group, expert): cnt[(g0 + g) E + j] = min(#tokens of group g
// that chose j, cap_g).  One workgroup per (group of the table, expert).
__global__ __launch_bounds__(256) void tc_count_kernel(const int32_t* __restrict__ flagT, int N,
                                                       int E, GroupTable tab, int g0,
                                                       int32_t* __restrict__ cnt) {
  __shared__ int red[4];
  const int g = blockIdx.x / E, j = blockIdx.x % E;
  const int off = tab.off[g], len = tab.len[g];
  const int32_t* f = flagT + (size_t)j * N + off;
  int c = 0;
  for (int i = threadIdx.x; i < len; i += 256) c += f[i];
  c = block_sum_256(c, red);
  if (threadIdx.x == 0) cnt[(size_t)(g0 + g) * E + j] = c < tab.k[g] ? c : tab.k[g];
}

// Offsets, one workgroup (thread j for expert j, E <= 256): expert j's packed
// rows start at rows[j] (rows[E] = all kept pairs); group g's tokens in expert
// j start at seg[g E + j]; the tiles of the two grouped products start at
// tiles13[j] and tiles2[j] (ceil(M_j / bm) row blocks times nt13 / nt2).
__global__ __launch_bounds__(256) void tc_offsets_kernel(const int32_t* __restrict__ cnt, int G,
                                                         int E, int bm, int nt13, int nt2,
                                                         int32_t* __restrict__ rows,
                                                         int32_t* __restrict__ seg,
                                                         int32_t* __restrict__ tiles13,
                                                         int32_t* __restrict__ tiles2) {
  __shared__ int sm[256], st[256];
  const int j = threadIdx.x;
  int m = 0;
  if (j < E)
    for (int g = 0; g < G; ++g) m += cnt[(size_t)g * E + j];
  sm[j] = m;
  st[j] = (m + bm - 1) / bm;
  __syncthreads();
  if (j == 0) {   // E <= 256 sequential prefix sums
    int r = 0, tt = 0;
    for (int q = 0; q < E; ++q) {
      const int mq = sm[q], tq = st[q];
      sm[q] = r;
      st[q] = tt;
      r += mq;
      tt += tq;
    }
    rows[E] = r;
    tiles13[E] = tt * nt13;
    tiles2[E] = tt * nt2;
  }
  __syncthreads();
  if (j < E) {
    rows[j] = sm[j];
    tiles13[j] = st[j] * nt13;
    tiles2[j] = st[j] * nt2;
    int r = sm[j];
    for (int g = 0; g < G; ++g) {
      seg[(size_t)g * E + j] = r;
      r += cnt[(size_t)g * E + j];
    }
  }
}

// Placement, one workgroup per (group of the table, expert): the group's
// tokens that chose expert j, in ascending order; the first cap_g take rows
// seg + 0, 1, ... of the packed buffer (slotT[j, i] = row, sel[row] = i), the
// others are dropped (slotT = -1, G[i, j] = 0); tokens that did not choose j get
// slotT = -1.  slotT holds the choice flags on entry.
__global__ __launch_bounds__(256) void tc_place_kernel(int32_t* __restrict__ slotT,
                                                       float* __restrict__ G, int N, int E,
                                                       GroupTable tab, int g0,
                                                       const int32_t* __restrict__ seg,
                                                       int32_t* __restrict__ sel) {
  __shared__ int wsum[4];
  const int g = blockIdx.x / E, j = blockIdx.x % E;
  const int off = tab.off[g], len = tab.len[g], cap = tab.k[g];
  const int base_row = seg[(size_t)(g0 + g) * E + j];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int32_t* f = slotT + (size_t)j * N + off;
  int base = 0;
  for (int c0 = 0; c0 < len; c0 += 256) {
    const int i = c0 + threadIdx.x;
    const int flag = (i < len) ? f[i] : 0;
    // exclusive prefix of the flags inside the block
    const uint64_t bal = __ballot(flag != 0);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wave] = __popcll(bal);
    __syncthreads();
    int pre = 0;
    for (int w = 0; w < wave; ++w) pre += wsum[w];
    const int total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
    if (i < len) {
      const int pos = base + pre + before;
      if (flag && pos < cap) {
        const int row = base_row + pos;
        f[i] = row;
        sel[row] = off + i;
      } else {
        f[i] = -1;
        if (flag) G[(size_t)(off + i) * E + j] = 0.f;
      }
    }
    base += total;
  }
}

}  // namespace

hipError_t launch_tc_topk(const float* S, int N, int E, int k, float* G, int32_t* flagT,
                          hipStream_t st) {
  if (N == 0) return hipSuccess;
  const int grid = (N + TC_TOK - 1) / TC_TOK;
  if (E <= 64)
    tc_topk_kernel<4><<<grid, 256, 0, st>>>(S, N, E, k, G, flagT);
  else
    tc_topk_kernel<16><<<grid, 256, 0, st>>>(S, N, E, k, G, flagT);
  return hipGetLastError();
}

hipError_t launch_tc_count(const int32_t* flagT, int N, int E, const GroupTable& tab, int g0,
                           int32_t* cnt, hipStream_t st) {
  if (tab.n == 0) return hipSuccess;
  tc_count_kernel<<<tab.n * E, 256, 0, st>>>(flagT, N, E, tab, g0, cnt);
  return hipGetLastError();
}

hipError_t launch_tc_offsets(const int32_t* cnt, int G, int E, int bm, int nt13, int nt2,
                             int32_t* rows, int32_t* seg, int32_t* tiles13, int32_t* tiles2,
                             hipStream_t st) {
  tc_offsets_kernel<<<1, 256, 0, st>>>(cnt, G, E, bm, nt13, nt2, rows, seg, tiles13, tiles2);
  return hipGetLastError();
}

hipError_t launch_tc_place(int32_t* slotT, float* G, int N, int E, const GroupTable& tab, int g0,
                           const int32_t* seg, int32_t* sel, hipStream_t st) {
  if (tab.n == 0) return hipSuccess;
  tc_place_kernel<<<tab.n * E, 256, 0, st>>>(slotT, G, N, E, tab, g0, seg, sel);
  return hipGetLastError();
}

}  // namespace ec
