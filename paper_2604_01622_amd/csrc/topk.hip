// Expert-choice selection (Section 2.2, T_j = TopC_i(S_ij); the pool of each
// expert is one sequence, Section 5.2): for every (group g, expert j) the k_g
// tokens of the group with the largest score, equal scores going to the lower
// token index, emitted in ascending token order.
//
// One workgroup per (group, expert) column of ST (contiguous).  The scores are
// mapped to order-preserving uint32 keys and the k-th largest key is found by
// a 4-pass 8-bit radix select with an LDS histogram (integer counts, so the
// result does not depend on the order of the LDS atomics).  A final pass in
// token order keeps every key above the threshold plus the first (k - #above)
// keys equal to it, and compacts them with two block-wide prefix sums.
#include "ec_common.h"
#include "ec_kernels.h"

namespace ec {

namespace {

constexpr int TK_THREADS = 256;
constexpr int TK_IPT = 8;                         // tokens per thread in the compaction pass
constexpr int TK_TILE = TK_THREADS * TK_IPT;
constexpr int TK_MAX_CACHED = 12288;              // column length kept in LDS (48 KiB)

__device__ __forceinline__ float key_to_f32(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k ^ 0x80000000u) : ~k);
}

// Exclusive prefix sum over the workgroup; *total receives the sum.
__device__ __forceinline__ int block_excl_scan(int v, int* sbuf, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sbuf[wave] = x;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < TK_THREADS / 64; ++w) {
    const int s = sbuf[w];
    before += (w < wave) ? s : 0;
    tot += s;
  }
  *total = tot;
  return before + x - v;
}

template <bool CACHED>
__global__ __launch_bounds__(TK_THREADS) void topk_kernel(const float* __restrict__ ST, int N,
                                                          int E, int K, GroupTable tab,
                                                          int32_t* __restrict__ sel_token,
                                                          float* __restrict__ sel_gate,
                                                          int32_t* __restrict__ slotT) {
  extern __shared__ uint32_t skeys[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_digit, s_kleft;
  __shared__ int sbuf0[TK_THREADS / 64], sbuf1[TK_THREADS / 64];

  const int j = blockIdx.x;
  const int gi = blockIdx.y;
  const int off = tab.off[gi], L = tab.len[gi], k = tab.k[gi], seg = tab.seg[gi];
  const int tid = threadIdx.x;
  const float* col = ST + (size_t)j * N + off;

  if (CACHED) {
    for (int i = tid; i < L; i += TK_THREADS) skeys[i] = f32_order_key(col[i]);
    __syncthreads();
  }

  // ---- radix select of the k-th largest key ----
  uint32_t prefix = 0, mask = 0;
  int kleft = k;
  if (k > 0) {
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      hist[tid] = 0;
      __syncthreads();
      for (int i = tid; i < L; i += TK_THREADS) {
        const uint32_t key = CACHED ? skeys[i] : f32_order_key(col[i]);
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid < 64) {
        // lane l owns digits 4l .. 4l+3; count the keys with a larger digit
        const uint32_t c0 = hist[4 * tid], c1 = hist[4 * tid + 1], c2 = hist[4 * tid + 2],
                       c3 = hist[4 * tid + 3];
        const uint32_t local = c0 + c1 + c2 + c3;
        uint32_t s = local;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t y = __shfl_down(s, o, 64);
          if (tid + o < 64) s += y;
        }
        const uint32_t above = s - local;  // keys whose digit is in a higher lane
        const uint32_t kl = (uint32_t)kleft;
        uint32_t gt = above;
        const uint32_t cnt[4] = {c3, c2, c1, c0};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (gt < kl && kl <= gt + cnt[q]) {
            s_digit = (uint32_t)(4 * tid + 3 - q);
            s_kleft = kl - gt;
          }
          gt += cnt[q];
        }
      }
      __syncthreads();
      prefix |= s_digit << shift;
      mask |= 255u << shift;
      kleft = (int)s_kleft;
      __syncthreads();
    }
  } else {
    prefix = 0xffffffffu;  // nothing is above it and no equal key is taken
  }
  const uint32_t thr = prefix;
  const int need_eq = (k > 0) ? kleft : 0;

  // ---- ordered compaction ----
  int eq_before = 0, sel_before = 0;
  int32_t* sel_row = sel_token + (size_t)j * K + seg;
  float* gate_row = sel_gate ? sel_gate + (size_t)j * K + seg : nullptr;
  int32_t* slot_row = slotT + (size_t)j * N + off;
  for (int t0 = 0; t0 < L; t0 += TK_TILE) {
    const int i0 = t0 + tid * TK_IPT;
    uint32_t keys[TK_IPT];
    int n_eq = 0, n_gt = 0;
#pragma unroll
    for (int q = 0; q < TK_IPT; ++q) {
      const int i = i0 + q;
      uint32_t key = 0;
      if (i < L) key = CACHED ? skeys[i] : f32_order_key(col[i]);
      keys[q] = key;
      n_gt += (i < L && key > thr);
      n_eq += (i < L && key == thr);
    }
    int tot_eq;
    const int eq_excl = block_excl_scan(n_eq, sbuf0, &tot_eq);
    int eq_rank = eq_before + eq_excl;
    uint32_t take = 0;
    int n_sel = 0;
#pragma unroll
    for (int q = 0; q < TK_IPT; ++q) {
      const int i = i0 + q;
      bool s = false;
      if (i < L) {
        if (keys[q] > thr) s = true;
        else if (keys[q] == thr) { s = eq_rank < need_eq; ++eq_rank; }
      }
      take |= (uint32_t)s << q;
      n_sel += s;
    }
    int tot_sel;
    const int sel_excl = block_excl_scan(n_sel, sbuf1, &tot_sel);
    int pos = sel_before + sel_excl;
#pragma unroll
    for (int q = 0; q < TK_IPT; ++q) {
      const int i = i0 + q;
      if (i < L) {
        if ((take & (1u << q)) && pos < k) {
          sel_row[pos] = off + i;
          if (gate_row) gate_row[pos] = key_to_f32(keys[q]);
          slot_row[i] = seg + pos;
          ++pos;
        } else {
          slot_row[i] = -1;
        }
      }
    }
    eq_before += tot_eq;
    sel_before += tot_sel;
    __syncthreads();  // sbuf reuse in the next tile
  }
}

}  // namespace

hipError_t launch_topk(const float* ST, int N, int E, int K, const GroupTable& tab,
                       int32_t* sel_token, float* sel_gate, int32_t* slotT, hipStream_t st) {
  if (tab.n == 0 || E == 0) return hipSuccess;
  int maxL = 0;
  for (int g = 0; g < tab.n; ++g) maxL = tab.len[g] > maxL ? tab.len[g] : maxL;
  const dim3 grid(E, tab.n);
  if (maxL <= TK_MAX_CACHED) {
    const size_t lds = (size_t)(maxL > 0 ? maxL : 1) * sizeof(uint32_t);
    topk_kernel<true><<<grid, TK_THREADS, lds, st>>>(ST, N, E, K, tab, sel_token, sel_gate, slotT);
  } else {
    topk_kernel<false><<<grid, TK_THREADS, 0, st>>>(ST, N, E, K, tab, sel_token, sel_gate, slotT);
  }
  return hipGetLastError();
}

}  // namespace ec
