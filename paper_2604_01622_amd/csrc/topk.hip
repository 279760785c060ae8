// Expert-choice selection (Section 2.2, T_j = TopC_i(S_ij); the pool of each
// expert is one sequence, Section 5.2): for every (group g, expert j) the k_g
// tokens of the group with the largest score, equal scores going to the lower
// token index, emitted in ascending token order.  Scores are compared as
// order-preserving uint32 keys (larger float, larger key), so the selection is
// an integer computation.
//
// Columns of up to 4096 tokens (every sequence length of the workloads): 1, 4
// or 8 waves per (group, expert) column, 8 keys per lane held in registers
// (each wave a contiguous token range, token q*64 + lane of it in slot q, so
// loads and slot-map stores are coalesced).  The column's min and max skip the
// key bits every token shares; 8-bit radix passes over the next bits build a
// shared LDS histogram (integer counts: the result does not depend on the order
// of the LDS atomics) until the bucket holding the k-th largest key holds
// exactly the keys still needed, or every bit is resolved (exact ties).  The
// ordered compaction uses ballots within a wave and the lower waves' counts.
//
// Longer columns: one workgroup per column, the keys cached in LDS (up to 12288,
// else re-read), a 4-pass 8-bit radix select with a shared histogram, and an
// ordered compaction with two block-wide prefix sums.
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

// ------------------------------------------------------------- wave per column

// NW waves per column, KPL keys per lane: wave w holds the contiguous tokens
// [w KPL 64, (w+1) KPL 64), token (w KPL + q) 64 + lane in its slot q.
template <int KPL, int NW>
__global__ __launch_bounds__(64 * NW) void topk_col_kernel(const float* __restrict__ ST, int N,
                                                           int K, GroupTable tab,
                                                           int32_t* __restrict__ sel_token,
                                                           float* __restrict__ sel_gate,
                                                           int32_t* __restrict__ slotT) {
  // 256 digit bins, then one bin per lane index that takes the adds of keys
  // outside the current prefix (branch-free adds without conflicts)
  __shared__ __attribute__((aligned(16))) uint32_t hist[256 + 64];
  __shared__ uint32_t s_mn[NW], s_mx[NW], s_take[NW], s_eq[NW];
  const int j = blockIdx.x;
  const int gi = blockIdx.y;
  const int off = tab.off[gi], L = tab.len[gi], k = tab.k[gi], seg = tab.seg[gi];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (L <= 0) return;                             // an empty group selects nothing
  const float* col = ST + (size_t)j * N + off;
  const int t0 = wave * KPL * 64;                 // the wave's first token
  auto tok = [&](int q) { return t0 + q * 64 + lane; };

  // every load is issued unconditionally: a lane past the column's end reads its
  // last score, a duplicate that leaves the minimum and maximum unchanged
  uint32_t key[KPL];
#pragma unroll
  for (int q = 0; q < KPL; ++q) key[q] = f32_order_key(col[tok(q) < L ? tok(q) : L - 1]);

  // Selection: every valid key >= T; in the tie case (`ties`) the keys > T and
  // the first `need_eq` keys == T in token order.  k = 0 takes nothing.
  uint32_t T = 0u;
  bool ties = false;
  int need_eq = 0;
  if (k > 0 && k < L) {
    uint32_t mn = key[0], mx = key[0];
#pragma unroll
    for (int q = 1; q < KPL; ++q) {
      mn = key[q] < mn ? key[q] : mn;
      mx = key[q] > mx ? key[q] : mx;
    }
    wave_minmax_u32(mn, mx, &mn, &mx);
    if (t0 >= L) { mn = 0xffffffffu; mx = 0u; }   // a wave past the column: no keys
    if (lane == 0) { s_mn[wave] = mn; s_mx[wave] = mx; }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t a = s_mn[w], b = s_mx[w];
      mn = a < mn ? a : mn;
      mx = b > mx ? b : mx;
    }
    if (mn == mx) {                               // one value: the first k tokens
      T = mx; ties = true; need_eq = k;
    } else {
      int top = 32 - __clz(mn ^ mx);              // bits >= top are common to every key
      uint32_t hp = top >= 32 ? 0u : mx >> top;   // their value
      int kleft = k;
      for (;;) {
        const int w = top >= 8 ? 8 : top;         // digit width and shift
        const int s = top - w;
        const uint32_t dmask = (1u << w) - 1u;
        const uint32_t hmask = top >= 32 ? 0u : (0xffffffffu << top);
        const uint32_t hval = top >= 32 ? 0u : (hp << top);
        for (int b = tid; b < 256; b += 64 * NW) hist[b] = 0u;
        __syncthreads();
        uint32_t idx[KPL];                        // all bins first, then all adds
#pragma unroll
        for (int q = 0; q < KPL; ++q) {
          const bool in = (tok(q) < L) & ((key[q] & hmask) == hval);
          idx[q] = in ? (key[q] >> s) & dmask : 256u + lane;
        }
#pragma unroll
        for (int q = 0; q < KPL; ++q) atomicAdd(&hist[idx[q]], 1u);
        __syncthreads();
        // every wave finds the same digit: lane l owns digits 4l .. 4l+3; the
        // keys with a larger digit are those of the higher lanes and of the
        // lane's own higher digits
        const uint4 c = *reinterpret_cast<const uint4*>(&hist[4 * lane]);
        const uint32_t local = c.x + c.y + c.z + c.w;
        uint32_t gt = wave_excl_suffix_u32(local);
        const uint32_t kl = (uint32_t)kleft;
        int digit = -1;
        uint32_t above = 0, cnt = 0;
        const uint32_t cc[4] = {c.w, c.z, c.y, c.x};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (digit < 0 && gt < kl && kl <= gt + cc[q]) {
            digit = 4 * lane + 3 - q;
            above = gt;
            cnt = cc[q];
          }
          gt += cc[q];
        }
        const uint64_t who = __ballot(digit >= 0);   // exactly one lane
        const int src = __ffsll((unsigned long long)who) - 1;
        digit = __builtin_amdgcn_readlane(digit, src);
        above = __builtin_amdgcn_readlane(above, src);
        cnt = __builtin_amdgcn_readlane(cnt, src);
        __syncthreads();                          // the histogram is read before the next clear
        kleft -= (int)above;
        hp = (hp << w) | (uint32_t)digit;
        top = s;
        if ((int)cnt == kleft) {                  // the bucket's keys are exactly those needed
          T = hp << s;
          break;
        }
        if (s == 0) {                             // every bit resolved: equal keys, first kleft
          T = hp; ties = true; need_eq = kleft;
          break;
        }
      }
    }
  }

  // Ordered compaction.  Each wave counts its takes (and, for ties, its keys
  // equal to T), the counts of the lower waves give its first output position.
  int32_t* sel_row = sel_token + (size_t)j * K + seg;
  float* gate_row = sel_gate ? sel_gate + (size_t)j * K + seg : nullptr;
  int32_t* slot_row = slotT + (size_t)j * N + off;
  uint64_t eqm[KPL];
  uint32_t n_eq = 0;
  if (ties) {
#pragma unroll
    for (int q = 0; q < KPL; ++q) {
      eqm[q] = __ballot((tok(q) < L) & (key[q] == T));
      n_eq += __popcll(eqm[q]);
    }
    if (lane == 0) s_eq[wave] = n_eq;
    __syncthreads();
  }
  int eq_before = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) eq_before += (ties && w < wave) ? (int)s_eq[w] : 0;
  uint64_t tm[KPL];
  uint32_t n_take = 0;
#pragma unroll
  for (int q = 0; q < KPL; ++q) {
    bool take;
    if (!ties) {
      take = (tok(q) < L) & (k > 0) & (key[q] >= T);
    } else {
      const int eq_rank = __builtin_amdgcn_mbcnt_hi(
          (uint32_t)(eqm[q] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)eqm[q], eq_before));
      const bool eq = (tok(q) < L) & (key[q] == T);
      take = (tok(q) < L) & ((key[q] > T) | (eq & (eq_rank < need_eq)));
      eq_before += __popcll(eqm[q]);
    }
    tm[q] = __ballot(take);
    n_take += __popcll(tm[q]);
  }
  if (lane == 0) s_take[wave] = n_take;
  __syncthreads();
  int sel_before = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) sel_before += w < wave ? (int)s_take[w] : 0;
#pragma unroll
  for (int q = 0; q < KPL; ++q) {
    const int i = tok(q);
    const bool take = (tm[q] >> lane) & 1u;
    const int pos = __builtin_amdgcn_mbcnt_hi((uint32_t)(tm[q] >> 32),
                                              __builtin_amdgcn_mbcnt_lo((uint32_t)tm[q], sel_before));
    const bool put = take & (pos < k);
    if (put) {
      sel_row[pos] = off + i;
      if (gate_row) gate_row[pos] = key_to_f32(key[q]);
    }
    if (i < L) slot_row[i] = put ? seg + pos : -1;
    sel_before += __popcll(tm[q]);
  }
}

// ------------------------------------------------------------- workgroup per column

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
  if (maxL <= 512) {
    topk_col_kernel<8, 1><<<grid, 64, 0, st>>>(ST, N, K, tab, sel_token, sel_gate, slotT);
  } else if (maxL <= 2048) {
    topk_col_kernel<8, 4><<<grid, 256, 0, st>>>(ST, N, K, tab, sel_token, sel_gate, slotT);
  } else if (maxL <= 4096) {
    topk_col_kernel<8, 8><<<grid, 512, 0, st>>>(ST, N, K, tab, sel_token, sel_gate, slotT);
  } else if (maxL <= TK_MAX_CACHED) {
    const size_t lds = (size_t)(maxL > 0 ? maxL : 1) * sizeof(uint32_t);
    topk_kernel<true><<<grid, TK_THREADS, lds, st>>>(ST, N, E, K, tab, sel_token, sel_gate, slotT);
  } else {
    topk_kernel<false><<<grid, TK_THREADS, 0, st>>>(ST, N, E, K, tab, sel_token, sel_gate, slotT);
  }
  return hipGetLastError();
}

}  // namespace ec
