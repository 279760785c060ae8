// Router: logits Z = X Wg^T (Wg stored [E, d]) and S = softmax(Z / tau) over the
// experts of each token (the score matrix S of Section 2.2).  Writes S [N, E]
// and its transpose ST [E, N]; the column top-k reads ST so that each
// (group, expert) column is contiguous.
//
// bf16: one workgroup = 64 tokens, 4 groups of 16 tokens, each group split
// over KS waves that take disjoint K ranges.  Each wave streams its 16 token
// rows straight from HBM into MFMA A-fragments (every X element is used by
// exactly one wave, so it never touches LDS); the router matrix is staged
// through LDS in 64-wide K chunks (double buffered per split) and shared by the
// 4 groups.  v_mfma_f32_16x16x32_bf16 with fp32 accumulation; the splits are
// summed in a fixed order through LDS, then softmax in the epilogue with the 16
// lanes that hold one token's logits.
#include "ec_common.h"
#include "ec_kernels.h"

namespace ec {

namespace {

constexpr int RT_KC = 64;     // K chunk
constexpr int RT_LDK = RT_KC + 8;  // padded LDS row (bf16 elements)
constexpr int RT_PX = 4;      // X chunks in flight per wave

// A workgroup takes TG wave-rows of 16 tokens (TG = 4, or 1 when the tokens
// would not fill every CU with 4-row workgroups), each repeated KS times over
// disjoint K ranges, so that KS * TG waves stream X concurrently (more loads in
// flight per CU); fewer splits for many experts keep the router-matrix LDS
// tiles within 160 KiB.
template <int ET> struct RouterCfg { static constexpr int KS = ET <= 4 ? 4 : (ET <= 8 ? 2 : 1); };

template <int ET, int TG>
constexpr int router_lds_bytes() {
  constexpr int KS = RouterCfg<ET>::KS;
  constexpr int w = KS * 2 * ET * 16 * RT_LDK * 2;     // router tiles
  constexpr int r = KS > 1 ? KS * TG * 64 * ET * 4 * 4 : 0;   // split partial sums
  return w > r ? w : r;
}

template <int ET, int TG>
__global__ __launch_bounds__(64 * TG * RouterCfg<ET>::KS) void router_softmax_bf16_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wg, float* __restrict__ S,
    float* __restrict__ ST, int N, int d, int E, float inv_tau) {
  constexpr int EP = ET * 16;
  constexpr int KS = RouterCfg<ET>::KS;
  constexpr int NT = 64 * TG * KS;
  constexpr int RT_ROWS = 16 * TG;               // tokens per workgroup
  __shared__ __attribute__((aligned(16))) char smem[router_lds_bytes<ET, TG>()];
  __shared__ float sT[EP][RT_ROWS + 1];
  bf16_t* sW = reinterpret_cast<bf16_t*>(smem);   // [KS][2][EP * RT_LDK]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int tg = wave % TG, ks = wave / TG;     // token group, K split
  const int row0 = blockIdx.x * RT_ROWS;
  const int myrow = row0 + tg * 16 + (lane & 15);
  const int xrow = myrow < N ? myrow : N - 1;
  const bf16_t* xp = X + (size_t)xrow * d + (lane >> 4) * 16;
  const int nk = d / RT_KC;
  const int cps = (nk + KS - 1) / KS;            // chunks per split
  // chunk c of split q, or -1 past the split's share
  auto chunk_of = [&](int q, int i) { const int c = q * cps + i; return c < nk ? c : -1; };

  // router tiles of iteration i for every split: KS * EP rows x 8 chunks of 16 B
  constexpr int WPT = (KS * EP * 8 + NT - 1) / NT;
  auto load_w = [&](int i, uint4* regs) {
#pragma unroll
    for (int q = 0; q < WPT; ++q) {
      const int c = (tid + q * NT) % (KS * EP * 8);
      const int sp = c / (EP * 8), r = (c >> 3) % EP, ch = c & 7;
      const int kc = chunk_of(sp, i);
      const bool ok = r < E && kc >= 0;
      const uint4 v = *reinterpret_cast<const uint4*>(
          Wg + (size_t)(r < E ? r : E - 1) * d + (kc >= 0 ? kc : 0) * RT_KC + ch * 8);
      regs[q] = ok ? v : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_w = [&](int buf, const uint4* regs) {
#pragma unroll
    for (int q = 0; q < WPT; ++q) {
      const int c = tid + q * NT;
      if (c < KS * EP * 8) {
        const int sp = c / (EP * 8), r = (c >> 3) % EP, ch = c & 7;
        *reinterpret_cast<uint4*>(&sW[(sp * 2 + buf) * EP * RT_LDK + r * RT_LDK + ch * 8]) = regs[q];
      }
    }
  };
  auto load_x = [&](int i, uint4& a, uint4& b) {
    const int kc = chunk_of(ks, i);
    const bf16_t* q = xp + (kc >= 0 ? kc : 0) * RT_KC;
    a = *reinterpret_cast<const uint4*>(q);
    b = *reinterpret_cast<const uint4*>(q + 8);
  };

  f32x4 acc[ET];
#pragma unroll
  for (int t = 0; t < ET; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // X: a ring of RT_PX chunks per wave in registers, so RT_PX chunks of the
  // wave's rows are in flight; the ring index is static (the loop is unrolled by
  // RT_PX).  Router tiles: chunk i+1 goes to LDS at the start of iteration i
  // (its loads were issued an iteration earlier) and chunk i+2 is loaded.
  // X is the critical path: its ring is requested at once (the first router
  // tile just before it, so that its LDS store waits only for that tile's loads).
  uint4 wreg[WPT];
  load_w(0, wreg);
  uint4 xr[RT_PX][2];
#pragma unroll
  for (int u = 0; u < RT_PX; ++u) load_x(u, xr[u][0], xr[u][1]);
  store_w(0, wreg);
  load_w(1, wreg);
  __syncthreads();

  for (int i0 = 0; i0 < cps; i0 += RT_PX) {
#pragma unroll
    for (int u = 0; u < RT_PX; ++u) {
      const int i = i0 + u;
      if (i < cps) {                             // uniform over the workgroup
        const int buf = i & 1;
        if (i + 1 < cps) store_w(buf ^ 1, wreg); // chunk i+1; buffer last read in iteration i-1
        load_w(i + 2 < cps ? i + 2 : i, wreg);
        const bool live = chunk_of(ks, i) >= 0;
        const uint4 z = make_uint4(0, 0, 0, 0);
        const bf16x8 a0 = __builtin_bit_cast(bf16x8, live ? xr[u][0] : z);
        const bf16x8 a1 = __builtin_bit_cast(bf16x8, live ? xr[u][1] : z);
        load_x(i + RT_PX < cps ? i + RT_PX : i, xr[u][0], xr[u][1]);
        const bf16_t* sWb = &sW[(ks * 2 + buf) * EP * RT_LDK];
#pragma unroll
        for (int t = 0; t < ET; ++t) {
          const bf16_t* wp = &sWb[(t * 16 + (lane & 15)) * RT_LDK + (lane >> 4) * 16];
          const bf16x8 b0 = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(wp));
          const bf16x8 b1 = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(wp + 8));
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b0, acc[t], 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, acc[t], 0, 0, 0);
        }
        __syncthreads();
      }
    }
  }

  // sum the K splits of each token group (fixed order), in the lane layout of the
  // accumulators: lane holds tokens 4*(lane/16)+i of its 16, experts t*16 + lane%16
  if constexpr (KS > 1) {
    float* red = reinterpret_cast<float*>(smem);   // [KS][4 groups][64 lanes][ET][4]
#pragma unroll
    for (int t = 0; t < ET; ++t)
      *reinterpret_cast<f32x4*>(&red[(((ks * TG + tg) * 64 + lane) * ET + t) * 4]) = acc[t];
    __syncthreads();
    if (ks == 0) {
#pragma unroll
      for (int t = 0; t < ET; ++t) {
        f32x4 v = acc[t];
        for (int q = 1; q < KS; ++q)
          v += *reinterpret_cast<const f32x4*>(&red[(((q * TG + tg) * 64 + lane) * ET + t) * 4]);
        acc[t] = v;
      }
    }
  }

  if (ks == 0) {
    const int col = lane & 15;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int lr = tg * 16 + (lane >> 4) * 4 + i;  // local row in the workgroup
      const int row = row0 + lr;
      float v[ET];
      float m = -INFINITY;
#pragma unroll
      for (int t = 0; t < ET; ++t) {
        const bool ok = t * 16 + col < E;
        v[t] = ok ? acc[t][i] * inv_tau : -INFINITY;
        m = fmaxf(m, v[t]);
      }
      m = row16_max(m);          // the token's 16 lanes form one DPP row
      float s = 0.f;
#pragma unroll
      for (int t = 0; t < ET; ++t) {
        v[t] = (t * 16 + col < E) ? expf(v[t] - m) : 0.f;
        s += v[t];
      }
      s = row16_sum(s);
#pragma unroll
      for (int t = 0; t < ET; ++t) {
        const int e = t * 16 + col;
        const float p = v[t] / s;
        if (e < E) {
          if (row < N) S[(size_t)row * E + e] = p;
          sT[e][lr] = p;
        }
      }
    }
  }
  __syncthreads();
  // transposed, coalesced write of ST[e][row0 .. row0+64)
  for (int c = tid; c < E * RT_ROWS; c += NT) {
    const int e = c / RT_ROWS, r = c % RT_ROWS;
    if (row0 + r < N) ST[(size_t)e * N + row0 + r] = sT[e][r];
  }
}

// fp32 storage: plain fp32 FMA, fp32 sums of 32-wide K chunks added in K order.
constexpr int RF_ROWS = 32;
constexpr int RF_KC = 32;

__global__ __launch_bounds__(256) void router_softmax_f32_kernel(
    const float* __restrict__ X, const float* __restrict__ Wg, float* __restrict__ S,
    float* __restrict__ ST, int N, int d, int E, float inv_tau) {
  __shared__ float sX[RF_ROWS][RF_KC + 1];
  __shared__ float sW[256][RF_KC + 1];
  __shared__ float sZ[RF_ROWS][257];
  const int tid = threadIdx.x;
  const int row0 = blockIdx.x * RF_ROWS;
  const int nout = RF_ROWS * E;
  float acc[32];
#pragma unroll
  for (int q = 0; q < 32; ++q) acc[q] = 0.f;
  for (int kc = 0; kc < d; kc += RF_KC) {
    for (int c = tid; c < RF_ROWS * RF_KC; c += 256) {
      const int r = c / RF_KC, k = c % RF_KC;
      const int row = row0 + r;
      sX[r][k] = (row < N) ? X[(size_t)row * d + kc + k] : 0.f;
    }
    for (int c = tid; c < E * RF_KC; c += 256) {
      const int e = c / RF_KC, k = c % RF_KC;
      sW[e][k] = Wg[(size_t)e * d + kc + k];
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 32; ++q) {
      const int o = tid + q * 256;
      if (o < nout) {
        const int r = o / E, e = o % E;
        // two-level sum: each K chunk in its own partial, the partials added in
        // K order (rounding error grows with the chunk and chunk counts, not d)
        float a = 0.f;
        for (int k = 0; k < RF_KC; ++k) a = fmaf(sX[r][k], sW[e][k], a);
        acc[q] += a;
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int q = 0; q < 32; ++q) {
    const int o = tid + q * 256;
    if (o < nout) sZ[o / E][o % E] = acc[q] * inv_tau;
  }
  __syncthreads();
  const int lane = tid & 63, wave = tid >> 6;
  for (int r = wave; r < RF_ROWS; r += 4) {
    const int row = row0 + r;
    if (row >= N) break;
    float m = -INFINITY;
    for (int e = lane; e < E; e += 64) m = fmaxf(m, sZ[r][e]);
    for (int o = 1; o < 64; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    float s = 0.f;
    for (int e = lane; e < E; e += 64) s += expf(sZ[r][e] - m);
    for (int o = 1; o < 64; o <<= 1) s += __shfl_xor(s, o, 64);
    for (int e = lane; e < E; e += 64) {
      const float p = expf(sZ[r][e] - m) / s;
      S[(size_t)row * E + e] = p;
      ST[(size_t)e * N + row] = p;
    }
  }
}


template <int ET, int TG>
hipError_t run_router(const bf16_t* x, const bf16_t* w, float* S, float* ST, int N, int d, int E,
                      float inv_tau, hipStream_t st) {
  const int grid = (N + 16 * TG - 1) / (16 * TG);
  router_softmax_bf16_kernel<ET, TG><<<grid, 64 * TG * RouterCfg<ET>::KS, 0, st>>>(x, w, S, ST, N,
                                                                                 d, E, inv_tau);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_router_softmax(int dtype, const void* X, const void* Wg, float* S, float* ST,
                                 int N, int d, int E, float inv_tau, hipStream_t st) {
  if (N == 0) return hipSuccess;
  if (dtype == DT_F32) {
    const int grid = (N + RF_ROWS - 1) / RF_ROWS;
    router_softmax_f32_kernel<<<grid, 256, 0, st>>>((const float*)X, (const float*)Wg, S, ST, N,
                                                    d, E, inv_tau);
    return hipGetLastError();
  }
  const bf16_t* x = (const bf16_t*)X;
  const bf16_t* w = (const bf16_t*)Wg;
  // 64-token workgroups when they fill every CU (256), else 16-token ones
  if (N >= 256 * 64) {
    if (E <= 16) return run_router<1, 4>(x, w, S, ST, N, d, E, inv_tau, st);
    if (E <= 32) return run_router<2, 4>(x, w, S, ST, N, d, E, inv_tau, st);
    if (E <= 64) return run_router<4, 4>(x, w, S, ST, N, d, E, inv_tau, st);
    if (E <= 128) return run_router<8, 4>(x, w, S, ST, N, d, E, inv_tau, st);
    return run_router<16, 4>(x, w, S, ST, N, d, E, inv_tau, st);
  }
  if (E <= 16) return run_router<1, 1>(x, w, S, ST, N, d, E, inv_tau, st);
  if (E <= 32) return run_router<2, 1>(x, w, S, ST, N, d, E, inv_tau, st);
  if (E <= 64) return run_router<4, 1>(x, w, S, ST, N, d, E, inv_tau, st);
  if (E <= 128) return run_router<8, 1>(x, w, S, ST, N, d, E, inv_tau, st);
  return run_router<16, 1>(x, w, S, ST, N, d, E, inv_tau, st);
}

}  // namespace ec
