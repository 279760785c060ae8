// Router: logits Z = X Wg^T (Wg stored [E, d]) and S = softmax(Z / tau) over the
// experts of each token (the score matrix S of Section 2.2).  Writes S [N, E]
// and its transpose ST [E, N]; the column top-k reads ST so that each
// (group, expert) column is contiguous.
//
// bf16: one workgroup = 64 tokens, 4 waves x 16 tokens.  Each wave streams its
// own 16 token rows straight from HBM into MFMA A-fragments (every X element is
// used by exactly one wave, so it never touches LDS); the router matrix is
// staged through LDS in 64-wide K chunks (double buffered) and shared by the
// 4 waves.  v_mfma_f32_16x16x32_bf16 with fp32 accumulation; softmax in the
// epilogue with the 16 lanes that hold one token's logits.
#include "ec_common.h"
#include "ec_kernels.h"

namespace ec {

namespace {

constexpr int RT_ROWS = 64;   // tokens per workgroup
constexpr int RT_KC = 64;     // K chunk
constexpr int RT_LDK = RT_KC + 8;  // padded LDS row (bf16 elements)

template <int ET>
__global__ __launch_bounds__(256) void router_softmax_bf16_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ Wg, float* __restrict__ S,
    float* __restrict__ ST, int N, int d, int E, float inv_tau) {
  constexpr int EP = ET * 16;
  __shared__ __attribute__((aligned(16))) bf16_t sW[2][EP * RT_LDK];
  __shared__ float sT[EP][RT_ROWS + 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int row0 = blockIdx.x * RT_ROWS;
  const int myrow = row0 + wave * 16 + (lane & 15);
  const int xrow = myrow < N ? myrow : N - 1;
  const bf16_t* xp = X + (size_t)xrow * d + (lane >> 4) * 16;

  // Wg chunk loader: EP rows x 8 chunks of 16 bytes
  auto load_w = [&](int kc, uint4* regs) {
#pragma unroll
    for (int q = 0; q < (EP * 8 + 255) / 256; ++q) {
      const int c = tid + q * 256;
      if (c < EP * 8) {
        const int r = c >> 3, ch = c & 7;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (r < E) v = *reinterpret_cast<const uint4*>(Wg + (size_t)r * d + kc + ch * 8);
        regs[q] = v;
      }
    }
  };
  auto store_w = [&](int buf, const uint4* regs) {
#pragma unroll
    for (int q = 0; q < (EP * 8 + 255) / 256; ++q) {
      const int c = tid + q * 256;
      if (c < EP * 8) {
        const int r = c >> 3, ch = c & 7;
        *reinterpret_cast<uint4*>(&sW[buf][r * RT_LDK + ch * 8]) = regs[q];
      }
    }
  };

  f32x4 acc[ET];
#pragma unroll
  for (int t = 0; t < ET; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  uint4 wreg[(EP * 8 + 255) / 256];
  load_w(0, wreg);
  uint4 xa0 = *reinterpret_cast<const uint4*>(xp);
  uint4 xa1 = *reinterpret_cast<const uint4*>(xp + 8);
  store_w(0, wreg);
  __syncthreads();

  const int nk = d / RT_KC;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    uint4 xb0 = xa0, xb1 = xa1;
    if (kt + 1 < nk) {
      load_w((kt + 1) * RT_KC, wreg);
      xa0 = *reinterpret_cast<const uint4*>(xp + (kt + 1) * RT_KC);
      xa1 = *reinterpret_cast<const uint4*>(xp + (kt + 1) * RT_KC + 8);
    }
    const bf16x8 a0 = __builtin_bit_cast(bf16x8, xb0);
    const bf16x8 a1 = __builtin_bit_cast(bf16x8, xb1);
#pragma unroll
    for (int t = 0; t < ET; ++t) {
      const bf16_t* wp = &sW[buf][(t * 16 + (lane & 15)) * RT_LDK + (lane >> 4) * 16];
      const bf16x8 b0 = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(wp));
      const bf16x8 b1 = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(wp + 8));
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b0, acc[t], 0, 0, 0);
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, acc[t], 0, 0, 0);
    }
    if (kt + 1 < nk) store_w(buf ^ 1, wreg);
    __syncthreads();
  }

  // Epilogue: lane holds logits of tokens 4*(lane/16)+i (i = 0..3) of this
  // wave's 16, for experts t*16 + lane%16.
  const int col = lane & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lr = wave * 16 + (lane >> 4) * 4 + i;  // local row in the workgroup
    const int row = row0 + lr;
    float v[ET];
    float m = -INFINITY;
#pragma unroll
    for (int t = 0; t < ET; ++t) {
      const bool ok = t * 16 + col < E;
      v[t] = ok ? acc[t][i] * inv_tau : -INFINITY;
      m = fmaxf(m, v[t]);
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    float s = 0.f;
#pragma unroll
    for (int t = 0; t < ET; ++t) {
      v[t] = (t * 16 + col < E) ? expf(v[t] - m) : 0.f;
      s += v[t];
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) s += __shfl_xor(s, o, 64);
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
  __syncthreads();
  // transposed, coalesced write of ST[e][row0 .. row0+64)
  for (int c = tid; c < E * RT_ROWS; c += 256) {
    const int e = c / RT_ROWS, r = c % RT_ROWS;
    if (row0 + r < N) ST[(size_t)e * N + row0 + r] = sT[e][r];
  }
}

// fp32 storage: plain fp32 FMA (exact products, fp32 sums in K order).
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
        float a = acc[q];
        for (int k = 0; k < RF_KC; ++k) a = fmaf(sX[r][k], sW[e][k], a);
        acc[q] = a;
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
  const int grid = (N + RT_ROWS - 1) / RT_ROWS;
  const bf16_t* x = (const bf16_t*)X;
  const bf16_t* w = (const bf16_t*)Wg;
  if (E <= 16)
    router_softmax_bf16_kernel<1><<<grid, 256, 0, st>>>(x, w, S, ST, N, d, E, inv_tau);
  else if (E <= 32)
    router_softmax_bf16_kernel<2><<<grid, 256, 0, st>>>(x, w, S, ST, N, d, E, inv_tau);
  else if (E <= 64)
    router_softmax_bf16_kernel<4><<<grid, 256, 0, st>>>(x, w, S, ST, N, d, E, inv_tau);
  else if (E <= 128)
    router_softmax_bf16_kernel<8><<<grid, 256, 0, st>>>(x, w, S, ST, N, d, E, inv_tau);
  else
    router_softmax_bf16_kernel<16><<<grid, 256, 0, st>>>(x, w, S, ST, N, d, E, inv_tau);
  return hipGetLastError();
}

}  // namespace ec
