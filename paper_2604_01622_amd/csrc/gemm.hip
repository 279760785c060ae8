// Grouped GEMMs of the SwiGLU experts (Appendix E) over the E expert buffers.
// Expert-choice gives every expert the same number of rows M = K_tot
// (Section 2.2: each expert processes exactly its capacity), so the group is
// a uniform batch of E problems; ragged per-group capacities only change M.
//
// bf16: v_mfma_f32_32x32x16_bf16, fp32 accumulation.  A workgroup of 4 waves
// (2 x 2) computes a BM x BN tile; K advances in 64-wide steps through two LDS
// buffers (padded rows, conflict-free 16-byte fragment reads) while the next
// step's global loads are in flight.  Operands stored K-contiguous are copied
// as 16-byte rows; operands stored M/N-contiguous (the backward's transposed
// products) are loaded as 8 x 8 blocks and transposed in registers on their
// way into LDS, so every MFMA fragment is one 16-byte LDS read.  Tiles are
// numbered so that consecutive ones share an expert and stay on one XCD.
//
// fp32: a plain LDS-tiled FMA kernel with the same operand conventions.
#include "ec_common.h"
#include "ec_kernels.h"

namespace ec {

namespace {

constexpr int GBK = 64;
constexpr int GLDK = GBK + 8;  // padded LDS row in bf16 elements (144 bytes)

enum { EPI_STORE = 0, EPI_SWIGLU = 1, EPI_SWIGLU_BWD = 2 };

struct GemmParams {
  // A operand, element (m, k) of batch e:
  //   K-contiguous:  A[e*a_bs + m*lda + k];   M-contiguous: A[e*a_bs + k*lda + m]
  const void* A;
  long a_bs;
  int lda;
  // B operand, element (n, k) of batch e:
  //   K-contiguous:  B[e*b_bs + n*ldb + k]  (SwiGLU: rows of W1 and W3 side by side)
  //   N-contiguous:  B[e*b_bs + k*ldb + n] for k < k_split, else B2[e*b_bs + (k-k_split)*ldb + n]
  const void* B;
  const void* B2;
  long b_bs;
  int ldb;
  int k_split;
  int M, N, K;        // per batch (SwiGLU: N = h, the output width)
  int kv_a, kv_b;     // k >= kv reads as zero
  int batches, MT, NT;
  // output (dtype, or fp32 when out_f32): rows m >= c_split go to C2 at m - c_split
  void* C;
  void* C2;
  long c_bs;
  int ldc;
  int c_split;
  // SwiGLU: H1/H3 [batch][M][h] saved (forward, optional) or read (backward)
  void* H1;
  void* H3;
  long h_bs;
  int ldh;
};

// ------------------------------------------------------------------ bf16 MFMA

__device__ __forceinline__ void transpose8x8(const u32x4 in[8], u32x4 out[8]) {
  // in[kq] holds 8 bf16 along m for k = kq; out[mm] holds 8 bf16 along k for m = mm
#pragma unroll
  for (int p = 0; p < 4; ++p) {       // source dword p holds m = 2p, 2p+1
#pragma unroll
    for (int q = 0; q < 4; ++q) {     // dest dword q holds k = 2q, 2q+1
      const uint32_t lo = in[2 * q][p], hi = in[2 * q + 1][p];
      out[2 * p][q] = (lo & 0xffffu) | (hi << 16);
      out[2 * p + 1][q] = (lo >> 16) | (hi & 0xffff0000u);
    }
  }
}

template <int R, bool KC, int NT>
struct TileRegs {
  static constexpr int N = KC ? (R * 8 + NT - 1) / NT : 8 * ((R + NT - 1) / NT);
};

// Loads one 64-wide K step of an operand tile of R rows into registers.
//   KC:  row r (0..R) -> pointer row_ptr(r) (K-contiguous), chunk of 8 k.
//   !KC: element (r, k) at col_base + k*ld + r, rows r >= r_valid zero.
// K-contiguous operand: chunk c = tid + q*NT covers row c/8, k-chunk c%8.  The
// K extent of such operands is a multiple of 64, so no K predicate is needed.
template <int R, int NT>
__device__ __forceinline__ void load_kc(u32x4* regs, const bf16_t* const* rowp, int k0) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < TileRegs<R, true, NT>::N; ++q) {
    const int c = tid + q * NT;
    if (R * 8 % NT == 0 || c < R * 8)
      regs[q] = *reinterpret_cast<const u32x4*>(rowp[q] + k0 + (c & 7) * 8);
  }
}

template <int R, int NT>
__device__ __forceinline__ void store_kc(bf16_t* s, const u32x4* regs) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < TileRegs<R, true, NT>::N; ++q) {
    const int c = tid + q * NT;
    if (R * 8 % NT == 0 || c < R * 8)
      *reinterpret_cast<u32x4*>(s + (c >> 3) * GLDK + (c & 7) * 8) = regs[q];
  }
}

template <int R, int NT>
__device__ __forceinline__ void store_mn(bf16_t* s, const u32x4* regs) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < (R + NT - 1) / NT; ++q) {
    const int b = tid + q * NT;
    if (b < R) {
      const int kb = b & 7, rc = b >> 3;
      u32x4 t[8];
      transpose8x8(regs + 8 * q, t);
#pragma unroll
      for (int mm = 0; mm < 8; ++mm)
        *reinterpret_cast<u32x4*>(s + (rc * 8 + mm) * GLDK + kb * 8) = t[mm];
    }
  }
}

template <int BM, int BN, int WGM, int WGN, bool A_KC, bool B_KC, int EPI, bool OUT_F32>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void gemm_bf16_kernel(GemmParams p) {
  constexpr int NT = 64 * WGM * WGN;   // threads
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int MB = WM / 32, NB = WN / 32;
  constexpr int A_N = TileRegs<BM, A_KC, NT>::N, B_N = TileRegs<BN, B_KC, NT>::N;
  static_assert(EPI != EPI_SWIGLU || (NB % 2 == 0), "SwiGLU needs W1 and W3 blocks per wave");
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * (BM + BN) * GLDK];
  bf16_t* As = smem;
  bf16_t* Bs = smem + 2 * BM * GLDK;

  const int ntile = p.batches * p.MT * p.NT;
  const int t = xcd_tile_id(blockIdx.x, gridDim.x);
  if (t >= ntile) return;
  const int per_b = p.MT * p.NT;
  const int e = t / per_b;
  const int rem = t - e * per_b;
  const int mt = rem % p.MT, nt = rem / p.MT;
  const int m0 = mt * BM;
  const int n0 = (EPI == EPI_SWIGLU) ? nt * (BN / 2) : nt * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WGM, wn = wave / WGM;

  const bf16_t* Ab = reinterpret_cast<const bf16_t*>(p.A) + (size_t)e * p.a_bs;
  const bf16_t* Bb = reinterpret_cast<const bf16_t*>(p.B) + (size_t)e * p.b_bs;
  const bf16_t* B2b = p.B2 ? reinterpret_cast<const bf16_t*>(p.B2) + (size_t)e * p.b_bs : nullptr;

  // per-thread row pointers of the K-contiguous operands (fixed over K)
  const bf16_t* arow[A_KC ? A_N : 1];
  const bf16_t* brow[B_KC ? B_N : 1];
  if constexpr (A_KC) {
#pragma unroll
    for (int q = 0; q < A_N; ++q) {
      int r = m0 + ((tid + q * NT) >> 3);
      r = r < p.M ? r : p.M - 1;
      arow[q] = Ab + (size_t)r * p.lda;
    }
  }
  if constexpr (B_KC) {
#pragma unroll
    for (int q = 0; q < B_N; ++q) {
      const int lr = (tid + q * NT) >> 3;
      if constexpr (EPI == EPI_SWIGLU) {
        const int half = lr / (BN / 2);
        int r = n0 + lr % (BN / 2);
        r = r < p.N ? r : p.N - 1;
        brow[q] = (half ? B2b : Bb) + (size_t)r * p.ldb;
      } else {
        int r = n0 + lr;
        r = r < p.N ? r : p.N - 1;
        brow[q] = Bb + (size_t)r * p.ldb;
      }
    }
  }

  // M/N-contiguous operand: 8 x 8 block b = tid + q*NT covers k-rows kb*8.. and
  // columns rc*8..; rows past kv (the ragged K tail) and columns past `cols` read 0.
  auto load_mn = [&](u32x4* regs, auto src_row, int R, int r0, int cols, int k0, int kv) {
#pragma unroll
    for (int q = 0; q < 8 * ((R + NT - 1) / NT) / 8; ++q) {
      const int b = tid + q * NT;
      const int kb = b & 7, rc = b >> 3;
      const int c = r0 + rc * 8;
      const bool full = (k0 + GBK <= kv);
#pragma unroll
      for (int kq = 0; kq < 8; ++kq) {
        const int k = k0 + kb * 8 + kq;
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if ((R % NT == 0 || b < R) && (full || k < kv) && c < cols)
          v = *reinterpret_cast<const u32x4*>(src_row(k) + c);
        regs[8 * q + kq] = v;
      }
    }
  };
  auto load_a = [&](int k0, u32x4* regs) {
    if constexpr (A_KC) {
      load_kc<BM, NT>(regs, arow, k0);
    } else {
      load_mn(regs, [&](int k) { return Ab + (size_t)k * p.lda; }, BM, m0, p.M, k0, p.kv_a);
    }
  };
  auto load_b = [&](int k0, u32x4* regs) {
    if constexpr (B_KC) {
      load_kc<BN, NT>(regs, brow, k0);
    } else {
      load_mn(regs,
              [&](int k) {
                return (k < p.k_split) ? Bb + (size_t)k * p.ldb
                                       : B2b + (size_t)(k - p.k_split) * p.ldb;
              },
              BN, n0, p.N, k0, p.kv_b);
    }
  };
  auto store_a = [&](int buf, const u32x4* regs) {
    if constexpr (A_KC) store_kc<BM, NT>(As + buf * BM * GLDK, regs);
    else store_mn<BM, NT>(As + buf * BM * GLDK, regs);
  };
  auto store_b = [&](int buf, const u32x4* regs) {
    if constexpr (B_KC) store_kc<BN, NT>(Bs + buf * BN * GLDK, regs);
    else store_mn<BN, NT>(Bs + buf * BN * GLDK, regs);
  };

  // LDS row of this wave's B block ni
  auto b_lds_row = [&](int ni) -> int {
    if constexpr (EPI == EPI_SWIGLU) {
      constexpr int HWN = BN / 2 / WGN;  // W1 (and W3) columns per wave
      return (ni < NB / 2) ? wn * HWN + ni * 32 : BN / 2 + wn * HWN + (ni - NB / 2) * 32;
    } else {
      return wn * WN + ni * 32;
    }
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int mi = 0; mi < MB; ++mi)
#pragma unroll
    for (int ni = 0; ni < NB; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.f;

  u32x4 ra[A_N], rb[B_N];
  load_a(0, ra);
  load_b(0, rb);
  store_a(0, ra);
  store_b(0, rb);
  __syncthreads();

  const int KT = (p.K + GBK - 1) / GBK;
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) {
      load_a((kt + 1) * GBK, ra);
      load_b((kt + 1) * GBK, rb);
    }
    const bf16_t* as = As + buf * BM * GLDK;
    const bf16_t* bs = Bs + buf * BN * GLDK;
#pragma unroll
    for (int kk = 0; kk < GBK / 16; ++kk) {
      const int ko = kk * 16 + (lane >> 5) * 8;
      bf16x8 af[MB], bfr[NB];
#pragma unroll
      for (int mi = 0; mi < MB; ++mi)
        af[mi] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(as + (wm * WM + mi * 32 + (lane & 31)) * GLDK + ko));
#pragma unroll
      for (int ni = 0; ni < NB; ++ni)
        bfr[ni] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(bs + (b_lds_row(ni) + (lane & 31)) * GLDK + ko));
#pragma unroll
      for (int mi = 0; mi < MB; ++mi)
#pragma unroll
        for (int ni = 0; ni < NB; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bfr[ni], acc[mi][ni], 0, 0, 0);
    }
    if (kt + 1 < KT) {
      store_a(buf ^ 1, ra);
      store_b(buf ^ 1, rb);
    }
    __syncthreads();
  }

  // ---- epilogue: stage 32-row slices of the wave tile through LDS ----
  constexpr int SLD = WN + 4;
  float* stage = reinterpret_cast<float*>(smem) + wave * 32 * SLD;
#pragma unroll
  for (int mi = 0; mi < MB; ++mi) {
#pragma unroll
    for (int ni = 0; ni < NB; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        stage[row * SLD + ni * 32 + (lane & 31)] = acc[mi][ni][r];
      }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): staged values visible to the wave
    __builtin_amdgcn_wave_barrier();
    const int mbase = m0 + wm * WM + mi * 32;
    if constexpr (EPI == EPI_STORE) {
      constexpr int CPR = WN / 8;  // 8-wide chunks per staged row
#pragma unroll
      for (int q = 0; q < (32 * CPR) / 64; ++q) {
        const int c = lane + q * 64;
        const int row = c / CPR, cc = c % CPR;
        const int m = mbase + row;
        const int n = n0 + wn * WN + cc * 8;
        if (m < p.M && n < p.N) {
          const float* v = stage + row * SLD + cc * 8;
          float vv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) vv[u] = v[u];
          const bool second = m >= p.c_split;
          const int mm = second ? m - p.c_split : m;
          const size_t off = (size_t)e * p.c_bs + (size_t)mm * p.ldc + n;
          if constexpr (OUT_F32) Elem<float>::store8((float*)(second ? p.C2 : p.C) + off, vv);
          else Elem<bf16_t>::store8((bf16_t*)(second ? p.C2 : p.C) + off, vv);
        }
      }
    } else if constexpr (EPI == EPI_SWIGLU) {
      constexpr int HW = WN / 2;    // h1 columns staged, then h3 columns
      constexpr int CPR = HW / 8;
#pragma unroll
      for (int q = 0; q < (32 * CPR + 63) / 64; ++q) {
        const int c = lane + q * 64;
        const int row = c / CPR, cc = c % CPR;
        const int m = mbase + row;
        const int n = n0 + wn * HW + cc * 8;
        if (c < 32 * CPR && m < p.M && n < p.N) {
          const float* v1 = stage + row * SLD + cc * 8;
          const float* v3 = v1 + HW;
          float a[8], h1[8], h3[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            h1[u] = v1[u];
            h3[u] = v3[u];
            a[u] = silu_f(h1[u]) * h3[u];
          }
          const size_t off = (size_t)e * p.c_bs + (size_t)m * p.ldc + n;
          Elem<bf16_t>::store8((bf16_t*)p.C + off, a);
          if (p.H1) {
            const size_t ho = (size_t)e * p.h_bs + (size_t)m * p.ldh + n;
            Elem<bf16_t>::store8((bf16_t*)p.H1 + ho, h1);
            Elem<bf16_t>::store8((bf16_t*)p.H3 + ho, h3);
          }
        }
      }
    } else {  // EPI_SWIGLU_BWD: acc = dA; dH1 -> C, dH3 -> C2
      constexpr int CPR = WN / 8;
#pragma unroll
      for (int q = 0; q < (32 * CPR) / 64; ++q) {
        const int c = lane + q * 64;
        const int row = c / CPR, cc = c % CPR;
        const int m = mbase + row;
        const int n = n0 + wn * WN + cc * 8;
        if (m < p.M && n < p.N) {
          const float* v = stage + row * SLD + cc * 8;
          const size_t ho = (size_t)e * p.h_bs + (size_t)m * p.ldh + n;
          float h1[8], h3[8], d1[8], d3[8];
          Elem<bf16_t>::load8((const bf16_t*)p.H1 + ho, h1);
          Elem<bf16_t>::load8((const bf16_t*)p.H3 + ho, h3);
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const float da = v[u];
            const float sg = sigmoid_f(h1[u]);
            d3[u] = da * h1[u] * sg;
            d1[u] = da * h3[u] * sg * (1.0f + h1[u] * (1.0f - sg));
          }
          const size_t off = (size_t)e * p.c_bs + (size_t)m * p.ldc + n;
          Elem<bf16_t>::store8((bf16_t*)p.C + off, d1);
          Elem<bf16_t>::store8((bf16_t*)p.C2 + off, d3);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// ------------------------------------------------------------------ bf16 MFMA, pipelined
// Both operands K-contiguous (the forward products).  K advances 32 at a time
// through a ring of STAGES LDS buffers filled directly from global memory by
// global_load_lds_dwordx4 (no VGPR staging), STAGES-1 K steps ahead of the
// MFMAs.  Each 64-byte LDS row holds one operand row's 32 k values as four
// 16-byte chunks, XOR-swizzled by row so that the 32-lane fragment reads are
// free of bank conflicts.

constexpr int DBK = 32;

__device__ __forceinline__ int dma_swz(int row) { return ((row >> 1) ^ (row >> 3)) & 3; }

// 16 bytes per lane from global memory straight into LDS at lds + 16 * lane.
// (The builtin exists only for the device; the host pass must not see it or it
// drops the kernel's launch stub.)
__device__ __forceinline__ void dma16(const void* g, void* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
#endif
}

constexpr int vmcnt_imm(int n) { return (n & 15) | (((n >> 4) & 3) << 14) | (7 << 4) | (15 << 8); }

template <int BM, int BN, int WGM, int WGN, int STAGES, int KSTEP, int EPI>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void gemm_nt_dma_kernel(GemmParams p) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int MB = WM / 32, NB = WN / 32;
  constexpr int KK = KSTEP / 16;                // MFMA k-steps per stage
  constexpr int CPR = KSTEP / 8;                // 16-byte chunks per LDS row
  constexpr int ROWB = KSTEP * 2;               // bytes per LDS row
  constexpr int ROWS = BM + BN;                 // LDS rows per stage (A then B)
  constexpr int STAGE_BYTES = ROWS * ROWB;
  constexpr int RPL = 1024 / ROWB;              // rows per 1 KiB load block
  constexpr int LOADS = ROWS * CPR / NT;        // 16-byte chunks per thread per stage
  constexpr int SLD = WN + 4;
  constexpr int STAGE_EPI = NT / 64 * 32 * SLD * 4;
  constexpr int SMEM = STAGES * STAGE_BYTES > STAGE_EPI ? STAGES * STAGE_BYTES : STAGE_EPI;
  static_assert(ROWS * CPR % NT == 0, "whole 16-byte chunks per thread");
  static_assert(KSTEP == 32 || KSTEP == 64, "K step");
  static_assert(EPI != EPI_SWIGLU || (NB % 2 == 0), "SwiGLU needs W1 and W3 blocks per wave");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  const int ntile = p.batches * p.MT * p.NT;
  const int t = xcd_tile_id(blockIdx.x, gridDim.x);
  if (t >= ntile) return;
  const int per_b = p.MT * p.NT;
  const int e = t / per_b;
  const int rem = t - e * per_b;
  const int mt = rem % p.MT, nt = rem / p.MT;
  const int m0 = mt * BM;
  const int n0 = (EPI == EPI_SWIGLU) ? nt * (BN / 2) : nt * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WGM, wn = wave / WGM;
  const bf16_t* Ab = reinterpret_cast<const bf16_t*>(p.A) + (size_t)e * p.a_bs;
  const bf16_t* Bb = reinterpret_cast<const bf16_t*>(p.B) + (size_t)e * p.b_bs;
  const bf16_t* B2b = p.B2 ? reinterpret_cast<const bf16_t*>(p.B2) + (size_t)e * p.b_bs : nullptr;

  // swizzle: physical chunk = logical chunk ^ swz(row), conflict-free 32-lane
  // fragment reads for 32 and 64 LDS banks
  auto swz = [](int row) -> int {
    if constexpr (KSTEP == 32) return ((row >> 1) ^ (row >> 3)) & 3;
    else return (row ^ (row >> 3)) & 7;
  };

  // The q-th load of this thread fills 1 KiB block (wave * LOADS + q) of a stage.
  const bf16_t* src[LOADS];
#pragma unroll
  for (int q = 0; q < LOADS; ++q) {
    const int row = (wave * LOADS + q) * RPL + lane / CPR;
    const int lc = (lane % CPR) ^ swz(row);
    const bf16_t* rp;
    if (row < BM) {
      int r = m0 + row;
      r = r < p.M ? r : p.M - 1;
      rp = Ab + (size_t)r * p.lda;
    } else {
      const int lr = row - BM;
      if constexpr (EPI == EPI_SWIGLU) {
        int r = n0 + lr % (BN / 2);
        r = r < p.N ? r : p.N - 1;
        rp = (lr < BN / 2 ? Bb : B2b) + (size_t)r * p.ldb;
      } else {
        int r = n0 + lr;
        r = r < p.N ? r : p.N - 1;
        rp = Bb + (size_t)r * p.ldb;
      }
    }
    src[q] = rp + lc * 8;
  }
  auto issue = [&](int kt, int stage) {
    char* base = smem + stage * STAGE_BYTES + wave * LOADS * 1024;
#pragma unroll
    for (int q = 0; q < LOADS; ++q) dma16(src[q] + kt * KSTEP, base + q * 1024);
  };

  auto b_lds_row = [&](int ni) -> int {
    if constexpr (EPI == EPI_SWIGLU) {
      constexpr int HWN = BN / 2 / WGN;
      return (ni < NB / 2) ? wn * HWN + ni * 32 : BN / 2 + wn * HWN + (ni - NB / 2) * 32;
    } else {
      return wn * WN + ni * 32;
    }
  };
  int aoff[MB], boff[NB], aswz[MB], bswz[NB];
#pragma unroll
  for (int mi = 0; mi < MB; ++mi) {
    const int row = wm * WM + mi * 32 + (lane & 31);
    aoff[mi] = row * ROWB;
    aswz[mi] = swz(row);
  }
#pragma unroll
  for (int ni = 0; ni < NB; ++ni) {
    const int row = BM + b_lds_row(ni) + (lane & 31);
    boff[ni] = row * ROWB;
    bswz[ni] = swz(row);
  }
  bf16x8 af[2][MB], bfr[2][NB];
  auto load_frags = [&](int buf, int stage, int kk) {
    const char* sb = smem + stage * STAGE_BYTES;
    const int lc = kk * 2 + (lane >> 5);
#pragma unroll
    for (int mi = 0; mi < MB; ++mi)
      af[buf][mi] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(sb + aoff[mi] + ((lc ^ aswz[mi]) << 4)));
#pragma unroll
    for (int ni = 0; ni < NB; ++ni)
      bfr[buf][ni] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(sb + boff[ni] + ((lc ^ bswz[ni]) << 4)));
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int mi = 0; mi < MB; ++mi)
#pragma unroll
    for (int ni = 0; ni < NB; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.f;

  // Waits until this wave's loads of K step `kt` have landed, given how many
  // younger steps have been issued after it.
  auto wait_step = [&](int kt, int KT) {
    const int younger = KT - 1 - kt < STAGES - 2 ? KT - 1 - kt : STAGES - 2;
    static_assert(STAGES <= 5, "wait cases");
    if (younger >= 3) __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * LOADS));
    else if (younger == 2) __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LOADS));
    else if (younger == 1) __builtin_amdgcn_s_waitcnt(vmcnt_imm(LOADS));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  };

  // Ring: steps 0..STAGES-1 are issued up front; the end of step kt refills
  // stage kt % STAGES with step kt + STAGES once every wave has read it.  When
  // waiting for step j, the steps issued after it number
  // min(STAGES-1, KT-1-j) for j = 0 and min(STAGES-2, KT-1-j) afterwards.
  const int KT = p.K / KSTEP;
#pragma unroll
  for (int s = 0; s < STAGES; ++s)
    if (s < KT) issue(s, s);
  if (KT > 0) {
    const int younger = KT - 1 < STAGES - 1 ? KT - 1 : STAGES - 1;
    if (younger >= 3) __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * LOADS));
    else if (younger == 2) __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LOADS));
    else if (younger == 1) __builtin_amdgcn_s_waitcnt(vmcnt_imm(LOADS));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __builtin_amdgcn_s_barrier();
    load_frags(0, 0, 0);
  }
  // Each k-step: the first half of its MFMAs, then the next k-step's fragment
  // reads (at a stage end: the barrier, the refill of this stage and the next
  // stage's first fragments), then the second half, so that the LDS latency
  // is covered by MFMAs already in flight.
  constexpr int NMF = MB * NB;
  auto mfma_range = [&](int cur, int lo, int hi) {
#pragma unroll
    for (int q = 0; q < NMF; ++q) {
      if (q < lo || q >= hi) continue;
      const int mi = q / NB, ni = q % NB;
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][mi], bfr[cur][ni],
                                                              acc[mi][ni], 0, 0, 0);
    }
  };
  for (int kt = 0; kt < KT; ++kt) {
    const int stage = kt % STAGES;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const int cur = kk & 1;
      mfma_range(cur, 0, NMF / 2);
      __builtin_amdgcn_sched_barrier(0);
      if (kk + 1 < KK) {
        load_frags(cur ^ 1, stage, kk + 1);
      } else {
        // after the final step this reads a stale stage, harmlessly, which
        // keeps the loop body uniform
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): this wave's reads are done
        if (kt + 1 < KT) wait_step(kt + 1, KT);
        __builtin_amdgcn_s_barrier();
        if (kt + STAGES < KT) issue(kt + STAGES, stage);
        load_frags(cur ^ 1, (kt + 1) % STAGES, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      mfma_range(cur, NMF / 2, NMF);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  __syncthreads();

  // ---- epilogue (same as gemm_bf16_kernel) ----
  float* stage_f = reinterpret_cast<float*>(smem) + wave * 32 * SLD;
#pragma unroll
  for (int mi = 0; mi < MB; ++mi) {
#pragma unroll
    for (int ni = 0; ni < NB; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        stage_f[row * SLD + ni * 32 + (lane & 31)] = acc[mi][ni][r];
      }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    const int mbase = m0 + wm * WM + mi * 32;
    if constexpr (EPI == EPI_STORE) {
      constexpr int CPR = WN / 8;
#pragma unroll
      for (int q = 0; q < (32 * CPR) / 64; ++q) {
        const int c = lane + q * 64;
        const int row = c / CPR, cc = c % CPR;
        const int m = mbase + row;
        const int n = n0 + wn * WN + cc * 8;
        if (m < p.M && n < p.N) {
          const float* v = stage_f + row * SLD + cc * 8;
          float vv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) vv[u] = v[u];
          Elem<bf16_t>::store8((bf16_t*)p.C + (size_t)e * p.c_bs + (size_t)m * p.ldc + n, vv);
        }
      }
    } else {
      constexpr int HW = WN / 2;
      constexpr int CPR = HW / 8;
#pragma unroll
      for (int q = 0; q < (32 * CPR + 63) / 64; ++q) {
        const int c = lane + q * 64;
        const int row = c / CPR, cc = c % CPR;
        const int m = mbase + row;
        const int n = n0 + wn * HW + cc * 8;
        if (c < 32 * CPR && m < p.M && n < p.N) {
          const float* v1 = stage_f + row * SLD + cc * 8;
          const float* v3 = v1 + HW;
          float a[8], h1[8], h3[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            h1[u] = v1[u];
            h3[u] = v3[u];
            a[u] = silu_f(h1[u]) * h3[u];
          }
          Elem<bf16_t>::store8((bf16_t*)p.C + (size_t)e * p.c_bs + (size_t)m * p.ldc + n, a);
          if (p.H1) {
            const size_t ho = (size_t)e * p.h_bs + (size_t)m * p.ldh + n;
            Elem<bf16_t>::store8((bf16_t*)p.H1 + ho, h1);
            Elem<bf16_t>::store8((bf16_t*)p.H3 + ho, h3);
          }
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

template <int BM, int BN, int WGM, int WGN, int STAGES, int KSTEP, int EPI>
hipError_t run_nt_dma(GemmParams p, hipStream_t st) {
  p.MT = (p.M + BM - 1) / BM;
  p.NT = (EPI == EPI_SWIGLU) ? (p.N + BN / 2 - 1) / (BN / 2) : (p.N + BN - 1) / BN;
  const long ntile = (long)p.batches * p.MT * p.NT;
  if (ntile == 0) return hipSuccess;
  const long grid = (ntile + 7) / 8 * 8;
  gemm_nt_dma_kernel<BM, BN, WGM, WGN, STAGES, KSTEP, EPI>
      <<<dim3((unsigned)grid), 64 * WGM * WGN, 0, st>>>(p);
  return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN, bool A_KC, bool B_KC, int EPI, bool OUT_F32>
hipError_t run_bf16(GemmParams p, hipStream_t st) {
  p.MT = (p.M + BM - 1) / BM;
  p.NT = (EPI == EPI_SWIGLU) ? (p.N + BN / 2 - 1) / (BN / 2) : (p.N + BN - 1) / BN;
  const long ntile = (long)p.batches * p.MT * p.NT;
  if (ntile == 0) return hipSuccess;
  const long grid = (ntile + 7) / 8 * 8;
  gemm_bf16_kernel<BM, BN, WGM, WGN, A_KC, B_KC, EPI, OUT_F32>
      <<<dim3((unsigned)grid), 64 * WGM * WGN, 0, st>>>(p);
  return hipGetLastError();
}

// ------------------------------------------------------------------ fp32 FMA

constexpr int FT = 64;   // tile
constexpr int FK = 16;   // K step

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmParams p, int a_kc, int b_kc) {
  __shared__ float sA[FK][FT + 1];
  __shared__ float sB[FK][FT + 1];
  __shared__ float sB3[FK][FT + 1];
  const int e = blockIdx.z;
  const int m0 = blockIdx.y * FT, n0 = blockIdx.x * FT;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const float* A = (const float*)p.A + (size_t)e * p.a_bs;
  const float* B = (const float*)p.B + (size_t)e * p.b_bs;
  const float* B2 = p.B2 ? (const float*)p.B2 + (size_t)e * p.b_bs : nullptr;
  float acc[4][4] = {}, acc3[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += FK) {
    for (int c = tid; c < FK * FT; c += 256) {
      const int kk = c / FT, r = c % FT;
      const int k = k0 + kk, m = m0 + r, n = n0 + r;
      float va = 0.f, vb = 0.f, vb3 = 0.f;
      if (k < p.kv_a && m < p.M) va = a_kc ? A[(size_t)m * p.lda + k] : A[(size_t)k * p.lda + m];
      if (k < p.kv_b && n < p.N) {
        if (b_kc) {
          vb = B[(size_t)n * p.ldb + k];
          if (EPI == EPI_SWIGLU) vb3 = B2[(size_t)n * p.ldb + k];
        } else {
          vb = (k < p.k_split) ? B[(size_t)k * p.ldb + n] : B2[(size_t)(k - p.k_split) * p.ldb + n];
        }
      }
      sA[kk][r] = va;
      sB[kk][r] = vb;
      sB3[kk][r] = vb3;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < FK; ++kk) {
      float a[4], b[4], b3[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = sA[kk][ty * 4 + i];
        b[i] = sB[kk][tx * 4 + i];
        b3[i] = sB3[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          acc[i][jj] = fmaf(a[i], b[jj], acc[i][jj]);
          if (EPI == EPI_SWIGLU) acc3[i][jj] = fmaf(a[i], b3[jj], acc3[i][jj]);
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + jj;
      if (m >= p.M || n >= p.N) continue;
      if (EPI == EPI_STORE) {
        const bool second = m >= p.c_split;
        const int mm = second ? m - p.c_split : m;
        ((float*)(second ? p.C2 : p.C))[(size_t)e * p.c_bs + (size_t)mm * p.ldc + n] = acc[i][jj];
      } else if (EPI == EPI_SWIGLU) {
        const float h1 = acc[i][jj], h3 = acc3[i][jj];
        ((float*)p.C)[(size_t)e * p.c_bs + (size_t)m * p.ldc + n] = silu_f(h1) * h3;
        if (p.H1) {
          const size_t ho = (size_t)e * p.h_bs + (size_t)m * p.ldh + n;
          ((float*)p.H1)[ho] = h1;
          ((float*)p.H3)[ho] = h3;
        }
      } else {
        const size_t ho = (size_t)e * p.h_bs + (size_t)m * p.ldh + n;
        const float h1 = ((const float*)p.H1)[ho], h3 = ((const float*)p.H3)[ho];
        const float da = acc[i][jj];
        const float sg = sigmoid_f(h1);
        const size_t off = (size_t)e * p.c_bs + (size_t)m * p.ldc + n;
        ((float*)p.C)[off] = da * h3 * sg * (1.0f + h1 * (1.0f - sg));
        ((float*)p.C2)[off] = da * h1 * sg;
      }
    }
}

template <int EPI>
hipError_t run_f32(GemmParams p, int a_kc, int b_kc, hipStream_t st) {
  if (p.batches == 0 || p.M == 0 || p.N == 0) return hipSuccess;
  const dim3 grid((p.N + FT - 1) / FT, (p.M + FT - 1) / FT, p.batches);
  gemm_f32_kernel<EPI><<<grid, 256, 0, st>>>(p, a_kc, b_kc);
  return hipGetLastError();
}

GemmParams base_params() {
  GemmParams p = {};
  p.k_split = 1 << 30;
  p.c_split = 1 << 30;
  return p;
}

// deterministic split-K reduction: out[i] = sum_s part[s * n + i] (fixed s order)
__global__ void splitk_reduce_kernel(const float* __restrict__ part, float* __restrict__ out,
                                     int splits, long n, int rows_in, int rows_out, int cols) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)rows_out * cols) return;
  const long r = i / cols, c = i % cols;
  float s = 0.f;
  for (int q = 0; q < splits; ++q) s += part[(size_t)q * n + r * cols + c];
  out[i] = s;
  (void)rows_in;
}

}  // namespace

// ---------------------------------------------------------------- launchers

hipError_t launch_gemm_w13(int dtype, const void* Xe, const void* W1, const void* W3, void* A,
                           void* H1, void* H3, int E, int M, int d, int h, hipStream_t st) {
  GemmParams p = base_params();
  p.A = Xe; p.a_bs = (long)M * d; p.lda = d;
  p.B = W1; p.B2 = W3; p.b_bs = (long)h * d; p.ldb = d;
  p.M = M; p.N = h; p.K = d; p.kv_a = d; p.kv_b = d; p.batches = E;
  p.C = A; p.c_bs = (long)M * h; p.ldc = h;
  p.H1 = H1; p.H3 = H3; p.h_bs = (long)M * h; p.ldh = h;
  if (M == 0) return hipSuccess;
  if (dtype == DT_F32) return run_f32<EPI_SWIGLU>(p, 1, 1, st);
  return run_nt_dma<256, 256, 4, 2, 2, 64, EPI_SWIGLU>(p, st);
}

hipError_t launch_gemm_w2(int dtype, const void* A, const void* W2, void* O, int E, int M, int d,
                          int h, hipStream_t st) {
  GemmParams p = base_params();
  p.A = A; p.a_bs = (long)M * h; p.lda = h;
  p.B = W2; p.b_bs = (long)d * h; p.ldb = h;
  p.M = M; p.N = d; p.K = h; p.kv_a = h; p.kv_b = h; p.batches = E;
  p.C = O; p.c_bs = (long)M * d; p.ldc = d;
  if (M == 0) return hipSuccess;
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 1, 1, st);
  return run_nt_dma<256, 256, 4, 2, 2, 64, EPI_STORE>(p, st);
}

hipError_t launch_gemm_dA(int dtype, const void* dO, const void* W2, const void* H1,
                          const void* H3, void* dH, int E, int M, int d, int h, hipStream_t st) {
  // dA[m, n] = sum_k dO[m, k] W2[k, n]  (k over d, n over h); epilogue -> dH1, dH3
  GemmParams p = base_params();
  p.A = dO; p.a_bs = (long)M * d; p.lda = d;
  p.B = W2; p.b_bs = (long)d * h; p.ldb = h;
  p.M = M; p.N = h; p.K = d; p.kv_a = d; p.kv_b = d; p.batches = E;
  const size_t esz = dtype == DT_F32 ? 4 : 2;
  p.C = dH; p.C2 = (char*)dH + (size_t)h * esz; p.c_bs = (long)M * 2 * h; p.ldc = 2 * h;
  p.H1 = (void*)H1; p.H3 = (void*)H3; p.h_bs = (long)M * h; p.ldh = h;
  if (M == 0) return hipSuccess;
  if (dtype == DT_F32) return run_f32<EPI_SWIGLU_BWD>(p, 1, 0, st);
  return run_bf16<256, 256, 4, 2, true, false, EPI_SWIGLU_BWD, false>(p, st);
}

hipError_t launch_gemm_dXe(int dtype, const void* dH, const void* W1, const void* W3, void* dXe,
                           int E, int M, int d, int h, hipStream_t st) {
  // dXe[m, n] = sum_k dH[m, k] W13[k, n], k < h from W1, k >= h from W3
  GemmParams p = base_params();
  p.A = dH; p.a_bs = (long)M * 2 * h; p.lda = 2 * h;
  p.B = W1; p.B2 = W3; p.b_bs = (long)h * d; p.ldb = d; p.k_split = h;
  p.M = M; p.N = d; p.K = 2 * h; p.kv_a = 2 * h; p.kv_b = 2 * h; p.batches = E;
  p.C = dXe; p.c_bs = (long)M * d; p.ldc = d;
  if (M == 0) return hipSuccess;
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 1, 0, st);
  return run_bf16<256, 256, 4, 2, true, false, EPI_STORE, false>(p, st);
}

hipError_t launch_gemm_dW2(int dtype, const void* dO, const void* A, void* dW2, int E, int M,
                           int d, int h, hipStream_t st) {
  // dW2[m, n] = sum_k dO[k, m] A[k, n]  (m over d, n over h, k over the M expert rows)
  GemmParams p = base_params();
  p.A = dO; p.a_bs = (long)M * d; p.lda = d;
  p.B = A; p.b_bs = (long)M * h; p.ldb = h;
  p.M = d; p.N = h; p.K = M; p.kv_a = M; p.kv_b = M; p.batches = E;
  p.C = dW2; p.c_bs = (long)d * h; p.ldc = h;
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 0, 0, st);
  return run_bf16<256, 128, 4, 2, false, false, EPI_STORE, false>(p, st);
}

hipError_t launch_gemm_dW13(int dtype, const void* dH, const void* Xe, void* dW1, void* dW3,
                            int E, int M, int d, int h, hipStream_t st) {
  // [dW1; dW3][m, n] = sum_k dH[k, m] Xe[k, n]  (m over 2h, n over d)
  GemmParams p = base_params();
  p.A = dH; p.a_bs = (long)M * 2 * h; p.lda = 2 * h;
  p.B = Xe; p.b_bs = (long)M * d; p.ldb = d;
  p.M = 2 * h; p.N = d; p.K = M; p.kv_a = M; p.kv_b = M; p.batches = E;
  p.C = dW1; p.C2 = dW3; p.c_split = h; p.c_bs = (long)h * d; p.ldc = d;
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 0, 0, st);
  return run_bf16<256, 128, 4, 2, false, false, EPI_STORE, false>(p, st);
}

hipError_t launch_router_dx(int dtype, const void* dZ, const void* Wg, void* dX, int N, int E,
                            int EP, int d, hipStream_t st) {
  // dX[i, n] = sum_j dZ[i, j] Wg[j, n]; dZ is [N, EP] (bf16, zero padded) or [N, E] fp32
  GemmParams p = base_params();
  p.A = dZ; p.a_bs = 0; p.lda = (dtype == DT_F32) ? E : EP;
  p.B = Wg; p.b_bs = 0; p.ldb = d;
  p.M = N; p.N = d; p.K = (dtype == DT_F32) ? E : EP; p.kv_a = p.K; p.kv_b = E; p.batches = 1;
  p.C = dX; p.c_bs = 0; p.ldc = d;
  if (N == 0) return hipSuccess;
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 1, 0, st);
  return run_bf16<256, 128, 2, 2, true, false, EPI_STORE, false>(p, st);
}

int router_dwg_splits(int N, int E, int d) {
  (void)E;
  int tiles = (d + 127) / 128;
  int s = (512 + tiles - 1) / tiles;
  int maxs = (N + 255) / 256;
  if (s > maxs) s = maxs;
  return s < 1 ? 1 : s;
}

hipError_t launch_router_dwg(int dtype, const void* dZ, const void* X, float* dWg, float* part,
                             int splits, int N, int E, int EP, int d, hipStream_t st) {
  // dWg[j, n] = sum_i dZ[i, j] X[i, n], split over i in `splits` chunks
  if (N == 0 || splits < 1) return launch_zero(dWg, (size_t)E * d * sizeof(float), st);
  const int chunk = (N + splits - 1) / splits;
  GemmParams p = base_params();
  const size_t xs = dtype == DT_F32 ? 4 : 2;
  p.A = dZ; p.a_bs = (long)chunk * ((dtype == DT_F32) ? E : EP); p.lda = (dtype == DT_F32) ? E : EP;
  p.B = X; p.b_bs = (long)chunk * d; p.ldb = d;
  p.M = E; p.N = d; p.K = chunk; p.batches = splits;
  p.C = part; p.c_bs = (long)E * d; p.ldc = d;
  (void)xs;
  // each split sees rows [s*chunk, min(N, (s+1)*chunk)); the last may be short
  const int last = N - (splits - 1) * chunk;
  hipError_t err;
  if (last == chunk) {
    p.kv_a = chunk; p.kv_b = chunk;
    if (dtype == DT_F32) err = run_f32<EPI_STORE>(p, 0, 0, st);
    else err = run_bf16<256, 128, 2, 2, false, false, EPI_STORE, true>(p, st);
  } else {
    GemmParams p1 = p;
    p1.batches = splits - 1; p1.kv_a = chunk; p1.kv_b = chunk;
    err = (splits > 1) ? ((dtype == DT_F32) ? run_f32<EPI_STORE>(p1, 0, 0, st)
                                            : run_bf16<256, 128, 2, 2, false, false, EPI_STORE, true>(p1, st))
                       : hipSuccess;
    if (err != hipSuccess) return err;
    GemmParams p2 = p;
    const long ao = (long)(splits - 1) * p.a_bs, bo = (long)(splits - 1) * p.b_bs;
    p2.A = (const char*)p.A + ao * ((dtype == DT_F32) ? 4 : 2);
    p2.B = (const char*)p.B + bo * ((dtype == DT_F32) ? 4 : 2);
    p2.C = part + (size_t)(splits - 1) * E * d;
    p2.batches = 1; p2.kv_a = last; p2.kv_b = last;
    err = (dtype == DT_F32) ? run_f32<EPI_STORE>(p2, 0, 0, st)
                            : run_bf16<256, 128, 2, 2, false, false, EPI_STORE, true>(p2, st);
  }
  if (err != hipSuccess) return err;
  const long n = (long)E * d;
  splitk_reduce_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(part, dWg, splits, n, E, E, d);
  return hipGetLastError();
}

}  // namespace ec
