// Grouped GEMMs of the SwiGLU experts (Appendix E) over the E expert buffers.
// Expert-choice gives every expert the same number of rows M = K_tot
// (Section 2.2: each expert processes exactly its capacity), so the group is
// a uniform batch of E problems; ragged per-group capacities only change M.
//
// bf16: one pipelined kernel (gemm_dma_kernel) for every product of the
// forward and backward.  v_mfma_f32_32x32x16_bf16 with fp32 accumulation; a
// 256 x 256 output tile per workgroup of 8 waves (2 per SIMD, 64 x 128 or
// 128 x 64 each; the forward products take 192- or 128-row tiles, 96 x 64 or
// 64 x 64 per wave, when those pad short expert buffers less);
// K advances 64 at a time through a 2-stage LDS ring filled straight from
// global memory by global_load_lds_dwordx4 (no VGPR staging).  K-contiguous
// operands sit in LDS as 128-byte rows with XOR-swizzled 16-byte chunks
// (conflict-free fragment reads); K-major operands (the weight gradients'
// token-row contractions, and the weights in the dA and dX products) stay
// K-major in LDS and are read with the transposing ds_read_b64_tr_b16.  The MFMAs of each k-step alternate with the
// next step's fragment reads and, once the barrier has freed a stage, with its
// refill's DMA (for K-contiguous products half of it then, half in the next
// step's first sub-step), so LDS latency hides behind MFMAs in flight.  The
// MFMAs take the B fragment first, so each lane ends with four consecutive
// output columns of a row, staged through LDS with 16-byte writes for
// coalesced stores.  Tiles are numbered so that consecutive ones share an
// expert and stay on one XCD.
//
// The products that read the selected tokens' rows (of X, or of the output
// gradient dY) gather them in the operand load: the W1/W3 and dA products per
// row of their K-contiguous A, the dW2 and dW1/dW3 products per k row of their
// K-major operand, so no gathered copy is ever written.
//
// fp32: a plain LDS-tiled FMA kernel with the same operand conventions.
#include <type_traits>

#include "ec_common.h"
#include "ec_kernels.h"

namespace ec {

namespace {

enum { EPI_STORE = 0, EPI_SWIGLU = 1, EPI_SWIGLU_BWD = 2, EPI_STORE_ADD = 3 };

// Stage tags: every product gets its own kernel symbol, so that traces and
// counters attribute each launch to its stage.
enum { G_W13 = 1, G_W2, G_DA, G_DXE, G_DW2, G_DW13, G_ROUTER_DX, G_ROUTER_DWG,
       G_SH_W13, G_SH_W2, G_SH_DA, G_SH_DXE, G_SH_DW2, G_SH_DW13, G_TC_W13, G_TC_W2 };

struct GemmParams {
  // A operand, element (m, k) of batch e:
  //   K-contiguous:  A[e*a_bs + m*lda + k];   M-contiguous: A[e*a_bs + k*lda + m]
  const void* A;
  long a_bs;
  int lda;
  // bf16 K-contiguous A only (may be null): row m of batch e is row
  // a_rows[e*a_rows_bs + r0 + m] of A itself (r0: the batch's first packed row
  // with var_rows, else 0), so the gather of the selected tokens happens in the
  // operand load
  const int32_t* a_rows;
  long a_rows_bs;
  // B operand, element (n, k) of batch e:
  //   K-contiguous:  B[e*b_bs + n*ldb + k]  (SwiGLU: rows of W1 and W3 side by side)
  //   N-contiguous:  B[e*b_bs + k*ldb + n]; rows k >= k_split come from B2
  //                  instead (B2[e*b_bs + (k-k_split)*ldb + n]; the bf16 kernel
  //                  needs k_split to be a multiple of its k-step)
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
  // bf16 K-major operands (used with the OPT_GA / OPT_GB instantiations): row k
  // of batch e's A is row ka_rows[e*k_rows_bs + k] of A itself (kb_rows: of
  // B), so the gather of the selected tokens happens in the operand load when
  // the contraction runs over an expert's rows
  const int32_t* ka_rows;
  const int32_t* kb_rows;
  long k_rows_bs;
  // SwiGLU forward and backward, uniform batches only (may be null): a factor
  // per output row, g = gate[e*gate_bs + m] for row m of batch e.  The forward
  // writes A = g SiLU(H1) H3 (H1, H3 unscaled); the backward takes dA = g (the
  // product) before the SwiGLU backward.
  const float* gate;
  long gate_bs;
  // SwiGLU backward only (may be null): the gate-gradient partials.  For row m
  // of batch e and each column block q of the output (128 columns in the bf16
  // kernel, 64 in the fp32 one), dsp[(e M + m) dsp_ld + q] = sum over the block
  // of dA * A with dA as above and A = SiLU(H1) H3 recomputed from the saved
  // H1, H3 (so the sum over all blocks is g times the gate's gradient when the
  // product is dY W2).
  float* dsp;
  int dsp_ld;
  // Variable rows per batch (token choice): batch e owns rows
  // [var_rows[e], var_rows[e+1]) of A, C and H (row strides lda, ldc, ldh) and
  // tiles [var_tiles[e], var_tiles[e+1]) of the launch; both device arrays of
  // batches + 1 entries, null for a uniform batch of M rows.
  const int* var_rows;
  const int* var_tiles;
};

// Where one output tile sits: batch, row and column block, the batch's rows,
// and the element offsets of the batch in A, C and H.
struct TileCoord {
  int e, mt, nt, M, MT, NT, row0;
  size_t a_off, c_off, h_off;
};

// ------------------------------------------------------------------ bf16 MFMA, pipelined

// 16 bytes per lane from global memory straight into LDS at lds + 16 * lane.
// (The builtin exists only for the device; the host pass must not see it or it
// drops the kernel's launch stub.)
__device__ __forceinline__ void dma16(const void* g, void* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
#endif
}

constexpr int vmcnt_imm(int n) { return (n & 15) | (((n >> 4) & 3) << 14) | (7 << 4) | (15 << 8); }

// Each operand is K-contiguous (stored [rows][K]) or K-major (stored
// [K][rows]: the backward's transposed products).  A K-major tile is kept
// K-major in LDS (64 rows of k, its columns contiguous, 16-byte chunks
// XOR-swizzled by k) and read with the transposing ds_read_b64_tr_b16: in each 16-lane group, lane j addresses the
// 4 consecutive columns 4*(j%4).. of row kbase + j/4, and lane i receives
// column i of rows kbase..kbase+3 -- two such reads make one MFMA fragment.
// Rows past the valid K (ragged tail) and columns past the operand's width are
// fetched from a zero block, so the MFMAs see exact zeros there.

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

__device__ __attribute__((aligned(16))) bf16_t g_zero_block[4096];  // stays zero

__device__ __forceinline__ v4i16 ds_read_tr16(const char* __restrict__ p) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p));
#else
  return v4i16{0, 0, 0, 0};
#endif
}

template <int R, bool KC, int NT, int KSTEP>
struct DmaOperand {
  static constexpr int BYTES = R * KSTEP * 2;               // per stage
  static constexpr int LOADS = R * KSTEP / 8 / NT;          // 16-byte chunks per thread
  static constexpr int CPR = KC ? KSTEP / 8 : R / 8;        // chunks per LDS row
  static_assert(R * KSTEP / 8 % NT == 0, "whole chunks per thread");
  static_assert(KC || (R % 128 == 0), "K-major tiles are multiples of 128 wide");
};

// Chunk swizzles, chosen by measuring the fragment-read pattern on gfx950:
// K-contiguous rows of 64 or 128 bytes, and K-major rows (by k).
template <int KSTEP>
__device__ __forceinline__ int kc_swz(int row) {
  if constexpr (KSTEP == 64) return (row ^ (row >> 3)) & 7;
  else return ((row >> 1) ^ (row >> 2)) & 3;
}
__device__ __forceinline__ int km_swz(int k) { return (k & 3) << 2; }

// Options of an instantiation (bf16; see GemmParams): OPT_GA / OPT_GB gather
// the rows of a K-major A / B through p.ka_rows / p.kb_rows.
enum { OPT_GA = 1, OPT_GB = 2 };
template <int BM, int BN, int WGM, int WGN, int KSTEP, int STAGES, bool A_KC, bool B_KC, int EPI,
          bool OUT_F32, int OPT>
__device__ __forceinline__ void gemm_dma_tile(const GemmParams& p, const TileCoord& tc,
                                              char* smem) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int MB = WM / 32, NB = WN / 32;
  constexpr int KK = KSTEP / 16;
  static_assert(KSTEP == 32 || KSTEP == 64, "K step");
  static_assert(STAGES >= 2 && STAGES <= 5, "ring depth");
  using OA = DmaOperand<BM, A_KC, NT, KSTEP>;
  using OB = DmaOperand<BN, B_KC, NT, KSTEP>;
  constexpr int STAGE_BYTES = OA::BYTES + OB::BYTES;
  constexpr int LOADS = OA::LOADS + OB::LOADS;
  constexpr int SLD = WN + 4;
  static_assert(EPI != EPI_SWIGLU || (NB % 2 == 0), "SwiGLU needs W1 and W3 blocks per wave");
  static_assert(EPI != EPI_SWIGLU || B_KC, "SwiGLU forward has K-contiguous weights");
  const int e = tc.e, mt = tc.mt, nt = tc.nt, M = tc.M;
  const int m0 = mt * BM;
  const int n0 = (EPI == EPI_SWIGLU) ? nt * (BN / 2) : nt * BN;

  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index is uniform: read into a scalar register so that the LDS
  // destinations of the DMA loads (M0) are formed with scalar arithmetic
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WGM, wn = wave / WGM;
  // SwiGLU: the row factors of this wave's rows (lane l holds row wm*WM + 64 t
  // + l), read before the main loop so the epilogue finds them in registers
  constexpr bool GATED = EPI == EPI_SWIGLU || EPI == EPI_SWIGLU_BWD;
  constexpr int GR = GATED ? (WM + 63) / 64 : 1;
  float gate_r[GR];
  if constexpr (GATED) {
#pragma unroll
    for (int t = 0; t < GR; ++t) {
      const int m = m0 + wm * WM + 64 * t + lane;
      gate_r[t] = (p.gate && m < M) ? p.gate[(size_t)e * p.gate_bs + m] : 1.f;
    }
  }
  const bf16_t* Ab = reinterpret_cast<const bf16_t*>(p.A) + tc.a_off;
  const bf16_t* Bb = reinterpret_cast<const bf16_t*>(p.B) + (size_t)e * p.b_bs;
  const bf16_t* B2b = p.B2 ? reinterpret_cast<const bf16_t*>(p.B2) + (size_t)e * p.b_bs : nullptr;

  // ---- DMA sources.  Load q of a thread fills 1 KiB block (wave*L + q) of
  // the operand's stage area: 64 chunks, lane -> chunk.
  // K-contiguous: the row pointer of the chunk, offset by kt * KSTEP per step.
  // K-major: the chunk's address at k-step 0 (or the zero block for columns
  // past the operand), advanced by KSTEP rows after every issue; rows past the
  // valid K read the zero block instead.  K-major gathered (OPT_GA / OPT_GB):
  // the chunk's column in row 0 of the operand (clamped into the row: columns
  // past the width produce outputs that are not stored); the source rows of
  // the next k-step's 64 rows are held one per lane (fetched one step ahead,
  // the first two at set-up so that the prologue waits for no index) and each
  // load takes its row's with a lane read.  Rows past the valid K re-read a
  // valid row: the other operand, never gathered, reads zeros there.
  constexpr bool GA = (OPT & OPT_GA) != 0 && !A_KC, GB = (OPT & OPT_GB) != 0 && !B_KC;
  static_assert(((OPT & OPT_GA) == 0 || GA) && ((OPT & OPT_GB) == 0 || GB), "K-major gathers");
  static_assert(!(GA && GB), "one gathered operand: the other zero-fills the ragged K");
  static_assert((!GA || OA::CPR == 32) && (!GB || OB::CPR == 32),
                "a gathered load covers two k rows of 256 columns");
  static_assert(!(GA || GB) || KSTEP == 64, "one source row per lane and k-step");
  const bf16_t* a_src[OA::LOADS];
  int a_row[OA::LOADS];
  long a_step[OA::LOADS];
  const bf16_t* b_src[OB::LOADS];
  int b_row[OB::LOADS];
  long b_step[OB::LOADS];
  // source row of row k (< K) of a gathered operand; rows past kv re-read the
  // last valid one (their loads take the zero block)
  auto k_row = [&](const int32_t* rows, int k, int kv) -> int {
    return rows[(size_t)e * p.k_rows_bs + (k < kv ? k : kv - 1)];
  };
  int a_kidx = 0, a_kidx1 = 0, b_kidx = 0, b_kidx1 = 0;
  if constexpr (GA) {
    if (p.kv_a > 0) {
      a_kidx = k_row(p.ka_rows, lane, p.kv_a);
      a_kidx1 = k_row(p.ka_rows, KSTEP + lane, p.kv_a);
    }
  }
  if constexpr (GB) {
    if (p.kv_b > 0) {
      b_kidx = k_row(p.kb_rows, lane, p.kv_b);
      b_kidx1 = k_row(p.kb_rows, KSTEP + lane, p.kv_b);
    }
  }
  // the source row of k row 2 j + (lane >= 32) of the step (j uniform)
  auto pick_row = [&](int kidx, int j) -> int {
    const int lo = __builtin_amdgcn_readlane(kidx, 2 * j);
    const int hi = __builtin_amdgcn_readlane(kidx, 2 * j + 1);
    return lane < 32 ? lo : hi;
  };
#pragma unroll
  for (int q = 0; q < OA::LOADS; ++q) {
    const int id = (wave * OA::LOADS + q) * 64 + lane;
    if constexpr (A_KC) {
      const int row = id / OA::CPR, lc = (id % OA::CPR) ^ kc_swz<KSTEP>(row);
      int r = m0 + row;
      r = r < M ? r : M - 1;
      if (p.a_rows) {
        const int tok = p.a_rows[(size_t)e * p.a_rows_bs + tc.row0 + r];
        a_src[q] = reinterpret_cast<const bf16_t*>(p.A) + (size_t)tok * p.lda + lc * 8;
      } else {
        a_src[q] = Ab + (size_t)r * p.lda + lc * 8;
      }
    } else {
      const int row = id / OA::CPR, lc = (id % OA::CPR) ^ km_swz(row);
      const int col = m0 + lc * 8;   // first column of the chunk
      a_row[q] = row;                // k within the step
      if constexpr (GA) {
        a_src[q] = reinterpret_cast<const bf16_t*>(p.A) + (col < M ? col : M - 8);
      } else {
        a_src[q] = col < M ? Ab + (size_t)row * p.lda + col : g_zero_block;
        a_step[q] = col < M ? (long)KSTEP * p.lda : 0;
      }
    }
  }
#pragma unroll
  for (int q = 0; q < OB::LOADS; ++q) {
    const int id = (wave * OB::LOADS + q) * 64 + lane;
    if constexpr (B_KC) {
      const int row = id / OB::CPR, lc = (id % OB::CPR) ^ kc_swz<KSTEP>(row);
      const bf16_t* rp;
      if constexpr (EPI == EPI_SWIGLU) {
        int r = n0 + row % (BN / 2);
        r = r < p.N ? r : p.N - 1;
        rp = (row < BN / 2 ? Bb : B2b) + (size_t)r * p.ldb;
      } else {
        int r = n0 + row;
        r = r < p.N ? r : p.N - 1;
        rp = Bb + (size_t)r * p.ldb;
      }
      b_src[q] = rp + lc * 8;
    } else {
      const int row = id / OB::CPR, lc = (id % OB::CPR) ^ km_swz(row);
      const int col = n0 + lc * 8;
      b_row[q] = row;
      if constexpr (GB) {
        b_src[q] = reinterpret_cast<const bf16_t*>(p.B) + (col < p.N ? col : p.N - 8);
      } else {
        b_src[q] = col < p.N ? Bb + (size_t)row * p.ldb + col : g_zero_block;
        b_step[q] = col < p.N ? (long)KSTEP * p.ldb : 0;
      }
    }
  }
  // K-major B split at k_split: from row k_split of B to row 0 of B2
  const long b_jump =
      (!B_KC && B2b) ? (long)(((intptr_t)B2b - (intptr_t)(Bb + (size_t)p.k_split * p.ldb)) /
                              (intptr_t)sizeof(bf16_t))
                     : 0;
  // Issues k-step kt; the calls come with kt = 0, 1, 2, ... in order.
  // Loads [lo, hi) of k-step kt (A's loads first, then B's); each load of a
  // k-step is issued exactly once and the k-steps in order.
  // K-major rows past the valid K read the zero block; with full_step (a step
  // known to lie below both kv) the per-load check is skipped.  first: k-step
  // 0 (its successor's source rows are already at hand).
  auto issue_part = [&](int kt, int stage, int lo, int hi, auto full_step, auto first) {
    constexpr bool FULL = decltype(full_step)::value;
    constexpr bool FIRST = decltype(first)::value;
    char* base = smem + stage * STAGE_BYTES;
#pragma unroll
    for (int q = 0; q < OA::LOADS; ++q) {
      if (q < lo || q >= hi) continue;
      const bf16_t* g;
      if constexpr (A_KC) {
        g = a_src[q] + kt * KSTEP;
      } else if constexpr (GA) {
        g = a_src[q] + (size_t)pick_row(a_kidx, wave * OA::LOADS + q) * p.lda;
      } else {
        g = (FULL || kt * KSTEP + a_row[q] < p.kv_a) ? a_src[q] : g_zero_block;
        a_src[q] += a_step[q];
      }
      dma16(g, base + (wave * OA::LOADS + q) * 1024);
    }
    if constexpr (GA) {   // every A load of step kt has gone out: rows of step kt + 1
      if (hi >= OA::LOADS)
        a_kidx = FIRST ? a_kidx1 : k_row(p.ka_rows, (kt + 1) * KSTEP + lane, p.kv_a);
    }
#pragma unroll
    for (int q = 0; q < OB::LOADS; ++q) {
      if (OA::LOADS + q < lo || OA::LOADS + q >= hi) continue;
      const bf16_t* g;
      if constexpr (B_KC) {
        g = b_src[q] + kt * KSTEP;
      } else if constexpr (GB) {
        g = b_src[q] + (size_t)pick_row(b_kidx, wave * OB::LOADS + q) * p.ldb;
      } else {
        g = (FULL || kt * KSTEP + b_row[q] < p.kv_b) ? b_src[q] : g_zero_block;
        // the next step's row; at k_split it continues in row 0 of B2
        const bool jump = (kt + 1) * KSTEP == p.k_split && b_step[q] != 0;
        b_src[q] += b_step[q] + (jump ? b_jump : 0);
      }
      dma16(g, base + OA::BYTES + (wave * OB::LOADS + q) * 1024);
    }
    if constexpr (GB) {
      if (hi >= OA::LOADS + OB::LOADS)
        b_kidx = FIRST ? b_kidx1 : k_row(p.kb_rows, (kt + 1) * KSTEP + lane, p.kv_b);
    }
  };
  auto issue = [&](int kt, int stage, auto first) {
    issue_part(kt, stage, 0, OA::LOADS + OB::LOADS, std::false_type{}, first);
  };

  auto b_lds_col = [&](int ni) -> int {
    if constexpr (EPI == EPI_SWIGLU) {
      constexpr int HWN = BN / 2 / WGN;
      return (ni < NB / 2) ? wn * HWN + ni * 32 : BN / 2 + wn * HWN + (ni - NB / 2) * 32;
    } else {
      return wn * WN + ni * 32;
    }
  };
  // Fragment addressing.  K-contiguous: lane l reads row base + l % 32 of the
  // tile, base a multiple of 32 (uniform over the wave), so the row's chunk
  // swizzle is one per-lane value combined with a uniform one.  K-major: lane l
  // reads 4 columns from column base + lp of k rows km_k and km_k + 4 (of each
  // 16-wide step); with base a multiple of 32 the swizzled chunk is base / 8
  // XOR a per-lane value.  Nothing per fragment is held in registers.
  const int g16 = lane >> 4, j16 = lane & 15;
  const int l31 = lane & 31;
  const int swz_lane = (l31 & 7) ^ (l31 >> 3);
  auto kc_sw = [&](int base) -> int {
    if constexpr (KSTEP == 64) return swz_lane ^ ((base >> 3) & 7);
    else return kc_swz<KSTEP>(base + l31);
  };
  const int km_k = 8 * (g16 >> 1) + (j16 >> 2);   // k row (within a 16-step) of a K-major read
  const int km_lp = 16 * (g16 & 1) + 4 * (j16 & 3);
  const int km_inner = (km_lp & 7) * 2;             // byte offset inside the chunk
  const int km_u = (km_lp >> 3) | km_swz(km_k);     // chunk bits from the lane and the k swizzle

  bf16x8 af[2][MB], bfr[2][NB];
  auto km_frag = [&](const char* tile, int rowbytes, int base, int kk) -> bf16x8 {
    const char* p0 = tile + (kk * 16 + km_k) * rowbytes + (((base >> 3) ^ km_u) << 4) + km_inner;
    const v4i16 lo = ds_read_tr16(p0);
    const v4i16 hi = ds_read_tr16(p0 + 4 * rowbytes);
    const v4i16 both[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, both);
  };
  auto load_frags = [&](int buf, int stage, int kk) {
    const char* sa = smem + stage * STAGE_BYTES;
    const char* sbb = sa + OA::BYTES;
    const int lc = kk * 2 + (lane >> 5);
#pragma unroll
    for (int mi = 0; mi < MB; ++mi) {
      if constexpr (A_KC) {
        const int base = wm * WM + mi * 32;
        af[buf][mi] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(sa + (base + l31) * (KSTEP * 2) +
                                                    ((lc ^ kc_sw(base)) << 4)));
      } else
        af[buf][mi] = km_frag(sa, BM * 2, wm * WM + mi * 32, kk);
    }
#pragma unroll
    for (int ni = 0; ni < NB; ++ni) {
      if constexpr (B_KC) {
        const int base = b_lds_col(ni);
        bfr[buf][ni] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(sbb + (base + l31) * (KSTEP * 2) +
                                                    ((lc ^ kc_sw(base)) << 4)));
      } else {
        bfr[buf][ni] = km_frag(sbb, BN * 2, b_lds_col(ni), kk);
      }
    }
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int mi = 0; mi < MB; ++mi)
#pragma unroll
    for (int ni = 0; ni < NB; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.f;

  // Ring: steps 0..STAGES-1 are issued up front; the end of step kt refills
  // stage kt % STAGES with step kt + STAGES once every wave has read it.  When
  // waiting for step j, the steps issued after it number min(STAGES-1, KT-1-j)
  // for j = 0 and min(STAGES-2, KT-1-j) afterwards (vmcnt counts this wave's
  // outstanding loads, which complete in order).
  auto wait_younger = [&](int younger) {
    if (younger >= 3) __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * LOADS));
    else if (younger == 2) __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LOADS));
    else if (younger == 1) __builtin_amdgcn_s_waitcnt(vmcnt_imm(LOADS));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  };
  static_assert(3 * LOADS <= 63, "vmcnt range");
  const int KT = (p.K + KSTEP - 1) / KSTEP;
  if (KT > 0) issue(0, 0, std::true_type{});
#pragma unroll
  for (int s2 = 1; s2 < STAGES; ++s2)
    if (s2 < KT) issue(s2, s2, std::false_type{});
  if (KT > 0) {
    wait_younger(KT - 1 < STAGES - 1 ? KT - 1 : STAGES - 1);
    __builtin_amdgcn_s_barrier();
    load_frags(0, 0, 0);
  }
  constexpr int NMF = MB * NB;
  auto mfma_range = [&](int cur, int lo, int hi) {
#pragma unroll
    for (int q = 0; q < NMF; ++q) {
      if (q < lo || q >= hi) continue;
      const int mi = q / NB, ni = q % NB;
      // B fragment first: the 32 x 32 block comes out transposed, each lane
      // holding four consecutive output columns of one row (16-byte staging
      // writes in the epilogue)
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cur][ni], af[cur][mi],
                                                              acc[mi][ni], 0, 0, 0);
    }
  };


  // Fragment-read instructions per 16-wide k step (a K-major fragment takes
  // two).  Inside a stage the MFMAs on the current fragments alternate with
  // the reads of the next ones (one MFMA, one read, ...).  At a stage end: half
  // the MFMAs, then this wave's waits and the barrier, then the other half
  // alternating with the refill's DMA and the next stage's first reads.  Steps
  // with and without a refill (or a refill's second half) run in separate
  // straight-line segments, so that no branch splits an interleaved group.
  constexpr int NRD = MB * (A_KC ? 1 : 2) + NB * (B_KC ? 1 : 2);
  constexpr int HALF = NMF / 2;
  // A stage's refill is issued in two parts: DMA_HEAD loads after the barrier
  // that frees the stage, the rest in the next step's first sub-step (two
  // stages only: the wait at every step end is then for all outstanding loads).
  constexpr bool SPLIT_DMA = STAGES == 2 && KK > 1;
  // (measured: half after the barrier and half in one sub-step beats a quarter
  // then three sub-steps, none after the barrier, or two tail sub-steps)
  constexpr int DMA_HEAD = SPLIT_DMA ? LOADS / 2 : LOADS;
  constexpr int TAIL_SUBS = 1;
  constexpr int TAIL_PER = (LOADS - DMA_HEAD + TAIL_SUBS - 1) / TAIL_SUBS;
  auto kstep = [&](int kt, auto refill, auto tail_part, auto full_refill) {
    constexpr bool RF = decltype(refill)::value;
    constexpr bool TAIL = SPLIT_DMA && decltype(tail_part)::value;
    const int stage = kt % STAGES;
    // TAIL: the second part of the previous step's refill goes out in this
    // step's first 16-wide sub-step (it still has a whole step to land)
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const int cur = kk & 1;
      if (kk < TAIL_SUBS && TAIL) {
        mfma_range(cur, 0, NMF);
        {
          const int q0 = DMA_HEAD + kk * TAIL_PER;
          const int q1 = q0 + TAIL_PER < LOADS ? q0 + TAIL_PER : LOADS;
          issue_part(kt - 1 + STAGES, (kt - 1) % STAGES, q0, q1, full_refill,
                     std::false_type{});
        }
        load_frags(cur ^ 1, stage, kk + 1);
#pragma unroll
        for (int q = 0; q < NMF; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                 // MFMA
          __builtin_amdgcn_sched_group_barrier(0x010, (TAIL_PER + NMF - 1) / NMF, 0);         // DMA
          __builtin_amdgcn_sched_group_barrier(0x100, (NRD + NMF - 1) / NMF, 0);             // LDS read
        }
        __builtin_amdgcn_sched_barrier(0);
      } else if (kk + 1 < KK) {
        mfma_range(cur, 0, NMF);
        load_frags(cur ^ 1, stage, kk + 1);
#pragma unroll
        for (int q = 0; q < NRD; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NMF > NRD ? NMF - NRD : 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      } else {
        mfma_range(cur, 0, HALF);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): this wave's reads are done
        if (kt + 1 < KT) wait_younger(KT - 2 - kt < STAGES - 2 ? KT - 2 - kt : STAGES - 2);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        mfma_range(cur, HALF, NMF);
        if constexpr (RF) issue_part(kt + STAGES, stage, 0, DMA_HEAD, full_refill, std::false_type{});
        // after the final step this reads a stale stage, harmlessly
        load_frags(cur ^ 1, (kt + 1) % STAGES, 0);
#pragma unroll
        for (int q = 0; q < HALF; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                           // MFMA
          if constexpr (RF) __builtin_amdgcn_sched_group_barrier(0x010, (DMA_HEAD + HALF - 1) / HALF, 0);  // DMA
          __builtin_amdgcn_sched_group_barrier(0x100, (NRD + HALF - 1) / HALF, 0);     // LDS read
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  // Straight-line segments, so that no branch splits an interleaved group:
  // step 0 (refill, no tail), steps that refill and finish the previous
  // refill, the step that only finishes it, then the last steps.
  {
    using T_ = std::true_type;
    using F_ = std::false_type;
    int kt = 0;
    // refills of the steps below KT - 1 skip the K-major row check when
    // every such step lies below both kv (the usual case: only the last step
    // is ragged); with a split refill, so does the second half of such a
    // refill in the next step
    const bool full_ok = p.kv_a >= (KT - 1) * KSTEP && p.kv_b >= (KT - 1) * KSTEP;
    const int n_full = full_ok ? KT - STAGES - 1 : 0;
    if constexpr (SPLIT_DMA) {
      if (KT > STAGES) {
        kstep(0, T_{}, F_{}, F_{});
        if constexpr (!A_KC || !B_KC)
          for (kt = 1; kt < n_full; ++kt) kstep(kt, T_{}, T_{}, T_{});
        for (kt = kt > 1 ? kt : 1; kt + STAGES < KT; ++kt) kstep(kt, T_{}, T_{}, F_{});
        kstep(kt, F_{}, T_{}, F_{});
        ++kt;
      }
    } else {
      for (; kt < n_full; ++kt) kstep(kt, T_{}, F_{}, T_{});
      for (; kt + STAGES < KT; ++kt) kstep(kt, T_{}, F_{}, F_{});
    }
    for (; kt < KT; ++kt) kstep(kt, F_{}, F_{}, F_{});
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  __syncthreads();

  // ---- epilogue: stage 32-row slices of the wave tile through LDS ----
  // The accumulators of a slice go to LDS (fp32, row-major); then every lane
  // reads its 16-byte output chunks back in batches of EQ with no branch
  // between the reads (their LDS addresses always lie inside the slice), and
  // only then converts and stores the chunks that fall inside the matrix.
  float* stage_f = reinterpret_cast<float*>(smem) + wave * 32 * SLD;
  constexpr int HW = WN / 2;                                    // SwiGLU: outputs per row
  constexpr int CPR = (EPI == EPI_SWIGLU) ? HW / 8 : WN / 8;    // chunks per slice row
  constexpr int NCH = 32 * CPR;                                 // chunks per slice
  constexpr int NQ = (NCH + 63) / 64;                           // chunks per lane
  constexpr int EQ = (EPI == EPI_SWIGLU_BWD && NQ > 4) ? 4 : NQ;  // chunks per batch
  static_assert(NQ % EQ == 0, "whole batches");
  static_assert(EPI != EPI_SWIGLU_BWD || (CPR == 16 && NCH % 64 == 0),
                "the chunks of a 128-column block of a row sit in one 16-lane DPP row");
  // SwiGLU backward: the H1/H3 chunks of slice 0 are loaded before it is
  // staged; those of slice mi + 1 batch by batch as slice mi's batches finish
  // with theirs, so their latency overlaps slice mi's work (rows or columns past
  // the matrix read element 0 and are not stored).
  constexpr int HQ = (EPI == EPI_SWIGLU_BWD) ? NQ : 1;
  u32x4 h1raw[2][HQ], h3raw[2][HQ];
  auto load_h = [&](int mi, int q) {
    if constexpr (EPI == EPI_SWIGLU_BWD) {
      const int mb = m0 + wm * WM + mi * 32;
      const int c = lane + q * 64;
      const int m = mb + c / CPR, n = n0 + wn * WN + (c % CPR) * 8;
      const size_t ho = (m < M && n < p.N) ? tc.h_off + (size_t)m * p.ldh + n : 0;
      // read once: streaming loads
      h1raw[mi & 1][q] =
          __builtin_nontemporal_load(reinterpret_cast<const u32x4*>((const bf16_t*)p.H1 + ho));
      h3raw[mi & 1][q] =
          __builtin_nontemporal_load(reinterpret_cast<const u32x4*>((const bf16_t*)p.H3 + ho));
    }
  };
  if constexpr (EPI == EPI_SWIGLU_BWD) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) load_h(0, q);
  }
#pragma unroll
  for (int mi = 0; mi < MB; ++mi) {
    const int mbase = m0 + wm * WM + mi * 32;
    // acc[mi][ni][4 g + i] is row lane % 32 of the slice, column
    // 32 ni + 8 g + 4 (lane / 32) + i
#pragma unroll
    for (int ni = 0; ni < NB; ++ni)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(&stage_f[(lane & 31) * SLD + ni * 32 + g * 8 + (lane >> 5) * 4]) =
            f32x4{acc[mi][ni][4 * g], acc[mi][ni][4 * g + 1], acc[mi][ni][4 * g + 2],
                  acc[mi][ni][4 * g + 3]};
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int q0 = 0; q0 < NQ; q0 += EQ) {
      // chunk q of this lane: slice row c / CPR, columns (c % CPR) * 8 .. + 7
      float v[EQ][8], v3[EPI == EPI_SWIGLU ? EQ : 1][8];
#pragma unroll
      for (int e = 0; e < EQ; ++e) {
        int c = lane + (q0 + e) * 64;
        c = c < NCH ? c : NCH - 1;
        const float* src = stage_f + (c / CPR) * SLD + (c % CPR) * 8;
#pragma unroll
        for (int u = 0; u < 8; ++u) v[e][u] = src[u];
        if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
          for (int u = 0; u < 8; ++u) v3[e][u] = src[HW + u];
        }
      }
      float dots[EPI == EPI_SWIGLU_BWD ? EQ : 1];
#pragma unroll
      for (int e = 0; e < (EPI == EPI_SWIGLU_BWD ? EQ : 1); ++e) dots[e] = 0.f;
#pragma unroll
      for (int e = 0; e < EQ; ++e) {
        const int q = q0 + e;
        const int c = lane + q * 64;
        const int m = mbase + c / CPR;
        const int n = n0 + wn * (EPI == EPI_SWIGLU ? HW : WN) + (c % CPR) * 8;
        // the row factor, from the lane that holds it (every lane takes part)
        float g = 1.f;
        if constexpr (GATED) {
          const int rr = (c < NCH ? c : NCH - 1) / CPR;   // row within the slice
          g = __shfl(gate_r[(mi * 32) / 64], (mi * 32) % 64 + rr, 64);
        }
        if (c >= NCH || m >= M || n >= p.N) continue;
        if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_ADD) {
          const bool second = m >= p.c_split;
          const int mm = second ? m - p.c_split : m;
          const size_t off = tc.c_off + (size_t)mm * p.ldc + n;
          if constexpr (OUT_F32) {
            float* dst = (float*)(second ? p.C2 : p.C) + off;
            if constexpr (EPI == EPI_STORE_ADD) {
              float old[8];
              Elem<float>::load8(dst, old);
#pragma unroll
              for (int u = 0; u < 8; ++u) v[e][u] += old[u];
            }
            Elem<float>::store8(dst, v[e]);
          } else {
            bf16_t* dst = (bf16_t*)(second ? p.C2 : p.C) + off;
            if constexpr (EPI == EPI_STORE_ADD) {
              float old[8];
              Elem<bf16_t>::load8(dst, old);
#pragma unroll
              for (int u = 0; u < 8; ++u) v[e][u] += old[u];
            }
            Elem<bf16_t>::store8(dst, v[e]);
          }
        } else if constexpr (EPI == EPI_SWIGLU) {
          float a[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) a[u] = silu_f(v[e][u]) * v3[e][u] * g;
          Elem<bf16_t>::store8((bf16_t*)p.C + tc.c_off + (size_t)m * p.ldc + n, a);
          if (p.H1) {
            const size_t ho = tc.h_off + (size_t)m * p.ldh + n;
            Elem<bf16_t>::store8((bf16_t*)p.H1 + ho, v[e]);
            Elem<bf16_t>::store8((bf16_t*)p.H3 + ho, v3[e]);
          }
        } else {  // EPI_SWIGLU_BWD
          float d1[8], d3[8];
          float dot = 0.f;
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const uint32_t w1 = h1raw[mi & 1][q][u >> 1], w3 = h3raw[mi & 1][q][u >> 1];
            const float h1 = bf16_to_f32((u & 1) ? (w1 >> 16) : (w1 & 0xffffu));
            const float h3 = bf16_to_f32((u & 1) ? (w3 >> 16) : (w3 & 0xffffu));
            const float da = v[e][u] * g;
            const float sg = sigmoid_f(h1);
            const float s1 = h1 * sg;   // SiLU(h1)
            d3[u] = da * s1;
            d1[u] = da * h3 * sg * (1.0f + h1 * (1.0f - sg));
            dot = fmaf(da, s1 * h3, dot);
          }
          dots[e] = dot;
          const size_t off = tc.c_off + (size_t)m * p.ldc + n;
          Elem<bf16_t>::store8((bf16_t*)p.C + off, d1);
          Elem<bf16_t>::store8((bf16_t*)p.C2 + off, d3);
        }
      }
      if constexpr (EPI == EPI_SWIGLU_BWD) {
        // gate-gradient partials: the 16 lanes of a DPP row hold the chunks of
        // one row's 128-column block (columns past N hold clamped duplicates
        // and count as zero)
        if (p.dsp) {
#pragma unroll
          for (int e = 0; e < EQ; ++e) {
            const int c = lane + (q0 + e) * 64;
            const int m = mbase + c / CPR;
            const int n = n0 + wn * WN + (c % CPR) * 8;
            const float t = row16_sum(n < p.N ? dots[e] : 0.f);
            if ((lane & 15) == 0 && m < M && n < p.N)
              p.dsp[((size_t)tc.e * p.M + m) * p.dsp_ld + (n >> 7)] = t;
          }
        }
        if (mi + 1 < MB) {
#pragma unroll
          for (int e = 0; e < EQ; ++e) load_h(mi + 1, q0 + e);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// smem bytes of gemm_dma_tile's configuration
template <int BM, int BN, int WGM, int WGN, int KSTEP, int STAGES, bool A_KC, bool B_KC>
constexpr int dma_smem_bytes() {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int STAGE_BYTES = (BM + BN) * KSTEP * 2;
  constexpr int STAGE_EPI = NT / 64 * 32 * (BN / WGN + 4) * 4;
  return STAGES * STAGE_BYTES > STAGE_EPI ? STAGES * STAGE_BYTES : STAGE_EPI;
}

// One output tile per workgroup; consecutive tile ids (same expert) are kept
// on one XCD so that its L2 serves their shared A rows and B columns.
template <int BM, int BN, int WGM, int WGN, int KSTEP, int STAGES, bool A_KC, bool B_KC, int EPI,
          bool OUT_F32, int TAG, int OPT>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void gemm_dma_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(1024)))
  char smem[dma_smem_bytes<BM, BN, WGM, WGN, KSTEP, STAGES, A_KC, B_KC>()];
  TileCoord tc;
  int rem, MT;
  if (p.var_rows) {
    // the tile count is known only on the device: the grid is an upper bound,
    // and the XCD-contiguous numbering uses the actual count
    const int total = p.var_tiles[p.batches];
    const int per_xcd = (total + 7) >> 3;
    const int j = blockIdx.x >> 3;
    if (j >= per_xcd) return;
    const int t = (blockIdx.x & 7) * per_xcd + j;
    if (t >= total) return;
    int lo = 0, hi = p.batches;          // var_tiles[lo] <= t < var_tiles[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (p.var_tiles[mid] <= t) lo = mid; else hi = mid;
    }
    const int row0 = p.var_rows[lo];
    tc.e = lo;
    tc.row0 = row0;
    tc.M = p.var_rows[lo + 1] - row0;
    MT = (tc.M + BM - 1) / BM;
    rem = t - p.var_tiles[lo];
    tc.a_off = (size_t)row0 * p.lda;
    tc.c_off = (size_t)row0 * p.ldc;
    tc.h_off = (size_t)row0 * p.ldh;
  } else {
    const int t = xcd_tile_id(blockIdx.x, gridDim.x);
    if (t >= p.batches * p.MT * p.NT) return;
    const int per_b = p.MT * p.NT;
    tc.e = t / per_b;
    tc.row0 = 0;
    tc.M = p.M;
    MT = p.MT;
    rem = t - tc.e * per_b;
    tc.a_off = (size_t)tc.e * p.a_bs;
    tc.c_off = (size_t)tc.e * p.c_bs;
    tc.h_off = (size_t)tc.e * p.h_bs;
  }
  // Tiles go in groups of GROUP_M row blocks, row block fastest inside a
  // group: the workgroups resident on one XCD then share few A row blocks and
  // B column blocks at a time (fewer L2 misses than a full column of row blocks).
  constexpr int GROUP_M = 3;
  const int grp = rem / (GROUP_M * p.NT), in_grp = rem - grp * GROUP_M * p.NT;
  const int gm = (MT - grp * GROUP_M) < GROUP_M ? (MT - grp * GROUP_M) : GROUP_M;
  tc.mt = grp * GROUP_M + in_grp % gm;
  tc.nt = in_grp / gm;
  tc.MT = MT;
  tc.NT = p.NT;
  gemm_dma_tile<BM, BN, WGM, WGN, KSTEP, STAGES, A_KC, B_KC, EPI, OUT_F32, OPT>(p, tc, smem);
}

// OPT: the options of the instantiation; the pointers of each option must be
// set exactly when it is.
template <int BM, int BN, int WGM, int WGN, int KSTEP, int STAGES, bool A_KC, bool B_KC, int EPI,
          bool OUT_F32, int TAG, int OPT = 0>
hipError_t run_dma(GemmParams p, hipStream_t st) {
  if (((OPT & OPT_GA) != 0) != (p.ka_rows != nullptr) ||
      ((OPT & OPT_GB) != 0) != (p.kb_rows != nullptr))
    return hipErrorInvalidValue;
  p.MT = (p.M + BM - 1) / BM;
  p.NT = (EPI == EPI_SWIGLU) ? (p.N + BN / 2 - 1) / (BN / 2) : (p.N + BN - 1) / BN;
  const long ntile = (long)p.batches * p.MT * p.NT;
  if (ntile == 0) return hipSuccess;
  const long grid = (ntile + 7) / 8 * 8;
  gemm_dma_kernel<BM, BN, WGM, WGN, KSTEP, STAGES, A_KC, B_KC, EPI, OUT_F32, TAG, OPT>
      <<<dim3((unsigned)grid), 64 * WGM * WGN, 0, st>>>(p);
  return hipGetLastError();
}

// Variable rows per batch (p.var_rows / p.var_tiles on the device): the grid
// covers max_rows rows in total plus one partial row block per batch.
template <int BM, int BN, int WGM, int WGN, int KSTEP, int STAGES, bool A_KC, bool B_KC, int EPI,
          bool OUT_F32, int TAG>
hipError_t run_dma_var(GemmParams p, long max_rows, hipStream_t st) {
  p.MT = 0;
  p.NT = (EPI == EPI_SWIGLU) ? (p.N + BN / 2 - 1) / (BN / 2) : (p.N + BN - 1) / BN;
  const long ntile = ((max_rows + BM - 1) / BM + p.batches) * p.NT;
  if (ntile == 0 || p.batches == 0) return hipSuccess;
  const long grid = (ntile + 7) / 8 * 8;
  gemm_dma_kernel<BM, BN, WGM, WGN, KSTEP, STAGES, A_KC, B_KC, EPI, OUT_F32, TAG, 0>
      <<<dim3((unsigned)grid), 64 * WGM * WGN, 0, st>>>(p);
  return hipGetLastError();
}

// Row blocks of the forward expert products: 192 when they pad the expert
// buffers enough less than blocks of 256 (one 2048-token sequence at c(t) =
// 12 - 8t has 373 rows per expert: 384 computed instead of 512), 128 for
// buffers of at most 128 rows (that sequence at t = 1).  A 192-row tile (96 x 64
// per wave) does three quarters of a 256-row tile's work in 0.875 of its time,
// a 128-row tile (64 x 64 per wave) half the work in 0.74 of the time (W1/W3),
// so a computed row costs 7/6 and 1.47 times as much.  Every choice keeps an
// expert's row blocks side by side on one XCD, so its weights are fetched once.
int fwd_block_rows(int M) {
  if (M <= 128) return 128;
  const long r256 = (M + 255) / 256 * 256L, r192 = (M + 191) / 192 * 192L;
  return r192 * 7 < r256 * 6 ? 192 : 256;
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
  // rows of this batch: uniform (M), or [var_rows[e], var_rows[e+1]) of packed buffers
  int M = p.M;
  size_t a_off = (size_t)e * p.a_bs, c_off = (size_t)e * p.c_bs, h_off = (size_t)e * p.h_bs;
  if (p.var_rows) {
    const int row0 = p.var_rows[e];
    M = p.var_rows[e + 1] - row0;
    a_off = (size_t)row0 * p.lda;
    c_off = (size_t)row0 * p.ldc;
    h_off = (size_t)row0 * p.ldh;
  }
  if (m0 >= M) return;
  const float* A = (const float*)p.A + a_off;
  const float* B = (const float*)p.B + (size_t)e * p.b_bs;
  const float* B2 = p.B2 ? (const float*)p.B2 + (size_t)e * p.b_bs : nullptr;
  float acc[4][4] = {}, acc3[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += FK) {
    for (int c = tid; c < FK * FT; c += 256) {
      const int kk = c / FT, r = c % FT;
      const int k = k0 + kk, m = m0 + r, n = n0 + r;
      float va = 0.f, vb = 0.f, vb3 = 0.f;
      if (k < p.kv_a && m < M) va = a_kc ? A[(size_t)m * p.lda + k] : A[(size_t)k * p.lda + m];
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
  float dsum[4] = {0.f, 0.f, 0.f, 0.f};   // SwiGLU backward: gate-gradient partials per row
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + jj;
      if (m >= M || n >= p.N) continue;
      if (EPI == EPI_STORE || EPI == EPI_STORE_ADD) {
        const bool second = m >= p.c_split;
        const int mm = second ? m - p.c_split : m;
        float* dst = (float*)(second ? p.C2 : p.C) + c_off + (size_t)mm * p.ldc + n;
        *dst = (EPI == EPI_STORE_ADD) ? *dst + acc[i][jj] : acc[i][jj];
      } else if (EPI == EPI_SWIGLU) {
        const float h1 = acc[i][jj], h3 = acc3[i][jj];
        const float g = p.gate ? p.gate[(size_t)e * p.gate_bs + m] : 1.f;
        ((float*)p.C)[c_off + (size_t)m * p.ldc + n] = silu_f(h1) * h3 * g;
        if (p.H1) {
          const size_t ho = h_off + (size_t)m * p.ldh + n;
          ((float*)p.H1)[ho] = h1;
          ((float*)p.H3)[ho] = h3;
        }
      } else {
        const size_t ho = h_off + (size_t)m * p.ldh + n;
        const float h1 = ((const float*)p.H1)[ho], h3 = ((const float*)p.H3)[ho];
        const float da = acc[i][jj] * (p.gate ? p.gate[(size_t)e * p.gate_bs + m] : 1.f);
        const float sg = sigmoid_f(h1);
        const size_t off = c_off + (size_t)m * p.ldc + n;
        ((float*)p.C)[off] = da * h3 * sg * (1.0f + h1 * (1.0f - sg));
        ((float*)p.C2)[off] = da * h1 * sg;
        dsum[i] = fmaf(da, h1 * sg * h3, dsum[i]);
      }
    }
  if (EPI == EPI_SWIGLU_BWD && p.dsp) {
    // the 16 threads of a row (tx, consecutive lanes) hold its 64 columns
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float t = dsum[i];
      t += __shfl_xor(t, 1, 64);
      t += __shfl_xor(t, 2, 64);
      t += __shfl_xor(t, 4, 64);
      t += __shfl_xor(t, 8, 64);
      const int m = m0 + ty * 4 + i;
      if (tx == 0 && m < M) p.dsp[((size_t)e * p.M + m) * p.dsp_ld + blockIdx.x] = t;
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

// deterministic split-K reduction into the storage dtype, with the output's
// row split: row r < c_split goes to C, the others to C2 at r - c_split.
template <typename T>
__global__ void splitk_store_kernel(const float* __restrict__ part, int splits, int M, int N,
                                    int c_split, T* __restrict__ C, T* __restrict__ C2, int ldc) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)M * N) return;
  const int r = (int)(i / N), c = (int)(i % N);
  float s = 0.f;
  for (int q = 0; q < splits; ++q) s += part[(size_t)q * M * N + i];
  if (r < c_split) Elem<T>::store1(C + (size_t)r * ldc + c, s);
  else Elem<T>::store1(C2 + (size_t)(r - c_split) * ldc + c, s);
}

}  // namespace

// ---------------------------------------------------------------- launchers

int dsp_parts(int dtype, int h) { return dtype == DT_F32 ? (h + 63) / 64 : (h + 127) / 128; }

hipError_t launch_gemm_w13(int dtype, const void* Xe, const void* W1, const void* W3, void* A,
                           void* H1, void* H3, int E, int M, int d, int h, hipStream_t st,
                           bool shared, const int32_t* rows, const float* gate) {
  GemmParams p = base_params();
  p.gate = gate; p.gate_bs = M;
  p.A = Xe; p.a_bs = (long)M * d; p.lda = d;
  if (rows) {   // Xe is X itself, row m of expert e is X[rows[e M + m]]
    p.a_bs = 0; p.a_rows = rows; p.a_rows_bs = M;
  }
  p.B = W1; p.B2 = W3; p.b_bs = (long)h * d; p.ldb = d;
  p.M = M; p.N = h; p.K = d; p.kv_a = d; p.kv_b = d; p.batches = E;
  p.C = A; p.c_bs = (long)M * h; p.ldc = h;
  p.H1 = H1; p.H3 = H3; p.h_bs = (long)M * h; p.ldh = h;
  if (M == 0) return hipSuccess;
  if (dtype == DT_F32) {
    if (rows) return hipErrorInvalidValue;   // fp32 reads a gathered Xe
    return run_f32<EPI_SWIGLU>(p, 1, 1, st);
  }
  if (shared) {
    if (rows) return hipErrorInvalidValue;   // the shared experts read X as is
    return run_dma<256, 256, 2, 4, 64, 2, true, true, EPI_SWIGLU, false, G_SH_W13>(p, st);
  }
  switch (fwd_block_rows(M)) {
    case 128: return run_dma<128, 256, 2, 4, 64, 2, true, true, EPI_SWIGLU, false, G_W13>(p, st);
    case 192: return run_dma<192, 256, 2, 4, 64, 2, true, true, EPI_SWIGLU, false, G_W13>(p, st);
    default: return run_dma<256, 256, 2, 4, 64, 2, true, true, EPI_SWIGLU, false, G_W13>(p, st);
  }
}

hipError_t launch_gemm_w2(int dtype, const void* A, const void* W2, void* O, int E, int M, int d,
                          int h, hipStream_t st, bool shared) {
  GemmParams p = base_params();
  p.A = A; p.a_bs = (long)M * h; p.lda = h;
  p.B = W2; p.b_bs = (long)d * h; p.ldb = h;
  p.M = M; p.N = d; p.K = h; p.kv_a = h; p.kv_b = h; p.batches = E;
  p.C = O; p.c_bs = (long)M * d; p.ldc = d;
  if (M == 0) return hipSuccess;
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 1, 1, st);
  if (shared) return run_dma<256, 256, 4, 2, 64, 2, true, true, EPI_STORE, false, G_SH_W2>(p, st);
  switch (fwd_block_rows(M)) {
    case 128: return run_dma<128, 256, 2, 4, 64, 2, true, true, EPI_STORE, false, G_W2>(p, st);
    case 192: return run_dma<192, 256, 2, 4, 64, 2, true, true, EPI_STORE, false, G_W2>(p, st);
    default: return run_dma<256, 256, 4, 2, 64, 2, true, true, EPI_STORE, false, G_W2>(p, st);
  }
}

hipError_t launch_gemm_dA(int dtype, const void* dO, const void* W2, const void* H1,
                          const void* H3, void* dH, int E, int M, int d, int h, hipStream_t st,
                          bool shared, float* dsp, const int32_t* rows, const float* gate) {
  // dA[m, n] = g_m sum_k dO[m, k] W2[k, n]  (k over d, n over h); epilogue -> dH1, dH3
  GemmParams p = base_params();
  p.A = dO; p.a_bs = (long)M * d; p.lda = d;
  if (rows) {   // dO is dY itself, row m of expert e is dY[rows[e M + m]]
    p.a_bs = 0; p.a_rows = rows; p.a_rows_bs = M;
  }
  p.gate = gate; p.gate_bs = M;
  p.B = W2; p.b_bs = (long)d * h; p.ldb = h;
  p.M = M; p.N = h; p.K = d; p.kv_a = d; p.kv_b = d; p.batches = E;
  const size_t esz = dtype == DT_F32 ? 4 : 2;
  p.C = dH; p.C2 = (char*)dH + (size_t)h * esz; p.c_bs = (long)M * 2 * h; p.ldc = 2 * h;
  p.H1 = (void*)H1; p.H3 = (void*)H3; p.h_bs = (long)M * h; p.ldh = h;
  p.dsp = dsp; p.dsp_ld = dsp_parts(dtype, h);
  if (M == 0) return hipSuccess;
  if (dtype == DT_F32) {
    if (rows) return hipErrorInvalidValue;   // fp32 reads a gathered dO
    return run_f32<EPI_SWIGLU_BWD>(p, 1, 0, st);
  }
  if (shared && rows) return hipErrorInvalidValue;
  // B = W2 K-major: B(n, k) = W2[k, n]
  if (shared)
    return run_dma<256, 256, 4, 2, 64, 2, true, false, EPI_SWIGLU_BWD, false, G_SH_DA>(p, st);
  return run_dma<256, 256, 4, 2, 64, 2, true, false, EPI_SWIGLU_BWD, false, G_DA>(p, st);
}

hipError_t launch_gemm_dXe(int dtype, const void* dH, const void* W1, const void* W3, void* dXe,
                           int E, int M, int d, int h, hipStream_t st, bool shared) {
  // dXe[m, n] = sum_k dH[m, k] W13[k, n], k < h from W1, k >= h from W3
  GemmParams p = base_params();
  p.A = dH; p.a_bs = (long)M * 2 * h; p.lda = 2 * h;
  p.B = W1; p.B2 = W3; p.b_bs = (long)h * d; p.ldb = d; p.k_split = h;
  p.M = M; p.N = d; p.K = 2 * h; p.kv_a = 2 * h; p.kv_b = 2 * h; p.batches = E;
  p.C = dXe; p.c_bs = (long)M * d; p.ldc = d;
  if (M == 0) return hipSuccess;
  if (dtype == DT_F32) return shared ? run_f32<EPI_STORE_ADD>(p, 1, 0, st)
                                     : run_f32<EPI_STORE>(p, 1, 0, st);
  // bf16: B K-major, rows k >= h from W3 (h is a multiple of the k-step); the
  // shared experts' input gradient is added to dX
  if (h % 64 != 0) return hipErrorInvalidValue;
  if (shared)
    return run_dma<256, 256, 4, 2, 64, 2, true, false, EPI_STORE_ADD, false, G_SH_DXE>(p, st);
  return run_dma<256, 256, 4, 2, 64, 2, true, false, EPI_STORE, false, G_DXE>(p, st);
}

hipError_t launch_gemm_dW2(int dtype, const void* dO, const void* A, void* dW2, int E, int M,
                           int d, int h, hipStream_t st, const int32_t* rows) {
  // dW2[m, n] = sum_k dO[k, m] A[k, n]  (m over d, n over h, k over the M expert rows)
  GemmParams p = base_params();
  p.A = dO; p.a_bs = (long)M * d; p.lda = d;
  p.B = A; p.b_bs = (long)M * h; p.ldb = h;
  p.M = d; p.N = h; p.K = M; p.kv_a = M; p.kv_b = M; p.batches = E;
  p.C = dW2; p.c_bs = (long)d * h; p.ldc = h;
  if (rows) {   // dO is dY itself, row k of expert e is dY[rows[e M + k]]
    if (dtype == DT_F32) return hipErrorInvalidValue;
    p.a_bs = 0; p.ka_rows = rows; p.k_rows_bs = M;
    return run_dma<256, 256, 4, 2, 64, 2, false, false, EPI_STORE, false, G_DW2, OPT_GA>(p, st);
  }
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 0, 0, st);
  return run_dma<256, 256, 4, 2, 64, 2, false, false, EPI_STORE, false, G_DW2>(p, st);
}

hipError_t launch_gemm_dW13(int dtype, const void* dH, const void* Xe, void* dW1, void* dW3,
                            int E, int M, int d, int h, hipStream_t st, const int32_t* rows) {
  // [dW1; dW3][m, n] = sum_k dH[k, m] Xe[k, n]  (m over 2h, n over d)
  GemmParams p = base_params();
  p.A = dH; p.a_bs = (long)M * 2 * h; p.lda = 2 * h;
  p.B = Xe; p.b_bs = (long)M * d; p.ldb = d;
  p.M = 2 * h; p.N = d; p.K = M; p.kv_a = M; p.kv_b = M; p.batches = E;
  p.C = dW1; p.C2 = dW3; p.c_split = h; p.c_bs = (long)h * d; p.ldc = d;
  if (rows) {   // Xe is X itself, row k of expert e is X[rows[e M + k]]
    if (dtype == DT_F32) return hipErrorInvalidValue;
    p.b_bs = 0; p.kb_rows = rows; p.k_rows_bs = M;
    return run_dma<256, 256, 4, 2, 64, 2, false, false, EPI_STORE, false, G_DW13, OPT_GB>(p, st);
  }
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 0, 0, st);
  return run_dma<256, 256, 4, 2, 64, 2, false, false, EPI_STORE, false, G_DW13>(p, st);
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
  return run_dma<256, 256, 4, 2, 64, 2, true, false, EPI_STORE, false, G_ROUTER_DX>(p, st);
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
    else err = run_dma<128, 256, 2, 4, 64, 2, false, false, EPI_STORE, true, G_ROUTER_DWG>(p, st);
  } else {
    GemmParams p1 = p;
    p1.batches = splits - 1; p1.kv_a = chunk; p1.kv_b = chunk;
    err = (splits > 1) ? ((dtype == DT_F32) ? run_f32<EPI_STORE>(p1, 0, 0, st)
                                            : run_dma<128, 256, 2, 4, 64, 2, false, false, EPI_STORE, true, G_ROUTER_DWG>(p1, st))
                       : hipSuccess;
    if (err != hipSuccess) return err;
    GemmParams p2 = p;
    const long ao = (long)(splits - 1) * p.a_bs, bo = (long)(splits - 1) * p.b_bs;
    p2.A = (const char*)p.A + ao * ((dtype == DT_F32) ? 4 : 2);
    p2.B = (const char*)p.B + bo * ((dtype == DT_F32) ? 4 : 2);
    p2.C = part + (size_t)(splits - 1) * E * d;
    p2.batches = 1; p2.kv_a = last; p2.kv_b = last;
    err = (dtype == DT_F32) ? run_f32<EPI_STORE>(p2, 0, 0, st)
                            : run_dma<128, 256, 2, 4, 64, 2, false, false, EPI_STORE, true, G_ROUTER_DWG>(p2, st);
  }
  if (err != hipSuccess) return err;
  const long n = (long)E * d;
  splitk_reduce_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(part, dWg, splits, n, E, E, d);
  return hipGetLastError();
}

int wgrad_splits(int M, int N, int K) {
  const int tiles = ((M + 255) / 256) * ((N + 255) / 256);
  int s = (512 + tiles - 1) / tiles;
  const int maxs = (K + 255) / 256;
  if (s > maxs) s = maxs;
  return s < 1 ? 1 : s;
}

namespace {

// C[m, n] = sum_k A[k, m] B[k, n] over K rows (both operands K-major), split
// over the rows into `splits` fp32 partials (part [splits, M, N]) added in a
// fixed order into C (rows < c_split) and C2 (the others).  One batch only.
template <int TAG>
hipError_t run_wgrad_splitk(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                            void* C, void* C2, int c_split, int ldc, float* part, int splits,
                            hipStream_t st) {
  if (K == 0 || splits < 1) {
    // no rows: the gradient is zero
    hipError_t e = launch_zero(C, (size_t)(c_split < M ? c_split : M) * ldc * 2, st);
    if (e != hipSuccess || c_split >= M) return e;
    return launch_zero(C2, (size_t)(M - c_split) * ldc * 2, st);
  }
  const int chunk = ((K + splits - 1) / splits + 63) / 64 * 64;
  const int full = K / chunk;                 // splits with chunk rows
  const int last = K - full * chunk;          // rows of the final short split (may be 0)
  const int nsplit = full + (last > 0 ? 1 : 0);
  GemmParams p = base_params();
  p.A = A; p.a_bs = (long)chunk * lda; p.lda = lda;
  p.B = B; p.b_bs = (long)chunk * ldb; p.ldb = ldb;
  p.M = M; p.N = N; p.K = chunk; p.kv_a = chunk; p.kv_b = chunk;
  p.C = part; p.c_bs = (long)M * N; p.ldc = N;
  hipError_t err = hipSuccess;
  if (full > 0) {
    p.batches = full;
    err = run_dma<256, 256, 4, 2, 64, 2, false, false, EPI_STORE, true, TAG>(p, st);
    if (err != hipSuccess) return err;
  }
  if (last > 0) {
    GemmParams q = p;
    q.A = (const bf16_t*)A + (size_t)full * chunk * lda;
    q.B = (const bf16_t*)B + (size_t)full * chunk * ldb;
    q.C = part + (size_t)full * M * N;
    q.K = last; q.kv_a = last; q.kv_b = last; q.batches = 1;
    err = run_dma<256, 256, 4, 2, 64, 2, false, false, EPI_STORE, true, TAG>(q, st);
    if (err != hipSuccess) return err;
  }
  const long n = (long)M * N;
  splitk_store_kernel<bf16_t><<<(unsigned)((n + 255) / 256), 256, 0, st>>>(
      part, nsplit, M, N, c_split, (bf16_t*)C, (bf16_t*)C2, ldc);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_shared_dW2(int dtype, const void* dY, const void* A, void* dW2, int N, int d,
                             int h, float* part, int splits, hipStream_t st) {
  // dW2[m, n] = sum_i dY[i, m] A[i, n]  (m over d, n over h, i over all N tokens)
  if (dtype == DT_F32) return launch_gemm_dW2(dtype, dY, A, dW2, 1, N, d, h, st);
  return run_wgrad_splitk<G_SH_DW2>(dY, d, A, h, d, h, N, dW2, dW2, 1 << 30, h, part, splits, st);
}

hipError_t launch_shared_dW13(int dtype, const void* dH, const void* X, void* dW1, void* dW3,
                              int N, int d, int h, float* part, int splits, hipStream_t st) {
  // [dW1; dW3][m, n] = sum_i dH[i, m] X[i, n]  (m over 2h, n over d)
  if (dtype == DT_F32) return launch_gemm_dW13(dtype, dH, X, dW1, dW3, 1, N, d, h, st);
  return run_wgrad_splitk<G_SH_DW13>(dH, 2 * h, X, d, 2 * h, d, N, dW1, dW3, h, d, part, splits,
                                     st);
}

int tc_col_blocks_w13(int h) { return (h + 127) / 128; }
int tc_col_blocks_w2(int d) { return (d + 255) / 256; }

hipError_t launch_gemm_w13_var(int dtype, const void* Xe, const void* W1, const void* W3, void* A,
                               int E, const int32_t* rows, const int32_t* tiles, long max_rows,
                               int max_rows_per_expert, int d, int h, hipStream_t st,
                               const int32_t* sel) {
  GemmParams p = base_params();
  p.A = Xe; p.lda = d;
  if (sel) {   // Xe is X itself, packed row r is X[sel[r]]
    if (dtype == DT_F32) return hipErrorInvalidValue;
    p.a_rows = sel; p.a_rows_bs = 0;
  }
  p.B = W1; p.B2 = W3; p.b_bs = (long)h * d; p.ldb = d;
  p.M = max_rows_per_expert; p.N = h; p.K = d; p.kv_a = d; p.kv_b = d; p.batches = E;
  p.C = A; p.ldc = h; p.ldh = h;
  p.var_rows = rows; p.var_tiles = tiles;
  if (max_rows == 0) return hipSuccess;
  if (dtype == DT_F32) return run_f32<EPI_SWIGLU>(p, 1, 1, st);
  return run_dma_var<256, 256, 2, 4, 64, 2, true, true, EPI_SWIGLU, false, G_TC_W13>(p, max_rows,
                                                                                     st);
}

hipError_t launch_gemm_w2_var(int dtype, const void* A, const void* W2, void* O, int E,
                              const int32_t* rows, const int32_t* tiles, long max_rows,
                              int max_rows_per_expert, int d, int h, hipStream_t st) {
  GemmParams p = base_params();
  p.A = A; p.lda = h;
  p.B = W2; p.b_bs = (long)d * h; p.ldb = h;
  p.M = max_rows_per_expert; p.N = d; p.K = h; p.kv_a = h; p.kv_b = h; p.batches = E;
  p.C = O; p.ldc = d;
  p.var_rows = rows; p.var_tiles = tiles;
  if (max_rows == 0) return hipSuccess;
  if (dtype == DT_F32) return run_f32<EPI_STORE>(p, 1, 1, st);
  return run_dma_var<256, 256, 4, 2, 64, 2, true, true, EPI_STORE, false, G_TC_W2>(p, max_rows,
                                                                                   st);
}

}  // namespace ec
