// Bandwidth-bound stages of the layer: the gather of selected tokens into
// expert-contiguous buffers, the gate-weighted combine (Section 2.2,
// y_i = sum_j g_ij FFN_j(x_i) with g_ij = S_ij), and their backward
// counterparts.  No floating-point atomics: every output row is produced by
// one wave that sums its expert contributions in ascending expert order.
#include "ec_common.h"
#include "ec_kernels.h"

namespace ec {

namespace {

// ---------------------------------------------------------------- gather
// One wave per expert row; 16-byte vectors, all loads of a row issued before
// its stores.
// With rows_dev the row count is read from device memory (rows is then the
// launch's upper bound).
template <int U>
__global__ __launch_bounds__(256) void gather_kernel(const uint4* __restrict__ X,
                                                     const int32_t* __restrict__ sel,
                                                     uint4* __restrict__ Xe, long rows, int vpr,
                                                     int N, const int32_t* rows_dev) {
  const int lane = threadIdx.x & 63;
  const long r = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (rows_dev && r >= *rows_dev) return;
  if (r >= rows) return;
  const int i = sel[r];
  if ((unsigned)i >= (unsigned)N) return;  // never for a valid selection
  const uint4* src = X + (size_t)i * vpr;
  uint4* dst = Xe + (size_t)r * vpr;
  for (int v0 = 0; v0 < vpr; v0 += 64 * U) {
    uint4 t[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + u * 64 + lane;
      if (v < vpr) t[u] = src[v];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + u * 64 + lane;
      if (v < vpr) dst[v] = t[u];
    }
  }
}

// ---------------------------------------------------------------- combine
constexpr int CB_TOK = 4;    // tokens per workgroup (one per wave)
constexpr int CB_Q = 4;      // 8-element chunks per lane per column block

// A row of zeros as wide as the widest fp32 row the library accepts (d <= 16384):
// the padding rows of a combine step read it (it stays zero).
__device__ __attribute__((aligned(16))) uint4 cb_zero_row[16384 * 4 / 16];

// Builds, for one token, the ascending list of (expert, row) it was selected
// by, with the gate values; returns the list length.  Lists are wave-private.
// Rows at or past K are treated as unselected (never for a valid selection).
template <int MAXE>
__device__ __forceinline__ int token_expert_list(const int32_t* sslot, const float* sgate,
                                                 int t, int E, int K, int2* list, float* lgate) {
  const int lane = threadIdx.x & 63;
  int n = 0;
  for (int j0 = 0; j0 < E; j0 += 64) {
    const int j = j0 + lane;
    int r = (j < E) ? sslot[j * CB_TOK + t] : -1;
    r = (r < K) ? r : -1;  // never for a valid selection
    const uint64_t m = __ballot(r >= 0);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (r >= 0) {
      list[n + before] = make_int2(j, r);
      lgate[n + before] = sgate ? sgate[t * MAXE + j] : 1.0f;
    }
    n += __popcll(m);
  }
  __builtin_amdgcn_wave_barrier();
  return n;
}

// Y[i] = (Xr[i] if Xr) + sum_j g_ij Src[j kstride + slot_ij] in ascending j;
// with S == nullptr the gates are 1 (backward combine of dXe).  kstride is the
// rows of one expert's buffer (0 when slot holds rows of one packed buffer);
// slot values are below K.  Each step loads U expert rows (16 or 8 16-byte
// loads per lane in flight) with no branch between the loads and their FMAs:
// entries past the token's last expert read the zero row with gate 0, and lanes
// past the row's end read its last chunk and store nothing.
// BWD: the backward combine of dXe (its own kernel symbol, so that traces and
// counters tell the two stages apart).
template <typename T, int MAXE, bool BWD>
__global__ __launch_bounds__(256) void combine_kernel(const T* __restrict__ Src,
                                                      const float* __restrict__ S,
                                                      const int32_t* __restrict__ slotT,
                                                      const T* Xr, T* Y, int N, int E, int K,
                                                      int d, long kstride) {
  constexpr int U = sizeof(T) == 2 ? 4 : 2;   // expert rows per step
  __shared__ int32_t sslot[MAXE * CB_TOK];
  __shared__ float sgate[CB_TOK * MAXE];
  __shared__ int2 slist[4][MAXE];
  __shared__ float sglist[4][MAXE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i0 = blockIdx.x * CB_TOK;
  for (int c = tid; c < E * CB_TOK; c += 256) {
    const int j = c / CB_TOK, t = c % CB_TOK;
    sslot[c] = (i0 + t < N) ? slotT[(size_t)j * N + i0 + t] : -1;
  }
  if (S) {
    for (int c = tid; c < CB_TOK * E; c += 256) {
      const int t = c / E, j = c % E;
      sgate[t * MAXE + j] = (i0 + t < N) ? S[(size_t)(i0 + t) * E + j] : 0.f;
    }
  }
  __syncthreads();
  const int nch = d >> 3;
  for (int t = wave; t < CB_TOK; t += 4) {
    const int i = i0 + t;
    if (i >= N) break;
    const int n = token_expert_list<MAXE>(sslot, S ? sgate : nullptr, t, E, K, slist[wave],
                                          sglist[wave]);
    for (int c0 = 0; c0 < nch; c0 += 64 * CB_Q) {
      int cc[CB_Q];
#pragma unroll
      for (int q = 0; q < CB_Q; ++q) {
        const int c = c0 + q * 64 + lane;
        cc[q] = c < nch ? c : nch - 1;
      }
      float acc[CB_Q][8];
#pragma unroll
      for (int q = 0; q < CB_Q; ++q) {
        if (Xr) {
          Elem<T>::load8(Xr + (size_t)i * d + cc[q] * 8, acc[q]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[q][e] = 0.f;
        }
      }
      for (int p = 0; p < n; p += U) {
        typename Elem<T>::Raw v[U][CB_Q];
        float g[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const bool pad = p + u >= n;
          const int2 jr = slist[wave][pad ? n - 1 : p + u];
          const T* src = pad ? reinterpret_cast<const T*>(cb_zero_row)
                             : Src + ((size_t)jr.x * kstride + jr.y) * d;
          g[u] = pad ? 0.f : sglist[wave][p + u];
#pragma unroll
          for (int q = 0; q < CB_Q; ++q) v[u][q] = Elem<T>::load_raw(src + cc[q] * 8);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int q = 0; q < CB_Q; ++q) Elem<T>::fma_raw(acc[q], g[u], v[u][q]);   // ascending j
      }
#pragma unroll
      for (int q = 0; q < CB_Q; ++q) {
        const int c = c0 + q * 64 + lane;
        if (c < nch) Elem<T>::store8(Y + (size_t)i * d + c * 8, acc[q]);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

template <typename T, bool BWD>
hipError_t run_combine(const T* Src, const float* S, const int32_t* slotT, const T* Xr, T* Y,
                       int N, int E, int K, int d, hipStream_t st, long kstride) {
  const int grid = (N + CB_TOK - 1) / CB_TOK;
  if (E <= 64)
    combine_kernel<T, 64, BWD><<<grid, 256, 0, st>>>(Src, S, slotT, Xr, Y, N, E, K, d, kstride);
  else if (E <= 128)
    combine_kernel<T, 128, BWD><<<grid, 256, 0, st>>>(Src, S, slotT, Xr, Y, N, E, K, d, kstride);
  else
    combine_kernel<T, 256, BWD><<<grid, 256, 0, st>>>(Src, S, slotT, Xr, Y, N, E, K, d, kstride);
  return hipGetLastError();
}

// ---------------------------------------------------------------- router dZ
// dZ[i, :] = S_i * (dS_i - <S_i, dS_i>) / tau = (u_i - S_i sum_j u_ij) / tau with
// u_ij = S_ij dS_ij: on the selection the sum of the dA product's partials of
// row (j, slot_ij) (they carry the gate: dA = S_ij dY_i W2), 0 off it; dS
// itself is never formed.  Writes fp32 dZ [N, E] and, if dZb is given,
// a bf16 copy [N, EP] whose columns E..EP-1 are zero.  A workgroup stages a
// tile of `tok` (<= RZ_TOK) tokens through LDS so that every global access is
// coalesced; the tile keeps the dynamic LDS under 64 KiB for any E <= 256.
constexpr int RZ_TOK = 32;
constexpr int RZ_B = 8;       // (expert, token) entries per thread per batch

// NP > 0: rows of exactly NP partials (NP a multiple of 4: 16-byte aligned rows),
// read as float4 vectors; NP = 0: any count, read one by one.  Either way each
// batch first loads the slots of its RZ_B entries, then every partial they
// select, so the loads are in flight together; the partials of a row are then
// added in a fixed order (0, 1, ...).
template <int NP>
__global__ __launch_bounds__(256) void router_dz_kernel(const float* __restrict__ S,
                                                        const float* __restrict__ dsp,
                                                        int nparts,
                                                        const int32_t* __restrict__ slotT,
                                                        float* __restrict__ dZ,
                                                        bf16_t* __restrict__ dZb, int N, int E,
                                                        int EP, int K, float inv_tau, int tok) {
  extern __shared__ float rz_lds[];
  const int LD = E + 1;
  float* sS = rz_lds;              // [tok][E+1]
  float* sU = rz_lds + tok * LD;   // [tok][E+1]
  __shared__ float sdot[RZ_TOK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i0 = blockIdx.x * tok;
  const int nt = N - i0 < tok ? N - i0 : tok;
  // S tile (contiguous rows), RZ_B loads per thread in flight together
  for (int c0 = 0; c0 < nt * E; c0 += 256 * RZ_B) {
    float v[RZ_B];
#pragma unroll
    for (int b = 0; b < RZ_B; ++b) {
      const int c = c0 + b * 256 + tid;
      v[b] = S[(size_t)i0 * E + (c < nt * E ? c : nt * E - 1)];
    }
#pragma unroll
    for (int b = 0; b < RZ_B; ++b) {
      const int c = c0 + b * 256 + tid;
      if (c < nt * E) sS[(c / E) * LD + c % E] = v[b];
    }
  }
  const int total = E * tok;                            // slot tile: tok tokens per expert
  for (int c0 = 0; c0 < total; c0 += 256 * RZ_B) {
    int row[RZ_B];
    bool sel[RZ_B];
#pragma unroll
    for (int b = 0; b < RZ_B; ++b) {
      const int c = c0 + b * 256 + tid;
      const int j = c / tok, t = c % tok;
      const bool in = c < total && t < nt;
      const int r = slotT[(size_t)(in ? j : 0) * N + i0 + (in ? t : 0)];   // always in range
      sel[b] = in && K > 0 && r >= 0 && r < K;
      row[b] = sel[b] ? j * K + r : 0;
    }
    float u[RZ_B];
    if constexpr (NP > 0) {
      // unconditional loads (an entry off the selection reads row 0, a valid row
      // whenever K > 0) so that none waits behind a branch; K = 0 is uniform
      float4 v[RZ_B][NP / 4];
      if (K > 0) {
#pragma unroll
        for (int b = 0; b < RZ_B; ++b)
#pragma unroll
          for (int w = 0; w < NP / 4; ++w)
            v[b][w] = *reinterpret_cast<const float4*>(dsp + (size_t)row[b] * NP + 4 * w);
      }
#pragma unroll
      for (int b = 0; b < RZ_B; ++b)
#pragma unroll
        for (int w = 0; w < NP / 4; ++w)
          if (!sel[b]) v[b][w] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int b = 0; b < RZ_B; ++b) {
        float x = 0.f;
#pragma unroll
        for (int w = 0; w < NP / 4; ++w) {
          x += v[b][w].x; x += v[b][w].y; x += v[b][w].z; x += v[b][w].w;
        }
        u[b] = x;
      }
    } else {
#pragma unroll
      for (int b = 0; b < RZ_B; ++b) {
        float x = 0.f;
        if (sel[b]) {
          const float* pp = dsp + (size_t)row[b] * nparts;
          for (int q = 0; q < nparts; ++q) x += pp[q];
        }
        u[b] = x;
      }
    }
#pragma unroll
    for (int b = 0; b < RZ_B; ++b) {
      const int c = c0 + b * 256 + tid;
      if (c < total) sU[(c % tok) * LD + c / tok] = u[b];
    }
  }
  __syncthreads();
  for (int t = wave; t < nt; t += 4) {                 // <S_t, dS_t> = sum_j u_tj, a wave per token
    float v = 0.f;
    for (int j = lane; j < E; j += 64) v += sU[t * LD + j];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) sdot[t] = v;
  }
  __syncthreads();
  for (int c = tid; c < nt * E; c += 256) {
    const int t = c / E, j = c % E;
    dZ[(size_t)i0 * E + c] = (sU[t * LD + j] - sS[t * LD + j] * sdot[t]) * inv_tau;
  }
  if (dZb) {
    for (int c = tid; c < nt * EP; c += 256) {
      const int t = c / EP, j = c % EP;
      const float z = (j < E) ? (sU[t * LD + j] - sS[t * LD + j] * sdot[t]) * inv_tau : 0.f;
      dZb[(size_t)i0 * EP + c] = (bf16_t)f32_to_bf16(z);
    }
  }
}

// Token drop statistic (Appendix D: tokens that no routed expert chose).
// cnt[i] = number of experts j with slotT[j, i] >= 0; one thread per token,
// coalesced over i for every expert row of the slot map.
__global__ __launch_bounds__(256) void coverage_count_kernel(const int32_t* __restrict__ slotT,
                                                              int N, int E,
                                                              int32_t* __restrict__ cnt) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= N) return;
  int c = 0;
  for (int j = 0; j < E; ++j) c += slotT[(size_t)j * N + i] >= 0;
  cnt[i] = c;
}

// dropped[g] = tokens of group g with cnt == 0; one workgroup per group of the table.
__global__ __launch_bounds__(256) void coverage_drop_kernel(const int32_t* __restrict__ cnt,
                                                             GroupTable tab,
                                                             int32_t* __restrict__ dropped) {
  __shared__ int part[4];
  const int g = blockIdx.x;
  const int off = tab.off[g], len = tab.len[g];
  int z = 0;
  for (int i = threadIdx.x; i < len; i += 256) z += cnt[off + i] == 0;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) z += __shfl_xor(z, m);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = z;
  __syncthreads();
  if (threadIdx.x == 0) dropped[g] = part[0] + part[1] + part[2] + part[3];
}

__global__ void zero_kernel(uint4* p, size_t n16, unsigned char* tail, size_t ntail) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    p[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0 && threadIdx.x < ntail) tail[threadIdx.x] = 0;
}

}  // namespace

hipError_t launch_gather(int dtype, const void* X, const int32_t* sel_token, void* Xe, long rows,
                         int d, int N, hipStream_t st, const int32_t* rows_dev) {
  if (rows == 0) return hipSuccess;
  const int vpr = d * (dtype == DT_F32 ? 4 : 2) / 16;
  const long grid = (rows + 3) / 4;
  gather_kernel<4><<<dim3((unsigned)grid), 256, 0, st>>>((const uint4*)X, sel_token, (uint4*)Xe,
                                                         rows, vpr, N, rows_dev);
  return hipGetLastError();
}

hipError_t launch_combine(int dtype, const void* O, const float* S, const int32_t* slotT,
                          const void* Xr, void* Y, int N, int E, int K, int d, hipStream_t st,
                          long kstride) {
  if (N == 0) return hipSuccess;
  if (kstride < 0) kstride = K;
  if (dtype == DT_F32)
    return run_combine<float, false>((const float*)O, S, slotT, (const float*)Xr, (float*)Y, N, E,
                                     K, d, st, kstride);
  return run_combine<bf16_t, false>((const bf16_t*)O, S, slotT, (const bf16_t*)Xr, (bf16_t*)Y, N,
                                    E, K, d, st, kstride);
}

hipError_t launch_bwd_combine(int dtype, const void* dXe, const int32_t* slotT, const void* Xr,
                              void* dX, int N, int E, int K, int d, hipStream_t st) {
  if (N == 0) return hipSuccess;
  if (dtype == DT_F32)
    return run_combine<float, true>((const float*)dXe, nullptr, slotT, (const float*)Xr,
                                    (float*)dX, N, E, K, d, st, K);
  return run_combine<bf16_t, true>((const bf16_t*)dXe, nullptr, slotT, (const bf16_t*)Xr,
                                   (bf16_t*)dX, N, E, K, d, st, K);
}

hipError_t launch_router_dz(const float* S, const float* dsp, int nparts, const int32_t* slotT,
                            float* dZ, uint16_t* dZb, int N, int E, int EP, int K, float inv_tau,
                            hipStream_t st) {
  if (N == 0) return hipSuccess;
  const int tok = E > 128 ? RZ_TOK / 2 : RZ_TOK;
  const size_t lds = (size_t)2 * tok * (E + 1) * sizeof(float);
  const int grid = (N + tok - 1) / tok;
  switch (nparts) {
    case 4:
      router_dz_kernel<4><<<grid, 256, lds, st>>>(S, dsp, nparts, slotT, dZ, dZb, N, E, EP, K,
                                                  inv_tau, tok);
      break;
    case 8:
      router_dz_kernel<8><<<grid, 256, lds, st>>>(S, dsp, nparts, slotT, dZ, dZb, N, E, EP, K,
                                                  inv_tau, tok);
      break;
    case 16:
      router_dz_kernel<16><<<grid, 256, lds, st>>>(S, dsp, nparts, slotT, dZ, dZb, N, E, EP, K,
                                                   inv_tau, tok);
      break;
    default:
      router_dz_kernel<0><<<grid, 256, lds, st>>>(S, dsp, nparts, slotT, dZ, dZb, N, E, EP, K,
                                                  inv_tau, tok);
  }
  return hipGetLastError();
}

hipError_t launch_coverage_count(const int32_t* slotT, int N, int E, int32_t* cnt,
                                 hipStream_t st) {
  if (N == 0) return hipSuccess;
  coverage_count_kernel<<<(N + 255) / 256, 256, 0, st>>>(slotT, N, E, cnt);
  return hipGetLastError();
}

hipError_t launch_coverage_drop(const int32_t* cnt, const GroupTable& tab, int32_t* dropped,
                                hipStream_t st) {
  if (tab.n == 0) return hipSuccess;
  coverage_drop_kernel<<<tab.n, 256, 0, st>>>(cnt, tab, dropped);
  return hipGetLastError();
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  const size_t n16 = bytes / 16;
  const size_t ntail = bytes - n16 * 16;
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks == 0) blocks = 1;
  zero_kernel<<<(unsigned)blocks, 256, 0, st>>>((uint4*)p, n16, (unsigned char*)p + n16 * 16, ntail);
  return hipGetLastError();
}

}  // namespace ec
