// Device-side helpers shared by the expert-choice MoE kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ec {

typedef uint16_t bf16_t;  // bf16 storage: the upper 16 bits of an fp32

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest, ties to even (v_cvt_pk_bf16_f32; NaN stays NaN).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Storage-type traits: load/store 8 consecutive elements as fp32.
template <typename T> struct Elem;

template <> struct Elem<float> {
  struct Raw { float4 a, b; };
  static __device__ __forceinline__ Raw load_raw(const float* p) {
    return Raw{*reinterpret_cast<const float4*>(p), *reinterpret_cast<const float4*>(p + 4)};
  }
  static __device__ __forceinline__ void fma_raw(float acc[8], float g, const Raw& r) {
    acc[0] = fmaf(g, r.a.x, acc[0]); acc[1] = fmaf(g, r.a.y, acc[1]);
    acc[2] = fmaf(g, r.a.z, acc[2]); acc[3] = fmaf(g, r.a.w, acc[3]);
    acc[4] = fmaf(g, r.b.x, acc[4]); acc[5] = fmaf(g, r.b.y, acc[5]);
    acc[6] = fmaf(g, r.b.z, acc[6]); acc[7] = fmaf(g, r.b.w, acc[7]);
  }
  static __device__ __forceinline__ void load8(const float* p, float v[8]) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
  static __device__ __forceinline__ void store8(float* p, const float v[8]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
  static __device__ __forceinline__ float load1(const float* p) { return *p; }
  static __device__ __forceinline__ void store1(float* p, float v) { *p = v; }
};

template <> struct Elem<bf16_t> {
  typedef uint4 Raw;
  // a streaming (non-temporal) load: the combines read each expert row once
  // (measured: -6-7% on both)
  static __device__ __forceinline__ Raw load_raw(const bf16_t* p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
  }
  static __device__ __forceinline__ void fma_raw(float acc[8], float g, const Raw& r) {
    acc[0] = fmaf(g, bf16_to_f32(r.x & 0xffffu), acc[0]); acc[1] = fmaf(g, bf16_to_f32(r.x >> 16), acc[1]);
    acc[2] = fmaf(g, bf16_to_f32(r.y & 0xffffu), acc[2]); acc[3] = fmaf(g, bf16_to_f32(r.y >> 16), acc[3]);
    acc[4] = fmaf(g, bf16_to_f32(r.z & 0xffffu), acc[4]); acc[5] = fmaf(g, bf16_to_f32(r.z >> 16), acc[5]);
    acc[6] = fmaf(g, bf16_to_f32(r.w & 0xffffu), acc[6]); acc[7] = fmaf(g, bf16_to_f32(r.w >> 16), acc[7]);
  }
  static __device__ __forceinline__ void load8(const bf16_t* p, float v[8]) {
    const uint4 a = *reinterpret_cast<const uint4*>(p);
    v[0] = bf16_to_f32(a.x & 0xffffu); v[1] = bf16_to_f32(a.x >> 16);
    v[2] = bf16_to_f32(a.y & 0xffffu); v[3] = bf16_to_f32(a.y >> 16);
    v[4] = bf16_to_f32(a.z & 0xffffu); v[5] = bf16_to_f32(a.z >> 16);
    v[6] = bf16_to_f32(a.w & 0xffffu); v[7] = bf16_to_f32(a.w >> 16);
  }
  static __device__ __forceinline__ void store8(bf16_t* p, const float v[8]) {
    uint4 a;
    a.x = pack_bf16x2(v[0], v[1]); a.y = pack_bf16x2(v[2], v[3]);
    a.z = pack_bf16x2(v[4], v[5]); a.w = pack_bf16x2(v[6], v[7]);
    // a streaming (non-temporal) store: no kernel re-reads its own output within
    // the same launch (later launches do: W2 and dW2 read A, dA reads H1/H3, the
    // combine reads O), and the hint keeps the written lines from displacing the
    // launch's operands in the caches (measured: combines -8-9%, dA -2%)
    __builtin_nontemporal_store(u32x4{a.x, a.y, a.z, a.w}, reinterpret_cast<u32x4*>(p));
  }
  static __device__ __forceinline__ float load1(const bf16_t* p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ void store1(bf16_t* p, float v) { *p = (bf16_t)f32_to_bf16(v); }
};

// Hardware exp2 and reciprocal (about 1 ulp each): the activations feed bf16
// stores or fp32 sums whose tolerance is far wider.
__device__ __forceinline__ float sigmoid_f(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

__device__ __forceinline__ float silu_f(float z) { return z * sigmoid_f(z); }

// Sum over the 16 lanes of a DPP row (lanes 16 r .. 16 r + 15); every lane of
// the row ends with the total.  Quad swaps (xor 1, xor 2) then row rotations
// by 4 and 8 lanes, all in registers (no LDS permute).
__device__ __forceinline__ float dpp_add(float t, int ctrl_id) {
  int v = __builtin_bit_cast(int, t);
  switch (ctrl_id) {
    case 0: v = __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false); break;   // quad [1,0,3,2]
    case 1: v = __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false); break;   // quad [2,3,0,1]
    case 2: v = __builtin_amdgcn_update_dpp(0, v, 0x124, 0xF, 0xF, false); break;  // row_ror:4
    default: v = __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false); break; // row_ror:8
  }
  return t + __builtin_bit_cast(float, v);
}
__device__ __forceinline__ float row16_sum(float t) {
  return dpp_add(dpp_add(dpp_add(dpp_add(t, 0), 1), 2), 3);
}

// DPP move of a 32-bit value within rows of 16 lanes; lanes whose source is
// outside the row read 0 (bound_ctrl).  Controls used here: quad_perm
// [1,0,3,2] = 0xB1 and [2,3,0,1] = 0x4E, row_shl:n = 0x100 + n, row_ror:n = 0x120 + n.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(float, dpp_u32<CTRL>(__builtin_bit_cast(uint32_t, v)));
}

// Maximum over the 16 lanes of a DPP row; every lane of the row ends with it.
__device__ __forceinline__ float row16_max(float t) {
  t = fmaxf(t, dpp_f32<0xB1>(t));
  t = fmaxf(t, dpp_f32<0x4E>(t));
  t = fmaxf(t, dpp_f32<0x124>(t));
  return fmaxf(t, dpp_f32<0x128>(t));
}

// Minimum and maximum of an unsigned value over the whole wave (uniform results).
__device__ __forceinline__ void wave_minmax_u32(uint32_t mn, uint32_t mx, uint32_t* out_mn,
                                                uint32_t* out_mx) {
  uint32_t a, b;
  a = dpp_u32<0xB1>(mn); mn = a < mn ? a : mn;  b = dpp_u32<0xB1>(mx); mx = b > mx ? b : mx;
  a = dpp_u32<0x4E>(mn); mn = a < mn ? a : mn;  b = dpp_u32<0x4E>(mx); mx = b > mx ? b : mx;
  a = dpp_u32<0x124>(mn); mn = a < mn ? a : mn; b = dpp_u32<0x124>(mx); mx = b > mx ? b : mx;
  a = dpp_u32<0x128>(mn); mn = a < mn ? a : mn; b = dpp_u32<0x128>(mx); mx = b > mx ? b : mx;
  uint32_t rmn = __builtin_amdgcn_readlane(mn, 0), rmx = __builtin_amdgcn_readlane(mx, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    const uint32_t c = __builtin_amdgcn_readlane(mn, r), d = __builtin_amdgcn_readlane(mx, r);
    rmn = c < rmn ? c : rmn;
    rmx = d > rmx ? d : rmx;
  }
  *out_mn = rmn;
  *out_mx = rmx;
}

// Exclusive suffix sum over the wave's lanes: the sum of v over lanes > lane.
__device__ __forceinline__ uint32_t wave_excl_suffix_u32(uint32_t v) {
  uint32_t x = v;                       // inclusive suffix within the row of 16
  x += dpp_u32<0x101>(x);
  x += dpp_u32<0x102>(x);
  x += dpp_u32<0x104>(x);
  x += dpp_u32<0x108>(x);
  const uint32_t t1 = __builtin_amdgcn_readlane(x, 16), t2 = __builtin_amdgcn_readlane(x, 32),
                 t3 = __builtin_amdgcn_readlane(x, 48);
  const int row = (threadIdx.x & 63) >> 4;
  const uint32_t later = row == 0 ? t1 + t2 + t3 : (row == 1 ? t2 + t3 : (row == 2 ? t3 : 0u));
  return x - v + later;
}

// Order-preserving map from fp32 to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t f32_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int wave_lane() { return threadIdx.x & 63; }

// Remap a linear workgroup id so that consecutive tile ids land on the same XCD.
// Workgroups are dispatched round-robin over the 8 XCDs; the launch pads the
// grid to a multiple of 8 and ids >= n_tiles exit.
__device__ __forceinline__ int xcd_tile_id(int bid, int grid) {
  const int per_xcd = grid >> 3;
  return (bid & 7) * per_xcd + (bid >> 3);
}

}  // namespace ec
