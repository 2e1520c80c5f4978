// Building blocks of the dequantising GEMV, shared by the dense decode kernel
// and the grouped expert kernels.
//
// A lane owns one 32-input group of a row per step: one 128-bit load of 16
// code bytes plus its fp16 scale.  Per 32-bit word (8 nibbles, inputs
// k0..k7, k0 in the low nibble) the nibbles become fp16 values by OR-ing them
// into the mantissa of 1024.0 (0x6400):
//   A = (w & 0x000F000F) | 0x6400_6400  ->  (1024 + u0,  1024 + u4)
//   B = (w & 0x00F000F0) | 0x6400_6400  ->  (1024 + 16 u1, 1024 + 16 u5)
//   C, D the same on w >> 8             ->  inputs (2, 6) and (3, 7)
// so four ALU ops cover eight weights.  v_dot2_f32_f16 multiplies each pair
// with the matching activation pair and accumulates in fp32 (all products are
// exact: 11-bit by 11-bit).  With S_e, S_o the even- and odd-input sums and
// X_e, X_o the matching activation sums, the group's exact partial is
//   sum_k q_k x_k = S_e - 1032 X_e + S_o / 16 - 72 X_o      (q = u - 8),
// and it is scaled by the group's fp16 scale in fp32.  Activations are
// permuted once per group to the (k, k+4) pairing, and X_e, X_o are shared by
// every row of the wave.
#pragma once

#include "common.h"

namespace atsi {
namespace gemv {

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr uint32_t kMagic = 0x64006400u;  // fp16 1024.0 in both halves
constexpr uint32_t kOnes = 0x3C003C00u;   // fp16 (1.0, 1.0)

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, a), __builtin_bit_cast(half2_t, b), c, false);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Cross-lane sums on the DPP and permlane paths (no LDS traffic).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xF, false));
}
// Sum over each row of 16 lanes, left in every lane of the row.
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f<0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x141, 0xF>(v);  // row_half_mirror
  v += dpp_f<0x140, 0xF>(v);  // row_mirror
  return v;
}
// Sum over the wave, returned in every lane.
__device__ __forceinline__ float wave_total(float v) {
  v = row16_sum(v);
  v += dpp_f<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
  v += dpp_f<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Sums V per-lane values over the wave at once.  Two butterfly levels swap
// half the values between lane halves (permlane32) and row pairs (permlane16),
// so each level halves the count of values a lane carries; the last V/4
// values are summed inside each row of 16.  On return v[i] (i < V/4), in
// every lane of row r, holds the total of value i + (V/4)(r & 1) + (V/2)(r >> 1).
template <int V>
__device__ __forceinline__ void transpose_reduce(float (&v)[V]) {
  static_assert(V >= 4 && (V & (V - 1)) == 0, "a power of two, at least 4");
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
  for (int i = 0; i < V / 2; ++i) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[i]), __float_as_uint(v[i + V / 2]), false, false);
    v[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
#pragma unroll
  for (int i = 0; i < V / 4; ++i) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[i]), __float_as_uint(v[i + V / 4]), false, false);
    v[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
#endif
#pragma unroll
  for (int i = 0; i < V / 4; ++i) v[i] = row16_sum(v[i]);
}

// Activations of one 32-input group: 16 pairs in nibble order and the
// correction 1032 X_e + 72 X_o.
struct XGroup {
  uint32_t p[16];
  float corr;
};

// Raw activation bytes of one group (64 B).
struct XRaw {
  uint4 d[4];
};

__device__ __forceinline__ void load_xraw(XRaw& r, const __half* __restrict__ xrow, int c) {
  const uint4* src = reinterpret_cast<const uint4*>(xrow + (size_t)c * kGroup);
#pragma unroll
  for (int b = 0; b < 4; ++b) r.d[b] = src[b];
}

// Permute to (k, k+4) pairs and form the correction; optionally add the sum of
// squares (for a fused RMS norm).
__device__ __forceinline__ void prep_x(XGroup& g, const XRaw& r, bool want_sq, float& sq) {
  float xe = 0.f, xo = 0.f;
#pragma unroll
  for (int b = 0; b < 4; ++b) {  // 8 inputs per 16 bytes
    const uint4 d = r.d[b];
    g.p[4 * b + 0] = __builtin_amdgcn_perm(d.z, d.x, 0x05040100u);  // (x0, x4)
    g.p[4 * b + 1] = __builtin_amdgcn_perm(d.z, d.x, 0x07060302u);  // (x1, x5)
    g.p[4 * b + 2] = __builtin_amdgcn_perm(d.w, d.y, 0x05040100u);  // (x2, x6)
    g.p[4 * b + 3] = __builtin_amdgcn_perm(d.w, d.y, 0x07060302u);  // (x3, x7)
    xe = dot2(g.p[4 * b + 0], kOnes, xe);
    xo = dot2(g.p[4 * b + 1], kOnes, xo);
    xe = dot2(g.p[4 * b + 2], kOnes, xe);
    xo = dot2(g.p[4 * b + 3], kOnes, xo);
  }
  g.corr = fmaf(1032.f, xe, 72.f * xo);
  if (want_sq) {
#pragma unroll
    for (int i = 0; i < 16; ++i) sq = dot2(g.p[i], g.p[i], sq);
  }
}

// sum_k q_k x_k over one group (exact products, fp32 sums).
__device__ __forceinline__ float group_dot(const uint4& cw, const XGroup& g) {
  float se = 0.f, so = 0.f;
  const uint32_t w4[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t w = w4[i];
    const uint32_t w8 = w >> 8;
    const uint32_t a = (w & 0x000F000Fu) | kMagic;   // inputs 8i+0, 8i+4
    const uint32_t b = (w & 0x00F000F0u) | kMagic;   // 8i+1, 8i+5 (x16)
    const uint32_t c = (w8 & 0x000F000Fu) | kMagic;  // 8i+2, 8i+6
    const uint32_t d = (w8 & 0x00F000F0u) | kMagic;  // 8i+3, 8i+7 (x16)
    se = dot2(a, g.p[4 * i + 0], se);
    so = dot2(b, g.p[4 * i + 1], so);
    se = dot2(c, g.p[4 * i + 2], se);
    so = dot2(d, g.p[4 * i + 3], so);
  }
  return fmaf(so, 0.0625f, se - g.corr);
}

// Unpack masks held in scalar registers and the 1024.0 pattern in a vector
// register, so that each mask-and-or is one v_and_or_b32 (its VOP3 encoding
// takes no literal constant and reads at most one scalar register).
struct UnpackMasks {
  uint32_t lo, hi, magic;
};
__device__ __forceinline__ UnpackMasks unpack_masks() {
  uint32_t lo, hi, mg;
  asm volatile("s_mov_b32 %0, %1" : "=s"(lo) : "i"(0x000F000Fu));
  asm volatile("s_mov_b32 %0, %1" : "=s"(hi) : "i"(0x00F000F0u));
  asm volatile("v_mov_b32 %0, %1" : "=v"(mg) : "i"(kMagic));
  return UnpackMasks{lo, hi, mg};
}
// v_dot2_f32_f16 with a zero addend (saves zeroing an accumulator)
__device__ __forceinline__ float dot2_0(uint32_t a, uint32_t b) {
  float r;
  asm("v_dot2_f32_f16 %0, %1, %2, 0" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
// group_dot with the masks in registers (same arithmetic and order)
__device__ __forceinline__ float group_dot_m(const uint4& cw, const XGroup& g, const UnpackMasks& k) {
  float se = 0.f, so = 0.f;
  const uint32_t w4[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t w = w4[i];
    const uint32_t w8 = w >> 8;
    const uint32_t a = (w & k.lo) | k.magic;
    const uint32_t b = (w & k.hi) | k.magic;
    const uint32_t c = (w8 & k.lo) | k.magic;
    const uint32_t d = (w8 & k.hi) | k.magic;
    if (i == 0) {
      se = dot2_0(a, g.p[0]);
      so = dot2_0(b, g.p[1]);
    } else {
      se = dot2(a, g.p[4 * i + 0], se);
      so = dot2(b, g.p[4 * i + 1], so);
    }
    se = dot2(c, g.p[4 * i + 2], se);
    so = dot2(d, g.p[4 * i + 3], so);
  }
  return fmaf(so, 0.0625f, se - g.corr);
}

}  // namespace gemv
}  // namespace atsi
