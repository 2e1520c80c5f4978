// Building blocks of the dequantising GEMV, shared by the dense decode kernel
// and the grouped expert kernels: a lane streams one 32-input group (16 code
// bytes, one 128-bit load) per step, turns nibbles into fp16 1024 + u by
// OR-ing them into the mantissa of 0x6400, multiplies pairs against
// activations with v_dot2_f32_f16 (fp32 accumulation), removes the 1032 offset
// with the group sum of x, and scales by the group's fp16 scale in fp32.
#pragma once

#include "common.h"

namespace atsi {
namespace gemv {

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr uint32_t kMagic = 0x64006400u;  // fp16 1024.0 in both halves

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, a), __builtin_bit_cast(half2_t, b), c, false);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// x pairs of one 32-input group in nibble order, plus the group sum.
template <int MT>
struct XChunk {
  uint32_t p[MT][16];
  float sum[MT];
};

template <int MT>
__device__ __forceinline__ void load_x(XChunk<MT>& xc, const __half* __restrict__ x, int K, int M, int c,
                                       bool norm, float (&sq)[MT]) {
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if (m < M) {
      const uint4* src = reinterpret_cast<const uint4*>(x + (size_t)m * K + (size_t)c * kGroup);
#pragma unroll
      for (int b = 0; b < 4; ++b) {       // 8 inputs per 16 bytes
        uint4 d = src[b];
        xc.p[m][4 * b + 0] = __builtin_amdgcn_perm(d.z, d.x, 0x05040100u);  // (x0, x4)
        xc.p[m][4 * b + 1] = __builtin_amdgcn_perm(d.z, d.x, 0x07060302u);  // (x1, x5)
        xc.p[m][4 * b + 2] = __builtin_amdgcn_perm(d.w, d.y, 0x05040100u);  // (x2, x6)
        xc.p[m][4 * b + 3] = __builtin_amdgcn_perm(d.w, d.y, 0x07060302u);  // (x3, x7)
      }
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) s = dot2(xc.p[m][i], 0x3C003C00u, s);  // (1.0, 1.0)
      xc.sum[m] = s;
      if (norm) {
        float q = sq[m];
#pragma unroll
        for (int i = 0; i < 16; ++i) q = dot2(xc.p[m][i], xc.p[m][i], q);
        sq[m] = q;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) xc.p[m][i] = 0u;
      xc.sum[m] = 0.f;
    }
  }
}

// sum_k (1024 + u_k) x_k over one group, per token.
template <int MT>
__device__ __forceinline__ void group_dot(const uint4& cw, const XChunk<MT>& xc, float (&part)[MT]) {
#pragma unroll
  for (int m = 0; m < MT; ++m) part[m] = 0.f;
  const uint32_t w4[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t w = w4[i];
    const uint32_t t0 = (w & 0x000F000Fu) | kMagic;          // inputs 8i+0, 8i+4
    const uint32_t t1 = ((w >> 4) & 0x000F000Fu) | kMagic;   // 8i+1, 8i+5
    const uint32_t t2 = ((w >> 8) & 0x000F000Fu) | kMagic;   // 8i+2, 8i+6
    const uint32_t t3 = ((w >> 12) & 0x000F000Fu) | kMagic;  // 8i+3, 8i+7
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float a = part[m];
      a = dot2(t0, xc.p[m][4 * i + 0], a);
      a = dot2(t1, xc.p[m][4 * i + 1], a);
      a = dot2(t2, xc.p[m][4 * i + 2], a);
      a = dot2(t3, xc.p[m][4 * i + 3], a);
      part[m] = a;
    }
  }
}


}  // namespace gemv
}  // namespace atsi
