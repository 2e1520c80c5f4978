// Int4 code words as MFMA operands, shared by the batched-decode kernels and
// the light-expert kernels: one 32-bit word (8 nibbles of one 8-input chunk)
// becomes the eight fp16 B-operand values of v_mfma_f32_16x16x32_f16, eight
// activations are permuted to the same pair order, and a 4 x 4 word
// transpose across a wave's 16-lane rows moves code words loaded row by row
// into the MFMA operand layout.
#pragma once

#include "q4_gemv_core.h"

namespace atsi {
namespace gemv {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// Eight exact fp16 integers q = u - 8 from one code word, in the pair order
// (k0, k4), (k1, k5), (k2, k6), (k3, k7): the B operand of an MFMA that sums
// one group's exact products.
__device__ __forceinline__ half8_t unpack_q(uint32_t w, const UnpackMasks& k) {
  const uint32_t w8 = w >> 8;
  const half2_t off = {(_Float16)-1032.f, (_Float16)-1032.f};
  const half2_t sh = {(_Float16)0.0625f, (_Float16)0.0625f};
  const half2_t off16 = {(_Float16)-72.f, (_Float16)-72.f};
  // (1024 + u) - 1032 and (1024 + 16 u) / 16 - 72 are exact in fp16
  const half2_t a = __builtin_bit_cast(half2_t, (w & k.lo) | k.magic) + off;
  const half2_t b = __builtin_bit_cast(half2_t, (w & k.hi) | k.magic) * sh + off16;
  const half2_t c = __builtin_bit_cast(half2_t, (w8 & k.lo) | k.magic) + off;
  const half2_t d = __builtin_bit_cast(half2_t, (w8 & k.hi) | k.magic) * sh + off16;
  const u32x4_t r = {__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b), __builtin_bit_cast(uint32_t, c),
                     __builtin_bit_cast(uint32_t, d)};
  return __builtin_bit_cast(half8_t, r);
}

// Eight consecutive fp16 activations reordered to the same pair order.
__device__ __forceinline__ half8_t perm_x(u32x4_t d) {
  const u32x4_t r = {__builtin_amdgcn_perm(d.z, d.x, 0x05040100u), __builtin_amdgcn_perm(d.z, d.x, 0x07060302u),
                     __builtin_amdgcn_perm(d.w, d.y, 0x05040100u), __builtin_amdgcn_perm(d.w, d.y, 0x07060302u)};
  return __builtin_bit_cast(half8_t, r);
}

// 4 x 4 transpose of words across the four 16-lane rows of the wave: on entry
// row r holds X[r][0..3] in v[0..3]; on return row r holds X[0..3][r].
__device__ __forceinline__ void transpose_rows4(uint32_t (&v)[4]) {
#if defined(__HIP_DEVICE_COMPILE__)
  // 2 x 2 blocks of rows {0, 1} and {2, 3} trade places (lane halves) ...
  const auto a = __builtin_amdgcn_permlane32_swap(v[0], v[2], false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(v[1], v[3], false, false);
  // ... then each block is transposed between neighbouring rows
  const auto c = __builtin_amdgcn_permlane16_swap(a[0], b[0], false, false);
  const auto d = __builtin_amdgcn_permlane16_swap(a[1], b[1], false, false);
  v[0] = c[0];
  v[1] = c[1];
  v[2] = d[0];
  v[3] = d[1];
#endif
}

}  // namespace gemv
}  // namespace atsi
