// Main loop of the dequantising fp16-MFMA GEMM tile, shared by the dense
// linear kernels and the grouped expert kernels.
//
//   * a 256-thread workgroup owns a BM x BN tile of outputs; its four waves
//     own (BM/WM) x (BN/WN) sub-tiles built from 32x32x16 fp16 MFMAs with
//     fp32 accumulators;
//   * per K step of 64 (two scale groups) the activation tile is copied to LDS
//     and the weight tile is dequantised into LDS as fp16: nibble -> 1024 + u
//     by mantissa OR, minus 1032 (exact), times the group scale (one rounding);
//     activations stay fp16, so the only operand rounding is w = RNE16(s * q);
//   * global loads run two K steps ahead of the MFMAs through two register
//     stages, and LDS is double-buffered; loads past the last K step repeat
//     it, so every iteration issues the same loads and the compiler's wait
//     counts stay exact;
//   * LDS rows are padded by 16 bytes so the 16-byte fragment reads of a
//     wavefront hit distinct banks;
//   * activation rows come from per-thread row pointers, so a tile can gather
//     its rows (tokens routed to one expert) from anywhere;
//   * with SWI the B tile interleaves 32-row blocks of two tensors (gate, up)
//     so one lane ends up holding g and u of the same output;
//   * with NORM the row sums of squares are gathered while staging the
//     activations and 1/rms per row lands in LDS for the epilogue.
#pragma once

#include "common.h"

namespace atsi {

typedef _Float16 g_half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 g_half2_t __attribute__((ext_vector_type(2)));
typedef float g_float16_t __attribute__((ext_vector_type(16)));

constexpr int kGemmBlock = 256;
constexpr int kBK = 64;          // K per LDS stage = two scale groups
constexpr int kLDSP = kBK + 8;   // padded LDS row length in halves
constexpr int kPre = 2;          // register stages of global loads in flight

__device__ __forceinline__ uint32_t pk_sub_mul(uint32_t t, g_half2_t off, g_half2_t s) {
  g_half2_t v = __builtin_bit_cast(g_half2_t, t);
  v = (v - off) * s;  // q exactly, then one rounding of s * q
  return __builtin_bit_cast(uint32_t, v);
}

// Dequantise one group (16 code bytes) into 32 fp16 weights in natural k order.
__device__ __forceinline__ void dequant_group(const uint4& cw, uint16_t sbits, uint4 (&out)[4]) {
  constexpr uint32_t kMagic = 0x64006400u;  // fp16 1024.0 in both halves
  const _Float16 s = __builtin_bit_cast(_Float16, sbits);
  const g_half2_t s2 = {s, s};
  const g_half2_t off = {(_Float16)1032.0f, (_Float16)1032.0f};
  const uint32_t w4[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t w = w4[i];
    const uint32_t t0 = pk_sub_mul((w & 0x000F000Fu) | kMagic, off, s2);          // (k0, k4)
    const uint32_t t1 = pk_sub_mul(((w >> 4) & 0x000F000Fu) | kMagic, off, s2);   // (k1, k5)
    const uint32_t t2 = pk_sub_mul(((w >> 8) & 0x000F000Fu) | kMagic, off, s2);   // (k2, k6)
    const uint32_t t3 = pk_sub_mul(((w >> 12) & 0x000F000Fu) | kMagic, off, s2);  // (k3, k7)
    out[i].x = __builtin_amdgcn_perm(t1, t0, 0x05040100u);  // (k0, k1)
    out[i].y = __builtin_amdgcn_perm(t3, t2, 0x05040100u);  // (k2, k3)
    out[i].z = __builtin_amdgcn_perm(t1, t0, 0x07060302u);  // (k4, k5)
    out[i].w = __builtin_amdgcn_perm(t3, t2, 0x07060302u);  // (k6, k7)
  }
}


template <int BM, int BN, int WM, int WN, bool SWI, bool NORM = false>
struct GemmCore {
  static_assert(WM * WN == 4, "four waves");
  static constexpr int SM = BM / WM, SN = BN / WN;  // wave sub-tile
  static constexpr int FM = SM / 32, FN = SN / 32;  // 32x32 fragments per wave
  static_assert(FM >= 1 && FN >= 1, "sub-tile at least 32x32");
  static_assert(!SWI || (SN % 64) == 0, "SwiGLU pairs gate/up fragments inside a wave");
  static constexpr int XV = BM * kBK / 8 / kGemmBlock;                 // 16-byte activation chunks per thread
  static constexpr int WG = (BN * 2 + kGemmBlock - 1) / kGemmBlock;    // weight groups per thread
  static_assert(XV >= 1 && (BM * kBK / 8) % kGemmBlock == 0, "activation tile must split evenly");
  static constexpr int NOUT = SWI ? BN / 2 : BN;                       // output columns per tile

  struct Smem {
    _Float16 As[2][BM * kLDSP];
    _Float16 Bs[2][BN * kLDSP];
    float rowinv[BM];
  };

  // activation tile row of chunk i of this thread
  __device__ static int xrow(int i) { return (threadIdx.x + i * kGemmBlock) / (kBK / 8); }

  // arow[i]: pointer to activation row xrow(i) (K halves), or nullptr for a row
  // outside the tile; safe: any readable 16-byte activation chunk.  Weight
  // rows n0 .. (n0 + NOUT) of w (and w2).
  __device__ static void run(Smem& sm, const __half* const (&arow)[XV], const __half* safe, const QView& w,
                             const QView& w2, int n0, int K, float eps, g_float16_t (&acc)[FM][FN]) {
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int ngrp = K / 32;
    const int nk = (K + kBK - 1) / kBK;

    uint4 xr[kPre][XV];
    uint4 cr[kPre][WG];
    uint16_t sr[kPre][WG];
    uint32_t sok[kPre][WG];  // 0xFFFF for a group inside the tensor, else 0
    float sq[XV];
#pragma unroll
    for (int i = 0; i < XV; ++i) sq[i] = 0.f;

    // global loads of K step kt (clamped to the last one) into stage st
    auto gload = [&](int st, int kt) {
      const int k0 = (kt < nk ? kt : nk - 1) * kBK;
#pragma unroll
      for (int i = 0; i < XV; ++i) {
        // loads are unconditional (rows outside the tile read `safe`, K past
        // the end its last chunk) and zeroed afterwards, so that every lane
        // issues the same loads
        const int cchunk = (tid + i * kGemmBlock) % (kBK / 8);
        const int k = k0 + cchunk * 8;
        const bool ok = arow[i] != nullptr && k < K;
        const __half* p = arow[i] != nullptr ? arow[i] + (k < K ? k : K - 8) : safe;
        const uint4 v = ldg16(p);
        xr[st][i] = ok ? v : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < WG; ++i) {
        // every thread loads (threads past the tile repeat its last group);
        // groups outside the tensor get scale 0 when dequantised
        const int idx = min(tid + i * kGemmBlock, BN * 2 - 1);
        const int br = idx >> 1, g = (k0 >> 5) + (idx & 1);
        int n;
        const QView* src = &w;
        if constexpr (SWI) {
          const int b32 = br >> 5;
          n = n0 + (b32 >> 1) * 32 + (br & 31);
          if (b32 & 1) src = &w2;
        } else {
          n = n0 + br;
        }
        const int nc = n < w.N ? n : w.N - 1, gc = g < ngrp ? g : ngrp - 1;
        cr[st][i] = ldg16(src->codes + (size_t)nc * (K / 2) + (size_t)gc * 16);
        sr[st][i] = ldg2(src->scales + (size_t)nc * ngrp + gc);
        sok[st][i] = n < w.N && g < ngrp ? 0xFFFFu : 0u;
      }
    };
    // stage st into LDS buffer buf (activations as they are, weights
    // dequantised); sq gathers row sums of squares once per K step
    auto lstore = [&](int st, int buf, float count) {
#pragma unroll
      for (int i = 0; i < XV; ++i) {
        const int idx = tid + i * kGemmBlock;
        const int r = idx / (kBK / 8), cchunk = idx % (kBK / 8);
        *reinterpret_cast<uint4*>(&sm.As[buf][r * kLDSP + cchunk * 8]) = xr[st][i];
        if constexpr (NORM) {
          const g_half2_t* h = reinterpret_cast<const g_half2_t*>(&xr[st][i]);
          float q = 0.f;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float a = (float)h[j][0], b = (float)h[j][1];
            q = fmaf(a, a, fmaf(b, b, q));
          }
          sq[i] = fmaf(count, q, sq[i]);  // count 0 for a repeated K step
        }
      }
#pragma unroll
      for (int i = 0; i < WG; ++i) {
        const int idx = tid + i * kGemmBlock;
        if constexpr ((BN * 2) % kGemmBlock != 0) {
          if (idx >= BN * 2) break;
        }
        const int r = idx >> 1, gl = idx & 1;
        uint4 o[4];
        dequant_group(cr[st][i], (uint16_t)(sr[st][i] & sok[st][i]), o);  // scale 0: weights 0
        uint4* dst = reinterpret_cast<uint4*>(&sm.Bs[buf][r * kLDSP + gl * 32]);
#pragma unroll
        for (int j = 0; j < 4; ++j) dst[j] = o[j];
      }
    };

#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // stage s and LDS buffer s hold K steps s, s + 2, s + 4, ...  The steady
    // state is one basic block per K step (MFMAs on one LDS buffer, the next
    // step's dequantisation into the other, the refill loads), so the
    // scheduler can overlap the dequantising VALU work with the MFMAs.
    gload(0, 0);
    gload(1, 1);
    lstore(0, 0, 1.f);
    gload(0, 2);
    __syncthreads();

    const int frow = lane & 31, fk = (lane >> 5) * 8;
    auto mfma_step = [&](int buf) {
#pragma unroll
      for (int ks = 0; ks < kBK / 16; ++ks) {
        g_half8_t a[FM], b[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i)
          a[i] = *reinterpret_cast<const g_half8_t*>(&sm.As[buf][(wm * SM + i * 32 + frow) * kLDSP + ks * 16 + fk]);
#pragma unroll
        for (int j = 0; j < FN; ++j)
          b[j] = *reinterpret_cast<const g_half8_t*>(&sm.Bs[buf][(wn * SN + j * 32 + frow) * kLDSP + ks * 16 + fk]);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
    };
    // K step kt on buffer st: MFMAs, stage st ^ 1 (K step kt + 1) into LDS,
    // refill stage st ^ 1 with K step kt + 3 (clamped, so every step issues
    // the same loads and the compiler waits for exactly one stage)
    int kt = 0;
    for (; kt + 2 <= nk; kt += 2) {
      mfma_step(0);
      lstore(1, 1, kt + 1 < nk ? 1.f : 0.f);
      gload(1, kt + 3);
      __syncthreads();
      mfma_step(1);
      lstore(0, 0, kt + 2 < nk ? 1.f : 0.f);
      gload(0, kt + 4);
      __syncthreads();
    }
    if (kt < nk) mfma_step(0);

    if constexpr (NORM) {
#pragma unroll
      for (int i = 0; i < XV; ++i) {
        float q = sq[i];
        q += __shfl_xor(q, 1, 64);
        q += __shfl_xor(q, 2, 64);
        q += __shfl_xor(q, 4, 64);
        const int idx = tid + i * kGemmBlock;
        if ((idx % (kBK / 8)) == 0) sm.rowinv[idx / (kBK / 8)] = 1.f / sqrtf(q / (float)K + eps);
      }
      __syncthreads();
    }
  }

  // Output coordinates of accumulator v of fragment (i, j): tile row and
  // output column (relative to n0).  D layout of a 32x32 MFMA block: lane l
  // holds column l % 32; accumulator v holds row 8 * (v / 4) + 4 * (l / 32) + v % 4.
  __device__ static int frag_row(int i, int v) {
    const int lane = threadIdx.x & 63, wm = (threadIdx.x >> 6) / WN;
    return wm * SM + i * 32 + 8 * (v >> 2) + (lane >> 5) * 4 + (v & 3);
  }
  __device__ static int frag_col(int j) {
    const int lane = threadIdx.x & 63, wn = (threadIdx.x >> 6) % WN;
    if constexpr (SWI) return ((wn * SN / 32 + j) >> 1) * 32 + (lane & 31);
    else return wn * SN + j * 32 + (lane & 31);
  }
};

}  // namespace atsi
