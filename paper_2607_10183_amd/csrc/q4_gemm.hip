// Prefill-path dequantising GEMM for block-int4 weights on CDNA4 (gfx950).
//
// Prefill runs a whole chunk of tokens through each linear (Sec. 2.2, chunked
// prefill in Sec. 5.1), a dense contraction, so it runs on the matrix cores:
//   * a 256-thread workgroup owns a BM x BN output tile; its four waves own
//     (BM/WM) x (BN/WN) sub-tiles built from 32x32x16 fp16 MFMAs with fp32
//     accumulators;
//   * per K step of 64 (two scale groups) the activation tile is copied to LDS
//     and the weight tile is dequantised into LDS as fp16: nibble -> 1024 + u
//     by mantissa OR, minus 1032 (exact), times the group scale (one rounding);
//     activations stay fp16, so the only operand rounding is w = RNE16(s * q);
//   * the next K step's global loads are issued before the current step's
//     MFMAs (register double-buffering) and LDS is double-buffered;
//   * LDS rows are padded by 16 bytes so the 16-byte fragment reads of a
//     wavefront hit distinct banks;
//   * workgroup ids are remapped so that the M tiles sharing one weight tile
//     run on the same XCD and reuse it from that XCD's L2.
// Like the GEMV, one launch covers several tensors sharing an input and fuses
// RMS normalisation (row sums of squares gathered while staging activations,
// applied to the fp32 accumulators), SwiGLU (the B tile interleaves 32-row
// blocks of gate and up so one lane holds g and u of the same output), the
// residual add and grouped-query head expansion.
#include <algorithm>

#include "common.h"

namespace atsi {
namespace {

constexpr int kBlock = 256;
constexpr int BK = 64;           // K per LDS stage = two scale groups
constexpr int LDSP = BK + 8;     // padded LDS row length in halves
constexpr uint32_t kMagic = 0x64006400u;

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef float float16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint32_t pk_sub_mul(uint32_t t, half2_t off, half2_t s) {
  half2_t v = __builtin_bit_cast(half2_t, t);
  v = (v - off) * s;  // q exactly, then one rounding of s * q
  return __builtin_bit_cast(uint32_t, v);
}

// Dequantise one group (16 code bytes) into 32 fp16 weights in natural k order.
__device__ __forceinline__ void dequant_group(const uint4& cw, uint16_t sbits, uint4 (&out)[4]) {
  const _Float16 s = __builtin_bit_cast(_Float16, sbits);
  const half2_t s2 = {s, s};
  const half2_t off = {(_Float16)1032.0f, (_Float16)1032.0f};
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

__device__ __forceinline__ float silu_f(float g) { return g / (1.f + expf(-g)); }

struct TileMap {
  int end[kMaxSeg];    // cumulative tile counts per segment
  int tiles_n[kMaxSeg];
  int tiles_m;
  int total;
};

template <int BM, int BN, int WM, int WN, bool SWI>
__global__ __launch_bounds__(kBlock, 2) void q4_gemm_kernel(LinOp op, TileMap tm_) {
  static_assert(WM * WN == 4, "four waves");
  constexpr int SM = BM / WM, SN = BN / WN;  // wave sub-tile
  constexpr int FM = SM / 32, FN = SN / 32;  // 32x32 fragments per wave
  static_assert(FM >= 1 && FN >= 1, "sub-tile at least 32x32");
  static_assert(!SWI || (SN % 64) == 0, "SwiGLU pairs gate/up fragments inside a wave");
  constexpr int XV = BM * BK / 8 / kBlock;            // uint4 of activations per thread
  constexpr int WG = (BN * 2 + kBlock - 1) / kBlock;  // weight groups per thread (BN rows x 2 groups)
  static_assert(XV >= 1 && (BM * BK / 8) % kBlock == 0, "activation tile must split evenly");
  constexpr int NOUT = SWI ? BN / 2 : BN;             // output columns per tile

  __shared__ __attribute__((aligned(16))) _Float16 As[2][BM * LDSP];
  __shared__ __attribute__((aligned(16))) _Float16 Bs[2][BN * LDSP];
  __shared__ float rowinv[BM];

  // XCD-aware tile order: consecutive ids land on different XCDs (8-way
  // round robin); give each XCD a contiguous run of tiles, M fastest.
  int bid = blockIdx.x;
  if ((tm_.total & 7) == 0) bid = (bid & 7) * (tm_.total >> 3) + (bid >> 3);
  int s = 0;
  while (s < op.nseg - 1 && bid >= tm_.end[s]) ++s;
  const int local = bid - (s ? tm_.end[s - 1] : 0);
  const int tmi = local % tm_.tiles_m, tni = local / tm_.tiles_m;
  const Seg& sg = op.seg[s];
  const QView w = sg.w, w2 = sg.w2;
  const int m0 = tmi * BM, n0 = tni * NOUT;
  const int M = op.M;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int K = op.K;
  const int ngrp = K / 32;
  const int nk = (K + BK - 1) / BK;

  uint4 xr[XV];
  uint4 cr[WG];
  uint16_t sr[WG];
  float sq[XV];
#pragma unroll
  for (int i = 0; i < XV; ++i) sq[i] = 0.f;

  auto gload = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = tid + i * kBlock;    // 8-half chunk index within the tile
      const int r = idx / (BK / 8), cchunk = idx % (BK / 8);
      const int m = m0 + r, k = k0 + cchunk * 8;
      if (m < M && k < K)
        xr[i] = *reinterpret_cast<const uint4*>(op.x + (size_t)m * K + k);
      else
        xr[i] = make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < WG; ++i) {
      const int idx = tid + i * kBlock;
      if (idx >= BN * 2) break;
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
      if (n < w.N && g < ngrp) {
        cr[i] = *reinterpret_cast<const uint4*>(src->codes + (size_t)n * (K / 2) + (size_t)g * 16);
        sr[i] = src->scales[(size_t)n * ngrp + g];
      } else {
        cr[i] = make_uint4(0x88888888u, 0x88888888u, 0x88888888u, 0x88888888u);  // q = 0
        sr[i] = 0;
      }
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int idx = tid + i * kBlock;
      const int r = idx / (BK / 8), cchunk = idx % (BK / 8);
      *reinterpret_cast<uint4*>(&As[buf][r * LDSP + cchunk * 8]) = xr[i];
      if (op.norm) {
        const half2_t* h = reinterpret_cast<const half2_t*>(&xr[i]);
        float q = sq[i];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float a = (float)h[j][0], b = (float)h[j][1];
          q = fmaf(a, a, fmaf(b, b, q));
        }
        sq[i] = q;
      }
    }
#pragma unroll
    for (int i = 0; i < WG; ++i) {
      const int idx = tid + i * kBlock;
      if (idx >= BN * 2) break;
      const int r = idx >> 1, gl = idx & 1;
      uint4 o[4];
      dequant_group(cr[i], sr[i], o);
      uint4* dst = reinterpret_cast<uint4*>(&Bs[buf][r * LDSP + gl * 32]);
#pragma unroll
      for (int j = 0; j < 4; ++j) dst[j] = o[j];
    }
  };

  float16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  gload(0);
  lstore(0);
  __syncthreads();

  const int frow = lane & 31, fk = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      half8_t a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = *reinterpret_cast<const half8_t*>(&As[buf][(wm * SM + i * 32 + frow) * LDSP + ks * 16 + fk]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = *reinterpret_cast<const half8_t*>(&Bs[buf][(wn * SN + j * 32 + frow) * LDSP + ks * 16 + fk]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      lstore(buf ^ 1);
      __syncthreads();
    }
  }

  // fused RMS normalisation: 1 / sqrt(mean(x^2) + eps) per row of the tile
  if (op.norm) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      float q = sq[i];
      q += __shfl_xor(q, 1, 64);
      q += __shfl_xor(q, 2, 64);
      q += __shfl_xor(q, 4, 64);
      const int idx = tid + i * kBlock;
      if ((idx % (BK / 8)) == 0) rowinv[idx / (BK / 8)] = 1.f / sqrtf(q / (float)K + op.eps);
    }
    __syncthreads();
  }

  // D layout of a 32x32 MFMA block: lane l holds column l % 32; accumulator v
  // holds row 8 * (v / 4) + 4 * (l / 32) + v % 4.
  const int col = lane & 31, rq = (lane >> 5) * 4;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      if (SWI && (j & 1)) continue;
      int n;
      if constexpr (SWI) n = n0 + ((wn * SN / 32 + j) >> 1) * 32 + col;
      else n = n0 + wn * SN + j * 32 + col;
      if (n >= w.N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int ml = wm * SM + i * 32 + 8 * (v >> 2) + rq + (v & 3);
        const int m = m0 + ml;
        if (m >= M) continue;
        const float sc = op.norm ? rowinv[ml] : 1.f;
        float o = acc[i][j][v] * sc;
        if constexpr (SWI) o = silu_f(o) * (acc[i][j + 1][v] * sc);
        if (sg.expand > 1) {
          const int hd = op.head_dim, jh = n / hd, d = n % hd;
          const __half h = __float2half_rn(o);
          for (int g = 0; g < sg.expand; ++g)
            sg.y[(size_t)m * sg.ldy + (size_t)(jh * sg.expand + g) * hd + d] = h;
        } else {
          const size_t at = (size_t)m * sg.ldy + n;
          if (op.res && s == 0) o += __half2float(op.res[at]);
          sg.y[at] = __float2half_rn(o);
        }
      }
    }
}

template <int BM, int BN, int WM, int WN, bool SWI>
hipError_t launch_tile(const LinOp& op, hipStream_t st) {
  constexpr int NOUT = SWI ? BN / 2 : BN;
  TileMap tm{};
  tm.tiles_m = (op.M + BM - 1) / BM;
  int total = 0;
  for (int s = 0; s < op.nseg; ++s) {
    tm.tiles_n[s] = (op.seg[s].w.N + NOUT - 1) / NOUT;
    total += tm.tiles_m * tm.tiles_n[s];
    tm.end[s] = total;
  }
  tm.total = total;
  hipLaunchKernelGGL((q4_gemm_kernel<BM, BN, WM, WN, SWI>), dim3(total), dim3(kBlock), 0, st, op, tm);
  return hipGetLastError();
}

// unpack kernel for the debug export: q[n][k] = nibble - 8
__global__ void unpack_kernel(QView w, int8_t* q) {
  const size_t total = (size_t)w.N * (w.K / 2);
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const uint8_t b = w.codes[i];
    q[2 * i] = (int8_t)((b & 0xF) - 8);
    q[2 * i + 1] = (int8_t)((b >> 4) - 8);
  }
}

}  // namespace

hipError_t launch_gemm(const LinOp& op, hipStream_t st) {
  long n = 0;
  for (int s = 0; s < op.nseg; ++s) n += op.seg[s].w.N;
  if (op.swiglu) {
    if (op.M <= 64) return launch_tile<64, 128, 2, 2, true>(op, st);
    return launch_tile<128, 128, 2, 2, true>(op, st);
  }
  // Prefer 128x128 tiles; narrower tiles when the grid would leave most of
  // the 256 CUs idle.
  const long t128 = (long)((op.M + 127) / 128) * ((n + 127) / 128);
  if (op.M <= 64) return launch_tile<64, 64, 2, 2, false>(op, st);
  if (t128 >= 256) return launch_tile<128, 128, 2, 2, false>(op, st);
  return launch_tile<128, 64, 2, 2, false>(op, st);
}

hipError_t launch_unpack(const QView& w, int8_t* q, hipStream_t s) {
  const size_t total = (size_t)w.N * (w.K / 2);
  const int blocks = (int)std::min<size_t>((total + 255) / 256, 4096);
  hipLaunchKernelGGL(unpack_kernel, dim3(blocks), dim3(256), 0, s, w, q);
  return hipGetLastError();
}

}  // namespace atsi
