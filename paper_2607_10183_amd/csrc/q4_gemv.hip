// Decode-path dequantising GEMV for block-int4 weights on CDNA4 (gfx950).
//
// y[m][n] = sum_g s[n][g] * sum_{k in g} q[n][k] * x[m][k] for M <= 4 tokens.
// Decode reads every weight byte once per token (the memory-bound phase,
// Sec. 2.2), so the kernel is organised around streaming the packed codes at
// HBM rate:
//   * a wavefront owns RW consecutive rows; lane l handles groups l, l+64, ...
//     of every row, so one 128-bit load per lane covers one whole group of 32
//     inputs and a wave instruction reads 1 KiB contiguous from a row;
//   * nibbles become fp16 values 1024 + u by OR-ing them into the mantissa of
//     0x6400 (two per 32-bit register), then v_dot2_f32_f16 multiplies two of
//     them by two activations and accumulates in fp32;
//   * the +1032 offset of (1024 + u) against q = u - 8 is removed once per
//     group with the group sum of x, computed once per chunk and reused by the
//     RW rows; the group partial is scaled by its fp16 scale in fp32;
//   * activations are read once per wave and permuted in registers to the
//     (k, k+4) pairing the nibble extraction yields;
//   * lanes reduce across the wavefront with DPP/shuffles; one lane per
//     (row, token) rounds to fp16 once.
// One launch can cover several tensors that read the same input (Q, K and V;
// the gate/up pair of a SwiGLU FFN) and fuses the RMS normalisation of the
// input (the sum of squares rides along the activation loads), the SwiGLU
// product, the residual add and the grouped-query head expansion of a
// context-length-1 attention into the epilogue.
#include "q4_gemv_core.h"

namespace atsi {
namespace {

using namespace gemv;

struct BlockMap {
  int end[kMaxSeg];  // cumulative block counts per segment
};

template <int MT, int RW, bool SWI>
__global__ __launch_bounds__(kBlock) void q4_gemv_kernel(LinOp op, BlockMap bm) {
  int s = 0;
  while (s < op.nseg - 1 && (int)blockIdx.x >= bm.end[s]) ++s;
  const int local = (int)blockIdx.x - (s ? bm.end[s - 1] : 0);
  const Seg& sg = op.seg[s];
  const QView w = sg.w;
  const QView w2 = sg.w2;

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int row0 = (local * (kBlock / kWave) + wave) * RW;
  if (row0 >= w.N) return;
  const int K = op.K, M = op.M;
  const int nchunk = K / kGroup;
  const size_t rbytes = (size_t)K / 2;

  float acc[RW][MT], acc2[SWI ? RW : 1][MT], sq[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    sq[m] = 0.f;
#pragma unroll
    for (int r = 0; r < RW; ++r) acc[r][m] = 0.f;
#pragma unroll
    for (int r = 0; r < (SWI ? RW : 1); ++r) acc2[r][m] = 0.f;
  }

  for (int c = lane; c < nchunk; c += kWave) {
    uint4 cw[RW], cw2[SWI ? RW : 1];
    float sc[RW], sc2[SWI ? RW : 1];
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      const int row = min(row0 + r, w.N - 1);  // clamped rows are computed, never stored
      cw[r] = *reinterpret_cast<const uint4*>(w.codes + (size_t)row * rbytes + (size_t)c * 16);
      sc[r] = __half2float(__ushort_as_half(w.scales[(size_t)row * nchunk + c]));
      if constexpr (SWI) {
        cw2[r] = *reinterpret_cast<const uint4*>(w2.codes + (size_t)row * rbytes + (size_t)c * 16);
        sc2[r] = __half2float(__ushort_as_half(w2.scales[(size_t)row * nchunk + c]));
      }
    }
    XChunk<MT> xc;
    load_x<MT>(xc, op.x, K, M, c, op.norm != 0, sq);
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      float part[MT];
      group_dot<MT>(cw[r], xc, part);
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = fmaf(sc[r], part[m] - 1032.f * xc.sum[m], acc[r][m]);
      if constexpr (SWI) {
        group_dot<MT>(cw2[r], xc, part);
#pragma unroll
        for (int m = 0; m < MT; ++m) acc2[r][m] = fmaf(sc2[r], part[m] - 1032.f * xc.sum[m], acc2[r][m]);
      }
    }
  }

  float inv_r[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) inv_r[m] = op.norm ? 1.f / sqrtf(wave_sum(sq[m]) / (float)K + op.eps) : 1.f;

#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float v = wave_sum(acc[r][m]) * inv_r[m];
      if constexpr (SWI) {
        const float u = wave_sum(acc2[r][m]) * inv_r[m];
        v = silu_f(v) * u;
      }
      const int row = row0 + r;
      if (lane == r * MT + m && row < w.N && m < M) {
        if (sg.expand > 1) {
          const int hd = op.head_dim, j = row / hd, d = row % hd;
          const __half o = __float2half_rn(v);
          for (int g = 0; g < sg.expand; ++g) sg.y[(size_t)m * sg.ldy + (size_t)(j * sg.expand + g) * hd + d] = o;
        } else {
          const size_t at = (size_t)m * sg.ldy + row;
          if (op.res && s == 0) v += __half2float(op.res[at]);
          sg.y[at] = __float2half_rn(v);
        }
      }
    }
}

template <int MT, int RW, bool SWI>
hipError_t launch_cfg(const LinOp& op, hipStream_t st) {
  const int rows_per_block = (kBlock / kWave) * RW;
  BlockMap bm{};
  int total = 0;
  for (int s = 0; s < op.nseg; ++s) {
    total += (op.seg[s].w.N + rows_per_block - 1) / rows_per_block;
    bm.end[s] = total;
  }
  hipLaunchKernelGGL((q4_gemv_kernel<MT, RW, SWI>), dim3(total), dim3(kBlock), 0, st, op, bm);
  return hipGetLastError();
}

template <int MT, bool SWI>
hipError_t launch_mt(const LinOp& op, hipStream_t st) {
  int n = 0;
  for (int s = 0; s < op.nseg; ++s) n += op.seg[s].w.N;
  // rows per wave: at least ~2 blocks per CU when N allows, more bytes in
  // flight per wave when it does not matter
  if (n >= 8192 && !SWI) return launch_cfg<MT, 4, SWI>(op, st);
  if (n >= 4096) return launch_cfg<MT, 2, SWI>(op, st);
  return launch_cfg<MT, 1, SWI>(op, st);
}

template <bool SWI>
hipError_t launch_sw(const LinOp& op, hipStream_t st) {
  if (op.M == 1) return launch_mt<1, SWI>(op, st);
  if (op.M == 2) return launch_mt<2, SWI>(op, st);
  return launch_mt<4, SWI>(op, st);
}

}  // namespace

hipError_t launch_gemv(const LinOp& op, hipStream_t st) {
  return op.swiglu ? launch_sw<true>(op, st) : launch_sw<false>(op, st);
}

}  // namespace atsi
