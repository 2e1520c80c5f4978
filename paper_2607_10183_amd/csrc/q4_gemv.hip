// Decode-path dequantising GEMV for block-int4 weights on CDNA4 (gfx950).
//
// y[m][n] = sum_g s[n][g] * sum_{k in g} q[n][k] * x[m][k] for M <= 4 tokens.
// Decode reads every weight byte once per token (the memory-bound phase,
// Sec. 2.2), so the kernel is built to keep HBM busy:
//   * the first step's weight loads are issued before anything else; then the
//     workgroup stages its activations once in LDS, already permuted to the
//     (k, k+4) pairs the nibble extraction yields, with each group's offset
//     correction (and, for a fused RMS norm, the sum of squares);
//   * a wavefront walks SPW steps of RW rows; lane l handles groups l, l+64, ...
//     of a row, so one 128-bit load covers one 32-input group and a wave
//     instruction reads 1 KiB contiguous from a row;
//   * steps alternate between two register buffers: the next step's codes and
//     scales are loaded (unconditionally, rows and groups clamped, so the
//     compiler counts outstanding loads exactly) before the current step is
//     computed, keeping a step of loads in flight per wave; steps per wave
//     are a compile-time constant, so no load is issued past a wave's last
//     step (those rows belong to the next workgroup and would be read twice);
//   * arithmetic per group: four ALU ops make eight fp16 weights-plus-offset
//     values, v_dot2_f32_f16 accumulates exact products in fp32, one FMA
//     removes the offset and one applies the fp16 scale (q4_gemv_core.h);
//   * lanes reduce across the wavefront with shuffles; one lane per
//     (row, token) rounds to fp16 once.
// One launch can cover several tensors that read the same input (Q, K and V;
// the gate/up pair of a SwiGLU FFN) and fuses the RMS normalisation of the
// input, the SwiGLU product, the residual add and the grouped-query head
// expansion of a context-length-1 attention into the epilogue.
#include "q4_gemv_core.h"

namespace atsi {
namespace {

using namespace gemv;

struct BlockMap {
  int end[kMaxSeg];  // cumulative block counts per segment
  int rows_per_block;
};

// LDS layout: activation pairs as uint4 [word b][token m][group c]
// (consecutive lanes read consecutive 16-byte words), then the float offset
// corrections [m][c].
template <int MT>
__device__ __forceinline__ void stage_x(char* smem, const __half* __restrict__ x, int K, int M, bool norm,
                                        float (&inv_r)[MT], float eps) {
  __shared__ float red[kBlock / kWave][MT];
  const int nchunk = K / kGroup;
  uint4* xw = reinterpret_cast<uint4*>(smem);
  float* xc = reinterpret_cast<float*>(smem + (size_t)4 * MT * nchunk * 16);
  float sq[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) sq[m] = 0.f;
  for (int c = threadIdx.x; c < nchunk; c += kBlock) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      XRaw r;
      XGroup g;
      if (m < M) {
        load_xraw(r, x + (size_t)m * K, c);
      } else {
#pragma unroll
        for (int b = 0; b < 4; ++b) r.d[b] = make_uint4(0, 0, 0, 0);
      }
      prep_x(g, r, norm, sq[m]);
#pragma unroll
      for (int b = 0; b < 4; ++b)
        xw[((size_t)b * MT + m) * nchunk + c] = make_uint4(g.p[4 * b], g.p[4 * b + 1], g.p[4 * b + 2], g.p[4 * b + 3]);
      xc[(size_t)m * nchunk + c] = g.corr;
    }
  }
  if (norm) {
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const float v = wave_sum(sq[m]);
      if (lane == 0) red[wave][m] = v;
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < kBlock / kWave; ++w) t += red[w][m];
      inv_r[m] = 1.f / sqrtf(t / (float)K + eps);
    }
  } else {
#pragma unroll
    for (int m = 0; m < MT; ++m) inv_r[m] = 1.f;
  }
  __syncthreads();
}

// codes and scales of one step: RW rows (of two tensors for SwiGLU), CPL groups per lane
template <int RW, int CPL, bool SWI>
struct Step {
  uint4 c[SWI ? 2 : 1][RW][CPL];
  uint16_t s[SWI ? 2 : 1][RW][CPL];
};

template <int RW, int CPL, bool SWI>
__device__ __forceinline__ void load_step(Step<RW, CPL, SWI>& st, const QView& w, const QView& w2, int row0, int lane,
                                          int nchunk) {
  const size_t rbytes = (size_t)nchunk * 16;
#pragma unroll
  for (int t = 0; t < (SWI ? 2 : 1); ++t) {
    const QView& v = t ? w2 : w;
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      const int row = min(row0 + r, v.N - 1);  // clamped rows are computed, never stored
      const uint8_t* cr = v.codes + (size_t)row * rbytes;
      const uint16_t* sr = v.scales + (size_t)row * nchunk;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c = min(lane + j * kWave, nchunk - 1);  // groups past the row end are not used
        st.c[t][r][j] = ldg16(cr + (size_t)c * 16);
        st.s[t][r][j] = ldg2(sr + c);
      }
    }
  }
}

template <int MT>
struct GemvCtx {
  const uint4* xw;
  const float* xc;
  int nchunk, lane;
  float inv_r[MT];
};

// Compute one step from its loaded codes and write its RW x MT outputs.
template <int MT, int RW, int CPL, bool SWI>
__device__ __forceinline__ void compute_step(const Step<RW, CPL, SWI>& cur, const GemvCtx<MT>& gc, const LinOp& op,
                                             const Seg& sg, int s, int row0, int M, int N) {
  constexpr int NT = SWI ? 2 : 1;
  const int lane = gc.lane, nchunk = gc.nchunk;
  float acc[NT][RW][MT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[t][r][m] = 0.f;
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int c = lane + j * kWave;
    const bool ok = c < nchunk;
    const int cc = ok ? c : nchunk - 1;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      XGroup g;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const uint4 v = gc.xw[((size_t)b * MT + m) * nchunk + cc];
        g.p[4 * b] = v.x;
        g.p[4 * b + 1] = v.y;
        g.p[4 * b + 2] = v.z;
        g.p[4 * b + 3] = v.w;
      }
      g.corr = gc.xc[(size_t)m * nchunk + cc];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < RW; ++r) {
          const float sc = ok ? __half2float(__ushort_as_half(cur.s[t][r][j])) : 0.f;
          acc[t][r][m] = fmaf(sc, group_dot(cur.c[t][r][j], g), acc[t][r][m]);
        }
    }
  }
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float v = wave_sum(acc[0][r][m]) * gc.inv_r[m];
      if constexpr (SWI) {
        const float u = wave_sum(acc[NT - 1][r][m]) * gc.inv_r[m];
        v = silu_f(v) * u;
      }
      const int row = row0 + r;
      if (lane == r * MT + m && row < N && m < M) emit_out(op, sg, s, m, row, v);
    }
}

template <int MT, int RW, int CPL, bool SWI, int SPW>
__global__ __launch_bounds__(kBlock) void q4_gemv_kernel(LinOp op, BlockMap bm) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int s = 0;
  while (s < op.nseg - 1 && (int)blockIdx.x >= bm.end[s]) ++s;
  const int local = (int)blockIdx.x - (s ? bm.end[s - 1] : 0);
  const Seg& sg = op.seg[s];
  const QView w = sg.w;
  const QView w2 = sg.w2;
  const int K = op.K, M = op.M;
  const int nchunk = K / kGroup;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  constexpr int NW = kBlock / kWave;
  const int blk_row0 = local * bm.rows_per_block;
  // step i of this wave covers rows blk_row0 + (i * NW + wave) * RW + [0, RW)
  auto step_row = [&](int i) { return blk_row0 + (i * NW + wave) * RW; };

  // weight loads of the first step go out before the activations are staged
  Step<RW, CPL, SWI> buf[2];
  load_step(buf[0], w, w2, step_row(0), lane, nchunk);

  GemvCtx<MT> gc;
  stage_x<MT>(smem, op.x, K, M, op.norm != 0, gc.inv_r, op.eps);
  gc.xw = reinterpret_cast<const uint4*>(smem);
  gc.xc = reinterpret_cast<const float*>(smem + (size_t)4 * MT * nchunk * 16);
  gc.nchunk = nchunk;
  gc.lane = lane;

  // the next step's loads go out before the current step is computed
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    if (i + 1 < SPW) load_step(buf[(i + 1) & 1], w, w2, step_row(i + 1), lane, nchunk);
    if (step_row(i) < w.N) compute_step(buf[i & 1], gc, op, sg, s, step_row(i), M, w.N);
  }
}

template <int MT, int RW, int CPL, bool SWI, int SPW>
hipError_t launch_cfg(const LinOp& op, hipStream_t st) {
  BlockMap bm{};
  bm.rows_per_block = (kBlock / kWave) * RW * SPW;
  int total = 0;
  for (int s = 0; s < op.nseg; ++s) {
    total += (op.seg[s].w.N + bm.rows_per_block - 1) / bm.rows_per_block;
    bm.end[s] = total;
  }
  const int nchunk = op.K / kGroup;
  const size_t lds = (size_t)4 * MT * nchunk * 16 + (size_t)MT * nchunk * 4;
  // HIP admits dynamic LDS up to the device's per-workgroup limit without a
  // function attribute
  if (lds > lds_limit()) return hipErrorInvalidValue;  // callers check gemv_tokens()
  hipLaunchKernelGGL((q4_gemv_kernel<MT, RW, CPL, SWI, SPW>), dim3(total), dim3(kBlock), lds, st, op, bm);
  return hipGetLastError();
}

template <int MT, int RW, int CPL, bool SWI>
hipError_t launch_spw(const LinOp& op, int spw, hipStream_t st) {
  if (spw >= 2) return launch_cfg<MT, RW, CPL, SWI, 2>(op, st);
  return launch_cfg<MT, RW, CPL, SWI, 1>(op, st);
}

// Groups per lane (CPL) follow K; one row per step.
template <int MT, bool SWI>
hipError_t launch_mt(const LinOp& op, int spw, hipStream_t st) {
  const int nchunk = op.K / kGroup;
  if (nchunk <= 64) return launch_spw<MT, 1, 1, SWI>(op, spw, st);
  if (nchunk <= 128) return launch_spw<MT, 1, 2, SWI>(op, spw, st);
  if (nchunk <= 256) return launch_spw<MT, 1, 4, SWI>(op, spw, st);
  if (nchunk <= 448) return launch_spw<MT, 1, 7, SWI>(op, spw, st);
  if (nchunk <= 512) return launch_spw<MT, 1, 8, SWI>(op, spw, st);
  return launch_spw<MT, 1, 16, SWI>(op, spw, st);
}

template <bool SWI>
hipError_t launch_sw(const LinOp& op, int spw, hipStream_t st) {
  if (op.M == 1) return launch_mt<1, SWI>(op, spw, st);
  if (op.M == 2) return launch_mt<2, SWI>(op, spw, st);
  return launch_mt<4, SWI>(op, spw, st);
}

// Steps per wave, measured on MI355X (batch 1): two for plain tensors of
// 2048+ rows; one for the fused gate/up pair (each step already covers a row
// of both tensors) and for small tensors, where the grid would be too small.
int default_spw(const LinOp& op) {
  int n = 0;
  for (int s = 0; s < op.nseg; ++s) n += op.seg[s].w.N;
  if (op.swiglu) return 1;
  return n >= 2048 ? 2 : 1;
}

}  // namespace

size_t lds_limit() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 64 * 1024;
  if (!cached[dev]) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0)
      v = 64 * 1024;
    cached[dev] = v;
  }
  return (size_t)cached[dev];
}

int gemv_tokens(int K) {
  const size_t per_token = (size_t)(K / kGroup) * 68;
  const size_t lim = lds_limit();
  for (int mt = kGemvMaxTokens; mt >= 1; mt /= 2)
    if (mt * per_token <= lim) return mt;
  return 0;
}

hipError_t launch_gemv(const LinOp& op, hipStream_t st) {
  const int spw = default_spw(op);
  return op.swiglu ? launch_sw<true>(op, spw, st) : launch_sw<false>(op, spw, st);
}

}  // namespace atsi
