// Decode-path dequantising GEMV for block-int4 weights on CDNA4 (gfx950).
//
// y[m][n] = sum_g s[n][g] * sum_{k in g} q[n][k] * x[m][k].  Decode reads
// every weight byte once per token (the memory-bound phase, Sec. 2.2), so
// both kernels here are built to keep HBM busy while the arithmetic hides
// under the loads.
//
// One token (q4_gemv1_kernel):
//   * a workgroup of S x P waves owns R = P x C consecutive rows; wave (s, p)
//     takes K-slice s (groups 64 s .. 64 s + 63, one group per lane, so one
//     128-bit load per lane reads 1 KiB of a row contiguously) of rows
//     r0 + p + P i, i < C; the P waves of a slice read neighbouring rows;
//   * the workgroup stages the activations once in LDS, already permuted to
//     the (k, k+4) pairs the nibble extraction yields, with each group's
//     offset correction (and the sum of squares for a fused RMS norm); each
//     lane then keeps its one group in registers for all C rows;
//   * the first D - 1 rows' loads are issued before the staging, and each row
//     refills the register buffer consumed by the previous one, so D - 1 rows
//     stay in flight per wave; loads are non-temporal buffer loads whose
//     out-of-range lanes (rows past N, groups past K) read zeros;
//   * per group: four ALU ops make eight fp16 weight-plus-offset values,
//     v_dot2_f32_f16 accumulates exact products in fp32, one FMA removes the
//     offset and one applies the fp16 scale (q4_gemv_core.h);
//   * a lane carries one partial per (row, tensor); after the last row the
//     wave sums all of them at once with a transposed butterfly (permlane32
//     and permlane16 swaps, then DPP inside rows of 16 lanes), and the S
//     slices meet in LDS, where one thread per row applies the epilogue.
// Up to 4 tokens (q4_gemv_kernel, used where the batched-decode kernel does
// not apply): a wavefront walks rows with lane l on groups l, l+64, ..., the
// activations staged in LDS per token and read back per row.
// One launch can cover several tensors that read the same input (Q, K and V;
// the gate/up pair of a SwiGLU FFN) and fuses the RMS normalisation of the
// input, the SwiGLU product, the residual add and the grouped-query head
// expansion of a context-length-1 attention into the epilogue.
#include <algorithm>
#include <cmath>

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

// ---------------------------------------------------------------- one token

constexpr uint32_t kOobOff = 0x80000000u;  // an offset past every buffer here

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

constexpr int kNtBits = 2;  // cache policy of the weight loads: non-temporal

struct Gemv1Map {
  int end[kMaxSeg];  // cumulative workgroup counts per segment
  int S;             // K slices (waves per row)
  int P;             // row partitions
};

constexpr int pad_pow2(int v) { return v <= 4 ? 4 : (v <= 8 ? 8 : 16); }

template <int C, bool SWI, int D>
__global__ __launch_bounds__(1024) void q4_gemv1_kernel(LinOp op, Gemv1Map m) {
  constexpr int NT = SWI ? 2 : 1;
  constexpr int V = pad_pow2(NT * C);
  static_assert(NT * C <= V, "one partial per row and tensor: at most 16 per lane");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ float sq_wave[16];
  int sgi = 0;
  while (sgi < op.nseg - 1 && (int)blockIdx.x >= m.end[sgi]) ++sgi;
  const int local = (int)blockIdx.x - (sgi ? m.end[sgi - 1] : 0);
  const Seg& sg = op.seg[sgi];
  const int K = op.K, G = K / kGroup, N = sg.w.N;
  const int S = m.S, P = m.P;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int s = wave % S, p = wave / S;
  const int r0 = local * P * C;
  const int g = 64 * s + lane;
  const bool gok = g < G;

  __amdgpu_buffer_rsrc_t rc[NT], rs[NT];
  rc[0] = buf_rsrc(sg.w.codes, (uint32_t)((size_t)N * K / 2));
  rs[0] = buf_rsrc(sg.w.scales, (uint32_t)((size_t)N * G * 2));
  if constexpr (SWI) {
    rc[1] = buf_rsrc(sg.w2.codes, (uint32_t)((size_t)N * K / 2));
    rs[1] = buf_rsrc(sg.w2.scales, (uint32_t)((size_t)N * G * 2));
  }
  struct Ld {
    u32x4_g c[NT];
    uint32_t s[NT];
  };
  // row i of this wave (rows past the block or the tensor read zeros)
  auto load = [&](Ld& b, int i) {
    const int row = i < C ? r0 + p + P * i : N;
    const uint32_t co = gok ? (uint32_t)row * (uint32_t)(K / 2) + (uint32_t)g * 16 : kOobOff;
    const uint32_t so = gok ? ((uint32_t)row * (uint32_t)G + (uint32_t)g) * 2 : kOobOff;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      b.c[t] = __builtin_bit_cast(u32x4_g, __builtin_amdgcn_raw_buffer_load_b128(rc[t], co, 0, kNtBits));
      b.s[t] = __builtin_amdgcn_raw_buffer_load_b16(rs[t], so, 0, kNtBits);
    }
  };
  Ld buf[D];
#pragma unroll
  for (int d = 0; d < D - 1; ++d) load(buf[d], d);

  // activations: [group][16 pairs + correction], then the slice partials [S][P][V]
  uint32_t* xs = reinterpret_cast<uint32_t*>(smem);
  float* red = reinterpret_cast<float*>(smem + (size_t)G * 68);
  float sq = 0.f;
  for (int c = threadIdx.x; c < G; c += S * P * kWave) {
    XRaw r;
    XGroup gx;
    load_xraw(r, op.x, c);
    prep_x(gx, r, op.norm != 0, sq);
#pragma unroll
    for (int i = 0; i < 16; ++i) xs[c * 17 + i] = gx.p[i];
    xs[c * 17 + 16] = __float_as_uint(gx.corr);
  }
  if (op.norm) {
    const float t = wave_total(sq);
    if (lane == 0) sq_wave[wave] = t;
  }
  __syncthreads();
  float inv_r = 1.f;
  if (op.norm) {
    float t = 0.f;
    for (int w = 0; w < S * P; ++w) t += sq_wave[w];
    inv_r = 1.f / sqrtf(t / (float)K + op.eps);
  }
  XGroup xg;
  {
    const int c = gok ? g : 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) xg.p[i] = xs[c * 17 + i];
    xg.corr = __uint_as_float(xs[c * 17 + 16]);
  }
  const UnpackMasks um = unpack_masks();

  float part[V];
#pragma unroll
  for (int i = 0; i < V; ++i) part[i] = 0.f;
#pragma unroll
  for (int i = 0; i < C; ++i) {
    load(buf[(i + D - 1) % D], i + D - 1);
    const Ld& cur = buf[i % D];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float sc = gok ? __half2float(__ushort_as_half((uint16_t)cur.s[t])) : 0.f;
      const uint4 cw = make_uint4(cur.c[t].x, cur.c[t].y, cur.c[t].z, cur.c[t].w);
      part[t * C + i] = sc * group_dot_m(cw, xg, um);
    }
  }
  transpose_reduce<V>(part);
  if ((lane & 15) == 0) {
    const int rr = lane >> 4;
#pragma unroll
    for (int i = 0; i < V / 4; ++i) red[(s * P + p) * V + i + (V / 4) * (rr & 1) + (V / 2) * (rr >> 1)] = part[i];
  }
  __syncthreads();
  const int tid = threadIdx.x;
  if (tid < P * C) {
    const int pp = tid % P, i = tid / P;
    const int row = r0 + pp + P * i;
    float a[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      float sum = 0.f;
      for (int ss = 0; ss < S; ++ss) sum += red[(ss * P + pp) * V + t * C + i];
      a[t] = sum * inv_r;
    }
    float v = a[0];
    if constexpr (SWI) v = silu_f(a[0]) * a[NT - 1];
    if (row < N) emit_out(op, sg, sgi, 0, row, v);
  }
}

// Rows per wave C (compile time) and row partitions P for a batch-1 launch:
// about two workgroups per CU over all segments (256 CUs), at most 16 waves
// per workgroup.  Measured on MI355X: 7 rows per wave with 4 partitions for
// the 4096 x 14336 gate/up pair, 4 x 2 for 4096 x 4096 and 14336 x 4096,
// 2 x 2 for 4096 x 1024.
struct Gemv1Shape {
  int C, P;
};
Gemv1Shape gemv1_shape(long rows, int S) {
  const int pmax = std::max(1, 16 / S);
  const double target = std::max(4.0, (double)rows / 512.0);
  const int cs[4] = {7, 4, 8, 2};  // ties go to the earlier entry
  Gemv1Shape best{2, 1};
  double berr = 1e30;
  for (int ci = 0; ci < 4; ++ci)
    for (int P = 1; P <= pmax; ++P) {
      const double err = std::fabs(cs[ci] * P - target) / target + (cs[ci] * P > 2 * target ? 1.0 : 0.0);
      if (err < berr - 1e-9) {
        berr = err;
        best = Gemv1Shape{cs[ci], P};
      }
    }
  return best;
}

template <int C, bool SWI, int D>
hipError_t launch_gemv1_cfg(const LinOp& op, int S, int P, hipStream_t st) {
  Gemv1Map m{};
  m.S = S;
  m.P = P;
  int total = 0;
  for (int s = 0; s < op.nseg; ++s) {
    total += (op.seg[s].w.N + P * C - 1) / (P * C);
    m.end[s] = total;
  }
  constexpr int V = pad_pow2((SWI ? 2 : 1) * C);
  const size_t lds = (size_t)(op.K / kGroup) * 68 + (size_t)S * P * V * 4;
  if (lds > lds_limit()) return hipErrorInvalidValue;
  hipLaunchKernelGGL((q4_gemv1_kernel<C, SWI, D>), dim3(total), dim3(S * P * kWave), lds, st, op, m);
  return hipGetLastError();
}

template <bool SWI>
hipError_t launch_gemv1(const LinOp& op, hipStream_t st) {
  const int G = op.K / kGroup;
  const int S = (G + 63) / 64;
  long rows = 0;
  for (int s = 0; s < op.nseg; ++s) rows += op.seg[s].w.N;
  const Gemv1Shape sh = gemv1_shape(rows, S);
  switch (sh.C) {
    case 8: return launch_gemv1_cfg<8, SWI, 4>(op, S, sh.P, st);
    case 7: return launch_gemv1_cfg<7, SWI, 4>(op, S, sh.P, st);
    case 4: return launch_gemv1_cfg<4, SWI, 3>(op, S, sh.P, st);
    default: return launch_gemv1_cfg<2, SWI, 3>(op, S, sh.P, st);
  }
}

// One-token launches need 32-bit buffer offsets and at most 16 slices.
bool gemv1_supported(const LinOp& op) {
  if (op.M != 1 || op.K % kGroup || op.K / kGroup > 16 * 64) return false;
  for (int s = 0; s < op.nseg; ++s) {
    const QView* v[2] = {&op.seg[s].w, &op.seg[s].w2};
    for (int t = 0; t < (op.swiglu ? 2 : 1); ++t)
      if ((size_t)v[t]->N * v[t]->K / 2 + (size_t)v[t]->K >= kOobOff) return false;
  }
  return true;
}

// Read-only streaming probe: every 16-byte chunk of the buffer is loaded once
// with non-temporal buffer loads; a workgroup reads U contiguous 4 KiB runs
// per round (U loads per thread in flight), and the rounds stride over the
// grid.  The XOR of the data is stored only if it equals a fixed value, so
// the loads are kept and the sink is practically never written.
template <int U>
__global__ __launch_bounds__(256) void read_probe_kernel(const void* __restrict__ p, uint32_t n16, unsigned* sink) {
  const __amdgpu_buffer_rsrc_t r = buf_rsrc(p, n16 * 16u);
  unsigned acc = 0;
  const uint32_t step = gridDim.x * 256u * U;
  for (uint32_t i = blockIdx.x * 256u * U + threadIdx.x; i < n16; i += step) {
    u32x4_g v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = __builtin_bit_cast(u32x4_g, __builtin_amdgcn_raw_buffer_load_b128(r, (i + u * 256u) * 16u, 0, kNtBits));
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (acc == 0x9E3779B9u) *sink = acc;
}

}  // namespace

hipError_t launch_read_probe(const void* p, size_t bytes, unsigned* sink, hipStream_t st) {
  // chunks past the buffer read zeros (buffer bounds), so rounds need no tail
  if (!p || !sink || bytes % 16 || (uintptr_t)p % 16 || bytes >= kOobOff) return hipErrorInvalidValue;
  int cus = 256, dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                               hipSuccess || cus < 1)
    cus = 256;
  constexpr int U = 4;
  const size_t n16 = bytes / 16;
  const size_t need = (n16 + 256 * U - 1) / (256 * U);
  const int grid = (int)std::max<size_t>(1, std::min<size_t>((size_t)cus * 8, need));
  hipLaunchKernelGGL((read_probe_kernel<U>), dim3(grid), dim3(256), 0, st, p, (uint32_t)n16, sink);
  return hipGetLastError();
}

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
  if (gemv1_supported(op)) return op.swiglu ? launch_gemv1<true>(op, st) : launch_gemv1<false>(op, st);
  const int spw = default_spw(op);
  return op.swiglu ? launch_sw<true>(op, spw, st) : launch_sw<false>(op, spw, st);
}

}  // namespace atsi
