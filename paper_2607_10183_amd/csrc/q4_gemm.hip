// Prefill-path dequantising GEMM for block-int4 weights on CDNA4 (gfx950).
//
// Prefill runs a whole chunk of tokens through each linear (Sec. 2.2, chunked
// prefill in Sec. 5.1), a dense contraction, so it runs on the matrix cores
// (tile main loop in q4_gemm_core.h).  One launch covers up to three tensors
// sharing an input and fuses RMS normalisation of the input, the SwiGLU
// product, the residual add and the grouped-query head expansion of a
// context-length-1 attention into the epilogue.  Workgroup ids are remapped so
// that the M tiles sharing one weight tile run on the same XCD and reuse it
// from that XCD's L2.
#include <algorithm>

#include "q4_gemm_core.h"

namespace atsi {
namespace {

struct TileMap {
  int end[kMaxSeg];  // cumulative tile counts per segment
  int tiles_m;
  int total;
};

template <int BM, int BN, int WM, int WN, bool SWI, bool NORM>
__global__ __launch_bounds__(kGemmBlock, 2) void q4_gemm_kernel(LinOp op, TileMap tm_) {
  using Core = GemmCore<BM, BN, WM, WN, SWI, NORM>;
  __shared__ __attribute__((aligned(16))) typename Core::Smem sm;

  // XCD-aware order: consecutive ids go to different XCDs (8-way round
  // robin); give each XCD a contiguous run of tiles, M fastest.
  int bid = blockIdx.x;
  if ((tm_.total & 7) == 0) bid = (bid & 7) * (tm_.total >> 3) + (bid >> 3);
  int s = 0;
  while (s < op.nseg - 1 && bid >= tm_.end[s]) ++s;
  const int local = bid - (s ? tm_.end[s - 1] : 0);
  const int tmi = local % tm_.tiles_m, tni = local / tm_.tiles_m;
  const Seg& sg = op.seg[s];
  const int m0 = tmi * BM, n0 = tni * Core::NOUT;
  const int M = op.M, K = op.K;

  const __half* arow[Core::XV];
#pragma unroll
  for (int i = 0; i < Core::XV; ++i) {
    const int m = m0 + Core::xrow(i);
    arow[i] = m < M ? op.x + (size_t)m * K : nullptr;
  }
  g_float16_t acc[Core::FM][Core::FN];
  Core::run(sm, arow, op.x, sg.w, sg.w2, n0, K, op.eps, acc);

#pragma unroll
  for (int i = 0; i < Core::FM; ++i)
#pragma unroll
    for (int j = 0; j < Core::FN; ++j) {
      if (SWI && (j & 1)) continue;
      const int n = n0 + Core::frag_col(j);
      if (n >= sg.w.N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int ml = Core::frag_row(i, v);
        const int m = m0 + ml;
        if (m >= M) continue;
        const float sc = NORM ? sm.rowinv[ml] : 1.f;
        float o = acc[i][j][v] * sc;
        if constexpr (SWI) o = silu_f(o) * (acc[i][j + 1][v] * sc);
        if (sg.expand > 1) {
          const int hd = op.head_dim, jh = n / hd, d = n % hd;
          const __half h = __float2half_rn(o);
          for (int g = 0; g < sg.expand; ++g) sg.y[(size_t)m * sg.ldy + (size_t)(jh * sg.expand + g) * hd + d] = h;
        } else {
          const size_t at = (size_t)m * sg.ldy + n;
          if (op.res && s == 0) o += __half2float(op.res[at]);
          if (op.y32 && s == 0)
            op.y32[at] = o;
          else
            sg.y[at] = __float2half_rn(o);
        }
      }
    }
}

template <int BM, int BN, int WM, int WN, bool SWI, bool NORM>
hipError_t launch_tile_n(const LinOp& op, hipStream_t st) {
  constexpr int NOUT = GemmCore<BM, BN, WM, WN, SWI>::NOUT;
  TileMap tm{};
  tm.tiles_m = (op.M + BM - 1) / BM;
  int total = 0;
  for (int s = 0; s < op.nseg; ++s) {
    total += tm.tiles_m * ((op.seg[s].w.N + NOUT - 1) / NOUT);
    tm.end[s] = total;
  }
  tm.total = total;
  hipLaunchKernelGGL((q4_gemm_kernel<BM, BN, WM, WN, SWI, NORM>), dim3(total), dim3(kGemmBlock), 0, st, op, tm);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, bool SWI>
hipError_t launch_tile(const LinOp& op, hipStream_t st) {
  return op.norm ? launch_tile_n<BM, BN, WM, WN, SWI, true>(op, st) : launch_tile_n<BM, BN, WM, WN, SWI, false>(op, st);
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
