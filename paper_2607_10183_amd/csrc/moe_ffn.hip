// Grouped SwiGLU expert FFN and the weighted combine.
//
// Routed pairs are bucketed by expert (moe_route.hip), so each expert sees a
// contiguous run of rows; its tokens are gathered row by row straight from
// the token matrix.  Work is a list of row tiles (expert, first row), ordered
// heavy-first: the expert with the most tokens starts first, so the Zipf head
// does not finish last.  Only experts some token selected are ever read.
//   gate/up : h[i] = silu(x[t] Wg_e) * (x[t] Wu_e) for bucket row i of pair
//             (t, j), on the MFMA tile (prefill) or a GEMV (decode; with
//             every expert resident the row is the pair id itself);
//   down    : out[k*t + j] = h[i] Wd_e, stored by pair id (fp16);
//   combine : y[t] = sum_j p[t][j] * out[k*t + j] in fp32, slot order, one
//             rounding to fp16 -- no atomics, so results are deterministic.
// A launch reads expert weights either from the device table (HBM-resident
// experts) or, for a batch of experts streamed into temporary buffers, from
// its own arguments.
#include "moe.h"
#include "q4_gemm_core.h"
#include "q4_gemv_core.h"

namespace atsi {
namespace {

__device__ __forceinline__ bool fetch_tile(const MoeArgs& a, int tix, int& e, int& row0, ExpertW& w) {
  if (a.nb > 0) {
    if (tix >= a.nb) return false;
    const int2 t = a.btiles[tix];
    e = a.bexp[t.x];
    row0 = t.y;
    w = a.bw[t.x];
    return true;
  }
  if (tix >= *a.n_tiles) return false;
  e = a.tiles[2 * tix];
  row0 = a.tiles[2 * tix + 1];
  w = a.table[e];
  return true;
}

// GEMV tile: the h row i and pair id pr it computes, and the expert's weights.
// Pair-indexed launches read one table entry per tile; bucketed ones follow
// the tile list, the bucket offsets and the permutation.
__device__ __forceinline__ bool fetch_row(const MoeArgs& a, int tix, int& i, int& pr, ExpertW& w) {
  if (a.pair_expert) {
    if (tix >= a.n_pairs) return false;
    const int e = a.pair_expert[tix];
    if ((unsigned)e >= (unsigned)a.n_experts) return false;
    w = a.table[e];
    i = pr = tix;
    return true;
  }
  int e, row0;
  if (!fetch_tile(a, tix, e, row0, w)) return false;
  i = a.offsets[e] + row0;
  pr = a.perm[i];
  return true;
}

constexpr int EBM = 64;   // rows per expert tile on the MFMA path
constexpr int EBN = 128;

// ---------------------------------------------------------------- MFMA path

__global__ __launch_bounds__(kGemmBlock, 2) void expert_gateup_gemm(MoeArgs a, int tile_bound) {
  using Core = GemmCore<EBM, EBN, 2, 2, true>;
  __shared__ __attribute__((aligned(16))) Core::Smem sm;
  const int tix = blockIdx.x % tile_bound, tn = blockIdx.x / tile_bound;
  int e, row0;
  ExpertW w;
  if (!fetch_tile(a, tix, e, row0, w)) return;
  const int cnt = a.counts[e], base = a.offsets[e] + row0;
  const int rows = min(EBM, cnt - row0);
  const int n0 = tn * Core::NOUT;
  const __half* arow[Core::XV];
#pragma unroll
  for (int i = 0; i < Core::XV; ++i) {
    const int r = Core::xrow(i);
    arow[i] = r < rows ? a.x + (size_t)(a.perm[base + r] / a.k) * a.H : nullptr;
  }
  g_float16_t acc[Core::FM][Core::FN];
  Core::run(sm, arow, a.x, w.gate, w.up, n0, a.H, 0.f, acc);
#pragma unroll
  for (int i = 0; i < Core::FM; ++i)
#pragma unroll
    for (int j = 0; j < Core::FN; j += 2) {
      const int n = n0 + Core::frag_col(j);
      if (n >= a.I) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = Core::frag_row(i, v);
        if (r < rows) {
          // RMS-normalised input: scale both products by the token's factor
          const float sc = a.inv_r ? a.inv_r[a.perm[base + r] / a.k] : 1.f;
          a.h[(size_t)(base + r) * a.I + n] = __float2half_rn(silu_f(acc[i][j][v] * sc) * (acc[i][j + 1][v] * sc));
        }
      }
    }
}

__global__ __launch_bounds__(kGemmBlock, 2) void expert_down_gemm(MoeArgs a, int tile_bound) {
  using Core = GemmCore<EBM, EBN, 2, 2, false>;
  __shared__ __attribute__((aligned(16))) Core::Smem sm;
  const int tix = blockIdx.x % tile_bound, tn = blockIdx.x / tile_bound;
  int e, row0;
  ExpertW w;
  if (!fetch_tile(a, tix, e, row0, w)) return;
  const int cnt = a.counts[e], base = a.offsets[e] + row0;
  const int rows = min(EBM, cnt - row0);
  const int n0 = tn * Core::NOUT;
  const __half* arow[Core::XV];
#pragma unroll
  for (int i = 0; i < Core::XV; ++i) {
    const int r = Core::xrow(i);
    arow[i] = r < rows ? a.h + (size_t)(base + r) * a.I : nullptr;
  }
  g_float16_t acc[Core::FM][Core::FN];
  Core::run(sm, arow, a.h, w.down, w.down, n0, a.I, 0.f, acc);
#pragma unroll
  for (int i = 0; i < Core::FM; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = Core::frag_row(i, v);
      if (r >= rows) continue;
      const size_t prow = (size_t)a.perm[base + r] * a.H;
#pragma unroll
      for (int j = 0; j < Core::FN; ++j) {
        const int n = n0 + Core::frag_col(j);
        if (n < a.H) a.out[prow + n] = __float2half_rn(acc[i][j][v]);
      }
    }
}

// ---------------------------------------------------------------- GEMV path (one row per tile)

// Sums over the wave of RW rows n0 .. n0 + RW - 1 of w1 (and of w2 when TWO)
// against one K-wide input row xr: lane l takes groups l, l + 64, ...; rows
// past N repeat the last row and are discarded by the caller.
template <int RW, bool TWO>
__device__ __forceinline__ void expert_rows(const QView& w1, const QView& w2, const __half* xr, int n0, int N, int K,
                                            int lane, float (&g)[RW], float (&u)[RW]) {
  using namespace gemv;
  constexpr int CH = 2;
  constexpr int R2 = TWO ? RW : 1;
  const int nchunk = K / kGroup;
  const size_t rbytes = (size_t)K / 2;
  float acc[RW], acc2[R2], sq = 0.f;
#pragma unroll
  for (int r = 0; r < RW; ++r) acc[r] = 0.f;
#pragma unroll
  for (int r = 0; r < R2; ++r) acc2[r] = 0.f;
  for (int c0 = lane; c0 < nchunk; c0 += kWave * CH) {
    uint4 cw[CH][RW], cw2[CH][R2];
    uint16_t sc[CH][RW], sc2[CH][R2];
    XRaw xv[CH];
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      const int c = c0 + h * kWave;
      if (c >= nchunk) continue;
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        const int row = min(n0 + r, N - 1);
        cw[h][r] = ldg16(w1.codes + (size_t)row * rbytes + (size_t)c * 16);
        sc[h][r] = ldg2(w1.scales + (size_t)row * nchunk + c);
        if constexpr (TWO) {
          cw2[h][r] = ldg16(w2.codes + (size_t)row * rbytes + (size_t)c * 16);
          sc2[h][r] = ldg2(w2.scales + (size_t)row * nchunk + c);
        }
      }
      load_xraw(xv[h], xr, c);
    }
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      if (c0 + h * kWave >= nchunk) break;
      XGroup gx;
      prep_x(gx, xv[h], false, sq);
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        acc[r] = fmaf(__half2float(__ushort_as_half(sc[h][r])), group_dot(cw[h][r], gx), acc[r]);
        if constexpr (TWO) acc2[r] = fmaf(__half2float(__ushort_as_half(sc2[h][r])), group_dot(cw2[h][r], gx), acc2[r]);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    g[r] = wave_total(acc[r]);
    u[r] = TWO ? wave_total(acc2[R2 > 1 ? r : 0]) : 0.f;
  }
}

template <int RW, bool DOWN>
__global__ __launch_bounds__(gemv::kBlock) void expert_gemv(MoeArgs a, int tile_bound) {
  using namespace gemv;
  const int tix = blockIdx.x % tile_bound, nb = blockIdx.x / tile_bound;
  int i, pr;
  ExpertW w;
  if (!fetch_row(a, tix, i, pr, w)) return;
  const int K = DOWN ? a.I : a.H, N = DOWN ? a.H : a.I;
  const __half* xr = DOWN ? a.h + (size_t)i * a.I : a.x + (size_t)(pr / a.k) * a.H;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int n0 = (nb * (kBlock / kWave) + wave) * RW;
  if (n0 >= N) return;
  float g[RW], u[RW];
  expert_rows<RW, !DOWN>(DOWN ? w.down : w.gate, w.up, xr, n0, N, K, lane, g, u);
  const float sc = (!DOWN && a.inv_r) ? a.inv_r[pr / a.k] : 1.f;  // RMS-normalised input
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const int n = n0 + r;
    if (lane == r && n < N) {
      if (DOWN)
        a.out[(size_t)pr * a.H + n] = __float2half_rn(g[r] * sc);
      else
        a.h[(size_t)i * a.I + n] = __float2half_rn(silu_f(g[r] * sc) * (u[r] * sc));
    }
  }
}

// Down projection and combine in one launch (decode, every expert resident,
// pair-indexed h): a workgroup owns kDcRows output rows of one token and
// computes them for all k routed experts of that token (wave task = expert j,
// RW rows), rounds each expert output to fp16 as the separate down launch
// stores it, and sums p_j * out_j in slot order in fp32 plus the residual, as
// the combine does.  y may alias res: each element is read, then written, by
// one thread.
constexpr int kDcRows = 8;
constexpr int kDcRW = 4;  // rows per wave task
constexpr int kDcThreads = 1024;

template <int RW>
__global__ __launch_bounds__(kDcThreads) void expert_down_combine(MoeArgs a, const float* __restrict__ p,
                                                                  const __half* res, __half* y) {
  using namespace gemv;
  static_assert(kDcRows % RW == 0, "whole wave tasks per row block");
  constexpr int SUB = kDcRows / RW;
  __shared__ float outs[kMaxTopK][kDcRows];
  const int t = blockIdx.y, nb = blockIdx.x * kDcRows;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  for (int task = wave; task < a.k * SUB; task += kDcThreads / kWave) {
    const int j = task / SUB, n0 = nb + (task % SUB) * RW;
    const int pr = t * a.k + j;
    const int e = a.pair_expert[pr];
    float g[RW], u[RW];
    if ((unsigned)e < (unsigned)a.n_experts) {
      expert_rows<RW, false>(a.table[e].down, a.table[e].down, a.h + (size_t)pr * a.I, n0, a.H, a.I, lane, g, u);
    } else {
#pragma unroll
      for (int r = 0; r < RW; ++r) g[r] = 0.f;
    }
    if (lane == 0) {
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        const __half o = __float2half_rn(g[r]);
        outs[j][(task % SUB) * RW + r] = __half2float(o);
        if (a.store_out && n0 + r < a.H) a.out[(size_t)pr * a.H + n0 + r] = o;
      }
    }
  }
  __syncthreads();
  const int n = nb + (int)threadIdx.x;
  if (threadIdx.x < kDcRows && n < a.H) {
    float acc = 0.f;
    for (int j = 0; j < a.k; ++j) acc = fmaf(p[(size_t)t * a.k + j], outs[j][threadIdx.x], acc);
    if (res) acc += __half2float(res[(size_t)t * a.H + n]);
    y[(size_t)t * a.H + n] = __float2half_rn(acc);
  }
}

constexpr int kGemvRW = 2;

// ---------------------------------------------------------------- combine, table patch

__global__ void combine_kernel(const __half* __restrict__ out, const float* __restrict__ p, int M, int k, int H,
                               const __half* res, __half* y) {
  const int c8 = H / 8;
  const size_t total = (size_t)M * c8;
  for (size_t q = (size_t)blockIdx.x * blockDim.x + threadIdx.x; q < total; q += (size_t)gridDim.x * blockDim.x) {
    const int t = (int)(q / c8), c = (int)(q % c8);
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 < k; j0 += 8) {  // loads of 8 slots first, then the fixed-order sum
      float pj[8];
      uint4 v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j0 + j < k) {
          pj[j] = p[(size_t)t * k + j0 + j];
          v[j] = *reinterpret_cast<const uint4*>(out + ((size_t)t * k + j0 + j) * H + (size_t)c * 8);
        }
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j0 + j < k) {
          const __half* hv = reinterpret_cast<const __half*>(&v[j]);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[i] = fmaf(pj[j], __half2float(hv[i]), acc[i]);
        }
    }
    if (res) {  // y = res + sum (y may alias res: each element is read, then written, by one thread)
      const uint4 rv = *reinterpret_cast<const uint4*>(res + (size_t)t * H + (size_t)c * 8);
      const __half* hr = reinterpret_cast<const __half*>(&rv);
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] += __half2float(hr[i]);
    }
    uint4 o;
    __half* ho = reinterpret_cast<__half*>(&o);
#pragma unroll
    for (int i = 0; i < 8; ++i) ho[i] = __float2half_rn(acc[i]);
    *reinterpret_cast<uint4*>(y + (size_t)t * H + (size_t)c * 8) = o;
  }
}

__global__ void gather_rows_kernel(const uint4* __restrict__ src, const int32_t* __restrict__ perm, int rows, int c16,
                                   uint4* __restrict__ dst) {
  const size_t total = (size_t)rows * c16;
  for (size_t q = (size_t)blockIdx.x * blockDim.x + threadIdx.x; q < total; q += (size_t)gridDim.x * blockDim.x) {
    const int i = (int)(q / c16), c = (int)(q % c16);
    const int to = perm ? perm[i] : i;
    if ((unsigned)to < (unsigned)rows) dst[(size_t)to * c16 + c] = src[q];
  }
}

struct TablePatch {
  int e0, n;
  ExpertW w[16];
  uint8_t r[16];
};

__global__ void table_patch_kernel(ExpertW* table, uint8_t* resident, TablePatch tp) {
  const int i = threadIdx.x;
  if (i < tp.n) {
    table[tp.e0 + i] = tp.w[i];
    resident[tp.e0 + i] = tp.r[i];
  }
}

}  // namespace

int expert_tile_rows(bool gemv) { return gemv ? 1 : EBM; }

hipError_t launch_expert_gateup(const MoeArgs& a, int tile_bound, bool gemv, hipStream_t s) {
  if (tile_bound <= 0) return hipSuccess;
  if (gemv) {
    const int nblk = (a.I + 4 * kGemvRW - 1) / (4 * kGemvRW);
    hipLaunchKernelGGL((expert_gemv<kGemvRW, false>), dim3(tile_bound * nblk), dim3(gemv::kBlock), 0, s, a,
                       tile_bound);
  } else {
    const int tn = (a.I + EBN / 2 - 1) / (EBN / 2);
    hipLaunchKernelGGL(expert_gateup_gemm, dim3(tile_bound * tn), dim3(kGemmBlock), 0, s, a, tile_bound);
  }
  return hipGetLastError();
}

hipError_t launch_expert_down(const MoeArgs& a, int tile_bound, bool gemv, hipStream_t s) {
  if (tile_bound <= 0) return hipSuccess;
  if (gemv) {
    const int nblk = (a.H + 4 * kGemvRW - 1) / (4 * kGemvRW);
    hipLaunchKernelGGL((expert_gemv<kGemvRW, true>), dim3(tile_bound * nblk), dim3(gemv::kBlock), 0, s, a,
                       tile_bound);
  } else {
    const int tn = (a.H + EBN - 1) / EBN;
    hipLaunchKernelGGL(expert_down_gemm, dim3(tile_bound * tn), dim3(kGemmBlock), 0, s, a, tile_bound);
  }
  return hipGetLastError();
}

hipError_t launch_expert_down_combine(const MoeArgs& a, int M, const float* p, const __half* res, __half* y,
                                      hipStream_t s) {
  if (!a.pair_expert || M < 1 || a.k > kMaxTopK) return hipErrorInvalidValue;
  hipLaunchKernelGGL((expert_down_combine<kDcRW>), dim3((a.H + kDcRows - 1) / kDcRows, M), dim3(kDcThreads), 0, s, a,
                     p, res, y);
  return hipGetLastError();
}

hipError_t launch_combine(const __half* out, const float* p, int M, int k, int H, const __half* res, __half* y,
                          hipStream_t s) {
  const size_t total = (size_t)M * (H / 8);
  const int blocks = (int)std::min<size_t>((total + 255) / 256, 2048);
  hipLaunchKernelGGL(combine_kernel, dim3(blocks), dim3(256), 0, s, out, p, M, k, H, res, y);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const __half* src, const int32_t* perm, int rows, int cols, __half* dst, hipStream_t s) {
  if (rows < 1 || cols % 8) return hipErrorInvalidValue;
  const size_t total = (size_t)rows * (cols / 8);
  const int blocks = (int)std::min<size_t>((total + 255) / 256, 4096);
  hipLaunchKernelGGL(gather_rows_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<const uint4*>(src), perm, rows,
                     cols / 8, reinterpret_cast<uint4*>(dst));
  return hipGetLastError();
}

hipError_t launch_table_patch(ExpertW* table, uint8_t* resident, int e0, int n, const ExpertW* w, const uint8_t* r,
                              hipStream_t s) {
  TablePatch tp{};
  tp.e0 = e0;
  tp.n = n;
  for (int i = 0; i < n; ++i) {
    tp.w[i] = w[i];
    tp.r[i] = r[i];
  }
  hipLaunchKernelGGL(table_patch_kernel, dim3(1), dim3(64), 0, s, table, resident, tp);
  return hipGetLastError();
}

}  // namespace atsi
