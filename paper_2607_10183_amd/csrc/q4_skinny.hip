// Batched-decode dequantising GEMM for block-int4 weights on CDNA4 (gfx950):
// y[m][n] = sum_g s[n][g] * sum_{k in g} q[n][k] * x[m][k] for 2..16 tokens.
//
// Decode over a small batch still reads every weight byte once per step
// (Sec. 2.2), but per weight it now needs one product per token.  The
// dot2-based GEMV spends about four ALU ops per eight weights per token, which
// outruns the HBM time from about four tokens on; here the products go to the
// matrix cores instead and the ALU work per weight no longer depends on the
// batch:
//   * one v_mfma_f32_16x16x32_f16 covers 16 weight rows x one 32-input group
//     x up to 16 tokens: the A operand holds the tokens' activations, the B
//     operand the group's codes, so every MFMA sums exactly one group;
//   * each lane turns one 32-bit code word (8 nibbles) into eight exact fp16
//     integers q = u - 8 with two mask-and-or ops per pair of inputs and one
//     packed fp16 add (or fma, for the nibbles shifted by four) per pair; the
//     products q * x are exact and the MFMA sums them in fp32, and the group's
//     fp16 scale multiplies the group sum in fp32, as the GEMV does;
//   * the (k, k+4) pair order that nibble extraction yields is matched by
//     permuting the activations of each lane's 8 inputs the same way;
//   * a workgroup owns 16 weight rows; its waves split K into contiguous
//     stretches, each wave keeping D - 1 steps of four groups in flight, and
//     their partial sums meet in LDS;
//   * the MFMA operand layout puts four different rows (or tokens) in every
//     four consecutive lanes, which defeats load coalescing (each lane's
//     access becomes a cache access of its own), so the loads use a layout
//     where four consecutive lanes read one contiguous run and each wave
//     restages the data through its own slice of LDS;
//   * all loads are buffer loads whose out-of-range lanes read zeros: rows
//     past N, tokens past M and steps past K need no clamping or branches;
//   * a fused RMS norm takes the per-token sum of squares from one more MFMA
//     per group (the activations times themselves; the diagonal of the
//     product is what is kept).
// The epilogue is the GEMV's: SwiGLU product, residual, fp32 output, KV-head
// expansion, over up to three tensors sharing the input.
#include "q4_mfma_unpack.h"

namespace atsi {
namespace {

using namespace gemv;

typedef half8_t h8_t;
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef u32x4_t u4_t;

constexpr int kRows = 16;  // weight rows per workgroup: the MFMA's N
constexpr uint32_t kOob = 0x80000000u;  // an offset past every buffer here

struct SkinnyMap {
  int end[kMaxSeg];  // cumulative workgroup counts per segment
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

// One step is four consecutive groups (128 inputs) of the wave's 16 rows.
// Global loads are laid out for coalescing, four consecutive lanes reading
// one contiguous run, and each wave restages them through its own LDS into
// the MFMA lanes' layout (lane n + 16 c takes row n, 8-input chunk c):
//   codes   lane l: row l/4, group l%4 of the step, 16 bytes;
//   scales  lane l: row l/4, group l%4, 2 bytes;
//   x       lane l of load i: token l/16 + 4 i, 16 bytes (chunk l%16) of the
//           step's 128 inputs, permuted to the codes' pair order on the way.
constexpr int kCStride = 80;   // LDS bytes per row of staged codes (64 + pad)
constexpr int kXStride = 272;  // LDS bytes per token of staged x (256 + pad)

template <bool SWI, int MX>
struct StepLd {
  u4_t c[SWI ? 2 : 1];      // 16 code bytes (gate and up for SwiGLU)
  uint32_t s[SWI ? 2 : 1];  // one scale in the low half
  u4_t x[MX];               // 8 activations of a token
};

template <bool SWI, int MX>
struct WaveLds {
  static constexpr int NT = SWI ? 2 : 1;
  static constexpr int XR = 4 * MX + 1;  // staged tokens and a zero row
  __attribute__((aligned(16))) uint8_t codes[NT][16 * kCStride];
  __attribute__((aligned(16))) uint8_t x[XR * kXStride];
  __attribute__((aligned(16))) uint16_t sc[NT][16 * 4];
};

template <int NW, int D, int MX, bool SWI, bool NORM>
__global__ __launch_bounds__(NW * 64) void q4_skinny_kernel(LinOp op, SkinnyMap bm) {
  constexpr int NT = SWI ? 2 : 1;
  __shared__ WaveLds<SWI, MX> wl[NW];
  __shared__ f4_t red[NT][NW][64];
  __shared__ float sq[NW][16];
  __shared__ float inv_r[16];
  int s = 0;
  while (s < op.nseg - 1 && (int)blockIdx.x >= bm.end[s]) ++s;
  const int local = (int)blockIdx.x - (s ? bm.end[s - 1] : 0);
  const Seg& sg = op.seg[s];
  const int K = op.K, G = K / kGroup, M = op.M, N = sg.w.N;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: step offsets stay scalar
  const int j = lane & 15, kb = lane >> 4;  // MFMA roles: B column (row) / A row (token); 8-input chunk
  const int row0 = local * kRows;
  WaveLds<SWI, MX>& L = wl[wave];

  __amdgpu_buffer_rsrc_t rc[NT], rs[NT];
  rc[0] = rsrc(sg.w.codes, (uint32_t)((size_t)N * K / 2));
  rs[0] = rsrc(sg.w.scales, (uint32_t)((size_t)N * G * 2));
  if constexpr (SWI) {
    rc[1] = rsrc(sg.w2.codes, (uint32_t)((size_t)N * K / 2));
    rs[1] = rsrc(sg.w2.scales, (uint32_t)((size_t)N * G * 2));
  }
  const __amdgpu_buffer_rsrc_t rx = rsrc(op.x, (uint32_t)((size_t)M * K * 2));
  // load roles: codes/scales row lr, group lg of the step; x token xm + 4 i, chunk xc
  const int lr = lane >> 2, lg = lane & 3, xm = lane >> 4, xc = lane & 15;
  const uint32_t oc = (uint32_t)(row0 + lr) * (uint32_t)(K / 2) + (uint32_t)lg * 16;  // + 64 per step
  const uint32_t os = ((uint32_t)(row0 + lr) * (uint32_t)G + (uint32_t)lg) * 2;     // + 8 per step
  const uint32_t ox = ((uint32_t)xm * (uint32_t)K + (uint32_t)xc * 8) * 2;           // + 256 per step

  // wave w owns steps [s0, s1) of ceil(G / 4): a contiguous stretch of its
  // rows, so the waves of a workgroup read different parts of them at once
  const int nstep = G / 4;  // K % 128 == 0
  const int spw = (nstep + NW - 1) / NW;
  const int s0 = wave * spw, s1 = min(s0 + spw, nstep);
  auto load = [&](StepLd<SWI, MX>& b, int st) {
    const bool ok = st < s1;  // uniform; past the stretch every load reads zeros
    const uint32_t dc = ok ? (uint32_t)st * 64 : kOob, ds = ok ? (uint32_t)st * 8 : kOob,
                   dx = ok ? (uint32_t)st * 256 : kOob;
#pragma unroll
    for (int t = 0; t < NT; ++t) b.c[t] = __builtin_amdgcn_raw_buffer_load_b128(rc[t], oc + dc, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) b.s[t] = __builtin_amdgcn_raw_buffer_load_b16(rs[t], os + ds, 0, 0);
#pragma unroll
    for (int i = 0; i < MX; ++i)
      b.x[i] = __builtin_amdgcn_raw_buffer_load_b128(rx, ox + (uint32_t)i * 4 * K * 2 + dx, 0, 0);
  };
  // staging writes: codes at [row][group] 16 B, scales [row][group], x [token][128 inputs]
  auto stage = [&](const StepLd<SWI, MX>& b) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      *reinterpret_cast<u4_t*>(&L.codes[t][lr * kCStride + lg * 16]) = b.c[t];
      L.sc[t][lr * 4 + lg] = (uint16_t)b.s[t];
    }
#pragma unroll
    for (int i = 0; i < MX; ++i) {
      *reinterpret_cast<h8_t*>(&L.x[(xm + 4 * i) * kXStride + xc * 16]) = perm_x(b.x[i]);
    }
  };
  // the zero row: A rows past the staged tokens read it
  if (lane < kXStride / 16)
    *reinterpret_cast<u4_t*>(&L.x[4 * MX * kXStride + lane * 16]) = u4_t{0u, 0u, 0u, 0u};
  const int arow = j < 4 * MX ? j : 4 * MX;
  const uint8_t* xa = &L.x[arow * kXStride + kb * 16];   // + 64 per group
  const UnpackMasks uk = unpack_masks();

  const f4_t zero = {0.f, 0.f, 0.f, 0.f};
  f4_t acc[NT], gram = zero;
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = zero;
  // compute one staged step: four MFMAs per tensor, each one group
  // (all LDS reads of the step go out before the first MFMA needs one)
  auto compute = [&]() {
    uint2 sv[NT];
    u4_t xa4[4];
    uint32_t w4[NT][4];
#pragma unroll
    for (int g = 0; g < 4; ++g) xa4[g] = *reinterpret_cast<const u4_t*>(xa + g * 64);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int g = 0; g < 4; ++g)
        w4[t][g] = *reinterpret_cast<const uint32_t*>(&L.codes[t][j * kCStride + g * 16 + kb * 4]);
      sv[t] = *reinterpret_cast<const uint2*>(&L.sc[t][j * 4]);
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const h8_t a = __builtin_bit_cast(h8_t, xa4[g]);
      if constexpr (NORM) gram = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, a, gram, 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const f4_t p = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, unpack_q(w4[t][g], uk), zero, 0, 0, 0);
        const uint32_t pair = g < 2 ? sv[t].x : sv[t].y;
        const float sc = __half2float(__ushort_as_half((uint16_t)((g & 1) ? pair >> 16 : pair)));
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[t][v] = fmaf(sc, p[v], acc[t][v]);
      }
    }
  };

  // Software pipeline over steps, one region per step with nothing moved
  // across regions: stage step st from its registers into LDS, refill those
  // registers with step st + D, compute step st.  Loads keep one order, so
  // each region waits for its own step only and D - 1 steps stay in flight.
  StepLd<SWI, MX> buf[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    load(buf[d], s0 + d);
    __builtin_amdgcn_sched_barrier(0);
  }
  const int nit = (spw + D - 1) / D;
  for (int it = 0; it < nit; ++it) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      stage(buf[d]);
      load(buf[d], s0 + (it + 1) * D + d);
      compute();
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // partial sums of the waves meet in LDS; D[m][n] sits in lane n + 16 (m / 4), item m % 4
#pragma unroll
  for (int t = 0; t < NT; ++t) red[t][wave][lane] = acc[t];
  if constexpr (NORM) {
    if (kb == (j >> 2)) sq[wave][j] = gram[j & 3];  // the diagonal: token j's sum of squares
  }
  __syncthreads();
  if constexpr (NORM) {
    if (threadIdx.x < 16) {
      float tot = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) tot += sq[w][threadIdx.x];
      inv_r[threadIdx.x] = 1.f / sqrtf(tot / (float)K + op.eps);
    }
    __syncthreads();
  }
  const int row = row0 + j;
  if (wave != 0 || row >= N) return;
  f4_t v[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    v[t] = red[t][0][lane];
#pragma unroll
    for (int w = 1; w < NW; ++w) v[t] += red[t][w][lane];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = 4 * kb + i;
    if (m >= M) break;
    const float r = NORM ? inv_r[m] : 1.f;
    float o = v[0][i] * r;
    if constexpr (SWI) o = silu_f(o) * (v[NT - 1][i] * r);
    emit_out(op, sg, s, m, row, o);
  }
}

template <int NW, int D, int MX, bool SWI, bool NORM>
hipError_t launch_cfg(const LinOp& op, hipStream_t st) {
  SkinnyMap bm{};
  int total = 0;
  for (int s = 0; s < op.nseg; ++s) {
    total += (op.seg[s].w.N + kRows - 1) / kRows;
    bm.end[s] = total;
  }
  hipLaunchKernelGGL((q4_skinny_kernel<NW, D, MX, SWI, NORM>), dim3(total), dim3(NW * 64), 0, st, op, bm);
  return hipGetLastError();
}

template <int MX, bool SWI>
hipError_t launch_mx(const LinOp& op, hipStream_t st) {
  // eight waves, two steps of loads in flight while a step is computed:
  // the fastest of 4 / 8 waves and 2 / 3 / 4 steps measured on MI355X
  return op.norm ? launch_cfg<8, 2, MX, SWI, true>(op, st) : launch_cfg<8, 2, MX, SWI, false>(op, st);
}

template <bool SWI>
hipError_t launch_sw(const LinOp& op, hipStream_t st) {
  if (op.M <= 4) return launch_mx<1, SWI>(op, st);
  if (op.M <= 8) return launch_mx<2, SWI>(op, st);
  return launch_mx<4, SWI>(op, st);
}

}  // namespace

bool skinny_supported(const LinOp& op) {
  if (op.M < 1 || op.M > kSkinnyMaxTokens || op.K % (4 * kGroup)) return false;
  // 32-bit buffer offsets
  if ((size_t)op.M * op.K * 2 >= kOob) return false;
  for (int s = 0; s < op.nseg; ++s) {
    const QView* v[2] = {&op.seg[s].w, &op.seg[s].w2};
    for (int t = 0; t < (op.swiglu ? 2 : 1); ++t)
      if ((size_t)(v[t]->N + kRows) * v[t]->K / 2 >= kOob) return false;
  }
  return true;
}

hipError_t launch_skinny(const LinOp& op, hipStream_t st) {
  if (!skinny_supported(op)) return hipErrorInvalidValue;
  return op.swiglu ? launch_sw<true>(op, st) : launch_sw<false>(op, st);
}

}  // namespace atsi
