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
//     stretches of groups, each wave keeping D - 1 groups of loads in flight,
//     and their partial sums meet in LDS;
//   * all loads are buffer loads whose out-of-range lanes read zeros: rows
//     past N, tokens past M and groups past K need no clamping or branches;
//   * a fused RMS norm takes the per-token sum of squares from one more MFMA
//     per group (the activations times themselves; the diagonal of the
//     product is what is kept).
// The epilogue is the GEMV's: SwiGLU product, residual, fp32 output, KV-head
// expansion, over up to three tensors sharing the input.
#include "q4_gemv_core.h"

namespace atsi {
namespace {

using namespace gemv;

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef unsigned u4_t __attribute__((ext_vector_type(4)));

constexpr int kRows = 16;  // weight rows per workgroup: the MFMA's N
constexpr uint32_t kOob = 0x80000000u;  // an offset past every buffer here

struct SkinnyMap {
  int end[kMaxSeg];  // cumulative workgroup counts per segment
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

// Masks in scalar registers and the 1024.0 pattern in a vector register, so
// that each mask-and-or is one v_and_or_b32 (its encoding takes no literal
// constant and reads at most one scalar register).
struct UnpackK {
  uint32_t lo, hi, magic;
};

__device__ __forceinline__ uint32_t sgpr_const(uint32_t v) {
  uint32_t r;
  asm volatile("s_mov_b32 %0, %1" : "=s"(r) : "i"(v));
  return r;
}

__device__ __forceinline__ uint32_t vgpr_const(uint32_t v) {
  uint32_t r;
  asm volatile("v_mov_b32 %0, %1" : "=v"(r) : "i"(v));
  return r;
}

__device__ __forceinline__ UnpackK unpack_consts() {
  return UnpackK{sgpr_const(0x000F000Fu), sgpr_const(0x00F000F0u), vgpr_const(kMagic)};
}

// Eight exact fp16 integers q = u - 8 from one code word, in the pair order
// (k0, k4), (k1, k5), (k2, k6), (k3, k7).
__device__ __forceinline__ h8_t unpack_q(uint32_t w, const UnpackK& k) {
  const uint32_t w8 = w >> 8;
  const half2_t off = {(_Float16)-1032.f, (_Float16)-1032.f};
  const half2_t sh = {(_Float16)0.0625f, (_Float16)0.0625f};
  const half2_t off16 = {(_Float16)-72.f, (_Float16)-72.f};
  // (1024 + u) - 1032 and (1024 + 16 u) / 16 - 72 are exact in fp16
  const half2_t a = __builtin_bit_cast(half2_t, (w & k.lo) | k.magic) + off;
  const half2_t b = __builtin_bit_cast(half2_t, (w & k.hi) | k.magic) * sh + off16;
  const half2_t c = __builtin_bit_cast(half2_t, (w8 & k.lo) | k.magic) + off;
  const half2_t d = __builtin_bit_cast(half2_t, (w8 & k.hi) | k.magic) * sh + off16;
  const u4_t r = {__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b), __builtin_bit_cast(uint32_t, c),
                  __builtin_bit_cast(uint32_t, d)};
  return __builtin_bit_cast(h8_t, r);
}

// Eight consecutive fp16 activations reordered to the same pair order.
__device__ __forceinline__ h8_t perm_x(u4_t d) {
  const u4_t r = {__builtin_amdgcn_perm(d.z, d.x, 0x05040100u), __builtin_amdgcn_perm(d.z, d.x, 0x07060302u),
                  __builtin_amdgcn_perm(d.w, d.y, 0x05040100u), __builtin_amdgcn_perm(d.w, d.y, 0x07060302u)};
  return __builtin_bit_cast(h8_t, r);
}

// Loads of one group for one lane.
template <bool SWI>
struct GroupLd {
  uint32_t c[SWI ? 2 : 1];  // code word of its row (gate and up for SwiGLU)
  uint16_t s[SWI ? 2 : 1];  // the row's scale of the group
  u4_t x;                   // its token's 8 activations
};

template <int NW, int D, bool SWI, bool NORM>
__global__ __launch_bounds__(NW * 64) void q4_skinny_kernel(LinOp op, SkinnyMap bm) {
  constexpr int NT = SWI ? 2 : 1;
  __shared__ f4_t red[NT][NW][64];
  __shared__ float sq[NW][16];
  __shared__ float inv_r[16];
  int s = 0;
  while (s < op.nseg - 1 && (int)blockIdx.x >= bm.end[s]) ++s;
  const int local = (int)blockIdx.x - (s ? bm.end[s - 1] : 0);
  const Seg& sg = op.seg[s];
  const int K = op.K, G = K / kGroup, M = op.M, N = sg.w.N;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: group offsets stay scalar
  const int j = lane & 15, kb = lane >> 4;  // B column (weight row) / A row (token); 8-input chunk
  const int row = local * kRows + j;

  __amdgpu_buffer_rsrc_t rc[NT], rs[NT];
  rc[0] = rsrc(sg.w.codes, (uint32_t)((size_t)N * K / 2));
  rs[0] = rsrc(sg.w.scales, (uint32_t)((size_t)N * G * 2));
  if constexpr (SWI) {
    rc[1] = rsrc(sg.w2.codes, (uint32_t)((size_t)N * K / 2));
    rs[1] = rsrc(sg.w2.scales, (uint32_t)((size_t)N * G * 2));
  }
  const __amdgpu_buffer_rsrc_t rx = rsrc(op.x, (uint32_t)((size_t)M * K * 2));
  const uint32_t oc = (uint32_t)row * (uint32_t)(K / 2) + (uint32_t)kb * 4;
  const uint32_t os = (uint32_t)row * (uint32_t)G * 2;
  const uint32_t ox = ((uint32_t)j * (uint32_t)K + (uint32_t)kb * 8) * 2;

  // Wave w owns groups [w * ngw, (w + 1) * ngw): at any moment the waves of a
  // workgroup read different stretches of their rows, so the requests in
  // flight spread over the HBM channels (waves taking interleaved groups all
  // hit the same few bytes of rows 2 KiB apart, and the channels behind
  // those addresses).  Past the wave's last group every offset is out of
  // range: the load reads zeros and moves no data.
  const int ngw = (G + NW - 1) / NW;
  const int g0 = wave * ngw, g1 = min(g0 + ngw, G);
  auto load = [&](GroupLd<SWI>& b, int i) {
    const int g = g0 + i;
    const bool ok = g < g1;
    const uint32_t gc = ok ? (uint32_t)g * 16 : kOob, gs = ok ? (uint32_t)g * 2 : kOob,
                   gx = ok ? (uint32_t)g * 64 : kOob;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      b.c[t] = __builtin_amdgcn_raw_buffer_load_b32(rc[t], oc + gc, 0, 0);
      b.s[t] = __builtin_amdgcn_raw_buffer_load_b16(rs[t], os + gs, 0, 0);
    }
    b.x = __builtin_amdgcn_raw_buffer_load_b128(rx, ox + gx, 0, 0);
  };

  // Software pipeline, one region per group with nothing moved across
  // regions: region i computes group i's MFMA, applies the previous group's
  // scale (its MFMA has finished by then), and refills the buffer it used
  // with group i + D.  Loads keep one order, so each region waits for its own
  // group's loads only and D - 1 groups stay in flight.
  const int nit = (ngw + D - 1) / D;
  const UnpackK uk = unpack_consts();
  GroupLd<SWI> buf[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    load(buf[d], d);
    __builtin_amdgcn_sched_barrier(0);
  }

  const f4_t zero = {0.f, 0.f, 0.f, 0.f};
  f4_t acc[NT], prev[NT], gram = zero;
  float prev_s[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    acc[t] = zero;
    prev[t] = zero;
    prev_s[t] = 0.f;
  }
  for (int it = 0; it < nit; ++it) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      GroupLd<SWI>& b = buf[d];
      const h8_t a = perm_x(b.x);
      if constexpr (NORM) gram = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, a, gram, 0, 0, 0);
      f4_t p[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) p[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, unpack_q(b.c[t], uk), zero, 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[t][v] = fmaf(prev_s[t], prev[t][v], acc[t][v]);
        prev[t] = p[t];
        prev_s[t] = __half2float(__ushort_as_half(b.s[t]));
      }
      load(b, (it + 1) * D + d);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[t][v] = fmaf(prev_s[t], prev[t][v], acc[t][v]);

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

template <int NW, int D, bool SWI, bool NORM>
hipError_t launch_cfg(const LinOp& op, hipStream_t st) {
  SkinnyMap bm{};
  int total = 0;
  for (int s = 0; s < op.nseg; ++s) {
    total += (op.seg[s].w.N + kRows - 1) / kRows;
    bm.end[s] = total;
  }
  hipLaunchKernelGGL((q4_skinny_kernel<NW, D, SWI, NORM>), dim3(total), dim3(NW * 64), 0, st, op, bm);
  return hipGetLastError();
}

template <bool SWI>
hipError_t launch_sw(const LinOp& op, hipStream_t st) {
  return op.norm ? launch_cfg<8, 8, SWI, true>(op, st) : launch_cfg<8, 8, SWI, false>(op, st);
}

}  // namespace

bool skinny_supported(const LinOp& op) {
  if (op.M < 1 || op.M > kSkinnyMaxTokens || op.K % kGroup) return false;
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
