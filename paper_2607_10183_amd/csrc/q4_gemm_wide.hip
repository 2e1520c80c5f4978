// Prefill dequantising GEMM with 512-row tiles for block-int4 weights on
// CDNA4 (gfx950): each weight is dequantised once per 512 activation rows.
//
// The dense contraction of a prefill chunk (Sec. 2.2; chunked prefill, Sec.
// 5.1) runs on the matrix cores.  Dequantisation is ALU work per weight, so
// the tile spans as many activation rows as the accumulators allow:
//   * a 512-thread workgroup owns a 512 x 128 output tile; its 8 waves are
//     stacked along M, each owning 64 rows x 128 columns as 2 x 4 blocks of
//     v_mfma_f32_32x32x16_f16 (the fp16 shape that runs at the full rate;
//     16x16x32 runs at half of it on gfx950);
//   * weights: per K step of 64 (two scale groups) each lane dequantises 16
//     weights (nibble -> 1024 + u by a byte permute and a mask-and-or, minus
//     1032 exactly, times the group scale with one rounding) into a shared,
//     double-buffered LDS tile in natural k order; the codes come from a
//     ring of register buffers three steps ahead;
//   * activations: each wave loads its own 64 rows with coalesced 16-byte
//     loads (8 rows x 128 B per instruction: the MFMA operand layout, 32 rows
//     x 32 B per instruction, delivers 3.4x less bandwidth from L2) one step
//     ahead into registers, and writes them into its own LDS rows after the
//     last fragment read of the step;
//   * LDS rows are padded to 144 B, which makes the 16-byte fragment reads
//     conflict-free (183 B/clk per CU measured, against 32 at a 128 B pitch);
//   * each 16-deep substep is one fenced phase: the next substep's fragment
//     reads, this substep's 8 MFMAs, then a slice of the dequantisation,
//     activation staging and code loads, which runs under the MFMAs;
//   * workgroup ids are remapped so each XCD takes a contiguous run of tiles;
//   * where the output has too few tiles to occupy the CUs (the O and down
//     projections of a 512-token chunk have 32), K is split into up to 8
//     ranges: each workgroup writes its raw fp32 sums for one range, and a
//     second kernel adds the ranges in order and applies the epilogue.
// One launch covers up to three tensors sharing the input, and fuses RMS
// normalisation of the input (rows scaled by precomputed 1/rms values, so the
// main loop carries no sums of squares), the SwiGLU product, the residual add
// and the grouped-query head expansion of a context-length-1 attention.
#include <algorithm>

#include "common.h"

namespace atsi {
namespace {

typedef _Float16 w_h8_t __attribute__((ext_vector_type(8)));
typedef _Float16 w_h2_t __attribute__((ext_vector_type(2)));
typedef float w_f16_t __attribute__((ext_vector_type(16)));
typedef unsigned w_u4_t __attribute__((ext_vector_type(4)));

constexpr uint32_t kOob = 0x80000000u;  // an offset past every buffer here
constexpr int kBM = 512;                // tile rows
constexpr int kBN = 128;                // tile columns (weight rows)
constexpr int kBK = 64;                 // K per step: two scale groups
constexpr int kPitch = 72;              // LDS row pitch in halves (64 + 8)
constexpr int kRows = 64;               // activation rows per wave
constexpr int kRing = 4;                // code buffers (steps in flight)
constexpr int kThreads = 512;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

// One 32-bit code word (k0..k7, k0 in the low nibble) -> eight fp16 weights
// s * q in natural order: byte b of w and of w >> 4 are permuted into the low
// and high halves, masked to one nibble each, offset to (1024 + u_2b,
// 1024 + u_2b+1) by OR-ing the exponent of 1024, then (v - 1032) * s.
__device__ __forceinline__ w_u4_t dq_word(uint32_t w, w_h2_t s2, uint32_t mask, uint32_t magic) {
  const uint32_t w4 = w >> 4;
  const w_h2_t off = {(_Float16)1032.f, (_Float16)1032.f};
  w_u4_t r;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const uint32_t sel = (uint32_t)b | 0x0C00u | ((uint32_t)(4 + b) << 16) | 0x0C000000u;
    const uint32_t t = __builtin_amdgcn_perm(w4, w, sel);
    w_h2_t h = __builtin_bit_cast(w_h2_t, (t & mask) | magic);
    h = (h - off) * s2;  // q exactly, then one rounding of s * q
    r[b] = __builtin_bit_cast(uint32_t, h);
  }
  return r;
}

// silu(g) = g / (1 + e^-g) with the hardware exponential and reciprocal
__device__ __forceinline__ float silu_fast(float g) { return g * __builtin_amdgcn_rcpf(1.f + __expf(-g)); }

struct WideMap {
  int end[kMaxSeg];  // cumulative tile counts per segment
  int tiles_m;
  int total;         // output tiles
  int splits;        // K ranges per tile (workgroups = total * splits)
  int tiles_n;       // tile columns over all segments (partial rows hold tiles_n * kBN floats)
};

// K steps of range r out of `splits` over nk steps
__device__ __forceinline__ int range_begin(int r, int nk, int splits) { return (int)(((long)r * nk) / splits); }

// SPLIT: write the raw sums of K range blockIdx / total to part[range][m][tile column]
// (NORM is then applied by the reduction).
template <bool SWI, bool NORM, bool SPLIT>
__global__ __launch_bounds__(kThreads, 1) void q4_gemm_wide_kernel(LinOp op, WideMap tm, float* __restrict__ part) {
  constexpr int NOUT = SWI ? kBN / 2 : kBN;
  __shared__ __attribute__((aligned(16))) _Float16 Bs[2][kBN * kPitch];
  __shared__ __attribute__((aligned(16))) _Float16 As[8 * kRows * kPitch];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nwg = tm.total * tm.splits;
  int bid = blockIdx.x;
  if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  // range-major order: the workgroups of one XCD share a K range of the activations
  const int range = bid / tm.total;
  bid -= range * tm.total;
  int sgi = 0;
  while (sgi < op.nseg - 1 && bid >= tm.end[sgi]) ++sgi;
  const int local = bid - (sgi ? tm.end[sgi - 1] : 0);
  const int tmi = local % tm.tiles_m, tni = local / tm.tiles_m;
  const Seg& sg = op.seg[sgi];
  const int M = op.M, K = op.K, N = sg.w.N, G = K / kGroup;
  const int m0 = tmi * kBM, n0 = tni * NOUT;
  const int nk_all = (K + kBK - 1) / kBK;
  const int kb = range_begin(range, nk_all, tm.splits);
  const int nk = range_begin(range + 1, nk_all, tm.splits) - kb;  // steps of this range
  // the buffers start at the range; inputs past klim (the range's end, or K) read zeros
  const int klim = min(K - kb * kBK, nk * kBK), glim = klim / kGroup;
  const size_t ka = (size_t)kb * kBK;

  const __amdgpu_buffer_rsrc_t ra = rsrc(op.x + ka, (uint32_t)(((size_t)M * K - ka) * 2));
  __amdgpu_buffer_rsrc_t rc[2], rs[2];
  rc[0] = rsrc(sg.w.codes + ka / 2, (uint32_t)((size_t)N * K / 2 - ka / 2));
  rs[0] = rsrc(sg.w.scales + ka / kGroup, (uint32_t)(((size_t)N * G - ka / kGroup) * 2));
  if constexpr (SWI) {
    rc[1] = rsrc(sg.w2.codes + ka / 2, (uint32_t)((size_t)N * K / 2 - ka / 2));
    rs[1] = rsrc(sg.w2.scales + ka / kGroup, (uint32_t)(((size_t)N * G - ka / kGroup) * 2));
  } else {
    rc[1] = rc[0];
    rs[1] = rs[0];
  }
  _Float16* Aw = As + wave * kRows * kPitch;

  // ---- activations: instruction r covers rows 8 r + l/8 of the wave's 64,
  // 16-byte chunk l%8 of the step's 128 bytes
  w_u4_t ax[8];
  auto load_ax = [&](int kt) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int row = m0 + kRows * wave + 8 * r + (lane >> 3);
      const int k = kt * kBK + 8 * (lane & 7);
      const uint32_t off = (row < M && k < klim) ? ((uint32_t)row * (uint32_t)K + (uint32_t)k) * 2 : kOob;
      ax[r] = __builtin_bit_cast(w_u4_t, __builtin_amdgcn_raw_buffer_load_b128(ra, off, 0, 0));
    }
  };
  auto store_ax = [&]() {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      *reinterpret_cast<w_u4_t*>(Aw + (8 * r + (lane >> 3)) * kPitch + 8 * (lane & 7)) = ax[r];
    }
  };
  // fragment (i, ks): lane l holds row 32 i + l%32, k 16 ks + 8 (l/32) .. +7
  auto afrag = [&](int i, int ks) -> w_h8_t {
    return *reinterpret_cast<const w_h8_t*>(Aw + (32 * i + (lane & 31)) * kPitch + 16 * ks + 8 * (lane >> 5));
  };

  // ---- weights: lane task = tile row tid/4, group (tid/2)%2 of the step, half tid%2 (16 weights).
  // Tile rows come in chunks of 32; for SwiGLU the chunks alternate gate / up
  // rows of the same 32 outputs.  A wave's lanes cover 16 rows of one chunk,
  // so the tensor a load reads is uniform across the wave.
  const int br = tid >> 2, bg = (tid >> 1) & 1, bh = tid & 1;
  const int bch = wave >> 1;
  const int bt = SWI ? (bch & 1) : 0;
  const int bn = SWI ? n0 + 32 * (bch >> 1) + (br & 31) : n0 + br;
  struct BCode {
    uint32_t c0, c1, s;
  };
  auto load_b = [&](BCode& b, int kt) {
    const int gg = 2 * kt + bg;
    const bool ok = bn < N && gg < glim;
    const uint32_t co = ok ? (uint32_t)bn * (uint32_t)(K / 2) + (uint32_t)gg * 16 + 8u * bh : kOob;
    const uint32_t so = ok ? ((uint32_t)bn * (uint32_t)G + (uint32_t)gg) * 2 : kOob;
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(rc[bt], co, 0, 2);
    b.c0 = v[0];
    b.c1 = v[1];
    b.s = __builtin_amdgcn_raw_buffer_load_b16(rs[bt], so, 0, 2);
  };
  uint32_t mask, magic;
  asm volatile("s_mov_b32 %0, %1" : "=s"(mask) : "i"(0x000F000Fu));
  asm volatile("v_mov_b32 %0, %1" : "=v"(magic) : "i"(0x64006400u));
  _Float16* bdst = &Bs[0][br * kPitch + 32 * bg + 16 * bh];
  auto dq_store = [&](const BCode& b, int buf, int w) {
    const _Float16 sv = __builtin_bit_cast(_Float16, (uint16_t)b.s);
    const w_h2_t s2 = {sv, sv};
    *reinterpret_cast<w_u4_t*>(bdst + buf * (kBN * kPitch) + 8 * w) = dq_word(w ? b.c1 : b.c0, s2, mask, magic);
  };
  auto bfrag = [&](int buf, int ks, int j) -> w_h8_t {
    return *reinterpret_cast<const w_h8_t*>(&Bs[buf][(32 * j + (lane & 31)) * kPitch + 16 * ks + 8 * (lane >> 5)]);
  };

  w_f16_t acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  BCode ring[kRing];
#pragma unroll
  for (int d = 0; d < kRing - 1; ++d) load_b(ring[d], d);
  load_ax(0);
  store_ax();
  load_ax(1);
  dq_store(ring[0], 0, 0);
  dq_store(ring[0], 0, 1);
  __syncthreads();

  // Step s of the range (ring slot rq = s % kRing at compile time): MFMAs on weight buffer
  // s % 2; step s + 1's weights are dequantised into the other buffer, the
  // codes of step s + kRing - 1 are loaded into the slot step s - 1 used, and
  // step s + 1's activations are staged once this step's fragments are read.
  // Steps past the range read zeros (out-of-range buffer loads) and add zeros.
  auto step = [&](int s, int rq) {
    const int buf = s & 1;
    w_h8_t bf[2][4], af[2][2];
#pragma unroll
    for (int j = 0; j < 4; ++j) bf[0][j] = bfrag(buf, 0, j);
#pragma unroll
    for (int i = 0; i < 2; ++i) af[0][i] = afrag(i, 0);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int c = ks & 1;
      if (ks + 1 < 4) {
#pragma unroll
        for (int j = 0; j < 4; ++j) bf[c ^ 1][j] = bfrag(buf, ks + 1, j);
#pragma unroll
        for (int i = 0; i < 2; ++i) af[c ^ 1][i] = afrag(i, ks + 1);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[c][i], bf[c][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (ks == 0) dq_store(ring[(rq + 1) % kRing], buf ^ 1, 0);
      if (ks == 1) dq_store(ring[(rq + 1) % kRing], buf ^ 1, 1);
      if (ks == 2) load_b(ring[(rq + kRing - 1) % kRing], s + kRing - 1);
      if (ks == 3) {
        store_ax();
        load_ax(s + 2);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
  };
  for (int s = 0; s < nk; s += kRing) {
    step(s + 0, 0);
    step(s + 1, 1);
    step(s + 2, 2);
    step(s + 3, 3);
  }

  // D of a 32x32 block: lane l holds column l % 32, item v row 8 (v/4) + 4 (l/32) + v % 4.
  if constexpr (SPLIT) {
    // raw sums, restaged 8 rows at a time through the wave's LDS rows so that
    // each lane writes 16 consecutive floats of one row
    float* stage = reinterpret_cast<float*>(Aw);  // [8][kBN] fp32
    const size_t pc = (size_t)tm.tiles_n * kBN;
    const int tcol = ((sgi ? tm.end[sgi - 1] : 0) / tm.tiles_m + tni) * kBN;
    float* dst = part + (size_t)range * M * pc + tcol;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int vv = 0; vv < 4; ++vv)
#pragma unroll
          for (int j = 0; j < 4; ++j) stage[(4 * (lane >> 5) + vv) * kBN + 32 * j + (lane & 31)] = acc[i][j][4 * q + vv];
        const int rl = lane >> 3, c0 = 16 * (lane & 7);
        const int m = m0 + kRows * wave + 32 * i + 8 * q + rl;
        if (m < M) {
#pragma unroll
          for (int e = 0; e < 16; e += 4)
            *reinterpret_cast<float4*>(dst + (size_t)m * pc + c0 + e) =
                *reinterpret_cast<const float4*>(&stage[rl * kBN + c0 + e]);
        }
      }
    return;
  }
  auto out_at = [&](int i, int v, int j, int& m, int& n, float& o) {
    const int ml = kRows * wave + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    m = m0 + ml;
    n = SWI ? n0 + 32 * (j >> 1) + (lane & 31) : n0 + 32 * j + (lane & 31);
    const float sc = NORM ? (m < M ? op.rinv[m] : 0.f) : 1.f;
    o = acc[i][j][v] * sc;
    if constexpr (SWI) o = silu_fast(o) * (acc[i][j + 1][v] * sc);
  };
  if (sg.expand > 1) {
    // grouped-query expansion: each output goes to several query heads
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (SWI && (j & 1)) continue;
          int m, n;
          float o;
          out_at(i, v, j, m, n, o);
          if (m >= M || n >= N) continue;
          const int hd = op.head_dim, jh = n / hd, d = n % hd;
          const __half h = __float2half_rn(o);
          for (int e = 0; e < sg.expand; ++e) sg.y[(size_t)m * sg.ldy + (size_t)(jh * sg.expand + e) * hd + d] = h;
        }
    return;
  }
  // Otherwise restage 8 rows at a time through the wave's own LDS rows (free
  // now) as fp32, so that each lane adds the residual and rounds 8 or 16
  // consecutive outputs of one row and stores them in one or two 16-byte
  // stores instead of one 2-byte store per output.
  constexpr int W = NOUT;                      // outputs per tile row
  constexpr int PER = W / 8;                   // outputs per lane per pass (8 lanes per row)
  float* stage = reinterpret_cast<float*>(Aw);  // [8][W] fp32 (4 KiB of the wave's 9 KiB)
  const bool full_cols = n0 + W <= N && (sg.ldy % 8) == 0;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma unroll
      for (int vv = 0; vv < 4; ++vv)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (SWI && (j & 1)) continue;
          int m, n;
          float o;
          out_at(i, 4 * q + vv, j, m, n, o);
          stage[(4 * (lane >> 5) + vv) * W + (n - n0)] = o;
        }
      // row 8 q + (l/8) of this block, outputs PER * (l % 8) .. +PER
      const int rl = lane >> 3, c0 = PER * (lane & 7);
      const int m = m0 + kRows * wave + 32 * i + 8 * q + rl;
      float o[PER];
#pragma unroll
      for (int e = 0; e < PER; e += 4) {
        const float4 t = *reinterpret_cast<const float4*>(&stage[rl * W + c0 + e]);
        o[e] = t.x;
        o[e + 1] = t.y;
        o[e + 2] = t.z;
        o[e + 3] = t.w;
      }
      if (m < M) {
        const size_t at = (size_t)m * sg.ldy + n0 + c0;
        if (full_cols) {
          if (op.res && sgi == 0) {
#pragma unroll
            for (int e = 0; e < PER; e += 8) {
              const uint4 r = *reinterpret_cast<const uint4*>(op.res + at + e);
              const __half* rh = reinterpret_cast<const __half*>(&r);
#pragma unroll
              for (int t = 0; t < 8; ++t) o[e + t] += __half2float(rh[t]);
            }
          }
          if (op.y32 && sgi == 0) {
#pragma unroll
            for (int e = 0; e < PER; e += 4)
              *reinterpret_cast<float4*>(op.y32 + at + e) = make_float4(o[e], o[e + 1], o[e + 2], o[e + 3]);
          } else {
#pragma unroll
            for (int e = 0; e < PER; e += 8) {
              uint4 w;
              __half* wh = reinterpret_cast<__half*>(&w);
#pragma unroll
              for (int t = 0; t < 8; ++t) wh[t] = __float2half_rn(o[e + t]);
              *reinterpret_cast<uint4*>(sg.y + at + e) = w;
            }
          }
        } else {
#pragma unroll
          for (int e = 0; e < PER; ++e) {
            if (n0 + c0 + e >= N) break;
            float v = o[e];
            if (op.res && sgi == 0) v += __half2float(op.res[at + e]);
            if (op.y32 && sgi == 0)
              op.y32[at + e] = v;
            else
              sg.y[at + e] = __float2half_rn(v);
          }
        }
      }
    }
}

// Sum of the K ranges of a split launch, in range order, then the epilogue of
// the single-range kernel: one thread per 4 consecutive outputs of a row
// (16-byte loads of each range's partial sums).
template <bool SWI, bool NORM>
__global__ __launch_bounds__(256) void wide_reduce_kernel(LinOp op, WideMap tm, const float* __restrict__ part) {
  constexpr int NOUT = SWI ? kBN / 2 : kBN;
  constexpr int Q = NOUT / 4;  // quads per tile row
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long total = (long)op.M * tm.tiles_n * Q;
  if (idx >= total) return;
  const int o = 4 * (int)(idx % Q);
  const long rest = idx / Q;
  const int T = (int)(rest % tm.tiles_n), m = (int)(rest / tm.tiles_n);
  int sgi = 0;
  while (sgi < op.nseg - 1 && T >= tm.end[sgi] / tm.tiles_m) ++sgi;
  const int tni = T - (sgi ? tm.end[sgi - 1] / tm.tiles_m : 0);
  const Seg& sg = op.seg[sgi];
  const int n = tni * NOUT + o;
  if (n >= sg.w.N) return;
  const size_t pc = (size_t)tm.tiles_n * kBN;
  const int col = T * kBN + (SWI ? 64 * (o >> 5) + (o & 31) : o);  // 4 columns in one 32-column chunk
  const float* p = part + (size_t)m * pc + col;
  const size_t stride = (size_t)op.M * pc;
  typedef float f4_t __attribute__((ext_vector_type(4)));
  f4_t g = {0.f, 0.f, 0.f, 0.f}, u = g;
  for (int r = 0; r < tm.splits; ++r) {
    g += __builtin_nontemporal_load(reinterpret_cast<const f4_t*>(p + r * stride));
    if constexpr (SWI) u += __builtin_nontemporal_load(reinterpret_cast<const f4_t*>(p + r * stride + 32));
  }
  const float sc = NORM ? op.rinv[m] : 1.f;
  const float gv[4] = {g.x, g.y, g.z, g.w}, uv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (n + e >= sg.w.N) break;
    float v = gv[e] * sc;
    if constexpr (SWI) v = silu_fast(v) * (uv[e] * sc);
    emit_out(op, sg, sgi, m, n + e, v);
  }
}

template <bool SWI, bool NORM>
hipError_t launch_wide(const LinOp& op, const WideMap& tm, float* part, hipStream_t st) {
  if (tm.splits == 1) {
    hipLaunchKernelGGL((q4_gemm_wide_kernel<SWI, NORM, false>), dim3(tm.total), dim3(kThreads), 0, st, op, tm,
                       nullptr);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((q4_gemm_wide_kernel<SWI, false, true>), dim3(tm.total * tm.splits), dim3(kThreads), 0, st, op,
                     tm, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long quads = (long)op.M * tm.tiles_n * (SWI ? kBN / 8 : kBN / 4);
  hipLaunchKernelGGL((wide_reduce_kernel<SWI, NORM>), dim3((unsigned)((quads + 255) / 256)), dim3(256), 0, st, op, tm,
                     part);
  return hipGetLastError();
}

WideMap wide_map(const LinOp& op, int splits) {
  const int nout = op.swiglu ? kBN / 2 : kBN;
  WideMap tm{};
  tm.tiles_m = (op.M + kBM - 1) / kBM;
  int total = 0, tn = 0;
  for (int s = 0; s < op.nseg; ++s) {
    const int t = (op.seg[s].w.N + nout - 1) / nout;
    tn += t;
    total += tm.tiles_m * t;
    tm.end[s] = total;
  }
  tm.total = total;
  tm.tiles_n = tn;
  tm.splits = splits;
  return tm;
}

bool wide_offsets_ok(const LinOp& op) {
  // 32-bit buffer offsets for the activations and every tensor
  if ((size_t)op.M * op.K * 2 >= kOob) return false;
  for (int s = 0; s < op.nseg; ++s) {
    const QView* v[2] = {&op.seg[s].w, &op.seg[s].w2};
    for (int t = 0; t < (op.swiglu ? 2 : 1); ++t)
      if ((size_t)v[t]->N * v[t]->K / 2 + (size_t)v[t]->K >= kOob) return false;
  }
  return true;
}

}  // namespace

// One range when the tiles fill three quarters of the CUs; otherwise the
// fewest ranges that do, keeping at least 8 K steps (512 inputs) per range.
int gemm_wide_splits(const LinOp& op) {
  if (op.M < 256 || !wide_offsets_ok(op)) return 0;
  const int tiles = wide_map(op, 1).total;
  if (tiles >= kWideMinTiles) return 1;
  const int nk = (op.K + kBK - 1) / kBK;
  const int want = (kWideMinTiles + tiles - 1) / tiles;
  const int splits = std::min(std::min(want, kWideMaxSplits), nk / 8);
  return splits >= 2 ? splits : 0;
}

size_t gemm_wide_part_bytes(const LinOp& op, int splits) {
  if (splits <= 1) return 0;
  return (size_t)splits * op.M * wide_map(op, splits).tiles_n * kBN * sizeof(float);
}

hipError_t launch_gemm_wide(const LinOp& op, int splits, float* part, hipStream_t st) {
  if (splits < 1 || splits > kWideMaxSplits || !wide_offsets_ok(op) || (splits > 1 && !part) ||
      (op.norm && !op.rinv))
    return hipErrorInvalidValue;
  const WideMap tm = wide_map(op, splits);
  if (op.swiglu)
    return op.norm ? launch_wide<true, true>(op, tm, part, st) : launch_wide<true, false>(op, tm, part, st);
  return op.norm ? launch_wide<false, true>(op, tm, part, st) : launch_wide<false, false>(op, tm, part, st);
}

}  // namespace atsi
