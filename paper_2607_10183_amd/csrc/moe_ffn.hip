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
#include "q4_mfma_unpack.h"

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

// ---------------------------------------------------------------- light experts

// Under a Zipf load most experts of a prefill call are routed a few tokens
// and a few many.  On the fixed 64-row MFMA tile of the grouped GEMM the
// light ones spend their K loop staging padding, and every tile walks K in
// short LDS-staged steps whose load latency the pipeline does not cover.
// Here an expert's tiles have 16, 32 or 64 rows (1, 2 or 4 token blocks of
// 16: the fewest that cover its count), every height in one launch with a
// code path per height, and the weights stream through registers once per
// tile:
//   * work items are (tile, block of output columns) in tile-major order; a
//     workgroup (one per CU) takes a contiguous run of one height's items, so
//     it mostly stays on one tile and its activations, and a ring of loads
//     runs on across items, so the next item's weights are in flight while an
//     item finishes; the item metadata comes through scalar loads, so waiting
//     for it leaves the ring's vector loads in flight;
//   * wavefront (ks, cg) takes K-slice ks (GS groups of 32 inputs) of the
//     light_steps(MT) 16-row steps of column group cg of an item (gate/up:
//     steps of gate rows, then the matching steps of up rows);
//   * the tile's activations for the K-slice stay in registers as the A
//     operands of v_mfma_f32_16x16x32_f16, one per token block and group
//     (lane n + 16 c holds token row n of the block, inputs 8c .. 8c + 7 of
//     the group, permuted to the nibble pair order);
//   * per step a lane loads GS / 4 x 16 code bytes of its weight row (groups
//     c, c + 4, ... of the slice: four lanes read 64 contiguous bytes) and the
//     row's scales of the slice; a 4 x 4 transpose of words across the four
//     16-lane rows (permlane32 and permlane16 swaps) gives every lane the code
//     word of its 8-input chunk for each group;
//   * with one token block each word becomes eight exact fp16 integers, one
//     MFMA per group sums that group's exact products and the group's fp16
//     scale multiplies the sums in fp32 (the batched-decode arithmetic); with
//     two or four blocks each word becomes eight weights w = RNE16(s * q) (q
//     exact, one rounding of the product: the grouped GEMM's operand), so the
//     ALU work per weight does not grow with the tile's rows, and the group
//     sums of every block accumulate in the MFMA's fp32 accumulator;
//   * each finished step's partial sums go to LDS; after a barrier the
//     K-slices are summed in slice order and the epilogue (SwiGLU and the RMS
//     factor, or the store by pair id) runs on every thread.
#ifndef LIGHT_D1
#define LIGHT_D1 8
#endif
#ifndef LIGHT_D2
#define LIGHT_D2 4
#endif
#ifndef LIGHT_D4
#define LIGHT_D4 4
#endif
#ifndef LIGHT_MT16
#define LIGHT_MT16 2
#endif
constexpr int kLightWaves = 8;  // at most, per workgroup (one workgroup per CU)
constexpr uint32_t kLightOob = 0x80000000u;  // an offset past every buffer here
// 16-row steps per item (the partial sums of an item fill at most 16 KB of
// LDS per wavefront) and steps of loads in flight (dividing the steps)
__host__ __device__ constexpr int light_steps(int mt) { return mt == 4 ? 4 : 8; }
constexpr int light_d(int gs, int mt) { return gs == 16 ? 2 : (mt == 1 ? LIGHT_D1 : (mt == 2 ? LIGHT_D2 : LIGHT_D4)); }

typedef float lf4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t light_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

template <typename T>
__device__ __forceinline__ T* uniform_ptr(T* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
  return reinterpret_cast<T*>(lo | (hi << 32));
}

// Loads through the global address space (a generic load would also count
// against the LDS wait counter, and its wait drains every load in flight).
template <typename T>
__device__ __forceinline__ T ld_global(const T* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  return *reinterpret_cast<const __attribute__((address_space(1))) T*>(reinterpret_cast<uintptr_t>(p));
#else
  return *p;
#endif
}

// Wave-uniform loads through the scalar data cache, for the tables an earlier
// launch wrote (that cache is invalidated when a launch starts).  Their wait
// counts against the scalar/LDS counter, so it leaves the vector loads in
// flight: waiting for a vector load here would wait for every weight load
// issued before it.  Addresses are wave-uniform and 4-byte aligned.
typedef int sint2_t __attribute__((ext_vector_type(2)));
typedef int sint4_t __attribute__((ext_vector_type(4)));

// Three consecutive ints in one round of loads.
__device__ __forceinline__ sint4_t s_ld3(const int32_t* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  sint2_t v;
  int w;
  asm volatile("s_load_dwordx2 %0, %2, 0x0\n\ts_load_dword %1, %2, 0x8\n\ts_waitcnt lgkmcnt(0)"
               : "=&s"(v), "=&s"(w)
               : "s"(p)
               : "memory");
  return sint4_t{v.x, v.y, w, 0};
#else
  return sint4_t{p[0], p[1], p[2], 0};
#endif
}

__device__ __forceinline__ sint2_t s_ld2(const int32_t* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  sint2_t v;
  asm volatile("s_load_dwordx2 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=&s"(v) : "s"(p) : "memory");
  return v;
#else
  return sint2_t{p[0], p[1]};
#endif
}

// One int from each of two tables, in one round of loads.
__device__ __forceinline__ sint2_t s_ld2_pair(const int32_t* pa, const int32_t* pb) {
#if defined(__HIP_DEVICE_COMPILE__)
  int va, vb;
  asm volatile("s_load_dword %0, %2, 0x0\n\ts_load_dword %1, %3, 0x0\n\ts_waitcnt lgkmcnt(0)"
               : "=&s"(va), "=&s"(vb)
               : "s"(pa), "s"(pb)
               : "memory");
  return sint2_t{va, vb};
#else
  return sint2_t{*pa, *pb};
#endif
}

// The code and scale pointers of two QViews of one ExpertW (byte offsets O0
// and O1), and one int from each of two tables, in one round of loads.
template <int O0, int O1>
__device__ __forceinline__ void s_ld_item(const ExpertW* w, const int32_t* pa, const int32_t* pb, sint4_t& q0,
                                          sint4_t& q1, int& va, int& vb) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile(
      "s_load_dwordx4 %0, %4, %7\n\t"
      "s_load_dwordx4 %1, %4, %8\n\t"
      "s_load_dword %2, %5, 0x0\n\t"
      "s_load_dword %3, %6, 0x0\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&s"(q0), "=&s"(q1), "=&s"(va), "=&s"(vb)
      : "s"(w), "s"(pa), "s"(pb), "i"(O0), "i"(O1)
      : "memory");
#else
  const char* b = reinterpret_cast<const char*>(w);
  q0 = *reinterpret_cast<const sint4_t*>(b + O0);
  q1 = *reinterpret_cast<const sint4_t*>(b + O1);
  va = *pa;
  vb = *pb;
#endif
}

template <typename T>
__device__ __forceinline__ T* ptr_of(int lo, int hi) {
  return reinterpret_cast<T*>((uint64_t)(uint32_t)lo | ((uint64_t)(uint32_t)hi << 32));
}

// Eight weights w = RNE16(s * q) from one code word, in the pair order of
// unpack_q (q exact, then one rounding of the product).
__device__ __forceinline__ gemv::half8_t dequant_word(uint32_t w, gemv::half2_t s2, const gemv::UnpackMasks& k) {
  const gemv::half8_t q = gemv::unpack_q(w, k);
  const gemv::half8_t s8 = {s2.x, s2.y, s2.x, s2.y, s2.x, s2.y, s2.x, s2.y};
  return q * s8;
}

// One work item of a light launch, all of it uniform.  Past the workgroup's
// items the pointers are null and every load of the ring reads zeros.
struct LightItem {
  const uint8_t* c0;    // codes / scales of gate (or down) and up
  const uint16_t* s0;
  const uint8_t* c1;
  const uint16_t* s1;
  int tix, cb, base, rows;
};

template <bool DOWN, int MT>
__device__ __forceinline__ LightItem light_item(const MoeArgs& a, int t0, int i, int i1, int ncb) {
  LightItem it;
  if (i >= i1) {
    it.c0 = it.c1 = nullptr;
    it.s0 = it.s1 = nullptr;
    it.tix = -1;
    it.cb = it.base = it.rows = 0;
    return it;
  }
  it.tix = i / ncb;
  it.cb = i % ncb;
  // scalar loads only: the ring's weight loads stay in flight meanwhile
  constexpr int O0 = DOWN ? (int)offsetof(ExpertW, down) : (int)offsetof(ExpertW, gate);
  constexpr int O1 = DOWN ? (int)offsetof(ExpertW, down) : (int)offsetof(ExpertW, up);
  static_assert(offsetof(QView, codes) == 0 && offsetof(QView, scales) == 8, "QView pointer layout");
  int e, row0, off, cnt;
  if (a.nb > 0) {
    // the batch's weights sit in the launch arguments
    const int2 t = a.btiles[it.tix];
    e = a.bexp[t.x];
    row0 = t.y;
    const ExpertW& w = a.bw[t.x];
    const QView& w0 = DOWN ? w.down : w.gate;
    const QView& w1 = DOWN ? w.down : w.up;
    it.c0 = uniform_ptr(w0.codes);
    it.s0 = uniform_ptr(w0.scales);
    it.c1 = uniform_ptr(w1.codes);
    it.s1 = uniform_ptr(w1.scales);
    const sint2_t oc = s_ld2_pair(uniform_ptr(a.offsets + e), uniform_ptr(a.counts + e));
    off = oc.x;
    cnt = oc.y;
  } else {
    const sint2_t t = s_ld2(uniform_ptr(a.tiles + 2 * (t0 + it.tix)));
    e = t.x;
    row0 = t.y;
    sint4_t q0, q1;
    s_ld_item<O0, O1>(uniform_ptr(a.table + e), uniform_ptr(a.offsets + e), uniform_ptr(a.counts + e), q0, q1, off,
                      cnt);
    it.c0 = ptr_of<const uint8_t>(q0.x, q0.y);
    it.s0 = ptr_of<const uint16_t>(q0.z, q0.w);
    it.c1 = ptr_of<const uint8_t>(q1.x, q1.y);
    it.s1 = ptr_of<const uint16_t>(q1.z, q1.w);
  }
  it.base = off + row0;
  it.rows = min(kLightTileRows * MT, cnt - row0);
  return it;
}

// Items i0 .. i1 - 1 of the tiles of height 16 MT listed from t0 (wave
// uniform), with red the partial-sum LDS ([wave][step][token block][lane])
// and row_dst / row_scale 16 MT entries of LDS each.
template <bool DOWN, int GS, int MT>
__device__ __forceinline__ void light_run(const MoeArgs& a, int t0, int i0, int i1, int ncb, int nk, int nc,
                                          lf4_t* red, int* row_dst, float* row_scale) {
  using namespace gemv;
  constexpr int S = light_steps(MT), D = light_d(GS, MT), RT = kLightTileRows * MT;
  static_assert(S % D == 0, "the ring restarts at every item");
  const int K = DOWN ? a.I : a.H, N = DOWN ? a.H : a.I, G = K / kGroup;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int ks = wave % nk, cg = wave / nk;
  const int n = lane & 15, c = lane >> 4;
  const int g0 = ks * GS;
  constexpr int OUTS = DOWN ? 16 * S : 8 * S;  // output columns per column group and item
  const uint32_t cbytes = (uint32_t)((size_t)N * K / 2), sbytes = (uint32_t)((size_t)N * G * 2);

  struct Ld {
    u32x4_t c[GS / 4];  // groups c, c + 4, ... of the slice
    u32x4_t s[GS / 8];  // the row's scales of the slice's groups
  };
  // step st of item it: weight row col0 + 16 st + n (gate/up: gate rows for
  // the first half of the steps, up rows after)
  auto load = [&](Ld& b, const LightItem& it, int st) {
    const bool second = !DOWN && st >= S / 2;
    const int row = (it.cb * nc + cg) * OUTS + 16 * (DOWN ? st : (st % (S / 2))) + n;
    const bool live = it.tix >= 0;
    const bool ok = row < N && live;
    const uint32_t co = ok ? (uint32_t)row * (uint32_t)(K / 2) + (uint32_t)(g0 + c) * 16 : kLightOob;
    const uint32_t so = ok ? ((uint32_t)row * (uint32_t)G + (uint32_t)g0) * 2 : kLightOob;
    const __amdgpu_buffer_rsrc_t rc = light_rsrc(second ? it.c1 : it.c0, live ? cbytes : 0);
    const __amdgpu_buffer_rsrc_t rs = light_rsrc(second ? it.s1 : it.s0, live ? sbytes : 0);
#pragma unroll
    for (int q = 0; q < GS / 4; ++q)
      b.c[q] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rc, co + 64 * q, 0, 0));
#pragma unroll
    for (int q = 0; q < GS / 8; ++q)
      b.s[q] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, so + 16 * q, 0, 0));
  };
  // A operands: token block t, row 16 t + n of the tile (zeros past its
  // rows); gate/up looks the rows' pair ids up before the ring's loads go
  // out, so that waiting for them does not wait for those
  const __amdgpu_buffer_rsrc_t rx = DOWN ? light_rsrc(a.h, (uint32_t)((size_t)a.M * a.k * a.I * 2))
                                         : light_rsrc(a.x, (uint32_t)((size_t)a.M * a.H * 2));
  half8_t xa[MT][GS];
  int prs[MT];
  auto pairs_of = [&](const LightItem& it) {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int m = kLightTileRows * t + n;
      prs[t] = DOWN ? 0 : ld_global(a.perm + it.base + (m < it.rows ? m : 0));
    }
  };
  auto load_x = [&](const LightItem& it) {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int m = kLightTileRows * t + n;
      const bool has_row = m < it.rows;
      const uint32_t rowoff =
          DOWN ? (uint32_t)(it.base + m) * (uint32_t)a.I * 2 : (uint32_t)(prs[t] / a.k) * (uint32_t)a.H * 2;
      const uint32_t xo = rowoff + (uint32_t)(g0 * kGroup + c * 8) * 2;
#pragma unroll
      for (int g = 0; g < GS; ++g) {
        const u32x4_t v = __builtin_bit_cast(
            u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rx, has_row ? xo + (uint32_t)g * kGroup * 2 : kLightOob, 0, 0));
        xa[t][g] = perm_x(v);
      }
    }
  };
  // output row and RMS factor of tile row m = threadIdx.x, loaded into
  // registers when a tile starts and stored to LDS at the end of each item's
  // steps, so that their wait comes after the ring's loads of that item
  int rdst = 0;
  float rsc = 1.f;
  auto row_info = [&](const LightItem& it) {
    if (threadIdx.x < (unsigned)RT) {
      const int m = threadIdx.x;
      if constexpr (DOWN) {
        rdst = ld_global(a.perm + it.base + (m < it.rows ? m : 0));
      } else {
        int p = prs[0];
#pragma unroll
        for (int t = 1; t < MT; ++t)
          if ((m >> 4) == t) p = prs[t];
        rdst = it.base + m;
        rsc = a.inv_r ? ld_global(a.inv_r + p / a.k) : 1.f;
      }
    }
  };
  // the next item: the same tile's metadata with another column block, or a
  // new tile's
  auto next_item = [&](const LightItem& p, int i) {
    if (i < i1 && i / ncb == p.tix) {
      LightItem it = p;
      it.cb = i % ncb;
      return it;
    }
    return light_item<DOWN, MT>(a, t0, i, i1, ncb);
  };

  // the tile's activations go out before the ring's weight loads, so that
  // the first step's wait for them leaves those in flight
  LightItem cur = light_item<DOWN, MT>(a, t0, i0, i1, ncb);
  pairs_of(cur);
  load_x(cur);
  __builtin_amdgcn_sched_barrier(0);
  Ld buf[D];
#pragma unroll
  for (int d = 0; d < D; ++d) load(buf[d], cur, d);
  __builtin_amdgcn_sched_barrier(0);
  row_info(cur);
  LightItem nxt = next_item(cur, i0 + 1);

  const UnpackMasks um = unpack_masks();
  const lf4_t zero = {0.f, 0.f, 0.f, 0.f};
  lf4_t* mine = red + (size_t)wave * S * MT * 64 + lane;
  constexpr int SPO = DOWN ? S : S / 2;  // steps per set of outputs
  const int nent = nc * SPO * MT * 64;

  for (int i = i0; i < i1; ++i) {
#pragma unroll
    for (int st = 0; st < S; ++st) {
      Ld& b = buf[st % D];
      uint32_t t4[GS / 4][4];
#pragma unroll
      for (int q = 0; q < GS / 4; ++q) {
        t4[q][0] = b.c[q].x;
        t4[q][1] = b.c[q].y;
        t4[q][2] = b.c[q].z;
        t4[q][3] = b.c[q].w;
      }
      u32x4_t sv[GS / 8];
#pragma unroll
      for (int q = 0; q < GS / 8; ++q) sv[q] = b.s[q];
      // refill: a later step of this item, or an early one of the next
      if (st + D < S)
        load(b, cur, st + D);
      else
        load(b, nxt, st + D - S);
#pragma unroll
      for (int q = 0; q < GS / 4; ++q) transpose_rows4(t4[q]);
      lf4_t acc[MT];
      if constexpr (MT == 1) {
        // one token block: exact group sums (independent MFMAs, integer
        // weights), each scaled by its group's scale in fp32
        acc[0] = zero;
#pragma unroll
        for (int h = 0; h < GS / 4; ++h) {
          lf4_t p[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int g = 4 * h + j;
            p[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[0][g], unpack_q(t4[h][j], um), zero, 0, 0, 0);
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int g = 4 * h + j;
            const uint32_t pair = sv[g >> 3][(g & 7) >> 1];
            const float sc = __half2float(__ushort_as_half((uint16_t)((g & 1) ? pair >> 16 : pair)));
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[0][v] = fmaf(sc, p[j][v], acc[0][v]);
          }
        }
      } else {
        // several token blocks share each dequantised weight: w = RNE16(s q),
        // the group sums accumulating in the MFMA
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[t] = zero;
#pragma unroll
        for (int g = 0; g < GS; ++g) {
          const uint32_t pair = sv[g >> 3][(g & 7) >> 1];
          const uint32_t sb = (g & 1) ? pair >> 16 : pair & 0xFFFFu;
          const half8_t wq = dequant_word(t4[g >> 2][g & 3], __builtin_bit_cast(half2_t, sb * 0x10001u), um);
#pragma unroll
          for (int t = 0; t < MT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[t][g], wq, acc[t], 0, 0, 0);
        }
      }
#pragma unroll
      for (int t = 0; t < MT; ++t) mine[(st * MT + t) * 64] = acc[t];
    }
    if (threadIdx.x < (unsigned)RT) {
      row_dst[threadIdx.x] = rdst;
      row_scale[threadIdx.x] = rsc;
    }
    __syncthreads();

    // slices summed in order; D[m][n] of a token block sits in lane
    // n + 16 (m / 4), item m % 4
    for (int q = threadIdx.x; q < nent; q += blockDim.x) {
      const int l = q & 63, t = (q >> 6) % MT, sidx = (q >> 6) / MT % SPO, cgq = (q >> 6) / MT / SPO;
      const int col = (cur.cb * nc + cgq) * OUTS + 16 * sidx + (l & 15);
      if (col >= N) continue;
      const lf4_t* r0 = red + (size_t)cgq * nk * S * MT * 64 + t * 64 + l;
      lf4_t v = r0[sidx * MT * 64], u = zero;
      if constexpr (!DOWN) u = r0[(sidx + SPO) * MT * 64];
      for (int k2 = 1; k2 < nk; ++k2) {
        v += r0[((size_t)k2 * S + sidx) * MT * 64];
        if constexpr (!DOWN) u += r0[((size_t)k2 * S + sidx + SPO) * MT * 64];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = kLightTileRows * t + 4 * (l >> 4) + j;
        if (m >= cur.rows) break;
        if constexpr (DOWN) {
          a.out[(size_t)row_dst[m] * a.H + col] = __float2half_rn(v[j]);
        } else {
          // RMS-normalised input: scale both products by the token's factor
          const float sc = row_scale[m];
          a.h[(size_t)row_dst[m] * a.I + col] = __float2half_rn(silu_f(v[j] * sc) * (u[j] * sc));
        }
      }
    }
    __syncthreads();
    if (i + 1 < i1) {
      if (nxt.tix != cur.tix) {
        pairs_of(nxt);
        load_x(nxt);
        row_info(nxt);
      }
      cur = nxt;
      nxt = next_item(cur, i + 2);
    }
  }
}

// One tile height per launch: the batch's tiles, or one class of the light list.
template <bool DOWN, int GS, int MT>
__global__ __launch_bounds__(kLightWaves * 64) void expert_light(MoeArgs a, int nk, int nc, int ncb) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int row_dst[kLightTileRows * MT];    // output row of tile row m (pair id / bucket row)
  __shared__ float row_scale[kLightTileRows * MT];  // gate/up: the token's RMS factor
  const int cls = light_class(MT);
  int t0 = 0, ntiles = a.nb;
  if (a.nb == 0) {
    static_assert(kLightClasses == 3, "one round of loads reads the three class counts");
    const sint4_t nt = s_ld3(uniform_ptr(a.n_tiles));
    t0 = (cls > 0 ? nt.x : 0) + (cls > 1 ? nt.y : 0);
    ntiles = cls == 0 ? nt.x : (cls == 1 ? nt.y : nt.z);
  }
  const int total = ntiles * ncb;
  const int per = (total + (int)gridDim.x - 1) / (int)gridDim.x;
  const int i0 = (int)blockIdx.x * per, i1 = min(i0 + per, total);
  if (i0 >= i1) return;
  light_run<DOWN, GS, MT>(a, t0, i0, i1, ncb, nk, nc, reinterpret_cast<lf4_t*>(smem), row_dst, row_scale);
}

// Relative cost of one item of each tile height (light_steps 16-row steps,
// 1, 2 or 4 token blocks) within one launch, from per-item times measured on
// MI355X with one workgroup per CU: with 8-group slices (hidden 2048, 512 and
// 2048 tokens) about 7.75 us for 16-row items, 9 us for 32-row items and 6 us
// for 64-row items (half the steps); with 16-group slices (hidden 4096, 512
// tokens) 14.4 us for 16-row and 21 us for 32-row items.
__host__ __device__ constexpr int light_item_cost(int gs, int mt) {
  return gs == 16 ? (mt == 2 ? 44 : 30) : (mt == 4 ? 24 : (mt == 2 ? 36 : 31));
}
__host__ __device__ inline int light_ncb(int N, int mt, int nc, bool down) {
  const int outs = (down ? 16 : 8) * light_steps(mt) * nc;
  return (N + outs - 1) / outs;
}

// Every tile height of the light list in one launch (classes MTMAX and
// below): the grid is shared among the classes in proportion to their items'
// cost, and each workgroup runs a contiguous range of one class's items, so
// the classes' start-up and tails overlap instead of following each other.
template <bool DOWN, int GS, int MTMAX>
__global__ __launch_bounds__(kLightWaves * 64) void expert_light_all(MoeArgs a, int nk, int nc) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int row_dst[kLightTileRows * MTMAX];
  __shared__ float row_scale[kLightTileRows * MTMAX];
  static_assert(kLightClasses == 3, "one round of loads reads the three class counts");
  const sint4_t nt = s_ld3(uniform_ptr(a.n_tiles));
  const int N = DOWN ? a.H : a.I, grid = (int)gridDim.x;
  const int cls0 = light_class(MTMAX);
  // items and cost per class (0: 64-row tiles, 1: 32, 2: 16), all uniform
  const int n0 = cls0 <= 0 ? nt.x * light_ncb(N, 4, nc, DOWN) : 0;
  const int n1 = cls0 <= 1 ? nt.y * light_ncb(N, 2, nc, DOWN) : 0;
  const int n2 = nt.z * light_ncb(N, 1, nc, DOWN);
  constexpr int w0 = light_item_cost(GS, 4), w1 = light_item_cost(GS, 2), w2 = light_item_cost(GS, 1);
  const long long tot = (long long)n0 * w0 + (long long)n1 * w1 + (long long)n2 * w2;
  if (tot == 0) return;
  // workgroups per class: the proportional share rounded down (at least one
  // for a class with items), then the rest one by one to the class whose
  // workgroups carry the most
  auto share = [&](int n, int w) { return n ? max(1, (int)((long long)grid * n * w / tot)) : 0; };
  int g0 = share(n0, w0), g1 = share(n1, w1), g2 = share(n2, w2);
  auto load_of = [](int n, int g, int w) { return g ? (n + g - 1) / g * w : 0; };
  while (g0 + g1 + g2 > grid) {  // only where the grid is smaller than the classes need
    if (g0 > 1 && g0 >= g1 && g0 >= g2) --g0;
    else if (g1 > 1 && g1 >= g2) --g1;
    else if (g2 > 1) --g2;
    else break;
  }
  while (g0 + g1 + g2 < grid) {
    const int l0 = load_of(n0, g0, w0), l1 = load_of(n1, g1, w1), l2 = load_of(n2, g2, w2);
    if (l0 >= l1 && l0 >= l2) ++g0;
    else if (l1 >= l2) ++g1;
    else ++g2;
  }
  const int b = (int)blockIdx.x;
  const int c = b < g0 ? 0 : (b < g0 + g1 ? 1 : 2);
  const int lb = b - (c == 0 ? 0 : (c == 1 ? g0 : g0 + g1));
  const int nc_items = c == 0 ? n0 : (c == 1 ? n1 : n2), gc = c == 0 ? g0 : (c == 1 ? g1 : g2);
  if (lb >= gc) return;
  const int per = (nc_items + gc - 1) / gc;
  const int i0 = __builtin_amdgcn_readfirstlane(lb * per);
  const int i1 = __builtin_amdgcn_readfirstlane(min(lb * per + per, nc_items));
  if (i0 >= i1) return;
  const int t0 = __builtin_amdgcn_readfirstlane((c > 0 ? nt.x : 0) + (c > 1 ? nt.y : 0));
  lf4_t* red = reinterpret_cast<lf4_t*>(smem);
  if constexpr (MTMAX >= 4)
    if (c == 0) return light_run<DOWN, GS, 4>(a, t0, i0, i1, light_ncb(N, 4, nc, DOWN), nk, nc, red, row_dst, row_scale);
  if (c == 1) return light_run<DOWN, GS, 2>(a, t0, i0, i1, light_ncb(N, 2, nc, DOWN), nk, nc, red, row_dst, row_scale);
  light_run<DOWN, GS, 1>(a, t0, i0, i1, light_ncb(N, 1, nc, DOWN), nk, nc, red, row_dst, row_scale);
}

// groups per K-slice: 8, or 16 where 8 would take more than kLightWaves slices
int light_gs(int K) { return K / kGroup / 8 <= kLightWaves ? 8 : 16; }
// token blocks per tile the kernels hold: 4 with 8-group slices, 2 with 16
// (the activations of 16 groups x 2 blocks fill 128 registers)
int light_mtmax_k(int K) { return light_gs(K) == 8 ? 4 : LIGHT_MT16; }

template <bool DOWN, int GS, int MT>
hipError_t launch_light_cfg(const MoeArgs& a, int tile_bound, int nk, int nc, hipStream_t s) {
  const int N = DOWN ? a.H : a.I;
  const int outs = (DOWN ? 16 : 8) * light_steps(MT) * nc;
  const int ncb = (N + outs - 1) / outs;
  const size_t lds = (size_t)nk * nc * light_steps(MT) * MT * 64 * sizeof(lf4_t);
  if (lds + 2 * kLightTileRows * MT * 4 > lds_limit()) return hipErrorInvalidValue;
  // one workgroup per CU: each holds its loads in flight in registers
  int cus = 256;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                               hipSuccess || cus < 1)
    cus = 256;
  const int grid = std::min(tile_bound * ncb, cus);
  hipLaunchKernelGGL((expert_light<DOWN, GS, MT>), dim3(grid), dim3(nk * nc * 64), lds, s, a, nk, nc, ncb);
  return hipGetLastError();
}

template <bool DOWN>
hipError_t launch_light(const MoeArgs& a, int cls, int tile_bound, hipStream_t s) {
  if (tile_bound <= 0) return hipSuccess;
  if (!light_supported(a.H, a.I) || cls < 0 || cls >= kLightClasses) return hipErrorInvalidValue;
  const int K = DOWN ? a.I : a.H;
  const int gs = light_gs(K);
  const int nk = K / (gs * kGroup);
  const int nc = std::max(1, kLightWaves / nk);
  if (gs == 16) {
    if (cls == 2) return launch_light_cfg<DOWN, 16, 1>(a, tile_bound, nk, nc, s);
    if (cls == 1) return launch_light_cfg<DOWN, 16, 2>(a, tile_bound, nk, nc, s);
    return hipErrorInvalidValue;
  }
  if (cls == 0) return launch_light_cfg<DOWN, 8, 4>(a, tile_bound, nk, nc, s);
  if (cls == 1) return launch_light_cfg<DOWN, 8, 2>(a, tile_bound, nk, nc, s);
  return launch_light_cfg<DOWN, 8, 1>(a, tile_bound, nk, nc, s);
}

template <bool DOWN, int GS, int MTMAX>
hipError_t launch_light_all_cfg(const MoeArgs& a, int tile_bound, int nk, int nc, hipStream_t s) {
  const int N = DOWN ? a.H : a.I;
  size_t lds = 0;
  for (int mt = 1; mt <= MTMAX; mt *= 2)
    lds = std::max(lds, (size_t)nk * nc * light_steps(mt) * mt * 64 * sizeof(lf4_t));
  if (lds + 2 * kLightTileRows * MTMAX * 4 > lds_limit()) return hipErrorInvalidValue;
  int cus = 256;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                               hipSuccess || cus < 1)
    cus = 256;
  // at least one workgroup per class; 64-row items are the most per tile
  const int grid = std::max(kLightClasses, std::min(tile_bound * light_ncb(N, MTMAX, nc, DOWN), cus));
  hipLaunchKernelGGL((expert_light_all<DOWN, GS, MTMAX>), dim3(grid), dim3(nk * nc * 64), lds, s, a, nk, nc);
  return hipGetLastError();
}

template <bool DOWN>
hipError_t launch_light_all(const MoeArgs& a, int mtmax, int tile_bound, hipStream_t s) {
  if (tile_bound <= 0) return hipSuccess;
  if (mtmax == 1) return launch_light<DOWN>(a, light_class(1), tile_bound, s);
  if (!light_supported(a.H, a.I) || a.nb != 0 || (mtmax != 2 && mtmax != 4)) return hipErrorInvalidValue;
  const int K = DOWN ? a.I : a.H;
  const int gs = light_gs(K);
  if (mtmax > light_mtmax_k(K)) return hipErrorInvalidValue;
  const int nk = K / (gs * kGroup);
  const int nc = std::max(1, kLightWaves / nk);
  if (gs == 16) return launch_light_all_cfg<DOWN, 16, 2>(a, tile_bound, nk, nc, s);
  if (mtmax == 4) return launch_light_all_cfg<DOWN, 8, 4>(a, tile_bound, nk, nc, s);
  return launch_light_all_cfg<DOWN, 8, 2>(a, tile_bound, nk, nc, s);
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

bool light_supported(int H, int I) {
  // K-slices of 8 or 16 groups, at most kLightWaves of them
  auto ok = [](int K) {
    if (K % (8 * kGroup)) return false;
    const int G = K / kGroup, gs = light_gs(K);
    return G % gs == 0 && G / gs <= kLightWaves;
  };
  return ok(H) && ok(I);
}

// the gate/up and down launches share the tile list
int light_mtmax(int H, int I) { return std::min(light_mtmax_k(H), light_mtmax_k(I)); }

hipError_t launch_light_gateup(const MoeArgs& a, int cls, int tile_bound, hipStream_t s) {
  return launch_light<false>(a, cls, tile_bound, s);
}

hipError_t launch_light_down(const MoeArgs& a, int cls, int tile_bound, hipStream_t s) {
  return launch_light<true>(a, cls, tile_bound, s);
}

hipError_t launch_light_all_gateup(const MoeArgs& a, int mtmax, int tile_bound, hipStream_t s) {
  return launch_light_all<false>(a, mtmax, tile_bound, s);
}

hipError_t launch_light_all_down(const MoeArgs& a, int mtmax, int tile_bound, hipStream_t s) {
  return launch_light_all<true>(a, mtmax, tile_bound, s);
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
