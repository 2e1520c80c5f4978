// Fused batch-1 decode step of one 8B-shaped dense decoder layer in a single
// persistent launch.
//
// At batch 1 the layer is four dependent GEMVs over 122.7 MB of weights
// (Sec. 2.2: decode reads every weight once per token): q, k, v = rms(h)
// [Wq Wk Wv]; h += attn Wo; f = silu(rms(h) Wg) * (rms(h) Wu); h += f Wd.
// Four launches pay four ramp-ups and drains.  Here one workgroup per CU
// walks the four phases with grid barriers between them, and because weights
// do not depend on activations each wavefront keeps its next weight loads in
// flight across a barrier: HBM keeps streaming while the grid synchronises
// and restages its input.
//
// Each phase is the one-token GEMV of q4_gemv.hip in a fixed shape: a
// workgroup of 14 wavefronts owns R consecutive output rows; wavefront
// (s, p) takes K-slice s (groups 64 s + lane, one 16-byte load per lane and
// row) of rows p + P i, i < C; the input is staged in LDS and held in
// registers; partials are summed by the transposed butterfly and the slices
// meet in LDS in slice order.  The per-row arithmetic is the standalone
// GEMV's, so both paths give the same bits.
//
//   phase  rows                 K      S x P   R (rows per workgroup)   C
//   q/k/v  4096 + 1024 + 1024   4096   2 x 7   24                       4
//   o      4096                 4096   2 x 7   16                       3
//   gate/up 14336 (x 2)         4096   2 x 7   56                       8
//   down   4096                 14336  7 x 2   16                       8
//
// Loads run through a ring of kRing steps in flight per wavefront, numbered
// across the phases, so the first loads of a phase are issued during the
// previous one.  Activations that cross workgroups are stored and loaded at
// agent scope; the grid barrier counts arrivals per XCD, then across XCDs.  Every wait is bounded: a barrier that
// does not complete sets an error flag and lets the launch finish.  The
// launch is an ordinary one of exactly one workgroup per CU, which the
// launcher checks fits; co-residency then holds on an otherwise idle GPU, and
// the bounded wait covers the case where it does not.
//
// Measured on MI355X, each grid barrier (three chained cross-XCD atomic round
// trips, then the poll) costs more than the kernel boundary it replaces: the
// layer takes 41 us here against 32.6 us as four graph-replayed launches, so
// the library runs it only on request (ATSI_FUSED_DECODE_LAYER=1).
#include "layer.h"
#include "q4_gemv_core.h"


namespace atsi {
namespace {

using namespace gemv;

// shape of the fused layer
constexpr int kH = 4096, kHq = 4096, kHkv = 1024, kI = 14336;
constexpr int kWG = 256;               // workgroups (one per CU)
constexpr int kWaves = 14;
constexpr int kThreads = kWaves * kWave;
constexpr int kRing = 4;               // steps in flight per wavefront
constexpr unsigned kSpinLimit = 1u << 20;  // polls of the generation word (each a memory round trip)

struct PhaseShape {
  int K, N, S, P, R, C, NT, first;  // first: global index of the phase's first step
};
constexpr PhaseShape kPh[4] = {
    {kH, kHq + 2 * kHkv, 2, 7, 24, 4, 1, 0},
    {kHq, kH, 2, 7, 16, 3, 1, 4},
    {kH, kI, 2, 7, 56, 8, 2, 7},
    {kI, kH, 7, 2, 16, 8, 1, 15},
};
constexpr int kSteps = 23;
static_assert(kPh[0].P * kPh[0].C >= kPh[0].R && kPh[1].P * kPh[1].C >= kPh[1].R, "rows covered");
static_assert(kPh[2].P * kPh[2].C >= kPh[2].R && kPh[3].P * kPh[3].C >= kPh[3].R, "rows covered");
static_assert(kPh[0].R * kWG >= kPh[0].N && kPh[1].R * kWG >= kPh[1].N, "grid covers the rows");
static_assert(kPh[2].R * kWG >= kPh[2].N && kPh[3].R * kWG >= kPh[3].N, "grid covers the rows");
static_assert(kPh[0].S * kPh[0].P == kWaves && kPh[3].S * kPh[3].P == kWaves, "every wave has a slice");
static_assert(kPh[3].first + kPh[3].C == kSteps, "step numbering");

constexpr int phase_of(int step) { return step < 4 ? 0 : (step < 7 ? 1 : (step < 15 ? 2 : 3)); }

// barrier words, 128 bytes apart: per-XCD arrival counts, the cross-XCD
// count, the generation and the error flag
constexpr int kBarXcdStride = 32;
constexpr int kBarGlobal = 8 * kBarXcdStride;
constexpr int kBarGen = kBarGlobal + kBarXcdStride;
constexpr int kBarErr = kBarGen + kBarXcdStride;
static_assert(kBarErr == kLayerBarrierErrWord && kBarErr < (int)kLayerBarrierWords, "barrier word layout");

constexpr uint32_t kOobOff = 0x80000000u;  // an offset past every buffer here

__device__ __forceinline__ unsigned ld_agent(const unsigned* p) {
  return __hip_atomic_load(const_cast<unsigned*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Activations that cross workgroups inside the launch (attention output,
// residual stream, SwiGLU activation) are written and read at agent scope, so
// no XCD's L2 serves a stale copy of a line other XCDs wrote parts of.
__device__ __forceinline__ void st_agent(__half* p, __half v) {
  __hip_atomic_store(reinterpret_cast<unsigned short*>(p), __half_as_ushort(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent_h(const __half* p) {
  const unsigned short u = __hip_atomic_load(reinterpret_cast<unsigned short*>(const_cast<__half*>(p)),
                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return __half2float(__ushort_as_half(u));
}

// Grid barrier: every thread's agent-scope stores complete (workgroup
// barrier), one thread arrives (per XCD, then across XCDs; the last arrival
// advances the generation), waits for the generation to change (bounded) and
// acquires.  The counts are reset by their last arrival, ready for the next.
__device__ __forceinline__ void grid_sync(unsigned* bar) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned nb = gridDim.x, x = blockIdx.x & 7u;
    const unsigned nx = (nb + 7u - x) / 8u, nxcd = nb < 8u ? nb : 8u;
    const unsigned gen0 = ld_agent(bar + kBarGen);
    if (__hip_atomic_fetch_add(bar + x * kBarXcdStride, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nx - 1u) {
      __hip_atomic_store(bar + x * kBarXcdStride, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (__hip_atomic_fetch_add(bar + kBarGlobal, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nxcd - 1u) {
        __hip_atomic_store(bar + kBarGlobal, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(bar + kBarGen, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    unsigned n = 0;
    while (ld_agent(bar + kBarGen) == gen0) {
      if (++n == kSpinLimit) {
        __hip_atomic_store(bar + kBarErr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_of(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

struct Ld {
  u32x4_g c[2];
  uint32_t s[2];
};

struct Weights {
  const uint8_t* codes[kLayerTensors];
  const uint16_t* scales[kLayerTensors];
};

// Issue the loads of global step `step` of this wavefront (compile-time after
// unrolling).  Rows past the workgroup's block or the phase read zeros.
__device__ __forceinline__ void issue(Ld& b, int step, const Weights& W, int wg, int wave, int lane) {
  if (step >= kSteps) return;
  const int ph = phase_of(step);
  const PhaseShape& P = kPh[ph];
  const int i = step - P.first;
  const int s = wave % P.S, p = wave / P.S;
  const int G = P.K / kGroup, g = 64 * s + lane;
  const int local = p + P.P * i;
  int row = wg * P.R + local;
  const bool ok = local < P.R && row < P.N && g < G;
  // the tensor: constant per phase, except q / k / v by row (a select between
  // fixed fields, never a run-time index into the argument aggregate)
  const uint8_t* codes[2];
  const uint16_t* scales[2];
  int n_rows = P.N;
  if (ph == 0) {
    const bool q = row < kHq, k = !q && row < kHq + kHkv;
    codes[0] = q ? W.codes[kQ] : (k ? W.codes[kK] : W.codes[kV]);
    scales[0] = q ? W.scales[kQ] : (k ? W.scales[kK] : W.scales[kV]);
    row -= q ? 0 : (k ? kHq : kHq + kHkv);
    n_rows = q ? kHq : kHkv;
  } else if (ph == 1) {
    codes[0] = W.codes[kO];
    scales[0] = W.scales[kO];
  } else if (ph == 2) {
    codes[0] = W.codes[kGate];
    scales[0] = W.scales[kGate];
    codes[1] = W.codes[kUp];
    scales[1] = W.scales[kUp];
  } else {
    codes[0] = W.codes[kDown];
    scales[0] = W.scales[kDown];
  }
  row = __builtin_amdgcn_readfirstlane(row);
  n_rows = __builtin_amdgcn_readfirstlane(n_rows);
  const uint32_t co = ok ? (uint32_t)row * (uint32_t)(P.K / 2) + (uint32_t)g * 16 : kOobOff;
  const uint32_t so = ok ? ((uint32_t)row * (uint32_t)G + (uint32_t)g) * 2 : kOobOff;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (t >= P.NT) break;
    const auto rc = rsrc_of(codes[t], (uint32_t)((size_t)n_rows * P.K / 2));
    const auto rs = rsrc_of(scales[t], (uint32_t)((size_t)n_rows * G * 2));
    b.c[t] = __builtin_bit_cast(u32x4_g, __builtin_amdgcn_raw_buffer_load_b128(rc, co, 0, 2));
    b.s[t] = __builtin_amdgcn_raw_buffer_load_b16(rs, so, 0, 2);
  }
}

// Stage a phase's K-wide input in LDS ([group][16 pairs + correction]) and
// return the RMS-norm factor (norm) or 1; the input was written by other
// workgroups before the last barrier.
__device__ __forceinline__ float stage(uint32_t* xs, float* sq_wave, const __half* x, int K, bool norm, float eps) {
  const int G = K / kGroup, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float sq = 0.f;
  for (int c = threadIdx.x; c < G; c += kThreads) {
    const unsigned* src = reinterpret_cast<const unsigned*>(x + (size_t)c * kGroup);
    unsigned wd[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) wd[i] = ld_agent(src + i);
    XRaw r;
#pragma unroll
    for (int b = 0; b < 4; ++b) r.d[b] = make_uint4(wd[4 * b], wd[4 * b + 1], wd[4 * b + 2], wd[4 * b + 3]);
    XGroup gx;
    prep_x(gx, r, norm, sq);
#pragma unroll
    for (int i = 0; i < 16; ++i) xs[c * 17 + i] = gx.p[i];
    xs[c * 17 + 16] = __float_as_uint(gx.corr);
  }
  if (norm) {
    const float t = wave_total(sq);
    if (lane == 0) sq_wave[wave] = t;
  }
  __syncthreads();
  float inv_r = 1.f;
  if (norm) {
    float t = 0.f;
    for (int w = 0; w < kWaves; ++w) t += sq_wave[w];
    inv_r = 1.f / sqrtf(t / (float)K + eps);
  }
  return inv_r;
}

__device__ __forceinline__ void load_xg(XGroup& xg, const uint32_t* xs, int g, int G) {
  const int c = g < G ? g : 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) xg.p[i] = xs[c * 17 + i];
  xg.corr = __uint_as_float(xs[c * 17 + 16]);
}

// An output is rounded to fp32 and then once to fp16, as the standalone GEMV
// does.  The empty asm keeps the compiler from fusing the last multiply (or
// add) with the conversion into one mixed-precision FMA, whose single
// rounding straight to fp16 differs in rare double-rounding cases.
__device__ __forceinline__ __half to_half(float v) {
  asm volatile("" : "+v"(v));
  return __float2half_rn(v);
}

struct LayerOut {
  __half* h;
  __half* q_out;
  __half* k_out;
  __half* oin;
  __half* hf;
  int head_dim, expand;
  float eps;
};

// One phase: compute its steps (issuing the loads kRing - 1 steps ahead),
// reduce, and let one thread per row apply the epilogue.
template <int PH>
__device__ __forceinline__ void run_phase(Ld (&ring)[kRing], const Weights& W, const LayerOut& o, uint32_t* xs,
                                          float* sq_wave, float* red, int wg, int wave, int lane,
                                          const UnpackMasks& um) {
  constexpr PhaseShape P = kPh[PH];
  constexpr int V = P.NT * P.C <= 4 ? 4 : (P.NT * P.C <= 8 ? 8 : 16);
  static_assert(P.NT * P.C <= V, "one partial per row and tensor");
  const __half* x = PH == 0 ? o.h : (PH == 1 ? o.oin : (PH == 2 ? o.h : o.hf));
  const float inv_r = stage(xs, sq_wave, x, P.K, PH == 0 || PH == 2, o.eps);
  const int s = wave % P.S, p = wave / P.S;
  const int G = P.K / kGroup, g = 64 * s + lane;
  XGroup xg;
  load_xg(xg, xs, g, G);
  float part[V];
#pragma unroll
  for (int i = 0; i < V; ++i) part[i] = 0.f;
#pragma unroll
  for (int i = 0; i < P.C; ++i) {
    const int step = P.first + i;
    issue(ring[(step + kRing - 1) % kRing], step + kRing - 1, W, wg, wave, lane);
    const Ld& cur = ring[step % kRing];
#pragma unroll
    for (int t = 0; t < P.NT; ++t) {
      const float sc = g < G ? __half2float(__ushort_as_half((uint16_t)cur.s[t])) : 0.f;
      const uint4 cw = make_uint4(cur.c[t].x, cur.c[t].y, cur.c[t].z, cur.c[t].w);
      part[t * P.C + i] = sc * group_dot_m(cw, xg, um);
    }
  }
  transpose_reduce<V>(part);
  if ((lane & 15) == 0) {
    const int rr = lane >> 4;
#pragma unroll
    for (int i = 0; i < V / 4; ++i) red[(s * P.P + p) * V + i + (V / 4) * (rr & 1) + (V / 2) * (rr >> 1)] = part[i];
  }
  __syncthreads();
  const int tid = threadIdx.x;
  if (tid < P.P * P.C) {
    const int pp = tid % P.P, i = tid / P.P;
    const int local = pp + P.P * i;
    const int row = wg * P.R + local;
    if (local < P.R && row < P.N) {
      float a[2];
#pragma unroll
      for (int t = 0; t < P.NT; ++t) {
        float sum = 0.f;
        for (int ss = 0; ss < P.S; ++ss) sum += red[(ss * P.P + pp) * V + t * P.C + i];
        a[t] = sum * inv_r;
      }
      if (PH == 0) {
        const __half v = to_half(a[0]);
        if (row < kHq) {
          o.q_out[row] = v;
        } else if (row < kHq + kHkv) {
          o.k_out[row - kHq] = v;
        } else {
          // context-length-1 attention: every query head of the group takes v
          const int rv = row - kHq - kHkv, jh = rv / o.head_dim, d = rv % o.head_dim;
          for (int e = 0; e < o.expand; ++e) st_agent(o.oin + (size_t)(jh * o.expand + e) * o.head_dim + d, v);
        }
      } else if (PH == 2) {
        st_agent(o.hf + row, to_half(silu_f(a[0]) * a[1]));
      } else {  // o and down: residual
        st_agent(o.h + row, to_half(a[0] + ld_agent_h(o.h + row)));
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void decode_layer_kernel(Weights W, LayerOut o, unsigned* __restrict__ bar) {
  __shared__ __attribute__((aligned(16))) uint32_t xs[(kI / kGroup) * 17];
  __shared__ float sq_wave[kWaves];
  __shared__ float red[kWaves * 16];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int wg = blockIdx.x;
  const UnpackMasks um = unpack_masks();
  Ld ring[kRing];
#pragma unroll
  for (int d = 0; d < kRing - 1; ++d) issue(ring[d], d, W, wg, wave, lane);
  run_phase<0>(ring, W, o, xs, sq_wave, red, wg, wave, lane, um);
  grid_sync(bar);
  run_phase<1>(ring, W, o, xs, sq_wave, red, wg, wave, lane, um);
  grid_sync(bar);
  run_phase<2>(ring, W, o, xs, sq_wave, red, wg, wave, lane, um);
  grid_sync(bar);
  run_phase<3>(ring, W, o, xs, sq_wave, red, wg, wave, lane, um);
}

}  // namespace

hipError_t launch_decode_layer(LayerArgs a, hipStream_t st) {
  if (a.H != kH || a.Hq != kHq || a.Hkv != kHkv || a.I != kI || a.head_dim < 1 || kHkv % a.head_dim ||
      a.expand < 1 || a.expand * kHkv != kHq)
    return hipErrorInvalidConfiguration;
  for (int t = 0; t < kLayerTensors; ++t) {
    const int K = t == kO ? kHq : (t == kDown ? kI : kH);
    const int N = t == kQ ? kHq : (t == kK || t == kV ? kHkv : (t == kDown || t == kO ? kH : kI));
    if (a.w[t].K != K || a.w[t].N != N || !a.w[t].codes || !a.w[t].scales) return hipErrorInvalidConfiguration;
  }
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_layer_kernel, kThreads, 0);
  if (e != hipSuccess) return e;
  if (cus != kWG || per_cu < 1) return hipErrorInvalidConfiguration;
  Weights W{};
  for (int t = 0; t < kLayerTensors; ++t) {
    W.codes[t] = a.w[t].codes;
    W.scales[t] = a.w[t].scales;
  }
  LayerOut o{a.h, a.q_out, a.k_out, a.oin, a.hf, a.head_dim, a.expand, a.eps};
  hipLaunchKernelGGL(decode_layer_kernel, dim3(kWG), dim3(kThreads), 0, st, W, o, a.bar);
  return hipGetLastError();
}

}  // namespace atsi
