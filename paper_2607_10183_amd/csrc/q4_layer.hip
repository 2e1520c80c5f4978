// Fused decode step of one dense decoder layer (batch 1) in a single
// cooperative launch.
//
// At batch 1 the layer is four dependent GEMVs over 122.7 MB of weights
// (8B-shaped layer): q, k, v = rms(h) [Wq Wk Wv]; h += attn Wo;
// f = silu(rms(h) Wg) * (rms(h) Wu); h += f Wd.  Issued as four launches,
// each one pays the ramp-up and drain of a short HBM-bound kernel.  Here one
// persistent grid walks all four phases with grid-wide barriers between
// them, and since weights do not depend on activations, every wavefront
// keeps loading the next weights across a barrier: HBM stays busy while the
// grid synchronises and restages its input.
//
// Work layout: phase p has nrows[p] output rows; wavefront w owns rows
// [w * rpw[p], (w + 1) * rpw[p]).  A wavefront step is one 64-group chunk of
// one row of one tensor: lane l loads the 16 code bytes and the scale of
// group 64 c + l, exactly the lane/group assignment and summation order of
// the standalone GEMV, so both paths give bit-identical outputs.  Each
// wavefront first writes the table of its steps (addresses and what to do
// after each) into LDS, all 64 lanes at once; the main loop then only reads
// the table.  Steps flow through a ring of D register buffers: the load of
// step s + D is issued as soon as step s has been computed, regardless of
// phase boundaries.  Every wavefront has the same number of steps per phase
// (rows past the end are loaded and discarded), so barriers are uniform.
//
// Activations that cross workgroups inside the kernel (attention output,
// residual stream, SwiGLU activation) are written and read with agent-scope
// coherent accesses, so the barrier needs no L2 writeback or invalidation;
// the barrier itself counts arrivals per XCD, then across XCDs, and resets
// its counters for the next use.  Every wait in it is bounded: a barrier
// that does not complete sets an error flag and lets the kernel finish.
#include "layer.h"
#include "q4_gemv_core.h"

namespace atsi {
namespace {

using namespace gemv;

constexpr int kWaves = kBlock / kWave;
constexpr int kRing = 8;             // steps in flight per wavefront
constexpr int kResidMax = 1024;      // residual inputs a workgroup stages per phase
constexpr unsigned kSpinLimit = 1u << 22;

// One step: where lane 0 reads (the lane adds 16 B per lane, clamped to the
// valid lanes), and what the compute side does with it.
struct Step {
  const uint8_t* codes;
  const uint16_t* scales;
  int row;     // output row of the phase, -1 for a discarded row
  int xv;      // first group (bits 0-19) | valid lanes - 1 (bits 20-25)
  int flags;   // bit 0: second tensor of the row, 1: last step of the row,
               // 2: first step of its phase, 4-5: phase
  int pad;
};
static_assert(sizeof(Step) == 32, "step table entries are 32 bytes");

// barrier words, 128 bytes apart: per-XCD arrival counts, the cross-XCD
// count, the generation and the error flag
constexpr int kBarXcdStride = 32;
constexpr int kBarGlobal = 8 * kBarXcdStride;
constexpr int kBarGen = kBarGlobal + kBarXcdStride;
constexpr int kBarErr = kBarGen + kBarXcdStride;

__device__ __forceinline__ unsigned ld_coh(const unsigned* p) {
  return __hip_atomic_load(const_cast<unsigned*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(__half* p, __half v) {
  __hip_atomic_store(reinterpret_cast<unsigned short*>(p), __half_as_ushort(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coh_f(const __half* p) {
  const unsigned short u = __hip_atomic_load(reinterpret_cast<unsigned short*>(const_cast<__half*>(p)),
                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return __half2float(__ushort_as_half(u));
}

// Grid barrier.  Every wave first waits for its own stores to complete; then
// one thread per workgroup arrives.
__device__ __forceinline__ void grid_barrier(unsigned* bar) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned nb = gridDim.x, x = blockIdx.x & 7u;
    const unsigned nx = (nb + 7u - x) / 8u, nxcd = nb < 8u ? nb : 8u;
    const unsigned gen0 = ld_coh(bar + kBarGen);
    __builtin_amdgcn_s_waitcnt(0);
    if (__hip_atomic_fetch_add(bar + x * kBarXcdStride, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nx - 1u) {
      __hip_atomic_store(bar + x * kBarXcdStride, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_waitcnt(0);
      if (__hip_atomic_fetch_add(bar + kBarGlobal, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nxcd - 1u) {
        __hip_atomic_store(bar + kBarGlobal, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_s_waitcnt(0);
        __hip_atomic_fetch_add(bar + kBarGen, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    unsigned n = 0;
    while (ld_coh(bar + kBarGen) == gen0) {
      __builtin_amdgcn_s_sleep(1);
      if (++n == kSpinLimit) {
        __hip_atomic_store(bar + kBarErr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
  }
  __syncthreads();
}

// Stage a phase's input (x, K wide) in LDS, permuted to nibble pairs with its
// offset corrections (same layout and arithmetic as the standalone GEMV,
// M = 1), and return the RMS-norm factor (1 without a norm).  x may have been
// written by other workgroups of this launch: it is read coherently.
__device__ __forceinline__ float stage(char* smem, float* red, const __half* __restrict__ x, int K, bool norm,
                                   float eps) {
  const int nch = K / kGroup;
  uint4* xw = reinterpret_cast<uint4*>(smem);
  float* xc = reinterpret_cast<float*>(smem + (size_t)4 * nch * 16);
  float sq = 0.f;
  for (int c = threadIdx.x; c < nch; c += kBlock) {
    const unsigned* src = reinterpret_cast<const unsigned*>(x + (size_t)c * kGroup);
    unsigned w[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) w[i] = ld_coh(src + i);
    XRaw r;
#pragma unroll
    for (int b = 0; b < 4; ++b) r.d[b] = make_uint4(w[4 * b], w[4 * b + 1], w[4 * b + 2], w[4 * b + 3]);
    XGroup g;
    prep_x(g, r, norm, sq);
#pragma unroll
    for (int b = 0; b < 4; ++b)
      xw[(size_t)b * nch + c] = make_uint4(g.p[4 * b], g.p[4 * b + 1], g.p[4 * b + 2], g.p[4 * b + 3]);
    xc[c] = g.corr;
  }
  float inv_r = 1.f;
  if (norm) {
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const float v = wave_sum(sq);
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t += red[w];
    inv_r = 1.f / sqrtf(t / (float)K + eps);
  }
  __syncthreads();
  return inv_r;
}

// The kernel takes scalar arguments and its helpers take scalars by value:
// choosing between fields of an aggregate with a run-time index makes the
// compiler read the aggregate from computed addresses, which puts it in
// scratch memory (whose accesses would queue behind the weight loads).
#define LAYER_W                                                                                                   \
  const uint8_t *__restrict__ qc, const uint16_t *__restrict__ qs, const uint8_t *__restrict__ kc,                \
      const uint16_t *__restrict__ ks, const uint8_t *__restrict__ vc, const uint16_t *__restrict__ vs,           \
      const uint8_t *__restrict__ oc, const uint16_t *__restrict__ os, const uint8_t *__restrict__ gc,            \
      const uint16_t *__restrict__ gs, const uint8_t *__restrict__ uc, const uint16_t *__restrict__ us,           \
      const uint8_t *__restrict__ dc, const uint16_t *__restrict__ ds
#define LAYER_W_ARGS qc, qs, kc, ks, vc, vs, oc, os, gc, gs, uc, us, dc, ds
#define LAYER_DIMS int H, int Hq, int Hkv, int I, int rpw0, int rpw1, int rpw2, int rpw3
#define LAYER_DIMS_ARGS H, Hq, Hkv, I, rpw0, rpw1, rpw2, rpw3

// Table entries per wavefront: the loop runs whole rounds of kRing steps and
// each step also reads the entry kRing ahead.
__host__ __device__ constexpr int table_steps(int total) { return (total + kRing - 1) / kRing * kRing + kRing; }

// 64-group chunks per row of a K-wide input
__device__ __forceinline__ int chunks(int K) { return (K / kGroup + kWave - 1) / kWave; }

// Table entry of step s of wavefront gw (computed by one lane).
__device__ __forceinline__ Step make_step(int gw, int s, int total, LAYER_W, LAYER_DIMS) {
  if (s >= total) s = total - 1;  // loads past the end repeat the last one
  const int n0 = rpw0 * chunks(H), n1 = rpw1 * chunks(Hq), n2 = rpw2 * 2 * chunks(H);
  const int p = s < n0 ? 0 : (s < n0 + n1 ? 1 : (s < n0 + n1 + n2 ? 2 : 3));
  const int base = p == 0 ? 0 : (p == 1 ? n0 : (p == 2 ? n0 + n1 : n0 + n1 + n2));
  const int K = p == 1 ? Hq : (p == 3 ? I : H);
  const int T = p == 2 ? 2 : 1;
  const int C = chunks(K);
  const int rpw = p == 0 ? rpw0 : (p == 1 ? rpw1 : (p == 2 ? rpw2 : rpw3));
  const int nrows = p == 0 ? Hq + 2 * Hkv : (p == 2 ? I : H);
  const int local = s - base;
  const int j = local / (T * C), rem = local % (T * C);
  const int c = rem / T, t = rem % T;
  const int out_row = gw * rpw + j;
  int row = out_row < nrows ? out_row : nrows - 1;
  const uint8_t* codes;
  const uint16_t* scales;
  if (p == 0) {
    if (row < Hq) {
      codes = qc; scales = qs;
    } else if (row < Hq + Hkv) {
      codes = kc; scales = ks; row -= Hq;
    } else {
      codes = vc; scales = vs; row -= Hq + Hkv;
    }
  } else if (p == 1) {
    codes = oc; scales = os;
  } else if (p == 2) {
    codes = t ? uc : gc; scales = t ? us : gs;
  } else {
    codes = dc; scales = ds;
  }
  const int nch = K / kGroup, g0 = c * kWave;
  const int valid = nch - g0 < kWave ? nch - g0 : kWave;
  Step st;
  st.codes = codes + (size_t)row * (K / 2) + (size_t)g0 * 16;
  st.scales = scales + (size_t)row * nch + g0;
  st.row = out_row < nrows ? out_row : -1;
  st.xv = g0 | ((valid - 1) << 20);
  st.flags = t | ((c == C - 1 && t == T - 1) << 1) | ((local == 0 && p > 0) << 2) | (p << 4);
  st.pad = 0;
  return st;
}

struct Buf {
  uint4 c;
  uint16_t s;
};

__device__ __forceinline__ void load_step(Buf& b, const Step* tab, int s, int lane) {
  const uint4* e = reinterpret_cast<const uint4*>(tab + s);
  const uint4 e0 = e[0], e1 = e[1];
  // readfirstlane returns int: widen the low words as unsigned
  const uint64_t cp = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane(e0.y) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane(e0.x);
  const uint64_t sp = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane(e0.w) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane(e0.z);
  const int vmax = __builtin_amdgcn_readfirstlane(e1.y) >> 20;
  const int l = lane < vmax ? lane : vmax;
  // global address space: a generic (flat) load would also count against the
  // LDS wait counter, so every LDS wait would drain the weight ring
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = reinterpret_cast<const __attribute__((address_space(1))) u32x4*>(cp)[l];
  b.c = make_uint4(v.x, v.y, v.z, v.w);
  b.s = reinterpret_cast<const __attribute__((address_space(1))) uint16_t*>(sp)[l];
}

__global__ __launch_bounds__(kBlock) void decode_layer_kernel(LAYER_W, __half* __restrict__ h,
                                                              __half* __restrict__ q_out, __half* __restrict__ k_out,
                                                              __half* __restrict__ oin, __half* __restrict__ hf,
                                                              unsigned* __restrict__ bar, int head_dim, int expand,
                                                              float eps, int xmax, int total, LAYER_DIMS) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ float red[kWaves];
  // residual inputs of the workgroup's rows, read before the phase starts so
  // that no global load (whose wait would drain the weight ring) sits in the
  // row epilogue
  __shared__ float resid[kResidMax];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int gw = blockIdx.x * kWaves + wave;
  const int xbytes = xmax / kGroup * 68;
  const int ntab = table_steps(total);
  Step* tab = reinterpret_cast<Step*>(smem + xbytes) + wave * ntab;

  for (int s = lane; s < ntab; s += kWave) tab[s] = make_step(gw, s, total, LAYER_W_ARGS, LAYER_DIMS_ARGS);
  __syncthreads();

  Buf buf[kRing];
#pragma unroll
  for (int d = 0; d < kRing; ++d) load_step(buf[d], tab, d, lane);

  float inv_r = stage(smem, red, h, H, true, eps);
  int nch = H / kGroup;
  const uint4* xw = reinterpret_cast<const uint4*>(smem);
  const float* xc = reinterpret_cast<const float*>(smem + (size_t)4 * nch * 16);
  int rbase = 0;  // first output row of the workgroup in the current phase
  float acc0 = 0.f, acc1 = 0.f;

  for (int i = 0; i < total; i += kRing) {
#pragma unroll
    for (int d = 0; d < kRing; ++d) {
      const int s = i + d;
      if (s < total) {
        const uint4 m = reinterpret_cast<const uint4*>(tab + s)[1];
        const int row = __builtin_amdgcn_readfirstlane(m.x);
        const int xv = __builtin_amdgcn_readfirstlane(m.y);
        const int flags = __builtin_amdgcn_readfirstlane(m.z);
        const int p = flags >> 4;
        if (flags & 4) {
          // first step of a phase: every row of the previous one is written
          grid_barrier(bar);
          const int K = p == 1 ? Hq : (p == 3 ? I : H);
          const int rpw = p == 1 ? rpw1 : (p == 3 ? rpw3 : rpw2);
          rbase = blockIdx.x * kWaves * rpw;
          if (p != 2) {
            const int nr = kWaves * rpw;
            for (int t = threadIdx.x; t < nr; t += kBlock) resid[t] = rbase + t < H ? ld_coh_f(h + rbase + t) : 0.f;
          }
          inv_r = stage(smem, red, p == 1 ? oin : (p == 2 ? h : hf), K, p == 2, eps);
          nch = K / kGroup;
          xc = reinterpret_cast<const float*>(smem + (size_t)4 * nch * 16);
        }
        const int g0 = xv & 0xFFFFF, vmax = xv >> 20;
        const bool ok = lane <= vmax;
        const int gg = g0 + (ok ? lane : vmax);
        XGroup xg;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const uint4 v = xw[(size_t)b * nch + gg];
          xg.p[4 * b] = v.x;
          xg.p[4 * b + 1] = v.y;
          xg.p[4 * b + 2] = v.z;
          xg.p[4 * b + 3] = v.w;
        }
        xg.corr = xc[gg];
        const float sc = ok ? __half2float(__ushort_as_half(buf[d].s)) : 0.f;
        if (flags & 1)
          acc1 = fmaf(sc, group_dot(buf[d].c, xg), acc1);
        else
          acc0 = fmaf(sc, group_dot(buf[d].c, xg), acc0);
        if (flags & 2) {
          // one store instruction per row (lanes pick the copies), so that
          // the number of memory operations behind each weight load is fixed
          const float v = wave_sum(acc0) * inv_r;
          const float u = p == 2 ? wave_sum(acc1) * inv_r : 0.f;
          if (row >= 0) {
            if (p == 0) {
              const __half o = __float2half_rn(v);
              if (row < Hq) {
                if (lane == 0) q_out[row] = o;
              } else if (row < Hq + Hkv) {
                if (lane == 0) k_out[row - Hq] = o;
              } else {
                // context-length-1 attention: each query head of the group takes v
                const int rv = row - Hq - Hkv, jh = rv / head_dim, dd = rv % head_dim;
                if (lane < expand) st_coh(oin + (size_t)(jh * expand + lane) * head_dim + dd, o);
              }
            } else if (p == 2) {
              if (lane == 0) st_coh(hf + row, __float2half_rn(silu_f(v) * u));
            } else {  // o and down: residual
              if (lane == 0) st_coh(h + row, __float2half_rn(v + resid[row - rbase]));
            }
          }
          acc0 = acc1 = 0.f;
        }
      }
      load_step(buf[d], tab, s + kRing, lane);
    }
  }
}

}  // namespace

size_t decode_layer_lds(const LayerArgs& a, int total) {
  int kmax = a.H > a.Hq ? a.H : a.Hq;
  kmax = kmax > a.I ? kmax : a.I;
  return (size_t)(kmax / kGroup) * 68 + (size_t)kWaves * table_steps(total) * sizeof(Step);
}

hipError_t launch_decode_layer(LayerArgs a, hipStream_t st) {
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  int xmax = a.H > a.Hq ? a.H : a.Hq;
  xmax = xmax > a.I ? xmax : a.I;
  // two workgroups per CU, or one if two do not fit
  for (int per = 2; per >= 1; --per) {
    const int grid = cus * per;
    const int waves = grid * kWaves;
    const int rows[kLayerPhases] = {a.Hq + 2 * a.Hkv, a.H, a.I, a.H};
    const int Ks[kLayerPhases] = {a.H, a.Hq, a.H, a.I};
    int total = 0;
    for (int p = 0; p < kLayerPhases; ++p) {
      a.rpw[p] = (rows[p] + waves - 1) / waves;
      total += a.rpw[p] * (p == 2 ? 2 : 1) * ((Ks[p] / kGroup + kWave - 1) / kWave);
    }
    if (kWaves * a.rpw[1] > kResidMax || kWaves * a.rpw[3] > kResidMax) continue;
    const size_t lds = decode_layer_lds(a, total);
    if (lds > kLayerMaxLds) continue;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_layer_kernel, kBlock, lds);
    if (e != hipSuccess) return e;
    if (per_cu < per) continue;
    QView* w = a.w;
    void* args[] = {&w[kQ].codes,    &w[kQ].scales,   &w[kK].codes,    &w[kK].scales, &w[kV].codes,
                    &w[kV].scales,   &w[kO].codes,    &w[kO].scales,   &w[kGate].codes, &w[kGate].scales,
                    &w[kUp].codes,   &w[kUp].scales,  &w[kDown].codes, &w[kDown].scales, &a.h,
                    &a.q_out,        &a.k_out,        &a.oin,          &a.hf,          &a.bar,
                    &a.head_dim,     &a.expand,       &a.eps,          &xmax,          &total,
                    &a.H,            &a.Hq,           &a.Hkv,          &a.I,           &a.rpw[0],
                    &a.rpw[1],       &a.rpw[2],       &a.rpw[3]};
    e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(decode_layer_kernel), dim3(grid), dim3(kBlock), args,
                                   (unsigned)lds, st);
    if (e != hipSuccess) return e;
    return hipGetLastError();
  }
  return hipErrorInvalidConfiguration;
}

}  // namespace atsi
