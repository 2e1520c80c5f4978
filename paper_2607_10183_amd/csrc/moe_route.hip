// MoE routing on CDNA4: router logits, top-k selection with renormalised
// softmax weights, and deterministic token-to-expert bucketing.
//
// The paper moves a MoE layer's expert weights only after routing is known
// and only for the experts the current tokens selected (Sec. 4.2.2; Sec.
// 4.4.1 counts only activated experts); these kernels produce that routing.
//
//   router_partial  logits of a 16-token tile for all experts over one K
//                   slice, on 16x16x32 fp16 MFMAs; the router slice is staged
//                   through LDS transposed so each lane reads 8 consecutive
//                   inputs of one expert; fp32 partials per slice.
//                   A launch of at most 16 tokens routes them in its last
//                   workgroup to finish (partials stored and loaded at agent
//                   scope around a counter that the last one resets), and
//                   computes the tokens' RMS-norm factors there when asked,
//                   from sums of squares each slice's workgroup leaves beside
//                   its partials; that workgroup's 256 threads fetch every
//                   partial in one round of loads.
//   router_topk     one wavefront per token: sums the K-slice partials in a
//                   fixed order, adds the bias, selects the top k by (logit
//                   descending, expert id ascending) with a pruned bitonic
//                   network over 64-bit keys (DPP and permlane swaps, no
//                   data-dependent branches), and writes the softmax over the
//                   selected logits.
//   bucket          one workgroup: per-expert counts (LDS integer atomics),
//                   exclusive scan, then a stable scatter of pair ids k*t + j
//                   ordered by (expert, token): each 64-token chunk builds a
//                   64-bit token mask per expert, a pair's rank is the
//                   popcount of the lower lanes' bits plus the counts of the
//                   earlier chunks.  Results do not depend on atomics order.
//                   Also ranks experts heavy-first and lists the row tiles of
//                   the HBM-resident experts for the grouped expert GEMM.
#include "moe.h"

namespace atsi {
namespace {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kRT = 16;  // tokens per router tile

// The partials of a fused launch cross workgroups on other XCDs: they are
// stored and loaded at agent scope, so no XCD's L2 keeps or serves a stale
// copy of them and no workgroup has to write back or invalidate its L2.
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// sum of squares of row t over the wave: each lane adds its 8-input chunks
// lane, lane + 64, ... in order; up to 8 chunks per lane are loaded in one
// round (chunks past H count as zeros, which leaves the sums unchanged)
__device__ __forceinline__ float row_sumsq(const __half* __restrict__ x, int t, int H) {
  const int lane = threadIdx.x & 63;
  const __half* xr = x + (size_t)t * H;
  float q = 0.f;
  for (int c0 = 0; c0 < H; c0 += 64 * 8 * 8) {
    uint4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = c0 + (j * 64 + lane) * 8;
      v[j] = c < H ? *reinterpret_cast<const uint4*>(xr + c) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const __half* hv = reinterpret_cast<const __half*>(&v[j]);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float f = __half2float(hv[i]);
        q = fmaf(f, f, q);
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
  return q;
}

// 1 / sqrt(mean(x[t]^2) + eps) for one token, computed by one wavefront and
// returned to every lane (the same arithmetic for every caller)
__device__ __forceinline__ float token_inv_rms(const __half* __restrict__ x, int t, int H, float eps) {
  return 1.f / sqrtf(row_sumsq(x, t, H) / (float)H + eps);
}

// Top k of one token's logits by (value descending, expert id ascending), by
// one wavefront holding experts lane and lane + 64 (-inf past E).  Each
// candidate is a 64-bit key, larger is better: the logit's bits mapped to an
// unsigned order in the high word (-0 taken as +0), the complement of the
// expert id in the low word.  A pruned bitonic network finds the top C (C = 8
// for k <= 8, else 16) without data-dependent branches: both registers sort
// their C-lane chunks descending; the elementwise maximum of a descending and
// an ascending chunk holds the top C of the two and is bitonic, so one merge
// sorts it; pairing each lane's two keys, then chunks across mirror distances
// 2C - 1 (up to 63) leaves the top C sorted in lanes 0 .. C - 1.  Lanes j < k
// write the ids and the softmax over the selected logits (normaliser summed
// in rank order).
__device__ __forceinline__ uint64_t topk_key(float v, int id) {
  unsigned u = __float_as_uint(v + 0.f);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (unsigned)~id;
}

template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t x) {
  const unsigned lo = (unsigned)__builtin_amdgcn_update_dpp(0, (int)(unsigned)x, CTRL, 0xF, 0xF, false);
  const unsigned hi = (unsigned)__builtin_amdgcn_update_dpp(0, (int)(unsigned)(x >> 32), CTRL, 0xF, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}

// the key of lane l ^ 16 (W = 16) or l ^ 32 (W = 32): the swap of a register
// with itself returns the lane's own word and its partner's; the partner's is
// the second result where l & W is 0, else the first
template <int W>
__device__ __forceinline__ uint64_t swap64(uint64_t x, int lane) {
  const unsigned lo = (unsigned)x, hi = (unsigned)(x >> 32);
  unsigned plo, phi;
  if constexpr (W == 16) {
    const auto a = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto b = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    plo = (lane & 16) ? a[0] : a[1];
    phi = (lane & 16) ? b[0] : b[1];
  } else {
    const auto a = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
    plo = (lane & 32) ? a[0] : a[1];
    phi = (lane & 32) ? b[0] : b[1];
  }
  return ((uint64_t)phi << 32) | plo;
}

// the key of lane l ^ J
template <int J>
__device__ __forceinline__ uint64_t lane_xor(uint64_t x, int lane) {
  if constexpr (J == 1) return dpp64<0xB1>(x);                  // quad_perm 1,0,3,2
  else if constexpr (J == 2) return dpp64<0x4E>(x);             // quad_perm 2,3,0,1
  else if constexpr (J == 3) return dpp64<0x1B>(x);             // quad_perm 3,2,1,0
  else if constexpr (J == 7) return dpp64<0x141>(x);            // row_half_mirror
  else if constexpr (J == 15) return dpp64<0x140>(x);           // row_mirror
  else if constexpr (J == 4) return dpp64<0x1B>(dpp64<0x141>(x));  // (l ^ 7) ^ 3
  else if constexpr (J == 8) return dpp64<0x141>(dpp64<0x140>(x));  // (l ^ 15) ^ 7
  else if constexpr (J == 31) return swap64<16>(dpp64<0x140>(x), lane);
  else if constexpr (J == 63) return swap64<32>(swap64<16>(dpp64<0x140>(x), lane), lane);
  else static_assert(J == 1, "no cross-lane path for this distance");
}

// compare-exchange with lane l ^ J: the lane keeps the larger key iff
// (l & D) == 0
template <int J, int D>
__device__ __forceinline__ uint64_t cx(uint64_t x, int lane) {
  const uint64_t p = lane_xor<J>(x, lane);
  return ((p > x) == ((lane & D) == 0)) ? p : x;
}

template <int J>
__device__ __forceinline__ uint64_t kmax(uint64_t x, int lane) {
  const uint64_t p = lane_xor<J>(x, lane);
  return p > x ? p : x;
}

// sorts a bitonic C-lane chunk descending (half-cleaners C/2 .. 1)
template <int C>
__device__ __forceinline__ uint64_t bitonic_merge(uint64_t x, int lane) {
  if constexpr (C >= 16) x = cx<8, 8>(x, lane);
  if constexpr (C >= 8) x = cx<4, 4>(x, lane);
  x = cx<2, 2>(x, lane);
  return cx<1, 1>(x, lane);
}

// sorts each C-lane chunk descending: stage s compares mirror partners
// (l ^ (s - 1)), then merges the halves
template <int C>
__device__ __forceinline__ uint64_t chunk_sort(uint64_t x, int lane) {
  x = cx<1, 1>(x, lane);
  x = cx<3, 2>(x, lane);
  x = cx<1, 1>(x, lane);
  x = cx<7, 4>(x, lane);
  x = bitonic_merge<4>(x, lane);
  if constexpr (C == 16) {
    x = cx<15, 8>(x, lane);
    x = bitonic_merge<8>(x, lane);
  }
  return x;
}

template <int C>
__device__ __forceinline__ uint64_t topk_network(uint64_t a, uint64_t b, int lane) {
  a = chunk_sort<C>(a, lane);
  b = chunk_sort<C>(b, lane);
  // lane's two chunks: a descending against b mirrored (ascending)
  const uint64_t bm = lane_xor<C - 1>(b, lane);
  a = a > bm ? a : bm;
  a = bitonic_merge<C>(a, lane);
  if constexpr (C == 8) {
    a = bitonic_merge<8>(kmax<15>(a, lane), lane);
  }
  a = bitonic_merge<C>(kmax<31>(a, lane), lane);
  return bitonic_merge<C>(kmax<63>(a, lane), lane);
}

__device__ __forceinline__ void select_topk(float v0, float v1, int E, int k, int t, int32_t* __restrict__ idx,
                                            float* __restrict__ p) {
  const int lane = threadIdx.x & 63;
  const uint64_t a = lane < E ? topk_key(v0, lane) : 0ull;
  const uint64_t b = lane + 64 < E ? topk_key(v1, lane + 64) : 0ull;
  const uint64_t key = k <= 8 ? topk_network<8>(a, b, lane) : topk_network<16>(a, b, lane);
  const unsigned hi = (unsigned)(key >> 32);
  const float v = __uint_as_float((hi & 0x80000000u) ? (hi & 0x7fffffffu) : ~hi);
  const int id = (int)~(unsigned)key;
  const float v_top = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));  // lane 0: rank 0
  const float ev = lane < k ? expf(v - v_top) : 0.f;
  float den = 0.f;
  for (int j = 0; j < k; ++j) den += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ev), j));
  if (lane < k) {
    idx[(size_t)t * k + lane] = id;
    p[(size_t)t * k + lane] = ev / den;
  }
}

// Routing of token t by one wavefront (E <= 128, two candidates per lane):
// the K-slice partial logits summed in slice order, times the norm factor rs
// when norm is set, plus the bias; then the top k and their softmax.
__device__ __forceinline__ void route_token(const float* __restrict__ part, int n_split, int M, int t, bool norm,
                                            float rs, const float* __restrict__ bias, int E, int k,
                                            int32_t* __restrict__ idx, float* __restrict__ p,
                                            float* __restrict__ logits_out) {
  const int lane = threadIdx.x & 63;
  float v[2] = {0.f, 0.f};
  const int id[2] = {lane, lane + 64};
  // every global load is issued before the first wait: the bias, then the
  // K-slice partials, 16 slices of both experts per round, added in slice
  // order
  float bv[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) bv[h] = (bias && id[h] < E) ? bias[id[h]] : 0.f;
  for (int sp0 = 0; sp0 < n_split; sp0 += 16) {
    float pv[2][16];
#pragma unroll
    for (int j = 0; j < 16; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        pv[h][j] = (sp0 + j < n_split && id[h] < E) ? part[((size_t)(sp0 + j) * M + t) * E + id[h]] : 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (sp0 + j < n_split) v[h] += pv[h][j];
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int e = id[h];
    if (e < E) {
      float s = v[h];
      if (norm) s *= rs;  // RMS-normalised input: scale the product once
      if (bias) s += bv[h];
      v[h] = s;
      if (logits_out) logits_out[(size_t)t * E + e] = s;
    } else {
      v[h] = -INFINITY;
    }
  }
  select_topk(v[0], v[1], E, k, t, idx, p);
}

// Outputs of the routing of one launch: the last workgroup of a single-tile
// launch (FUSED) routes the tile's tokens itself.
struct RouteOut {
  unsigned* counter;        // zero between launches; counts finished workgroups
  const float* inv_r;       // per-token norm factors given by the caller, or null
  float* inv_r_out;         // non-null: compute them here (and write them)
  float eps;
  const float* bias;
  int k;
  int32_t* idx;
  float* p;
  float* logits;
};

constexpr int kChunk = 32;  // partials a thread of the routing workgroup fetches per round

// Routing of a whole tile (at most 16 tokens) by the 256 threads of the last
// workgroup.  Every input is fetched in one round of loads where it fits:
// g threads per (token, expert) each sum a contiguous run of K slices in
// slice order and the g runs are added in order; the squares of the inputs
// (per slice, written by the slices' workgroups) are summed the same way
// for the norm factor.  Then one wavefront per token selects the top k.
// pbuf holds at least 2048 floats.
__device__ void route_tile(const float* __restrict__ part, int n_split, int M, int t0, int H, int E, const RouteOut& ro,
                           float* pbuf) {
  __shared__ float lg[kRT * 128];
  __shared__ float sqb[256];
  __shared__ float rsq[kRT];
  const int tid = threadIdx.x;
  const int Mt = min(kRT, M - t0);
  const int items = Mt * E;
  int g = 1;
  while (2 * g * items <= 256 && 2 * g <= n_split) g *= 2;
  const int chunk = n_split / g;
  const float* sq = part + (size_t)n_split * M * E;  // per-slice sums of squares, [slice][token]
  int g2 = 1;
  while (n_split / g2 > kChunk) g2 *= 2;
  const int chunk2 = n_split / g2;
  const bool make = ro.inv_r_out != nullptr;
  const bool norm = make || ro.inv_r != nullptr;

  // issued first, consumed last: this thread's squares run, its first
  // item's bias and the given norm factors
  // loads are unpredicated (indexes clamped into the run, the extra values
  // dropped when summing) with 32-bit offsets from the launch's base, so
  // they issue back to back
  float qv[kChunk];
  const bool has_q = make && tid < Mt * g2;
  if (has_q) {
    const int t = t0 + tid / g2, s0 = (tid % g2) * chunk2;
#pragma unroll
    for (int j = 0; j < kChunk; ++j) qv[j] = ld_agent(sq + (unsigned)(min(s0 + j, s0 + chunk2 - 1) * M + t));
  }
  const float b0 = (ro.bias && tid < items) ? ro.bias[tid % E] : 0.f;
  if (!make && ro.inv_r && tid < Mt) rsq[tid] = ro.inv_r[t0 + tid];

  const unsigned stride = (unsigned)(M * E);
  for (int w = tid; w < items * g; w += 256) {
    const int item = w / g, sub = w % g;
    const unsigned base = (unsigned)((t0 + item / E) * E + item % E);
    const int end = (sub + 1) * chunk;
    float s = 0.f;
    for (int c0 = sub * chunk; c0 < end; c0 += kChunk) {
      float pv[kChunk];
#pragma unroll
      for (int j = 0; j < kChunk; ++j) pv[j] = ld_agent(part + (base + (unsigned)min(c0 + j, end - 1) * stride));
#pragma unroll
      for (int j = 0; j < kChunk; ++j)
        if (c0 + j < end) s += pv[j];
    }
    pbuf[w] = s;
  }
  if (has_q) {
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < kChunk; ++j)
      if (j < chunk2) q += qv[j];
    sqb[tid] = q;
  }
  __syncthreads();
  if (make && tid < Mt) {
    float q = 0.f;
    for (int j = 0; j < g2; ++j) q += sqb[tid * g2 + j];
    const float rs = 1.f / sqrtf(q / (float)H + ro.eps);
    rsq[tid] = rs;
    ro.inv_r_out[t0 + tid] = rs;
  }
  __syncthreads();
  for (int item = tid; item < items; item += 256) {
    const int tt = item / E, e = item % E;
    float s = 0.f;
    for (int j = 0; j < g; ++j) s += pbuf[item * g + j];
    if (norm) s *= rsq[tt];  // RMS-normalised input: scale the product once
    if (ro.bias) s += item == tid ? b0 : ro.bias[e];
    lg[item] = s;
    if (ro.logits) ro.logits[(size_t)(t0 + tt) * E + e] = s;
  }
  __syncthreads();
  const int lane = tid & 63, wave = tid >> 6;
  for (int tt = wave; tt < Mt; tt += 4) {
    const float v0 = lane < E ? lg[tt * E + lane] : -INFINITY;
    const float v1 = lane + 64 < E ? lg[tt * E + lane + 64] : -INFINITY;
    select_topk(v0, v1, E, ro.k, t0 + tt, ro.idx, ro.p);
  }
}

// grid: (ceil(M/16), n_split); block 256 = 4 waves x 32 experts (E <= 128).
// Requires E % 16 == 0, E <= 128, ks % 32 == 0.  The global loads of the
// next 32-input step are issued before the MFMAs of the current one.
template <bool FUSED>
__global__ __launch_bounds__(256) void router_partial_kernel(const __half* __restrict__ x, const __half* __restrict__ wr,
                                                             int M, int H, int E, int ks, float* __restrict__ part,
                                                             RouteOut ro) {
  __shared__ __attribute__((aligned(16))) _Float16 Bt[128 * (32 + 8)];  // [expert][k] of one 32-k step
  const int t0 = blockIdx.x * kRT;
  const int k_begin = blockIdx.y * ks, k_end = k_begin + ks;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tr = lane & 15, kq = (lane >> 4) * 8;
  // staging roles: k row kk of the step, experts e8 .. e8 + 7 and 64 above
  // (a wave's 2-byte LDS stores then cover 16 consecutive dwords twice,
  // 32 banks apart: no bank conflicts)
  const int kk = threadIdx.x & 31, e8 = (threadIdx.x >> 5) * 8;
  const bool wl = e8 < E, wl2 = e8 + 64 < E;
  const int t = t0 + tr;
  // squares of the slice's inputs, for the norm factors the routing makes
  const bool sq = ro.inv_r_out && wave == 0;
  float4_t acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  float q = 0.f;
  uint4 w0 = {0, 0, 0, 0}, w1 = {0, 0, 0, 0};
  half8_t a = {0, 0, 0, 0, 0, 0, 0, 0};
  auto fetch = [&](int k0) {
    // W_r row k0 + kk, 8 experts from e8 and from e8 + 64; x[t][k0 + kq ..]
    if (wl) w0 = *reinterpret_cast<const uint4*>(wr + (size_t)(k0 + kk) * E + e8);
    if (wl2) w1 = *reinterpret_cast<const uint4*>(wr + (size_t)(k0 + kk) * E + e8 + 64);
    if (t < M) a = *reinterpret_cast<const half8_t*>(x + (size_t)t * H + k0 + kq);
  };
  fetch(k_begin);
  for (int k0 = k_begin; k0 < k_end; k0 += 32) {
    __syncthreads();  // the previous step's reads of Bt are done
    const _Float16* h0 = reinterpret_cast<const _Float16*>(&w0);
    const _Float16* h1 = reinterpret_cast<const _Float16*>(&w1);
    if (wl) {
#pragma unroll
      for (int i = 0; i < 8; ++i) Bt[(e8 + i) * 40 + kk] = h0[i];
    }
    if (wl2) {
#pragma unroll
      for (int i = 0; i < 8; ++i) Bt[(e8 + 64 + i) * 40 + kk] = h1[i];
    }
    const half8_t ac = a;
    if (k0 + 32 < k_end) fetch(k0 + 32);
    __syncthreads();
    if (sq) {
#pragma unroll
      for (int i = 0; i < 8; ++i) q = fmaf((float)ac[i], (float)ac[i], q);
    }
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int e = wave * 32 + nb * 16 + tr;
      if (wave * 32 + nb * 16 < E) {
        const half8_t b = *reinterpret_cast<const half8_t*>(&Bt[e * 40 + kq]);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ac, b, acc[nb], 0, 0, 0);
      }
    }
  }
  // 16x16 D layout: lane l holds column l % 16, rows 4 * (l / 16) + i
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int e = wave * 32 + nb * 16 + (lane & 15);
    if (wave * 32 + nb * 16 >= E) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tt = t0 + 4 * (lane >> 4) + i;
      if (tt < M) {
        float* dst = part + ((size_t)blockIdx.y * M + tt) * E + e;
        if constexpr (FUSED) st_agent(dst, acc[nb][i]); else *dst = acc[nb][i];
      }
    }
  }
  if (sq) {
    // lanes tr, tr + 16, tr + 32, tr + 48 hold token tr's four 8-input groups
    q += __shfl_xor(q, 16, 64);
    q += __shfl_xor(q, 32, 64);
    if (lane < 16 && t < M) {
      float* dst = part + (size_t)gridDim.y * M * E + (size_t)blockIdx.y * M + t;
      if constexpr (FUSED) st_agent(dst, q); else *dst = q;
    }
  }
  if constexpr (FUSED) {
    // The last workgroup to finish routes the tile.  Every thread waits until
    // its agent-scope stores are performed, then one thread counts the
    // workgroup in; the last one resets the count for the next launch and
    // reads the partials back at agent scope.
    __shared__ unsigned ticket;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) ticket = __hip_atomic_fetch_add(ro.counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (ticket != gridDim.y - 1) return;
    if (threadIdx.x == 0) __hip_atomic_store(ro.counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    route_tile(part, gridDim.y, M, t0, H, E, ro, reinterpret_cast<float*>(Bt));
  }
}

// one wave per token; E <= 128 (two candidates per lane)
// With inv_r_out the norm factors come from the partial kernel's per-slice
// sums of squares (summed here over the slices, lane by lane, then across the
// wave) and are written out for the expert launches.
__global__ __launch_bounds__(256) void router_topk_kernel(const float* __restrict__ part, int n_split,
                                                          const float* __restrict__ inv_r, float* __restrict__ inv_r_out,
                                                          int H, float eps, const float* __restrict__ bias, int M,
                                                          int E, int k, int32_t* __restrict__ idx,
                                                          float* __restrict__ p, float* __restrict__ logits_out) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= M) return;
  float rs = 1.f;
  if (inv_r_out) {
    const int lane = threadIdx.x & 63;
    const float* sq = part + (size_t)n_split * M * E;  // [slice][token]
    float q = 0.f;
    for (int s = lane; s < n_split; s += 64) q += sq[(size_t)s * M + t];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
    q = __shfl(q, 0, 64);  // lane 0's sum in every lane: one factor for all experts
    rs = 1.f / sqrtf(q / (float)H + eps);
    if (lane == 0) inv_r_out[t] = rs;
  } else if (inv_r) {
    rs = inv_r[t];
  }
  route_token(part, n_split, M, t, inv_r_out != nullptr || inv_r != nullptr, rs, bias, E, k, idx, p, logits_out);
}

// Single workgroup of 1024 threads.  Up to 16 chunks of 64 tokens are ranked
// per pass; masks live in LDS.
// Exclusive prefix sum of v over experts 0..E-1 (E <= 128) by wave 0: lane l
// owns experts 2l and 2l+1.  Returns the total; out[e] = sum_{f < e} v[f].
__device__ int scan128(const int* v, int* out, int E) {
  const int lane = threadIdx.x & 63;
  int total = 0;
  if (threadIdx.x < 64) {
    const int a = (2 * lane < E) ? v[2 * lane] : 0;
    const int b = (2 * lane + 1 < E) ? v[2 * lane + 1] : 0;
    int incl = a + b;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    const int excl = incl - a - b;
    if (2 * lane < E) out[2 * lane] = excl;
    if (2 * lane + 1 < E) out[2 * lane + 1] = excl + a;
    total = __shfl(incl, 63, 64);
  }
  return total;
}

// Single workgroup of 1024 threads.  Up to 16 chunks of 64 tokens are ranked
// per pass; masks live in LDS.
constexpr int kBucketThreads = 1024;
// up to this many routed pairs the scatter writes perm into LDS and copies it
// out in order (64 KB): scattered 4-byte stores from the one workgroup took
// most of the kernel's time
constexpr int kBucketStage = 16384;
__global__ __launch_bounds__(kBucketThreads) void bucket_kernel(const int32_t* __restrict__ idx, int M, int k, int E,
                                                      const uint8_t* __restrict__ resident, int bm_rows,
                                                      int light_rows, int light_mtmax, int32_t* __restrict__ counts,
                                                      int32_t* __restrict__ offsets, int32_t* __restrict__ perm,
                                                      int32_t* __restrict__ inv_perm, int32_t* __restrict__ order,
                                                      int32_t* __restrict__ tiles, int32_t* __restrict__ n_tiles,
                                                      int32_t* __restrict__ ltiles, int32_t* __restrict__ n_ltiles) {
  __shared__ int cnt[kMaxExperts];
  __shared__ int base[kMaxExperts];
  __shared__ unsigned long long mask[16][kMaxExperts];
  __shared__ int pre[16][kMaxExperts];
  __shared__ int ord[kMaxExperts];
  __shared__ int ntile[kMaxExperts];   // tiles of the expert at rank r
  __shared__ int tstart[kMaxExperts];
  __shared__ int nlt[kMaxExperts];     // light tiles of the expert at rank r
  __shared__ int lstart[kMaxExperts];
  __shared__ int lclass[kLightClasses];
  __shared__ int rpart[8][kMaxExperts];
  extern __shared__ int sperm[];  // perm, staged (pairs <= kBucketStage)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int pairs = M * k;
  const bool stage = pairs <= kBucketStage;
  // inv_perm rows of four pairs go out as one 16-byte store where aligned
  const bool inv4 = (k & 3) == 0 && (reinterpret_cast<uintptr_t>(inv_perm) & 15) == 0;
  for (int e = tid; e < E; e += blockDim.x) cnt[e] = 0;
  __syncthreads();
  // every load of a round of 8 is issued before its first count
  for (int i0 = 0; i0 < pairs; i0 += 8 * kBucketThreads) {
    int ev[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int i = i0 + r * kBucketThreads + tid;
      ev[r] = i < pairs ? idx[i] : -1;
    }
#pragma unroll
    for (int r = 0; r < 8; ++r)
      if ((unsigned)ev[r] < (unsigned)E) atomicAdd(&cnt[ev[r]], 1);
  }
  __syncthreads();
  const int total = scan128(cnt, base, E);
  __syncthreads();
  for (int e = tid; e < E; e += blockDim.x) {
    offsets[e] = base[e];
    counts[e] = cnt[e];
  }
  if (tid == 0) offsets[E] = total;
  // stable scatter, 16 chunks of 64 tokens per pass
  for (int c0 = 0; c0 * 64 < M; c0 += 16) {
    for (int i = tid; i < 16 * E; i += blockDim.x) mask[i / E][i % E] = 0ull;
    __syncthreads();
    const int t = (c0 + wave) * 64 + lane;
    int et[kMaxTopK];  // the token's k experts, loaded once (-1 past k or M)
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) et[j] = (t < M && j < k) ? idx[(size_t)t * k + j] : -1;
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j)
      if ((unsigned)et[j] < (unsigned)E) atomicOr(&mask[wave][et[j]], 1ull << lane);
    __syncthreads();
    for (int e = tid; e < E; e += blockDim.x) {
      int run = base[e];
      for (int c = 0; c < 16; ++c) {
        pre[c][e] = run;
        run += __popcll(mask[c][e]);
      }
      base[e] = run;
    }
    __syncthreads();
    if (t < M) {
      const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      int iv[kMaxTopK];
#pragma unroll
      for (int j = 0; j < kMaxTopK; ++j) {
        const int e = et[j];
        iv[j] = -1;
        if ((unsigned)e >= (unsigned)E) continue;
        const int pos = pre[wave][e] + __popcll(mask[wave][e] & below);
        iv[j] = pos;
        if (stage)
          sperm[pos] = t * k + j;
        else
          perm[pos] = t * k + j;
      }
      if (inv4) {
#pragma unroll
        for (int q = 0; q < kMaxTopK / 4; ++q)
          if (4 * q < k)
            *reinterpret_cast<int4*>(inv_perm + (size_t)t * k + 4 * q) =
                make_int4(iv[4 * q], iv[4 * q + 1], iv[4 * q + 2], iv[4 * q + 3]);
      } else {
#pragma unroll
        for (int j = 0; j < kMaxTopK; ++j)
          if (j < k && iv[j] >= 0) inv_perm[t * k + j] = iv[j];
      }
    }
    __syncthreads();
  }
  if (stage) {  // staged perm out in order
    if ((reinterpret_cast<uintptr_t>(perm) & 15) == 0) {
      for (int i = 4 * tid; i < pairs; i += 4 * kBucketThreads) {
        if (i + 3 < pairs)
          *reinterpret_cast<int4*>(perm + i) = make_int4(sperm[i], sperm[i + 1], sperm[i + 2], sperm[i + 3]);
        else
          for (int q = i; q < pairs; ++q) perm[q] = sperm[q];
      }
    } else {
      for (int i = tid; i < pairs; i += kBucketThreads) perm[i] = sperm[i];
    }
  }
  // heavy-first expert order: (count descending, id ascending); eight
  // threads per expert each count the experts ahead of it in an eighth of
  // the others (E is a multiple of 16)
  if (tid < 8 * E) {
    const int e = tid % E, part = tid / E, span = E / 8;
    const int ce = cnt[e];
    int r = 0;
    for (int f = part * span; f < (part + 1) * span; ++f) {
      const int cf = cnt[f];
      r += (cf > ce) || (cf == ce && f < e);
    }
    rpart[part][e] = r;
  }
  __syncthreads();
  if (tid < E) {
    int r = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) r += rpart[q][tid];
    ord[r] = tid;
    order[r] = tid;
  }
  __syncthreads();
  // row tiles of resident experts in heavy-first order: tile -> (expert, first
  // row); experts routed at most light_rows pairs get light tiles in the
  // second list instead (their class never rises along the list)
  if (tid < kLightClasses) lclass[tid] = 0;
  __syncthreads();
  for (int r = tid; r < E; r += blockDim.x) {
    const int e = ord[r];
    const bool res = resident == nullptr || resident[e];
    const bool light = cnt[e] <= light_rows;
    const int lrows = kLightTileRows * light_mt(cnt[e], light_mtmax);
    ntile[r] = (res && !light) ? (cnt[e] + bm_rows - 1) / bm_rows : 0;
    nlt[r] = (res && light) ? (cnt[e] + lrows - 1) / lrows : 0;
    if (nlt[r]) atomicAdd(&lclass[light_class(light_mt(cnt[e], light_mtmax))], nlt[r]);
  }
  __syncthreads();
  const int nt = scan128(ntile, tstart, E);
  scan128(nlt, lstart, E);
  if (tid == 0) *n_tiles = nt;
  if (n_ltiles && tid < kLightClasses) n_ltiles[tid] = lclass[tid];
  __syncthreads();
  // one thread per rank writes that expert's tiles
  for (int r = tid; r < E; r += blockDim.x) {
    const int e = ord[r], t0 = tstart[r], l0 = lstart[r];
    for (int i = 0; i < ntile[r]; ++i) {
      tiles[2 * (t0 + i)] = e;
      tiles[2 * (t0 + i) + 1] = i * bm_rows;
    }
    const int lrows = kLightTileRows * light_mt(cnt[e], light_mtmax);
    for (int i = 0; i < nlt[r]; ++i) {
      ltiles[2 * (l0 + i)] = e;
      ltiles[2 * (l0 + i) + 1] = i * lrows;
    }
  }
}

// one wavefront per token: inv_r[t] = 1 / sqrt(mean(x[t]^2) + eps)
__global__ __launch_bounds__(256) void rms_inv_kernel(const __half* __restrict__ x, int M, int H, float eps,
                                                      float* __restrict__ inv_r) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= M) return;
  const float r = token_inv_rms(x, t, H, eps);
  if ((threadIdx.x & 63) == 0) inv_r[t] = r;
}

// one wavefront per token: y[t] = x[t] * inv_r (one fp16 rounding); y may alias x
__global__ __launch_bounds__(256) void rmsnorm_kernel(const __half* x, int M, int H, float eps, __half* y) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= M) return;
  const float inv = token_inv_rms(x, t, H, eps);
  for (int c = lane * 8; c < H; c += 64 * 8) {
    const uint4 v = *reinterpret_cast<const uint4*>(x + (size_t)t * H + c);
    const __half* hv = reinterpret_cast<const __half*>(&v);
    uint4 o;
    __half* ho = reinterpret_cast<__half*>(&o);
#pragma unroll
    for (int i = 0; i < 8; ++i) ho[i] = __float2half_rn(__half2float(hv[i]) * inv);
    *reinterpret_cast<uint4*>(y + (size_t)t * H + c) = o;
  }
}

// the same from an fp32 input (a residual sum that may exceed the fp16 range):
// one workgroup per token, every thread loading kNv float4 of the row in one
// round (held in registers when the row fits, else re-read), the sum of
// squares reduced per wave and then over the four waves in a fixed order
constexpr int kNv = 4;
__global__ __launch_bounds__(256) void rmsnorm32_kernel(const float* __restrict__ x, int M, int H, float eps,
                                                        __half* __restrict__ y) {
  __shared__ float wsum[4];
  const int t = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* xr = x + (size_t)t * H;
  __half* yr = y + (size_t)t * H;
  constexpr int kRound = 256 * 4 * kNv;  // inputs per round
  float4 v[kNv];
  float q = 0.f;
  for (int c0 = 0; c0 < H; c0 += kRound) {
#pragma unroll
    for (int j = 0; j < kNv; ++j) {
      const int c = c0 + (j * 256 + tid) * 4;
      v[j] = c < H ? *reinterpret_cast<const float4*>(xr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int j = 0; j < kNv; ++j) {
      q = fmaf(v[j].x, v[j].x, q);
      q = fmaf(v[j].y, v[j].y, q);
      q = fmaf(v[j].z, v[j].z, q);
      q = fmaf(v[j].w, v[j].w, q);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
  if (lane == 0) wsum[wave] = q;
  __syncthreads();
  const float inv = 1.f / sqrtf((((wsum[0] + wsum[1]) + wsum[2]) + wsum[3]) / (float)H + eps);
  for (int c0 = 0; c0 < H; c0 += kRound) {
    if (H > kRound) {  // the row did not fit in one round: read this round again
#pragma unroll
      for (int j = 0; j < kNv; ++j) {
        const int c = c0 + (j * 256 + tid) * 4;
        if (c < H) v[j] = *reinterpret_cast<const float4*>(xr + c);
      }
    }
#pragma unroll
    for (int j = 0; j < kNv; ++j) {
      const int c = c0 + (j * 256 + tid) * 4;
      if (c < H) {
        __half2 lo = __halves2half2(__float2half_rn(v[j].x * inv), __float2half_rn(v[j].y * inv));
        __half2 hi = __halves2half2(__float2half_rn(v[j].z * inv), __float2half_rn(v[j].w * inv));
        uint2 o;
        o.x = *reinterpret_cast<const unsigned*>(&lo);
        o.y = *reinterpret_cast<const unsigned*>(&hi);
        *reinterpret_cast<uint2*>(yr + c) = o;
      }
    }
  }
}

}  // namespace

hipError_t launch_rmsnorm32(const float* x, int M, int H, float eps, __half* y, hipStream_t s) {
  if (H % 4 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rmsnorm32_kernel, dim3(M), dim3(256), 0, s, x, M, H, eps, y);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const __half* x, int M, int H, float eps, __half* y, hipStream_t s) {
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((M + 3) / 4), dim3(256), 0, s, x, M, H, eps, y);
  return hipGetLastError();
}

hipError_t launch_rms_inv(const __half* x, int M, int H, float eps, float* inv_r, hipStream_t s) {
  hipLaunchKernelGGL(rms_inv_kernel, dim3((M + 3) / 4), dim3(256), 0, s, x, M, H, eps, inv_r);
  return hipGetLastError();
}

hipError_t launch_router(const __half* x, const float* inv_r, float* inv_r_out, float eps, const __half* wr,
                         const float* bias, int M, int H, int E, int k, float* part, int32_t* idx, float* p,
                         float* logits, unsigned* counter, hipStream_t s) {
  // K slice per workgroup: enough workgroups to cover the chip, slices of >= 64
  const int tiles = (M + kRT - 1) / kRT;
  // a single tile may go down to one 32-input step per workgroup while the
  // routing workgroup still gathers each logit in one round (<= 64 slices)
  const int min_ks = (tiles == 1 && H / 32 <= 64) ? 32 : 64;
  int ks = H;
  while (ks > min_ks && (long)tiles * (H / ks) < 512 && (ks / 2) % 32 == 0 && H % (ks / 2) == 0) ks /= 2;
  const int n_split = H / ks;
  RouteOut ro{counter, inv_r, inv_r_out, eps, bias, k, idx, p, logits};
  if (tiles == 1 && counter && n_split <= 512) {
    // one tile: its last workgroup routes (no second launch); at most 16
    // threads per token then fetch its squares (32 slices each)
    hipLaunchKernelGGL(router_partial_kernel<true>, dim3(tiles, n_split), dim3(256), 0, s, x, wr, M, H, E, ks, part,
                       ro);
    return hipGetLastError();
  }
  // with inv_r_out the partial launch also stores per-slice sums of squares
  // and the top-k launch makes the norm factors from them
  hipLaunchKernelGGL(router_partial_kernel<false>, dim3(tiles, n_split), dim3(256), 0, s, x, wr, M, H, E, ks, part,
                     ro);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(router_topk_kernel, dim3((M + 3) / 4), dim3(256), 0, s, part, n_split, inv_r_out ? nullptr : inv_r,
                     inv_r_out, H, eps, bias, M, E, k, idx, p, logits);
  return hipGetLastError();
}

size_t router_partial_floats(int M, int H, int E) {
  // upper bound of n_split * M * (E + 1): the logit partials, then the
  // squares partials of the fused routing (n_split <= H / 32 + 1)
  return (size_t)(H / 32 + 1) * M * (E + 1);
}

hipError_t launch_bucket(const int32_t* idx, int M, int k, int E, const uint8_t* resident, int bm_rows,
                         int light_rows, int light_mtmax, int32_t* counts, int32_t* offsets, int32_t* perm,
                         int32_t* inv_perm, int32_t* order, int32_t* tiles, int32_t* n_tiles, int32_t* ltiles,
                         int32_t* n_ltiles, hipStream_t s) {
  if (k < 1 || k > kMaxTopK || (light_rows > 0 && (!ltiles || !n_ltiles || light_mtmax < 1)))
    return hipErrorInvalidValue;
  const size_t lds = (size_t)M * k <= (size_t)kBucketStage ? (size_t)M * k * sizeof(int32_t) : 0;
  hipLaunchKernelGGL(bucket_kernel, dim3(1), dim3(kBucketThreads), lds, s, idx, M, k, E, resident, bm_rows, light_rows,
                     light_mtmax, counts, offsets, perm, inv_perm, order, tiles, n_tiles, ltiles, n_ltiles);
  return hipGetLastError();
}

}  // namespace atsi
