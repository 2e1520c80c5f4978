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
//                   workgroup to finish (release/acquire fences around a
//                   counter that the last one resets), and computes the
//                   tokens' RMS-norm factors there when asked.
//   router_topk     one wavefront per token: sums the K-slice partials in a
//                   fixed order, adds the bias, selects the top k by (logit
//                   descending, expert id ascending) with k wave-wide argmax
//                   rounds (DPP inside rows of 16 lanes, scalar reads across
//                   rows), and writes the softmax over the selected logits.
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

// 1 / sqrt(mean(x[t]^2) + eps) for one token, computed by one wavefront and
// returned to every lane (the same arithmetic for every caller)
__device__ __forceinline__ float token_inv_rms(const __half* __restrict__ x, int t, int H, float eps) {
  const int lane = threadIdx.x & 63;
  float q = 0.f;
  for (int c = lane * 8; c < H; c += 64 * 8) {
    const uint4 v = *reinterpret_cast<const uint4*>(x + (size_t)t * H + c);
    const __half* hv = reinterpret_cast<const __half*>(&v);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float f = __half2float(hv[i]);
      q = fmaf(f, f, q);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
  return 1.f / sqrtf(q / (float)H + eps);
}

__device__ __forceinline__ void wave_best(float& v, int& i);

// Routing of token t by one wavefront (E <= 128, two candidates per lane):
// the K-slice partial logits summed in slice order, times the norm factor rs
// when norm is set, plus the bias; the top k by (logit descending, expert id
// ascending) in k argmax rounds; the softmax over the selected logits.
__device__ __forceinline__ void route_token(const float* __restrict__ part, int n_split, int M, int t, bool norm,
                                            float rs, const float* __restrict__ bias, int E, int k,
                                            int32_t* __restrict__ idx, float* __restrict__ p,
                                            float* __restrict__ logits_out) {
  const int lane = threadIdx.x & 63;
  float v[2] = {0.f, 0.f};
  int id[2] = {lane, lane + 64};
  // every global load is issued before the first wait: the bias, then the
  // K-slice partials, 16 slices of both experts per round (the partials come
  // from other XCDs' writes, a memory round trip each), added in slice order
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
  float sel_v[16];
  int sel_i[16];
  for (int j = 0; j < k; ++j) {
    // best of this lane: larger value, then lower id
    float bv2 = v[0];
    int bi = id[0];
    if (v[1] > bv2 || (v[1] == bv2 && id[1] < bi)) { bv2 = v[1]; bi = id[1]; }
    if (bi >= E) bi = 0x7fffffff;
    wave_best(bv2, bi);
    sel_v[j] = bv2;
    sel_i[j] = bi;
    if (bi == id[0]) v[0] = -INFINITY, id[0] = 0x7fffffff;
    if (bi == id[1]) v[1] = -INFINITY, id[1] = 0x7fffffff;
  }
  if (lane == 0) {
    float den = 0.f;
    for (int j = 0; j < k; ++j) den += expf(sel_v[j] - sel_v[0]);
    for (int j = 0; j < k; ++j) {
      idx[(size_t)t * k + j] = sel_i[j];
      p[(size_t)t * k + j] = expf(sel_v[j] - sel_v[0]) / den;
    }
  }
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

// grid: (ceil(M/16), n_split); block 256 = 4 waves x 32 experts (E <= 128).
// Requires E % 16 == 0, E <= 128, ks % 32 == 0.
template <bool FUSED>
__global__ __launch_bounds__(256) void router_partial_kernel(const __half* __restrict__ x, const __half* __restrict__ wr,
                                                             int M, int H, int E, int ks, float* __restrict__ part,
                                                             RouteOut ro) {
  __shared__ __attribute__((aligned(16))) _Float16 Bt[128 * (32 + 8)];  // [expert][k] of one 32-k step
  const int t0 = blockIdx.x * kRT;
  const int k_begin = blockIdx.y * ks;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tr = lane & 15, kq = (lane >> 4) * 8;
  float4_t acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  for (int k0 = k_begin; k0 < k_begin + ks; k0 += 32) {
    // stage W_r[k0 .. k0+31][0 .. E) transposed: thread -> (k = tid / 16, 8 experts)
    __syncthreads();
    {
      const int kk = threadIdx.x >> 4, e8 = (threadIdx.x & 15) * 8;
      if (e8 < E) {
        const uint4 v = *reinterpret_cast<const uint4*>(wr + (size_t)(k0 + kk) * E + e8);
        const _Float16* hv = reinterpret_cast<const _Float16*>(&v);
#pragma unroll
        for (int i = 0; i < 8; ++i) Bt[(e8 + i) * 40 + kk] = hv[i];
      }
      if (kk + 16 < 32) {
        const int k2 = kk + 16;
        if (e8 < E) {
          const uint4 v = *reinterpret_cast<const uint4*>(wr + (size_t)(k0 + k2) * E + e8);
          const _Float16* hv = reinterpret_cast<const _Float16*>(&v);
#pragma unroll
          for (int i = 0; i < 8; ++i) Bt[(e8 + i) * 40 + k2] = hv[i];
        }
      }
    }
    __syncthreads();
    half8_t a;
    const int t = t0 + tr;
    if (t < M)
      a = *reinterpret_cast<const half8_t*>(x + (size_t)t * H + k0 + kq);
    else
      a = half8_t{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int e = wave * 32 + nb * 16 + tr;
      if (wave * 32 + nb * 16 < E) {
        const half8_t b = *reinterpret_cast<const half8_t*>(&Bt[e * 40 + kq]);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[nb], 0, 0, 0);
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
      const int t = t0 + 4 * (lane >> 4) + i;
      if (t < M) part[((size_t)blockIdx.y * M + t) * E + e] = acc[nb][i];
    }
  }
  if constexpr (FUSED) {
    // The last workgroup to finish routes the tile: every workgroup makes its
    // partials visible device-wide (release) before it counts itself; the last
    // one acquires them all, resets the count for the next launch and routes.
    __shared__ unsigned ticket;
    __threadfence();
    if (threadIdx.x == 0) ticket = atomicAdd(ro.counter, 1u);
    __syncthreads();
    if (ticket != gridDim.y - 1) return;
    __threadfence();
    if (threadIdx.x == 0) atomicExch(ro.counter, 0u);
    for (int tt = wave; tt < kRT; tt += 4) {
      const int t = t0 + tt;
      if (t >= M) break;
      float rs = 1.f;
      if (ro.inv_r_out) {
        rs = token_inv_rms(x, t, H, ro.eps);
        if (lane == 0) ro.inv_r_out[t] = rs;
      } else if (ro.inv_r) {
        rs = ro.inv_r[t];
      }
      route_token(part, gridDim.y, M, t, ro.inv_r_out || ro.inv_r, rs, ro.bias, E, ro.k, ro.idx, ro.p, ro.logits);
    }
  }
}

// (value, id) of the best candidate of the wave, by (value descending, id
// ascending), returned to every lane: DPP steps inside rows of 16 lanes
// (swap neighbours, swap pairs, mirror within 8, mirror within 16), then the
// four row results read back as scalars.  Needs all 64 lanes active.
__device__ __forceinline__ void wave_best(float& v, int& i) {
  auto better = [](float av, int ai, float bv, int bi) { return av > bv || (av == bv && ai < bi); };
#define ATSI_BEST_STEP(CTRL)                                                                             \
  {                                                                                                      \
    const float ov = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false)); \
    const int oi = __builtin_amdgcn_update_dpp(0, i, CTRL, 0xF, 0xF, false);                             \
    if (better(ov, oi, v, i)) {                                                                          \
      v = ov;                                                                                            \
      i = oi;                                                                                            \
    }                                                                                                    \
  }
  ATSI_BEST_STEP(0xB1)   // quad_perm 1,0,3,2
  ATSI_BEST_STEP(0x4E)   // quad_perm 2,3,0,1
  ATSI_BEST_STEP(0x141)  // row_half_mirror
  ATSI_BEST_STEP(0x140)  // row_mirror
#undef ATSI_BEST_STEP
  float bv = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  int bi = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) {
    const float ov = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16 * r));
    const int oi = __builtin_amdgcn_readlane(i, 16 * r);
    if (better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
  v = bv;
  i = bi;
}

// one wave per token; E <= 128 (two candidates per lane)
__global__ __launch_bounds__(256) void router_topk_kernel(const float* __restrict__ part, int n_split,
                                                          const float* __restrict__ inv_r,
                                                          const float* __restrict__ bias, int M, int E, int k,
                                                          int32_t* __restrict__ idx, float* __restrict__ p,
                                                          float* __restrict__ logits_out) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= M) return;
  const float rs = inv_r ? inv_r[t] : 1.f;
  route_token(part, n_split, M, t, inv_r != nullptr, rs, bias, E, k, idx, p, logits_out);
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
__global__ __launch_bounds__(1024) void bucket_kernel(const int32_t* __restrict__ idx, int M, int k, int E,
                                                      const uint8_t* __restrict__ resident, int bm_rows,
                                                      int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
                                                      int32_t* __restrict__ perm, int32_t* __restrict__ inv_perm,
                                                      int32_t* __restrict__ order, int32_t* __restrict__ tiles,
                                                      int32_t* __restrict__ n_tiles) {
  __shared__ int cnt[kMaxExperts];
  __shared__ int base[kMaxExperts];
  __shared__ unsigned long long mask[16][kMaxExperts];
  __shared__ int pre[16][kMaxExperts];
  __shared__ int ord[kMaxExperts];
  __shared__ int ntile[kMaxExperts];   // tiles of the expert at rank r
  __shared__ int tstart[kMaxExperts];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int pairs = M * k;
  for (int e = tid; e < E; e += blockDim.x) cnt[e] = 0;
  __syncthreads();
  for (int i = tid; i < pairs; i += blockDim.x) {
    const int e = idx[i];
    if ((unsigned)e < (unsigned)E) atomicAdd(&cnt[e], 1);
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
    if (t < M)
      for (int j = 0; j < k; ++j) {
        const int e = idx[(size_t)t * k + j];
        if ((unsigned)e < (unsigned)E) atomicOr(&mask[wave][e], 1ull << lane);
      }
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
      for (int j = 0; j < k; ++j) {
        const int e = idx[(size_t)t * k + j];
        if ((unsigned)e >= (unsigned)E) continue;
        const int pos = pre[wave][e] + __popcll(mask[wave][e] & below);
        perm[pos] = t * k + j;
        inv_perm[t * k + j] = pos;
      }
    }
    __syncthreads();
  }
  // heavy-first expert order: (count descending, id ascending)
  for (int e = tid; e < E; e += blockDim.x) {
    const int ce = cnt[e];
    int r = 0;
    for (int f0 = 0; f0 < E; f0 += 16) {  // E is a multiple of 16
      int cf[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) cf[j] = cnt[f0 + j];
#pragma unroll
      for (int j = 0; j < 16; ++j) r += (cf[j] > ce) || (cf[j] == ce && f0 + j < e);
    }
    ord[r] = e;
    order[r] = e;
  }
  __syncthreads();
  // row tiles of resident experts in heavy-first order: tile -> (expert, first row)
  for (int r = tid; r < E; r += blockDim.x) {
    const int e = ord[r];
    ntile[r] = (resident == nullptr || resident[e]) ? (cnt[e] + bm_rows - 1) / bm_rows : 0;
  }
  __syncthreads();
  const int nt = scan128(ntile, tstart, E);
  if (tid == 0) *n_tiles = nt;
  __syncthreads();
  for (int r = wave; r < E; r += blockDim.x / 64) {
    const int e = ord[r];
    for (int i = lane; i < ntile[r]; i += 64) {
      tiles[2 * (tstart[r] + i)] = e;
      tiles[2 * (tstart[r] + i) + 1] = i * bm_rows;
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
  float q = 0.f;
  for (int c = lane * 8; c < H; c += 64 * 8) {
    const uint4 v = *reinterpret_cast<const uint4*>(x + (size_t)t * H + c);
    const __half* hv = reinterpret_cast<const __half*>(&v);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float f = __half2float(hv[i]);
      q = fmaf(f, f, q);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
  const float inv = 1.f / sqrtf(q / (float)H + eps);
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

// the same from an fp32 input (a residual sum that may exceed the fp16 range)
__global__ __launch_bounds__(256) void rmsnorm32_kernel(const float* __restrict__ x, int M, int H, float eps,
                                                        __half* __restrict__ y) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= M) return;
  float q = 0.f;
  for (int c = lane * 4; c < H; c += 64 * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + (size_t)t * H + c);
    q = fmaf(v.x, v.x, q);
    q = fmaf(v.y, v.y, q);
    q = fmaf(v.z, v.z, q);
    q = fmaf(v.w, v.w, q);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
  const float inv = 1.f / sqrtf(q / (float)H + eps);
  for (int c = lane * 4; c < H; c += 64 * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + (size_t)t * H + c);
    y[(size_t)t * H + c] = __float2half_rn(v.x * inv);
    y[(size_t)t * H + c + 1] = __float2half_rn(v.y * inv);
    y[(size_t)t * H + c + 2] = __float2half_rn(v.z * inv);
    y[(size_t)t * H + c + 3] = __float2half_rn(v.w * inv);
  }
}

}  // namespace

hipError_t launch_rmsnorm32(const float* x, int M, int H, float eps, __half* y, hipStream_t s) {
  hipLaunchKernelGGL(rmsnorm32_kernel, dim3((M + 3) / 4), dim3(256), 0, s, x, M, H, eps, y);
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
  int ks = H;
  while (ks > 64 && (long)tiles * (H / ks) < 512 && (ks / 2) % 32 == 0 && H % (ks / 2) == 0) ks /= 2;
  const int n_split = H / ks;
  RouteOut ro{counter, inv_r, inv_r_out, eps, bias, k, idx, p, logits};
  if (tiles == 1 && counter) {
    // one tile: its last workgroup routes (no second launch)
    hipLaunchKernelGGL(router_partial_kernel<true>, dim3(tiles, n_split), dim3(256), 0, s, x, wr, M, H, E, ks, part,
                       ro);
    return hipGetLastError();
  }
  if (inv_r_out) {
    hipLaunchKernelGGL(rms_inv_kernel, dim3((M + 3) / 4), dim3(256), 0, s, x, M, H, eps, inv_r_out);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    inv_r = inv_r_out;
  }
  hipLaunchKernelGGL(router_partial_kernel<false>, dim3(tiles, n_split), dim3(256), 0, s, x, wr, M, H, E, ks, part,
                     ro);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(router_topk_kernel, dim3((M + 3) / 4), dim3(256), 0, s, part, n_split, inv_r, bias, M, E, k,
                     idx, p, logits);
  return hipGetLastError();
}

size_t router_partial_floats(int M, int H, int E) {
  // upper bound of n_split * M * E (n_split <= H / 64)
  return (size_t)(H / 64 + 1) * M * E;
}

hipError_t launch_bucket(const int32_t* idx, int M, int k, int E, const uint8_t* resident, int bm_rows,
                         int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* inv_perm, int32_t* order,
                         int32_t* tiles, int32_t* n_tiles, hipStream_t s) {
  hipLaunchKernelGGL(bucket_kernel, dim3(1), dim3(1024), 0, s, idx, M, k, E, resident, bm_rows, counts, offsets, perm,
                     inv_perm, order, tiles, n_tiles);
  return hipGetLastError();
}

}  // namespace atsi
