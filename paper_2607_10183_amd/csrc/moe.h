// Internal definitions of the MoE path: routing, bucketing, grouped expert
// kernels and the combine.
#pragma once

#include "common.h"

namespace atsi {

constexpr int kMaxExperts = 128;   // experts per layer handled by one launch
constexpr int kMaxTopK = 16;
constexpr int kBatchExp = 4;       // streamed experts per batch launch
constexpr int kBatchTiles = 64;    // row tiles per batch launch
constexpr int kLightTileRows = 16; // rows per token block of the light-expert kernels
constexpr int kMoeLightRowsMax = 1 << 20;
constexpr int kLightClasses = 3;     // tiles of 4, 2 and 1 token blocks, in that order in the tile list
constexpr int kLightTallPairs = 16;  // taller light tiles only above this many pairs per expert on average

// Token blocks of 16 rows per light tile of an expert routed cnt pairs: the
// smallest of 1, 2, 4 that covers cnt, at most mtmax.
__host__ __device__ inline int light_mt(int cnt, int mtmax) {
  int mt = 1;
  while (mt < mtmax && mt < 4 && mt * kLightTileRows < cnt) mt *= 2;
  return mt;
}
// class of a tile of mt token blocks: 0 for 4, 1 for 2, 2 for 1
__host__ __device__ inline int light_class(int mt) { return mt == 4 ? 0 : (mt == 2 ? 1 : 2); }

// The three weight tensors of one SwiGLU expert.
struct ExpertW {
  QView gate, up, down;
};

// One grouped-expert launch.  A "tile" is (expert, first row) over the rows
// of that expert's bucket (rows offsets[e] .. offsets[e+1] of the routed
// pairs ordered by expert); rows hold pair ids k*t + j.
struct MoeArgs {
  const ExpertW* table;        // device table indexed by expert id (resident launches)
  const int32_t* tiles;        // device list of (expert, row0) (resident launches)
  const int32_t* n_tiles;      // device count of that list
  int nb;                      // > 0: batch launch over btiles with weights bw
  int2 btiles[kBatchTiles];    // (index into bexp/bw, row0)
  int bexp[kBatchExp];
  ExpertW bw[kBatchExp];
  const int32_t* counts;
  const int32_t* offsets;
  const int32_t* perm;
  const __half* x;             // tokens [M][H]
  __half* h;                   // SwiGLU activations [M*k][I], row = bucket position
  __half* out;                 // expert outputs [M*k][H], row = pair id
  const float* inv_r;          // per-token RMS-norm factor of x, or nullptr
  int k, H, I;
  int M;                       // tokens (rows of x)
  // decode with every expert HBM-resident (GEMV path only): tile t is routed
  // pair t, whose expert is pair_expert[t]; its rows in h and out are t, so no
  // bucketing sits between routing and the expert loads
  const int32_t* pair_expert;
  int n_pairs;
  int n_experts;               // table entries (a pair naming another expert is skipped)
  int store_out;               // the fused down/combine launch also stores the expert outputs in out
};

// router: logits = x W_r + b (fp32 accumulation), top-k with renormalised
// softmax.  Per-token norm factors: given (inv_r), computed here (inv_r_out,
// with eps), or none.  counter: a word that is zero between launches (the
// launch leaves it so); with it, up to 16 tokens are routed in one launch.
hipError_t launch_router(const __half* x, const float* inv_r, float* inv_r_out, float eps, const __half* wr,
                         const float* bias, int M, int H, int E, int k, float* part, int32_t* idx, float* p,
                         float* logits, unsigned* counter, hipStream_t s);
// inv_r[t] = 1 / sqrt(mean_k x[t][k]^2 + eps) (fp32)
hipError_t launch_rms_inv(const __half* x, int M, int H, float eps, float* inv_r, hipStream_t s);
// y[t] = x[t] * inv_r[t] in fp16 (y may alias x)
hipError_t launch_rmsnorm(const __half* x, int M, int H, float eps, __half* y, hipStream_t s);
hipError_t launch_rmsnorm32(const float* x, int M, int H, float eps, __half* y, hipStream_t s);
size_t router_partial_floats(int M, int H, int E);

// bucketing (single workgroup): counts, offsets, perm, inv_perm, heavy-first
// expert order and the row tiles of experts with resident[e] != 0: tiles of
// bm_rows rows for experts routed more than light_rows pairs; for the others
// light tiles of 16 * light_mt(cnt, light_mtmax) rows in ltiles, with the
// number of tiles of each class in n_ltiles[0 .. kLightClasses) (ltiles and
// n_ltiles may be null when light_rows is 0)
hipError_t launch_bucket(const int32_t* idx, int M, int k, int E, const uint8_t* resident, int bm_rows,
                         int light_rows, int light_mtmax, int32_t* counts, int32_t* offsets, int32_t* perm,
                         int32_t* inv_perm, int32_t* order, int32_t* tiles, int32_t* n_tiles, int32_t* ltiles,
                         int32_t* n_ltiles, hipStream_t s);

// rows per tile of the grouped expert kernels (1 on the GEMV path)
int expert_tile_rows(bool gemv);
// grouped SwiGLU gate/up and grouped down; tile_bound = grid size in tiles
hipError_t launch_expert_gateup(const MoeArgs& a, int tile_bound, bool gemv, hipStream_t s);
hipError_t launch_expert_down(const MoeArgs& a, int tile_bound, bool gemv, hipStream_t s);
// light experts: the tiles of one class of a.tiles (the light list, counts
// per class at a.n_tiles) or of a.btiles (all of that class): the grouped
// GEMM's products, on kernels that stream each weight once per tile; shapes
// where light_supported(H, I) holds, with tiles of at most
// light_mtmax(H, I) token blocks
bool light_supported(int H, int I);
int light_mtmax(int H, int I);
hipError_t launch_light_gateup(const MoeArgs& a, int cls, int tile_bound, hipStream_t s);
hipError_t launch_light_down(const MoeArgs& a, int cls, int tile_bound, hipStream_t s);
// Every light tile height up to 16 mtmax rows in one launch (resident tile
// list only; mtmax 1 is the one class of 16-row tiles).
hipError_t launch_light_all_gateup(const MoeArgs& a, int mtmax, int tile_bound, hipStream_t s);
hipError_t launch_light_all_down(const MoeArgs& a, int mtmax, int tile_bound, hipStream_t s);
// pair-indexed decode (a.pair_expert set): the down projections of all k
// experts of each of the M tokens and the combine, in one launch; the same
// results as launch_expert_down followed by launch_combine
hipError_t launch_expert_down_combine(const MoeArgs& a, int M, const float* p, const __half* res, __half* y,
                                      hipStream_t s);
// y[t] = sum_j p[t][j] * out[k*t + j] (fp32, slot order) -> fp16
hipError_t launch_combine(const __half* out, const float* p, int M, int k, int H, const __half* res, __half* y,
                          hipStream_t s);
// dst[perm[i]] = src[i] for rows i < rows of `cols` fp16 (dst[i] = src[i] when
// perm is null); cols % 8 == 0
hipError_t launch_gather_rows(const __half* src, const int32_t* perm, int rows, int cols, __half* dst, hipStream_t s);
// write table entries e0 .. e0+n-1 (n <= 16) and their residency flags
hipError_t launch_table_patch(ExpertW* table, uint8_t* resident, int e0, int n, const ExpertW* w, const uint8_t* r,
                              hipStream_t s);

}  // namespace atsi
