// Internal definitions shared by the HIP kernels and the C-ABI layer.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace atsi {

constexpr int kGroup = 32;  // inputs per fp16 scale
constexpr int kMaxCallRows = 65536;  // activation rows (tokens) one call may take
constexpr int kMaxSeg = 3;  // tensors fused into one launch

// Location of one block-int4 tensor as a kernel sees it.
struct QView {
  const uint8_t* codes;    // [N][K/2]
  const uint16_t* scales;  // [N][K/32] fp16 bits
  int K;
  int N;
};

// One output segment of a fused launch: a tensor (or a gate/up pair), where
// its outputs go and how they are laid out.
struct Seg {
  QView w;       // the tensor (gate for SwiGLU)
  QView w2;      // up tensor for SwiGLU, unused otherwise
  __half* y;     // output [M][ldy]
  int ldy;
  int expand;    // >1: output row n = (j, d) of a KV head is written to
                 // query heads j*expand .. j*expand+expand-1 (context-length-1
                 // attention of grouped-query heads); 1: plain
};

// A fused linear launch over up to kMaxSeg tensors sharing one input x.
struct LinOp {
  Seg seg[kMaxSeg];
  int nseg;
  const __half* x;   // [M][K], K common to all segments
  int M;
  int K;
  int swiglu;        // 1: segment 0 is a (gate, up) pair, output silu(g) * u
  int norm;          // 1: input is RMS-normalised (unit gain) before the product
  float eps;
  const __half* res; // residual added to segment 0's output (may alias its y)
  float* y32;        // non-null: segment 0's output goes here in fp32 instead of y
  int head_dim;      // granularity of `expand`
  const float* rinv; // norm: per-row 1 / rms of x precomputed (the 512-row GEMM needs it), or null
};

__device__ __forceinline__ float silu_f(float g) { return g / (1.f + expf(-g)); }

// Epilogue of one output v of row `row` (output n) of token m in segment s:
// grouped-query expansion, or residual add (segment 0), then fp32 or fp16.
__device__ __forceinline__ void emit_out(const LinOp& op, const Seg& sg, int s, int m, int row, float v) {
  if (sg.expand > 1) {
    const int hd = op.head_dim, jh = row / hd, d = row % hd;
    const __half o = __float2half_rn(v);
    for (int g = 0; g < sg.expand; ++g) sg.y[(size_t)m * sg.ldy + (size_t)(jh * sg.expand + g) * hd + d] = o;
    return;
  }
  const size_t at = (size_t)m * sg.ldy + row;
  if (op.res && s == 0) v += __half2float(op.res[at]);
  if (op.y32 && s == 0)
    op.y32[at] = v;
  else
    sg.y[at] = __float2half_rn(v);
}

// Loads through the global address space.  Pointers read from memory (expert
// tables, step tables) are otherwise generic, and a generic load also counts
// against the LDS wait counter: every LDS wait would then drain the loads in
// flight.
typedef unsigned u32x4_g __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg16(const void* p) {
  const u32x4_g v = *reinterpret_cast<const __attribute__((address_space(1))) u32x4_g*>(reinterpret_cast<uintptr_t>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint16_t ldg2(const uint16_t* p) {
  return *reinterpret_cast<const __attribute__((address_space(1))) uint16_t*>(reinterpret_cast<uintptr_t>(p));
}

// ---- launchers (each returns hipGetLastError() of its launch) ----
// LDS one workgroup may use on the current device (160 KiB on gfx950)
size_t lds_limit();
// Tokens one decode-GEMV launch takes for inputs K wide: 4, 2 or 1, the most
// whose staged activations fit in LDS (0 if not even one does).  Calls with
// up to 4 tokens run as GEMV launches of at most that many tokens.
int gemv_tokens(int K);
constexpr int kGemvMaxTokens = 4;
hipError_t launch_gemv(const LinOp& op, hipStream_t s);
// batched decode on the matrix cores: 1 <= M <= kSkinnyMaxTokens, K
// divisible by 128, tensors below 2 GiB
constexpr int kSkinnyMaxTokens = 16;
constexpr int kSkinnyMinTokens = 2;  // a single token goes to the GEMV
bool skinny_supported(const LinOp& op);
hipError_t launch_skinny(const LinOp& op, hipStream_t s);
hipError_t launch_gemm(const LinOp& op, hipStream_t s);
// 512-row-tile prefill GEMM.  K ranges per output tile: 1 when the launch
// has a tile for most CUs, up to 8 (fp32 partial sums, reduced by a second
// kernel in a fixed order) when it does not, 0 when the 512-row tiles do not
// apply (fewer than 256 rows, too little K to split, offsets beyond 32 bits).
constexpr int kWideMinTiles = 192;  // three quarters of the 256 CUs
constexpr int kWideMaxSplits = 8;
int gemm_wide_splits(const LinOp& op);
// bytes of fp32 partial sums a launch with `splits` K ranges needs (0 for 1)
size_t gemm_wide_part_bytes(const LinOp& op, int splits);
hipError_t launch_gemm_wide(const LinOp& op, int splits, float* part, hipStream_t s);
hipError_t launch_unpack(const QView& w, int8_t* q, hipStream_t s);
// read-only streaming probe over bytes (16-byte aligned, a multiple of 16)
hipError_t launch_read_probe(const void* p, size_t bytes, unsigned* sink, hipStream_t s);

// single-tensor helpers
inline LinOp plain_op(const QView& w, const __half* x, int M, __half* y) {
  LinOp op{};
  op.seg[0].w = w;
  op.seg[0].y = y;
  op.seg[0].ldy = w.N;
  op.seg[0].expand = 1;
  op.nseg = 1;
  op.x = x;
  op.M = M;
  op.K = w.K;
  op.head_dim = 1;
  return op;
}

}  // namespace atsi
