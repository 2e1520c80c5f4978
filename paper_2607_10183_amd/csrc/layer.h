// Fused batch-1 decode of an 8B-shaped dense decoder layer (one persistent
// launch of one workgroup per CU, grid barriers between its four phases).
#pragma once

#include "common.h"

namespace atsi {

enum LayerTensor { kQ = 0, kK, kV, kO, kGate, kUp, kDown, kLayerTensors };

// barrier words the fused kernel keeps in device memory (zero-initialised
// once; the barrier leaves them ready for the next launch, except the error
// flag, which stays set after a barrier that timed out)
constexpr size_t kLayerBarrierWords = 352;
constexpr int kLayerBarrierErrWord = 8 * 32 + 64;
// a word of the same block the read probe may write (never read)
constexpr int kProbeSinkWord = kLayerBarrierErrWord + 16;
static_assert(kProbeSinkWord < (int)kLayerBarrierWords, "probe sink inside the block");

struct LayerArgs {
  QView w[kLayerTensors];
  __half* h;      // [H] residual stream, read and updated in place
  __half* q_out;  // [Hq]
  __half* k_out;  // [Hkv]
  __half* oin;    // [Hq] attention output (v expanded to the query heads)
  __half* hf;     // [I] SwiGLU activation
  unsigned* bar;  // kLayerBarrierWords words of barrier state
  int H, Hq, Hkv, I, head_dim, expand;
  float eps;
};

// hipErrorInvalidConfiguration when the layer is not the shape the fused
// kernel is built for (hidden 4096, 32 x 128 query and 8 x 128 KV heads,
// SwiGLU 14336) or the device does not have 256 CUs for one workgroup each
hipError_t launch_decode_layer(LayerArgs a, hipStream_t s);

}  // namespace atsi
