// Fused batch-1 decode of a dense decoder layer (one cooperative launch).
#pragma once

#include "common.h"

namespace atsi {

constexpr int kLayerPhases = 4;  // q/k/v, o, gate/up, down
enum LayerTensor { kQ = 0, kK, kV, kO, kGate, kUp, kDown, kLayerTensors };

// barrier words the fused kernel keeps in device memory (zero-initialised
// once; the barrier leaves them ready for the next launch, except the error
// flag, which stays set after a barrier that timed out)
constexpr size_t kLayerBarrierWords = 352;
constexpr int kLayerBarrierErrWord = 8 * 32 + 64;
constexpr size_t kLayerMaxLds = 96 * 1024;

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
  int rpw[kLayerPhases];  // rows per wavefront, filled by the launcher
};

// LDS bytes the fused kernel needs per workgroup for `total` steps per wave
size_t decode_layer_lds(const LayerArgs& a, int total);
// hipErrorInvalidConfiguration when the layer does not fit the fused kernel
hipError_t launch_decode_layer(LayerArgs a, hipStream_t s);

}  // namespace atsi
