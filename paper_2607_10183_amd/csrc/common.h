// Internal definitions shared by the HIP kernels and the C-ABI layer.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace atsi {

constexpr int kGroup = 32;  // inputs per fp16 scale

// Location of one block-int4 tensor as a kernel sees it.
struct QView {
  const uint8_t* codes;    // [N][K/2]
  const uint16_t* scales;  // [N][K/32] fp16 bits
  int K;
  int N;
};

// Epilogues of the linear kernels.
enum Epilogue : int {
  kStore = 0,        // y = acc
  kResidual = 1,     // y = acc + res (res may alias y)
};

// ---- launchers (each returns hipGetLastError() of its launch) ----
hipError_t launch_gemv(const QView& w, const __half* x, int M, __half* y, int ldy,
                       Epilogue ep, const __half* res, hipStream_t s);
hipError_t launch_gemm(const QView& w, const __half* x, int M, __half* y, int ldy,
                       Epilogue ep, const __half* res, hipStream_t s);
hipError_t launch_unpack(const QView& w, int8_t* q, hipStream_t s);

}  // namespace atsi
