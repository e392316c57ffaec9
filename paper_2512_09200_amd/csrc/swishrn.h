// Device helpers of the SwishRN activation (Section 3.3.4): the self-gate
// (logistic sigmoid, or the hard sigmoid that replaces it to avoid the
// exponential, Section 3.5.3) and its derivative.  Used by the GEMM's fused
// BlockNorm epilogue and by the row kernels of swishrn.hip.
#pragma once
#include "common.h"

namespace lat {

enum NormGate { GATE_NONE = 0, GATE_SIGMOID = 1, GATE_HARD = 2 };
constexpr int NORM_TILE = 128;  // BlockNorm group: the GEMM's 128-column tile

template <int GATE>
__device__ inline float gate_fn(float z) {
  if constexpr (GATE == GATE_SIGMOID) {
    return 1.f / (1.f + __expf(-z));
  } else {
    return fminf(fmaxf(fmaf(z, 1.f / 6.f, 0.5f), 0.f), 1.f);
  }
}

// derivative at z, given s = gate_fn(z); the hard gate's is 1/6 strictly
// inside (-3, 3)
template <int GATE>
__device__ inline float gate_deriv(float z, float s) {
  if constexpr (GATE == GATE_SIGMOID) {
    return s * (1.f - s);
  } else {
    return fabsf(z) < 3.f ? 1.f / 6.f : 0.f;
  }
}

// Sum over the 16 lanes of an aligned 16-lane group (8 columns per lane: one
// 128-column norm group).  The butterfly gives every lane the same bits.
__device__ inline float sum16(float x) {
  x += __shfl_xor(x, 1, 64);
  x += __shfl_xor(x, 2, 64);
  x += __shfl_xor(x, 4, 64);
  x += __shfl_xor(x, 8, 64);
  return x;
}

__device__ inline float sum64(float x) {
  x += __shfl_xor(x, 32, 64);
  x += __shfl_xor(x, 16, 64);
  return sum16(x);
}

}  // namespace lat
