// Device helpers of the SwishRN activation (Section 3.3.4): the self-gate
// (logistic sigmoid, or the hard sigmoid that replaces it to avoid the
// exponential, Section 3.5.3) and its derivative.  Used by the GEMM's fused
// BlockNorm epilogue and by the row kernels of swishrn.hip.
#pragma once
#include "common.h"

namespace lat {

enum NormGate { GATE_NONE = 0, GATE_SIGMOID = 1, GATE_HARD = 2 };
constexpr int NORM_TILE = 128;  // BlockNorm group: the GEMM's 128-column tile

// The sigmoid from the hardware exponential and reciprocal (about 1 ulp
// each; exp(-z) = inf for very negative z gives 0).
template <int GATE>
__device__ inline float gate_fn(float z) {
  if constexpr (GATE == GATE_SIGMOID) {
    return __builtin_amdgcn_rcpf(1.f + __expf(-z));
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

// g_a and g_b of the 8 columns c.. of a layer of width N (gain = [g_a; g_b],
// two rows of N); zeros past N.  Two 16-byte loads each when aligned.
__device__ __forceinline__ void load_gains8(const float* gain, int N, int c, float* ga, float* gb) {
  if (c + 8 <= N && (N & 3) == 0 && ((uintptr_t)gain & 15) == 0) {
    const f32x4* a = reinterpret_cast<const f32x4*>(gain + c);
    const f32x4* b = reinterpret_cast<const f32x4*>(gain + N + c);
    const f32x4 a0 = a[0], a1 = a[1], b0 = b[0], b1 = b[1];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      ga[t] = a0[t];
      ga[4 + t] = a1[t];
      gb[t] = b0[t];
      gb[4 + t] = b1[t];
    }
  } else {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const bool ok = c + t < N;
      const int k = ok ? c + t : 0;
      const float x = gain[k], y = gain[N + k];
      ga[t] = ok ? x : 0.f;
      gb[t] = ok ? y : 0.f;
    }
  }
}

// 1 / (number of columns of the 128-column group holding column c)
__device__ __forceinline__ float inv_group_size(int c, int N) {
  const int cnt = max(1, min(NORM_TILE, N - (c / NORM_TILE) * NORM_TILE));
  return cnt == NORM_TILE ? 1.f / NORM_TILE : __builtin_amdgcn_rcpf((float)cnt);
}

__device__ inline float sum64(float x) {
  x += __shfl_xor(x, 32, 64);
  x += __shfl_xor(x, 16, 64);
  return sum16(x);
}

}  // namespace lat
