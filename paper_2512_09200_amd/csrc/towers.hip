// Heads of per-objective towers (Section 3.3.3): the last hidden layer of the
// top MLP holds T groups of H units, one group per objective, and objective
// t's logit reads only its group:
//   z[b, t] = sum_j h[b, t*H + j] w[t, j] + bias[t]            (w: [T, H])
// backward, from the logits' gradient g (storage dtype, the GEMM-operand
// copy of the loss gradient):
//   dh[b, t*H + j] = g[b, t] w[t, j]   (times [mask > 0]: the ReLU of h)
//   dw[t, j] = sum_b g[b, t] h[b, t*H + j],   dbias[t] = sum_b g[b, t].
// Block-diagonal products of a few MACs per output: memory-bound, no MFMA.
// One thread per (sample, objective) in the forward and the input
// gradient, its H values as 16-byte vectors; the weight gradient is a
// column sum over samples (64 columns x 256 samples per block, summed in a
// fixed order, then the blocks in order).  H % 8 == 0.
#include "common.h"
#include "kernels.h"

namespace lat {

template <typename T>
__device__ __forceinline__ void ld8v(const T* p, float* v) {
  if constexpr (sizeof(T) == 2) {
    Vec16<bf16_t>::unpack(ldg16(p), v);
  } else {
    Vec16<float>::unpack(ldg16(p), v);
    Vec16<float>::unpack(ldg16(p + 4), v + 4);
  }
}

template <typename T>
__device__ __forceinline__ void st8v(T* p, const float* v) {
  if constexpr (sizeof(T) == 2) {
    stg16(p, Vec16<bf16_t>::pack(v));
  } else {
    stg16(p, Vec16<float>::pack(v));
    stg16(p + 4, Vec16<float>::pack(v + 4));
  }
}

template <typename T>
__global__ __launch_bounds__(256) void tower_head_fwd_kernel(const T* __restrict__ h, int64_t ldh,
                                                             int B, int NT, int H,
                                                             const T* __restrict__ w,
                                                             const float* __restrict__ bias,
                                                             float* __restrict__ z) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * NT) return;
  const int64_t b = i / NT;
  const int t = (int)(i - b * NT);
  const T* hp = h + b * ldh + (int64_t)t * H;
  const T* wp = w + (int64_t)t * H;
  float acc = 0.f;
  for (int j = 0; j < H; j += 8) {  // in order of j
    float hv[8], wv[8];
    ld8v(hp + j, hv);
    ld8v(wp + j, wv);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += hv[e] * wv[e];
  }
  z[i] = acc + (bias ? bias[t] : 0.f);
}

template <typename T>
__global__ __launch_bounds__(256) void tower_head_dgrad_kernel(const T* __restrict__ g, int64_t ldg,
                                                               int B, int NT, int H,
                                                               const T* __restrict__ w,
                                                               const T* __restrict__ mask, int64_t ldm,
                                                               T* __restrict__ dh, int64_t ldd) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * NT) return;
  const int64_t b = i / NT;
  const int t = (int)(i - b * NT);
  const float gv = ld(g + b * ldg + t);
  const T* wp = w + (int64_t)t * H;
  T* dp = dh + b * ldd + (int64_t)t * H;
  const T* mp = mask ? mask + b * ldm + (int64_t)t * H : nullptr;
  for (int j = 0; j < H; j += 8) {
    float wv[8], o[8];
    ld8v(wp + j, wv);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = gv * wv[e];
    if (mp) {
      float mv[8];
      ld8v(mp + j, mv);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = mv[e] > 0.f ? o[e] : 0.f;
    }
    st8v(dp + j, o);
  }
}

constexpr int TW_ROWS = 256;

// block (x, y): columns x*64 .. x*64+63 of the T*H, samples y*256 ..; thread
// = 8 columns (one objective: H % 8 == 0) x every 32nd sample
template <typename T>
__global__ __launch_bounds__(256) void tower_wgrad_partial_kernel(const T* __restrict__ g, int64_t ldg,
                                                                  const T* __restrict__ h, int64_t ldh,
                                                                  int B, int NT, int H,
                                                                  float* __restrict__ part) {
  __shared__ float red[32][65];
  const int cg = threadIdx.x & 7, rl = threadIdx.x >> 3;
  const int TH = NT * H;
  const int col0 = blockIdx.x * 64 + cg * 8;
  const int r0 = blockIdx.y * TW_ROWS, r1 = min(B, r0 + TW_ROWS);
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  if (col0 < TH) {
    const int t = col0 / H;
    // straight line over the thread's 8 samples (loads in flight together);
    // samples past B read sample r0 and count as zero
#pragma unroll
    for (int q = 0; q < TW_ROWS / 32; ++q) {
      const int r = r0 + rl + 32 * q;
      const bool ok = r < r1;
      const int64_t rr = ok ? r : r0;
      float hv[8];
      ld8v(h + rr * ldh + col0, hv);
      const float gv = ok ? ld(g + rr * ldg + t) : 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += gv * hv[e];
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rl][cg * 8 + e] = acc[e];
  __syncthreads();
  if (threadIdx.x < 64) {
    const int col = blockIdx.x * 64 + threadIdx.x;
    float s = 0.f;
    for (int q = 0; q < 32; ++q) s += red[q][threadIdx.x];
    if (col < TH) part[(int64_t)blockIdx.y * TH + col] = s;
  }
}

__global__ __launch_bounds__(256) void tower_wgrad_final_kernel(const float* __restrict__ part,
                                                                int chunks, int TH,
                                                                float* __restrict__ dw) {
  const int col = blockIdx.x * 256 + threadIdx.x;
  if (col >= TH) return;
  const float* p = part + col;
  float s = 0.f;
  int c = 0;
  for (; c + 8 <= chunks; c += 8) {  // in order; 8 loads issued before their adds
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = p[(int64_t)(c + q) * TH];
#pragma unroll
    for (int q = 0; q < 8; ++q) s += v[q];
  }
  for (; c < chunks; ++c) s += p[(int64_t)c * TH];
  dw[col] = s;
}

static bool a16(const void* p) { return ((uintptr_t)p & 15) == 0; }

static hipError_t tower_check(DType dt, const void* h, int64_t ldh, int H, const void* w) {
  const int64_t e = dt == DT_BF16 ? 8 : 4;
  if (H % 8 || ldh % e || !a16(h) || !a16(w)) {
    set_error("tower heads: units per tower must be a multiple of 8, rows and weights 16-byte aligned");
    return hipErrorInvalidValue;
  }
  return hipSuccess;
}

hipError_t tower_head_fwd(DType dt, const void* h, int64_t ldh, int B, int NT, int H, const void* w,
                          const float* bias, float* z, hipStream_t s) {
  if (B == 0 || NT == 0) return hipSuccess;
  hipError_t e = tower_check(dt, h, ldh, H, w);
  if (e != hipSuccess) return e;
  const int grid = cdiv((int64_t)B * NT, 256);
  if (dt == DT_BF16)
    tower_head_fwd_kernel<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)h, ldh, B, NT, H, (const bf16_t*)w, bias, z);
  else
    tower_head_fwd_kernel<float><<<grid, 256, 0, s>>>((const float*)h, ldh, B, NT, H, (const float*)w, bias, z);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t tower_head_dgrad(DType dt, const void* g, int64_t ldg, int B, int NT, int H, const void* w,
                            const void* mask, int64_t ldm, void* dh, int64_t ldd, hipStream_t s) {
  if (B == 0 || NT == 0) return hipSuccess;
  hipError_t e = tower_check(dt, dh, ldd, H, w);
  if (e == hipSuccess && mask) e = tower_check(dt, mask, ldm, H, w);
  if (e != hipSuccess) return e;
  const int grid = cdiv((int64_t)B * NT, 256);
  if (dt == DT_BF16)
    tower_head_dgrad_kernel<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)g, ldg, B, NT, H, (const bf16_t*)w,
                                                         (const bf16_t*)mask, ldm, (bf16_t*)dh, ldd);
  else
    tower_head_dgrad_kernel<float><<<grid, 256, 0, s>>>((const float*)g, ldg, B, NT, H, (const float*)w,
                                                        (const float*)mask, ldm, (float*)dh, ldd);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

size_t tower_wgrad_workspace(int B, int NT, int H) {
  return (size_t)cdiv(B > 0 ? B : 1, TW_ROWS) * NT * H * sizeof(float);
}

hipError_t tower_wgrad(DType dt, const void* g, int64_t ldg, const void* h, int64_t ldh, int B, int NT,
                       int H, float* dw, void* ws, hipStream_t s) {
  const int TH = NT * H;
  if (TH == 0 || !dw) return hipSuccess;
  hipError_t e = tower_check(dt, h, ldh, H, h);
  if (e != hipSuccess) return e;
  const int chunks = B > 0 ? cdiv(B, TW_ROWS) : 0;
  float* part = (float*)ws;
  if (chunks > 0) {
    const dim3 grid(cdiv(TH, 64), chunks);
    if (dt == DT_BF16)
      tower_wgrad_partial_kernel<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)g, ldg, (const bf16_t*)h, ldh,
                                                              B, NT, H, part);
    else
      tower_wgrad_partial_kernel<float><<<grid, 256, 0, s>>>((const float*)g, ldg, (const float*)h, ldh,
                                                             B, NT, H, part);
    LAT_LAUNCH_CHECK();
  }
  tower_wgrad_final_kernel<<<cdiv(TH, 256), 256, 0, s>>>(part, chunks, TH, dw);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
