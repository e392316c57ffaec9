// Feature interaction over the stacked per-sample vectors X_b [n, d]
// (Section 3.3.2): dot-product Gram (strict upper triangle) and the
// factorization-machine block O_b = X_b (X_b^T W), forward and backward.
//
// These kernels stage one sample's vectors in LDS as fp32 and compute with
// fp32 FMAs; storage rounding happens exactly where the products are stored
// (P = X^T W and the output O for FM; the pair values for DOT), matching the
// precision policy of the whole step.  The FM weight gradient is summed per
// block over a fixed set of samples and then over blocks in a fixed order.
#include "common.h"
#include "kernels.h"

namespace lat {

// ---------------------------------------------------------------------------
// DOT
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void dot_fwd_kernel(const T* __restrict__ X, int n, int d,
                                                      T* __restrict__ out, int64_t ostride,
                                                      int emit0) {
  extern __shared__ float xs[];  // [n][d+1]
  const int b = blockIdx.x;
  const int ldx = d + 1;
  const T* Xb = X + (int64_t)b * n * d;
  for (int e = threadIdx.x; e < n * d; e += 256) xs[(e / d) * ldx + (e % d)] = ld(Xb + e);
  __syncthreads();
  T* ob = out + (int64_t)b * ostride;
  int off = 0;
  if (emit0) {
    for (int a = threadIdx.x; a < d; a += 256) ob[a] = Xb[a];
    off = d;
  }
  for (int q = threadIdx.x; q < n * n; q += 256) {
    const int i = q / n, j = q % n;
    if (j <= i) continue;
    float s = 0.f;
    for (int a = 0; a < d; ++a) s = fmaf(xs[i * ldx + a], xs[j * ldx + a], s);
    const int m = i * n - i * (i + 1) / 2 + (j - i - 1);
    st(ob + off + m, s);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void dot_bwd_kernel(const T* __restrict__ X, int n, int d,
                                                      const T* __restrict__ dout,
                                                      int64_t dstride, int emit0,
                                                      T* __restrict__ dX) {
  extern __shared__ float sm[];  // xs [n][d+1], S [n][n+1]
  const int b = blockIdx.x;
  const int ldx = d + 1, lds = n + 1;
  float* xs = sm;
  float* S = sm + n * ldx;
  const T* Xb = X + (int64_t)b * n * d;
  const T* gb = dout + (int64_t)b * dstride;
  const int off = emit0 ? d : 0;
  for (int e = threadIdx.x; e < n * d; e += 256) xs[(e / d) * ldx + (e % d)] = ld(Xb + e);
  for (int q = threadIdx.x; q < n * n; q += 256) {
    const int i = q / n, j = q % n;
    float v = 0.f;
    if (i != j) {
      const int lo = i < j ? i : j, hi = i < j ? j : i;
      v = ld(gb + off + lo * n - lo * (lo + 1) / 2 + (hi - lo - 1));
    }
    S[i * lds + j] = v;
  }
  __syncthreads();
  T* dXb = dX + (int64_t)b * n * d;
  for (int e = threadIdx.x; e < n * d; e += 256) {
    const int i = e / d, a = e % d;
    float s = 0.f;
    for (int j = 0; j < n; ++j) s = fmaf(S[i * lds + j], xs[j * ldx + a], s);
    if (emit0 && i == 0) s += ld(gb + a);
    st(dXb + e, s);
  }
}

// ---------------------------------------------------------------------------
// FM
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void fm_fwd_kernel(const T* __restrict__ X, const T* __restrict__ W,
                                                     int n, int d, int k, T* __restrict__ out,
                                                     int64_t ostride, int emit0) {
  extern __shared__ float sm[];  // xs [n][d+1], ws [n][k], ps [d][k+1]
  const int b = blockIdx.x;
  const int ldx = d + 1, ldp = k + 1;
  float* xs = sm;
  float* ws = xs + n * ldx;
  float* ps = ws + n * k;
  const T* Xb = X + (int64_t)b * n * d;
  for (int e = threadIdx.x; e < n * d; e += 256) xs[(e / d) * ldx + (e % d)] = ld(Xb + e);
  for (int e = threadIdx.x; e < n * k; e += 256) ws[e] = ld(W + e);
  __syncthreads();
  for (int e = threadIdx.x; e < d * k; e += 256) {
    const int a = e / k, c = e % k;
    float s = 0.f;
    for (int j = 0; j < n; ++j) s = fmaf(xs[j * ldx + a], ws[j * k + c], s);
    ps[a * ldp + c] = ld_round<T>(s);  // P is stored at storage precision
  }
  __syncthreads();
  T* ob = out + (int64_t)b * ostride;
  int off = 0;
  if (emit0) {
    for (int a = threadIdx.x; a < d; a += 256) ob[a] = Xb[a];
    off = d;
  }
  for (int e = threadIdx.x; e < n * k; e += 256) {
    const int j = e / k, c = e % k;
    float s = 0.f;
    for (int a = 0; a < d; ++a) s = fmaf(xs[j * ldx + a], ps[a * ldp + c], s);
    st(ob + off + e, s);
  }
}

// Backward of O = X (X^T W) given G = dO:  P = rnd(X^T W), dP = rnd(X^T G),
// dX = G P^T + W dP^T (+ addend), dW = sum_b X dP.  Persistent over samples:
// block z handles samples z, z + gridDim.x, ...; its dW partial goes to
// dw_part[z].
template <typename T, typename DXT>
__global__ __launch_bounds__(256) void fm_bwd_kernel(const T* __restrict__ X, const T* __restrict__ W,
                                                     int B, int n, int d, int k,
                                                     const T* __restrict__ dout, int64_t dstride,
                                                     int emit0, const float* __restrict__ addend,
                                                     DXT* __restrict__ dX,
                                                     float* __restrict__ dw_part) {
  extern __shared__ float sm[];  // xs [n][d+1], ws [n][k], gs [n][k], ps [d][k+1], dps [d][k+1]
  const int ldx = d + 1, ldp = k + 1;
  float* xs = sm;
  float* ws = xs + n * ldx;
  float* gs = ws + n * k;
  float* ps = gs + n * k;
  float* dps = ps + d * ldp;
  for (int e = threadIdx.x; e < n * k; e += 256) ws[e] = ld(W + e);
  constexpr int MAXW = 64;  // dW elements per thread (n*k <= 256*MAXW)
  float dw[MAXW];
#pragma unroll
  for (int i = 0; i < MAXW; ++i) dw[i] = 0.f;
  const int off = emit0 ? d : 0;
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    __syncthreads();
    const T* Xb = X + (int64_t)b * n * d;
    const T* gb = dout + (int64_t)b * dstride;
    for (int e = threadIdx.x; e < n * d; e += 256) xs[(e / d) * ldx + (e % d)] = ld(Xb + e);
    for (int e = threadIdx.x; e < n * k; e += 256) gs[e] = ld(gb + off + e);
    __syncthreads();
    for (int e = threadIdx.x; e < d * k; e += 256) {
      const int a = e / k, c = e % k;
      float s = 0.f, t = 0.f;
      for (int j = 0; j < n; ++j) {
        s = fmaf(xs[j * ldx + a], ws[j * k + c], s);
        t = fmaf(xs[j * ldx + a], gs[j * k + c], t);
      }
      ps[a * ldp + c] = ld_round<T>(s);
      dps[a * ldp + c] = ld_round<T>(t);
    }
    __syncthreads();
    DXT* dXb = dX + (int64_t)b * n * d;
    for (int e = threadIdx.x; e < n * d; e += 256) {
      const int j = e / d, a = e % d;
      float s = 0.f;
      for (int c = 0; c < k; ++c) s = fmaf(gs[j * k + c], ps[a * ldp + c], s);
      for (int c = 0; c < k; ++c) s = fmaf(ws[j * k + c], dps[a * ldp + c], s);
      if (addend) s += addend[(int64_t)b * n * d + e];
      if (emit0 && j == 0) s += ld(gb + a);
      st(dXb + e, s);
    }
#pragma unroll
    for (int i = 0; i < MAXW; ++i) {
      const int e = threadIdx.x + i * 256;
      if (e < n * k) {
        const int j = e / k, c = e % k;
        float s = 0.f;
        for (int a = 0; a < d; ++a) s = fmaf(xs[j * ldx + a], dps[a * ldp + c], s);
        dw[i] += s;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < MAXW; ++i) {
    const int e = threadIdx.x + i * 256;
    if (e < n * k) dw_part[(int64_t)blockIdx.x * n * k + e] = dw[i];
  }
}

__global__ __launch_bounds__(256) void sum_parts_kernel(const float* __restrict__ part, int parts,
                                                        int64_t len, float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= len) return;
  float s = 0.f;
  for (int p = 0; p < parts; ++p) s += part[(int64_t)p * len + i];
  out[i] = s;
}

constexpr int FM_BWD_BLOCKS = 512;

size_t fm_bwd_workspace(int n, int k) { return (size_t)FM_BWD_BLOCKS * n * k * sizeof(float); }

static hipError_t set_lds(const void* fn, size_t bytes) {
  if (bytes > 65536) LAT_HIP_CHECK(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes));
  return hipSuccess;
}

hipError_t dot_fwd(DType dt, const void* X, int B, int n, int d, void* out, int64_t ostride,
                   int emit0, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const size_t lds = (size_t)n * (d + 1) * 4;
  if (dt == DT_BF16) {
    auto fn = dot_fwd_kernel<bf16_t>;
    if (set_lds((const void*)fn, lds) != hipSuccess) return hipErrorInvalidValue;
    fn<<<B, 256, lds, s>>>((const bf16_t*)X, n, d, (bf16_t*)out, ostride, emit0);
  } else {
    auto fn = dot_fwd_kernel<float>;
    if (set_lds((const void*)fn, lds) != hipSuccess) return hipErrorInvalidValue;
    fn<<<B, 256, lds, s>>>((const float*)X, n, d, (float*)out, ostride, emit0);
  }
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t dot_bwd(DType dt, const void* X, int B, int n, int d, const void* dout,
                   int64_t dstride, int emit0, void* dX, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const size_t lds = ((size_t)n * (d + 1) + (size_t)n * (n + 1)) * 4;
  if (dt == DT_BF16) {
    auto fn = dot_bwd_kernel<bf16_t>;
    if (set_lds((const void*)fn, lds) != hipSuccess) return hipErrorInvalidValue;
    fn<<<B, 256, lds, s>>>((const bf16_t*)X, n, d, (const bf16_t*)dout, dstride, emit0, (bf16_t*)dX);
  } else {
    auto fn = dot_bwd_kernel<float>;
    if (set_lds((const void*)fn, lds) != hipSuccess) return hipErrorInvalidValue;
    fn<<<B, 256, lds, s>>>((const float*)X, n, d, (const float*)dout, dstride, emit0, (float*)dX);
  }
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

size_t dot_lds_bytes(int n, int d) { return ((size_t)n * (d + 1) + (size_t)n * (n + 1)) * 4; }
size_t fm_lds_bytes(int n, int d, int k) {
  return ((size_t)n * (d + 1) + 2 * (size_t)n * k + 2 * (size_t)d * (k + 1)) * 4;
}

hipError_t fm_fwd(DType dt, const void* X, const void* W, int B, int n, int d, int k, void* out,
                  int64_t ostride, int emit0, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const size_t lds = ((size_t)n * (d + 1) + (size_t)n * k + (size_t)d * (k + 1)) * 4;
  if (dt == DT_BF16) {
    auto fn = fm_fwd_kernel<bf16_t>;
    if (set_lds((const void*)fn, lds) != hipSuccess) return hipErrorInvalidValue;
    fn<<<B, 256, lds, s>>>((const bf16_t*)X, (const bf16_t*)W, n, d, k, (bf16_t*)out, ostride, emit0);
  } else {
    auto fn = fm_fwd_kernel<float>;
    if (set_lds((const void*)fn, lds) != hipSuccess) return hipErrorInvalidValue;
    fn<<<B, 256, lds, s>>>((const float*)X, (const float*)W, n, d, k, (float*)out, ostride, emit0);
  }
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t fm_bwd(DType dt, const void* X, const void* W, int B, int n, int d, int k,
                  const void* dout, int64_t dstride, int emit0, const float* addend,
                  void* dX, DType dxt, float* dW, void* ws, hipStream_t s) {
  const int blocks = B < FM_BWD_BLOCKS ? (B > 0 ? B : 1) : FM_BWD_BLOCKS;
  const size_t lds = fm_lds_bytes(n, d, k);
  float* part = (float*)ws;
  if (B > 0) {
#define LAT_FMB(TT, DT2)                                                                         \
  {                                                                                              \
    auto fn = fm_bwd_kernel<TT, DT2>;                                                            \
    if (set_lds((const void*)fn, lds) != hipSuccess) return hipErrorInvalidValue;                \
    fn<<<blocks, 256, lds, s>>>((const TT*)X, (const TT*)W, B, n, d, k, (const TT*)dout, dstride, \
                                emit0, addend, (DT2*)dX, part);                                  \
  }
    if (dt == DT_BF16 && dxt == DT_BF16) LAT_FMB(bf16_t, bf16_t)
    else if (dt == DT_BF16) LAT_FMB(bf16_t, float)
    else if (dxt == DT_BF16) LAT_FMB(float, bf16_t)
    else LAT_FMB(float, float)
#undef LAT_FMB
    LAT_LAUNCH_CHECK();
  }
  const int64_t len = (int64_t)n * k;
  sum_parts_kernel<<<cdiv(len, 256), 256, 0, s>>>(part, B > 0 ? blocks : 0, len, dW);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
