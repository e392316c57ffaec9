// Stacked interaction of the deep workload: L fusion blocks (DHEN/Wukong,
// Section 3.3.2) of
//   F = X (X^T W)                      (FM block, rank k)
//   H_F = vec(F) A^T                   (its projection to nv - nL vectors of dim d, no bias)
//   H_L = L X                          (linear compression block, nL vectors; nL = 0: none)
//   u = [H_F; H_L] + R,  R = C X or X  (residual; C a linear projection)
//   X' = LayerNorm_gamma(u)            (per vector over d, gain only, fp32 math)
// and the exact backward.  The contractions run on the bf16 MFMA GEMM (the
// projection vec(F) A^T optionally in FP8 e4m3 with row-wise scales, the
// backward then taking it as the identity of its bf16 operands)
// (batched over samples where they are per-sample products, K-segmented
// where they sum over samples); LayerNorm forward/backward are one wave per
// vector.  Storage points: P = X^T W, F, X' and the GEMM operand copy of the
// LayerNorm input gradient are bf16; H, R, u, dX between layers are fp32.
#include "common.h"
#include "kernels.h"

namespace lat {

// The weight gradients summed over samples (dW, dC) have tiny outputs and a
// contraction over B*d: split K widely so the whole chip takes part.
constexpr int SAMPLE_SUM_SPLITS = 256;

// ---------------------------------------------------------------------------
// LayerNorm over d (= 64*E elements per vector), one wave per vector
// ---------------------------------------------------------------------------
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// u = H[v] + res[v]; out[v] = bf16(gamma * (u - mean) * rstd); saves mean, rstd.
// Vector v = b*nv + i lives at H + v*d, res + v*d, out + b*out_stride + i*d.
template <int E, typename RT>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const float* __restrict__ H,
                                                     const RT* __restrict__ res,
                                                     const float* __restrict__ gamma, int64_t nvec,
                                                     int nv, float eps, bf16_t* __restrict__ out,
                                                     int64_t out_stride, float* __restrict__ mean,
                                                     float* __restrict__ rstd) {
  constexpr int D = 64 * E;
  const int lane = threadIdx.x & 63;
  const int64_t v = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (v >= nvec) return;
  float u[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int a = lane + 64 * e;
    u[e] = H[v * D + a] + ld(res + v * D + a);
  }
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) s += u[e];
  const float mu = wave_sum(s) / D;
  float q = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) q += (u[e] - mu) * (u[e] - mu);
  const float r = 1.f / sqrtf(wave_sum(q) / D + eps);
  const int64_t b = v / nv, i = v % nv;
  bf16_t* o = out + b * out_stride + i * D;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int a = lane + 64 * e;
    o[a] = f2bf(gamma[a] * (u[e] - mu) * r);
  }
  if (lane == 0) {
    mean[v] = mu;
    rstd[v] = r;
  }
}

// du = rstd * (dxh - mean(dxh) - xhat * mean(dxh * xhat)), dxh = dY * gamma;
// du (fp32) and its bf16 copy; per-block partial sums of dY * xhat (dgamma).
// Persistent grid: wave w of block z handles vectors z*4 + w, + 4*gridDim, ...
template <int E, typename RT, typename YT>
__global__ __launch_bounds__(256) void ln_bwd_kernel(
    const float* __restrict__ H, const RT* __restrict__ res, const float* __restrict__ gamma,
    const float* __restrict__ mean, const float* __restrict__ rstd, const YT* __restrict__ dY,
    int64_t dy_stride, int64_t nvec, int nv, float* __restrict__ du, bf16_t* __restrict__ duR,
    float* __restrict__ dgamma_part) {
  constexpr int D = 64 * E;
  __shared__ float red[4][D];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float g[E], dg[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    g[e] = gamma[lane + 64 * e];
    dg[e] = 0.f;
  }
  for (int64_t v = (int64_t)blockIdx.x * 4 + w; v < nvec; v += (int64_t)gridDim.x * 4) {
    const float mu = mean[v], r = rstd[v];
    const int64_t b = v / nv, i = v % nv;
    float xh[E], dxh[E];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int a = lane + 64 * e;
      xh[e] = (H[v * D + a] + ld(res + v * D + a) - mu) * r;
      const float dy = ld(dY + b * dy_stride + i * D + a);
      dg[e] += dy * xh[e];
      dxh[e] = dy * g[e];
      s1 += dxh[e];
      s2 += dxh[e] * xh[e];
    }
    const float m1 = wave_sum(s1) / D, m2 = wave_sum(s2) / D;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int a = lane + 64 * e;
      const float x = r * (dxh[e] - m1 - xh[e] * m2);
      du[v * D + a] = x;
      duR[v * D + a] = f2bf(x);
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) red[w][lane + 64 * e] = dg[e];
  __syncthreads();
  for (int a = threadIdx.x; a < D; a += 256)
    dgamma_part[(int64_t)blockIdx.x * D + a] = red[0][a] + red[1][a] + red[2][a] + red[3][a];
}

// out[i] = sum over p of part[p][i]: one block per output, thread t adds
// parts t, t + 256, ..., then a fixed-shape tree (deterministic order).
__global__ __launch_bounds__(256) void stack_sum_parts_kernel(const float* __restrict__ part,
                                                              int parts, int64_t len,
                                                              float* __restrict__ out) {
  __shared__ float red[256];
  const int64_t i = blockIdx.x;
  float s = 0.f;
  for (int p = threadIdx.x; p < parts; p += 256) s += part[(int64_t)p * len + i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[i] = red[0];
}

constexpr int LN_BWD_BLOCKS = 1024;

// ---------------------------------------------------------------------------
// plan of the saved state (forward -> backward) and the backward scratch
// ---------------------------------------------------------------------------
static size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

StackPlan stack_plan(const StackShape& sh, int B) {
  StackPlan p{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t r = off; off += al(bytes); return r; };
  const int64_t nvd = (int64_t)sh.nv * sh.d;
  for (int l = 0; l < sh.L; ++l) {
    const int n = l == 0 ? sh.n0 : sh.nv;
    p.P[l] = take((size_t)B * sh.d * sh.k * 2);
    p.F[l] = take((size_t)B * n * sh.k * 2);
    p.H[l] = take((size_t)B * nvd * 4);
    p.mean[l] = take((size_t)B * sh.nv * 4);
    p.rstd[l] = take((size_t)B * sh.nv * 4);
    p.Xn[l] = l + 1 < sh.L ? take((size_t)B * nvd * 2) : 0;
  }
  p.R0 = sh.has_C0 ? take((size_t)B * nvd * 4) : 0;
  p.state_bytes = off;
  // backward scratch
  const int nmax = sh.n0 > sh.nv ? sh.n0 : sh.nv;
  p.du = take((size_t)B * nvd * 4);
  p.duR = take((size_t)B * nvd * 2);
  p.dF = take((size_t)B * nmax * sh.k * 2);
  p.dP = take((size_t)B * sh.d * sh.k * 2);
  p.dXf = take((size_t)B * nmax * sh.d * 4);
  p.dgp = take((size_t)LN_BWD_BLOCKS * sh.d * 4);
  // split-K partials of the sample-summed weight gradients
  size_t gw = 0;
  for (int l = 0; l < sh.L; ++l) {
    const int n = l == 0 ? sh.n0 : sh.nv;
    GemmArgs g;
    g.max_splits = 16;
    g.M = (int)nvd; g.N = n * sh.k; g.K = B;
    gw = gw > gemm_workspace(g) ? gw : gemm_workspace(g);
    g.max_splits = SAMPLE_SUM_SPLITS;
    g.M = n; g.N = sh.k; g.K = B * sh.d;
    gw = gw > gemm_workspace(g) ? gw : gemm_workspace(g);
    if (l == 0 && sh.has_C0) {
      g.M = sh.nv; g.N = sh.n0; g.K = B * sh.d;
      gw = gw > gemm_workspace(g) ? gw : gemm_workspace(g);
    }
    if (sh.nL > 0) {
      g.M = sh.nL; g.N = n; g.K = B * sh.d;
      gw = gw > gemm_workspace(g) ? gw : gemm_workspace(g);
    }
  }
  p.gemm_ws = take(gw);
  if (sh.fp8) {
    // codes of the widest vec(F) and A (layer 0 when n0 > nv), reused by every layer
    const int nmx = sh.n0 > sh.nv ? sh.n0 : sh.nv;
    const size_t ldq = ((size_t)nmx * sh.k + 15) / 16 * 16;
    const size_t rowsA = (size_t)(sh.nv - sh.nL) * sh.d;
    p.qF = take((size_t)B * ldq);
    p.sF = take((size_t)B * 4);
    p.qA = take(rowsA * ldq);
    p.sA = take(rowsA * 4);
  }
  p.total_bytes = off;
  return p;
}

#define STK_CHECK(...)                  \
  do {                                  \
    hipError_t e_ = (__VA_ARGS__);      \
    if (e_ != hipSuccess) return e_;    \
  } while (0)

template <typename RT>
static hipError_t ln_fwd_launch(int E, const float* H, const RT* res, const float* gamma,
                                int64_t nvec, int nv, float eps, bf16_t* out, int64_t ostride,
                                float* mean, float* rstd, hipStream_t s) {
  const int grid = cdiv(nvec, 4);
  if (E == 1) ln_fwd_kernel<1, RT><<<grid, 256, 0, s>>>(H, res, gamma, nvec, nv, eps, out, ostride, mean, rstd);
  else if (E == 2) ln_fwd_kernel<2, RT><<<grid, 256, 0, s>>>(H, res, gamma, nvec, nv, eps, out, ostride, mean, rstd);
  else ln_fwd_kernel<4, RT><<<grid, 256, 0, s>>>(H, res, gamma, nvec, nv, eps, out, ostride, mean, rstd);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

template <typename RT, typename YT>
static hipError_t ln_bwd_launch(int E, const float* H, const RT* res, const float* gamma,
                                const float* mean, const float* rstd, const YT* dY,
                                int64_t dy_stride, int64_t nvec, int nv, float* du, bf16_t* duR,
                                float* dgp, float* dgamma, int d, hipStream_t s) {
  const int grid = (int)(nvec < (int64_t)LN_BWD_BLOCKS * 4 ? cdiv(nvec, 4) : LN_BWD_BLOCKS);
  if (E == 1) ln_bwd_kernel<1, RT, YT><<<grid, 256, 0, s>>>(H, res, gamma, mean, rstd, dY, dy_stride, nvec, nv, du, duR, dgp);
  else if (E == 2) ln_bwd_kernel<2, RT, YT><<<grid, 256, 0, s>>>(H, res, gamma, mean, rstd, dY, dy_stride, nvec, nv, du, duR, dgp);
  else ln_bwd_kernel<4, RT, YT><<<grid, 256, 0, s>>>(H, res, gamma, mean, rstd, dY, dy_stride, nvec, nv, du, duR, dgp);
  LAT_LAUNCH_CHECK();
  stack_sum_parts_kernel<<<d, 256, 0, s>>>(dgp, grid, d, dgamma);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

bool stack_supported(const StackShape& sh) {
  return sh.L >= 1 && sh.L <= 8 && (sh.d == 64 || sh.d == 128 || sh.d == 256) && sh.k >= 1 &&
         sh.n0 >= 1 && sh.nv >= 1 && (sh.has_C0 || sh.n0 == sh.nv) && sh.k % 8 == 0 &&
         sh.n0 % 2 == 0 && sh.nv % 2 == 0 && sh.nL >= 0 && sh.nL < sh.nv;
}

// Forward.  X [B, n0, d] bf16; out rows (stride out_stride) receive vec(X_L).
hipError_t stack_fwd(const StackShape& sh, const StackLayer* Ls, int B, const void* X, void* out,
                     int64_t out_stride, void* state, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const StackPlan p = stack_plan(sh, B);
  char* base = (char*)state;
  const int d = sh.d, k = sh.k, nv = sh.nv;
  const int64_t nvd = (int64_t)nv * d;
  const bf16_t* Xl = (const bf16_t*)X;
  for (int l = 0; l < sh.L; ++l) {
    const int n = l == 0 ? sh.n0 : nv;
    bf16_t* P = (bf16_t*)(base + p.P[l]);
    bf16_t* F = (bf16_t*)(base + p.F[l]);
    float* H = (float*)(base + p.H[l]);
    // P_b = round(X_b^T W): M = d (a), N = k (c), K = n (j)
    GemmArgs g1;
    g1.A = Xl; g1.lda = d; g1.ta = 1; g1.sA = (int64_t)n * d;
    g1.B = Ls[l].W; g1.ldb = k; g1.tb = 1;
    g1.C = P; g1.ldc = k; g1.c_dt = DT_BF16; g1.sC = (int64_t)d * k;
    g1.M = d; g1.N = k; g1.K = n; g1.batch = B;
    STK_CHECK(gemm(g1, nullptr, s));
    // F_b = round(X_b P_b): M = n (j), N = k (c), K = d (a)
    GemmArgs g2;
    g2.A = Xl; g2.lda = d; g2.sA = (int64_t)n * d;
    g2.B = P; g2.ldb = k; g2.tb = 1; g2.sB = (int64_t)d * k;
    g2.C = F; g2.ldc = k; g2.c_dt = DT_BF16; g2.sC = (int64_t)n * k;
    g2.M = n; g2.N = k; g2.K = d; g2.batch = B;
    STK_CHECK(gemm(g2, nullptr, s));
    // H_F = vec(F) A^T: M = B, N = (nv - nL)*d, K = n*k (the first nv - nL vectors of H)
    const int nF = nv - sh.nL;
    if (sh.fp8) {
      // FP8 linear layer (Section 3.5.2): vec(F) quantised per sample and A
      // per output unit (one launch), then the e4m3 product with both scales
      const int64_t ldq = ((int64_t)n * k + 15) / 16 * 16;
      uint8_t* qF = (uint8_t*)(base + p.qF);
      uint8_t* qA = (uint8_t*)(base + p.qA);
      float* sF = (float*)(base + p.sF);
      float* sA = (float*)(base + p.sA);
      const Fp8RowJob jobs[2] = {{F, (int64_t)n * k, B, n * k, qF, ldq, sF},
                                 {Ls[l].A, (int64_t)n * k, nF * d, n * k, qA, ldq, sA}};
      STK_CHECK(fp8_quantize_rows(DT_BF16, jobs, 2, s));
      STK_CHECK(gemm_fp8(qF, ldq, sF, 1, qA, ldq, sA, 1, nullptr, H, DT_F32, nvd, B, nF * d, n * k, 0,
                         sh.fp8 == 2, s));
    } else {
      GemmArgs g3;
      g3.A = F; g3.lda = (int64_t)n * k;
      g3.B = Ls[l].A; g3.ldb = (int64_t)n * k;
      g3.C = H; g3.ldc = nvd; g3.c_dt = DT_F32;
      g3.M = B; g3.N = nF * d; g3.K = n * k;
      STK_CHECK(gemm(g3, nullptr, s));
    }
    if (sh.nL > 0) {
      // H_L,b = L X_b (the last nL vectors of H): M = nL, N = d, K = n
      GemmArgs gl;
      gl.A = Ls[l].Lc; gl.lda = n;
      gl.B = Xl; gl.ldb = d; gl.tb = 1; gl.sB = (int64_t)n * d;
      gl.C = H + (int64_t)nF * d; gl.ldc = d; gl.c_dt = DT_F32; gl.sC = nvd;
      gl.M = sh.nL; gl.N = d; gl.K = n; gl.batch = B;
      STK_CHECK(gemm(gl, nullptr, s));
    }
    bf16_t* Xn = l + 1 < sh.L ? (bf16_t*)(base + p.Xn[l]) : (bf16_t*)out;
    const int64_t ostr = l + 1 < sh.L ? nvd : out_stride;
    float* mean = (float*)(base + p.mean[l]);
    float* rstd = (float*)(base + p.rstd[l]);
    if (l == 0 && sh.has_C0) {
      // R_b = C X_b: M = nv (v), N = d (a), K = n0 (u)
      float* R = (float*)(base + p.R0);
      GemmArgs g4;
      g4.A = Ls[0].C; g4.lda = sh.n0;
      g4.B = Xl; g4.ldb = d; g4.tb = 1; g4.sB = (int64_t)sh.n0 * d;
      g4.C = R; g4.ldc = d; g4.c_dt = DT_F32; g4.sC = nvd;
      g4.M = nv; g4.N = d; g4.K = sh.n0; g4.batch = B;
      STK_CHECK(gemm(g4, nullptr, s));
      STK_CHECK(ln_fwd_launch<float>(d / 64, H, R, Ls[l].gamma, (int64_t)B * nv, nv, sh.eps, Xn,
                                     ostr, mean, rstd, s));
    } else {
      STK_CHECK(ln_fwd_launch<bf16_t>(d / 64, H, Xl, Ls[l].gamma, (int64_t)B * nv, nv, sh.eps,
                                      Xn, ostr, mean, rstd, s));
    }
    Xl = Xn;
  }
  return hipSuccess;
}

// Backward.  d_out rows (stride d_out_stride, bf16) = dL/dvec(X_L); writes
// dX [B, n0, d] (bf16) and every layer's dW, dA, dC, dgamma.
hipError_t stack_bwd(const StackShape& sh, const StackLayer* Ls, int B, const void* X,
                     const void* d_out, int64_t d_out_stride, void* dX, void* state,
                     hipStream_t s) {
  const StackPlan p = stack_plan(sh, B);
  char* base = (char*)state;
  const int d = sh.d, k = sh.k, nv = sh.nv;
  const int64_t nvd = (int64_t)nv * d;
  float* du = (float*)(base + p.du);
  bf16_t* duR = (bf16_t*)(base + p.duR);
  bf16_t* dF = (bf16_t*)(base + p.dF);
  bf16_t* dP = (bf16_t*)(base + p.dP);
  float* dXf = (float*)(base + p.dXf);
  const float* dY = dXf;
  float* dgp = (float*)(base + p.dgp);
  void* gws = base + p.gemm_ws;
  for (int l = sh.L - 1; l >= 0; --l) {
    const int n = l == 0 ? sh.n0 : nv;
    const bf16_t* Xl = l == 0 ? (const bf16_t*)X : (const bf16_t*)(base + p.Xn[l - 1]);
    const bf16_t* P = (const bf16_t*)(base + p.P[l]);
    const bf16_t* F = (const bf16_t*)(base + p.F[l]);
    const float* H = (const float*)(base + p.H[l]);
    const float* mean = (const float*)(base + p.mean[l]);
    const float* rstd = (const float*)(base + p.rstd[l]);
    const int64_t nvec = (int64_t)B * nv;
    // LayerNorm backward (dY: bf16 top-input gradient for the last layer, fp32 after)
    const bool c_res = l == 0 && sh.has_C0;
    if (l == sh.L - 1) {
      if (c_res)
        STK_CHECK(ln_bwd_launch<float, bf16_t>(d / 64, H, (const float*)(base + p.R0), Ls[l].gamma, mean, rstd,
                                               (const bf16_t*)d_out, d_out_stride, nvec, nv, du, duR, dgp, Ls[l].dgamma, d, s));
      else
        STK_CHECK(ln_bwd_launch<bf16_t, bf16_t>(d / 64, H, Xl, Ls[l].gamma, mean, rstd,
                                                (const bf16_t*)d_out, d_out_stride, nvec, nv, du, duR, dgp, Ls[l].dgamma, d, s));
    } else {
      if (c_res)
        STK_CHECK(ln_bwd_launch<float, float>(d / 64, H, (const float*)(base + p.R0), Ls[l].gamma, mean, rstd,
                                              dY, nvd, nvec, nv, du, duR, dgp, Ls[l].dgamma, d, s));
      else
        STK_CHECK(ln_bwd_launch<bf16_t, float>(d / 64, H, Xl, Ls[l].gamma, mean, rstd, dY, nvd,
                                               nvec, nv, du, duR, dgp, Ls[l].dgamma, d, s));
    }
    // the FM block's part of du: its first nF vectors
    const int nF = nv - sh.nL;
    // dA = duR_F^T vec(F): M = nF*d, N = n*k, K = B
    GemmArgs a1;
    a1.A = duR; a1.lda = nvd; a1.ta = 1;
    a1.B = F; a1.ldb = (int64_t)n * k; a1.tb = 1;
    a1.C = Ls[l].dA; a1.ldc = (int64_t)n * k; a1.c_dt = DT_F32;
    a1.M = nF * d; a1.N = n * k; a1.K = B; a1.max_splits = 16;
    STK_CHECK(gemm(a1, gws, s));
    // dF = round(duR_F A): M = B, N = n*k, K = nF*d
    GemmArgs a2;
    a2.A = duR; a2.lda = nvd;
    a2.B = Ls[l].A; a2.ldb = (int64_t)n * k; a2.tb = 1;
    a2.C = dF; a2.ldc = (int64_t)n * k; a2.c_dt = DT_BF16;
    a2.M = B; a2.N = n * k; a2.K = nF * d;
    STK_CHECK(gemm(a2, nullptr, s));
    // dP_b = round(X_b^T G_b): M = d, N = k, K = n
    GemmArgs f1;
    f1.A = Xl; f1.lda = d; f1.ta = 1; f1.sA = (int64_t)n * d;
    f1.B = dF; f1.ldb = k; f1.tb = 1; f1.sB = (int64_t)n * k;
    f1.C = dP; f1.ldc = k; f1.c_dt = DT_BF16; f1.sC = (int64_t)d * k;
    f1.M = d; f1.N = k; f1.K = n; f1.batch = B;
    STK_CHECK(gemm(f1, nullptr, s));
    // dX_b = G_b P_b^T (+ du for an identity residual): M = n, N = d, K = k
    const bool last = l == 0;
    GemmArgs f2;
    f2.A = dF; f2.lda = k; f2.sA = (int64_t)n * k;
    f2.B = P; f2.ldb = k; f2.sB = (int64_t)d * k;
    f2.C = dXf; f2.ldc = d; f2.c_dt = DT_F32; f2.sC = (int64_t)n * d;
    f2.M = n; f2.N = d; f2.K = k; f2.batch = B;
    if (!c_res) {
      f2.addend = du; f2.ld_add = d; f2.s_add = nvd;
    }
    STK_CHECK(gemm(f2, nullptr, s));
    if (sh.nL > 0) {
      const bf16_t* duL = duR + (int64_t)nF * d;
      // dX_b += L^T duR_L,b: M = n, N = d, K = nL
      GemmArgs l2;
      l2.A = Ls[l].Lc; l2.lda = n; l2.ta = 1;
      l2.B = duL; l2.ldb = d; l2.tb = 1; l2.sB = nvd;
      l2.C = dXf; l2.ldc = d; l2.c_dt = DT_F32; l2.sC = (int64_t)n * d; l2.accumulate = 1;
      l2.M = n; l2.N = d; l2.K = sh.nL; l2.batch = B;
      STK_CHECK(gemm(l2, nullptr, s));
      // dL = sum_b duR_L,b X_b^T: M = nL, N = n, K = (b, a)
      GemmArgs l1;
      l1.A = duL; l1.lda = d; l1.kseg = d; l1.ksA = nvd;
      l1.B = Xl; l1.ldb = d; l1.ksB = (int64_t)n * d;
      l1.C = Ls[l].dL; l1.ldc = n; l1.c_dt = DT_F32;
      l1.M = sh.nL; l1.N = n; l1.K = B * d; l1.max_splits = SAMPLE_SUM_SPLITS;
      STK_CHECK(gemm(l1, gws, s));
    }
    // dX_b += W dP_b^T: M = n, N = d, K = k  (bf16 output when this ends the chain)
    GemmArgs f3;
    f3.A = Ls[l].W; f3.lda = k;
    f3.B = dP; f3.ldb = k; f3.sB = (int64_t)d * k;
    f3.M = n; f3.N = d; f3.K = k; f3.batch = B;
    if (last && !c_res) {
      f3.C = dX; f3.ldc = d; f3.c_dt = DT_BF16; f3.sC = (int64_t)n * d;
      f3.addend = dXf; f3.ld_add = d; f3.s_add = (int64_t)n * d;
    } else {
      f3.C = dXf; f3.ldc = d; f3.c_dt = DT_F32; f3.sC = (int64_t)n * d; f3.accumulate = 1;
    }
    STK_CHECK(gemm(f3, nullptr, s));
    // dW = sum_b X_b dP_b: M = n (j), N = k (c), K = (b, a)
    GemmArgs w1;
    w1.A = Xl; w1.lda = d; w1.kseg = d; w1.ksA = (int64_t)n * d;
    w1.B = dP; w1.ldb = k; w1.tb = 1; w1.ksB = (int64_t)d * k;
    w1.C = Ls[l].dW; w1.ldc = k; w1.c_dt = DT_F32;
    w1.M = n; w1.N = k; w1.K = B * d; w1.max_splits = SAMPLE_SUM_SPLITS;
    STK_CHECK(gemm(w1, gws, s));
    if (c_res) {
      // dC = sum_b duR_b X_b^T: M = nv (v), N = n0 (u), K = (b, a)
      GemmArgs c1;
      c1.A = duR; c1.lda = d; c1.kseg = d; c1.ksA = nvd;
      c1.B = Xl; c1.ldb = d; c1.ksB = (int64_t)sh.n0 * d;
      c1.C = Ls[0].dC; c1.ldc = sh.n0; c1.c_dt = DT_F32;
      c1.M = nv; c1.N = sh.n0; c1.K = B * d; c1.max_splits = SAMPLE_SUM_SPLITS;
      STK_CHECK(gemm(c1, gws, s));
      // dX_b = C^T duR_b + dXf_b: M = n0 (u), N = d (a), K = nv (v)
      GemmArgs c2;
      c2.A = Ls[0].C; c2.lda = sh.n0; c2.ta = 1;
      c2.B = duR; c2.ldb = d; c2.tb = 1; c2.sB = nvd;
      c2.M = sh.n0; c2.N = d; c2.K = nv; c2.batch = B;
      c2.addend = dXf; c2.ld_add = d; c2.s_add = (int64_t)sh.n0 * d;
      if (last) {
        c2.C = dX; c2.ldc = d; c2.c_dt = DT_BF16; c2.sC = (int64_t)sh.n0 * d;
      } else {
        c2.C = dXf; c2.ldc = d; c2.c_dt = DT_F32; c2.sC = (int64_t)sh.n0 * d;
      }
      STK_CHECK(gemm(c2, nullptr, s));
    }
    // the next layer down reads this layer's input gradient (fp32 [B, nv, d]) from dXf;
    // its LayerNorm backward consumes it before anything overwrites dXf
  }
  return hipSuccess;
}

}  // namespace lat
