// Factorization-machine block O_b = X_b (X_b^T W) (Section 3.3.2) on bf16 MFMA
// (v_mfma_f32_32x32x16_bf16), forward and backward, for n <= 96 vectors,
// d in {64, 128}, rank k in {32, 64}.
//
// Each block of 8 waves loops over samples.  A sample's X [n, d] is read once
// with coalesced 4-byte loads (8 rows x 2 columns per thread) into registers
// one sample ahead (the next sample's loads are in flight while the current
// one is computed), transposed in registers, and staged in LDS twice --
// row-major X[j][a] and transposed X^T[a][j] -- so every MFMA operand is read
// as k-contiguous 16-byte fragments.  Storage rounding matches the rest of the step: P = X^T W and
// dP = X^T G are rounded to bf16 before use, O and dX are stored in bf16.
//   forward : P = X^T W (contraction over j), O = X P (over a)
//   backward: P, dP and dP^T (= G^T X, the dW operand) share the staged
//             fragments; dX = [G | W] [P | dP]^T is one contraction over 2k;
//             dW += X dP accumulates in the waves' registers across the
//             block's samples (fixed order), and the per-block partials are
//             summed in block order afterwards.
#include "common.h"
#include "kernels.h"
#include "mfma_tile.h"

namespace lat {

template <int NP, int D, int K>
__global__ __launch_bounds__(512) void fm_fwd_mfma_kernel(const bf16_t* __restrict__ X,
                                                          const bf16_t* __restrict__ W, int B,
                                                          int n, bf16_t* __restrict__ out,
                                                          int64_t ostride, int emit0) {
  constexpr int LX = D + 8, LT = NP + 8, LP = D + 8, LR = K + 8;
  __shared__ __attribute__((aligned(16))) bf16_t Xs[NP * LX];
  __shared__ __attribute__((aligned(16))) bf16_t XT[D * LT];
  __shared__ __attribute__((aligned(16))) bf16_t PT[K * LP];
  __shared__ __attribute__((aligned(16))) bf16_t WR[NP * LR];
  __shared__ __attribute__((aligned(16))) bf16_t WT[K * LT];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  {
    Stager<NP, K, 512> sw;
    sw.load(W, K, n);
    sw.store(WR, LR, WT, LT);
  }
  const int off = emit0 ? D : 0;
  Stager<NP, D, 512> sx;
  if (blockIdx.x < B) sx.load(X + (int64_t)blockIdx.x * n * D, D, n);
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    sx.store(Xs, LX, XT, LT);
    __syncthreads();
    // the next sample's X is in flight while this one is computed
    if (b + (int)gridDim.x < B) sx.load(X + (int64_t)(b + gridDim.x) * n * D, D, n);
    // P[a][c] = sum_j X^T[a][j] W^T[c][j]; tile (ta, tc) per wave
    constexpr int PT_TILES = (D / 32) * (K / 32);
    for (int t = w; t < PT_TILES; t += 8) {
      const int ta = t / (K / 32), tc = t % (K / 32);
      f32x16 acc;
      zero16(acc);
      mfma_tile<NP>(acc, XT + ta * 32 * LT, LT, WT + tc * 32 * LT, LT);
      const int c = tc * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) PT[c * LP + ta * 32 + frag_row(r)] = f2bf(acc[r]);
    }
    __syncthreads();
    // O[j][c] = sum_a X[j][a] P^T[c][a]
    bf16_t* ob = out + (int64_t)b * ostride;
    constexpr int O_TILES = (NP / 32) * (K / 32);
    for (int t = w; t < O_TILES; t += 8) {
      const int tj = t / (K / 32), tc = t % (K / 32);
      f32x16 acc;
      zero16(acc);
      mfma_tile<D>(acc, Xs + tj * 32 * LX, LX, PT + tc * 32 * LP, LP);
      const int c = tc * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = tj * 32 + frag_row(r);
        if (j < n) ob[off + j * K + c] = f2bf(acc[r]);
      }
    }
    if (emit0)
      for (int a = threadIdx.x; a < D; a += blockDim.x) ob[a] = Xs[a];
    __syncthreads();
  }
}

// Backward.  dX_f32 (optional) receives the unrounded fp32 dX instead of dX.
template <int NP, int D, int K>
__global__ __launch_bounds__(512) void fm_bwd_mfma_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int B, int n,
    const bf16_t* __restrict__ dout, int64_t dstride, int emit0, const float* __restrict__ addend,
    bf16_t* __restrict__ dX, float* __restrict__ dX_f32, float* __restrict__ dw_part) {
  constexpr int LX = D + 8, LT = NP + 8, LG = 2 * K + 8, LPD = 2 * K + 8, LDT = D + 8;
  __shared__ __attribute__((aligned(16))) bf16_t Xs[NP * LX];
  __shared__ __attribute__((aligned(16))) bf16_t XT[D * LT];
  __shared__ __attribute__((aligned(16))) bf16_t PT_[K * LDT];  // dP^T [K][LDT]
  __shared__ __attribute__((aligned(16))) bf16_t GW[NP * LG];   // [j][ G (K) | W (K) ]
  __shared__ __attribute__((aligned(16))) bf16_t GT[K * LT];
  __shared__ __attribute__((aligned(16))) bf16_t WT[K * LT];
  __shared__ __attribute__((aligned(16))) bf16_t PD[D * LPD];   // [a][ P (K) | dP (K) ]
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  {
    Stager<NP, K, 512> sw;
    sw.load(W, K, n);
    sw.store(GW + K, LG, WT, LT);
  }
  constexpr int DW_TILES = (NP / 32) * (K / 32);
  f32x16 dw[(DW_TILES + 7) / 8];
#pragma unroll
  for (int i = 0; i < (DW_TILES + 7) / 8; ++i) zero16(dw[i]);
  const int off = emit0 ? D : 0;
  Stager<NP, D, 512> sx;
  Stager<NP, K, 512> sg;
  if (blockIdx.x < B) {
    sx.load(X + (int64_t)blockIdx.x * n * D, D, n);
    sg.load(dout + (int64_t)blockIdx.x * dstride + off, K, n);
  }
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    const bf16_t* gb = dout + (int64_t)b * dstride;
    sx.store(Xs, LX, XT, LT);
    sg.store(GW, LG, GT, LT);
    __syncthreads();
    // the next sample's X and G are in flight while this one is computed
    if (b + (int)gridDim.x < B) {
      sx.load(X + (int64_t)(b + gridDim.x) * n * D, D, n);
      sg.load(dout + (int64_t)(b + gridDim.x) * dstride + off, K, n);
    }
    // P = X^T W and dP = X^T G into PD[a][P | dP], and dP^T[c][a] = G^T X
    // into DT (the dW operand), all rounded to bf16
    constexpr int P_TILES = (D / 32) * (K / 32);
    bf16_t* DT = PT_;
    for (int t = w; t < 3 * P_TILES; t += 8) {
      const int which = t / P_TILES, tt = t % P_TILES;
      f32x16 acc;
      zero16(acc);
      if (which < 2) {
        const int ta = tt / (K / 32), tc = tt % (K / 32);
        mfma_tile<NP>(acc, XT + ta * 32 * LT, LT, (which ? GT : WT) + tc * 32 * LT, LT);
        const int c = tc * 32 + (lane & 31) + which * K;
#pragma unroll
        for (int r = 0; r < 16; ++r) PD[(ta * 32 + frag_row(r)) * LPD + c] = f2bf(acc[r]);
      } else {
        const int tc = tt / (D / 32), ta = tt % (D / 32);
        mfma_tile<NP>(acc, GT + tc * 32 * LT, LT, XT + ta * 32 * LT, LT);
        const int a = ta * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) DT[(tc * 32 + frag_row(r)) * LDT + a] = f2bf(acc[r]);
      }
    }
    __syncthreads();
    // dX[j][a] = sum_kk GW[j][kk] PD[a][kk]  (+ addend, + slot-0 gradient)
    constexpr int DX_TILES = (NP / 32) * (D / 32);
    for (int t = w; t < DX_TILES; t += 8) {
      const int tj = t / (D / 32), ta = t % (D / 32);
      f32x16 acc;
      zero16(acc);
      mfma_tile<2 * K>(acc, GW + tj * 32 * LG, LG, PD + ta * 32 * LPD, LPD);
      const int a = ta * 32 + (lane & 31);
      const int64_t sbase = (int64_t)b * n * D;  // this sample's [n, D] block
      const float g0 = (emit0 && tj == 0) ? bf2f(gb[a]) : 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = tj * 32 + frag_row(r);
        if (j < n) {
          float v = acc[r];
          const int e = j * D + a;
          if (addend) v += addend[sbase + e];
          if (j == 0) v += g0;
          if (dX_f32) dX_f32[sbase + e] = v;
          else dX[sbase + e] = f2bf(v);
        }
      }
    }
    // dW[j][c] += sum_a X[j][a] dP^T[c][a]
    for (int t = w, i = 0; t < DW_TILES; t += 8, ++i) {
      const int tj = t / (K / 32), tc = t % (K / 32);
      mfma_tile<D>(dw[i], Xs + tj * 32 * LX, LX, DT + tc * 32 * LDT, LDT);
    }
    __syncthreads();
  }
  for (int t = w, i = 0; t < DW_TILES; t += 8, ++i) {
    const int tj = t / (K / 32), tc = t % (K / 32);
    const int c = tc * 32 + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = tj * 32 + frag_row(r);
      if (j < n) dw_part[((int64_t)blockIdx.x * n + j) * K + c] = dw[i][r];
    }
  }
}

__global__ __launch_bounds__(256) void sum_parts_unrolled_kernel(const float* __restrict__ part,
                                                                 int parts, int64_t len,
                                                                 float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= len) return;
  float s = 0.f;
  int p = 0;
  for (; p + 8 <= parts; p += 8) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = part[(int64_t)(p + q) * len + i];
#pragma unroll
    for (int q = 0; q < 8; ++q) s += v[q];
  }
  for (; p < parts; ++p) s += part[(int64_t)p * len + i];
  out[i] = s;
}

constexpr int FM_MFMA_BLOCKS = 256;

bool fm_mfma_supported(int n, int d, int k) {
  if (n < 1) return false;
  if (k == 32) return n <= 96 && (d == 64 || d == 128);
  if (k == 64) return n <= 64 && d == 128;
  return false;
}

size_t fm_mfma_bwd_workspace(int n, int k) { return (size_t)FM_MFMA_BLOCKS * n * k * sizeof(float); }

template <int NP, int D, int K>
static hipError_t fm_mfma_launch(bool fwd, const void* X, const void* W, int B, int n, void* out,
                                 int64_t ostride, int emit0, const void* dout, int64_t dstride,
                                 const float* addend, void* dX, float* dX_f32, float* dW,
                                 void* ws, hipStream_t s) {
  const int blocks = B < FM_MFMA_BLOCKS ? (B > 0 ? B : 1) : FM_MFMA_BLOCKS;
  if (fwd) {
    if (B == 0) return hipSuccess;
    // the forward fits two blocks per compute unit
    const int fblocks = B < 2 * FM_MFMA_BLOCKS ? B : 2 * FM_MFMA_BLOCKS;
    fm_fwd_mfma_kernel<NP, D, K><<<fblocks, 512, 0, s>>>((const bf16_t*)X, (const bf16_t*)W, B, n,
                                                        (bf16_t*)out, ostride, emit0);
    LAT_LAUNCH_CHECK();
    return hipSuccess;
  }
  float* part = (float*)ws;
  if (B > 0) {
    fm_bwd_mfma_kernel<NP, D, K><<<blocks, 512, 0, s>>>(
        (const bf16_t*)X, (const bf16_t*)W, B, n, (const bf16_t*)dout, dstride, emit0, addend,
        (bf16_t*)dX, dX_f32, part);
    LAT_LAUNCH_CHECK();
  }
  const int64_t len = (int64_t)n * K;
  sum_parts_unrolled_kernel<<<cdiv(len, 256), 256, 0, s>>>(part, B > 0 ? blocks : 0, len, dW);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t fm_mfma(bool fwd, const void* X, const void* W, int B, int n, int d, int k, void* out,
                   int64_t ostride, int emit0, const void* dout, int64_t dstride,
                   const float* addend, void* dX, float* dX_f32, float* dW, void* ws,
                   hipStream_t s) {
#define LAT_FMM(NPV, DV, KV)                                                                    \
  if (n <= NPV && d == DV && k == KV)                                                           \
    return fm_mfma_launch<NPV, DV, KV>(fwd, X, W, B, n, out, ostride, emit0, dout, dstride,     \
                                       addend, dX, dX_f32, dW, ws, s);
  LAT_FMM(32, 128, 32) LAT_FMM(64, 128, 32) LAT_FMM(96, 128, 32)
  LAT_FMM(32, 64, 32) LAT_FMM(64, 64, 32) LAT_FMM(96, 64, 32)
  LAT_FMM(32, 128, 64) LAT_FMM(64, 128, 64)
#undef LAT_FMM
  set_error("FM MFMA path: unsupported shape n=%d d=%d k=%d", n, d, k);
  return hipErrorInvalidValue;
}

}  // namespace lat
