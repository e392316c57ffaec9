// Dot-product interaction on bf16 MFMA (v_mfma_f32_32x32x16_bf16), forward
// and backward, for n <= 128 vectors and d in {64, 128}: the pairwise inner
// products of a sample's vectors, strict upper triangle packed row by row
// (Section 3.3.2; the DLRM-style baseline of Section 4).
//
// Each block of 4 waves loops over samples; a sample's X [n, d] is loaded
// one sample ahead into registers (the next sample's loads are in flight
// while the current one is computed).
//   forward : X staged row-major; the tiles on or above the diagonal of
//             X X^T are computed, the pairs i < j rounded to bf16 into a
//             packed LDS row, which is then written out with 16-byte stores.
//   backward: the symmetric gradient matrix S (S[i][j] = S[j][i] = g of the
//             pair, zero diagonal) is built in LDS from the packed gradient;
//             dX = S X is one contraction over j, with X staged transposed.
// Accumulation is fp32; the pair values and dX are rounded to bf16 once,
// where they are stored.
#include "common.h"
#include "kernels.h"
#include "mfma_tile.h"

namespace lat {

constexpr int DOT_THREADS = 256;
constexpr int DOT_BLOCKS = 512;

// first packed position of row i (pairs (i, i+1) .. (i, n-1))
__device__ inline int pair_start(int i, int n) { return i * n - i * (i + 1) / 2; }

template <int NP, int D>
__global__ __launch_bounds__(DOT_THREADS) void dot_fwd_mfma_kernel(const bf16_t* __restrict__ X,
                                                                   int B, int n,
                                                                   bf16_t* __restrict__ out,
                                                                   int64_t ostride, int emit0) {
  constexpr int LX = D + 8;
  constexpr int TT = NP / 32;
  constexpr int ZT = TT * (TT + 1) / 2;  // 32x32 tiles on or above the diagonal
  constexpr int PMAX = NP * (NP - 1) / 2;
  __shared__ __attribute__((aligned(16))) bf16_t Xs[NP * LX];
  __shared__ __attribute__((aligned(16))) bf16_t Zp[(PMAX + 7) / 8 * 8];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int P = n * (n - 1) / 2;
  const int off = emit0 ? D : 0;
  Stager<NP, D, DOT_THREADS> sx;
  if (blockIdx.x < B) sx.load(X + (int64_t)blockIdx.x * n * D, D, n);
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    sx.store(Xs, LX, nullptr, 0, n);
    __syncthreads();
    if (b + (int)gridDim.x < B) sx.load(X + (int64_t)(b + gridDim.x) * n * D, D, n);
    for (int t = w; t < ZT; t += DOT_THREADS / 64) {
      int ti = 0, rem = t;
      while (rem >= TT - ti) {
        rem -= TT - ti;
        ++ti;
      }
      const int tj = ti + rem;
      f32x16 acc;
      zero16(acc);
      mfma_tile<D>(acc, Xs + ti * 32 * LX, LX, Xs + tj * 32 * LX, LX);
      const int j = tj * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = ti * 32 + frag_row(r);
        if (i < j && j < n) Zp[pair_start(i, n) + (j - i - 1)] = f2bf(acc[r]);
      }
    }
    __syncthreads();
    bf16_t* ob = out + (int64_t)b * ostride;
    if (emit0)
      for (int a = threadIdx.x; a < D; a += DOT_THREADS) ob[a] = Xs[a];
    bf16_t* dst = ob + off;
    int done = 0;
    if ((reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
      const int nv = P / 8;
      for (int v = threadIdx.x; v < nv; v += DOT_THREADS)
        *reinterpret_cast<u32x4*>(dst + v * 8) = *reinterpret_cast<const u32x4*>(Zp + v * 8);
      done = nv * 8;
    }
    for (int m = done + threadIdx.x; m < P; m += DOT_THREADS) dst[m] = Zp[m];
    __syncthreads();  // Xs and Zp are rewritten for the next sample
  }
}

// LDS writes of this wave visible to its own reads (wave-private patches)
__device__ inline void dot_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int NP, int D>
__global__ __launch_bounds__(DOT_THREADS, 2) void dot_bwd_mfma_kernel(
    const bf16_t* __restrict__ X, int B, int n, const bf16_t* __restrict__ dout, int64_t dstride,
    int emit0, bf16_t* __restrict__ dX) {
  constexpr int LT = NP + 8, LS = NP + 8;
  constexpr int TT = NP / 32;
  constexpr int PMAX = NP * (NP - 1) / 2;
  constexpr int Q = (PMAX + DOT_THREADS - 1) / DOT_THREADS;  // pairs per thread
  __shared__ __attribute__((aligned(16))) bf16_t XT[D * LT];
  __shared__ __attribute__((aligned(16))) bf16_t S[NP * LS];
  // per-wave 32 x 32 patch: dX tiles leave as 16-byte row segments
  constexpr int LQ = 32 + 8;
  __shared__ __attribute__((aligned(16))) bf16_t DQ[DOT_THREADS / 64][32 * LQ];
  const bool vec_dx = (reinterpret_cast<uintptr_t>(dX) & 15) == 0;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int P = n * (n - 1) / 2;
  const int off = emit0 ? D : 0;
  // diagonal and padding of S stay zero; every sample rewrites all pairs
  for (int e = threadIdx.x; e < NP * LS; e += DOT_THREADS) S[e] = 0;
  // this thread's pairs m = tid + q * THREADS as 16-bit i | j << 8, two per
  // register (the same for every sample): the row is the largest i with
  // pair_start(i) <= m
  uint32_t ijp[(Q + 1) / 2];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int m = threadIdx.x + q * DOT_THREADS;
    uint32_t v = 0;
    if (m < P) {
      const float c = 2.f * n - 1.f;
      int i = (int)((c - sqrtf(fmaxf(c * c - 8.f * m, 0.f))) * 0.5f);
      i = max(0, min(i, n - 2));
      while (i > 0 && pair_start(i, n) > m) --i;
      while (i + 1 <= n - 2 && pair_start(i + 1, n) <= m) ++i;
      const int j = m - pair_start(i, n) + i + 1;
      v = (uint32_t)i | ((uint32_t)j << 8);
    }
    if (q % 2 == 0) ijp[q / 2] = v;
    else ijp[q / 2] |= v << 16;
  }
  Stager<NP, D, DOT_THREADS> sx;
  if (blockIdx.x < B) sx.load(X + (int64_t)blockIdx.x * n * D, D, n);
  __syncthreads();
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    // the pair gradients of this sample, then S and X^T into LDS
    const bf16_t* gb = dout + (int64_t)b * dstride + off;
    // straight-line loads (a pair past the last reads pair 0 and is not
    // used): selecting the loaded value would make each load wait alone
    uint32_t gv[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int m = threadIdx.x + q * DOT_THREADS;
      gv[q] = gb[m < P ? m : 0];
    }
    sx.store(nullptr, 0, XT, LT, n);
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int m = threadIdx.x + q * DOT_THREADS;
      if (m < P) {
        const uint32_t v = (ijp[q / 2] >> (16 * (q % 2))) & 0xffffu;
        const int i = v & 0xff, j = v >> 8;
        S[i * LS + j] = (bf16_t)gv[q];
        S[j * LS + i] = (bf16_t)gv[q];
      }
    }
    __syncthreads();
    // the slot-0 gradient of the column this wave's first tile covers, read
    // before the next sample's loads are issued (a wait for it then does not
    // wait for them); used only with emit0, by the tiles of row block 0
    const bf16_t* g0 = dout + (int64_t)b * dstride;
    const bf16_t g0raw = g0[(w % (D / 32)) * 32 + (lane & 31)];
    if (b + (int)gridDim.x < B) sx.load(X + (int64_t)(b + gridDim.x) * n * D, D, n);
    bf16_t* dxb = dX + (int64_t)b * n * D;
    bf16_t* pq = DQ[w];
    for (int t = w; t < TT * (D / 32); t += DOT_THREADS / 64) {
      const int ti = t / (D / 32), ta = t % (D / 32);
      f32x16 acc;
      zero16(acc);
      mfma_tile<NP>(acc, S + ti * 32 * LS, LS, XT + ta * 32 * LT, LT);
      const float gz = (emit0 && ti == 0) ? bf2f(g0raw) : 0.f;  // ti == 0: t == w
      if (vec_dx) {
        // tile -> patch (row frag_row(r), column lane % 32) -> 16-byte row segments
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int il = frag_row(r);
          const float v = (ti == 0 && il == 0) ? acc[r] + gz : acc[r];
          pq[il * LQ + (lane & 31)] = f2bf(v);
        }
        dot_wave_sync();
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int rl = half * 16 + (lane >> 2), c8 = (lane & 3) * 8;
          const int i = ti * 32 + rl;
          if (i < n) stg16(dxb + i * D + ta * 32 + c8, *reinterpret_cast<const u32x4*>(pq + rl * LQ + c8));
        }
        dot_wave_sync();
        continue;
      }
      const int a = ta * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = ti * 32 + frag_row(r);
        if (i < n) {
          float v = acc[r];
          if (i == 0) v += gz;
          dxb[i * D + a] = f2bf(v);
        }
      }
    }
    __syncthreads();  // S and XT are rewritten for the next sample
  }
}

bool dot_mfma_supported(int n, int d) { return n >= 1 && n <= 128 && (d == 64 || d == 128); }

template <int NP, int D>
static hipError_t dot_mfma_launch(bool fwd, const void* X, int B, int n, void* out,
                                  int64_t ostride, int emit0, const void* dout, int64_t dstride,
                                  void* dX, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const int blocks = B < DOT_BLOCKS ? B : DOT_BLOCKS;
  if (fwd)
    dot_fwd_mfma_kernel<NP, D><<<blocks, DOT_THREADS, 0, s>>>((const bf16_t*)X, B, n,
                                                             (bf16_t*)out, ostride, emit0);
  else
    dot_bwd_mfma_kernel<NP, D><<<blocks, DOT_THREADS, 0, s>>>(
        (const bf16_t*)X, B, n, (const bf16_t*)dout, dstride, emit0, (bf16_t*)dX);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t dot_mfma(bool fwd, const void* X, int B, int n, int d, void* out, int64_t ostride,
                    int emit0, const void* dout, int64_t dstride, void* dX, hipStream_t s) {
#define LAT_DOTM(NPV, DV)                                                                  \
  if (n <= NPV && d == DV)                                                                 \
    return dot_mfma_launch<NPV, DV>(fwd, X, B, n, out, ostride, emit0, dout, dstride, dX, s);
  LAT_DOTM(32, 64) LAT_DOTM(64, 64) LAT_DOTM(96, 64) LAT_DOTM(128, 64)
  LAT_DOTM(32, 128) LAT_DOTM(64, 128) LAT_DOTM(96, 128) LAT_DOTM(128, 128)
#undef LAT_DOTM
  set_error("DOT MFMA path: unsupported shape n=%d d=%d", n, d);
  return hipErrorInvalidValue;
}

}  // namespace lat
