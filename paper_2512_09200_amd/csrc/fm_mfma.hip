// Factorization-machine block O_b = X_b (X_b^T W) (Section 3.3.2) on bf16 MFMA
// (v_mfma_f32_32x32x16_bf16), forward and backward, for up to 96 vectors in
// tiles (97 with a head row, below), d in {64, 128}, rank k in {32, 64}.
//
// Each block of 8 waves loops over samples.  A sample's X [n, d] is read once
// with coalesced 4-byte loads (8 rows x 2 columns per thread) into registers
// one sample ahead (the next sample's loads are in flight while the current
// one is computed), transposed in registers, and staged in LDS twice --
// row-major X[j][a] and transposed X^T[a][j] -- so every MFMA operand is read
// as k-contiguous 16-byte fragments.  Where it lets three blocks share a
// compute unit, the forward runs 4-wave blocks that stage X once and read
// the X^T operand of P = X^T W from it with transposed LDS reads
// (ds_read_b64_tr_b16): three samples in flight per unit instead of two
// (n = 65, d = 128, k = 32: 43 -> 38 us).  Storage rounding matches the rest of the step: P = X^T W and
// dP = X^T G are rounded to bf16 before use, O and dX are stored in bf16.
//   forward : P = X^T W (contraction over j), O = X P (over a)
//   backward: P, dP and dP^T (= G^T X, the dW operand) share the staged
//             fragments; dX = [G | W] [P | dP]^T is one contraction over 2k;
//             dW += X dP accumulates in the waves' registers across the
//             block's samples (fixed order), and the per-block partials are
//             summed in block order afterwards.
// Head row: when n = 32 t + 1 (the dense vector plus 32 t features), row 0 is
// taken out of the tiles (HEAD): the MFMA tiles cover rows 1 .. n-1 exactly
// instead of padding to the next multiple of 32, and row 0's rank-1 terms
// (x0^T w0, x0^T g0) and its own outputs (O[0], dX[0], dW[0]) are a few
// hundred FMAs per sample on the vector units, reduced in a fixed order.
#include "common.h"
#include "kernels.h"
#include "mfma_tile.h"

namespace lat {

// sum over the 16 lanes of an aligned lane group, in a fixed butterfly order
__device__ inline float group16_sum(float v) {
  v += __shfl_xor(v, 8, 64);
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 2, 64);
  v += __shfl_xor(v, 1, 64);
  return v;
}

// LDS writes of this wave visible to its own reads (wave-private patches)
__device__ inline void fm_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Head row in registers one sample ahead: thread t < COLS/2 holds columns
// 2t, 2t+1 of row 0 (bf16 pair).
template <int COLS>
struct HeadRow {
  uint32_t v = 0;
  // straight-line (threads past the row re-read its first pair)
  __device__ inline void load(const bf16_t* __restrict__ g, int tid = threadIdx.x) {
    v = *reinterpret_cast<const uint32_t*>(g + 2 * (tid < COLS / 2 ? tid : 0));
  }
  __device__ inline void store_bf16(bf16_t* dst, int tid = threadIdx.x) const {
    if (tid < COLS / 2) *reinterpret_cast<uint32_t*>(dst + 2 * tid) = v;
  }
  __device__ inline void store(float* dst, int tid = threadIdx.x) const {
    if (tid < COLS / 2) {
      dst[2 * tid] = __uint_as_float(v << 16);
      dst[2 * tid + 1] = __uint_as_float(v & 0xffff0000u);
    }
  }
};

// NW waves per block; TR: X is staged once (row-major) and the X^T operand
// of P = X^T W is read from it with transposed LDS reads, so the block's LDS
// holds no X^T copy, and W only as W^T, the operand of P (with 4 waves,
// three blocks fit a compute unit: three samples in flight instead of two).
template <int NP, int D, int K, bool HEAD, int NW = 8, bool TR = false>
__global__ __launch_bounds__(NW * 64) void fm_fwd_mfma_kernel(const bf16_t* __restrict__ X,
                                                          const bf16_t* __restrict__ W, int B,
                                                          int n, bf16_t* __restrict__ out,
                                                          int64_t ostride, int emit0) {
  constexpr int LX = D + 8, LT = NP + 8, LP = D + 8;
  constexpr int H = HEAD ? 1 : 0;  // rows ahead of the MFMA rows
  constexpr int THREADS = NW * 64;
  __shared__ __attribute__((aligned(16))) bf16_t Xs[NP * LX];
  __shared__ __attribute__((aligned(16))) bf16_t XT[TR ? 8 : D * LT];
  __shared__ __attribute__((aligned(16))) bf16_t PT[K * LP];
  __shared__ __attribute__((aligned(16))) bf16_t WT[K * LT];
  __shared__ float X0[HEAD ? D : 1], W0[HEAD ? K : 1];
  // per-wave 32 x 32 patch: an O tile leaves as 16-byte row segments (its
  // rows are contiguous in the output) instead of 2-byte columns, where the
  // patches leave room for two blocks per compute unit
  constexpr int LQ = 32 + 8;
  constexpr int OT = (NP / 32) * (K / 32);  // O tiles (OT <= 8), one patch per wave that has one
  constexpr int NQ = OT < NW ? OT : NW;
  constexpr size_t BASE = 2 * ((size_t)NP * LX + (TR ? 0 : D * LT) + K * LP + K * LT) +
                          4 * ((HEAD ? D : 1) + (HEAD ? K : 1));
  constexpr bool VEC = BASE + (size_t)NQ * 2 * 32 * LQ <= 80 * 1024;
  __shared__ __attribute__((aligned(16))) bf16_t OQ[VEC ? NQ : 1][VEC ? 32 * LQ : 8];
  const bool vec_out = VEC && (reinterpret_cast<uintptr_t>(out) & 15) == 0 && (ostride & 7) == 0;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nm = n - H;  // rows in the tiles
  {
    Stager<NP, K, THREADS> sw;
    sw.load(W + H * K, K, nm);
    sw.store(nullptr, 0, WT, LT, nm);  // only W^T is an operand here
    if (HEAD)
      for (int c = threadIdx.x; c < K; c += blockDim.x) W0[c] = bf2f(W[c]);
  }
  const int off = emit0 ? D : 0;
  Stager<NP, D, THREADS> sx;
  HeadRow<D> hx;
  if (blockIdx.x < B) {
    const bf16_t* xb = X + (int64_t)blockIdx.x * n * D;
    sx.load(xb + H * D, D, nm);
    if (HEAD) hx.load(xb);
  }
  for (int b = blockIdx.x; b < B; b += gridDim.x) {
    sx.store(Xs, LX, TR ? nullptr : XT, LT, nm);
    if (HEAD) hx.store(X0);
    __syncthreads();
    // the next sample's X is in flight while this one is computed
    if (b + (int)gridDim.x < B) {
      const bf16_t* xb = X + (int64_t)(b + gridDim.x) * n * D;
      sx.load(xb + H * D, D, nm);
      if (HEAD) hx.load(xb);
    }
    // P[a][c] = sum_j X^T[a][j] W^T[c][j] (+ x0[a] w0[c]); tile (ta, tc) per wave
    constexpr int PT_TILES = (D / 32) * (K / 32);
    for (int t = w; t < PT_TILES; t += NW) {
      const int ta = t / (K / 32), tc = t % (K / 32);
      f32x16 acc;
      zero16(acc);
      if constexpr (TR) mfma_tile_kmA<NP>(acc, Xs, LX, ta * 32, WT + tc * 32 * LT, LT);
      else mfma_tile<NP>(acc, XT + ta * 32 * LT, LT, WT + tc * 32 * LT, LT);
      const int c = tc * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int a = ta * 32 + frag_row(r);
        const float v = HEAD ? acc[r] + X0[a] * W0[c] : acc[r];
        PT[c * LP + a] = f2bf(v);
      }
    }
    __syncthreads();
    // O[j][c] = sum_a X[j][a] P^T[c][a]
    bf16_t* ob = out + (int64_t)b * ostride;
    constexpr int O_TILES = (NP / 32) * (K / 32);
    for (int t = w; t < O_TILES; t += NW) {
      const int tj = t / (K / 32), tc = t % (K / 32);
      f32x16 acc;
      zero16(acc);
      mfma_tile<D>(acc, Xs + tj * 32 * LX, LX, PT + tc * 32 * LP, LP);
      const int c = tc * 32 + (lane & 31);
      if (vec_out) {
        bf16_t* pq = OQ[VEC ? w : 0];
#pragma unroll
        for (int r = 0; r < 16; ++r) pq[frag_row(r) * LQ + (lane & 31)] = f2bf(acc[r]);
        fm_wave_sync();
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int rl = half * 16 + (lane >> 2), c8 = (lane & 3) * 8;
          const int j = tj * 32 + rl;
          if (j < nm)
            stg16(ob + off + (j + H) * K + tc * 32 + c8, *reinterpret_cast<const u32x4*>(pq + rl * LQ + c8));
        }
        fm_wave_sync();
        continue;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = tj * 32 + frag_row(r);
        if (j < nm) ob[off + (j + H) * K + c] = f2bf(acc[r]);
      }
    }
    if (HEAD) {
      // O[0][c] = sum_a x0[a] P[a][c]: 16 lanes per c, D/16 terms each
      const int q = threadIdx.x & 15;
#pragma unroll
      for (int c = threadIdx.x >> 4; c < K; c += THREADS / 16) {
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < D / 16; ++i) {
          const int a = q * (D / 16) + i;
          sum += X0[a] * bf2f(PT[c * LP + a]);
        }
        sum = group16_sum(sum);
        if (q == 0) ob[off + c] = f2bf(sum);
      }
      if (emit0)
        for (int a = threadIdx.x; a < D; a += blockDim.x) ob[a] = f2bf(X0[a]);
    } else if (emit0) {
      for (int a = threadIdx.x; a < D; a += blockDim.x) ob[a] = Xs[a];
    }
    __syncthreads();
  }
}

// Backward.  dX_f32 (optional) receives the unrounded fp32 dX instead of dX.
// SPB samples per block iteration (their buffers side by side in LDS): each
// phase then has SPB times the tiles to spread over the 8 waves between the
// same barriers.
template <int NP, int D, int K, bool HEAD, int SPB>
struct FmBwdLds {
  static constexpr int LX = D + 8, LT = NP + 8, LG = 2 * K + 8, LPD = 2 * K + 8, LDT = D + 8;
  static constexpr size_t bytes =
      2 * ((size_t)SPB * (NP * LX + D * LT + K * LDT + NP * LG + K * LT + D * LPD) + K * LT) +
      4 * (size_t)SPB * (HEAD ? D + 2 * K : 2);
};

template <int NP, int D, int K, bool HEAD, int SPB>
__global__ __launch_bounds__(512) void fm_bwd_mfma_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int B, int n,
    const bf16_t* __restrict__ dout, int64_t dstride, int emit0, const float* __restrict__ addend,
    bf16_t* __restrict__ dX, float* __restrict__ dX_f32, float* __restrict__ dw_part) {
  using L = FmBwdLds<NP, D, K, HEAD, SPB>;
  constexpr int LX = L::LX, LT = L::LT, LG = L::LG, LPD = L::LPD, LDT = L::LDT;
  constexpr int H = HEAD ? 1 : 0;
  __shared__ __attribute__((aligned(16))) bf16_t Xs[SPB][NP * LX];
  __shared__ __attribute__((aligned(16))) bf16_t XT[SPB][D * LT];
  __shared__ __attribute__((aligned(16))) bf16_t DT[SPB][K * LDT];  // dP^T [K][LDT]
  __shared__ __attribute__((aligned(16))) bf16_t GW[SPB][NP * LG];  // [j][ G (K) | W (K) ]
  __shared__ __attribute__((aligned(16))) bf16_t GT[SPB][K * LT];
  __shared__ __attribute__((aligned(16))) bf16_t WT[K * LT];
  __shared__ __attribute__((aligned(16))) bf16_t PD[SPB][D * LPD];  // [a][ P (K) | dP (K) ]
  __shared__ float X0[SPB][HEAD ? D : 1], GW0[SPB][HEAD ? 2 * K : 1];  // head row: x0, [g0 | w0]
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nm = n - H;
  {
    Stager<NP, K, 512> sw;
    sw.load(W + H * K, K, nm);
    for (int q = 0; q < SPB; ++q) sw.store(GW[q] + K, LG, q == 0 ? WT : nullptr, LT, nm);
    if (HEAD)
      for (int c = threadIdx.x; c < K; c += blockDim.x)
        for (int q = 0; q < SPB; ++q) GW0[q][K + c] = bf2f(W[c]);
  }
  constexpr int DW_TILES = (NP / 32) * (K / 32);
  f32x16 dw[(DW_TILES + 7) / 8];
#pragma unroll
  for (int i = 0; i < (DW_TILES + 7) / 8; ++i) zero16(dw[i]);
  // head row of dW, accumulated over the block's samples: lane group
  // tid / 16 owns columns c = tid / 16 + 32 i
  float dw0[(K + 31) / 32];
#pragma unroll
  for (int i = 0; i < (K + 31) / 32; ++i) dw0[i] = 0.f;
  const int off = emit0 ? D : 0;
  Stager<NP, D, 512> sx[SPB];
  Stager<NP, K, 512> sg[SPB];
  HeadRow<D> hx[SPB];
  HeadRow<K> hg[SPB];
  auto prefetch = [&](int b0) {
#pragma unroll
    for (int q = 0; q < SPB; ++q) {
      const int bb = b0 + q;
      if (bb >= B) break;
      const bf16_t* xb = X + (int64_t)bb * n * D;
      const bf16_t* gb = dout + (int64_t)bb * dstride + off;
      sx[q].load(xb + H * D, D, nm);
      sg[q].load(gb + H * K, K, nm);
      if (HEAD) {
        hx[q].load(xb);
        hg[q].load(gb);
      }
    }
  };
  const int step = gridDim.x * SPB;
  if (blockIdx.x * SPB < B) prefetch(blockIdx.x * SPB);
  for (int b0 = blockIdx.x * SPB; b0 < B; b0 += step) {
    const int ns = B - b0 < SPB ? B - b0 : SPB;  // samples in this iteration
#pragma unroll
    for (int q = 0; q < SPB; ++q) {
      if (q >= ns) break;
      sx[q].store(Xs[q], LX, XT[q], LT, nm);
      sg[q].store(GW[q], LG, GT[q], LT, nm);
      if (HEAD) {
        hx[q].store(X0[q]);
        hg[q].store(GW0[q]);
      }
    }
    __syncthreads();
    // the next samples' X and G are in flight while these are computed
    if (b0 + step < B) prefetch(b0 + step);
    // P = X^T W and dP = X^T G into PD[a][P | dP], and dP^T[c][a] = G^T X
    // into DT (the dW operand), all rounded to bf16 (+ the head row's
    // rank-1 terms)
    constexpr int P_TILES = (D / 32) * (K / 32);
    for (int t = w; t < ns * 3 * P_TILES; t += 8) {
      const int q = t / (3 * P_TILES), which = (t / P_TILES) % 3, tt = t % P_TILES;
      f32x16 acc;
      zero16(acc);
      if (which < 2) {
        const int ta = tt / (K / 32), tc = tt % (K / 32);
        mfma_tile<NP>(acc, XT[q] + ta * 32 * LT, LT, (which ? GT[q] : WT) + tc * 32 * LT, LT);
        const int c = tc * 32 + (lane & 31);
        const float h = HEAD ? GW0[q][which ? c : K + c] : 0.f;  // g0[c] or w0[c]
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int a = ta * 32 + frag_row(r);
          const float v = HEAD ? acc[r] + X0[q][a] * h : acc[r];
          PD[q][a * LPD + c + which * K] = f2bf(v);
        }
      } else {
        const int tc = tt / (D / 32), ta = tt % (D / 32);
        mfma_tile<NP>(acc, GT[q] + tc * 32 * LT, LT, XT[q] + ta * 32 * LT, LT);
        const int a = ta * 32 + (lane & 31);
        const float x0 = HEAD ? X0[q][a] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int c = tc * 32 + frag_row(r);
          const float v = HEAD ? acc[r] + GW0[q][c] * x0 : acc[r];
          DT[q][c * LDT + a] = f2bf(v);
        }
      }
    }
    __syncthreads();
    // dX[j][a] = sum_kk GW[j][kk] PD[a][kk]  (+ addend, + slot-0 gradient).
    // Plain bf16 output: each tile is rounded into XT (free after the phase
    // above) as [j][a] and the sample's rows j >= H are then written with
    // 16-byte stores (they are contiguous in dX).
    constexpr int DX_TILES = (NP / 32) * (D / 32);
    constexpr int LY = NP * (D + 8) <= D * LT ? D + 8 : D;  // row stride of the staged dX
    static_assert(NP * LY <= D * LT, "staged dX must fit in X^T");
    const bool staged = !addend && !dX_f32 && (reinterpret_cast<uintptr_t>(dX) & 15) == 0;
    for (int t = w; t < ns * DX_TILES; t += 8) {
      const int q = t / DX_TILES, tj = (t % DX_TILES) / (D / 32), ta = t % (D / 32);
      const int b = b0 + q;
      const int64_t sbase = (int64_t)b * n * D;  // this sample's [n, D] block
      f32x16 acc;
      zero16(acc);
      mfma_tile<2 * K>(acc, GW[q] + tj * 32 * LG, LG, PD[q] + ta * 32 * LPD, LPD);
      const int a = ta * 32 + (lane & 31);
      const float g0 = (!HEAD && emit0 && tj == 0) ? bf2f(dout[(int64_t)b * dstride + a]) : 0.f;
      if (staged) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = tj * 32 + frag_row(r);
          const float v = (!HEAD && j == 0) ? acc[r] + g0 : acc[r];
          XT[q][j * LY + a] = f2bf(v);
        }
        continue;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = tj * 32 + frag_row(r);
        if (j < nm) {
          float v = acc[r];
          const int e = (j + H) * D + a;
          if (addend) v += addend[sbase + e];
          if (!HEAD && j == 0) v += g0;
          if (dX_f32) dX_f32[sbase + e] = v;
          else dX[sbase + e] = f2bf(v);
        }
      }
    }
    if (HEAD) {
      // dX[0][a] = sum_kk [g0 | w0][kk] PD[a][kk]: 4 lanes per a, K/2 terms
      // each, then the slot-0 gradient and the addend
      const int a = threadIdx.x >> 2, qq = threadIdx.x & 3;
#pragma unroll
      for (int q = 0; q < SPB; ++q) {
        if (q >= ns) break;
        const int b = b0 + q;
        const int64_t sbase = (int64_t)b * n * D;
        if (a < D) {
          float sum = 0.f;
#pragma unroll
          for (int i = 0; i < 2 * K / 4; ++i) {
            const int kk = qq * (2 * K / 4) + i;
            sum += GW0[q][kk] * bf2f(PD[q][a * LPD + kk]);
          }
          sum += __shfl_xor(sum, 2, 64);
          sum += __shfl_xor(sum, 1, 64);
          if (qq == 0) {
            if (addend) sum += addend[sbase + a];
            if (emit0) sum += bf2f(dout[(int64_t)b * dstride + a]);
            if (dX_f32) dX_f32[sbase + a] = sum;
            else dX[sbase + a] = f2bf(sum);
          }
        }
      }
    }
    // dW[j][c] += sum_a X[j][a] dP^T[c][a], the samples in order
    for (int t = w, i = 0; t < DW_TILES; t += 8, ++i) {
      const int tj = t / (K / 32), tc = t % (K / 32);
#pragma unroll
      for (int q = 0; q < SPB; ++q) {
        if (q >= ns) break;
        mfma_tile<D>(dw[i], Xs[q] + tj * 32 * LX, LX, DT[q] + tc * 32 * LDT, LDT);
      }
    }
    if (HEAD) {
      // dW[0][c] += sum_a x0[a] dP[a][c]: 16 lanes per c, the samples in order
      const int qq = threadIdx.x & 15;
#pragma unroll
      for (int i0 = 0; i0 < (K + 31) / 32; ++i0) {
        const int c = (threadIdx.x >> 4) + 32 * i0;
        if (c < K) {
#pragma unroll
          for (int q = 0; q < SPB; ++q) {
            if (q >= ns) break;
            float sum = 0.f;
#pragma unroll
            for (int i = 0; i < D / 16; ++i) {
              const int a = qq * (D / 16) + i;
              sum += X0[q][a] * bf2f(DT[q][c * LDT + a]);
            }
            dw0[i0] += group16_sum(sum);
          }
        }
      }
    }
    __syncthreads();
    if (staged) {
      // rows H .. n-1 of each sample: nm * D contiguous bf16, 8 per store
      for (int q = 0; q < ns; ++q) {
        bf16_t* dst = dX + (int64_t)(b0 + q) * n * D + H * D;
        for (int v = threadIdx.x; v < nm * D / 8; v += blockDim.x) {
          const int j = v / (D / 8), a = (v % (D / 8)) * 8;
          stg16(dst + j * D + a, *reinterpret_cast<const u32x4*>(XT[q] + j * LY + a));
        }
      }
      __syncthreads();  // X^T is restaged for the next samples
    }
  }
  for (int t = w, i = 0; t < DW_TILES; t += 8, ++i) {
    const int tj = t / (K / 32), tc = t % (K / 32);
    const int c = tc * 32 + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = tj * 32 + frag_row(r);
      if (j < nm) dw_part[((int64_t)blockIdx.x * n + j + H) * K + c] = dw[i][r];
    }
  }
  if (HEAD && (threadIdx.x & 15) == 0)
#pragma unroll
    for (int i0 = 0; i0 < (K + 31) / 32; ++i0) {
      const int c = (threadIdx.x >> 4) + 32 * i0;
      if (c < K) dw_part[(int64_t)blockIdx.x * n * K + c] = dw0[i0];
    }
}

// Backward for d = 128 with the products chained through registers.  Four
// waves work on one sample, wave ta on the columns a in [32 ta, 32 ta + 32);
// SPB samples per block iteration.  A wave computes its tiles of P^T (c x a),
// dP^T (c x a) and dP (a x c) from the staged X^T, G^T and W^T, rounds them
// to bf16 and uses them directly as MFMA operands: a result tile's lane
// holds one column and, for rows 16 s .. 16 s + 15, the rows
// 16 s + 4 h + {0..3} and 16 s + 8 + 4 h + {0..3} (h = lane / 32), which is
// an operand fragment of the k step s with its k order permuted; the other
// operand is read from LDS in the same order (two 8-byte reads).  So
//   dX[j][a] += sum_c G[j][c] P^T[c][a] + W[j][c] dP^T[c][a]   (rows j of G, W)
//   dW[j][c] += sum_{a in the wave's columns} X[j][a] dP[a][c]   (rows j of X)
// need no LDS round trip for P, dP and dP^T, and an iteration has two
// barriers.  dW accumulates in the waves' registers across the block's
// samples; at the end the eight waves' partial tiles are added in wave order
// through LDS into the block's partial.
__device__ inline bf16x8 ld_perm(const bf16_t* p) {
  const u32x2 lo = *reinterpret_cast<const u32x2*>(p);
  const u32x2 hi = *reinterpret_cast<const u32x2*>(p + 8);
  return __builtin_bit_cast(bf16x8, (u32x4{lo[0], lo[1], hi[0], hi[1]}));
}

// bf16 fragment of result rows 16 s .. 16 s + 15 (values r = 8 s .. 8 s + 7)
__device__ inline bf16x8 frag_of(const f32x16& v, int s) {
  return __builtin_bit_cast(
      bf16x8, (u32x4{pack_bf2(v[8 * s], v[8 * s + 1]), pack_bf2(v[8 * s + 2], v[8 * s + 3]),
                     pack_bf2(v[8 * s + 4], v[8 * s + 5]), pack_bf2(v[8 * s + 6], v[8 * s + 7])}));
}

// LDS of the chained kernel, one buffer: the staged operands during the
// sample loop; afterwards the first bytes hold the dW reduction.
// operand fragment with v (a bf16 value held as fp32) in the first k slot of
// the lane's row and zeros elsewhere
__device__ inline bf16x8 slot0(float v) {
  const uint32_t lo = ((threadIdx.x & 63) >> 5) == 0 ? (uint32_t)f2bf(v) : 0u;
  return __builtin_bit_cast(bf16x8, (u32x4{lo, 0u, 0u, 0u}));
}

// operand fragment of row 0 only: the row at p in the permuted k order for
// lane 0 / 32 (rows 0 of the tile), zeros for the other rows
__device__ inline bf16x8 row0(const bf16_t* p) {
  return (threadIdx.x & 31) == 0 ? ld_perm(p) : __builtin_bit_cast(bf16x8, (u32x4{0u, 0u, 0u, 0u}));
}

template <int NP, int K, bool HEAD, int SPB>
struct FmChainLds {
  static constexpr int D = 128, NW = SPB * 4;
  static constexpr int LT = NP + 8, LX = D + 4, LG = K + 4;
  static constexpr size_t al(size_t b) { return (b + 15) / 16 * 16; }
  // byte offsets
  static constexpr size_t XT = 0;                                   // [SPB][D][LT]  X^T
  static constexpr size_t XS = XT + al(2 * (size_t)SPB * D * LT);   // [SPB][NP][LX] X
  static constexpr size_t GT = XS + al(2 * (size_t)SPB * NP * LX);  // [SPB][K][LT]  G^T
  static constexpr size_t GS = GT + al(2 * (size_t)SPB * K * LT);   // [SPB][NP][LG] G
  static constexpr size_t WT = GS + al(2 * (size_t)SPB * NP * LG);  // [K][LT]       W^T
  static constexpr size_t WS = WT + al(2 * (size_t)K * LT);         // [NP][LG]      W
  static constexpr size_t X0 = WS + al(2 * (size_t)NP * LG);        // [SPB][D] f32  head x0
  static constexpr size_t G0 = X0 + al(4 * (size_t)SPB * D);        // [SPB][K] f32  head g0
  static constexpr size_t W0 = G0 + al(4 * (size_t)SPB * K);        // [K] f32       head w0
  static constexpr size_t G0B = W0 + al(4 * (size_t)K);             // [SPB][K + 8]  head g0, bf16
  static constexpr size_t W0B = G0B + al(2 * (size_t)SPB * (K + 8)); // [K + 8]      head w0, bf16
  static constexpr size_t S0 = W0B + al(2 * (size_t)(K + 8));       // [SPB][D] f32  slot-0 gradient
  static constexpr int LQ = 32 + 8;                                 // dX patch row stride
  static constexpr size_t DQ = S0 + al(4 * (size_t)SPB * D);        // [NW][32][LQ]  per-wave dX patch
  static constexpr size_t stage_bytes = DQ + al(2 * (size_t)NW * 32 * LQ);
  static constexpr size_t red_bytes = 4 * ((size_t)NW * 16 * 64 + (size_t)NW * K);
  static constexpr size_t bytes = stage_bytes > red_bytes ? stage_bytes : red_bytes;
};

// PLAIN: a bf16 dX (16-byte aligned), no addend, no fp32 copy
template <int NP, int K, bool HEAD, int SPB, bool PLAIN>
__global__ __launch_bounds__(SPB * 256) void fm_bwd_chain_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int B, int n,
    const bf16_t* __restrict__ dout, int64_t dstride, int emit0, const float* __restrict__ addend,
    bf16_t* __restrict__ dX, float* __restrict__ dX_f32, float* __restrict__ dw_part) {
  constexpr int D = 128, THREADS = SPB * 256, NW = THREADS / 64;
  constexpr int NJ = NP / 32, NC = K / 32;
  using L = FmChainLds<NP, K, HEAD, SPB>;
  constexpr int LT = L::LT, LX = L::LX, LG = L::LG;
  constexpr int H = HEAD ? 1 : 0;
  __shared__ __attribute__((aligned(16))) unsigned char smem[L::bytes];
  auto XT = [&](int qq) { return reinterpret_cast<bf16_t*>(smem + L::XT) + (size_t)qq * D * LT; };
  auto Xs = [&](int qq) { return reinterpret_cast<bf16_t*>(smem + L::XS) + (size_t)qq * NP * LX; };
  auto GT = [&](int qq) { return reinterpret_cast<bf16_t*>(smem + L::GT) + (size_t)qq * K * LT; };
  auto Gs = [&](int qq) { return reinterpret_cast<bf16_t*>(smem + L::GS) + (size_t)qq * NP * LG; };
  bf16_t* WT = reinterpret_cast<bf16_t*>(smem + L::WT);
  bf16_t* Ws = reinterpret_cast<bf16_t*>(smem + L::WS);
  auto X0 = [&](int qq) { return reinterpret_cast<float*>(smem + L::X0) + qq * D; };
  auto G0 = [&](int qq) { return reinterpret_cast<float*>(smem + L::G0) + qq * K; };
  float* W0 = reinterpret_cast<float*>(smem + L::W0);
  auto G0b = [&](int qq) { return reinterpret_cast<bf16_t*>(smem + L::G0B) + qq * (K + 8); };
  bf16_t* W0b = reinterpret_cast<bf16_t*>(smem + L::W0B);
  auto S0 = [&](int qq) { return reinterpret_cast<float*>(smem + L::S0) + qq * D; };
  constexpr int LQ = L::LQ;
  // this wave's 32 x 32 patch for transposing dX tiles to row segments
  bf16_t* dq = reinterpret_cast<bf16_t*>(smem + L::DQ) + (threadIdx.x >> 6) * 32 * LQ;
  // PLAIN: tiles leave as 16-byte row segments through the patch instead of
  // 2-byte column stores
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = w >> 2, ta = w & 3;  // this wave's sample and column block
  const int h = lane >> 5, l32 = lane & 31;
  const int nm = n - H;
  {
    Stager<NP, K, THREADS> sw;
    sw.load(W + H * K, K, nm);
    sw.store(Ws, LG, WT, LT, nm);
    if (HEAD)
      for (int c = threadIdx.x; c < K; c += THREADS) {
        W0[c] = bf2f(W[c]);
        W0b[c] = W[c];
      }
  }
  f32x16 dw[NJ][NC];
#pragma unroll
  for (int tj = 0; tj < NJ; ++tj)
#pragma unroll
    for (int tc = 0; tc < NC; ++tc) zero16(dw[tj][tc]);
  float dw0[NC];
#pragma unroll
  for (int tc = 0; tc < NC; ++tc) dw0[tc] = 0.f;
  const int off = emit0 ? D : 0;
  Stager<NP, D, THREADS> sx[SPB];
  Stager<NP, K, THREADS> sg[SPB];
  HeadRow<D> hx[SPB];
  HeadRow<K> hg[SPB];
  HeadRow<D> hs[SPB];  // slot-0 gradient (emit0): staged like the operands, so
                       // the compute reads no global memory
  auto prefetch = [&](int b0) {
#pragma unroll
    for (int qq = 0; qq < SPB; ++qq) {
      // a valid sample for every qq (stored only if b0 + qq < B): the loads
      // are straight-line code
      const int bb = b0 + qq < B ? b0 + qq : B - 1;
      const bf16_t* xb = X + (int64_t)bb * n * D;
      const bf16_t* gb = dout + (int64_t)bb * dstride + off;
      sx[qq].load(xb + H * D, D, nm);
      sg[qq].load(gb + H * K, K, nm);
      if (HEAD) {
        hx[qq].load(xb);
        hg[qq].load(gb);
      }
      if (emit0) hs[qq].load(dout + (int64_t)bb * dstride);
    }
  };
  const int step = gridDim.x * SPB;
  if (blockIdx.x * SPB < B) prefetch(blockIdx.x * SPB);
  for (int b0 = blockIdx.x * SPB; b0 < B; b0 += step) {
    const int ns = B - b0 < SPB ? B - b0 : SPB;
#pragma unroll
    for (int qq = 0; qq < SPB; ++qq) {
      if (qq >= ns) break;
      sx[qq].store(Xs(qq), LX, XT(qq), LT, nm);
      sg[qq].store(Gs(qq), LG, GT(qq), LT, nm);
      if (HEAD) {
        hx[qq].store(X0(qq));
        hg[qq].store(G0(qq));
        hg[qq].store_bf16(G0b(qq));
      }
      if (emit0) hs[qq].store(S0(qq));
    }
    __syncthreads();
    if (b0 + step < B) prefetch(b0 + step);
    if (q < ns) {
      const int b = b0 + q;
      const int64_t sbase = (int64_t)b * n * D;
      const int a = ta * 32 + l32;  // this lane's column of dX
      const bf16_t* xt_a = XT(q) + ta * 32 * LT;
      f32x16 ax[NJ];
#pragma unroll
      for (int tj = 0; tj < NJ; ++tj) zero16(ax[tj]);
      const float x0a = HEAD ? X0(q)[a] : 0.f;
      // One product at a time (its tile, then its bf16 fragments -- the
      // rounding of P and dP -- then the MFMAs that take them), and dX
      // finished before dP is formed, so few tiles are live at once.  The head row's rank-1 terms are one more
      // MFMA per product whose operands hold x0[a], w0[c] or g0[c] in their
      // first k slot (zero elsewhere), and its dX row is a tile whose A
      // operand is zero except row 0 (g0 or w0).
      f32x16 axh;
      zero16(axh);
#pragma unroll
      for (int tc = 0; tc < NC; ++tc) {
        const float w0c = HEAD ? W0[tc * 32 + l32] : 0.f, g0c = HEAD ? G0(q)[tc * 32 + l32] : 0.f;
        // P^T [c][a] (+ w0[c] x0[a]) -> dX += G P^T
        {
          f32x16 t;
          zero16(t);
          mfma_tile<NP>(t, WT + tc * 32 * LT, LT, xt_a, LT);
          if (HEAD) t = __builtin_amdgcn_mfma_f32_32x32x16_bf16(slot0(w0c), slot0(x0a), t, 0, 0, 0);
#pragma unroll
          for (int s = 0; s < 2; ++s) {
            const bf16x8 f = frag_of(t, s);
            const int kc = tc * 32 + 16 * s + 4 * h;
#pragma unroll
            for (int tj = 0; tj < NJ; ++tj)
              ax[tj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_perm(Gs(q) + (tj * 32 + l32) * LG + kc),
                                                               f, ax[tj], 0, 0, 0);
            if (HEAD)
              axh = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row0(G0b(q) + kc), f, axh, 0, 0, 0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        // dP^T [c][a] (+ g0[c] x0[a]) -> dX += W dP^T
        {
          f32x16 t;
          zero16(t);
          mfma_tile<NP>(t, GT(q) + tc * 32 * LT, LT, xt_a, LT);
          if (HEAD) t = __builtin_amdgcn_mfma_f32_32x32x16_bf16(slot0(g0c), slot0(x0a), t, 0, 0, 0);
#pragma unroll
          for (int s = 0; s < 2; ++s) {
            const bf16x8 f = frag_of(t, s);
            const int kc = tc * 32 + 16 * s + 4 * h;
#pragma unroll
            for (int tj = 0; tj < NJ; ++tj)
              ax[tj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_perm(Ws + (tj * 32 + l32) * LG + kc),
                                                               f, ax[tj], 0, 0, 0);
            if (HEAD) axh = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row0(W0b + kc), f, axh, 0, 0, 0);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      float hx0 = axh[0];  // dX[0][a] in the lanes with h == 0
      // dX rows (+ addend, + slot-0 gradient on row 0 when it is in the tiles)
      {
        const float g0v = emit0 ? S0(q)[a] : 0.f;
        const float g0 = HEAD ? 0.f : g0v;
#pragma unroll
        for (int tj = 0; tj < NJ; ++tj) {
          if constexpr (PLAIN) {
            // tile -> patch (row frag_row(r), column l32), then lane l writes
            // row l / 4 (+ 16) columns 8 (l % 4) .. + 7 of the tile
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int jl = frag_row(r);
              const float v = (!HEAD && tj == 0 && jl == 0) ? ax[tj][r] + g0 : ax[tj][r];
              dq[jl * LQ + l32] = f2bf(v);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
            for (int half = 0; half < 2; ++half) {
              const int jl = half * 16 + (lane >> 2), c8 = (lane & 3) * 8;
              const int j = tj * 32 + jl;
              const u32x4 v = *reinterpret_cast<const u32x4*>(dq + jl * LQ + c8);
              if (j < nm) stg16(dX + sbase + (int64_t)(j + H) * D + ta * 32 + c8, v);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
          } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int j = tj * 32 + frag_row(r);
              if (j < nm) {
                float v = ax[tj][r];
                const int e = (j + H) * D + a;
                if (addend) v += addend[sbase + e];
                if (!HEAD && j == 0) v += g0;
                if (dX_f32) dX_f32[sbase + e] = v;
                else dX[sbase + e] = f2bf(v);
              }
            }
          }
        }
        if (HEAD) {
          if (h == 0) {
            if (!PLAIN && addend) hx0 += addend[sbase + a];
            hx0 += g0v;
            if (!PLAIN && dX_f32) dX_f32[sbase + a] = hx0;
            else dX[sbase + a] = f2bf(hx0);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      // dP [a][c] (+ x0[a] g0[c]) -> dW += X dP
#pragma unroll
      for (int tc = 0; tc < NC; ++tc) {
        const float g0c = HEAD ? G0(q)[tc * 32 + l32] : 0.f;
        f32x16 t;
        zero16(t);
        mfma_tile<NP>(t, xt_a, LT, GT(q) + tc * 32 * LT, LT);
        if (HEAD) t = __builtin_amdgcn_mfma_f32_32x32x16_bf16(slot0(x0a), slot0(g0c), t, 0, 0, 0);
        float d0 = 0.f;  // with the bf16-rounded dP (the operand the fragments carry)
        if (HEAD)
#pragma unroll
          for (int r = 0; r < 16; ++r) d0 += X0(q)[ta * 32 + frag_row(r)] * bf2f(f2bf(t[r]));
        if (HEAD) {
          d0 += __shfl_xor(d0, 32, 64);
          dw0[tc] += d0;
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const bf16x8 f = frag_of(t, s);
          const int ka = ta * 32 + 16 * s + 4 * h;
#pragma unroll
          for (int tj = 0; tj < NJ; ++tj)
            dw[tj][tc] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                ld_perm(Xs(q) + (tj * 32 + l32) * LX + ka), f, dw[tj][tc], 0, 0, 0);
        }
      }
    }
    __syncthreads();  // the LDS is restaged for the next samples
  }
  // block partial of dW: the waves' tiles added in wave order
  float* red = reinterpret_cast<float*>(smem);  // [NW][16][64], then [NW][K]
  float* red0 = red + NW * 16 * 64;
#pragma unroll
  for (int tj = 0; tj < NJ; ++tj)
#pragma unroll
    for (int tc = 0; tc < NC; ++tc) {
#pragma unroll
      for (int r = 0; r < 16; ++r) red[(w * 16 + r) * 64 + lane] = dw[tj][tc][r];
      __syncthreads();
      for (int e = threadIdx.x; e < 16 * 64; e += THREADS) {
        float v = red[e];
        for (int ww = 1; ww < NW; ++ww) v += red[ww * 16 * 64 + e];
        const int r = e >> 6, ln = e & 63;
        const int j = tj * 32 + 8 * (r >> 2) + 4 * (ln >> 5) + (r & 3);
        const int c = tc * 32 + (ln & 31);
        if (j < nm) dw_part[((int64_t)blockIdx.x * n + j + H) * K + c] = v;
      }
      __syncthreads();
    }
  if (HEAD) {
    if (h == 0)
#pragma unroll
      for (int tc = 0; tc < NC; ++tc) red0[w * K + tc * 32 + l32] = dw0[tc];
    __syncthreads();
    for (int c = threadIdx.x; c < K; c += THREADS) {
      float v = red0[c];
      for (int ww = 1; ww < NW; ++ww) v += red0[ww * K + c];
      dw_part[(int64_t)blockIdx.x * n * K + c] = v;
    }
  }
}

// out[i] = sum over the blocks' partials part[p][i], in a fixed order: the
// parts are split into 8 consecutive groups, each summed in part order by
// one thread (16 loads in flight), and the 8 group sums are added in group
// order.  A block covers 32 outputs.
__global__ __launch_bounds__(256) void sum_parts_grouped_kernel(const float* __restrict__ part,
                                                                int parts, int64_t len,
                                                                float* __restrict__ out) {
  __shared__ float gs[8][33];
  const int c = threadIdx.x & 31, g = threadIdx.x >> 5;
  const int64_t i = (int64_t)blockIdx.x * 32 + c;
  const int per = (parts + 7) / 8;
  const int p0 = g * per, p1 = min(parts, p0 + per);
  float s = 0.f;
  if (i < len) {
    int p = p0;
    for (; p + 16 <= p1; p += 16) {
      float v[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) v[q] = part[(int64_t)(p + q) * len + i];
#pragma unroll
      for (int q = 0; q < 16; ++q) s += v[q];
    }
    for (; p < p1; ++p) s += part[(int64_t)p * len + i];
  }
  gs[g][c] = s;
  __syncthreads();
  if (g == 0 && i < len) {
    float t = gs[0][c];
#pragma unroll
    for (int q = 1; q < 8; ++q) t += gs[q][c];
    out[i] = t;
  }
}

constexpr int FM_MFMA_BLOCKS = 256;

bool fm_mfma_supported(int n, int d, int k) {
  if (n < 1) return false;
  // up to three (k = 32) or two (k = 64) tiles of 32 rows, plus a head row
  // when n = 32 t + 1
  if (k == 32) return n <= 97 && (d == 64 || d == 128);
  if (k == 64) return n <= 65 && d == 128;
  return false;
}

size_t fm_mfma_bwd_workspace(int n, int k) { return (size_t)FM_MFMA_BLOCKS * n * k * sizeof(float); }

template <int NP, int D, int K, bool HEAD>
static hipError_t fm_mfma_launch(bool fwd, const void* X, const void* W, int B, int n, void* out,
                                 int64_t ostride, int emit0, const void* dout, int64_t dstride,
                                 const float* addend, void* dX, float* dX_f32, float* dW,
                                 void* ws, hipStream_t s) {
  const int blocks = B < FM_MFMA_BLOCKS ? (B > 0 ? B : 1) : FM_MFMA_BLOCKS;
  if (fwd) {
    if (B == 0) return hipSuccess;
    // 4-wave blocks without the X^T copy where three fit a compute unit's
    // LDS (three samples in flight), else 8-wave blocks, two per unit
    constexpr int LX = D + 8, LT = NP + 8, LP = D + 8, LQ = 40;
    constexpr int NQ4 = (NP / 32) * (K / 32) < 4 ? (NP / 32) * (K / 32) : 4;
    constexpr size_t LDS4 = 2 * ((size_t)NP * LX + K * LP + K * LT) + 4 * (HEAD ? D + K : 2) +
                            (size_t)NQ4 * 2 * 32 * LQ;
    if constexpr (3 * LDS4 <= 160 * 1024) {
      const int fblocks = B < 3 * FM_MFMA_BLOCKS ? B : 3 * FM_MFMA_BLOCKS;
      fm_fwd_mfma_kernel<NP, D, K, HEAD, 4, true><<<fblocks, 256, 0, s>>>(
          (const bf16_t*)X, (const bf16_t*)W, B, n, (bf16_t*)out, ostride, emit0);
    } else {
      const int fblocks = B < 2 * FM_MFMA_BLOCKS ? B : 2 * FM_MFMA_BLOCKS;
      fm_fwd_mfma_kernel<NP, D, K, HEAD><<<fblocks, 512, 0, s>>>((const bf16_t*)X, (const bf16_t*)W, B, n,
                                                          (bf16_t*)out, ostride, emit0);
    }
    LAT_LAUNCH_CHECK();
    return hipSuccess;
  }
  float* part = (float*)ws;
  int bblocks = 0;
  // the chained kernel where its registers fit (up to 64 rows in tiles; not
  // rank 64 with a head row)
  constexpr bool CHAIN = D == 128 && NP <= 64 && !(K == 64 && HEAD);
  if constexpr (CHAIN) {
    // two samples per block iteration (8 waves)
    constexpr int SPB = 2;
    static_assert(FmChainLds<NP, K, HEAD, SPB>::bytes <= 160 * 1024, "FM chain LDS");
    const int iters = (B + SPB - 1) / SPB;
    bblocks = iters < FM_MFMA_BLOCKS ? (iters > 0 ? iters : 1) : FM_MFMA_BLOCKS;
    if (B > 0) {
      if (!addend && !dX_f32 && (reinterpret_cast<uintptr_t>(dX) & 15) == 0)
        fm_bwd_chain_kernel<NP, K, HEAD, SPB, true><<<bblocks, SPB * 256, 0, s>>>(
            (const bf16_t*)X, (const bf16_t*)W, B, n, (const bf16_t*)dout, dstride, emit0, addend,
            (bf16_t*)dX, dX_f32, part);
      else
        fm_bwd_chain_kernel<NP, K, HEAD, SPB, false><<<bblocks, SPB * 256, 0, s>>>(
            (const bf16_t*)X, (const bf16_t*)W, B, n, (const bf16_t*)dout, dstride, emit0, addend,
            (bf16_t*)dX, dX_f32, part);
      LAT_LAUNCH_CHECK();
    }
  } else {
    // two samples per block iteration when both fit in LDS
    constexpr int SPB = FmBwdLds<NP, D, K, HEAD, 2>::bytes <= 160 * 1024 ? 2 : 1;
    bblocks = (B + SPB - 1) / SPB < FM_MFMA_BLOCKS ? ((B + SPB - 1) / SPB > 0 ? (B + SPB - 1) / SPB : 1)
                                                   : FM_MFMA_BLOCKS;
    if (B > 0) {
      fm_bwd_mfma_kernel<NP, D, K, HEAD, SPB><<<bblocks, 512, 0, s>>>(
          (const bf16_t*)X, (const bf16_t*)W, B, n, (const bf16_t*)dout, dstride, emit0, addend,
          (bf16_t*)dX, dX_f32, part);
      LAT_LAUNCH_CHECK();
    }
  }
  const int64_t len = (int64_t)n * K;
  sum_parts_grouped_kernel<<<cdiv(len, 32), 256, 0, s>>>(part, B > 0 ? bblocks : 0, len, dW);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t fm_mfma(bool fwd, const void* X, const void* W, int B, int n, int d, int k, void* out,
                   int64_t ostride, int emit0, const void* dout, int64_t dstride,
                   const float* addend, void* dX, float* dX_f32, float* dW, void* ws,
                   hipStream_t s) {
  // n = 32 t + 1: row 0 outside the tiles (exactly t tiles of rows)
  const bool head = n > 1 && (n - 1) % 32 == 0;
#define LAT_FMM(NPV, DV, KV)                                                                    \
  if (head && n - 1 == NPV && d == DV && k == KV)                                               \
    return fm_mfma_launch<NPV, DV, KV, true>(fwd, X, W, B, n, out, ostride, emit0, dout,        \
                                             dstride, addend, dX, dX_f32, dW, ws, s);           \
  if (!head && n <= NPV && d == DV && k == KV)                                                  \
    return fm_mfma_launch<NPV, DV, KV, false>(fwd, X, W, B, n, out, ostride, emit0, dout,       \
                                              dstride, addend, dX, dX_f32, dW, ws, s);
  LAT_FMM(32, 128, 32) LAT_FMM(64, 128, 32) LAT_FMM(96, 128, 32)
  LAT_FMM(32, 64, 32) LAT_FMM(64, 64, 32) LAT_FMM(96, 64, 32)
  LAT_FMM(32, 128, 64) LAT_FMM(64, 128, 64)
#undef LAT_FMM
  set_error("FM MFMA path: unsupported shape n=%d d=%d k=%d", n, d, k);
  return hipErrorInvalidValue;
}

}  // namespace lat
