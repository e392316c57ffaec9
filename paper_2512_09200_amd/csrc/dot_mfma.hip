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
constexpr int DOT_MASK_WORDS = 4;  // slot bitmask words per sample (n <= 128)

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

// ---------------------------------------------------------------------------
// Listed slots only (forward).  A per-sample bitmask of DOT_MASK_WORDS
// words (bit s of word s / 32: slot s may be non-zero; bits at or past n are
// ignored) lets the forward work on the listed slots: the caller guarantees
// that every unlisted slot holds a zero vector (absent features are
// zero-padded, Section 3.2), so a pair touching one is exactly 0.  With na
// listed slots (row r of the compact matrix = the r-th listed slot,
// ascending) the listed rows are staged compactly, only the tiles on or above
// the diagonal of the compact Gram matrix are computed (for n = 97 with 42
// listed: 3 tiles instead of 10), and the pairs are scattered into the
// zero-filled packed row; the results equal the full kernel's.  The lists of
// the next sample are built in LDS one iteration ahead, so the prefetch of
// its rows reads its slots from there, and its mask words are loaded one
// more iteration ahead.  (A backward over the listed slots, S [n, na] times
// the compact X, measured slower than the full backward: 156 against 121 us
// at n = 97 with 42 listed, so the backward always runs over every slot.)
struct SlotMask {
  uint32_t m[DOT_MASK_WORDS];
  int na;
};

// sample b's mask words, as a vector load (issued with the row prefetch and
// counted in order with it; a scalar load would be waited for at the next
// barrier).  The offset is a zero held in a vector register the compiler
// cannot see through, so the address stays per lane.
__device__ inline u32x4 slot_mask_load(const uint32_t* __restrict__ mask, int b) {
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  return *reinterpret_cast<const u32x4*>(mask + (int64_t)b * DOT_MASK_WORDS + z);
}

// the mask with the bits at or past n cleared, and its count
__device__ inline SlotMask slot_mask_of(const u32x4 raw, int n) {
  SlotMask sm;
  sm.na = 0;
#pragma unroll
  for (int w = 0; w < DOT_MASK_WORDS; ++w) {
    const int lim = n - 32 * w;
    const uint32_t valid = lim >= 32 ? 0xffffffffu : (lim <= 0 ? 0u : (1u << lim) - 1u);
    sm.m[w] = raw[w] & valid;
    sm.na += __popc(sm.m[w]);
  }
  return sm;
}

// lst[r] = r-th listed slot (r < na).  Thread t handles slot t (t < n).
__device__ inline void slot_lists(const SlotMask& sm, int n, uint8_t* lst) {
  const int t = threadIdx.x;
  if (t >= n) return;
  const int w = t >> 5, bit = t & 31;
  uint32_t mw = sm.m[0];
  int below = 0;
#pragma unroll
  for (int k = 1; k < DOT_MASK_WORDS; ++k)
    if (w >= k) {
      below += __popc(mw);
      mw = sm.m[k];
    }
  const bool on = (mw >> bit) & 1u;
  const int r = below + __popc(mw & ((1u << bit) - 1u));
  if (on) lst[r] = (uint8_t)t;
}

// Stager over the listed rows: compact row r reads slot lst[r] of the
// sample (r < na), rows past na read slot 0 and are stored as zeros.
template <int RP, int COLS, int THREADS>
struct ListStager {
  static constexpr int ITEMS = (RP / 8) * (COLS / 2);
  static constexpr int PER = (ITEMS + THREADS - 1) / THREADS;
  uint32_t v[PER][8];
  __device__ inline void load(const bf16_t* __restrict__ g, const uint8_t* lst, int na) {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      int it = threadIdx.x + q * THREADS;
      it = it < ITEMS ? it : ITEMS - 1;
      const int j0 = (it / (COLS / 2)) * 8, c = (it % (COLS / 2)) * 2;
      const uint2 sl = *reinterpret_cast<const uint2*>(lst + j0);  // 8 slots
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t word = i < 4 ? sl.x : sl.y;
        const int slot = j0 + i < na ? (int)((word >> (8 * (i & 3))) & 0xffu) : 0;
        v[q][i] = *reinterpret_cast<const uint32_t*>(g + (int64_t)slot * COLS + c);
      }
    }
  }
  __device__ inline void store(bf16_t* R, int ldr, bf16_t* T, int ldt, int na) const {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int it = threadIdx.x + q * THREADS;
      if (it < ITEMS) {
        const int j0 = (it / (COLS / 2)) * 8, c = (it % (COLS / 2)) * 2;
        uint32_t x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = j0 + i < na ? v[q][i] : 0u;
        if (R)
#pragma unroll
          for (int i = 0; i < 8; ++i) *reinterpret_cast<uint32_t*>(R + (j0 + i) * ldr + c) = x[i];
        if (!T) continue;
        u32x4 lo, hi;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          lo[i] = __builtin_amdgcn_perm(x[2 * i + 1], x[2 * i], 0x05040100u);
          hi[i] = __builtin_amdgcn_perm(x[2 * i + 1], x[2 * i], 0x07060302u);
        }
        *reinterpret_cast<u32x4*>(T + c * ldt + j0) = lo;
        *reinterpret_cast<u32x4*>(T + (c + 1) * ldt + j0) = hi;
      }
    }
  }
};

template <int NP, int D>
__global__ __launch_bounds__(DOT_THREADS) void dot_fwd_listed_kernel(const bf16_t* __restrict__ X,
                                                                     int B, int n,
                                                                     const uint32_t* __restrict__ mask,
                                                                     bf16_t* __restrict__ out,
                                                                     int64_t ostride, int emit0) {
  constexpr int LX = D + 8;
  constexpr int PMAX = NP * (NP - 1) / 2;
  __shared__ __attribute__((aligned(16))) bf16_t Xs[NP * LX];
  __shared__ __attribute__((aligned(16))) bf16_t Zp[(PMAX + 7) / 8 * 8];
  __shared__ __attribute__((aligned(16))) uint8_t lst[2][NP];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int P = n * (n - 1) / 2;
  const int off = emit0 ? D : 0;
  ListStager<NP, D, DOT_THREADS> sx;
  const int G = (int)gridDim.x;
  int na_next = 0;
  u32x4 mraw = {0u, 0u, 0u, 0u};  // mask words of the sample after the next
  if (blockIdx.x < B) {
    const SlotMask sm = slot_mask_of(slot_mask_load(mask, blockIdx.x), n);
    slot_lists(sm, n, lst[0]);
    na_next = sm.na;
  }
  if (blockIdx.x + G < B) mraw = slot_mask_load(mask, blockIdx.x + G);
  __syncthreads();
  if (blockIdx.x < B) sx.load(X + (int64_t)blockIdx.x * n * D, lst[0], na_next);
  int cur = 0;
  for (int b = blockIdx.x; b < B; b += G, cur ^= 1) {
    const int na = na_next;
    const int nb = b + G;
    sx.store(Xs, LX, nullptr, 0, na);
    for (int v = threadIdx.x; v < (P + 7) / 8; v += DOT_THREADS)
      *reinterpret_cast<u32x4*>(Zp + v * 8) = u32x4{0u, 0u, 0u, 0u};
    if (nb < B) {
      const SlotMask sm = slot_mask_of(mraw, n);
      slot_lists(sm, n, lst[cur ^ 1]);
      na_next = sm.na;
    }
    __syncthreads();
    if (nb + G < B) mraw = slot_mask_load(mask, nb + G);
    if (nb < B) sx.load(X + (int64_t)nb * n * D, lst[cur ^ 1], na_next);
    const int TA = (na + 31) / 32;
    const int ZA = TA * (TA + 1) / 2;
    const uint8_t* L = lst[cur];
    for (int t = w; t < ZA; t += DOT_THREADS / 64) {
      int ti = 0, rem = t;
      while (rem >= TA - ti) {
        rem -= TA - ti;
        ++ti;
      }
      const int tj = ti + rem;
      f32x16 acc;
      zero16(acc);
      mfma_tile<D>(acc, Xs + ti * 32 * LX, LX, Xs + tj * 32 * LX, LX);
      const int rj = tj * 32 + (lane & 31);
      const int j = rj < na ? L[rj] : 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ri = ti * 32 + frag_row(r);
        if (ri < rj && rj < na) {
          const int i = L[ri];
          Zp[pair_start(i, n) + (j - i - 1)] = f2bf(acc[r]);
        }
      }
    }
    __syncthreads();
    bf16_t* ob = out + (int64_t)b * ostride;
    if (emit0)
      for (int a = threadIdx.x; a < D; a += DOT_THREADS) ob[a] = X[(int64_t)b * n * D + a];
    bf16_t* dst = ob + off;
    int done = 0;
    if ((reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
      const int nv = P / 8;
      for (int v = threadIdx.x; v < nv; v += DOT_THREADS)
        *reinterpret_cast<u32x4*>(dst + v * 8) = *reinterpret_cast<const u32x4*>(Zp + v * 8);
      done = nv * 8;
    }
    for (int m = done + threadIdx.x; m < P; m += DOT_THREADS) dst[m] = Zp[m];
    __syncthreads();  // Xs, Zp and this sample's list are rewritten next
  }
}

// Slot masks of a batch (feature-major bags): bit 0 when has0 (the dense
// vector), and bit first + f for every feature f whose bag is non-empty.
// Thread (word w, sample b) builds word w of sample b.
__global__ __launch_bounds__(256) void dot_slot_mask_kernel(const int32_t* __restrict__ offsets, int F,
                                                            int B, int first, int has0,
                                                            uint32_t* __restrict__ mask) {
  const int64_t tid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (tid >= (int64_t)DOT_MASK_WORDS * B) return;
  const int wd = (int)(tid / B), b = (int)(tid - (int64_t)wd * B);
  uint32_t m = (has0 && wd == 0) ? 1u : 0u;
  const int s0 = 32 * wd;
  const int f0 = max(0, s0 - first), cnt = min(F, s0 + 32 - first) - f0;
  if (cnt > 0) {
    // the word's (up to 32) bags: both ends of each loaded as straight-line
    // code from clamped positions, so all loads are in flight together
    int32_t lo[32], hi[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      const int64_t o = (int64_t)(f0 + min(k, cnt - 1)) * B + b;
      lo[k] = offsets[o];
      hi[k] = offsets[o + 1];
    }
#pragma unroll
    for (int k = 0; k < 32; ++k)
      if (k < cnt && hi[k] > lo[k]) m |= 1u << (first + f0 + k - s0);
  }
  mask[(int64_t)b * DOT_MASK_WORDS + wd] = m;
}

hipError_t dot_slot_mask(const int32_t* offsets, int F, int B, int first, int has0, uint32_t* mask,
                         hipStream_t s) {
  if (B == 0) return hipSuccess;
  if (first + F > DOT_MASK_WORDS * 32 || first < 0) {
    set_error("DOT slot mask: slots up to %d exceed %d", first + F, DOT_MASK_WORDS * 32);
    return hipErrorInvalidValue;
  }
  dot_slot_mask_kernel<<<cdiv((int64_t)DOT_MASK_WORDS * B, 256), 256, 0, s>>>(offsets, F, B, first, has0, mask);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

bool dot_mfma_supported(int n, int d) { return n >= 1 && n <= 128 && (d == 64 || d == 128); }

template <int NP, int D>
static hipError_t dot_mfma_launch(bool fwd, const void* X, int B, int n, void* out,
                                  int64_t ostride, int emit0, const void* dout, int64_t dstride,
                                  void* dX, const uint32_t* mask, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const int blocks = B < DOT_BLOCKS ? B : DOT_BLOCKS;
  if (fwd && mask)
    dot_fwd_listed_kernel<NP, D><<<blocks, DOT_THREADS, 0, s>>>((const bf16_t*)X, B, n, mask,
                                                               (bf16_t*)out, ostride, emit0);
  else if (fwd)
    dot_fwd_mfma_kernel<NP, D><<<blocks, DOT_THREADS, 0, s>>>((const bf16_t*)X, B, n,
                                                             (bf16_t*)out, ostride, emit0);
  else
    dot_bwd_mfma_kernel<NP, D><<<blocks, DOT_THREADS, 0, s>>>(
        (const bf16_t*)X, B, n, (const bf16_t*)dout, dstride, emit0, (bf16_t*)dX);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t dot_mfma(bool fwd, const void* X, int B, int n, int d, void* out, int64_t ostride,
                    int emit0, const void* dout, int64_t dstride, void* dX, const uint32_t* mask,
                    hipStream_t s) {
#define LAT_DOTM(NPV, DV)                                                                  \
  if (n <= NPV && d == DV)                                                                 \
    return dot_mfma_launch<NPV, DV>(fwd, X, B, n, out, ostride, emit0, dout, dstride, dX, mask, s);
  LAT_DOTM(32, 64) LAT_DOTM(64, 64) LAT_DOTM(96, 64) LAT_DOTM(128, 64)
  LAT_DOTM(32, 128) LAT_DOTM(64, 128) LAT_DOTM(96, 128) LAT_DOTM(128, 128)
#undef LAT_DOTM
  set_error("DOT MFMA path: unsupported shape n=%d d=%d", n, d);
  return hipErrorInvalidValue;
}

}  // namespace lat
