// Dense contractions of the MLPs and heads:
//   C[m, n] = epilogue( sum_k A(m, k) * B(n, k) )
// with A(m,k) = A[m*lda + k] (K-contiguous) or A[k*lda + m] (M-contiguous),
// and likewise for B, so the forward (X W^T), input-gradient (dY W) and
// weight-gradient (dY^T X) products all map onto one kernel family without
// materialised transposes.
//
// bf16 path (gfx950 MFMA): block tile 128x128, K step 32, 256 threads as a
// 2x2 grid of waves each owning a 64x64 sub-tile = 2x2 fragments of
// v_mfma_f32_32x32x16_bf16.  Operands are staged through LDS in [row][k]
// layout (k contiguous, rows padded to 40 elements so 16-byte fragment reads
// of 16 lanes hit 64 distinct banks).  A K-contiguous operand is copied with
// 16-byte loads; an M-contiguous operand is read as 2-element pairs along M
// (coalesced across the wave) and transposed in registers before the LDS
// write.  Global loads of step k+1 overlap the MFMAs of step k (double
// buffer).  Split-K writes fp32 partials that a second kernel sums in a fixed
// order, so results are deterministic.
//
// Epilogue: + bias[n], ReLU, or multiply by (mask[m, n] > 0) (the ReLU
// derivative read from a stored activation), then round to the output dtype.
#include "common.h"
#include "kernels.h"

namespace lat {

constexpr int GBM = 128, GBN = 128, GBK = 32, GPAD = 8, GLD = GBK + GPAD;

struct Epi {
  const float* bias;    // [N] or null
  int relu;
  const void* mask;     // activation whose sign gates the output, or null
  DType mask_dt;
  int64_t ldm, s_mask;
  const float* addend;  // + addend[m*ld_add + n] (fp32) or null
  int64_t ld_add, s_add;
  int accumulate;       // + the existing (fp32) C
};

template <typename CT>
__device__ inline void epi_store(CT* C, int64_t ldc, int row, int col, float v, const Epi& e,
                                 int64_t bz) {
  if (e.bias) v += e.bias[col];
  if (e.addend) v += e.addend[bz * e.s_add + (int64_t)row * e.ld_add + col];
  if (e.accumulate) v += ld(C + (int64_t)row * ldc + col);
  if (e.relu) v = v > 0.f ? v : 0.f;
  if (e.mask) {
    const int64_t mi = bz * e.s_mask + (int64_t)row * e.ldm + col;
    float g = e.mask_dt == DT_BF16 ? bf2f(((const bf16_t*)e.mask)[mi]) : ((const float*)e.mask)[mi];
    v = g > 0.f ? v : 0.f;
  }
  st(C + (int64_t)row * ldc + col, v);
}

// An operand: element (r, k) of A(m,k) / B(n,k).  K-contiguous: p[r*ld + koff(k)];
// MN-contiguous: p[koff(k)*... + r] with koff(k) counted in rows of length ld.
// K segmentation splits k into (k / kseg, k % kseg): the segment index moves by
// ks elements (batched sums over samples as one contraction).
struct Opnd {
  const bf16_t* p;
  int64_t ld;
  int kseg;     // 0: no segmentation
  int64_t ks;
};
template <bool MN>
__device__ inline int64_t koff(const Opnd& o, int k) {
  if (o.kseg == 0) return MN ? (int64_t)k * o.ld : (int64_t)k;
  const int q = k / o.kseg, r = k - q * o.kseg;
  return (int64_t)q * o.ks + (MN ? (int64_t)r * o.ld : (int64_t)r);
}

// --- operand tile loaders: fill S[rows][GLD] (k contiguous) for rows r0.., k k0.. ---
// K-contiguous, 16-byte vectors: 128 rows x 32 k = 4 vectors per row, 2 per thread.
struct LoadK {
  u32x4 r[2];
  __device__ void load(const Opnd& o, int R, int K, int r0, int k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int v = threadIdx.x + i * 256;
      const int rr = v >> 2, kc = (v & 3) * 8;
      const int gr = r0 + rr, gk = k0 + kc;
      if (gr < R && gk < K) r[i] = ldg16(o.p + (int64_t)gr * o.ld + koff<false>(o, gk));
      else r[i] = u32x4{0, 0, 0, 0};
    }
  }
  __device__ void store(bf16_t* S) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int v = threadIdx.x + i * 256;
      *reinterpret_cast<u32x4*>(S + (v >> 2) * GLD + (v & 3) * 8) = r[i];
    }
  }
};
// MN-contiguous: thread owns rows (2p, 2p+1) and 8 consecutive k (wave w -> k 8w..8w+7),
// read as 4-byte row pairs (coalesced across the wave) and transposed in registers.
struct LoadMN {
  uint32_t r[8];
  __device__ void load(const Opnd& o, int R, int K, int r0, int k0) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int gr = r0 + 2 * lane;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int gk = k0 + w * 8 + i;
      if (gk < K && gr < R) r[i] = *reinterpret_cast<const uint32_t*>(o.p + koff<true>(o, gk) + gr);
      else r[i] = 0u;
    }
  }
  __device__ void store(bf16_t* S) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    u32x4 lo, hi;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // r[k] = (row 2p at k) | (row 2p+1 at k) << 16
      lo[i] = __builtin_amdgcn_perm(r[2 * i + 1], r[2 * i], 0x05040100u);  // low halves
      hi[i] = __builtin_amdgcn_perm(r[2 * i + 1], r[2 * i], 0x07060302u);  // high halves
    }
    *reinterpret_cast<u32x4*>(S + (2 * lane) * GLD + w * 8) = lo;
    *reinterpret_cast<u32x4*>(S + (2 * lane + 1) * GLD + w * 8) = hi;
  }
};
// Generic element loader (any alignment / transposition).
template <bool MN>
struct LoadElem {
  bf16_t r[16];
  __device__ void load(const Opnd& o, int R, int K, int r0, int k0) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int e = threadIdx.x + i * 256;
      const int rr = e >> 5, kk = e & 31;
      const int gr = r0 + rr, gk = k0 + kk;
      bf16_t v = 0;
      if (gr < R && gk < K) v = MN ? o.p[koff<true>(o, gk) + gr] : o.p[(int64_t)gr * o.ld + koff<false>(o, gk)];
      r[i] = v;
    }
  }
  __device__ void store(bf16_t* S) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int e = threadIdx.x + i * 256;
      S[(e >> 5) * GLD + (e & 31)] = r[i];
    }
  }
};
template <bool MN, bool VEC> struct LoaderSel;
template <> struct LoaderSel<false, true> { using T = LoadK; };
template <> struct LoaderSel<true, true> { using T = LoadMN; };
template <bool MN> struct LoaderSel<MN, false> { using T = LoadElem<MN>; };

// blockIdx.z: split index (split-K) or batch index (batched; never both)
template <bool TA, bool TB, bool VA, bool VB, typename CT>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(
    Opnd A, Opnd Bm, CT* __restrict__ C, int64_t ldc, int M, int N, int K, int k_per_split,
    float* __restrict__ partial, Epi epi, int64_t sA, int64_t sB, int64_t sC, int batched) {
  __shared__ __attribute__((aligned(16))) bf16_t As[2][GBM * GLD];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][GBN * GLD];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int m0 = blockIdx.y * GBM, n0 = blockIdx.x * GBN;
  const int64_t bz = batched ? blockIdx.z : 0;
  if (batched) {
    A.p += bz * sA;
    Bm.p += bz * sB;
    C += bz * sC;
  }
  const int kbeg = batched ? 0 : blockIdx.z * k_per_split;
  const int kend = batched ? K : min(K, kbeg + k_per_split);

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  typename LoaderSel<TA, VA>::T la;
  typename LoaderSel<TB, VB>::T lb;
  const int ktiles = (kend - kbeg + GBK - 1) / GBK;
  if (ktiles > 0) {
    la.load(A, M, kend, m0, kbeg);
    lb.load(Bm, N, kend, n0, kbeg);
    la.store(As[0]);
    lb.store(Bs[0]);
  }
  __syncthreads();
  const int frow = lane & 31, fk = (lane >> 5) * 8;
  for (int kt = 0; kt < ktiles; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < ktiles;
    if (more) {
      la.load(A, M, kend, m0, kbeg + (kt + 1) * GBK);
      lb.load(Bm, N, kend, n0, kbeg + (kt + 1) * GBK);
    }
    const bf16_t* as = As[cur] + (wm * 64 + frow) * GLD + fk;
    const bf16_t* bs = Bs[cur] + (wn * 64 + frow) * GLD + fk;
#pragma unroll
    for (int ks = 0; ks < GBK; ks += 16) {
      bf16x8 a0 = *reinterpret_cast<const bf16x8*>(as + ks);
      bf16x8 a1 = *reinterpret_cast<const bf16x8*>(as + 32 * GLD + ks);
      bf16x8 b0 = *reinterpret_cast<const bf16x8*>(bs + ks);
      bf16x8 b1 = *reinterpret_cast<const bf16x8*>(bs + 32 * GLD + ks);
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
    }
    if (more) {
      la.store(As[cur ^ 1]);
      lb.store(Bs[cur ^ 1]);
    }
    __syncthreads();
  }

  // D[i][j] of a 32x32 fragment: lane holds column (lane & 31), rows
  // 8*(r/4) + 4*(lane/32) + r%4 for r = 0..15.
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < M && col < N) {
          if (partial) partial[((int64_t)blockIdx.z * M + row) * N + col] = acc[i][j][r];
          else epi_store<CT>(C, ldc, row, col, acc[i][j][r], epi, bz);
        }
      }
    }
  }
}

template <typename CT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ partial,
                                                            int splits, int M, int N,
                                                            CT* __restrict__ C, int64_t ldc,
                                                            Epi epi) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)M * N) return;
  const int row = (int)(i / N), col = (int)(i % N);
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += partial[(int64_t)z * M * N + i];
  epi_store<CT>(C, ldc, row, col, s, epi, 0);
}

// --- fp32 VALU GEMM (fp32 workloads): 64x64 tile, 4x4 per thread, any layout ---
template <typename CT>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int64_t lda,
                                                       int ta, const float* __restrict__ Bm,
                                                       int64_t ldb, int tb, CT* __restrict__ C,
                                                       int64_t ldc, int M, int N, int K,
                                                       Epi epi) {
  constexpr int T = 64, KS = 16;
  __shared__ float As[KS][T + 1];
  __shared__ float Bs[KS][T + 1];
  const int m0 = blockIdx.y * T, n0 = blockIdx.x * T;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += KS) {
    for (int e = threadIdx.x; e < KS * T; e += 256) {
      const int kk = e / T, r = e % T;
      const int gk = k0 + kk;
      const int gm = m0 + r, gn = n0 + r;
      As[kk][r] = (gm < M && gk < K) ? (ta ? A[(int64_t)gk * lda + gm] : A[(int64_t)gm * lda + gk]) : 0.f;
      Bs[kk][r] = (gn < N && gk < K) ? (tb ? Bm[(int64_t)gk * ldb + gn] : Bm[(int64_t)gn * ldb + gk]) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
      if (row < M && col < N) epi_store<CT>(C, ldc, row, col, acc[i][j], epi, 0);
    }
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }
static bool aligned4(const void* p) { return ((uintptr_t)p & 3) == 0; }

int gemm_splits(const GemmArgs& g) {
  if (g.dt != DT_BF16 || g.batch > 1) return 1;
  const int tiles = cdiv(g.M, GBM) * cdiv(g.N, GBN);
  int s = 1;
  // fill the 256 compute units at least twice over when K is long enough
  while (tiles * s < 512 && g.K / (s * 2) >= 512 && s * 2 <= g.max_splits) s *= 2;
  return s;
}

size_t gemm_workspace(const GemmArgs& g) {
  int splits = gemm_splits(g);
  return splits > 1 ? (size_t)splits * g.M * g.N * sizeof(float) : 0;
}

static Epi make_epi(const GemmArgs& g) {
  return Epi{g.bias, g.relu, g.mask, g.mask_dt, g.ldm, g.s_mask, g.addend, g.ld_add, g.s_add,
             g.accumulate};
}

template <bool TA, bool TB, bool VA, bool VB>
static hipError_t gemm_bf16_launch(const GemmArgs& g, float* ws, hipStream_t st) {
  const int splits = gemm_splits(g);
  if (splits > 1 && !ws) {
    set_error("split-K GEMM without a workspace");
    return hipErrorInvalidValue;
  }
  int kps = (g.K + splits - 1) / splits;
  kps = ((kps + GBK - 1) / GBK) * GBK;
  const int batched = g.batch > 1 ? 1 : 0;
  dim3 grid(cdiv(g.N, GBN), cdiv(g.M, GBM), batched ? g.batch : splits);
  Epi epi = make_epi(g);
  Opnd a{(const bf16_t*)g.A, g.lda, g.kseg, g.ksA};
  Opnd b{(const bf16_t*)g.B, g.ldb, g.kseg, g.ksB};
  float* partial = splits > 1 ? ws : nullptr;
  if (g.c_dt == DT_BF16)
    gemm_bf16_kernel<TA, TB, VA, VB, bf16_t><<<grid, 256, 0, st>>>(
        a, b, (bf16_t*)g.C, g.ldc, g.M, g.N, g.K, kps, partial, epi, g.sA, g.sB, g.sC, batched);
  else
    gemm_bf16_kernel<TA, TB, VA, VB, float><<<grid, 256, 0, st>>>(
        a, b, (float*)g.C, g.ldc, g.M, g.N, g.K, kps, partial, epi, g.sA, g.sB, g.sC, batched);
  LAT_LAUNCH_CHECK();
  if (splits > 1) {
    const int64_t n = (int64_t)g.M * g.N;
    if (g.c_dt == DT_BF16)
      splitk_reduce_kernel<bf16_t><<<cdiv(n, 256), 256, 0, st>>>(ws, splits, g.M, g.N, (bf16_t*)g.C, g.ldc, epi);
    else
      splitk_reduce_kernel<float><<<cdiv(n, 256), 256, 0, st>>>(ws, splits, g.M, g.N, (float*)g.C, g.ldc, epi);
    LAT_LAUNCH_CHECK();
  }
  return hipSuccess;
}

template <bool TA, bool TB>
static hipError_t gemm_bf16_dispatch(const GemmArgs& g, float* ws, hipStream_t st) {
  // 16-byte K-vectors need 8-aligned rows (and segments); M-pairs need even rows
  // and 4-byte alignment.  Batch strides must keep the same alignment.
  const bool seg_ok = g.kseg == 0 || (g.kseg % 8 == 0 && g.ksA % 8 == 0 && g.ksB % 8 == 0);
  const bool va = TA ? (g.lda % 2 == 0 && aligned4(g.A) && g.M % 2 == 0 && g.sA % 2 == 0 &&
                        (g.kseg == 0 || g.ksA % 2 == 0))
                     : (g.lda % 8 == 0 && aligned16(g.A) && g.K % 8 == 0 && g.sA % 8 == 0 && seg_ok);
  const bool vb = TB ? (g.ldb % 2 == 0 && aligned4(g.B) && g.N % 2 == 0 && g.sB % 2 == 0 &&
                        (g.kseg == 0 || g.ksB % 2 == 0))
                     : (g.ldb % 8 == 0 && aligned16(g.B) && g.K % 8 == 0 && g.sB % 8 == 0 && seg_ok);
  if (va && vb) return gemm_bf16_launch<TA, TB, true, true>(g, ws, st);
  if (va) return gemm_bf16_launch<TA, TB, true, false>(g, ws, st);
  if (vb) return gemm_bf16_launch<TA, TB, false, true>(g, ws, st);
  return gemm_bf16_launch<TA, TB, false, false>(g, ws, st);
}

hipError_t gemm(const GemmArgs& g, void* ws, hipStream_t st) {
  if (g.M == 0 || g.N == 0 || g.batch == 0) return hipSuccess;
  if (g.accumulate && g.c_dt != DT_F32) {
    set_error("accumulating GEMM needs an fp32 output");
    return hipErrorInvalidValue;
  }
  if (g.dt == DT_BF16) {
    float* w = (float*)ws;
    if (!g.ta && !g.tb) return gemm_bf16_dispatch<false, false>(g, w, st);
    if (!g.ta && g.tb) return gemm_bf16_dispatch<false, true>(g, w, st);
    if (g.ta && !g.tb) return gemm_bf16_dispatch<true, false>(g, w, st);
    return gemm_bf16_dispatch<true, true>(g, w, st);
  }
  if (g.batch > 1 || g.kseg) {
    set_error("fp32 GEMM: batching / K segmentation not supported");
    return hipErrorInvalidValue;
  }
  dim3 grid(cdiv(g.N, 64), cdiv(g.M, 64));
  Epi epi = make_epi(g);
  if (g.c_dt == DT_F32)
    gemm_f32_kernel<float><<<grid, 256, 0, st>>>((const float*)g.A, g.lda, g.ta, (const float*)g.B,
                                                 g.ldb, g.tb, (float*)g.C, g.ldc, g.M, g.N, g.K, epi);
  else
    gemm_f32_kernel<bf16_t><<<grid, 256, 0, st>>>((const float*)g.A, g.lda, g.ta, (const float*)g.B,
                                                  g.ldb, g.tb, (bf16_t*)g.C, g.ldc, g.M, g.N, g.K, epi);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

// --- deterministic column sums: out[n] = sum_m G[m*ld + n] (bias gradients) ---
// Block: 64 columns as 8 groups of 8, 32 row lanes, CS_ROWS rows; partial sums
// combined in a fixed order in LDS, then over row chunks in a second kernel.
constexpr int CS_ROWS = 256;
template <typename T>
__global__ __launch_bounds__(256) void colsum_partial_kernel(const T* __restrict__ G, int64_t ldG,
                                                             int M, int N, int vec,
                                                             float* __restrict__ part) {
  constexpr int VE = 16 / sizeof(T);
  __shared__ float red[32][65];
  const int cg = threadIdx.x & 7, rl = threadIdx.x >> 3;
  const int col0 = blockIdx.x * 64 + cg * 8;
  const int r0 = blockIdx.y * CS_ROWS, r1 = min(M, r0 + CS_ROWS);
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  if (vec && col0 + 8 <= N) {
#pragma unroll 4
    for (int r = r0 + rl; r < r1; r += 32) {
      const T* g = G + (int64_t)r * ldG + col0;
#pragma unroll
      for (int h = 0; h < 8; h += VE) {
        float t[VE];
        Vec16<T>::unpack(ldg16(g + h), t);
#pragma unroll
        for (int i = 0; i < VE; ++i) acc[h + i] += t[i];
      }
    }
  } else {
    for (int r = r0 + rl; r < r1; r += 32)
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (col0 + i < N) acc[i] += ld(G + (int64_t)r * ldG + col0 + i);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) red[rl][cg * 8 + i] = acc[i];
  __syncthreads();
  if (threadIdx.x < 64) {
    const int col = blockIdx.x * 64 + threadIdx.x;
    float s = 0.f;
    for (int i = 0; i < 32; ++i) s += red[i][threadIdx.x];
    if (col < N) part[(int64_t)blockIdx.y * N + col] = s;
  }
}
__global__ __launch_bounds__(256) void colsum_final_kernel(const float* __restrict__ part,
                                                           int chunks, int N,
                                                           float* __restrict__ out) {
  const int col = blockIdx.x * 256 + threadIdx.x;
  if (col >= N) return;
  float s = 0.f;
  for (int c = 0; c < chunks; ++c) s += part[(int64_t)c * N + col];
  out[col] = s;
}

size_t colsum_workspace(int M, int N) { return (size_t)cdiv(M > 0 ? M : 1, CS_ROWS) * N * sizeof(float); }

hipError_t colsum(const void* G, DType dt, int64_t ld, int M, int N, float* out, void* ws,
                  hipStream_t st) {
  if (N == 0) return hipSuccess;
  const int chunks = cdiv(M > 0 ? M : 1, CS_ROWS);
  float* part = (float*)ws;
  if (M == 0) {
    colsum_final_kernel<<<cdiv(N, 256), 256, 0, st>>>(part, 0, N, out);
    LAT_LAUNCH_CHECK();
    return hipSuccess;
  }
  dim3 grid(cdiv(N, 64), chunks);
  const int ve = dt == DT_BF16 ? 8 : 4;
  const int vec = (ld % ve == 0) && (((uintptr_t)G & 15) == 0);
  if (dt == DT_BF16)
    colsum_partial_kernel<bf16_t><<<grid, 256, 0, st>>>((const bf16_t*)G, ld, M, N, vec, part);
  else
    colsum_partial_kernel<float><<<grid, 256, 0, st>>>((const float*)G, ld, M, N, vec, part);
  LAT_LAUNCH_CHECK();
  colsum_final_kernel<<<cdiv(N, 256), 256, 0, st>>>(part, chunks, N, out);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
