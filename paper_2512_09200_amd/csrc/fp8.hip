// FP8 (OCP e4m3) linear layers with tensor-wise or row-wise scaling
// (Section 3.5.2: FP8 GEMMs for the linear layers, tensor- or row-wise
// scalers rather than block-wise ones; normalisation stays in fp32).
//
// Quantisation of a matrix X [rows, cols]: s = amax / 448 over a row
// (row-wise) or over the whole matrix (tensor-wise), s = 1 for an all-zero
// row / matrix, r = 1 / s, and q = e4m3(x * r) with s, r and x * r fp32
// (correctly rounded) and the product rounded to the nearest e4m3 value, ties
// to even, saturating at +-448.  The rounding is the hardware conversion
// (v_cvt_pk_fp8_f32), measured on gfx950 to give round-to-nearest-even
// e4m3 codes for every finite fp32 value of magnitude up to 448 (1 + 2^-20)
// (|x * r| stays below 448 (1 + 2^-22)); the product is clamped to +-448
// first, so an overflowing reciprocal scale saturates as well.  Codes are
// stored row-major with a row stride of ldq bytes (a multiple of 16); bytes
// past cols are written as zeros.  Several matrices of one dtype can be
// quantised row-wise in one launch (the forward of an FP8 MLP quantises its
// input and every layer's weights together).
//
// Linear layer: Y[m, n] = act( (sum_k qa[m,k] qw[n,k]) * sa[m] * sw[n] + b[n] )
// with the contraction on v_mfma_scale_f32_32x32x64_f8f6f4 (fp8 x fp8, unit
// block scales: the row / tensor scales are applied in the epilogue), block
// tile 128 x 128, K step 128 bytes, 2 x 2 waves of 64 x 64, operands staged
// through LDS two K steps ahead as in the bf16 kernel.
//
// Accumulation.  Measured on gfx950, this instruction adds its 64 products
// and the incoming accumulator after aligning them to the largest exponent
// among them, keeping about 13 fraction bits: 1 + 2^-13 survives, 1 + 2^-14
// does not, and an accumulator of ~1000 absorbs products at the 2^-3 level.
// Chaining the accumulator through the whole K ("fast accumulation") thus
// loses low bits relative to the running sum (the paper trains with fast
// accumulation off and serves with it on).  The precise mode therefore
// starts every 128-k block from zero (two chained instructions) and adds
// its result to the fp32 accumulator with an ordinary fp32 add: each block's
// alignment is relative to its own 128 products only.
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace lat {

typedef int i32x8 __attribute__((ext_vector_type(8)));

// Four fp32 values (already scaled) -> four e4m3 codes in one word, byte e
// = value e: round to nearest even, saturating at +-448.
__device__ inline uint32_t e4m3x4(float a, float b, float c, float d) {
  auto cl = [](float v) { return __builtin_amdgcn_fmed3f(v, -448.f, 448.f); };
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(cl(a), cl(b), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(cl(c), cl(d), w, true);
  return (uint32_t)w;
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

template <typename IT>
__device__ inline float ldf(const IT* p) { return ld(p); }

// Row-wise: one wave per row; the row is read once with 16-byte loads (8
// bf16 or 4 fp32 per load, kept in registers for rows of up to 64 * 8 * RV
// elements), its amax reduced across the wave, then the codes written 8 per
// lane-step.  Longer rows take the generic loop.  Tensor-wise: the same
// kernel with a given scale (scale_in), after the two amax kernels below.
// A launch covers the jobs of Fp8Jobs, job k taking blocks blk0[k] ..
// blk0[k+1]-1 (four rows per block).
template <typename IT, bool ROWWISE>
__global__ __launch_bounds__(256) void fp8_quant_kernel(Fp8Jobs J, const float* __restrict__ scale_in) {
  constexpr int RV = 6;                      // 8-element chunks per lane kept in registers
  const int lane = threadIdx.x & 63;
  int k = 0;
#pragma unroll
  for (int t = 1; t < FP8_MAX_JOBS; ++t)
    if (t < J.n && (int)blockIdx.x >= J.blk0[t]) k = t;
  const Fp8RowJob& jb = J.j[k];
  const int rows = jb.rows, cols = jb.cols;
  const int64_t ld = jb.ld, ldq = jb.ldq;
  const int row = __builtin_amdgcn_readfirstlane(((int)blockIdx.x - J.blk0[k]) * 4 + (threadIdx.x >> 6));
  if (row >= rows) return;
  const IT* xr = static_cast<const IT*>(jb.x) + (int64_t)row * ld;
  uint8_t* qr = jb.q + (int64_t)row * ldq;
  float* scales = jb.scales;
  const bool vec = cols >= 8 && (cols % 8 == 0) && (ld % 8 == 0) && ((uintptr_t)jb.x % 16 == 0) && cols <= 64 * 8 * RV;
  if (vec) {
    float v[RV][8];
    float m = 0.f;
    // straight-line loads from clamped addresses (a load inside a branch
    // would be waited for right there); chunks past the row count as zero
#pragma unroll
    for (int i = 0; i < RV; ++i) {
      const int c0 = (lane + 64 * i) * 8;
      const int cc = c0 < cols ? c0 : cols - 8;
      if constexpr (sizeof(IT) == 2) {
        Vec16<bf16_t>::unpack(ldg16(reinterpret_cast<const bf16_t*>(xr) + cc), v[i]);
      } else {
        const f32x4 a = *reinterpret_cast<const f32x4*>(xr + cc);
        const f32x4 b = *reinterpret_cast<const f32x4*>(xr + cc + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) { v[i][e] = a[e]; v[i][4 + e] = b[e]; }
      }
    }
#pragma unroll
    for (int i = 0; i < RV; ++i) {
      const bool ok = (lane + 64 * i) * 8 < cols;
#pragma unroll
      for (int e = 0; e < 8; ++e) m = fmaxf(m, ok ? fabsf(v[i][e]) : 0.f);
    }
    float s;
    if (ROWWISE) {
      m = wave_max(m);
      s = m > 0.f ? m / 448.f : 1.f;
      if (lane == 0) scales[row] = s;
    } else {
      s = scale_in[0];
    }
    const float rs = 1.f / s;
#pragma unroll
    for (int i = 0; i < RV; ++i) {
      const int c0 = (lane + 64 * i) * 8;
      if (c0 < cols) {
        const float* t = v[i];
        const uint32_t w0 = e4m3x4(t[0] * rs, t[1] * rs, t[2] * rs, t[3] * rs);
        const uint32_t w1 = e4m3x4(t[4] * rs, t[5] * rs, t[6] * rs, t[7] * rs);
        *reinterpret_cast<u32x2*>(qr + c0) = u32x2{w0, w1};
      }
    }
    // zero padding of the code row (cols .. ldq-1)
    for (int c0 = cols + lane * 8; c0 < ldq; c0 += 512) *reinterpret_cast<u32x2*>(qr + c0) = u32x2{0u, 0u};
    return;
  }
  const bool vec_long = cols % 8 == 0 && ld % 8 == 0 && (uintptr_t)jb.x % 16 == 0 && cols > 64 * 8 * RV;
  if (vec_long) {
    // rows too long for the registers: two passes of 16-byte loads (the
    // second re-reads the wave's row, mostly from cache)
    auto ld8 = [&](int c0, float* v) {
      if constexpr (sizeof(IT) == 2) {
        Vec16<bf16_t>::unpack(ldg16(reinterpret_cast<const bf16_t*>(xr) + c0), v);
      } else {
        const f32x4 a = *reinterpret_cast<const f32x4*>(xr + c0);
        const f32x4 b = *reinterpret_cast<const f32x4*>(xr + c0 + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) { v[e] = a[e]; v[4 + e] = b[e]; }
      }
    };
    float s;
    if (ROWWISE) {
      float m = 0.f;
      for (int c0 = lane * 8; c0 < cols; c0 += 512) {
        float v[8];
        ld8(c0, v);
#pragma unroll
        for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(v[e]));
      }
      m = wave_max(m);
      s = m > 0.f ? m / 448.f : 1.f;
      if (lane == 0) scales[row] = s;
    } else {
      s = scale_in[0];
    }
    const float rs = 1.f / s;
    for (int c0 = lane * 8; c0 < cols; c0 += 512) {
      float v[8];
      ld8(c0, v);
      const uint32_t w0 = e4m3x4(v[0] * rs, v[1] * rs, v[2] * rs, v[3] * rs);
      const uint32_t w1 = e4m3x4(v[4] * rs, v[5] * rs, v[6] * rs, v[7] * rs);
      *reinterpret_cast<u32x2*>(qr + c0) = u32x2{w0, w1};
    }
    for (int c0 = cols + lane * 8; c0 < ldq; c0 += 512) *reinterpret_cast<u32x2*>(qr + c0) = u32x2{0u, 0u};
    return;
  }
  float s;
  if (ROWWISE) {
    float m = 0.f;
    for (int c = lane; c < cols; c += 64) m = fmaxf(m, fabsf(ldf(xr + c)));
    m = wave_max(m);
    s = m > 0.f ? m / 448.f : 1.f;
    if (lane == 0) scales[row] = s;
  } else {
    s = scale_in[0];
  }
  const float rs = 1.f / s;
  // four codes per lane and step, written as one 32-bit word (zeros past cols)
  for (int c0 = lane * 4; c0 < ldq; c0 += 256) {
    float t[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) t[e] = c0 + e < cols ? ldf(xr + c0 + e) * rs : 0.f;
    *reinterpret_cast<uint32_t*>(qr + c0) = e4m3x4(t[0], t[1], t[2], t[3]);
  }
}

// Tensor-wise amax: per-block maxima, then one block takes their maximum
// (max is exact in any order, so the result does not depend on the split).
template <typename IT>
__global__ __launch_bounds__(256) void fp8_amax_partial_kernel(const IT* __restrict__ x, int64_t ld,
                                                               int rows, int cols,
                                                               float* __restrict__ part) {
  float m = 0.f;
  const int64_t n = (int64_t)rows * cols;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / cols, c = i - r * cols;
    m = fmaxf(m, fabsf(ldf(x + r * ld + c)));
  }
  m = wave_max(m);
  __shared__ float wm[4];
  if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = fmaxf(fmaxf(wm[0], wm[1]), fmaxf(wm[2], wm[3]));
}

__global__ __launch_bounds__(256) void fp8_amax_final_kernel(const float* __restrict__ part, int n,
                                                             float* __restrict__ scale) {
  float m = 0.f;
  for (int i = threadIdx.x; i < n; i += 256) m = fmaxf(m, part[i]);
  m = wave_max(m);
  __shared__ float wm[4];
  if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    m = fmaxf(fmaxf(wm[0], wm[1]), fmaxf(wm[2], wm[3]));
    scale[0] = m > 0.f ? m / 448.f : 1.f;
  }
}

constexpr int FP8_AMAX_BLOCKS = 1024;

size_t fp8_quantize_workspace() { return (size_t)FP8_AMAX_BLOCKS * sizeof(float); }

template <bool ROWWISE>
static void fp8_quant_launch(DType xdt, const Fp8Jobs& J, int blocks, const float* scale_in, hipStream_t s) {
  if (xdt == DT_BF16)
    fp8_quant_kernel<bf16_t, ROWWISE><<<blocks, 256, 0, s>>>(J, scale_in);
  else
    fp8_quant_kernel<float, ROWWISE><<<blocks, 256, 0, s>>>(J, scale_in);
}

hipError_t fp8_quantize_rows(DType xdt, const Fp8RowJob* jobs, int njobs, hipStream_t s) {
  if (njobs < 1 || njobs > FP8_MAX_JOBS) {
    set_error("fp8_quantize_rows: 1 .. %d matrices per launch", FP8_MAX_JOBS);
    return hipErrorInvalidValue;
  }
  Fp8Jobs J{};
  int blocks = 0;
  for (int k = 0; k < njobs; ++k) {
    J.j[J.n] = jobs[k];
    J.blk0[J.n] = blocks;
    if (jobs[k].rows <= 0) continue;
    blocks += cdiv(jobs[k].rows, 4);
    ++J.n;
  }
  if (blocks == 0) return hipSuccess;
  fp8_quant_launch<true>(xdt, J, blocks, nullptr, s);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t fp8_quantize(const void* x, DType xdt, int rows, int cols, int64_t ld, int rowwise,
                        uint8_t* q, int64_t ldq, float* scales, void* ws, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const Fp8RowJob job{x, ld, rows, cols, q, ldq, scales};
  if (rowwise) return fp8_quantize_rows(xdt, &job, 1, s);
  float* part = static_cast<float*>(ws);
  const int64_t n = (int64_t)rows * cols;
  int pg = cdiv(n, 256);
  pg = pg < 1 ? 1 : (pg > FP8_AMAX_BLOCKS ? FP8_AMAX_BLOCKS : pg);
  if (xdt == DT_BF16)
    fp8_amax_partial_kernel<bf16_t><<<pg, 256, 0, s>>>((const bf16_t*)x, ld, rows, cols, part);
  else
    fp8_amax_partial_kernel<float><<<pg, 256, 0, s>>>((const float*)x, ld, rows, cols, part);
  LAT_LAUNCH_CHECK();
  fp8_amax_final_kernel<<<1, 256, 0, s>>>(part, pg, scales);
  LAT_LAUNCH_CHECK();
  Fp8Jobs J{};
  J.j[0] = Fp8RowJob{x, ld, rows, cols, q, ldq, nullptr};
  J.n = 1;
  fp8_quant_launch<false>(xdt, J, cdiv(rows, 4), scales, s);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// FP8 GEMM, C = act(A B^T * sa sw + b): A [M, K] and B [N, K] e4m3 codes with
// row strides lda / ldb bytes (multiples of 16).
// ---------------------------------------------------------------------------
constexpr int F8M = 128, F8N = 128, F8K = 128, F8PAD = 16, F8LD = F8K + F8PAD;  // bytes
constexpr int F8CLD = F8N + 4;
constexpr size_t FP8_GEMM_LDS = (size_t)2 * (F8M + F8N) * F8LD;  // 73,728 B
static_assert((size_t)F8M * F8CLD * sizeof(float) <= FP8_GEMM_LDS, "C staging fits the operand stages");

// 128 rows x 128 bytes of one operand: 1024 16-byte vectors, 4 per thread.
// Straight-line loads: a vector outside the matrix reads the first one
// instead and is zeroed at the LDS store; a vector reaching past K has its
// tail bytes zeroed.
struct F8Tile {
  u32x4 r[4];
  int R_, K_, r0_, k0_;
  bool edge_;
  __device__ inline void load(const uint8_t* p, int64_t ld, int R, int K, int r0, int k0, bool edge) {
    R_ = R; K_ = K; r0_ = r0; k0_ = k0; edge_ = edge;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = threadIdx.x + i * 256;
      const int rr = v >> 3, kc = (v & 7) * 16;
      const int gr = r0 + rr, gk = k0 + kc;
      const bool ok = !edge || (gr < R && gk < K);
      r[i] = *reinterpret_cast<const u32x4*>(p + (ok ? (int64_t)gr * ld + gk : 0));
    }
  }
  __device__ inline void store(uint8_t* S) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = threadIdx.x + i * 256;
      const int rr = v >> 3, kc = (v & 7) * 16;
      u32x4 x = r[i];
      if (edge_) {
        const int gr = r0_ + rr, gk = k0_ + kc;
        if (!(gr < R_ && gk < K_)) {
          x = u32x4{0, 0, 0, 0};
        } else if (gk + 16 > K_) {
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (gk + e >= K_) x[e >> 2] &= ~(0xffu << (8 * (e & 3)));
        }
      }
      *reinterpret_cast<u32x4*>(S + rr * F8LD + kc) = x;
    }
  }
};

// 128 k of fp8 MFMAs on the staged tiles: each wave 2 x 2 fragments of 32 x 32;
// a lane supplies row (lane % 32) and 32 consecutive k of each half (lane / 32).
template <bool PRECISE>
__device__ inline void mma_fp8_k128(const uint8_t* As, const uint8_t* Bs, int wm, int wn, int lane,
                                    f32x16 (&acc)[2][2]) {
  const int frow = lane & 31, fk = (lane >> 5) * 32;
  const uint8_t* as = As + (wm * 64 + frow) * F8LD + fk;
  const uint8_t* bs = Bs + (wn * 64 + frow) * F8LD + fk;
  auto opnd = [&](const uint8_t* p) {
    const u32x4 lo = *reinterpret_cast<const u32x4*>(p);
    const u32x4 hi = *reinterpret_cast<const u32x4*>(p + 16);
    return i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  };
  const f32x16 zero = {};
  if constexpr (PRECISE) {
    // all four fragments' two chained halves from zero first, then their
    // fp32 adds: the adds of one fragment overlap the MFMAs of the others
    f32x16 c[2][2];
    i32x8 a1[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const i32x8 a0 = opnd(as + i * 32 * F8LD);
      a1[i] = opnd(as + i * 32 * F8LD + 64);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        c[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a0, opnd(bs + j * 32 * F8LD), zero,
                                                                 0, 0, 0, 127, 0, 127);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const i32x8 b1 = opnd(bs + j * 32 * F8LD + 64);
#pragma unroll
      for (int i = 0; i < 2; ++i)
        c[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a1[i], b1, c[i][j], 0, 0, 0, 127, 0, 127);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] += c[i][j][r];
    return;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    // one 32-row fragment of A against both of B: the k = 0..63 and 64..127
    // halves chained through the accumulator
    const i32x8 a0 = opnd(as + i * 32 * F8LD), a1 = opnd(as + i * 32 * F8LD + 64);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const i32x8 b0 = opnd(bs + j * 32 * F8LD), b1 = opnd(bs + j * 32 * F8LD + 64);
      // formats 0 / 0: e4m3 operands; E8M0 block scales 127 = 2^0
      f32x16 c = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a0, b0, acc[i][j], 0, 0, 0, 127, 0, 127);
      acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a1, b1, c, 0, 0, 0, 127, 0, 127);
    }
  }
}

template <typename CT, bool RELU, bool PRECISE>
__global__ __launch_bounds__(256, 2) void gemm_fp8_kernel(
    const uint8_t* __restrict__ A, int64_t lda, const float* __restrict__ sa, int sa_rowwise,
    const uint8_t* __restrict__ Bm, int64_t ldb, const float* __restrict__ sb, int sb_rowwise,
    const float* __restrict__ bias, CT* __restrict__ C, int64_t ldc, int M, int N, int K) {
  extern __shared__ __attribute__((aligned(16))) unsigned char f8_smem[];
  uint8_t* As[2];
  uint8_t* Bs[2];
  As[0] = f8_smem;
  Bs[0] = As[0] + F8M * F8LD;
  As[1] = Bs[0] + F8N * F8LD;
  Bs[1] = As[1] + F8M * F8LD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int tiles_n = (N + F8N - 1) / F8N;
  const int tile = xcd_block(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * F8M, n0 = (tile % tiles_n) * F8N;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int ktiles = (K + F8K - 1) / F8K;
  const bool edge_m = m0 + F8M > M, edge_n = n0 + F8N > N;
  auto load = [&](F8Tile& la, F8Tile& lb, int kt) {
    const int k0 = kt * F8K;
    const bool edge_k = k0 + F8K > K;
    la.load(A, lda, M, K, m0, k0, edge_m || edge_k);
    lb.load(Bm, ldb, N, K, n0, k0, edge_n || edge_k);
  };
  if constexpr (PRECISE) {
    // One register stage (the per-block partial sums take the registers of
    // the second): the next K step's tiles are loaded while the MFMAs consume
    // the current LDS stage, then written to the other LDS stage.
    F8Tile la, lb;
    if (ktiles > 0) {
      load(la, lb, 0);
      la.store(As[0]);
      lb.store(Bs[0]);
    }
    __syncthreads();
    for (int kt = 0; kt < ktiles; ++kt) {
      const int cur = kt & 1;
      if (kt + 1 < ktiles) load(la, lb, kt + 1);
      mma_fp8_k128<true>(As[cur], Bs[cur], wm, wn, lane, acc);
      if (kt + 1 < ktiles) {
        la.store(As[cur ^ 1]);
        lb.store(Bs[cur ^ 1]);
      }
      __syncthreads();
    }
  } else {
    // Two register stages and two LDS stages: while the MFMAs consume LDS
    // stage s, the registers of the other stage receive the tile two K steps
    // ahead (as in the bf16 kernel).
    F8Tile la0, la1, lb0, lb1;
    if (ktiles > 0) load(la0, lb0, 0);
    if (ktiles > 1) load(la1, lb1, 1);
    if (ktiles > 0) {
      la0.store(As[0]);
      lb0.store(Bs[0]);
    }
    __syncthreads();
    int kt = 0;
    for (; kt + 2 <= ktiles; kt += 2) {
      if (kt + 2 < ktiles) load(la0, lb0, kt + 2);
      mma_fp8_k128<false>(As[0], Bs[0], wm, wn, lane, acc);
      la1.store(As[1]);
      lb1.store(Bs[1]);
      __syncthreads();
      if (kt + 3 < ktiles) load(la1, lb1, kt + 3);
      mma_fp8_k128<false>(As[1], Bs[1], wm, wn, lane, acc);
      if (kt + 2 < ktiles) {
        la0.store(As[0]);
        lb0.store(Bs[0]);
      }
      __syncthreads();
    }
    if (kt < ktiles) {
      mma_fp8_k128<false>(As[0], Bs[0], wm, wn, lane, acc);
      __syncthreads();
    }
  }
  // stage the fp32 tile, then rows of 8 columns: dequantise, bias, ReLU, store
  float* Cs = reinterpret_cast<float*>(f8_smem);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int cl = wn * 64 + j * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        Cs[rl * F8CLD + cl] = acc[i][j][r];
      }
    }
  __syncthreads();
  const float sb0 = sb[0];
#pragma unroll
  for (int q = 0; q < (F8M * F8N / 8) / 256; ++q) {
    const int chunk = threadIdx.x + q * 256;
    const int rl = chunk / (F8N / 8), cl = (chunk % (F8N / 8)) * 8;
    const int row = m0 + rl, col = n0 + cl;
    if (row >= M || col >= N) continue;
    const float ra = sa_rowwise ? sa[row] : sa[0];
    float v[8], cs[8], bs[8];
    if (col + 8 <= N && (N & 3) == 0) {     // 16-byte loads of the column scales and bias
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4 x4 = sb_rowwise ? *reinterpret_cast<const f32x4*>(sb + col + 4 * h) : f32x4{sb0, sb0, sb0, sb0};
        const f32x4 b4 = bias ? *reinterpret_cast<const f32x4*>(bias + col + 4 * h) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) { cs[4 * h + e] = x4[e]; bs[4 * h + e] = b4[e]; }
      }
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int c = col + t < N ? col + t : N - 1;
        cs[t] = sb_rowwise ? sb[c] : sb0;
        bs[t] = bias ? bias[c] : 0.f;
      }
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      float y = Cs[rl * F8CLD + cl + t] * ra;
      y *= cs[t];
      y += bs[t];
      if (RELU) y = y > 0.f ? y : 0.f;
      v[t] = y;
    }
    CT* c = C + (int64_t)row * ldc + col;
    if (col + 8 <= N && ((ldc * (int64_t)sizeof(CT)) & 15) == 0 && ((uintptr_t)C & 15) == 0) {
      if constexpr (sizeof(CT) == 2) {
        stg16(c, Vec16<bf16_t>::pack(v));
      } else {
        stg16(c, Vec16<float>::pack(v));
        stg16(c + 4, Vec16<float>::pack(v + 4));
      }
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (col + t < N) st(c + t, v[t]);
    }
  }
}

hipError_t gemm_fp8(const uint8_t* A, int64_t lda, const float* sa, int sa_rowwise, const uint8_t* B,
                    int64_t ldb, const float* sb, int sb_rowwise, const float* bias, void* C,
                    DType cdt, int64_t ldc, int M, int N, int K, int relu, int fast_accum,
                    hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  static std::once_flag once;
  std::call_once(once, [] {
    const int lds = (int)FP8_GEMM_LDS;
    const void* ks[] = {(const void*)gemm_fp8_kernel<bf16_t, true, true>, (const void*)gemm_fp8_kernel<bf16_t, false, true>,
                        (const void*)gemm_fp8_kernel<float, true, true>, (const void*)gemm_fp8_kernel<float, false, true>,
                        (const void*)gemm_fp8_kernel<bf16_t, true, false>, (const void*)gemm_fp8_kernel<bf16_t, false, false>,
                        (const void*)gemm_fp8_kernel<float, true, false>, (const void*)gemm_fp8_kernel<float, false, false>};
    for (const void* k : ks) (void)hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  });
  const int grid = cdiv(M, F8M) * cdiv(N, F8N);
#define LAT_F8(CTT, RL, PR)                                                                      \
  gemm_fp8_kernel<CTT, RL, PR><<<grid, 256, FP8_GEMM_LDS, s>>>(A, lda, sa, sa_rowwise, B, ldb, sb, \
                                                               sb_rowwise, bias, (CTT*)C, ldc, M, N, K)
#define LAT_F8P(CTT, RL) \
  do { if (fast_accum) LAT_F8(CTT, RL, false); else LAT_F8(CTT, RL, true); } while (0)
  if (cdt == DT_BF16) {
    if (relu) LAT_F8P(bf16_t, true); else LAT_F8P(bf16_t, false);
  } else {
    if (relu) LAT_F8P(float, true); else LAT_F8P(float, false);
  }
#undef LAT_F8P
#undef LAT_F8
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
