// The objective heads of the training step: the last (linear) layer of the
// top MLP fused with the masked multi-objective binary cross-entropy (an
// impression trains only the heads it is routed to, Section 3.2.1) and with
// that layer's input gradient, for bf16 models with at most 64 heads.
// The generic GEMM would give these skinny products (N or K = T = 4..64)
// 128-wide tiles of which a few columns are used, and the loss two more
// passes over the logits; here each product is a few MFMAs per 32 rows.
//
// head_fwd_kernel: z = h W^T + b (fp32).  One block per 32 rows; its eight
//   waves take interleaved 16-wide K steps of v_mfma_f32_32x32x16_bf16 (the
//   heads padded to 32 columns with zeros) and their partial tiles are added
//   in wave order through LDS.  Each block writes its partial sums of the
//   masked loss terms max(z,0) - z y + log1p(exp(-|z|)) and of the mask.
// head_bwd_kernel: N = max(1, sum m) and the loss (sum / N) from all blocks'
//   partials (every wave adds them in the same fixed order); dz = m (sigmoid(z) - y) / N in fp32 and
//   its bf16 operand copy; then the layer's input gradient
//   g = (dz_bf16 W) ⊙ [mask > 0] (mask: the layer's input, i.e. the previous
//   layer's ReLU output, or none) in bf16, one MFMA per 32 x 32 tile and 16
//   heads, the dz fragments built in registers in the operand layout; the
//   mask is read and the gradient written as 16-byte row segments through a
//   per-wave LDS patch (not as 2-byte columns of the MFMA layout).
#include "common.h"
#include "kernels.h"
#include "mfma_tile.h"

namespace lat {

constexpr int HEAD_ROWS = 32;
constexpr int HEAD_THREADS = 512;
constexpr int HEAD_WAVES = HEAD_THREADS / 64;
constexpr int HEAD_SPW = 4;  // forward: K steps per wave and chunk (K <= 512: one chunk)
// backward: 32-column tiles per wave and chunk (fewer with more heads, to
// keep the prefetched fragments in registers)
template <int TS> constexpr int head_kpw() { return TS <= 1 ? 2 : 1; }

// Each wave reads every fragment of its chunk before the first MFMA, and
// the loss operands before the chunk loop, so the few global round trips of
// a block overlap instead of following one another.
// NT: 32-column tiles of heads (T <= 32 NT)
template <int NT>
__global__ __launch_bounds__(HEAD_THREADS) void head_fwd_kernel(
    const bf16_t* __restrict__ h, int64_t ldh, int B, int K, const bf16_t* __restrict__ W,
    const float* __restrict__ bias, int T, const float* __restrict__ y,
    const uint8_t* __restrict__ m, float* __restrict__ z, float* __restrict__ part) {
  constexpr int EPT = NT * 1024 / HEAD_THREADS;  // output elements per thread
  __shared__ float red[HEAD_WAVES][NT][16][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r0 = blockIdx.x * HEAD_ROWS;
  const int row = r0 + (lane & 31);
  const int kofs = (lane >> 5) * 8;
  // this thread's outputs after the reduction: element e = threadIdx.x + j *
  // HEAD_THREADS of the tiles, in the MFMA output layout
  int oi[EPT];
  float yv[EPT], bv0[EPT];
  uint8_t mv[EPT];
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int e = threadIdx.x + j * HEAD_THREADS;
    const int tt = e >> 10, r = (e >> 6) & 15, ln = e & 63;
    const int rr = r0 + 8 * (r >> 2) + 4 * (ln >> 5) + (r & 3);
    const int t = tt * 32 + (ln & 31);
    const bool ok = rr < B && t < T;
    oi[j] = ok ? rr * T + t : -1;
    yv[j] = (ok && y) ? y[(int64_t)rr * T + t] : 0.f;  // no labels (forward alone): no loss terms
    mv[j] = (ok && m) ? m[(int64_t)rr * T + t] : 0;
    bv0[j] = (ok && bias) ? bias[t] : 0.f;
  }
  f32x16 acc[NT];
#pragma unroll
  for (int tt = 0; tt < NT; ++tt) zero16(acc[tt]);
  const bf16_t* hr = h + (int64_t)(row < B ? row : 0) * ldh;
  const int steps = (K + 15) / 16;
  for (int c0 = 0; c0 < steps; c0 += HEAD_WAVES * HEAD_SPW) {
    u32x4 av[HEAD_SPW], bw[HEAD_SPW][NT];
#pragma unroll
    for (int i = 0; i < HEAD_SPW; ++i) {
      const int k = (c0 + w + i * HEAD_WAVES) * 16 + kofs;  // K % 8 == 0: k < K means k + 8 <= K
      av[i] = (row < B && k < K) ? ldg16(hr + k) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const int t = tt * 32 + (lane & 31);
        bw[i][tt] = (t < T && k < K) ? ldg16(W + (int64_t)t * K + k) : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int i = 0; i < HEAD_SPW; ++i)
#pragma unroll
      for (int tt = 0; tt < NT; ++tt)
        acc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av[i]),
                                                          __builtin_bit_cast(bf16x8, bw[i][tt]),
                                                          acc[tt], 0, 0, 0);
  }
#pragma unroll
  for (int tt = 0; tt < NT; ++tt)
#pragma unroll
    for (int r = 0; r < 16; ++r) red[w][tt][r][lane] = acc[tt][r];
  __syncthreads();
  float ls = 0.f, cs = 0.f;
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const int e = threadIdx.x + j * HEAD_THREADS;
    const int tt = e >> 10, r = (e >> 6) & 15, ln = e & 63;
    float v = red[0][tt][r][ln];
#pragma unroll
    for (int q = 1; q < HEAD_WAVES; ++q) v += red[q][tt][r][ln];
    if (oi[j] >= 0) {
      v += bv0[j];
      z[oi[j]] = v;
      if (mv[j]) {
        ls += fmaxf(v, 0.f) - v * yv[j] + log1pf(expf(-fabsf(v)));
        cs += 1.f;
      }
    }
  }
  // block sums in a fixed order: butterfly within each wave, then the waves
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    ls += __shfl_xor(ls, o, 64);
    cs += __shfl_xor(cs, o, 64);
  }
  if (lane == 0) {
    red[w][0][0][0] = ls;
    red[w][0][0][1] = cs;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float a = 0.f, c = 0.f;
    for (int q = 0; q < HEAD_WAVES; ++q) {
      a += red[q][0][0][0];
      c += red[q][0][0][1];
    }
    part[blockIdx.x] = a;
    part[gridDim.x + blockIdx.x] = c;
  }
}

constexpr int HEAD_LQ = 32 + 8;  // patch row stride (bf16)

// LDS writes of this wave visible to its reads (the patch is wave-private)
__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// TS: 16-wide steps of heads (T <= 16 TS)
template <int TS>
__global__ __launch_bounds__(HEAD_THREADS) void head_bwd_kernel(
    const float* __restrict__ z, const float* __restrict__ y, const uint8_t* __restrict__ m,
    int B, int T, const float* __restrict__ part, const bf16_t* __restrict__ W, int K,
    const bf16_t* __restrict__ mask, int64_t ldm, float* __restrict__ loss,
    float* __restrict__ dz, bf16_t* __restrict__ dz_op, bf16_t* __restrict__ g, int64_t ldg) {
  const int parts = gridDim.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r0 = blockIdx.x * HEAD_ROWS;
  const int row = r0 + (lane & 31);
  const int tofs = (lane >> 5) * 8;
  __shared__ __attribute__((aligned(16))) bf16_t patch[HEAD_WAVES][32 * HEAD_LQ];
  bf16_t* pq = patch[w];  // this wave's 32 x 32 transposition patch
  // loss operands of this lane's dz fragment (row, heads ts*16 + tofs + j)
  float zv[TS][8], yv[TS][8];
  uint8_t mv[TS][8];
#pragma unroll
  for (int ts = 0; ts < TS; ++ts)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int t = ts * 16 + tofs + j;
      const bool ok = row < B && t < T;
      const int64_t i = (int64_t)row * T + t;
      zv[ts][j] = ok ? z[i] : 0.f;
      yv[ts][j] = ok ? y[i] : 0.f;
      mv[ts][j] = ok ? m[i] : 0;
    }
  // this wave's first chunk of W^T fragments and mask values, in flight
  // while the loss is reduced and dz computed
  constexpr int HEAD_KPW = head_kpw<TS>();
  const int ktiles = (K + 31) / 32;
  uint32_t bw[HEAD_KPW][TS][4];
  // mask rows of each tile as 16-byte segments: lane l holds row
  // half * 16 + l / 4, columns 8 (l % 4) .. + 7 (no mask: all positive)
  u32x4 mk[HEAD_KPW][2];
  auto load_chunk = [&](int c0) {
#pragma unroll
    for (int i = 0; i < HEAD_KPW; ++i) {
      const int kb = (c0 + w + i * HEAD_WAVES) * 32;
      const int k = kb + (lane & 31);
#pragma unroll
      for (int ts = 0; ts < TS; ++ts)
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
          const int t0 = ts * 16 + tofs + j;
          const uint32_t b0 = (k < K && t0 < T) ? W[(int64_t)t0 * K + k] : 0u;
          const uint32_t b1 = (k < K && t0 + 1 < T) ? W[(int64_t)(t0 + 1) * K + k] : 0u;
          bw[i][ts][j / 2] = b0 | (b1 << 16);
        }
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int rr = r0 + half * 16 + (lane >> 2), c8 = kb + (lane & 3) * 8;
        const bool ok = mask && rr < B && c8 < K;
        // (an address inside the mask whatever ok is; the value is used only if ok)
        const u32x4 v = mask ? ldg16(mask + (ok ? (int64_t)rr * ldm + c8 : 0)) : u32x4{0u, 0u, 0u, 0u};
        mk[i][half] = ok ? v : u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};
      }
    }
  };
  load_chunk(0);
  // N = max(1, sum m) and the loss sum from the partials, by every wave in
  // the same fixed order (lane-strided sums, then a butterfly)
  float c = 0.f, l = 0.f;
  for (int i = lane; i < parts; i += 64) {
    l += part[i];
    c += part[parts + i];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    l += __shfl_xor(l, o, 64);
    c += __shfl_xor(c, o, 64);
  }
  const float N = fmaxf(1.f, c);
  if (blockIdx.x == 0 && threadIdx.x == 0) loss[0] = l / N;
  // dz fragment (the A operand of the input-gradient MFMA); wave 0 writes
  // it out (each element once)
  bf16x8 a[TS];
#pragma unroll
  for (int ts = 0; ts < TS; ++ts) {
    float gv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float gg = 0.f;
      if (mv[ts][j]) {
        const float zz = zv[ts][j];
        const float e = expf(-fabsf(zz));
        const float sg = zz >= 0.f ? 1.f / (1.f + e) : e / (1.f + e);
        gg = (sg - yv[ts][j]) / N;
      }
      gv[j] = gg;
      const int t = ts * 16 + tofs + j;
      if (w == 0 && row < B && t < T) {
        const int64_t i = (int64_t)row * T + t;
        dz[i] = gg;
        dz_op[i] = f2bf(gg);
      }
    }
    a[ts] = __builtin_bit_cast(bf16x8, (u32x4{pack_bf2(gv[0], gv[1]), pack_bf2(gv[2], gv[3]),
                                               pack_bf2(gv[4], gv[5]), pack_bf2(gv[6], gv[7])}));
  }
  // g[row][k] = sum_t dz[row][t] W[t][k], tiles of 32 rows x 32 columns
  for (int c0 = 0; c0 < ktiles; c0 += HEAD_WAVES * HEAD_KPW) {
    f32x16 acc[HEAD_KPW];
#pragma unroll
    for (int i = 0; i < HEAD_KPW; ++i) {
      zero16(acc[i]);
#pragma unroll
      for (int ts = 0; ts < TS; ++ts)
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            a[ts],
            __builtin_bit_cast(bf16x8, (u32x4{bw[i][ts][0], bw[i][ts][1], bw[i][ts][2], bw[i][ts][3]})),
            acc[i], 0, 0, 0);
    }
    u32x4 mc[HEAD_KPW][2];
#pragma unroll
    for (int i = 0; i < HEAD_KPW; ++i) {
      mc[i][0] = mk[i][0];
      mc[i][1] = mk[i][1];
    }
    if (c0 + HEAD_WAVES * HEAD_KPW < ktiles) load_chunk(c0 + HEAD_WAVES * HEAD_KPW);
#pragma unroll
    for (int i = 0; i < HEAD_KPW; ++i) {
      const int kb = (c0 + w + i * HEAD_WAVES) * 32;
      if (kb >= K) continue;  // wave-uniform
      // mask rows into the patch, read back in the tile's layout; the masked
      // gradient written there and read out as 16-byte row segments
#pragma unroll
      for (int half = 0; half < 2; ++half)
        *reinterpret_cast<u32x4*>(pq + (half * 16 + (lane >> 2)) * HEAD_LQ + (lane & 3) * 8) = mc[i][half];
      wave_sync();
      bf16_t gv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int jl = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        gv[r] = f2bf(bf2f(pq[jl * HEAD_LQ + (lane & 31)]) > 0.f ? acc[i][r] : 0.f);
      }
      wave_sync();
#pragma unroll
      for (int r = 0; r < 16; ++r) pq[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * HEAD_LQ + (lane & 31)] = gv[r];
      wave_sync();
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int rl = half * 16 + (lane >> 2), c8 = (lane & 3) * 8;
        const u32x4 v = *reinterpret_cast<const u32x4*>(pq + rl * HEAD_LQ + c8);
        if (r0 + rl < B && kb + c8 < K) stg16(g + (int64_t)(r0 + rl) * ldg + kb + c8, v);
      }
      wave_sync();
    }
  }
}

static bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

bool head_fusable(int T, int K, const void* h, int64_t ldh, const void* W) {
  return T >= 1 && T <= HEAD_MAX_T && K >= 8 && K % 8 == 0 && ldh % 8 == 0 && al16(h) && al16(W);
}

size_t head_workspace(int B) { return (size_t)2 * cdiv(B > 0 ? B : 1, HEAD_ROWS) * sizeof(float); }

hipError_t head_fwd(const bf16_t* h, int64_t ldh, int B, int K, const bf16_t* W,
                    const float* bias, int T, const float* y, const uint8_t* m, float* z,
                    void* ws, hipStream_t s) {
  const int blocks = cdiv(B > 0 ? B : 1, HEAD_ROWS);
  float* part = (float*)ws;
  if (T <= 32)
    head_fwd_kernel<1><<<blocks, HEAD_THREADS, 0, s>>>(h, ldh, B, K, W, bias, T, y, m, z, part);
  else
    head_fwd_kernel<2><<<blocks, HEAD_THREADS, 0, s>>>(h, ldh, B, K, W, bias, T, y, m, z, part);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t head_bwd(const float* z, const float* y, const uint8_t* m, int B, int T,
                    const bf16_t* W, int K, const bf16_t* mask, int64_t ldm, float* loss,
                    float* dz, bf16_t* dz_op, bf16_t* g, int64_t ldg, const void* ws,
                    hipStream_t s) {
  const int blocks = cdiv(B > 0 ? B : 1, HEAD_ROWS);
  const float* part = (const float*)ws;
#define LAT_HEAD_BWD(TSV)                                                                    \
  head_bwd_kernel<TSV><<<blocks, HEAD_THREADS, 0, s>>>(z, y, m, B, T, part, W, K, mask, ldm, \
                                                       loss, dz, dz_op, g, ldg)
  if (T <= 16) LAT_HEAD_BWD(1);
  else if (T <= 32) LAT_HEAD_BWD(2);
  else if (T <= 48) LAT_HEAD_BWD(3);
  else LAT_HEAD_BWD(4);
#undef LAT_HEAD_BWD
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
