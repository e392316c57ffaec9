// Masked multi-objective binary cross-entropy on the logits (impressions
// train only the heads they are routed to, Section 3.2.1):
//   N = max(1, sum m),  loss = sum m*(max(z,0) - z*y + log1p(exp(-|z|))) / N,
//   dz = m*(sigmoid(z) - y) / N.
// Two passes with fixed-order block reductions (deterministic): per-block
// partial loss sums and mask counts, then every block reads all partials,
// writes its dz slice (fp32 and the storage-dtype operand copy) and block 0
// writes the loss.
#include "common.h"
#include "kernels.h"

namespace lat {

constexpr int BCE_THREADS = 256;
// two logits per thread: the passes are latency-bound (one exp/log1p chain
// per element), so many small blocks beat few long ones
constexpr int BCE_TILE = 512;

__device__ inline float block_sum_f(float v, float* lds) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  if (lane == 0) lds[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < BCE_THREADS / 64; ++i) s += lds[i];
  __syncthreads();
  return s;
}

__global__ __launch_bounds__(BCE_THREADS) void bce_partial_kernel(
    const float* __restrict__ z, const float* __restrict__ y, const uint8_t* __restrict__ m,
    int64_t n, float* __restrict__ part_loss, float* __restrict__ part_cnt) {
  __shared__ float lds[BCE_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * BCE_TILE;
  float ls = 0.f, cs = 0.f;
  for (int i = threadIdx.x; i < BCE_TILE; i += BCE_THREADS) {
    const int64_t k = base + i;
    if (k < n && m[k]) {
      const float zz = z[k];
      ls += fmaxf(zz, 0.f) - zz * y[k] + log1pf(expf(-fabsf(zz)));
      cs += 1.f;
    }
  }
  ls = block_sum_f(ls, lds);
  cs = block_sum_f(cs, lds);
  if (threadIdx.x == 0) {
    part_loss[blockIdx.x] = ls;
    part_cnt[blockIdx.x] = cs;
  }
}

template <typename OT>
__global__ __launch_bounds__(BCE_THREADS) void bce_final_kernel(
    const float* __restrict__ z, const float* __restrict__ y, const uint8_t* __restrict__ m,
    int64_t n, const float* __restrict__ part_loss, const float* __restrict__ part_cnt, int parts,
    float* __restrict__ loss, float* __restrict__ dz, OT* __restrict__ dz_op) {
  __shared__ float lds[BCE_THREADS / 64];
  float c = 0.f, l = 0.f;
  for (int i = threadIdx.x; i < parts; i += BCE_THREADS) {
    c += part_cnt[i];
    l += part_loss[i];
  }
  c = block_sum_f(c, lds);
  l = block_sum_f(l, lds);
  const float N = fmaxf(1.f, c);
  if (blockIdx.x == 0 && threadIdx.x == 0) loss[0] = l / N;
  const int64_t base = (int64_t)blockIdx.x * BCE_TILE;
  for (int i = threadIdx.x; i < BCE_TILE; i += BCE_THREADS) {
    const int64_t k = base + i;
    if (k < n) {
      float g = 0.f;
      if (m[k]) {
        const float zz = z[k];
        const float e = expf(-fabsf(zz));
        const float sg = zz >= 0.f ? 1.f / (1.f + e) : e / (1.f + e);
        g = (sg - y[k]) / N;
      }
      dz[k] = g;
      if (dz_op) st(dz_op + k, g);
    }
  }
}

size_t bce_workspace(int64_t n) { return (size_t)2 * (cdiv(n > 0 ? n : 1, BCE_TILE)) * sizeof(float); }

hipError_t bce(const float* z, const float* y, const uint8_t* m, int64_t n, float* loss, float* dz,
               void* dz_op, DType op_dt, void* ws, hipStream_t s) {
  const int parts = cdiv(n > 0 ? n : 1, BCE_TILE);
  float* pl = (float*)ws;
  float* pc = pl + parts;
  bce_partial_kernel<<<parts, BCE_THREADS, 0, s>>>(z, y, m, n, pl, pc);
  LAT_LAUNCH_CHECK();
  if (op_dt == DT_BF16)
    bce_final_kernel<bf16_t><<<parts, BCE_THREADS, 0, s>>>(z, y, m, n, pl, pc, parts, loss, dz, (bf16_t*)dz_op);
  else
    bce_final_kernel<float><<<parts, BCE_THREADS, 0, s>>>(z, y, m, n, pl, pc, parts, loss, dz, (float*)dz_op);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
