// SwishRN activation of a feed-forward layer (Section 3.3.4) over a stored
// pre-activation h [M, N]:
//   rho = 1 / sqrt(mean over the group of h^2 + eps),  n = h rho,
//   out = (g_a n) * gate(g_b n)
// with the groups either the whole row (RMSNorm) or consecutive 128-column
// groups (BlockNorm, Section 3.5.3: the statistic of one GEMM tile, which
// the bf16 GEMM computes in its epilogue instead; these row kernels are the
// unfused path: fp32 models and whole-row norms).  gain = [g_a; g_b], two
// rows of N fp32.
//
// Backward, from the stored h (pre), rho (rinv) and the output gradient go:
//   dn = go (g_a s + g_b a gate'(z)),  dh = rho (dn - n mean_G(dn n)),
//   d g_a = sum over rows of go s n,  d g_b = sum over rows of go a gate'(z) n.
//
// Row kernels: one wave per row, 8 consecutive columns per lane (16-byte
// vectors when rows are aligned), so a 128-column group is one aligned
// 16-lane group and its sums are shuffles within it.  The gain gradients
// are column sums: 64-column x 256-row blocks summed in a fixed order, then
// the row blocks in order (deterministic).
#include <initializer_list>
#include <utility>

#include "common.h"
#include "kernels.h"
#include "swishrn.h"

namespace lat {

template <typename T>
__device__ __forceinline__ void load8(const T* p, int c, int N, int vec, float* v) {
  if (vec && c + 8 <= N) {
    if constexpr (sizeof(T) == 2) {
      Vec16<bf16_t>::unpack(ldg16(p + c), v);
    } else {
      Vec16<float>::unpack(ldg16(p + c), v);
      Vec16<float>::unpack(ldg16(p + c + 4), v + 4);
    }
  } else {
#pragma unroll
    for (int t = 0; t < 8; ++t) v[t] = c + t < N ? ld(p + c + t) : 0.f;
  }
}

template <typename T>
__device__ __forceinline__ void store8(T* p, int c, int N, int vec, const float* v) {
  if (vec && c + 8 <= N) {
    if constexpr (sizeof(T) == 2) {
      stg16(p + c, Vec16<bf16_t>::pack(v));
    } else {
      stg16(p + c, Vec16<float>::pack(v));
      stg16(p + c + 4, Vec16<float>::pack(v + 4));
    }
  } else {
#pragma unroll
    for (int t = 0; t < 8; ++t)
      if (c + t < N) st(p + c + t, v[t]);
  }
}

// out of 8 columns from h (zero past N), rho and the columns' gains
template <int GATE>
__device__ __forceinline__ void swish8(const float* h, float r, const float* ga, const float* gb,
                                       float* o) {
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const float n = h[t] * r;
    o[t] = (ga[t] * n) * gate_fn<GATE>(gb[t] * n);
  }
}

// dn and n of 8 columns (g and h zero past N, so are n and dn there)
template <int GATE>
__device__ __forceinline__ void dn8(const float* g, const float* h, float r, const float* ga,
                                    const float* gb, float* n, float* dn) {
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    n[t] = h[t] * r;
    const float a = ga[t] * n[t], z = gb[t] * n[t];
    const float s = gate_fn<GATE>(z);
    dn[t] = g[t] * (ga[t] * s + gb[t] * a * gate_deriv<GATE>(z, s));
  }
}

template <typename T, int GATE, bool FULL>
__global__ __launch_bounds__(256) void swishrn_fwd_rows_kernel(const T* __restrict__ pre, int64_t ldp,
                                                               int M, int N,
                                                               const float* __restrict__ gain,
                                                               float eps, T* __restrict__ out,
                                                               int64_t ldo, float* __restrict__ rinv,
                                                               int nblk, int vec) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;  // whole wave
  const T* p = pre + (int64_t)row * ldp;
  T* o = out + (int64_t)row * ldo;
  if constexpr (FULL) {
    float ss = 0.f;
    for (int c = lane * 8; c < N; c += 512) {
      float v[8];
      load8(p, c, N, vec, v);
#pragma unroll
      for (int t = 0; t < 8; ++t) ss += v[t] * v[t];
    }
    ss = sum64(ss);
    const float r = rsqrtf(ss * __builtin_amdgcn_rcpf((float)N) + eps);
    if (lane == 0) rinv[(int64_t)row * nblk] = r;
    for (int c = lane * 8; c < N; c += 512) {
      float v[8], y[8], ga[8], gb[8];
      load8(p, c, N, vec, v);
      load_gains8(gain, N, c, ga, gb);
      swish8<GATE>(v, r, ga, gb, y);
      store8(o, c, N, vec, y);
    }
  } else {
    for (int c0 = 0; c0 < N; c0 += 512) {
      const int c = c0 + lane * 8;
      float v[8], y[8], ga[8], gb[8];
      load8(p, c, N, vec, v);
      load_gains8(gain, N, c, ga, gb);
      float ss = 0.f;
#pragma unroll
      for (int t = 0; t < 8; ++t) ss += v[t] * v[t];
      ss = sum16(ss);
      const float r = rsqrtf(ss * inv_group_size(c, N) + eps);
      if (c < N) {
        if ((lane & 15) == 0) rinv[(int64_t)row * nblk + c / NORM_TILE] = r;
        swish8<GATE>(v, r, ga, gb, y);
        store8(o, c, N, vec, y);
      }
    }
  }
}

template <typename T, int GATE, bool FULL>
__global__ __launch_bounds__(256) void swishrn_bwd_rows_kernel(
    const T* __restrict__ go, int64_t ldg, const T* __restrict__ pre, int64_t ldp,
    const float* __restrict__ rinv, int nblk, int M, int N, const float* __restrict__ gain,
    T* __restrict__ dh, int64_t ldd, int vec) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;  // whole wave
  const T* g = go + (int64_t)row * ldg;
  const T* p = pre + (int64_t)row * ldp;
  T* d = dh + (int64_t)row * ldd;
  if constexpr (FULL) {
    const float r = rinv[(int64_t)row * nblk];
    float acc = 0.f;
    for (int c = lane * 8; c < N; c += 512) {
      float gv[8], hv[8], n[8], dn[8], ga[8], gb[8];
      load8(g, c, N, vec, gv);
      load8(p, c, N, vec, hv);
      load_gains8(gain, N, c, ga, gb);
      dn8<GATE>(gv, hv, r, ga, gb, n, dn);
#pragma unroll
      for (int t = 0; t < 8; ++t) acc += dn[t] * n[t];
    }
    const float m = sum64(acc) * __builtin_amdgcn_rcpf((float)N);
    for (int c = lane * 8; c < N; c += 512) {
      float gv[8], hv[8], n[8], dn[8], y[8], ga[8], gb[8];
      load8(g, c, N, vec, gv);
      load8(p, c, N, vec, hv);
      load_gains8(gain, N, c, ga, gb);
      dn8<GATE>(gv, hv, r, ga, gb, n, dn);
#pragma unroll
      for (int t = 0; t < 8; ++t) y[t] = r * (dn[t] - n[t] * m);
      store8(d, c, N, vec, y);
    }
  } else {
    for (int c0 = 0; c0 < N; c0 += 512) {
      const int c = c0 + lane * 8;
      const int blk = c / NORM_TILE;
      const float r = c < N ? rinv[(int64_t)row * nblk + blk] : 0.f;
      float gv[8], hv[8], n[8], dn[8], y[8], ga[8], gb[8];
      load8(g, c, N, vec, gv);
      load8(p, c, N, vec, hv);
      load_gains8(gain, N, c, ga, gb);
      dn8<GATE>(gv, hv, r, ga, gb, n, dn);
      float acc = 0.f;
#pragma unroll
      for (int t = 0; t < 8; ++t) acc += dn[t] * n[t];
      const float m = sum16(acc) * inv_group_size(c, N);
      if (c < N) {
#pragma unroll
        for (int t = 0; t < 8; ++t) y[t] = r * (dn[t] - n[t] * m);
        store8(d, c, N, vec, y);
      }
    }
  }
}

// Gain gradients, first pass: block (x, y) sums rows y*256 .. of columns
// x*64 .. x*64+63 (8 groups of 8 columns, 32 row lanes) in a fixed order;
// part[y][k] receives d g_a[k], part[y][N + k] d g_b[k].
constexpr int GG_ROWS = 256;
template <typename T, int GATE>
__global__ __launch_bounds__(256) void swishrn_gain_partial_kernel(
    const T* __restrict__ go, int64_t ldg, const T* __restrict__ pre, int64_t ldp,
    const float* __restrict__ rinv, int nblk, int block, int M, int N,
    const float* __restrict__ gain, int vec, float* __restrict__ part) {
  __shared__ float red[2][32][65];
  const int cg = threadIdx.x & 7, rl = threadIdx.x >> 3;
  const int col0 = blockIdx.x * 64 + cg * 8;
  const int r0 = blockIdx.y * GG_ROWS, r1 = min(M, r0 + GG_ROWS);
  const int blk = block ? col0 / block : 0;
  float sa[8], sb[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) sa[t] = sb[t] = 0.f;
  if (col0 < N) {
    float ga[8], gb[8];
    load_gains8(gain, N, col0, ga, gb);
    // straight line over the thread's GG_ROWS / 32 rows (all loads in
    // flight together); rows past M read row r0 and count as zero
#pragma unroll
    for (int i = 0; i < GG_ROWS / 32; ++i) {
      const int row = r0 + rl + 32 * i;
      const bool ok = row < r1;
      const int rr = ok ? row : r0;
      float gv[8], hv[8];
      load8(go + (int64_t)rr * ldg, col0, N, vec, gv);
      load8(pre + (int64_t)rr * ldp, col0, N, vec, hv);
      const float r = ok ? rinv[(int64_t)rr * nblk + blk] : 0.f;
#pragma unroll
      for (int t = 0; t < 8; ++t) {   // zero past N (gv, hv and the gains are) and past M
        gv[t] = ok ? gv[t] : 0.f;
        const float n = hv[t] * r;
        const float a = ga[t] * n, z = gb[t] * n;
        const float s = gate_fn<GATE>(z);
        sa[t] += gv[t] * s * n;
        sb[t] += gv[t] * a * gate_deriv<GATE>(z, s) * n;
      }
    }
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    red[0][rl][cg * 8 + t] = sa[t];
    red[1][rl][cg * 8 + t] = sb[t];
  }
  __syncthreads();
  if (threadIdx.x < 128) {
    const int w = threadIdx.x >> 6, c = threadIdx.x & 63;
    const int col = blockIdx.x * 64 + c;
    float s = 0.f;
    for (int i = 0; i < 32; ++i) s += red[w][i][c];
    if (col < N) part[((int64_t)blockIdx.y * 2 + w) * N + col] = s;
  }
}

__global__ __launch_bounds__(256) void swishrn_gain_final_kernel(const float* __restrict__ part,
                                                                 int chunks, int N,
                                                                 float* __restrict__ dgain) {
  const int j = blockIdx.x * 256 + threadIdx.x;  // j < 2N: [g_a; g_b]
  if (j >= 2 * N) return;
  const int w = j / N, col = j - w * N;
  const float* p = part + (int64_t)w * N + col;
  const int64_t stride = 2 * (int64_t)N;
  // chunks in order; the loads of 8 chunks are issued before their adds
  float s = 0.f;
  int c = 0;
  for (; c + 8 <= chunks; c += 8) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = p[(c + q) * stride];
#pragma unroll
    for (int q = 0; q < 8; ++q) s += v[q];
  }
  for (; c < chunks; ++c) s += p[c * stride];
  dgain[j] = s;
}

int swishrn_groups(int N, int block) { return (block <= 0 || block >= N) ? 1 : cdiv(N, block); }

static int vec_ok(DType dt, std::initializer_list<std::pair<const void*, int64_t>> rows) {
  const int64_t e = dt == DT_BF16 ? 8 : 4;
  for (const auto& r : rows)
    if (((uintptr_t)r.first & 15) || r.second % e) return 0;
  return 1;
}

template <typename T, int GATE>
static void fwd_launch(bool full, const void* pre, int64_t ldp, int M, int N, const float* gain,
                       float eps, void* out, int64_t ldo, float* rinv, int nblk, int vec,
                       hipStream_t s) {
  const dim3 grid(cdiv(M, 4));
  if (full)
    swishrn_fwd_rows_kernel<T, GATE, true><<<grid, 256, 0, s>>>((const T*)pre, ldp, M, N, gain, eps,
                                                                (T*)out, ldo, rinv, nblk, vec);
  else
    swishrn_fwd_rows_kernel<T, GATE, false><<<grid, 256, 0, s>>>((const T*)pre, ldp, M, N, gain, eps,
                                                                 (T*)out, ldo, rinv, nblk, vec);
}

hipError_t swishrn_fwd_rows(DType dt, const void* pre, int64_t ldp, int M, int N, int block, int gate,
                            const float* gain, float eps, void* out, int64_t ldo, float* rinv,
                            hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  if ((block != 0 && block != NORM_TILE) || (gate != GATE_SIGMOID && gate != GATE_HARD)) {
    set_error("SwishRN: block must be 0 or %d, gate 1 or 2", NORM_TILE);
    return hipErrorInvalidValue;
  }
  const int nblk = swishrn_groups(N, block);
  const bool full = nblk == 1 && block == 0;
  const int vec = vec_ok(dt, {{pre, ldp}, {out, ldo}});
  if (dt == DT_BF16) {
    if (gate == GATE_SIGMOID) fwd_launch<bf16_t, GATE_SIGMOID>(full, pre, ldp, M, N, gain, eps, out, ldo, rinv, nblk, vec, s);
    else fwd_launch<bf16_t, GATE_HARD>(full, pre, ldp, M, N, gain, eps, out, ldo, rinv, nblk, vec, s);
  } else {
    if (gate == GATE_SIGMOID) fwd_launch<float, GATE_SIGMOID>(full, pre, ldp, M, N, gain, eps, out, ldo, rinv, nblk, vec, s);
    else fwd_launch<float, GATE_HARD>(full, pre, ldp, M, N, gain, eps, out, ldo, rinv, nblk, vec, s);
  }
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

template <typename T, int GATE>
static void bwd_launch(bool full, const void* go, int64_t ldg, const void* pre, int64_t ldp,
                       const float* rinv, int nblk, int M, int N, const float* gain, void* dh,
                       int64_t ldd, int vec, hipStream_t s) {
  const dim3 grid(cdiv(M, 4));
  if (full)
    swishrn_bwd_rows_kernel<T, GATE, true><<<grid, 256, 0, s>>>((const T*)go, ldg, (const T*)pre, ldp,
                                                                rinv, nblk, M, N, gain, (T*)dh, ldd, vec);
  else
    swishrn_bwd_rows_kernel<T, GATE, false><<<grid, 256, 0, s>>>((const T*)go, ldg, (const T*)pre, ldp,
                                                                 rinv, nblk, M, N, gain, (T*)dh, ldd, vec);
}

hipError_t swishrn_bwd_rows(DType dt, const void* go, int64_t ldg, const void* pre, int64_t ldp,
                            const float* rinv, int M, int N, int block, int gate, const float* gain,
                            void* dh, int64_t ldd, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  if ((block != 0 && block != NORM_TILE) || (gate != GATE_SIGMOID && gate != GATE_HARD)) {
    set_error("SwishRN: block must be 0 or %d, gate 1 or 2", NORM_TILE);
    return hipErrorInvalidValue;
  }
  const int nblk = swishrn_groups(N, block);
  const bool full = nblk == 1 && block == 0;
  const int vec = vec_ok(dt, {{go, ldg}, {pre, ldp}, {dh, ldd}});
  if (dt == DT_BF16) {
    if (gate == GATE_SIGMOID) bwd_launch<bf16_t, GATE_SIGMOID>(full, go, ldg, pre, ldp, rinv, nblk, M, N, gain, dh, ldd, vec, s);
    else bwd_launch<bf16_t, GATE_HARD>(full, go, ldg, pre, ldp, rinv, nblk, M, N, gain, dh, ldd, vec, s);
  } else {
    if (gate == GATE_SIGMOID) bwd_launch<float, GATE_SIGMOID>(full, go, ldg, pre, ldp, rinv, nblk, M, N, gain, dh, ldd, vec, s);
    else bwd_launch<float, GATE_HARD>(full, go, ldg, pre, ldp, rinv, nblk, M, N, gain, dh, ldd, vec, s);
  }
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

size_t swishrn_gain_workspace(int M, int N) {
  return (size_t)cdiv(M > 0 ? M : 1, GG_ROWS) * 2 * (size_t)N * sizeof(float);
}

template <typename T, int GATE>
static void gain_launch(dim3 grid, const void* go, int64_t ldg, const void* pre, int64_t ldp,
                        const float* rinv, int nblk, int block, int M, int N, const float* gain,
                        int vec, float* part, hipStream_t s) {
  swishrn_gain_partial_kernel<T, GATE><<<grid, 256, 0, s>>>((const T*)go, ldg, (const T*)pre, ldp, rinv,
                                                            nblk, block, M, N, gain, vec, part);
}

hipError_t swishrn_gain_grad(DType dt, const void* go, int64_t ldg, const void* pre, int64_t ldp,
                             const float* rinv, int M, int N, int block, int gate,
                             const float* gain, float* dgain, void* ws, hipStream_t s) {
  if (N == 0 || !dgain) return hipSuccess;
  if ((block != 0 && block != NORM_TILE) || (gate != GATE_SIGMOID && gate != GATE_HARD)) {
    set_error("SwishRN: block must be 0 or %d, gate 1 or 2", NORM_TILE);
    return hipErrorInvalidValue;
  }
  const int chunks = M > 0 ? cdiv(M, GG_ROWS) : 0;
  float* part = (float*)ws;
  if (chunks > 0) {
    const int nblk = swishrn_groups(N, block);
    const int blk = nblk == 1 ? 0 : block;
    const dim3 grid(cdiv(N, 64), chunks);
    const int vec = vec_ok(dt, {{go, ldg}, {pre, ldp}});
    if (dt == DT_BF16) {
      if (gate == GATE_SIGMOID) gain_launch<bf16_t, GATE_SIGMOID>(grid, go, ldg, pre, ldp, rinv, nblk, blk, M, N, gain, vec, part, s);
      else gain_launch<bf16_t, GATE_HARD>(grid, go, ldg, pre, ldp, rinv, nblk, blk, M, N, gain, vec, part, s);
    } else {
      if (gate == GATE_SIGMOID) gain_launch<float, GATE_SIGMOID>(grid, go, ldg, pre, ldp, rinv, nblk, blk, M, N, gain, vec, part, s);
      else gain_launch<float, GATE_HARD>(grid, go, ldg, pre, ldp, rinv, nblk, blk, M, N, gain, vec, part, s);
    }
    LAT_LAUNCH_CHECK();
  }
  swishrn_gain_final_kernel<<<cdiv(2 * (int64_t)N, 256), 256, 0, s>>>(part, chunks, N, dgain);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
