// Dense contractions of the MLPs and heads:
//   C[m, n] = epilogue( sum_k A(m, k) * B(n, k) )
// with A(m,k) = A[m*lda + k] (K-contiguous) or A[k*lda + m] (M-contiguous),
// and likewise for B, so the forward (X W^T), input-gradient (dY W) and
// weight-gradient (dY^T X) products all map onto one kernel family without
// materialised transposes.
//
// bf16 path (gfx950 MFMA): block tile 128x128, K step 64, 256 threads as a
// 2x2 grid of waves each owning a 64x64 sub-tile = 2x2 fragments of
// v_mfma_f32_32x32x16_bf16.  Operands are staged through LDS in [row][k]
// layout (k contiguous, rows padded to 72 elements).  A K-contiguous operand
// is copied with 16-byte loads; an M-contiguous operand is read with 16-byte
// loads along M (8 rows x 4 k per thread) and transposed in registers before
// the LDS write.  Products without K segmentation whose operands span less
// than 2 GiB load through buffer resources: a thread's offsets are fixed at
// the start and a K step adds one uniform count, and what lies past the
// operand reads zero in hardware, so the K loop carries no per-load address
// arithmetic or bounds branches (the top MLP's products 10-15% faster than
// with per-load pointers and selects).  There an M-contiguous operand is
// staged k-major (16-byte copies of whole k rows, no register transpose) and
// its MFMA fragments are read with gfx950's transposed LDS reads
// (ds_read_b64_tr_b16): the weight-gradient product of top layer 1 went from
// 105 to 73 us, its input gradient from 71 to 61 us.  On the buffer path the
// K loop runs unchecked while four more tiles remain (no K tail, no
// conditional load or store, one basic block), and the next tile's global
// loads and the other LDS stage's stores are issued in four parts, each after
// one 16-k slice of MFMAs and fenced there against the scheduler (which
// otherwise gathers the loads at the end of the step and shortens the
// prefetch): the 256x256 products of the deep stack went from 4.7-4.8 to
// 3.7-3.9 ms, top layer 1 forward 52.7 -> 48 us; the last tiles finish in
// the checked loop.  Global loads run two K steps ahead of the MFMAs (two
// register stages, two LDS stages).  Tiles are numbered so that each XCD works
// through whole row panels of A (one L2 keeps the panel while the XCD sweeps
// the columns).  The finished tile is staged through LDS as fp32 so that the
// epilogue reads and writes rows with 16-byte vectors.  Split-K writes fp32
// partials that a second kernel sums in a fixed order, so results are
// deterministic.
//
// Epilogue: + bias[n], + addend[m, n], + C (accumulate), ReLU, or multiply by
// (mask[m, n] > 0) (the ReLU derivative read from a stored activation), then
// round to the output dtype.
//
// BlockNorm epilogue (SwishRN, Sections 3.3.4 and 3.5.3): the pre-activation
// h = acc + bias is normalised over each row's 128-column group -- exactly
// the columns of one 128x128 tile (half a 256x256 tile), so the statistic
// needs no data from another workgroup -- and C = (g_a n) * gate(g_b n) with
// n = h / sqrt(mean h^2 + eps); h (rounded to C's dtype) and the group's
// 1 / sqrt(...) are stored for the backward.  The 8 columns of a thread
// belong to one aligned 16-lane group per 128 columns, so the sum of squares
// is a 16-lane butterfly.
#include <mutex>
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "swishrn.h"

namespace lat {

constexpr int GBM = 128, GBN = 128, GBK = 64, GPAD = 8, GLD = GBK + GPAD;
constexpr int CLD = GBN + 4;  // fp32 row stride of the staged C tile
constexpr size_t GEMM_LDS = (size_t)2 * (GBM + GBN) * GLD * sizeof(uint16_t);  // 73,728 B
static_assert((size_t)GBM * CLD * sizeof(float) <= GEMM_LDS, "C staging must fit the operand stages");

struct Epi {
  const float* bias;    // [N] or null
  int relu;
  const void* mask;     // activation whose sign gates the output, or null
  DType mask_dt;
  int64_t ldm, s_mask;
  const float* addend;  // + addend[m*ld_add + n] (fp32) or null
  int64_t ld_add, s_add;
  int accumulate;       // + the existing (fp32) C
  // BlockNorm / SwishRN (kernels instantiated with NORM = gate): gain [2, N],
  // pre [M, ldp] (C's dtype), rinv [M, nblk]
  const float* gain;
  float eps;
  void* pre;
  int64_t ldp;
  float* rinv;
  int nblk;
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

__device__ inline void ld8f(const float* p, float* v) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i] = a[i];
    v[4 + i] = b[i];
  }
}

// Per-thread coefficients of the BlockNorm epilogue: a thread stores the
// same 8 columns col.. in every row it handles, so bias, g_a, g_b (zeros
// past N) and 1 / |group| are loaded once.
struct NormCoef {
  float b[8], ga[8], gb[8];
  float inv_cnt;
};

__device__ inline void load_norm_coef(const Epi& e, int col, int N, NormCoef& c) {
  load_gains8(e.gain, N, col, c.ga, c.gb);
  if (e.bias && col + 8 <= N && ((uintptr_t)e.bias & 15) == 0) {
    ld8f(e.bias + col, c.b);
  } else {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const bool ok = e.bias && col + t < N;
      c.b[t] = ok ? e.bias[ok ? col + t : 0] : 0.f;
    }
  }
  c.inv_cnt = inv_group_size(col, N);
}

// SwishRN with BlockNorm on 8 columns col.. of row `row` of the finished
// fp32 tile (see the header comment).  Every lane of the wave calls it (the
// shuffles need the whole 16-lane group); rows past M and columns past N
// store nothing.
template <typename CT, int GATE>
__device__ inline void epi_blocknorm8(CT* C, int64_t ldc, int row, int col, int M, int N, float* v,
                                      const Epi& e, const NormCoef& nc, int vec) {
  float ss = 0.f;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    v[t] = col + t < N ? v[t] + nc.b[t] : 0.f;
    ss += v[t] * v[t];
  }
  ss = sum16(ss);
  const float r = rsqrtf(ss * nc.inv_cnt + e.eps);
  if (row >= M || col >= N) return;
  if (col % NORM_TILE == 0) e.rinv[(int64_t)row * e.nblk + col / NORM_TILE] = r;
  float o[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const float n = v[t] * r;
    o[t] = (nc.ga[t] * n) * gate_fn<GATE>(nc.gb[t] * n);
  }
  CT* c = C + (int64_t)row * ldc + col;
  CT* p = reinterpret_cast<CT*>(e.pre) + (int64_t)row * e.ldp + col;
  if (vec && col + 8 <= N) {
    if constexpr (sizeof(CT) == 2) {
      stg16(c, Vec16<bf16_t>::pack(o));
      stg16(p, Vec16<bf16_t>::pack(v));
    } else {
      stg16(c, Vec16<float>::pack(o));
      stg16(c + 4, Vec16<float>::pack(o + 4));
      stg16(p, Vec16<float>::pack(v));
      stg16(p + 4, Vec16<float>::pack(v + 4));
    }
  } else {
#pragma unroll
    for (int t = 0; t < 8; ++t)
      if (col + t < N) {
        st(c + t, o[t]);
        st(p + t, v[t]);
      }
  }
}


// Epilogue of 8 consecutive columns of one row with 16-byte vectors (the
// caller guarantees alignment and col + 8 <= N).
template <typename CT>
__device__ inline void epi_store8(CT* C, int64_t ldc, int row, int col, float* v, const Epi& e,
                                  int64_t bz) {
  float t[8];
  if (e.bias) {
    ld8f(e.bias + col, t);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += t[i];
  }
  if (e.addend) {
    ld8f(e.addend + bz * e.s_add + (int64_t)row * e.ld_add + col, t);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += t[i];
  }
  CT* c = C + (int64_t)row * ldc + col;
  if (e.accumulate) {  // fp32 C only
    ld8f(reinterpret_cast<const float*>(c), t);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += t[i];
  }
  if (e.relu) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = v[i] > 0.f ? v[i] : 0.f;
  }
  if (e.mask) {
    const int64_t mi = bz * e.s_mask + (int64_t)row * e.ldm + col;
    if (e.mask_dt == DT_BF16) {
      Vec16<bf16_t>::unpack(ldg16(reinterpret_cast<const bf16_t*>(e.mask) + mi), t);
    } else {
      ld8f(reinterpret_cast<const float*>(e.mask) + mi, t);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = t[i] > 0.f ? v[i] : 0.f;
  }
  if constexpr (sizeof(CT) == 2) {
    stg16(c, Vec16<bf16_t>::pack(v));
  } else {
    stg16(c, Vec16<float>::pack(v));
    stg16(c + 4, Vec16<float>::pack(v + 4));
  }
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
// K-contiguous, 16-byte vectors: ROWS rows x 64 k = 8 vectors per row,
// ROWS / 32 per thread.
// The loads are straight-line code: an element outside the matrix reads
// element (0, 0) instead (its address is selected, not its value) and
// store() writes zeros for it.  A load inside a branch, or whose value is
// selected at once, makes the compiler wait there for it and for every load
// issued before it, which would cut the prefetch distance to one step.
template <int ROWS = GBM, int THREADS = 256>
struct LoadK {
  static constexpr int NV = ROWS * 8 / THREADS;
  u32x4 r[NV];
  int R_, K_, r0_, k0_;
  bool edge_;
  // edge: the tile may reach past R rows or K columns (uniform per block and step)
  __device__ inline void load(const Opnd& o, int R, int K, int r0, int k0, bool edge) {
    R_ = R; K_ = K; r0_ = r0; k0_ = k0; edge_ = edge;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = threadIdx.x + i * THREADS;
      const int rr = v >> 3, kc = (v & 7) * 8;
      const int gr = r0 + rr, gk = k0 + kc;
      const bool ok = !edge || (gr < R && gk < K);
      r[i] = ldg16(o.p + (ok ? (int64_t)gr * o.ld + koff<false>(o, gk) : 0));
    }
  }
  __device__ inline void store(bf16_t* S) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = threadIdx.x + i * THREADS;
      const int rr = v >> 3, kc = (v & 7) * 8;
      u32x4 x = r[i];
      if (edge_) {
        const int gr = r0_ + rr, gk = k0_ + kc;
        if (!(gr < R_ && gk < K_)) {
          x = u32x4{0, 0, 0, 0};
        } else if (gk + 8 > K_) {
          // a vector reaching past K (rows padded to 8 elements): zero the tail
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (gk + e >= K_) x[e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
        }
      }
      *reinterpret_cast<u32x4*>(S + rr * GLD + kc) = x;
    }
  }
};
// MN-contiguous, 16-byte vectors along M: a thread holds 8 consecutive rows x
// 4 consecutive k (four 16-byte loads), transposed in registers to 4-k pieces
// per row (8-byte LDS writes).  Wave w, lane l: row group mg = 4w + l/16,
// k group kg = l%16, so one load instruction reads 64 contiguous bytes of
// each of 16 k-rows, and the 16 lanes of a group write one row's 128 bytes.
// In general item it = thread + q * THREADS is row group it / 16, k group
// it % 16 (ROWS / 8 row groups x 16 k groups).
template <int ROWS = GBM, int THREADS = 256>
struct LoadMN {
  static constexpr int NI = ROWS * 2 / THREADS;
  u32x4 r[NI][4];
  int R_, K_, r0_, k0_;
  bool edge_;
  __device__ inline void load(const Opnd& o, int R, int K, int r0, int k0, bool edge) {
    R_ = R; K_ = K; r0_ = r0; k0_ = k0; edge_ = edge;
#pragma unroll
    for (int q = 0; q < NI; ++q) {
      const int it = threadIdx.x + q * THREADS;
      const int gr = r0 + (it >> 4) * 8, kb = k0 + (it & 15) * 4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int gk = kb + i;
        const bool ok = !edge || (gk < K && gr < R);
        r[q][i] = ldg16(o.p + (ok ? koff<true>(o, gk) + gr : 0));
      }
    }
  }
  __device__ inline void store(bf16_t* S) {
#pragma unroll
    for (int q = 0; q < NI; ++q) {
      const int it = threadIdx.x + q * THREADS;
      u32x4 x[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[i] = r[q][i];
        if (edge_) {
          const int gr = r0_ + (it >> 4) * 8, gk = k0_ + (it & 15) * 4 + i;
          if (!(gk < K_ && gr < R_)) x[i] = u32x4{0, 0, 0, 0};
        }
      }
      bf16_t* s = S + ((it >> 4) * 8) * GLD + (it & 15) * 4;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        // row j of the group: (k0, k1, k2, k3) = half (j & 1) of word j/2 of x[0..3]
        const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t lo = __builtin_amdgcn_perm(x[1][j >> 1], x[0][j >> 1], sel);
        const uint32_t hi = __builtin_amdgcn_perm(x[3][j >> 1], x[2][j >> 1], sel);
        *reinterpret_cast<uint2*>(s + j * GLD) = uint2{lo, hi};
      }
    }
  }
};
// Generic element loader (any alignment / transposition).  Consecutive lanes
// take consecutive elements in memory: along k for a K-contiguous operand,
// along the rows for an MN-contiguous one.  It holds no tile in registers:
// load() records the tile and store() reads it from memory straight into LDS
// (2-byte loads would otherwise pin 32 registers per stage).
template <bool MN>
struct LoadElem {
  const Opnd* o;
  int R, K, r0, k0;
  __device__ static inline void at(int e, int& rr, int& kk) {
    if (MN) {
      rr = e & (GBM - 1);
      kk = e / GBM;
    } else {
      rr = e >> 6;
      kk = e & 63;
    }
  }
  __device__ inline void load(const Opnd& o_, int R_, int K_, int r0_, int k0_, bool /*edge*/) {
    o = &o_;
    R = R_;
    K = K_;
    r0 = r0_;
    k0 = k0_;
  }
  __device__ inline void store(bf16_t* S) {
    // all 32 loads in flight at once (two elements per register), then the writes
    uint32_t r[16];
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      int rr, kk;
      at(threadIdx.x + i * 256, rr, kk);
      const int gr = r0 + rr, gk = k0 + kk;
      uint32_t v = 0;
      if (gr < R && gk < K)
        v = MN ? o->p[koff<true>(*o, gk) + gr] : o->p[(int64_t)gr * o->ld + koff<false>(*o, gk)];
      if (i & 1) r[i >> 1] |= v << 16;
      else r[i >> 1] = v;
    }
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      int rr, kk;
      at(threadIdx.x + i * 256, rr, kk);
      S[rr * GLD + kk] = (bf16_t)((i & 1) ? (r[i >> 1] >> 16) : (r[i >> 1] & 0xffffu));
    }
  }
};
// Buffer-resource loaders (16-byte vectors, no K segmentation, each operand
// spanning less than 2 GiB).  The addressing (resource and a thread's byte
// offsets at k = kbeg) is set up once and shared by the register stages;
// each K step adds one uniform byte count.  The resource's size ends at the
// operand's last element in the block's K range, so a vector past it reads
// zeros in hardware: rows past R of a K-contiguous operand (their offsets
// are pushed past 2 GiB) and k rows past kend of an MN-contiguous one.
// What stays inside the range but lies past kend (the K tail of a
// K-contiguous row, read from the next row) is zeroed at the LDS store of
// the last step; MN-contiguous rows past R (inside a padded k row) only
// reach output rows or columns that are never written.
template <bool MN, int ROWS = GBM, int THREADS = 256>
struct BufAddr {
  static constexpr int NV = MN ? ROWS * 2 / THREADS : ROWS * 8 / THREADS;
  __amdgpu_buffer_rsrc_t rs;
  uint32_t voff[NV];
  uint32_t kbytes;  // bytes per unit of k
  int kbeg, kend;
  __device__ inline void init(const Opnd& o, int R, int kbeg_, int kend_, int r0) {
    kbeg = kbeg_;
    kend = kend_;
    int64_t last;
    if (MN) last = kend > 0 ? (int64_t)(kend - 1) * o.ld + ((R + 7) & ~7) : 0;
    else last = R > 0 ? (int64_t)(R - 1) * o.ld + ((kend + 7) & ~7) : 0;
    rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(o.p), 0, (int)(uint32_t)(last * 2),
                                           BUF_RSRC_WORD3);
    kbytes = MN ? (uint32_t)(o.ld * 2) : 2u;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = threadIdx.x + i * THREADS;
      if (MN) {
        const int gr = r0 + (v >> 4) * 8, kq = kbeg + (v & 15) * 4;
        voff[i] = (uint32_t)(((int64_t)kq * o.ld + gr) * 2);
      } else {
        const int gr = r0 + (v >> 3), kc = (v & 7) * 8;
        voff[i] = gr < R ? (uint32_t)(((int64_t)gr * o.ld + kbeg + kc) * 2) : 0x80000000u;
      }
    }
  }
};
template <int ROWS = GBM, int THREADS = 256>
struct BufK {
  using Addr = BufAddr<false, ROWS, THREADS>;
  static constexpr int NV = Addr::NV;
  u32x4 r[NV];
  int k0_;
  bool tail_;
  __device__ inline void load(const Addr& a, int k0, bool tail) {
    k0_ = k0;
    tail_ = tail;
    const uint32_t d = (uint32_t)(k0 - a.kbeg) * 2u;
#pragma unroll
    for (int i = 0; i < NV; ++i) r[i] = __builtin_amdgcn_raw_buffer_load_b128(a.rs, (int)(a.voff[i] + d), 0, 0);
  }
  // part p of P of a load or of an LDS store (the unchecked loop, whose
  // tiles have no K tail); the load records the tile for store()
  __device__ inline void load_part(const Addr& a, int k0, int p, int P) {
    if (p == 0) {
      k0_ = k0;
      tail_ = k0 + GBK > a.kend;
    }
    const uint32_t d = (uint32_t)(k0 - a.kbeg) * 2u;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (i * P / NV == p) r[i] = __builtin_amdgcn_raw_buffer_load_b128(a.rs, (int)(a.voff[i] + d), 0, 0);
  }
  __device__ inline void store_part(const Addr& /*a*/, bf16_t* S, int p, int P) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (i * P / NV != p) continue;
      const int v = threadIdx.x + i * THREADS;
      *reinterpret_cast<u32x4*>(S + (v >> 3) * GLD + (v & 7) * 8) = r[i];
    }
  }
  __device__ inline void store(const Addr& a, bf16_t* S) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = threadIdx.x + i * THREADS;
      const int rr = v >> 3, kc = (v & 7) * 8;
      u32x4 x = r[i];
      if (tail_) {
        const int gk = k0_ + kc;
        if (gk >= a.kend) {
          x = u32x4{0, 0, 0, 0};
        } else if (gk + 8 > a.kend) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (gk + e >= a.kend) x[e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
        }
      }
      *reinterpret_cast<u32x4*>(S + rr * GLD + kc) = x;
    }
  }
};
template <int ROWS = GBM, int THREADS = 256>
struct BufMN {
  using Addr = BufAddr<true, ROWS, THREADS>;
  static constexpr int NI = Addr::NV;
  u32x4 r[NI][4];
  __device__ inline void load(const Addr& a, int k0, bool /*tail*/) {
    const uint32_t d = (uint32_t)(k0 - a.kbeg) * a.kbytes;
#pragma unroll
    for (int q = 0; q < NI; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        r[q][i] = __builtin_amdgcn_raw_buffer_load_b128(a.rs, (int)(a.voff[q] + d + (uint32_t)i * a.kbytes), 0, 0);
  }
  __device__ inline void load_part(const Addr& a, int k0, int p, int P) {
    const uint32_t d = (uint32_t)(k0 - a.kbeg) * a.kbytes;
#pragma unroll
    for (int q = 0; q < NI; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if ((q * 4 + i) * P / (4 * NI) == p)
          r[q][i] = __builtin_amdgcn_raw_buffer_load_b128(a.rs, (int)(a.voff[q] + d + (uint32_t)i * a.kbytes), 0, 0);
  }
  __device__ inline void store_part(const Addr& /*a*/, bf16_t* S, int p, int P) {
#pragma unroll
    for (int q = 0; q < NI; ++q) {
      const int it = threadIdx.x + q * THREADS;
      bf16_t* s = S + ((it >> 4) * 8) * GLD + (it & 15) * 4;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if ((q * 8 + j) * P / (8 * NI) != p) continue;
        // row j of the group: (k0, k1, k2, k3) = half (j & 1) of word j/2 of the four vectors
        const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t lo = __builtin_amdgcn_perm(r[q][1][j >> 1], r[q][0][j >> 1], sel);
        const uint32_t hi = __builtin_amdgcn_perm(r[q][3][j >> 1], r[q][2][j >> 1], sel);
        *reinterpret_cast<uint2*>(s + j * GLD) = uint2{lo, hi};
      }
    }
  }
  __device__ inline void store(const Addr& a, bf16_t* S) {
#pragma unroll
    for (int p = 0; p < 4; ++p) store_part(a, S, p, 4);
  }
};

// An MN-contiguous operand staged k-major (buffer path): S[k][r] with r
// contiguous, ROWS rows per k row and no padding, copied with 16-byte loads
// and 16-byte LDS writes (no register transpose; a load instruction reads
// whole k rows: four of 256 bytes for 128-row tiles, two of 512 for 256).
// The 16-byte units of k row k are XOR-swizzled by 4 (k mod 4), so that the
// four consecutive k rows a transposed fragment read touches fall on
// disjoint banks (rows start on a 256-byte boundary, and the swizzle moves
// a 64-byte group of units to another quarter of the bank window).  Thread
// t holds unit t mod (ROWS / 8) of k rows t / (ROWS / 8) + (THREADS * 8 /
// ROWS) i.
template <int LD>
__device__ inline int km_off(int k, int r) { return k * LD + ((((r >> 3) ^ ((k & 3) << 2))) << 3) + (r & 7); }
template <int ROWS = GBM, int THREADS = 256>
struct BufMNK {
  static constexpr int UNITS = ROWS / 8;              // 16-byte units per k row
  static constexpr int KPI = THREADS / UNITS;         // k rows per load instruction round
  static constexpr int NV = ROWS * GBK / 8 / THREADS; // vectors per thread
  struct Addr {
    __amdgpu_buffer_rsrc_t rs;
    uint32_t voff;   // byte offset of the thread's unit in k row kbeg + t / UNITS
    uint32_t kbytes;
    int kbeg;
    __device__ inline void init(const Opnd& o, int R, int kbeg_, int kend, int r0) {
      kbeg = kbeg_;
      const int64_t last = kend > 0 ? (int64_t)(kend - 1) * o.ld + ((R + 7) & ~7) : 0;
      rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(o.p), 0, (int)(uint32_t)(last * 2),
                                             BUF_RSRC_WORD3);
      kbytes = (uint32_t)(o.ld * 2);
      const int k = kbeg + threadIdx.x / UNITS, u = threadIdx.x % UNITS;
      voff = (uint32_t)(((int64_t)k * o.ld + r0 + u * 8) * 2);
    }
  };
  u32x4 r[NV];
  __device__ inline void load(const Addr& a, int k0, bool /*tail*/) {
    const uint32_t d = (uint32_t)(k0 - a.kbeg) * a.kbytes;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      r[i] = __builtin_amdgcn_raw_buffer_load_b128(a.rs, (int)(a.voff + d + (uint32_t)(KPI * i) * a.kbytes), 0, 0);
  }
  __device__ inline void load_part(const Addr& a, int k0, int p, int P) {
    const uint32_t d = (uint32_t)(k0 - a.kbeg) * a.kbytes;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (i * P / NV == p)
        r[i] = __builtin_amdgcn_raw_buffer_load_b128(a.rs, (int)(a.voff + d + (uint32_t)(KPI * i) * a.kbytes), 0, 0);
  }
  __device__ inline void store_part(const Addr& /*a*/, bf16_t* S, int p, int P) {
    const int k = threadIdx.x / UNITS, u = threadIdx.x % UNITS;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (i * P / NV == p) *reinterpret_cast<u32x4*>(S + km_off<ROWS>(k + KPI * i, u * 8)) = r[i];
  }
  __device__ inline void store(const Addr& a, bf16_t* S) {
#pragma unroll
    for (int p = 0; p < 4; ++p) store_part(a, S, p, 4);
  }
  // row sums: the thread's 8 rows over its k rows of the step (k rows past
  // the range read zero)
  __device__ inline void rowsum(float (&rs)[8]) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float v[8];
      Vec16<bf16_t>::unpack(r[i], v);
#pragma unroll
      for (int e = 0; e < 8; ++e) rs[e] += v[e];
    }
  }
  // after the K loop: row sums added over the KPI k classes in class order
  // (LDS scratch `red` of KPI * ROWS floats; a barrier inside); thread t < ROWS
  // returns row t's sum
  __device__ inline static float rowsum_combine(const float (&rs)[8], float* red) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red[(threadIdx.x / UNITS) * ROWS + (threadIdx.x % UNITS) * 8 + e] = rs[e];
    __syncthreads();
    float s = 0.f;
    if (threadIdx.x < ROWS) {
#pragma unroll
      for (int c = 0; c < KPI; ++c) s += red[c * ROWS + threadIdx.x];
    }
    __syncthreads();
    return s;
  }
};

// MFMA operand fragment (32 rows from rbase, 8 k from ks) of a k-major tile
// by two transposed LDS reads (ds_read_b64_tr_b16).  Within each 16-lane
// group the read returns to lane j, as its element e, element j % 4 of the
// 8-byte piece addressed by lane 4e + j / 4; lane 4e + q therefore addresses
// rows rbase + 16 (g % 2) + 4q .. +3 of k row ks + 8 (g / 2) + e (g = lane /
// 16), and lane j receives row rbase + lane % 32 at four consecutive k.
typedef short i16x4 __attribute__((ext_vector_type(4)));
template <int LD>
__device__ inline bf16x8 frag_km(const bf16_t* S, int rbase, int ks, int lane) {
  const int g = lane >> 4, j = lane & 15;
  const int r = rbase + 16 * (g & 1) + 4 * (j & 3);
  const int k = ks + 8 * (g >> 1) + (j >> 2);
  typedef __attribute__((address_space(3))) i16x4 lds_v4;
  const lds_v4* p0 = (const lds_v4*)(S + km_off<LD>(k, r));
  const lds_v4* p1 = (const lds_v4*)(S + km_off<LD>(k + 4, r));
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_v4*>(p0));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_v4*>(p1));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Plain-pointer loaders behind the same interface (any K segmentation or span):
// the addressing is the operand and its bounds.
struct PlainAddr {
  Opnd o;
  int R, r0, kend;
  __device__ inline void init(const Opnd& o_, int R_, int /*kbeg*/, int kend_, int r0_) {
    o = o_;
    R = R_;
    r0 = r0_;
    kend = kend_;
  }
};
template <typename L>
struct PlainStage {
  using Addr = PlainAddr;
  L l;
  __device__ inline void load(const Addr& a, int k0, bool edge) { l.load(a.o, a.R, a.kend, a.r0, k0, edge); }
  __device__ inline void store(const Addr& /*a*/, bf16_t* S) { l.store(S); }
};

template <bool MN, bool VEC> struct LoaderSel;
template <> struct LoaderSel<false, true> { using T = LoadK<>; };
template <> struct LoaderSel<true, true> { using T = LoadMN<>; };
template <bool MN> struct LoaderSel<MN, false> { using T = LoadElem<MN>; };
// the register stage of an operand: buffer loaders (BUF) or plain ones
template <bool MN, bool VEC, bool BUF> struct StageSel { using T = PlainStage<typename LoaderSel<MN, VEC>::T>; };
template <> struct StageSel<false, true, true> { using T = BufK<>; };
template <> struct StageSel<true, true, true> { using T = BufMNK<>; };

// 64 k of MFMAs on the staged tiles: each wave 2x2 fragments of 32x32.
// KA / KB: that operand's tile is k-major (transposed fragment reads).
struct NoSide {
  __device__ inline void operator()(int) const {}
};
// side(q), q = 0..3, runs after the MFMAs of 16-k slice q (the next tile's
// loads and the other LDS stage's stores, overlapping the matrix work)
template <bool KA = false, bool KB = false, typename Side = NoSide>
__device__ inline void mma_k64(const bf16_t* As, const bf16_t* Bs, int wm, int wn, int lane,
                               f32x16 (&acc)[2][2], Side side = Side()) {
  const int frow = lane & 31, fk = (lane >> 5) * 8;
  const bf16_t* as = As + (wm * 64 + frow) * GLD + fk;
  const bf16_t* bs = Bs + (wn * 64 + frow) * GLD + fk;
#pragma unroll
  for (int ks = 0; ks < GBK; ks += 16) {
    const bf16x8 a0 = KA ? frag_km<GBM>(As, wm * 64, ks, lane) : *reinterpret_cast<const bf16x8*>(as + ks);
    const bf16x8 a1 = KA ? frag_km<GBM>(As, wm * 64 + 32, ks, lane) : *reinterpret_cast<const bf16x8*>(as + 32 * GLD + ks);
    const bf16x8 b0 = KB ? frag_km<GBN>(Bs, wn * 64, ks, lane) : *reinterpret_cast<const bf16x8*>(bs + ks);
    const bf16x8 b1 = KB ? frag_km<GBN>(Bs, wn * 64 + 32, ks, lane) : *reinterpret_cast<const bf16x8*>(bs + 32 * GLD + ks);
    acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
    acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
    acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
    acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
    side(ks / 16);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Grouped products (parameter untying): blockIdx.z = group.  Rows (gk = 0):
// group z is rows off[z] .. off[z+1]-1 of A, C and the epilogue operands,
// with its own B operand (+ z sB), bias (+ z N) and gains (+ z 2N); blocks
// past a group's rows exit at once.  K (gk = 1): group z sums k = off[z] ..
// off[z+1]-1 into its own C (+ z sC) and row sums (+ z M).
constexpr int GEMM_MAX_GROUPS = 16;
struct GroupSpec {
  int n;    // 0: not grouped
  int gk;
  int off[GEMM_MAX_GROUPS + 1];
  int64_t sB, sC;
};

// grid: x = M tiles * N tiles (renumbered per XCD), z = split index (split-K)
// or batch index (batched) or group (grouped; never two of them).  vec:
// 16-byte epilogue vectors allowed.
// rowsum (optional, not batched): rowsum[m] = sum over k of A[m][k], added in
// k order by the blocks of the first N tile from their LDS A tiles; with
// split-K each split's sum goes to rs_partial[split][m].
template <bool TA, bool TB, bool VA, bool VB, typename CT, int NORM = 0, bool BUF = false>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(
    Opnd A, Opnd Bm, CT* __restrict__ C, int64_t ldc, int M, int N, int K, int k_per_split,
    float* __restrict__ partial, Epi epi, int64_t sA, int64_t sB, int64_t sC, int batched, int vec,
    float* __restrict__ rowsum, float* __restrict__ rs_partial, GroupSpec grp) {
  extern __shared__ __attribute__((aligned(16))) unsigned char gemm_smem[];
  bf16_t* As[2];
  bf16_t* Bs[2];
  As[0] = reinterpret_cast<bf16_t*>(gemm_smem);
  Bs[0] = As[0] + GBM * GLD;
  As[1] = Bs[0] + GBN * GLD;
  Bs[1] = As[1] + GBM * GLD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int tiles_n = (N + GBN - 1) / GBN;
  const int tile = xcd_block(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * GBM, n0 = (tile % tiles_n) * GBN;
  const int64_t bz = batched ? blockIdx.z : 0;
  if (batched) {
    A.p += bz * sA;
    Bm.p += bz * sB;
    C += bz * sC;
  }
  int kbeg = batched ? 0 : blockIdx.z * k_per_split;
  int kend = batched ? K : min(K, kbeg + k_per_split);
  if (grp.n > 0) {
    const int gz = blockIdx.z;
    Bm.p += gz * grp.sB;
    if (grp.gk) {
      kbeg = grp.off[gz];
      kend = grp.off[gz + 1];
      C += gz * grp.sC;
      if (rowsum) rowsum += (int64_t)gz * M;
    } else {
      kbeg = 0;  // (blockIdx.z is the group, not a split index)
      kend = K;
      const int r0 = grp.off[gz];
      M = grp.off[gz + 1] - r0;
      if (m0 >= M) return;  // the whole block: past this group's rows
      A.p += TA ? (int64_t)r0 : (int64_t)r0 * A.ld;
      C += (int64_t)r0 * ldc;
      if (epi.bias) epi.bias += (int64_t)gz * N;
      if (epi.gain) epi.gain += (int64_t)gz * 2 * N;
      if (epi.pre) epi.pre = reinterpret_cast<CT*>(epi.pre) + (int64_t)r0 * epi.ldp;
      if (epi.rinv) epi.rinv += (int64_t)r0 * epi.nblk;
      if (epi.mask)
        epi.mask = reinterpret_cast<const char*>(epi.mask) + (int64_t)r0 * epi.ldm * (epi.mask_dt == DT_BF16 ? 2 : 4);
      if (epi.addend) epi.addend += (int64_t)r0 * epi.ld_add;
    }
  }

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  using SA = typename StageSel<TA, VA, BUF>::T;
  using SB = typename StageSel<TB, VB, BUF>::T;
  typename SA::Addr adA;
  typename SB::Addr adB;
  adA.init(A, M, kbeg, kend, m0);
  adB.init(Bm, N, kbeg, kend, n0);
  SA la0, la1;
  SB lb0, lb1;
  const int ktiles = kend > kbeg ? (kend - kbeg + GBK - 1) / GBK : 0;
  // tiles reaching past the matrix edge take the checked loads (uniform)
  const bool edge_m = m0 + GBM > M, edge_n = n0 + GBN > N;
  auto load = [&](auto& la, auto& lb, int kt) {
    const int k0 = kbeg + kt * GBK;
    const bool edge_k = k0 + GBK > kend;
    la.load(adA, k0, (BUF ? false : edge_m) || edge_k);
    lb.load(adB, k0, (BUF ? false : edge_n) || edge_k);
  };
  // row sums of A: thread t adds 32 k of row t/2 of each LDS A tile, or
  // (A staged k-major) its 8 rows over its k rows from the registers it
  // stores, combined over the threads after the loop
  constexpr bool KA = BUF && TA && VA, KB = BUF && TB && VB;
  const bool rs_on = rowsum != nullptr && n0 == 0;
  float rs = 0.f;
  float rsv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) rsv[e] = 0.f;
  auto stage_a = [&](auto& la, bf16_t* S) {
    if constexpr (KA) {
      if (rs_on) la.rowsum(rsv);
    }
    la.store(adA, S);
  };
  auto rowsum_step = [&](const bf16_t* as) {
    if (!KA && rs_on) {
      const bf16_t* p = as + (threadIdx.x >> 1) * GLD + (threadIdx.x & 1) * 32;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const u32x4 x = *reinterpret_cast<const u32x4*>(p + v * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          rs += __uint_as_float(x[e] << 16);
          rs += __uint_as_float(x[e] & 0xffff0000u);
        }
      }
    }
  };
  if (ktiles > 0) load(la0, lb0, 0);
  if (ktiles > 1) load(la1, lb1, 1);
  if (ktiles > 0) {
    stage_a(la0, As[0]);
    lb0.store(adB, Bs[0]);
  }
  __syncthreads();
  // Two register stages and two LDS stages: while the MFMAs consume LDS stage
  // s, the registers of the other stage receive the tile two steps ahead.
  // The loop body is two steps with no early exit (so the accumulators keep
  // their registers); an odd last step follows the loop.
  int kt = 0;
  if constexpr (BUF) {
    // unchecked steady state while tiles kt .. kt + 3 exist (no K tail, no
    // conditional load or store): the next tile's loads and the other
    // stage's stores are issued between the MFMA slices
    for (; kt + 4 <= ktiles; kt += 2) {
      const int k2 = kbeg + (kt + 2) * GBK, k3 = k2 + GBK;
      mma_k64<KA, KB>(As[0], Bs[0], wm, wn, lane, acc, [&](int q) {
        la0.load_part(adA, k2, q, 4);
        lb0.load_part(adB, k2, q, 4);
        if constexpr (KA) {
          if (q == 0 && rs_on) la1.rowsum(rsv);
        }
        la1.store_part(adA, As[1], q, 4);
        lb1.store_part(adB, Bs[1], q, 4);
      });
      rowsum_step(As[0]);
      __syncthreads();
      mma_k64<KA, KB>(As[1], Bs[1], wm, wn, lane, acc, [&](int q) {
        la1.load_part(adA, k3, q, 4);
        lb1.load_part(adB, k3, q, 4);
        if constexpr (KA) {
          if (q == 0 && rs_on) la0.rowsum(rsv);
        }
        la0.store_part(adA, As[0], q, 4);
        lb0.store_part(adB, Bs[0], q, 4);
      });
      rowsum_step(As[1]);
      __syncthreads();
    }
  }
  for (; kt + 2 <= ktiles; kt += 2) {
    if (kt + 2 < ktiles) load(la0, lb0, kt + 2);
    mma_k64<KA, KB>(As[0], Bs[0], wm, wn, lane, acc);
    rowsum_step(As[0]);
    stage_a(la1, As[1]);
    lb1.store(adB, Bs[1]);
    __syncthreads();
    if (kt + 3 < ktiles) load(la1, lb1, kt + 3);
    mma_k64<KA, KB>(As[1], Bs[1], wm, wn, lane, acc);
    rowsum_step(As[1]);
    if (kt + 2 < ktiles) {
      stage_a(la0, As[0]);
      lb0.store(adB, Bs[0]);
    }
    __syncthreads();
  }
  if (kt < ktiles) {
    mma_k64<KA, KB>(As[0], Bs[0], wm, wn, lane, acc);
    rowsum_step(As[0]);
    __syncthreads();
  }
  if (rs_on) {
    int row;
    if constexpr (KA) {
      // the k classes of each row added in class order (LDS is free: the
      // loop ended with a barrier)
      rs = BufMNK<>::rowsum_combine(rsv, reinterpret_cast<float*>(gemm_smem));
      row = threadIdx.x < GBM ? m0 + threadIdx.x : M;
    } else {
      rs += __shfl_xor(rs, 1, 64);  // the two halves of the row, in a fixed order
      row = (threadIdx.x & 1) == 0 ? m0 + (threadIdx.x >> 1) : M;
    }
    if (row < M) {
      if (rs_partial) rs_partial[(int64_t)blockIdx.z * M + row] = rs;
      else rowsum[row] = rs;
    }
  }

  // Stage the fp32 tile in LDS.  D[i][j] of a 32x32 fragment: lane holds
  // column (lane & 31), rows 8*(r/4) + 4*(lane/32) + r%4 for r = 0..15.
  float* Cs = reinterpret_cast<float*>(gemm_smem);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int cl = wn * 64 + j * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        Cs[rl * CLD + cl] = acc[i][j][r];
      }
    }
  __syncthreads();
  if constexpr (NORM != 0) {
    // one 128-column norm group per tile row: 16 lanes per row, the same
    // 8 columns for a thread in every row
    const int cl = (threadIdx.x % (GBN / 8)) * 8;
    NormCoef nc;
    load_norm_coef(epi, n0 + cl, N, nc);
#pragma unroll
    for (int q = 0; q < (GBM * GBN / 8) / 256; ++q) {
      const int rl = (threadIdx.x + q * 256) / (GBN / 8);
      float v[8];
      ld8f(Cs + rl * CLD + cl, v);
      epi_blocknorm8<CT, NORM>(C, ldc, m0 + rl, n0 + cl, M, N, v, epi, nc, vec);
    }
    return;
  }
  // Rows of the tile, 8 columns per thread.
#pragma unroll
  for (int q = 0; q < (GBM * GBN / 8) / 256; ++q) {
    const int chunk = threadIdx.x + q * 256;
    const int rl = chunk / (GBN / 8), cl = (chunk % (GBN / 8)) * 8;
    const int row = m0 + rl, col = n0 + cl;
    if (row >= M || col >= N) continue;
    float v[8];
    ld8f(Cs + rl * CLD + cl, v);
    if (partial) {
      float* pp = partial + ((int64_t)blockIdx.z * M + row) * N + col;
      if ((N & 3) == 0 && col + 8 <= N) {
        stg16(pp, Vec16<float>::pack(v));
        stg16(pp + 4, Vec16<float>::pack(v + 4));
      } else {
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (col + t < N) pp[t] = v[t];
      }
    } else if (vec && col + 8 <= N) {
      epi_store8<CT>(C, ldc, row, col, v, epi, bz);
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (col + t < N) epi_store<CT>(C, ldc, row, col + t, v[t], epi, bz);
    }
  }
}

// Sum of the splits' partials in split order; the loads of 16 splits are
// issued before their adds (a split's partial is a separate [M, N] slice, so
// a plain loop would wait for one load at a time).
__device__ inline float sum_splits(const float* __restrict__ p, int splits, int64_t stride) {
  float s = 0.f;
  int z = 0;
  for (; z + 16 <= splits; z += 16) {
    float v[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q] = p[(int64_t)(z + q) * stride];
#pragma unroll
    for (int q = 0; q < 16; ++q) s += v[q];
  }
  for (; z < splits; ++z) s += p[(int64_t)z * stride];
  return s;
}

template <typename CT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ partial,
                                                            int splits, int M, int N,
                                                            CT* __restrict__ C, int64_t ldc,
                                                            Epi epi, const float* __restrict__ rs_partial,
                                                            float* __restrict__ rowsum) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (rowsum && i < M) rowsum[i] = sum_splits(rs_partial + i, splits, M);
  if (i >= (int64_t)M * N) return;
  const int row = (int)(i / N), col = (int)(i % N);
  epi_store<CT>(C, ldc, row, col, sum_splits(partial + i, splits, (int64_t)M * N), epi, 0);
}

// --- large products: block tile 256x256, 4 waves of 128x128 (4x4 fragments) or 8 of 128x64 ---
// Twice the MFMA work per byte read from LDS of the 128x128 kernel (whose
// 64x64 wave tiles keep the LDS port as busy as the matrix cores), for
// products with enough 256x256 tiles to fill the chip.  Same staging (two
// register and two LDS stages, 16-byte vector loaders only), same epilogue;
// the fp32 tile is staged through LDS in two halves of 128 rows.  No split-K
// and no batching.
constexpr int BBM = 256, BBN = 256, BCLD = BBN + 4;
constexpr size_t GEMM_BIG_LDS = (size_t)2 * (BBM + BBN) * GLD * sizeof(uint16_t);  // 147,456 B
static_assert((size_t)(BBM / 2) * BCLD * sizeof(float) <= GEMM_BIG_LDS, "C staging must fit");

// NW waves as 2 (M) x NW/2 (N): each wave 128 x 1024/NW, 4 x FN fragments
template <bool MN, int THREADS, bool BUF> struct BigLoader;
template <int THREADS> struct BigLoader<false, THREADS, false> { using T = PlainStage<LoadK<BBM, THREADS>>; };
template <int THREADS> struct BigLoader<true, THREADS, false> { using T = PlainStage<LoadMN<BBM, THREADS>>; };
template <int THREADS> struct BigLoader<false, THREADS, true> { using T = BufK<BBM, THREADS>; };
template <int THREADS> struct BigLoader<true, THREADS, true> { using T = BufMNK<BBM, THREADS>; };

template <int FN, bool KA = false, bool KB = false, typename Side = NoSide>
__device__ inline void mma_big_k64(const bf16_t* As, const bf16_t* Bs, int wm, int wn, int lane,
                                   f32x16 (&acc)[4][FN], Side side = Side()) {
  const int frow = lane & 31, fk = (lane >> 5) * 8;
  const bf16_t* as = As + (wm * 128 + frow) * GLD + fk;
  const bf16_t* bs = Bs + (wn * FN * 32 + frow) * GLD + fk;
#pragma unroll
  for (int ks = 0; ks < GBK; ks += 16) {
    bf16x8 a[4], b[FN];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = KA ? frag_km<BBM>(As, wm * 128 + i * 32, ks, lane) : *reinterpret_cast<const bf16x8*>(as + i * 32 * GLD + ks);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      b[j] = KB ? frag_km<BBN>(Bs, wn * FN * 32 + j * 32, ks, lane) : *reinterpret_cast<const bf16x8*>(bs + j * 32 * GLD + ks);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    side(ks / 16);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <bool TA, bool TB, typename CT, int NW, int NORM = 0, bool BUF = false>
__global__ __launch_bounds__(NW * 64, 1) void gemm_big_kernel(Opnd A, Opnd Bm, CT* __restrict__ C,
                                                              int64_t ldc, int M, int N, int K,
                                                              Epi epi, int vec,
                                                              float* __restrict__ rowsum) {
  constexpr int THREADS = NW * 64;
  constexpr int FN = 8 / NW * 2;  // fragments along N per wave: 4 (4 waves) or 2 (8 waves)
  extern __shared__ __attribute__((aligned(16))) unsigned char gemm_smem[];
  bf16_t* As[2];
  bf16_t* Bs[2];
  As[0] = reinterpret_cast<bf16_t*>(gemm_smem);
  Bs[0] = As[0] + BBM * GLD;
  As[1] = Bs[0] + BBN * GLD;
  Bs[1] = As[1] + BBM * GLD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / (NW / 2), wn = w % (NW / 2);
  const int tiles_n = (N + BBN - 1) / BBN;
  const int tile = xcd_block(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * BBM, n0 = (tile % tiles_n) * BBN;

  f32x16 acc[4][FN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // k-major staging for B when M-contiguous, for A only when B is too (A
  // k-major beside a K-contiguous B, or both k-major, costs registers in the
  // K loop); otherwise the register transpose
  constexpr bool KA = BUF && TA && TB, KB = BUF && TB && !TA;
  using SA = typename std::conditional<BUF && TA && !KA, BufMN<BBM, THREADS>,
                                       typename BigLoader<TA, THREADS, BUF>::T>::type;
  using SB = typename std::conditional<BUF && TB && !KB, BufMN<BBM, THREADS>,
                                       typename BigLoader<TB, THREADS, BUF>::T>::type;
  typename SA::Addr adA;
  typename SB::Addr adB;
  adA.init(A, M, 0, K, m0);
  adB.init(Bm, N, 0, K, n0);
  SA la0, la1;
  SB lb0, lb1;
  const int ktiles = (K + GBK - 1) / GBK;
  const bool edge_m = m0 + BBM > M, edge_n = n0 + BBN > N;
  auto load = [&](auto& la, auto& lb, int kt) {
    const int k0 = kt * GBK;
    const bool edge_k = k0 + GBK > K;
    la.load(adA, k0, (BUF ? false : edge_m) || edge_k);
    lb.load(adB, k0, (BUF ? false : edge_n) || edge_k);
  };
  // row sums of A (blocks of the first N tile): THREADS / 256 threads per
  // row, each adding 64 / (THREADS / 256) consecutive k
  constexpr int TPR = THREADS / BBM;
  const bool rs_on = rowsum != nullptr && n0 == 0;
  float rs = 0.f;
  float rsv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) rsv[e] = 0.f;
  auto stage_a = [&](auto& la, bf16_t* S) {
    if constexpr (KA) {
      if (rs_on) la.rowsum(rsv);
    }
    la.store(adA, S);
  };
  auto rowsum_step = [&](const bf16_t* as) {
    if (!KA && rs_on) {
      const bf16_t* p = as + (threadIdx.x / TPR) * GLD + (threadIdx.x % TPR) * (GBK / TPR);
#pragma unroll
      for (int v = 0; v < GBK / TPR / 8; ++v) {
        const u32x4 x = *reinterpret_cast<const u32x4*>(p + v * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          rs += __uint_as_float(x[e] << 16);
          rs += __uint_as_float(x[e] & 0xffff0000u);
        }
      }
    }
  };
  if (ktiles > 0) load(la0, lb0, 0);
  if (ktiles > 1) load(la1, lb1, 1);
  if (ktiles > 0) {
    stage_a(la0, As[0]);
    lb0.store(adB, Bs[0]);
  }
  __syncthreads();
  int kt = 0;
  if constexpr (BUF) {
    // unchecked steady state, as in the 128x128 kernel
    for (; kt + 4 <= ktiles; kt += 2) {
      const int k2 = (kt + 2) * GBK, k3 = k2 + GBK;
      mma_big_k64<FN, KA, KB>(As[0], Bs[0], wm, wn, lane, acc, [&](int q) {
        la0.load_part(adA, k2, q, 4);
        lb0.load_part(adB, k2, q, 4);
        if constexpr (KA) {
          if (q == 0 && rs_on) la1.rowsum(rsv);
        }
        la1.store_part(adA, As[1], q, 4);
        lb1.store_part(adB, Bs[1], q, 4);
      });
      rowsum_step(As[0]);
      __syncthreads();
      mma_big_k64<FN, KA, KB>(As[1], Bs[1], wm, wn, lane, acc, [&](int q) {
        la1.load_part(adA, k3, q, 4);
        lb1.load_part(adB, k3, q, 4);
        if constexpr (KA) {
          if (q == 0 && rs_on) la0.rowsum(rsv);
        }
        la0.store_part(adA, As[0], q, 4);
        lb0.store_part(adB, Bs[0], q, 4);
      });
      rowsum_step(As[1]);
      __syncthreads();
    }
  }
  for (; kt + 2 <= ktiles; kt += 2) {
    if (kt + 2 < ktiles) load(la0, lb0, kt + 2);
    mma_big_k64<FN, KA, KB>(As[0], Bs[0], wm, wn, lane, acc);
    rowsum_step(As[0]);
    stage_a(la1, As[1]);
    lb1.store(adB, Bs[1]);
    __syncthreads();
    if (kt + 3 < ktiles) load(la1, lb1, kt + 3);
    mma_big_k64<FN, KA, KB>(As[1], Bs[1], wm, wn, lane, acc);
    rowsum_step(As[1]);
    if (kt + 2 < ktiles) {
      stage_a(la0, As[0]);
      lb0.store(adB, Bs[0]);
    }
    __syncthreads();
  }
  if (kt < ktiles) {
    mma_big_k64<FN, KA, KB>(As[0], Bs[0], wm, wn, lane, acc);
    rowsum_step(As[0]);
    __syncthreads();
  }
  if (rs_on) {
    if constexpr (KA) {
      rs = BufMNK<BBM, THREADS>::rowsum_combine(rsv, reinterpret_cast<float*>(gemm_smem));
      const int row = m0 + threadIdx.x;
      if (threadIdx.x < BBM && row < M) rowsum[row] = rs;
    } else {
      if (TPR == 2) rs += __shfl_xor(rs, 1, 64);  // the two halves of the row, fixed order
      const int row = m0 + threadIdx.x / TPR;
      if (threadIdx.x % TPR == 0 && row < M) rowsum[row] = rs;
    }
  }

  // epilogue in two halves of 128 rows: the waves of row half h stage their
  // fp32 fragments, then all threads write the half's rows, 8 columns each
  float* Cs = reinterpret_cast<float*>(gemm_smem);
#pragma unroll 1
  for (int h = 0; h < 2; ++h) {
    if (wm == h) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int cl = wn * FN * 32 + j * 32 + (lane & 31);
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int rl = i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            Cs[rl * BCLD + cl] = acc[i][j][r];
          }
        }
    }
    __syncthreads();
    if constexpr (NORM != 0) {
      // two 128-column norm groups per tile row: lanes 0-15 and 16-31 of
      // each 32-lane row; a thread keeps its 8 columns in every row
      const int cl = (threadIdx.x % (BBN / 8)) * 8;
      NormCoef nc;
      load_norm_coef(epi, n0 + cl, N, nc);
#pragma unroll 4
      for (int q = 0; q < (BBM / 2) * BBN / 8 / THREADS; ++q) {
        const int rl = (threadIdx.x + q * THREADS) / (BBN / 8);
        float v[8];
        ld8f(Cs + rl * BCLD + cl, v);
        epi_blocknorm8<CT, NORM>(C, ldc, m0 + h * 128 + rl, n0 + cl, M, N, v, epi, nc, vec);
      }
      __syncthreads();
      continue;
    }
#pragma unroll 4
    for (int q = 0; q < (BBM / 2) * BBN / 8 / THREADS; ++q) {
      const int chunk = threadIdx.x + q * THREADS;
      const int rl = chunk / (BBN / 8), cl = (chunk % (BBN / 8)) * 8;
      const int row = m0 + h * 128 + rl, col = n0 + cl;
      if (row >= M || col >= N) continue;
      float v[8];
      ld8f(Cs + rl * BCLD + cl, v);
      if (vec && col + 8 <= N) {
        epi_store8<CT>(C, ldc, row, col, v, epi, 0);
      } else {
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (col + t < N) epi_store<CT>(C, ldc, row, col + t, v[t], epi, 0);
      }
    }
    __syncthreads();
  }
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

// Split-K factor by an estimated time: ceil(blocks / 512) waves (two blocks
// per CU) of K / s each, in K steps, plus the fp32 partials each split writes
// and the reduction reads back, M * N / 375000 K steps per split (fitted to
// the step's weight-gradient products at K = 8192: the 512 x 1024 product
// takes 26 us at 8 splits and 32 us at 16), so any factor (not only powers
// of two) that balances the waves is considered; ties keep fewer splits.
int gemm_splits(const GemmArgs& g) {
  if (g.dt != DT_BF16 || g.batch > 1 || g.max_splits <= 1) return 1;
  const int64_t tiles = (int64_t)cdiv(g.M, GBM) * cdiv(g.N, GBN);
  double best = 0.0;
  int best_s = 1;
  for (int s = 1; s <= g.max_splits; ++s) {
    const int64_t kps = ((int64_t)cdiv(g.K, s) + GBK - 1) / GBK * GBK;
    if (s > 1 && kps < 4 * GBK) break;          // at least four K steps per split
    if ((int64_t)(s - 1) * kps >= g.K) continue;  // the last split would be empty
    const double waves = (double)cdiv(tiles * s, (int64_t)512);
    const double cost = waves * (double)(kps / GBK) +
                        (s > 1 ? (double)s * g.M * g.N / 3.75e5 : 0.0);
    if (s == 1 || cost < 0.98 * best) {
      best = cost;
      best_s = s;
    }
  }
  return best_s;
}

// split-K partial tiles [splits][M][N], then the row-sum partials [splits][M]
size_t gemm_workspace(const GemmArgs& g) {
  int splits = gemm_splits(g);
  return splits > 1 ? (size_t)splits * ((size_t)g.M * g.N + g.M) * sizeof(float) : 0;
}

static Epi make_epi(const GemmArgs& g) {
  return Epi{g.bias,   g.relu,     g.mask, g.mask_dt, g.ldm,  g.s_mask, g.addend,
             g.ld_add, g.s_add,    g.accumulate,      g.gain, g.eps,    g.pre,
             g.ldp,    g.rinv,     g.nblk};
}

static bool a16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// 16-byte epilogue vectors: every row of C and of the epilogue operands
// (bias, addend, mask) starts 16-byte aligned.
static int epi_vec_ok(const GemmArgs& g) {
  const int64_t ce = g.c_dt == DT_BF16 ? 8 : 4;
  if (!a16(g.C) || g.ldc % ce || g.sC % ce) return 0;
  if (g.accumulate && (g.ldc % 4)) return 0;
  if (g.bias && !a16(g.bias)) return 0;
  if (g.addend && (!a16(g.addend) || g.ld_add % 4 || g.s_add % 4)) return 0;
  if (g.mask) {
    const int64_t me = g.mask_dt == DT_BF16 ? 8 : 4;
    if (!a16(g.mask) || g.ldm % me || g.s_mask % me) return 0;
  }
  if (g.norm_gate && (!a16(g.pre) || g.ldp % ce)) return 0;
  return 1;
}

// The 256x256 kernel takes products with vector loaders (and no batching)
// when its estimated time is lower.  In units of one CU doing a 128x128xK
// tile alone at the small kernel's rate: the small kernel runs waves of 512
// tiles (two blocks per CU, K / splits each), 2K / splits per wave; the large
// kernel runs waves of 256 tiles (one per CU, no split) of four times the
// work at about 1.3x the rate, 3.08K per wave.
static bool gemm_use_big(const GemmArgs& g) {
  if (g.batch > 1 || g.ngroups > 0) return false;
  const int64_t s = gemm_splits(g);
  const int64_t big_waves = cdiv((int64_t)cdiv(g.M, BBM) * cdiv(g.N, BBN), 256);
  const int64_t small_waves = cdiv((int64_t)cdiv(g.M, GBM) * cdiv(g.N, GBN) * s, 512);
  return 308 * big_waves * s < 200 * small_waves;
}

// Bytes from an operand's first element to the end of its last one (one
// batch): R rows (or columns) of K, K-contiguous (rows of ld) or not.
static int64_t operand_span(int64_t ld, int R, int K, bool mn) {
  if (R <= 0 || K <= 0) return 0;
  return mn ? ((int64_t)(K - 1) * ld + (R + 7) / 8 * 8) * 2 : ((int64_t)(R - 1) * ld + (K + 7) / 8 * 8) * 2;
}
// Buffer loaders: no K segmentation and both operands within 2 GiB,
// counting the 64 k rows a last K step may address past the range (their
// byte offsets must stay below 2^32, out of the resource's range, so that
// they read zero rather than wrap back into it).
static bool gemm_use_buf(const GemmArgs& g) {
  const int64_t lim = (int64_t)1 << 31;
  auto reach = [](int64_t ld, int R, int K, bool mn) { return operand_span(ld, R, K, mn) + (mn ? 64 * ld * 2 : 128); };
  return g.kseg == 0 && reach(g.lda, g.M, g.K, g.ta) < lim && reach(g.ldb, g.N, g.K, g.tb) < lim;
}

template <bool TA, bool TB, int NORM>
static hipError_t gemm_big_launch(const GemmArgs& g, hipStream_t st) {
  // 8 waves of 128 x 64 (two per SIMD) where both operands load without the
  // register transpose or one is staged k-major: 3% faster than 4 waves of
  // 128 x 128 on the deep stack's projection products; with both operands
  // M-contiguous the 8-wave kernel spills (51 VGPRs) and 4 waves stay
  constexpr int NW = (TA && TB) ? 4 : 8;
  Epi epi = make_epi(g);
  Opnd a{(const bf16_t*)g.A, g.lda, g.kseg, g.ksA};
  Opnd b{(const bf16_t*)g.B, g.ldb, g.kseg, g.ksB};
  const int vec = epi_vec_ok(g);
  const dim3 grid(cdiv(g.N, BBN) * cdiv(g.M, BBM));
  static std::once_flag once[2][2];
  auto launch = [&](auto kern, auto* c, std::once_flag& of) {
    std::call_once(of, [&] {
      (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)GEMM_BIG_LDS);
    });
    kern<<<grid, NW * 64, GEMM_BIG_LDS, st>>>(a, b, c, g.ldc, g.M, g.N, g.K, epi, vec, g.rowsum);
  };
  const bool buf = gemm_use_buf(g);
  if (g.c_dt == DT_BF16) {
    if (buf) launch(gemm_big_kernel<TA, TB, bf16_t, NW, NORM, true>, (bf16_t*)g.C, once[0][1]);
    else launch(gemm_big_kernel<TA, TB, bf16_t, NW, NORM, false>, (bf16_t*)g.C, once[0][0]);
  } else {
    if (buf) launch(gemm_big_kernel<TA, TB, float, NW, NORM, true>, (float*)g.C, once[1][1]);
    else launch(gemm_big_kernel<TA, TB, float, NW, NORM, false>, (float*)g.C, once[1][0]);
  }
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

template <bool TA, bool TB, bool VA, bool VB, int NORM>
static hipError_t gemm_bf16_launch(const GemmArgs& g, float* ws, hipStream_t st) {
  if constexpr (VA && VB) {
    if (gemm_use_big(g)) return gemm_big_launch<TA, TB, NORM>(g, st);
  }
  constexpr bool can_buf = VA && VB;
  const bool buf = can_buf && gemm_use_buf(g);
  const int splits = gemm_splits(g);
  if (splits > 1 && !ws) {
    set_error("split-K GEMM without a workspace");
    return hipErrorInvalidValue;
  }
  int kps = (g.K + splits - 1) / splits;
  kps = ((kps + GBK - 1) / GBK) * GBK;
  const int batched = g.batch > 1 ? 1 : 0;
  GroupSpec grp{};
  int grid_m = g.M;
  if (g.ngroups > 0) {
    grp.n = g.ngroups;
    grp.gk = g.gk;
    grp.sB = g.gsB;
    grp.sC = g.gsC;
    int maxrows = 0;
    for (int i = 0; i <= g.ngroups; ++i) grp.off[i] = (int)g.goff[i];
    for (int i = 0; i < g.ngroups; ++i) maxrows = std::max(maxrows, grp.off[i + 1] - grp.off[i]);
    if (!g.gk) grid_m = std::max(maxrows, 1);
  }
  dim3 grid(cdiv(g.N, GBN) * cdiv(grid_m, GBM), 1, g.ngroups > 0 ? g.ngroups : (batched ? g.batch : splits));
  Epi epi = make_epi(g);
  Opnd a{(const bf16_t*)g.A, g.lda, g.kseg, g.ksA};
  Opnd b{(const bf16_t*)g.B, g.ldb, g.kseg, g.ksB};
  float* partial = splits > 1 ? ws : nullptr;
  float* rs_partial = (splits > 1 && g.rowsum) ? ws + (size_t)splits * g.M * g.N : nullptr;
  const int vec = epi_vec_ok(g);
  // The kernels use 72 KiB of dynamic LDS (above the 64 KiB default limit).
  static std::once_flag once[2][2];
  auto launch = [&](auto kern, auto* c, std::once_flag& of) {
    std::call_once(of, [&] {
      (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)GEMM_LDS);
    });
    kern<<<grid, 256, GEMM_LDS, st>>>(a, b, c, g.ldc, g.M, g.N, g.K, kps, partial, epi, g.sA, g.sB, g.sC,
                                      batched, vec, g.rowsum, rs_partial, grp);
  };
  if (g.c_dt == DT_BF16) {
    if (buf) launch(gemm_bf16_kernel<TA, TB, VA, VB, bf16_t, NORM, can_buf>, (bf16_t*)g.C, once[0][1]);
    else launch(gemm_bf16_kernel<TA, TB, VA, VB, bf16_t, NORM, false>, (bf16_t*)g.C, once[0][0]);
  } else {
    if (buf) launch(gemm_bf16_kernel<TA, TB, VA, VB, float, NORM, can_buf>, (float*)g.C, once[1][1]);
    else launch(gemm_bf16_kernel<TA, TB, VA, VB, float, NORM, false>, (float*)g.C, once[1][0]);
  }
  LAT_LAUNCH_CHECK();
  if (splits > 1) {
    const int64_t n = (int64_t)g.M * g.N;
    if (g.c_dt == DT_BF16)
      splitk_reduce_kernel<bf16_t><<<cdiv(n, 256), 256, 0, st>>>(ws, splits, g.M, g.N, (bf16_t*)g.C,
                                                                  g.ldc, epi, rs_partial, g.rowsum);
    else
      splitk_reduce_kernel<float><<<cdiv(n, 256), 256, 0, st>>>(ws, splits, g.M, g.N, (float*)g.C,
                                                                 g.ldc, epi, rs_partial, g.rowsum);
    LAT_LAUNCH_CHECK();
  }
  return hipSuccess;
}

template <bool TA, bool TB, int NORM = 0>
static hipError_t gemm_bf16_dispatch(const GemmArgs& g, float* ws, hipStream_t st) {
  // 16-byte vectors (along K, or along M/N for a transposed operand) need
  // 8-element-aligned rows, segments and batch strides.
  // A length not a multiple of 8 is fine when the rows are padded to one: the
  // last vector then stays inside its row (the K-contiguous loader zeroes the
  // elements past K; rows past M or N only feed discarded outputs).
  const bool seg_ok = g.kseg == 0 || (g.kseg % 8 == 0 && g.ksA % 8 == 0 && g.ksB % 8 == 0);
  auto fits = [&](int len, int64_t ld) { return len % 8 == 0 || (g.kseg == 0 && ld >= (len + 7) / 8 * 8); };
  const bool va = TA ? (g.lda % 8 == 0 && aligned16(g.A) && fits(g.M, g.lda) && g.sA % 8 == 0 &&
                        (g.kseg == 0 || g.ksA % 8 == 0))
                     : (g.lda % 8 == 0 && aligned16(g.A) && fits(g.K, g.lda) && g.sA % 8 == 0 && seg_ok);
  const bool vb = TB ? (g.ldb % 8 == 0 && aligned16(g.B) && fits(g.N, g.ldb) && g.sB % 8 == 0 &&
                        (g.kseg == 0 || g.ksB % 8 == 0))
                     : (g.ldb % 8 == 0 && aligned16(g.B) && fits(g.K, g.ldb) && g.sB % 8 == 0 && seg_ok);
  if (va && vb) return gemm_bf16_launch<TA, TB, true, true, NORM>(g, ws, st);
  if (va) return gemm_bf16_launch<TA, TB, true, false, NORM>(g, ws, st);
  if (vb) return gemm_bf16_launch<TA, TB, false, true, NORM>(g, ws, st);
  return gemm_bf16_launch<TA, TB, false, false, NORM>(g, ws, st);
}

hipError_t gemm(const GemmArgs& g0, void* ws, hipStream_t st) {
  GemmArgs g = g0;
  if (g.M == 0 || g.N == 0 || g.batch == 0) return hipSuccess;
  if (g.ngroups > 0) {
    if (g.dt != DT_BF16 || g.batch > 1 || g.kseg || g.ngroups > GEMM_MAX_GROUPS || !g.goff ||
        g.goff[0] != 0 || g.goff[g.ngroups] != (g.gk ? g.K : g.M)) {
      set_error("grouped GEMM: bf16, not batched, at most %d groups covering %s", GEMM_MAX_GROUPS,
                g.gk ? "K" : "M");
      return hipErrorInvalidValue;
    }
    g.max_splits = 1;  // each group's K range or rows in one pass
  }
  if (g.accumulate && g.c_dt != DT_F32) {
    set_error("accumulating GEMM needs an fp32 output");
    return hipErrorInvalidValue;
  }
  if (g.rowsum && (g.dt != DT_BF16 || g.batch > 1)) {
    set_error("GEMM row sums: bf16 and not batched only");
    return hipErrorInvalidValue;
  }
  if (g.norm_gate) {
    // the BlockNorm epilogue: forward products (A and B K-contiguous), one
    // product, K not split, pre-activation and statistics stored
    if (g.dt != DT_BF16 || g.ta || g.tb || g.batch > 1 || g.kseg || g.max_splits > 1 || g.mask ||
        g.addend || g.accumulate || g.relu || g.rowsum || !g.gain || !g.pre || !g.rinv ||
        g.nblk != cdiv(g.N, NORM_TILE) ||
        (g.norm_gate != GATE_SIGMOID && g.norm_gate != GATE_HARD)) {
      set_error("BlockNorm GEMM epilogue: unsupported arguments");
      return hipErrorInvalidValue;
    }
    if (g.norm_gate == GATE_SIGMOID) return gemm_bf16_dispatch<false, false, GATE_SIGMOID>(g, (float*)ws, st);
    return gemm_bf16_dispatch<false, false, GATE_HARD>(g, (float*)ws, st);
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
