// Per-sample MFMA building blocks shared by the interaction kernels: 32x32
// output tiles of v_mfma_f32_32x32x16_bf16 over operands staged in LDS with
// the contraction dimension contiguous, and a register-staged loader that
// writes a sample's [rows][cols] bf16 matrix to LDS row-major and/or
// transposed.
#pragma once
#include "common.h"

namespace lat {

// acc += A[32 rows][K] * B[32 rows][K]^T, operands in LDS with k contiguous.
// D element r of a lane is row 8*(r/4) + 4*(lane/32) + r%4, column lane%32.
template <int K>
__device__ inline void mfma_tile(f32x16& acc, const bf16_t* A, int lda, const bf16_t* B, int ldb) {
  const int lane = threadIdx.x & 63;
  const bf16_t* a = A + (lane & 31) * lda + (lane >> 5) * 8;
  const bf16_t* b = B + (lane & 31) * ldb + (lane >> 5) * 8;
#pragma unroll
  for (int k = 0; k < K; k += 16) {
    const bf16x8 av = *reinterpret_cast<const bf16x8*>(a + k);
    const bf16x8 bv = *reinterpret_cast<const bf16x8*>(b + k);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
  }
}

// acc += A[32 rows from rbase][K] * B[32 rows][K]^T with A stored k-major in
// LDS (Akm[k * ldk + r], r contiguous), read with the transposed LDS read
// ds_read_b64_tr_b16: within each 16-lane group it returns to lane j, as its
// element e, element j % 4 of the 8-byte piece addressed by lane 4e + j / 4,
// so lane 4e + q addresses rows rbase + 16 (g % 2) + 4q .. +3 of k row
// 8 (g / 2) + e (g = lane / 16) and lane j receives row rbase + lane % 32 at
// four consecutive k; two reads make the 8-k fragment.  ldk and rbase must
// be multiples of 4 (8-byte aligned pieces).
typedef short i16x4_t __attribute__((ext_vector_type(4)));
template <int K>
__device__ inline void mfma_tile_kmA(f32x16& acc, const bf16_t* Akm, int ldk, int rbase, const bf16_t* B,
                                     int ldb) {
  typedef __attribute__((address_space(3))) i16x4_t lds_v4;
  const int lane = threadIdx.x & 63, g = lane >> 4, j = lane & 15;
  const bf16_t* a = Akm + (8 * (g >> 1) + (j >> 2)) * ldk + rbase + 16 * (g & 1) + 4 * (j & 3);
  const bf16_t* b = B + (lane & 31) * ldb + (lane >> 5) * 8;
#pragma unroll
  for (int k = 0; k < K; k += 16) {
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(a + k * ldk));
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(a + (k + 4) * ldk));
    const bf16x8 av = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    const bf16x8 bv = *reinterpret_cast<const bf16x8*>(b + k);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
  }
}

__device__ inline void zero16(f32x16& a) {
#pragma unroll
  for (int r = 0; r < 16; ++r) a[r] = 0.f;
}

__device__ inline int frag_row(int r) { return 8 * (r >> 2) + 4 * ((threadIdx.x & 63) >> 5) + (r & 3); }

// Stage a [rows][cols] bf16 matrix (row stride gld, rows >= nrows read as 0)
// into LDS twice: R[j][c] (stride ldr) and T[c][j] (stride ldt).  Items are
// (group of 8 rows, pair of columns); RP = padded row count (multiple of 8).
// load() fetches this thread's items into registers (so the next sample can
// be in flight while the current one is computed), store() writes them.
// load() is straight-line code: rows past nrows and items past the last
// read a valid element (nrows >= 1) and store() writes zeros for them.  A
// load inside a branch, or whose value is selected at once, makes the
// compiler wait for it (and for every load issued before it) right there,
// which would serialise the prefetch with the compute.
template <int RP, int COLS, int THREADS>
struct Stager {
  static constexpr int ITEMS = (RP / 8) * (COLS / 2);
  static constexpr int PER = (ITEMS + THREADS - 1) / THREADS;
  uint32_t v[PER][8];
  __device__ inline void load(const bf16_t* __restrict__ g, int64_t gld, int nrows) {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      int it = threadIdx.x + q * THREADS;
      it = it < ITEMS ? it : ITEMS - 1;
      const int j0 = (it / (COLS / 2)) * 8, c = (it % (COLS / 2)) * 2;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int row = j0 + i < nrows ? j0 + i : 0;
        v[q][i] = *reinterpret_cast<const uint32_t*>(g + (int64_t)row * gld + c);
      }
    }
  }
  // R or T may be null (that layout is not written); nrows as in load()
  __device__ inline void store(bf16_t* R, int ldr, bf16_t* T, int ldt, int nrows) const {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int it = threadIdx.x + q * THREADS;
      if (it < ITEMS) {
        const int j0 = (it / (COLS / 2)) * 8, c = (it % (COLS / 2)) * 2;
        uint32_t x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = j0 + i < nrows ? v[q][i] : 0u;
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

}  // namespace lat
