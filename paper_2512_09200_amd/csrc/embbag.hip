// Pooled embedding lookup over jagged multi-hot bags (Section 3.3.1) and its
// deterministic row-coalesced gradient with an optional fused row-sparse SGD
// update.
//
// Forward: one wavefront per bag.  A table row is split into 16-byte lane
// chunks (a 256-byte bf16 row of d=128 is 16 lanes); the wave's 64 lanes form
// G = 64/LP groups that each take every G-th entry of the bag, and every group
// issues U row loads before using any of them, so each wave keeps G*U rows in
// flight.  The groups' fp32 partial sums are combined with a fixed butterfly
// (deterministic), and the first group writes the pooled row.
//
// Backward (no floating-point atomics):
//   keys     : key = row_base[f] + index, value = bag id, per position
//   sort     : stable LSD radix sort by key (ties keep position order)
//   segments : run boundaries -> unique rows ascending, run offsets, and the
//              segment id at each chunk start
//   chunks   : the sorted occurrences are cut into fixed chunks of 64; one
//              block per chunk gathers its 64 dX rows into LDS (all loads in
//              flight at once), then each thread walks one column in order.
//              Runs that end inside the chunk are final (written to G and/or
//              applied as SGD); runs cut by a chunk boundary leave a partial
//   fixup    : each run that spans chunks sums its partials in chunk order
// Work per block is uniform whatever the Zipf skew of the rows.
#include "common.h"
#include "kernels.h"

namespace lat {

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <typename TT, typename XT, int LP>
__global__ __launch_bounds__(256) void embbag_fwd_kernel(
    const TT* __restrict__ E, const int64_t* __restrict__ row_base,
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ indices, int F, int B,
    int dim, int mean, XT* __restrict__ X, int n_slots, int first_slot, int* __restrict__ keys,
    int* __restrict__ vals) {
  constexpr int VE = 16 / sizeof(TT);  // table elements per 16-byte lane chunk
  constexpr int G = 64 / LP;           // row groups per wave
  constexpr int U = (16 / G) > 0 ? (16 / G) : 1;  // loads in flight per group
  const int lane = threadIdx.x & 63;
  const int64_t bag = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (bag >= (int64_t)F * B) return;
  const int f = (int)(bag / B), b = (int)(bag % B);
  const int g = lane / LP, sub = lane % LP;
  const bool active = sub * VE < dim;
  const int start = offsets[bag], end = offsets[bag + 1];
  const TT* Ef = E + row_base[f] * (int64_t)dim + sub * VE;

  if (keys) {  // sort keys of the backward (global row) and values (bag id), coalesced
    const int rb = (int)row_base[f];
    for (int q = start + lane; q < end; q += 64) {
      keys[q] = rb + indices[q];
      vals[q] = (int)bag;
    }
  }
  float acc[VE];
#pragma unroll
  for (int i = 0; i < VE; ++i) acc[i] = 0.f;

  for (int p = start + g; p < end; p += G * U) {
    int idx[U];
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int q = p + u * G;
      idx[u] = (q < end) ? indices[q] : -1;
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (idx[u] >= 0 && active) v[u] = ldg16(Ef + (int64_t)idx[u] * dim);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (idx[u] >= 0 && active) {
        float t[VE];
        Vec16<TT>::unpack(v[u], t);
#pragma unroll
        for (int i = 0; i < VE; ++i) acc[i] += t[i];
      }
    }
  }
#pragma unroll
  for (int o = LP; o < 64; o <<= 1) {
#pragma unroll
    for (int i = 0; i < VE; ++i) acc[i] += __shfl_xor(acc[i], o, 64);
  }
  if (g == 0 && active) {
    if (mean && end > start) {
      const float len = (float)(end - start);
#pragma unroll
      for (int i = 0; i < VE; ++i) acc[i] = acc[i] / len;
    }
    XT* out = X + ((int64_t)b * n_slots + first_slot + f) * dim + sub * VE;
    if constexpr (sizeof(XT) == sizeof(TT)) {
      stg16(out, Vec16<XT>::pack(acc));
    } else {
#pragma unroll
      for (int i = 0; i < VE; ++i) st(out + i, acc[i]);
    }
  }
}

template <typename TT, typename XT>
static hipError_t embbag_fwd_t(const void* E, int dim, const int64_t* row_base,
                               const int32_t* offsets, const int32_t* indices, int F, int B,
                               int mean, void* X, int n_slots, int first_slot, int* keys,
                               int* vals, hipStream_t s) {
  const int64_t bags = (int64_t)F * B;
  if (bags == 0) return hipSuccess;
  const int lanes = (int)((dim * sizeof(TT) + 15) / 16);
  const int grid = cdiv(bags, 4);
#define LAT_FWD(LPV)                                                                       \
  embbag_fwd_kernel<TT, XT, LPV><<<grid, 256, 0, s>>>(                                    \
      (const TT*)E, row_base, offsets, indices, F, B, dim, mean, (XT*)X, n_slots, first_slot, keys, vals)
  if (lanes <= 1) LAT_FWD(1);
  else if (lanes <= 2) LAT_FWD(2);
  else if (lanes <= 4) LAT_FWD(4);
  else if (lanes <= 8) LAT_FWD(8);
  else if (lanes <= 16) LAT_FWD(16);
  else if (lanes <= 32) LAT_FWD(32);
  else LAT_FWD(64);
#undef LAT_FWD
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t embbag_fwd(const void* E, DType edt, int dim, const int64_t* row_base,
                      const int32_t* offsets, const int32_t* indices, int F, int B, int mean,
                      void* X, DType xdt, int n_slots, int first_slot, hipStream_t s, int* keys,
                      int* vals) {
  if (edt == DT_BF16 && xdt == DT_BF16)
    return embbag_fwd_t<bf16_t, bf16_t>(E, dim, row_base, offsets, indices, F, B, mean, X, n_slots, first_slot, keys, vals, s);
  if (edt == DT_BF16 && xdt == DT_F32)
    return embbag_fwd_t<bf16_t, float>(E, dim, row_base, offsets, indices, F, B, mean, X, n_slots, first_slot, keys, vals, s);
  if (edt == DT_F32 && xdt == DT_F32)
    return embbag_fwd_t<float, float>(E, dim, row_base, offsets, indices, F, B, mean, X, n_slots, first_slot, keys, vals, s);
  return embbag_fwd_t<float, bf16_t>(E, dim, row_base, offsets, indices, F, B, mean, X, n_slots, first_slot, keys, vals, s);
}

// ---------------------------------------------------------------------------
// backward: keys
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void embbag_keys_kernel(const int64_t* __restrict__ row_base,
                                                          const int32_t* __restrict__ offsets,
                                                          const int32_t* __restrict__ indices,
                                                          int F, int B, int* __restrict__ keys,
                                                          int* __restrict__ vals) {
  const int lane = threadIdx.x & 63;
  const int64_t bag = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (bag >= (int64_t)F * B) return;
  const int f = (int)(bag / B);
  const int start = offsets[bag], end = offsets[bag + 1];
  const int rb = (int)row_base[f];
  for (int p = start + lane; p < end; p += 64) {
    keys[p] = rb + indices[p];
    vals[p] = (int)bag;
  }
}

// ---------------------------------------------------------------------------
// backward: segment bookkeeping over sorted keys
// ---------------------------------------------------------------------------
constexpr int SEG_THREADS = 256;
constexpr int SEG_ITEMS = 16;
constexpr int SEG_TILE = SEG_THREADS * SEG_ITEMS;
constexpr int CHUNK = 64;  // occurrences per reduction chunk

__device__ inline int seg_flag(const int* k, int64_t i) { return (i == 0 || k[i] != k[i - 1]) ? 1 : 0; }

__device__ inline int block_sum_scan(int v, int* lds, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds[w] = x;
  __syncthreads();
  int wb = 0, tot = 0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) {
    if (i < w) wb += lds[i];
    tot += lds[i];
  }
  __syncthreads();
  *total = tot;
  return wb + x - v;
}

__global__ __launch_bounds__(SEG_THREADS) void seg_count_kernel(const int* __restrict__ keys, int n,
                                                                int* __restrict__ tile_counts) {
  __shared__ int lds[SEG_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * SEG_TILE;
  int c = 0;
#pragma unroll
  for (int i = 0; i < SEG_ITEMS; ++i) {
    int64_t k = base + (int64_t)i * SEG_THREADS + threadIdx.x;
    if (k < n) c += seg_flag(keys, k);
  }
  int tot;
  block_sum_scan(c, lds, &tot);
  if (threadIdx.x == 0) tile_counts[blockIdx.x] = tot;
}

__global__ __launch_bounds__(SEG_THREADS) void seg_write_kernel(
    const int* __restrict__ keys, int n, const int* __restrict__ tile_base,
    int* __restrict__ unique_rows, int* __restrict__ seg_offsets, int* __restrict__ num_unique,
    int* __restrict__ chunk_uid) {
  __shared__ int lds[SEG_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * SEG_TILE + (int64_t)threadIdx.x * SEG_ITEMS;
  int fl[SEG_ITEMS];
  int c = 0;
#pragma unroll
  for (int i = 0; i < SEG_ITEMS; ++i) {
    fl[i] = (base + i < n) ? seg_flag(keys, base + i) : 0;
    c += fl[i];
  }
  int tot;
  int run = block_sum_scan(c, lds, &tot) + tile_base[blockIdx.x];
#pragma unroll
  for (int i = 0; i < SEG_ITEMS; ++i) {
    const int64_t k = base + i;
    if (k < n) {
      run += fl[i];
      const int u = run - 1;  // segment id of position k
      if (fl[i]) {
        unique_rows[u] = keys[k];
        seg_offsets[u] = (int)k;
      }
      if (k % CHUNK == 0) chunk_uid[k / CHUNK] = u;
      if (k == n - 1) {
        num_unique[0] = u + 1;
        seg_offsets[u + 1] = n;
      }
    }
  }
}

__global__ void set_empty_kernel(int* num_unique, int* seg_offsets) {
  num_unique[0] = 0;
  seg_offsets[0] = 0;
}

// ---------------------------------------------------------------------------
// backward: chunked segmented reduction (+ fused SGD)
// ---------------------------------------------------------------------------
template <typename ET>
__device__ inline void finalize_row(int u, int row, float g, int a, int dim, float* grad_rows,
                                    ET* E, float lr) {
  if (grad_rows) grad_rows[(int64_t)u * dim + a] = g;
  if (E) {
    ET* e = E + (int64_t)row * dim + a;
    st(e, ld(e) - lr * g);
  }
}

// One block per chunk of CHUNK consecutive sorted occurrences.
//  1. wave 0: keys and bags of the chunk; run boundaries by ballot; the
//     pieces (maximal runs inside the chunk) with their end position, segment
//     id and kind (complete run, or cut by the chunk start / end)
//  2. all threads: gather the chunk's dX rows into LDS (fp32) and, at the same
//     time, load the table rows of the complete runs that the SGD updates
//  3. work items (piece, 8 columns): sum the piece's rows in position order
//     and write the row gradient / apply the SGD / store the partial
template <typename DT, typename ET>
__global__ __launch_bounds__(256) void chunk_reduce_kernel(
    const int* __restrict__ skeys, const int* __restrict__ sbags, int n,
    const DT* __restrict__ dX, int B, int n_slots, int first_slot, int dim,
    const int32_t* __restrict__ offsets, int mean, const int* __restrict__ chunk_uid,
    float* __restrict__ part, int* __restrict__ part_uid, int* __restrict__ span_list,
    int* __restrict__ span_count, float* __restrict__ grad_rows, ET* __restrict__ E, float lr) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  DT* rows = reinterpret_cast<DT*>(smem_raw);  // [CHUNK][dim], the gathered dX rows as stored
  __shared__ int k_s[CHUNK];
  __shared__ int b_s[CHUNK];
  __shared__ float sc_s[CHUNK];
  __shared__ int pend_s[CHUNK];    // end position of piece i
  __shared__ int pkind_s[CHUNK];   // 1: complete run, 2: cut at chunk start (slot 0), 3: cut at end only (slot 1)
  __shared__ int pu_s[CHUNK];      // segment id of piece i
  __shared__ int npieces_s;
  const int c = blockIdx.x;
  const int64_t p0 = (int64_t)c * CHUNK;
  const int cnt = (int)((n - p0) < CHUNK ? (n - p0) : CHUNK);
  const int tid = threadIdx.x;
  if (tid < CHUNK) {
    const int key = tid < cnt ? skeys[p0 + tid] : -1;
    const int prev = p0 > 0 ? skeys[p0 - 1] : -1;
    const int next = (p0 + cnt < n) ? skeys[p0 + cnt] : -1;
    const int key_prev = __shfl_up(key, 1, 64);
    const bool starts = tid < cnt && tid > 0 && key != key_prev;
    const uint64_t smask = __ballot(starts);
    const uint64_t le = (tid == 63) ? ~0ull : ((2ull << tid) - 1);
    const int u = chunk_uid[c] + __popcll(smask & le);
    const int key_next = __shfl_down(key, 1, 64);
    const bool ends = tid < cnt && (tid == cnt - 1 || key_next != key);
    const uint64_t emask = __ballot(ends);
    const bool starts_before = p0 > 0 && prev == __shfl(key, 0, 64);
    const bool touch_start = (smask & le) == 0 && starts_before;
    const bool touch_end = (tid == cnt - 1) && next == key;
    if (tid < cnt) {
      k_s[tid] = key;
      const int bag = sbags[p0 + tid];
      b_s[tid] = bag;
      sc_s[tid] = mean ? 1.f / (float)(offsets[bag + 1] - offsets[bag]) : 1.f;
    }
    if (ends) {
      const int i = __popcll(emask & (le >> 1));  // pieces ending before tid
      pend_s[i] = tid;
      pkind_s[i] = (!touch_start && !touch_end) ? 1 : (touch_start ? 2 : 3);
      pu_s[i] = u;
    }
    if (tid == 0) npieces_s = __popcll(emask);
    if (ends && tid == cnt - 1) {
      part_uid[c] = touch_end ? u : -1;
      if (touch_end && !touch_start) span_list[atomicAdd(span_count, 1)] = c;
    }
  }
  __syncthreads();

  constexpr int VE = 16 / sizeof(DT);
  const int vpr = dim / VE;
  const int total = cnt * vpr;
  const int np = npieces_s;
  const int ipr = dim / 8;          // work items per piece (8 columns each)
  const int items = np * ipr;
  // table rows of this thread's complete pieces: loads in flight with the gather
  constexpr int EV = 8 * sizeof(ET) / 16;  // 16-byte vectors per 8 columns
  u32x4 ev[4][EV];
  if (E) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int it = tid + q * 256;
      if (it < items) {
        const int i = it / ipr, a = (it - i * ipr) * 8;
        if (pkind_s[i] == 1) {
          const ET* e = E + (int64_t)k_s[pend_s[i]] * dim + a;
#pragma unroll
          for (int h = 0; h < EV; ++h) ev[q][h] = ldg16(e + h * (16 / sizeof(ET)));
        }
      }
    }
  }
  for (int v0 = tid; v0 < total; v0 += 256 * 4) {
    u32x4 buf[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int v = v0 + q * 256;
      if (v < total) {
        const int r = v / vpr, col = (v % vpr) * VE;
        const int bag = b_s[r];
        const int f = bag / B, b = bag % B;
        buf[q] = ldg16(dX + ((int64_t)b * n_slots + first_slot + f) * dim + col);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int v = v0 + q * 256;
      if (v < total) {
        const int r = v / vpr, col = (v % vpr) * VE;
        *reinterpret_cast<u32x4*>(rows + r * dim + col) = buf[q];
      }
    }
  }
  __syncthreads();

  // items beyond the first 1024 (dim > 128) load their table rows in place
  for (int base = 0; base < items; base += 1024) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int it = base + tid + q * 256;
      if (it >= items) continue;
      const int i = it / ipr, a = (it - i * ipr) * 8;
      const int pe = pend_s[i], ps = i == 0 ? 0 : pend_s[i - 1] + 1;
      const int kind = pkind_s[i];
      if (base > 0 && E && kind == 1) {
        const ET* e = E + (int64_t)k_s[pe] * dim + a;
#pragma unroll
        for (int h = 0; h < EV; ++h) ev[q][h] = ldg16(e + h * (16 / sizeof(ET)));
      }
      float g[8];
#pragma unroll
      for (int h = 0; h < 8; ++h) g[h] = 0.f;
      for (int p = ps; p <= pe; ++p) {
        float x[8];
#pragma unroll
        for (int h = 0; h < 8; h += VE)
          Vec16<DT>::unpack(*reinterpret_cast<const u32x4*>(rows + p * dim + a + h), x + h);
        const float scl = sc_s[p];
#pragma unroll
        for (int h = 0; h < 8; ++h) g[h] += mean ? x[h] * scl : x[h];
      }
      if (kind == 1) {
        if (grad_rows) {
          float* gr = grad_rows + (int64_t)pu_s[i] * dim + a;
          stg16(gr, u32x4{__float_as_uint(g[0]), __float_as_uint(g[1]), __float_as_uint(g[2]), __float_as_uint(g[3])});
          stg16(gr + 4, u32x4{__float_as_uint(g[4]), __float_as_uint(g[5]), __float_as_uint(g[6]), __float_as_uint(g[7])});
        }
        if (E) {
          constexpr int PV = 16 / sizeof(ET);
          ET* e = E + (int64_t)k_s[pe] * dim + a;
#pragma unroll
          for (int h = 0; h < EV; ++h) {
            float x[PV];
            Vec16<ET>::unpack(ev[q][h], x);
#pragma unroll
            for (int t = 0; t < PV; ++t) x[t] = x[t] - lr * g[h * PV + t];
            stg16(e + h * PV, Vec16<ET>::pack(x));
          }
        }
      } else {
        float* pp = part + ((int64_t)c * 2 + (kind - 2)) * dim + a;
        stg16(pp, u32x4{__float_as_uint(g[0]), __float_as_uint(g[1]), __float_as_uint(g[2]), __float_as_uint(g[3])});
        stg16(pp + 4, u32x4{__float_as_uint(g[4]), __float_as_uint(g[5]), __float_as_uint(g[6]), __float_as_uint(g[7])});
      }
    }
  }
}

// One wave per spanning run (persistent grid of 4-wave blocks): the run's
// partials are summed in chunk order; lane l owns columns 2l, 2l+1.
template <typename ET>
__global__ __launch_bounds__(256) void chunk_fixup_kernel(
    const int* __restrict__ span_list, const int* __restrict__ span_count,
    const int* __restrict__ part_uid, const int* __restrict__ seg_offsets,
    const int* __restrict__ unique_rows, const float* __restrict__ part, int dim,
    float* __restrict__ grad_rows, ET* __restrict__ E, float lr) {
  const int nspan = *span_count;
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6), nwaves = gridDim.x * 4;
  for (int i = wave; i < nspan; i += nwaves) {
    const int c0 = span_list[i];
    const int u = part_uid[c0];
    const int end = seg_offsets[u + 1];
    const int ce = (end - 1) / CHUNK;
    const int Q = ce - c0 + 1;  // pieces: slot 1 of c0, slot 0 of c0+1..ce
    for (int a = 2 * lane; a < dim; a += 128) {
      float s0 = 0.f, s1 = 0.f;
      int q = 0;
      for (; q + 8 <= Q; q += 8) {
        float2 v[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int qq = q + t;
          const int64_t slot = (qq == 0) ? ((int64_t)c0 * 2 + 1) : ((int64_t)(c0 + qq) * 2);
          v[t] = *reinterpret_cast<const float2*>(part + slot * dim + a);
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) { s0 += v[t].x; s1 += v[t].y; }
      }
      for (; q < Q; ++q) {
        const int64_t slot = (q == 0) ? ((int64_t)c0 * 2 + 1) : ((int64_t)(c0 + q) * 2);
        const float2 v = *reinterpret_cast<const float2*>(part + slot * dim + a);
        s0 += v.x;
        s1 += v.y;
      }
      const int row = unique_rows[u];
      finalize_row<ET>(u, row, s0, a, dim, grad_rows, E, lr);
      finalize_row<ET>(u, row, s1, a + 1, dim, grad_rows, E, lr);
    }
  }
}

__global__ void zero_int_kernel(int* p, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t embbag_bwd_workspace(int64_t nnz, int dim) {
  const int64_t n = nnz > 0 ? nnz : 1;
  const int64_t chunks = cdiv(n, CHUNK);
  size_t s = 0;
  s += 2 * align256((size_t)n * 4);                 // keys, vals (unsorted)
  s += align256((size_t)n * 4);                     // sorted keys
  s += align256(radix_sort_workspace(n));
  s += align256((size_t)(cdiv(n, SEG_TILE) + 1) * 4);  // segment tile counts
  s += align256((size_t)chunks * 4);                // chunk_uid
  s += align256((size_t)chunks * 4);                // part_uid
  s += align256((size_t)chunks * 4);                // span_list
  s += align256(4);                                 // span_count
  s += align256((size_t)chunks * 2 * dim * 4);      // partial rows
  return s;
}

template <typename DT, typename ET>
static hipError_t embbag_bwd_reduce(const int* skeys, const int* sbags, int n, const void* dX,
                                    int B, int n_slots, int first_slot, int dim,
                                    const int32_t* offsets, int mean, const int* chunk_uid,
                                    float* part, int* part_uid, int* span_list, int* span_count,
                                    const int* seg_offsets, const int* unique_rows,
                                    float* grad_rows, void* E, float lr, hipStream_t s) {
  const int chunks = cdiv(n, CHUNK);
  zero_int_kernel<<<1, 64, 0, s>>>(span_count, 1);
  LAT_LAUNCH_CHECK();
  const size_t lds = (size_t)CHUNK * dim * sizeof(DT);
  if (lds > 48 * 1024)
    LAT_HIP_CHECK(hipFuncSetAttribute((const void*)chunk_reduce_kernel<DT, ET>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
  chunk_reduce_kernel<DT, ET><<<chunks, 256, lds, s>>>(
      skeys, sbags, n, (const DT*)dX, B, n_slots, first_slot, dim, offsets, mean, chunk_uid,
      part, part_uid, span_list, span_count, grad_rows, (ET*)E, lr);
  LAT_LAUNCH_CHECK();
  const int fix_grid = chunks < 2048 ? chunks : 2048;
  chunk_fixup_kernel<ET><<<fix_grid, 256, 0, s>>>(span_list, span_count, part_uid,
                                                         seg_offsets, unique_rows, part, dim,
                                                         grad_rows, (ET*)E, lr);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t embbag_bwd(const int64_t* row_base, int64_t total_rows, const int32_t* offsets,
                      const int32_t* indices, int F, int B, int64_t nnz, int mean,
                      const void* dX, DType dxt, int n_slots, int first_slot, int dim,
                      int* unique_rows, int* seg_offsets, int* sorted_bags, int* num_unique,
                      float* grad_rows, void* E, DType et, float lr, void* ws, hipStream_t s,
                      const int* keys_in, const int* vals_in) {
  if (nnz == 0) {
    set_empty_kernel<<<1, 1, 0, s>>>(num_unique, seg_offsets);
    LAT_LAUNCH_CHECK();
    return hipSuccess;
  }
  const int n = (int)nnz;
  const int64_t chunks = cdiv(n, CHUNK);
  char* p = static_cast<char*>(ws);
  auto take = [&](size_t bytes) { char* q = p; p += align256(bytes); return q; };
  int* keys = (int*)take((size_t)n * 4);
  int* vals = (int*)take((size_t)n * 4);
  int* skeys = (int*)take((size_t)n * 4);
  void* sort_ws = take(radix_sort_workspace(n));
  int* tile_counts = (int*)take((size_t)(cdiv(n, SEG_TILE) + 1) * 4);
  int* chunk_uid = (int*)take((size_t)chunks * 4);
  int* part_uid = (int*)take((size_t)chunks * 4);
  int* span_list = (int*)take((size_t)chunks * 4);
  int* span_count = (int*)take(4);
  float* part = (float*)take((size_t)chunks * 2 * dim * 4);

  const int64_t bags = (int64_t)F * B;
  if (keys_in && vals_in) {
    keys = const_cast<int*>(keys_in);  // read-only from here on
    vals = const_cast<int*>(vals_in);
  } else {
    embbag_keys_kernel<<<cdiv(bags, 4), 256, 0, s>>>(row_base, offsets, indices, F, B, keys, vals);
    LAT_LAUNCH_CHECK();
  }
  hipError_t e = radix_sort_pairs(keys, vals, n, total_rows - 1, skeys, sorted_bags, sort_ws, s);
  if (e != hipSuccess) return e;
  const int tiles = cdiv(n, SEG_TILE);
  seg_count_kernel<<<tiles, SEG_THREADS, 0, s>>>(skeys, n, tile_counts);
  LAT_LAUNCH_CHECK();
  e = exclusive_scan_inplace_small(tile_counts, tiles, s);
  if (e != hipSuccess) return e;
  seg_write_kernel<<<tiles, SEG_THREADS, 0, s>>>(skeys, n, tile_counts, unique_rows, seg_offsets,
                                                 num_unique, chunk_uid);
  LAT_LAUNCH_CHECK();
  void* Eupd = lr != 0.f ? E : nullptr;
#define LAT_RED(DTT, ETT)                                                                     \
  return embbag_bwd_reduce<DTT, ETT>(skeys, sorted_bags, n, dX, B, n_slots, first_slot, dim,   \
                                     offsets, mean, chunk_uid, part, part_uid, span_list,      \
                                     span_count, seg_offsets, unique_rows, grad_rows, Eupd, lr, s)
  if (dxt == DT_BF16 && et == DT_BF16) LAT_RED(bf16_t, bf16_t);
  if (dxt == DT_BF16 && et == DT_F32) LAT_RED(bf16_t, float);
  if (dxt == DT_F32 && et == DT_BF16) LAT_RED(float, bf16_t);
  LAT_RED(float, float);
#undef LAT_RED
}

// ---------------------------------------------------------------------------
// batch validation
// ---------------------------------------------------------------------------
__global__ void validate_init_kernel(unsigned long long* r) {
  r[0] = ~0ull;
  r[1] = ~0ull;
}

__global__ __launch_bounds__(256) void validate_kernel(const int64_t* __restrict__ row_base,
                                                       const int32_t* __restrict__ offsets,
                                                       const int32_t* __restrict__ indices, int F,
                                                       int B, int64_t nnz,
                                                       unsigned long long* __restrict__ bad) {
  const int64_t bags = (int64_t)F * B;
  const int64_t bag = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (bag == 0 && offsets[0] != 0) atomicMin(&bad[0], 0ull);
  if (bag == 0 && offsets[bags] != nnz) atomicMin(&bad[0], (unsigned long long)bags);
  if (bag >= bags) return;
  const int64_t lo = offsets[bag], hi = offsets[bag + 1];
  if (hi < lo || lo < 0 || hi > nnz) {
    atomicMin(&bad[0], (unsigned long long)(bag + 1));
    return;
  }
  const int f = (int)(bag / B);
  const int64_t rows = row_base[f + 1] - row_base[f];
  for (int64_t j = lo; j < hi; ++j) {
    const int64_t v = indices[j];
    if (v < 0 || v >= rows) {
      atomicMin(&bad[1], (unsigned long long)j);
      break;
    }
  }
}

hipError_t validate_batch(const int64_t* row_base, const int32_t* offsets,
                          const int32_t* indices, int F, int B, int64_t nnz,
                          unsigned long long* dev_result, hipStream_t s) {
  validate_init_kernel<<<1, 1, 0, s>>>(dev_result);
  LAT_LAUNCH_CHECK();
  const int64_t bags = (int64_t)F * B;
  validate_kernel<<<cdiv(bags + 1, 256), 256, 0, s>>>(row_base, offsets, indices, F, B, nnz,
                                                       dev_result);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
