// Pooled embedding lookup over jagged multi-hot bags (Section 3.3.1) and its
// deterministic row-coalesced gradient with an optional fused row-sparse SGD
// update.
//
// Forward: one wavefront per 16 consecutive bags, walking their lookups one
// table row per step (each lane holds a 4..16-byte slice of the row), with
// the rows of 8..32 lookups in flight at once; each bag is summed in position
// order in fp32 and stored when it ends.
//
// Backward (no floating-point atomics):
//   keys     : key = row_base[f] + index, value = bag id, per position
//   sort     : stable LSD radix sort by key (ties keep position order); the
//              positions are grouped by feature, so each feature's segment is
//              sorted by its local row and only the largest table's row bits
//              need digit passes
//   segments : run boundaries -> unique rows ascending, run offsets, and the
//              run id before every 256-position range
//   reduce   : one wave per range of 256 sorted occurrences; dX rows are
//              gathered into registers chunk by chunk and summed by an
//              in-register segmented scan in a fixed order, with the running
//              sum carried from chunk to chunk.  Runs that start and end in
//              the range are final (written to G and/or applied as SGD); a
//              run cut by a range boundary leaves a partial sum
//   fixup    : each run that crosses ranges sums its partials in range order
// Work per wave is uniform whatever the Zipf skew of the rows.
#include "common.h"
#include "kernels.h"

namespace lat {

// N consecutive elements of T held by one lane, as raw 32-bit words.
template <typename T, int N>
struct Frag {
  static constexpr int NB = N * (int)sizeof(T);
  static constexpr int W = NB >= 4 ? NB / 4 : 1;
  uint32_t w[W];
  __device__ inline void load(const T* p) {
    if constexpr (NB == 2) {
      w[0] = *reinterpret_cast<const uint16_t*>(p);
    } else if constexpr (NB == 4) {
      w[0] = *reinterpret_cast<const uint32_t*>(p);
    } else if constexpr (NB == 8) {
      const uint2 v = *reinterpret_cast<const uint2*>(p);
      w[0] = v.x;
      w[1] = v.y;
    } else {
#pragma unroll
      for (int q = 0; q < W / 4; ++q) {
        const u32x4 v = ldg16(reinterpret_cast<const uint32_t*>(p) + 4 * q);
#pragma unroll
        for (int t = 0; t < 4; ++t) w[4 * q + t] = v[t];
      }
    }
  }
  // streaming (non-temporal) access: data touched once, kept out of the caches' way
  __device__ inline void load_nt(const T* p) {
    if constexpr (NB == 4) {
      w[0] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
    } else {
      load(p);
    }
  }
  // element i as fp32
  __device__ inline float get(int i) const {
    if constexpr (sizeof(T) == 2)
      return __uint_as_float((i & 1) ? (w[i >> 1] & 0xffff0000u) : (w[i >> 1] << 16));
    else
      return __uint_as_float(w[i]);
  }
  // stores v[0..N) rounded to T, non-temporal where the width allows
  __device__ static inline void store_nt(T* p, const float* v) {
    if constexpr (NB == 4 && sizeof(T) == 2) {
      __builtin_nontemporal_store(pack_bf2(v[0], v[1]), reinterpret_cast<uint32_t*>(p));
    } else if constexpr (NB == 4) {
      __builtin_nontemporal_store(__float_as_uint(v[0]), reinterpret_cast<uint32_t*>(p));
    } else {
      store(p, v);
    }
  }
  // stores v[0..N) rounded to T
  __device__ static inline void store(T* p, const float* v) {
    uint32_t o[W];
    if constexpr (sizeof(T) == 2) {
      if constexpr (N == 1) {
        *reinterpret_cast<uint16_t*>(p) = f2bf(v[0]);
        return;
      } else {
#pragma unroll
        for (int t = 0; t < W; ++t) o[t] = pack_bf2(v[2 * t], v[2 * t + 1]);
      }
    } else {
#pragma unroll
      for (int t = 0; t < W; ++t) o[t] = __float_as_uint(v[t]);
    }
    if constexpr (NB == 4) {
      *reinterpret_cast<uint32_t*>(p) = o[0];
    } else if constexpr (NB == 8) {
      *reinterpret_cast<uint2*>(p) = uint2{o[0], o[1]};
    } else if constexpr (NB >= 16) {
#pragma unroll
      for (int q = 0; q < W / 4; ++q)
        stg16(reinterpret_cast<uint32_t*>(p) + 4 * q, u32x4{o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]});
    }
  }
};

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
constexpr int FWD_BAGS = 16;  // bags per wave in the forward

// S consecutive lookups of a chunk starting at chunk row s0 (all inside the
// chunk when CHECK is false): their table rows are loaded together, then
// added to the running sum in order; a bag end stores and resets the sum.
template <typename TT, typename XT, int EPL, int S, bool MEAN, bool FULL, bool CHECK>
__device__ inline void fwd_group(int s0, int cnt, uint64_t emask, int grow, int xrow, float inv_len,
                                 const char* Eb, int64_t row_bytes, int lane_b, XT* X, int dim,
                                 int col, bool active, float* acc) {
  Frag<TT, EPL> xf[S];
  const uint64_t em = emask >> s0;  // the group's bag ends at positions 0 .. S-1
#pragma unroll
  for (int i = 0; i < S; ++i) {
    const int r = s0 + i;
    if (CHECK && r >= cnt) break;
    const int gr = __builtin_amdgcn_readlane(grow, r);
    const char* rowp = Eb + (FULL ? ((int64_t)gr << 8) : (int64_t)gr * row_bytes);
    if (FULL || active) xf[i].load(reinterpret_cast<const TT*>(rowp + lane_b));
  }
#pragma unroll
  for (int i = 0; i < S; ++i) {
    const int r = s0 + i;
    if (CHECK && r >= cnt) break;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] += xf[i].get(e);
    if ((em >> i) & 1) {
      if (MEAN) {
        const float il = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(inv_len), r));
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] *= il;
      }
      XT* out = X + (int64_t)__builtin_amdgcn_readlane(xrow, r) * dim + col;
      if (FULL || active) Frag<XT, EPL>::store(out, acc);
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
    }
  }
}

// One wave per FWD_BAGS consecutive bags (feature-major, so a wave's bags are
// consecutive samples of one or two features).  The wave walks their lookups
// in position order one table row per step: lane l holds bytes
// [l*BPL, (l+1)*BPL) of the row, so bag ends are the same for every lane and
// the pooled sum is one fp32 accumulator per column, stored and reset at each
// bag end.  Per chunk of 64 positions: indices (one per lane), their bags, the
// global rows and the destination slots; then in groups of S positions the S
// table rows are loaded together and summed in order.  Empty bags are written
// as zeros.
template <typename TT, typename XT, int BPL, bool MEAN, bool FULL>
__global__ __launch_bounds__(256) void embbag_fwd_kernel(
    const TT* __restrict__ E, const int64_t* __restrict__ row_base,
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ indices, int F, int B,
    int dim, XT* __restrict__ X, int n_slots, int first_slot) {
  constexpr int EPL = BPL / (int)sizeof(TT);
  constexpr int S = BPL == 4 ? 32 : (BPL == 8 ? 16 : 8);
  const int lane = threadIdx.x & 63;
  // Each XCD pools a contiguous span of bags (whole tables), so a table's hot
  // rows are cached in one L2.  Wave-uniform values are scalar: uniform
  // control flow throughout.
  const int wave = __builtin_amdgcn_readfirstlane(xcd_block(blockIdx.x, gridDim.x) * 4 + (threadIdx.x >> 6));
  const int nbags = F * B;
  const int b0 = wave * FWD_BAGS;
  if (b0 >= nbags) return;
  const int nb = nbags - b0 < FWD_BAGS ? nbags - b0 : FWD_BAGS;
  // lane k <= nb holds offsets[b0 + k]
  const int offv = lane <= nb ? offsets[b0 + lane] : 0;
  const int p_begin = __builtin_amdgcn_readlane(offv, 0);
  const int p_end = __builtin_amdgcn_readlane(offv, nb);
  const int col = lane * EPL;
  const bool active = col < dim;
  const int lane_b = lane * BPL;
  const int64_t row_bytes = (int64_t)dim * (int64_t)sizeof(TT);
  const char* Eb = reinterpret_cast<const char*>(E);

  float acc[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
  // bag (index k within the wave's bags) of position p
  auto bag_of = [&](int p) {
    int k = 0;
    for (int q = 1; q < nb; ++q) k += p >= __builtin_amdgcn_readlane(offv, q) ? 1 : 0;
    return k;
  };
  // a chunk's indices and table bases are loaded one chunk ahead: while the
  // rows of one chunk are summed, the next chunk's row numbers are in flight
  int k = 0, idx = 0;
  int64_t rb = 0;
  if (p_begin + lane < p_end) {
    k = bag_of(p_begin + lane);
    idx = indices[p_begin + lane];
    rb = row_base[(b0 + k) / B];
  }
  for (int p0 = p_begin; p0 < p_end; p0 += 64) {
    const int cnt = p_end - p0 < 64 ? p_end - p0 : 64;
    const int p = p0 + lane;
    const bool valid = lane < cnt;
    int nk = 0, nidx = 0;
    int64_t nrb = 0;
    if (p + 64 < p_end) {
      nk = bag_of(p + 64);
      nidx = indices[p + 64];
      nrb = row_base[(b0 + nk) / B];
    }
    // (shuffles stay outside divergent code: a shuffle from a lane that is
    // switched off reads nothing)
    const int next_off = __shfl(offv, k + 1, 64);
    const int this_off = __shfl(offv, k, 64);
    const uint64_t emask = __ballot(valid && p + 1 == next_off);  // last position of its bag
    const int bag = b0 + k;
    const int f = bag / B, b = bag - f * B;
    int grow = 0, xrow = 0;
    float inv_len = 1.f;
    if (valid) {
      grow = (int)(rb + idx);
      xrow = b * n_slots + first_slot + f;
      if (MEAN) inv_len = 1.f / (float)(next_off - this_off);
    }
    int s0 = 0;
    for (; s0 + S <= cnt; s0 += S)
      fwd_group<TT, XT, EPL, S, MEAN, FULL, false>(s0, cnt, emask, grow, xrow, inv_len, Eb, row_bytes,
                                                    lane_b, X, dim, col, active, acc);
    if (s0 < cnt)
      fwd_group<TT, XT, EPL, S, MEAN, FULL, true>(s0, cnt, emask, grow, xrow, inv_len, Eb, row_bytes,
                                                   lane_b, X, dim, col, active, acc);
    k = nk;
    idx = nidx;
    rb = nrb;
  }
  // empty bags pool to zero
  for (int q = 0; q < nb; ++q) {
    if (__builtin_amdgcn_readlane(offv, q) == __builtin_amdgcn_readlane(offv, q + 1)) {
      const int bag = b0 + q, f = bag / B, b = bag - f * B;
      float z[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) z[e] = 0.f;
      if (FULL || active) Frag<XT, EPL>::store(X + ((int64_t)b * n_slots + first_slot + f) * dim + col, z);
    }
  }
}

template <typename TT, typename XT>
static hipError_t embbag_fwd_t(const void* E, int dim, const int64_t* row_base,
                               const int32_t* offsets, const int32_t* indices, int F, int B,
                               int mean, void* X, int n_slots, int first_slot, hipStream_t s) {
  const int64_t bags = (int64_t)F * B;
  if (bags == 0) return hipSuccess;
  const int row_bytes = dim * (int)sizeof(TT);
  const int grid = cdiv(cdiv(bags, FWD_BAGS), 4);
#define LAT_FWD(BPLV, MV, FV)                                                              \
  embbag_fwd_kernel<TT, XT, BPLV, MV, FV><<<grid, 256, 0, s>>>(                           \
      (const TT*)E, row_base, offsets, indices, F, B, dim, (XT*)X, n_slots, first_slot)
  if (row_bytes == 256) {
    if (mean) LAT_FWD(4, true, true); else LAT_FWD(4, false, true);
  } else if (row_bytes < 256) {
    if (mean) LAT_FWD(4, true, false); else LAT_FWD(4, false, false);
  } else if (row_bytes <= 512) {
    if (mean) LAT_FWD(8, true, false); else LAT_FWD(8, false, false);
  } else {
    if (mean) LAT_FWD(16, true, false); else LAT_FWD(16, false, false);
  }
#undef LAT_FWD
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

hipError_t embbag_fwd(const void* E, DType edt, int dim, const int64_t* row_base,
                      const int32_t* offsets, const int32_t* indices, int F, int B, int mean,
                      void* X, DType xdt, int n_slots, int first_slot, hipStream_t s) {
  if (edt == DT_BF16 && xdt == DT_BF16)
    return embbag_fwd_t<bf16_t, bf16_t>(E, dim, row_base, offsets, indices, F, B, mean, X, n_slots, first_slot, s);
  if (edt == DT_BF16 && xdt == DT_F32)
    return embbag_fwd_t<bf16_t, float>(E, dim, row_base, offsets, indices, F, B, mean, X, n_slots, first_slot, s);
  if (edt == DT_F32 && xdt == DT_F32)
    return embbag_fwd_t<float, float>(E, dim, row_base, offsets, indices, F, B, mean, X, n_slots, first_slot, s);
  return embbag_fwd_t<float, bf16_t>(E, dim, row_base, offsets, indices, F, B, mean, X, n_slots, first_slot, s);
}

// ---------------------------------------------------------------------------
// backward: segment bookkeeping over sorted keys
// ---------------------------------------------------------------------------
constexpr int SEG_THREADS = 256;
constexpr int SEG_ITEMS = 16;
constexpr int SEG_TILE = SEG_THREADS * SEG_ITEMS;
// Sorted occurrences per wave in the segmented reduction.  Partial sums only
// arise where a run crosses a multiple of RANGE.
constexpr int RANGE = 256;

// The keys of a tile's SEG_ITEMS stripes and of the positions before them,
// loaded as straight-line code from clamped positions (n >= 1), so that all
// of them are in flight together: a load in a branch, or whose value is
// selected at once, makes the compiler wait for it right there.
__device__ inline void seg_load(const int* __restrict__ keys, int n, int64_t base,
                                int (&key)[SEG_ITEMS], int (&prev)[SEG_ITEMS]) {
#pragma unroll
  for (int i = 0; i < SEG_ITEMS; ++i) {
    const int64_t k = base + (int64_t)i * SEG_THREADS + threadIdx.x;
    const int64_t kc = k < n ? k : n - 1;
    key[i] = keys[kc];
    prev[i] = keys[kc > 0 ? kc - 1 : 0];
  }
}

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
  int key[SEG_ITEMS], prev[SEG_ITEMS];
  seg_load(keys, n, base, key, prev);
  int c = 0;
#pragma unroll
  for (int i = 0; i < SEG_ITEMS; ++i) {
    const int64_t k = base + (int64_t)i * SEG_THREADS + threadIdx.x;
    c += (k < n && (k == 0 || key[i] != prev[i])) ? 1 : 0;
  }
  int tot;
  block_sum_scan(c, lds, &tot);
  if (threadIdx.x == 0) tile_counts[blockIdx.x] = tot;
}

// Run starts of one tile, visited as SEG_ITEMS consecutive 256-position
// stripes (coalesced); a stripe's starts are ranked by wave ballots.  Writes
// the unique rows and run offsets, num_unique, and for every RANGE-aligned
// position k the id of the run holding position k-1 (-1 at k = 0).
__global__ __launch_bounds__(SEG_THREADS) void seg_write_kernel(
    const int* __restrict__ keys, int n, const int* __restrict__ tile_base,
    int* __restrict__ unique_rows, int* __restrict__ seg_offsets, int* __restrict__ num_unique,
    int* __restrict__ range_ubefore) {
  __shared__ int wsum[SEG_THREADS / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  int run = tile_base[blockIdx.x];
  const int64_t base = (int64_t)blockIdx.x * SEG_TILE;
  int keyv[SEG_ITEMS], prev[SEG_ITEMS];
  seg_load(keys, n, base, keyv, prev);
#pragma unroll
  for (int i = 0; i < SEG_ITEMS; ++i) {
    const int64_t k = base + (int64_t)i * SEG_THREADS + threadIdx.x;
    const bool in = k < n;
    const int key = keyv[i];
    const int fl = in && (k == 0 || key != prev[i]) ? 1 : 0;
    const uint64_t m = __ballot(fl);
    if (lane == 0) wsum[w] = __popcll(m);
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < SEG_THREADS / 64; ++q) {
      off += q < w ? wsum[q] : 0;
      tot += wsum[q];
    }
    __syncthreads();
    if (in) {
      const int u = run + off + __popcll(m & lt) + fl - 1;  // run id of position k
      if (fl) {
        unique_rows[u] = key;
        seg_offsets[u] = (int)k;
      }
      if (k % RANGE == 0) range_ubefore[k / RANGE] = u - fl;
      if (k == n - 1) {
        num_unique[0] = u + 1;
        seg_offsets[u + 1] = n;
      }
    }
    run += tot;
  }
}

__global__ void set_empty_kernel(int* num_unique, int* seg_offsets) {
  num_unique[0] = 0;
  seg_offsets[0] = 0;
}

// ---------------------------------------------------------------------------
// backward: segmented reduction over the sorted occurrences (+ fused SGD)
// ---------------------------------------------------------------------------
// One wave per RANGE consecutive sorted occurrences.  The wave walks the
// occurrences one dX row per step: lane l holds bytes [l*BPL, (l+1)*BPL) of
// the row, so run starts and ends are the same for every lane and the
// segmented sum is a single running fp32 accumulator per column, added to in
// position order and cleared after each piece end (uniform branches, no
// cross-lane arithmetic).  Per chunk of 64 occurrences:
//   1. keys and bag ids (one per lane, prefetched a chunk ahead); run starts
//      and ends by comparing neighbouring keys (ballots)
//   2. in groups of S occurrences: the S dX rows, and the table rows of the
//      runs that end there and started inside this range, all loads in
//      flight together; then the S steps of the running sum
//   3. at each run end: a complete run writes its row gradient and/or applies
//      the SGD update; the run cut by the range start (no start inside the
//      range) goes to partial slot 0, the run cut by the range end to slot 1
// No floating-point atomics; every sum is taken in position order.
// FULL: the dX row is exactly 64*BPL bytes (every lane active, no predication).
// SGD: table rows are updated.  The step is bound by instruction issue as much
// as by memory, so the per-occurrence work is kept to a few instructions: row
// offsets are read from lanes (v_readlane) straight into the scalar offset of
// a buffer access, group positions are compile-time constants in full chunks,
// and the table is addressed through a buffer resource based at the range's
// first row whenever the range's rows span less than 4 GiB (EBUF).
template <typename DT, typename ET, int BPL, bool MEAN, bool FULL, bool SGD>
struct SegWave {
  static constexpr int EPL = BPL / (int)sizeof(DT);              // columns per lane
  static constexpr int S = BPL == 4 ? 32 : (BPL == 8 ? 16 : 8);  // rows in flight
  static constexpr int ENB = EPL * (int)sizeof(ET);              // table bytes per lane
  // constants of the wave
  __amdgpu_buffer_rsrc_t dXr;  // dX (< 4 GiB, checked by the launcher)
  const char* dXb;
  ET* E;
  float *grad_rows, *part;
  float lr;
  int wave, dim, col, lane_b, lane_e;
  int64_t erow_bytes;
  bool active;
  // running state: this lane's accumulators; wave-uniform run bookkeeping
  float acc[EPL];
  bool started;  // a run started at or after the range start
  int u_before;  // run id of the run before the current chunk

  // NB bytes of a buffer at byte offset voff + soff (streamed: each table row
  // is read and written exactly once)
  template <int NB>
  __device__ static inline void buf_load(uint32_t* w, __amdgpu_buffer_rsrc_t r, int voff, int soff) {
    if constexpr (NB == 2) {
      w[0] = __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, BUF_NT);
    } else if constexpr (NB == 4) {
      w[0] = __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, BUF_NT);
    } else if constexpr (NB == 8) {
      const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, BUF_NT);
      w[0] = v[0];
      w[1] = v[1];
    } else {
#pragma unroll
      for (int q = 0; q < NB / 16; ++q) {
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff + 16 * q, soff, BUF_NT);
#pragma unroll
        for (int t = 0; t < 4; ++t) w[4 * q + t] = v[t];
      }
    }
  }
  template <int NB>
  __device__ static inline void buf_store(const uint32_t* w, __amdgpu_buffer_rsrc_t r, int voff, int soff) {
    if constexpr (NB == 2) {
      __builtin_amdgcn_raw_buffer_store_b16((uint16_t)w[0], r, voff, soff, BUF_NT);
    } else if constexpr (NB == 4) {
      __builtin_amdgcn_raw_buffer_store_b32(w[0], r, voff, soff, BUF_NT);
    } else if constexpr (NB == 8) {
      __builtin_amdgcn_raw_buffer_store_b64(u32x2{w[0], w[1]}, r, voff, soff, BUF_NT);
    } else {
#pragma unroll
      for (int q = 0; q < NB / 16; ++q)
        __builtin_amdgcn_raw_buffer_store_b128(u32x4{w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]},
                                               r, voff + 16 * q, soff, BUF_NT);
    }
  }
  // the updated row values rounded to ET, as 32-bit words
  __device__ static inline void pack(uint32_t* o, const float* v) {
    if constexpr (sizeof(ET) == 2) {
      if constexpr (EPL == 1) {
        o[0] = f2bf(v[0]);
      } else {
#pragma unroll
        for (int t = 0; t < EPL / 2; ++t) o[t] = pack_bf2(v[2 * t], v[2 * t + 1]);
      }
    } else {
#pragma unroll
      for (int t = 0; t < EPL; ++t) o[t] = __float_as_uint(v[t]);
    }
  }

  // One group of S occurrences starting at chunk row s0 (s0 + S <= cnt when
  // CHECK is false).  Per lane (= chunk row): xoff, the byte offset of the
  // occurrence's dX row; erow, its table row as a byte offset into er (EBUF)
  // or as a row number (otherwise); scl, its bag's 1/length (MEAN).
  template <bool CHECK, bool EBUF>
  __device__ inline void group(const int s0, const int cnt, const uint64_t smask,
                               const uint64_t cmask, const uint64_t pmask, const int xoff,
                               const int erow, const float scl, const __amdgpu_buffer_rsrc_t er) {
    Frag<DT, EPL> xf[S];
    Frag<ET, EPL> ef[S];
    // the group's run bits at positions 0 .. S-1 (constant-position tests below)
    static_assert(S <= 32, "group masks are 32-bit");
    const uint32_t cm = (uint32_t)(cmask >> s0), pm = (uint32_t)(pmask >> s0);
#pragma unroll
    for (int i = 0; i < S; ++i) {
      const int r = s0 + i;
      if (CHECK && r >= cnt) break;
      const int xr = __builtin_amdgcn_readlane(xoff, r);
      if constexpr (FULL) {
        xf[i].w[0] = __builtin_amdgcn_raw_buffer_load_b32(dXr, lane_b, xr, 0);
      } else {
        if (active) xf[i].load(reinterpret_cast<const DT*>(dXb + (uint32_t)xr + lane_b));
      }
      if (SGD && ((cm >> i) & 1)) {
        const int er_r = __builtin_amdgcn_readlane(erow, r);
        if (FULL || active) {
          if constexpr (EBUF) {
            buf_load<ENB>(ef[i].w, er, lane_e, er_r);
          } else {
            const char* p = reinterpret_cast<const char*>(E) + (int64_t)er_r * erow_bytes + lane_e;
            ef[i].load_nt(reinterpret_cast<const ET*>(p));
          }
        }
      }
    }
    // the table row offsets are read from their lanes again at the update, and
    // the run-end bits tested again, rather than held in 2*S scalar registers
    // across the group (opaque copies the compiler cannot fold into the loads')
    int erow2 = erow;
    uint32_t cm2 = cm;
    if constexpr (SGD) asm volatile("" : "+v"(erow2), "+s"(cm2));
#pragma unroll
    for (int i = 0; i < S; ++i) {
      const int r = s0 + i;
      if (CHECK && r >= cnt) break;
      if (MEAN) {
        const float sc = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(scl), r));
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] += xf[i].get(e) * sc;
      } else {
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] += xf[i].get(e);
      }
      if ((pm >> i) & 1) {  // a piece ends here
        const uint64_t le = (r == 63) ? ~0ull : ((2ull << r) - 1);
        if ((cm2 >> i) & 1) {  // ... completing its run
          if (grad_rows && (FULL || active))
            Frag<float, EPL>::store(grad_rows + (int64_t)(u_before + __popcll(smask & le)) * dim + col, acc);
          if constexpr (SGD) {
            float upd[EPL];
#pragma unroll
            for (int e = 0; e < EPL; ++e) upd[e] = ef[i].get(e) - lr * acc[e];
            const int er_r = __builtin_amdgcn_readlane(erow2, r);
            if (FULL || active) {
              if constexpr (EBUF) {
                uint32_t o[Frag<ET, EPL>::W];
                pack(o, upd);
                buf_store<ENB>(o, er, lane_e, er_r);
              } else {
                Frag<ET, EPL>::store_nt(reinterpret_cast<ET*>(reinterpret_cast<char*>(E) +
                                                              (int64_t)er_r * erow_bytes + lane_e),
                                        upd);
              }
            }
          }
        } else {
          const bool has_start = started || (smask & le);
          if (FULL || active)
            Frag<float, EPL>::store(part + ((int64_t)wave * 2 + (has_start ? 1 : 0)) * dim + col, acc);
        }
        // the next occurrence starts a new run (or lies past the range)
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
      }
    }
  }

  // The range's occurrences [r0, rend), chunk by chunk.  EBUF: er covers the
  // table rows from row k_first on.
  template <bool EBUF>
  __device__ inline void run(const int* __restrict__ skeys, const int* __restrict__ sbags, int n,
                             int r0, int rend, int B, int n_slots, int first_slot, int row_bytes,
                             const int32_t* __restrict__ offsets, int lane, int k_first,
                             __amdgpu_buffer_rsrc_t er, int* __restrict__ part_uid,
                             int* __restrict__ span_list, int* __restrict__ span_count) {
    int prev_key = r0 > 0 ? __builtin_amdgcn_readfirstlane(skeys[r0 - 1]) : -1;
    int last_nxt = -1;
    int p0 = r0;
    int key = -1, bag = 0, nxt;
    {
      const int cnt = rend - p0 < 64 ? rend - p0 : 64;
      if (lane < cnt) {
        key = skeys[p0 + lane];
        bag = sbags[p0 + lane];
      }
      nxt = p0 + cnt < n ? __builtin_amdgcn_readfirstlane(skeys[p0 + cnt]) : -1;
    }
    while (p0 < rend) {
      const int cnt = rend - p0 < 64 ? rend - p0 : 64;
      const bool valid = lane < cnt;
      const int q0 = p0 + cnt;
      int nkey = -1, nbag = 0, nnxt = -1;
      if (q0 < rend) {
        const int ncnt = rend - q0 < 64 ? rend - q0 : 64;
        if (lane < ncnt) {
          nkey = skeys[q0 + lane];
          nbag = sbags[q0 + lane];
        }
        nnxt = q0 + ncnt < n ? __builtin_amdgcn_readfirstlane(skeys[q0 + ncnt]) : -1;
      }
      int kp = __shfl_up(key, 1, 64);
      if (lane == 0) kp = prev_key;
      int kn = __shfl_down(key, 1, 64);
      if (lane == cnt - 1) kn = nxt;
      const uint64_t smask = __ballot(valid && key != kp);  // run starts
      const uint64_t emask = __ballot(valid && key != kn);  // run ends
      // runs ending here are complete if a start lies at or before them in the range
      const uint64_t ge_first = smask ? ~((smask & (~smask + 1)) - 1) : 0ull;
      const uint64_t cmask = emask & (started ? ~0ull : ge_first);
      const uint64_t pmask = emask | (q0 == rend ? (1ull << (cnt - 1)) : 0ull);  // piece ends
      int xoff = 0, erow = 0;
      float scl = 1.f;
      if (valid) {
        const int f = bag / B, b = bag - f * B;
        xoff = (int)((uint32_t)(b * n_slots + first_slot + f) * (uint32_t)row_bytes);  // < 2^32
        erow = EBUF ? (int)((uint32_t)(key - k_first) * (uint32_t)erow_bytes) : key;   // < 2^32
        if (MEAN) scl = 1.f / (float)(offsets[bag + 1] - offsets[bag]);
      }
      // full chunks: the groups unrolled with constant positions (not for the
      // far-apart-rows fallback of the SGD path, which is rare)
      if ((!SGD || EBUF) && cnt == 64) {
#pragma unroll
        for (int g = 0; g < 64 / S; ++g)
          group<false, EBUF>(g * S, 64, smask, cmask, pmask, xoff, erow, scl, er);
      } else {
        for (int s0 = 0; s0 < cnt; s0 += S)
          group<true, EBUF>(s0, cnt, smask, cmask, pmask, xoff, erow, scl, er);
      }
      started = started || smask != 0;
      prev_key = __builtin_amdgcn_readlane(key, cnt - 1);
      u_before += __popcll(smask);
      last_nxt = nxt;
      key = nkey;
      bag = nbag;
      nxt = nnxt;
      p0 = q0;
    }
    if (lane == 0) {
      const bool touch_end = rend < n && last_nxt == prev_key;
      part_uid[wave] = touch_end ? u_before : -1;
      if (touch_end && started) span_list[atomicAdd(span_count, 1)] = wave;
    }
  }
};

template <typename DT, typename ET, int BPL, bool MEAN, bool FULL, bool SGD>
__global__ __launch_bounds__(256) void seg_reduce_kernel(
    const int* __restrict__ skeys, const int* __restrict__ sbags, int n,
    const DT* __restrict__ dX, int B, int n_slots, int first_slot, int dim,
    const int32_t* __restrict__ offsets, const int* __restrict__ range_ubefore,
    float* __restrict__ part, int* __restrict__ part_uid, int* __restrict__ span_list,
    int* __restrict__ span_count, float* __restrict__ grad_rows, ET* __restrict__ E, float lr) {
  using W = SegWave<DT, ET, BPL, MEAN, FULL, SGD>;
  const int lane = threadIdx.x & 63;
  // Each XCD takes a contiguous span of ranges, so the dX rows of one table's
  // occurrences stay in that XCD's L2 while it works through them.  Wave-
  // uniform values are made scalar explicitly: all control flow below is
  // uniform branching.
  const int wave = __builtin_amdgcn_readfirstlane(xcd_block(blockIdx.x, gridDim.x) * 4 + (threadIdx.x >> 6));
  const int r0 = wave * RANGE;
  if (r0 >= n) return;
  const int rend = n - r0 < RANGE ? n : r0 + RANGE;
  W w;
  w.wave = wave;
  w.dim = dim;
  w.col = lane * W::EPL;
  w.active = w.col < dim;
  w.lane_b = lane * BPL;
  w.lane_e = w.col * (int)sizeof(ET);
  w.erow_bytes = (int64_t)dim * (int64_t)sizeof(ET);
  w.dXb = reinterpret_cast<const char*>(dX);
  w.dXr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<DT*>(dX), (short)0,
      (int)(uint32_t)((uint64_t)B * n_slots * dim * sizeof(DT) < 0xffffffffull
                          ? (uint64_t)B * n_slots * dim * sizeof(DT) : 0xffffffffull),
      BUF_RSRC_WORD3);
  w.E = E;
  w.grad_rows = grad_rows;
  w.part = part;
  w.lr = lr;
#pragma unroll
  for (int e = 0; e < W::EPL; ++e) w.acc[e] = 0.f;
  w.started = false;
  w.u_before = __builtin_amdgcn_readfirstlane(range_ubefore[wave]);
  const int row_bytes = dim * (int)sizeof(DT);
  if constexpr (SGD) {
    // the range's keys are sorted: its table rows lie in [k_first, k_last]
    const int k_first = __builtin_amdgcn_readfirstlane(skeys[r0]);
    const int k_last = __builtin_amdgcn_readfirstlane(skeys[rend - 1]);
    const uint64_t span = (uint64_t)(k_last - k_first + 1) * (uint64_t)w.erow_bytes;
    if (span <= 0xffffffffull) {
      const __amdgpu_buffer_rsrc_t er = __builtin_amdgcn_make_buffer_rsrc(
          reinterpret_cast<char*>(E) + (int64_t)k_first * w.erow_bytes, (short)0,
          (int)(uint32_t)span, BUF_RSRC_WORD3);
      w.template run<true>(skeys, sbags, n, r0, rend, B, n_slots, first_slot, row_bytes, offsets,
                           lane, k_first, er, part_uid, span_list, span_count);
      return;
    }
  }
  w.template run<false>(skeys, sbags, n, r0, rend, B, n_slots, first_slot, row_bytes, offsets,
                        lane, 0, w.dXr, part_uid, span_list, span_count);
}

// One wave per run that crosses a range boundary: its partial sums (slot 1 of
// the range where it starts, slot 0 of every later range it reaches) are
// added in range order by S interleaved streams of dim/4 lanes each, then the
// streams are combined in stream order; the total goes to the row gradient
// and/or the SGD update.  A wave takes FIX_U runs per round and loads their
// index chains (run -> its row id -> run end and table row), each stream's
// first partial sum and the table values straight-line, all in flight
// together (a round's positions past the last run re-read its first run, and
// a null table reads the partials in its place; neither value is used), then
// finishes the runs one by one: each run's arithmetic is that of a wave
// taking it alone.
constexpr int FIX_U = 4;
template <typename ET>
__global__ __launch_bounds__(256) void seg_fixup_kernel(
    const int* __restrict__ span_list, const int* __restrict__ span_count,
    const int* __restrict__ part_uid, const int* __restrict__ seg_offsets,
    const int* __restrict__ unique_rows, const float* __restrict__ part, int dim,
    float* __restrict__ grad_rows, ET* __restrict__ E, float lr) {
  const int nspan = *span_count;
  const int lane = threadIdx.x & 63;
  const int CL = dim / 4;  // 4-column groups (dim % 8 == 0, dim <= 256)
  const int S = 64 / CL;   // streams
  const int cq = lane % CL, s = lane / CL;
  const bool act = s < S;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6), nwaves = gridDim.x * 4;
  const ET* eb = E ? E : reinterpret_cast<const ET*>(part);
  for (int i0 = wave; i0 < nspan; i0 += FIX_U * nwaves) {
    int c0[FIX_U], u[FIX_U], Q[FIX_U];
    int64_t erow[FIX_U];
#pragma unroll
    for (int t = 0; t < FIX_U; ++t) {
      const int i = i0 + t * nwaves;
      c0[t] = span_list[i < nspan ? i : i0];
    }
#pragma unroll
    for (int t = 0; t < FIX_U; ++t) u[t] = part_uid[c0[t]];
#pragma unroll
    for (int t = 0; t < FIX_U; ++t) {
      Q[t] = (seg_offsets[u[t] + 1] - 1) / RANGE - c0[t] + 1;
      erow[t] = E ? (int64_t)unique_rows[u[t]] * dim : 0;
    }
    // stream s's first partial sum (q = s; the run's first slot where the
    // run does not reach it) and the run's table values
    f32x4 a0[FIX_U];
    float ev[FIX_U][4];
#pragma unroll
    for (int t = 0; t < FIX_U; ++t) {
      const int q = s < Q[t] ? s : 0;
      const int64_t slot = q == 0 ? (int64_t)c0[t] * 2 + 1 : (int64_t)(c0[t] + q) * 2;
      a0[t] = *reinterpret_cast<const f32x4*>(part + slot * dim + cq * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) ev[t][e] = ld(eb + erow[t] + cq * 4 + e);
    }
#pragma unroll
    for (int t = 0; t < FIX_U; ++t) {
      if (i0 + t * nwaves >= nspan) break;  // wave-uniform
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
      if (act && s < Q[t]) {
        a += a0[t];
        int q = s + S;
        for (; q + 3 * S < Q[t]; q += 4 * S) {
          f32x4 v[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int64_t slot = (int64_t)(c0[t] + q + k * S) * 2;
            v[k] = *reinterpret_cast<const f32x4*>(part + slot * dim + cq * 4);
          }
#pragma unroll
          for (int k = 0; k < 4; ++k) a += v[k];
        }
        for (; q < Q[t]; q += S) a += *reinterpret_cast<const f32x4*>(part + (int64_t)(c0[t] + q) * 2 * dim + cq * 4);
      }
      f32x4 t4 = {0.f, 0.f, 0.f, 0.f};
      for (int ss = 0; ss < S; ++ss) {
#pragma unroll
        for (int e = 0; e < 4; ++e) t4[e] += __shfl(a[e], ss * CL + cq, 64);
      }
      if (s == 0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int c = cq * 4 + e;
          if (grad_rows) grad_rows[(int64_t)u[t] * dim + c] = t4[e];
          if (E) st(E + erow[t] + c, ev[t][e] - lr * t4[e]);
        }
      }
    }
  }
}

__global__ void zero_int_kernel(int* p, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t embbag_bwd_workspace(int64_t nnz, int dim, int F) {
  const int64_t n = nnz > 0 ? nnz : 1;
  const int64_t ranges = cdiv(n, RANGE);
  size_t s = 0;
  s += align256((size_t)n * 4);                        // sorted keys
  s += align256(radix_sort_segments_workspace(n, F));
  s += align256((size_t)(cdiv(n, SEG_TILE) + 1) * 4);  // segment tile counts
  s += 3 * align256((size_t)ranges * 4);               // range_ubefore, part_uid, span_list
  s += align256(4);                                    // span_count
  s += align256((size_t)ranges * 2 * dim * 4);         // partial sums
  return s;
}

template <typename DT, typename ET>
static hipError_t embbag_bwd_reduce(const int* skeys, const int* sbags, int n, const void* dX,
                                    int B, int n_slots, int first_slot, int dim,
                                    const int32_t* offsets, int mean, const int* range_ubefore,
                                    float* part, int* part_uid, int* span_list, int* span_count,
                                    const int* seg_offsets, const int* unique_rows,
                                    float* grad_rows, void* E, float lr, hipStream_t s,
                                    void* const* ev) {
  // ev (optional): 4 events, begin / end of the reduction and of the fixup
  // (null entries are not recorded)
  auto record = [&](int i) -> hipError_t {
    return ev && ev[i] ? hipEventRecord((hipEvent_t)ev[i], s) : hipSuccess;
  };
  const int ranges = cdiv(n, RANGE);
  LAT_HIP_CHECK(record(0));
  const int row_bytes = dim * (int)sizeof(DT);
  const int grid = cdiv(ranges, 4);
#define LAT_SEG(BPLV, MV, FV)                                                                \
  do {                                                                                      \
    if (E)                                                                                  \
      seg_reduce_kernel<DT, ET, BPLV, MV, FV, true><<<grid, 256, 0, s>>>(                   \
          skeys, sbags, n, (const DT*)dX, B, n_slots, first_slot, dim, offsets, range_ubefore, \
          part, part_uid, span_list, span_count, grad_rows, (ET*)E, lr);                    \
    else                                                                                    \
      seg_reduce_kernel<DT, ET, BPLV, MV, FV, false><<<grid, 256, 0, s>>>(                  \
          skeys, sbags, n, (const DT*)dX, B, n_slots, first_slot, dim, offsets, range_ubefore, \
          part, part_uid, span_list, span_count, grad_rows, (ET*)E, lr);                    \
  } while (0)
  if (row_bytes == 256) {
    if (mean) LAT_SEG(4, true, true); else LAT_SEG(4, false, true);
  } else if (row_bytes < 256) {
    if (mean) LAT_SEG(4, true, false); else LAT_SEG(4, false, false);
  } else if (row_bytes <= 512) {
    if (mean) LAT_SEG(8, true, false); else LAT_SEG(8, false, false);
  } else {
    if (mean) LAT_SEG(16, true, false); else LAT_SEG(16, false, false);
  }
#undef LAT_SEG
  LAT_LAUNCH_CHECK();
  LAT_HIP_CHECK(record(1));
  LAT_HIP_CHECK(record(2));
  // every wave resident (5 blocks of 4 waves per compute unit at the
  // kernel's 88-96 VGPRs): each then takes its runs in rounds of FIX_U
  const int fix_grid = grid < 1280 ? grid : 1280;
  seg_fixup_kernel<ET><<<fix_grid, 256, 0, s>>>(span_list, span_count, part_uid, seg_offsets,
                                                unique_rows, part, dim, grad_rows, (ET*)E, lr);
  LAT_LAUNCH_CHECK();
  LAT_HIP_CHECK(record(3));
  return hipSuccess;
}

// The sparse gradient's workspace, shared by its two phases.
struct EmbBwdWs {
  int* skeys;
  void* sort_ws;
  int *tile_counts, *range_ubefore, *part_uid, *span_list, *span_count;
  float* part;
};
static EmbBwdWs emb_bwd_ws(void* ws, int64_t nnz, int dim, int F) {
  const int64_t n = nnz > 0 ? nnz : 1;
  const int64_t ranges = cdiv(n, RANGE);
  char* p = static_cast<char*>(ws);
  auto take = [&](size_t bytes) { char* q = p; p += align256(bytes); return q; };
  EmbBwdWs w;
  w.skeys = (int*)take((size_t)n * 4);
  w.sort_ws = take(radix_sort_segments_workspace(n, F));
  w.tile_counts = (int*)take((size_t)(cdiv(n, SEG_TILE) + 1) * 4);
  w.range_ubefore = (int*)take((size_t)ranges * 4);
  w.part_uid = (int*)take((size_t)ranges * 4);
  w.span_list = (int*)take((size_t)ranges * 4);
  w.span_count = (int*)take(4);
  w.part = (float*)take((size_t)ranges * 2 * dim * 4);
  return w;
}

hipError_t embbag_bwd_sort(const int64_t* row_base, int64_t max_local_rows, const int32_t* offsets,
                           const int32_t* indices, int F, int B, int64_t nnz, int dim,
                           int* unique_rows, int* seg_offsets, int* sorted_bags, int* num_unique,
                           void* ws, hipStream_t s, void* const* ev) {
  // ev (optional): 4 events, begin / end of the sort and of the run bookkeeping
  // (null entries are not recorded)
  auto record = [&](int i) -> hipError_t {
    return ev && ev[i] ? hipEventRecord((hipEvent_t)ev[i], s) : hipSuccess;
  };
  LAT_HIP_CHECK(record(0));
  if (nnz == 0) {
    LAT_HIP_CHECK(record(1));
    LAT_HIP_CHECK(record(2));
    set_empty_kernel<<<1, 1, 0, s>>>(num_unique, seg_offsets);
    LAT_LAUNCH_CHECK();
    LAT_HIP_CHECK(record(3));
    return hipSuccess;
  }
  const int n = (int)nnz;
  EmbBwdWs w = emb_bwd_ws(ws, nnz, dim, F);
  hipError_t e = radix_sort_segments(indices, n, offsets, F, B, row_base, max_local_rows,
                                     w.skeys, sorted_bags, w.sort_ws, s);
  if (e != hipSuccess) return e;
  LAT_HIP_CHECK(record(1));
  LAT_HIP_CHECK(record(2));
  const int tiles = cdiv(n, SEG_TILE);
  zero_int_kernel<<<1, 64, 0, s>>>(w.span_count, 1);
  LAT_LAUNCH_CHECK();
  seg_count_kernel<<<tiles, SEG_THREADS, 0, s>>>(w.skeys, n, w.tile_counts);
  LAT_LAUNCH_CHECK();
  e = exclusive_scan_inplace_small(w.tile_counts, tiles, s);
  if (e != hipSuccess) return e;
  seg_write_kernel<<<tiles, SEG_THREADS, 0, s>>>(w.skeys, n, w.tile_counts, unique_rows,
                                                 seg_offsets, num_unique, w.range_ubefore);
  LAT_LAUNCH_CHECK();
  LAT_HIP_CHECK(record(3));
  return hipSuccess;
}

hipError_t embbag_bwd_apply(const int32_t* offsets, int F, int B, int64_t nnz, int mean,
                            const void* dX, DType dxt, int n_slots, int first_slot, int dim,
                            const int* unique_rows, const int* seg_offsets, const int* sorted_bags,
                            float* grad_rows, void* E, DType et, float lr, void* ws, hipStream_t s,
                            void* const* ev) {
  if (nnz == 0) {
    if (ev)
      for (int i = 0; i < 4; ++i)
        if (ev[i]) LAT_HIP_CHECK(hipEventRecord((hipEvent_t)ev[i], s));
    return hipSuccess;
  }
  const int n = (int)nnz;
  if ((int64_t)B * n_slots * dim * (dxt == DT_BF16 ? 2 : 4) > (int64_t)UINT32_MAX) {
    set_error("dX of %lld bytes: the sparse gradient addresses dX with 32-bit offsets",
              (long long)B * n_slots * dim * (dxt == DT_BF16 ? 2 : 4));
    return hipErrorInvalidValue;
  }
  EmbBwdWs w = emb_bwd_ws(ws, nnz, dim, F);
  void* Eupd = lr != 0.f ? E : nullptr;
#define LAT_RED(DTT, ETT)                                                                       \
  return embbag_bwd_reduce<DTT, ETT>(w.skeys, sorted_bags, n, dX, B, n_slots, first_slot, dim,   \
                                     offsets, mean, w.range_ubefore, w.part, w.part_uid,          \
                                     w.span_list, w.span_count, seg_offsets, unique_rows,         \
                                     grad_rows, Eupd, lr, s, ev)
  if (dxt == DT_BF16 && et == DT_BF16) LAT_RED(bf16_t, bf16_t);
  if (dxt == DT_BF16 && et == DT_F32) LAT_RED(bf16_t, float);
  if (dxt == DT_F32 && et == DT_BF16) LAT_RED(float, bf16_t);
  LAT_RED(float, float);
#undef LAT_RED
}

hipError_t embbag_bwd(const int64_t* row_base, int64_t max_local_rows, const int32_t* offsets,
                      const int32_t* indices, int F, int B, int64_t nnz, int mean,
                      const void* dX, DType dxt, int n_slots, int first_slot, int dim,
                      int* unique_rows, int* seg_offsets, int* sorted_bags, int* num_unique,
                      float* grad_rows, void* E, DType et, float lr, void* ws, hipStream_t s) {
  hipError_t e = embbag_bwd_sort(row_base, max_local_rows, offsets, indices, F, B, nnz, dim,
                                 unique_rows, seg_offsets, sorted_bags, num_unique, ws, s, nullptr);
  if (e != hipSuccess) return e;
  return embbag_bwd_apply(offsets, F, B, nnz, mean, dX, dxt, n_slots, first_slot, dim, unique_rows,
                          seg_offsets, sorted_bags, grad_rows, E, et, lr, ws, s, nullptr);
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
                                                       int B, int64_t nnz, int64_t max_rows,
                                                       unsigned long long* __restrict__ bad) {
  const int64_t bags = (int64_t)F * B;
  const int64_t bag = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (max_rows > 0 && bag < F && row_base[bag + 1] - row_base[bag] > max_rows)
    atomicMin(&bad[0], (unsigned long long)(bags + 1 + bag));
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
                          const int32_t* indices, int F, int B, int64_t nnz, int64_t max_rows,
                          unsigned long long* dev_result, hipStream_t s) {
  validate_init_kernel<<<1, 1, 0, s>>>(dev_result);
  LAT_LAUNCH_CHECK();
  const int64_t bags = (int64_t)F * B;
  const int64_t threads = (bags + 1 > F ? bags + 1 : F);
  validate_kernel<<<cdiv(threads, 256), 256, 0, s>>>(row_base, offsets, indices, F, B, nnz,
                                                     max_rows, dev_result);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

}  // namespace lat
