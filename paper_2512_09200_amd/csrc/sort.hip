// Stable LSD radix sort of the occurrences of a jagged batch by table row
// (int32 key, int32 bag id), used by the deterministic embedding backward to
// group the occurrences of each row.
//
// One histogram pass over the batch's indices counts every digit of every
// pass per feature segment (the counts of a digit do not depend on the order
// the previous passes leave).  Each sort pass is then a single kernel: a tile
// of 8192 items is ranked with wave ballots (items with equal digits keep
// their order), its digit counts are published, and its output offsets come
// from the segment's digit bases plus the counts of the segment's earlier
// tiles, read by decoupled look-back over the tiles' published counts (the
// single-pass prefix scan of Merrill and Garland, "Single-pass Parallel
// Prefix Scan with Decoupled Look-back", NVIDIA technical report NVR-2016-002,
// implemented here from its description; tiles take their ids in the order
// they start, so every tile looked back at is running and publishes without
// waiting).
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace lat {

// 512 threads x 16 items: a scatter block holds 73 KB of LDS, so two fit a
// CU and one leaving frees room for a 72 KB GEMM block of the dense stages
// that run beside the sort (with 4096-item tiles four 37 KB blocks filled the
// LDS and a freed slot was always refilled by the next sort block).
constexpr int SORT_THREADS = 512;
constexpr int SORT_ITEMS = 16;
constexpr int SORT_TILE = SORT_THREADS * SORT_ITEMS;  // 8192
constexpr int RADIX_BITS = 8;
constexpr int RADIX = 1 << RADIX_BITS;

constexpr int SCAN_THREADS = 256;
static_assert(SORT_THREADS >= RADIX, "one thread per digit in the scatter's tile scan");

// ---------------------------------------------------------------------------
// block-wide and small exclusive scans of int32 (counts fit int32: totals < 2^31)
// ---------------------------------------------------------------------------
__device__ inline int block_exclusive_scan(int v, int* lds, int* total) {
  // lds: at least SCAN_THREADS/64 ints
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds[w] = x;
  __syncthreads();
  int wbase = 0, tot = 0;
  const int nw = blockDim.x >> 6;
  for (int i = 0; i < nw; ++i) {
    int s = lds[i];
    if (i < w) wbase += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return wbase + x - v;
}

// single block: exclusive scan of the tile sums in place (n >= 1).  Thread t
// owns elements [t*per, (t+1)*per); they are read SCAN_REG at a time from
// clamped positions (straight-line loads, all in flight together), and kept
// in registers for the second sweep when per <= SCAN_REG.
constexpr int SCAN_REG = 4;
__global__ __launch_bounds__(1024) void scan_sums_kernel(int* __restrict__ sums, int n) {
  __shared__ int lds[1024 / 64];
  const int per = (n + blockDim.x - 1) / blockDim.x;
  const int lo = threadIdx.x * per;
  int v[SCAN_REG];
  int s = 0;
  for (int i0 = 0; i0 < per; i0 += SCAN_REG) {
#pragma unroll
    for (int r = 0; r < SCAN_REG; ++r) {
      const int i = lo + i0 + r;
      v[r] = sums[i < n ? i : n - 1];
    }
#pragma unroll
    for (int r = 0; r < SCAN_REG; ++r)
      if (i0 + r < per && lo + i0 + r < n) s += v[r];
  }
  int tot;
  int run = block_exclusive_scan(s, lds, &tot);
  for (int i0 = 0; i0 < per; i0 += SCAN_REG) {
    if (per > SCAN_REG) {
#pragma unroll
      for (int r = 0; r < SCAN_REG; ++r) {
        const int i = lo + i0 + r;
        v[r] = sums[i < n ? i : n - 1];
      }
    }
#pragma unroll
    for (int r = 0; r < SCAN_REG; ++r) {
      const int i = lo + i0 + r;
      if (i0 + r < per && i < n) {
        sums[i] = run;
        run += v[r];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// radix sort
// ---------------------------------------------------------------------------
static int key_bits(int64_t max_key) {
  int b = 0;
  while (b < 31 && ((int64_t)1 << b) <= max_key) ++b;
  return b;
}

// ---------------------------------------------------------------------------
// segmented radix sort (positions grouped by feature)
// ---------------------------------------------------------------------------
// The occurrences of a jagged batch are feature-major, so segment f (positions
// offsets[f*B] .. offsets[(f+1)*B]) holds all keys of table f, and those keys
// lie in [row_base[f], row_base[f] + rows_f).  Sorting every segment by its
// local row (key - row_base[f]) is therefore a sort by global key, and needs
// only as many digit passes as the largest table has row bits.  Tiles never
// straddle segments; a pass scatters each tile inside its own segment.

// tiles per segment (tile_base, scanned afterwards); also clears zero[0 .. nzero)
__global__ __launch_bounds__(256) void seg_ntiles_kernel(const int32_t* __restrict__ offsets, int F,
                                                         int B, int* __restrict__ tile_base,
                                                         int* __restrict__ zero, int nzero) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < nzero) zero[i] = 0;
  if (i <= F)
    tile_base[i] = i < F ? (offsets[(int64_t)(i + 1) * B] - offsets[(int64_t)i * B] + SORT_TILE - 1) / SORT_TILE : 0;
}

// tile -> segment map: block f fills its segment's tiles
__global__ __launch_bounds__(256) void seg_tilemap_kernel(const int* __restrict__ tile_base,
                                                          int* __restrict__ tile_seg) {
  const int f = blockIdx.x;
  for (int t = tile_base[f] + threadIdx.x; t < tile_base[f + 1]; t += 256) tile_seg[t] = f;
}

// tile -> first bag: every non-empty bag writes its index to the tiles that
// start inside it (each tile start lies in exactly one non-empty bag)
__global__ __launch_bounds__(256) void seg_tilebag_kernel(const int32_t* __restrict__ offsets,
                                                          int F, int B,
                                                          const int* __restrict__ tile_base,
                                                          int* __restrict__ tile_bag0) {
  const int64_t bag = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (bag >= (int64_t)F * B) return;
  const int f = (int)(bag / B);
  const int seg0 = offsets[(int64_t)f * B];
  const int lo = offsets[bag], hi = offsets[bag + 1];
  if (lo == hi) return;
  for (int lt = (lo - seg0 + SORT_TILE - 1) / SORT_TILE; seg0 + lt * SORT_TILE < hi; ++lt)
    tile_bag0[tile_base[f] + lt] = (int)bag;
}

struct SegTile {
  int f, lt, base, cnt;  // segment, tile within it, first position, items
  int64_t key0;          // row_base[f]
};

__device__ inline void seg_tile(int tix, const int* tile_base, const int* tile_seg,
                                const int32_t* offsets, const int64_t* row_base, int B, SegTile& t) {
  t.f = tile_seg[tix];
  t.lt = tix - tile_base[t.f];
  const int s0 = offsets[(int64_t)t.f * B], s1 = offsets[(int64_t)(t.f + 1) * B];
  t.base = s0 + t.lt * SORT_TILE;
  t.cnt = s1 - t.base < SORT_TILE ? s1 - t.base : SORT_TILE;
  t.key0 = row_base[t.f];
}

// Digit counts of every pass per segment, ghist[pass][f][digit] (zeroed
// before), from the batch's indices (rows local to the segment's table); each
// tile also clears its look-back words of every pass.
__global__ __launch_bounds__(SORT_THREADS) void radix_hist_all_kernel(
    const int32_t* __restrict__ indices, const int32_t* __restrict__ offsets,
    const int64_t* __restrict__ row_base, int F, int B, const int* __restrict__ tile_base,
    const int* __restrict__ tile_seg, int passes, int dbits, int tmax, int* __restrict__ ghist,
    uint32_t* __restrict__ state) {
  __shared__ int hist[4][RADIX];
  const int tix = blockIdx.x;
  if (tix >= tile_base[F]) return;
  const int radix = 1 << dbits;
  SegTile t;
  seg_tile(tix, tile_base, tile_seg, offsets, row_base, B, t);
  for (int i = threadIdx.x; i < passes * radix; i += SORT_THREADS) {
    hist[i / radix][i % radix] = 0;
    state[((int64_t)(i / radix) * tmax + tix) * radix + i % radix] = 0u;
  }
  __syncthreads();
  // all of the thread's indices in flight together (positions past the
  // tile's end read position 0 and are not counted)
  uint32_t rv[SORT_ITEMS];
#pragma unroll
  for (int i = 0; i < SORT_ITEMS; ++i) {
    const int k = i * SORT_THREADS + threadIdx.x;
    rv[i] = (uint32_t)indices[t.base + (k < t.cnt ? k : 0)];
  }
#pragma unroll
  for (int i = 0; i < SORT_ITEMS; ++i) {
    const int k = i * SORT_THREADS + threadIdx.x;
    if (k < t.cnt)
      for (int p = 0; p < passes; ++p) atomicAdd(&hist[p][(rv[i] >> (p * dbits)) & (radix - 1)], 1);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < passes * radix; i += SORT_THREADS) {
    const int c = hist[i / radix][i % radix];
    if (c) atomicAdd(&ghist[((int64_t)(i / radix) * F + t.f) * radix + i % radix], c);
  }
}

// Look-back words: bits 30-31 = 0 (not yet published), 1 (the tile's own
// count of the digit), 2 (inclusive count over the segment's tiles up to
// this one); bits 0-29 the count (< 2^30 occurrences).
constexpr uint32_t LB_AGG = 1u << 30, LB_INC = 2u << 30, LB_VAL = (1u << 30) - 1;
constexpr int LB_WIN = 8;
// tile counters of the sort passes, one per (pass, segment), 128 bytes apart
constexpr int CTR_STRIDE = 32;

__device__ inline void lb_store(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint32_t lb_load(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One sort pass.  FIRST (the first pass): keys_in are the batch's indices
// (local rows) and vals_in is unused: the keys become global rows (+ row_base
// of the segment) and the values the bag ids, expanded from the offsets of the
// bags the tile covers (tile_bag0: the first of them).
template <bool FIRST, int DB>
__global__ __launch_bounds__(SORT_THREADS) void radix_scatter_seg_kernel(
    const int* __restrict__ keys_in, const int* __restrict__ vals_in,
    const int* __restrict__ tile_bag0, const int32_t* __restrict__ offsets,
    const int64_t* __restrict__ row_base, int F, int B, const int* __restrict__ tile_base,
    const int* __restrict__ tile_seg, int pass, int dbits, int tmax,
    const int* __restrict__ ghist, uint32_t* __restrict__ state, int* __restrict__ tile_ctr,
    int* __restrict__ keys_out, int* __restrict__ vals_out) {
  constexpr int NW = SORT_THREADS / 64;
  constexpr int CHUNK = SORT_TILE / NW;  // 1024 consecutive items per wave
  constexpr int ROUNDS = CHUNK / 64;     // 16
  __shared__ int wcnt[NW][RADIX];        // per-wave digit counts, then per-wave bases in the tile
  __shared__ int dbase[RADIX];           // output position of tile position 0 of each digit
  __shared__ int scan_tmp[SORT_THREADS / 64];
  __shared__ int lkeys[SORT_TILE];
  __shared__ int lvals[SORT_TILE];
  __shared__ int s_tix;
  // Block b works on a tile of the segment static tile b lies in; which one
  // is the order the segment's blocks start in (one counter per segment and
  // pass: a single device-wide counter serialises every block's start)
  if ((int)blockIdx.x >= tile_base[F]) return;
  if (threadIdx.x == 0) {
    const int f0 = tile_seg[blockIdx.x];
    s_tix = tile_base[f0] + atomicAdd(&tile_ctr[((int64_t)pass * F + f0) * CTR_STRIDE], 1);
  }
  __syncthreads();
  const int tix = s_tix;
  constexpr int radix = 1 << DB;  // the digit width is a template argument (dbits == DB)
  const int shift = pass * DB;
  SegTile t;
  seg_tile(tix, tile_base, tile_seg, offsets, row_base, B, t);
  const int key0 = (int)t.key0;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < NW * RADIX; i += SORT_THREADS) (&wcnt[0][0])[i] = 0;
  __syncthreads();
  if constexpr (FIRST) {
    // bag id of every tile position, staged in lvals (free until the ranks
    // are known): bag0 + i for i = thread, thread + 256, ... until the bags
    // start past the tile
    const int tend = t.base + t.cnt, bag_end = (t.f + 1) * B;
    for (int bag = tile_bag0[tix] + threadIdx.x; bag < bag_end; bag += SORT_THREADS) {
      const int lo = offsets[bag];
      if (lo >= tend) break;
      const int hi = offsets[bag + 1] < tend ? offsets[bag + 1] : tend;
      for (int q = lo > t.base ? lo : t.base; q < hi; ++q) lvals[q - t.base] = bag;
    }
    __syncthreads();
  }
  const int cbase = w * CHUNK;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int key[ROUNDS], val[ROUNDS], rank[ROUNDS];
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int k = cbase + r * 64 + lane;
    const bool valid = k < t.cnt;
    // a lane past the tile's end reads position 0 (its key and value are
    // never used): no select on the loaded value, so the loads of all
    // rounds are in flight together
    const int kk = valid ? k : 0;
    if constexpr (FIRST) {
      key[r] = keys_in[t.base + kk] + key0;
      val[r] = lvals[kk];
    } else {
      key[r] = keys_in[t.base + kk];
      val[r] = vals_in[t.base + kk];
    }
  }
  // stable rank of each item among the wave's items with the same digit
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int k = cbase + r * 64 + lane;
    const bool valid = k < t.cnt;
    const uint32_t d = ((uint32_t)(key[r] - key0) >> shift) & (radix - 1);
    // lanes whose digit equals this lane's: for each bit, the ballot of the
    // lanes holding it set, kept where this lane's bit is set and inverted
    // where it is clear (sb: the bit spread over a word; unrolled over the
    // digit's bits)
    const uint64_t vm = __ballot(valid);
    uint32_t plo = (uint32_t)vm, phi = (uint32_t)(vm >> 32);
#pragma unroll
    for (int b = 0; b < DB; ++b) {
      const uint32_t sb = (uint32_t)((int32_t)(d << (31 - b)) >> 31);
      const uint64_t m = __ballot(sb != 0u);
      plo &= ~((uint32_t)m ^ sb);
      phi &= ~((uint32_t)(m >> 32) ^ sb);
    }
    const uint64_t peers = ((uint64_t)phi << 32) | plo;
    const int before = __popcll(peers & lt_mask);
    const int cnt = __popcll(peers);
    const int base = valid ? wcnt[w][d] : 0;
    rank[r] = base + before;
    __builtin_amdgcn_wave_barrier();
    if (valid && before == 0) wcnt[w][d] = base + cnt;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  }
  __syncthreads();
  {
    const int d = threadIdx.x;  // SORT_THREADS >= RADIX >= radix
    int tot = 0;
    if (d < radix)
      for (int i = 0; i < NW; ++i) tot += wcnt[i][d];
    // publish this tile's count of digit d, then add up the counts of the
    // segment's earlier tiles: back over published counts until an
    // inclusive one (the segment's first tile publishes its count as such)
    uint32_t* st = state + (int64_t)pass * tmax * radix;
    int excl = 0;
    if (d < radix) {
      lb_store(st + (int64_t)tix * radix + d, (t.lt == 0 ? LB_INC : LB_AGG) | (uint32_t)tot);
      if (t.lt > 0) {
        // LB_WIN predecessors read per round trip, nearest first; a word not
        // yet published ends the round (it is read again next round)
        const int jlo = tix - t.lt;  // the segment's first tile
        for (int j = tix - 1;;) {
          uint32_t v[LB_WIN];
#pragma unroll
          for (int q = 0; q < LB_WIN; ++q)
            v[q] = j - q >= jlo ? lb_load(st + (int64_t)(j - q) * radix + d) : LB_INC;
          bool done = false;
          int q = 0;
#pragma unroll
          for (; q < LB_WIN; ++q) {
            if ((v[q] & ~LB_VAL) == 0u) break;
            excl += (int)(v[q] & LB_VAL);
            if (v[q] & LB_INC) {
              done = true;
              break;
            }
          }
          if (done) break;
          j -= q;
          if (q < LB_WIN) __builtin_amdgcn_s_sleep(1);
        }
        lb_store(st + (int64_t)tix * radix + d, LB_INC | (uint32_t)(excl + tot));
      }
    }
    // the segment's bucket of digit d starts after the segment's items of
    // smaller digits
    const int g = d < radix ? ghist[((int64_t)pass * F + t.f) * radix + d] : 0;
    int all;
    const int gex = block_exclusive_scan(g, scan_tmp, &all);
    // tile-level digit starts (exclusive scan over digits) and per-wave bases
    const int tst = block_exclusive_scan(tot, scan_tmp, &all);
    if (d < radix) dbase[d] = offsets[(int64_t)t.f * B] + gex + excl - tst;
    int run = tst;
    if (d < radix)
      for (int i = 0; i < NW; ++i) {
        const int c = wcnt[i][d];
        wcnt[i][d] = run;
        run += c;
      }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int k = cbase + r * 64 + lane;
    if (k < t.cnt) {
      const uint32_t d = ((uint32_t)(key[r] - key0) >> shift) & (radix - 1);
      const int pos = wcnt[w][d] + rank[r];
      lkeys[pos] = key[r];
      lvals[pos] = val[r];
    }
  }
  __syncthreads();
  // consecutive threads write consecutive positions of each digit's run
  for (int i = threadIdx.x; i < t.cnt; i += SORT_THREADS) {
    const int kk = lkeys[i];
    const uint32_t d = ((uint32_t)(kk - key0) >> shift) & (radix - 1);
    const int pos = dbase[d] + i;
    keys_out[pos] = kk;
    vals_out[pos] = lvals[i];
  }
}

static int seg_sort_tiles_max(int64_t n, int F) { return cdiv(n, SORT_TILE) + F; }
constexpr int MAX_PASSES = 4;  // 31-bit rows, digits of up to 8 bits

size_t radix_sort_segments_workspace(int64_t n, int F) {
  const int64_t tmax = seg_sort_tiles_max(n > 0 ? n : 1, F);
  return 2 * (size_t)(n > 0 ? n : 1) * sizeof(int)              // ping-pong keys/vals
         + (size_t)MAX_PASSES * RADIX * tmax * sizeof(uint32_t)  // look-back words
         + (size_t)MAX_PASSES * F * RADIX * sizeof(int)          // digit counts per segment
         + (size_t)MAX_PASSES * F * CTR_STRIDE * sizeof(int)     // tile counters
         + (size_t)(F + 1 + 2 * tmax) * sizeof(int) + 1024;      // tile_base, tile_seg, tile_bag0
}

hipError_t radix_sort_segments(const int32_t* indices, int64_t n, const int32_t* offsets, int F,
                               int B, const int64_t* row_base, int64_t max_local_rows,
                               int* keys_out, int* vals_out, void* ws, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int tmax = seg_sort_tiles_max(n, F);
  char* p = static_cast<char*>(ws);
  int* kb = reinterpret_cast<int*>(p); p += (size_t)n * sizeof(int);
  int* vb = reinterpret_cast<int*>(p); p += (size_t)n * sizeof(int);
  uint32_t* state = reinterpret_cast<uint32_t*>(p); p += (size_t)MAX_PASSES * RADIX * tmax * sizeof(uint32_t);
  int* ghist = reinterpret_cast<int*>(p); p += (size_t)MAX_PASSES * F * RADIX * sizeof(int);
  int* tile_ctr = reinterpret_cast<int*>(p); p += (size_t)MAX_PASSES * F * CTR_STRIDE * sizeof(int);
  int* tile_base = reinterpret_cast<int*>(p); p += (size_t)(F + 1) * sizeof(int);
  int* tile_seg = reinterpret_cast<int*>(p); p += (size_t)tmax * sizeof(int);
  int* tile_bag0 = reinterpret_cast<int*>(p);

  const int bits = key_bits(max_local_rows > 0 ? max_local_rows - 1 : 0);
  const int passes = bits == 0 ? 1 : (bits + RADIX_BITS - 1) / RADIX_BITS;
  const int dbits = bits == 0 ? 1 : (bits + passes - 1) / passes;

  // the digit counts and tile id counters (ghist and tile_ctr are adjacent)
  const int nzero = MAX_PASSES * F * (RADIX + CTR_STRIDE);
  seg_ntiles_kernel<<<cdiv(nzero, 256), 256, 0, s>>>(offsets, F, B, tile_base, ghist, nzero);
  LAT_LAUNCH_CHECK();
  hipError_t e = exclusive_scan_inplace_small(tile_base, F + 1, s);
  if (e != hipSuccess) return e;
  seg_tilemap_kernel<<<F, 256, 0, s>>>(tile_base, tile_seg);
  LAT_LAUNCH_CHECK();
  seg_tilebag_kernel<<<cdiv((int64_t)F * B, 256), 256, 0, s>>>(offsets, F, B, tile_base, tile_bag0);
  LAT_LAUNCH_CHECK();
  radix_hist_all_kernel<<<tmax, SORT_THREADS, 0, s>>>(indices, offsets, row_base, F, B, tile_base,
                                                      tile_seg, passes, dbits, tmax, ghist, state);
  LAT_LAUNCH_CHECK();

  const int* src_k = indices;
  const int* src_v = nullptr;
  for (int pass = 0; pass < passes; ++pass) {
    const bool last = pass == passes - 1;
    const int remaining = passes - 1 - pass;
    int* dst_k = last ? keys_out : ((remaining % 2 == 1) ? kb : keys_out);
    int* dst_v = last ? vals_out : ((remaining % 2 == 1) ? vb : vals_out);
    auto launch = [&](auto first, auto db) {
      radix_scatter_seg_kernel<decltype(first)::value, decltype(db)::value><<<tmax, SORT_THREADS, 0, s>>>(
          src_k, src_v, tile_bag0, offsets, row_base, F, B, tile_base, tile_seg, pass, dbits, tmax,
          ghist, state, tile_ctr, dst_k, dst_v);
    };
    auto by_width = [&](auto first) {
      switch (dbits) {
        case 1: launch(first, std::integral_constant<int, 1>{}); break;
        case 2: launch(first, std::integral_constant<int, 2>{}); break;
        case 3: launch(first, std::integral_constant<int, 3>{}); break;
        case 4: launch(first, std::integral_constant<int, 4>{}); break;
        case 5: launch(first, std::integral_constant<int, 5>{}); break;
        case 6: launch(first, std::integral_constant<int, 6>{}); break;
        case 7: launch(first, std::integral_constant<int, 7>{}); break;
        default: launch(first, std::integral_constant<int, 8>{}); break;
      }
    };
    if (pass == 0) by_width(std::true_type{});
    else by_width(std::false_type{});
    LAT_LAUNCH_CHECK();
    src_k = dst_k; src_v = dst_v;
  }
  return hipSuccess;
}

}  // namespace lat

namespace lat {
hipError_t exclusive_scan_inplace_small(int* a, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  scan_sums_kernel<<<1, 1024, 0, s>>>(a, n);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}
}  // namespace lat
