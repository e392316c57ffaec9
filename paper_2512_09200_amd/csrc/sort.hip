// Stable LSD radix sort of (int32 key, int32 value) pairs and a device-wide
// exclusive scan, used by the deterministic embedding backward to group the
// occurrences of each table row.
//
// Sort pass (digit of up to 8 bits):
//   hist    : per tile of 4096 items, digit histogram in LDS -> counts
//   scan    : exclusive scan of the counts -> global bucket offsets
//   scatter : each wave ranks its contiguous 1024-item chunk with ballots
//             (items with equal digits keep their order), waves are ordered
//             within the tile, tiles within the bucket: a stable pass.
#include "common.h"
#include "kernels.h"

namespace lat {

constexpr int SORT_THREADS = 256;
constexpr int SORT_ITEMS = 16;
constexpr int SORT_TILE = SORT_THREADS * SORT_ITEMS;  // 4096
constexpr int RADIX_BITS = 8;
constexpr int RADIX = 1 << RADIX_BITS;

constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 16;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;  // 4096
static_assert(SORT_THREADS == RADIX, "one thread per digit in the scatter's tile scan");

// ---------------------------------------------------------------------------
// device-wide exclusive scan of int32 (counts fit int32: totals < 2^31)
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

__global__ __launch_bounds__(SCAN_THREADS) void scan_reduce_kernel(const int* __restrict__ in, int n,
                                                                    int* __restrict__ sums) {
  __shared__ int lds[SCAN_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
  int s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    int64_t k = base + (int64_t)i * SCAN_THREADS + threadIdx.x;
    if (k < n) s += in[k];
  }
  int tot;
  block_exclusive_scan(s, lds, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

// single block: exclusive scan of the tile sums in place
__global__ __launch_bounds__(1024) void scan_sums_kernel(int* __restrict__ sums, int n) {
  __shared__ int lds[1024 / 64];
  const int per = (n + blockDim.x - 1) / blockDim.x;
  const int lo = threadIdx.x * per;
  int s = 0;
  for (int i = 0; i < per; ++i)
    if (lo + i < n) s += sums[lo + i];
  int tot;
  int run = block_exclusive_scan(s, lds, &tot);
  for (int i = 0; i < per; ++i) {
    if (lo + i < n) {
      int v = sums[lo + i];
      sums[lo + i] = run;
      run += v;
    }
  }
}

// sums: the tile totals (not scanned); each block adds up those before it
__global__ __launch_bounds__(SCAN_THREADS) void scan_apply_kernel(const int* __restrict__ in, int n,
                                                                   const int* __restrict__ sums,
                                                                   int* __restrict__ out) {
  __shared__ int lds[SCAN_THREADS / 64];
  int p = 0;
  for (int i = threadIdx.x; i < (int)blockIdx.x; i += SCAN_THREADS) p += sums[i];
  int prefix;
  block_exclusive_scan(p, lds, &prefix);
  // blocked arrangement: thread t owns items [t*ITEMS, (t+1)*ITEMS) of the tile
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + (int64_t)threadIdx.x * SCAN_ITEMS;
  int v[SCAN_ITEMS];
  int s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    v[i] = (base + i < n) ? in[base + i] : 0;
    s += v[i];
  }
  int tot;
  int run = block_exclusive_scan(s, lds, &tot) + prefix;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
}

size_t scan_workspace(int64_t n) { return (size_t)(cdiv(n, SCAN_TILE) + 1) * sizeof(int); }

hipError_t exclusive_scan(const int* in, int* out, int64_t n, int* tmp, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int tiles = cdiv(n, SCAN_TILE);
  scan_reduce_kernel<<<tiles, SCAN_THREADS, 0, s>>>(in, (int)n, tmp);
  LAT_LAUNCH_CHECK();
  scan_apply_kernel<<<tiles, SCAN_THREADS, 0, s>>>(in, (int)n, tmp, out);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
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
// straddle segments; a pass scatters each tile inside its own segment, with
// bucket offsets from one device-wide scan of the counts laid out as
// [segment][digit][tile of the segment].

__global__ __launch_bounds__(256) void seg_ntiles_kernel(const int32_t* __restrict__ offsets, int F,
                                                         int B, int* __restrict__ tile_base) {
  const int f = blockIdx.x * 256 + threadIdx.x;
  if (f > F) return;
  tile_base[f] = f < F ? (offsets[(int64_t)(f + 1) * B] - offsets[(int64_t)f * B] + SORT_TILE - 1) / SORT_TILE : 0;
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
  int f, lt, nt, base, cnt, cb;  // segment, tile within it, its tile count, first position, items, count base
  int64_t key0;                  // row_base[f]
};

__device__ inline bool seg_tile(const int* tile_base, const int* tile_seg, const int32_t* offsets,
                                const int64_t* row_base, int F, int B, int radix, SegTile& t) {
  const int tix = blockIdx.x;
  if (tix >= tile_base[F]) return false;
  t.f = tile_seg[tix];
  const int tb = tile_base[t.f];
  t.lt = tix - tb;
  t.nt = tile_base[t.f + 1] - tb;
  const int s0 = offsets[(int64_t)t.f * B], s1 = offsets[(int64_t)(t.f + 1) * B];
  t.base = s0 + t.lt * SORT_TILE;
  t.cnt = s1 - t.base < SORT_TILE ? s1 - t.base : SORT_TILE;
  t.cb = tb * radix;
  t.key0 = row_base[t.f];
  return true;
}

// keys: global rows, or (local = 1, the first pass) the batch's indices,
// i.e. rows local to the segment's table
__global__ __launch_bounds__(SORT_THREADS) void radix_hist_seg_kernel(
    const int* __restrict__ keys, int local, const int32_t* __restrict__ offsets,
    const int64_t* __restrict__ row_base, int F, int B, const int* __restrict__ tile_base,
    const int* __restrict__ tile_seg, int shift, int dbits, int* __restrict__ counts) {
  __shared__ int hist[RADIX];
  const int radix = 1 << dbits;
  SegTile t;
  if (!seg_tile(tile_base, tile_seg, offsets, row_base, F, B, radix, t)) {
    // blocks past the last tile clear the unused tail of the counts
    for (int d = threadIdx.x; d < radix; d += SORT_THREADS) counts[(int64_t)blockIdx.x * radix + d] = 0;
    return;
  }
  for (int i = threadIdx.x; i < radix; i += SORT_THREADS) hist[i] = 0;
  __syncthreads();
  const int key0 = local ? 0 : (int)t.key0;
#pragma unroll
  for (int i = 0; i < SORT_ITEMS; ++i) {
    const int k = i * SORT_THREADS + threadIdx.x;
    if (k < t.cnt) atomicAdd(&hist[((uint32_t)(keys[t.base + k] - key0) >> shift) & (radix - 1)], 1);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < radix; d += SORT_THREADS) counts[t.cb + (int64_t)d * t.nt + t.lt] = hist[d];
}

// FIRST (the first pass): keys_in are the batch's indices (local rows) and
// vals_in is unused: the keys become global rows (+ row_base of the
// segment) and the values the bag ids, expanded from the offsets of the
// bags the tile covers (tile_bag0: the first of them).
template <bool FIRST>
__global__ __launch_bounds__(SORT_THREADS) void radix_scatter_seg_kernel(
    const int* __restrict__ keys_in, const int* __restrict__ vals_in,
    const int* __restrict__ tile_bag0, const int32_t* __restrict__ offsets,
    const int64_t* __restrict__ row_base, int F, int B, const int* __restrict__ tile_base,
    const int* __restrict__ tile_seg, int shift, int dbits, const int* __restrict__ coffs,
    int* __restrict__ keys_out, int* __restrict__ vals_out) {
  constexpr int NW = SORT_THREADS / 64;
  constexpr int CHUNK = SORT_TILE / NW;  // 1024 consecutive items per wave
  constexpr int ROUNDS = CHUNK / 64;     // 16
  __shared__ int wcnt[NW][RADIX];        // per-wave digit counts, then per-wave bases in the tile
  __shared__ int dbase[RADIX];           // output position of tile position 0 of each digit
  __shared__ int scan_tmp[SORT_THREADS / 64];
  __shared__ int lkeys[SORT_TILE];
  __shared__ int lvals[SORT_TILE];
  const int radix = 1 << dbits;
  SegTile t;
  if (!seg_tile(tile_base, tile_seg, offsets, row_base, F, B, radix, t)) return;
  const int key0 = (int)t.key0;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < NW * RADIX; i += SORT_THREADS) (&wcnt[0][0])[i] = 0;
  __syncthreads();
  if constexpr (FIRST) {
    // bag id of every tile position, staged in lvals (free until the ranks
    // are known): bag0 + i for i = thread, thread + 256, ... until the bags
    // start past the tile
    const int tend = t.base + t.cnt, bag_end = (t.f + 1) * B;
    for (int bag = tile_bag0[blockIdx.x] + threadIdx.x; bag < bag_end; bag += SORT_THREADS) {
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
    if constexpr (FIRST) {
      key[r] = valid ? keys_in[t.base + k] + key0 : 0;
      val[r] = valid ? lvals[k] : 0;
    } else {
      key[r] = valid ? keys_in[t.base + k] : 0;
      val[r] = valid ? vals_in[t.base + k] : 0;
    }
  }
  // stable rank of each item among the wave's items with the same digit
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int k = cbase + r * 64 + lane;
    const bool valid = k < t.cnt;
    const uint32_t d = ((uint32_t)(key[r] - key0) >> shift) & (radix - 1);
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < dbits; ++b) {
      const uint64_t m = __ballot((d >> b) & 1u);
      peers &= ((d >> b) & 1u) ? m : ~m;
    }
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
  // tile-level digit starts (exclusive scan over digits) and per-wave bases
  {
    const int d = threadIdx.x;  // SORT_THREADS == RADIX >= radix
    int tot = 0;
    if (d < radix)
      for (int i = 0; i < NW; ++i) tot += wcnt[i][d];
    int all;
    const int st = block_exclusive_scan(tot, scan_tmp, &all);
    if (d < radix) dbase[d] = coffs[t.cb + (int64_t)d * t.nt + t.lt] - st;
    int run = st;
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

size_t radix_sort_segments_workspace(int64_t n, int F) {
  const int64_t tmax = seg_sort_tiles_max(n > 0 ? n : 1, F);
  const size_t c = (size_t)RADIX * tmax;
  return 2 * (size_t)(n > 0 ? n : 1) * sizeof(int)  // ping-pong keys/vals
         + 2 * c * sizeof(int)                        // counts + offsets
         + scan_workspace((int64_t)c)
         + (size_t)(F + 1 + 2 * tmax) * sizeof(int) + 1024;  // tile_base, tile_seg, tile_bag0
}

hipError_t radix_sort_segments(const int32_t* indices, int64_t n, const int32_t* offsets, int F,
                               int B, const int64_t* row_base, int64_t max_local_rows,
                               int* keys_out, int* vals_out, void* ws, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int tmax = seg_sort_tiles_max(n, F);
  const size_t c = (size_t)RADIX * tmax;
  char* p = static_cast<char*>(ws);
  int* kb = reinterpret_cast<int*>(p); p += (size_t)n * sizeof(int);
  int* vb = reinterpret_cast<int*>(p); p += (size_t)n * sizeof(int);
  int* counts = reinterpret_cast<int*>(p); p += c * sizeof(int);
  int* offs = reinterpret_cast<int*>(p); p += c * sizeof(int);
  int* tmp = reinterpret_cast<int*>(p); p += scan_workspace((int64_t)c);
  int* tile_base = reinterpret_cast<int*>(p); p += (size_t)(F + 1) * sizeof(int);
  int* tile_seg = reinterpret_cast<int*>(p); p += (size_t)tmax * sizeof(int);
  int* tile_bag0 = reinterpret_cast<int*>(p);

  seg_ntiles_kernel<<<cdiv(F + 1, 256), 256, 0, s>>>(offsets, F, B, tile_base);
  LAT_LAUNCH_CHECK();
  hipError_t e = exclusive_scan_inplace_small(tile_base, F + 1, s);
  if (e != hipSuccess) return e;
  seg_tilemap_kernel<<<F, 256, 0, s>>>(tile_base, tile_seg);
  LAT_LAUNCH_CHECK();
  seg_tilebag_kernel<<<cdiv((int64_t)F * B, 256), 256, 0, s>>>(offsets, F, B, tile_base, tile_bag0);
  LAT_LAUNCH_CHECK();

  const int bits = key_bits(max_local_rows > 0 ? max_local_rows - 1 : 0);
  const int passes = bits == 0 ? 1 : (bits + RADIX_BITS - 1) / RADIX_BITS;
  const int dbits = bits == 0 ? 1 : (bits + passes - 1) / passes;
  const int radix = 1 << dbits;
  const int* src_k = indices;
  const int* src_v = nullptr;
  for (int pass = 0; pass < passes; ++pass) {
    const bool last = pass == passes - 1;
    const int remaining = passes - 1 - pass;
    int* dst_k = last ? keys_out : ((remaining % 2 == 1) ? kb : keys_out);
    int* dst_v = last ? vals_out : ((remaining % 2 == 1) ? vb : vals_out);
    const int shift = pass * dbits;
    radix_hist_seg_kernel<<<tmax, SORT_THREADS, 0, s>>>(src_k, pass == 0, offsets, row_base, F, B,
                                                         tile_base, tile_seg, shift, dbits, counts);
    LAT_LAUNCH_CHECK();
    e = exclusive_scan(counts, offs, (int64_t)radix * tmax, tmp, s);
    if (e != hipSuccess) return e;
    if (pass == 0)
      radix_scatter_seg_kernel<true><<<tmax, SORT_THREADS, 0, s>>>(
          src_k, src_v, tile_bag0, offsets, row_base, F, B, tile_base, tile_seg, shift, dbits, offs,
          dst_k, dst_v);
    else
      radix_scatter_seg_kernel<false><<<tmax, SORT_THREADS, 0, s>>>(
          src_k, src_v, tile_bag0, offsets, row_base, F, B, tile_base, tile_seg, shift, dbits, offs,
          dst_k, dst_v);
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
