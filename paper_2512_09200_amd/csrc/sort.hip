// Stable LSD radix sort of (int32 key, int32 value) pairs and a device-wide
// exclusive scan, used by the deterministic embedding backward to group the
// occurrences of each table row.
//
// Sort pass (8-bit digit):
//   hist    : per tile of 4096 items, digit histogram in LDS -> counts[d][tile]
//   scan    : exclusive scan of counts (digit-major) -> global bucket offsets
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

__global__ __launch_bounds__(SCAN_THREADS) void scan_apply_kernel(const int* __restrict__ in, int n,
                                                                   const int* __restrict__ sums,
                                                                   int* __restrict__ out) {
  __shared__ int lds[SCAN_THREADS / 64];
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
  int run = block_exclusive_scan(s, lds, &tot) + sums[blockIdx.x];
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
  scan_sums_kernel<<<1, 1024, 0, s>>>(tmp, tiles);
  LAT_LAUNCH_CHECK();
  scan_apply_kernel<<<tiles, SCAN_THREADS, 0, s>>>(in, (int)n, tmp, out);
  LAT_LAUNCH_CHECK();
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// radix sort
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(SORT_THREADS) void radix_hist_kernel(const int* __restrict__ keys, int n,
                                                                   int shift, int tiles,
                                                                   int* __restrict__ counts) {
  __shared__ int hist[RADIX];
  for (int i = threadIdx.x; i < RADIX; i += SORT_THREADS) hist[i] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * SORT_TILE;
#pragma unroll
  for (int i = 0; i < SORT_ITEMS; ++i) {
    int64_t k = base + (int64_t)i * SORT_THREADS + threadIdx.x;
    if (k < n) atomicAdd(&hist[((uint32_t)keys[k] >> shift) & (RADIX - 1)], 1);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < RADIX; d += SORT_THREADS) counts[(int64_t)d * tiles + blockIdx.x] = hist[d];
}

__global__ __launch_bounds__(SORT_THREADS) void radix_scatter_kernel(
    const int* __restrict__ keys_in, const int* __restrict__ vals_in, int n, int shift, int tiles,
    const int* __restrict__ offsets, int* __restrict__ keys_out, int* __restrict__ vals_out) {
  constexpr int NW = SORT_THREADS / 64;
  constexpr int CHUNK = SORT_TILE / NW;  // 1024 consecutive items per wave
  constexpr int ROUNDS = CHUNK / 64;     // 16
  __shared__ int wcnt[NW][RADIX];        // per-wave digit counts, then per-wave bases in the tile
  __shared__ int dstart[RADIX];          // first tile position of each digit
  __shared__ int scan_tmp[SORT_THREADS / 64];
  __shared__ int lkeys[SORT_TILE];
  __shared__ int lvals[SORT_TILE];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < NW * RADIX; i += SORT_THREADS) (&wcnt[0][0])[i] = 0;
  __syncthreads();

  const int64_t tbase = (int64_t)blockIdx.x * SORT_TILE;
  const int64_t cbase = tbase + (int64_t)w * CHUNK;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int key[ROUNDS], val[ROUNDS], rank[ROUNDS];
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    int64_t k = cbase + (int64_t)r * 64 + lane;
    bool valid = k < n;
    key[r] = valid ? keys_in[k] : 0;
    val[r] = valid ? vals_in[k] : 0;
  }
  // stable rank of each item among the wave's items with the same digit
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    int64_t k = cbase + (int64_t)r * 64 + lane;
    bool valid = k < n;
    uint32_t d = ((uint32_t)key[r] >> shift) & (RADIX - 1);
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < RADIX_BITS; ++b) {
      uint64_t m = __ballot((d >> b) & 1u);
      peers &= ((d >> b) & 1u) ? m : ~m;
    }
    int before = __popcll(peers & lt_mask);
    int cnt = __popcll(peers);
    int base = valid ? wcnt[w][d] : 0;
    rank[r] = base + before;
    __builtin_amdgcn_wave_barrier();
    if (valid && before == 0) wcnt[w][d] = base + cnt;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  }
  __syncthreads();
  // tile-level digit starts (exclusive scan over digits) and per-wave bases
  {
    const int d = threadIdx.x;  // SORT_THREADS == RADIX
    int tot = 0;
    for (int i = 0; i < NW; ++i) tot += wcnt[i][d];
    int all;
    const int st = block_exclusive_scan(tot, scan_tmp, &all);
    dstart[d] = st;
    int run = st;
    for (int i = 0; i < NW; ++i) {
      const int c = wcnt[i][d];
      wcnt[i][d] = run;
      run += c;
    }
  }
  __syncthreads();
  // the tile in stable digit order in LDS
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    int64_t k = cbase + (int64_t)r * 64 + lane;
    if (k < n) {
      uint32_t d = ((uint32_t)key[r] >> shift) & (RADIX - 1);
      const int pos = wcnt[w][d] + rank[r];
      lkeys[pos] = key[r];
      lvals[pos] = val[r];
    }
  }
  __syncthreads();
  // consecutive threads write consecutive positions of each digit's run
  const int tn = (int)((n - tbase) < SORT_TILE ? (n - tbase) : SORT_TILE);
  for (int i = threadIdx.x; i < tn; i += SORT_THREADS) {
    const int kk = lkeys[i];
    const uint32_t d = ((uint32_t)kk >> shift) & (RADIX - 1);
    const int pos = offsets[(int64_t)d * tiles + blockIdx.x] + (i - dstart[d]);
    keys_out[pos] = kk;
    vals_out[pos] = lvals[i];
  }
}

static int key_bits(int64_t max_key) {
  int b = 0;
  while (b < 31 && ((int64_t)1 << b) <= max_key) ++b;
  return b;
}

size_t radix_sort_workspace(int64_t n) {
  const int tiles = cdiv(n, SORT_TILE);
  size_t c = (size_t)RADIX * tiles;
  return 2 * (size_t)n * sizeof(int)            // ping-pong keys/vals (second buffer pair)
         + 2 * c * sizeof(int)                  // counts + offsets
         + scan_workspace((int64_t)c) + 256;
}

// Sorts (keys, vals) of length n with keys in [0, max_key].  keys/vals are
// clobbered; the sorted result is written to keys_out / vals_out.
hipError_t radix_sort_pairs(int* keys, int* vals, int64_t n, int64_t max_key, int* keys_out,
                            int* vals_out, void* ws, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int tiles = cdiv(n, SORT_TILE);
  const size_t c = (size_t)RADIX * tiles;
  char* p = static_cast<char*>(ws);
  int* kb = reinterpret_cast<int*>(p); p += (size_t)n * sizeof(int);
  int* vb = reinterpret_cast<int*>(p); p += (size_t)n * sizeof(int);
  int* counts = reinterpret_cast<int*>(p); p += c * sizeof(int);
  int* offs = reinterpret_cast<int*>(p); p += c * sizeof(int);
  int* tmp = reinterpret_cast<int*>(p);

  const int bits = key_bits(max_key);
  const int passes = bits == 0 ? 1 : (bits + RADIX_BITS - 1) / RADIX_BITS;
  // ping-pong so that the final pass lands in keys_out / vals_out
  int* src_k = keys; int* src_v = vals;
  for (int pass = 0; pass < passes; ++pass) {
    const bool last = pass == passes - 1;
    // passes remaining after this one decide the buffer so the last is *_out
    const int remaining = passes - 1 - pass;
    int* dst_k = last ? keys_out : ((remaining % 2 == 1) ? kb : keys_out);
    int* dst_v = last ? vals_out : ((remaining % 2 == 1) ? vb : vals_out);
    const int shift = pass * RADIX_BITS;
    radix_hist_kernel<<<tiles, SORT_THREADS, 0, s>>>(src_k, (int)n, shift, tiles, counts);
    LAT_LAUNCH_CHECK();
    hipError_t e = exclusive_scan(counts, offs, (int64_t)c, tmp, s);
    if (e != hipSuccess) return e;
    radix_scatter_kernel<<<tiles, SORT_THREADS, 0, s>>>(src_k, src_v, (int)n, shift, tiles, offs,
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
