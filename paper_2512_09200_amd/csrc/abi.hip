// C ABI of the training-step library: argument checks, the public entry
// points, and lattice_step, which runs the whole forward + backward on one
// stream over a caller-provided workspace whose layout lattice_step_plan
// reports.
#include <cstdarg>
#include <cstdio>
#include <cmath>
#include <cstring>
#include <mutex>

#include "../../include/lattice.h"
#include "common.h"
#include "kernels.h"
#include "swishrn.h"

namespace lat {
static thread_local char g_err[1024] = "";
void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}
}  // namespace lat

using namespace lat;

#define FAIL(code, ...)         \
  do {                          \
    ::lat::set_error(__VA_ARGS__); \
    return code;                \
  } while (0)
#define REQUIRE(cond, ...) \
  do {                     \
    if (!(cond)) FAIL(LATTICE_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)
#define HIPRET(expr)                                  \
  do {                                                \
    hipError_t e__ = (expr);                          \
    if (e__ != hipSuccess) return LATTICE_ERR_HIP;    \
  } while (0)
// inside helpers that return a hipError_t
#define HIP_TRY(expr)                                 \
  do {                                                \
    hipError_t e__ = (expr);                          \
    if (e__ != hipSuccess) return e__;                \
  } while (0)

static inline DType dt_of(lattice_dtype d) { return d == LATTICE_BF16 ? DT_BF16 : DT_F32; }
static inline size_t esize(lattice_dtype d) { return d == LATTICE_BF16 ? 2 : 4; }
static inline hipStream_t strm(void* s) { return reinterpret_cast<hipStream_t>(s); }
static inline size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

static lattice_status check_dim(int dim, lattice_dtype dt) {
  if (dim <= 0 || dim > 256) FAIL(LATTICE_ERR_UNSUPPORTED, "dim %d outside 1..256", dim);
  if (dim % 8) FAIL(LATTICE_ERR_UNSUPPORTED, "dim %d not a multiple of 8", dim);
  (void)dt;
  return LATTICE_OK;
}

// rows of the largest table (max_rows when given, else the total row count)
static int64_t local_rows_bound(const lattice_tables* t) {
  return t->max_rows > 0 ? t->max_rows : t->total_rows;
}

static lattice_status check_tables(const lattice_tables* t, const lattice_jagged* j) {
  REQUIRE(t && j, "null tables or bags");
  REQUIRE(j->num_features >= 0 && j->batch >= 0 && j->nnz >= 0, "negative sizes");
  REQUIRE(j->nnz < ((int64_t)1 << 31), "nnz must be < 2^31");
  if (j->nnz > 0) REQUIRE(j->indices, "null indices");
  if ((int64_t)j->num_features * j->batch > 0) REQUIRE(j->offsets && t->row_base && t->data, "null pointer in batch/tables");
  REQUIRE(t->dtype == LATTICE_F32 || t->dtype == LATTICE_BF16, "bad table dtype");
  if (t->total_rows >= ((int64_t)1 << 31)) FAIL(LATTICE_ERR_UNSUPPORTED, "total_rows must be < 2^31");
  REQUIRE(t->max_rows >= 0 && t->max_rows <= t->total_rows, "max_rows outside 0 .. total_rows");
  return check_dim(t->dim, t->dtype);
}

// Parameter gradients of an empty batch are sums over no samples: zero.  A
// fill kernel (not hipMemsetAsync) so that a captured graph replays it.
__global__ void zero_f32_kernel(float* p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

static hipError_t zero_f32(float* p, int64_t n, hipStream_t s) {
  if (!p || n <= 0) return hipSuccess;
  zero_f32_kernel<<<cdiv(n, 256), 256, 0, s>>>(p, n);
  return hipGetLastError();
}

// layer i applies SwishRN
static bool swish_layer(const lattice_mlp_desc* d, int i) {
  return d->act != LATTICE_ACT_RELU && (i < d->n_layers - 1 || d->relu_last);
}

// layer i is the heads of per-objective towers (W [T, H], H = in / T)
static bool tower_layer(const lattice_mlp_desc* d, int i) {
  return d->tower_heads && i == d->n_layers - 1;
}

static int64_t w_elems(const lattice_mlp_desc* d, int i) {
  const lattice_linear& L = d->layers[i];
  return tower_layer(d, i) ? (int64_t)L.in_dim : (int64_t)L.out_dim * L.in_dim;
}

static hipError_t zero_mlp_grads(const lattice_mlp_desc* d, hipStream_t s) {
  for (int i = 0; i < d->n_layers; ++i) {
    const lattice_linear& L = d->layers[i];
    const int64_t sets = (d->n_domains > 1 && i < d->untied_layers) ? d->n_domains : 1;
    hipError_t e = zero_f32(L.dW, sets * w_elems(d, i), s);
    if (e == hipSuccess) e = zero_f32(L.db, sets * L.out_dim, s);
    if (e == hipSuccess && swish_layer(d, i)) e = zero_f32(L.dgain, sets * 2 * (int64_t)L.out_dim, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

static hipError_t zero_interact_grads(const lattice_interact_desc* d, hipStream_t s) {
  if (d->kind == LATTICE_INTERACT_FM) return zero_f32(d->fm_dW, (int64_t)d->n * d->rank, s);
  if (d->kind != LATTICE_INTERACT_STACK) return hipSuccess;
  int n_in = d->n;
  for (int l = 0; l < d->n_layers; ++l) {
    const lattice_stack_layer& L = d->layers[l];
    const int64_t nd = (int64_t)(d->stack_n - d->lcb_n) * d->dim;
    hipError_t e = zero_f32(L.dW, (int64_t)n_in * d->rank, s);
    if (e == hipSuccess) e = zero_f32(L.dA, nd * n_in * d->rank, s);
    if (e == hipSuccess && L.C) e = zero_f32(L.dC, (int64_t)d->stack_n * n_in, s);
    if (e == hipSuccess && d->lcb_n > 0) e = zero_f32(L.dL, (int64_t)d->lcb_n * n_in, s);
    if (e == hipSuccess) e = zero_f32(L.dgamma, d->dim, s);
    if (e != hipSuccess) return e;
    n_in = d->stack_n;
  }
  return hipSuccess;
}

extern "C" {

const char* lattice_status_string(lattice_status s) {
  switch (s) {
    case LATTICE_OK: return "ok";
    case LATTICE_ERR_INVALID_ARG: return "invalid argument";
    case LATTICE_ERR_UNSUPPORTED: return "unsupported";
    case LATTICE_ERR_WORKSPACE: return "workspace too small";
    case LATTICE_ERR_BAD_INPUT: return "malformed input";
    case LATTICE_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}
const char* lattice_last_error(void) { return g_err; }
int lattice_abi_version(void) { return LATTICE_ABI_VERSION; }

// ---------------------------------------------------------------------------
lattice_status lattice_embbag_fwd(const lattice_tables* tables, const lattice_jagged* bags,
                                  lattice_pool pool, void* X, lattice_dtype x_dtype,
                                  int32_t n_slots, int32_t first_slot, void* stream) {
  lattice_status st = check_tables(tables, bags);
  if (st != LATTICE_OK) return st;
  REQUIRE(x_dtype == LATTICE_F32 || x_dtype == LATTICE_BF16, "bad X dtype");
  REQUIRE(pool == LATTICE_POOL_SUM || pool == LATTICE_POOL_MEAN, "bad pool mode");
  REQUIRE(first_slot >= 0 && first_slot + bags->num_features <= n_slots, "slots out of range");
  if ((int64_t)bags->num_features * bags->batch == 0) return LATTICE_OK;
  REQUIRE(X, "null X");
  HIPRET(embbag_fwd(tables->data, dt_of(tables->dtype), tables->dim, tables->row_base,
                    bags->offsets, bags->indices, bags->num_features, bags->batch,
                    pool == LATTICE_POOL_MEAN, X, dt_of(x_dtype), n_slots, first_slot,
                    strm(stream)));
  return LATTICE_OK;
}

size_t lattice_embbag_bwd_workspace(const lattice_tables* tables, const lattice_jagged* bags) {
  if (!tables || !bags) return 0;
  return embbag_bwd_workspace(bags->nnz, tables->dim, bags->num_features);
}

lattice_status lattice_embbag_bwd(const lattice_tables* tables, const lattice_jagged* bags,
                                  lattice_pool pool, const void* dX, lattice_dtype dx_dtype,
                                  int32_t n_slots, int32_t first_slot,
                                  const lattice_sparse_grad* out, float lr, void* ws,
                                  size_t ws_bytes, void* stream) {
  lattice_status st = check_tables(tables, bags);
  if (st != LATTICE_OK) return st;
  REQUIRE(out && out->unique_rows && out->seg_offsets && out->sorted_bags && out->num_unique,
          "null sparse-gradient output");
  REQUIRE(dx_dtype == LATTICE_F32 || dx_dtype == LATTICE_BF16, "bad dX dtype");
  REQUIRE(pool == LATTICE_POOL_SUM || pool == LATTICE_POOL_MEAN, "bad pool mode");
  REQUIRE(first_slot >= 0 && first_slot + bags->num_features <= n_slots, "slots out of range");
  if (bags->nnz > 0) REQUIRE(dX, "null dX");
  if ((int64_t)bags->batch * n_slots * tables->dim * (int64_t)esize(dx_dtype) > (int64_t)UINT32_MAX)
    FAIL(LATTICE_ERR_UNSUPPORTED, "dX larger than 4 GiB");
  const size_t need = embbag_bwd_workspace(bags->nnz, tables->dim, bags->num_features);
  if (ws_bytes < need || (need && !ws)) FAIL(LATTICE_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
  HIPRET(embbag_bwd(tables->row_base, local_rows_bound(tables), bags->offsets, bags->indices,
                    bags->num_features, bags->batch, bags->nnz, pool == LATTICE_POOL_MEAN, dX,
                    dt_of(dx_dtype), n_slots, first_slot, tables->dim, out->unique_rows,
                    out->seg_offsets, out->sorted_bags, out->num_unique, out->grad_rows,
                    tables->data, dt_of(tables->dtype), lr, ws, strm(stream)));
  return LATTICE_OK;
}

// ---------------------------------------------------------------------------
// The sparse gradient without a caller workspace: its scratch (sort buffers,
// run bookkeeping, partial sums of runs crossing reduction ranges) is one
// file-scope device array per GPU, held until the process ends.  In host
// code `scratch` names a host-side stand-in, never the device memory: the
// device address comes from hipGetSymbolAddress, taken once per device with
// that device current, and only that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[LATTICE_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of this device's scratch array (set up on first use).
lattice_status scratch_of(hipStream_t s, void** out) {
  hipDevice_t dev = 0;
  if (s) {
    if (hipStreamGetDevice(s, &dev) != hipSuccess) FAIL(LATTICE_ERR_HIP, "hipStreamGetDevice failed");
  } else {
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) FAIL(LATTICE_ERR_HIP, "hipGetDevice failed");
    dev = cur;
  }
  REQUIRE(dev >= 0 && dev < kMaxScratchDevices, "device %d out of range", (int)dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) FAIL(LATTICE_ERR_HIP, "hipGetDevice failed");
    if (cur != dev && hipSetDevice(dev) != hipSuccess) FAIL(LATTICE_ERR_HIP, "hipSetDevice failed");
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !ptr)
      FAIL(LATTICE_ERR_HIP, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return LATTICE_OK;
}
}  // namespace

lattice_status lattice_embbag_bwd_noalloc(const lattice_tables* tables, const lattice_jagged* bags,
                                          lattice_pool pool, const void* dX, lattice_dtype dx_dtype,
                                          int32_t n_slots, int32_t first_slot,
                                          const lattice_sparse_grad* out, float lr, void* stream) {
  lattice_status st = check_tables(tables, bags);
  if (st != LATTICE_OK) return st;
  REQUIRE(out && out->unique_rows && out->seg_offsets && out->sorted_bags && out->num_unique,
          "null sparse-gradient output");
  REQUIRE(dx_dtype == LATTICE_F32 || dx_dtype == LATTICE_BF16, "bad dX dtype");
  REQUIRE(pool == LATTICE_POOL_SUM || pool == LATTICE_POOL_MEAN, "bad pool mode");
  REQUIRE(first_slot >= 0 && first_slot + bags->num_features <= n_slots, "slots out of range");
  if (bags->nnz > 0) REQUIRE(dX, "null dX");
  if ((int64_t)bags->batch * n_slots * tables->dim * (int64_t)esize(dx_dtype) > (int64_t)UINT32_MAX)
    FAIL(LATTICE_ERR_UNSUPPORTED, "dX larger than 4 GiB");
  const size_t need = embbag_bwd_workspace(bags->nnz, tables->dim, bags->num_features);
  if (need > (size_t)LATTICE_NOALLOC_SCRATCH_BYTES)
    FAIL(LATTICE_ERR_UNSUPPORTED,
         "the sparse gradient of %lld lookups (dim %d, %d features) needs %zu bytes of scratch; "
         "the allocation-free entry point holds %zu (use lattice_embbag_bwd with a workspace)",
         (long long)bags->nnz, tables->dim, bags->num_features, need,
         (size_t)LATTICE_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  st = scratch_of(strm(stream), &ws);
  if (st != LATTICE_OK) return st;
  HIPRET(embbag_bwd(tables->row_base, local_rows_bound(tables), bags->offsets, bags->indices,
                    bags->num_features, bags->batch, bags->nnz, pool == LATTICE_POOL_MEAN, dX,
                    dt_of(dx_dtype), n_slots, first_slot, tables->dim, out->unique_rows,
                    out->seg_offsets, out->sorted_bags, out->num_unique, out->grad_rows,
                    tables->data, dt_of(tables->dtype), lr, ws, strm(stream)));
  return LATTICE_OK;
}

__device__ unsigned long long g_validate_result[2];
static std::mutex g_validate_mu;

lattice_status lattice_validate_batch(const lattice_tables* tables, const lattice_jagged* bags,
                                      int64_t* first_bad, void* stream) {
  lattice_status st = check_tables(tables, bags);
  if (st != LATTICE_OK) return st;
  REQUIRE(first_bad, "null first_bad");
  *first_bad = 0;
  if ((int64_t)bags->num_features * bags->batch == 0) return LATTICE_OK;
  std::lock_guard<std::mutex> lock(g_validate_mu);
  void* ptr = nullptr;
  if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(g_validate_result)) != hipSuccess)
    FAIL(LATTICE_ERR_HIP, "hipGetSymbolAddress failed");
  HIPRET(validate_batch(tables->row_base, bags->offsets, bags->indices, bags->num_features,
                        bags->batch, bags->nnz, tables->max_rows, (unsigned long long*)ptr,
                        strm(stream)));
  unsigned long long host[2];
  if (hipMemcpyAsync(host, ptr, sizeof(host), hipMemcpyDeviceToHost, strm(stream)) != hipSuccess ||
      hipStreamSynchronize(strm(stream)) != hipSuccess)
    FAIL(LATTICE_ERR_HIP, "validate copy failed");
  if (host[0] != ~0ull) {
    *first_bad = -1 - (int64_t)host[0];
    const int64_t nbags = (int64_t)bags->num_features * bags->batch;
    if ((int64_t)host[0] > nbags)
      FAIL(LATTICE_ERR_BAD_INPUT, "table %lld has more than max_rows rows", (long long)host[0] - nbags - 1);
    FAIL(LATTICE_ERR_BAD_INPUT, "malformed offsets at position %lld", (long long)host[0]);
  }
  if (host[1] != ~0ull) {
    *first_bad = (int64_t)host[1];
    FAIL(LATTICE_ERR_BAD_INPUT, "index out of range at position %lld", (long long)host[1]);
  }
  return LATTICE_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// interaction
// ---------------------------------------------------------------------------
static StackShape stack_shape(const lattice_interact_desc* d) {
  StackShape sh;
  sh.L = d->n_layers;
  sh.n0 = d->n;
  sh.nv = d->stack_n;
  sh.d = d->dim;
  sh.k = d->rank;
  sh.has_C0 = (d->layers && d->n_layers > 0 && d->layers[0].C) ? 1 : 0;
  sh.eps = d->ln_eps;
  sh.nL = d->lcb_n;
  sh.fp8 = d->fp8_proj;
  return sh;
}

static void stack_layers(const lattice_interact_desc* d, StackLayer* out) {
  for (int l = 0; l < d->n_layers; ++l) {
    const lattice_stack_layer& L = d->layers[l];
    out[l] = StackLayer{L.W, L.A, L.C, L.gamma, L.dW, L.dA, L.dC, L.dgamma, L.L, L.dL};
  }
}

static lattice_status check_interact(const lattice_interact_desc* d, int32_t B) {
  REQUIRE(d, "null interaction descriptor");
  REQUIRE(B >= 0, "negative batch");
  REQUIRE(d->dtype == LATTICE_F32 || d->dtype == LATTICE_BF16, "bad dtype");
  REQUIRE(d->n >= 1 && d->dim >= 1, "bad n/dim");
  lattice_status st = check_dim(d->dim, d->dtype);
  if (st != LATTICE_OK) return st;
  REQUIRE(d->skip_absent == 0 || d->skip_absent == 1, "skip_absent must be 0 or 1");
  REQUIRE(d->fp8_proj >= 0 && d->fp8_proj <= 2, "fp8_proj must be 0, 1 or 2");
  if (d->fp8_proj) REQUIRE(d->kind == LATTICE_INTERACT_STACK, "fp8_proj is for the STACK interaction only");
  if (d->skip_absent) REQUIRE(d->kind == LATTICE_INTERACT_DOT, "skip_absent is for the DOT interaction only");
  if (d->slot_mask) {
    REQUIRE(d->kind == LATTICE_INTERACT_DOT, "slot_mask is for the DOT interaction only");
    REQUIRE(d->n <= 128, "slot_mask needs n <= 128");
    REQUIRE(((uintptr_t)d->slot_mask & 15) == 0, "slot_mask must be 16-byte aligned");
  }
  if (d->kind == LATTICE_INTERACT_DOT) {
    if (dot_lds_bytes(d->n, d->dim) > 160 * 1024)
      FAIL(LATTICE_ERR_UNSUPPORTED, "DOT with n=%d, dim=%d exceeds LDS", d->n, d->dim);
  } else if (d->kind == LATTICE_INTERACT_FM) {
    REQUIRE(d->rank >= 1 && d->fm_W, "FM needs rank and W");
    if (fm_lds_bytes(d->n, d->dim, d->rank) > 160 * 1024 || d->n * d->rank > 256 * 64)
      FAIL(LATTICE_ERR_UNSUPPORTED, "FM with n=%d, dim=%d, rank=%d exceeds LDS", d->n, d->dim, d->rank);
  } else if (d->kind == LATTICE_INTERACT_STACK) {
    if (d->dtype != LATTICE_BF16) FAIL(LATTICE_ERR_UNSUPPORTED, "STACK runs in bf16 only");
    REQUIRE(d->n_layers >= 1 && d->n_layers <= LATTICE_MAX_LAYERS && d->layers, "STACK needs 1..%d layers",
            LATTICE_MAX_LAYERS);
    REQUIRE(d->rank >= 1 && d->stack_n >= 1 && d->ln_eps > 0.f, "STACK needs rank, stack_n, ln_eps > 0");
    REQUIRE(!d->emit_slot0, "STACK does not emit slot 0");
    REQUIRE(d->lcb_n >= 0 && d->lcb_n < d->stack_n, "lcb_n must be in 0 .. stack_n - 1");
    for (int l = 0; l < d->n_layers; ++l) {
      const lattice_stack_layer& L = d->layers[l];
      REQUIRE(L.W && L.A && L.gamma, "STACK layer %d: null W/A/gamma", l);
      if (d->lcb_n > 0) REQUIRE(L.L, "STACK layer %d: lcb_n > 0 needs L", l);
      if (l == 0 && d->n != d->stack_n) REQUIRE(L.C, "STACK layer 0 needs C when n != stack_n");
      if (l > 0) REQUIRE(!L.C, "STACK layer %d: only layer 0 may have C", l);
    }
    if (!stack_supported(stack_shape(d)))
      FAIL(LATTICE_ERR_UNSUPPORTED, "STACK shape n=%d stack_n=%d dim=%d rank=%d not supported", d->n,
           d->stack_n, d->dim, d->rank);
  } else {
    FAIL(LATTICE_ERR_UNSUPPORTED, "interaction kind %d not supported", (int)d->kind);
  }
  return LATTICE_OK;
}

static int64_t interact_width(const lattice_interact_desc* d) {
  if (d->kind == LATTICE_INTERACT_STACK) return (int64_t)d->stack_n * d->dim;
  int64_t w = d->kind == LATTICE_INTERACT_DOT ? (int64_t)d->n * (d->n - 1) / 2
                                              : (int64_t)d->n * d->rank;
  return w + (d->emit_slot0 ? d->dim : 0);
}

// The MFMA path reads and writes rows with 4-byte accesses: row strides must
// keep every row 16-byte aligned.
static bool fm_uses_mfma(const lattice_interact_desc* d, int64_t stride = 8) {
  return d->dtype == LATTICE_BF16 && fm_mfma_supported(d->n, d->dim, d->rank) && stride % 8 == 0;
}

// DOT on MFMA: bf16, n <= 128, d in {64, 128}, X rows read with 4-byte loads
static bool dot_uses_mfma(const lattice_interact_desc* d, const void* X) {
  return d->dtype == LATTICE_BF16 && dot_mfma_supported(d->n, d->dim) &&
         ((uintptr_t)X & 3) == 0;
}

// bytes of the step's DOT slot masks (B x 4 words) when its DOT runs on MFMA
static size_t step_dot_mask_bytes(const lattice_model_desc* m, int B) {
  const lattice_interact_desc* d = &m->interact;
  if (!d->skip_absent || d->kind != LATTICE_INTERACT_DOT || d->dtype != LATTICE_BF16 ||
      !dot_mfma_supported(d->n, d->dim))
    return 0;
  return al256((size_t)B * 16);
}

static size_t interact_ws(const lattice_interact_desc* d, int B) {
  if (d->kind == LATTICE_INTERACT_STACK) return stack_plan(stack_shape(d), B).total_bytes;
  if (d->kind != LATTICE_INTERACT_FM) return 0;
  return std::max(fm_mfma_bwd_workspace(d->n, d->rank), fm_bwd_workspace(d->n, d->rank));
}

static hipError_t interact_fwd_impl(const lattice_interact_desc* d, int B, const void* X,
                                    void* out, int64_t os, void* ws, hipStream_t s) {
  if (d->kind == LATTICE_INTERACT_STACK) {
    StackLayer Ls[LATTICE_MAX_LAYERS];
    stack_layers(d, Ls);
    return stack_fwd(stack_shape(d), Ls, B, X, out, os, ws, s);
  }
  if (d->kind == LATTICE_INTERACT_DOT) {
    if (dot_uses_mfma(d, X))
      return dot_mfma(true, X, B, d->n, d->dim, out, os, d->emit_slot0, nullptr, 0, nullptr, d->slot_mask, s);
    return dot_fwd(dt_of(d->dtype), X, B, d->n, d->dim, out, os, d->emit_slot0, s);
  }
  if (fm_uses_mfma(d, os))
    return fm_mfma(true, X, d->fm_W, B, d->n, d->dim, d->rank, out, os, d->emit_slot0, nullptr, 0,
                   nullptr, nullptr, nullptr, nullptr, nullptr, s);
  return fm_fwd(dt_of(d->dtype), X, d->fm_W, B, d->n, d->dim, d->rank, out, os, d->emit_slot0, s);
}

static hipError_t interact_bwd_impl(const lattice_interact_desc* d, int B, const void* X,
                                    const void* dout, int64_t ds, void* dX, void* ws,
                                    hipStream_t s) {
  if (d->kind == LATTICE_INTERACT_STACK) {
    StackLayer Ls[LATTICE_MAX_LAYERS];
    stack_layers(d, Ls);
    return stack_bwd(stack_shape(d), Ls, B, X, dout, ds, dX, ws, s);
  }
  if (d->kind == LATTICE_INTERACT_DOT) {
    if (dot_uses_mfma(d, X))
      return dot_mfma(false, X, B, d->n, d->dim, nullptr, 0, d->emit_slot0, dout, ds, dX, d->slot_mask, s);
    return dot_bwd(dt_of(d->dtype), X, B, d->n, d->dim, dout, ds, d->emit_slot0, dX, s);
  }
  if (fm_uses_mfma(d, ds))
    return fm_mfma(false, X, d->fm_W, B, d->n, d->dim, d->rank, nullptr, 0, d->emit_slot0, dout, ds,
                   nullptr, dX, nullptr, d->fm_dW, ws, s);
  return fm_bwd(dt_of(d->dtype), X, d->fm_W, B, d->n, d->dim, d->rank, dout, ds, d->emit_slot0,
                nullptr, dX, dt_of(d->dtype), d->fm_dW, ws, s);
}

extern "C" {

size_t lattice_interact_workspace(const lattice_interact_desc* desc, int32_t B) {
  return (desc && check_interact(desc, B) == LATTICE_OK) ? interact_ws(desc, B) : 0;
}

lattice_status lattice_interact_fwd(const lattice_interact_desc* desc, int32_t B, const void* X,
                                    void* out, int64_t out_stride, void* ws, size_t ws_bytes,
                                    void* stream) {
  lattice_status st = check_interact(desc, B);
  if (st != LATTICE_OK) return st;
  if (B == 0) return LATTICE_OK;
  REQUIRE(X && out, "null X/out");
  REQUIRE(out_stride >= interact_width(desc), "out_stride %lld < row width %lld",
          (long long)out_stride, (long long)interact_width(desc));
  const size_t need = desc->kind == LATTICE_INTERACT_STACK ? interact_ws(desc, B) : 0;
  if (ws_bytes < need || (need && !ws)) FAIL(LATTICE_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
  HIPRET(interact_fwd_impl(desc, B, X, out, out_stride, ws, strm(stream)));
  return LATTICE_OK;
}

lattice_status lattice_interact_state(const lattice_interact_desc* desc, int32_t B,
                                      lattice_stack_state* out) {
  REQUIRE(out, "null output");
  lattice_status st = check_interact(desc, B);
  if (st != LATTICE_OK) return st;
  for (int l = 0; l < LATTICE_MAX_LAYERS; ++l)
    out->P[l] = out->F[l] = out->H[l] = out->mean[l] = out->rstd[l] = out->Xn[l] = -1;
  if (desc->kind != LATTICE_INTERACT_STACK) return LATTICE_OK;
  const StackShape sh = stack_shape(desc);
  const StackPlan p = stack_plan(sh, B);
  for (int l = 0; l < sh.L; ++l) {
    out->P[l] = (int64_t)p.P[l];
    out->F[l] = (int64_t)p.F[l];
    out->H[l] = (int64_t)p.H[l];
    out->mean[l] = (int64_t)p.mean[l];
    out->rstd[l] = (int64_t)p.rstd[l];
    out->Xn[l] = l + 1 < sh.L ? (int64_t)p.Xn[l] : -1;
  }
  return LATTICE_OK;
}

lattice_status lattice_interact_bwd(const lattice_interact_desc* desc, int32_t B, const void* X,
                                    const void* d_out, int64_t d_out_stride, void* dX, void* ws,
                                    size_t ws_bytes, void* stream) {
  lattice_status st = check_interact(desc, B);
  if (st != LATTICE_OK) return st;
  if (desc->kind == LATTICE_INTERACT_FM) REQUIRE(desc->fm_dW, "FM backward needs fm_dW");
  if (desc->kind == LATTICE_INTERACT_STACK)
    for (int l = 0; l < desc->n_layers; ++l) {
      const lattice_stack_layer& L = desc->layers[l];
      REQUIRE(L.dW && L.dA && L.dgamma && (!L.C || L.dC), "STACK layer %d: null gradient buffer", l);
    }
  const size_t need = interact_ws(desc, B);
  if (ws_bytes < need || (need && !ws)) FAIL(LATTICE_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
  if (B == 0) {
    HIPRET(zero_interact_grads(desc, strm(stream)));
    return LATTICE_OK;
  }
  REQUIRE(X && d_out && dX, "null X/d_out/dX");
  REQUIRE(d_out_stride >= interact_width(desc), "d_out_stride too small");
  HIPRET(interact_bwd_impl(desc, B, X, d_out, d_out_stride, dX, ws, strm(stream)));
  return LATTICE_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// FP8 linear layers
// ---------------------------------------------------------------------------
extern "C" {

size_t lattice_fp8_quantize_workspace(void) { return fp8_quantize_workspace(); }

lattice_status lattice_fp8_quantize(const void* x, lattice_dtype x_dtype, int64_t rows, int64_t cols,
                                    int64_t ld, lattice_fp8_scaling scaling, uint8_t* q, int64_t ldq,
                                    float* scales, void* ws, size_t ws_bytes, void* stream) {
  REQUIRE(rows >= 0 && cols >= 0 && rows < ((int64_t)1 << 31) && cols < ((int64_t)1 << 31),
          "bad rows/cols");
  REQUIRE(x_dtype == LATTICE_F32 || x_dtype == LATTICE_BF16, "bad dtype");
  REQUIRE(scaling == LATTICE_FP8_ROWWISE || scaling == LATTICE_FP8_TENSORWISE, "bad scaling");
  REQUIRE(ld >= cols, "ld < cols");
  REQUIRE(ldq >= cols && ldq % 16 == 0, "ldq must be >= cols and a multiple of 16");
  if (rows == 0) return LATTICE_OK;
  REQUIRE(x && q && scales, "null x/q/scales");
  REQUIRE(((uintptr_t)q & 15) == 0, "q must be 16-byte aligned");
  if (scaling == LATTICE_FP8_TENSORWISE && (ws_bytes < fp8_quantize_workspace() || !ws))
    FAIL(LATTICE_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, fp8_quantize_workspace());
  HIPRET(fp8_quantize(x, dt_of(x_dtype), (int)rows, (int)cols, ld, scaling == LATTICE_FP8_ROWWISE, q,
                      ldq, scales, ws, strm(stream)));
  return LATTICE_OK;
}

lattice_status lattice_linear_fp8_fwd(const uint8_t* qA, int64_t lda, const float* sA,
                                      lattice_fp8_scaling a_scaling, const uint8_t* qW, int64_t ldw,
                                      const float* sW, lattice_fp8_scaling w_scaling,
                                      const float* bias, int32_t M, int32_t N, int32_t K,
                                      int32_t relu, int32_t fast_accum, void* Y,
                                      lattice_dtype y_dtype, int64_t ldy, void* stream) {
  REQUIRE(M >= 0 && N >= 0 && K >= 0, "negative size");
  REQUIRE(y_dtype == LATTICE_F32 || y_dtype == LATTICE_BF16, "bad output dtype");
  REQUIRE(a_scaling == LATTICE_FP8_ROWWISE || a_scaling == LATTICE_FP8_TENSORWISE, "bad a_scaling");
  REQUIRE(w_scaling == LATTICE_FP8_ROWWISE || w_scaling == LATTICE_FP8_TENSORWISE, "bad w_scaling");
  const int64_t kpad = ((int64_t)K + 15) / 16 * 16;
  REQUIRE(lda >= kpad && ldw >= kpad && lda % 16 == 0 && ldw % 16 == 0,
          "lda/ldw must be multiples of 16 and >= K rounded up to 16");
  REQUIRE(ldy >= N, "ldy < N");
  if ((int64_t)M * N == 0) return LATTICE_OK;
  REQUIRE(qA && sA && qW && sW && Y, "null operand");
  REQUIRE(((uintptr_t)qA & 15) == 0 && ((uintptr_t)qW & 15) == 0, "codes must be 16-byte aligned");
  HIPRET(gemm_fp8(qA, lda, sA, a_scaling == LATTICE_FP8_ROWWISE, qW, ldw, sW,
                  w_scaling == LATTICE_FP8_ROWWISE, bias, Y, dt_of(y_dtype), ldy, M, N, K,
                  relu != 0, fast_accum != 0, strm(stream)));
  return LATTICE_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// MLP + heads
// ---------------------------------------------------------------------------
static lattice_status check_mlp(const lattice_mlp_desc* d, int32_t B) {
  REQUIRE(d && d->layers, "null MLP descriptor");
  REQUIRE(B >= 0, "negative batch");
  REQUIRE(d->n_layers >= 1 && d->n_layers <= LATTICE_MAX_LAYERS, "n_layers %d outside 1..%d",
          d->n_layers, LATTICE_MAX_LAYERS);
  REQUIRE(d->dtype == LATTICE_F32 || d->dtype == LATTICE_BF16, "bad dtype");
  REQUIRE(d->act == LATTICE_ACT_RELU || d->act == LATTICE_ACT_SWISHRN ||
              d->act == LATTICE_ACT_HARDSWISHRN, "bad activation %d", (int)d->act);
  if (d->act != LATTICE_ACT_RELU) {
    REQUIRE(d->norm_block == 0 || d->norm_block == LATTICE_BLOCKNORM_COLS,
            "norm_block must be 0 or %d", LATTICE_BLOCKNORM_COLS);
    REQUIRE(d->norm_eps >= 0.f && d->norm_eps < INFINITY, "norm_eps must be finite and >= 0");
  }
  for (int i = 0; i < d->n_layers; ++i) {
    const lattice_linear& L = d->layers[i];
    REQUIRE(L.in_dim >= 1 && L.out_dim >= 1 && L.W, "layer %d: bad dims or null W", i);
    if (i > 0) REQUIRE(L.in_dim == d->layers[i - 1].out_dim, "layer %d: in_dim mismatch", i);
    if (swish_layer(d, i)) REQUIRE(L.gain, "layer %d: SwishRN needs gains", i);
  }
  if (d->tower_heads) {
    const lattice_linear& L = d->layers[d->n_layers - 1];
    REQUIRE(!d->relu_last, "tower heads need a linear last layer");
    REQUIRE(L.in_dim % L.out_dim == 0 && (L.in_dim / L.out_dim) % 8 == 0,
            "tower heads: in_dim must be out_dim x H with H a multiple of 8");
  }
  REQUIRE(d->n_domains >= 0, "negative n_domains");
  if (d->n_domains > 1) {
    REQUIRE(d->untied_layers >= 0 && d->untied_layers <= d->n_layers - (d->tower_heads ? 1 : 0),
            "untied_layers %d outside 0..%d", d->untied_layers, d->n_layers - (d->tower_heads ? 1 : 0));
  }
  return LATTICE_OK;
}


static int gate_of(const lattice_mlp_desc* d) {
  return d->act == LATTICE_ACT_SWISHRN ? GATE_SIGMOID : GATE_HARD;
}

// Where the SwishRN layers keep what the backward needs: per layer, the
// pre-activation, rho, and (backward) the gradient of the layer's output.
struct ActBufs {
  void* pre[LATTICE_MAX_LAYERS] = {};
  float* rinv[LATTICE_MAX_LAYERS] = {};
  void* gout[LATTICE_MAX_LAYERS] = {};
};

// Parameter untying (Section 3.3.4): samples grouped by domain, host
// offsets off[0..n] (off[0] = 0, off[n] = B); layers i < untied_layers hold
// n_domains parameter sets, stacked, and the samples of domain g use set g.
struct Domains {
  int n = 1;
  const int64_t* off = nullptr;
};

static bool untied(const lattice_mlp_desc* d, int i) {
  return d->n_domains > 1 && i < d->untied_layers;
}

// Host domain offsets: off[0] = 0, non-decreasing, off[n] = B.
static lattice_status check_domains(const lattice_mlp_desc* d, const int64_t* off, int B, Domains* dom) {
  dom->n = 1;
  dom->off = nullptr;
  if (d->n_domains <= 1 || d->untied_layers == 0) return LATTICE_OK;
  REQUIRE(off, "untied layers need domain offsets");
  REQUIRE(off[0] == 0 && off[d->n_domains] == B, "domain offsets must run from 0 to B = %d", B);
  for (int g = 0; g < d->n_domains; ++g) REQUIRE(off[g + 1] >= off[g], "domain offsets decrease at %d", g);
  dom->n = d->n_domains;
  dom->off = off;
  return LATTICE_OK;
}

// SwishRN statistic groups of layer i (columns of its rho rows)
static int rinv_cols(const lattice_mlp_desc* d, int i) {
  return swishrn_groups(d->layers[i].out_dim, d->norm_block);
}

// The MLP seen by the samples of domain g: every untied layer's parameters
// (and gradients) point at set g.
struct MlpView {
  lattice_mlp_desc d;
  lattice_linear L[LATTICE_MAX_LAYERS];
};

static void domain_view(const lattice_mlp_desc* d, int g, MlpView* v) {
  v->d = *d;
  const int64_t es = (int64_t)esize(d->dtype);
  for (int i = 0; i < d->n_layers; ++i) {
    lattice_linear L = d->layers[i];
    if (untied(d, i)) {
      const int64_t wn = w_elems(d, i), o = L.out_dim;
      L.W = (const char*)L.W + g * wn * es;
      if (L.b) L.b += g * o;
      if (L.dW) L.dW += g * wn;
      if (L.db) L.db += g * o;
      if (L.gain) L.gain += g * 2 * o;
      if (L.dgain) L.dgain += g * 2 * o;
    }
    v->L[i] = L;
  }
  v->d.layers = v->L;
}

static const void* row_at(const void* p, int64_t r0, int64_t ld, int64_t es) {
  return p ? (const char*)p + r0 * ld * es : nullptr;
}
static void* row_at(void* p, int64_t r0, int64_t ld, int64_t es) {
  return p ? (char*)p + r0 * ld * es : nullptr;
}

// Rows r0.. of the activations (storage dtype; a linear last layer's fp32
// logits) and of the SwishRN buffers.
struct RowView {
  const void* acts[LATTICE_MAX_LAYERS];
  void* wacts[LATTICE_MAX_LAYERS];
  ActBufs ab;
};

static void row_view(const lattice_mlp_desc* d, const void* const* acts, const int64_t* strides,
                     const ActBufs* ab, int64_t r0, RowView* v) {
  const int64_t es = (int64_t)esize(d->dtype);
  for (int i = 0; i < d->n_layers; ++i) {
    const bool logits = i == d->n_layers - 1 && !d->relu_last;
    const int64_t e = logits ? 4 : es;
    v->acts[i] = acts ? row_at(acts[i], r0, strides[i], e) : nullptr;
    v->wacts[i] = const_cast<void*>(v->acts[i]);
    const int64_t o = d->layers[i].out_dim;
    v->ab.pre[i] = ab ? row_at(ab->pre[i], r0, o, es) : nullptr;
    v->ab.rinv[i] = ab && ab->rinv[i] ? (float*)row_at(ab->rinv[i], r0, rinv_cols(d, i), 4) : nullptr;
    v->ab.gout[i] = ab ? row_at(ab->gout[i], r0, o, es) : nullptr;
  }
}

// f(desc, r0, rows) over the whole batch, or once per domain with that
// domain's parameters when `split` (segments of no samples are skipped).
template <typename F>
static hipError_t per_domain(const lattice_mlp_desc* d, const Domains* dom, bool split, int B, F&& f) {
  if (!split || !dom || dom->n <= 1) return f(d, (int64_t)0, B);
  for (int g = 0; g < dom->n; ++g) {
    const int64_t r0 = dom->off[g], rows = dom->off[g + 1] - r0;
    if (rows <= 0) continue;
    MlpView v;
    domain_view(d, g, &v);
    hipError_t e = f(&v.d, r0, (int)rows);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// split-K bound of the MLP backward products (the factor itself comes from
// gemm_splits' time estimate)
constexpr int MLP_MAX_SPLITS = 64;

static size_t mlp_bwd_ws(const lattice_mlp_desc* d, int B) {
  size_t s = 0;
  for (int i = 0; i < d->n_layers; ++i) {
    const lattice_linear& L = d->layers[i];
    GemmArgs g;
    g.dt = dt_of(d->dtype);
    g.max_splits = MLP_MAX_SPLITS;
    g.M = L.out_dim; g.N = L.in_dim; g.K = B;
    s = std::max(s, gemm_workspace(g));
    g.M = B; g.N = L.in_dim; g.K = L.out_dim;
    s = std::max(s, gemm_workspace(g));
    s = std::max(s, colsum_workspace(B, L.out_dim));
    if (swish_layer(d, i)) s = std::max(s, swishrn_gain_workspace(B, L.out_dim));
    if (tower_layer(d, i)) s = std::max(s, tower_wgrad_workspace(B, L.out_dim, L.in_dim / L.out_dim));
  }
  return al256(s);
}

static size_t mlp_gbuf_elems(const lattice_mlp_desc* d, int B) {
  int64_t w = 1;
  for (int i = 1; i < d->n_layers; ++i) w = std::max<int64_t>(w, d->layers[i].in_dim);
  w = std::max<int64_t>(w, d->layers[d->n_layers - 1].out_dim);
  return (size_t)w * B;
}

// Layer i's forward on B rows: A [B, in] -> C [B, out] (and the SwishRN
// buffers ab).  SwishRN layers: bf16 models with BlockNorm groups take the
// statistic in the GEMM's epilogue; otherwise the GEMM stores the
// pre-activation and a row kernel normalises it.
// The domains of an untied bf16 layer as the groups of one grouped GEMM (or
// null: the layer is tied, or the model fp32 -- then per domain).
static const Domains* gemm_groups(const lattice_mlp_desc* d, int i, const Domains* dom) {
  return (untied(d, i) && dom && dom->n > 1 && dom->n <= 16 && d->dtype == LATTICE_BF16) ? dom : nullptr;
}

static hipError_t mlp_forward_layer(const lattice_mlp_desc* d, int i, int B, const void* A,
                                    int64_t lda, void* C, int64_t ldc, const ActBufs* ab,
                                    hipStream_t s, const Domains* grp = nullptr) {
  const DType dt = dt_of(d->dtype);
  const lattice_linear& L = d->layers[i];
  const bool last = i == d->n_layers - 1;
  GemmArgs g;
  g.dt = dt;
  g.A = A; g.lda = lda;
  g.B = L.W; g.ldb = L.in_dim;
  g.C = C; g.ldc = ldc;
  g.c_dt = (last && !d->relu_last) ? DT_F32 : dt;
  g.M = B; g.N = L.out_dim; g.K = L.in_dim;
  g.bias = L.b;
  if (grp) {  // every domain's rows with its own W, b and gains, one launch
    g.ngroups = grp->n;
    g.goff = grp->off;
    g.gsB = (int64_t)L.out_dim * L.in_dim;
  }
  if (tower_layer(d, i)) {
    if (ldc != L.out_dim) {
      set_error("tower heads write contiguous logits");
      return hipErrorInvalidValue;
    }
    return tower_head_fwd(dt, A, lda, B, L.out_dim, L.in_dim / L.out_dim, L.W, L.b, (float*)C, s);
  }
  if (swish_layer(d, i)) {
    if (dt == DT_BF16 && d->norm_block == LATTICE_BLOCKNORM_COLS) {
      g.norm_gate = gate_of(d);
      g.gain = L.gain;
      g.eps = d->norm_eps;
      g.pre = ab->pre[i];
      g.ldp = L.out_dim;
      g.rinv = ab->rinv[i];
      g.nblk = cdiv(L.out_dim, LATTICE_BLOCKNORM_COLS);
      return gemm(g, nullptr, s);
    }
    g.C = ab->pre[i];
    g.ldc = L.out_dim;
    hipError_t e = gemm(g, nullptr, s);
    if (e != hipSuccess) return e;
    const int64_t es = (int64_t)esize(d->dtype);
    return per_domain(d, grp, grp != nullptr, B, [&](const lattice_mlp_desc* dv, int64_t r0, int rows) {
      const lattice_linear& Lv = dv->layers[i];
      return swishrn_fwd_rows(dt, row_at(ab->pre[i], r0, L.out_dim, es), L.out_dim, rows, L.out_dim,
                              d->norm_block, gate_of(d), Lv.gain, d->norm_eps, row_at(C, r0, ldc, es), ldc,
                              (float*)row_at(ab->rinv[i], r0, rinv_cols(d, i), 4), s);
    });
  }
  g.relu = (!last || d->relu_last) ? 1 : 0;
  return gemm(g, nullptr, s);  // forward GEMMs never split K
}

static hipError_t mlp_forward(const lattice_mlp_desc* d, int B, const void* in, int64_t in_stride,
                              void* const* acts, const int64_t* strides, const ActBufs* ab,
                              hipStream_t s, const Domains* dom = nullptr) {
  const int64_t es = (int64_t)esize(d->dtype);
  for (int i = 0; i < d->n_layers; ++i) {
    if (const Domains* grp = gemm_groups(d, i, dom)) {
      hipError_t e = mlp_forward_layer(d, i, B, i == 0 ? in : acts[i - 1], i == 0 ? in_stride : strides[i - 1],
                                       acts[i], strides[i], ab, s, grp);
      if (e != hipSuccess) return e;
      continue;
    }
    hipError_t e = per_domain(d, dom, untied(d, i), B, [&](const lattice_mlp_desc* dv, int64_t r0, int rows) {
      RowView v;
      row_view(dv, acts, strides, ab, r0, &v);
      const void* A = i == 0 ? row_at(in, r0, in_stride, es) : v.acts[i - 1];
      return mlp_forward_layer(dv, i, rows, A, i == 0 ? in_stride : strides[i - 1], v.wacts[i],
                               strides[i], &v.ab, s);
    });
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// FP8 forward of hidden ReLU layers (bf16 model): the input and every
// layer's weights quantised row-wise to e4m3 in one launch, then per layer
// the FP8 GEMM with bias and ReLU into the layer's bf16 activation, and the
// next layer's input quantised.  Workspace: codes of the widest input
// [B, ldq] and its scales (reused layer after layer), then each layer's
// weight codes [out, ldq] and scales.
static int64_t fp8_ldq(int cols) { return ((int64_t)cols + 15) / 16 * 16; }

struct Fp8MlpWs {
  uint8_t* qa;
  float* sa;
  uint8_t* qw[LATTICE_MAX_LAYERS];
  float* sw[LATTICE_MAX_LAYERS];
  size_t bytes;
};

static Fp8MlpWs fp8_mlp_ws(const lattice_mlp_desc* d, int B, void* ws) {
  int64_t kmax = 1;
  for (int i = 0; i < d->n_layers; ++i) kmax = std::max<int64_t>(kmax, fp8_ldq(d->layers[i].in_dim));
  Fp8MlpWs w{};
  char* base = (char*)ws;
  size_t o = 0;
  w.qa = (uint8_t*)(base + o); o += al256((size_t)B * kmax);
  w.sa = (float*)(base + o);   o += al256((size_t)B * 4);
  for (int i = 0; i < d->n_layers; ++i) {
    const lattice_linear& L = d->layers[i];
    w.qw[i] = (uint8_t*)(base + o); o += al256((size_t)L.out_dim * fp8_ldq(L.in_dim));
    w.sw[i] = (float*)(base + o);   o += al256((size_t)L.out_dim * 4);
  }
  w.bytes = o;
  return w;
}

static size_t fp8_mlp_workspace(const lattice_mlp_desc* d, int B) { return fp8_mlp_ws(d, B, nullptr).bytes; }

static hipError_t mlp_forward_fp8(const lattice_mlp_desc* d, int B, const void* in, int64_t in_stride,
                                  void* const* acts, const int64_t* strides, void* ws, int fast,
                                  hipStream_t s) {
  const Fp8MlpWs w = fp8_mlp_ws(d, B, ws);
  static_assert(LATTICE_MAX_LAYERS + 1 <= FP8_MAX_JOBS, "input and every weight in one launch");
  Fp8RowJob jobs[FP8_MAX_JOBS];
  int nj = 0;
  jobs[nj++] = Fp8RowJob{in, in_stride, B, d->layers[0].in_dim, w.qa, fp8_ldq(d->layers[0].in_dim), w.sa};
  for (int i = 0; i < d->n_layers; ++i) {
    const lattice_linear& L = d->layers[i];
    jobs[nj++] = Fp8RowJob{L.W, L.in_dim, L.out_dim, L.in_dim, w.qw[i], fp8_ldq(L.in_dim), w.sw[i]};
  }
  hipError_t e = fp8_quantize_rows(DT_BF16, jobs, nj, s);
  for (int i = 0; i < d->n_layers && e == hipSuccess; ++i) {
    const lattice_linear& L = d->layers[i];
    const int64_t ldq = fp8_ldq(L.in_dim);
    if (i > 0) {
      const Fp8RowJob a{acts[i - 1], strides[i - 1], B, L.in_dim, w.qa, ldq, w.sa};
      e = fp8_quantize_rows(DT_BF16, &a, 1, s);
      if (e != hipSuccess) break;
    }
    e = gemm_fp8(w.qa, ldq, w.sa, 1, w.qw[i], ldq, w.sw[i], 1, L.b, acts[i], DT_BF16, strides[i], B,
                 L.out_dim, L.in_dim, 1, fast, s);
  }
  return e;
}

// Weight and bias gradients of layer i: dW = gᵀ · in (fp32), db = Σ_b g.
static hipError_t mlp_layer_wgrad(const lattice_mlp_desc* d, int i, int B, const void* g,
                                  int64_t gs, const void* in_i, int64_t ld_in, void* ws,
                                  hipStream_t s, const Domains* grp = nullptr) {
  const lattice_linear& L = d->layers[i];
  const DType dt = dt_of(d->dtype);
  if (tower_layer(d, i)) {
    hipError_t e = tower_wgrad(dt, g, gs, in_i, ld_in, B, L.out_dim, L.in_dim / L.out_dim, L.dW, ws, s);
    if (e == hipSuccess && L.db) e = colsum(g, dt, gs, B, L.out_dim, L.db, ws, s);
    return e;
  }
  bool db_done = false;
  if (L.dW) {
    GemmArgs w;
    w.dt = dt;
    w.A = g; w.lda = gs; w.ta = 1;
    w.B = in_i; w.ldb = ld_in; w.tb = 1;
    w.C = L.dW; w.ldc = L.in_dim; w.c_dt = DT_F32;
    w.M = L.out_dim; w.N = L.in_dim; w.K = B;
    w.max_splits = MLP_MAX_SPLITS;
    if (grp) {  // every domain's samples into its own dW (and db), one launch
      w.ngroups = grp->n;
      w.goff = grp->off;
      w.gk = 1;
      w.gsC = (int64_t)L.out_dim * L.in_dim;
    }
    // bf16: db is the row sum of A = gᵀ, taken by the same GEMM
    if (dt == DT_BF16 && L.db) {
      w.rowsum = L.db;
      db_done = true;
    }
    hipError_t e = gemm(w, ws, s);
    if (e != hipSuccess) return e;
  }
  if (L.db && !db_done) return colsum(g, dt, gs, B, L.out_dim, L.db, ws, s);
  return hipSuccess;
}

// Input gradient of layer i: dst = (g · W) ⊙ [mask > 0] (mask: the layer's
// input activation, i.e. the previous layer's ReLU output; null: no mask).
static hipError_t mlp_layer_dgrad(const lattice_mlp_desc* d, int i, int B, const void* g,
                                  int64_t gs, void* dst, int64_t dst_ld, const void* mask,
                                  int64_t ldm, void* ws, hipStream_t s, const Domains* grp = nullptr) {
  const lattice_linear& L = d->layers[i];
  GemmArgs x;
  x.dt = dt_of(d->dtype);
  x.A = g; x.lda = gs;
  x.B = L.W; x.ldb = L.in_dim; x.tb = 1;
  x.C = dst; x.ldc = dst_ld; x.c_dt = x.dt;
  x.M = B; x.N = L.in_dim; x.K = L.out_dim;
  x.max_splits = MLP_MAX_SPLITS;
  if (grp) {  // every domain's rows with its own W, one launch
    x.ngroups = grp->n;
    x.goff = grp->off;
    x.gsB = (int64_t)L.out_dim * L.in_dim;
  }
  if (mask) {
    x.mask = mask;
    x.mask_dt = x.dt;
    x.ldm = ldm;
  }
  return gemm(x, ws, s);
}

// Gradient of layer j's pre-activation from the gradient of its output
// (layer j applies SwishRN): the row kernel of the SwishRN backward.
static hipError_t swish_back(const lattice_mlp_desc* d, int j, int B, const void* gout,
                             int64_t gout_ld, const ActBufs* ab, void* dst, int64_t dst_ld,
                             hipStream_t s) {
  const lattice_linear& L = d->layers[j];
  return swishrn_bwd_rows(dt_of(d->dtype), gout, gout_ld, ab->pre[j], L.out_dim, ab->rinv[j], B,
                          L.out_dim, d->norm_block, gate_of(d), L.gain, dst, dst_ld, s);
}

static hipError_t swish_gain_grad(const lattice_mlp_desc* d, int j, int B, const void* gout,
                                  int64_t gout_ld, const ActBufs* ab, void* ws, hipStream_t s) {
  const lattice_linear& L = d->layers[j];
  return swishrn_gain_grad(dt_of(d->dtype), gout, gout_ld, ab->pre[j], L.out_dim, ab->rinv[j], B,
                           L.out_dim, d->norm_block, gate_of(d), L.gain, L.dgain, ws, s);
}

// Gradient of layer i-1's pre-activation (i > 0) or of the MLP's input
// (i == 0) from g, the gradient of layer i's pre-activation: g W_i, then
// through layer i-1's activation (ReLU mask, or the SwishRN backward via its
// output gradient ab->gout[i-1]).
static hipError_t mlp_chain_step(const lattice_mlp_desc* d, int i, int B, const void* g, int64_t gs,
                                 const void* const* acts, const int64_t* strides, const ActBufs* ab,
                                 void* dst, int64_t dst_ld, void* ws, hipStream_t s) {
  if (tower_layer(d, i)) {
    const lattice_linear& L = d->layers[i];
    const DType dt = dt_of(d->dtype);
    const int T = L.out_dim, H = L.in_dim / L.out_dim;
    if (i > 0 && swish_layer(d, i - 1)) {
      hipError_t e = tower_head_dgrad(dt, g, gs, B, T, H, L.W, nullptr, 0, ab->gout[i - 1], L.in_dim, s);
      if (e != hipSuccess) return e;
      return swish_back(d, i - 1, B, ab->gout[i - 1], L.in_dim, ab, dst, dst_ld, s);
    }
    return tower_head_dgrad(dt, g, gs, B, T, H, L.W, i > 0 ? acts[i - 1] : nullptr,
                            i > 0 ? strides[i - 1] : 0, dst, dst_ld, s);
  }
  if (i > 0 && swish_layer(d, i - 1)) {
    const int64_t ldo = d->layers[i - 1].out_dim;
    hipError_t e = mlp_layer_dgrad(d, i, B, g, gs, ab->gout[i - 1], ldo, nullptr, 0, ws, s);
    if (e != hipSuccess) return e;
    return swish_back(d, i - 1, B, ab->gout[i - 1], ldo, ab, dst, dst_ld, s);
  }
  return mlp_layer_dgrad(d, i, B, g, gs, dst, dst_ld, i > 0 ? acts[i - 1] : nullptr,
                         i > 0 ? strides[i - 1] : 0, ws, s);
}

// The chain step of layer i (see mlp_chain_step) over the batch, per domain
// where layer i or the activation below it has untied parameters.
static hipError_t chain_step_all(const lattice_mlp_desc* d, const Domains* dom, int i, int B,
                                 const void* g, int64_t gs, const void* const* acts,
                                 const int64_t* strides, const ActBufs* ab, void* dst, int64_t dst_ld,
                                 void* ws, hipStream_t s) {
  const int64_t es = (int64_t)esize(d->dtype);
  if (const Domains* grp = gemm_groups(d, i, dom)) {
    // one grouped product for every domain's rows; then the activation
    // below (ReLU: in the product's epilogue; SwishRN: its row kernel, per
    // domain when that layer is untied)
    if (i > 0 && swish_layer(d, i - 1)) {
      const int64_t ldo = d->layers[i - 1].out_dim;
      hipError_t e = mlp_layer_dgrad(d, i, B, g, gs, ab->gout[i - 1], ldo, nullptr, 0, ws, s, grp);
      if (e != hipSuccess) return e;
      return per_domain(d, dom, untied(d, i - 1), B, [&](const lattice_mlp_desc* dv, int64_t r0, int rows) {
        RowView v;
        row_view(dv, nullptr, nullptr, ab, r0, &v);
        return swish_back(dv, i - 1, rows, v.ab.gout[i - 1], ldo, &v.ab, row_at(dst, r0, dst_ld, es), dst_ld, s);
      });
    }
    return mlp_layer_dgrad(d, i, B, g, gs, dst, dst_ld, i > 0 ? acts[i - 1] : nullptr,
                           i > 0 ? strides[i - 1] : 0, ws, s, grp);
  }
  const bool split = untied(d, i) || (i > 0 && untied(d, i - 1));
  return per_domain(d, dom, split, B, [&](const lattice_mlp_desc* dv, int64_t r0, int rows) {
    RowView v;
    row_view(dv, acts, strides, ab, r0, &v);
    return mlp_chain_step(dv, i, rows, row_at(g, r0, gs, es), gs, v.acts, strides, &v.ab,
                          row_at(dst, r0, dst_ld, es), dst_ld, ws, s);
  });
}

static hipError_t wgrad_all(const lattice_mlp_desc* d, const Domains* dom, int i, int B, const void* g,
                            int64_t gs, const void* in_i, int64_t ld_in, void* ws, hipStream_t s) {
  const int64_t es = (int64_t)esize(d->dtype);
  if (const Domains* grp = gemm_groups(d, i, dom))
    return mlp_layer_wgrad(d, i, B, g, gs, in_i, ld_in, ws, s, grp);
  return per_domain(d, dom, untied(d, i), B, [&](const lattice_mlp_desc* dv, int64_t r0, int rows) {
    return mlp_layer_wgrad(dv, i, rows, row_at(g, r0, gs, es), gs, row_at(in_i, r0, ld_in, es), ld_in,
                           ws, s);
  });
}

static hipError_t gain_grad_all(const lattice_mlp_desc* d, const Domains* dom, int j, int B,
                                const ActBufs* ab, void* ws, hipStream_t s) {
  return per_domain(d, dom, untied(d, j), B, [&](const lattice_mlp_desc* dv, int64_t r0, int rows) {
    RowView v;
    row_view(dv, nullptr, nullptr, ab, r0, &v);
    return swish_gain_grad(dv, j, rows, v.ab.gout[j], dv->layers[j].out_dim, &v.ab, ws, s);
  });
}

// g_last: gradient of the last layer's pre-activation (already taken through
// its activation where it has one).  Layer by layer (weights, gains of the
// layer below, then input gradient); hidden gradients alternate between
// gbuf0 and gbuf1.
static hipError_t mlp_backward(const lattice_mlp_desc* d, int B, const void* in, int64_t in_stride,
                               const void* const* acts, const int64_t* strides,
                               const void* g_last, int64_t g_last_stride, void* d_in,
                               int64_t d_in_stride, void* gbuf0, void* gbuf1, const ActBufs* ab,
                               void* ws, hipStream_t s, const Domains* dom = nullptr) {
  const void* g = g_last;
  int64_t gs = g_last_stride;
  for (int i = d->n_layers - 1; i >= 0; --i) {
    const lattice_linear& L = d->layers[i];
    const void* in_i = i == 0 ? in : acts[i - 1];
    const int64_t ld_in = i == 0 ? in_stride : strides[i - 1];
    hipError_t e = wgrad_all(d, dom, i, B, g, gs, in_i, ld_in, ws, s);
    if (e != hipSuccess) return e;
    if (i > 0 || d_in) {
      void* dst = i > 0 ? ((d->n_layers - 1 - i) % 2 == 0 ? gbuf0 : gbuf1) : d_in;
      const int64_t dst_ld = i > 0 ? L.in_dim : d_in_stride;
      e = chain_step_all(d, dom, i, B, g, gs, acts, strides, ab, dst, dst_ld, ws, s);
      if (e == hipSuccess && i > 0 && swish_layer(d, i - 1)) e = gain_grad_all(d, dom, i - 1, B, ab, ws, s);
      if (e != hipSuccess) return e;
      g = dst;
      gs = dst_ld;
    }
  }
  return hipSuccess;
}

// The gradient chain alone: hidden gradients into gl[i] (gradient of layer
// i's pre-activation, [B, out_i], i < n-1) and the input gradient into d_in
// (if any).
static hipError_t mlp_backward_data(const lattice_mlp_desc* d, int B, const void* const* acts,
                                    const int64_t* strides, const void* g_last,
                                    int64_t g_last_stride, void* d_in, int64_t d_in_stride,
                                    void* const* gl, const ActBufs* ab, void* ws, hipStream_t s,
                                    const Domains* dom = nullptr) {
  const void* g = g_last;
  int64_t gs = g_last_stride;
  for (int i = d->n_layers - 1; i >= 0; --i) {
    if (i == 0 && !d_in) break;
    void* dst = i > 0 ? gl[i - 1] : d_in;
    const int64_t dst_ld = i > 0 ? d->layers[i].in_dim : d_in_stride;
    hipError_t e = chain_step_all(d, dom, i, B, g, gs, acts, strides, ab, dst, dst_ld, ws, s);
    if (e != hipSuccess) return e;
    g = dst;
    gs = dst_ld;
  }
  return hipSuccess;
}

// Weight and bias gradients of every layer from the stored chain, and the
// gains of the hidden SwishRN layers from their stored output gradients.
static hipError_t mlp_backward_weights(const lattice_mlp_desc* d, int B, const void* in,
                                       int64_t in_stride, const void* const* acts,
                                       const int64_t* strides, const void* g_last,
                                       int64_t g_last_stride, void* const* gl, const ActBufs* ab,
                                       void* ws, hipStream_t s, const Domains* dom = nullptr) {
  for (int i = d->n_layers - 1; i >= 0; --i) {
    const void* g = i == d->n_layers - 1 ? g_last : gl[i];
    const int64_t gs = i == d->n_layers - 1 ? g_last_stride : d->layers[i].out_dim;
    hipError_t e = wgrad_all(d, dom, i, B, g, gs, i == 0 ? in : acts[i - 1],
                             i == 0 ? in_stride : strides[i - 1], ws, s);
    if (e == hipSuccess && i < d->n_layers - 1 && swish_layer(d, i)) e = gain_grad_all(d, dom, i, B, ab, ws, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// bf16, 8 elements per thread with 16-byte accesses (N, gs and as multiples
// of 8, pointers 16-byte aligned): the gradient masked by act > 0
__global__ __launch_bounds__(256) void relu_mask8_kernel(const bf16_t* __restrict__ g, int64_t gs,
                                                         const bf16_t* __restrict__ act, int64_t as,
                                                         int B, int N, bf16_t* __restrict__ out) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (i >= (int64_t)B * N) return;
  const int64_t r = i / N, c = i - r * N;
  const u32x4 gv = ldg16(g + r * gs + c), av = ldg16(act + r * as + c);
  u32x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t a = av[e], v = gv[e];
    const uint32_t lo = __uint_as_float(a << 16) > 0.f ? (v & 0xffffu) : 0u;
    const uint32_t hi = __uint_as_float(a & 0xffff0000u) > 0.f ? (v & 0xffff0000u) : 0u;
    o[e] = lo | hi;
  }
  stg16(out + i, o);
}

static hipError_t relu_mask(const void* g, int64_t gs, const void* act, int64_t as, int B, int N,
                            bool bf, void* out, hipStream_t s);

__global__ void relu_mask_kernel(const void* g, int64_t gs, const void* act, int64_t as, int B,
                                 int N, int bf, void* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)B * N) return;
  const int64_t r = i / N, c = i % N;
  if (bf) {
    const float a = bf2f(((const bf16_t*)act)[r * as + c]);
    const bf16_t v = ((const bf16_t*)g)[r * gs + c];
    ((bf16_t*)out)[i] = a > 0.f ? v : (bf16_t)0;
  } else {
    const float a = ((const float*)act)[r * as + c];
    ((float*)out)[i] = a > 0.f ? ((const float*)g)[r * gs + c] : 0.f;
  }
}

static hipError_t relu_mask(const void* g, int64_t gs, const void* act, int64_t as, int B, int N,
                            bool bf, void* out, hipStream_t s) {
  if (B == 0 || N == 0) return hipSuccess;
  const bool vec = bf && N % 8 == 0 && gs % 8 == 0 && as % 8 == 0 && ((uintptr_t)g & 15) == 0 &&
                   ((uintptr_t)act & 15) == 0 && ((uintptr_t)out & 15) == 0;
  if (vec)
    relu_mask8_kernel<<<cdiv((int64_t)B * N / 8, 256), 256, 0, s>>>((const bf16_t*)g, gs, (const bf16_t*)act,
                                                                   as, B, N, (bf16_t*)out);
  else
    relu_mask_kernel<<<cdiv((int64_t)B * N, 256), 256, 0, s>>>(g, gs, act, as, B, N, bf, out);
  return hipGetLastError();
}

static size_t mlp_heads_ws(const lattice_mlp_desc* d, int B) {
  const size_t g = al256(mlp_gbuf_elems(d, B) * esize(d->dtype));
  const int T = d->layers[d->n_layers - 1].out_dim;
  return mlp_bwd_ws(d, B) + 4 * g + al256(bce_workspace((int64_t)B * T));
}

// The caller's per-layer SwishRN buffers (lattice_linear.pre / rinv).
static lattice_status layer_bufs(const lattice_mlp_desc* d, int B, ActBufs* ab) {
  for (int i = 0; i < d->n_layers; ++i) {
    if (!swish_layer(d, i)) continue;
    const lattice_linear& L = d->layers[i];
    REQUIRE((L.pre && L.rinv) || B == 0, "layer %d: SwishRN needs pre and rinv buffers", i);
    ab->pre[i] = L.pre;
    ab->rinv[i] = L.rinv;
  }
  return LATTICE_OK;
}

extern "C" {

size_t lattice_mlp_heads_workspace(const lattice_mlp_desc* desc, int32_t B) {
  if (check_mlp(desc, B) != LATTICE_OK) return 0;
  return mlp_heads_ws(desc, B);
}

lattice_status lattice_mlp_heads_fwd(const lattice_mlp_desc* desc, int32_t B, const void* in,
                                     int64_t in_stride, void* const* acts,
                                     const int64_t* act_strides, const lattice_loss_desc* loss,
                                     void* ws, size_t ws_bytes, void* stream) {
  lattice_status st = check_mlp(desc, B);
  if (st != LATTICE_OK) return st;
  REQUIRE(acts && act_strides, "null acts");
  REQUIRE(in || B == 0, "null input");
  REQUIRE(in_stride >= desc->layers[0].in_dim, "in_stride too small");
  for (int i = 0; i < desc->n_layers; ++i)
    REQUIRE((acts[i] || B == 0) && act_strides[i] >= desc->layers[i].out_dim, "bad act %d", i);
  const int T = desc->layers[desc->n_layers - 1].out_dim;
  if (loss) {
    REQUIRE(!desc->relu_last, "the loss needs a linear last layer");
    REQUIRE(act_strides[desc->n_layers - 1] == T, "logits must be contiguous for the loss");
    REQUIRE(loss->labels && loss->mask && loss->loss && loss->d_logits, "null loss buffers");
    const size_t need = bce_workspace((int64_t)B * T);
    if (ws_bytes < need || !ws) FAIL(LATTICE_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
  }
  ActBufs ab;
  st = layer_bufs(desc, B, &ab);
  if (st != LATTICE_OK) return st;
  Domains dom;
  st = check_domains(desc, desc->domain_offsets, B, &dom);
  if (st != LATTICE_OK) return st;
  if (B > 0) HIPRET(mlp_forward(desc, B, in, in_stride, acts, act_strides, &ab, strm(stream), &dom));
  if (loss)
    HIPRET(bce((const float*)acts[desc->n_layers - 1], loss->labels, loss->mask, (int64_t)B * T,
               loss->loss, loss->d_logits, loss->d_logits_op, dt_of(desc->dtype), ws,
               strm(stream)));
  return LATTICE_OK;
}

lattice_status lattice_mlp_heads_bwd(const lattice_mlp_desc* desc, int32_t B, const void* in,
                                     int64_t in_stride, const void* const* acts,
                                     const int64_t* act_strides, const void* d_out,
                                     int64_t d_out_stride, void* d_in, int64_t d_in_stride,
                                     void* ws, size_t ws_bytes, void* stream) {
  lattice_status st = check_mlp(desc, B);
  if (st != LATTICE_OK) return st;
  REQUIRE(acts && act_strides, "null acts");
  const size_t need = mlp_heads_ws(desc, B);
  if (ws_bytes < need || !ws) FAIL(LATTICE_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
  if (B > 0) REQUIRE(in && d_out, "null in/d_out");
  const int L = desc->n_layers;
  const int T = desc->layers[L - 1].out_dim;
  REQUIRE(d_out_stride >= T, "d_out_stride too small");
  if (d_in) REQUIRE(d_in_stride >= desc->layers[0].in_dim, "d_in_stride too small");
  if (B == 0) {
    HIPRET(zero_mlp_grads(desc, strm(stream)));
    return LATTICE_OK;
  }
  ActBufs ab;
  st = layer_bufs(desc, B, &ab);
  if (st != LATTICE_OK) return st;
  Domains dom;
  st = check_domains(desc, desc->domain_offsets, B, &dom);
  if (st != LATTICE_OK) return st;
  char* p = (char*)ws;
  void* gemm_ws = p; p += mlp_bwd_ws(desc, B);
  const size_t g = al256(mlp_gbuf_elems(desc, B) * esize(desc->dtype));
  void* gb0 = p; p += g;
  void* gb1 = p; p += g;
  void* masked = p; p += g;
  void* gout = p;  // gradient of a hidden SwishRN layer's output (one at a time)
  for (int i = 0; i + 1 < L; ++i) ab.gout[i] = gout;
  const void* g_last = d_out;
  int64_t g_ld = d_out_stride;
  hipStream_t s = strm(stream);
  if (desc->relu_last && swish_layer(desc, L - 1)) {
    // the last layer's SwishRN backward from d_out (per domain if untied)
    const int64_t es = (int64_t)esize(desc->dtype);
    HIPRET(per_domain(desc, &dom, untied(desc, L - 1), B, [&](const lattice_mlp_desc* dv, int64_t r0, int rows) {
      RowView v;
      row_view(dv, nullptr, nullptr, &ab, r0, &v);
      const void* go = row_at(d_out, r0, d_out_stride, es);
      hipError_t e = swish_gain_grad(dv, L - 1, rows, go, d_out_stride, &v.ab, gemm_ws, s);
      if (e == hipSuccess) e = swish_back(dv, L - 1, rows, go, d_out_stride, &v.ab, row_at(masked, r0, T, es), T, s);
      return e;
    }));
    g_last = masked;
    g_ld = T;
  } else if (desc->relu_last) {
    if (relu_mask(d_out, d_out_stride, acts[L - 1], act_strides[L - 1], B, T, desc->dtype == LATTICE_BF16,
                  masked, s) != hipSuccess)
      FAIL(LATTICE_ERR_HIP, "relu mask launch failed");
    g_last = masked;
    g_ld = T;
  }
  HIPRET(mlp_backward(desc, B, in, in_stride, acts, act_strides, g_last, g_ld, d_in, d_in_stride,
                      gb0, gb1, &ab, gemm_ws, s, &dom));
  return LATTICE_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// whole step
// ---------------------------------------------------------------------------
struct Plan {
  lattice_step_layout L;
  int n, T, t_stride;
  size_t gbuf_top, gbuf_bot, scratch;
  // offset inside the dense scratch of the bottom backward's own part (it
  // runs on the side stream while the top weight gradients use the rest)
  size_t scratch_bottom;
  // per hidden layer i: gradient of its output [B, out_i]; g_masked: the
  // ReLU-masked gradient of the bottom MLP's output [B, dim]
  int64_t g_top[LATTICE_MAX_LAYERS], g_bot[LATTICE_MAX_LAYERS], g_masked;
};

static lattice_status check_model(const lattice_model_desc* m, int B) {
  REQUIRE(m, "null model");
  REQUIRE(B >= 0, "negative batch");
  REQUIRE(m->dtype == LATTICE_F32 || m->dtype == LATTICE_BF16, "bad dtype");
  REQUIRE(m->tables.dtype == m->dtype, "table dtype must equal the model dtype");
  lattice_status st = check_dim(m->tables.dim, m->dtype);
  if (st != LATTICE_OK) return st;
  const int d = m->tables.dim;
  const int n = m->num_features + (m->dense_in > 0 ? 1 : 0);
  REQUIRE(m->num_features >= 1, "need at least one feature");
  if (m->dense_in > 0) {
    st = check_mlp(&m->bottom, B);
    if (st != LATTICE_OK) return st;
    REQUIRE(m->bottom.relu_last == 1, "bottom MLP must apply ReLU on every layer");
    REQUIRE(m->bottom.layers[0].in_dim == m->dense_in, "bottom input width != dense_in");
    REQUIRE(m->bottom.layers[m->bottom.n_layers - 1].out_dim == d, "bottom output width != dim");
    REQUIRE(m->bottom.dtype == m->dtype, "bottom dtype");
    if (m->bottom.act != LATTICE_ACT_RELU)
      FAIL(LATTICE_ERR_UNSUPPORTED, "the step's bottom MLP uses ReLU (SwishRN: top MLP)");
    if (m->bottom.n_domains > 1 && m->bottom.untied_layers > 0)
      FAIL(LATTICE_ERR_UNSUPPORTED, "the step's bottom MLP is tied (untying: top MLP)");
  }
  st = check_mlp(&m->top, B);
  if (st != LATTICE_OK) return st;
  REQUIRE(m->top.relu_last == 0, "top MLP last layer must be linear");
  REQUIRE(m->top.dtype == m->dtype, "top dtype");
  st = check_interact(&m->interact, B);
  if (st != LATTICE_OK) return st;
  REQUIRE(m->interact.n == n && m->interact.dim == d && m->interact.dtype == m->dtype,
          "interaction shape/dtype mismatch");
  const int want_emit = (m->dense_in > 0 && m->interact.kind != LATTICE_INTERACT_STACK) ? 1 : 0;
  REQUIRE(m->interact.emit_slot0 == want_emit, "emit_slot0 must be %d", want_emit);
  REQUIRE(m->top.layers[0].in_dim == interact_width(&m->interact), "top input width %d != %lld",
          m->top.layers[0].in_dim, (long long)interact_width(&m->interact));
  if ((int64_t)B * n * d * (int64_t)esize(m->dtype) > (int64_t)UINT32_MAX)
    FAIL(LATTICE_ERR_UNSUPPORTED, "stacked vectors of %lld bytes exceed 4 GiB",
         (long long)B * n * d * (int64_t)esize(m->dtype));
  return LATTICE_OK;
}

static lattice_status make_plan(const lattice_model_desc* m, int B, int64_t nnz,
                                const lattice_step_opts* o, Plan* P) {
  lattice_status st = check_model(m, B);
  if (st != LATTICE_OK) return st;
  REQUIRE(nnz >= 0 && nnz < ((int64_t)1 << 31), "bad nnz");
  if (o && o->fp8_top) {
    REQUIRE(o->fp8_top == 1 || o->fp8_top == 2, "fp8_top must be 0, 1 or 2");
    if (m->dtype != LATTICE_BF16) FAIL(LATTICE_ERR_UNSUPPORTED, "fp8_top needs a bf16 model");
    if (m->top.act != LATTICE_ACT_RELU) FAIL(LATTICE_ERR_UNSUPPORTED, "fp8_top needs ReLU layers");
    if (m->top.n_domains > 1 && m->top.untied_layers > 0)
      FAIL(LATTICE_ERR_UNSUPPORTED, "fp8_top needs tied layers");
  }
  const size_t es = esize(m->dtype);
  const int d = m->tables.dim;
  P->n = m->interact.n;
  P->T = m->top.layers[m->top.n_layers - 1].out_dim;
  P->t_stride = (int)((m->top.layers[0].in_dim + 7) / 8 * 8);
  lattice_step_layout& L = P->L;
  for (int i = 0; i < LATTICE_MAX_LAYERS; ++i) L.bottom_act[i] = L.top_act[i] = -1;
  int64_t off = 0;
  auto take = [&](size_t bytes) { int64_t r = off; off += (int64_t)al256(bytes); return r; };
  L.X = take((size_t)B * P->n * d * es);
  L.t = take((size_t)B * P->t_stride * es);
  L.t_stride = P->t_stride;
  if (m->dense_in > 0)
    for (int i = 0; i + 1 < m->bottom.n_layers; ++i) L.bottom_act[i] = take((size_t)B * m->bottom.layers[i].out_dim * es);
  for (int i = 0; i + 1 < m->top.n_layers; ++i) L.top_act[i] = take((size_t)B * m->top.layers[i].out_dim * es);
  for (int i = 0; i < LATTICE_MAX_LAYERS; ++i) L.top_pre[i] = L.top_rinv[i] = L.top_gout[i] = -1;
  if (m->top.act != LATTICE_ACT_RELU)
    for (int i = 0; i + 1 < m->top.n_layers; ++i) {
      const int o = m->top.layers[i].out_dim;
      L.top_pre[i] = take((size_t)B * o * es);
      L.top_rinv[i] = take((size_t)B * swishrn_groups(o, m->top.norm_block) * 4);
      L.top_gout[i] = take((size_t)B * o * es);
    }
  L.logits = take((size_t)B * P->T * 4);
  L.d_logits = take((size_t)B * P->T * 4);
  L.d_logits_op = take((size_t)B * P->T * es);
  L.loss = take(4);
  L.d_t = take((size_t)B * P->t_stride * es);
  L.dX = take((size_t)B * P->n * d * es);
  for (int i = 0; i < LATTICE_MAX_LAYERS; ++i) P->g_top[i] = P->g_bot[i] = -1;
  for (int i = 0; i + 1 < m->top.n_layers; ++i) P->g_top[i] = take((size_t)B * m->top.layers[i].out_dim * es);
  P->g_masked = -1;
  if (m->dense_in > 0) {
    for (int i = 0; i + 1 < m->bottom.n_layers; ++i)
      P->g_bot[i] = take((size_t)B * m->bottom.layers[i].out_dim * es);
    P->g_masked = take((size_t)B * d * es);
  }
  for (int i = 0; i < LATTICE_MAX_LAYERS; ++i) L.top_grad[i] = L.bottom_grad[i] = -1;
  for (int i = 0; i + 1 < m->top.n_layers; ++i) L.top_grad[i] = P->g_top[i];
  L.top_grad[m->top.n_layers - 1] = L.d_logits_op;
  if (m->dense_in > 0) {
    for (int i = 0; i + 1 < m->bottom.n_layers; ++i) L.bottom_grad[i] = P->g_bot[i];
    L.bottom_grad[m->bottom.n_layers - 1] = P->g_masked;
  }
  const int64_t nn = nnz > 0 ? nnz : 1;
  L.unique_rows = take((size_t)nn * 4);
  L.seg_offsets = take((size_t)(nn + 1) * 4);
  L.sorted_bags = take((size_t)nn * 4);
  L.num_unique = take(4);
  L.grad_rows = (o && o->emit_grad_rows) ? take((size_t)nn * d * 4) : -1;
  size_t sc = 0;
  sc = std::max(sc, mlp_bwd_ws(&m->top, B));
  sc = std::max(sc, bce_workspace((int64_t)B * P->T));
  sc = std::max(sc, head_workspace(B));
  // the bottom backward's part follows the top's: the two run concurrently
  P->scratch_bottom = al256(sc);
  sc = P->scratch_bottom + (m->dense_in > 0 ? mlp_bwd_ws(&m->bottom, B) : 0);
  L.interact = take(interact_ws(&m->interact, B) + step_dot_mask_bytes(m, B));
  L.scratch = take(sc);
  L.scratch_bytes = (int64_t)sc;
  // the sparse gradient's scratch is its own: its first half may run on the
  // side stream while the dense stages use `scratch`
  const size_t sp = embbag_bwd_workspace(nnz, d, m->num_features);
  L.sparse = take(sp);
  L.sparse_bytes = (int64_t)sp;
  L.fp8 = -1;
  L.fp8_bytes = 0;
  if (o && o->fp8_top) {
    const size_t f8 = fp8_mlp_workspace(&m->top, B);
    L.fp8 = take(f8);
    L.fp8_bytes = (int64_t)f8;
  }
  L.total_bytes = off;
  return LATTICE_OK;
}

// The caller's side stream and its fork / join events (see lattice.h).
namespace {
struct SideStream {
  hipStream_t s = nullptr;
  // fork at the step's start, after the pooled lookups and after the
  // interaction backward; join of the bottom MLP's forward, of the sort and
  // run bookkeeping and of the dense weight gradients
  hipEvent_t fork_start = nullptr, fork_fwd = nullptr, fork_bwd = nullptr;
  hipEvent_t bottom_done = nullptr, sorted = nullptr, done = nullptr;
};
static_assert(LATTICE_STEP_SIDE_EVENTS == 6, "side events");
}  // namespace

extern "C" {

lattice_status lattice_step_plan(const lattice_model_desc* model, int32_t B, int64_t nnz,
                                 const lattice_step_opts* opts, lattice_step_layout* layout) {
  REQUIRE(layout, "null layout");
  Plan P;
  const int64_t cap = (opts && opts->nnz_capacity > nnz) ? opts->nnz_capacity : nnz;
  lattice_status st = make_plan(model, B, cap, opts, &P);
  if (st != LATTICE_OK) return st;
  *layout = P.L;
  return LATTICE_OK;
}

}  // extern "C"

// The step (forward_only = false) or its forward alone (lattice_forward).
static lattice_status step_impl(const lattice_model_desc* m, const lattice_batch_desc* batch,
                                const lattice_step_opts* opts, void* ws, size_t ws_bytes,
                                void* stream, bool forward_only) {
  REQUIRE(m && batch && opts, "null model/batch/opts");
  const int B = batch->bags.batch;
  REQUIRE(batch->bags.num_features == m->num_features, "batch features != model features");
  REQUIRE(opts->nnz_capacity == 0 || batch->bags.nnz <= opts->nnz_capacity,
          "batch nnz %lld exceeds nnz_capacity %lld", (long long)batch->bags.nnz,
          (long long)opts->nnz_capacity);
  Plan P;
  const int64_t cap = opts->nnz_capacity > 0 ? opts->nnz_capacity : batch->bags.nnz;
  lattice_status st = make_plan(m, B, cap, opts, &P);
  if (st != LATTICE_OK) return st;
  st = check_tables(&m->tables, &batch->bags);
  if (st != LATTICE_OK) return st;
  if (ws_bytes < (size_t)P.L.total_bytes || !ws)
    FAIL(LATTICE_ERR_WORKSPACE, "workspace %zu < %lld", ws_bytes, (long long)P.L.total_bytes);
  REQUIRE((batch->labels && batch->mask) || B == 0 || forward_only, "null labels/mask");
  Domains dom;
  st = check_domains(&m->top, batch->domain_offsets, B, &dom);
  if (st != LATTICE_OK) return st;
  if (m->dense_in > 0) REQUIRE(batch->dense || B == 0, "null dense input");
  if (opts->side_stream && opts->side_stream != stream) {
    REQUIRE(opts->side_events, "side_stream needs side_events");
    for (int i = 0; i < LATTICE_STEP_SIDE_EVENTS; ++i)
      REQUIRE(opts->side_events[i], "side_events[%d] is null", i);
  }
  if (B == 0 && forward_only) return LATTICE_OK;
  if (B == 0) {
    // sums over an empty batch: every parameter gradient, the loss and the
    // unique-row count are zero; the tables are untouched
    hipStream_t s0 = strm(stream);
    char* base0 = (char*)ws;
    if (m->dense_in > 0) HIPRET(zero_mlp_grads(&m->bottom, s0));
    HIPRET(zero_mlp_grads(&m->top, s0));
    HIPRET(zero_interact_grads(&m->interact, s0));
    HIPRET(zero_f32((float*)(base0 + P.L.loss), 1, s0));
    HIPRET(zero_f32((float*)(base0 + P.L.num_unique), 1, s0));
    return LATTICE_OK;
  }

  hipStream_t s = strm(stream);
  void* const* ev = opts->stage_events;
  auto stage_ev = [&](int i) -> void* const* { return ev ? ev + 2 * i : nullptr; };
  auto begin = [&](int i) -> hipError_t {
    return ev && ev[2 * i] ? hipEventRecord((hipEvent_t)ev[2 * i], s) : hipSuccess;
  };
  auto end = [&](int i) -> hipError_t {
    return ev && ev[2 * i + 1] ? hipEventRecord((hipEvent_t)ev[2 * i + 1], s) : hipSuccess;
  };
  char* base = (char*)ws;
  auto at = [&](int64_t o) -> void* { return o < 0 ? nullptr : base + o; };
  const lattice_step_layout& L = P.L;
  const DType dt = dt_of(m->dtype);
  const int d = m->tables.dim, n = P.n, T = P.T;
  const int s0 = m->dense_in > 0 ? 1 : 0;
  void* X = at(L.X);
  void* t = at(L.t);
  void* scratch = at(L.scratch);
  void* sparse = at(L.sparse);
  const int64_t nnz = batch->bags.nnz;
  // first half of the sparse gradient: sort of the forward's (row, bag)
  // pairs, unique rows and run offsets (stages EMBBAG_SORT and EMBBAG_RUNS)
  auto sparse_sort = [&](hipStream_t on) -> hipError_t {
    return embbag_bwd_sort(m->tables.row_base, local_rows_bound(&m->tables), batch->bags.offsets,
                           batch->bags.indices, m->num_features, B, nnz, d,
                           (int*)at(L.unique_rows), (int*)at(L.seg_offsets),
                           (int*)at(L.sorted_bags), (int*)at(L.num_unique), sparse, on,
                           stage_ev(LATTICE_STAGE_EMBBAG_SORT));
  };

  SideStream side_;
  SideStream* side = nullptr;
  if (opts->side_stream && strm(opts->side_stream) != s) {
    side_.s = strm(opts->side_stream);
    hipEvent_t* evs[LATTICE_STEP_SIDE_EVENTS] = {&side_.fork_start, &side_.fork_fwd, &side_.fork_bwd,
                                                 &side_.bottom_done, &side_.sorted, &side_.done};
    for (int i = 0; i < LATTICE_STEP_SIDE_EVENTS; ++i) *evs[i] = (hipEvent_t)opts->side_events[i];
    side = &side_;
  }
  // 2. bottom MLP -> slot 0 of X.  It needs only the dense input, so with the
  // side stream it runs there beside the pooled lookups (latency-bound small
  // GEMMs next to a bandwidth-bound gather); slot 0 of a row is its own
  // cache lines, which the lookups do not write.
  void* bacts[LATTICE_MAX_LAYERS];
  int64_t bstr[LATTICE_MAX_LAYERS];
  auto bottom_forward = [&](hipStream_t on) -> hipError_t {
    if (ev && ev[2 * LATTICE_STAGE_BOTTOM_FWD])
      HIP_TRY(hipEventRecord((hipEvent_t)ev[2 * LATTICE_STAGE_BOTTOM_FWD], on));
    if (m->dense_in > 0) {
      const int nb = m->bottom.n_layers;
      for (int i = 0; i + 1 < nb; ++i) {
        bacts[i] = at(L.bottom_act[i]);
        bstr[i] = m->bottom.layers[i].out_dim;
      }
      bacts[nb - 1] = X;
      bstr[nb - 1] = (int64_t)n * d;
      const ActBufs none;
      HIP_TRY(mlp_forward(&m->bottom, B, batch->dense, m->dense_in, bacts, bstr, &none, on));
    }
    if (ev && ev[2 * LATTICE_STAGE_BOTTOM_FWD + 1])
      HIP_TRY(hipEventRecord((hipEvent_t)ev[2 * LATTICE_STAGE_BOTTOM_FWD + 1], on));
    return hipSuccess;
  };
  const bool bottom_on_side = side && m->dense_in > 0;
  if (bottom_on_side) {
    HIPRET(hipEventRecord(side->fork_start, s));
    HIPRET(hipStreamWaitEvent(side->s, side->fork_start, 0));
    HIPRET(bottom_forward(side->s));
    HIPRET(hipEventRecord(side->bottom_done, side->s));
  }
  // 1. pooled lookups -> embedding slots of X
  HIPRET(begin(LATTICE_STAGE_EMBBAG_FWD));
  HIPRET(embbag_fwd(m->tables.data, dt, d, m->tables.row_base, batch->bags.offsets,
                    batch->bags.indices, m->num_features, B, m->pool == LATTICE_POOL_MEAN, X, dt,
                    n, s0, s));
  HIPRET(end(LATTICE_STAGE_EMBBAG_FWD));
  // fork: the sort and run bookkeeping go to the side stream, overlapping
  // the dense stages
  if (side && !forward_only) {
    HIPRET(hipEventRecord(side->fork_fwd, s));
    HIPRET(hipStreamWaitEvent(side->s, side->fork_fwd, 0));
    HIPRET(sparse_sort(side->s));
    HIPRET(hipEventRecord(side->sorted, side->s));
  }
  if (bottom_on_side) HIPRET(hipStreamWaitEvent(s, side->bottom_done, 0));
  else HIPRET(bottom_forward(s));
  // 3. interaction -> top input t = [X[:,0,:], interaction]
  HIPRET(begin(LATTICE_STAGE_INTERACT_FWD));
  lattice_interact_desc idesc = m->interact;
  if (step_dot_mask_bytes(m, B)) {
    // DOT with absent features: the slots whose bag is empty are zero
    // vectors, which the forward skips
    idesc.slot_mask = (const uint32_t*)at(L.interact);
    HIPRET(dot_slot_mask(batch->bags.offsets, m->num_features, B, s0, m->dense_in > 0,
                         (uint32_t*)at(L.interact), s));
  }
  HIPRET(interact_fwd_impl(&idesc, B, X, t, P.t_stride, at(L.interact), s));
  HIPRET(end(LATTICE_STAGE_INTERACT_FWD));
  // 4. top MLP -> logits; 5. masked BCE.  bf16 models with at most 64 heads
  // run the last layer as the fused heads: its forward with the loss
  // partials, then dz, the loss and the last layer's input gradient (which
  // starts the gradient chain of 6.) in the loss stage.
  HIPRET(begin(LATTICE_STAGE_TOP_FWD));
  const int nt = m->top.n_layers;
  void* tacts[LATTICE_MAX_LAYERS];
  int64_t tstr[LATTICE_MAX_LAYERS];
  for (int i = 0; i + 1 < nt; ++i) {
    tacts[i] = at(L.top_act[i]);
    tstr[i] = m->top.layers[i].out_dim;
  }
  tacts[nt - 1] = at(L.logits);
  tstr[nt - 1] = T;
  void* gtop[LATTICE_MAX_LAYERS];
  for (int i = 0; i < LATTICE_MAX_LAYERS; ++i) gtop[i] = at(P.g_top[i]);
  ActBufs tab;  // SwishRN hidden layers: pre-activations, statistics, output gradients
  for (int i = 0; i < LATTICE_MAX_LAYERS; ++i) {
    tab.pre[i] = at(L.top_pre[i]);
    tab.rinv[i] = (float*)at(L.top_rinv[i]);
    tab.gout[i] = at(L.top_gout[i]);
  }
  const bool top_swish = m->top.act != LATTICE_ACT_RELU;
  const lattice_linear& head = m->top.layers[nt - 1];
  const void* head_in = nt > 1 ? tacts[nt - 2] : t;
  const int64_t head_ld = nt > 1 ? tstr[nt - 2] : P.t_stride;
  const bool fused_heads = dt == DT_BF16 && !m->top.tower_heads &&
                           head_fusable(T, head.in_dim, head_in, head_ld, head.W);
  lattice_mlp_desc hidden = m->top;  // the layers before the heads
  hidden.n_layers = nt - 1;
  hidden.relu_last = 1;
  if (fused_heads) {
    if (nt > 1 && opts->fp8_top)
      HIPRET(mlp_forward_fp8(&hidden, B, t, P.t_stride, tacts, tstr, at(L.fp8), opts->fp8_top == 2, s));
    else if (nt > 1)
      HIPRET(mlp_forward(&hidden, B, t, P.t_stride, tacts, tstr, &tab, s, &dom));
    HIPRET(head_fwd((const bf16_t*)head_in, head_ld, B, head.in_dim, (const bf16_t*)head.W, head.b,
                    T, forward_only ? nullptr : batch->labels, forward_only ? nullptr : batch->mask,
                    (float*)at(L.logits), scratch, s));
  } else {
    if (opts->fp8_top) FAIL(LATTICE_ERR_UNSUPPORTED, "fp8_top needs the fused bf16 heads (<= 64 objectives)");
    HIPRET(mlp_forward(&m->top, B, t, P.t_stride, tacts, tstr, &tab, s, &dom));
  }
  HIPRET(end(LATTICE_STAGE_TOP_FWD));
  // the forward alone ends here (a bottom MLP on the side stream was joined
  // before the interaction)
  if (forward_only) return LATTICE_OK;
  HIPRET(begin(LATTICE_STAGE_LOSS));
  if (fused_heads) {
    // the heads' input gradient: masked by the ReLU, or (SwishRN) the
    // gradient of the last hidden layer's output, taken through the SwishRN
    // backward at the start of the top backward
    void* g_head = nt > 1 ? (top_swish ? tab.gout[nt - 2] : gtop[nt - 2]) : at(L.d_t);
    const int64_t g_ld = nt > 1 ? head.in_dim : P.t_stride;
    HIPRET(head_bwd((const float*)at(L.logits), batch->labels, batch->mask, B, T,
                    (const bf16_t*)head.W, head.in_dim,
                    nt > 1 && !top_swish ? (const bf16_t*)head_in : nullptr, head_ld,
                    (float*)at(L.loss), (float*)at(L.d_logits), (bf16_t*)at(L.d_logits_op),
                    (bf16_t*)g_head, g_ld, scratch, s));
  } else {
    HIPRET(bce((const float*)at(L.logits), batch->labels, batch->mask, (int64_t)B * T,
               (float*)at(L.loss), (float*)at(L.d_logits), at(L.d_logits_op), dt, scratch, s));
  }
  HIPRET(end(LATTICE_STAGE_LOSS));
  // 6. top backward, gradient chain only -> d_t (weight gradients: 8.)
  HIPRET(begin(LATTICE_STAGE_TOP_BWD));
  if (fused_heads) {
    if (nt > 1 && top_swish) {
      const int64_t es = (int64_t)esize(m->dtype);
      HIPRET(per_domain(&hidden, &dom, untied(&hidden, nt - 2), B,
                        [&](const lattice_mlp_desc* dv, int64_t r0, int rows) {
                          RowView v;
                          row_view(dv, nullptr, nullptr, &tab, r0, &v);
                          return swish_back(dv, nt - 2, rows, v.ab.gout[nt - 2], head.in_dim, &v.ab,
                                            row_at(gtop[nt - 2], r0, head.in_dim, es), head.in_dim, s);
                        }));
    }
    if (nt > 1)
      HIPRET(mlp_backward_data(&hidden, B, tacts, tstr, gtop[nt - 2], head.in_dim, at(L.d_t),
                               P.t_stride, gtop, &tab, scratch, s, &dom));
  } else {
    HIPRET(mlp_backward_data(&m->top, B, tacts, tstr, at(L.d_logits_op), T, at(L.d_t), P.t_stride,
                             gtop, &tab, scratch, s, &dom));
  }
  HIPRET(end(LATTICE_STAGE_TOP_BWD));
  // 7. interaction backward -> dX (slot 0 gets d_t[:, :d] added, then the bottom ReLU mask)
  HIPRET(begin(LATTICE_STAGE_INTERACT_BWD));
  void* dX = at(L.dX);
  HIPRET(interact_bwd_impl(&idesc, B, X, at(L.d_t), P.t_stride, dX, at(L.interact), s));
  HIPRET(end(LATTICE_STAGE_INTERACT_BWD));
  // 8./9. The bottom backward and the weight gradients of the top MLP need
  // nothing the sparse gradient writes.  The top weight gradients run on the
  // caller's stream before the segmented reduction (beside the reduction they
  // were starved of compute units: 0.59 ms against 0.17 ms alone), the
  // bottom backward on the side stream beside them and the reduction, with a
  // scratch part of its own.  (Forking them before the interaction backward
  // measured no faster and costs one more cross-stream event.)
  hipStream_t ws_stream = s;
  if (side) {
    HIPRET(hipEventRecord(side->fork_bwd, s));
    HIPRET(hipStreamWaitEvent(side->s, side->fork_bwd, 0));
    ws_stream = side->s;
  }
  auto wbegin = [&](int i) -> hipError_t {
    return ev && ev[2 * i] ? hipEventRecord((hipEvent_t)ev[2 * i], ws_stream) : hipSuccess;
  };
  auto wend = [&](int i) -> hipError_t {
    return ev && ev[2 * i + 1] ? hipEventRecord((hipEvent_t)ev[2 * i + 1], ws_stream) : hipSuccess;
  };
  // 9. bottom backward (gradient of the post-ReLU output, masked by slot 0 > 0)
  HIPRET(wbegin(LATTICE_STAGE_BOTTOM_BWD));
  if (m->dense_in > 0) {
    void* masked = at(P.g_masked);
    if (relu_mask(dX, (int64_t)n * d, X, (int64_t)n * d, B, d, dt == DT_BF16, masked, ws_stream) != hipSuccess)
      FAIL(LATTICE_ERR_HIP, "relu mask launch failed");
    void* gbot[LATTICE_MAX_LAYERS];
    for (int i = 0; i < LATTICE_MAX_LAYERS; ++i) gbot[i] = at(P.g_bot[i]);
    const ActBufs none;
    void* bscratch = (char*)scratch + P.scratch_bottom;
    HIPRET(mlp_backward_data(&m->bottom, B, bacts, bstr, masked, d, nullptr, 0, gbot, &none, bscratch,
                             ws_stream));
    HIPRET(mlp_backward_weights(&m->bottom, B, batch->dense, m->dense_in, bacts, bstr, masked, d,
                                gbot, &none, bscratch, ws_stream));
  }
  HIPRET(wend(LATTICE_STAGE_BOTTOM_BWD));
  HIPRET(begin(LATTICE_STAGE_TOP_WGRAD));
  HIPRET(mlp_backward_weights(&m->top, B, t, P.t_stride, tacts, tstr, at(L.d_logits_op), T, gtop,
                              &tab, scratch, s, &dom));
  HIPRET(end(LATTICE_STAGE_TOP_WGRAD));
  // 10. row-coalesced embedding gradient (+ row-sparse SGD) once the sort is done
  if (side) {
    HIPRET(hipEventRecord(side->done, side->s));
    HIPRET(hipStreamWaitEvent(s, side->sorted, 0));
  } else {
    HIPRET(sparse_sort(s));
  }
  HIPRET(embbag_bwd_apply(batch->bags.offsets, m->num_features, B, nnz,
                          m->pool == LATTICE_POOL_MEAN, dX, dt, n, s0, d,
                          (const int*)at(L.unique_rows), (const int*)at(L.seg_offsets),
                          (const int*)at(L.sorted_bags), (float*)at(L.grad_rows), m->tables.data,
                          dt, opts->lr_tables, sparse, s, stage_ev(LATTICE_STAGE_EMBBAG_REDUCE)));
  // join: the caller's stream passes this point after all of the step's work
  if (side) HIPRET(hipStreamWaitEvent(s, side->done, 0));
  return LATTICE_OK;
}


extern "C" {

lattice_status lattice_step(const lattice_model_desc* m, const lattice_batch_desc* batch,
                            const lattice_step_opts* opts, void* ws, size_t ws_bytes,
                            void* stream) {
  return step_impl(m, batch, opts, ws, ws_bytes, stream, false);
}

lattice_status lattice_forward(const lattice_model_desc* m, const lattice_batch_desc* batch,
                               const lattice_step_opts* opts, void* ws, size_t ws_bytes,
                               void* stream) {
  return step_impl(m, batch, opts, ws, ws_bytes, stream, true);
}

}  // extern "C"
