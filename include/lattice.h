/*
 * lattice.h -- C ABI of the MI355X (gfx950) training-step library for the
 * sparse-dense core of the Lattice Network (Meta Lattice, arXiv 2512.09200).
 *
 * One training step of that core is: pooled embedding lookups over jagged
 * multi-hot categorical features (Section 3.3.1), the dense-feature MLP
 * (Section 3.3.1), the pairwise feature interaction -- dot-product Gram, the
 * factorization-machine block, or a stack of FM blocks with linear
 * compression, residual and LayerNorm (the DHEN/Wukong fusion block,
 * Section 3.3.2) -- the task modules with one logit per objective
 * (Section 3.3.3), the masked multi-objective loss (impressions train only
 * their routed heads, Section 3.2.1), and the backward pass including the
 * row-coalesced embedding gradient and a row-sparse SGD update of the tables.
 *
 * Conventions shared by every entry point
 *  - Pointers are DEVICE pointers unless marked "host".  Every buffer is owned
 *    by the caller; the library never allocates or frees device memory.
 *    Scratch memory is a caller-provided workspace whose size the matching
 *    *_workspace / lattice_step_plan call reports.
 *  - Layouts are row-major and contiguous unless a row stride (in elements)
 *    is given.  Weights are [out, in].
 *  - Storage dtype: LATTICE_F32 keeps every tensor in fp32.  LATTICE_BF16
 *    stores tables, weights, activations and activation gradients (all GEMM
 *    operands) in bf16, rounded to nearest even from fp32 accumulators;
 *    biases, LayerNorm gains, logits, the loss and all parameter gradients are
 *    fp32 (mixed precision with bf16 GEMMs and fp32 normalisation,
 *    Section 3.5.2).
 *  - `stream` is a hipStream_t (NULL = default stream).  All work is enqueued
 *    on it in order; nothing synchronises except lattice_validate_batch.
 *  - Results are deterministic: identical inputs give bitwise-identical
 *    outputs (no floating-point atomics anywhere).
 *  - Every function returns a lattice_status; nothing aborts or prints.
 *    Arguments are checked before anything is launched; on failure
 *    lattice_last_error() holds a message (thread-local).  The hot path does
 *    NOT bounds-check embedding indices: out-of-range indices give undefined
 *    results; lattice_validate_batch checks a batch.
 *  - B = 0 or nnz = 0 are valid and produce the mathematically defined
 *    (zero / empty) results.
 */
#ifndef LATTICE_H_
#define LATTICE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LATTICE_ABI_VERSION 10
#define LATTICE_MAX_LAYERS 8

typedef enum {
  LATTICE_OK = 0,
  LATTICE_ERR_INVALID_ARG = 1,  /* null pointer, negative or inconsistent size */
  LATTICE_ERR_UNSUPPORTED = 2,  /* valid but not supported (dim, dtype, size limits) */
  LATTICE_ERR_WORKSPACE = 3,    /* workspace too small */
  LATTICE_ERR_BAD_INPUT = 4,    /* malformed batch (lattice_validate_batch) */
  LATTICE_ERR_HIP = 5           /* a HIP call or kernel launch failed */
} lattice_status;

typedef enum { LATTICE_F32 = 0, LATTICE_BF16 = 1 } lattice_dtype;
typedef enum { LATTICE_POOL_SUM = 0, LATTICE_POOL_MEAN = 1 } lattice_pool;
typedef enum {
  LATTICE_INTERACT_DOT = 0,    /* pairwise dot products, strict upper triangle */
  LATTICE_INTERACT_FM = 1,     /* factorization-machine block X (X^T W) */
  LATTICE_INTERACT_STACK = 2   /* stacked FM -> linear -> residual -> LayerNorm */
} lattice_interact_kind;

/* ------------------------------------------------------------------------ */
/* Jagged categorical batch and embedding tables (Section 3.3.1)            */
/* ------------------------------------------------------------------------ */

/* Feature-major jagged batch: bag f*B+b holds the indices of feature f for
 * sample b at positions offsets[f*B+b] .. offsets[f*B+b+1]-1.  Indices are
 * table-local row ids.  An empty bag is a feature the record does not carry
 * (zero-padded in the unified dataset, Section 3.2) and pools to zero. */
typedef struct {
  int32_t num_features;     /* F >= 0 */
  int32_t batch;            /* B >= 0 */
  const int32_t* offsets;   /* device [F*B+1], offsets[0] = 0, non-decreasing */
  const int32_t* indices;   /* device [nnz] */
  int64_t nnz;              /* host copy of offsets[F*B]; < 2^31 */
} lattice_jagged;

/* All tables stacked in one buffer; table f occupies global rows
 * row_base[f] .. row_base[f+1]-1 (row_base non-decreasing).  Embedding
 * dimension d is uniform across features (Section 3.3.1). */
typedef struct {
  void* data;                /* device [total_rows, dim], dtype */
  lattice_dtype dtype;
  int32_t dim;               /* d: multiple of 8, <= 256 */
  int64_t total_rows;        /* < 2^31 */
  const int64_t* row_base;   /* device [F+1] */
  int64_t max_rows;          /* rows of the largest table, or 0 (unknown: total_rows
                                is used).  The backward sorts each feature's lookups
                                by their row within its table, so its cost grows with
                                the bits of this bound.  Must be >= every table's rows
                                (lattice_validate_batch checks it). */
} lattice_tables;

/* Pooled lookup: X[b, first_slot+f, :] = sum (or mean) over j in bag(f,b) of
 * table row row_base[f] + indices[j], accumulated in fp32, stored in x_dtype.
 * X is [B, n_slots, dim]; slots outside first_slot .. first_slot+F-1 are not
 * touched.  Errors: INVALID_ARG (nulls, first_slot+F > n_slots), UNSUPPORTED
 * (dim), HIP. */
lattice_status lattice_embbag_fwd(const lattice_tables* tables, const lattice_jagged* bags,
                                  lattice_pool pool, void* X, lattice_dtype x_dtype,
                                  int32_t n_slots, int32_t first_slot, void* stream);

/* Row-coalesced sparse gradient of the pooled lookup, deterministic
 * (sort-by-row segmented reduction, no atomics). */
typedef struct {
  int32_t* unique_rows;  /* device [nnz]: global rows that occur, ascending; first *num_unique valid */
  int32_t* seg_offsets;  /* device [nnz+1]: run start of each unique row in sorted order; [num_unique] = nnz */
  int32_t* sorted_bags;  /* device [nnz]: bag id f*B+b of each occurrence, by (row, position) */
  int32_t* num_unique;   /* device [1] */
  float* grad_rows;      /* device [nnz, dim] fp32 or NULL: G[u] = sum of dX over row u's occurrences */
} lattice_sparse_grad;

size_t lattice_embbag_bwd_workspace(const lattice_tables* tables, const lattice_jagged* bags);

/* G[u] = sum over occurrences j of global row unique_rows[u] of
 * dX[b(j), first_slot+f(j), :] (divided by the bag length for mean pooling),
 * summed in fp32 in a fixed order.  If lr != 0 the occurring rows of
 * tables->data are updated in place: E[r] <- round(E[r] - lr * G[r]); other
 * rows are untouched.  dX is [B, n_slots, dim] in dx_dtype.  Errors:
 * INVALID_ARG, UNSUPPORTED (dim, total_rows >= 2^31, dX larger than 4 GiB),
 * WORKSPACE, HIP. */
lattice_status lattice_embbag_bwd(const lattice_tables* tables, const lattice_jagged* bags,
                                  lattice_pool pool, const void* dX, lattice_dtype dx_dtype,
                                  int32_t n_slots, int32_t first_slot,
                                  const lattice_sparse_grad* out, float lr,
                                  void* ws, size_t ws_bytes, void* stream);

/* The same computation as lattice_embbag_bwd, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving or
 * training loops, harnesses that forbid allocation): no workspace argument
 * and no hipMalloc / hipFree or other allocating call.  The scratch lives in
 * one device array of LATTICE_NOALLOC_SCRATCH_BYTES per GPU, part of the
 * library's code object, held until the process ends; its address is looked
 * up once per device on the first call there.  Every call on a GPU shares
 * that GPU's array: calls that overlap on one GPU (concurrent streams or
 * threads) race and give undefined results; calls ordered on one stream are
 * fine (the kernels clear what they need).  Errors: as lattice_embbag_bwd,
 * plus UNSUPPORTED when the batch needs more scratch than the array holds
 * (lattice_embbag_bwd_workspace(...) > LATTICE_NOALLOC_SCRATCH_BYTES: about
 * 16.1M lookups at dim 128 and 64 features) and HIP if the address lookup
 * fails. */
#define LATTICE_NOALLOC_SCRATCH_BYTES (256u << 20)
lattice_status lattice_embbag_bwd_noalloc(const lattice_tables* tables, const lattice_jagged* bags,
                                          lattice_pool pool, const void* dX, lattice_dtype dx_dtype,
                                          int32_t n_slots, int32_t first_slot,
                                          const lattice_sparse_grad* out, float lr, void* stream);

/* Synchronous check of a batch against the tables: offsets[0] == 0,
 * non-decreasing, offsets[F*B] == nnz, 0 <= indices[j] < rows of its
 * table, and (if max_rows != 0) no table has more than max_rows rows.
 * Returns BAD_INPUT with *first_bad (host) = first bad offset position (as
 * -1 - position), first bad index position, or -1 - (F*B + 1 + f) for a
 * table f larger than max_rows. */
lattice_status lattice_validate_batch(const lattice_tables* tables, const lattice_jagged* bags,
                                      int64_t* first_bad, void* stream);

/* ------------------------------------------------------------------------ */
/* Interaction (Section 3.3.2)                                              */
/* ------------------------------------------------------------------------ */

/* One layer of the stacked fusion blocks (DHEN/Wukong fusion block, Section
 * 3.3.2): the factorization-machine block F = X (X^T W) (rank k), H_F =
 * A vec(F) reshaped to [n_out - n_lcb, dim] (no bias: bias-less backbone,
 * Section 3.3.4); with n_lcb > 0 the linear compression block H_L = L X
 * ([n_lcb, dim]) is concatenated after it, H = [H_F; H_L]; residual R = C X
 * (C != NULL, a linear projection) or R = X; output LayerNorm_gamma(H + R)
 * per vector over dim (gain only, fp32 math). */
typedef struct {
  const void* W;        /* device [n_in, rank] */
  const void* A;        /* device [(n_out - n_lcb)*dim, n_in*rank] */
  const void* C;        /* device [n_out, n_in] or NULL (requires n_in == n_out) */
  const float* gamma;   /* device [dim] */
  float* dW;            /* device fp32 grads, same shapes (bwd) */
  float* dA;
  float* dC;
  float* dgamma;
  const void* L;        /* device [n_lcb, n_in] (n_lcb > 0), else ignored */
  float* dL;            /* device [n_lcb, n_in] fp32 (bwd) */
} lattice_stack_layer;

typedef struct {
  lattice_interact_kind kind;
  lattice_dtype dtype;
  int32_t n;             /* vectors per sample entering the interaction */
  int32_t dim;           /* d */
  int32_t rank;          /* k (FM, STACK) */
  int32_t emit_slot0;    /* DOT/FM: out row = [X[b,0,:], interaction] (dense vector first) */
  const void* fm_W;      /* FM: device [n, rank] */
  float* fm_dW;          /* FM: device [n, rank] fp32 (bwd) */
  int32_t n_layers;      /* STACK: layers (<= LATTICE_MAX_LAYERS) */
  int32_t stack_n;       /* STACK: vectors per layer output */
  float ln_eps;          /* STACK: LayerNorm epsilon */
  const lattice_stack_layer* layers;  /* host [n_layers] */
  int32_t lcb_n;         /* STACK: output vectors of each layer's linear compression
                            block (0: FM block only; < stack_n) */
  const uint32_t* slot_mask; /* DOT, optional: device [B, 4] per-sample bitmask (16-byte
                            aligned), bit s of word s/32 set when slot s may be
                            non-zero (bits >= n ignored).  The caller guarantees
                            that every slot whose bit is clear holds a zero vector
                            (absent features are zero-padded, Section 3.2); the
                            forward then skips those slots (their pairs are written
                            as 0), with results equal to the full computation's;
                            the backward computes every slot.  Needs n <= 128;
                            NULL: every slot is computed.  lattice_step builds its
                            own (see skip_absent): leave NULL in the model. */
  int32_t fp8_proj;      /* STACK: the FM blocks' projection vec(F) A^T as an FP8 linear layer
                            (Section 3.5.2): 0 = bf16; 1 = e4m3 with row-wise scales
                            (vec(F) per sample, A per output unit, quantised every
                            call), fast accumulation off; 2 = the same with fast
                            accumulation on.  The backward stays bf16 and takes the
                            quantisation as the identity. */
  int32_t skip_absent;   /* DOT in lattice_step: 1 when whole features may be absent from
                            a sample (empty bags, as in multi-domain batches, Section
                            3.2): the step builds each sample's slot mask from the
                            batch and the forward skips the empty slots; 0: none */
} lattice_interact_desc;

/* DOT: out[b, m(i,j)] = <X[b,i], X[b,j]> for i<j, m(i,j) row-major over the
 * strict upper triangle.  FM: out[b] = vec_rowmajor(X_b (X_b^T W)), [n, k].
 * STACK: out[b] = vec(X_{L+1}), [stack_n, dim].  X is [B, n, dim]; out rows
 * have stride out_stride (elements) and start with X[b,0,:] when emit_slot0.
 * The workspace holds what the backward needs (STACK) and must be passed
 * unchanged to lattice_interact_bwd.  Errors: INVALID_ARG, UNSUPPORTED,
 * WORKSPACE, HIP. */
size_t lattice_interact_workspace(const lattice_interact_desc* desc, int32_t B);
lattice_status lattice_interact_fwd(const lattice_interact_desc* desc, int32_t B, const void* X,
                                    void* out, int64_t out_stride, void* ws, size_t ws_bytes,
                                    void* stream);

/* STACK: byte offsets inside the interaction workspace of the state the
 * forward saves for the backward, per layer l < n_layers (-1: absent):
 * P = X_l^T W [B, dim, rank] (bf16), F = X_l P [B, n_l, rank] (bf16),
 * H = [H_F; H_L] [B, stack_n * dim] (fp32, the LayerNorm input before the
 * residual), mean and rstd [B, stack_n] (fp32, of the LayerNorm), and the
 * layer's output X_{l+1} [B, stack_n, dim] (bf16; the last layer's output is
 * the caller's out, so -1).  For inspection and tests; other kinds: all -1.
 * Errors: INVALID_ARG, UNSUPPORTED. */
typedef struct {
  int64_t P[LATTICE_MAX_LAYERS], F[LATTICE_MAX_LAYERS], H[LATTICE_MAX_LAYERS];
  int64_t mean[LATTICE_MAX_LAYERS], rstd[LATTICE_MAX_LAYERS], Xn[LATTICE_MAX_LAYERS];
} lattice_stack_state;
lattice_status lattice_interact_state(const lattice_interact_desc* desc, int32_t B,
                                      lattice_stack_state* out);

/* Gradient of lattice_interact_fwd: given d_out (same layout as out, storage
 * dtype), writes dX [B, n, dim] (storage dtype; with emit_slot0 the slot-0
 * part of d_out is added to dX[:,0,:] in fp32 before rounding) and the
 * parameter gradients named in desc (fp32, overwritten, summed over the batch
 * in a fixed order). */
lattice_status lattice_interact_bwd(const lattice_interact_desc* desc, int32_t B, const void* X,
                                    const void* d_out, int64_t d_out_stride, void* dX,
                                    void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* MLPs and multi-objective heads (Sections 3.3.1, 3.3.3, 3.2.1)            */
/* ------------------------------------------------------------------------ */

/* Activation of the hidden layers of an MLP.
 *
 * SwishRN (Section 3.3.4) replaces the ReLU of a feed-forward layer: with
 * the layer's pre-activation h = x W^T + b split into normalisation groups
 * G of its features,
 *   rho_G = 1 / sqrt(mean_{j in G} h_j^2 + eps),  n = h rho_G,
 *   out   = (g_a n) * gate(g_b n),
 * two per-feature gains (g_a of the normalised value, g_b of the RMSNorm
 * that feeds the self-gate; both share rho).  gate is the logistic sigmoid
 * (SWISHRN) or the hard sigmoid clip(z/6 + 1/2, 0, 1), which avoids the
 * exponential (HARDSWISHRN, Section 3.5.3).  The groups are the whole row
 * (norm_block = 0: RMSNorm) or BlockNorm's groups of 128 consecutive
 * features (norm_block = 128, Section 3.5.3: the columns of one GEMM tile,
 * so bf16 models compute the statistic in the GEMM's epilogue without
 * data from other workgroups); the last group is shorter when 128 does not
 * divide the width.  The forward stores h (storage dtype) and every
 * group's rho (fp32) for the backward. */
typedef enum {
  LATTICE_ACT_RELU = 0,
  LATTICE_ACT_SWISHRN = 1,
  LATTICE_ACT_HARDSWISHRN = 2
} lattice_activation;

#define LATTICE_BLOCKNORM_COLS 128

typedef struct {
  int32_t in_dim, out_dim;
  const void* W;    /* device [out_dim, in_dim], storage dtype */
  const float* b;   /* device [out_dim] or NULL */
  float* dW;        /* device [out_dim, in_dim] fp32 (bwd, overwritten) */
  float* db;        /* device [out_dim] fp32 or NULL (bwd, overwritten) */
  /* SwishRN layers only (ignored otherwise): */
  const float* gain;  /* device [2, out_dim] fp32: g_a, then g_b */
  float* dgain;       /* device [2, out_dim] fp32 or NULL (bwd, overwritten) */
  void* pre;          /* lattice_mlp_heads_fwd/bwd: device [B, out_dim] storage dtype,
                         the pre-activation h (fwd writes, bwd reads); lattice_step
                         keeps it in its workspace instead */
  float* rinv;        /* lattice_mlp_heads_fwd/bwd: device [B, groups] fp32, rho of
                         every row and group (fwd writes, bwd reads) */
} lattice_linear;

typedef struct {
  lattice_dtype dtype;
  int32_t n_layers;                 /* 1 .. LATTICE_MAX_LAYERS */
  const lattice_linear* layers;     /* host [n_layers] */
  int32_t relu_last;                /* 1: the activation on every layer (bottom MLP);
                                       0: last layer linear, fp32 output (heads) */
  lattice_activation act;           /* activation of the activated layers */
  int32_t norm_block;               /* SwishRN groups: 0 (whole row) or 128 (BlockNorm) */
  float norm_eps;                   /* SwishRN eps (>= 0) */
  int32_t tower_heads;              /* 1: per-objective towers (Section 3.3.3): the last
                                       (linear) layer's input holds T = out_dim groups of
                                       H = in_dim / out_dim units, one tower per objective,
                                       and output t reads only group t: its W and dW are
                                       [T, H] (not [T, in_dim]); H % 8 == 0, the logits
                                       contiguous.  0: a dense last layer. */
  int32_t n_domains;                /* parameter untying (Section 3.3.4): >= 2 gives each of
                                       the first untied_layers layers one parameter set per
                                       domain, stacked: W [n_domains, out, in], b, gain and
                                       their gradients likewise; the samples of domain g use
                                       set g.  0 or 1: every layer tied. */
  int32_t untied_layers;            /* layers 0 .. untied_layers-1 are untied (not the
                                       towers' heads) */
  const int64_t* domain_offsets;    /* lattice_mlp_heads_fwd/bwd with untied layers: host
                                       [n_domains + 1], samples grouped by domain, domain g
                                       = rows off[g] .. off[g+1]-1 (off[0] = 0, non-
                                       decreasing, off[n_domains] = B).  lattice_step uses
                                       the batch's offsets instead. */
} lattice_mlp_desc;

/* Masked multi-objective BCE with logits z [B, T]: with N = max(1, sum m),
 * loss = sum m*(max(z,0) - z*y + log1p(exp(-|z|))) / N and
 * d_logits = m*(sigmoid(z) - y)/N, so masked heads get exactly zero. */
typedef struct {
  const float* labels;   /* device [B, T] */
  const uint8_t* mask;   /* device [B, T], 0/1 */
  float* loss;           /* device [1] */
  float* d_logits;       /* device [B, T] fp32 */
  void* d_logits_op;     /* device [B, T] storage dtype (backward GEMM operand) or NULL */
} lattice_loss_desc;

/* Workspace of lattice_mlp_heads_fwd and lattice_mlp_heads_bwd (the larger
 * of the two). */
size_t lattice_mlp_heads_workspace(const lattice_mlp_desc* desc, int32_t B);

/* Forward: acts[i] (host array of device pointers) receives layer i's output
 * [B, out_i] with row stride act_strides[i] (host array, elements): the
 * activation (ReLU or SwishRN, then storage rounding) on hidden layers; fp32
 * logits on a linear last layer.  SwishRN layers also write their pre and
 * rinv buffers (lattice_linear).  If
 * loss != NULL the masked BCE is evaluated on the logits (which must then be
 * contiguous, act_strides[last] == T).  `in` is [B, in_0] with row stride
 * in_stride, storage dtype.  Errors: INVALID_ARG, WORKSPACE, HIP. */
lattice_status lattice_mlp_heads_fwd(const lattice_mlp_desc* desc, int32_t B, const void* in,
                                     int64_t in_stride, void* const* acts,
                                     const int64_t* act_strides, const lattice_loss_desc* loss,
                                     void* ws, size_t ws_bytes, void* stream);

/* Backward: d_out is the gradient of the last layer's output (storage dtype;
 * for relu_last the gradient of the activated output, taken through the
 * activation here: masked by acts[last] > 0, or the SwishRN backward).
 * Writes dW/db (and dgain of SwishRN layers) of every layer (fp32,
 * overwritten, summed over the batch in a fixed order) and, if d_in != NULL,
 * the input gradient
 * [B, in_0] (stride d_in_stride, storage dtype, unmasked).  Errors:
 * INVALID_ARG, WORKSPACE, HIP. */
lattice_status lattice_mlp_heads_bwd(const lattice_mlp_desc* desc, int32_t B, const void* in,
                                     int64_t in_stride, const void* const* acts,
                                     const int64_t* act_strides, const void* d_out,
                                     int64_t d_out_stride, void* d_in, int64_t d_in_stride,
                                     void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* FP8 linear layers (Section 3.5.2)                                        */
/* ------------------------------------------------------------------------ */

/* Linear-layer GEMMs in FP8 with tensor-wise or row-wise scales (not
 * block-wise), the format the paper uses for FP8 training and inference;
 * normalisation stays in fp32.  The FP8 format is OCP e4m3 (bias 7, largest
 * finite value 448, no infinities). */
typedef enum {
  LATTICE_FP8_ROWWISE = 0,     /* one scale per row of the matrix */
  LATTICE_FP8_TENSORWISE = 1   /* one scale for the whole matrix */
} lattice_fp8_scaling;

/* Quantise x [rows, cols] (row stride ld elements, bf16 or fp32): s = amax /
 * 448 over each row (ROWWISE, scales [rows]) or over the matrix (TENSORWISE,
 * scales [1]), s = 1 where the amax is 0; q = e4m3(x * (1 / s)), with s, 1 / s
 * and the product in fp32 (correctly rounded) and the product rounded to the
 * nearest e4m3 value, ties to even, saturating at +-448 (x must be finite).  q is [rows, ldq] bytes,
 * ldq a multiple of 16 and >= cols, 16-byte aligned; bytes cols .. ldq-1 of
 * each row are written as 0.  TENSORWISE needs a workspace of
 * lattice_fp8_quantize_workspace() bytes.  Errors: INVALID_ARG, WORKSPACE,
 * HIP. */
size_t lattice_fp8_quantize_workspace(void);
lattice_status lattice_fp8_quantize(const void* x, lattice_dtype x_dtype, int64_t rows, int64_t cols,
                                    int64_t ld, lattice_fp8_scaling scaling, uint8_t* q, int64_t ldq,
                                    float* scales, void* ws, size_t ws_bytes, void* stream);

/* Y[m, n] = act((sum_k qA[m,k] qW[n,k]) * sA[m or 0] * sW[n or 0] + bias[n]):
 * a linear layer Y = X W^T + b on quantised X [M, K] and W [N, K] (codes from
 * lattice_fp8_quantize, row strides lda / ldw bytes: multiples of 16, >= K
 * rounded up to 16, 16-byte aligned).  The matrix instruction adds 64
 * products and its incoming partial sum after aligning them to the largest
 * exponent among them with about 13 fraction bits.  fast_accum = 1 chains
 * the partial sum through all of K (fastest; low bits are lost relative to
 * the running sum: inference); fast_accum = 0 starts every 64-k instruction
 * from zero and adds the partial sums in fp32 (training).  The sum is scaled by sA then
 * sW, in fp32.  bias may be NULL; relu != 0 applies ReLU; Y is [M, ldy] in
 * y_dtype (bf16 rounded to nearest even).  Errors: INVALID_ARG, HIP. */
lattice_status lattice_linear_fp8_fwd(const uint8_t* qA, int64_t lda, const float* sA,
                                      lattice_fp8_scaling a_scaling, const uint8_t* qW, int64_t ldw,
                                      const float* sW, lattice_fp8_scaling w_scaling,
                                      const float* bias, int32_t M, int32_t N, int32_t K,
                                      int32_t relu, int32_t fast_accum, void* Y,
                                      lattice_dtype y_dtype, int64_t ldy, void* stream);

/* ------------------------------------------------------------------------ */
/* Whole training step                                                      */
/* ------------------------------------------------------------------------ */

typedef struct {
  lattice_dtype dtype;
  lattice_pool pool;
  lattice_tables tables;
  int32_t num_features;        /* F */
  int32_t dense_in;            /* dense inputs (0: no dense path, no bottom MLP) */
  lattice_mlp_desc bottom;     /* relu_last = 1, ReLU, tied, output width = dim */
  lattice_interact_desc interact;  /* n = F + (dense_in > 0); emit_slot0 = dense_in > 0 (DOT/FM) */
  lattice_mlp_desc top;        /* relu_last = 0, output width = T; hidden layers ReLU
                                  or SwishRN (act), tied or untied per domain; dense or
                                  tower heads */
} lattice_model_desc;

typedef struct {
  lattice_jagged bags;
  const void* dense;           /* device [B, dense_in], storage dtype */
  const float* labels;         /* device [B, T] */
  const uint8_t* mask;         /* device [B, T] */
  const int64_t* domain_offsets;  /* host [top.n_domains + 1] when the top MLP has untied
                                     layers (samples grouped by domain, see
                                     lattice_mlp_desc), else ignored */
} lattice_batch_desc;

/* Stages of lattice_step, in order (for optional per-stage timing). */
typedef enum {
  LATTICE_STAGE_EMBBAG_FWD = 0,
  LATTICE_STAGE_BOTTOM_FWD,
  LATTICE_STAGE_INTERACT_FWD,
  LATTICE_STAGE_TOP_FWD,
  LATTICE_STAGE_LOSS,
  LATTICE_STAGE_TOP_BWD,         /* gradient chain of the top MLP down to its input */
  LATTICE_STAGE_INTERACT_BWD,
  LATTICE_STAGE_TOP_WGRAD,       /* weight and bias gradients of the top MLP */
  LATTICE_STAGE_BOTTOM_BWD,
  LATTICE_STAGE_EMBBAG_SORT,     /* sparse gradient: sort of (row, bag) pairs */
  LATTICE_STAGE_EMBBAG_RUNS,     /* sparse gradient: unique rows and run offsets */
  LATTICE_STAGE_EMBBAG_REDUCE,   /* sparse gradient: segmented reduction (+ SGD) */
  LATTICE_STAGE_EMBBAG_FIXUP,    /* sparse gradient: runs crossing reduction ranges */
  LATTICE_STEP_STAGES
} lattice_step_stage;

/* Streams.  The sort and run bookkeeping of the sparse gradient need only
 * the batch, and the dense weight gradients (top MLP weights, bottom MLP
 * backward) are not needed by the sparse gradient, so lattice_step can run
 * them on a second stream that the CALLER provides (side_stream, a
 * hipStream_t of the same device, default priority) together with
 * LATTICE_STEP_SIDE_EVENTS events (hipEvent_t, created by the caller; timing
 * may be disabled) that it uses to fork work from `stream` onto the side
 * stream and to join it back: the bottom MLP's forward is forked at the
 * step's start and runs beside the pooled lookups; the sort is forked after
 * the pooled lookups and overlaps the dense forward and backward; the bottom
 * MLP's backward is forked after the interaction backward and overlaps the
 * top MLP's weight gradients and the segmented reduction (which waits for
 * the sort), both on `stream`.  All work is still ordered
 * after the caller's prior work on `stream`, and the call's work is complete
 * when `stream` reaches the end of it, as with a single stream.  The library
 * keeps no stream or event of its own.  Two calls that share a side stream
 * or events must not be enqueued concurrently from different host threads
 * (they would interleave their event records).  side_stream = NULL (or equal
 * to `stream`) keeps every stage on `stream`; results are bit-identical
 * either way. */
#define LATTICE_STEP_SIDE_EVENTS 6

typedef struct {
  float lr_tables;             /* row-sparse SGD step on the tables (0: none) */
  int32_t emit_grad_rows;      /* 1: also write the [nnz, dim] fp32 row gradients */
  int64_t nnz_capacity;        /* lookups the workspace is planned for (0: the batch's nnz);
                                  plan and step must use the same value */
  void* const* stage_events;   /* host array of 2*LATTICE_STEP_STAGES hipEvent_t or NULL:
                                  [2s] is recorded when stage s begins and [2s+1] when
                                  it ends, on the stream that runs the stage (the side
                                  stream for BOTTOM_FWD, EMBBAG_SORT, EMBBAG_RUNS and
                                  BOTTOM_BWD when a side stream is given);
                                  NULL entries are not recorded (each record costs a
                                  few microseconds of GPU time) */
  void* side_stream;           /* hipStream_t or NULL (see above) */
  void* const* side_events;    /* host array of LATTICE_STEP_SIDE_EVENTS hipEvent_t;
                                  required when side_stream is used */
  int32_t fp8_top;             /* mixed FP8 / BF16 training (Section 3.5.2), bf16 models:
                                  0 = off; 1 = the forward GEMMs of the top MLP's hidden
                                  layers in FP8 e4m3 with row-wise scales (inputs per
                                  sample, weights per output unit, quantised every step)
                                  and fast accumulation off; 2 = the same with fast
                                  accumulation on.  The objective heads, every backward
                                  GEMM and all stored activations stay bf16; the
                                  gradients treat quantisation as the identity.  Plan
                                  and step must use the same value. */
} lattice_step_opts;

/* Byte offsets of every intermediate inside the step workspace (-1: absent). */
typedef struct {
  int64_t total_bytes;
  int64_t X;            /* [B, n, dim] stacked vectors (dense slot 0, then features) */
  int64_t t;            /* [B, t_stride] top-MLP input */
  int64_t t_stride;     /* elements */
  int64_t logits;       /* [B, T] fp32 */
  int64_t d_logits;     /* [B, T] fp32 */
  int64_t d_logits_op;  /* [B, T] storage dtype */
  int64_t loss;         /* [1] fp32 */
  int64_t d_t;          /* [B, t_stride] gradient of the top input */
  int64_t dX;           /* [B, n, dim] gradient of the stacked vectors */
  int64_t bottom_act[LATTICE_MAX_LAYERS];   /* [B, out_i] hidden bottom outputs (last: in X) */
  int64_t top_act[LATTICE_MAX_LAYERS];      /* [B, out_i] hidden top outputs (last: logits) */
  /* Gradient chain, storage dtype, [B, out_i]: the gradient of layer i's
   * pre-activation (its output's gradient masked by the ReLU, or taken
   * through the SwishRN backward), i.e. the left operand of that layer's
   * weight gradient dW_i = g_i^T h_i.  top_grad[last] is d_logits_op; bottom_grad[last]
   * is the masked gradient of the bottom output (slot 0 of X). */
  int64_t top_grad[LATTICE_MAX_LAYERS];
  int64_t bottom_grad[LATTICE_MAX_LAYERS];
  /* SwishRN hidden top layers (else -1): the pre-activation h [B, out_i]
   * (storage dtype), rho [B, groups_i] (fp32), and the gradient of the layer's
   * output [B, out_i] (storage dtype) from which top_grad[i] is taken through
   * the SwishRN backward. */
  int64_t top_pre[LATTICE_MAX_LAYERS];
  int64_t top_rinv[LATTICE_MAX_LAYERS];
  int64_t top_gout[LATTICE_MAX_LAYERS];
  int64_t unique_rows, seg_offsets, sorted_bags, num_unique, grad_rows;
  int64_t interact;     /* interaction workspace (saved state from forward to backward) */
  int64_t scratch;      /* scratch shared by the dense stages */
  int64_t scratch_bytes;
  int64_t sparse;       /* scratch of the sparse gradient (sort, runs, reduction) */
  int64_t sparse_bytes;
  int64_t fp8;          /* e4m3 codes and scales of the FP8 forward (fp8_top), or -1 */
  int64_t fp8_bytes;
} lattice_step_layout;

/* Workspace layout for batches of B samples and at most
 * max(nnz, opts->nnz_capacity) lookups. */
lattice_status lattice_step_plan(const lattice_model_desc* model, int32_t B, int64_t nnz,
                                 const lattice_step_opts* opts, lattice_step_layout* layout);

/* One forward + backward step: pooled lookups, bottom MLP, interaction, top
 * MLP, masked BCE, and the backward of all of them; parameter gradients go to
 * the dW/db/... pointers in `model`; the row-coalesced table gradient goes to
 * the workspace (see lattice_step_layout); with lr_tables != 0 the tables are
 * updated in place.  ws must be lattice_step_plan(...)->total_bytes long for
 * the same opts; the batch's nnz must not exceed opts->nnz_capacity (when
 * set).  Errors: INVALID_ARG, UNSUPPORTED (also: stacked vectors X larger
 * than 4 GiB), WORKSPACE, HIP. */
lattice_status lattice_step(const lattice_model_desc* model, const lattice_batch_desc* batch,
                            const lattice_step_opts* opts, void* ws, size_t ws_bytes,
                            void* stream);

/* The forward of lattice_step alone, for inference (Section 3.5.2 serves
 * with FP8 and fast accumulation: opts->fp8_top = 2): pooled lookups, bottom
 * MLP, interaction and top MLP, writing the logits ([B, T] fp32 at
 * layout.logits) and the forward intermediates of the layout.  No loss,
 * gradient or table update; batch->labels and batch->mask are not read (may
 * be NULL).  Same model, plan, workspace and opts as lattice_step (a side
 * stream, if given, runs the bottom MLP beside the pooled lookups; lr_tables
 * and emit_grad_rows are ignored).  Errors as lattice_step. */
lattice_status lattice_forward(const lattice_model_desc* model, const lattice_batch_desc* batch,
                               const lattice_step_opts* opts, void* ws, size_t ws_bytes,
                               void* stream);

/* ------------------------------------------------------------------------ */
const char* lattice_status_string(lattice_status s);
const char* lattice_last_error(void);
int lattice_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* LATTICE_H_ */
