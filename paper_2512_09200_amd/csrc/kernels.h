// Internal launchers (namespace lat).  Every launcher enqueues on the given
// stream and returns the first HIP error (with lat::set_error detail).
#pragma once
#include "common.h"

namespace lat {

// sort.hip
hipError_t exclusive_scan_inplace_small(int* a, int n, hipStream_t s);
// Sort of a jagged batch's (global row, bag) pairs whose positions are grouped
// by feature: each feature segment is sorted by its local row (< max_local_rows).
// The first pass reads the batch's indices directly (keys = row_base[f] +
// index, values = bag ids expanded from the offsets).
size_t radix_sort_segments_workspace(int64_t n, int F);
hipError_t radix_sort_segments(const int32_t* indices, int64_t n, const int32_t* offsets, int F,
                               int B, const int64_t* row_base, int64_t max_local_rows,
                               int* keys_out, int* vals_out, void* ws, hipStream_t s);

// embbag.hip
hipError_t embbag_fwd(const void* E, DType edt, int dim, const int64_t* row_base,
                      const int32_t* offsets, const int32_t* indices, int F, int B, int mean,
                      void* X, DType xdt, int n_slots, int first_slot, hipStream_t s);
size_t embbag_bwd_workspace(int64_t nnz, int dim, int F);
// max_local_rows: rows of the largest table (bounds every local index).
// The sparse gradient in two phases over one workspace: embbag_bwd_sort needs
// only the batch -- sort, unique rows, run offsets; embbag_bwd_apply needs
// dX -- segmented reduction and SGD.
// ev (optional): 4 events each, begin/end of the phase's two parts (null
// entries are not recorded).
hipError_t embbag_bwd_sort(const int64_t* row_base, int64_t max_local_rows, const int32_t* offsets,
                           const int32_t* indices, int F, int B, int64_t nnz, int dim,
                           int* unique_rows, int* seg_offsets, int* sorted_bags, int* num_unique,
                           void* ws, hipStream_t s, void* const* ev);
hipError_t embbag_bwd_apply(const int32_t* offsets, int F, int B, int64_t nnz, int mean,
                            const void* dX, DType dxt, int n_slots, int first_slot, int dim,
                            const int* unique_rows, const int* seg_offsets, const int* sorted_bags,
                            float* grad_rows, void* E, DType et, float lr, void* ws, hipStream_t s,
                            void* const* ev);
hipError_t embbag_bwd(const int64_t* row_base, int64_t max_local_rows, const int32_t* offsets,
                      const int32_t* indices, int F, int B, int64_t nnz, int mean,
                      const void* dX, DType dxt, int n_slots, int first_slot, int dim,
                      int* unique_rows, int* seg_offsets, int* sorted_bags, int* num_unique,
                      float* grad_rows, void* E, DType et, float lr, void* ws, hipStream_t s);
hipError_t validate_batch(const int64_t* row_base, const int32_t* offsets,
                          const int32_t* indices, int F, int B, int64_t nnz, int64_t max_rows,
                          unsigned long long* dev_result, hipStream_t s);

// gemm.hip
struct GemmArgs {
  DType dt = DT_BF16;          // operand dtype
  const void* A = nullptr; int64_t lda = 0; int ta = 0;
  const void* B = nullptr; int64_t ldb = 0; int tb = 0;
  void* C = nullptr; int64_t ldc = 0; DType c_dt = DT_F32;
  int M = 0, N = 0, K = 0;
  const float* bias = nullptr;
  int relu = 0;
  const void* mask = nullptr; DType mask_dt = DT_BF16; int64_t ldm = 0, s_mask = 0;
  const float* addend = nullptr; int64_t ld_add = 0, s_add = 0;  // epilogue + addend[m][n]
  int accumulate = 0;          // epilogue + existing C (fp32 C only)
  int max_splits = 1;          // split-K only when the caller provides gemm_workspace()
  int batch = 1;               // batched: blockIdx.z = batch index; strides in elements
  int64_t sA = 0, sB = 0, sC = 0;
  int kseg = 0;                // K segmentation: k -> (k / kseg) * ks + k % kseg (0: none)
  int64_t ksA = 0, ksB = 0;
  float* rowsum = nullptr;     // bf16, not batched: rowsum[m] = sum_k A[m][k] (fp32, k order)
  // BlockNorm epilogue (SwishRN over 128-column groups): gate 1 = sigmoid,
  // 2 = hard sigmoid; gain [2, N] (g_a; g_b); pre [M, ldp] receives h =
  // acc + bias in C's dtype, rinv [M, nblk = ceil(N / 128)] each group's
  // 1 / sqrt(mean h^2 + eps)
  // Grouped product (parameter untying), bf16 only: ngroups groups with
  // host offsets goff[0..ngroups] over the rows of A and C (gk = 0; B, bias
  // and gains per group, B + z gsB) or over K (gk = 1; C + z gsC, row sums
  // + z M).  At most 16 groups.
  int ngroups = 0;
  const int64_t* goff = nullptr;
  int gk = 0;
  int64_t gsB = 0, gsC = 0;
  int norm_gate = 0;
  const float* gain = nullptr;
  float eps = 0.f;
  void* pre = nullptr;
  int64_t ldp = 0;
  float* rinv = nullptr;
  int nblk = 0;
};
int gemm_splits(const GemmArgs& g);
size_t gemm_workspace(const GemmArgs& g);
hipError_t gemm(const GemmArgs& g, void* ws, hipStream_t s);
size_t colsum_workspace(int M, int N);
hipError_t colsum(const void* G, DType dt, int64_t ld, int M, int N, float* out, void* ws,
                  hipStream_t s);

// swishrn.hip (SwishRN rows: the unfused forward, the backward chain and the
// gain gradients; block = 0: the whole row, 128: BlockNorm groups; gate 1 =
// sigmoid, 2 = hard sigmoid; rinv [M, swishrn_groups(N, block)])
int swishrn_groups(int N, int block);
hipError_t swishrn_fwd_rows(DType dt, const void* pre, int64_t ldp, int M, int N, int block, int gate,
                            const float* gain, float eps, void* out, int64_t ldo, float* rinv,
                            hipStream_t s);
hipError_t swishrn_bwd_rows(DType dt, const void* go, int64_t ldg, const void* pre, int64_t ldp,
                            const float* rinv, int M, int N, int block, int gate, const float* gain,
                            void* dh, int64_t ldd, hipStream_t s);
size_t swishrn_gain_workspace(int M, int N);
hipError_t swishrn_gain_grad(DType dt, const void* go, int64_t ldg, const void* pre, int64_t ldp,
                             const float* rinv, int M, int N, int block, int gate,
                             const float* gain, float* dgain, void* ws, hipStream_t s);

// towers.hip (heads of per-objective towers: objective t reads only units
// t*H .. t*H+H-1 of its input; w [T, H]; H % 8 == 0)
hipError_t tower_head_fwd(DType dt, const void* h, int64_t ldh, int B, int NT, int H, const void* w,
                          const float* bias, float* z, hipStream_t s);
hipError_t tower_head_dgrad(DType dt, const void* g, int64_t ldg, int B, int NT, int H, const void* w,
                            const void* mask, int64_t ldm, void* dh, int64_t ldd, hipStream_t s);
size_t tower_wgrad_workspace(int B, int NT, int H);
hipError_t tower_wgrad(DType dt, const void* g, int64_t ldg, const void* h, int64_t ldh, int B, int NT,
                       int H, float* dw, void* ws, hipStream_t s);

// interact.hip
size_t dot_lds_bytes(int n, int d);
size_t fm_lds_bytes(int n, int d, int k);
hipError_t dot_fwd(DType dt, const void* X, int B, int n, int d, void* out, int64_t ostride,
                   int emit0, hipStream_t s);
hipError_t dot_bwd(DType dt, const void* X, int B, int n, int d, const void* dout,
                   int64_t dstride, int emit0, void* dX, hipStream_t s);
hipError_t fm_fwd(DType dt, const void* X, const void* W, int B, int n, int d, int k, void* out,
                  int64_t ostride, int emit0, hipStream_t s);
size_t fm_bwd_workspace(int n, int k);
hipError_t fm_bwd(DType dt, const void* X, const void* W, int B, int n, int d, int k,
                  const void* dout, int64_t dstride, int emit0, const float* addend,
                  void* dX, DType dxt, float* dW, void* ws, hipStream_t s);

// fm_mfma.hip (bf16 MFMA path of the FM block)
bool fm_mfma_supported(int n, int d, int k);
size_t fm_mfma_bwd_workspace(int n, int k);
hipError_t fm_mfma(bool fwd, const void* X, const void* W, int B, int n, int d, int k, void* out,
                   int64_t ostride, int emit0, const void* dout, int64_t dstride,
                   const float* addend, void* dX, float* dX_f32, float* dW, void* ws,
                   hipStream_t s);

// dot_mfma.hip (bf16 MFMA path of the DOT interaction)
bool dot_mfma_supported(int n, int d);
hipError_t dot_mfma(bool fwd, const void* X, int B, int n, int d, void* out, int64_t ostride,
                    int emit0, const void* dout, int64_t dstride, void* dX, const uint32_t* mask,
                    hipStream_t s);
// per-sample DOT slot bitmasks (4 words) of a batch: the dense slot and the non-empty bags
hipError_t dot_slot_mask(const int32_t* offsets, int F, int B, int first, int has0, uint32_t* mask,
                         hipStream_t s);

// stack.hip (stacked FM -> linear -> residual -> LayerNorm interaction)
struct StackShape {
  int L, n0, nv, d, k;  // layers, input vectors, vectors per layer output, dim, FM rank
  int has_C0;           // layer 0 uses a projection residual C [nv, n0]
  float eps;
  int nL;               // output vectors of the linear compression block (0: none)
  int fp8;              // FM projection in FP8 e4m3: 0 = bf16, 1 = precise, 2 = fast accumulation
};
struct StackLayer {
  const void* W;        // [n, k] bf16
  const void* A;        // [(nv - nL)*d, n*k] bf16
  const void* C;        // [nv, n0] bf16 (layer 0) or null
  const float* gamma;   // [d]
  float* dW; float* dA; float* dC; float* dgamma;
  const void* Lc;       // [nL, n] bf16 (nL > 0)
  float* dL;
};
struct StackPlan {       // byte offsets inside the interaction workspace
  size_t P[8], F[8], H[8], mean[8], rstd[8], Xn[8], R0, state_bytes;
  size_t qF, sF, qA, sA;  // FP8 projection: codes and row scales of vec(F) and A (fp8 only)
  size_t du, duR, dF, dP, dXf, dgp, gemm_ws, total_bytes;
};
bool stack_supported(const StackShape& sh);
StackPlan stack_plan(const StackShape& sh, int B);
hipError_t stack_fwd(const StackShape& sh, const StackLayer* Ls, int B, const void* X, void* out,
                     int64_t out_stride, void* state, hipStream_t s);
hipError_t stack_bwd(const StackShape& sh, const StackLayer* Ls, int B, const void* X,
                     const void* d_out, int64_t d_out_stride, void* dX, void* state,
                     hipStream_t s);

// loss.hip
size_t bce_workspace(int64_t n);
hipError_t bce(const float* z, const float* y, const uint8_t* m, int64_t n, float* loss, float* dz,
               void* dz_op, DType op_dt, void* ws, hipStream_t s);

// head.hip (bf16 objective heads: last top layer fused with the masked BCE
// and with its input gradient; workspace: per-block partials, written by
// head_fwd and read by head_bwd)
constexpr int HEAD_MAX_T = 64;
bool head_fusable(int T, int K, const void* h, int64_t ldh, const void* W);
size_t head_workspace(int B);
hipError_t head_fwd(const bf16_t* h, int64_t ldh, int B, int K, const bf16_t* W,
                    const float* bias, int T, const float* y, const uint8_t* m, float* z,
                    void* ws, hipStream_t s);
hipError_t head_bwd(const float* z, const float* y, const uint8_t* m, int B, int T,
                    const bf16_t* W, int K, const bf16_t* mask, int64_t ldm, float* loss,
                    float* dz, bf16_t* dz_op, bf16_t* g, int64_t ldg, const void* ws,
                    hipStream_t s);

// fp8.hip (OCP e4m3 linear layers, tensor- or row-wise scales)
size_t fp8_quantize_workspace();
// one matrix of a row-wise quantisation launch (codes q [rows, ldq], scales [rows])
struct Fp8RowJob {
  const void* x;
  int64_t ld;
  int rows, cols;
  uint8_t* q;
  int64_t ldq;
  float* scales;
};
constexpr int FP8_MAX_JOBS = 9;
struct Fp8Jobs {
  Fp8RowJob j[FP8_MAX_JOBS];
  int blk0[FP8_MAX_JOBS];
  int n;
};
hipError_t fp8_quantize_rows(DType xdt, const Fp8RowJob* jobs, int njobs, hipStream_t s);
hipError_t fp8_quantize(const void* x, DType xdt, int rows, int cols, int64_t ld, int rowwise,
                        uint8_t* q, int64_t ldq, float* scales, void* ws, hipStream_t s);
hipError_t gemm_fp8(const uint8_t* A, int64_t lda, const float* sa, int sa_rowwise, const uint8_t* B,
                    int64_t ldb, const float* sb, int sb_rowwise, const float* bias, void* C,
                    DType cdt, int64_t ldc, int M, int N, int K, int relu, int fast_accum,
                    hipStream_t s);

}  // namespace lat
