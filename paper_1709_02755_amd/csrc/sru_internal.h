// Internal launch interface between the C ABI (sru_api.hip) and the kernels.
// Launchers assume validated arguments and only enqueue work.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sru {

// The v/b gradient sums over the batch: `rows` rows of per-sequence partials
// [rows, 4, nfeat] (q = dv_f, dv_r, db_f, db_r) summed in a fixed order into
// the four [nfeat] outputs, from q = qlo (the linear recurrence has no v:
// qlo = 2).  partial == nullptr: nothing to do.
struct VbSum {
  const float* partial = nullptr;
  int rows = 0, nfeat = 0, qlo = 0;
  float* out[4] = {nullptr, nullptr, nullptr, nullptr};
};
// Blocks of 256 threads the sums take (64 outputs per block).
inline int vb_sum_blocks(const VbSum& v) { return ((4 - v.qlo) * v.nfeat + 63) / 64; }
hipError_t vb_sum_launch(const VbSum& v, hipStream_t stream);

// A split-K sum: partials [splits, M, N] (fp32) summed in split order into
// C (row pitch ldc), plus up to two addend rows (add, add + add_off; pitch
// add_ld).
struct SplitSum {
  const float* part = nullptr;
  int splits = 0, M = 0, N = 0;
  float* C = nullptr;
  long long ldc = 0;
  const float* add = nullptr;
  long long add_ld = 0, add_off = 0;
  int add_count = 0;
};

// ----------------------------------------------------------------- GEMM
// C[M,N] = sum_k A(m,k) B(n,k), fp32 result, MFMA compute.
//   A(m,k) = a_kc ? A[m*lda + k] : A[k*lda + m]
//   B(n,k) = b_kc ? B[n*ldb + k] : B[k*ldb + n]
// Each operand is fp32 or bf16 (raw uint16 bits) in memory (a_bf16, b_bf16);
// bf16 operands require bf16 compute (bf16 == true).  fp32 operands are
// rounded to bf16 (RNE) when staged, in bf16 compute mode.
// With splits > 1 the reduction is cut into `splits` contiguous K ranges;
// each writes a partial [M,N] (ld = N) at `partials` + s*M*N, and a second
// kernel sums them in split order into C.  The optional addend adds
//   add[m*add_ld + n] (+ add[m*add_ld + add_off + n] when add_count == 2)
// to the result (used for the highway gradient of dX).
struct GemmDesc {
  const void* A;
  const void* B;
  float* C;
  int M, N, K;
  long long lda, ldb, ldc;
  bool a_kc, b_kc;
  bool a_bf16, b_bf16;
  bool bf16;
  int splits;
  float* partials;
  // a K-contiguous product may be split over K too (register-staged path,
  // when its tiles would leave CUs idle); partials must then be given
  bool kc_split;
  const float* add;
  long long add_ld, add_off;
  int add_count;
  // Optional bf16 (RNE) copy of the result, row pitch ldcb; C may then be
  // nullptr (bf16 result only).  Direct path only, both operands
  // K-contiguous, no addend, no split; ldcb % 4 == 0, 8-byte aligned.
  uint16_t* Cb;
  long long ldcb;
  const char* label;  // name for the measurement hook (nullptr: by layout)
  // v/b sums to run with this product (vb.partial != nullptr): in the same
  // launch as the split-K sum when there is one, else right after the product
  VbSum vb;
  // defer_sum: a split product leaves its split sum to a later product's
  // launch (the caller hands gemm_split_sum(this) to that product as
  // `extra`, and keeps the two products' partials apart).  extra: another
  // product's deferred split sum, run in the same launch as this product's
  // (on its own when this product is not split).
  bool defer_sum;
  SplitSum extra;
};

// The split sum gemm_launch would run after g (its partials, split count,
// output and addend).
SplitSum gemm_split_sum(const GemmDesc& g);

// fp32 -> bf16 (RNE) copy of a [rows, cols] matrix; transposed ([cols, rows])
// when `transpose`.
hipError_t to_bf16_launch(const float* src, int rows, int cols, uint16_t* dst, bool transpose,
                          hipStream_t stream, const char* label);
// The same for n contiguous elements (n up to 2^40).
hipError_t to_bf16_n_launch(const float* src, long long n, uint16_t* dst, hipStream_t stream,
                            const char* label);
// Transposed copy [cols, rows] in bf16 (RNE) of a [rows, cols] matrix held in
// fp32, or in bf16 (src_bf16; then an exact copy of its values).
hipError_t to_bf16_t_launch(const void* src, bool src_bf16, int rows, int cols, uint16_t* dst,
                            hipStream_t stream, const char* label);

// Number of K splits the launcher will use for this product (>= 1) and the
// partial-buffer bytes it then needs.
int gemm_splits(const GemmDesc& g);
// whether gemm_launch runs g on the direct (global -> LDS) bf16 kernel
bool gemm_is_direct(const GemmDesc& g);
size_t gemm_partial_bytes(int M, int N, int splits);
hipError_t gemm_launch(const GemmDesc& g, hipStream_t stream);

// ------------------------------------------- fused projection + forward scan
// Inference with bf16 products: U = X Wcat^T and Eq. 1-4 in one kernel; U
// and C are not stored.  Needs k = 3 or 4, L <= 256 / bb, d % 64 == 0,
// d_in % 8 == 0, 16-byte aligned bf16 operands smaller than 2 GiB (a_bytes,
// b_bytes: their sizes).
struct FusedFwdArgs {
  const uint16_t* Xb;  // X in bf16 [L*B, d_in]
  const uint16_t* Wb;  // Wcat in bf16 [ndir*k*d, d_in]
  unsigned a_bytes, b_bytes;
  const float* X;      // X in fp32: the highway input x_t when k = 3
  const float* v_f;
  const float* v_r;
  const float* b_f;
  const float* b_r;
  const float* c0;
  const uint8_t* mask;
  float* H;
  uint16_t* Hb;
  float* c_last;
  int L, B, d_in, d, ndir, k, direction;
  int bb;                 // sequences per tile: a tile holds 256 / bb steps of each
  int ngroups, nbgroups;  // d / 64 unit groups; ceil(B / bb) sequence groups
  float alpha;
  int reset_new, linear;
};
hipError_t proj_scan_forward_launch(const FusedFwdArgs& a, hipStream_t stream);

// ----------------------------------------------------------------- scans
struct ScanShape {
  int L, B, d_in, d, ndir, k, direction;
  float alpha;    // highway scale (Sec. 3.2); 1 = Eq. 4 as printed
  int reset_new;  // reset gate reads c_t (Algorithm 1) instead of c_{t-1} (Eq. 3)
  int linear;     // v * c_{t-1} removed from both gates (ablation (1), Sec. 4.5);
                  // v_f, v_r, dv_f, dv_r are then unused
};

// Work plan of the time-chunked scans of the linear recurrence: nw waves per
// workgroup, groups lane groups of 64, time cut into nseg segments of
// seg_steps steps (whole blocks), one workgroup per (group, segment).
struct LinPlan {
  int nw, groups, nseg, seg_steps;
};

struct ScanFwdArgs {
  const float* U;
  const float* X;
  const float* v_f;
  const float* v_r;
  const float* b_f;
  const float* b_r;
  const float* c0;
  const uint8_t* mask;
  float* H;
  float* C;
  float* c_last;
  uint16_t* Hb;  // optional bf16 (RNE) copy of H
  void* scratch;  // linear recurrence: the segment maps (scan_forward_scratch_bytes)
};

struct ScanBwdArgs {
  const float* U;
  const float* X;
  const float* C;
  const float* dH;
  const float* dc_last;
  const float* v_f;
  const float* v_r;
  const float* b_f;
  const float* b_r;
  const float* c0;
  const uint8_t* mask;
  void* dU;        // fp32, or bf16 bits when du_bf16
  bool du_bf16;
  float* dxh;
  float* partial;  // per-sequence sums of the v/b gradients (and, for the
                   // linear recurrence, the segment maps): scan_backward_partial_bytes
  float* dc0;
  float* dv_f;
  float* dv_r;
  float* db_f;
  float* db_r;
  // the caller runs the v/b sums (scan_backward_vb) instead of
  // scan_backward_launch
  bool defer_vb = false;
};

hipError_t scan_forward_launch(const ScanShape& s, const ScanFwdArgs& a, hipStream_t stream);
// Scratch the forward scan needs (the linear recurrence's segment maps; the
// gated one needs none).  Depends on the sizes only.
size_t scan_forward_scratch_bytes(const ScanShape& s);
// Enqueues the reverse scan and (unless a.defer_vb) the fixed-order
// reduction of `partial`; scan_backward_vb describes that reduction.
hipError_t scan_backward_launch(const ScanShape& s, const ScanBwdArgs& a, hipStream_t stream);
size_t scan_backward_partial_bytes(const ScanShape& s);
VbSum scan_backward_vb(const ScanShape& s, const ScanBwdArgs& a);

// ----------------------------------------------------------------- timing
// Measurement hook: while a caller has armed it (sru_timing_begin), every
// kernel launch is bracketed by two hipEventRecord calls on its stream and
// labelled.  Disarmed (the default) it costs one thread-local load.
void timing_before(const char* label, hipStream_t stream);
void timing_after(hipStream_t stream);

}  // namespace sru
