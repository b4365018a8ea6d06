/*
 * sru.h -- C ABI of libsru.so, an MI355X (gfx950) implementation of one
 * Simple Recurrent Unit layer (Lei et al., "Simple Recurrent Units for Highly
 * Parallelizable Recurrence", EMNLP 2018).
 *
 * The layer (Sec. 3, Eq. 1-4), per direction, for t in the direction's order:
 *   f_t = sigma(W_f x_t + v_f * c_{t-1} + b_f)
 *   c_t = f_t * c_{t-1} + (1 - f_t) * (W x_t)
 *   r_t = sigma(W_r x_t + v_r * c_{t-1} + b_r)
 *   h_t = r_t * c_t + (1 - r_t) * x_hat_t
 * computed as in Sec. 3.1: one matrix product U = X [W; W_f; W_r]^T over all
 * L*B tokens, then one fused element-wise scan, parallel over (batch, hidden
 * unit, direction) and sequential over t (Algorithm 1).  The reset gate reads
 * c_{t-1} as Eq. 3 writes it.
 *
 * x_hat: when d_in == d there are k = 3 weight blocks and x_hat_t = x_t
 * (Eq. 4).  When d_in != d, Eq. 4 is undefined; a fourth block W_h supplies
 * x_hat_t = W_h x_t (k = 4).  k is implied by (d_in, d).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout: row-major, contiguous, fp32 unless stated.  ndir = 2 for
 *   SRU_DIR_BI, else 1.  M = L*B tokens, N = ndir*k*d projection columns.
 *     X        [L, B, d_in]
 *     W        [ndir, k, d, d_in]   (block order W, W_f, W_r[, W_h])
 *     v_f, v_r, b_f, b_r            [ndir, d]
 *     c0, c_last, dc0, dc_last      [B, ndir*d]
 *     U        [L, B, ndir, k, d]   (= [M, N], the batched projection)
 *     H, C, dH [L, B, ndir*d]       (features: forward direction first)
 *     pad_mask [L, B] uint8, nonzero = padded position, or NULL (no padding)
 *   A padded (t, b) leaves c unchanged and writes h = 0 (C holds the carried
 *   state there); its dH is ignored and it adds nothing to any gradient.
 *   SRU_DIR_REV and the second half of SRU_DIR_BI visit t = L-1 .. 0.
 * Memory: every pointer is caller-owned DEVICE memory except where stated;
 *   inputs and outputs must not alias.  The library never allocates, frees
 *   or synchronises; the caller supplies a workspace of at least the queried
 *   size (device memory, any contents, 256-byte aligned) and a stream.
 * Precision: the ABI is fp32.  SRU_GEMM_BF16 rounds the operands of the
 *   matrix products (X and W for U; dU and W for dX; dU and X for dW) to
 *   bfloat16, round-to-nearest-even, accumulating in fp32.  The scan (state,
 *   gates, highway term) is fp32 in both modes.
 * Errors: every function returns an sru_status.  All arguments are checked
 *   before anything is enqueued; on error nothing is enqueued and no output
 *   is touched.  SRU_OK means "enqueued on `stream`": execution errors
 *   surface at the caller's next synchronisation.  After SRU_E_HIP,
 *   sru_last_hip_error() returns the hipError_t (per calling thread).
 * Gradients are overwritten, never accumulated.  Results are deterministic:
 *   the same inputs give bit-identical outputs (no floating-point atomics).
 */
#ifndef SRU_H_
#define SRU_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#if defined(__GNUC__)
#define SRU_API __attribute__((visibility("default")))
#else
#define SRU_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SRU_OK = 0,
  SRU_E_NULLPTR = 1,   /* a required pointer is NULL                         */
  SRU_E_SHAPE = 2,     /* a size is <= 0, too large, or inconsistent         */
  SRU_E_FLAG = 3,      /* unknown direction / gemm dtype / gemm op           */
  SRU_E_WORKSPACE = 4, /* workspace NULL or smaller than the queried size    */
  SRU_E_HIP = 5,       /* a HIP launch failed; see sru_last_hip_error()      */
  SRU_E_ALIGN = 6      /* a pointer is not 4-byte (fp32) / 256-byte aligned  */
} sru_status;

typedef enum { SRU_DIR_FWD = 0, SRU_DIR_REV = 1, SRU_DIR_BI = 2 } sru_direction;
typedef enum { SRU_GEMM_FP32 = 0, SRU_GEMM_BF16 = 1 } sru_gemm_dtype;

/* Gate variants.  Every layer and scan call takes a `const sru_options*`;
 * NULL means Eq. 1-4 as printed: highway_scale = 1, the reset gate on
 * c_{t-1} (Eq. 3) and the gated recurrence.  The same options must be
 * passed to the forward and the backward call of a layer.  Host memory,
 * read during the call only.
 *   highway_scale: alpha in h_t = r_t c_t + (1 - r_t) alpha x_hat, the
 *     scaling correction of Sec. 3.2 (sqrt(3), or sqrt(1 + 2 e^b) for a
 *     reset-gate bias b, Appendix A).  Must be finite.
 *   reset_state: SRU_RESET_PREV, r_t = sigma(W_r x_t + v_r c_{t-1} + b_r)
 *     (Eq. 3); SRU_RESET_NEW, r_t reads c_t: the order of Algorithm 1.
 *     Anything else is SRU_E_FLAG.
 *   recurrence: SRU_RECURRENCE_GATED, Eq. 1-4; SRU_RECURRENCE_LINEAR,
 *     ablation (1) of Sec. 4.5: the point-wise v_f * c_{t-1} and
 *     v_r * c_{t-1} terms are removed from both gates, so
 *       f_t = sigma(W_f x_t + b_f),  r_t = sigma(W_r x_t + b_r)
 *     and c_t = f_t c_{t-1} + (1 - f_t) W x_t is linear in c.  v_f and v_r
 *     are then not read, dv_f and dv_r not written (all may be NULL), and
 *     reset_state has no effect (r reads no state).  The scans then run in
 *     parallel over chunks of time as well as over (b, direction, j), which
 *     keeps the GPU busy when B*ndir*d is small; with fewer than 128*64
 *     such lanes, time is also cut into segments run by separate
 *     workgroups, whose maps are kept in the workspace (the queried sizes
 *     always include this scratch, so the gated recurrence may be passed a
 *     workspace sized for either).  Anything else is SRU_E_FLAG. */
typedef enum { SRU_RESET_PREV = 0, SRU_RESET_NEW = 1 } sru_reset_state;
typedef enum { SRU_RECURRENCE_GATED = 0, SRU_RECURRENCE_LINEAR = 1 } sru_recurrence;
typedef struct {
  float highway_scale;
  int reset_state;
  int recurrence;
} sru_options;

/* Human-readable name of a status code (static string, never NULL). */
SRU_API const char* sru_status_string(int status);

/* hipError_t of the last SRU_E_HIP returned to the calling thread. */
SRU_API int sru_last_hip_error(void);

/* ABI version: (major << 16) | minor. */
SRU_API int sru_version(void);

/* Workspace bytes sru_forward / sru_backward need for these sizes (0 means
 * none; NULL may then be passed).  Returns 0 for invalid arguments as well;
 * the compute call reports those.  The sizes cover both recurrences; an
 * fp32 forward of the gated recurrence needs none and accepts NULL. */
SRU_API size_t sru_forward_workspace_bytes(int L, int B, int d_in, int d, int direction,
                                   int gemm_dtype);
SRU_API size_t sru_backward_workspace_bytes(int L, int B, int d_in, int d, int direction,
                                    int gemm_dtype);

/*
 * Forward pass of one layer (Sec. 3 Eq. 1-4, organised as Sec. 3.1 /
 * Algorithm 1).
 *   in : X, W, v_f, v_r, b_f, b_r; c0 (NULL = zeros); pad_mask (NULL = none)
 *   out: U [M, N] -- the batched projection, kept by the caller for
 *        sru_backward;
 *        H [L, B, ndir*d];
 *        C [L, B, ndir*d] -- every state c_t, needed by sru_backward
 *        (NULL = do not store: inference);
 *        U may be NULL too when C is NULL and sru_forward_fused_available
 *        says so (bf16 products, d % 64 == 0): the projection and the scan
 *        then run as one kernel and U never reaches memory (H and c_last
 *        are bit-identical to the unfused call's).  Otherwise a NULL U is
 *        SRU_E_NULLPTR;
 *        c_last [B, ndir*d] -- state after each sequence's last valid step
 *        (NULL = do not store).
 *   bf16 companions (gemm_dtype = SRU_GEMM_BF16 only, else they must be
 *   NULL; each may be NULL; 16-byte aligned device buffers of uint16 bf16
 *   bit patterns, rounded to nearest even):
 *        X_bf16 [M, d_in] in -- X rounded to bf16, e.g. the H_bf16 of the
 *        layer below; it must equal that rounding of X (it replaces X as the
 *        projection operand).  NULL: X is rounded into the workspace.
 *        W_bf16 [N, d_in] out -- Wcat rounded to bf16, for sru_backward.
 *        With W = NULL it is an input instead: the weights already rounded
 *        (e.g. held in bf16 across inference calls, rounded once with
 *        sru_round_bf16); the forward reads them and rounds nothing.  A
 *        NULL W with a NULL W_bf16, or in fp32 mode, is SRU_E_NULLPTR.
 *        H_bf16 [L, B, ndir*d] out -- H rounded to bf16 (the next layer's
 *        X_bf16).
 */
/* 1 when sru_forward accepts U = NULL with C = NULL for these sizes (the
 * fused projection + scan of inference), else 0: bf16 products, d % 64 == 0,
 * d_in % 8 == 0, bf16 operands below 2 GiB, and either L <= 128 or
 * ndir * (d / 64) * ceil(B / 2) >= 256 (enough tiles of two sequences to
 * give every CU of the chip one; with fewer, the separate projection and
 * scan are faster on long sequences). */
SRU_API int sru_forward_fused_available(int L, int B, int d_in, int d, int direction,
                                        int gemm_dtype);

SRU_API int sru_forward(const float* X, const float* W,
                const float* v_f, const float* v_r, const float* b_f, const float* b_r,
                const float* c0, int L, int B, int d_in, int d, int direction,
                const uint8_t* pad_mask, int gemm_dtype, const sru_options* options,
                float* U, float* H, float* C, float* c_last,
                const uint16_t* X_bf16, uint16_t* W_bf16, uint16_t* H_bf16,
                void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * sru_forward without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid allocation): the same arguments, results and errors as
 * sru_forward, minus workspace and workspace_bytes.  Its workspace lives in
 * a static device array of SRU_NOALLOC_SCRATCH_BYTES (128 MiB) that each GPU
 * the library runs on holds until the process ends; the call itself
 * allocates and frees nothing.  Shapes whose forward workspace
 * (sru_forward_workspace_bytes) exceeds that size return SRU_E_WORKSPACE
 * before anything is enqueued.  It runs on the current device, which
 * `stream` must belong to; the first call on a device looks up the array's
 * address there (a HIP failure then returns SRU_E_HIP).  Every call on one
 * device shares that device's array: calls whose execution overlaps on one
 * GPU (other streams, other threads) race on it and must be serialised by
 * the caller.  The array keeps the last call's contents; nothing in it needs
 * to start at zero.
 */
#define SRU_NOALLOC_SCRATCH_BYTES (128u << 20)
SRU_API int sru_forward_noalloc(const float* X, const float* W,
                const float* v_f, const float* v_r, const float* b_f, const float* b_r,
                const float* c0, int L, int B, int d_in, int d, int direction,
                const uint8_t* pad_mask, int gemm_dtype, const sru_options* options,
                float* U, float* H, float* C, float* c_last,
                const uint16_t* X_bf16, uint16_t* W_bf16, uint16_t* H_bf16,
                hipStream_t stream);

/*
 * Backward pass of one layer: the chain rule of Eq. 1-4 taken in reverse
 * step order (the paper trains by back-propagation but does not state it).
 *   in : the forward inputs, U and C from sru_forward on those inputs,
 *        dH [L, B, ndir*d] (gradient of the loss w.r.t. H), dc_last
 *        [B, ndir*d] (w.r.t. c_last; NULL = zeros).
 *   out: dX [L, B, d_in], dW [ndir, k, d, d_in], dv_f, dv_r, db_f, db_r
 *        [ndir, d], dc0 [B, ndir*d] (NULL = do not compute).
 *   bf16 companions (SRU_GEMM_BF16 only, else NULL; each may be NULL; as
 *   in sru_forward): X_bf16 = X rounded to bf16; W_bf16 = Wcat rounded to
 *   bf16 (the W_bf16 sru_forward wrote; the dX product reads its transposed
 *   copy, made in the workspace).  NULL: rounded into the workspace.  W
 *   may be NULL when W_bf16 is given (weights held in bf16, as in
 *   sru_forward); dW is still written in fp32.
 * With the gated recurrence, a sequence cut into consecutive calls
 * (c_last -> c0 forward, dc0 -> dc_last backward) gives one call's results
 * bit for bit, except the backward with 8,192 to 32,767 lanes
 * (B * ndir * d): there the reverse scan runs in time-parallel chunks (the
 * gradient recurrence is affine given C), and the calls agree with one
 * call to fp32 rounding, as the linear recurrence's chunked scans do at
 * every size.
 */
SRU_API int sru_backward(const float* X, const float* W,
                 const float* v_f, const float* v_r, const float* b_f, const float* b_r,
                 const float* c0, int L, int B, int d_in, int d, int direction,
                 const uint8_t* pad_mask, int gemm_dtype, const sru_options* options,
                 const float* U, const float* C, const float* dH, const float* dc_last,
                 float* dX, float* dW, float* dv_f, float* dv_r, float* db_f, float* db_r,
                 float* dc0, const uint16_t* X_bf16, const uint16_t* W_bf16,
                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Low-rank projection: the bottleneck trick of Sec. 4.4, the stacked weights
 * re-parameterised as a product of two smaller matrices:
 *     Wcat [ndir*k*d, d_in] = P Q^T,  Q [d_in, dp],  P [ndir, k, d, dp].
 * (The text prints P^T Q, which does not compose with the shapes it states;
 * P Q^T is the reading taken.)  The layer is otherwise the one of
 * sru_forward / sru_backward, with the same conventions and options.
 *   forward : T = X Q [L, B, dp] -- an output, kept by the caller for the
 *             backward -- then U = T P^T and the scan.
 *   backward: the reverse scan, then dT = dU P, dX = dT Q^T (+ the highway
 *             gradient when k = 3), dP = dU^T T and dQ = X^T dT.
 * bf16 mode rounds the operands of each product (X and Q, T and P, dU and
 * P, dT and Q, dU and T, X and dT), and needs d_in, dp and ndir*k*d to be
 * multiples of 8 (else SRU_E_SHAPE).  Workspace as queried.
 * bf16 companions (SRU_GEMM_BF16 only, else NULL; each may be NULL; as for
 * sru_forward / sru_backward): X_bf16 [M, d_in] in -- X rounded to bf16
 * (e.g. the H_bf16 of the layer below); T_bf16 [M, dp] -- out of the
 * forward (T rounded to bf16, written with T), in to the backward (it must
 * be that rounding of T); H_bf16 [L, B, ndir*d] out -- H rounded to bf16.
 */
SRU_API size_t sru_forward_lowrank_workspace_bytes(int L, int B, int d_in, int d, int dp,
                                                   int direction, int gemm_dtype);
SRU_API size_t sru_backward_lowrank_workspace_bytes(int L, int B, int d_in, int d, int dp,
                                                    int direction, int gemm_dtype);
SRU_API int sru_forward_lowrank(const float* X, const float* Q, const float* P,
                        const float* v_f, const float* v_r, const float* b_f, const float* b_r,
                        const float* c0, int L, int B, int d_in, int d, int dp, int direction,
                        const uint8_t* pad_mask, int gemm_dtype, const sru_options* options,
                        float* T, float* U, float* H, float* C, float* c_last,
                        const uint16_t* X_bf16, uint16_t* T_bf16, uint16_t* H_bf16,
                        void* workspace, size_t workspace_bytes, hipStream_t stream);
SRU_API int sru_backward_lowrank(const float* X, const float* Q, const float* P,
                         const float* v_f, const float* v_r, const float* b_f, const float* b_r,
                         const float* c0, int L, int B, int d_in, int d, int dp, int direction,
                         const uint8_t* pad_mask, int gemm_dtype, const sru_options* options,
                         const float* T, const float* U, const float* C, const float* dH,
                         const float* dc_last, float* dX, float* dQ, float* dP,
                         float* dv_f, float* dv_r, float* db_f, float* db_r, float* dc0,
                         const uint16_t* X_bf16, const uint16_t* T_bf16,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Component entry points: the individual steps of the two calls above, with
 * the same conventions, for testing and per-kernel measurement.
 * ------------------------------------------------------------------------- */

typedef enum {
  SRU_OP_NT = 0, /* C[M,N] = A[M,K] * B[N,K]^T   (U = X W^T)     */
  SRU_OP_NN = 1, /* C[M,N] = A[M,K] * B[K,N]     (dX = dU W)     */
  SRU_OP_TN = 2  /* C[M,N] = A[K,M]^T * B[K,N]   (dW = dU^T X)   */
} sru_gemm_op;

/* bf16 rounding (round to nearest even) of n fp32 values: the operand copy
 * the bf16 companions expect.  A caller that feeds the same X to a layer's
 * forward and backward rounds it once here and passes the copy as X_bf16 to
 * both.  src, dst: device memory, 16-byte aligned, not overlapping; n >= 0
 * (0 enqueues nothing). */
SRU_API int sru_round_bf16(const float* src, size_t n, uint16_t* dst, hipStream_t stream);

/* Matrix product on the MFMA units (the batched projection of Sec. 3.1 and
 * its two backward products).  Row-major operands with leading dimensions
 * lda, ldb, ldc (elements).  gemm_dtype as above.  TN may split the
 * reduction; it then needs sru_gemm_workspace_bytes of workspace. */
SRU_API size_t sru_gemm_workspace_bytes(int op, int M, int N, int K, int gemm_dtype);
SRU_API int sru_gemm(int op, int gemm_dtype, int M, int N, int K,
             const float* A, int lda, const float* B, int ldb, float* C, int ldc,
             void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The fused forward scan (Algorithm 1 with the Eq. 3 reading) on a given U.
 * X is read only when k = 3 (d_in == d).  C, c_last and H_bf16 (bf16 copy
 * of H, 2-byte aligned) may be NULL.  Workspace:
 * sru_scan_forward_workspace_bytes, used by the linear recurrence only (the
 * gated one accepts NULL); 256-byte aligned. */
SRU_API size_t sru_scan_forward_workspace_bytes(int L, int B, int d_in, int d, int direction);
SRU_API int sru_scan_forward(const float* U, const float* X,
                     const float* v_f, const float* v_r, const float* b_f, const float* b_r,
                     const float* c0, int L, int B, int d_in, int d, int direction,
                     const uint8_t* pad_mask, const sru_options* options, float* H, float* C,
                     float* c_last, uint16_t* H_bf16, void* workspace, size_t workspace_bytes,
                     hipStream_t stream);

/* The reverse-time gradient scan on a given U, C, dH.
 *   out: dU [L, B, ndir, k, d] (gradient w.r.t. the projections; when k = 4
 *        block 3 holds the highway gradient), dxh [L, B, ndir, d] (highway
 *        gradient w.r.t. x_t when k = 3; must be NULL when k = 4), dv_f,
 *        dv_r, db_f, db_r [ndir, d], dc0 (NULL = skip).
 * Workspace: sru_scan_backward_workspace_bytes. */
SRU_API size_t sru_scan_backward_workspace_bytes(int L, int B, int d_in, int d, int direction);
SRU_API int sru_scan_backward(const float* U, const float* X, const float* C, const float* dH,
                      const float* dc_last,
                      const float* v_f, const float* v_r, const float* b_f, const float* b_r,
                      const float* c0, int L, int B, int d_in, int d, int direction,
                      const uint8_t* pad_mask, const sru_options* options,
                      float* dU, float* dxh, float* dv_f, float* dv_r, float* db_f,
                      float* db_r, float* dc0,
                      void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Measurement hook, per calling thread.  sru_timing_begin arms it with
 * `capacity` events the caller created (hipEventCreate, timing enabled).
 * Every kernel this thread then enqueues through the calls above is
 * bracketed by two of them, recorded on the kernel's stream in launch order:
 * kernel i runs between events[2i] and events[2i+1].  When the events run
 * out, further kernels are not bracketed.  sru_timing_end disarms the hook
 * and returns the number of kernels bracketed; sru_timing_label(i) names
 * kernel i until the next sru_timing_begin ("" out of range):
 *   products: "gemm_u", "gemm_dx", "gemm_dw" (layer calls), "gemm_t",
 *     "gemm_dt", "gemm_dp", "gemm_dq" (low-rank calls), "gemm_nt",
 *     "gemm_nn", "gemm_tn" (sru_gemm), "splitk_reduce";
 *   bf16 operand copies: "bf16_w", "bf16_x", "bf16_wt", "bf16_q", "bf16_p",
 *     "bf16_t";
 *   scans: "scan_fwd", "scan_bwd", "reduce_vb", and "proj_scan_fwd" (the
 *     fused projection + scan of inference).
 * The caller owns the events and reads them after synchronising.
 * Disarmed (the default), launches record nothing.
 * ------------------------------------------------------------------------- */
SRU_API int sru_timing_begin(hipEvent_t* events, int capacity);
SRU_API int sru_timing_end(void);
SRU_API const char* sru_timing_label(int i);

#ifdef __cplusplus
}
#endif

#endif /* SRU_H_ */
