// C ABI of libsru.so: argument validation, workspace layout and dispatch.
// Every check runs before anything is enqueued; nothing here allocates,
// frees or synchronises.
#include <limits.h>

#include <cmath>

#include <algorithm>
#include <initializer_list>
#include <mutex>
#include <vector>

#include "../../include/sru.h"
#include "sru_internal.h"

namespace {

// Per-thread state of the measurement hook.
struct TimingState {
  hipEvent_t* events = nullptr;
  int capacity = 0;  // events available
  int used = 0;      // events recorded
  std::vector<const char*> labels;
};
thread_local TimingState g_timing;

thread_local int g_last_hip_error = 0;

constexpr size_t kAlign = 256;
constexpr long long kMaxElems = 1LL << 40;  // per tensor, far beyond any HBM size
// dX (fp32) above this size runs after dW in the backward (see sru_backward)
constexpr long long kDxLastBytes = 32LL << 20;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool valid_direction(int d) { return d == SRU_DIR_FWD || d == SRU_DIR_REV || d == SRU_DIR_BI; }
bool valid_dtype(int t) { return t == SRU_GEMM_FP32 || t == SRU_GEMM_BF16; }

bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3) == 0; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// The optional bf16 companions: only with bf16 GEMMs, 16-byte aligned.
int check_bf16_side(int gemm_dtype, std::initializer_list<const void*> ptrs) {
  for (const void* p : ptrs) {
    if (!p) continue;
    if (gemm_dtype != SRU_GEMM_BF16) return SRU_E_FLAG;
    if (!aligned16(p)) return SRU_E_ALIGN;
  }
  return SRU_OK;
}

struct Dims {
  int L, B, d_in, d, ndir, k;
  long long M, N, nfeat;
};

// dX runs after dW when it is large: the layer below's backward scan reads
// it as dH next, and then still finds much of it in the caches (measured:
// L 256, B 64, d 1024 and L 128, B 128, d 2048 ran 0.6 % and 1.1 % faster
// per step; with dX of 8 MB, at B 8, 0.8 % slower, so small ones keep dX
// first)
bool dx_last(const Dims& s) { return 4LL * s.M * s.d_in > kDxLastBytes; }

// Shape checks shared by every layer entry point.  Sizes must be positive,
// products must fit the 32-bit indices the kernels use for tokens, columns
// and lanes, and no tensor may exceed kMaxElems elements.
int make_dims(int L, int B, int d_in, int d, int direction, Dims& s) {
  if (!valid_direction(direction)) return SRU_E_FLAG;
  if (L <= 0 || B <= 0 || d_in <= 0 || d <= 0) return SRU_E_SHAPE;
  s.L = L;
  s.B = B;
  s.d_in = d_in;
  s.d = d;
  s.ndir = direction == SRU_DIR_BI ? 2 : 1;
  s.k = d_in == d ? 3 : 4;
  s.M = (long long)L * B;
  s.N = (long long)s.ndir * s.k * d;
  s.nfeat = (long long)s.ndir * d;
  if (s.M > INT_MAX || s.N > INT_MAX || (long long)B * s.nfeat > INT_MAX) return SRU_E_SHAPE;
  if (s.M * s.N > kMaxElems || s.M * d_in > kMaxElems) return SRU_E_SHAPE;
  return SRU_OK;
}

// The gate variants of an entry point (NULL = Eq. 1-4 as printed).
struct Opts {
  float alpha = 1.0f;
  int reset_new = 0;
  int linear = 0;  // v * c_{t-1} removed: v_f, v_r, dv_f, dv_r unused (may be NULL)
};

int read_options(const sru_options* o, Opts& op) {
  if (!o) return SRU_OK;
  if (!std::isfinite(o->highway_scale)) return SRU_E_FLAG;
  if (o->reset_state != SRU_RESET_PREV && o->reset_state != SRU_RESET_NEW) return SRU_E_FLAG;
  if (o->recurrence != SRU_RECURRENCE_GATED && o->recurrence != SRU_RECURRENCE_LINEAR)
    return SRU_E_FLAG;
  op.alpha = o->highway_scale;
  op.linear = o->recurrence == SRU_RECURRENCE_LINEAR;
  // without v the reset gate reads no state, so the two orders coincide
  op.reset_new = !op.linear && o->reset_state == SRU_RESET_NEW;
  return SRU_OK;
}

sru::ScanShape scan_shape(const Dims& s, int direction, const Opts& op = Opts()) {
  return sru::ScanShape{s.L, s.B, s.d_in, s.d, s.ndir, s.k, direction, op.alpha, op.reset_new,
                        op.linear};
}

// v_f, v_r (and dv_f, dv_r) are required by the gated recurrence only
bool missing_v(const Opts& op, const void* a, const void* b) { return !op.linear && (!a || !b); }

int hip_status(hipError_t e) {
  if (e == hipSuccess) return SRU_OK;
  g_last_hip_error = (int)e;
  return SRU_E_HIP;
}

sru::GemmDesc gemm_desc(int op, bool bf16, int M, int N, int K, const void* A, long long lda,
                        const void* B, long long ldb, float* C, long long ldc) {
  sru::GemmDesc g{};
  g.A = A;
  g.B = B;
  g.C = C;
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.a_kc = op != SRU_OP_TN;
  g.b_kc = op == SRU_OP_NT;
  g.bf16 = bf16;
  g.splits = 1;
  return g;
}

// Where inference (U and C not kept) runs the projection and the scan as one
// kernel: bf16 products, whole groups of 64 hidden units, whole 16-byte
// chunks of X rows, operands within the 2 GiB byte range of buffer loads.
// Every lane scans from its own accumulators, about 23 ns a step, and a
// workgroup carries c from one time block to the next, so any length runs;
// it is the faster organisation at up to 128 steps (1.3-2x, measured), and
// beyond that where tiles of two sequences give every CU a workgroup
// (1.2-1.65x at 256-512 steps; even at 128 workgroups, slower below).
constexpr int kFusedShortL = 128;
constexpr long long kFusedMinGroups = 256;
bool fused_ok(const Dims& s, int gemm_dtype) {
  const long long groups = (long long)s.ndir * (s.d / 64) * ((s.B + 1) / 2);
  return gemm_dtype == SRU_GEMM_BF16 && (s.L <= kFusedShortL || groups >= kFusedMinGroups) &&
         s.d % 64 == 0 && s.d_in % 8 == 0 && 2 * s.M * s.d_in < (1LL << 31) &&
         2 * s.N * s.d_in < (1LL << 31);
}

// Sequences per fused tile (bb = 2, 4 or 8: the tile holds 256 / bb steps of
// each, in time chunks of 32).  A workgroup runs its time blocks one after
// another, each a product (about 1.4 us per 64 of d_in, plus 4 us) and a
// serial scan of 256 / bb steps (about 25 ns each, plus 0.5 us per chunk
// for the hand-over of c); the workgroups fill the 256 CUs in rounds.  The
// plan with the least modelled time wins: on the 9 shapes measured it picked
// the fastest plan, or one within 2 % of it.
int fused_seqs_per_tile(const Dims& s) {
  int best = 2;
  long long best_cost = -1;
  for (int bb : {2, 4, 8}) {
    const long long tb = 256 / bb;
    const long long groups = (long long)s.ndir * (s.d / 64) * ((s.B + bb - 1) / bb);
    const long long rounds = (groups + 255) / 256;
    const long long blocks = (s.L + tb - 1) / tb;
    // in units of 25 ns
    const long long cost = rounds * blocks * (56 * ((s.d_in + 63) / 64) + 160 + tb + 20 * (tb / 32));
    if (best_cost < 0 || cost < best_cost) {
      best = bb;
      best_cost = cost;
    }
  }
  return best;
}

// Scratch of the scans.  The linear recurrence's scans cut time into
// segments when the lanes alone cannot fill the chip, and keep the segments'
// maps (and, backward, one row of partial sums per segment); the sizes
// depend on L, B, d and the number of directions only, and the workspace
// sizes cover both recurrences, so one size serves every option.
sru::ScanShape linear_shape(const Dims& s) {
  Opts op;
  op.linear = 1;
  return scan_shape(s, 0, op);
}
size_t scan_fwd_scratch(const Dims& s) {
  return align_up(sru::scan_forward_scratch_bytes(linear_shape(s)));
}
size_t scan_bwd_partial(const Dims& s) {
  return align_up(std::max(sru::scan_backward_partial_bytes(scan_shape(s, 0)),
                           sru::scan_backward_partial_bytes(linear_shape(s))));
}

// Forward workspace: [bf16 copies of W [N, d_in] and X [M, d_in] (bf16
// mode: the operands of the projection) | scan scratch].
size_t fwd_bf16_bytes(const Dims& s, int gemm_dtype) {
  if (gemm_dtype != SRU_GEMM_BF16) return 0;
  return align_up(2 * (size_t)s.N * (size_t)s.d_in) + align_up(2 * (size_t)s.M * (size_t)s.d_in);
}
size_t fwd_workspace(const Dims& s, int gemm_dtype) {
  return fwd_bf16_bytes(s, gemm_dtype) + scan_fwd_scratch(s);
}

// The dW product of sru_backward (the workspace is sized from this same
// descriptor, so the split count it is sized for is the one launched).
sru::GemmDesc dw_desc(const Dims& s, bool bf16, const void* dU, const void* X, float* dW) {
  sru::GemmDesc g = gemm_desc(SRU_OP_TN, bf16, (int)s.N, s.d_in, (int)s.M, dU, s.N, X, s.d_in,
                              dW, s.d_in);
  g.a_bf16 = g.b_bf16 = bf16;
  g.label = "gemm_dw";
  return g;
}

// Backward workspace layout:
//   [dU (fp32, or bf16 in bf16 mode) | dxh (k = 3) | v/b partials |
//    Wcat^T and X in bf16 (bf16 mode) | split partials]
// The split partials of dW and dX share one region, each product's sum
// running before the other product starts; when both are split and dX runs
// first, dX's sum runs in dW's split-sum launch (one launch less), and dX's
// partials then follow dW's.
struct BwdLayout {
  size_t dU, dxh, partial, wt, xb, splitk, splitk_dx, total;
  int splits, splits_dx;
  bool joint_sum;
};

// dX = dU Wcat (+ highway): NN on Wcat in fp32 mode; in bf16 mode NT on the
// bf16 Wcat^T.  Its tiles can be too few to fill the CUs (d_in of a few
// hundred, or few tokens: one GPU's share of a batch), so it may be split
// over K; the launcher's plan decides.
// With k = 3 the product adds every direction's highway gradient dxh.  The
// addend is part of the descriptor the workspace is sized from, since it
// decides the tile shape and with it the split count.
sru::GemmDesc dx_desc(const Dims& s, bool bf16, const void* dU, const void* W, const void* wt,
                      float* dX, const float* dxh) {
  sru::GemmDesc g = bf16 ? gemm_desc(SRU_OP_NT, true, (int)s.M, s.d_in, (int)s.N, dU, s.N, wt,
                                     s.N, dX, s.d_in)
                         : gemm_desc(SRU_OP_NN, false, (int)s.M, s.d_in, (int)s.N, dU, s.N, W,
                                     s.d_in, dX, s.d_in);
  g.a_bf16 = g.b_bf16 = bf16;
  g.kc_split = true;
  g.label = "gemm_dx";
  if (s.k == 3) {
    g.add = dxh;
    g.add_ld = s.nfeat;
    g.add_off = s.d;
    g.add_count = s.ndir;
  }
  return g;
}

BwdLayout bwd_layout(const Dims& s, int gemm_dtype) {
  const bool bf16 = gemm_dtype == SRU_GEMM_BF16;
  BwdLayout w{};
  size_t off = 0;
  w.dU = off;
  off += align_up((bf16 ? 2 : 4) * (size_t)s.M * (size_t)s.N);
  w.dxh = off;
  if (s.k == 3) off += align_up(sizeof(float) * (size_t)s.M * (size_t)s.nfeat);
  w.partial = off;
  off += scan_bwd_partial(s);
  w.wt = off;
  if (bf16) off += align_up(2 * (size_t)s.N * (size_t)s.d_in);
  w.xb = off;
  if (bf16) off += align_up(2 * (size_t)s.M * (size_t)s.d_in);
  w.splits = sru::gemm_splits(dw_desc(s, bf16, nullptr, nullptr, nullptr));
  w.splits_dx = sru::gemm_splits(dx_desc(s, bf16, nullptr, nullptr, nullptr, nullptr, nullptr));
  w.joint_sum = w.splits > 1 && w.splits_dx > 1 && !dx_last(s);
  const size_t pw = sru::gemm_partial_bytes((int)s.N, s.d_in, w.splits);
  const size_t px = sru::gemm_partial_bytes((int)s.M, s.d_in, w.splits_dx);
  w.splitk = off;
  if (w.joint_sum) {
    w.splitk_dx = off + align_up(pw);
    off += align_up(pw) + align_up(px);
  } else {
    w.splitk_dx = off;  // shared: the products run one after the other
    off += align_up(std::max(pw, px));
  }
  w.total = off;
  return w;
}

// ---------------------------------------------------------------- low rank
// Wcat = P Q^T (Sec. 4.4).  Products, with M = L*B, N = ndir*k*d, dp = d':
//   forward : T = X Q (K = d_in), U = T P^T (NT, K = dp)
//   backward: dT = dU P (K = N), dX = dT Q^T (NT, K = dp; + highway),
//             dP = dU^T T (TN, K = M), dQ = X^T dT (TN, K = M)
// fp32 mode runs T and dT as NN products.  bf16 mode rounds every operand
// (into the workspace unless the caller holds the copy) and runs each
// product on the direct kernel, which needs whole 16-byte chunks: T and dT
// as NT products on transposed bf16 copies of Q and P (K-contiguous, like
// the projection), T written in fp32 and bf16 at once, dT in bf16 only
// (only its rounding is ever read).
bool lowrank_dims_ok(const Dims& s, int dp, int gemm_dtype) {
  if (gemm_dtype != SRU_GEMM_BF16) return true;
  return s.d_in % 8 == 0 && dp % 8 == 0 && s.N % 8 == 0;
}

// [bf16 operands (bf16 mode) | scan scratch (last, so the gated
// recurrence needs only the first scr bytes)]
struct LrFwdLayout {
  size_t xb, qt, tb, pb, scr, total;
};
LrFwdLayout lr_fwd_layout(const Dims& s, int dp, int gemm_dtype) {
  LrFwdLayout w{};
  size_t off = 0;
  if (gemm_dtype == SRU_GEMM_BF16) {
    w.xb = off; off += align_up(2 * (size_t)s.M * s.d_in);
    w.qt = off; off += align_up(2 * (size_t)s.d_in * dp);  // Q^T [dp, d_in]
    w.tb = off; off += align_up(2 * (size_t)s.M * dp);
    w.pb = off; off += align_up(2 * (size_t)s.N * dp);
  }
  w.scr = off; off += scan_fwd_scratch(s);
  w.total = off;
  return w;
}

// The two reductions over tokens (dP, dQ), described for sizing and launch.
sru::GemmDesc lr_dp_desc(const Dims& s, int dp, bool bf16, const void* dU, const void* T,
                         float* dP) {
  sru::GemmDesc g = gemm_desc(SRU_OP_TN, bf16, (int)s.N, dp, (int)s.M, dU, s.N, T, dp, dP, dp);
  g.a_bf16 = g.b_bf16 = bf16;
  g.label = "gemm_dp";
  return g;
}
sru::GemmDesc lr_dq_desc(const Dims& s, int dp, bool bf16, const void* X, const void* dT,
                         float* dQ) {
  sru::GemmDesc g = gemm_desc(SRU_OP_TN, bf16, s.d_in, dp, (int)s.M, X, s.d_in, dT, dp, dQ, dp);
  g.a_bf16 = g.b_bf16 = bf16;
  g.label = "gemm_dq";
  return g;
}

struct LrBwdLayout {
  size_t dU, dxh, partial, dT, pt, qb, tb, xb, dtb, splitk, total;
  int splits_p, splits_q;
};
LrBwdLayout lr_bwd_layout(const Dims& s, int dp, int gemm_dtype) {
  const bool bf16 = gemm_dtype == SRU_GEMM_BF16;
  LrBwdLayout w{};
  size_t off = 0;
  w.dU = off; off += align_up((bf16 ? 2 : 4) * (size_t)s.M * s.N);
  w.dxh = off; if (s.k == 3) off += align_up(4 * (size_t)s.M * s.nfeat);
  w.partial = off; off += scan_bwd_partial(s);
  w.dT = off; if (!bf16) off += align_up(4 * (size_t)s.M * dp);  // bf16: dT in bf16 only
  if (bf16) {
    w.pt = off; off += align_up(2 * (size_t)s.N * dp);  // P^T [dp, N]
    w.qb = off; off += align_up(2 * (size_t)s.d_in * dp);
    w.tb = off; off += align_up(2 * (size_t)s.M * dp);
    w.xb = off; off += align_up(2 * (size_t)s.M * s.d_in);
    w.dtb = off; off += align_up(2 * (size_t)s.M * dp);
  }
  w.splits_p = sru::gemm_splits(lr_dp_desc(s, dp, bf16, nullptr, nullptr, nullptr));
  w.splits_q = sru::gemm_splits(lr_dq_desc(s, dp, bf16, nullptr, nullptr, nullptr));
  w.splitk = off;
  off += align_up(std::max(sru::gemm_partial_bytes((int)s.N, dp, w.splits_p),
                           sru::gemm_partial_bytes(s.d_in, dp, w.splits_q)));
  w.total = off;
  return w;
}

// Scratch of sru_forward_noalloc: the forward's workspace (bf16 operand
// copies, the linear recurrence's segment maps) in a file-scope device array,
// so that call allocates nothing.  Host code never passes the array's name to
// a kernel or a copy (on the host it is only a stand-in symbol): it uses the
// device address hipGetSymbolAddress returns, looked up once per device with
// that device current, on the device's first call.
__device__ __align__(256) unsigned char scratch[SRU_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 256;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device.
int scratch_on_current_device(void** out) {
  int dev = -1;
  if (int e = hip_status(hipGetDevice(&dev))) return e;
  if (dev < 0 || dev >= kMaxDevices) return SRU_E_SHAPE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (int e = hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)))) return e;
    if (!p) return SRU_E_NULLPTR;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SRU_OK;
}

}  // namespace

namespace sru {

void timing_before(const char* label, hipStream_t stream) {
  TimingState& t = g_timing;
  if (!t.events || t.used + 2 > t.capacity) return;
  hipEventRecord(t.events[t.used++], stream);
  t.labels.push_back(label);
}

void timing_after(hipStream_t stream) {
  TimingState& t = g_timing;
  // pairs with a timing_before that recorded (used is then odd)
  if (!t.events || (t.used & 1) == 0) return;
  hipEventRecord(t.events[t.used++], stream);
}

}  // namespace sru

extern "C" {

int sru_timing_begin(hipEvent_t* events, int capacity) {
  if (!events || capacity < 2) return SRU_E_NULLPTR;
  g_timing.events = events;
  g_timing.capacity = capacity;
  g_timing.used = 0;
  g_timing.labels.clear();
  return SRU_OK;
}

int sru_timing_end(void) {
  const int n = g_timing.used / 2;
  g_timing.events = nullptr;
  g_timing.capacity = 0;
  return n;
}

const char* sru_timing_label(int i) {
  if (i < 0 || i >= (int)g_timing.labels.size()) return "";
  return g_timing.labels[i];
}

const char* sru_status_string(int status) {
  switch (status) {
    case SRU_OK: return "SRU_OK";
    case SRU_E_NULLPTR: return "SRU_E_NULLPTR: a required pointer is NULL";
    case SRU_E_SHAPE: return "SRU_E_SHAPE: invalid or inconsistent size";
    case SRU_E_FLAG: return "SRU_E_FLAG: unknown direction, gemm dtype or gemm op";
    case SRU_E_WORKSPACE: return "SRU_E_WORKSPACE: workspace missing or too small";
    case SRU_E_HIP: return "SRU_E_HIP: a HIP launch failed";
    case SRU_E_ALIGN: return "SRU_E_ALIGN: misaligned pointer";
    default: return "unknown sru_status";
  }
}

int sru_last_hip_error(void) { return g_last_hip_error; }

int sru_version(void) { return (1 << 16) | 4; }

size_t sru_forward_workspace_bytes(int L, int B, int d_in, int d, int direction, int gemm_dtype) {
  Dims s;
  if (make_dims(L, B, d_in, d, direction, s) != SRU_OK || !valid_dtype(gemm_dtype)) return 0;
  return fwd_workspace(s, gemm_dtype);
}

size_t sru_backward_workspace_bytes(int L, int B, int d_in, int d, int direction,
                                    int gemm_dtype) {
  Dims s;
  if (make_dims(L, B, d_in, d, direction, s) != SRU_OK || !valid_dtype(gemm_dtype)) return 0;
  return bwd_layout(s, gemm_dtype).total;
}

int sru_forward_fused_available(int L, int B, int d_in, int d, int direction, int gemm_dtype) {
  Dims s;
  if (make_dims(L, B, d_in, d, direction, s) != SRU_OK || !valid_dtype(gemm_dtype)) return 0;
  return fused_ok(s, gemm_dtype) ? 1 : 0;
}

int sru_forward(const float* X, const float* W, const float* v_f, const float* v_r,
                const float* b_f, const float* b_r, const float* c0, int L, int B, int d_in,
                int d, int direction, const uint8_t* pad_mask, int gemm_dtype,
                const sru_options* options, float* U,
                float* H, float* C, float* c_last, const uint16_t* X_bf16, uint16_t* W_bf16,
                uint16_t* H_bf16, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  Dims s;
  int st = make_dims(L, B, d_in, d, direction, s);
  if (st != SRU_OK) return st;
  if (!valid_dtype(gemm_dtype)) return SRU_E_FLAG;
  Opts op;
  if (int e = read_options(options, op)) return e;
  // U may be omitted only where the fused projection + scan applies
  // (inference with bf16 products: C omitted too)
  const bool fused = !U && fused_ok(s, gemm_dtype) && !C;
  // bf16 products may take the weights already rounded: W = NULL, and
  // W_bf16 is then the input
  const bool w_rounded = !W && W_bf16 && gemm_dtype == SRU_GEMM_BF16;
  if (!X || (!W && !w_rounded) || missing_v(op, v_f, v_r) || !b_f || !b_r ||
      (!U && !fused) || !H)
    return SRU_E_NULLPTR;
  const void* ptrs[] = {X, W, v_f, v_r, b_f, b_r, c0, U, H, C, c_last};
  for (const void* p : ptrs)
    if (p && !aligned4(p)) return SRU_E_ALIGN;
  if (int e = check_bf16_side(gemm_dtype, {X_bf16, W_bf16, H_bf16})) return e;
  const bool bf16 = gemm_dtype == SRU_GEMM_BF16;
  const size_t bf16_bytes = fwd_bf16_bytes(s, gemm_dtype);
  const size_t need = bf16_bytes + (op.linear && !fused ? scan_fwd_scratch(s) : 0);
  if (need > 0) {
    if (!workspace || workspace_bytes < need) return SRU_E_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return SRU_E_ALIGN;
  }

  // U = X Wcat^T (Sec. 3.1).  bf16 mode: W and X rounded once (into
  // W_bf16 / the workspace, unless the caller holds X_bf16 or passes the
  // weights rounded), so both operands of the product are K-contiguous bf16.
  const void* Wop = W;
  const void* Xop = X;
  if (bf16) {
    uint16_t* wb = W_bf16 ? W_bf16 : static_cast<uint16_t*>(workspace);
    if (!w_rounded) {
      if (int e = hip_status(sru::to_bf16_launch(W, (int)s.N, d_in, wb, false, stream,
                                                 "bf16_w")))
        return e;
    }
    Wop = wb;
    if (X_bf16) {
      Xop = X_bf16;
    } else {
      uint16_t* xb = reinterpret_cast<uint16_t*>(static_cast<unsigned char*>(workspace) +
                                                 align_up(2 * (size_t)s.N * (size_t)d_in));
      if (int e = hip_status(sru::to_bf16_launch(X, (int)s.M, d_in, xb, false, stream, "bf16_x"))) return e;
      Xop = xb;
    }
  }
  if (fused) {
    sru::FusedFwdArgs f{};
    f.Xb = static_cast<const uint16_t*>(Xop);
    f.Wb = static_cast<const uint16_t*>(Wop);
    f.a_bytes = (unsigned)(2 * s.M * d_in);
    f.b_bytes = (unsigned)(2 * s.N * d_in);
    f.v_f = op.linear ? nullptr : v_f;
    f.v_r = op.linear ? nullptr : v_r;
    f.b_f = b_f;
    f.b_r = b_r;
    f.c0 = c0;
    f.mask = pad_mask;
    f.H = H;
    f.Hb = H_bf16;
    f.c_last = c_last;
    f.L = L;
    f.B = B;
    f.d_in = d_in;
    f.d = d;
    f.ndir = s.ndir;
    f.k = s.k;
    f.X = X;
    f.direction = direction;
    f.bb = fused_seqs_per_tile(s);
    f.ngroups = d / 64;
    f.nbgroups = (B + f.bb - 1) / f.bb;
    f.alpha = op.alpha;
    f.reset_new = op.reset_new;
    f.linear = op.linear;
    return hip_status(sru::proj_scan_forward_launch(f, stream));
  }
  sru::GemmDesc g = gemm_desc(SRU_OP_NT, bf16, (int)s.M, (int)s.N, d_in, Xop, d_in, Wop, d_in, U,
                              s.N);
  g.a_bf16 = g.b_bf16 = bf16;
  g.label = "gemm_u";
  if (int e = hip_status(sru::gemm_launch(g, stream))) return e;

  sru::ScanFwdArgs a{U, X, v_f, v_r, b_f, b_r, c0, pad_mask, H, C, c_last, H_bf16,
                     static_cast<unsigned char*>(workspace) + bf16_bytes};
  return hip_status(sru::scan_forward_launch(scan_shape(s, direction, op), a, stream));
}

int sru_forward_noalloc(const float* X, const float* W, const float* v_f, const float* v_r,
                        const float* b_f, const float* b_r, const float* c0, int L, int B,
                        int d_in, int d, int direction, const uint8_t* pad_mask, int gemm_dtype,
                        const sru_options* options, float* U, float* H, float* C,
                        float* c_last, const uint16_t* X_bf16, uint16_t* W_bf16,
                        uint16_t* H_bf16, hipStream_t stream) {
  Dims s;
  int st = make_dims(L, B, d_in, d, direction, s);
  if (st != SRU_OK) return st;
  if (!valid_dtype(gemm_dtype)) return SRU_E_FLAG;
  // the whole forward workspace must fit the array (checked before any HIP call)
  if (fwd_workspace(s, gemm_dtype) > (size_t)SRU_NOALLOC_SCRATCH_BYTES) return SRU_E_WORKSPACE;
  void* ws = nullptr;
  if (int e = scratch_on_current_device(&ws)) return e;
  return sru_forward(X, W, v_f, v_r, b_f, b_r, c0, L, B, d_in, d, direction, pad_mask,
                     gemm_dtype, options, U, H, C, c_last, X_bf16, W_bf16, H_bf16, ws,
                     (size_t)SRU_NOALLOC_SCRATCH_BYTES, stream);
}

int sru_backward(const float* X, const float* W, const float* v_f, const float* v_r,
                 const float* b_f, const float* b_r, const float* c0, int L, int B, int d_in,
                 int d, int direction, const uint8_t* pad_mask, int gemm_dtype,
                 const sru_options* options, const float* U,
                 const float* C, const float* dH, const float* dc_last, float* dX, float* dW,
                 float* dv_f, float* dv_r, float* db_f, float* db_r, float* dc0,
                 const uint16_t* X_bf16, const uint16_t* W_bf16, void* workspace,
                 size_t workspace_bytes, hipStream_t stream) {
  Dims s;
  int st = make_dims(L, B, d_in, d, direction, s);
  if (st != SRU_OK) return st;
  if (!valid_dtype(gemm_dtype)) return SRU_E_FLAG;
  Opts op;
  if (int e = read_options(options, op)) return e;
  // weights already rounded (bf16 products): W = NULL with W_bf16 given
  const bool w_ok = W || (W_bf16 && gemm_dtype == SRU_GEMM_BF16);
  if (!X || !w_ok || missing_v(op, v_f, v_r) || !b_f || !b_r || !U || !C || !dH || !dX || !dW ||
      missing_v(op, dv_f, dv_r) || !db_f || !db_r)
    return SRU_E_NULLPTR;
  const void* ptrs[] = {X, W, v_f, v_r, b_f, b_r, c0, U, C, dH, dc_last, dX, dW, dv_f, dv_r,
                        db_f, db_r, dc0};
  for (const void* p : ptrs)
    if (p && !aligned4(p)) return SRU_E_ALIGN;
  if (int e = check_bf16_side(gemm_dtype, {X_bf16, W_bf16})) return e;
  const BwdLayout lay = bwd_layout(s, gemm_dtype);
  if (!workspace || workspace_bytes < lay.total) return SRU_E_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return SRU_E_ALIGN;

  const bool bf16 = gemm_dtype == SRU_GEMM_BF16;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  void* dU = ws + lay.dU;
  float* dxh = s.k == 3 ? reinterpret_cast<float*>(ws + lay.dxh) : nullptr;
  float* partial = reinterpret_cast<float*>(ws + lay.partial);
  uint16_t* wt = reinterpret_cast<uint16_t*>(ws + lay.wt);
  float* splitk = reinterpret_cast<float*>(ws + lay.splitk);
  uint16_t* xb = reinterpret_cast<uint16_t*>(ws + lay.xb);
  const void* Xop = !bf16 ? static_cast<const void*>(X) : X_bf16 ? X_bf16 : xb;
  sru::GemmDesc gw = dw_desc(s, bf16, dU, Xop, dW);
  gw.partials = splitk;
  // the split partials were sized for lay.splits; refuse (before enqueueing
  // anything) rather than overrun if the launch plan ever differed
  if (sru::gemm_splits(gw) > lay.splits) return SRU_E_WORKSPACE;

  // 1. reverse gradient scan and the v/b sums; dU is written in the operand
  //    type of the products that read it
  sru::ScanBwdArgs a{U,   X,    C,   dH,      dc_last, v_f,  v_r,  b_f,  b_r,  c0,
                     pad_mask, dU, bf16, dxh, partial, dc0, dv_f, dv_r, db_f, db_r};
  // the v/b sums over the batch run with the dW product (in its split-K
  // sum's launch when it has one)
  a.defer_vb = true;
  gw.vb = sru::scan_backward_vb(scan_shape(s, direction, op), a);
  if (int e = hip_status(sru::scan_backward_launch(scan_shape(s, direction, op), a, stream)))
    return e;

  // 2-3. dW = dU^T X (reduction over all tokens, split over K) and dX = dU
  //    Wcat (+ the highway gradient of every direction when k = 3).  bf16
  //    mode: dW reads X in bf16 (X_bf16, or rounded into the workspace), both
  //    operands row-contiguous; dX reads Wcat^T rounded to bf16 into the
  //    workspace (a transposed copy of W_bf16 when the caller holds it, else
  //    rounded from W), both operands K-contiguous, so it runs at the speed
  //    of the projection.  Split partials: see BwdLayout (with both
  //    products split and dX first, one launch sums both).
  auto run_dw = [&]() -> int {
    if (bf16 && !X_bf16) {
      if (int e = hip_status(sru::to_bf16_launch(X, (int)s.M, d_in, xb, false, stream, "bf16_x")))
        return e;
    }
    return hip_status(sru::gemm_launch(gw, stream));
  };
  sru::GemmDesc gx = dx_desc(s, bf16, dU, W, wt, dX, dxh);
  gx.partials = reinterpret_cast<float*>(ws + lay.splitk_dx);
  // split as planned, else (a plan that differs at run time) not at all
  if (sru::gemm_splits(gx) > lay.splits_dx) gx.kc_split = false;
  if (lay.joint_sum && sru::gemm_splits(gx) > 1 && sru::gemm_splits(gw) > 1) {
    // dX runs first; its split sum runs in dW's split-sum launch
    gx.defer_sum = true;
    gw.extra = sru::gemm_split_sum(gx);
  }
  auto run_dx = [&]() -> int {
    if (bf16) {
      const hipError_t te = W_bf16
          ? sru::to_bf16_t_launch(W_bf16, true, (int)s.N, d_in, wt, stream, "bf16_wt")
          : sru::to_bf16_t_launch(W, false, (int)s.N, d_in, wt, stream, "bf16_wt");
      if (int e = hip_status(te)) return e;
    }
    return hip_status(sru::gemm_launch(gx, stream));
  };
  if (dx_last(s)) {
    if (int e = run_dw()) return e;
    return run_dx();
  }
  if (int e = run_dx()) return e;
  return run_dw();
}

int sru_round_bf16(const float* src, size_t n, uint16_t* dst, hipStream_t stream) {
  if (n == 0) return SRU_OK;
  if (!src || !dst) return SRU_E_NULLPTR;
  if (n > (size_t)kMaxElems) return SRU_E_SHAPE;
  if (!aligned16(src) || !aligned16(dst)) return SRU_E_ALIGN;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + 2 * n && d0 < s0 + 4 * n) return SRU_E_SHAPE;  // overlapping buffers
  return hip_status(sru::to_bf16_n_launch(src, (long long)n, dst, stream, "bf16_x"));
}

size_t sru_gemm_workspace_bytes(int op, int M, int N, int K, int gemm_dtype) {
  if (op < SRU_OP_NT || op > SRU_OP_TN || !valid_dtype(gemm_dtype)) return 0;
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  sru::GemmDesc g = gemm_desc(op, gemm_dtype == SRU_GEMM_BF16, M, N, K, nullptr, 0, nullptr, 0,
                              nullptr, 0);
  return align_up(sru::gemm_partial_bytes(M, N, sru::gemm_splits(g)));
}

int sru_gemm(int op, int gemm_dtype, int M, int N, int K, const float* A, int lda,
             const float* B, int ldb, float* C, int ldc, void* workspace,
             size_t workspace_bytes, hipStream_t stream) {
  if (op < SRU_OP_NT || op > SRU_OP_TN || !valid_dtype(gemm_dtype)) return SRU_E_FLAG;
  if (M <= 0 || N <= 0 || K <= 0) return SRU_E_SHAPE;
  if (!A || !B || !C) return SRU_E_NULLPTR;
  // leading dimensions cover a row of the stored layout
  const int a_row = op == SRU_OP_TN ? M : K;
  const int b_row = op == SRU_OP_NT ? K : N;
  if (lda < a_row || ldb < b_row || ldc < N) return SRU_E_SHAPE;
  if ((long long)M * N > kMaxElems) return SRU_E_SHAPE;
  if (!aligned4(A) || !aligned4(B) || !aligned4(C)) return SRU_E_ALIGN;
  sru::GemmDesc g = gemm_desc(op, gemm_dtype == SRU_GEMM_BF16, M, N, K, A, lda, B, ldb, C, ldc);
  const size_t need = align_up(sru::gemm_partial_bytes(M, N, sru::gemm_splits(g)));
  if (need > 0) {
    if (!workspace || workspace_bytes < need) return SRU_E_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return SRU_E_ALIGN;
    g.partials = static_cast<float*>(workspace);
  }
  return hip_status(sru::gemm_launch(g, stream));
}

size_t sru_scan_forward_workspace_bytes(int L, int B, int d_in, int d, int direction) {
  Dims s;
  if (make_dims(L, B, d_in, d, direction, s) != SRU_OK) return 0;
  return scan_fwd_scratch(s);
}

int sru_scan_forward(const float* U, const float* X, const float* v_f, const float* v_r,
                     const float* b_f, const float* b_r, const float* c0, int L, int B, int d_in,
                     int d, int direction, const uint8_t* pad_mask, const sru_options* options,
                     float* H, float* C, float* c_last, uint16_t* H_bf16, void* workspace,
                     size_t workspace_bytes, hipStream_t stream) {
  Dims s;
  int st = make_dims(L, B, d_in, d, direction, s);
  if (st != SRU_OK) return st;
  Opts op;
  if (int e = read_options(options, op)) return e;
  if (!U || missing_v(op, v_f, v_r) || !b_f || !b_r || !H) return SRU_E_NULLPTR;
  if (s.k == 3 && !X) return SRU_E_NULLPTR;
  const void* ptrs[] = {U, X, v_f, v_r, b_f, b_r, c0, H, C, c_last};
  for (const void* p : ptrs)
    if (p && !aligned4(p)) return SRU_E_ALIGN;
  if ((reinterpret_cast<uintptr_t>(H_bf16) & 1) != 0) return SRU_E_ALIGN;
  const size_t need = op.linear ? scan_fwd_scratch(s) : 0;
  if (need > 0) {
    if (!workspace || workspace_bytes < need) return SRU_E_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return SRU_E_ALIGN;
  }
  sru::ScanFwdArgs a{U, X, v_f, v_r, b_f, b_r, c0, pad_mask, H, C, c_last, H_bf16, workspace};
  return hip_status(sru::scan_forward_launch(scan_shape(s, direction, op), a, stream));
}

size_t sru_scan_backward_workspace_bytes(int L, int B, int d_in, int d, int direction) {
  Dims s;
  if (make_dims(L, B, d_in, d, direction, s) != SRU_OK) return 0;
  return scan_bwd_partial(s);
}

int sru_scan_backward(const float* U, const float* X, const float* C, const float* dH,
                      const float* dc_last, const float* v_f, const float* v_r, const float* b_f,
                      const float* b_r, const float* c0, int L, int B, int d_in, int d,
                      int direction, const uint8_t* pad_mask, const sru_options* options,
                      float* dU, float* dxh, float* dv_f, float* dv_r, float* db_f,
                      float* db_r, float* dc0, void* workspace, size_t workspace_bytes,
                      hipStream_t stream) {
  Dims s;
  int st = make_dims(L, B, d_in, d, direction, s);
  if (st != SRU_OK) return st;
  Opts op;
  if (int e = read_options(options, op)) return e;
  if (!U || !C || !dH || missing_v(op, v_f, v_r) || !b_f || !b_r || !dU ||
      missing_v(op, dv_f, dv_r) || !db_f || !db_r)
    return SRU_E_NULLPTR;
  if (s.k == 3 && (!X || !dxh)) return SRU_E_NULLPTR;
  if (s.k == 4 && dxh) return SRU_E_SHAPE;
  const void* ptrs[] = {U, X, C, dH, dc_last, v_f, v_r, b_f, b_r, c0, dU, dxh, dv_f, dv_r,
                        db_f, db_r, dc0};
  for (const void* p : ptrs)
    if (p && !aligned4(p)) return SRU_E_ALIGN;
  const sru::ScanShape sh = scan_shape(s, direction, op);
  const size_t need = align_up(sru::scan_backward_partial_bytes(sh));
  if (!workspace || workspace_bytes < need) return SRU_E_WORKSPACE;
  sru::ScanBwdArgs a{U,   X,   C,     dH,  dc_last,
                     v_f, v_r, b_f,   b_r, c0,
                     pad_mask, dU, false, dxh, static_cast<float*>(workspace),
                     dc0, dv_f, dv_r,  db_f, db_r};
  return hip_status(sru::scan_backward_launch(sh, a, stream));
}

size_t sru_forward_lowrank_workspace_bytes(int L, int B, int d_in, int d, int dp,
                                           int direction, int gemm_dtype) {
  Dims s;
  if (make_dims(L, B, d_in, d, direction, s) != SRU_OK || !valid_dtype(gemm_dtype) || dp <= 0)
    return 0;
  return lr_fwd_layout(s, dp, gemm_dtype).total;
}

size_t sru_backward_lowrank_workspace_bytes(int L, int B, int d_in, int d, int dp,
                                            int direction, int gemm_dtype) {
  Dims s;
  if (make_dims(L, B, d_in, d, direction, s) != SRU_OK || !valid_dtype(gemm_dtype) || dp <= 0)
    return 0;
  return lr_bwd_layout(s, dp, gemm_dtype).total;
}

int sru_forward_lowrank(const float* X, const float* Q, const float* P, const float* v_f,
                        const float* v_r, const float* b_f, const float* b_r, const float* c0,
                        int L, int B, int d_in, int d, int dp, int direction,
                        const uint8_t* pad_mask, int gemm_dtype, const sru_options* options,
                        float* T, float* U, float* H, float* C, float* c_last,
                        const uint16_t* X_bf16, uint16_t* T_bf16, uint16_t* H_bf16,
                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
  Dims s;
  int st = make_dims(L, B, d_in, d, direction, s);
  if (st != SRU_OK) return st;
  if (!valid_dtype(gemm_dtype)) return SRU_E_FLAG;
  Opts op;
  if (int e = read_options(options, op)) return e;
  if (dp <= 0 || s.M * dp > kMaxElems || s.N * dp > kMaxElems) return SRU_E_SHAPE;
  if (!lowrank_dims_ok(s, dp, gemm_dtype)) return SRU_E_SHAPE;
  if (!X || !Q || !P || missing_v(op, v_f, v_r) || !b_f || !b_r || !T || !U || !H)
    return SRU_E_NULLPTR;
  const void* ptrs[] = {X, Q, P, v_f, v_r, b_f, b_r, c0, T, U, H, C, c_last};
  for (const void* p : ptrs)
    if (p && !aligned4(p)) return SRU_E_ALIGN;
  if (int e = check_bf16_side(gemm_dtype, {X_bf16, T_bf16, H_bf16})) return e;
  const bool bf16 = gemm_dtype == SRU_GEMM_BF16;
  const LrFwdLayout lay = lr_fwd_layout(s, dp, gemm_dtype);
  const size_t need = op.linear ? lay.total : lay.scr;
  if (need > 0) {
    if (!workspace || workspace_bytes < need) return SRU_E_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return SRU_E_ALIGN;
  }
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  auto bf = [&](size_t off) { return reinterpret_cast<uint16_t*>(ws + off); };
  auto round = [&](const float* src, int rows, int cols, uint16_t* dst, const char* label) {
    return hip_status(sru::to_bf16_launch(src, rows, cols, dst, false, stream, label));
  };

  if (!bf16) {
    // T = X Q, U = T P^T
    sru::GemmDesc gt = gemm_desc(SRU_OP_NN, false, (int)s.M, dp, d_in, X, d_in, Q, dp, T, dp);
    gt.label = "gemm_t";
    if (int e = hip_status(sru::gemm_launch(gt, stream))) return e;
    sru::GemmDesc gu = gemm_desc(SRU_OP_NT, false, (int)s.M, (int)s.N, dp, T, dp, P, dp, U, s.N);
    gu.label = "gemm_u";
    if (int e = hip_status(sru::gemm_launch(gu, stream))) return e;
  } else {
    // T = X Q as X (Q^T)^T: both operands K-contiguous; T in fp32 and bf16
    const uint16_t* xb = X_bf16;
    if (!xb) {
      if (int e = round(X, (int)s.M, d_in, bf(lay.xb), "bf16_x")) return e;
      xb = bf(lay.xb);
    }
    if (int e = hip_status(sru::to_bf16_t_launch(Q, false, d_in, dp, bf(lay.qt), stream,
                                                 "bf16_q")))
      return e;
    uint16_t* tb = T_bf16 ? T_bf16 : bf(lay.tb);
    sru::GemmDesc gt = gemm_desc(SRU_OP_NT, true, (int)s.M, dp, d_in, xb, d_in, bf(lay.qt), d_in,
                                 T, dp);
    gt.a_bf16 = gt.b_bf16 = true;
    gt.Cb = tb;
    gt.ldcb = dp;
    gt.label = "gemm_t";
    if (int e = hip_status(sru::gemm_launch(gt, stream))) return e;
    // U = T P^T
    if (int e = round(P, (int)s.N, dp, bf(lay.pb), "bf16_p")) return e;
    sru::GemmDesc gu = gemm_desc(SRU_OP_NT, true, (int)s.M, (int)s.N, dp, tb, dp, bf(lay.pb), dp,
                                 U, s.N);
    gu.a_bf16 = gu.b_bf16 = true;
    gu.label = "gemm_u";
    if (int e = hip_status(sru::gemm_launch(gu, stream))) return e;
  }

  sru::ScanFwdArgs a{U, X, v_f, v_r, b_f, b_r, c0, pad_mask, H, C, c_last, H_bf16, ws + lay.scr};
  return hip_status(sru::scan_forward_launch(scan_shape(s, direction, op), a, stream));
}

int sru_backward_lowrank(const float* X, const float* Q, const float* P, const float* v_f,
                         const float* v_r, const float* b_f, const float* b_r, const float* c0,
                         int L, int B, int d_in, int d, int dp, int direction,
                         const uint8_t* pad_mask, int gemm_dtype, const sru_options* options,
                         const float* T, const float* U, const float* C, const float* dH,
                         const float* dc_last, float* dX, float* dQ, float* dP, float* dv_f,
                         float* dv_r, float* db_f, float* db_r, float* dc0,
                         const uint16_t* X_bf16, const uint16_t* T_bf16, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  Dims s;
  int st = make_dims(L, B, d_in, d, direction, s);
  if (st != SRU_OK) return st;
  if (!valid_dtype(gemm_dtype)) return SRU_E_FLAG;
  Opts op;
  if (int e = read_options(options, op)) return e;
  if (dp <= 0 || s.M * dp > kMaxElems || s.N * dp > kMaxElems) return SRU_E_SHAPE;
  if (!lowrank_dims_ok(s, dp, gemm_dtype)) return SRU_E_SHAPE;
  if (!X || !Q || !P || missing_v(op, v_f, v_r) || !b_f || !b_r || !T || !U || !C || !dH ||
      !dX || !dQ || !dP || missing_v(op, dv_f, dv_r) || !db_f || !db_r)
    return SRU_E_NULLPTR;
  const void* ptrs[] = {X, Q, P, v_f, v_r, b_f, b_r, c0, T, U, C, dH, dc_last, dX, dQ, dP, dv_f,
                        dv_r, db_f, db_r, dc0};
  for (const void* p : ptrs)
    if (p && !aligned4(p)) return SRU_E_ALIGN;
  if (int e = check_bf16_side(gemm_dtype, {X_bf16, T_bf16})) return e;
  const LrBwdLayout lay = lr_bwd_layout(s, dp, gemm_dtype);
  if (!workspace || workspace_bytes < lay.total) return SRU_E_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return SRU_E_ALIGN;

  const bool bf16 = gemm_dtype == SRU_GEMM_BF16;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  auto bf = [&](size_t off) { return reinterpret_cast<uint16_t*>(ws + off); };
  void* dU = ws + lay.dU;
  float* dxh = s.k == 3 ? reinterpret_cast<float*>(ws + lay.dxh) : nullptr;
  float* partial = reinterpret_cast<float*>(ws + lay.partial);
  float* dT = reinterpret_cast<float*>(ws + lay.dT);
  float* splitk = reinterpret_cast<float*>(ws + lay.splitk);
  const void* tb = !bf16 ? static_cast<const void*>(T) : T_bf16 ? T_bf16 : bf(lay.tb);
  const void* xb = !bf16 ? static_cast<const void*>(X) : X_bf16 ? X_bf16 : bf(lay.xb);
  sru::GemmDesc gp = lr_dp_desc(s, dp, bf16, dU, tb, dP);
  sru::GemmDesc gq = lr_dq_desc(s, dp, bf16, xb, bf16 ? (const void*)bf(lay.dtb) : dT, dQ);
  gp.partials = gq.partials = splitk;
  // the split partials were sized for these plans: refuse before enqueueing
  if (sru::gemm_splits(gp) > lay.splits_p || sru::gemm_splits(gq) > lay.splits_q)
    return SRU_E_WORKSPACE;
  auto round = [&](const float* src, int rows, int cols, uint16_t* dst, const char* label) {
    return hip_status(sru::to_bf16_launch(src, rows, cols, dst, false, stream, label));
  };

  // 1. reverse gradient scan (dU in the products' operand type); the v/b
  //    sums over the batch run with the dP product (in its split-K sum's
  //    launch when it has one)
  sru::ScanBwdArgs a{U,   X,    C,   dH,      dc_last, v_f,  v_r,  b_f,  b_r,  c0,
                     pad_mask, dU, bf16, dxh, partial, dc0, dv_f, dv_r, db_f, db_r};
  a.defer_vb = true;
  gp.vb = sru::scan_backward_vb(scan_shape(s, direction, op), a);
  if (int e = hip_status(sru::scan_backward_launch(scan_shape(s, direction, op), a, stream)))
    return e;
  // 2. dT = dU P (bf16: as dU (P^T)^T, written in bf16 only)
  sru::GemmDesc gd;
  if (bf16) {
    if (int e = hip_status(sru::to_bf16_t_launch(P, false, (int)s.N, dp, bf(lay.pt), stream,
                                                 "bf16_p")))
      return e;
    gd = gemm_desc(SRU_OP_NT, true, (int)s.M, dp, (int)s.N, dU, s.N, bf(lay.pt), s.N, nullptr,
                   dp);
    gd.a_bf16 = gd.b_bf16 = true;
    gd.Cb = bf(lay.dtb);
    gd.ldcb = dp;
  } else {
    gd = gemm_desc(SRU_OP_NN, false, (int)s.M, dp, (int)s.N, dU, s.N, P, dp, dT, dp);
  }
  gd.label = "gemm_dt";
  if (int e = hip_status(sru::gemm_launch(gd, stream))) return e;
  // 3. dX = dT Q^T (+ the highway gradient of every direction when k = 3)
  if (bf16) {
    if (int e = round(Q, d_in, dp, bf(lay.qb), "bf16_q")) return e;
  }
  sru::GemmDesc gx = gemm_desc(SRU_OP_NT, bf16, (int)s.M, d_in, dp,
                               bf16 ? (const void*)bf(lay.dtb) : dT, dp,
                               bf16 ? (const void*)bf(lay.qb) : Q, dp, dX, d_in);
  gx.a_bf16 = gx.b_bf16 = bf16;
  gx.label = "gemm_dx";
  if (s.k == 3) {
    gx.add = dxh;
    gx.add_ld = s.nfeat;
    gx.add_off = d;
    gx.add_count = s.ndir;
  }
  if (int e = hip_status(sru::gemm_launch(gx, stream))) return e;
  // 4. dP = dU^T T, 5. dQ = X^T dT (reductions over all tokens)
  if (bf16 && !T_bf16) {
    if (int e = round(T, (int)s.M, dp, bf(lay.tb), "bf16_t")) return e;
  }
  if (int e = hip_status(sru::gemm_launch(gp, stream))) return e;
  if (bf16 && !X_bf16) {
    if (int e = round(X, (int)s.M, d_in, bf(lay.xb), "bf16_x")) return e;
  }
  return hip_status(sru::gemm_launch(gq, stream));
}

}  // extern "C"
