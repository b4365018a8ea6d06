// Element-wise scans of the SRU layer on gfx950.
//
// Forward: the fused kernel of Sec. 3.1 / Algorithm 1.  One lane per
// (batch b, direction, hidden unit j), sequential over t, the state c held in
// a register.  Eq. 1-4 with the reset gate on c_{t-1} (Eq. 3), or on c_t
// (Algorithm 1's order, RN), and the highway term scaled by alpha (Sec. 3.2).
// Backward: the chain rule of Eq. 1-4 in reverse step order; one lane per
// (b, direction, j) again, the carried gradient dloss/dc in a register.
//
// Memory: per step a lane reads its U blocks (and x_t when k = 3) and writes
// h and c; a wavefront covers 64 consecutive j, so every access is a
// contiguous 256-byte segment per array.  The loads of step t do not depend on
// the recurrence, so they are issued PF steps ahead into a register ring (the
// wavefront keeps PF steps of loads in flight).  The main loop covers whole
// rings only, so it contains no data-dependent branch; the last L % PF steps
// run in a guarded tail.
#include <type_traits>

#include "sru_internal.h"

namespace sru {
namespace {

constexpr int kScanThreads = 64;

__device__ __forceinline__ float sigmoid_fast(float z) {
  // 1 / (1 + e^{-z}); saturates to exactly 0 (e^{-z} = inf) and 1 (e^{-z}
  // underflows) instead of producing NaN.
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

struct Lane {
  int gid, b, fidx, dir, j;
  bool rev;
};

__device__ __forceinline__ bool decode_lane(const ScanShape& s, Lane& ln) {
  const int nfeat = s.ndir * s.d;
  ln.gid = blockIdx.x * kScanThreads + threadIdx.x;
  if (ln.gid >= s.B * nfeat) return false;
  ln.b = ln.gid / nfeat;
  ln.fidx = ln.gid - ln.b * nfeat;
  ln.dir = ln.fidx / s.d;
  ln.j = ln.fidx - ln.dir * s.d;
  ln.rev = s.direction == 1 || (s.direction == 2 && ln.dir == 1);
  return true;
}

// ------------------------------------------------------------ forward scan
template <int KB, bool MASK, bool STORE_C, bool STORE_HB, bool RN, int PF>
__global__ __launch_bounds__(kScanThreads) void scan_fwd_kernel(ScanShape s, ScanFwdArgs a) {
  Lane ln;
  if (!decode_lane(s, ln)) return;
  const int L = s.L;
  const long long nfeat = (long long)s.ndir * s.d;
  const long long u_step = (long long)s.B * s.ndir * KB * s.d;
  const long long x_step = (long long)s.B * s.d_in;
  const long long h_step = (long long)s.B * nfeat;
  const float* up = a.U + ((long long)ln.b * s.ndir + ln.dir) * KB * s.d + ln.j;
  const float* xp = KB == 3 ? a.X + (long long)ln.b * s.d_in + ln.j : nullptr;
  const uint8_t* mp = MASK ? a.mask + ln.b : nullptr;
  float* hp = a.H + ln.gid;
  float* cp = STORE_C ? a.C + ln.gid : nullptr;
  uint16_t* hbp = STORE_HB ? a.Hb + ln.gid : nullptr;
  const int d = s.d;

  const float vf = a.v_f[ln.fidx], vr = a.v_r[ln.fidx];
  const float bf = a.b_f[ln.fidx], br = a.b_r[ln.fidx];
  const float alpha = s.alpha;
  float c = a.c0 ? a.c0[ln.gid] : 0.0f;

  float r0[PF], r1[PF], r2[PF], rx[PF];
  uint8_t rm[PF];
  (void)rm;

  auto tindex = [&](int st) { return ln.rev ? L - 1 - st : st; };
  auto load = [&](int st, float& u0, float& u1, float& u2, float& xh, uint8_t& m) {
    const long long t = tindex(st);
    const float* u = up + t * u_step;
    u0 = __builtin_nontemporal_load(u);
    u1 = __builtin_nontemporal_load(u + d);
    u2 = __builtin_nontemporal_load(u + 2 * d);
    if constexpr (KB == 4) xh = __builtin_nontemporal_load(u + 3 * d);
    else xh = xp[t * x_step];
    if constexpr (MASK) m = mp[t * s.B];
  };
  auto step = [&](int st, float u0, float u1, float u2, float xh, uint8_t m) {
    const long long t = tindex(st);
    const float f = sigmoid_fast(fmaf(vf, c, u1 + bf));   // Eq. 1
    const float cn = fmaf(f, c, (1.0f - f) * u0);         // Eq. 2
    const float r = sigmoid_fast(fmaf(vr, RN ? cn : c, u2 + br));  // Eq. 3
    float h = fmaf(r, cn, (1.0f - r) * (alpha * xh));     // Eq. 4 (Sec. 3.2)
    if constexpr (MASK) {
      const bool pad = m != 0;
      c = pad ? c : cn;
      h = pad ? 0.0f : h;
    } else {
      c = cn;
    }
    __builtin_nontemporal_store(h, hp + t * h_step);
    if constexpr (STORE_C) __builtin_nontemporal_store(c, cp + t * h_step);
    if constexpr (STORE_HB)
      __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (__bf16)h), hbp + t * h_step);
  };

#pragma unroll
  for (int p = 0; p < PF; ++p) load(p < L ? p : L - 1, r0[p], r1[p], r2[p], rx[p], rm[p]);

  int s0 = 0;
  for (; s0 + PF <= L; s0 += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      step(s0 + p, r0[p], r1[p], r2[p], rx[p], rm[p]);
      const int sn = s0 + p + PF < L ? s0 + p + PF : L - 1;
      load(sn, r0[p], r1[p], r2[p], rx[p], rm[p]);
      // keep each prefetch where it is: sunk loads shorten the distance
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (s0 + p < L) step(s0 + p, r0[p], r1[p], r2[p], rx[p], rm[p]);

  if (a.c_last) a.c_last[ln.gid] = c;
}

// ------------------------------------------------------------ backward scan
// Iteration i handles forward-order position pos = L-1-i.  With
// t = t(pos), c_p = C[t(pos-1)] (c0 at pos 0), c_t = C[t]:
//   f = sigma(u1 + v_f c_p + b_f), r = sigma(u2 + v_r c_p + b_r)
//   gc = g + dh r
//   dr = dh (c_t - x_hat) r (1 - r)        -> dU block 2
//   df = gc (c_p - u0) f (1 - f)           -> dU block 1
//   du0 = gc (1 - f)                       -> dU block 0
//   dx_hat = dh (1 - r)                    -> dxh (k = 3) / dU block 3 (k = 4)
//   v/b sums += (df c_p, dr c_p, df, dr);  g <- gc f + df v_f + dr v_r
// A padded step writes zeros and leaves g unchanged.
// DUB: store dU as bf16 (RNE), the operand type of bf16 matrix products.
template <int KB, bool MASK, bool DUB, bool RN, int PF>
__global__ __launch_bounds__(kScanThreads) void scan_bwd_kernel(ScanShape s, ScanBwdArgs a) {
  Lane ln;
  if (!decode_lane(s, ln)) return;
  const int L = s.L;
  const int d = s.d;
  const long long nfeat = (long long)s.ndir * s.d;
  const long long u_step = (long long)s.B * s.ndir * KB * s.d;
  const long long x_step = (long long)s.B * s.d_in;
  const long long h_step = (long long)s.B * nfeat;
  const long long u_off = ((long long)ln.b * s.ndir + ln.dir) * KB * s.d + ln.j;
  const float* up = a.U + u_off;
  using DuT = typename std::conditional<DUB, uint16_t, float>::type;
  DuT* dup = static_cast<DuT*>(a.dU) + u_off;
  const float* xp = KB == 3 ? a.X + (long long)ln.b * s.d_in + ln.j : nullptr;
  const uint8_t* mp = MASK ? a.mask + ln.b : nullptr;
  const float* cpp = a.C + ln.gid;
  const float* dhp = a.dH + ln.gid;
  float* dxp = KB == 3 ? a.dxh + ln.gid : nullptr;

  const float vf = a.v_f[ln.fidx], vr = a.v_r[ln.fidx];
  const float bf = a.b_f[ln.fidx], br = a.b_r[ln.fidx];
  const float alpha = s.alpha;
  const float c0v = a.c0 ? a.c0[ln.gid] : 0.0f;
  float g = a.dc_last ? a.dc_last[ln.gid] : 0.0f;
  float sum_df_c = 0.f, sum_dr_c = 0.f, sum_df = 0.f, sum_dr = 0.f;

  auto tpos = [&](int pos) { return ln.rev ? L - 1 - pos : pos; };
  float c_t = cpp[(long long)tpos(L - 1) * h_step];

  float r0[PF], r1[PF], r2[PF], rx[PF], rdh[PF], rcp[PF];
  uint8_t rm[PF];
  (void)rm;

  auto load = [&](int i, float& u0, float& u1, float& u2, float& xh, float& dh, float& cprev,
                  uint8_t& m) {
    const int pos = L - 1 - i;
    const long long t = tpos(pos);
    const float* u = up + t * u_step;
    u0 = __builtin_nontemporal_load(u);
    u1 = __builtin_nontemporal_load(u + d);
    u2 = __builtin_nontemporal_load(u + 2 * d);
    if constexpr (KB == 4) xh = __builtin_nontemporal_load(u + 3 * d);
    else xh = xp[t * x_step];
    dh = __builtin_nontemporal_load(dhp + t * h_step);
    const long long tp = tpos(pos > 0 ? pos - 1 : 0);
    cprev = cpp[tp * h_step];
    if constexpr (MASK) m = mp[t * s.B];
  };
  auto step = [&](int i, float u0, float u1, float u2, float xh, float dh, float cprev,
                  uint8_t m) {
    const int pos = L - 1 - i;
    const long long t = tpos(pos);
    const float c_p = pos > 0 ? cprev : c0v;
    const float c_r = RN ? c_t : c_p;  // the state the reset gate reads
    const float f = sigmoid_fast(fmaf(vf, c_p, u1 + bf));
    const float r = sigmoid_fast(fmaf(vr, c_r, u2 + br));
    bool pad = false;
    if constexpr (MASK) pad = m != 0;
    const float dhv = pad ? 0.0f : dh;
    const float rr = r * (1.0f - r);
    const float ff = f * (1.0f - f);
    float dr = dhv * (c_t - alpha * xh) * rr;
    // total gradient into c_t: from later steps, through h, and (RN)
    // through the reset gate
    const float gc = RN ? fmaf(dr, vr, fmaf(dhv, r, g)) : fmaf(dhv, r, g);
    float df = gc * (c_p - u0) * ff;
    float du0 = gc * (1.0f - f);
    float dx = dhv * (1.0f - r) * alpha;
    if constexpr (MASK) {
      dr = pad ? 0.0f : dr;
      df = pad ? 0.0f : df;
      du0 = pad ? 0.0f : du0;
      dx = pad ? 0.0f : dx;
    }
    sum_df_c = fmaf(df, c_p, sum_df_c);
    sum_dr_c = fmaf(dr, c_r, sum_dr_c);
    sum_df += df;
    sum_dr += dr;
    const float gn = RN ? fmaf(df, vf, gc * f) : fmaf(dr, vr, fmaf(df, vf, gc * f));
    g = pad ? g : gn;
    DuT* du = dup + t * u_step;
    auto put = [](float v, DuT* p) {
      if constexpr (DUB) __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (__bf16)v), p);
      else __builtin_nontemporal_store(v, p);
    };
    put(du0, du);
    put(df, du + d);
    put(dr, du + 2 * d);
    if constexpr (KB == 4) put(dx, du + 3 * d);
    else __builtin_nontemporal_store(dx, dxp + t * h_step);
    // c_t takes the value in a register of its own.  Were it to share
    // cprev's register, the ring's registers would shift by one slot per
    // step and the loop would copy still-loading values at its back edge.
    asm volatile("v_mov_b32 %0, %1" : "=v"(c_t) : "v"(cprev));
  };

#pragma unroll
  for (int p = 0; p < PF; ++p)
    load(p < L ? p : L - 1, r0[p], r1[p], r2[p], rx[p], rdh[p], rcp[p], rm[p]);
  int i0 = 0;
  for (; i0 + PF <= L; i0 += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      step(i0 + p, r0[p], r1[p], r2[p], rx[p], rdh[p], rcp[p], rm[p]);
      const int in = i0 + p + PF < L ? i0 + p + PF : L - 1;
      load(in, r0[p], r1[p], r2[p], rx[p], rdh[p], rcp[p], rm[p]);
      __builtin_amdgcn_sched_barrier(0);  // as in the forward scan
    }
  }
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (i0 + p < L) step(i0 + p, r0[p], r1[p], r2[p], rx[p], rdh[p], rcp[p], rm[p]);

  float* part = a.partial + (long long)ln.b * 4 * nfeat + ln.fidx;
  part[0] = sum_df_c;
  part[nfeat] = sum_dr_c;
  part[2 * nfeat] = sum_df;
  part[3 * nfeat] = sum_dr;
  if (a.dc0) a.dc0[ln.gid] = g;
}

// Sum of the per-sequence partials over b, in a fixed order (deterministic).
// A workgroup covers 64 consecutive outputs; its 8 waves take b = w, w+8,
// ... in sequence, and the 8 wave sums of an output are added as a fixed
// tree through LDS.  The loads of a lane are independent, so a launch costs
// about one memory round trip.
constexpr int kVbWaves = 8;
__global__ __launch_bounds__(64 * kVbWaves) void reduce_vb_kernel(const float* __restrict__ partial,
                                                                  int B, int nfeat, float* dv_f,
                                                                  float* dv_r, float* db_f,
                                                                  float* db_r) {
  __shared__ float red[kVbWaves][64];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int o = blockIdx.x * 64 + lane;  // output: q * nfeat + f
  const bool live = o < 4 * nfeat;
  const long long stride = 4LL * nfeat;
  float s = 0.f;
  if (live) {
    const float* p = partial + o;
#pragma unroll 8
    for (int b = w; b < B; b += kVbWaves) s += p[b * stride];
  }
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && live) {
    const float t = ((red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane])) +
                    ((red[4][lane] + red[5][lane]) + (red[6][lane] + red[7][lane]));
    const int q = o / nfeat;
    const int f = o - q * nfeat;
    float* out = q == 0 ? dv_f : q == 1 ? dv_r : q == 2 ? db_f : db_r;
    out[f] = t;
  }
}

constexpr int kFwdPF = 8;
constexpr int kBwdPF = 6;

template <int KB, bool MASK, bool STORE_C, bool STORE_HB>
hipError_t fwd_dispatch(const ScanShape& s, const ScanFwdArgs& a, hipStream_t st) {
  const int lanes = s.B * s.ndir * s.d;
  const int grid = (lanes + kScanThreads - 1) / kScanThreads;
  timing_before("scan_fwd", st);
  if (s.reset_new)
    hipLaunchKernelGGL((scan_fwd_kernel<KB, MASK, STORE_C, STORE_HB, true, kFwdPF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  else
    hipLaunchKernelGGL((scan_fwd_kernel<KB, MASK, STORE_C, STORE_HB, false, kFwdPF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  timing_after(st);
  return hipGetLastError();
}

template <int KB, bool MASK>
hipError_t fwd_dispatch_c(const ScanShape& s, const ScanFwdArgs& a, hipStream_t st) {
  if (a.Hb)
    return a.C ? fwd_dispatch<KB, MASK, true, true>(s, a, st)
               : fwd_dispatch<KB, MASK, false, true>(s, a, st);
  return a.C ? fwd_dispatch<KB, MASK, true, false>(s, a, st)
             : fwd_dispatch<KB, MASK, false, false>(s, a, st);
}

template <int KB, bool MASK>
hipError_t bwd_dispatch(const ScanShape& s, const ScanBwdArgs& a, hipStream_t st) {
  const int lanes = s.B * s.ndir * s.d;
  const int grid = (lanes + kScanThreads - 1) / kScanThreads;
  timing_before("scan_bwd", st);
  if (a.du_bf16 && s.reset_new)
    hipLaunchKernelGGL((scan_bwd_kernel<KB, MASK, true, true, kBwdPF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  else if (a.du_bf16)
    hipLaunchKernelGGL((scan_bwd_kernel<KB, MASK, true, false, kBwdPF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  else if (s.reset_new)
    hipLaunchKernelGGL((scan_bwd_kernel<KB, MASK, false, true, kBwdPF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  else
    hipLaunchKernelGGL((scan_bwd_kernel<KB, MASK, false, false, kBwdPF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  timing_after(st);
  return hipGetLastError();
}

}  // namespace

hipError_t scan_forward_launch(const ScanShape& s, const ScanFwdArgs& a, hipStream_t st) {
  const bool m = a.mask != nullptr;
  if (s.k == 3) return m ? fwd_dispatch_c<3, true>(s, a, st) : fwd_dispatch_c<3, false>(s, a, st);
  return m ? fwd_dispatch_c<4, true>(s, a, st) : fwd_dispatch_c<4, false>(s, a, st);
}

size_t scan_backward_partial_bytes(const ScanShape& s) {
  return sizeof(float) * 4ull * (size_t)s.B * (size_t)s.ndir * (size_t)s.d;
}

hipError_t scan_backward_launch(const ScanShape& s, const ScanBwdArgs& a, hipStream_t st) {
  const bool m = a.mask != nullptr;
  hipError_t e;
  if (s.k == 3) e = m ? bwd_dispatch<3, true>(s, a, st) : bwd_dispatch<3, false>(s, a, st);
  else e = m ? bwd_dispatch<4, true>(s, a, st) : bwd_dispatch<4, false>(s, a, st);
  if (e != hipSuccess) return e;
  const int nfeat = s.ndir * s.d;
  const int grid = (4 * nfeat + 63) / 64;
  timing_before("reduce_vb", st);
  hipLaunchKernelGGL(reduce_vb_kernel, dim3(grid), dim3(64 * kVbWaves), 0, st, a.partial, s.B,
                     nfeat, a.dv_f, a.dv_r, a.db_f, a.db_r);
  timing_after(st);
  return hipGetLastError();
}

}  // namespace sru
