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

#include "sru_device.h"
#include "sru_internal.h"

namespace sru {
namespace {

constexpr int kScanThreads = 64;
typedef __attribute__((address_space(3))) void lds_t;

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
  const int d = s.d;
  // Addresses are cursors that move one step at a time in the direction's
  // order (no per-step 64-bit products): the load cursors run PF steps
  // ahead of the store cursors and stop at the last step, so the loads past
  // the end of the sequence re-read it.
  const long long t0 = ln.rev ? L - 1 : 0;
  const long long sg = ln.rev ? -1 : 1;
  const long long su = sg * u_step, sx = sg * x_step, sh = sg * h_step, sm = sg * s.B;
  const float* lu = a.U + ((long long)ln.b * s.ndir + ln.dir) * KB * s.d + ln.j + t0 * u_step;
  const float* lx = KB == 3 ? a.X + (long long)ln.b * s.d_in + ln.j + t0 * x_step : nullptr;
  const uint8_t* lm = MASK ? a.mask + ln.b + t0 * s.B : nullptr;
  float* hp = a.H + ln.gid + t0 * h_step;
  float* cp = STORE_C ? a.C + ln.gid + t0 * h_step : nullptr;
  uint16_t* hbp = STORE_HB ? a.Hb + ln.gid + t0 * h_step : nullptr;
  int ls = 0;  // the step the load cursors point at

  // gate parameters scaled by -log2(e) (sigmoid_scaled)
  const float vfs = a.v_f[ln.fidx] * kNegLog2e, vrs = a.v_r[ln.fidx] * kNegLog2e;
  const float bfs = a.b_f[ln.fidx] * kNegLog2e, brs = a.b_r[ln.fidx] * kNegLog2e;
  const float alpha = s.alpha;
  float c = a.c0 ? a.c0[ln.gid] : 0.0f;

  float r0[PF], r1[PF], r2[PF], rx[PF];
  // mask bytes held one per register: a byte array would be packed four to
  // a register, and packing waits for the loads that fill it
  unsigned rm[PF];
  (void)rm;

  auto load = [&](float& u0, float& u1, float& u2, float& xh, unsigned& m) {
    u0 = __builtin_nontemporal_load(lu);
    u1 = __builtin_nontemporal_load(lu + d);
    u2 = __builtin_nontemporal_load(lu + 2 * d);
    if constexpr (KB == 4) xh = __builtin_nontemporal_load(lu + 3 * d);
    else xh = *lx;
    if constexpr (MASK) m = *lm;
    const bool adv = ls + 1 < L;  // the same for the whole wave
    ls += adv;
    lu = adv ? lu + su : lu;
    if constexpr (KB == 3) lx = adv ? lx + sx : lx;
    if constexpr (MASK) lm = adv ? lm + sm : lm;
  };
  // The chain from c to the next c: fma, exp2, add, rcp, fma, fma.  Eq. 2 is
  // f c + (u0 - f u0), which keeps f = 0 and f = 1 exact (c' = u0, c' = c).
  auto step = [&](float u0, float u1, float u2, float xh, unsigned m) {
    const float f = sigmoid_scaled(fmaf(vfs, c, fmaf(u1, kNegLog2e, bfs)));  // Eq. 1
    const float cn = fmaf(f, c, fmaf(-f, u0, u0));                           // Eq. 2
    const float r = sigmoid_scaled(fmaf(vrs, RN ? cn : c, fmaf(u2, kNegLog2e, brs)));  // Eq. 3
    float h = fmaf(r, cn, (1.0f - r) * (alpha * xh));     // Eq. 4 (Sec. 3.2)
    if constexpr (MASK) {
      const bool pad = m != 0;
      c = pad ? c : cn;
      h = pad ? 0.0f : h;
    } else {
      c = cn;
    }
    // Plain (write-back) stores: a wave's wait for a load also covers its
    // older stores, which complete sooner when the cache takes them than
    // when they stream to memory.  L 256, B 8, d 1024 (few lanes, each step
    // waiting on its loads): 36.1 -> 32.9 us; L 128, B 128, d 2048:
    // 180 -> 166 us.
    *hp = h;
    if constexpr (STORE_C) *cp = c;
    if constexpr (STORE_HB) *hbp = __builtin_bit_cast(uint16_t, (__bf16)h);
    hp += sh;
    if constexpr (STORE_C) cp += sh;
    if constexpr (STORE_HB) hbp += sh;
  };

#pragma unroll
  for (int p = 0; p < PF; ++p) load(r0[p], r1[p], r2[p], rx[p], rm[p]);

  auto ring = [&]() {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      step(r0[p], r1[p], r2[p], rx[p], rm[p]);
      load(r0[p], r1[p], r2[p], rx[p], rm[p]);  // PF steps ahead (or the last step)
      // keep each prefetch where it is: sunk loads shorten the distance
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // The first ring is peeled off the loop, so the loop is entered with the
  // memory operations of a whole ring in flight, as on its back edge: the
  // compiler derives each step's wait for its loads from both paths, and
  // from the prologue's loads alone the ring's first step would wait for
  // loads issued 3 steps back instead of PF (L 256, B 8, d 1024:
  // 33.0 -> 31.9 us).
  int s0 = 0;
  if (PF <= L) {
    ring();
    for (s0 = PF; s0 + PF <= L; s0 += PF) ring();
  }
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (s0 + p < L) step(r0[p], r1[p], r2[p], rx[p], rm[p]);

  if (a.c_last) a.c_last[ln.gid] = c;
}

// ------------------------------------------------ forward scan, LDS ring
// The same recurrence and arithmetic as scan_fwd_kernel (results equal bit
// for bit), organised for more memory parallelism.  A workgroup owns 256
// consecutive hidden units of one (sequence b, direction): four consumer
// waves (one unit per lane) run the recurrence, and one producer wave
// streams their inputs into a ring in LDS with buffer loads that write LDS
// directly, 1 KiB (64 lanes x 16 bytes) per instruction: per step one load
// per input segment (U blocks 0-2 and x for k = 3, U blocks 0-3 for
// k = 4) and, with padding, one byte load of the step's mask entry per
// lane.  The ring holds kRingSlots groups of kRingSteps steps; the producer
// keeps kRingSlots - 1 groups in flight (12 steps, 48 KiB per workgroup),
// about twice what the register ring of scan_fwd_kernel holds per unit.
// Hand-off per group: the producer waits for the group's loads, every wave
// meets at a barrier, the consumers read the group from LDS and the
// producer refills the slot the consumers finished before the barrier.
// Steps past the end of the sequence load with an out-of-range offset
// (zeros) and are not computed.  Operands must be smaller than 2 GiB (the
// buffer offsets are 32-bit; the top bit marks out-of-range).
constexpr int kRingUnits = 256;  // hidden units per workgroup (4 consumer waves)
constexpr int kRingSteps = 4;    // steps per hand-off
constexpr int kRingSlots = 4;    // groups in the ring
constexpr int kRingConsumers = kRingUnits / 64;
constexpr int kRingThreads = kRingUnits + 64;
constexpr int kRingSegBytes = kRingUnits * 4;  // one input segment of one step
constexpr unsigned kRingOOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t ring_rsrc(const void* p, unsigned bytes) {
  // dword 3 = 0x00020000: 32-bit data format, the raw-buffer setting of gfx9 parts
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                           0x00020000);
}

// Workgroup barrier of the ring: this wave's LDS accesses are complete
// (lgkmcnt 0), not its global stores (the release fence of __syncthreads
// would wait for those too).
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0) (vmcnt 63, expcnt 7)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt immediate for vmcnt <= n (expcnt 7, lgkmcnt 15)
constexpr int ring_vm_wait(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }

template <int KB, bool MASK, bool STORE_C, bool STORE_HB, bool RN>
__global__ __launch_bounds__(kRingThreads) void scan_fwd_ring_kernel(ScanShape s, ScanFwdArgs a,
                                                                     unsigned u_bytes,
                                                                     unsigned x_bytes,
                                                                     unsigned m_bytes) {
  constexpr int NSEG = 4;  // U blocks 0-2 and x (k = 3), or U blocks 0-3 (k = 4)
  constexpr int STEPB = NSEG * kRingSegBytes;
  constexpr int SLOTB = kRingSteps * STEPB;
  constexpr int IPG = kRingSteps * (NSEG + (MASK ? 1 : 0));  // loads per group
  static_assert((kRingSlots - 1) * IPG < 64, "vmcnt counts at most 63 loads");
  __shared__ __attribute__((aligned(1024))) unsigned char ring[kRingSlots * SLOTB];
  __shared__ __attribute__((aligned(256))) unsigned mring[kRingSlots][kRingSteps * 64];

  const int nblk = s.d / kRingUnits;
  const int jb = blockIdx.x % nblk;
  const int bd = blockIdx.x / nblk;
  const int dir = bd % s.ndir;
  const int b = bd / s.ndir;
  const bool rev = s.direction == 1 || (s.direction == 2 && dir == 1);
  const int L = s.L;
  const int G = (L + kRingSteps - 1) / kRingSteps;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;

  if (wave == kRingConsumers) {
    // ---- producer
    const __amdgpu_buffer_rsrc_t ru = ring_rsrc(a.U, u_bytes);
    const __amdgpu_buffer_rsrc_t rx = ring_rsrc(KB == 3 ? a.X : a.U, KB == 3 ? x_bytes : u_bytes);
    const __amdgpu_buffer_rsrc_t rm =
        ring_rsrc(MASK ? static_cast<const void*>(a.mask) : static_cast<const void*>(a.U),
                  MASK ? m_bytes : u_bytes);
    const unsigned u_step = (unsigned)s.B * s.ndir * KB * s.d * 4u;
    const unsigned x_step = (unsigned)s.B * s.d_in * 4u;
    const unsigned u_base =
        (unsigned)((((long long)b * s.ndir + dir) * KB * s.d + jb * kRingUnits) * 4) + lane * 16u;
    const unsigned x_base = (unsigned)(((long long)b * s.d_in + jb * kRingUnits) * 4) + lane * 16u;
    const unsigned seg = (unsigned)s.d * 4u;
    auto issue = [&](int gi) {
      unsigned char* slot = ring + (gi % kRingSlots) * SLOTB;
#pragma unroll
      for (int k = 0; k < kRingSteps; ++k) {
        const int step = gi * kRingSteps + k;
        const int t = rev ? L - 1 - step : step;
        const unsigned oob = step < L ? 0u : kRingOOB;
        const unsigned uo = ((unsigned)t * u_step + u_base) | oob;
#pragma unroll
        for (int q = 0; q < KB; ++q)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              ru, (lds_t*)(slot + k * STEPB + q * kRingSegBytes), 16, uo + q * seg, 0, 0, 0);
        if constexpr (KB == 3)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rx, (lds_t*)(slot + k * STEPB + 3 * kRingSegBytes), 16,
              ((unsigned)t * x_step + x_base) | oob, 0, 0, 0);
        if constexpr (MASK) {
          // lane 0 loads the step's mask byte into its dword slot; the
          // other lanes read out of range (zeros)
          const unsigned mo = lane == 0 ? (((unsigned)t * s.B + b) | oob) : kRingOOB;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rm, (lds_t*)(&mring[gi % kRingSlots][k * 64]), 1, mo, 0, 0, 0);
        }
      }
    };
    for (int gi = 0; gi < kRingSlots - 1 && gi < G; ++gi) issue(gi);
    for (int g = 0; g < G; ++g) {
      // group g has landed once at most the groups issued after it remain
      const int later = min(kRingSlots - 2, G - 1 - g);
      if (later >= 2) __builtin_amdgcn_s_waitcnt(ring_vm_wait(2 * IPG));
      else if (later == 1) __builtin_amdgcn_s_waitcnt(ring_vm_wait(IPG));
      else __builtin_amdgcn_s_waitcnt(ring_vm_wait(0));
      ring_barrier();
      // the slot of group g - 1, which every consumer finished before the barrier
      if (g + kRingSlots - 1 < G) issue(g + kRingSlots - 1);
    }
    return;
  }

  // ---- consumers: unit j of (b, dir), lane gid of the [B, ndir*d] state
  const int j = jb * kRingUnits + wave * 64 + lane;
  const int fidx = dir * s.d + j;
  const long long nfeat = (long long)s.ndir * s.d;
  const long long gid = (long long)b * nfeat + fidx;
  const long long h_step = (long long)s.B * nfeat;
  const long long t0 = rev ? L - 1 : 0;
  const long long sh = rev ? -h_step : h_step;
  float* hp = a.H + gid + t0 * h_step;
  float* cp = STORE_C ? a.C + gid + t0 * h_step : nullptr;
  uint16_t* hbp = STORE_HB ? a.Hb + gid + t0 * h_step : nullptr;
  const float vfs = a.v_f[fidx] * kNegLog2e, vrs = a.v_r[fidx] * kNegLog2e;
  const float bfs = a.b_f[fidx] * kNegLog2e, brs = a.b_r[fidx] * kNegLog2e;
  const float alpha = s.alpha;
  float c = a.c0 ? a.c0[gid] : 0.0f;
  const int ubyte = (wave * 64 + lane) * 4;

  auto step = [&](const float (&v)[NSEG], unsigned mk) {
    const float u0 = v[0], u1 = v[1], u2 = v[2], xh = v[3];
    const float f = sigmoid_scaled(fmaf(vfs, c, fmaf(u1, kNegLog2e, bfs)));  // Eq. 1
    const float cn = fmaf(f, c, fmaf(-f, u0, u0));                           // Eq. 2
    const float r = sigmoid_scaled(fmaf(vrs, RN ? cn : c, fmaf(u2, kNegLog2e, brs)));  // Eq. 3
    float h = fmaf(r, cn, (1.0f - r) * (alpha * xh));  // Eq. 4 (Sec. 3.2)
    if constexpr (MASK) {
      const bool pad = mk != 0;
      c = pad ? c : cn;
      h = pad ? 0.0f : h;
    } else {
      c = cn;
    }
    __builtin_nontemporal_store(h, hp);
    if constexpr (STORE_C) __builtin_nontemporal_store(c, cp);
    if constexpr (STORE_HB)
      __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (__bf16)h), hbp);
    hp += sh;
    if constexpr (STORE_C) cp += sh;
    if constexpr (STORE_HB) hbp += sh;
  };

  // Whole groups run without a bound check, so a group's LDS reads all go
  // out before its first step; the last, partial group checks each step.
  const int Gfull = L / kRingSteps;
  for (int g = 0; g < G; ++g) {
    ring_barrier();
    const unsigned char* slot = ring + (g % kRingSlots) * SLOTB;
    float in[kRingSteps][NSEG];
    unsigned m[kRingSteps];
#pragma unroll
    for (int k = 0; k < kRingSteps; ++k) {
#pragma unroll
      for (int q = 0; q < NSEG; ++q)
        in[k][q] = *reinterpret_cast<const float*>(slot + k * STEPB + q * kRingSegBytes + ubyte);
      m[k] = MASK ? (mring[g % kRingSlots][k * 64] & 0xFFu) : 0u;
    }
    if (g < Gfull) {
#pragma unroll
      for (int k = 0; k < kRingSteps; ++k) step(in[k], m[k]);
    } else {
#pragma unroll
      for (int k = 0; k < kRingSteps; ++k)
        if (g * kRingSteps + k < L) step(in[k], m[k]);
    }
  }
  if (a.c_last) a.c_last[gid] = c;
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
// ----------------------------------------- forward scan, narrow LDS ring
// The same recurrence and arithmetic again (results equal bit for bit), for
// few lanes, where each step of the register-ring scan waits on the one
// before.  A workgroup owns 64 consecutive hidden units of one (sequence,
// direction): one consumer wave runs the recurrence from LDS, one producer
// wave streams its inputs into a ring of kNrSlots groups of kNrSteps steps.
// A producer load covers four steps of one input segment (16 lanes x 16
// bytes per step), so a group takes 4 loads per segment and three groups
// stay in flight within the 63 loads vmcnt counts; the two waves meet at
// one barrier per group.  Mask bytes: lanes 0-15 load one step's byte each
// into their dword of the group's mask slot.
constexpr int kNrUnits = 64;
constexpr int kNrSteps = 16;  // steps per hand-off
constexpr int kNrSlots = 4;   // groups in the ring

template <int KB, bool MASK, bool STORE_C, bool STORE_HB, bool RN>
__global__ __launch_bounds__(128) void scan_fwd_nring_kernel(ScanShape s, ScanFwdArgs a,
                                                             unsigned u_bytes, unsigned x_bytes,
                                                             unsigned m_bytes) {
  constexpr int NSEG = 4;  // U blocks 0-2 and x (k = 3), or U blocks 0-3 (k = 4)
  constexpr int STEPB = kNrUnits * 4;        // one segment of one step
  constexpr int SEGB = kNrSteps * STEPB;     // one segment of a group
  constexpr int SLOTB = NSEG * SEGB;
  constexpr int IPG = NSEG * (kNrSteps / 4) + (MASK ? 1 : 0);  // loads per group
  static_assert((kNrSlots - 1) * IPG < 64, "vmcnt counts at most 63 loads");
  __shared__ __attribute__((aligned(1024))) unsigned char ring[kNrSlots * SLOTB];
  __shared__ __attribute__((aligned(256))) unsigned mring[kNrSlots][64];

  const int nblk = s.d / kNrUnits;
  const int jb = blockIdx.x % nblk;
  const int bd = blockIdx.x / nblk;
  const int dir = bd % s.ndir;
  const int b = bd / s.ndir;
  const bool rev = s.direction == 1 || (s.direction == 2 && dir == 1);
  const int L = s.L;
  const int G = (L + kNrSteps - 1) / kNrSteps;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;

  if (wave == 1) {
    // ---- producer
    const __amdgpu_buffer_rsrc_t ru = ring_rsrc(a.U, u_bytes);
    const __amdgpu_buffer_rsrc_t rx = ring_rsrc(KB == 3 ? a.X : a.U, KB == 3 ? x_bytes : u_bytes);
    const __amdgpu_buffer_rsrc_t rm =
        ring_rsrc(MASK ? static_cast<const void*>(a.mask) : static_cast<const void*>(a.U),
                  MASK ? m_bytes : u_bytes);
    const unsigned u_step = (unsigned)s.B * s.ndir * KB * s.d * 4u;
    const unsigned x_step = (unsigned)s.B * s.d_in * 4u;
    const int sub = lane >> 4;                    // step of the four an instruction loads
    const unsigned uc = (unsigned)(lane & 15) * 16u;  // the lane's four units
    const unsigned u_base =
        (unsigned)((((long long)b * s.ndir + dir) * KB * s.d + jb * kNrUnits) * 4) + uc;
    const unsigned x_base = (unsigned)(((long long)b * s.d_in + jb * kNrUnits) * 4) + uc;
    const unsigned seg = (unsigned)s.d * 4u;
    auto issue = [&](int gi) {
      unsigned char* slot = ring + (gi % kNrSlots) * SLOTB;
#pragma unroll
      for (int k4 = 0; k4 < kNrSteps / 4; ++k4) {
        const int step = gi * kNrSteps + 4 * k4 + sub;
        const bool in = step < L;
        const unsigned t = in ? (unsigned)(rev ? L - 1 - step : step) : 0u;
        const unsigned oob = in ? 0u : kRingOOB;
        const unsigned uo = (t * u_step + u_base) | oob;
#pragma unroll
        for (int q = 0; q < KB; ++q)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              ru, (lds_t*)(slot + q * SEGB + k4 * 4 * STEPB), 16, uo + q * seg, 0, 0, 0);
        if constexpr (KB == 3)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rx, (lds_t*)(slot + 3 * SEGB + k4 * 4 * STEPB), 16, (t * x_step + x_base) | oob, 0,
              0, 0);
      }
      if constexpr (MASK) {
        const int step = gi * kNrSteps + lane;
        const bool in = lane < kNrSteps && step < L;
        const unsigned t = in ? (unsigned)(rev ? L - 1 - step : step) : 0u;
        const unsigned mo = in ? t * (unsigned)s.B + (unsigned)b : kRingOOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rm, (lds_t*)(&mring[gi % kNrSlots][0]), 1, mo, 0,
                                                 0, 0);
      }
    };
    for (int gi = 0; gi < kNrSlots - 1 && gi < G; ++gi) issue(gi);
    for (int g = 0; g < G; ++g) {
      // group g has landed once at most the groups issued after it remain
      const int later = min(kNrSlots - 2, G - 1 - g);
      if (later >= 2) __builtin_amdgcn_s_waitcnt(ring_vm_wait(2 * IPG));
      else if (later == 1) __builtin_amdgcn_s_waitcnt(ring_vm_wait(IPG));
      else __builtin_amdgcn_s_waitcnt(ring_vm_wait(0));
      ring_barrier();
      // the slot of group g - 1, which the consumer finished before the barrier
      if (g + kNrSlots - 1 < G) issue(g + kNrSlots - 1);
    }
    return;
  }

  // ---- consumer: unit j of (b, dir), lane gid of the [B, ndir*d] state
  const int j = jb * kNrUnits + lane;
  const int fidx = dir * s.d + j;
  const long long nfeat = (long long)s.ndir * s.d;
  const long long gid = (long long)b * nfeat + fidx;
  const long long h_step = (long long)s.B * nfeat;
  const long long t0 = rev ? L - 1 : 0;
  const long long sh = rev ? -h_step : h_step;
  float* hp = a.H + gid + t0 * h_step;
  float* cp = STORE_C ? a.C + gid + t0 * h_step : nullptr;
  uint16_t* hbp = STORE_HB ? a.Hb + gid + t0 * h_step : nullptr;
  const float vfs = a.v_f[fidx] * kNegLog2e, vrs = a.v_r[fidx] * kNegLog2e;
  const float bfs = a.b_f[fidx] * kNegLog2e, brs = a.b_r[fidx] * kNegLog2e;
  const float alpha = s.alpha;
  float c = a.c0 ? a.c0[gid] : 0.0f;

  auto step = [&](float u0, float u1, float u2, float xh, unsigned mk) {
    const float f = sigmoid_scaled(fmaf(vfs, c, fmaf(u1, kNegLog2e, bfs)));  // Eq. 1
    const float cn = fmaf(f, c, fmaf(-f, u0, u0));                           // Eq. 2
    const float r = sigmoid_scaled(fmaf(vrs, RN ? cn : c, fmaf(u2, kNegLog2e, brs)));  // Eq. 3
    float h = fmaf(r, cn, (1.0f - r) * (alpha * xh));  // Eq. 4 (Sec. 3.2)
    if constexpr (MASK) {
      const bool pad = mk != 0;
      c = pad ? c : cn;
      h = pad ? 0.0f : h;
    } else {
      c = cn;
    }
    // non-temporal stores: the consumer never waits for them (plain ones
    // measured 2-3 % slower here)
    __builtin_nontemporal_store(h, hp);
    if constexpr (STORE_C) __builtin_nontemporal_store(c, cp);
    if constexpr (STORE_HB) __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (__bf16)h), hbp);
    hp += sh;
    if constexpr (STORE_C) cp += sh;
    if constexpr (STORE_HB) hbp += sh;
  };

  const int Gfull = L / kNrSteps;
  for (int g = 0; g < G; ++g) {
    ring_barrier();
    const unsigned char* slot = ring + (g % kNrSlots) * SLOTB + lane * 4;
    const unsigned* mslot = mring[g % kNrSlots];
    auto rd = [&](int q, int st) {
      return *reinterpret_cast<const float*>(slot + q * SEGB + st * STEPB);
    };
    if (g < Gfull) {
#pragma unroll
      for (int st = 0; st < kNrSteps; ++st)
        step(rd(0, st), rd(1, st), rd(2, st), rd(3, st), MASK ? (mslot[st] & 0xFFu) : 0u);
    } else {
#pragma unroll
      for (int st = 0; st < kNrSteps; ++st)
        if (g * kNrSteps + st < L)
          step(rd(0, st), rd(1, st), rd(2, st), rd(3, st), MASK ? (mslot[st] & 0xFFu) : 0u);
    }
  }
  if (a.c_last) a.c_last[gid] = c;
}

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
  using DuT = typename std::conditional<DUB, uint16_t, float>::type;
  const float* cpp = a.C + ln.gid;
  // Cursors, as in the forward scan, moving one step per load or store in
  // the reverse of the direction's order: the load cursors (U, x, dh, mask
  // at t(pos); C at t(pos - 1)) run PF steps ahead of the store cursors and
  // stop at the first position.
  auto tpos = [&](int pos) { return (long long)(ln.rev ? L - 1 - pos : pos); };
  const long long t0 = tpos(L - 1);
  const long long sg = ln.rev ? 1 : -1;
  const long long su = sg * u_step, sx = sg * x_step, sh = sg * h_step, sm = sg * s.B;
  const float* lu = a.U + u_off + t0 * u_step;
  const float* lx = KB == 3 ? a.X + (long long)ln.b * s.d_in + ln.j + t0 * x_step : nullptr;
  const uint8_t* lm = MASK ? a.mask + ln.b + t0 * s.B : nullptr;
  const float* ldh = a.dH + ln.gid + t0 * h_step;
  const float* lc = cpp + tpos(L > 1 ? L - 2 : 0) * h_step;
  DuT* dup = static_cast<DuT*>(a.dU) + u_off + t0 * u_step;
  float* dxp = KB == 3 ? a.dxh + ln.gid + t0 * h_step : nullptr;
  int nl = 0;  // loads issued
  int is = 0;  // steps done

  const float vf = a.v_f[ln.fidx], vr = a.v_r[ln.fidx];
  // the forward scan's gate arithmetic (sigmoid_scaled), so f and r are the
  // forward's values bit for bit
  const float vfs = vf * kNegLog2e, vrs = vr * kNegLog2e;
  const float bfs = a.b_f[ln.fidx] * kNegLog2e, brs = a.b_r[ln.fidx] * kNegLog2e;
  const float alpha = s.alpha;
  const float c0v = a.c0 ? a.c0[ln.gid] : 0.0f;
  float g = a.dc_last ? a.dc_last[ln.gid] : 0.0f;
  float sum_df_c = 0.f, sum_dr_c = 0.f, sum_df = 0.f, sum_dr = 0.f;

  float c_t = cpp[t0 * h_step];

  float r0[PF], r1[PF], r2[PF], rx[PF], rdh[PF], rcp[PF];
  // mask bytes held one per register: a byte array would be packed four to
  // a register, and packing waits for the loads that fill it
  unsigned rm[PF];
  (void)rm;

  auto load = [&](float& u0, float& u1, float& u2, float& xh, float& dh, float& cprev,
                  unsigned& m) {
    u0 = __builtin_nontemporal_load(lu);
    u1 = __builtin_nontemporal_load(lu + d);
    u2 = __builtin_nontemporal_load(lu + 2 * d);
    if constexpr (KB == 4) xh = __builtin_nontemporal_load(lu + 3 * d);
    else xh = *lx;
    dh = __builtin_nontemporal_load(ldh);
    cprev = *lc;
    if constexpr (MASK) m = *lm;
    // the same for the whole wave: load nl + 1 is at position L-2-nl, its
    // C one position earlier
    const bool adv = nl + 1 < L, advc = nl + 2 < L;
    ++nl;
    lu = adv ? lu + su : lu;
    if constexpr (KB == 3) lx = adv ? lx + sx : lx;
    ldh = adv ? ldh + sh : ldh;
    if constexpr (MASK) lm = adv ? lm + sm : lm;
    lc = advc ? lc + sh : lc;
  };
  auto step = [&](float u0, float u1, float u2, float xh, float dh, float cprev, unsigned m) {
    const float c_p = is + 1 < L ? cprev : c0v;  // position 0 starts from c0
    ++is;
    const float c_r = RN ? c_t : c_p;  // the state the reset gate reads
    const float f = sigmoid_scaled(fmaf(vfs, c_p, fmaf(u1, kNegLog2e, bfs)));
    const float r = sigmoid_scaled(fmaf(vrs, c_r, fmaf(u2, kNegLog2e, brs)));
    bool pad = false;
    if constexpr (MASK) pad = m != 0;
    const float dhv = pad ? 0.0f : dh;
    const float rr = r * (1.0f - r);
    const float ff = f * (1.0f - f);
    float dr = dhv * (c_t - alpha * xh) * rr;
    // total gradient into c_t: from later steps, through h, and (RN)
    // through the reset gate
    const float gc = RN ? fmaf(dr, vr, fmaf(dhv, r, g)) : fmaf(dhv, r, g);
    const float pf = (c_p - u0) * ff;  // df = gc pf
    float df = gc * pf;
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
    // g <- gc f + df v_f (+ dr v_r) = gc (f + pf v_f) (+ dr v_r): two
    // dependent operations from g to the next g
    const float gf = fmaf(pf, vf, f);
    const float gn = RN ? gc * gf : fmaf(gc, gf, dr * vr);
    g = pad ? g : gn;
    // bf16 dU goes through the cache: the products read it next (L 256,
    // B 64, d 1024: 97.4 -> 92.5 us, while dW, which runs next, takes 2-3 us
    // longer).  fp32 dU and the highway gradient, which is read only after
    // dW, stream to memory.
    auto put = [](float v, DuT* p) {
      if constexpr (DUB) *p = __builtin_bit_cast(uint16_t, (__bf16)v);
      else __builtin_nontemporal_store(v, p);
    };
    put(du0, dup);
    put(df, dup + d);
    put(dr, dup + 2 * d);
    if constexpr (KB == 4) put(dx, dup + 3 * d);
    else __builtin_nontemporal_store(dx, dxp);
    dup += su;
    if constexpr (KB == 3) dxp += sh;
    // c_t takes the value in a register of its own.  Were it to share
    // cprev's register, the ring's registers would shift by one slot per
    // step and the loop would copy still-loading values at its back edge.
    asm volatile("v_mov_b32 %0, %1" : "=v"(c_t) : "v"(cprev));
  };

#pragma unroll
  for (int p = 0; p < PF; ++p) load(r0[p], r1[p], r2[p], rx[p], rdh[p], rcp[p], rm[p]);
  // The loop is entered from the prologue, whose loads alone set the
  // waits of the first steps of every ring (a lead of 3 steps, not PF, on
  // the ring's first step).  With the first ring peeled off, every step
  // waits for loads PF steps back, and the scan was slower: more memory
  // operations per wave than the memory system serves best (L 256, B 64,
  // d 1024: 92.5 -> 96.7 us; L 400, B 32, d 128: 72.0 -> 78.9 us).
  int i0 = 0;
  for (; i0 + PF <= L; i0 += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      step(r0[p], r1[p], r2[p], rx[p], rdh[p], rcp[p], rm[p]);
      load(r0[p], r1[p], r2[p], rx[p], rdh[p], rcp[p], rm[p]);  // index i0 + p + PF (or the last)
      __builtin_amdgcn_sched_barrier(0);  // as in the forward scan
    }
  }
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (i0 + p < L) step(r0[p], r1[p], r2[p], rx[p], rdh[p], rcp[p], rm[p]);

  float* part = a.partial + (long long)ln.b * 4 * nfeat + ln.fidx;
  part[0] = sum_df_c;
  part[nfeat] = sum_dr_c;
  part[2 * nfeat] = sum_df;
  part[3 * nfeat] = sum_dr;
  if (a.dc0) a.dc0[ln.gid] = g;
}

// ------------------------------------------------- linear variant, chunked
// Ablation (1) of Sec. 4.5 removes v * c_{t-1} from both gates: f and r then
// depend on the projections only, and each step is an affine map of the
// state, c -> f c + (1 - f) u0.  Affine maps compose, so time can be split
// into chunks that are scanned in parallel:
//   1. every chunk folds its steps into one map (A, S) = (prod f, the state
//      reached from 0),
//   2. a chunk's incoming state is the previous state pushed through the
//      maps of the chunks before it,
//   3. every chunk rescans its steps from that state.
// A workgroup is 64 lanes (b, direction, j) times NW waves; it walks the
// direction's step order in blocks of NW * CH steps, wave w taking steps
// [w CH, (w + 1) CH) of a block.  Step 1 runs on the block's loads held in
// registers, the maps meet in LDS (step 2), and step 3 rescans the same
// registers, so every element is read and written once, as in the
// sequential scan.  The block's final state (after the rescan, held by
// the wave that owns the block's last step) is the next
// block's incoming state.  The backward pass does the
// same on the carried gradient, g -> f (g + dh r), in reverse step order.
// No wave leaves early: every wave reaches every barrier.
//
// When the lane groups alone would leave CUs idle (small B*ndir*d), time is
// also cut into segments of whole blocks, one workgroup per (group,
// segment).  A first kernel folds every segment but the last into its map;
// the chunked kernel then starts each segment from the maps of the segments
// before it composed onto c0 (dc_last backward).  That reads two of the
// inputs twice, and fills the chip.
constexpr int kLinMaxWaves = 16;

// Workgroup barrier for LDS hand-offs: waits for this wave's LDS accesses
// only (the release fence of __syncthreads would also drain every
// outstanding global store); the memory clobbers keep the compiler from
// moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0) (vmcnt 63, expcnt 7)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Lane of a chunked workgroup: as decode_lane, with the lane index taken
// from threadIdx.x mod 64.  Lanes past the end (live = false) take the last
// lane's coordinates, so every address they form is in range; they store
// nothing.
__device__ __forceinline__ bool decode_lane_lin(const ScanShape& s, Lane& ln, int group) {
  const int nfeat = s.ndir * s.d;
  const int total = s.B * nfeat;
  const int gid = group * 64 + (threadIdx.x & 63);
  const bool live = gid < total;
  ln.gid = live ? gid : total - 1;
  ln.b = ln.gid / nfeat;
  ln.fidx = ln.gid - ln.b * nfeat;
  ln.dir = ln.fidx / s.d;
  ln.j = ln.fidx - ln.dir * s.d;
  ln.rev = s.direction == 1 || (s.direction == 2 && ln.dir == 1);
  return live;
}

// The backward's segment maps follow its partial rows [nseg * B, 4, ndir*d].
__host__ __device__ __forceinline__ float2* lin_bwd_maps(float* partial, const ScanShape& s,
                                                        const LinPlan& pl) {
  return reinterpret_cast<float2*>(partial + (long long)pl.nseg * s.B * 4 * s.ndir * s.d);
}

// Segment maps: every segment but the last folded into (A, S) per lane, in
// the order of the chunked kernels' first phase (chunks of CH steps per wave,
// the waves' maps composed in wave order, block after block).  MAPB selects
// the backward's map, g -> f (g + dh r), in reverse step order.
template <bool MASK, bool MAPB, int CH>
__global__ __launch_bounds__(64 * kLinMaxWaves) void scan_lin_maps_kernel(ScanShape s,
                                                                          ScanFwdArgs fa,
                                                                          ScanBwdArgs ba,
                                                                          LinPlan pl) {
  __shared__ float2 red[kLinMaxWaves][64];
  Lane ln;
  const int group = blockIdx.x % pl.groups, seg = blockIdx.x / pl.groups;
  const bool live = decode_lane_lin(s, ln, group);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int NW = blockDim.x >> 6;
  const int L = s.L;
  const int d = s.d;
  const long long nfeat = (long long)s.ndir * s.d;
  const int KB = s.k;
  const long long u_step = (long long)s.B * s.ndir * KB * s.d;
  const long long h_step = (long long)s.B * nfeat;
  const float* up = (MAPB ? ba.U : fa.U) + ((long long)ln.b * s.ndir + ln.dir) * KB * s.d + ln.j;
  const uint8_t* mk = MAPB ? ba.mask : fa.mask;
  const uint8_t* mp = MASK ? mk + ln.b : nullptr;
  const float* dhp = MAPB ? ba.dH + ln.gid : nullptr;
  const float bf = (MAPB ? ba.b_f : fa.b_f)[ln.fidx];
  const float br = MAPB ? ba.b_r[ln.fidx] : 0.0f;
  // time index of a position of this segment in the pass's order
  auto tof = [&](int st) {
    const int pos = MAPB ? L - 1 - st : st;  // forward-order position
    return (long long)(ln.rev ? L - 1 - pos : pos);
  };
  const int sbeg = seg * pl.seg_steps, send = min(L, sbeg + pl.seg_steps);
  float A = 1.0f, S = 0.0f;
  for (int base = sbeg; base < send; base += NW * CH) {
    const int st0 = base + w * CH;
    float r1[CH], r2[CH], rd[CH];
    bool act[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const long long t = tof(st0 + i < send ? st0 + i : send - 1);
      r1[i] = __builtin_nontemporal_load(up + t * u_step + d);
      if constexpr (MAPB) {
        r2[i] = __builtin_nontemporal_load(up + t * u_step + 2 * d);
        rd[i] = __builtin_nontemporal_load(dhp + t * h_step);
      } else {
        r2[i] = __builtin_nontemporal_load(up + t * u_step);  // u0
        rd[i] = 0.0f;
      }
      act[i] = st0 + i < send;
      if constexpr (MASK) act[i] = act[i] && mp[t * s.B] == 0;
    }
    float Aw = 1.0f, Sw = 0.0f;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const float f = sigmoid_fast(r1[i] + bf);
      if (act[i]) {
        if constexpr (MAPB) {
          const float r = sigmoid_fast(r2[i] + br);
          Sw = f * fmaf(rd[i], r, Sw);
        } else {
          Sw = fmaf(f, Sw, (1.0f - f) * r2[i]);
        }
        Aw *= f;
      }
    }
    red[w][lane] = make_float2(Aw, Sw);
    lds_barrier();
    for (int m = 0; m < NW; ++m) {
      const float2 q = red[m][lane];
      S = fmaf(q.x, S, q.y);
      A *= q.x;
    }
    lds_barrier();  // before the next block's chunk maps
  }
  if (w == 0 && live) {
    float2* out = MAPB ? lin_bwd_maps(ba.partial, s, pl)
                       : reinterpret_cast<float2*>(fa.scratch);
    out[((long long)group * pl.nseg + seg) * 64 + lane] = make_float2(A, S);
  }
}

template <int KB, bool MASK, bool STORE_C, bool STORE_HB, int CH>
__global__ __launch_bounds__(64 * kLinMaxWaves) void scan_fwd_lin_kernel(ScanShape s,
                                                                         ScanFwdArgs a,
                                                                         LinPlan pl) {
  __shared__ float2 agg[2][kLinMaxWaves][64];  // (A, S) per block parity, wave, lane
  __shared__ float carry_lds[2][64];           // block's final state, per parity
  Lane ln;
  const int group = blockIdx.x % pl.groups, seg = blockIdx.x / pl.groups;
  const bool live = decode_lane_lin(s, ln, group);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int NW = blockDim.x >> 6;
  const int L = s.L;
  const int d = s.d;
  const long long nfeat = (long long)s.ndir * s.d;
  const long long u_step = (long long)s.B * s.ndir * KB * s.d;
  const long long x_step = (long long)s.B * s.d_in;
  const long long h_step = (long long)s.B * nfeat;
  const float* up = a.U + ((long long)ln.b * s.ndir + ln.dir) * KB * s.d + ln.j;
  const float* xp = KB == 3 ? a.X + (long long)ln.b * s.d_in + ln.j : nullptr;
  const uint8_t* mp = MASK ? a.mask + ln.b : nullptr;
  const float bf = a.b_f[ln.fidx], br = a.b_r[ln.fidx];
  const float alpha = s.alpha;
  // this workgroup's steps [sbeg, send) of the direction's order; the
  // incoming state: c0 through the maps of the segments before this one
  const int sbeg = seg * pl.seg_steps, send = min(L, sbeg + pl.seg_steps);
  float carry = a.c0 ? a.c0[ln.gid] : 0.0f;
  {
    const float2* sm = reinterpret_cast<const float2*>(a.scratch) + (long long)group * pl.nseg * 64;
    for (int q = 0; q < seg; ++q) {
      const float2 m = sm[q * 64 + lane];
      carry = fmaf(m.x, carry, m.y);
    }
  }
  auto tindex = [&](int st) { return ln.rev ? L - 1 - st : st; };

  int blk = 0;
  for (int base = sbeg; base < send; base += NW * CH, ++blk) {
    const int p = blk & 1;
    const int st0 = base + w * CH;
    float ru0[CH], rf[CH], ru2[CH], rx[CH];
    bool act[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int st = st0 + i < send ? st0 + i : send - 1;
      const long long t = tindex(st);
      const float* u = up + t * u_step;
      ru0[i] = __builtin_nontemporal_load(u);
      rf[i] = __builtin_nontemporal_load(u + d);
      ru2[i] = __builtin_nontemporal_load(u + 2 * d);
      if constexpr (KB == 4) rx[i] = __builtin_nontemporal_load(u + 3 * d);
      else rx[i] = xp[t * x_step];
      act[i] = st0 + i < send;
      if constexpr (MASK) act[i] = act[i] && mp[t * s.B] == 0;
    }
    // 1. this chunk's map
    float A = 1.0f, S = 0.0f;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const float f = sigmoid_fast(rf[i] + bf);  // Eq. 1 without v * c
      rf[i] = f;
      if (act[i]) {
        S = fmaf(f, S, (1.0f - f) * ru0[i]);
        A *= f;
      }
    }
    agg[p][w][lane] = make_float2(A, S);
    lds_barrier();
    // 2. incoming state: the previous block's final state through the maps
    //    of the chunks before this one
    float c = blk == 0 ? carry : carry_lds[p ^ 1][lane];
    for (int m = 0; m < w; ++m) {
      const float2 g = agg[p][m][lane];
      c = fmaf(g.x, c, g.y);
    }
    // 3. rescan
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      if (st0 + i >= send) break;
      const long long t = tindex(st0 + i);
      const float f = rf[i];
      const float cn = fmaf(f, c, (1.0f - f) * ru0[i]);            // Eq. 2
      const float r = sigmoid_fast(ru2[i] + br);                   // Eq. 3 without v * c
      float h = fmaf(r, cn, (1.0f - r) * (alpha * rx[i]));         // Eq. 4 (Sec. 3.2)
      if (act[i]) c = cn;
      else h = 0.0f;
      if (live) {
        __builtin_nontemporal_store(h, a.H + ln.gid + t * h_step);
        if constexpr (STORE_C) __builtin_nontemporal_store(c, a.C + ln.gid + t * h_step);
        if constexpr (STORE_HB)
          __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (__bf16)h),
                                      a.Hb + ln.gid + t * h_step);
      }
    }
    // the wave holding the block's last step publishes the rescanned state
    const int w_last = (min(send - base, NW * CH) - 1) / CH;
    if (w == w_last) {
      carry_lds[p][lane] = c;
      if (base + NW * CH >= send && send == L && live && a.c_last) a.c_last[ln.gid] = c;
    }
  }
}

// Backward of the variant.  Processing index i visits forward-order
// position pos = L-1-i.  cval(i) = C at position L-1-i (c0 for i = L), so
// step i has c_t = cval(i) and c_p = cval(i+1).  Per step:
//   gc = g + dh r;  du0 = gc (1 - f);  df = gc (c_p - u0) f (1 - f)
//   dr = dh (c_t - alpha x_hat) r (1 - r);  dx_hat = dh (1 - r) alpha
//   g <- gc f          (the map g -> f g + f dh r)
// b_f / b_r sums go to partial[b][2|3][feature] after a fixed-order sum
// over the workgroup's waves.
template <int KB, bool MASK, bool DUB, int CH>
__global__ __launch_bounds__(64 * kLinMaxWaves) void scan_bwd_lin_kernel(ScanShape s,
                                                                         ScanBwdArgs a,
                                                                         LinPlan pl) {
  __shared__ float2 agg[2][kLinMaxWaves][64];
  __shared__ float carry_lds[2][64];
  Lane ln;
  const int group = blockIdx.x % pl.groups, seg = blockIdx.x / pl.groups;
  const bool live = decode_lane_lin(s, ln, group);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int NW = blockDim.x >> 6;
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
  const float bf = a.b_f[ln.fidx], br = a.b_r[ln.fidx];
  const float alpha = s.alpha;
  const float c0v = a.c0 ? a.c0[ln.gid] : 0.0f;
  // processing indices [sbeg, send) of this workgroup; the incoming
  // gradient: dc_last through the maps of the segments before this one
  const int sbeg = seg * pl.seg_steps, send = min(L, sbeg + pl.seg_steps);
  float carry = a.dc_last ? a.dc_last[ln.gid] : 0.0f;
  {
    const float2* sm = lin_bwd_maps(a.partial, s, pl) + (long long)group * pl.nseg * 64;
    for (int q = 0; q < seg; ++q) {
      const float2 m = sm[q * 64 + lane];
      carry = fmaf(m.x, carry, m.y);
    }
  }
  float sum_df = 0.f, sum_dr = 0.f;
  // time index of processing index i (clamped into range)
  auto tproc = [&](int i) {
    const int pos = L - 1 - (i < L ? i : L - 1);
    return (long long)(ln.rev ? L - 1 - pos : pos);
  };

  int blk = 0;
  for (int base = sbeg; base < send; base += NW * CH, ++blk) {
    const int p = blk & 1;
    const int i0 = base + w * CH;
    float ru0[CH], rf[CH], rr[CH], rx[CH], rdh[CH], rc[CH + 1];
    bool act[CH];
#pragma unroll
    for (int m = 0; m < CH; ++m) {
      const long long t = tproc(i0 + m);
      const float* u = up + t * u_step;
      ru0[m] = __builtin_nontemporal_load(u);
      rf[m] = __builtin_nontemporal_load(u + d);
      rr[m] = __builtin_nontemporal_load(u + 2 * d);
      if constexpr (KB == 4) rx[m] = __builtin_nontemporal_load(u + 3 * d);
      else rx[m] = xp[t * x_step];
      rdh[m] = __builtin_nontemporal_load(dhp + t * h_step);
      rc[m] = cpp[t * h_step];
      act[m] = i0 + m < send;
      if constexpr (MASK) act[m] = act[m] && mp[t * s.B] == 0;
    }
    {
      const int ie = i0 + CH;  // c_p of the chunk's last step
      rc[CH] = ie < L ? cpp[tproc(ie) * h_step] : c0v;
    }
    // 1. this chunk's map on the carried gradient
    float A = 1.0f, S = 0.0f;
#pragma unroll
    for (int m = 0; m < CH; ++m) {
      const float f = sigmoid_fast(rf[m] + bf);
      const float r = sigmoid_fast(rr[m] + br);
      rf[m] = f;
      rr[m] = r;
      if (act[m]) {
        S = f * fmaf(rdh[m], r, S);
        A *= f;
      }
    }
    agg[p][w][lane] = make_float2(A, S);
    lds_barrier();
    // 2. incoming gradient
    float g = blk == 0 ? carry : carry_lds[p ^ 1][lane];
    for (int m = 0; m < w; ++m) {
      const float2 q = agg[p][m][lane];
      g = fmaf(q.x, g, q.y);
    }
    // 3. rescan
#pragma unroll
    for (int m = 0; m < CH; ++m) {
      if (i0 + m >= send) break;
      const long long t = tproc(i0 + m);
      const float f = rf[m], r = rr[m];
      const float c_t = rc[m];
      const float c_p = i0 + m + 1 < L ? rc[m + 1] : c0v;
      const float dh = act[m] ? rdh[m] : 0.0f;
      const float gc = fmaf(dh, r, g);
      float du0 = gc * (1.0f - f);
      float df = gc * (c_p - ru0[m]) * (f * (1.0f - f));
      float dr = dh * (c_t - alpha * rx[m]) * (r * (1.0f - r));
      float dx = dh * (1.0f - r) * alpha;
      if (act[m]) {
        g = gc * f;
      } else {
        du0 = df = dr = dx = 0.0f;
      }
      sum_df += df;
      sum_dr += dr;
      if (live) {
        DuT* du = dup + t * u_step;
        auto put = [](float v, DuT* q) {
          if constexpr (DUB)
            __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (__bf16)v), q);
          else
            __builtin_nontemporal_store(v, q);
        };
        put(du0, du);
        put(df, du + d);
        put(dr, du + 2 * d);
        if constexpr (KB == 4) put(dx, du + 3 * d);
        else __builtin_nontemporal_store(dx, a.dxh + ln.gid + t * h_step);
      }
    }
    const int w_last = (min(send - base, NW * CH) - 1) / CH;
    if (w == w_last) {
      carry_lds[p][lane] = g;
      if (base + NW * CH >= send && send == L && live && a.dc0) a.dc0[ln.gid] = g;
    }
  }
  // fixed-order sum of the waves' b sums (agg is free: every wave is past
  // its last read of it once it reaches this barrier)
  lds_barrier();
  agg[0][w][lane] = make_float2(sum_df, sum_dr);
  lds_barrier();
  if (w == 0 && live) {
    float sdf = 0.f, sdr = 0.f;
    for (int m = 0; m < NW; ++m) {
      const float2 q = agg[0][m][lane];
      sdf += q.x;
      sdr += q.y;
    }
    // one row of partials per (segment, sequence)
    float* part = a.partial + ((long long)seg * s.B + ln.b) * 4 * nfeat + ln.fidx;
    part[2 * nfeat] = sdf;
    part[3 * nfeat] = sdr;
  }
}

// ------------------------------------- gated backward, time-parallel
// Given the forward states C, the backward recurrence of the gated layer is
// affine in the carried gradient: a step maps g to A g + B with A = f +
// p_f v_f (p_f = (c_{t-1} - u0) f (1 - f)) and B = A (dh r) + dr v_r, or
// A (dh r + dr v_r) when the reset gate reads c_t; a padded step is the
// identity.  So the reverse scan splits into chunks like the linear
// recurrence's (scan_bwd_lin_kernel): every wave folds its CH steps into one
// map, a chunk's incoming gradient is the block's incoming gradient pushed
// through the maps of the chunks before it, and every wave rescans its steps
// with the sequential kernel's arithmetic from there.  The outputs of a step
// are then those of scan_bwd_kernel for the same incoming gradient, which
// differs from the sequential one by rounding only.  One workgroup per 64
// lanes covers the whole sequence (no time segments), so this serves shapes
// whose lane groups alone fill at least half the CUs and leave most SIMDs
// without a wave; there the sequential scan waits on its serial chain.
template <int KB, bool MASK, bool DUB, bool RN, int CH>
__global__ __launch_bounds__(64 * kLinMaxWaves) void scan_bwd_tp_kernel(ScanShape s,
                                                                        ScanBwdArgs a,
                                                                        LinPlan pl) {
  __shared__ float2 agg[2][kLinMaxWaves][64];
  __shared__ float carry_lds[2][64];
  Lane ln;
  const bool live = decode_lane_lin(s, ln, blockIdx.x);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int NW = blockDim.x >> 6;
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
  // the forward's gate arithmetic (sigmoid_scaled), as in scan_bwd_kernel
  const float vf = a.v_f[ln.fidx], vr = a.v_r[ln.fidx];
  const float vfs = vf * kNegLog2e, vrs = vr * kNegLog2e;
  const float bfs = a.b_f[ln.fidx] * kNegLog2e, brs = a.b_r[ln.fidx] * kNegLog2e;
  const float alpha = s.alpha;
  const float c0v = a.c0 ? a.c0[ln.gid] : 0.0f;
  float sum_df_c = 0.f, sum_dr_c = 0.f, sum_df = 0.f, sum_dr = 0.f;
  // time index of processing index i (reverse of the direction's order;
  // clamped into range)
  auto tproc = [&](int i) {
    const int pos = L - 1 - (i < L ? i : L - 1);
    return (long long)(ln.rev ? L - 1 - pos : pos);
  };

  int blk = 0;
  for (int base = 0; base < L; base += NW * CH, ++blk) {
    const int p = blk & 1;
    const int i0 = base + w * CH;
    float ru0[CH], rf[CH], rr[CH], rx[CH], rdh[CH], rc[CH + 1];
    bool act[CH], pad[CH];
#pragma unroll
    for (int m = 0; m < CH; ++m) {
      const long long t = tproc(i0 + m);
      const float* u = up + t * u_step;
      ru0[m] = __builtin_nontemporal_load(u);
      rf[m] = __builtin_nontemporal_load(u + d);
      rr[m] = __builtin_nontemporal_load(u + 2 * d);
      if constexpr (KB == 4) rx[m] = __builtin_nontemporal_load(u + 3 * d);
      else rx[m] = xp[t * x_step];
      rdh[m] = __builtin_nontemporal_load(dhp + t * h_step);
      rc[m] = cpp[t * h_step];
      act[m] = i0 + m < L;
      pad[m] = MASK ? mp[t * s.B] != 0 : false;
    }
    {
      const int ie = i0 + CH;  // c_{t-1} of the chunk's last step
      rc[CH] = ie < L ? cpp[tproc(ie) * h_step] : c0v;
    }
    // 1. this chunk's map on the carried gradient (f and r replace u1, u2)
    float A = 1.0f, S = 0.0f;
#pragma unroll
    for (int m = 0; m < CH; ++m) {
      const float c_t = rc[m];
      const float c_p = i0 + m + 1 < L ? rc[m + 1] : c0v;
      const float c_r = RN ? c_t : c_p;
      const float f = sigmoid_scaled(fmaf(vfs, c_p, fmaf(rf[m], kNegLog2e, bfs)));
      const float r = sigmoid_scaled(fmaf(vrs, c_r, fmaf(rr[m], kNegLog2e, brs)));
      rf[m] = f;
      rr[m] = r;
      if (act[m] && !pad[m]) {
        const float dh = rdh[m];
        const float dr = dh * (c_t - alpha * rx[m]) * (r * (1.0f - r));
        const float gf = fmaf((c_p - ru0[m]) * (f * (1.0f - f)), vf, f);
        const float bm = RN ? gf * fmaf(dr, vr, dh * r) : fmaf(gf, dh * r, dr * vr);
        S = fmaf(gf, S, bm);
        A *= gf;
      }
    }
    agg[p][w][lane] = make_float2(A, S);
    lds_barrier();
    // 2. incoming gradient of this chunk
    float g = blk == 0 ? (a.dc_last ? a.dc_last[ln.gid] : 0.0f) : carry_lds[p ^ 1][lane];
    for (int m = 0; m < w; ++m) {
      const float2 q = agg[p][m][lane];
      g = fmaf(q.x, g, q.y);
    }
    // 3. rescan: scan_bwd_kernel's step
#pragma unroll
    for (int m = 0; m < CH; ++m) {
      if (i0 + m >= L) break;
      const long long t = tproc(i0 + m);
      const float f = rf[m], r = rr[m];
      const float c_t = rc[m];
      const float c_p = i0 + m + 1 < L ? rc[m + 1] : c0v;
      const float c_r = RN ? c_t : c_p;
      const bool pd = pad[m];
      const float dhv = pd ? 0.0f : rdh[m];
      const float rrv = r * (1.0f - r);
      const float ff = f * (1.0f - f);
      float dr = dhv * (c_t - alpha * rx[m]) * rrv;
      const float gc = RN ? fmaf(dr, vr, fmaf(dhv, r, g)) : fmaf(dhv, r, g);
      const float pf = (c_p - ru0[m]) * ff;
      float df = gc * pf;
      float du0 = gc * (1.0f - f);
      float dx = dhv * (1.0f - r) * alpha;
      if constexpr (MASK) {
        dr = pd ? 0.0f : dr;
        df = pd ? 0.0f : df;
        du0 = pd ? 0.0f : du0;
        dx = pd ? 0.0f : dx;
      }
      sum_df_c = fmaf(df, c_p, sum_df_c);
      sum_dr_c = fmaf(dr, c_r, sum_dr_c);
      sum_df += df;
      sum_dr += dr;
      const float gf = fmaf(pf, vf, f);
      const float gn = RN ? gc * gf : fmaf(gc, gf, dr * vr);
      g = pd ? g : gn;
      if (live) {
        DuT* du = dup + t * u_step;
        // bf16 dU through the cache, as in scan_bwd_kernel
        auto put = [](float v, DuT* q) {
          if constexpr (DUB) *q = __builtin_bit_cast(uint16_t, (__bf16)v);
          else __builtin_nontemporal_store(v, q);
        };
        put(du0, du);
        put(df, du + d);
        put(dr, du + 2 * d);
        if constexpr (KB == 4) put(dx, du + 3 * d);
        else __builtin_nontemporal_store(dx, a.dxh + ln.gid + t * h_step);
      }
    }
    const int w_last = (min(L - base, NW * CH) - 1) / CH;
    if (w == w_last) {
      carry_lds[p][lane] = g;
      if (base + NW * CH >= L && live && a.dc0) a.dc0[ln.gid] = g;
    }
  }
  // fixed-order sum of the waves' v/b sums (agg is free: every wave is past
  // its last read of it once it reaches this barrier)
  lds_barrier();
  agg[0][w][lane] = make_float2(sum_df_c, sum_dr_c);
  agg[1][w][lane] = make_float2(sum_df, sum_dr);
  lds_barrier();
  if (w == 0 && live) {
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    for (int m = 0; m < NW; ++m) {
      const float2 q = agg[0][m][lane], q2 = agg[1][m][lane];
      s0 += q.x;
      s1 += q.y;
      s2 += q2.x;
      s3 += q2.y;
    }
    // one row of partials per sequence, as scan_bwd_kernel writes
    float* part = a.partial + (long long)ln.b * 4 * nfeat + ln.fidx;
    part[0] = s0;
    part[nfeat] = s1;
    part[2 * nfeat] = s2;
    part[3 * nfeat] = s3;
  }
}

// Sum of the per-sequence partials over b, in a fixed order (deterministic):
// vb_sum_block, 64 outputs per workgroup of 4 waves.  The loads of a lane
// are independent, so a launch costs about one memory round trip.  The same
// blocks can run inside the split-K sum of the dW product (sru_gemm.hip),
// which saves this launch; either way the sums are the same bits.
__global__ __launch_bounds__(256) void reduce_vb_kernel(VbSum v) {
  __shared__ float red[256];
  vb_sum_block(v.partial, v.rows, v.nfeat, v.qlo, v.out, blockIdx.x, red);
}

// Steps of loads a lane keeps in flight (its register ring).  Measured on
// MI355X over the workloads' shapes: deeper rings are slower once every SIMD
// holds a wave (the memory system is then saturated and shorter per-wave
// queues serve it better); with fewer waves than SIMDs the backward needs a
// ring of 6 to cover the memory latency, and the forward does best with 6
// everywhere.
constexpr int kFwdPF = 6;
constexpr int kBwdPF = 6;
constexpr int kBwdPFFull = 4;
constexpr int kFullLanes = 256 * 4 * 64;  // one wave on each of the 1024 SIMDs
constexpr int kFwdLinCH = 12;
constexpr int kBwdLinCH = 8;
constexpr int kBwdTpCH = 8;  // steps per wave chunk of the time-parallel gated backward

// Plan of the chunked scans: waves per workgroup so that the launch holds
// about 4096 waves (4 per SIMD), at most 16 per workgroup and no more chunks
// than the sequence has steps.  With lane groups for fewer than half the CUs,
// time is also cut into segments of whole blocks, for up to about two
// workgroups per CU: the segments' maps cost an extra pass over half of the
// scan's input, which pays where the scan is bound by its serial latency
// and not where half the chip already streams from HBM.
LinPlan lin_plan(const ScanShape& s, int ch) {
  LinPlan pl{};
  pl.groups = (s.B * s.ndir * s.d + 63) / 64;
  int nw = 1;
  while (nw < kLinMaxWaves && pl.groups * nw * 2 <= 4096 && nw * ch < s.L) nw *= 2;
  pl.nw = nw;
  const int block = nw * ch;
  const int nblk = (s.L + block - 1) / block;
  int nseg = 1;
  if (pl.groups < 128) nseg = std::min(nblk, (512 + pl.groups - 1) / pl.groups);
  pl.seg_steps = ((nblk + nseg - 1) / nseg) * block;
  pl.nseg = (s.L + pl.seg_steps - 1) / pl.seg_steps;
  return pl;
}

template <int KB, bool MASK, bool STORE_C, bool STORE_HB>
hipError_t fwd_lin_dispatch(const ScanShape& s, const ScanFwdArgs& a, hipStream_t st) {
  const LinPlan pl = lin_plan(s, kFwdLinCH);
  if (pl.nseg > 1) {
    timing_before("scan_maps", st);
    hipLaunchKernelGGL((scan_lin_maps_kernel<MASK, false, kFwdLinCH>),
                       dim3(pl.groups * (pl.nseg - 1)), dim3(64 * pl.nw), 0, st, s, a,
                       ScanBwdArgs{}, pl);
    timing_after(st);
    if (hipError_t e = hipGetLastError()) return e;
  }
  timing_before("scan_fwd", st);
  hipLaunchKernelGGL((scan_fwd_lin_kernel<KB, MASK, STORE_C, STORE_HB, kFwdLinCH>),
                     dim3(pl.groups * pl.nseg), dim3(64 * pl.nw), 0, st, s, a, pl);
  timing_after(st);
  return hipGetLastError();
}

// Where the LDS-ring forward scan runs: gated recurrence, whole groups of
// 256 units, operands inside the 2 GiB range of buffer offsets, enough
// lanes that the scan streams from HBM rather than waiting on its serial
// chain (below that, one wave per 64 units spreads better over the SIMDs),
// and few enough that every workgroup is resident at once (two per CU):
// with a second round of workgroups the register-ring scan, whose waves
// all fit at once, is faster.  Measured at L 256, B 64, d 1024 (256
// workgroups): 68 us against 72 us in the step, the same time cold; at
// L 128, B 128, d 2048 (1024 workgroups): 201 us against 185 us.
constexpr long long kRingMinLanes = 65536;
constexpr long long kRingMaxLanes = 2LL * 256 * kRingUnits;
bool ring_ok(const ScanShape& s, long long u_bytes, long long x_bytes) {
  const long long lanes = (long long)s.B * s.ndir * s.d;
  return !s.linear && s.d % kRingUnits == 0 && lanes >= kRingMinLanes &&
         lanes <= kRingMaxLanes &&
         u_bytes < (long long)kRingOOB && x_bytes < (long long)kRingOOB &&
         (long long)s.L * s.B < (long long)kRingOOB;
}

// Where the narrow LDS ring runs: fewer lanes than one wave per SIMD (there
// each step of the register-ring scan waits on the one before), whole groups
// of 64 units, operands inside the 2 GiB range of buffer offsets.
bool nring_ok(const ScanShape& s, long long u_bytes, long long x_bytes) {
  const long long lanes = (long long)s.B * s.ndir * s.d;
  return !s.linear && s.d % kNrUnits == 0 && lanes < kFullLanes &&
         u_bytes < (long long)kRingOOB && x_bytes < (long long)kRingOOB &&
         (long long)s.L * s.B < (long long)kRingOOB;
}

template <int KB, bool MASK, bool STORE_C, bool STORE_HB>
hipError_t fwd_dispatch(const ScanShape& s, const ScanFwdArgs& a, hipStream_t st) {
  const int lanes = s.B * s.ndir * s.d;
  const int grid = (lanes + kScanThreads - 1) / kScanThreads;
  const long long u_bytes = 4LL * s.L * s.B * s.ndir * KB * s.d;
  const long long x_bytes = KB == 3 ? 4LL * s.L * s.B * s.d_in : 0;
  // the LDS rings load 16 bytes per lane from U and x: their bases must be
  // 16-byte aligned (the interface asks 4 bytes of fp32 tensors)
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  const bool al = al16(a.U) && (KB != 3 || al16(a.X));
  if (al && nring_ok(s, u_bytes, x_bytes)) {
    const int ngrid = s.B * s.ndir * (s.d / kNrUnits);
    const unsigned m_bytes = (unsigned)((long long)s.L * s.B);
    timing_before("scan_fwd", st);
    if (s.reset_new)
      hipLaunchKernelGGL((scan_fwd_nring_kernel<KB, MASK, STORE_C, STORE_HB, true>), dim3(ngrid),
                         dim3(128), 0, st, s, a, (unsigned)u_bytes, (unsigned)x_bytes, m_bytes);
    else
      hipLaunchKernelGGL((scan_fwd_nring_kernel<KB, MASK, STORE_C, STORE_HB, false>), dim3(ngrid),
                         dim3(128), 0, st, s, a, (unsigned)u_bytes, (unsigned)x_bytes, m_bytes);
    timing_after(st);
    return hipGetLastError();
  }
  if (al && ring_ok(s, u_bytes, x_bytes)) {
    const int rgrid = s.B * s.ndir * (s.d / kRingUnits);
    const unsigned m_bytes = (unsigned)((long long)s.L * s.B);
    timing_before("scan_fwd", st);
    if (s.reset_new)
      hipLaunchKernelGGL((scan_fwd_ring_kernel<KB, MASK, STORE_C, STORE_HB, true>), dim3(rgrid),
                         dim3(kRingThreads), 0, st, s, a, (unsigned)u_bytes, (unsigned)x_bytes,
                         m_bytes);
    else
      hipLaunchKernelGGL((scan_fwd_ring_kernel<KB, MASK, STORE_C, STORE_HB, false>), dim3(rgrid),
                         dim3(kRingThreads), 0, st, s, a, (unsigned)u_bytes, (unsigned)x_bytes,
                         m_bytes);
    timing_after(st);
    return hipGetLastError();
  }
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
  if (s.linear) {
    if (a.Hb)
      return a.C ? fwd_lin_dispatch<KB, MASK, true, true>(s, a, st)
                 : fwd_lin_dispatch<KB, MASK, false, true>(s, a, st);
    return a.C ? fwd_lin_dispatch<KB, MASK, true, false>(s, a, st)
               : fwd_lin_dispatch<KB, MASK, false, false>(s, a, st);
  }
  if (a.Hb)
    return a.C ? fwd_dispatch<KB, MASK, true, true>(s, a, st)
               : fwd_dispatch<KB, MASK, false, true>(s, a, st);
  return a.C ? fwd_dispatch<KB, MASK, true, false>(s, a, st)
             : fwd_dispatch<KB, MASK, false, false>(s, a, st);
}

// Where the gated backward runs time-parallel (scan_bwd_tp_kernel): lane
// groups for at least half the CUs (one workgroup per group then covers the
// sequence without segments), and fewer lanes than half the SIMDs hold a
// wave each.  Measured at L 256, d 1024: 16,384 lanes 35.5 us against 48.5
// us sequential; 32,768 lanes 62.2 against 56.8 us (and sequential ahead up
// to 61,440 lanes).  Smaller shapes keep the sequential scan, whose results
// do not depend on how a sequence is cut into calls.
constexpr long long kTpMinLanes = 128 * 64;
constexpr long long kTpMaxLanes = 32768;  // exclusive
bool bwd_tp_ok(const ScanShape& s) {
  const long long lanes = (long long)s.B * s.ndir * s.d;
  return !s.linear && lanes >= kTpMinLanes && lanes < kTpMaxLanes &&
         lin_plan(s, kBwdTpCH).nseg == 1;
}

template <int KB, bool MASK, int PF>
void bwd_launch(const ScanShape& s, const ScanBwdArgs& a, int grid, hipStream_t st) {
  if (a.du_bf16 && s.reset_new)
    hipLaunchKernelGGL((scan_bwd_kernel<KB, MASK, true, true, PF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  else if (a.du_bf16)
    hipLaunchKernelGGL((scan_bwd_kernel<KB, MASK, true, false, PF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  else if (s.reset_new)
    hipLaunchKernelGGL((scan_bwd_kernel<KB, MASK, false, true, PF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
  else
    hipLaunchKernelGGL((scan_bwd_kernel<KB, MASK, false, false, PF>), dim3(grid),
                       dim3(kScanThreads), 0, st, s, a);
}

template <int KB, bool MASK>
hipError_t bwd_dispatch(const ScanShape& s, const ScanBwdArgs& a, hipStream_t st) {
  const int lanes = s.B * s.ndir * s.d;
  const int grid = (lanes + kScanThreads - 1) / kScanThreads;
  if (s.linear) {
    const LinPlan pl = lin_plan(s, kBwdLinCH);
    if (pl.nseg > 1) {
      timing_before("scan_maps", st);
      hipLaunchKernelGGL((scan_lin_maps_kernel<MASK, true, kBwdLinCH>),
                         dim3(pl.groups * (pl.nseg - 1)), dim3(64 * pl.nw), 0, st, s,
                         ScanFwdArgs{}, a, pl);
      timing_after(st);
      if (hipError_t e = hipGetLastError()) return e;
    }
    timing_before("scan_bwd", st);
    if (a.du_bf16)
      hipLaunchKernelGGL((scan_bwd_lin_kernel<KB, MASK, true, kBwdLinCH>),
                         dim3(pl.groups * pl.nseg), dim3(64 * pl.nw), 0, st, s, a, pl);
    else
      hipLaunchKernelGGL((scan_bwd_lin_kernel<KB, MASK, false, kBwdLinCH>),
                         dim3(pl.groups * pl.nseg), dim3(64 * pl.nw), 0, st, s, a, pl);
    timing_after(st);
    return hipGetLastError();
  }
  if (bwd_tp_ok(s)) {
    const LinPlan pl = lin_plan(s, kBwdTpCH);
    const dim3 g(pl.groups), b(64 * pl.nw);
    timing_before("scan_bwd", st);
    if (a.du_bf16 && s.reset_new)
      hipLaunchKernelGGL((scan_bwd_tp_kernel<KB, MASK, true, true, kBwdTpCH>), g, b, 0, st, s, a, pl);
    else if (a.du_bf16)
      hipLaunchKernelGGL((scan_bwd_tp_kernel<KB, MASK, true, false, kBwdTpCH>), g, b, 0, st, s, a, pl);
    else if (s.reset_new)
      hipLaunchKernelGGL((scan_bwd_tp_kernel<KB, MASK, false, true, kBwdTpCH>), g, b, 0, st, s, a, pl);
    else
      hipLaunchKernelGGL((scan_bwd_tp_kernel<KB, MASK, false, false, kBwdTpCH>), g, b, 0, st, s, a, pl);
    timing_after(st);
    return hipGetLastError();
  }
  timing_before("scan_bwd", st);
  if (lanes >= kFullLanes) bwd_launch<KB, MASK, kBwdPFFull>(s, a, grid, st);
  else bwd_launch<KB, MASK, kBwdPF>(s, a, grid, st);
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
  const size_t row = sizeof(float) * 4ull * (size_t)s.ndir * (size_t)s.d;
  if (!s.linear) return row * (size_t)s.B;
  const LinPlan pl = lin_plan(s, kBwdLinCH);
  return row * (size_t)s.B * (size_t)pl.nseg + sizeof(float2) * 64ull * pl.groups * pl.nseg;
}

size_t scan_forward_scratch_bytes(const ScanShape& s) {
  if (!s.linear) return 0;
  const LinPlan pl = lin_plan(s, kFwdLinCH);
  return pl.nseg > 1 ? sizeof(float2) * 64ull * pl.groups * pl.nseg : 0;
}

hipError_t scan_backward_launch(const ScanShape& s, const ScanBwdArgs& a, hipStream_t st) {
  const bool m = a.mask != nullptr;
  hipError_t e;
  if (s.k == 3) e = m ? bwd_dispatch<3, true>(s, a, st) : bwd_dispatch<3, false>(s, a, st);
  else e = m ? bwd_dispatch<4, true>(s, a, st) : bwd_dispatch<4, false>(s, a, st);
  if (e != hipSuccess) return e;
  if (a.defer_vb) return hipSuccess;
  return vb_sum_launch(scan_backward_vb(s, a), st);
}

VbSum scan_backward_vb(const ScanShape& s, const ScanBwdArgs& a) {
  VbSum v{};
  v.partial = a.partial;
  v.nfeat = s.ndir * s.d;
  v.qlo = s.linear ? 2 : 0;
  // the linear scans leave one row of partials per (segment, sequence)
  v.rows = s.linear ? s.B * lin_plan(s, kBwdLinCH).nseg : s.B;
  v.out[0] = a.dv_f;
  v.out[1] = a.dv_r;
  v.out[2] = a.db_f;
  v.out[3] = a.db_r;
  return v;
}

hipError_t vb_sum_launch(const VbSum& v, hipStream_t st) {
  timing_before("reduce_vb", st);
  hipLaunchKernelGGL(reduce_vb_kernel, dim3(vb_sum_blocks(v)), dim3(256), 0, st, v);
  timing_after(st);
  return hipGetLastError();
}

}  // namespace sru
