// Matrix products of the SRU layer on the gfx950 matrix cores (MFMA).
//
// The forward projection of Sec. 3.1 (U = X [W; W_f; W_r]^T over all L*B
// tokens at once) and the two products of the backward pass (dX = dU W and
// dW = dU^T X) are one kernel template:
//     C[M,N] = sum_k A(m,k) B(n,k)
// with each operand either K-contiguous ("KC": row-major [rows, K]) or
// row-contiguous ("RC": [K, rows]), and stored as fp32 or bf16.  The loader
// stages a tile into LDS in the compute type:
//   * bf16 mode: bf16 operands are copied, fp32 ones rounded to bf16 (RNE,
//     v_cvt_pk_bf16_f32); v_mfma_f32_32x32x16_bf16 with fp32 accumulation;
//   * fp32 mode: v_mfma_f32_32x32x2_f32.
// LDS always holds a tile K-contiguous per row ([rows][BK + 16 bytes]), so a
// lane's MFMA fragment is one 16-byte LDS read.  An RC operand is transposed
// in registers on its way into LDS: a thread owns a block of k-rows x rows,
// and packs the k-run of each row (the fp32 -> bf16 pack of a (k, k+1) pair
// does the transposition; bf16 pairs are joined with v_perm_b32).
//
// Loads never branch and are never masked after the fact: a chunk past the
// end of K is loaded from an out-of-range buffer offset (the hardware returns
// zeros), and a row past the end of the operand is clamped to its last row
// (that row only feeds outputs the epilogue discards), so the compiler issues
// every global load of a K step back to back and waits once.
// Pipelining: two LDS buffers; the global loads of tile k+1 are in flight
// while the MFMAs consume tile k; one barrier per K step.
// Work mapping: one workgroup per output tile (and K split).  Workgroups are
// dispatched round-robin over the 8 XCDs, so the linear tile order is
// remapped to give each XCD a contiguous run of tiles that share A panels in
// its own L2.
#include <algorithm>
#include <type_traits>

#include "sru_device.h"
#include "sru_internal.h"


namespace sru {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

template <int BM_, int BN_, int BK_, int WAVES_M_, int WAVES_N_, bool BF16_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_;
  static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int THREADS = WAVES_M * WAVES_N * 64;
  static constexpr bool BF16 = BF16_;
  static constexpr int ESZ = BF16 ? 2 : 4;    // bytes per LDS element
  static constexpr int KPACK = 16 / ESZ;       // elements per 16-byte fragment read
  static constexpr int KSLAB = 2 * KPACK;      // k covered by one fragment pair
  static constexpr int LDK = BK + KPACK;       // LDS row stride (16 bytes of padding)
  static constexpr int A_BYTES = BM * LDK * ESZ;
  static constexpr int B_BYTES = BN * LDK * ESZ;
  static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  static_assert(BK % KSLAB == 0, "BK must hold whole fragment pairs");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile is a grid of 32x32 MFMA tiles");
};

// bf16: tiles 256x256x64, 4 waves of 128x128.  fp32: 128x128x32, 4 waves of 64x64.
using CfgBF16 = Cfg<256, 256, 64, 2, 2, true>;
using CfgF32 = Cfg<128, 128, 32, 2, 2, false>;

// Source element types: fp32, or bf16 carried as raw 16-bit patterns.
template <class S> struct Src;
template <> struct Src<float> { static constexpr int E = 4; };     // elements per 16 bytes
template <> struct Src<uint16_t> { static constexpr int E = 8; };

__device__ __forceinline__ unsigned pack_bf16(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;  // RNE (v_cvt_pk_bf16_f32)
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(unsigned, v);
}

// Vector loads go through a buffer resource: the hardware returns zeros for
// any offset at or beyond its byte size, so an out-of-range chunk is loaded
// from the sentinel offset kOOB instead of being masked afterwards (no select
// on the loaded data, so nothing has to wait for it).  Operands must then be
// smaller than kOOB bytes; the launcher checks this.
constexpr unsigned kOOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, unsigned bytes) {
  // dword 3 = 0x00020000: 32-bit data format, the raw-buffer setting of gfx9 parts
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                           0x00020000);
}

// Resource for the bytes of an operand from `base` on (extent `bytes`),
// its range capped below kOOB so that sentinel offsets stay out of range.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t panel_rsrc(const void* p, long long base,
                                                             long long bytes) {
  return make_rsrc(static_cast<const unsigned char*>(p) + base,
                   (unsigned)min(bytes - base, (long long)kOOB - 1));
}

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// Element-wise variant for unaligned or ragged operands: element e is valid
// when e < valid.
template <class S>
__device__ __forceinline__ u32x4 load16_elems(const S* src, long long idx, int valid) {
  constexpr int E = Src<S>::E;
  S tmp[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool ok = e < valid;
    const S x = src[ok ? idx + e : 0];
    tmp[e] = ok ? x : S(0);
  }
  return __builtin_bit_cast(u32x4, tmp);
}

// Element e of a 16-byte chunk as fp32.  The element is copied to a scalar
// first: a bit cast applied directly to a vector-element lvalue reads element
// 0 with this compiler.
__device__ __forceinline__ float f32_of(const u32x4& v, int e) {
  const unsigned x = v[e];
  return __builtin_bit_cast(float, x);
}

// ---- loader for a K-contiguous operand: element (r, k) at src[r*ld + k]
template <class C, int R, class S, bool VEC>
struct LoaderKC {
  static constexpr int E = Src<S>::E;
  static constexpr int CPR = C::BK / E;  // 16-byte chunks per row
  static constexpr int PER = R * CPR / C::THREADS;
  static_assert(R * CPR % C::THREADS == 0, "tile must split evenly over the threads");
  static_assert(C::BF16 || std::is_same<S, float>::value, "fp32 compute takes fp32 operands");
  u32x4 v[PER];
  unsigned base[PER];  // VEC: byte offset of the chunk at k = 0 (rows clamped)

  __device__ __forceinline__ void init(long long ld, int r0, int rows, int tid) {
    if constexpr (VEC) {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int c = tid + i * C::THREADS;
        const int r = min(r0 + c / CPR, rows - 1);
        const int k = (c % CPR) * E;
        base[i] = (unsigned)(((long long)r * ld + k) * sizeof(S));
      }
    }
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, const S* src, long long ld,
                                       int r0, int rows, int k0, int K, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * C::THREADS;
      const int k = k0 + (c % CPR) * E;
      if constexpr (VEC) {
        const unsigned off = k < K ? base[i] + (unsigned)(k0 * sizeof(S)) : kOOB;
        v[i] = buf_load16(rs, off);
      } else {
        const int r = r0 + c / CPR;
        v[i] = load16_elems(src, (long long)r * ld + k, r < rows ? K - k : 0);
      }
    }
  }
  __device__ __forceinline__ void store(unsigned char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * C::THREADS;
      const int r = c / CPR;
      const int k = (c % CPR) * E;
      unsigned char* dst = lds + (r * C::LDK + k) * C::ESZ;
      if constexpr (C::BF16 && std::is_same<S, float>::value) {
        u32x2 w;
        w[0] = pack_bf16(f32_of(v[i], 0), f32_of(v[i], 1));
        w[1] = pack_bf16(f32_of(v[i], 2), f32_of(v[i], 3));
        *reinterpret_cast<u32x2*>(dst) = w;
      } else {
        *reinterpret_cast<u32x4*>(dst) = v[i];
      }
    }
  }
};

// ---- loader for a row-contiguous operand: element (r, k) at src[k*ld + r].
// A thread owns KB k-rows x E rows (one 16-byte chunk per k-row) and writes
// E LDS rows of KB elements (16 bytes each).  Consecutive threads take
// consecutive k-blocks of the same rows, so their LDS writes fall in
// distinct banks.
template <class C, int R, class S, bool VEC>
struct LoaderRC {
  static constexpr int E = Src<S>::E;              // rows per chunk
  static constexpr int KB = C::BF16 ? 8 : 4;       // k per LDS write (16 bytes)
  static constexpr int NKB = C::BK / KB;
  static constexpr int NMB = (R / E) * NKB;
  static constexpr int PER = NMB / C::THREADS;
  static_assert(NMB % C::THREADS == 0, "tile must split evenly over the threads");
  static_assert(C::BF16 || std::is_same<S, float>::value, "fp32 compute takes fp32 operands");
  u32x4 v[PER][KB];
  unsigned base[PER];  // VEC: byte offset of k-row kb*KB at k0 = 0 (rows clamped)

  __device__ __forceinline__ void init(long long ld, int r0, int rows, int tid) {
    if constexpr (VEC) {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int c = tid + i * C::THREADS;
        const int kb = c % NKB;
        // rows is a multiple of E here, so a clamped chunk stays whole
        const int r = min(r0 + (c / NKB) * E, rows - E);
        base[i] = (unsigned)(((long long)kb * KB * ld + r) * sizeof(S));
      }
    }
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, const S* src, long long ld,
                                       int r0, int rows, int k0, int K, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * C::THREADS;
      const int kb = c % NKB;
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) {
        const int k = k0 + kb * KB + kk;
        if constexpr (VEC) {
          const unsigned off =
              k < K ? base[i] + (unsigned)(((long long)k0 + kk) * ld * sizeof(S)) : kOOB;
          v[i][kk] = buf_load16(rs, off);
        } else {
          const int r = r0 + (c / NKB) * E;
          v[i][kk] = load16_elems(src, (long long)k * ld + r, k < K ? rows - r : 0);
        }
      }
    }
  }
  __device__ __forceinline__ void store(unsigned char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * C::THREADS;
      const int kb = c % NKB;
      const int r = (c / NKB) * E;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        unsigned char* dst = lds + ((r + e) * C::LDK + kb * KB) * C::ESZ;
        u32x4 w;
        if constexpr (!C::BF16) {
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) w[kk] = v[i][kk][e];
        } else if constexpr (std::is_same<S, float>::value) {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            w[j] = pack_bf16(f32_of(v[i][2 * j], e), f32_of(v[i][2 * j + 1], e));
        } else {
          // element e of chunk kk is half (e % 2) of dword e / 2; pair chunks
          // (2j, 2j+1) into dword j: low half from k = 2j, high from 2j+1.
          const unsigned sel = (e & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            w[j] = __builtin_amdgcn_perm(v[i][2 * j + 1][e >> 1], v[i][2 * j][e >> 1], sel);
        }
        *reinterpret_cast<u32x4*>(dst) = w;
      }
    }
  }
};

template <class C, int R, bool KC, class S, bool VEC>
using Loader =
    typename std::conditional<KC, LoaderKC<C, R, S, VEC>, LoaderRC<C, R, S, VEC>>::type;

struct KernelArgs {
  const void* A;
  const void* B;
  // operand extents in bytes: the register-staged kernels address whole
  // operands through buffer resources (VEC: extents below kOOB); the direct
  // kernel bases its resources at each workgroup's panels
  long long a_bytes, b_bytes;
  float* out;               // C, or the split partials
  long long lda, ldb, ldo;
  long long split_stride;   // elements between split outputs (0 when splits == 1)
  int M, N, K;
  int k_per_split;          // multiple of BK
  int tiles_m, tiles_n, splits;
  const float* add;
  long long add_ld, add_off;
  int add_count;
  int vec_out;  // output (and addend) rows allow 16-byte accesses: see write_tile_rows
  uint16_t* outb;  // bf16 copy of the result (direct kernel, OB), out may be nullptr
  long long ldob;
};

// Epilogue shared by the kernels.  32x32 accumulator layout: element e of
// lane l is row 8*(e/4) + 4*(l/32) + e%4, column l%32 of the MFMA tile.
// ADD = number of addend tensors (0..2, see KernelArgs).  For each MFMA
// tile the addend loads are issued together (rows and columns clamped into
// range, so no branch separates them) before the stores.
template <class C, int ADD>
__device__ __forceinline__ void write_tile_add(const KernelArgs& g,
                                               const floatx16 (&acc)[C::FM][C::FN], int m0,
                                               int n0, int wm0, int wn0, int lane, int split) {
  float* out = g.out + (long long)split * g.split_stride;
  const bool full = m0 + C::BM <= g.M && n0 + C::BN <= g.N;
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int n = n0 + wn0 + j * 32 + (lane & 31);
      const int mb = m0 + wm0 + i * 32 + (lane >> 5) * 4;
      float v[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] = acc[i][j][e];
      if constexpr (ADD > 0) {
        const int nc = min(n, g.N - 1);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int mc = min(mb + (e >> 2) * 8 + (e & 3), g.M - 1);
          const float* ar = g.add + (long long)mc * g.add_ld + nc;
          v[e] += ar[0];
          if constexpr (ADD > 1) v[e] += ar[g.add_off];
        }
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = mb + (e >> 2) * 8 + (e & 3);
        if (full || (m < g.M && n < g.N)) out[(long long)m * g.ldo + n] = v[e];
      }
    }
}

// Epilogue of the direct kernel, whose MFMAs take the B-operand fragment
// first and so accumulate the transposed tile: element e of lane l is row
// l%32, column 8*(e/4) + 4*(l/32) + e%4 of the 32x32 output tile.  Each
// group of four elements is four consecutive columns of one row, written
// (and its addend read) as one 16-byte access when the tile lies wholly
// inside the output and vec_out holds (16-byte aligned rows).
// OB: also (or, when g.out is null, only) write the bf16 rounding of the
// result to g.outb (four columns as one 8-byte store); no addend then.
template <class C, int ADD, bool OB = false>
__device__ __forceinline__ void write_tile_rows(const KernelArgs& g,
                                                const floatx16 (&acc)[C::FM][C::FN], int m0,
                                                int n0, int wm0, int wn0, int lane, int split) {
  static_assert(!OB || ADD == 0, "the bf16 result takes no addend");
  float* out = g.out ? g.out + (long long)split * g.split_stride : nullptr;
  const int cl = 4 * (lane >> 5);
  if constexpr (OB) {
    if (g.vec_out && m0 + C::BM <= g.M && n0 + C::BN <= g.N) {
#pragma unroll
      for (int i = 0; i < C::FM; ++i) {
        const int m = m0 + wm0 + i * 32 + (lane & 31);
        const long long col = n0 + wn0 + cl;
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float a0 = acc[i][j][4 * q], a1 = acc[i][j][4 * q + 1];
            const float a2 = acc[i][j][4 * q + 2], a3 = acc[i][j][4 * q + 3];
            u32x2 w;
            w[0] = pack_bf16(a0, a1);
            w[1] = pack_bf16(a2, a3);
            *reinterpret_cast<u32x2*>(g.outb + m * g.ldob + col + j * 32 + 8 * q) = w;
            if (out) {
              floatx4 v;
              v[0] = a0;
              v[1] = a1;
              v[2] = a2;
              v[3] = a3;
              *reinterpret_cast<floatx4*>(out + m * g.ldo + col + j * 32 + 8 * q) = v;
            }
          }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int j = 0; j < C::FN; ++j) {
        const int m = m0 + wm0 + i * 32 + (lane & 31);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int n = n0 + wn0 + j * 32 + 8 * (e >> 2) + cl + (e & 3);
          if (m < g.M && n < g.N) {
            const float v = acc[i][j][e];
            g.outb[(long long)m * g.ldob + n] = __builtin_bit_cast(uint16_t, (__bf16)v);
            if (out) out[(long long)m * g.ldo + n] = v;
          }
        }
      }
    return;
  }
  if constexpr (ADD > 0) {
    if (g.vec_out && m0 + C::BM <= g.M && n0 + C::BN <= g.N) {
      // Addends of one row of MFMA tiles are loaded one row ahead, before
      // the stores of the current row: the loads never wait behind stores
      // (which the compiler would otherwise keep in program order, since
      // it cannot rule out aliasing), so a wave has one exposed memory
      // round trip instead of one per MFMA tile.
      constexpr int NA = C::FN * 4;  // 16-byte addend chunks per tile row
      floatx4 buf[2][ADD][NA];
      auto load_row = [&](int i, floatx4 (&a)[ADD][NA]) {
        const int m = m0 + wm0 + i * 32 + (lane & 31);
        const float* arow = g.add + (long long)m * g.add_ld + n0 + wn0 + cl;
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            a[0][j * 4 + q] = *reinterpret_cast<const floatx4*>(arow + j * 32 + 8 * q);
            if constexpr (ADD > 1)
              a[1][j * 4 + q] =
                  *reinterpret_cast<const floatx4*>(arow + g.add_off + j * 32 + 8 * q);
          }
      };
      load_row(0, buf[0]);
#pragma unroll
      for (int i = 0; i < C::FM; ++i) {
        floatx4 v[NA];
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[j * 4 + q][e] = acc[i][j][4 * q + e];
            v[j * 4 + q] += buf[i & 1][0][j * 4 + q];
            if constexpr (ADD > 1) v[j * 4 + q] += buf[i & 1][1][j * 4 + q];
          }
        if (i + 1 < C::FM) load_row(i + 1, buf[(i + 1) & 1]);
        const int m = m0 + wm0 + i * 32 + (lane & 31);
        float* orow = out + (long long)m * g.ldo + n0 + wn0 + cl;
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *reinterpret_cast<floatx4*>(orow + j * 32 + 8 * q) = v[j * 4 + q];
      }
      return;
    }
  }
  if (ADD == 0 && g.vec_out && m0 + C::BM <= g.M && n0 + C::BN <= g.N) {
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
      const int m = m0 + wm0 + i * 32 + (lane & 31);
      float* orow = out + (long long)m * g.ldo + n0 + wn0 + cl;
      const float* arow = ADD > 0 ? g.add + (long long)m * g.add_ld + n0 + wn0 + cl : nullptr;
#pragma unroll
      for (int j = 0; j < C::FN; ++j) {
        floatx4 v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e) v[q][e] = acc[i][j][4 * q + e];
        if constexpr (ADD > 0) {
          floatx4 a0[4], a1[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            a0[q] = *reinterpret_cast<const floatx4*>(arow + j * 32 + 8 * q);
            if constexpr (ADD > 1)
              a1[q] = *reinterpret_cast<const floatx4*>(arow + g.add_off + j * 32 + 8 * q);
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            v[q] += a0[q];
            if constexpr (ADD > 1) v[q] += a1[q];
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) *reinterpret_cast<floatx4*>(orow + j * 32 + 8 * q) = v[q];
      }
    }
    return;
  }
  // edge tiles (or unaligned rows): element by element, inside the bounds
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int m = m0 + wm0 + i * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int n = n0 + wn0 + j * 32 + 8 * (e >> 2) + cl + (e & 3);
        if (m < g.M && n < g.N) {
          float v = acc[i][j][e];
          if constexpr (ADD > 0) {
            const float* ar = g.add + (long long)m * g.add_ld + n;
            v += ar[0];
            if constexpr (ADD > 1) v += ar[g.add_off];
          }
          out[(long long)m * g.ldo + n] = v;
        }
      }
    }
}

// fp32 epilogue of a whole tile through LDS.  The accumulator layout makes a
// direct store write 32 rows x 32 bytes; here each wave moves one row of
// MFMA tiles (32 x WN) at a time through its own LDS block and reads it back
// row by row, so that a store instruction writes 4 rows x 256 bytes, i.e.
// whole 128-byte lines, and the addends are read the same way.  The caller
// has ended every wave's reads of the operand stages (barrier).
constexpr int kStagePitch = 68;  // floats per staged row: 64 + 4 keeps 16-byte writes conflict-free
template <class C, int ADD>
__device__ __forceinline__ void write_tile_staged(const KernelArgs& g,
                                                  const floatx16 (&acc)[C::FM][C::FN],
                                                  unsigned char* smem, int m0, int n0, int wm0,
                                                  int wn0, int lane, int wave, int split) {
  static_assert(C::WN == 64 || C::WN == 96, "staged rows of 64 or 96 columns");
  float* out = g.out + (long long)split * g.split_stride;
  const int cl = 4 * (lane >> 5);
  if constexpr (C::WN == 96) {
    // 96-column wave blocks: rows of 24 16-byte chunks (pitch 100 floats, 4
    // past a multiple of 32 banks as for 64 columns), read back as 12 passes
    // of 64 consecutive chunks of the 32-row group (runs of 384 bytes)
    static_assert(ADD == 0, "the 96-column tiles serve products without an addend");
    constexpr int P = 100, CPR = 24;
    static_assert(C::WAVES * 32 * P * 4 <= C::LDS, "staging fits the operand stages");
    float* blk = reinterpret_cast<float*>(smem) + wave * 32 * P;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          floatx4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e];
          *reinterpret_cast<floatx4*>(blk + (lane & 31) * P + j * 32 + 8 * q + cl) = v;
        }
#pragma unroll
      for (int s = 0; s < 32 * CPR / 64; ++s) {
        const int ch = s * 64 + lane, r = ch / CPR, col = 4 * (ch % CPR);
        const long long mrow = m0 + wm0 + i * 32 + r;
        *reinterpret_cast<floatx4*>(out + mrow * g.ldo + n0 + wn0 + col) =
            *reinterpret_cast<const floatx4*>(blk + r * P + col);
      }
    }
    return;
  }
  static_assert(C::WAVES * 32 * kStagePitch * 4 <= C::LDS, "staging fits the operand stages");
  float* blk = reinterpret_cast<float*>(smem) + wave * 32 * kStagePitch;
  const int rr = lane >> 4, cc = 4 * (lane & 15);  // read-back: rows rr + 4 s, columns cc..cc+3
#pragma unroll
  for (int i = 0; i < C::FM; ++i) {
    const long long mrow = m0 + wm0 + i * 32 + rr;  // row of read-back s = 0
    floatx4 ad[ADD > 0 ? ADD : 1][8];
    if constexpr (ADD > 0) {
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const float* ar = g.add + (mrow + 4 * s) * g.add_ld + n0 + wn0 + cc;
        ad[0][s] = *reinterpret_cast<const floatx4*>(ar);
        if constexpr (ADD > 1) ad[1][s] = *reinterpret_cast<const floatx4*>(ar + g.add_off);
      }
    }
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        floatx4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e];
        *reinterpret_cast<floatx4*>(blk + (lane & 31) * kStagePitch + j * 32 + 8 * q + cl) = v;
      }
    // one wave's LDS accesses run in order: the reads below see the writes,
    // and the next row group's writes come after these reads
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      floatx4 v = *reinterpret_cast<const floatx4*>(blk + (rr + 4 * s) * kStagePitch + cc);
      if constexpr (ADD > 0) v += ad[0][s];
      if constexpr (ADD > 1) v += ad[1][s];
      *reinterpret_cast<floatx4*>(out + (mrow + 4 * s) * g.ldo + n0 + wn0 + cc) = v;
    }
  }
}

// XCD-aware remap of the linear workgroup id: workgroups are dispatched
// round-robin over the 8 XCDs; each XCD gets a contiguous run of tiles.
struct TileIdx {
  int split, tm, tn;
};
__device__ __forceinline__ TileIdx tile_of(const KernelArgs& g) {
  const int nwg = gridDim.x;
  const int w = blockIdx.x;
  const int q = nwg / 8, rmd = nwg % 8, x = w % 8;
  const int u = x * q + (x < rmd ? x : rmd) + w / 8;
  const int nt = g.tiles_m * g.tiles_n;
  TileIdx r;
  r.split = u / nt;
  const int t = u - r.split * nt;
  // tiles in groups of GM tile rows, column by column within a group: the
  // 32 tiles an XCD runs at once then span 4 A panels x 8 B panels instead
  // of 3 x 12 (gemm_u's 12 column tiles), fewer distinct panels in its L2
  // (measured: GM = 4 slightly ahead of 8, 16 behind)
  constexpr int GM = 4;
  const int gsz = GM * g.tiles_n;
  const int first = (t / gsz) * GM;
  const int rows = min(g.tiles_m - first, GM);
  const int tg = t - (t / gsz) * gsz;
  r.tm = first + tg % rows;
  r.tn = tg / rows;
  return r;
}

template <class C, bool A_KC, bool B_KC, class SA, class SB, bool VEC, int ADD>
__global__ __launch_bounds__(C::THREADS) void gemm_kernel(KernelArgs g) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * C::STAGE_BYTES];

  const TileIdx ti = tile_of(g);
  const int split = ti.split;
  const int m0 = ti.tm * C::BM;
  const int n0 = ti.tn * C::BN;
  const int kbeg = split * g.k_per_split;
  const int kend = min(g.K, kbeg + g.k_per_split);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm0 = (wave / C::WAVES_N) * C::WM;
  const int wn0 = (wave % C::WAVES_N) * C::WN;
  const SA* A = static_cast<const SA*>(g.A);
  const SB* B = static_cast<const SB*>(g.B);

  Loader<C, C::BM, A_KC, SA, VEC> la;
  Loader<C, C::BN, B_KC, SB, VEC> lb;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, (unsigned)g.a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(B, (unsigned)g.b_bytes);
  la.init(g.lda, m0, g.M, tid);
  lb.init(g.ldb, n0, g.N, tid);

  floatx16 acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  la.load(ra, A, g.lda, m0, g.M, kbeg, kend, tid);
  lb.load(rb, B, g.ldb, n0, g.N, kbeg, kend, tid);
  la.store(smem, tid);
  lb.store(smem + C::A_BYTES, tid);
  __syncthreads();

  int cur = 0;
  for (int k0 = kbeg; k0 < kend; k0 += C::BK) {
    const bool next = k0 + C::BK < kend;
    if (next) {
      la.load(ra, A, g.lda, m0, g.M, k0 + C::BK, kend, tid);
      lb.load(rb, B, g.ldb, n0, g.N, k0 + C::BK, kend, tid);
    }
    const unsigned char* As = smem + cur * C::STAGE_BYTES;
    const unsigned char* Bs = As + C::A_BYTES;
#pragma unroll
    for (int ks = 0; ks < C::BK; ks += C::KSLAB) {
      const int koff = ks + (lane >> 5) * C::KPACK;
      floatx4 af[C::FM], bfr[C::FN];
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
        af[i] = *reinterpret_cast<const floatx4*>(
            As + ((wm0 + i * 32 + (lane & 31)) * C::LDK + koff) * C::ESZ);
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
        bfr[j] = *reinterpret_cast<const floatx4*>(
            Bs + ((wn0 + j * 32 + (lane & 31)) * C::LDK + koff) * C::ESZ);
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
          if constexpr (C::BF16) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, af[i]), __builtin_bit_cast(bf16x8, bfr[j]), acc[i][j],
                0, 0, 0);
          } else {
            // Lane group h = lane/32 holds k = koff..koff+3 of its row; MFMA e
            // takes element e, so the 4 MFMAs cover the 8 k of this slab once.
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i][e], bfr[j][e], acc[i][j], 0,
                                                               0, 0);
          }
        }
    }
    if (next) {
      unsigned char* nb = smem + (cur ^ 1) * C::STAGE_BYTES;
      la.store(nb, tid);
      lb.store(nb + C::A_BYTES, tid);
    }
    __syncthreads();
    cur ^= 1;
  }

  write_tile_add<C, ADD>(g, acc, m0, n0, wm0, wn0, lane, split);
}

// ---------------------------------------------------------------------------
// bf16 x bf16 products with global -> LDS loads that bypass registers.
// Buffer loads with the LDS flag write each lane's 16 bytes straight into
// LDS at (wave-uniform base + 16 * lane); a ring of STAGES tiles lets the
// loads run STAGES-1 K steps ahead of the MFMAs at no register cost.  Both
// operands have the same layout, selected by RC:
//
// K-contiguous (RC = false; U = X W^T and dX = dU W as dU (W^T)^T):
//   row r of a tile holds BK k (2*BK bytes) at r*2*BK, its 16-byte k-chunks
//   permuted as slot = chunk ^ swz(r), which keeps the 16 rows of one
//   ds_read_b128 phase on distinct banks.  BK = 64 makes each row one whole
//   128-byte line of the operand: a wave load (8 rows, lane l: row l/8,
//   slot l%8) then touches 8 lines instead of 16 half lines, which is what
//   bounds the load rate.  A fragment is one ds_read_b128.
// Row-contiguous (RC = true; dW = dU^T X, both operands [K, rows]):
//   the tile is kept as loaded, k-row s at s*2R bytes (R rows of bf16), its
//   R/8 16-byte row-chunks permuted as slot = chunk ^ 4*(s & 3).  A wave
//   load fills 512/R k-rows.  A fragment (8 consecutive k of one row) is two
//   ds_read_b64_tr_b16: within each group of 16 lanes, input lane 4s+q names
//   k-row s, rows 4q..4q+3 of the group's 16 rows, and output lane i
//   receives that k-run of row i.  A k-row is a multiple of 256 bytes, so
//   its slot p sits on banks 4p..4p+3 (mod 64) whatever s is; the two groups
//   of a half wave read chunks c..c+3 (c a multiple of 4) of the same four
//   k-rows, and the XOR by 4*(s & 3) puts those 16 chunks on 16 distinct
//   slots mod 16, i.e. all 64 banks once.  (An XOR by 2*(s & 3) put both
//   groups on the same 8 slots: a two-way conflict on every read.)
//
// Each wave owns a 128 x 64 block of the tile (4 x 2 MFMA tiles of 32 x 32,
// 128 accumulator registers per lane); two waves share each SIMD, so one's
// LDS reads and barrier waits hide behind the other's MFMAs.  A 256 x 256
// tile (8 waves) loads a third fewer bytes per flop than 256 x 128 (4
// waves, two workgroups per CU); the loads, not the MFMAs, bound the
// smaller tile.
template <int BM_, int BN_, int BK_, int WAVES_M_, int WAVES_N_, int STAGES_, int SA_ = STAGES_>
struct DCfg {
  // STAGES: slots of the B operand's ring; SA: slots of the A operand's
  // ring (STAGES or STAGES + 1: A then loads one K step further ahead)
  static constexpr int BM = BM_, BN = BN_, BK = BK_, STAGES = STAGES_, SA = SA_;
  static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_, WAVES = WAVES_M * WAVES_N;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int KSLAB = 16, SLABS = BK / KSLAB;
  static constexpr int A_OPB = BM * BK * 2, B_OPB = BN * BK * 2;  // bytes per stage
  static constexpr int STB = A_OPB + B_OPB;
  static constexpr int A_BPW = A_OPB / 1024 / WAVES, B_BPW = B_OPB / 1024 / WAVES;
  static constexpr int IPS = A_BPW + B_BPW;  // load instructions per stage per wave
  static constexpr int LDS = SA * A_OPB + STAGES * B_OPB;  // A slots, then B slots
  static constexpr int OCC = LDS <= 80 * 1024 ? 2 : 1;  // workgroups per CU
  static_assert(SA == STAGES || SA == STAGES + 1, "A ring depth");
  static_assert(BK == 32 || BK == 64, "k per stage");
  static_assert((WM == 128 && WN == 64) || (WM == 64 && (WN == 96 || WN == 128)), "wave block");
  static_assert(A_BPW * 1024 * WAVES == A_OPB && B_BPW * 1024 * WAVES == B_OPB,
                "whole 1 KiB load blocks per wave");
  static_assert(LDS <= 160 * 1024 && IPS * (SA - 1) < 64, "LDS and vmcnt");
};
using DirectTall = DCfg<256, 128, 32, 2, 2, 3>;  // 4 waves, 2 workgroups per CU
using DirectWide = DCfg<256, 256, 32, 2, 4, 4>;  // 8 waves, 1 workgroup per CU
using DirectLine = DCfg<256, 256, 64, 2, 4, 2>;  // 8 waves, whole-line loads
using DirectLineA3 = DCfg<256, 256, 64, 2, 4, 2, 3>;  // the same, A two K steps ahead (160 KiB)
using DirectNarrow = DCfg<256, 128, 64, 2, 2, 2, 3>;  // 4 waves, whole-line loads, half the columns
using DirectN96 = DCfg<256, 96, 64, 4, 1, 2, 3>;  // 4 waves of 64 x 96

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_t;
typedef __attribute__((address_space(3))) v4i16 lds_v4;

// s_waitcnt immediate waiting for vmcnt <= n only (expcnt 7, lgkmcnt 15)
constexpr int vm_wait(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }

// One operand's part of the direct loads: R tile rows, this wave's BPW
// 1 KiB blocks.  off: byte offset at k0 = 0 from the panel's base (init:
// row r0 of a K-contiguous operand, k-row kbase of a row-contiguous one, see
// issue; init_rows: the operand's start); kk: k (within a stage) of the
// lane's data; oob: out-of-range bit for rows past the end (RC).
template <int R, bool RC, int BPW, int BK>
struct DirectOperand {
  static constexpr int LPR = BK / 8;    // KC: 16-byte chunks (lanes) per row
  static constexpr int RPB = 64 / LPR;  // KC: rows per 1 KiB block
  unsigned off[BPW], oob[BPW];
  int kk[BPW];

  __device__ __forceinline__ static int swz(int r) {
    if constexpr (BK == 32) return ((r >> 1) ^ (r >> 3)) & 3;
    else return (r >> 1) & 7;
  }
  __device__ __forceinline__ void init(int wave, int lane, int r0, int rows, long long ld) {
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      const int blk = wave * BPW + j;
      if constexpr (!RC) {
        const int r = blk * RPB + lane / LPR;
        const int chunk = (lane % LPR) ^ swz(r);
        kk[j] = chunk * 8;
        off[j] = (unsigned)(((long long)(min(r0 + r, rows - 1) - r0) * ld + chunk * 8) * 2);
        oob[j] = 0;  // rows past the end are clamped: they feed discarded outputs
      } else {
        constexpr int CPK = R / 8;  // 16-byte chunks per k-row
        static_assert(CPK >= 16, "the k-row swizzle XORs chunk indices with up to 12");
        const int srow = blk * (512 / R) + lane / CPK;
        const int chunk = (lane % CPK) ^ (4 * (srow & 3));
        const int r = r0 + chunk * 8;
        kk[j] = srow;
        off[j] = (unsigned)(((long long)srow * ld + min(r, rows - 8)) * 2);
        oob[j] = (unsigned)(r >= rows) << 31;  // rows % 8 == 0: chunks are whole
      }
    }
  }
  // K-contiguous operand whose tile row r is row row_of(r) of the operand,
  // or a row of zeros where row_of(r) < 0 (no memory is read for it).
  template <class F>
  __device__ __forceinline__ void init_rows(int wave, int lane, F row_of, long long ld) {
    static_assert(!RC, "row maps are for K-contiguous operands");
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      const int blk = wave * BPW + j;
      const int r = blk * RPB + lane / LPR;
      const int chunk = (lane % LPR) ^ swz(r);
      const long long gr = row_of(r);
      kk[j] = chunk * 8;
      off[j] = gr >= 0 ? (unsigned)((gr * ld + chunk * 8) * 2) : 0u;
      oob[j] = gr >= 0 ? 0u : kOOB;
    }
  }
  // Loads of the stage at k0 (RC: k-rows from kbase on lie at the panel's
  // base; KC: the base holds k = 0).
  __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t rs, unsigned char* lds, int wave,
                                        int k0, int kend, long long ld, int kbase) const {
    const unsigned dk = RC ? (unsigned)((long long)(k0 - kbase) * ld * 2) : (unsigned)(k0 * 2);
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      // past the end of K: an out-of-range offset, for which the hardware
      // writes zeros
      const unsigned kob = (unsigned)(k0 + kk[j] >= kend) << 31;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_t*)(lds + (wave * BPW + j) * 1024), 16,
                                               (off[j] + dk) | kob | oob[j], 0, 0, 0);
    }
  }
  // 16-byte MFMA fragment: k-chunk c (8 k) of tile row `row`
  __device__ __forceinline__ static floatx4 frag(const unsigned char* base, int row, int c,
                                                 int lane) {
    if constexpr (!RC) {
      return *reinterpret_cast<const floatx4*>(base + row * (2 * BK) + ((c ^ swz(row)) << 4));
    } else {
      // this lane's role in its 16-lane group: k-row s, rows 4q..4q+3
      const int gl = lane & 15;
      const int r = (row & ~15) + 4 * (gl & 3);
      const int kr = c * 8 + (gl >> 2);
      auto addr = [&](int k) {
        return base + k * (2 * R) + (((r >> 3) ^ (4 * (k & 3))) << 4) + (r & 7) * 2;
      };
      const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(addr(kr)));
      const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4*)(addr(kr + 4)));
      floatx4 f;
      f[0] = __builtin_bit_cast(float, __builtin_shufflevector(lo, lo, 0, 1));
      f[1] = __builtin_bit_cast(float, __builtin_shufflevector(lo, lo, 2, 3));
      f[2] = __builtin_bit_cast(float, __builtin_shufflevector(hi, hi, 0, 1));
      f[3] = __builtin_bit_cast(float, __builtin_shufflevector(hi, hi, 2, 3));
      return f;
    }
  }
};

// The main loop of the direct products: the tile whose operand loads la and
// lb were set up, accumulated over k in [kbeg, kend) into acc.  TRANS: the
// MFMAs take B first, so acc holds the transposed tile (lane l: tile row
// l % 32 of each 32 x 32 block); else lane l holds tile column l % 32, rows
// 8 (e / 4) + 4 (l / 32) + e % 4 of element e.
template <class C, bool TRANS = true, class OpA, class OpB>
__device__ __forceinline__ void direct_mainloop(unsigned char* smem, const OpA& la,
                                                const OpB& lb, __amdgpu_buffer_rsrc_t ra,
                                                __amdgpu_buffer_rsrc_t rb, long long lda,
                                                long long ldb, int kbeg, int kend, int wave,
                                                int lane, int wm0, int wn0,
                                                floatx16 (&acc)[C::FM][C::FN]) {
  constexpr int STAGES = C::STAGES, SA = C::SA;
  constexpr bool ALEAD = SA > STAGES;  // A loads one K step further ahead than B
  const int nk = (kend - kbeg + C::BK - 1) / C::BK;
  auto a_slot = [&](int kt) { return smem + (kt % SA) * C::A_OPB; };
  auto b_slot = [&](int kt) { return smem + SA * C::A_OPB + (kt % STAGES) * C::B_OPB; };
  auto issue_a = [&](int kt) {
    la.issue(ra, a_slot(kt), wave, kbeg + kt * C::BK, kend, lda, kbeg);
  };
  auto issue_b = [&](int kt) {
    lb.issue(rb, b_slot(kt), wave, kbeg + kt * C::BK, kend, ldb, kbeg);
  };
  auto issue = [&](int kt) {
    issue_a(kt);
    issue_b(kt);
  };

#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue(s);
  // the A ring's extra slot: A of step STAGES - 1 goes out with the prologue
  if constexpr (ALEAD)
    if (STAGES - 1 < nk) issue_a(STAGES - 1);

  // Wait until this wave's part of stage kt has landed: the loads of later
  // stages (IPS instructions per stage per wave) may stay in flight.  With
  // the deeper A ring the loads go out in the order A(kt+1) ... B(kt) A(kt+1)
  // B(kt+1) A(kt+2), so only A of step kt + 1 may remain (STAGES == 2).
  auto wait_stage = [&](int kt) {
    if constexpr (ALEAD) {
      static_assert(STAGES == 2, "A lead with a 2-slot B ring");
      if (kt + 1 < nk) __builtin_amdgcn_s_waitcnt(vm_wait(C::A_BPW));
      else __builtin_amdgcn_s_waitcnt(vm_wait(0));
      return;
    }
    const int later = min(STAGES - 2, nk - 1 - kt);
    if constexpr (STAGES >= 4) {
      if (later >= 2) {
        __builtin_amdgcn_s_waitcnt(vm_wait(2 * C::IPS));
        return;
      }
    }
    if constexpr (STAGES >= 3) {
      if (later >= 1) {
        __builtin_amdgcn_s_waitcnt(vm_wait(C::IPS));
        return;
      }
    }
    __builtin_amdgcn_s_waitcnt(vm_wait(0));
  };
  // Workgroup barrier without the release fence of __syncthreads (which
  // would wait for every outstanding vector memory operation, i.e. drain the
  // prefetched stages): this wave's LDS reads are waited for explicitly, the
  // stage's loads by wait_stage, and the memory clobbers keep the compiler
  // from moving LDS accesses across it.
  auto barrier = [] {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0) only (vmcnt 63, expcnt 7)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  struct Frags {
    floatx4 a[C::FM], b[C::FN];
  };
  auto load_frags = [&](Frags& f, int kt, int sl) {
    const unsigned char* As = a_slot(kt);
    const unsigned char* Bs = b_slot(kt);
    const int c = 2 * sl + (lane >> 5);
#pragma unroll
    for (int i = 0; i < C::FM; ++i) f.a[i] = OpA::frag(As, wm0 + i * 32 + (lane & 31), c, lane);
#pragma unroll
    for (int j = 0; j < C::FN; ++j) f.b[j] = OpB::frag(Bs, wn0 + j * 32 + (lane & 31), c, lane);
  };
  auto mfmas = [&](const Frags& f) {
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
        acc[i][j] = TRANS ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                __builtin_bit_cast(bf16x8, f.b[j]),
                                __builtin_bit_cast(bf16x8, f.a[i]), acc[i][j], 0, 0, 0)
                          : __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                __builtin_bit_cast(bf16x8, f.a[i]),
                                __builtin_bit_cast(bf16x8, f.b[j]), acc[i][j], 0, 0, 0);
  };

  // Software pipeline over the SLABS fragment slabs (16 k each) of a stage:
  // a slab's fragments are read from LDS before the MFMAs of the previous
  // slab are issued (f[0] and f[1] alternate; SLABS is even, so slab 0 of
  // every stage is f[0]).  The barrier that publishes stage kt+1 sits before
  // the MFMAs of the last slab of stage kt; it also ends every wave's reads
  // of stage kt, which frees that slot for the loads issued at the top of
  // the next iteration.  The last stage is peeled off so that no branch
  // separates the reads of the next f[0] from the MFMAs of the last slab: at
  // a join the compiler would count those newer reads into the wait.  A
  // scheduling barrier after each slab's reads keeps the compiler from
  // sinking them next to the MFMAs that consume them.
  Frags f[2];
  if (nk > 0) {
    wait_stage(0);
    barrier();
    load_frags(f[0], 0, 0);
    for (int kt = 0; kt + 1 < nk; ++kt) {
      if constexpr (ALEAD) {
        // slots of stage kt-1, free: B of the next step, then A of the one after
        if (kt + 1 < nk) issue_b(kt + 1);
        if (kt + 2 < nk) issue_a(kt + 2);
      } else {
        if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1);  // slot of stage kt-1, free
      }
#pragma unroll
      for (int sl = 0; sl + 1 < C::SLABS; ++sl) {
        load_frags(f[(sl + 1) & 1], kt, sl + 1);
        __builtin_amdgcn_sched_barrier(0);  // reads of the next slab stay ahead
        mfmas(f[sl & 1]);
      }
      wait_stage(kt + 1);
      barrier();
      load_frags(f[0], kt + 1, 0);
      __builtin_amdgcn_sched_barrier(0);  // reads of the next slab stay ahead
      mfmas(f[1]);
    }
#pragma unroll
    for (int sl = 0; sl < C::SLABS; ++sl) {
      if (sl + 1 < C::SLABS) load_frags(f[(sl + 1) & 1], nk - 1, sl + 1);
      __builtin_amdgcn_sched_barrier(0);  // reads of the next slab stay ahead
      mfmas(f[sl & 1]);
    }
  }
}

template <class C, int ADD, bool A_RC, bool B_RC, bool OB>
__global__ __launch_bounds__(C::THREADS, C::OCC) void gemm_direct_kernel(KernelArgs g) {
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS];

  const TileIdx ti = tile_of(g);
  const int m0 = ti.tm * C::BM;
  const int n0 = ti.tn * C::BN;
  const int kbeg = ti.split * g.k_per_split;
  const int kend = min(g.K, kbeg + g.k_per_split);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm0 = (wave / C::WAVES_N) * C::WM;
  const int wn0 = (wave % C::WAVES_N) * C::WN;
  // Buffer resources based at this workgroup's panels: a K-contiguous
  // operand at the tile's first row, a row-contiguous one at the split's
  // first k-row.  The loaders' offsets count from there, so they stay below
  // kOOB however large the operand is (the plan bounds the panels).
  const __amdgpu_buffer_rsrc_t ra =
      panel_rsrc(g.A, 2LL * (A_RC ? kbeg : m0) * g.lda, g.a_bytes);
  const __amdgpu_buffer_rsrc_t rb =
      panel_rsrc(g.B, 2LL * (B_RC ? kbeg : n0) * g.ldb, g.b_bytes);

  using OpA = DirectOperand<C::BM, A_RC, C::A_BPW, C::BK>;
  using OpB = DirectOperand<C::BN, B_RC, C::B_BPW, C::BK>;
  OpA la;
  OpB lb;
  la.init(wave, lane, m0, g.M, g.lda);
  lb.init(wave, lane, n0, g.N, g.ldb);
  floatx16 acc[C::FM][C::FN];
  direct_mainloop<C>(smem, la, lb, ra, rb, g.lda, g.ldb, kbeg, kend, wave, lane, wm0, wn0,
                     acc);
  if constexpr (!OB) {
    if (g.vec_out && m0 + C::BM <= g.M && n0 + C::BN <= g.N) {
      __builtin_amdgcn_s_waitcnt(0xC07F);  // this wave's LDS reads (lgkmcnt 0)
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();  // every wave is done with the operand stages
      asm volatile("" ::: "memory");
      write_tile_staged<C, ADD>(g, acc, smem, m0, n0, wm0, wn0, lane, wave, ti.split);
      return;
    }
  }
  write_tile_rows<C, ADD, OB>(g, acc, m0, n0, wm0, wn0, lane, ti.split);
}

// ---- fused projection + forward scan (inference: neither U nor C kept) ----
// One workgroup per (direction, group of 64 hidden units, group of bb
// sequences), bb = 2, 4 or 8.  Per time block of 256 / bb steps it computes
// the tile of U whose 256 rows are the block's (step, sequence) pairs and
// whose 64 k columns are the k gate blocks of the 64 units (k = 4: block 3
// is the highway input x_hat; k = 3 reads x_t from X).  The MFMAs leave the
// tile untransposed on 64 x 32k wave blocks, and the operand rows are mapped
// so that a lane's accumulators are the scan's inputs: lane l of wave
// (wm, wn) holds column l % 32 of each of its k 32-column MFMA blocks, i.e.
// the gates of unit 64 g + 32 wn + l % 32, and rows of one sequence (l / 32
// picks one of the wave's two), 16 consecutive steps per 32-row block, so 32
// steps in all.  The lane then runs Eq. 1-4 over those steps from its own
// registers: U is neither written to memory nor staged.  A block's 256 / bb
// steps lie in 8 / bb waves (time chunks of 32 steps), which scan one after
// the other and hand c over through LDS; c carries over from block to block
// the same way.  The scan arithmetic is the forward scan kernel's, in the
// same order, so H equals the unfused path's bit for bit.
// 8 waves of 64 x 32k, A two K steps ahead (a type of its own per k: two
// kernels instantiating the main loop on one configuration type trip the
// host compilation pass)
template <int KB>
struct FusedCfg : DCfg<256, 64 * KB, 64, 4, 2, 2, 3> {};

template <bool B_>
struct BoolC {
  static constexpr bool value = B_;
};

template <int KB>
__global__ __launch_bounds__(512, 1) void proj_scan_fwd_kernel(FusedFwdArgs a) {
  using C = FusedCfg<KB>;
  static_assert(C::THREADS == 512, "8 waves");
  static_assert(C::FM == 2 && C::FN == KB, "a lane: 2 row blocks, one column block per gate");
  static_assert(C::WAVES_M == 4 && C::WAVES_N == 2, "wave rows and columns");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS];

  // workgroup -> (direction, unit group, sequence group); XCD-aware, so the
  // workgroups of one XCD share the Wcat rows of a unit group
  const int nwg = gridDim.x, w = blockIdx.x;
  const int q8 = nwg / 8, rmd = nwg % 8, x8 = w % 8;
  const int wu = x8 * q8 + (x8 < rmd ? x8 : rmd) + w / 8;
  const int bg = wu % a.nbgroups;
  const int dg = wu / a.nbgroups;
  const int dir = dg / a.ngroups, g = dg % a.ngroups;
  const int nchunk = 8 / a.bb;  // time chunks of 32 steps per tile
  const int b0 = bg * a.bb;
  const bool rev = a.direction == 1 || (a.direction == 2 && dir == 1);
  const int L = a.L, Bs = a.B, d = a.d;
  const long long nfeat = (long long)a.ndir * d;

  // wave -> (time chunk, sequence pair, column half wn): the waves of one
  // chunk are consecutive, so they sit on different SIMDs (with two chunks,
  // waves 0-3 scan the first and waves 4-7 the second)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave & 1;
  const int pairs = 4 / nchunk;
  const int q2 = (wave >> 1) / pairs;
  const int pair = (wave >> 1) % pairs;
  const int wm = pair * nchunk + q2;  // the wave's 64-row block of the tile
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(a.Xb, a.a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(a.Wb, a.b_bytes);
  using OpA = DirectOperand<C::BM, false, C::A_BPW, C::BK>;
  using OpB = DirectOperand<C::BN, false, C::B_BPW, C::BK>;
  // tile column 32 k cw + 32 gate + u: gate block `gate` of unit 64 g + 32 cw + u
  OpB lb;
  lb.init_rows(
      wave, lane,
      [&](int col) -> long long {
        const int cw = col / (32 * KB), gate = (col >> 5) % KB;
        return (long long)(dir * KB + gate) * d + g * 64 + cw * 32 + (col & 31);
      },
      a.d_in);
  // this lane's scan: sequence sb, unit 64 g + 32 wn + lane % 32, time chunk
  // q2 of every block; c carries over from block to block
  const int sb = b0 + 2 * pair + (lane >> 5);
  const bool live = sb < Bs;
  const int unit = g * 64 + wn * 32 + (lane & 31);
  const long long fidx = (long long)dir * d + unit;
  float vf = 0.f, vr = 0.f, bf = 0.f, br = 0.f, c = 0.f;
  if (live) {
    if (!a.linear) {
      vf = a.v_f[fidx];
      vr = a.v_r[fidx];
    }
    bf = a.b_f[fidx];
    br = a.b_r[fidx];
    c = a.c0 ? a.c0[(long long)sb * nfeat + fidx] : 0.f;
  }
  // gate parameters scaled by -log2(e), as in the forward scan
  const float vfs = vf * kNegLog2e, vrs = vr * kNegLog2e;
  const float bfs = bf * kNegLog2e, brs = br * kNegLog2e;
  const float alpha = a.alpha;
  const bool rn = a.reset_new != 0;
  auto barrier = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);  // this wave's LDS accesses (lgkmcnt 0) only
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  // hand-over of c between the waves of consecutive chunks, in LDS, which is
  // free between a block's product and the next block's
  float* cx = reinterpret_cast<float*>(smem) + (pair * C::WAVES_N + wn) * 64 + lane;

  const int TB = 32 * nchunk;  // steps per block
  const int nblk = (L + TB - 1) / TB;
  int prev = -1;  // the time chunk scanned last (-1: none yet)
  for (int ib = 0; ib < nblk; ++ib) {
    const int t0 = (rev ? nblk - 1 - ib : ib) * TB;  // blocks in the direction's order
    // tile row r: wave row r / 64 = (sequence pair, time chunk); in a 32-row
    // block, row rr is sequence (rr / 4) % 2 of the pair at step
    // 4 (rr / 8) + rr % 4 of the block's 16 (the MFMA's row of element e)
    OpA la;
    la.init_rows(
        wave, lane,
        [&](int r) -> long long {
          const int wr = r >> 6, rr = r & 31;
          const int b = b0 + 2 * (wr / nchunk) + ((rr >> 2) & 1);
          const int t =
              t0 + 32 * (wr % nchunk) + 16 * ((r >> 5) & 1) + 4 * (rr >> 3) + (rr & 3);
          return t < L && b < Bs ? (long long)t * Bs + b : -1;
        },
        a.d_in);
    floatx16 acc[C::FM][C::FN];
    direct_mainloop<C, false>(smem, la, lb, ra, rb, a.d_in, a.d_in, 0, a.d_in, wave, lane,
                              wm * C::WM, wn * C::WN, acc);
    // k = 3: the highway input x_t of the wave's chunk, loaded now so that it
    // arrives while earlier chunks scan (steps past L re-read step L - 1)
    float xr[32];
    if constexpr (KB == 3) {
      if (live) {
        const float* xp = a.X + (long long)sb * a.d_in + unit;
        const long long xs = (long long)Bs * a.d_in;
#pragma unroll
        for (int tt = 0; tt < 32; ++tt) xr[tt] = xp[min(t0 + 32 * q2 + tt, L - 1) * xs];
      }
    }
    (void)xr;
    barrier();  // every wave is done with the operand stages

    // the 32 steps of the chunk from step tb (scan order: backward for a
    // reverse direction); steps at or past L are not computed.  A whole
    // chunk runs without a branch between its steps, so the compiler can
    // overlap one step's output (reset gate, h, stores) with the next step's
    // chain.
    auto scan_chunk = [&](auto rev_c, auto whole_c, auto hb_c, int tb) {
      constexpr bool RV = decltype(rev_c)::value, WHOLE = decltype(whole_c)::value;
      constexpr bool HB = decltype(hb_c)::value;
      const int nv = min(32, L - tb);
      // padding bits of the chunk's steps: lane u of each half reads step
      // tb + u of its sequence, and the ballot hands each half its 32 bits
      unsigned mbits = 0;
      if (a.mask) {
        const int tm = tb + (lane & 31);
        const bool pad = live && tm < L && a.mask[(long long)tm * Bs + sb] != 0;
        mbits = (unsigned)(__ballot(pad) >> (32 * (lane >> 5)));
      }
      if (!live) return;
      // output offset at the chunk's first step in scan order, moved one
      // step at a time (the empty asm keeps the compiler from precomputing
      // every step's offset)
      const int tt0 = RV ? (WHOLE ? 31 : nv - 1) : 0;
      long long o = ((long long)(tb + tt0) * Bs + sb) * nfeat + fidx;
      const long long dstep = (RV ? -1LL : 1LL) * Bs * nfeat;
      // A step carries c forward first (Eq. 1-2) and then finishes the
      // previous step's output (Eq. 3-4, the store), which no longer lies on
      // the chain from one c to the next.
      float p_cn = 0.f, p_rin = 0.f, p_zr = 0.f, p_xh = 0.f;
      bool p_pad = false, pend = false;
      auto emit = [&]() {
        const float r = sigmoid_scaled(fmaf(vrs, p_rin, p_zr));        // Eq. 3
        float h = fmaf(r, p_cn, (1.0f - r) * (alpha * p_xh));          // Eq. 4 (Sec. 3.2)
        h = p_pad ? 0.0f : h;
        __builtin_nontemporal_store(h, a.H + o);
        if constexpr (HB)
          __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (__bf16)h), a.Hb + o);
        o += dstep;
        asm volatile("" : "+v"(o));
      };
#pragma unroll
      for (int s = 0; s < 32; ++s) {
        const int tt = RV ? 31 - s : s;
        if (WHOLE || tt < nv) {
          const float u0 = acc[tt >> 4][0][tt & 15], u1 = acc[tt >> 4][1][tt & 15];
          const float u2 = acc[tt >> 4][2][tt & 15];
          float xh;
          if constexpr (KB == 4) xh = acc[tt >> 4][3][tt & 15];
          else xh = xr[tt];
          const float f = sigmoid_scaled(fmaf(vfs, c, fmaf(u1, kNegLog2e, bfs)));  // Eq. 1
          const float cn = fmaf(f, c, fmaf(-f, u0, u0));                           // Eq. 2
          const float rin = rn ? cn : c;
          const bool pad = (mbits >> tt) & 1u;
          c = pad ? c : cn;
          if (WHOLE ? s > 0 : pend) emit();
          p_cn = cn;
          p_rin = rin;
          p_zr = fmaf(u2, kNegLog2e, brs);
          p_xh = xh;
          p_pad = pad;
          pend = true;
        }
      }
      if (pend) emit();
    };
    // one instantiation per (direction of time, whole chunk, bf16 copy of H)
    auto scan_any = [&](auto rev_c, int tb) {
      const bool whole = L - tb >= 32;
      if (whole) {
        if (a.Hb) scan_chunk(rev_c, BoolC<true>{}, BoolC<true>{}, tb);
        else scan_chunk(rev_c, BoolC<true>{}, BoolC<false>{}, tb);
      } else {
        if (a.Hb) scan_chunk(rev_c, BoolC<false>{}, BoolC<true>{}, tb);
        else scan_chunk(rev_c, BoolC<false>{}, BoolC<false>{}, tb);
      }
    };
    for (int i = 0; i < nchunk; ++i) {
      const int q = rev ? nchunk - 1 - i : i;  // the chunk scanned now
      if (nchunk > 1 && prev >= 0) {
        // the wave of the previous chunk (of this block or the one before)
        // hands its c over
        if (q2 == prev) *cx = c;
        barrier();
        if (q2 == q) c = *cx;
      }
      if (q2 == q) {
        if (rev) scan_any(BoolC<true>{}, t0 + 32 * q);
        else scan_any(BoolC<false>{}, t0 + 32 * q);
      }
      prev = q;
    }
    barrier();  // the hand-over's LDS reads are done before the next block's loads
  }
  if (live && a.c_last && q2 == prev) a.c_last[(long long)sb * nfeat + fidx] = c;
}

template <class C, int ADD, bool A_RC, bool B_RC, bool OB = false>
void launch_direct(const KernelArgs& a, int nwg, hipStream_t st) {
  hipLaunchKernelGGL((gemm_direct_kernel<C, ADD, A_RC, B_RC, OB>), dim3(nwg), dim3(C::THREADS), 0, st,
                     a);
}

// Sum of split partials in split order, plus the optional addend.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part,
                                                            int splits, int M, int N,
                                                            float* C, long long ldc,
                                                            const float* add, long long add_ld,
                                                            long long add_off, int add_count) {
  const long long total = (long long)M * N;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (long long)gridDim.x * 256) {
    const int m = (int)(i / N);
    const int n = (int)(i - (long long)m * N);
    float s = 0.f;
    for (int z = 0; z < splits; ++z) s += part[(long long)z * total + i];
    if (add_count > 0) {
      const float* ar = add + (long long)m * add_ld + n;
      s += ar[0];
      if (add_count > 1) s += ar[add_off];
    }
    C[(long long)m * ldc + n] = s;
  }
}

// The same for rows of 16-byte aligned groups of 4 (N % 4 == 0): one group
// per thread, the partials read as 16-byte loads.  The per-element sum is
// the same sequence of additions, so the result is bit-identical.  Blocks
// from `main_blocks` on run the v/b sums of the backward pass instead
// (vb_sum_block: the same bits as their own launch).
__device__ __forceinline__ void split_sum4_block(const SplitSum& j, unsigned blk) {
  const long long total = (long long)j.M * j.N;
  const long long i = ((long long)blk * 256 + threadIdx.x) * 4;
  if (i >= total) return;
  const int m = (int)(i / j.N);
  const int n = (int)(i - (long long)m * j.N);
  floatx4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int z = 0; z < j.splits; ++z)
    s += *reinterpret_cast<const floatx4*>(j.part + z * total + i);
  if (j.add_count > 0) {
    const float* ar = j.add + (long long)m * j.add_ld + n;
    s += *reinterpret_cast<const floatx4*>(ar);
    if (j.add_count > 1) s += *reinterpret_cast<const floatx4*>(ar + j.add_off);
  }
  *reinterpret_cast<floatx4*>(j.C + (long long)m * j.ldc + n) = s;
}

// Blocks [0, n1) sum j1, [n1, n1 + n2) sum j2 (another product's deferred
// split sum: one launch instead of two), the rest the v/b sums.
__global__ __launch_bounds__(256) void splitk_reduce4_kernel(SplitSum j1, unsigned n1,
                                                             SplitSum j2, unsigned n2,
                                                             VbSum vb) {
  const unsigned b = blockIdx.x;
  if (b < n1) {
    split_sum4_block(j1, b);
  } else if (b < n1 + n2) {
    split_sum4_block(j2, b - n1);
  } else {
    __shared__ float red[256];
    vb_sum_block(vb.partial, vb.rows, vb.nfeat, vb.qlo, vb.out, b - n1 - n2, red);
  }
}

bool split_sum_vec(const SplitSum& j) {
  auto al16 = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  return j.N % 4 == 0 && j.ldc % 4 == 0 && al16(j.part) && al16(j.C) &&
         (j.add_count == 0 || (j.add_ld % 4 == 0 && j.add_off % 4 == 0 && al16(j.add)));
}

// Split sum j (if j.part), the deferred split sum `extra` (if extra.part) and
// the v/b sums (if vb.partial), in one launch where the rows allow 16-byte
// accesses.
hipError_t launch_splitk_reduce(const SplitSum& j, const SplitSum& extra, const VbSum& vb,
                                hipStream_t st) {
  const bool vec = (!j.part || split_sum_vec(j)) && (!extra.part || split_sum_vec(extra));
  if (!vec) {
    // one element per thread, each sum in its own launch
    for (const SplitSum* q : {&extra, &j}) {
      if (!q->part) continue;
      const long long total = (long long)q->M * q->N;
      const int grid = (int)std::min<long long>((total + 255) / 256, 8192);
      timing_before("splitk_reduce", st);
      hipLaunchKernelGGL(splitk_reduce_kernel, dim3(grid), dim3(256), 0, st, q->part, q->splits,
                         q->M, q->N, q->C, q->ldc, q->add, q->add_ld, q->add_off, q->add_count);
      timing_after(st);
      if (hipError_t e = hipGetLastError()) return e;
    }
    return vb.partial ? vb_sum_launch(vb, st) : hipSuccess;
  }
  auto blocks = [](const SplitSum& q) {
    return q.part ? (unsigned)(((long long)q.M * q.N / 4 + 255) / 256) : 0u;
  };
  const unsigned n1 = blocks(j), n2 = blocks(extra);
  const unsigned nv = vb.partial ? (unsigned)vb_sum_blocks(vb) : 0u;
  if (n1 + n2 + nv == 0) return hipSuccess;
  timing_before(n1 + n2 > 0 ? "splitk_reduce" : "reduce_vb", st);
  hipLaunchKernelGGL(splitk_reduce4_kernel, dim3(n1 + n2 + nv), dim3(256), 0, st, j, n1, extra,
                     n2, vb);
  timing_after(st);
  return hipGetLastError();
}

SplitSum split_sum_of(const GemmDesc& g, int splits) {
  SplitSum j;
  j.part = g.partials;
  j.splits = splits;
  j.M = g.M;
  j.N = g.N;
  j.C = g.C;
  j.ldc = g.ldc;
  j.add = g.add;
  j.add_ld = g.add_ld;
  j.add_off = g.add_off;
  j.add_count = g.add_count;
  return j;
}

// After a product: its split sum (unless deferred), the deferred split sum
// of an earlier product, and the v/b sums, in one launch.
hipError_t finish_product(const GemmDesc& g, int splits, hipStream_t st) {
  if (splits > 1 && g.defer_sum) return hipSuccess;
  const SplitSum own = splits > 1 ? split_sum_of(g, splits) : SplitSum{};
  return launch_splitk_reduce(own, g.extra, g.vb, st);
}

// fp32 -> bf16 conversions (RNE).  Plain copy: 8 elements per thread (two
// 16-byte loads, one 16-byte store).
__global__ __launch_bounds__(256) void to_bf16_kernel(const float* __restrict__ src,
                                                      long long n, uint16_t* __restrict__ dst) {
  const long long i = ((long long)blockIdx.x * 256 + threadIdx.x) * 8;
  if (i + 7 < n) {
    const floatx4 v0 = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(src + i));
    const floatx4 v1 = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(src + i + 4));
    u32x4 w;
    w[0] = pack_bf16(v0[0], v0[1]);
    w[1] = pack_bf16(v0[2], v0[3]);
    w[2] = pack_bf16(v1[0], v1[1]);
    w[3] = pack_bf16(v1[2], v1[3]);
    *reinterpret_cast<u32x4*>(dst + i) = w;
  } else {
    for (long long j = i; j < n; ++j)
      dst[j] = __builtin_bit_cast(uint16_t, (__bf16)src[j]);
  }
}

// Transposed: dst[c*rows + r] = bf16(src[r*cols + c]) through a 64x64 LDS tile.
// Source element as fp32: fp32 as is, bf16 (raw bits) widened exactly.
__device__ __forceinline__ float src_f32(float v) { return v; }
__device__ __forceinline__ float src_f32(uint16_t v) {
  return __builtin_bit_cast(float, (unsigned)v << 16);
}

template <class S>
__global__ __launch_bounds__(256) void to_bf16_t_kernel(const S* __restrict__ src, int rows,
                                                        int cols, uint16_t* __restrict__ dst) {
  __shared__ float tile[64][65];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    tile[i][tx] = (r < rows && c < cols) ? src_f32(src[(long long)r * cols + c]) : 0.f;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows)
      dst[(long long)c * rows + r] = __builtin_bit_cast(uint16_t, (__bf16)tile[tx][i]);
  }
}

// The same for whole 64 x 64 tiles with 16-byte accesses on both sides: each
// lane loads 16 bytes of a source row (4 fp32 or 8 bf16 elements) into the
// LDS tile, then packs 8 elements of a tile column into one 16-byte segment
// of an output row.  With the row pitch of 65 floats both the row writes and
// the column reads of the tile hit 64 distinct banks.
template <class S>
__global__ __launch_bounds__(256) void to_bf16_t_tiled_kernel(const S* __restrict__ src, int rows,
                                                              int cols, uint16_t* __restrict__ dst) {
  __shared__ float tile[64][65];
  constexpr int E = 16 / (int)sizeof(S);  // source elements per 16-byte load
  constexpr int TPR = 64 / E;             // lanes per tile row
  constexpr int RPR = 256 / TPR;          // tile rows per pass
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int t = threadIdx.x;
  const int lc = (t % TPR) * E;
  for (int i = t / TPR; i < 64; i += RPR) {
    const S* row = src + (long long)(r0 + i) * cols + c0 + lc;
    if constexpr (sizeof(S) == 4) {
      // loaded as floats: a bit cast of a vector element would read element 0
      const floatx4 v = *reinterpret_cast<const floatx4*>(row);
#pragma unroll
      for (int w = 0; w < 4; ++w) tile[i][lc + w] = v[w];
    } else {
      const u32x4 v = *reinterpret_cast<const u32x4*>(row);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const unsigned x = v[w];
        tile[i][lc + 2 * w] = __builtin_bit_cast(float, x << 16);
        tile[i][lc + 2 * w + 1] = __builtin_bit_cast(float, x & 0xFFFF0000u);
      }
    }
  }
  __syncthreads();
  const int q = t & 7;  // 8-element segment of the output row
  for (int c = t >> 3; c < 64; c += 32) {
    u32x4 w;
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = pack_bf16(tile[8 * q + 2 * j][c], tile[8 * q + 2 * j + 1][c]);
    *reinterpret_cast<u32x4*>(dst + (long long)(c0 + c) * rows + r0 + 8 * q) = w;
  }
}

template <class C>
int splits_for(const GemmDesc& g) {
  const int tiles = ((g.M + C::BM - 1) / C::BM) * ((g.N + C::BN - 1) / C::BN);
  // The K = tokens product (TN) is split.  A K-contiguous one is split only
  // on request and only when its tiles fill at most a quarter of the CUs:
  // the 32 tiles of the two-layer d = 256 stack's dX (K = 768) take 21 us
  // split six ways plus 6 us for the split sum, instead of 66 us; at 100-200
  // tiles the partials' extra pass costs what the split saves.
  if (g.a_kc && (!g.kc_split || tiles > 64)) return 1;
  const int kt = (g.K + C::BK - 1) / C::BK;  // K steps
  int s = (2 * 256 + tiles - 1) / tiles;     // aim for two workgroups per CU
  // fp32 accumulation chains stay short (<= 2048 terms per split)
  if (!C::BF16) s = max(s, (g.K + 2047) / 2048);
  s = min(s, max(1, kt / 4));                // at least 4 K steps per split
  return max(1, min(s, 64));
}

// Vector (buffer) loads need 16-byte aligned chunks that are either wholly
// inside or wholly outside the operand, i.e. the contiguous extent (K for KC,
// the row count for RC) and the leading dimension are multiples of a chunk,
// and an operand smaller than the out-of-range sentinel.
template <class S>
bool whole_chunks(const void* p, long long ld, int contiguous_extent) {
  constexpr int E = Src<S>::E;
  return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % E == 0 && contiguous_extent % E == 0;
}
template <class S>
bool vec_ok(const void* p, long long ld, int contiguous_extent, long long bytes) {
  return whole_chunks<S>(p, ld, contiguous_extent) && bytes > 0 && bytes < (long long)kOOB;
}

template <class C, bool A_KC, bool B_KC, class SA, class SB, bool VEC>
void launch_staged(const KernelArgs& a, int nwg, hipStream_t st) {
  if (a.add_count == 2)
    hipLaunchKernelGGL((gemm_kernel<C, A_KC, B_KC, SA, SB, VEC, 2>), dim3(nwg), dim3(C::THREADS), 0,
                       st, a);
  else if (a.add_count == 1)
    hipLaunchKernelGGL((gemm_kernel<C, A_KC, B_KC, SA, SB, VEC, 1>), dim3(nwg), dim3(C::THREADS), 0,
                       st, a);
  else
    hipLaunchKernelGGL((gemm_kernel<C, A_KC, B_KC, SA, SB, VEC, 0>), dim3(nwg), dim3(C::THREADS), 0,
                       st, a);
}

template <class C, bool A_KC, bool B_KC, class SA, class SB>
hipError_t launch_cfg(const GemmDesc& g, hipStream_t st) {
  const int splits = splits_for<C>(g);
  const int kt = (g.K + C::BK - 1) / C::BK;
  const int kps = ((kt + splits - 1) / splits) * C::BK;
  KernelArgs a;
  a.A = g.A;
  a.B = g.B;
  a.lda = g.lda;
  a.ldb = g.ldb;
  a.M = g.M;
  a.N = g.N;
  a.K = g.K;
  a.k_per_split = kps;
  a.tiles_m = (g.M + C::BM - 1) / C::BM;
  a.tiles_n = (g.N + C::BN - 1) / C::BN;
  // the real number of splits after rounding kps up to whole K steps
  a.splits = (g.K + kps - 1) / kps;
  if (a.splits > 1) {
    a.out = g.partials;
    a.ldo = g.N;
    a.split_stride = (long long)g.M * g.N;
    a.add = nullptr;
    a.add_count = 0;
    a.add_ld = a.add_off = 0;
  } else {
    a.out = g.C;
    a.ldo = g.ldc;
    a.split_stride = 0;
    a.add = g.add;
    a.add_count = g.add_count;
    a.add_ld = g.add_ld;
    a.add_off = g.add_off;
  }
  const int nwg = a.tiles_m * a.tiles_n * a.splits;
  // operand extents in bytes: rows x ld (KC) or K x ld (RC), last row exact
  const long long a_bytes =
      (long long)sizeof(SA) * (A_KC ? (long long)(g.M - 1) * g.lda + g.K
                                    : (long long)(g.K - 1) * g.lda + g.M);
  const long long b_bytes =
      (long long)sizeof(SB) * (B_KC ? (long long)(g.N - 1) * g.ldb + g.K
                                    : (long long)(g.K - 1) * g.ldb + g.N);
  const bool vec = vec_ok<SA>(g.A, g.lda, A_KC ? g.K : g.M, a_bytes) &&
                   vec_ok<SB>(g.B, g.ldb, B_KC ? g.K : g.N, b_bytes);
  a.a_bytes = vec ? a_bytes : 0;
  a.b_bytes = vec ? b_bytes : 0;
  timing_before(g.label ? g.label : !g.b_kc ? (g.a_kc ? "gemm_nn" : "gemm_tn") : "gemm_nt", st);
  if (vec)
    launch_staged<C, A_KC, B_KC, SA, SB, true>(a, nwg, st);
  else
    launch_staged<C, A_KC, B_KC, SA, SB, false>(a, nwg, st);
  timing_after(st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return finish_product(g, a.splits, st);
}

// ---- the direct path: plan (shared by workspace sizing and launch) ----
long long operand_bytes(bool kc, int rows, int K, long long ld, int esz) {
  return (long long)esz * (kc ? (long long)(rows - 1) * ld + K : (long long)(K - 1) * ld + rows);
}

// The direct kernel addresses each operand from its workgroup's panel (a
// tile's 256 rows of a K-contiguous operand, a split's k-rows of a
// row-contiguous one) with 32-bit offsets below kOOB.  Bytes a panel spans:
long long panel_bytes(bool kc, int rows, int K, long long ld, long long k_rows) {
  return 2 * (kc ? (long long)(min(rows, 256) - 1) * ld + K : (k_rows - 1) * ld + rows);
}
// The largest K range (whole 64-k stages) whose row-contiguous panel fits;
// 0 if not even one stage does.
long long rc_max_k(int rows, long long ld) {
  const long long room = (long long)kOOB - 1 - 2LL * rows;  // bytes for (k_rows - 1) * 2 ld
  if (room < 0) return 0;
  return ((room / (2 * ld) + 1) / 64) * 64;
}
bool split_allowed(const GemmDesc& g) { return !g.Cb && (!g.a_kc || g.kc_split); }

// bf16 x bf16 operands whose 16-byte chunks are whole (the contiguous
// extent and leading dimension are multiples of 8 elements) and whose
// panels fit the 32-bit offsets: a K-contiguous operand's 256 rows, a
// row-contiguous one's whole K when the product is not split, else one
// 64-k stage (the split count then keeps each split's panel in range, see
// direct_splits_cfg).  Layouts: both K-contiguous, both row-contiguous, or A
// K-contiguous with B row-contiguous.
bool direct_ok(const GemmDesc& g) {
  if (!g.bf16 || !g.a_bf16 || !g.b_bf16 || (!g.a_kc && g.b_kc)) return false;
  auto fits = [&](bool kc, int rows, long long ld) {
    if (kc) return panel_bytes(true, rows, g.K, ld, 0) < (long long)kOOB;
    return split_allowed(g) ? rc_max_k(rows, ld) >= 64 : rc_max_k(rows, ld) >= g.K;
  };
  return whole_chunks<uint16_t>(g.A, g.lda, g.a_kc ? g.K : g.M) &&
         whole_chunks<uint16_t>(g.B, g.ldb, g.b_kc ? g.K : g.N) && g.M > 0 && g.N > 0 &&
         g.K > 0 && fits(g.a_kc, g.M, g.lda) && fits(g.b_kc, g.N, g.ldb);
}

// Split count for the direct path: the K = tokens product (row-contiguous
// operands) is cut over K so that the CUs share the work evenly, and so is a
// K-contiguous product whose caller asks for it (kc_split: dX of a small
// batch, whose few tiles would leave most CUs idle).  A bf16 result (Cb) is
// never split.  The count
// minimises a cost in K steps: the rounds of workgroups over the CUs times
// the K steps of a split, plus the split partials' HBM traffic ((s + 1)
// fp32 outputs written and read) at kSplitBytesPerStep, the bytes HBM moves
// in the time of one K step (a 64 KiB stage takes ~2 us per CU; ~6 TB/s).
// At least 8 K steps per split.  E.g. 48 tiles x 256 steps: 5 splits (240
// workgroups, 52 steps); 192 tiles x 256 steps: 4 splits (768 workgroups,
// three rounds of 64 steps) rather than 192 workgroups of 256 steps.
constexpr double kSplitBytesPerStep = 11.0 * (1 << 20);
template <class C>
int direct_splits_cfg(const GemmDesc& g) {
  static_assert(C::BK == 64, "rc_max_k counts 64-k stages");
  if (!split_allowed(g)) return 1;
  const long long tiles = (long long)((g.M + C::BM - 1) / C::BM) * ((g.N + C::BN - 1) / C::BN);
  const int kt = (g.K + C::BK - 1) / C::BK;
  const long long slots = C::OCC * 256LL;  // workgroups the CUs run at once
  const double out_bytes = 4.0 * g.M * g.N;
  // fewest splits whose row-contiguous panels fit (direct_ok: one stage does)
  long long kmax = kt;
  if (!g.a_kc) kmax = min(kmax, rc_max_k(g.M, g.lda) / C::BK);
  if (!g.b_kc) kmax = min(kmax, rc_max_k(g.N, g.ldb) / C::BK);
  kmax = max(kmax, 1LL);
  const int s_min = (int)((kt + kmax - 1) / kmax);
  int best = s_min;
  double best_cost = 0.0;
  for (int s = s_min; s <= max(s_min, kt / 8); ++s) {
    const long long rounds = (tiles * s + slots - 1) / slots;
    const int steps = (kt + s - 1) / s;
    const double cost =
        (double)(rounds * steps) + (s > 1 ? (s + 1) * out_bytes / kSplitBytesPerStep : 0.0);
    if (s == s_min || cost < best_cost) {
      best = s;
      best_cost = cost;
    }
  }
  const int kps = ((kt + best - 1) / best) * C::BK;
  return (g.K + kps - 1) / kps;
}

using CfgDirect = DirectLine;
// Both operands K-contiguous (U = X W^T, dX = dU W on W^T): the A operand's
// ring gets the third slot, 5-6 % faster on the 256 x 256 tiles of these
// products; the row-contiguous dW product runs slower with it.
using CfgDirectKC = DirectLineA3;
// K-contiguous products whose 256 x 256 tiles would leave CUs idle (N of a
// few hundred, e.g. the rank-dp products of the projection trick, or few
// tokens, e.g. dX of one GPU's share of a batch) use 256 x 128 tiles: twice
// the workgroups, and fewer K splits where a split is planned (dX of 2,048
// tokens at d = 1024: 4 splits of 64 tiles instead of 6 of 32, a third less
// partial traffic).
using CfgNarrow = DirectNarrow;

bool use_narrow(const GemmDesc& g) {
  if (!g.a_kc || !g.b_kc) return false;
  const long long tiles = (long long)((g.M + CfgDirect::BM - 1) / CfgDirect::BM) *
                          ((g.N + CfgDirect::BN - 1) / CfgDirect::BN);
  return tiles < 256;
}

using CfgN96 = DirectN96;
// A product that is never split and has no addend (U = X W^T), whose
// 256 x 128 tiles still leave CUs idle and whose N is a whole number of
// 96-column tiles that fill more of them, runs on 256 x 96 tiles (one GPU's
// share of a batch: 2,048 tokens x 3,072 columns make 256 such tiles against
// 192 of 256 x 128).
bool use_n96(const GemmDesc& g) {
  if (!use_narrow(g) || split_allowed(g) || g.add_count != 0 || g.N % CfgN96::BN != 0)
    return false;
  const long long tm = (g.M + CfgN96::BM - 1) / CfgN96::BM;
  const long long t128 = tm * ((g.N + CfgNarrow::BN - 1) / CfgNarrow::BN);
  const long long t96 = tm * (g.N / CfgN96::BN);
  return t128 < 256 && t96 > t128 && t96 <= 256;
}

// The split count of the configuration gemm_launch runs g on.
int direct_splits(const GemmDesc& g) {
  if (!g.a_kc || !g.b_kc) return direct_splits_cfg<CfgDirect>(g);
  if (use_n96(g)) return 1;
  if (use_narrow(g)) return direct_splits_cfg<CfgNarrow>(g);
  return direct_splits_cfg<CfgDirectKC>(g);
}

// Explicit instantiations: the host pass did not emit the launch stubs of
// every specialisation referenced through launch_direct_cfg.
#define SRU_DIRECT_INST(CFG, ADD, ARC, BRC, OB) \
  template __global__ void gemm_direct_kernel<CFG, ADD, ARC, BRC, OB>(KernelArgs);
SRU_DIRECT_INST(CfgDirectKC, 0, false, false, false)
SRU_DIRECT_INST(CfgDirectKC, 1, false, false, false)
SRU_DIRECT_INST(CfgDirectKC, 2, false, false, false)
SRU_DIRECT_INST(CfgDirect, 0, true, true, false)
SRU_DIRECT_INST(CfgDirect, 1, true, true, false)
SRU_DIRECT_INST(CfgDirect, 2, true, true, false)
SRU_DIRECT_INST(CfgDirect, 0, false, true, false)
SRU_DIRECT_INST(CfgDirect, 1, false, true, false)
SRU_DIRECT_INST(CfgDirect, 2, false, true, false)
SRU_DIRECT_INST(CfgDirectKC, 0, false, false, true)
SRU_DIRECT_INST(CfgNarrow, 0, false, false, false)
SRU_DIRECT_INST(CfgN96, 0, false, false, false)
SRU_DIRECT_INST(CfgNarrow, 1, false, false, false)
SRU_DIRECT_INST(CfgNarrow, 2, false, false, false)
SRU_DIRECT_INST(CfgNarrow, 0, false, false, true)
#undef SRU_DIRECT_INST

template <class C, bool A_RC, bool B_RC, bool OB = false>
hipError_t launch_direct_cfg(const GemmDesc& g, hipStream_t st) {
  const int splits = direct_splits_cfg<C>(g);
  const int kt = (g.K + C::BK - 1) / C::BK;
  const int kps = ((kt + splits - 1) / splits) * C::BK;
  KernelArgs a{};
  a.A = g.A;
  a.B = g.B;
  a.lda = g.lda;
  a.ldb = g.ldb;
  a.M = g.M;
  a.N = g.N;
  a.K = g.K;
  a.a_bytes = operand_bytes(g.a_kc, g.M, g.K, g.lda, 2);
  a.b_bytes = operand_bytes(g.b_kc, g.N, g.K, g.ldb, 2);
  a.k_per_split = kps;
  a.tiles_m = (g.M + C::BM - 1) / C::BM;
  a.tiles_n = (g.N + C::BN - 1) / C::BN;
  a.splits = splits;
  if (splits > 1) {
    a.out = g.partials;
    a.ldo = g.N;
    a.split_stride = (long long)g.M * g.N;
  } else {
    a.out = g.C;
    a.ldo = g.ldc;
    a.add = g.add;
    a.add_count = g.add_count;
    a.add_ld = g.add_ld;
    a.add_off = g.add_off;
  }
  auto al16 = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  a.outb = g.Cb;
  a.ldob = g.ldcb;
  a.vec_out = a.ldo % 4 == 0 && a.split_stride % 4 == 0 && (!a.out || al16(a.out)) &&
              (a.add_count == 0 || (a.add_ld % 4 == 0 && a.add_off % 4 == 0 && al16(a.add))) &&
              (!OB || (a.ldob % 4 == 0 && ((uintptr_t)a.outb & 7) == 0));
  const int nwg = a.tiles_m * a.tiles_n * splits;
  timing_before(g.label ? g.label : !g.b_kc ? (g.a_kc ? "gemm_nn" : "gemm_tn") : "gemm_nt", st);
  if constexpr (OB) launch_direct<C, 0, A_RC, B_RC, true>(a, nwg, st);
  else if constexpr (C::WN == 96) launch_direct<C, 0, A_RC, B_RC>(a, nwg, st);  // no addend
  else if (a.add_count == 2) launch_direct<C, 2, A_RC, B_RC>(a, nwg, st);
  else if (a.add_count == 1) launch_direct<C, 1, A_RC, B_RC>(a, nwg, st);
  else launch_direct<C, 0, A_RC, B_RC>(a, nwg, st);
  timing_after(st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return finish_product(g, splits, st);
}

// Operand-type combinations that are instantiated: fp32 x fp32 for every
// layout in both compute modes, plus the bf16-operand products of the layer:
// U = X W^T (fp32 X, bf16 W), dX = dU W (bf16 dU, bf16 W^T, as NT) and
// dW = dU^T X (bf16 dU, fp32 X).
template <class C, bool A_KC, bool B_KC>
hipError_t launch_types(const GemmDesc& g, hipStream_t st) {
  if (!g.a_bf16 && !g.b_bf16) return launch_cfg<C, A_KC, B_KC, float, float>(g, st);
  if constexpr (C::BF16) {
    if constexpr (A_KC && B_KC) {
      if (!g.a_bf16 && g.b_bf16) return launch_cfg<C, true, true, float, uint16_t>(g, st);
      if (g.a_bf16 && g.b_bf16) return launch_cfg<C, true, true, uint16_t, uint16_t>(g, st);
    }
    if constexpr (!A_KC && !B_KC) {
      if (g.a_bf16 && !g.b_bf16) return launch_cfg<C, false, false, uint16_t, float>(g, st);
      if (g.a_bf16 && g.b_bf16) return launch_cfg<C, false, false, uint16_t, uint16_t>(g, st);
    }
  }
  return hipErrorInvalidValue;
}

template <class C>
hipError_t launch_layout(const GemmDesc& g, hipStream_t st) {
  if (g.a_kc && g.b_kc) return launch_types<C, true, true>(g, st);
  if (g.a_kc && !g.b_kc) return launch_types<C, true, false>(g, st);
  if (!g.a_kc && !g.b_kc) return launch_types<C, false, false>(g, st);
  return hipErrorInvalidValue;  // (row-contiguous A with K-contiguous B is not used)
}

}  // namespace

bool gemm_is_direct(const GemmDesc& g) { return direct_ok(g); }

int gemm_splits(const GemmDesc& g) {
  if (direct_ok(g)) return direct_splits(g);
  const int s = g.bf16 ? splits_for<CfgBF16>(g) : splits_for<CfgF32>(g);
  const int bk = g.bf16 ? CfgBF16::BK : CfgF32::BK;
  const int kt = (g.K + bk - 1) / bk;
  const int kps = ((kt + s - 1) / s) * bk;
  return (g.K + kps - 1) / kps;
}

SplitSum gemm_split_sum(const GemmDesc& g) { return split_sum_of(g, gemm_splits(g)); }

size_t gemm_partial_bytes(int M, int N, int splits) {
  return splits > 1 ? sizeof(float) * (size_t)splits * (size_t)M * (size_t)N : 0;
}

hipError_t gemm_launch(const GemmDesc& g, hipStream_t st) {
  if ((g.a_bf16 || g.b_bf16) && !g.bf16) return hipErrorInvalidValue;
  if (direct_ok(g)) {
    if (g.Cb) {
      // bf16 result: K-contiguous operands, no addend (never split)
      if (!g.a_kc || !g.b_kc || g.add_count != 0) return hipErrorInvalidValue;
      return use_narrow(g) ? launch_direct_cfg<CfgNarrow, false, false, true>(g, st)
                           : launch_direct_cfg<CfgDirectKC, false, false, true>(g, st);
    }
    if (!g.a_kc) return launch_direct_cfg<CfgDirect, true, true>(g, st);
    if (!g.b_kc) return launch_direct_cfg<CfgDirect, false, true>(g, st);
    if (use_n96(g)) return launch_direct_cfg<CfgN96, false, false>(g, st);
    if (use_narrow(g)) return launch_direct_cfg<CfgNarrow, false, false>(g, st);
    return launch_direct_cfg<CfgDirectKC, false, false>(g, st);
  }
  if (g.Cb) return hipErrorInvalidValue;  // a bf16 result needs the direct path
  return g.bf16 ? launch_layout<CfgBF16>(g, st) : launch_layout<CfgF32>(g, st);
}

template <class S>
void launch_transpose(const S* src, int rows, int cols, uint16_t* dst, hipStream_t st) {
  const dim3 grid((cols + 63) / 64, (rows + 63) / 64);
  const bool tiled = rows % 64 == 0 && cols % 64 == 0 &&
                     (reinterpret_cast<uintptr_t>(src) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(dst) & 15) == 0;
  if (tiled)
    hipLaunchKernelGGL(to_bf16_t_tiled_kernel<S>, grid, dim3(256), 0, st, src, rows, cols, dst);
  else
    hipLaunchKernelGGL(to_bf16_t_kernel<S>, grid, dim3(256), 0, st, src, rows, cols, dst);
}

hipError_t to_bf16_t_launch(const void* src, bool src_bf16, int rows, int cols, uint16_t* dst,
                            hipStream_t st, const char* label) {
  timing_before(label, st);
  if (src_bf16) launch_transpose(static_cast<const uint16_t*>(src), rows, cols, dst, st);
  else launch_transpose(static_cast<const float*>(src), rows, cols, dst, st);
  timing_after(st);
  return hipGetLastError();
}

void launch_copy(const float* src, long long n, uint16_t* dst, hipStream_t st) {
  const long long threads = (n + 7) / 8;
  hipLaunchKernelGGL(to_bf16_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st,
                     src, n, dst);
}

hipError_t to_bf16_launch(const float* src, int rows, int cols, uint16_t* dst, bool transpose,
                          hipStream_t st, const char* label) {
  timing_before(label, st);
  if (transpose) {
    launch_transpose(src, rows, cols, dst, st);
  } else {
    launch_copy(src, (long long)rows * cols, dst, st);
  }
  timing_after(st);
  return hipGetLastError();
}

hipError_t proj_scan_forward_launch(const FusedFwdArgs& a, hipStream_t st) {
  // a tile holds 256 / bb steps of bb sequences, in time chunks of 32 steps;
  // k = 3 reads x_t from X (d_in = d)
  if ((a.bb != 2 && a.bb != 4 && a.bb != 8) || (a.k != 3 && a.k != 4) ||
      (a.k == 3 && (!a.X || a.d_in != a.d)))
    return hipErrorInvalidValue;
  const int grid = a.ndir * a.ngroups * a.nbgroups;
  timing_before("proj_scan_fwd", st);
  if (a.k == 3)
    hipLaunchKernelGGL((proj_scan_fwd_kernel<3>), dim3(grid), dim3(512), 0, st, a);
  else
    hipLaunchKernelGGL((proj_scan_fwd_kernel<4>), dim3(grid), dim3(512), 0, st, a);
  timing_after(st);
  return hipGetLastError();
}

hipError_t to_bf16_n_launch(const float* src, long long n, uint16_t* dst, hipStream_t st,
                            const char* label) {
  timing_before(label, st);
  launch_copy(src, n, dst, st);
  timing_after(st);
  return hipGetLastError();
}

}  // namespace sru
