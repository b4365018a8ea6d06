// Matrix products of the SRU layer on the gfx950 matrix cores (MFMA).
//
// The forward projection of Sec. 2.1 (U = X [W; W_f; W_r]^T over all L*B
// tokens at once) and the two products of the backward pass (dX = dU W and
// dW = dU^T X) are one kernel template:
//     C[M,N] = sum_k A(m,k) B(n,k)
// with each operand either K-contiguous ("kc": row-major [rows, K]) or
// row-contiguous ([K, rows]).  Operands are fp32 in memory; the loader
// converts them to the compute type while staging a tile into LDS:
//   * bf16 mode: round-to-nearest-even bf16 (v_cvt_pk_bf16_f32) and
//     v_mfma_f32_32x32x16_bf16, fp32 accumulation;
//   * fp32 mode: v_mfma_f32_32x32x2_f32.
// LDS always holds a tile K-contiguous per row ([rows][BK + pad]), so the
// MFMA fragment of a lane is one 16-byte LDS read.  A row-contiguous source
// is transposed in registers on its way into LDS (8 k-rows x 4 rows per
// thread; the bf16 pack of (k, k+1) pairs does the transposition).
//
// Pipelining: two LDS buffers; the global loads of tile k+1 are in flight
// while the MFMAs consume tile k; one barrier per K step.
// Work mapping: one workgroup per output tile (and K split).  Workgroups are
// dispatched round-robin over the 8 XCDs, so the linear tile order is
// remapped to give each XCD a contiguous run of tiles that share A panels in
// its own L2.
#include <algorithm>
#include <type_traits>

#include "sru_internal.h"

namespace sru {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

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

// bf16 tiles 256x256x32, 4 waves of 128x128; fp32 tiles 128x128x32, 4 waves of 64x64.
using CfgBF16 = Cfg<256, 256, 32, 2, 2, true>;
using CfgF32 = Cfg<128, 128, 32, 2, 2, false>;

__device__ __forceinline__ floatx4 load4(const float* p, long long idx, int valid) {
  // valid = number of in-bounds elements starting at idx (<= 0: none)
  floatx4 v;
  v[0] = valid > 0 ? p[idx] : 0.f;
  v[1] = valid > 1 ? p[idx + 1] : 0.f;
  v[2] = valid > 2 ? p[idx + 2] : 0.f;
  v[3] = valid > 3 ? p[idx + 3] : 0.f;
  return v;
}

// ---- loader for a K-contiguous operand: element (r, k) at src[r*ld + k]
template <class C, int R, bool VEC>
struct LoaderKC {
  static constexpr int CPR = C::BK / 4;                 // float4 chunks per row
  static constexpr int PER = R * CPR / C::THREADS;
  static_assert(R * CPR % C::THREADS == 0, "tile must split evenly over the threads");
  floatx4 v[PER];

  __device__ __forceinline__ void load(const float* src, long long ld, int r0, int rows, int k0,
                                       int K, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * C::THREADS;
      const int r = r0 + c / CPR;
      const int k = k0 + (c % CPR) * 4;
      const long long idx = (long long)r * ld + k;
      if (VEC && r < rows && k + 3 < K) v[i] = *reinterpret_cast<const floatx4*>(src + idx);
      else v[i] = load4(src, idx, r < rows ? K - k : 0);
    }
  }
  __device__ __forceinline__ void store(unsigned char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * C::THREADS;
      const int r = c / CPR;
      const int k = (c % CPR) * 4;
      unsigned char* dst = lds + (r * C::LDK + k) * C::ESZ;
      if constexpr (C::BF16) {
        bf16x4 w;
        w[0] = (__bf16)v[i][0];
        w[1] = (__bf16)v[i][1];
        w[2] = (__bf16)v[i][2];
        w[3] = (__bf16)v[i][3];
        *reinterpret_cast<bf16x4*>(dst) = w;
      } else {
        *reinterpret_cast<floatx4*>(dst) = v[i];
      }
    }
  }
};

// ---- loader for a row-contiguous operand: element (r, k) at src[k*ld + r].
// Each thread owns KB k-rows x 4 rows and writes 4 K-contiguous LDS rows.
template <class C, int R, bool VEC>
struct LoaderRC {
  static constexpr int KB = C::BF16 ? 8 : 4;            // k per micro-block (16 LDS bytes)
  static constexpr int NMB = (R / 4) * (C::BK / KB);
  static constexpr int PER = NMB / C::THREADS;
  static_assert(NMB % C::THREADS == 0, "tile must split evenly over the threads");
  floatx4 v[PER][KB];

  __device__ __forceinline__ void load(const float* src, long long ld, int r0, int rows, int k0,
                                       int K, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * C::THREADS;
      const int r = r0 + (c % (R / 4)) * 4;
      const int kb = k0 + (c / (R / 4)) * KB;
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) {
        const int k = kb + kk;
        const long long idx = (long long)k * ld + r;
        if (VEC && k < K && r + 3 < rows) v[i][kk] = *reinterpret_cast<const floatx4*>(src + idx);
        else v[i][kk] = load4(src, idx, k < K ? rows - r : 0);
      }
    }
  }
  __device__ __forceinline__ void store(unsigned char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * C::THREADS;
      const int r = (c % (R / 4)) * 4;
      const int kb = (c / (R / 4)) * KB;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        unsigned char* dst = lds + ((r + e) * C::LDK + kb) * C::ESZ;
        if constexpr (C::BF16) {
          bf16x8 w;
#pragma unroll
          for (int kk = 0; kk < 8; ++kk) w[kk] = (__bf16)v[i][kk][e];
          *reinterpret_cast<bf16x8*>(dst) = w;
        } else {
          floatx4 w;
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) w[kk] = v[i][kk][e];
          *reinterpret_cast<floatx4*>(dst) = w;
        }
      }
    }
  }
};

template <class C, int R, bool KC, bool VEC>
using Loader = typename std::conditional<KC, LoaderKC<C, R, VEC>, LoaderRC<C, R, VEC>>::type;

struct KernelArgs {
  const float* A;
  const float* B;
  float* out;          // C, or the split partials
  long long lda, ldb, ldo;
  long long split_stride;  // elements between split outputs (0 when splits == 1)
  int M, N, K;
  int k_per_split;     // multiple of BK
  int tiles_m, tiles_n, splits;
  const float* add;
  long long add_ld, add_off;
  int add_count;
};

template <class C, bool A_KC, bool B_KC, bool VEC>
__global__ __launch_bounds__(C::THREADS) void gemm_kernel(KernelArgs g) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * C::STAGE_BYTES];

  // XCD-aware remap of the linear workgroup id (round-robin dispatch).
  const int nwg = gridDim.x;
  const int w = blockIdx.x;
  const int q = nwg / 8, rmd = nwg % 8, x = w % 8;
  const int u = x * q + (x < rmd ? x : rmd) + w / 8;
  const int nt = g.tiles_m * g.tiles_n;
  const int split = u / nt;
  const int t = u - split * nt;
  const int tm = t / g.tiles_n;
  const int tn = t - tm * g.tiles_n;
  const int m0 = tm * C::BM;
  const int n0 = tn * C::BN;
  const int kbeg = split * g.k_per_split;
  const int kend = min(g.K, kbeg + g.k_per_split);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm0 = (wave / C::WAVES_N) * C::WM;
  const int wn0 = (wave % C::WAVES_N) * C::WN;

  Loader<C, C::BM, A_KC, VEC> la;
  Loader<C, C::BN, B_KC, VEC> lb;

  floatx16 acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  la.load(g.A, g.lda, m0, g.M, kbeg, kend, tid);
  lb.load(g.B, g.ldb, n0, g.N, kbeg, kend, tid);
  la.store(smem, tid);
  lb.store(smem + C::A_BYTES, tid);
  __syncthreads();

  int cur = 0;
  for (int k0 = kbeg; k0 < kend; k0 += C::BK) {
    const bool next = k0 + C::BK < kend;
    if (next) {
      la.load(g.A, g.lda, m0, g.M, k0 + C::BK, kend, tid);
      lb.load(g.B, g.ldb, n0, g.N, k0 + C::BK, kend, tid);
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

  // Epilogue.  32x32 accumulator layout: element e of lane l is row
  // 8*(e/4) + 4*(l/32) + e%4, column l%32 of the MFMA tile.
  float* out = g.out + (long long)split * g.split_stride;
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int n = n0 + wn0 + j * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + wm0 + i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
        if (m < g.M && n < g.N) {
          float val = acc[i][j][e];
          if (g.add_count > 0) {
            const float* ar = g.add + (long long)m * g.add_ld + n;
            val += ar[0];
            if (g.add_count > 1) val += ar[g.add_off];
          }
          out[(long long)m * g.ldo + n] = val;
        }
      }
    }
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

template <class C>
int splits_for(const GemmDesc& g) {
  if (g.a_kc) return 1;  // only the K = tokens product (TN) is split
  const int tiles = ((g.M + C::BM - 1) / C::BM) * ((g.N + C::BN - 1) / C::BN);
  const int kt = (g.K + C::BK - 1) / C::BK;  // K steps
  int s = (2 * 256 + tiles - 1) / tiles;     // aim for two workgroups per CU
  // fp32 accumulation chains stay short (<= 2048 terms per split)
  if (!C::BF16) s = max(s, (g.K + 2047) / 2048);
  s = min(s, max(1, kt / 4));                // at least 4 K steps per split
  return max(1, min(s, 64));
}

template <class C, bool A_KC, bool B_KC>
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
  timing_before(!g.b_kc ? (g.a_kc ? "gemm_nn" : "gemm_tn") : "gemm_nt", st);
  const bool vec = ((reinterpret_cast<uintptr_t>(g.A) | reinterpret_cast<uintptr_t>(g.B)) & 15) == 0 &&
                   g.lda % 4 == 0 && g.ldb % 4 == 0;
  if (vec)
    hipLaunchKernelGGL((gemm_kernel<C, A_KC, B_KC, true>), dim3(nwg), dim3(C::THREADS), 0, st, a);
  else
    hipLaunchKernelGGL((gemm_kernel<C, A_KC, B_KC, false>), dim3(nwg), dim3(C::THREADS), 0, st, a);
  timing_after(st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  const long long total = (long long)g.M * g.N;
  const int grid = (int)std::min<long long>((total + 255) / 256, 8192);
  timing_before("splitk_reduce", st);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(grid), dim3(256), 0, st, g.partials, a.splits,
                     g.M, g.N, g.C, g.ldc, g.add, g.add_ld, g.add_off, g.add_count);
  timing_after(st);
  return hipGetLastError();
}

template <class C>
hipError_t launch_layout(const GemmDesc& g, hipStream_t st) {
  if (g.a_kc && g.b_kc) return launch_cfg<C, true, true>(g, st);
  if (g.a_kc && !g.b_kc) return launch_cfg<C, true, false>(g, st);
  if (!g.a_kc && !g.b_kc) return launch_cfg<C, false, false>(g, st);
  return hipErrorInvalidValue;  // (row-contiguous A with K-contiguous B is not used)
}

}  // namespace

int gemm_splits(const GemmDesc& g) {
  const int s = g.bf16 ? splits_for<CfgBF16>(g) : splits_for<CfgF32>(g);
  const int bk = g.bf16 ? CfgBF16::BK : CfgF32::BK;
  const int kt = (g.K + bk - 1) / bk;
  const int kps = ((kt + s - 1) / s) * bk;
  return (g.K + kps - 1) / kps;
}

size_t gemm_partial_bytes(int M, int N, int splits) {
  return splits > 1 ? sizeof(float) * (size_t)splits * (size_t)M * (size_t)N : 0;
}

hipError_t gemm_launch(const GemmDesc& g, hipStream_t st) {
  return g.bf16 ? launch_layout<CfgBF16>(g, st) : launch_layout<CfgF32>(g, st);
}

}  // namespace sru
