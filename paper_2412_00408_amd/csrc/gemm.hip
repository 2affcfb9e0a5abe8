// gemm.hip — quake_linear_gelu: y = GELU(x w^T) for bfloat16 or binary16
// x [m, k] and w [n, k] (both k-contiguous, the layout of a linear layer's
// input and weight), binary32 accumulation on the matrix cores, the GELU of
// Eq. 7 with QuAKE / QuAKE2 / EXACT applied to the binary32 accumulators in
// the epilogue, output in the input format. This is QuAKE inside a fused consumer: the GELU
// costs no HBM traffic of its own, and its VALU work runs beside the MFMAs.
//
// Tiling: a workgroup (4 waves) computes a 128 x BN tile of y (BN = 192 when
// n is a multiple of 192 and those tiles cover every CU, else 128), each wave
// a 64 x BN/2 quarter as 2 x BN/64 blocks of v_mfma_f32_32x32x16_bf16. The
// wider tile reads 17 % fewer
// LDS bytes per matrix-core operation (each A fragment feeds three blocks
// instead of two), which is what bounds this loop. K advances in slabs of 64:
// the next slab is loaded from HBM into registers while the current one is
// multiplied out of LDS (rows padded by 16 bytes so the 16-byte fragment reads
// of 8 consecutive rows hit distinct banks). With two workgroups per CU the
// other workgroup's products cover a slab's load latency; a grid of at most
// one tile per CU over a long k (>= 1024) has nothing to cover it, and there
// each slab is loaded two slabs ahead into a second register set.
// Operand lane layout of the 32x32x16 bf16 MFMA (checked on the device):
// lane l holds row (l mod 32) and k = 8 (l / 32) .. +7 of A, and column
// (l mod 32), the same k, of B; accumulator r of lane l is row
// 8 (r / 4) + 4 (l / 32) + (r mod 4), column l mod 32.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// one 32x32x16 matrix-core step on raw 16-bit operands of format DT
template <int DT>
__device__ __forceinline__ f32x16_t mfma16(u32x4 a, u32x4 b, f32x16_t c) {
  if constexpr (DT == BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                  __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}
template <int DT>
__device__ __forceinline__ uint16_t narrow16(float v) {
  if constexpr (DT == BF16)
    return __builtin_bit_cast(uint16_t, (__bf16)v);
  else
    return __builtin_bit_cast(uint16_t, (_Float16)v);
}

constexpr int kBM = 128, kBK = 64;
constexpr int kLdsRow = kBK + 8;   // bf16 elements per LDS row (144 bytes)
constexpr int kGemmThreads = 256;
constexpr int kMaxBN = 192;

struct GemmArgs {
  const uint16_t* x;
  const uint16_t* w;
  uint16_t* y;
  int32_t m, n, k;
  int64_t ldx, ldw, ldy;   // elements
  float c0, c1, a;         // GELU constants (Eq. 7 folded into Eq. 5)
  uint32_t tiles_m, tiles_n;
  uint32_t xcd_split;      // tiles_m % 4 == 0 and tiles_n % 2 == 0
};

// OCC: workgroups per CU the register budget is set for (3 at BN = 128: at
// most 168 VGPRs; 2 at BN = 192 and with two register sets). AHEAD: slabs
// in flight (1: the next slab, one register set; 2: two register sets).
template <int DT, int MODE, bool GELU, int BN, int OCC, int AHEAD>
__global__ __launch_bounds__(kGemmThreads, OCC) void gemm_kernel(GemmArgs g) {
  constexpr int TN = BN / 64;                     // 32 x 32 blocks per wave along n
  constexpr int VA = kBM * 8 / kGemmThreads;      // 16-byte vectors per thread per slab
  constexpr int VB = BN * 8 / kGemmThreads;
  static_assert(BN % 64 == 0 && BN <= kMaxBN && BN * 8 % kGemmThreads == 0, "tile width");
  __shared__ __attribute__((aligned(16))) uint16_t sx[kBM * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t sw[BN * kLdsRow];
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  // Workgroups go to the 8 XCDs round-robin (blockIdx mod 8). When the tile
  // grid splits into 4 x 2 equal blocks, XCD j gets block (j / 2, j mod 2),
  // so the rows of x and w its tiles share stay in its own L2.
  int tm, tn;
  if (g.xcd_split) {
    const uint32_t xcd = blockIdx.x & 7u, local = blockIdx.x >> 3;
    const uint32_t bm = g.tiles_m >> 2, bn = g.tiles_n >> 1;
    tm = (int)((xcd >> 1) * bm + local / bn);
    tn = (int)((xcd & 1u) * bn + local % bn);
  } else {
    tm = (int)(blockIdx.x / g.tiles_n);
    tn = (int)(blockIdx.x % g.tiles_n);
  }
  const int row0 = tm * kBM, col0 = tn * BN;

  // Slab loads: 8 16-byte vectors per row of each operand; thread t takes
  // vectors t + 256 i, i.e. row v / 8 and k-vector v mod 8. Rows past m (n)
  // re-read the last row; k past the end re-reads k-vector 0 and is replaced
  // by zeros when the slab is written to LDS (k is a multiple of 8). Nothing
  // consumes the loaded registers before that write, so the loads stay in
  // flight during the previous slab's MFMAs.
  u32x4 rxs[2][VA], rws[2][VB];
  const u32x4 zero = {0u, 0u, 0u, 0u};
  auto load_slab = [&](u32x4 (&rx)[VA], u32x4 (&rw)[VB], int k0) {
#pragma unroll
    for (int i = 0; i < VA; ++i) {
      const int v = t + kGemmThreads * i;
      const int r = v >> 3, kk = k0 + 8 * (v & 7);
      const int gm = min(row0 + r, g.m - 1);
      const int kc = kk < g.k ? kk : 0;
      rx[i] = *reinterpret_cast<const u32x4*>(g.x + (int64_t)gm * g.ldx + kc);
    }
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = t + kGemmThreads * i;
      const int r = v >> 3, kk = k0 + 8 * (v & 7);
      const int gn = min(col0 + r, g.n - 1);
      const int kc = kk < g.k ? kk : 0;
      rw[i] = *reinterpret_cast<const u32x4*>(g.w + (int64_t)gn * g.ldw + kc);
    }
  };
  auto store_slab = [&](const u32x4 (&rx)[VA], const u32x4 (&rw)[VB], int k0) {
#pragma unroll
    for (int i = 0; i < VA; ++i) {
      const int v = t + kGemmThreads * i;
      const int r = v >> 3, c = 8 * (v & 7);
      *reinterpret_cast<u32x4*>(sx + r * kLdsRow + c) = (k0 + c < g.k) ? rx[i] : zero;
    }
#pragma unroll
    for (int i = 0; i < VB; ++i) {
      const int v = t + kGemmThreads * i;
      const int r = v >> 3, c = 8 * (v & 7);
      *reinterpret_cast<u32x4*>(sw + r * kLdsRow + c) = (k0 + c < g.k) ? rw[i] : zero;
    }
  };

  f32x16_t acc[2][TN];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (g.k + kBK - 1) / kBK;
  // AHEAD = 2: two register sets, each slab's loads issued two slabs ahead.
  // Those loads are unconditional (past the end of k they re-read k-vector 0,
  // and nothing stores them), so the compiler's wait counts stay exact:
  // storing a slab waits only for its own set, the other set's loads stay in
  // flight.
  load_slab(rxs[0], rws[0], 0);
  __builtin_amdgcn_sched_barrier(0);   // set 0's loads all before set 1's
  if constexpr (AHEAD == 2) load_slab(rxs[1], rws[1], kBK);
  __builtin_amdgcn_sched_barrier(0);
  const int fr = lane & 31, fk = 8 * (lane >> 5);
  auto slab = [&](int kt, u32x4 (&rx)[VA], u32x4 (&rw)[VB]) {
    __syncthreads();   // every wave is done reading the previous slab
    store_slab(rx, rw, kt * kBK);
    __syncthreads();
    if constexpr (AHEAD == 2) load_slab(rx, rw, (kt + 2) * kBK);   // in flight for two slabs
    else if (kt + 1 < nk) load_slab(rxs[0], rws[0], (kt + 1) * kBK);   // one set: the next slab
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      u32x4 af[2], bf[TN];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const u32x4*>(sx + (wm * 64 + 32 * i + fr) * kLdsRow + ks * 16 + fk);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bf[j] = *reinterpret_cast<const u32x4*>(sw + (wn * 32 * TN + 32 * j + fr) * kLdsRow + ks * 16 + fk);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = mfma16<DT>(af[i], bf[j], acc[i][j]);
    }
  };
  // every way back to the loop head has issued both sets in the same order
  // (an exit taken before the second set would make the waits conservative)
  if constexpr (AHEAD == 2) {
    for (int kt = 0;; kt += 2) {
      slab(kt, rxs[0], rws[0]);
      if (kt + 1 >= nk) break;
      slab(kt + 1, rxs[1], rws[1]);
      if (kt + 2 >= nk) break;
    }
  } else {
    for (int kt = 0; kt < nk; ++kt) slab(kt, rxs[0], rws[0]);
  }

  // Epilogue: GELU on the binary32 accumulators, round to the 16-bit format,
  // store. Accumulator r of block (i, j) in lane l is row
  // 32 i + 8 (r / 4) + 4 (l / 32) + r mod 4 of the wave's rows and column
  // 32 j + l mod 32 of its columns: for each (i, r) a half-wave stores 64
  // contiguous bytes of one row. In a tile inside m and n (uniform) the row
  // base of each (i, r) is uniform and the lane adds a 32-bit offset, so the
  // stores need no per-element address arithmetic or bounds checks.
  // the wave index made uniform here keeps the row bases of the stores in
  // scalar registers (the main loop above is faster with its LDS fragment
  // addresses formed per lane)
  const int wu = __builtin_amdgcn_readfirstlane(wave);
  const int wrow = row0 + (wu >> 1) * 64, wcol = col0 + (wu & 1) * 32 * TN;
  if (row0 + kBM <= g.m && col0 + BN <= g.n && (int64_t)4 * g.ldy < INT32_MAX) {
    const uint32_t lo = (uint32_t)(4 * (lane >> 5)) * (uint32_t)g.ldy + (uint32_t)fr;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        uint16_t* yr = g.y + (int64_t)(wrow + 32 * i + 8 * (r >> 2) + (r & 3)) * g.ldy + wcol;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          float v = acc[i][j][r];
          if constexpr (GELU) v = gelu_q<MODE>(v, g.c0, g.c1, g.a);
          yr[lo + 32 * j] = narrow16<DT>(v);
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = wcol + 32 * j + fr;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wrow + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        float v = acc[i][j][r];
        if constexpr (GELU) v = gelu_q<MODE>(v, g.c0, g.c1, g.a);
        if (row < g.m && col < g.n)
          g.y[(int64_t)row * g.ldy + col] = narrow16<DT>(v);
      }
    }
}

template <int DT, int MODE, int BN, int OCC, int AHEAD>
void launch_gemm(int gelu, dim3 grid, hipStream_t s, const GemmArgs& g) {
  if (gelu)
    hipLaunchKernelGGL((gemm_kernel<DT, MODE, true, BN, OCC, AHEAD>), grid, dim3(kGemmThreads), 0, s, g);
  else
    hipLaunchKernelGGL((gemm_kernel<DT, MODE, false, BN, OCC, AHEAD>), grid, dim3(kGemmThreads), 0, s, g);
}

template <int DT>
void launch_gemm_dt(int mode, bool wide, bool ahead2, int gelu, dim3 grid, hipStream_t s,
                    const GemmArgs& g) {
#define QK_GEMM_CASE(M)                                      \
  if (mode == M) {                                           \
    if (ahead2) {                                            \
      if (wide)                                              \
        launch_gemm<DT, M, 192, 2, 2>(gelu, grid, s, g);     \
      else                                                   \
        launch_gemm<DT, M, 128, 2, 2>(gelu, grid, s, g);     \
    } else if (wide) {                                       \
      launch_gemm<DT, M, 192, 2, 1>(gelu, grid, s, g);       \
    } else {                                                 \
      launch_gemm<DT, M, 128, 3, 1>(gelu, grid, s, g);       \
    }                                                        \
  }
  QK_GEMM_CASE(EXACT) QK_GEMM_CASE(Q1) QK_GEMM_CASE(Q2) QK_GEMM_CASE(Q2M)
#undef QK_GEMM_CASE
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_linear_gelu(const void* x, const void* w, void* y, int64_t m,
                                          int64_t n, int64_t k, int64_t ldx, int64_t ldw,
                                          int64_t ldy, quake_dtype dtype, quake_mode mode,
                                          int gelu, void* stream) {
  if (dtype != QUAKE_BF16 && dtype != QUAKE_F16) return QUAKE_EDTYPE;
  if (!valid_mode(mode)) return QUAKE_EMODE;
  if (m < 0 || n < 0 || k < 0) return QUAKE_EINVAL;
  if (m == 0 || n == 0) return QUAKE_OK;
  if (k == 0 || k % 8 != 0 || x == nullptr || w == nullptr || y == nullptr) return QUAKE_EINVAL;
  if (ldx < k || ldw < k || ldy < n || ldx % 8 != 0 || ldw % 8 != 0) return QUAKE_EINVAL;
  if (!aligned16(x) || !aligned16(w)) return QUAKE_EINVAL;
  // 32-bit row, column and k arithmetic in the kernel: the last slab loaded
  // (two slabs ahead) starts below k + 2 kBK
  if (m > INT32_MAX - kBM || n > INT32_MAX - kMaxBN || k > INT32_MAX - 4 * kBK) return QUAKE_EINVAL;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  // the 128 x 192 tile where n allows it and its grid still covers every CU;
  // otherwise the 128 x 128 tile, whose grid is 1.5x larger (measured
  // 1.28x faster at 4096 x 768 x 3072, where the wide grid is 128 tiles)
  const bool wide = n % 192 == 0 && ((m + kBM - 1) / kBM) * (n / 192) >= cus;
  const int64_t bn = wide ? 192 : 128;
  const int64_t tiles_m = (m + kBM - 1) / kBM, tiles_n = (n + bn - 1) / bn;
  if (tiles_m * tiles_n > INT32_MAX) return QUAKE_EINVAL;
  const Affine af = gelu_affine(mode);
  GemmArgs g{static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w),
             static_cast<uint16_t*>(y), (int32_t)m, (int32_t)n, (int32_t)k, ldx, ldw, ldy,
             af.c0, af.c1, gelu_a(), (uint32_t)tiles_m, (uint32_t)tiles_n,
             (uint32_t)(tiles_m % 4 == 0 && tiles_n % 2 == 0)};
  const dim3 grid((uint32_t)(tiles_m * tiles_n));
  const hipStream_t s = static_cast<hipStream_t>(stream);
  // at most one tile per CU and a long k: slabs loaded two ahead (measured
  // 1.1-1.3x faster there; elsewhere the co-resident workgroup hides the
  // latency and the second set only costs registers)
  const bool ahead2 = tiles_m * tiles_n <= cus && k >= 1024;
  if (dtype == QUAKE_BF16)
    launch_gemm_dt<BF16>(mode, wide, ahead2, gelu, grid, s, g);
  else
    launch_gemm_dt<F16>(mode, wide, ahead2, gelu, grid, s, g);
  return launch_status();
}
