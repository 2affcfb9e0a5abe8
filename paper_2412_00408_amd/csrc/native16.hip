// native16.hip — quake_exp16: QuAKE / QuAKE2 built directly in the binary16
// or bfloat16 layout (arXiv:2412.00408, Sec. II-A: the construction holds for
// any IEEE-style format; Eq. 3 with that format's l_m and B, Algorithm 1 with
// its masks). No binary32 result is formed and nothing is narrowed:
//   l = fma(x, c0, c1) in binary32 (x widened exactly), clamped to
//       [0, (2^l_e - 1) 2^l_m]; z = (int) l is the 16-bit result of QuAKE;
//   QuAKE2 refines z's l_m-bit mantissa: a_m = (z & M) | (B << l_m) in [1, 2),
//       y_m = (a_m^2 + 2) / 3 in the format's arithmetic, joined to z's
//       exponent field.
// binary16 (l_e 5, l_m 10, B 15): two elements per dword through the packed
// v_pk_fma_f16 / v_pk_mul_f16 (each rounded once to binary16) and one
// v_and_or / v_bfi per pair. bfloat16 (l_e 8, l_m 7, B 127): the refinement
// runs in binary32 (t = a_m^2 + 2 is exact there) and is rounded to bfloat16
// by v_cvt_pk_bf16_f32, the hardware having no bfloat16 FMA.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));

struct N16Const {
  float c0, c1;
};

template <int DT>
struct N16Fmt;
template <>
struct N16Fmt<F16> {
  static constexpr int kLm = 10, kB = 15;
  static constexpr float kTop = 31744.0f;          // 31 * 2^10: the pattern of +inf
  static constexpr uint32_t kMant2 = 0x03FF03FFu;  // mantissa fields of a pair
  static constexpr uint32_t kExpB2 = 0x3C003C00u;  // exponent fields := B
};
template <>
struct N16Fmt<BF16> {
  static constexpr int kLm = 7, kB = 127;
  static constexpr float kTop = 32640.0f;          // 255 * 2^7
  static constexpr uint32_t kMant2 = 0x007F007Fu;
  static constexpr uint32_t kExpB2 = 0x3F803F80u;
};

// z of one element (Eq. 3 in the 16-bit layout), as an integer below 2^15.
template <int DT>
__device__ __forceinline__ uint32_t n16_z(float x, const N16Const& k) {
  const float l = __builtin_amdgcn_fmed3f(__builtin_fmaf(x, k.c0, k.c1), 0.0f, N16Fmt<DT>::kTop);
  return (uint32_t)(int32_t)l;
}

// Two elements (the low and high halves of one dword of input) to one dword
// of output patterns.
template <int DT, int MODE>
__device__ __forceinline__ uint32_t n16_pair(float xlo, float xhi, const N16Const& k) {
  const uint32_t zp = n16_z<DT>(xlo, k) | (n16_z<DT>(xhi, k) << 16);
  if constexpr (MODE == Q1) {
    return zp;
  } else if constexpr (DT == F16) {
    const h2_t am = __builtin_bit_cast(h2_t, (zp & N16Fmt<F16>::kMant2) | N16Fmt<F16>::kExpB2);
    const h2_t two = {(_Float16)2.0f, (_Float16)2.0f};
    const _Float16 th = (_Float16)(1.0f / 3.0f);   // fl16(1/3): 1/3 is not a tie in binary16
    const h2_t third = {th, th};
    const h2_t t = __builtin_elementwise_fma(am, am, two);   // v_pk_fma_f16, one rounding
    const h2_t ym = t * third;                               // v_pk_mul_f16
    return (zp & ~N16Fmt<F16>::kMant2) | (__builtin_bit_cast(uint32_t, ym) & N16Fmt<F16>::kMant2);
  } else {
    const uint32_t am2 = (zp & N16Fmt<BF16>::kMant2) | N16Fmt<BF16>::kExpB2;
    const float alo = as_f(am2 << 16), ahi = as_f(am2 & 0xFFFF0000u);
    const float plo = __builtin_fmaf(alo, alo, 2.0f) * kThird;  // t exact in binary32
    const float phi = __builtin_fmaf(ahi, ahi, 2.0f) * kThird;
    const uint32_t ym = pack_bf16(plo, phi);                   // round to bfloat16
    return (zp & ~N16Fmt<BF16>::kMant2) | (ym & N16Fmt<BF16>::kMant2);
  }
}

template <int DT>
__device__ __forceinline__ float n16_lo(uint32_t w) {
  return DT == F16 ? f16_lo(w) : bf16_lo(w);
}
template <int DT>
__device__ __forceinline__ float n16_hi(uint32_t w) {
  return DT == F16 ? f16_hi(w) : bf16_hi(w);
}

constexpr int kN16Block = 256;

// One 16-byte vector (8 elements) per lane; the last workgroup's first lanes
// also take the elements past the last whole vector.
template <int DT, int MODE>
__global__ __launch_bounds__(kN16Block) void exp16_vec_kernel(const u32x4* __restrict__ x,
                                                             u32x4* __restrict__ y,
                                                             uint32_t nvec, uint32_t tail,
                                                             N16Const k) {
  const uint32_t i = blockIdx.x * kN16Block + threadIdx.x;
  if (i < nvec) {
    const u32x4 v = __builtin_nontemporal_load(x + i);
    u32x4 o;
#pragma unroll
    for (int w = 0; w < 4; ++w) o[w] = n16_pair<DT, MODE>(n16_lo<DT>(v[w]), n16_hi<DT>(v[w]), k);
    __builtin_nontemporal_store(o, y + i);
  }
  if (tail && blockIdx.x == gridDim.x - 1 && threadIdx.x < tail) {
    const int64_t e = (int64_t)nvec * 8 + threadIdx.x;
    const uint16_t h = reinterpret_cast<const uint16_t*>(x)[e];
    const float xv = DT == F16 ? (float)__builtin_bit_cast(_Float16, h) : as_f((uint32_t)h << 16);
    reinterpret_cast<uint16_t*>(y)[e] = (uint16_t)(n16_pair<DT, MODE>(xv, 0.0f, k) & 0xFFFFu);
  }
}

// Buffers not both 16-byte aligned (element-aligned): y in aligned vectors,
// each assembled from the one or two aligned vectors of x that hold its bytes
// (d bytes into the first; d = 0 when x and y share their offset), the
// elements before y's first 16-byte boundary and after its last whole vector
// in the first and the last workgroup, one element per lane.
template <int DT, int MODE>
__device__ __forceinline__ uint16_t exp16_one(uint16_t h, const N16Const& k) {
  const float xv = DT == F16 ? (float)__builtin_bit_cast(_Float16, h) : as_f((uint32_t)h << 16);
  return (uint16_t)(n16_pair<DT, MODE>(xv, 0.0f, k) & 0xFFFFu);
}

template <int DT, int MODE>
__global__ __launch_bounds__(kN16Block) void exp16_realign_kernel(const uint16_t* __restrict__ x,
                                                                 uint16_t* __restrict__ y,
                                                                 uint32_t head, uint32_t nvec,
                                                                 uint32_t tail, uint32_t d,
                                                                 N16Const k) {
  const u32x4* xa =
      reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(x + head) - d);
  u32x4* ya = reinterpret_cast<u32x4*>(y + head);
  const uint32_t i = blockIdx.x * kN16Block + threadIdx.x;
  // d = 0: the vector is a itself, and the next aligned vector of x may lie
  // past its end; else a and b from aligned_pair
  u32x4 a, b;
  if (d == 0) {
    if (i < nvec) a = __builtin_nontemporal_load(xa + i);
    b = a;
  } else {
    aligned_pair(xa, i, nvec, a, b);
  }
  if (i < nvec) {
    const u32x4 v = realign(a, b, d);
    u32x4 o;
#pragma unroll
    for (int w = 0; w < 4; ++w) o[w] = n16_pair<DT, MODE>(n16_lo<DT>(v[w]), n16_hi<DT>(v[w]), k);
    __builtin_nontemporal_store(o, ya + i);
  }
  if (blockIdx.x == 0 && threadIdx.x < head) y[threadIdx.x] = exp16_one<DT, MODE>(x[threadIdx.x], k);
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x < tail) {
    const int64_t e = (int64_t)head + (int64_t)nvec * 8 + threadIdx.x;
    y[e] = exp16_one<DT, MODE>(x[e], k);
  }
}

// Buffers not element-aligned, or short: one element per lane, grid-stride.
template <int DT, int MODE>
__global__ __launch_bounds__(kN16Block) void exp16_scalar_kernel(const uint16_t* __restrict__ x,
                                                                uint16_t* __restrict__ y,
                                                                uint32_t n, N16Const k) {
  for (uint32_t i = blockIdx.x * kN16Block + threadIdx.x; i < n; i += gridDim.x * kN16Block) {
    const uint16_t h = x[i];
    const float xv = DT == F16 ? (float)__builtin_bit_cast(_Float16, h) : as_f((uint32_t)h << 16);
    y[i] = (uint16_t)(n16_pair<DT, MODE>(xv, 0.0f, k) & 0xFFFFu);
  }
}

constexpr int64_t kN16Chunk = int64_t(1) << 30;   // elements per launch, a multiple of 8

template <int DT, int MODE>
static quake_status exp16_launch(const void* x, void* y, int64_t n, const N16Const& k,
                                 hipStream_t s) {
  const uintptr_t ux = (uintptr_t)x, uy = (uintptr_t)y;
  if (((ux | uy) & 15u) != 0 && ux % 2 == 0 && uy % 2 == 0 && n >= 16 && n < (int64_t(1) << 31)) {
    const int64_t head = (int64_t)((16u - (uy & 15u)) & 15u) / 2;
    const int64_t nvec = (n - head) / 8, tail = (n - head) % 8;
    const uint32_t d = (uint32_t)((ux + head * 2) & 15u);
    const uint32_t grid = (uint32_t)std::max<int64_t>(1, (nvec + kN16Block - 1) / kN16Block);
    hipLaunchKernelGGL((exp16_realign_kernel<DT, MODE>), dim3(grid), dim3(kN16Block), 0, s,
                       static_cast<const uint16_t*>(x), static_cast<uint16_t*>(y),
                       (uint32_t)head, (uint32_t)nvec, (uint32_t)tail, d, k);
    return launch_status();
  }
  // x and y at the same offset from a 16-byte boundary, beyond that length
  // range: the elements before the first boundary take the scalar kernel, the
  // rest the vector kernel.
  if ((ux & 15u) != 0 && ((ux - uy) & 15u) == 0 && ux % 2 == 0) {
    const int64_t head = std::min<int64_t>(n, (int64_t)((16u - (ux & 15u)) & 15u) / 2);
    hipLaunchKernelGGL((exp16_scalar_kernel<DT, MODE>), dim3(1), dim3(kN16Block), 0, s,
                       static_cast<const uint16_t*>(x), static_cast<uint16_t*>(y),
                       (uint32_t)head, k);
    const quake_status st = launch_status();
    if (st != QUAKE_OK || head == n) return st;
    return exp16_launch<DT, MODE>(static_cast<const uint16_t*>(x) + head,
                                  static_cast<uint16_t*>(y) + head, n - head, k, s);
  }
  const bool vec = aligned16(x) && aligned16(y);
  for (int64_t o = 0; o < n; o += kN16Chunk) {
    const int64_t m = std::min(kN16Chunk, n - o);
    const uint16_t* xc = static_cast<const uint16_t*>(x) + o;
    uint16_t* yc = static_cast<uint16_t*>(y) + o;
    if (vec) {
      const uint32_t nvec = (uint32_t)(m / 8), tail = (uint32_t)(m % 8);
      const uint32_t grid = std::max<uint32_t>(1, (nvec + kN16Block - 1) / kN16Block);
      hipLaunchKernelGGL((exp16_vec_kernel<DT, MODE>), dim3(grid), dim3(kN16Block), 0, s,
                         reinterpret_cast<const u32x4*>(xc), reinterpret_cast<u32x4*>(yc), nvec,
                         tail, k);
    } else {
      const uint32_t grid = (uint32_t)std::min<int64_t>((m + kN16Block - 1) / kN16Block, 65536);
      hipLaunchKernelGGL((exp16_scalar_kernel<DT, MODE>), dim3(grid), dim3(kN16Block), 0, s, xc,
                         yc, (uint32_t)m, k);
    }
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_exp16(const void* x, void* y, int64_t n, quake_dtype dtype,
                                    quake_mode mode, float a, float b, void* stream) {
  if (dtype != QUAKE_F16 && dtype != QUAKE_BF16) return QUAKE_EDTYPE;
  if (mode != QUAKE_1 && mode != QUAKE_2) return QUAKE_EMODE;
  if (n < 0) return QUAKE_EINVAL;
  if (n > 0 && (x == nullptr || y == nullptr)) return QUAKE_EINVAL;
  if (!std::isfinite(a) || !std::isfinite(b)) return QUAKE_EINVAL;
  // Eq. 5 in the 16-bit layout: c0 = 2^l_m a / ln2, c1 = 2^l_m (B - beta + b / ln2)
  const double two_lm = dtype == QUAKE_F16 ? 1024.0 : 128.0;
  const double bias = dtype == QUAKE_F16 ? 15.0 : 127.0;
  const double beta = mode == QUAKE_1 ? kSchraudolph : 0.0;
  const N16Const k{(float)((a / kLn2) * two_lm), (float)(((bias - beta) + b / kLn2) * two_lm)};
  if (!std::isfinite(k.c0) || !std::isfinite(k.c1)) return QUAKE_EINVAL;
  if (n == 0) return QUAKE_OK;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == QUAKE_F16)
    return mode == QUAKE_1 ? exp16_launch<F16, Q1>(x, y, n, k, s) : exp16_launch<F16, Q2>(x, y, n, k, s);
  return mode == QUAKE_1 ? exp16_launch<BF16, Q1>(x, y, n, k, s) : exp16_launch<BF16, Q2>(x, y, n, k, s);
}
