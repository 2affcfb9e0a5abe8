// quake_device.hpp — device-side building blocks of libquake (gfx950 / CDNA4).
//
// The per-element arithmetic of QuAKE (arXiv:2412.00408):
//   Sec. III-A, Eq. 5   l = c0*x + c1, one v_fma_f32
//   (clamp)             l = med3(l, 0, 255*2^23), one v_med3_f32
//   Eq. 3               z = convert_to_int(l), one v_cvt_i32_f32 (truncating)
//   Eq. 2 (QuAKE)       result = bits of z
//   Alg. 1 (QuAKE2)     a_m = (z & 0x007FFFFF) | 0x3F800000   (v_and_or_b32)
//                       (QuAKE2M: the same with the minimax coefficients of Eq. 6)
//                       y_m = fma(a_m, a_m, 2) * fl(1/3)      (Eq. 6, a0=1/3, a2=2/3)
//                       result = (z & 0xFF800000) + bits(y_m) - 0x3F800000, which is
//                       one v_bfi_b32: y_m lies in [1, 2), so bits(y_m) - 0x3F800000
//                       is exactly y_m's mantissa field and the addition cannot
//                       carry into z's sign/exponent field.
// plus 16-byte vector I/O for binary32 / binary16 / bfloat16 and the 64-lane
// DPP reductions used by the softmax kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace qk {

enum Mode : int { EXACT = 0, Q1 = 1, Q2 = 2, Q2M = 3 };
enum Dt : int { F32 = 0, F16 = 1, BF16 = 2 };

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Clamp bound of l: biased exponent 255, mantissa 0 (the bits of +inf).
constexpr float kLHi = 2139095040.0f;                 // 255 * 2^23, exact
constexpr float kK127 = 1065353216.0f;                // 127 * 2^23, exact
constexpr float kThird = (float)(1.0 / 3.0);          // fl32(1/3)
constexpr uint32_t kMantMask = 0x007FFFFFu;           // Alg. 1: keep mantissa
constexpr uint32_t kSignExpMask = 0xFF800000u;        // Alg. 1: keep sign + exponent
constexpr uint32_t kExpB = 0x3F800000u;               // Alg. 1: exponent field := B
// Coefficients of Eq. 6 minimising max |y_m(a) 2^(1-a) - 1| over a in [1, 2]
// (the grid-search optimum of Sec. III-B): the Remez solution in double,
// 0.33718943461968731, -0.016742593503297265, 0.68127792209835503 (worst case
// 0.17247632 %), each rounded once to binary32.
constexpr float kQ2mA0 = 0x1.594830p-2f;
constexpr float kQ2mA1 = -0x1.124f86p-6f;
constexpr float kQ2mA2 = 0x1.5cd076p-1f;

__device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }

__device__ __forceinline__ float as_f(uint32_t u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ uint32_t as_u(float f) { return __builtin_bit_cast(uint32_t, f); }

// QuAKE / QuAKE2 from z, the truncated integer of the clamped argument
// (Eq. 3): Eq. 2 reads z as a binary32, Algorithm 1 refines its mantissa.
template <int MODE>
__device__ __forceinline__ float quake_of_z(uint32_t z) {
  if constexpr (MODE == Q1) {
    return as_f(z);
  } else if constexpr (MODE == Q2) {
    const float am = as_f((z & kMantMask) | kExpB);
    const float ym = __builtin_fmaf(am, am, 2.0f) * kThird;
    return as_f((z & kSignExpMask) | (as_u(ym) & kMantMask));
  } else {
    // minimax coefficients, Horner form; y_m in [1.0017, 1.9966) so the same
    // join applies. At a_m = 1 the result is z itself (y_m := 1): exact powers
    // of two, and 0 / +inf at the two ends of the clamp.
    const uint32_t mz = z & kMantMask;
    const float am = as_f(mz | kExpB);
    const float ym = __builtin_fmaf(__builtin_fmaf(kQ2mA0, am, kQ2mA1), am, kQ2mA2);
    const uint32_t j = (z & kSignExpMask) | (as_u(ym) & kMantMask);
    return as_f(mz == 0 ? z : j);
  }
}

// QuAKE / QuAKE2 of an already affine-mapped argument l (Eq. 5 applied).
template <int MODE>
__device__ __forceinline__ float quake_of_l(float l) {
  l = __builtin_amdgcn_fmed3f(l, 0.0f, kLHi);
  return quake_of_z<MODE>((uint32_t)(int32_t)l);
}

// The same for an argument l known to stay below 255 * 2^23 (Algorithm 2
// with a row constant |c1| < 2^54: for x <= m, l = fma(x, c0, c1) is at most
// 127 * 2^23 plus half an ulp of c1, < 2^29). v_cvt_u32_f32 truncates and
// saturates negative arguments to 0, which is the lower clamp, and the upper
// clamp cannot act, so the bits are those of quake_of_l with one instruction
// fewer.
template <int MODE>
__device__ __forceinline__ float quake_of_l_below(float l) {
  uint32_t z;
  asm("v_cvt_u32_f32 %0, %1" : "=v"(z) : "v"(l));
  return quake_of_z<MODE>(z);
}

// e^(p x + q) with c0, c1 folded on the host (Eq. 5). EXACT: the same fused
// binary32 argument in base 2, exponentiated by the hardware v_exp_f32.
template <int MODE>
__device__ __forceinline__ float qexp(float x, float c0, float c1) {
  const float l = __builtin_fmaf(x, c0, c1);
  if constexpr (MODE == EXACT) {
    return __builtin_amdgcn_exp2f(l);
  } else {
    return quake_of_l<MODE>(l);
  }
}

// qexp for Algorithm 2's exponentials, x <= the row max m: with BELOW (every
// lane's |c1| < 2^54, see quake_of_l_below) the clamp is folded into the
// conversion.
template <int MODE, bool BELOW>
__device__ __forceinline__ float qexp_row(float x, float c0, float c1) {
  if constexpr (MODE == EXACT || !BELOW) {
    return qexp<MODE>(x, c0, c1);
  } else {
    return quake_of_l_below<MODE>(__builtin_fmaf(x, c0, c1));
  }
}
// whether every lane of the wave may take qexp_row<MODE, true> with its c1
__device__ __forceinline__ bool row_c1_below(float c1) {
  return __all(__builtin_fabsf(c1) < 0x1p54f) != 0;
}

// num / (1 + e) with one v_rcp_f32. Both operands are scaled by 1/4 (exact
// in binary32) so that the reciprocal of 1 + e stays a normal number for every
// finite e (v_rcp_f32 flushes subnormal results): (num/4) * rcp((1 + e)/4),
// where (1 + e)/4 = fma(e, 1/4, 1/4) is exactly the rounded 1 + e scaled.
__device__ __forceinline__ float div_one_plus(float num, float e) {
  return (num * 0.25f) * __builtin_amdgcn_rcpf(__builtin_fmaf(e, 0.25f, 0.25f));
}

// GELU through Eq. 7: u = fma(x, x, 1/0.044715), w = x u, y = x / (1 + QuAKEx(w))
// with the folded constants c0 = -2^23 2 0.044715 sqrt(2/pi) / ln2 and c1.
template <int MODE>
__device__ __forceinline__ float gelu_q(float x, float c0, float c1, float a) {
  const float u = __builtin_fmaf(x, x, a);
  const float w = x * u;
  return div_one_plus(x, qexp<MODE>(w, c0, c1));
}

// ---------------------------------------------------------------------------
// Element formats. A 16-byte vector holds kV<DT> elements.
// ---------------------------------------------------------------------------
template <int DT>
constexpr int kV = (DT == F32) ? 4 : 8;
template <int DT>
constexpr int kEsz = (DT == F32) ? 4 : 2;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return as_f(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return as_f(w & 0xFFFF0000u); }
__device__ __forceinline__ float f16_lo(uint32_t w) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));
}
__device__ __forceinline__ float f16_hi(uint32_t w) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}

// Round-to-nearest-even narrowing of two binary32 values into one dword, one
// instruction each (v_cvt_pk_bf16_f32 / v_cvt_pk_f16_f32); converting the
// halves separately costs two conversions plus a shift-and-or per pair.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2_t));
}

template <int DT>
__device__ __forceinline__ void unpack(const u32x4 v, float* f) {
  if constexpr (DT == F32) {
#pragma unroll
    for (int k = 0; k < 4; ++k) f[k] = as_f(v[k]);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      f[2 * k] = (DT == BF16) ? bf16_lo(v[k]) : f16_lo(v[k]);
      f[2 * k + 1] = (DT == BF16) ? bf16_hi(v[k]) : f16_hi(v[k]);
    }
  }
}

template <int DT>
__device__ __forceinline__ u32x4 pack(const float* f) {
  u32x4 v;
  if constexpr (DT == F32) {
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = as_u(f[k]);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      v[k] = (DT == BF16) ? pack_bf16(f[2 * k], f[2 * k + 1]) : pack_f16(f[2 * k], f[2 * k + 1]);
  }
  return v;
}

// The 16 bytes that start d bytes into the aligned vector a and continue into
// the next aligned vector b (d uniform, 0 <= d < 16): one v_alignbyte per
// dword, so an unaligned run of memory is read as aligned vectors.
__device__ __forceinline__ u32x4 realign(const u32x4& a, const u32x4& b, uint32_t d) {
  const uint32_t w[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  const uint32_t rb = d & 3u;
  u32x4 o;
  auto take = [&](auto wq) {
    constexpr int Q = decltype(wq)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = __builtin_amdgcn_alignbyte(w[j + Q + 1], w[j + Q], rb);
  };
  switch (d >> 2) {
    case 0: take(std::integral_constant<int, 0>{}); break;
    case 1: take(std::integral_constant<int, 1>{}); break;
    case 2: take(std::integral_constant<int, 2>{}); break;
    default: take(std::integral_constant<int, 3>{}); break;
  }
  return o;
}

// The aligned vectors a and b that hold the 16 bytes starting d bytes into
// vector i of xa (d > 0): every lane loads its own a (past the last vector,
// the one after it, which still holds bytes of the operand) and takes b from
// the next lane (ds_bpermute), so each aligned vector is fetched once; the
// wave's last lane loads its b. Every lane of the wave must call this.
__device__ __forceinline__ void aligned_pair(const u32x4* xa, uint32_t i, uint32_t nvec, u32x4& a,
                                             u32x4& b) {
  a = __builtin_nontemporal_load(xa + (i < nvec ? i : nvec));
  const int src = (int)((((threadIdx.x & 63u) + 1u) & 63u) << 2);
#pragma unroll
  for (int j = 0; j < 4; ++j) b[j] = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)a[j]);
  if ((threadIdx.x & 63u) == 63u) b = __builtin_nontemporal_load(xa + (i + 1 < nvec ? i + 1 : nvec));
}

// A 16-byte vector of -inf in each format (masked lanes of a softmax row).
template <int DT>
__device__ __forceinline__ u32x4 neg_inf_vec() {
  constexpr uint32_t w = (DT == F32) ? 0xFF800000u : (DT == F16 ? 0xFC00FC00u : 0xFF80FF80u);
  const u32x4 v = {w, w, w, w};
  return v;
}

template <int DT>
__device__ __forceinline__ float load1(const void* p, int64_t i) {
  if constexpr (DT == F32) {
    return static_cast<const float*>(p)[i];
  } else {
    const uint16_t h = static_cast<const uint16_t*>(p)[i];
    return (DT == BF16) ? as_f((uint32_t)h << 16) : (float)__builtin_bit_cast(_Float16, h);
  }
}

template <int DT>
__device__ __forceinline__ void store1(void* p, int64_t i, float v) {
  if constexpr (DT == F32) {
    static_cast<float*>(p)[i] = v;
  } else if constexpr (DT == BF16) {
    static_cast<uint16_t*>(p)[i] = __builtin_bit_cast(uint16_t, (__bf16)v);
  } else {
    static_cast<uint16_t*>(p)[i] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

// ---------------------------------------------------------------------------
// 64-lane reductions. Four DPP steps make every lane of a 16-lane row hold the
// row's result (xor 1, xor 2 via quad_perm; xor 4 via row_half_mirror; xor 8
// via row_mirror); then row_bcast:15 combines rows 0 and 1 into row 1 and rows
// 2 and 3 into row 3, and row_bcast:31 row 1 into row 3, so lane 63 holds
// op(op(r0, r1), op(r2, r3)), the same tree (and, addition being commutative,
// the same bits) as combining the four row results pairwise; one v_readlane
// hands it to every lane. All 64 lanes must be active.
// ---------------------------------------------------------------------------
constexpr int kDppXor1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;   // row_half_mirror
constexpr int kDppMirror = 0x140;       // row_mirror
constexpr int kDppRowBcast15 = 0x142;   // lane 15 of each row to the next row
constexpr int kDppRowBcast31 = 0x143;   // lane 31 to rows 2 and 3

// v of the lane CTRL names; lanes of rows not in ROWS (or whose source is
// invalid) get `old`
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWS, 0xF, false);
}

template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ float dpp_f32(float v) {
  return as_f(dpp_u32<CTRL, ROWS>(0u, as_u(v)));
}

template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = dpp_u32<CTRL, ROWS>(0u, (uint32_t)u);
  const uint32_t hi = dpp_u32<CTRL, ROWS>(0u, (uint32_t)(u >> 32));
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ float readlane_f32(float v, int lane) {
  return as_f((uint32_t)__builtin_amdgcn_readlane((int)as_u(v), lane));
}

__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), lane);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// The wave maximum runs on order-preserving integer images of the values: a
// binary32 pattern with its magnitude bits flipped when negative compares as a
// signed int32 exactly as the floats compare (NaN aside), so each step is one
// v_max_i32 with a DPP operand. A float max would need the DPP value quieted
// (IEEE mode) first.
__device__ __forceinline__ int32_t ord_key(float v) {
  const int32_t u = (int32_t)as_u(v);
  return u ^ (int32_t)((uint32_t)(u >> 31) >> 1);
}
__device__ __forceinline__ float ord_val(int32_t k) {
  return as_f((uint32_t)(k ^ (int32_t)((uint32_t)(k >> 31) >> 1)));
}
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ int32_t dpp_max_i32(int32_t k) {
  const int32_t o = (int32_t)dpp_u32<CTRL, ROWS>((uint32_t)INT32_MIN, (uint32_t)k);
  return k > o ? k : o;
}

__device__ __forceinline__ float wave_max(float v) {
  int32_t k = ord_key(v);
  k = dpp_max_i32<kDppXor1>(k);
  k = dpp_max_i32<kDppXor2>(k);
  k = dpp_max_i32<kDppHalfMirror>(k);
  k = dpp_max_i32<kDppMirror>(k);
  k = dpp_max_i32<kDppRowBcast15, 0xA>(k);
  k = dpp_max_i32<kDppRowBcast31, 0xC>(k);
  return ord_val(__builtin_amdgcn_readlane(k, 63));
}

__device__ __forceinline__ float wave_sum_f32(float v) {
  v += dpp_f32<kDppXor1>(v);
  v += dpp_f32<kDppXor2>(v);
  v += dpp_f32<kDppHalfMirror>(v);
  v += dpp_f32<kDppMirror>(v);
  v += dpp_f32<kDppRowBcast15, 0xA>(v);   // rows 0 and 2 add the 0 `old`
  v += dpp_f32<kDppRowBcast31, 0xC>(v);
  return readlane_f32(v, 63);
}

__device__ __forceinline__ double wave_sum(double v) {
  v += dpp_f64<kDppXor1>(v);
  v += dpp_f64<kDppXor2>(v);
  v += dpp_f64<kDppHalfMirror>(v);
  v += dpp_f64<kDppMirror>(v);
  v += dpp_f64<kDppRowBcast15, 0xA>(v);
  v += dpp_f64<kDppRowBcast31, 0xC>(v);
  return readlane_f64(v, 63);
}

}  // namespace qk
