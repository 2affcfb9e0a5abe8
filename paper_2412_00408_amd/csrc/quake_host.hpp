// quake_host.hpp — host-side helpers of libquake: the folded constants of
// QuAKE (each evaluated in double from its definition and rounded once to
// binary32), argument validation, and launch bookkeeping.
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "quake.h"

namespace qk {

constexpr double kLn2 = 0.693147180559945309417232121458176568;
constexpr double kTwo23 = 8388608.0;      // 2^l_m, l_m = 23 (Sec. II-A)
constexpr double kBias = 127.0;           // B (Sec. II-A)
constexpr double kSchraudolph = 0.0436;   // bias of first-order QuAKE (Sec. III-A)
constexpr double kGeluC = 0.044715;       // Eq. 4
constexpr double kPi = 3.14159265358979323846264338327950288;

// The two constants of one QuAKE call (Eq. 5), or of its EXACT counterpart
// (the same affine map in base 2 without the 2^23 scale and 127 offset).
struct Affine {
  float c0, c1;
};

// e^(a x + b): p = a / ln2, q = b / ln2 in Eq. 5.
inline Affine exp_affine(double a, double b, int mode) {
  if (mode == QUAKE_EXACT) return {(float)(a / kLn2), (float)(b / kLn2)};
  const double beta = (mode == QUAKE_1) ? kSchraudolph : 0.0;
  return {(float)((a / kLn2) * kTwo23), (float)(((kBias - beta) + b / kLn2) * kTwo23)};
}

// Scale of the logistic argument in Eq. 7: 2 * 0.044715 * sqrt(2/pi).
inline double gelu_k() { return 2.0 * kGeluC * std::sqrt(2.0 / kPi); }

// 1/0.044715 + x^2 is one FMA with this addend (Eq. 7).
inline float gelu_a() { return (float)(1.0 / kGeluC); }

// e^(-k w) for w = x (1/0.044715 + x^2): Eq. 5 with p = -k.
inline Affine gelu_affine(int mode) { return exp_affine(-gelu_k(), 0.0, mode); }

// e^(-x) of the logistic function: Eq. 5 with p = -1.
inline Affine sigmoid_affine(int mode) { return exp_affine(-1.0, 0.0, mode); }

// Algorithm 2: c0 = 2^23 t / ln2 (EXACT: t / ln2); c1 is per row on the GPU.
inline float softmax_c0(double t, int mode) {
  if (mode == QUAKE_EXACT) return (float)(t / kLn2);
  return (float)((t / kLn2) * kTwo23);
}

inline bool valid_dtype(int d) { return d == QUAKE_F32 || d == QUAKE_F16 || d == QUAKE_BF16; }
inline bool valid_mode(int m) {
  return m == QUAKE_EXACT || m == QUAKE_1 || m == QUAKE_2 || m == QUAKE_2M;
}
inline int64_t elem_size(int d) { return d == QUAKE_F32 ? 4 : 2; }

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

inline quake_status launch_status() {
  return hipGetLastError() == hipSuccess ? QUAKE_OK : QUAKE_EHIP;
}

}  // namespace qk
