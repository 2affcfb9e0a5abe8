// elementwise.hip — quake_exp, quake_gelu, quake_sigmoid (Logistic / SiLU).
//
// One streaming kernel per (format, operator, mode): every lane moves UNROLL
// 16-byte vectors (4 binary32 or 8 binary16/bfloat16 elements each), all
// loads issued before any arithmetic, with non-temporal loads and stores (the
// data is touched once). A wave reads 1 KiB contiguous per load instruction.
// Elements past the last whole vector are handled by the last workgroup's
// first lanes with scalar accesses. Buffers that are not 16-byte aligned take
// a scalar grid-stride kernel with the same per-element arithmetic.
//
// Per-element arithmetic (Sec. III-A, III-B, III-D of arXiv:2412.00408):
//   exp      y = QuAKEx(x; c0, c1)                     (Eq. 5, Alg. 1)
//   GELU     u = fma(x, x, 1/0.044715); w = x*u; e = QuAKEx(w); y = x/(1+e)   (Eq. 7)
//   Logistic e = QuAKEx(x; -2^23/ln2, c1); y = 1/(1+e)
//   SiLU     y = x/(1+e)
#include <hip/hip_runtime.h>

#include <algorithm>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

enum Op : int { OP_EXP = 0, OP_GELU = 1, OP_SIGMOID = 2, OP_SILU = 3 };

struct EwParams {
  float c0, c1, a;  // folded constants; `a` is the FMA addend of GELU
};

template <int OP, int MODE>
__device__ __forceinline__ float ew_op(float x, const EwParams& p) {
  if constexpr (OP == OP_EXP) {
    return qexp<MODE>(x, p.c0, p.c1);
  } else if constexpr (OP == OP_GELU) {
    const float u = __builtin_fmaf(x, x, p.a);
    const float w = x * u;
    return div_one_plus(x, qexp<MODE>(w, p.c0, p.c1));
  } else if constexpr (OP == OP_SIGMOID) {
    return __builtin_amdgcn_rcpf(1.0f + qexp<MODE>(x, p.c0, p.c1));
  } else {
    return div_one_plus(x, qexp<MODE>(x, p.c0, p.c1));
  }
}

constexpr int kEwBlock = 256;

template <int DT, int OP, int MODE, int UNROLL>
__global__ __launch_bounds__(kEwBlock) void ew_vec_kernel(const u32x4* __restrict__ x,
                                                         u32x4* __restrict__ y, uint32_t nvec,
                                                         uint32_t tail, EwParams p) {
  constexpr int V = kV<DT>;
  const uint32_t base = blockIdx.x * (kEwBlock * UNROLL) + threadIdx.x;
  u32x4 v[UNROLL];
#pragma unroll
  for (int u = 0; u < UNROLL; ++u) {
    const uint32_t i = base + u * kEwBlock;
    if (i < nvec) v[u] = __builtin_nontemporal_load(x + i);
  }
#pragma unroll
  for (int u = 0; u < UNROLL; ++u) {
    const uint32_t i = base + u * kEwBlock;
    if (i < nvec) {
      float f[V];
      unpack<DT>(v[u], f);
#pragma unroll
      for (int k = 0; k < V; ++k) f[k] = ew_op<OP, MODE>(f[k], p);
      __builtin_nontemporal_store(pack<DT>(f), y + i);
    }
  }
  if (tail && blockIdx.x == gridDim.x - 1 && threadIdx.x < tail) {
    const int64_t e = (int64_t)nvec * V + threadIdx.x;
    store1<DT>(y, e, ew_op<OP, MODE>(load1<DT>(x, e), p));
  }
}

template <int DT, int OP, int MODE>
__global__ __launch_bounds__(kEwBlock) void ew_scalar_kernel(const void* __restrict__ x,
                                                            void* __restrict__ y, uint32_t n,
                                                            EwParams p) {
  for (uint32_t i = blockIdx.x * kEwBlock + threadIdx.x; i < n; i += gridDim.x * kEwBlock)
    store1<DT>(y, i, ew_op<OP, MODE>(load1<DT>(x, i), p));
}

constexpr int kEwUnroll = 2;
// Elements per launch: a multiple of every vector width, below 2^31.
constexpr int64_t kEwChunk = int64_t(1) << 30;

template <int DT, int OP, int MODE>
quake_status ew_launch(const void* x, void* y, int64_t n, const EwParams& p, hipStream_t s) {
  constexpr int V = kV<DT>;
  constexpr int64_t esz = kEsz<DT>;
  const bool vec = aligned16(x) && aligned16(y);
  for (int64_t off = 0; off < n; off += kEwChunk) {
    const int64_t m = std::min(kEwChunk, n - off);
    const char* xc = static_cast<const char*>(x) + off * esz;
    char* yc = static_cast<char*>(y) + off * esz;
    if (vec) {
      const uint32_t nvec = (uint32_t)(m / V);
      const uint32_t tail = (uint32_t)(m % V);
      const int64_t per_block = (int64_t)kEwBlock * kEwUnroll;
      uint32_t grid = (uint32_t)((nvec + per_block - 1) / per_block);
      if (grid == 0) grid = 1;
      hipLaunchKernelGGL((ew_vec_kernel<DT, OP, MODE, kEwUnroll>), dim3(grid), dim3(kEwBlock), 0,
                         s, reinterpret_cast<const u32x4*>(xc), reinterpret_cast<u32x4*>(yc),
                         nvec, tail, p);
    } else {
      const int64_t want = (m + kEwBlock - 1) / kEwBlock;
      const uint32_t grid = (uint32_t)std::min<int64_t>(want, 65536);
      hipLaunchKernelGGL((ew_scalar_kernel<DT, OP, MODE>), dim3(grid), dim3(kEwBlock), 0, s, xc,
                         yc, (uint32_t)m, p);
    }
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

template <int OP>
quake_status ew_dispatch(const void* x, void* y, int64_t n, int dt, int mode, const EwParams& p,
                         hipStream_t s) {
#define QK_EW_CASE(D, M) \
  if (dt == D && mode == M) return ew_launch<D, OP, M>(x, y, n, p, s);
  QK_EW_CASE(F32, EXACT) QK_EW_CASE(F32, Q1) QK_EW_CASE(F32, Q2)
  QK_EW_CASE(F16, EXACT) QK_EW_CASE(F16, Q1) QK_EW_CASE(F16, Q2)
  QK_EW_CASE(BF16, EXACT) QK_EW_CASE(BF16, Q1) QK_EW_CASE(BF16, Q2)
#undef QK_EW_CASE
  return QUAKE_EMODE;
}

static quake_status ew_check(const void* x, void* y, int64_t n, int dt, int mode) {
  if (!valid_dtype(dt)) return QUAKE_EDTYPE;
  if (!valid_mode(mode)) return QUAKE_EMODE;
  if (n < 0) return QUAKE_EINVAL;
  if (n > 0 && (x == nullptr || y == nullptr)) return QUAKE_EINVAL;
  return QUAKE_OK;
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_exp(const void* x, void* y, int64_t n, quake_dtype dtype,
                                  quake_mode mode, float a, float b, void* stream) {
  quake_status st = ew_check(x, y, n, dtype, mode);
  if (st != QUAKE_OK) return st;
  if (!std::isfinite(a) || !std::isfinite(b)) return QUAKE_EINVAL;
  const Affine af = exp_affine(a, b, mode);
  if (!std::isfinite(af.c0) || !std::isfinite(af.c1)) return QUAKE_EINVAL;
  if (n == 0) return QUAKE_OK;
  return ew_dispatch<OP_EXP>(x, y, n, dtype, mode, EwParams{af.c0, af.c1, 0.0f},
                             static_cast<hipStream_t>(stream));
}

extern "C" quake_status quake_gelu(const void* x, void* y, int64_t n, quake_dtype dtype,
                                   quake_mode mode, void* stream) {
  quake_status st = ew_check(x, y, n, dtype, mode);
  if (st != QUAKE_OK || n == 0) return st;
  const Affine af = gelu_affine(mode);
  return ew_dispatch<OP_GELU>(x, y, n, dtype, mode, EwParams{af.c0, af.c1, gelu_a()},
                              static_cast<hipStream_t>(stream));
}

extern "C" quake_status quake_sigmoid(const void* x, void* y, int64_t n, quake_dtype dtype,
                                      quake_mode mode, int silu, void* stream) {
  quake_status st = ew_check(x, y, n, dtype, mode);
  if (st != QUAKE_OK || n == 0) return st;
  const Affine af = sigmoid_affine(mode);
  const EwParams p{af.c0, af.c1, 0.0f};
  hipStream_t s = static_cast<hipStream_t>(stream);
  return silu ? ew_dispatch<OP_SILU>(x, y, n, dtype, mode, p, s)
              : ew_dispatch<OP_SIGMOID>(x, y, n, dtype, mode, p, s);
}
