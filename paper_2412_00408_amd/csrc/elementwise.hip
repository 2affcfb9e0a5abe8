// elementwise.hip — quake_exp, quake_gelu, quake_sigmoid (Logistic / SiLU).
//
// Streaming kernels per (format, operator, mode) over 16-byte vectors (4
// binary32 or 8 binary16/bfloat16 elements), with non-temporal loads and
// stores (the data is touched once); a wave reads 1 KiB contiguous per load
// instruction. Two launch shapes, chosen by size: a one-shot grid with one
// vector per lane for large inputs, and a resident, software-pipelined
// grid-stride loop for mid-size ones (where launch ramp and tail dominate).
// Elements past the last whole vector are handled by one workgroup's first
// lanes with scalar accesses. Buffers that are not both 16-byte aligned take
// a kernel that writes y in aligned vectors, each assembled from the aligned
// vectors of x that hold its bytes, with scalar accesses before y's first
// 16-byte boundary and after its last whole vector.
//
// Per-element arithmetic (Sec. III-A, III-B, III-D of arXiv:2412.00408):
//   exp      y = QuAKEx(x; c0, c1)                     (Eq. 5, Alg. 1)
//   GELU     u = fma(x, x, 1/0.044715); w = x*u; e = QuAKEx(w); y = x/(1+e)   (Eq. 7)
//   Logistic e = QuAKEx(x; -2^23/ln2, c1); y = 1/(1+e)
//   SiLU     y = x/(1+e)
//   GELU, unfused (the fusion study of Sec. V-A / Table IV): s = k*w with
//            k = 2*0.044715*sqrt(2/pi), e = e^-s through the standard constants
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

enum Op : int { OP_EXP = 0, OP_GELU = 1, OP_SIGMOID = 2, OP_SILU = 3, OP_GELU_UNFUSED = 4 };

struct EwParams {
  float c0, c1;  // constants of the exponential (folded, or the standard e^s)
  float a;       // FMA addend of GELU, 1/0.044715
  float k;       // unfused GELU only: scale 2*0.044715*sqrt(2/pi) applied before e^-s
};

template <int OP, int MODE>
__device__ __forceinline__ float ew_op(float x, const EwParams& p) {
  if constexpr (OP == OP_EXP) {
    return qexp<MODE>(x, p.c0, p.c1);
  } else if constexpr (OP == OP_GELU) {
    return gelu_q<MODE>(x, p.c0, p.c1, p.a);
  } else if constexpr (OP == OP_SIGMOID) {
    return __builtin_amdgcn_rcpf(1.0f + qexp<MODE>(x, p.c0, p.c1));
  } else if constexpr (OP == OP_SILU) {
    return div_one_plus(x, qexp<MODE>(x, p.c0, p.c1));
  } else {
    // plug-in form of the fusion study: s = k * w, then the standard e^-s
    const float u = __builtin_fmaf(x, x, p.a);
    const float w = x * u;
    const float sk = w * p.k;
    return div_one_plus(x, qexp<MODE>(-sk, p.c0, p.c1));
  }
}

constexpr int kEwBlock = 256;

// Large inputs: one 16-byte vector per lane, one workgroup per 256 vectors.
// Workgroups are retired and replaced continuously, which keeps the most
// requests in flight once the grid is many times the resident capacity.
template <int DT, int OP, int MODE>
__global__ __launch_bounds__(kEwBlock) void ew_oneshot_kernel(const u32x4* __restrict__ x,
                                                             u32x4* __restrict__ y, uint32_t nvec,
                                                             uint32_t tail, EwParams p) {
  constexpr int V = kV<DT>;
  const uint32_t i = blockIdx.x * kEwBlock + threadIdx.x;
  if (i < nvec) {
    const u32x4 v = __builtin_nontemporal_load(x + i);
    float f[V];
    unpack<DT>(v, f);
#pragma unroll
    for (int k = 0; k < V; ++k) f[k] = ew_op<OP, MODE>(f[k], p);
    __builtin_nontemporal_store(pack<DT>(f), y + i);
  }
  if (tail && blockIdx.x == gridDim.x - 1 && threadIdx.x < tail) {
    const int64_t e = (int64_t)nvec * V + threadIdx.x;
    store1<DT>(y, e, ew_op<OP, MODE>(load1<DT>(x, e), p));
  }
}

// Mid-size inputs: a resident grid (a few workgroups per CU) strides over the
// vectors, two per lane per step, and issues the next step's loads before the
// current step's arithmetic so every lane always has loads in flight.
template <int DT, int OP, int MODE>
__global__ __launch_bounds__(kEwBlock) void ew_pipe_kernel(const u32x4* __restrict__ x,
                                                          u32x4* __restrict__ y, uint32_t nvec,
                                                          uint32_t tail, EwParams p) {
  constexpr int V = kV<DT>;
  constexpr int U = 2;
  const uint32_t step = gridDim.x * (kEwBlock * U);
  uint32_t base = blockIdx.x * (kEwBlock * U) + threadIdx.x;
  u32x4 cur[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t i = base + u * kEwBlock;
    if (i < nvec) cur[u] = __builtin_nontemporal_load(x + i);
  }
  while (base < nvec) {
    const uint32_t nb = base + step;
    u32x4 nxt[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = nb + u * kEwBlock;
      if (i < nvec) nxt[u] = __builtin_nontemporal_load(x + i);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = base + u * kEwBlock;
      if (i < nvec) {
        float f[V];
        unpack<DT>(cur[u], f);
#pragma unroll
        for (int k = 0; k < V; ++k) f[k] = ew_op<OP, MODE>(f[k], p);
        __builtin_nontemporal_store(pack<DT>(f), y + i);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) cur[u] = nxt[u];
    base = nb;
  }
  if (tail && blockIdx.x == 0 && threadIdx.x < tail) {
    const int64_t e = (int64_t)nvec * V + threadIdx.x;
    store1<DT>(y, e, ew_op<OP, MODE>(load1<DT>(x, e), p));
  }
}

// Buffers that are not both 16-byte aligned: y is written in aligned 16-byte
// vectors, each built from the two aligned vectors of x that hold its bytes
// (d bytes into the first, d a multiple of the element size, uniform; d = 0
// when x and y sit at the same offset, and then one vector), so every access
// is an aligned vector access: an aligned vector never crosses a page, and a
// lane's second load is the next lane's first (served by the cache). The
// elements before y's first 16-byte boundary (head) and after its last whole
// vector (tail) take scalar accesses in the first and the last workgroup.
template <int DT, int OP, int MODE>
__global__ __launch_bounds__(kEwBlock) void ew_realign_kernel(const void* __restrict__ x,
                                                             void* __restrict__ y, uint32_t head,
                                                             uint32_t nvec, uint32_t tail,
                                                             uint32_t d, EwParams p) {
  constexpr int V = kV<DT>;
  constexpr int64_t esz = kEsz<DT>;
  // x's element at y's first 16-byte boundary sits d bytes past xa's start
  const u32x4* xa = reinterpret_cast<const u32x4*>(static_cast<const char*>(x) + head * esz - d);
  u32x4* ya = reinterpret_cast<u32x4*>(static_cast<char*>(y) + head * esz);
  const uint32_t i = blockIdx.x * kEwBlock + threadIdx.x;
  // d = 0 (x and y at the same offset): the vector is a itself, and the next
  // aligned vector of x may lie past its end; else a and b from aligned_pair
  u32x4 a, b;
  if (d == 0) {
    if (i < nvec) a = __builtin_nontemporal_load(xa + i);
    b = a;
  } else {
    aligned_pair(xa, i, nvec, a, b);
  }
  if (i < nvec) {
    float f[V];
    unpack<DT>(realign(a, b, d), f);
#pragma unroll
    for (int k = 0; k < V; ++k) f[k] = ew_op<OP, MODE>(f[k], p);
    __builtin_nontemporal_store(pack<DT>(f), ya + i);
  }
  if (blockIdx.x == 0 && threadIdx.x < head)
    store1<DT>(y, threadIdx.x, ew_op<OP, MODE>(load1<DT>(x, threadIdx.x), p));
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x < tail) {
    const int64_t e = (int64_t)head + (int64_t)nvec * V + threadIdx.x;
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

// Elements per launch: a multiple of every vector width, below 2^31.
constexpr int64_t kEwChunk = int64_t(1) << 30;
// Resident workgroups per CU for the strided kernel.
constexpr int kEwPipeBlocksPerCu = 8;
// At or above this many vectors per CU the one-shot kernel is used.
constexpr int64_t kEwOneShotVecPerCu = 64 * kEwBlock;

// Compute units of the current device (the runtime answers from its cached
// device properties; nothing is kept here).
static int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

template <int DT, int OP, int MODE>
quake_status ew_launch(const void* x, void* y, int64_t n, const EwParams& p, hipStream_t s) {
  constexpr int V = kV<DT>;
  constexpr int64_t esz = kEsz<DT>;
  const uintptr_t ux = (uintptr_t)x, uy = (uintptr_t)y;
  // not both 16-byte aligned (element-aligned): y in aligned vectors, each
  // assembled from aligned vectors of x, scalar head and tail, one launch
  if (((ux | uy) & 15u) != 0 && ux % esz == 0 && uy % esz == 0 && n >= 2 * V &&
      n < (int64_t(1) << 31)) {
    const int64_t head = (int64_t)((16u - (uy & 15u)) & 15u) / esz;
    const int64_t nvec = (n - head) / V, tail = (n - head) % V;
    const uint32_t d = (uint32_t)((ux + head * esz) & 15u);
    const uint32_t grid = (uint32_t)std::max<int64_t>(1, (nvec + kEwBlock - 1) / kEwBlock);
    hipLaunchKernelGGL((ew_realign_kernel<DT, OP, MODE>), dim3(grid), dim3(kEwBlock), 0, s, x, y,
                       (uint32_t)head, (uint32_t)nvec, (uint32_t)tail, d, p);
    return launch_status();
  }
  // x and y at the same offset from a 16-byte boundary, beyond that length
  // range: the few elements before the first boundary take the scalar
  // kernel, the rest the vector kernels.
  if ((ux & 15u) != 0 && ((ux - uy) & 15u) == 0 && ux % esz == 0) {
    const int64_t head = std::min<int64_t>(n, (int64_t)((16u - (ux & 15u)) & 15u) / esz);
    hipLaunchKernelGGL((ew_scalar_kernel<DT, OP, MODE>), dim3(1), dim3(kEwBlock), 0, s, x, y,
                       (uint32_t)head, p);
    const quake_status st = launch_status();
    if (st != QUAKE_OK || head == n) return st;
    return ew_launch<DT, OP, MODE>(static_cast<const char*>(x) + head * esz,
                                   static_cast<char*>(y) + head * esz, n - head, p, s);
  }
  const bool vec = aligned16(x) && aligned16(y);
  const int cus = device_cus();
  for (int64_t off = 0; off < n; off += kEwChunk) {
    const int64_t m = std::min(kEwChunk, n - off);
    const char* xc = static_cast<const char*>(x) + off * esz;
    char* yc = static_cast<char*>(y) + off * esz;
    if (vec) {
      const uint32_t nvec = (uint32_t)(m / V);
      const uint32_t tail = (uint32_t)(m % V);
      const u32x4* xv = reinterpret_cast<const u32x4*>(xc);
      u32x4* yv = reinterpret_cast<u32x4*>(yc);
      if ((int64_t)nvec >= kEwOneShotVecPerCu * cus) {
        const uint32_t grid = (uint32_t)((nvec + kEwBlock - 1) / kEwBlock);
        hipLaunchKernelGGL((ew_oneshot_kernel<DT, OP, MODE>), dim3(grid), dim3(kEwBlock), 0, s, xv,
                           yv, nvec, tail, p);
      } else {
        const int64_t want = ((int64_t)nvec + 2 * kEwBlock - 1) / (2 * kEwBlock);
        const uint32_t grid =
            (uint32_t)std::max<int64_t>(1, std::min<int64_t>(want, (int64_t)kEwPipeBlocksPerCu * cus));
        hipLaunchKernelGGL((ew_pipe_kernel<DT, OP, MODE>), dim3(grid), dim3(kEwBlock), 0, s, xv, yv,
                           nvec, tail, p);
      }
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
  QK_EW_CASE(F32, EXACT) QK_EW_CASE(F32, Q1) QK_EW_CASE(F32, Q2) QK_EW_CASE(F32, Q2M)
  QK_EW_CASE(F16, EXACT) QK_EW_CASE(F16, Q1) QK_EW_CASE(F16, Q2) QK_EW_CASE(F16, Q2M)
  QK_EW_CASE(BF16, EXACT) QK_EW_CASE(BF16, Q1) QK_EW_CASE(BF16, Q2) QK_EW_CASE(BF16, Q2M)
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
  return ew_dispatch<OP_EXP>(x, y, n, dtype, mode, EwParams{af.c0, af.c1, 0.0f, 0.0f},
                             static_cast<hipStream_t>(stream));
}

extern "C" quake_status quake_gelu(const void* x, void* y, int64_t n, quake_dtype dtype,
                                   quake_mode mode, void* stream) {
  quake_status st = ew_check(x, y, n, dtype, mode);
  if (st != QUAKE_OK || n == 0) return st;
  const Affine af = gelu_affine(mode);
  return ew_dispatch<OP_GELU>(x, y, n, dtype, mode, EwParams{af.c0, af.c1, gelu_a(), 0.0f},
                              static_cast<hipStream_t>(stream));
}

extern "C" quake_status quake_gelu_unfused(const void* x, void* y, int64_t n, quake_dtype dtype,
                                           quake_mode mode, void* stream) {
  quake_status st = ew_check(x, y, n, dtype, mode);
  if (st != QUAKE_OK || n == 0) return st;
  const Affine af = exp_affine(1.0, 0.0, mode);   // the standard e^s
  return ew_dispatch<OP_GELU_UNFUSED>(x, y, n, dtype, mode,
                                      EwParams{af.c0, af.c1, gelu_a(), (float)gelu_k()},
                                      static_cast<hipStream_t>(stream));
}

extern "C" quake_status quake_sigmoid(const void* x, void* y, int64_t n, quake_dtype dtype,
                                      quake_mode mode, int silu, void* stream) {
  quake_status st = ew_check(x, y, n, dtype, mode);
  if (st != QUAKE_OK || n == 0) return st;
  const Affine af = sigmoid_affine(mode);
  const EwParams p{af.c0, af.c1, 0.0f, 0.0f};
  hipStream_t s = static_cast<hipStream_t>(stream);
  return silu ? ew_dispatch<OP_SILU>(x, y, n, dtype, mode, p, s)
              : ew_dispatch<OP_SIGMOID>(x, y, n, dtype, mode, p, s);
}
