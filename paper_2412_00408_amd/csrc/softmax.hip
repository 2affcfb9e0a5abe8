// softmax.hip — quake_softmax: row-wise softmax(t * x), Algorithm 2 of
// arXiv:2412.00408 (SoftMax-QuAKEx), for gfx950.
//
// Algorithm 2 per row: m = max_j x_j; c0 = 2^23 t / ln2; c1 = 127*2^23 - c0 m;
// y_j = QuAKEx(x_j; c0, c1); y_j /= sum_j y_j. The temperature and the max
// subtraction are folded into c0 and c1, so each element costs one fma plus
// the bit construction. Every exponent of a row uses the row's final max.
//
// Kernels (all one read of x and one write of y from HBM):
//   sm_rows<NV, WAVES=1>  one wave per row, the row held in VGPRs as NV
//                         16-byte vectors per lane (rows up to 64*NV vectors);
//                         4 rows per 256-thread workgroup, no LDS, no barrier.
//   sm_rows<NV, WAVES=4>  one workgroup per row (rows up to 256*NV vectors),
//                         cross-wave max/sum through LDS.
//   sm_split<NV>          rows longer than a workgroup's registers: G
//                         workgroups per row each hold one chunk in VGPRs and
//                         exchange their chunk max, then their chunk sum,
//                         through a small device workspace (two arrivals on a
//                         per-row counter). The launch is cooperative, so all
//                         workgroups are co-resident and every wait ends; each
//                         wait is also bounded by a spin limit.
//   sm_generic            any alignment / stride / length: one workgroup per
//                         row, three passes (max, sum, normalise) with scalar
//                         accesses; the re-reads are served by the caches.
// Sums: fp32 within one 16-byte vector (at most 8 terms), then double across
// vectors, lanes, waves and workgroups, in a fixed order.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <utility>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

constexpr int kSmBlock = 256;

// Per-row c1 of Algorithm 2: fma(-c0, m, 127*2^23) (EXACT: -c0*m in base 2).
template <int MODE>
__device__ __forceinline__ float row_c1(float c0, float m) {
  if (m == -INFINITY) return 0.0f;   // fully masked row: every y_j becomes 0
  return __builtin_fmaf(-c0, m, MODE == EXACT ? 0.0f : kK127);
}

// ---------------------------------------------------------------------------
// Register-resident rows: one wave (WAVES = 1) or one workgroup (WAVES = 4).
// ---------------------------------------------------------------------------
template <int DT, int MODE, int NV, int WAVES>
__global__ __launch_bounds__(kSmBlock) void sm_rows_kernel(const char* __restrict__ x,
                                                          char* __restrict__ y, uint32_t rows,
                                                          uint32_t nvr, int64_t ldx_b,
                                                          int64_t ldy_b, float c0) {
  constexpr int V = kV<DT>;
  constexpr int LANES = 64 * WAVES;
  constexpr int ROWS_PER_BLOCK = kSmBlock / LANES;
  __shared__ float s_max[4];
  __shared__ double s_sum[4];

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lid = threadIdx.x % LANES;
  const uint32_t row = blockIdx.x * ROWS_PER_BLOCK + threadIdx.x / LANES;
  if (WAVES == 1 && row >= rows) return;   // uniform per wave

  const u32x4* xr = reinterpret_cast<const u32x4*>(x + (int64_t)row * ldx_b);
  u32x4* yr = reinterpret_cast<u32x4*>(y + (int64_t)row * ldy_b);

  // Every lane loads (vectors past the row end re-read the row's last vector,
  // which stays in one cache line) and padding lanes select -inf: no branch
  // around the loads, so the whole row stays in registers without merges.
  u32x4 raw[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k)
    raw[k] = __builtin_nontemporal_load(xr + umin32(k * LANES + lid, nvr - 1));
  float f[NV][V];
  float lmax = -INFINITY;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    unpack<DT>(raw[k], f[k]);
    const bool valid = k * LANES + lid < nvr;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      f[k][j] = valid ? f[k][j] : -INFINITY;
      lmax = fmaxf(lmax, f[k][j]);
    }
  }

  float m = wave_max(lmax);
  if constexpr (WAVES > 1) {
    if (lane == 0) s_max[wave] = m;
    __syncthreads();
    m = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
  }

  const float c1 = row_c1<MODE>(c0, m);
  double acc = 0.0;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      f[k][j] = qexp<MODE>(f[k][j], c0, c1);
      part += f[k][j];
    }
    acc += (double)part;
  }
  double total = wave_sum(acc);
  if constexpr (WAVES > 1) {
    if (lane == 0) s_sum[wave] = total;
    __syncthreads();
    total = (s_sum[0] + s_sum[1]) + (s_sum[2] + s_sum[3]);
  }
  const float r = (m == -INFINITY) ? 0.0f : (float)(1.0 / total);

#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = k * LANES + lid;
    if (vi < nvr) {
#pragma unroll
      for (int j = 0; j < V; ++j) f[k][j] *= r;
      __builtin_nontemporal_store(pack<DT>(f[k]), yr + vi);
    }
  }
}

// ---------------------------------------------------------------------------
// Split rows: G workgroups per row, exchanging chunk max and chunk sum.
// ---------------------------------------------------------------------------
struct SplitWs {
  float* pmax;      // [slots]   chunk maxima, index rr * G + g
  double* psum;     // [slots]   chunk sums
  uint32_t* cnt;    // [slots]   per-row arrival counters (zero between launches)
  uint32_t* err;    // [1]       set if a wait hit its spin limit
};

constexpr uint32_t kWsSlots = 8192;          // max rows * G per launch
constexpr uint32_t kSpinLimit = 1u << 20;    // about a second of polling; never reached when co-resident
constexpr int kMaxG = kSmBlock;              // chunk exchange goes through one LDS slot per lane

__device__ __forceinline__ void arrive_and_wait(uint32_t* cnt, uint32_t target, uint32_t* err) {
  __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  uint32_t spins = 0;
  while (__hip_atomic_load(cnt, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
    __builtin_amdgcn_s_sleep(1);
    if (++spins == kSpinLimit) {
      __hip_atomic_store(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
  }
}

template <int DT, int MODE, int NV>
__global__ __launch_bounds__(kSmBlock) void sm_split_kernel(const char* __restrict__ x,
                                                           char* __restrict__ y, uint32_t nvr,
                                                           int64_t ldx_b, int64_t ldy_b, float c0,
                                                           uint32_t G, SplitWs ws) {
  constexpr int V = kV<DT>;
  constexpr int CHV = kSmBlock * NV;   // vectors per chunk
  __shared__ float s_max[4];
  __shared__ double s_sum[4];
  __shared__ float s_pmax[kMaxG];
  __shared__ double s_psum[kMaxG];

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const uint32_t rr = blockIdx.x / G;
  const uint32_t g = blockIdx.x - rr * G;
  const uint32_t slot = rr * G + g;

  const u32x4* xr = reinterpret_cast<const u32x4*>(x + (int64_t)rr * ldx_b);
  u32x4* yr = reinterpret_cast<u32x4*>(y + (int64_t)rr * ldy_b);
  const uint32_t v0 = g * CHV;

  u32x4 raw[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k)
    raw[k] = __builtin_nontemporal_load(xr + umin32(v0 + k * kSmBlock + threadIdx.x, nvr - 1));
  float f[NV][V];
  float lmax = -INFINITY;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    unpack<DT>(raw[k], f[k]);
    const bool valid = v0 + k * kSmBlock + threadIdx.x < nvr;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      f[k][j] = valid ? f[k][j] : -INFINITY;
      lmax = fmaxf(lmax, f[k][j]);
    }
  }
  float m = wave_max(lmax);
  if (lane == 0) s_max[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    m = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
    __hip_atomic_store(&ws.pmax[slot], m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    arrive_and_wait(&ws.cnt[rr], G, ws.err);
  }
  __syncthreads();
  if (threadIdx.x < G)
    s_pmax[threadIdx.x] =
        __hip_atomic_load(&ws.pmax[rr * G + threadIdx.x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  m = -INFINITY;
  for (uint32_t q = 0; q < G; ++q) m = fmaxf(m, s_pmax[q]);

  const float c1 = row_c1<MODE>(c0, m);
  double acc = 0.0;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      f[k][j] = qexp<MODE>(f[k][j], c0, c1);
      part += f[k][j];
    }
    acc += (double)part;
  }
  double total = wave_sum(acc);
  if (lane == 0) s_sum[wave] = total;
  __syncthreads();
  if (threadIdx.x == 0) {
    total = (s_sum[0] + s_sum[1]) + (s_sum[2] + s_sum[3]);
    __hip_atomic_store(reinterpret_cast<uint64_t*>(&ws.psum[slot]),
                       __builtin_bit_cast(uint64_t, total), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    arrive_and_wait(&ws.cnt[rr], 2 * G, ws.err);
  }
  __syncthreads();
  if (threadIdx.x < G)
    s_psum[threadIdx.x] = __builtin_bit_cast(
        double, __hip_atomic_load(reinterpret_cast<uint64_t*>(&ws.psum[rr * G + threadIdx.x]),
                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  __syncthreads();
  if (threadIdx.x == 0) {
    // third arrival: this workgroup has finished reading the workspace; the
    // last one of the row returns the counter to zero for the next launch.
    const uint32_t old = __hip_atomic_fetch_add(&ws.cnt[rr], 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    if (old == 3 * G - 1) __hip_atomic_store(&ws.cnt[rr], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  total = 0.0;
  for (uint32_t q = 0; q < G; ++q) total += s_psum[q];
  const float r = (m == -INFINITY) ? 0.0f : (float)(1.0 / total);

#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = v0 + k * kSmBlock + threadIdx.x;
    if (vi < nvr) {
#pragma unroll
      for (int j = 0; j < V; ++j) f[k][j] *= r;
      __builtin_nontemporal_store(pack<DT>(f[k]), yr + vi);
    }
  }
}

__global__ void zero_u32_kernel(uint32_t* p, uint32_t n) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// ---------------------------------------------------------------------------
// Generic rows: any alignment, stride and length.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float block_max(float v, float* s) {
  v = wave_max(v);
  if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
}

__device__ __forceinline__ double block_sum(double v, double* s) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = v;
  __syncthreads();
  return (s[0] + s[1]) + (s[2] + s[3]);
}

template <int DT, int MODE>
__global__ __launch_bounds__(kSmBlock) void sm_generic_kernel(const void* __restrict__ x,
                                                             void* __restrict__ y, int64_t rows,
                                                             int64_t cols, int64_t ldx,
                                                             int64_t ldy, float c0) {
  __shared__ float s_max[4];
  __shared__ double s_sum[4];
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const int64_t bx = row * ldx, by = row * ldy;
    float lm = -INFINITY;
    for (int64_t j = threadIdx.x; j < cols; j += kSmBlock) lm = fmaxf(lm, load1<DT>(x, bx + j));
    const float m = block_max(lm, s_max);
    const float c1 = row_c1<MODE>(c0, m);
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < cols; j += kSmBlock)
      acc += (double)qexp<MODE>(load1<DT>(x, bx + j), c0, c1);
    const double total = block_sum(acc, s_sum);
    const float r = (m == -INFINITY) ? 0.0f : (float)(1.0 / total);
    for (int64_t j = threadIdx.x; j < cols; j += kSmBlock)
      store1<DT>(y, by + j, qexp<MODE>(load1<DT>(x, bx + j), c0, c1) * r);
    __syncthreads();   // s_max / s_sum are rewritten for the next row
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
struct WsKey {
  int dev;
  hipStream_t stream;
  bool operator<(const WsKey& o) const {
    return dev != o.dev ? dev < o.dev : (uintptr_t)stream < (uintptr_t)o.stream;
  }
};

static std::mutex g_ws_mu;
static std::map<WsKey, SplitWs> g_ws;

// Workspace of the split kernel for (current device, stream): allocated and
// zeroed on first use, kept until the process ends. Launches on one stream
// are ordered, so they may share it; different streams get their own.
static quake_status split_workspace(hipStream_t s, SplitWs* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return QUAKE_EHIP;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  auto it = g_ws.find(WsKey{dev, s});
  if (it != g_ws.end()) {
    *out = it->second;
    return QUAKE_OK;
  }
  const size_t n_pmax = kWsSlots * sizeof(float), n_psum = kWsSlots * sizeof(double);
  const size_t n_cnt = (kWsSlots + 64) * sizeof(uint32_t);
  char* base = nullptr;
  if (hipMalloc(&base, n_psum + n_pmax + n_cnt) != hipSuccess) return QUAKE_EHIP;
  SplitWs w;
  w.psum = reinterpret_cast<double*>(base);
  w.pmax = reinterpret_cast<float*>(base + n_psum);
  w.cnt = reinterpret_cast<uint32_t*>(base + n_psum + n_pmax);
  w.err = w.cnt + kWsSlots;
  hipLaunchKernelGGL(zero_u32_kernel, dim3(8), dim3(256), 0, s, w.cnt, kWsSlots + 64);
  if (hipGetLastError() != hipSuccess) return QUAKE_EHIP;
  g_ws.emplace(WsKey{dev, s}, w);
  *out = w;
  return QUAKE_OK;
}

// Co-resident workgroups of one kernel on the current device.
template <typename K>
static int coresident_blocks(K kernel) {
  int dev = 0, nb = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, kSmBlock, 0) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return nb * cus;
}

struct SmArgs {
  const char* x;
  char* y;
  int64_t rows, cols, ldx_b, ldy_b;
  float c0;
  hipStream_t s;
};

constexpr int64_t kRowChunk = int64_t(1) << 28;   // rows per launch (grid stays < 2^31)

template <int DT, int MODE, int NV, int WAVES>
static quake_status launch_rows(const SmArgs& a) {
  constexpr int V = kV<DT>;
  constexpr int RPB = kSmBlock / (64 * WAVES);
  const uint32_t nvr = (uint32_t)(a.cols / V);
  for (int64_t r0 = 0; r0 < a.rows; r0 += kRowChunk) {
    const int64_t nr = std::min(kRowChunk, a.rows - r0);
    const uint32_t grid = (uint32_t)((nr + RPB - 1) / RPB);
    hipLaunchKernelGGL((sm_rows_kernel<DT, MODE, NV, WAVES>), dim3(grid), dim3(kSmBlock), 0, a.s,
                       a.x + r0 * a.ldx_b, a.y + r0 * a.ldy_b, (uint32_t)nr, nvr, a.ldx_b, a.ldy_b,
                       a.c0);
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

template <int DT, int MODE>
static quake_status launch_generic(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                                   int64_t ldy, float c0, hipStream_t s) {
  const uint32_t grid = (uint32_t)std::min<int64_t>(rows, int64_t(1) << 20);
  hipLaunchKernelGGL((sm_generic_kernel<DT, MODE>), dim3(grid), dim3(kSmBlock), 0, s, x, y, rows,
                     cols, ldx, ldy, c0);
  return launch_status();
}

// Returns QUAKE_OK on success, or 1 + status on failure; -1 if the split path
// cannot be used (too many chunks per row) and the caller should fall back.
template <int DT, int MODE, int NV>
static int launch_split(const SmArgs& a) {
  constexpr int V = kV<DT>;
  constexpr int CHV = kSmBlock * NV;
  const uint32_t nvr = (uint32_t)(a.cols / V);
  const uint32_t G = (nvr + CHV - 1) / CHV;
  auto kern = sm_split_kernel<DT, MODE, NV>;
  static int cached[64] = {0};   // per device; a benign race only recomputes it
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 1 + QUAKE_EHIP;
  int cap = (dev >= 0 && dev < 64) ? cached[dev] : 0;
  if (cap == 0) {
    cap = std::min<int>(coresident_blocks(kern), (int)kWsSlots);
    if (dev >= 0 && dev < 64) cached[dev] = cap;
  }
  if (G > (uint32_t)kMaxG || cap < (int)G) return -1;
  SplitWs ws;
  quake_status st = split_workspace(a.s, &ws);
  if (st != QUAKE_OK) return 1 + st;
  const int64_t rows_per_launch = cap / G;
  for (int64_t r0 = 0; r0 < a.rows; r0 += rows_per_launch) {
    const int64_t nr = std::min(rows_per_launch, a.rows - r0);
    const char* xp = a.x + r0 * a.ldx_b;
    char* yp = a.y + r0 * a.ldy_b;
    int64_t ldx_b = a.ldx_b, ldy_b = a.ldy_b;
    float c0 = a.c0;
    uint32_t g = G;
    void* args[] = {&xp, &yp, const_cast<uint32_t*>(&nvr), &ldx_b, &ldy_b, &c0, &g, &ws};
    if (hipLaunchCooperativeKernel(reinterpret_cast<const void*>(kern), dim3((uint32_t)(nr * G)),
                                   dim3(kSmBlock), args, 0, a.s) != hipSuccess)
      return 1 + QUAKE_EHIP;
    st = launch_status();
    if (st != QUAKE_OK) return 1 + st;
  }
  return QUAKE_OK;
}

template <int DT, int MODE>
static quake_status sm_dispatch(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                                int64_t ldy, float c0, hipStream_t s) {
  constexpr int V = kV<DT>;
  constexpr int64_t esz = kEsz<DT>;
  const bool vec = aligned16(x) && aligned16(y) && (ldx * esz) % 16 == 0 && (ldy * esz) % 16 == 0 &&
                   cols % V == 0 && cols / V < (int64_t(1) << 30);
  if (!vec) return launch_generic<DT, MODE>(x, y, rows, cols, ldx, ldy, c0, s);
  const SmArgs a{static_cast<const char*>(x), static_cast<char*>(y), rows, cols, ldx * esz,
                 ldy * esz, c0, s};
  const int64_t nvr = cols / V;
  if (nvr <= 64) return launch_rows<DT, MODE, 1, 1>(a);
  if (nvr <= 128) return launch_rows<DT, MODE, 2, 1>(a);
  if (nvr <= 256) return launch_rows<DT, MODE, 4, 1>(a);
  if (nvr <= 512) return launch_rows<DT, MODE, 8, 1>(a);
  if (nvr <= 1024) return launch_rows<DT, MODE, 4, 4>(a);
  if (nvr <= 2048) return launch_rows<DT, MODE, 8, 4>(a);
  const int rc = launch_split<DT, MODE, 8>(a);
  if (rc >= 0) return rc == 0 ? QUAKE_OK : (quake_status)(rc - 1);
  return launch_generic<DT, MODE>(x, y, rows, cols, ldx, ldy, c0, s);
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_softmax(const void* x, void* y, int64_t rows, int64_t cols,
                                      int64_t ldx, int64_t ldy, quake_dtype dtype,
                                      quake_mode mode, float t, void* stream) {
  if (!valid_dtype(dtype)) return QUAKE_EDTYPE;
  if (!valid_mode(mode)) return QUAKE_EMODE;
  if (rows < 0 || cols < 0 || ldx < 0 || ldy < 0) return QUAKE_EINVAL;
  if (rows == 0) return QUAKE_OK;
  if (cols == 0 || ldx < cols || ldy < cols || x == nullptr || y == nullptr) return QUAKE_EINVAL;
  if (!std::isfinite(t) || !(t > 0.0f)) return QUAKE_EINVAL;
  const float c0 = softmax_c0(t, mode);
  if (!std::isfinite(c0) || c0 == 0.0f) return QUAKE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
#define QK_SM_CASE(D, M) \
  if ((int)dtype == D && (int)mode == M) return sm_dispatch<D, M>(x, y, rows, cols, ldx, ldy, c0, s);
  QK_SM_CASE(F32, EXACT) QK_SM_CASE(F32, Q1) QK_SM_CASE(F32, Q2)
  QK_SM_CASE(F16, EXACT) QK_SM_CASE(F16, Q1) QK_SM_CASE(F16, Q2)
  QK_SM_CASE(BF16, EXACT) QK_SM_CASE(BF16, Q1) QK_SM_CASE(BF16, Q2)
#undef QK_SM_CASE
  return QUAKE_EMODE;
}
