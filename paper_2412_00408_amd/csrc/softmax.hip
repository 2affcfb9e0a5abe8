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
//   sm_rows<NV, WAVES=4>  one workgroup per row (rows up to 256*NV vectors, i.e.
//                         16384 elements), cross-wave max/sum through LDS.
//   sm_split<NV>          rows longer than a workgroup's registers: G
//                         workgroups per row each hold one chunk in VGPRs and
//                         exchange their chunk max, then their chunk sum,
//                         through sentinel slots of a small device workspace
//                         (relaxed atomics, no fences). A launch never has more
//                         workgroups than fit on the device at once, so every
//                         wait ends; each wait is also bounded by a spin limit.
//   sm_generic            any alignment / stride / length: one workgroup per
//                         row, three passes (max, sum, normalise) with scalar
//                         accesses; the re-reads are served by the caches.
// Sums: fp32 within one 16-byte vector (at most 8 terms), then, in a fixed
// order, double across vectors, lanes, waves and workgroups for binary32
// outputs and fp32 for 16-bit outputs (double across split workgroups).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <map>
#include <mutex>
#include <utility>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

constexpr int kSmBlock = 256;

// Row sums: binary32 outputs accumulate in double across vectors, lanes and
// waves (the 1e-6 relative tolerance leaves no room for a long fp32 chain) and
// divide in double; 16-bit outputs accumulate in fp32 (error below 2^-20
// relative, far under half an ulp of the output) and take one v_rcp_f32.
template <int DT>
struct AccOf {
  typedef float T;
};
template <>
struct AccOf<F32> {
  typedef double T;
};
__device__ __forceinline__ double wave_sum_acc(double v) { return wave_sum(v); }
__device__ __forceinline__ float wave_sum_acc(float v) { return wave_sum_f32(v); }
__device__ __forceinline__ float inv_total(double t) { return (float)(1.0 / t); }
__device__ __forceinline__ float inv_total(float t) { return __builtin_amdgcn_rcpf(t); }

// Per-row c1 of Algorithm 2: fma(-c0, m, 127*2^23) (EXACT: -c0*m in base 2).
template <int MODE>
__device__ __forceinline__ float row_c1(float c0, float m) {
  if (m == -INFINITY) return 0.0f;   // fully masked row: every y_j becomes 0
  return __builtin_fmaf(-c0, m, MODE == EXACT ? 0.0f : kK127);
}

// Constants of one softmax call. Fused (Algorithm 2): c0 = 2^23 t / ln2 and
// the per-row c1. Unfused (the plug-in form of the fusion study, Sec. V-A /
// Table IV): s = (v - m) * t in binary32, then the standard exponential with
// c0 = 2^23 / ln2, c1 = c1s (EXACT: c0 = fl(1/ln2), c1 = 0).
struct SmConst {
  float c0, c1s, t;
};

template <int MODE, bool FUSE>
struct RowExp {
  float c0, c1, m, t;
  __device__ __forceinline__ float operator()(float v) const {
    if constexpr (FUSE) {
      return qexp<MODE>(v, c0, c1);
    } else {
      const float d = v - m;
      return qexp<MODE>(d * t, c0, c1);
    }
  }
};

template <int MODE, bool FUSE>
__device__ __forceinline__ RowExp<MODE, FUSE> row_exp(const SmConst& k, float m) {
  if constexpr (FUSE) {
    return RowExp<MODE, FUSE>{k.c0, row_c1<MODE>(k.c0, m), 0.0f, 0.0f};
  } else {
    return RowExp<MODE, FUSE>{k.c0, k.c1s, m == -INFINITY ? 0.0f : m, k.t};
  }
}

// Implicit causal mask: row r (global index) uses only its first
// L = clamp(r mod period + shift + 1, 0, cols) entries; the rest are not
// read and give 0, exactly what -inf entries give. row0_mod = (index of the
// launch's first row) mod period, so r mod period = (row0_mod + local) mod period.
struct CausalArg {
  uint32_t row0_mod, period;
  int64_t shift;
  uint32_t write_masked;   // 0: masked outputs are not stored
};

template <bool CAUSAL>
__device__ __forceinline__ int64_t live_len(const CausalArg& ca, uint32_t local_row, int64_t cols) {
  if constexpr (!CAUSAL) {
    return cols;
  } else {
    const int64_t r = (int64_t)((ca.row0_mod + local_row) % ca.period);
    const int64_t L = r + ca.shift + 1;
    return L < 0 ? 0 : (L > cols ? cols : L);
  }
}

// ---------------------------------------------------------------------------
// Register-resident rows: one wave (WAVES = 1) or one workgroup (WAVES = 4).
// ---------------------------------------------------------------------------
template <int DT, int MODE, bool FUSE, bool CAUSAL, int NV, int WAVES>
__global__ __launch_bounds__(kSmBlock) void sm_rows_kernel(const char* __restrict__ x,
                                                          char* __restrict__ y, uint32_t rows,
                                                          uint32_t nvr, int64_t ldx_b,
                                                          int64_t ldy_b, SmConst kc,
                                                          CausalArg ca) {
  constexpr int V = kV<DT>;
  constexpr int LANES = 64 * WAVES;
  constexpr int ROWS_PER_BLOCK = kSmBlock / LANES;
  using Acc = typename AccOf<DT>::T;
  __shared__ float s_max[4];
  __shared__ Acc s_sum[4];

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
  // With the causal mask only vectors holding live entries are read.
  const uint32_t L = (uint32_t)live_len<CAUSAL>(ca, row, (int64_t)nvr * V);
  const uint32_t nvl = CAUSAL ? (L + V - 1) / V : nvr;
  const uint32_t vlast = (nvl > 0 ? nvl : 1) - 1;
  u32x4 raw[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) raw[k] = __builtin_nontemporal_load(xr + umin32(k * LANES + lid, vlast));
  float f[NV][V];
  float lmax = -INFINITY;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = k * LANES + lid;
    // whole vectors past the row end become -inf before widening (one select
    // per word); only the causal boundary needs a per-element mask
    if (!CAUSAL && vi >= nvr) raw[k] = neg_inf_vec<DT>();
    unpack<DT>(raw[k], f[k]);
#pragma unroll
    for (int j = 0; j < V; ++j) {
      if constexpr (CAUSAL) f[k][j] = (vi * V + j < L) ? f[k][j] : -INFINITY;
      lmax = fmaxf(lmax, f[k][j]);
    }
  }

  float m = wave_max(lmax);
  if constexpr (WAVES > 1) {
    if (lane == 0) s_max[wave] = m;
    __syncthreads();
    m = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
  }

  const RowExp<MODE, FUSE> ex = row_exp<MODE, FUSE>(kc, m);
  Acc acc = 0;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      f[k][j] = ex(f[k][j]);
      part += f[k][j];
    }
    acc += (Acc)part;
  }
  Acc total = wave_sum_acc(acc);
  if constexpr (WAVES > 1) {
    if (lane == 0) s_sum[wave] = total;
    __syncthreads();
    total = (s_sum[0] + s_sum[1]) + (s_sum[2] + s_sum[3]);
  }
  const float r = (m == -INFINITY) ? 0.0f : inv_total(total);

#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = k * LANES + lid;
    if (vi < nvr && (!CAUSAL || ca.write_masked || vi < nvl)) {
#pragma unroll
      for (int j = 0; j < V; ++j) f[k][j] *= r;
      __builtin_nontemporal_store(pack<DT>(f[k]), yr + vi);
    }
  }
}

// ---------------------------------------------------------------------------
// Square causal blocks (period = cols = P, shift = 0): row r of a block has
// r + 1 live entries, so a wave that owns one row leaves most lanes idle in
// the block's upper rows. Here a wave owns two rows whose live vectors fit its
// 64 lanes together: r and M - 1 - r, with M = P - K and K = max(0, P - 63 V)
// (then ceil((r+1)/V) + ceil((M-r)/V) <= 64). Lanes [0, nA) hold row A's live
// vectors and lanes [nA, nA + nB) row B's; max and sum are reduced per row
// over its own lanes (the other lanes contribute the identity). Row B's
// partial sums are first rotated down by nA lanes (ds_bpermute), so both rows
// are summed over lanes 0, 1, ... in the one-row kernel's reduction tree and
// the results are bit-identical to it. Rows M .. P-1, and the middle row
// when M is odd, take a wave alone. Masked entries are neither read nor
// computed; with write_masked their outputs are stored as zeros.
// ---------------------------------------------------------------------------
// v of lane (lane + k) mod 64, for every lane (ds_bpermute).
__device__ __forceinline__ float lane_rotate(float v, uint32_t k) {
  const int src = (int)((((uint32_t)(threadIdx.x & 63) + k) & 63u) << 2);
  return as_f((uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)as_u(v)));
}
__device__ __forceinline__ double lane_rotate(double v, uint32_t k) {
  const int src = (int)((((uint32_t)(threadIdx.x & 63) + k) & 63u) << 2);
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)(uint32_t)u);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)(uint32_t)(u >> 32));
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

struct PairArg {
  uint32_t P;        // rows per block = cols
  uint32_t M;        // rows [0, M) are paired r <-> M - 1 - r
  uint32_t J;        // jobs (waves) per block: M / 2 + (M & 1) + (P - M)
  uint32_t jobs;     // jobs in this launch (whole blocks)
  uint32_t write_masked;
};

template <int DT, int MODE, bool FUSE>
__global__ __launch_bounds__(kSmBlock) void sm_causal_pair_kernel(const char* __restrict__ x,
                                                                 char* __restrict__ y,
                                                                 int64_t ldx_b, int64_t ldy_b,
                                                                 SmConst kc, PairArg pa) {
  constexpr int V = kV<DT>;
  using Acc = typename AccOf<DT>::T;
  const int lane = threadIdx.x & 63;
  const uint32_t job = blockIdx.x * (kSmBlock / 64) + (threadIdx.x >> 6);
  if (job >= pa.jobs) return;   // uniform per wave

  const uint32_t blk = job / pa.J;
  const uint32_t j = job - blk * pa.J;
  const uint32_t npairs = pa.M / 2;
  uint32_t rA, rB = 0;
  const bool pair = j < npairs;
  if (pair) {
    rA = j;
    rB = pa.M - 1 - j;
  } else {
    const uint32_t s = j - npairs;
    rA = (pa.M & 1) ? (s == 0 ? npairs : pa.M + s - 1) : pa.M + s;
  }
  const uint32_t nvr = pa.P / V;
  const uint32_t LA = rA + 1, LB = pair ? rB + 1 : 0;
  const uint32_t nA = (LA + V - 1) / V, nB = (LB + V - 1) / V;
  const bool inA = (uint32_t)lane < nA;
  const bool inB = !inA && (uint32_t)lane - nA < nB;
  // idle lanes re-read row A's last live vector (in bounds, no branch)
  const uint32_t row = inB ? rB : rA;
  const uint32_t vi = inA ? (uint32_t)lane : (inB ? (uint32_t)lane - nA : nA - 1);
  const uint32_t Lrow = inB ? LB : ((inA) ? LA : 0);

  const int64_t grow = (int64_t)blk * pa.P + row;
  const u32x4* xr = reinterpret_cast<const u32x4*>(x + grow * ldx_b);
  const u32x4 raw = __builtin_nontemporal_load(xr + vi);
  float f[V];
  unpack<DT>(raw, f);
  float lmax = -INFINITY;
#pragma unroll
  for (int e = 0; e < V; ++e) {
    f[e] = (vi * V + e < Lrow) ? f[e] : -INFINITY;
    lmax = fmaxf(lmax, f[e]);
  }
  const float mA = wave_max(inA ? lmax : -INFINITY);
  const float mB = pair ? wave_max(inB ? lmax : -INFINITY) : -INFINITY;
  const float m = inB ? mB : mA;

  const RowExp<MODE, FUSE> ex = row_exp<MODE, FUSE>(kc, m);
  float part = 0.0f;
#pragma unroll
  for (int e = 0; e < V; ++e) {
    f[e] = ex(f[e]);
    part += f[e];
  }
  const Acc acc = (Acc)part;
  const Acc tA = wave_sum_acc(inA ? acc : (Acc)0);
  const Acc tB = pair ? wave_sum_acc(lane_rotate(inB ? acc : (Acc)0, nA)) : (Acc)0;
  const float r = (m == -INFINITY) ? 0.0f : inv_total(inB ? tB : tA);

  if (inA || inB) {
    u32x4* yr = reinterpret_cast<u32x4*>(y + grow * ldy_b);
#pragma unroll
    for (int e = 0; e < V; ++e) f[e] *= r;
    __builtin_nontemporal_store(pack<DT>(f), yr + vi);
  }
  if (pa.write_masked) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    const int64_t gA = (int64_t)blk * pa.P + rA;
    if (nA + lane < nvr)
      __builtin_nontemporal_store(z, reinterpret_cast<u32x4*>(y + gA * ldy_b) + nA + lane);
    if (pair && nB + lane < nvr) {
      const int64_t gB = (int64_t)blk * pa.P + rB;
      __builtin_nontemporal_store(z, reinterpret_cast<u32x4*>(y + gB * ldy_b) + nB + lane);
    }
  }
}

// ---------------------------------------------------------------------------
// Split rows: G workgroups per row, exchanging chunk max and chunk sum.
//
// Exchange without fences: every chunk owns one 32-bit slot for its max and
// one 64-bit slot for its sum, both holding a sentinel between launches. A
// workgroup publishes its value with a relaxed agent-scope atomic store and
// polls the G slots of its row with relaxed agent-scope atomic loads until no
// sentinel is left. The value is itself the atomic object, so no release /
// acquire fence (and no L2 write-back or invalidate) is needed. After reading
// both rounds each workgroup counts itself done; the last one of the row puts
// the sentinels back, so the workspace is ready for the next launch (also on
// graph replay). Launches use at most as many workgroups as can be resident
// at once, so every polled value is eventually written; every wait is also
// bounded by a spin limit and then flags an error instead of hanging.
// ---------------------------------------------------------------------------
struct SplitWs {
  uint32_t* pmax;        // [kWsSlots]  chunk maxima (binary32 bits), index rr * G + g
  uint64_t* psum;        // [kWsSlots]  chunk sums (binary64 bits)
  uint32_t* done;        // [kWsSlots]  per-row count of finished workgroups
  uint32_t* err;         // [1]         number of waits that hit their spin limit
  uint32_t spin_limit;   // polls before a wait gives up
  uint32_t withhold;     // test hook: chunk 0 of every row never publishes
};

constexpr uint32_t kWsSlots = 8192;                 // max rows * G per launch
constexpr uint32_t kSpinLimit = 1u << 20;           // about a second of polling
constexpr uint32_t kTestSpinLimit = 1u << 12;       // short limit while a fault is injected
constexpr int kMaxG = kSmBlock;                     // one polling lane per chunk
constexpr uint32_t kSent32 = 0xFFFFFFFFu;           // a NaN never published
constexpr uint64_t kSent64 = 0xFFFFFFFFFFFFFFFFull; // a NaN never published

template <typename T>
__device__ __forceinline__ T poll_slot(T* slot, T sentinel, T fallback, const SplitWs& ws) {
  T v;
  uint32_t spins = 0;
  while ((v = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) == sentinel) {
    __builtin_amdgcn_s_sleep(1);
    if (++spins >= ws.spin_limit) {
      __hip_atomic_fetch_add(ws.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return fallback;
    }
  }
  return v;
}

template <int DT, int MODE, bool FUSE, bool CAUSAL, int NV>
__global__ __launch_bounds__(kSmBlock) void sm_split_kernel(const char* __restrict__ x,
                                                           char* __restrict__ y, uint32_t nvr,
                                                           int64_t ldx_b, int64_t ldy_b,
                                                           SmConst kc, CausalArg ca, uint32_t G,
                                                           SplitWs ws) {
  constexpr int V = kV<DT>;
  constexpr int CHV = kSmBlock * NV;   // vectors per chunk
  __shared__ float s_max[4];
  __shared__ double s_sum[4];
  __shared__ float s_pmax[kMaxG];
  __shared__ double s_psum[kMaxG];

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  // Chunk g of row rr. blockIdx round-robins over the 8 XCDs; with the rows a
  // multiple of 8, XCD x takes rows x, x + 8, ... with all their chunks, so a
  // row's exchange stays among the workgroups of one XCD.
  uint32_t rr, g;
  if ((gridDim.x / G) % 8u == 0) {
    const uint32_t sl = blockIdx.x >> 3;
    rr = (blockIdx.x & 7u) + 8u * (sl / G);
    g = sl % G;
  } else {
    rr = blockIdx.x / G;
    g = blockIdx.x - rr * G;
  }
  uint32_t* pm = ws.pmax + rr * G;
  uint64_t* ps = ws.psum + rr * G;

  const u32x4* xr = reinterpret_cast<const u32x4*>(x + (int64_t)rr * ldx_b);
  u32x4* yr = reinterpret_cast<u32x4*>(y + (int64_t)rr * ldy_b);
  const uint32_t v0 = g * CHV;

  const uint32_t L = (uint32_t)live_len<CAUSAL>(ca, rr, (int64_t)nvr * V);
  const uint32_t nvl = CAUSAL ? (L + V - 1) / V : nvr;
  const uint32_t vlast = (nvl > 0 ? nvl : 1) - 1;
  u32x4 raw[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k)
    raw[k] = __builtin_nontemporal_load(xr + umin32(v0 + k * kSmBlock + threadIdx.x, vlast));
  float f[NV][V];
  float lmax = -INFINITY;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = v0 + k * kSmBlock + threadIdx.x;
    if (!CAUSAL && vi >= nvr) raw[k] = neg_inf_vec<DT>();
    unpack<DT>(raw[k], f[k]);
#pragma unroll
    for (int j = 0; j < V; ++j) {
      if constexpr (CAUSAL) f[k][j] = (vi * V + j < L) ? f[k][j] : -INFINITY;
      lmax = fmaxf(lmax, f[k][j]);
    }
  }

  // first exchange: the chunk maxima
  float m = wave_max(lmax);
  if (lane == 0) s_max[wave] = m;
  __syncthreads();
  const bool publish = !(ws.withhold && g == 0);
  if (threadIdx.x == 0 && publish) {
    m = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
    const uint32_t mb = (m != m) ? as_u(-INFINITY) : as_u(m);
    __hip_atomic_store(pm + g, mb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (threadIdx.x < G)
    s_pmax[threadIdx.x] = as_f(poll_slot<uint32_t>(pm + threadIdx.x, kSent32, as_u(-INFINITY), ws));
  __syncthreads();
  m = -INFINITY;
  for (uint32_t q = 0; q < G; ++q) m = fmaxf(m, s_pmax[q]);

  // second exchange: the chunk sums against the row's final max
  const RowExp<MODE, FUSE> ex = row_exp<MODE, FUSE>(kc, m);
  double acc = 0.0;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      f[k][j] = ex(f[k][j]);
      part += f[k][j];
    }
    acc += (double)part;
  }
  double total = wave_sum(acc);
  if (lane == 0) s_sum[wave] = total;
  __syncthreads();
  if (threadIdx.x == 0 && publish) {
    total = (s_sum[0] + s_sum[1]) + (s_sum[2] + s_sum[3]);
    const uint64_t tb = (total != total) ? 0x7FF8000000000000ull : __builtin_bit_cast(uint64_t, total);
    __hip_atomic_store(ps + g, tb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (threadIdx.x < G)
    s_psum[threadIdx.x] = __builtin_bit_cast(double, poll_slot<uint64_t>(ps + threadIdx.x, kSent64, 0, ws));
  __syncthreads();
  if (threadIdx.x == 0) {
    // This workgroup has read both rounds (the values are in LDS); the last
    // workgroup of the row restores the sentinels for the next launch.
    const uint32_t old = __hip_atomic_fetch_add(ws.done + rr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == G - 1) {
      for (uint32_t q = 0; q < G; ++q) {
        __hip_atomic_store(pm + q, kSent32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(ps + q, kSent64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __hip_atomic_store(ws.done + rr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  total = 0.0;
  for (uint32_t q = 0; q < G; ++q) total += s_psum[q];
  const float r = (m == -INFINITY) ? 0.0f : (float)(1.0 / total);

#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = v0 + k * kSmBlock + threadIdx.x;
    if (vi < nvr && (!CAUSAL || ca.write_masked || vi < nvl)) {
#pragma unroll
      for (int j = 0; j < V; ++j) f[k][j] *= r;
      __builtin_nontemporal_store(pack<DT>(f[k]), yr + vi);
    }
  }
}

__global__ void split_ws_init_kernel(SplitWs w, uint32_t n) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    w.pmax[i] = kSent32;
    w.psum[i] = kSent64;
    w.done[i] = 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *w.err = 0;
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

template <int DT, int MODE, bool FUSE, bool CAUSAL>
__global__ __launch_bounds__(kSmBlock) void sm_generic_kernel(const void* __restrict__ x,
                                                             void* __restrict__ y, int64_t rows,
                                                             int64_t cols, int64_t ldx,
                                                             int64_t ldy, SmConst kc,
                                                             CausalArg ca) {
  __shared__ float s_max[4];
  __shared__ double s_sum[4];
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const int64_t bx = row * ldx, by = row * ldy;
    const int64_t L = live_len<CAUSAL>(ca, (uint32_t)row, cols);
    float lm = -INFINITY;
    for (int64_t j = threadIdx.x; j < L; j += kSmBlock) lm = fmaxf(lm, load1<DT>(x, bx + j));
    const float m = block_max(lm, s_max);
    const RowExp<MODE, FUSE> ex = row_exp<MODE, FUSE>(kc, m);
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < L; j += kSmBlock) acc += (double)ex(load1<DT>(x, bx + j));
    const double total = block_sum(acc, s_sum);
    const float r = (m == -INFINITY) ? 0.0f : (float)(1.0 / total);
    const int64_t jend = (CAUSAL && !ca.write_masked) ? L : cols;
    for (int64_t j = threadIdx.x; j < jend; j += kSmBlock)
      store1<DT>(y, by + j, j < L ? ex(load1<DT>(x, bx + j)) * r : 0.0f);
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
static std::atomic<int> g_test_fault{0};

// Workspace of the split kernel for (current device, stream): allocated and
// filled with sentinels on first use (on that stream), kept until the process
// ends. Launches on one stream are ordered, so they may share it; different
// streams get their own.
static quake_status split_workspace(hipStream_t s, SplitWs* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return QUAKE_EHIP;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  const bool fault = g_test_fault.load(std::memory_order_relaxed) != 0;
  auto it = g_ws.find(WsKey{dev, s});
  if (it != g_ws.end()) {
    *out = it->second;
    out->withhold = fault ? 1u : 0u;
    out->spin_limit = fault ? kTestSpinLimit : kSpinLimit;
    return QUAKE_OK;
  }
  const size_t n_psum = kWsSlots * sizeof(uint64_t), n_pmax = kWsSlots * sizeof(uint32_t);
  const size_t n_done = kWsSlots * sizeof(uint32_t), n_err = 256;
  char* base = nullptr;
  if (hipMalloc(&base, n_psum + n_pmax + n_done + n_err) != hipSuccess) return QUAKE_EHIP;
  SplitWs w;
  w.psum = reinterpret_cast<uint64_t*>(base);
  w.pmax = reinterpret_cast<uint32_t*>(base + n_psum);
  w.done = reinterpret_cast<uint32_t*>(base + n_psum + n_pmax);
  w.err = reinterpret_cast<uint32_t*>(base + n_psum + n_pmax + n_done);
  w.spin_limit = kSpinLimit;
  w.withhold = 0;
  hipLaunchKernelGGL(split_ws_init_kernel, dim3(8), dim3(256), 0, s, w, kWsSlots);
  if (hipGetLastError() != hipSuccess) return QUAKE_EHIP;
  g_ws.emplace(WsKey{dev, s}, w);
  *out = w;
  out->withhold = fault ? 1u : 0u;
  out->spin_limit = fault ? kTestSpinLimit : kSpinLimit;
  return QUAKE_OK;
}

static quake_status split_timeouts(hipStream_t s, int64_t* count) {
  *count = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return QUAKE_EHIP;
  uint32_t* err = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    auto it = g_ws.find(WsKey{dev, s});
    if (it == g_ws.end()) return QUAKE_OK;   // no split-row launch on this stream yet
    err = it->second.err;
  }
  uint32_t v = 0;
  if (hipStreamSynchronize(s) != hipSuccess) return QUAKE_EHIP;
  if (hipMemcpy(&v, err, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return QUAKE_EHIP;
  if (v != 0) {
    const uint32_t zero = 0;
    if (hipMemcpy(err, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess) return QUAKE_EHIP;
  }
  *count = v;
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
  SmConst kc;
  int64_t period, shift;   // causal mask (unused otherwise)
  uint32_t write_masked;
  hipStream_t s;
};

static CausalArg causal_at(const SmArgs& a, int64_t r0) {
  if (a.period <= 0) return CausalArg{0, 1, 0, 1};
  return CausalArg{(uint32_t)(r0 % a.period), (uint32_t)a.period, a.shift, a.write_masked};
}

constexpr int64_t kRowChunk = int64_t(1) << 28;   // rows per launch (grid stays < 2^31)

template <int DT, int MODE, bool FUSE, bool CAUSAL, int NV, int WAVES>
static quake_status launch_rows(const SmArgs& a) {
  constexpr int V = kV<DT>;
  constexpr int RPB = kSmBlock / (64 * WAVES);
  const uint32_t nvr = (uint32_t)(a.cols / V);
  for (int64_t r0 = 0; r0 < a.rows; r0 += kRowChunk) {
    const int64_t nr = std::min(kRowChunk, a.rows - r0);
    const uint32_t grid = (uint32_t)((nr + RPB - 1) / RPB);
    hipLaunchKernelGGL((sm_rows_kernel<DT, MODE, FUSE, CAUSAL, NV, WAVES>), dim3(grid),
                       dim3(kSmBlock), 0, a.s, a.x + r0 * a.ldx_b, a.y + r0 * a.ldy_b,
                       (uint32_t)nr, nvr, a.ldx_b, a.ldy_b, a.kc, causal_at(a, r0));
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

// Square causal blocks with rows of at most 64 vectors: the paired kernel on
// whole blocks. Returns false (nothing launched) when the shape does not apply.
template <int DT, int MODE, bool FUSE>
static bool pair_applies(const SmArgs& a) {
  constexpr int V = kV<DT>;
  return a.period == a.cols && a.shift == 0 && a.cols % V == 0 && a.cols / V <= 64 &&
         a.rows >= a.period;
}

template <int DT, int MODE, bool FUSE>
static quake_status launch_causal_pair(const SmArgs& a, int64_t* rows_done) {
  constexpr int V = kV<DT>;
  const uint32_t P = (uint32_t)a.cols;
  const uint32_t K = P > 63u * V ? P - 63u * V : 0u;
  PairArg pa;
  pa.P = P;
  pa.M = P - K;
  pa.J = pa.M / 2 + (pa.M & 1) + K;
  pa.write_masked = a.write_masked;
  const int64_t nblocks = a.rows / P;
  // blocks per launch: keep the job count (and the grid) below 2^31
  const int64_t per = std::max<int64_t>(1, (int64_t(1) << 30) / pa.J);
  for (int64_t b0 = 0; b0 < nblocks; b0 += per) {
    const int64_t nb = std::min(per, nblocks - b0);
    pa.jobs = (uint32_t)(nb * pa.J);
    const uint32_t grid = (pa.jobs + (kSmBlock / 64) - 1) / (kSmBlock / 64);
    const int64_t r0 = b0 * P;
    hipLaunchKernelGGL((sm_causal_pair_kernel<DT, MODE, FUSE>), dim3(grid), dim3(kSmBlock), 0, a.s,
                       a.x + r0 * a.ldx_b, a.y + r0 * a.ldy_b, a.ldx_b, a.ldy_b, a.kc, pa);
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  *rows_done = nblocks * P;
  return QUAKE_OK;
}

template <int DT, int MODE, bool FUSE, bool CAUSAL>
static quake_status launch_generic(const void* x, void* y, const SmArgs& a, int64_t ldx,
                                   int64_t ldy) {
  constexpr int64_t esz = kEsz<DT>;
  constexpr int64_t kGenericRows = int64_t(1) << 30;   // rows per launch (32-bit row index)
  for (int64_t r0 = 0; r0 < a.rows; r0 += kGenericRows) {
    const int64_t nr = std::min(kGenericRows, a.rows - r0);
    const uint32_t grid = (uint32_t)std::min<int64_t>(nr, int64_t(1) << 20);
    hipLaunchKernelGGL((sm_generic_kernel<DT, MODE, FUSE, CAUSAL>), dim3(grid), dim3(kSmBlock), 0,
                       a.s, static_cast<const char*>(x) + r0 * ldx * esz,
                       static_cast<char*>(y) + r0 * ldy * esz, nr, a.cols, ldx, ldy, a.kc,
                       causal_at(a, r0));
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

// Returns QUAKE_OK on success, or 1 + status on failure; -1 if the split path
// cannot be used (too many chunks per row) and the caller should fall back.
template <int DT, int MODE, bool FUSE, bool CAUSAL, int NV>
static int launch_split(const SmArgs& a) {
  constexpr int V = kV<DT>;
  constexpr int CHV = kSmBlock * NV;
  const uint32_t nvr = (uint32_t)(a.cols / V);
  const uint32_t G = (nvr + CHV - 1) / CHV;
  auto kern = sm_split_kernel<DT, MODE, FUSE, CAUSAL, NV>;
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
  // every workgroup of one launch fits on the device at once
  const int64_t rows_per_launch = cap / G;
  for (int64_t r0 = 0; r0 < a.rows; r0 += rows_per_launch) {
    const int64_t nr = std::min(rows_per_launch, a.rows - r0);
    hipLaunchKernelGGL((sm_split_kernel<DT, MODE, FUSE, CAUSAL, NV>), dim3((uint32_t)(nr * G)),
                       dim3(kSmBlock), 0, a.s, a.x + r0 * a.ldx_b, a.y + r0 * a.ldy_b, nvr, a.ldx_b,
                       a.ldy_b, a.kc, causal_at(a, r0), G, ws);
    st = launch_status();
    if (st != QUAKE_OK) return 1 + st;
  }
  return QUAKE_OK;
}

template <int DT, int MODE, bool FUSE, bool CAUSAL>
static quake_status sm_dispatch(const void* x, void* y, int64_t ldx, int64_t ldy, const SmArgs& ain) {
  constexpr int V = kV<DT>;
  constexpr int64_t esz = kEsz<DT>;
  const int64_t cols = ain.cols;
  const bool vec = aligned16(x) && aligned16(y) && (ldx * esz) % 16 == 0 && (ldy * esz) % 16 == 0 &&
                   cols % V == 0 && cols < (int64_t(1) << 31) - 16;
  if (!vec) return launch_generic<DT, MODE, FUSE, CAUSAL>(x, y, ain, ldx, ldy);
  SmArgs a = ain;
  a.x = static_cast<const char*>(x);
  a.y = static_cast<char*>(y);
  a.ldx_b = ldx * esz;
  a.ldy_b = ldy * esz;
  const int64_t nvr = cols / V;
  if constexpr (CAUSAL) {
    if (pair_applies<DT, MODE, FUSE>(a)) {
      int64_t done = 0;
      const quake_status st = launch_causal_pair<DT, MODE, FUSE>(a, &done);
      if (st != QUAKE_OK || done == a.rows) return st;
      // rows after the last whole block: the one-row kernel (r0 is a multiple of P)
      SmArgs rest = a;
      rest.x = a.x + done * a.ldx_b;
      rest.y = a.y + done * a.ldy_b;
      rest.rows = a.rows - done;
      return launch_rows<DT, MODE, FUSE, CAUSAL, 1, 1>(rest);
    }
  }
  if (nvr <= 64) return launch_rows<DT, MODE, FUSE, CAUSAL, 1, 1>(a);
  if (nvr <= 128) return launch_rows<DT, MODE, FUSE, CAUSAL, 2, 1>(a);
  if (nvr <= 256) return launch_rows<DT, MODE, FUSE, CAUSAL, 4, 1>(a);
  if (nvr <= 512) return launch_rows<DT, MODE, FUSE, CAUSAL, 8, 1>(a);
  if (nvr <= 1024) return launch_rows<DT, MODE, FUSE, CAUSAL, 4, 4>(a);
  if (nvr <= 2048) return launch_rows<DT, MODE, FUSE, CAUSAL, 8, 4>(a);
  if constexpr (DT == F32) {
    if (nvr <= 4096) return launch_rows<DT, MODE, FUSE, CAUSAL, 16, 4>(a);
  }
  // 64 elements per lane per chunk: 16 vectors of binary32 or 8 of 16-bit
  const int rc = launch_split<DT, MODE, FUSE, CAUSAL, (DT == F32 ? 16 : 8)>(a);
  if (rc >= 0) return rc == 0 ? QUAKE_OK : (quake_status)(rc - 1);
  return launch_generic<DT, MODE, FUSE, CAUSAL>(x, y, ain, ldx, ldy);
}

template <bool FUSE, bool CAUSAL>
static quake_status softmax_entry(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                                  int64_t ldy, int dtype, int mode, float t, int64_t period,
                                  int64_t shift, int write_masked, void* stream) {
  if (!valid_dtype(dtype)) return QUAKE_EDTYPE;
  if (!valid_mode(mode)) return QUAKE_EMODE;
  if (rows < 0 || cols < 0 || ldx < 0 || ldy < 0) return QUAKE_EINVAL;
  if (CAUSAL && (period <= 0 || period > INT32_MAX || shift < -(int64_t(1) << 40) ||
                 shift > (int64_t(1) << 40)))
    return QUAKE_EINVAL;
  if (rows == 0) return QUAKE_OK;
  if (cols == 0 || ldx < cols || ldy < cols || x == nullptr || y == nullptr) return QUAKE_EINVAL;
  if (!std::isfinite(t) || !(t > 0.0f)) return QUAKE_EINVAL;
  SmConst kc;
  if (FUSE) {
    kc = SmConst{softmax_c0(t, mode), 0.0f, t};
    if (!std::isfinite(kc.c0) || kc.c0 == 0.0f) return QUAKE_EINVAL;
  } else {
    const Affine af = exp_affine(1.0, 0.0, mode);   // the standard e^s
    kc = SmConst{af.c0, af.c1, t};
  }
  const SmArgs a{static_cast<const char*>(x), static_cast<char*>(y), rows, cols, 0, 0, kc,
                 CAUSAL ? period : 0, shift, (uint32_t)(write_masked != 0),
                 static_cast<hipStream_t>(stream)};
#define QK_SM_CASE(D, M) \
  if (dtype == D && mode == M) return sm_dispatch<D, M, FUSE, CAUSAL>(x, y, ldx, ldy, a);
  QK_SM_CASE(F32, EXACT) QK_SM_CASE(F32, Q1) QK_SM_CASE(F32, Q2) QK_SM_CASE(F32, Q2M)
  QK_SM_CASE(F16, EXACT) QK_SM_CASE(F16, Q1) QK_SM_CASE(F16, Q2) QK_SM_CASE(F16, Q2M)
  QK_SM_CASE(BF16, EXACT) QK_SM_CASE(BF16, Q1) QK_SM_CASE(BF16, Q2) QK_SM_CASE(BF16, Q2M)
#undef QK_SM_CASE
  return QUAKE_EMODE;
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_softmax(const void* x, void* y, int64_t rows, int64_t cols,
                                      int64_t ldx, int64_t ldy, quake_dtype dtype,
                                      quake_mode mode, float t, void* stream) {
  return softmax_entry<true, false>(x, y, rows, cols, ldx, ldy, dtype, mode, t, 0, 0, 1, stream);
}

extern "C" quake_status quake_softmax_unfused(const void* x, void* y, int64_t rows, int64_t cols,
                                              int64_t ldx, int64_t ldy, quake_dtype dtype,
                                              quake_mode mode, float t, void* stream) {
  return softmax_entry<false, false>(x, y, rows, cols, ldx, ldy, dtype, mode, t, 0, 0, 1, stream);
}

extern "C" quake_status quake_softmax_causal(const void* x, void* y, int64_t rows, int64_t cols,
                                             int64_t ldx, int64_t ldy, int64_t period,
                                             int64_t shift, int write_masked, quake_dtype dtype,
                                             quake_mode mode, float t, void* stream) {
  return softmax_entry<true, true>(x, y, rows, cols, ldx, ldy, dtype, mode, t, period, shift,
                                   write_masked, stream);
}

extern "C" quake_status quake_softmax_split_timeouts(void* stream, int64_t* count) {
  if (count == nullptr) return QUAKE_EINVAL;
  return split_timeouts(static_cast<hipStream_t>(stream), count);
}

extern "C" int quake_test_split_fault(int on) {
  return g_test_fault.exchange(on ? 1 : 0);
}
