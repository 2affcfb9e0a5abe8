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
//   sm_split<NV>          rows longer than a workgroup's registers, with a
//                         workspace from the caller: G workgroups per row each
//                         hold one chunk in VGPRs and exchange their chunk max,
//                         then their chunk sum, through the workspace's slots
//                         (relaxed atomics, no fences). A workgroup that waits
//                         too long for a peer computes the peer's value from x
//                         itself (same bits), so no wait depends on the peers
//                         being resident.
//   sm_res                the same rows without a workspace, up to 129024
//                         (binary32) or 131072 (16-bit) elements: one
//                         512-thread workgroup per row holds the row in VGPRs
//                         and LDS (one read, each exponential taken once).
//   sm_long               longer or causal rows without a workspace: one
//                         1024-thread workgroup per row, three passes (max,
//                         sum, normalise), the re-reads served by the caches.
//   shifted rows          rows whose start is not 16-byte aligned (a length
//                         that is not a multiple of the vector, an offset
//                         base) at the same offset in x and y: sm_rows and
//                         sm_res read the aligned vectors that cover each
//                         row, mask the elements outside it and store the
//                         row's first and last vectors element by element.
//   sm_generic            any other alignment / stride / length: one
//                         workgroup per row, three passes (max, sum,
//                         normalise) with scalar accesses; the re-reads are
//                         served by the caches.
// Sums: fp32 within one 16-byte vector (at most 8 terms), then, in a fixed
// order, double across vectors, lanes, waves and workgroups for binary32
// outputs and fp32 for 16-bit outputs in the row kernels (double in the split,
// resident and long kernels).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

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

// The exponential of one entry with the clamp folded into the conversion
// (BELOW: every entry is at most the row max and |c1| < 2^54, so the upper
// clamp cannot act): the bits of ex(v) with one instruction fewer.
template <bool BELOW, int MODE, bool FUSE>
__device__ __forceinline__ float row_exp_at(const RowExp<MODE, FUSE>& ex, float v) {
  if constexpr (FUSE && BELOW) return qexp_row<MODE, true>(v, ex.c0, ex.c1);
  else return ex(v);
}
// whether the wave may take row_exp_at<true>
template <int MODE, bool FUSE>
__device__ __forceinline__ bool row_exp_below(const RowExp<MODE, FUSE>& ex) {
  if constexpr (FUSE && MODE != EXACT) return row_c1_below(ex.c1);
  else return false;
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
// Rows whose start is not 16-byte aligned (a length that is not a multiple of
// the vector, or a shifted base): the row is read as the aligned 16-byte
// vectors that cover it, from the aligned address s elements before its start
// (s = 0 .. V-1). An aligned 16-byte vector never crosses a page, so reading
// the few elements around the row cannot fault; they are masked to -inf and
// never written. Element e of that vector space is row element e - s.
// ---------------------------------------------------------------------------
// -inf for the elements of vector vi outside the row [s, s + cols).
template <int V>
__device__ __forceinline__ void mask_outside(float* f, uint32_t vi, uint32_t s, uint32_t cols) {
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const uint32_t e = vi * V + j;
    if (e < s || e - s >= cols) f[j] = -INFINITY;
  }
}

// Stores the elements of vector vi that lie inside the row, one element at a
// time, with the rounding of the whole-vector store.
template <int DT>
__device__ __forceinline__ void store_inside(char* ya, uint32_t vi, uint32_t s, uint32_t cols,
                                             const float* f) {
  constexpr int V = kV<DT>;
  const u32x4 p = pack<DT>(f);
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const uint32_t e = vi * V + j;
    if (e >= s && e - s < cols) {
      if constexpr (DT == F32) {
        reinterpret_cast<uint32_t*>(ya)[e] = p[j];
      } else {
        const uint32_t w = p[j >> 1];
        reinterpret_cast<uint16_t*>(ya)[e] = (uint16_t)((j & 1) ? (w >> 16) : (w & 0xffffu));
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Register-resident rows: one wave (WAVES = 1) or one workgroup (WAVES = 4).
// ---------------------------------------------------------------------------
template <int DT, int MODE, bool FUSE, bool CAUSAL, int NV, int WAVES, bool FULL = false,
          bool SHIFT = false>
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

  // SHIFT: nvr carries the row length in elements; the row is read as the
  // aligned vectors that cover it (x and y rows share their offset s).
  const char* xrow = x + (int64_t)row * ldx_b;
  char* yrow = y + (int64_t)row * ldy_b;
  uint32_t s = 0, cols = 0;
  if constexpr (SHIFT) {
    s = (uint32_t)(((uintptr_t)xrow & 15u) / kEsz<DT>);
    cols = nvr;
    nvr = (s + cols + V - 1) / V;
    xrow -= s * kEsz<DT>;
    yrow -= s * kEsz<DT>;
  }
  const u32x4* xr = reinterpret_cast<const u32x4*>(xrow);
  u32x4* yr = reinterpret_cast<u32x4*>(yrow);

  // Every lane loads (vectors past the row end re-read the row's last vector,
  // which stays in one cache line) and padding lanes select -inf: no branch
  // around the loads, so the whole row stays in registers without merges.
  // With the causal mask only vectors holding live entries are read. FULL:
  // the row is exactly NV vectors per lane, so there is nothing to pad.
  // live entries: row elements [0, L) (the causal mask), i.e. elements
  // [s, s + L) of the vector space; nvl vectors hold them
  const uint32_t L = (uint32_t)live_len<CAUSAL>(ca, row, SHIFT ? (int64_t)cols : (int64_t)nvr * V);
  const uint32_t nvl = !CAUSAL ? nvr : L == 0 ? 0 : (s + L + V - 1) / V;
  const uint32_t vlast = (nvl > 0 ? nvl : 1) - 1;
  u32x4 raw[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k)
    raw[k] = __builtin_nontemporal_load(xr + (FULL ? k * LANES + lid : umin32(k * LANES + lid, vlast)));
  float f[NV][V];
  float lmax = -INFINITY;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = k * LANES + lid;
    // whole vectors past the row end become -inf before widening (one select
    // per word); only the causal boundary needs a per-element mask
    if (!FULL && !CAUSAL && vi >= nvr) raw[k] = neg_inf_vec<DT>();
    unpack<DT>(raw[k], f[k]);
    if constexpr (SHIFT && !CAUSAL) {
      if (vi == 0 || vi + 1 == nvr) mask_outside<V>(f[k], vi, s, cols);
    }
#pragma unroll
    for (int j = 0; j < V; ++j) {
      // with SHIFT, elements before the row start wrap to large values
      if constexpr (CAUSAL) f[k][j] = (vi * V + j - s < L) ? f[k][j] : -INFINITY;
      lmax = fmaxf(lmax, f[k][j]);
    }
  }

  float m = wave_max(lmax);
  if constexpr (WAVES > 1) {
    if (lane == 0) s_max[wave] = m;
    __syncthreads();
    m = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
  }

  // Partial sums start from their first term: every exponential is >= +0,
  // so 0 + e would be e exactly and the sums are the same bits.
  const RowExp<MODE, FUSE> ex = row_exp<MODE, FUSE>(kc, m);
  Acc acc = 0;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    f[k][0] = ex(f[k][0]);
    float part = f[k][0];
#pragma unroll
    for (int j = 1; j < V; ++j) {
      f[k][j] = ex(f[k][j]);
      part += f[k][j];
    }
    acc = (k == 0) ? (Acc)part : acc + (Acc)part;
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
    if ((FULL || vi < nvr) && (!CAUSAL || ca.write_masked || vi < nvl)) {
#pragma unroll
      for (int j = 0; j < V; ++j) f[k][j] *= r;
      if (SHIFT && (vi == 0 || vi + 1 == nvr))
        store_inside<DT>(yrow, vi, s, cols, f[k]);
      else
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
// Every exponent of a row needs the row's final max (Algorithm 2), so a row
// longer than one workgroup's registers is held by G workgroups that exchange
// their chunk maxima, then their chunk sums against the final max, through a
// workspace the caller owns. Each chunk has a 32-bit max slot and a 64-bit sum
// slot; a value is published as the complement of its bits with a relaxed
// agent-scope atomic store, so 0 means "not published yet" and a zero-filled
// workspace is the initial state. The value is itself the atomic object: no
// release / acquire fence (no L2 write-back or invalidate) is needed. After
// both rounds each workgroup counts itself done; the last one of the row puts
// the slots back to 0, so the workspace is ready for the next launch (also on
// graph replay).
//
// No wait depends on co-residency: a workgroup that has polled a slot for the
// wait limit (s_memrealtime ticks) without seeing it published computes that
// chunk's value itself from x, with the same loads, lane layout and summation
// order as the chunk's owner, so the bits are the same either way. A launch
// may therefore be larger than the device, and other streams may hold any
// number of CUs; only the speed changes. The limit 0xFFFFFFFF means no wait
// at all: every workgroup computes every chunk value of its row itself.
// ---------------------------------------------------------------------------
struct SplitWs {
  uint32_t* hdr;    // [0] wait limit in s_memrealtime ticks (0: the default)
                    // [1] count of chunk values recomputed after a wait gave up
  uint64_t* psum;   // [R*G] ~bits of chunk sums (binary64), 0 = not published
  uint32_t* pmax;   // [R*G] ~bits of chunk maxima (binary32), 0 = not published
  uint32_t* done;   // [R]   workgroups of the row past both exchanges
};

constexpr int kMaxG = kSmBlock;                    // one polling lane per chunk
constexpr uint64_t kDefaultWaitTicks = 10000;      // 100 us at the 100 MHz constant clock
constexpr size_t kWsHeader = 256;                  // bytes before the slot arrays

constexpr uint32_t kNoWait = 0xFFFFFFFFu;          // wait limit word: never wait

template <typename T>
__device__ __forceinline__ bool poll_slot(T* slot, uint64_t limit, T* out) {
  if (limit == kNoWait) return false;   // every peer value is computed from x
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  T v;
  while ((v = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) == 0) {
    if (__builtin_amdgcn_s_memrealtime() - t0 > limit) return false;
    __builtin_amdgcn_s_sleep(1);
  }
  *out = ~v;
  return true;
}

// One 16-byte vector of a row widened to binary32, masked as the register-
// resident kernels mask it: vectors past the row end are -inf, and with the
// causal mask entries at or past the live length L are -inf.
template <int DT, bool CAUSAL>
__device__ __forceinline__ void widen_masked(u32x4 raw, uint32_t vi, uint32_t nvr, uint32_t L,
                                             float* f) {
  constexpr int V = kV<DT>;
  if (!CAUSAL && vi >= nvr) raw = neg_inf_vec<DT>();
  unpack<DT>(raw, f);
  if constexpr (CAUSAL) {
#pragma unroll
    for (int j = 0; j < V; ++j) f[j] = (vi * V + j < L) ? f[j] : -INFINITY;
  }
}

// Chunk q's max and sum computed from x by the whole workgroup, for a chunk
// whose owner has not published in time: thread t takes vectors
// q*CHV + k*256 + t, k = 0 .. NV-1, as the owner's thread t holds them, so the
// per-vector partial sums, the per-lane double accumulation, the wave trees
// and the cross-wave pairing are the owner's, bit for bit.
template <int DT, bool CAUSAL, int NV, bool SHIFT>
__device__ float chunk_max_from_x(const u32x4* xr, uint32_t q, uint32_t nvr, uint32_t vlast,
                                  uint32_t L, float* s4, uint32_t s, uint32_t cols) {
  constexpr int V = kV<DT>;
  float lmax = -INFINITY;
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = q * (kSmBlock * NV) + k * kSmBlock + threadIdx.x;
    float f[V];
    widen_masked<DT, CAUSAL>(__builtin_nontemporal_load(xr + umin32(vi, vlast)), vi, nvr, L, f);
    if (SHIFT && (vi == 0 || vi + 1 == nvr)) mask_outside<V>(f, vi, s, cols);
#pragma unroll
    for (int j = 0; j < V; ++j) lmax = fmaxf(lmax, f[j]);
  }
  const float m = wave_max(lmax);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s4[threadIdx.x >> 6] = m;
  __syncthreads();
  return fmaxf(fmaxf(s4[0], s4[1]), fmaxf(s4[2], s4[3]));
}

template <int DT, int MODE, bool FUSE, bool CAUSAL, int NV, bool SHIFT>
__device__ double chunk_sum_from_x(const u32x4* xr, uint32_t q, uint32_t nvr, uint32_t vlast,
                                   uint32_t L, const RowExp<MODE, FUSE>& ex, double* s4,
                                   uint32_t s, uint32_t cols) {
  constexpr int V = kV<DT>;
  double acc = 0.0;
  for (int k = 0; k < NV; ++k) {
    const uint32_t vi = q * (kSmBlock * NV) + k * kSmBlock + threadIdx.x;
    float f[V];
    widen_masked<DT, CAUSAL>(__builtin_nontemporal_load(xr + umin32(vi, vlast)), vi, nvr, L, f);
    if (SHIFT && (vi == 0 || vi + 1 == nvr)) mask_outside<V>(f, vi, s, cols);
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < V; ++j) part += ex(f[j]);
    acc += (double)part;
  }
  const double ws = wave_sum(acc);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s4[threadIdx.x >> 6] = ws;
  __syncthreads();
  return (s4[0] + s4[1]) + (s4[2] + s4[3]);
}

template <int DT, int MODE, bool FUSE, bool CAUSAL, int NV, bool SHIFT = false>
__global__ __launch_bounds__(kSmBlock) void sm_split_kernel(const char* __restrict__ x,
                                                           char* __restrict__ y, uint32_t nvr,
                                                           int64_t ldx_b, int64_t ldy_b,
                                                           SmConst kc, CausalArg ca, uint32_t G,
                                                           uint32_t xcd_map, SplitWs ws) {
  constexpr int V = kV<DT>;
  constexpr int CHV = kSmBlock * NV;   // vectors per chunk
  __shared__ float s_max[4];
  __shared__ double s_sum[4];
  __shared__ float s_fmax[4];
  __shared__ double s_fsum[4];
  __shared__ float s_pmax[kMaxG];
  __shared__ double s_psum[kMaxG];
  __shared__ uint32_t s_missing;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  // Chunk g of row rr. blockIdx round-robins over the 8 XCDs; with xcd_map
  // (rows a multiple of 8, few chunks per row) XCD x takes rows x, x + 8, ...
  // with all their chunks, so a row's exchange stays within one XCD's L2.
  uint32_t rr, g;
  if (xcd_map) {
    const uint32_t sl = blockIdx.x >> 3;
    rr = (blockIdx.x & 7u) + 8u * (sl / G);
    g = sl % G;
  } else {
    rr = blockIdx.x / G;
    g = blockIdx.x - rr * G;
  }
  uint32_t* pm = ws.pmax + rr * G;
  uint64_t* ps = ws.psum + rr * G;
  const uint32_t lim_in = ws.hdr[0];
  const uint64_t limit = lim_in ? (uint64_t)lim_in : kDefaultWaitTicks;

  // SHIFT: nvr carries the row length in elements; the row is read as the
  // aligned vectors that cover it (x and y rows share their offset s). The
  // launch's chunk count covers the most vectors any row can span, so a
  // row's last chunk may hold no element of it (max -inf, sum 0).
  const char* xrow = x + (int64_t)rr * ldx_b;
  char* yrow = y + (int64_t)rr * ldy_b;
  uint32_t s = 0, cols = 0;
  if constexpr (SHIFT) {
    s = (uint32_t)(((uintptr_t)xrow & 15u) / kEsz<DT>);
    cols = nvr;
    nvr = (s + cols + V - 1) / V;
    xrow -= s * kEsz<DT>;
    yrow -= s * kEsz<DT>;
  }
  const u32x4* xr = reinterpret_cast<const u32x4*>(xrow);
  u32x4* yr = reinterpret_cast<u32x4*>(yrow);
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
    widen_masked<DT, CAUSAL>(raw[k], vi, nvr, L, f[k]);
    if constexpr (SHIFT) {
      if (vi == 0 || vi + 1 == nvr) mask_outside<V>(f[k], vi, s, cols);
    }
#pragma unroll
    for (int j = 0; j < V; ++j) lmax = fmaxf(lmax, f[k][j]);
  }

  // first exchange: the chunk maxima
  float m = wave_max(lmax);
  if (lane == 0) s_max[wave] = m;
  if (threadIdx.x == 0) s_missing = 0;
  __syncthreads();
  if (threadIdx.x == 0) {
    m = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
    const uint32_t mb = (m != m) ? as_u(-INFINITY) : as_u(m);
    __hip_atomic_store(pm + g, ~mb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (threadIdx.x < G) {
    uint32_t v;
    const bool ok = poll_slot<uint32_t>(pm + threadIdx.x, limit, &v);
    s_pmax[threadIdx.x] = ok ? as_f(v) : __builtin_nanf("");   // NaN: not published in time
    if (!ok) s_missing = 1;
  }
  __syncthreads();
  const bool missing_max = s_missing != 0;
  m = -INFINITY;
  for (uint32_t q = 0; q < G; ++q) m = fmaxf(m, s_pmax[q]);   // fmaxf skips the NaN marks
  if (missing_max) {   // uniform: every thread reads the same LDS words
    for (uint32_t q = 0; q < G; ++q) {
      if (s_pmax[q] != s_pmax[q])
        m = fmaxf(m, chunk_max_from_x<DT, CAUSAL, NV, SHIFT>(xr, q, nvr, vlast, L, s_fmax, s, cols));
    }
  }

  // second exchange: the chunk sums against the row's final max
  // the exponentials sit between the two exchanges, on the critical path: the
  // folded clamp where the row constant allows it (same bits)
  const RowExp<MODE, FUSE> ex = row_exp<MODE, FUSE>(kc, m);
  double acc = 0.0;
  auto exps = [&](auto below) {
    constexpr bool B = decltype(below)::value;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      float part = 0.0f;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        f[k][j] = row_exp_at<B>(ex, f[k][j]);
        part += f[k][j];
      }
      acc += (double)part;
    }
  };
  if (row_exp_below(ex))
    exps(std::true_type{});
  else
    exps(std::false_type{});
  double total = wave_sum(acc);
  if (lane == 0) s_sum[wave] = total;
  __syncthreads();
  if (threadIdx.x == 0) {
    s_missing = 0;
    total = (s_sum[0] + s_sum[1]) + (s_sum[2] + s_sum[3]);
    const uint64_t tb = (total != total) ? 0x7FF8000000000000ull : __builtin_bit_cast(uint64_t, total);
    __hip_atomic_store(ps + g, ~tb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (threadIdx.x < G) {
    uint64_t v;
    const bool ok = poll_slot<uint64_t>(ps + threadIdx.x, limit, &v);
    s_psum[threadIdx.x] = ok ? __builtin_bit_cast(double, v) : __builtin_nan("");
    if (!ok) s_missing = 1;
  }
  __syncthreads();
  const bool missing_sum = s_missing != 0;
  if (missing_sum) {
    for (uint32_t q = 0; q < G; ++q) {
      const double sq = s_psum[q];
      __syncthreads();   // every thread has read s_psum[q] before thread 0 may rewrite it
      if (sq != sq) {
        const double v = chunk_sum_from_x<DT, MODE, FUSE, CAUSAL, NV, SHIFT>(xr, q, nvr, vlast, L, ex,
                                                                             s_fsum, s, cols);
        if (threadIdx.x == 0) s_psum[q] = v;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (missing_max || missing_sum)
      __hip_atomic_fetch_add(ws.hdr + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // This workgroup's two publishing stores are complete before it counts
    // itself done, so no publish can land after the row's slots are cleared;
    // the last workgroup of the row clears them for the next launch.
    __builtin_amdgcn_s_waitcnt(0);
    const uint32_t old = __hip_atomic_fetch_add(ws.done + rr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == G - 1) {
      for (uint32_t q = 0; q < G; ++q) {
        __hip_atomic_store(pm + q, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(ps + q, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
      if (SHIFT && (vi == 0 || vi + 1 == nvr))
        store_inside<DT>(yrow, vi, s, cols, f[k]);
      else
        __builtin_nontemporal_store(pack<DT>(f[k]), yr + vi);
    }
  }
}

// ---------------------------------------------------------------------------
// Long rows without a workspace: one 1024-thread workgroup per row, three
// passes over the row (max; sum of the exponentials against it; normalise and
// store). The second and third reads are mostly served by the caches. No
// exchange between workgroups, so nothing but x and y is touched.
// ---------------------------------------------------------------------------
constexpr int kLongBlock = 1024;
constexpr int kLongUnroll = 4;

template <int DT, int MODE, bool FUSE, bool CAUSAL>
__global__ __launch_bounds__(kLongBlock) void sm_long_kernel(const char* __restrict__ x,
                                                            char* __restrict__ y, uint32_t nvr,
                                                            int64_t ldx_b, int64_t ldy_b,
                                                            SmConst kc, CausalArg ca) {
  constexpr int V = kV<DT>;
  constexpr int W = kLongBlock / 64;
  constexpr uint32_t STEP = kLongBlock * kLongUnroll;
  __shared__ float s_max[W];
  __shared__ double s_sum[W];
  const uint32_t rr = blockIdx.x;
  const u32x4* xr = reinterpret_cast<const u32x4*>(x + (int64_t)rr * ldx_b);
  u32x4* yr = reinterpret_cast<u32x4*>(y + (int64_t)rr * ldy_b);
  const uint32_t L = (uint32_t)live_len<CAUSAL>(ca, rr, (int64_t)nvr * V);
  const uint32_t nvl = CAUSAL ? (L + V - 1) / V : nvr;
  const uint32_t vlast = (nvl > 0 ? nvl : 1) - 1;

  float lmax = -INFINITY;
  for (uint32_t b = threadIdx.x; b < nvl; b += STEP) {
    u32x4 raw[kLongUnroll];
#pragma unroll
    for (int u = 0; u < kLongUnroll; ++u)
      raw[u] = __builtin_nontemporal_load(xr + umin32(b + u * kLongBlock, vlast));
#pragma unroll
    for (int u = 0; u < kLongUnroll; ++u) {
      float f[V];
      widen_masked<DT, CAUSAL>(raw[u], b + u * kLongBlock, nvr, L, f);
#pragma unroll
      for (int j = 0; j < V; ++j) lmax = fmaxf(lmax, f[j]);
    }
  }
  float m = wave_max(lmax);
  if ((threadIdx.x & 63) == 0) s_max[threadIdx.x >> 6] = m;
  __syncthreads();
  m = s_max[0];
  for (int w = 1; w < W; ++w) m = fmaxf(m, s_max[w]);

  const RowExp<MODE, FUSE> ex = row_exp<MODE, FUSE>(kc, m);
  double acc = 0.0;
  for (uint32_t b = threadIdx.x; b < nvl; b += STEP) {
    u32x4 raw[kLongUnroll];
#pragma unroll
    for (int u = 0; u < kLongUnroll; ++u)
      raw[u] = __builtin_nontemporal_load(xr + umin32(b + u * kLongBlock, vlast));
#pragma unroll
    for (int u = 0; u < kLongUnroll; ++u) {
      const uint32_t vi = b + u * kLongBlock;
      float f[V];
      widen_masked<DT, CAUSAL>(raw[u], vi, nvr, L, f);
      float part = 0.0f;
#pragma unroll
      for (int j = 0; j < V; ++j) part += ex(f[j]);
      if (vi < nvl) acc += (double)part;
    }
  }
  double total = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) s_sum[threadIdx.x >> 6] = total;
  __syncthreads();
  total = s_sum[0];
  for (int w = 1; w < W; ++w) total += s_sum[w];
  const float r = (m == -INFINITY) ? 0.0f : (float)(1.0 / total);

  const uint32_t nst = (!CAUSAL || ca.write_masked) ? nvr : nvl;
  for (uint32_t b = threadIdx.x; b < nst; b += STEP) {
    u32x4 raw[kLongUnroll];
#pragma unroll
    for (int u = 0; u < kLongUnroll; ++u)
      raw[u] = __builtin_nontemporal_load(xr + umin32(b + u * kLongBlock, vlast));
#pragma unroll
    for (int u = 0; u < kLongUnroll; ++u) {
      const uint32_t vi = b + u * kLongBlock;
      if (vi < nst) {
        float f[V];
        widen_masked<DT, CAUSAL>(raw[u], vi, nvr, L, f);
#pragma unroll
        for (int j = 0; j < V; ++j) f[j] = ex(f[j]) * r;
        __builtin_nontemporal_store(pack<DT>(f), yr + vi);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Rows without a workspace that fit one workgroup (up to 129024 binary32 or
// 131072 16-bit elements): one 512-thread workgroup per row reads the row once
// and keeps it, NK 16-byte vectors per thread in VGPRs and NL more per thread
// in LDS as binary32, so every exponential is taken once and nothing is read
// twice. Thread t holds vectors k * 512 + t. Whole blocks of 512 vectors past
// the row's end are skipped (a workgroup-uniform branch); inside the last
// block, lanes past the end load the last vector again, which leaves the max
// unchanged (SHIFT: masked to -inf like the elements outside the row), is
// left out of the sum and is never stored. REGFULL: every register block
// lies inside the row, so those loads are unconditional and the compiler's
// vmcnt waits stay per load. MINB: workgroups per CU the registers are
// budgeted for. The LDS part is loaded first, so the VGPRs it passes through
// are free again before the register part arrives. Sums as in sm_long: fp32
// within a vector, then double across vectors, lanes and waves in a fixed
// order.
// ---------------------------------------------------------------------------
constexpr int kResBlock = 512;

template <int DT, int MODE, bool FUSE, int NK, int NL, bool REGFULL, int MINB, bool SHIFT = false>
__global__ __launch_bounds__(kResBlock, MINB) void sm_res_kernel(const char* __restrict__ x,
                                                                char* __restrict__ y, uint32_t nvr,
                                                                int64_t ldx_b, int64_t ldy_b,
                                                                SmConst kc) {
  constexpr int V = kV<DT>;
  constexpr int B = kResBlock;
  constexpr int W = B / 64;
  __shared__ float s_max[W];
  __shared__ double s_sum[W];
  __shared__ __attribute__((aligned(16))) float s_row[NL > 0 ? NL * B * V : 4];
  const uint32_t t = threadIdx.x;
  // SHIFT: nvr carries the row length in elements; the row is read as the
  // aligned vectors that cover it (x and y rows share their offset s).
  const char* xrow = x + (int64_t)blockIdx.x * ldx_b;
  char* yrow = y + (int64_t)blockIdx.x * ldy_b;
  uint32_t s = 0, cols = 0;
  if constexpr (SHIFT) {
    s = (uint32_t)(((uintptr_t)xrow & 15u) / kEsz<DT>);
    cols = nvr;
    nvr = (s + cols + V - 1) / V;
    xrow -= s * kEsz<DT>;
    yrow -= s * kEsz<DT>;
  }
  const u32x4* xr = reinterpret_cast<const u32x4*>(xrow);
  u32x4* yr = reinterpret_cast<u32x4*>(yrow);
  const uint32_t vlast = nvr - 1;                              // nvr >= 1
  const uint32_t cnt = t < nvr ? (nvr - 1 - t) / B + 1 : 0;    // this thread's vectors in the row
  float* mine = s_row + t * V;                                 // LDS block k: mine + k * B * V

  float lmax = -INFINITY;
  {
    u32x4 raw[NL > 0 ? NL : 1];
#pragma unroll
    for (int k = 0; k < NL; ++k)
      if (REGFULL || (NK + k) * B < nvr)
        raw[k] = __builtin_nontemporal_load(xr + umin32((NK + k) * B + t, vlast));
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      if ((NK + k) * B >= nvr) continue;
      float g[V];
      unpack<DT>(raw[k], g);
      if constexpr (SHIFT) {
        const uint32_t vi = (NK + k) * B + t;
        if (vi + 1 >= nvr) mask_outside<V>(g, vi, s, cols);   // the last vector, or past it
      }
#pragma unroll
      for (int j = 0; j < V; ++j) {
        lmax = fmaxf(lmax, g[j]);
        mine[k * B * V + j] = g[j];
      }
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  u32x4 raw[NK];
#pragma unroll
  for (int k = 0; k < NK; ++k)
    if (REGFULL || k * B < nvr) raw[k] = __builtin_nontemporal_load(xr + umin32(k * B + t, vlast));
  float f[NK][V];
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    if (!REGFULL && k * B >= nvr) continue;
    unpack<DT>(raw[k], f[k]);
    if constexpr (SHIFT) {
      const uint32_t vi = k * B + t;
      if (vi == 0 || vi + 1 >= nvr) mask_outside<V>(f[k], vi, s, cols);
    }
#pragma unroll
    for (int j = 0; j < V; ++j) lmax = fmaxf(lmax, f[k][j]);
  }
  float m = wave_max(lmax);
  if ((t & 63) == 0) s_max[t >> 6] = m;
  __syncthreads();
  m = s_max[0];
  for (int w = 1; w < W; ++w) m = fmaxf(m, s_max[w]);

  const RowExp<MODE, FUSE> ex = row_exp<MODE, FUSE>(kc, m);
  double acc = 0.0;
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    if (!REGFULL && k * B >= nvr) continue;
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      f[k][j] = ex(f[k][j]);
      part += f[k][j];
    }
    if ((uint32_t)k < cnt) acc += (double)part;
  }
#pragma unroll
  for (int k = 0; k < NL; ++k) {
    if ((NK + k) * B >= nvr) continue;
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const float e = ex(mine[k * B * V + j]);
      mine[k * B * V + j] = e;
      part += e;
    }
    if ((uint32_t)(NK + k) < cnt) acc += (double)part;
  }
  double total = wave_sum(acc);
  if ((t & 63) == 0) s_sum[t >> 6] = total;
  __syncthreads();
  total = s_sum[0];
  for (int w = 1; w < W; ++w) total += s_sum[w];
  const float r = (m == -INFINITY) ? 0.0f : (float)(1.0 / total);

  // The store indexes come from an opaque copy of t: otherwise the compiler
  // keeps the load-side indexes (or their compares) live across the kernel,
  // and the row no longer fits the VGPRs.
  uint32_t ts = t;
  asm volatile("" : "+v"(ts));
#pragma unroll
  for (int k = 0; k < NK; ++k) {
    const uint32_t vi = k * B + ts;
    if (vi < nvr) {
#pragma unroll
      for (int j = 0; j < V; ++j) f[k][j] *= r;
      if (SHIFT && (vi == 0 || vi + 1 == nvr))
        store_inside<DT>(yrow, vi, s, cols, f[k]);
      else
        __builtin_nontemporal_store(pack<DT>(f[k]), yr + vi);
    }
  }
#pragma unroll
  for (int k = 0; k < NL; ++k) {
    const uint32_t vi = (NK + k) * B + ts;
    if (vi < nvr) {
      float g[V];
#pragma unroll
      for (int j = 0; j < V; ++j) g[j] = mine[k * B * V + j] * r;
      if (SHIFT && vi + 1 == nvr)
        store_inside<DT>(yrow, vi, s, cols, g);
      else
        __builtin_nontemporal_store(pack<DT>(g), yr + vi);
    }
  }
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
  const bool full = !CAUSAL && nvr == (uint32_t)(64 * WAVES * NV);
  for (int64_t r0 = 0; r0 < a.rows; r0 += kRowChunk) {
    const int64_t nr = std::min(kRowChunk, a.rows - r0);
    const uint32_t grid = (uint32_t)((nr + RPB - 1) / RPB);
    if (full)
      hipLaunchKernelGGL((sm_rows_kernel<DT, MODE, FUSE, CAUSAL, NV, WAVES, true>), dim3(grid),
                         dim3(kSmBlock), 0, a.s, a.x + r0 * a.ldx_b, a.y + r0 * a.ldy_b,
                         (uint32_t)nr, nvr, a.ldx_b, a.ldy_b, a.kc, causal_at(a, r0));
    else
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

// Register and LDS shapes of the row-resident kernel (vectors per thread):
// NK2 blocks in VGPRs at two workgroups per CU (at most 128 VGPRs); NK1 blocks
// at one workgroup per CU; NK1 blocks plus NL1 blocks in LDS (147-156 KB).
template <int DT>
struct ResShape {
  static constexpr int NK2 = (DT == F32) ? 24 : 12;
  static constexpr int NK1 = (DT == F32) ? 44 : 23;
  static constexpr int NL1 = (DT == F32) ? 19 : 9;
  static constexpr uint32_t kMax = (uint32_t)((NK1 + NL1) * kResBlock);
};

template <int DT, int MODE, bool FUSE, bool CAUSAL>
static quake_status launch_long(const SmArgs& a) {
  constexpr int V = kV<DT>;
  constexpr int64_t kLongRows = int64_t(1) << 30;      // rows per launch (one workgroup each)
  typedef ResShape<DT> RS;
  const uint32_t nvr = (uint32_t)(a.cols / V);
  for (int64_t r0 = 0; r0 < a.rows; r0 += kLongRows) {
    const int64_t nr = std::min(kLongRows, a.rows - r0);
    const char* xp = a.x + r0 * a.ldx_b;
    char* yp = a.y + r0 * a.ldy_b;
    const dim3 grid((uint32_t)nr);
    if (!CAUSAL && nvr <= (uint32_t)(RS::NK2 * kResBlock))
      hipLaunchKernelGGL((sm_res_kernel<DT, MODE, FUSE, RS::NK2, 0, false, 2>), grid,
                         dim3(kResBlock), 0, a.s, xp, yp, nvr, a.ldx_b, a.ldy_b, a.kc);
    else if (!CAUSAL && nvr <= (uint32_t)(RS::NK1 * kResBlock))
      hipLaunchKernelGGL((sm_res_kernel<DT, MODE, FUSE, RS::NK1, 0, false, 1>), grid,
                         dim3(kResBlock), 0, a.s, xp, yp, nvr, a.ldx_b, a.ldy_b, a.kc);
    else if (!CAUSAL && nvr <= RS::kMax)   // every register block inside the row
      hipLaunchKernelGGL((sm_res_kernel<DT, MODE, FUSE, RS::NK1, RS::NL1, true, 1>), grid,
                         dim3(kResBlock), 0, a.s, xp, yp, nvr, a.ldx_b, a.ldy_b, a.kc);
    else
      hipLaunchKernelGGL((sm_long_kernel<DT, MODE, FUSE, CAUSAL>), grid, dim3(kLongBlock), 0,
                         a.s, xp, yp, nvr, a.ldx_b, a.ldy_b, a.kc, causal_at(a, r0));
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

// Split-row geometry: 64 elements per lane per chunk (16 vectors of binary32,
// 8 of 16-bit), 256 lanes per workgroup, so a chunk is 16384 elements; rows of
// more than one chunk and at most kMaxG chunks exchange through a workspace.
constexpr int64_t kChunkElems = 16384;
constexpr int64_t kSplitRows = 1024;   // rows per launch: the workspace holds their slots

static bool split_chunks(int64_t cols, uint32_t* G) {
  if (cols <= kChunkElems || cols > kChunkElems * kMaxG) return false;
  *G = (uint32_t)((cols + kChunkElems - 1) / kChunkElems);
  return true;
}

static int64_t split_ws_bytes(int64_t rows, int64_t cols) {
  uint32_t G = 0;
  if (rows <= 0 || !split_chunks(cols, &G)) return 0;
  const int64_t R = std::min(rows, kSplitRows);
  const int64_t b = (int64_t)kWsHeader + R * G * 12 + R * 4;
  return (b + 255) / 256 * 256;
}

static SplitWs split_ws_view(char* base, int64_t rows, uint32_t G) {
  const int64_t S = std::min(rows, kSplitRows) * G;
  SplitWs w;
  w.hdr = reinterpret_cast<uint32_t*>(base);
  w.psum = reinterpret_cast<uint64_t*>(base + kWsHeader);
  w.pmax = reinterpret_cast<uint32_t*>(base + kWsHeader + 8 * S);
  w.done = reinterpret_cast<uint32_t*>(base + kWsHeader + 12 * S);
  return w;
}

// SHIFT: rows not 16-byte aligned; the chunk count (and the workspace's
// layout) is the one of cols, which the caller has checked covers the most
// vectors such a row can span.
template <int DT, int MODE, bool FUSE, bool CAUSAL, bool SHIFT = false>
static quake_status launch_split(const SmArgs& a, char* ws) {
  constexpr int V = kV<DT>;
  constexpr int NV = (DT == F32) ? 16 : 8;
  static_assert(kSmBlock * NV * V == kChunkElems, "chunk geometry");
  uint32_t G = 0;
  if (!split_chunks(a.cols, &G)) return QUAKE_EINVAL;
  const uint32_t nvr = SHIFT ? (uint32_t)a.cols : (uint32_t)(a.cols / V);
  const SplitWs w = split_ws_view(ws, a.rows, G);
  for (int64_t r0 = 0; r0 < a.rows; r0 += kSplitRows) {
    const int64_t nr = std::min(kSplitRows, a.rows - r0);
    const uint32_t xcd = (nr % 8 == 0 && G <= 32) ? 1u : 0u;
    hipLaunchKernelGGL((sm_split_kernel<DT, MODE, FUSE, CAUSAL, NV, SHIFT>), dim3((uint32_t)(nr * G)),
                       dim3(kSmBlock), 0, a.s, a.x + r0 * a.ldx_b, a.y + r0 * a.ldy_b, nvr, a.ldx_b,
                       a.ldy_b, a.kc, causal_at(a, r0), G, xcd, w);
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

// Rows whose start is not 16-byte aligned, at the same offset in x and y:
// the register-row kernels (up to 16384 elements, also with the implicit
// causal mask) and the row-resident kernel (up to its capacity) read the
// aligned vectors that cover each row. Classes by the most vectors a row of
// this length can cover, (cols + 2V - 2) / V.
template <int DT>
static bool shifted_fits(const void* x, const void* y, int64_t rows, int64_t cols, int64_t ldx,
                         int64_t ldy) {
  constexpr int64_t esz = kEsz<DT>;
  const uintptr_t ux = (uintptr_t)x, uy = (uintptr_t)y;
  return ux % esz == 0 && uy % esz == 0 && ((ux - uy) & 15u) == 0 &&
         (rows <= 1 || (((ldx & 15) * esz) & 15) == (((ldy & 15) * esz) & 15)) &&
         cols < (int64_t(1) << 31);
}

template <int DT, int MODE, bool CAUSAL, int NV, int WAVES>
static quake_status launch_rows_shifted(const SmArgs& a) {
  constexpr int RPB = kSmBlock / (64 * WAVES);
  for (int64_t r0 = 0; r0 < a.rows; r0 += kRowChunk) {
    const int64_t nr = std::min(kRowChunk, a.rows - r0);
    const uint32_t grid = (uint32_t)((nr + RPB - 1) / RPB);
    hipLaunchKernelGGL((sm_rows_kernel<DT, MODE, true, CAUSAL, NV, WAVES, false, true>),
                       dim3(grid), dim3(kSmBlock), 0, a.s, a.x + r0 * a.ldx_b,
                       a.y + r0 * a.ldy_b, (uint32_t)nr, (uint32_t)a.cols, a.ldx_b, a.ldy_b,
                       a.kc, causal_at(a, r0));
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

template <int DT, int MODE>
static quake_status launch_res_shifted(const SmArgs& a) {
  constexpr int V = kV<DT>;
  constexpr int64_t kResRows = int64_t(1) << 30;       // rows per launch (one workgroup each)
  typedef ResShape<DT> RS;
  const int64_t nvm = (a.cols + 2 * V - 2) / V;
  const uint32_t cols = (uint32_t)a.cols;
  for (int64_t r0 = 0; r0 < a.rows; r0 += kResRows) {
    const int64_t nr = std::min(kResRows, a.rows - r0);
    const char* xp = a.x + r0 * a.ldx_b;
    char* yp = a.y + r0 * a.ldy_b;
    const dim3 grid((uint32_t)nr);
    if (nvm <= RS::NK2 * kResBlock)
      hipLaunchKernelGGL((sm_res_kernel<DT, MODE, true, RS::NK2, 0, false, 2, true>), grid,
                         dim3(kResBlock), 0, a.s, xp, yp, cols, a.ldx_b, a.ldy_b, a.kc);
    else if (nvm <= RS::NK1 * kResBlock)
      hipLaunchKernelGGL((sm_res_kernel<DT, MODE, true, RS::NK1, 0, false, 1, true>), grid,
                         dim3(kResBlock), 0, a.s, xp, yp, cols, a.ldx_b, a.ldy_b, a.kc);
    else
      hipLaunchKernelGGL((sm_res_kernel<DT, MODE, true, RS::NK1, RS::NL1, true, 1, true>), grid,
                         dim3(kResBlock), 0, a.s, xp, yp, cols, a.ldx_b, a.ldy_b, a.kc);
    const quake_status st = launch_status();
    if (st != QUAKE_OK) return st;
  }
  return QUAKE_OK;
}

// Whether the shifted-row kernels take rows of this length (the implicit
// causal mask only in the register-row kernels).
template <int DT, bool CAUSAL>
static bool shifted_length(int64_t cols) {
  constexpr int V = kV<DT>;
  const int64_t nvm = (cols + 2 * V - 2) / V;
  if (CAUSAL) return nvm <= (DT == F32 ? 4096 : 2048);
  return nvm <= (int64_t)ResShape<DT>::kMax;
}

template <int DT, int MODE, bool CAUSAL>
static quake_status launch_shifted(const SmArgs& a) {
  constexpr int V = kV<DT>;
  const int64_t nvm = (a.cols + 2 * V - 2) / V;
  if (nvm <= 64) return launch_rows_shifted<DT, MODE, CAUSAL, 1, 1>(a);
  if (nvm <= 128) return launch_rows_shifted<DT, MODE, CAUSAL, 2, 1>(a);
  if (nvm <= 256) return launch_rows_shifted<DT, MODE, CAUSAL, 4, 1>(a);
  if (nvm <= 512) return launch_rows_shifted<DT, MODE, CAUSAL, 8, 1>(a);
  if (nvm <= 1024) return launch_rows_shifted<DT, MODE, CAUSAL, 4, 4>(a);
  if (nvm <= 2048) return launch_rows_shifted<DT, MODE, CAUSAL, 8, 4>(a);
  if constexpr (DT == F32) {
    if (nvm <= 4096) return launch_rows_shifted<DT, MODE, CAUSAL, 16, 4>(a);
  }
  if constexpr (CAUSAL) return QUAKE_EINVAL;   // excluded by shifted_length
  else return launch_res_shifted<DT, MODE>(a);
}

template <int DT, int MODE, bool FUSE, bool CAUSAL>
static quake_status sm_dispatch(const void* x, void* y, int64_t ldx, int64_t ldy, const SmArgs& ain,
                                char* ws) {
  constexpr int V = kV<DT>;
  constexpr int64_t esz = kEsz<DT>;
  const int64_t cols = ain.cols;
  const bool vec = aligned16(x) && aligned16(y) && (ldx * esz) % 16 == 0 && (ldy * esz) % 16 == 0 &&
                   cols % V == 0 && cols < (int64_t(1) << 31) - 16;
  SmArgs a = ain;
  a.x = static_cast<const char*>(x);
  a.y = static_cast<char*>(y);
  a.ldx_b = ldx * esz;
  a.ldy_b = ldy * esz;
  if (!vec) {
    if constexpr (FUSE) {
      if (shifted_fits<DT>(x, y, a.rows, cols, ldx, ldy)) {
        if constexpr (!CAUSAL) {
          // longer than the register-row kernels, with a workspace: the split
          // rows, when cols' chunk count covers every row's vectors
          const int64_t nvm = (cols + 2 * V - 2) / V;
          uint32_t G = 0, Gs = 0;
          if (ws != nullptr && nvm > (DT == F32 ? 4096 : 2048) && split_chunks(cols, &G) &&
              split_chunks(nvm * V, &Gs) && Gs == G)
            return launch_split<DT, MODE, FUSE, CAUSAL, true>(a, ws);
        }
        if (shifted_length<DT, CAUSAL>(cols)) return launch_shifted<DT, MODE, CAUSAL>(a);
      }
    }
    return launch_generic<DT, MODE, FUSE, CAUSAL>(x, y, ain, ldx, ldy);
  }
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
  // Longer rows: chunks exchanged between workgroups through the caller's
  // workspace, or, without one, a workgroup per row holding the whole row in
  // VGPRs and LDS (sm_res), or reading it three times when it does not fit or
  // is causal (sm_long).
  if constexpr (FUSE && !CAUSAL) {
    uint32_t G = 0;
    if (ws != nullptr && split_chunks(cols, &G)) return launch_split<DT, MODE, FUSE, CAUSAL>(a, ws);
  }
  return launch_long<DT, MODE, FUSE, CAUSAL>(a);
}

template <bool FUSE, bool CAUSAL>
static quake_status softmax_entry(const void* x, void* y, int64_t rows, int64_t cols, int64_t ldx,
                                  int64_t ldy, int dtype, int mode, float t, int64_t period,
                                  int64_t shift, int write_masked, void* ws, int64_t ws_bytes,
                                  void* stream, bool check_only = false) {
  if (!valid_dtype(dtype)) return QUAKE_EDTYPE;
  if (!valid_mode(mode)) return QUAKE_EMODE;
  if (rows < 0 || cols < 0 || ldx < 0 || ldy < 0 || ws_bytes < 0) return QUAKE_EINVAL;
  if (CAUSAL && (period <= 0 || period > INT32_MAX || shift < -(int64_t(1) << 40) ||
                 shift > (int64_t(1) << 40)))
    return QUAKE_EINVAL;
  if (ws != nullptr && (((uintptr_t)ws & 15u) != 0 || ws_bytes < split_ws_bytes(rows, cols)))
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
  if (check_only) return QUAKE_OK;
  const SmArgs a{static_cast<const char*>(x), static_cast<char*>(y), rows, cols, 0, 0, kc,
                 CAUSAL ? period : 0, shift, (uint32_t)(write_masked != 0),
                 static_cast<hipStream_t>(stream)};
  char* w = static_cast<char*>(ws);
#define QK_SM_CASE(D, M) \
  if (dtype == D && mode == M) return sm_dispatch<D, M, FUSE, CAUSAL>(x, y, ldx, ldy, a, w);
  QK_SM_CASE(F32, EXACT) QK_SM_CASE(F32, Q1) QK_SM_CASE(F32, Q2) QK_SM_CASE(F32, Q2M)
  QK_SM_CASE(F16, EXACT) QK_SM_CASE(F16, Q1) QK_SM_CASE(F16, Q2) QK_SM_CASE(F16, Q2M)
  QK_SM_CASE(BF16, EXACT) QK_SM_CASE(BF16, Q1) QK_SM_CASE(BF16, Q2) QK_SM_CASE(BF16, Q2M)
#undef QK_SM_CASE
  return QUAKE_EMODE;
}

// ---------------------------------------------------------------------------
// Fixed scratch for callers that cannot allocate (quake_softmax_noalloc): the
// split-row exchange's workspace as a device array of the library, one copy
// per device, zero at load and zeroed once more at set-up on each device.
// ---------------------------------------------------------------------------
constexpr int64_t kScratchBytes = 256 * 1024;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
static std::mutex g_scratch_mu;
static char* g_scratch_ptr[kMaxScratchDevices];   // device address of `scratch`, per device

__global__ void scratch_zero_kernel(uint32_t* p, uint32_t n) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0u;
}

// Device address of the current device's scratch. The first call on a device
// looks the array up (its name is only a host-side stand-in) and clears it
// with a kernel on `s`, ahead of the caller's own kernels on that stream.
static quake_status scratch_on_current_device(hipStream_t s, char** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return QUAKE_EHIP;
  if (dev < 0 || dev >= kMaxScratchDevices) return QUAKE_EHIP;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return QUAKE_EHIP;
    hipLaunchKernelGGL(scratch_zero_kernel, dim3(64), dim3(256), 0, s, static_cast<uint32_t*>(p),
                       (uint32_t)(kScratchBytes / 4));
    if (hipGetLastError() != hipSuccess) return QUAKE_EHIP;
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return QUAKE_OK;
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_softmax_noalloc(const void* x, void* y, int64_t rows, int64_t cols,
                                              int64_t ldx, int64_t ldy, quake_dtype dtype,
                                              quake_mode mode, float t, void* stream) {
  quake_status st = softmax_entry<true, false>(x, y, rows, cols, ldx, ldy, dtype, mode, t, 0, 0, 1,
                                               nullptr, 0, stream, true);
  if (st != QUAKE_OK || rows == 0) return st;
  const int64_t need = split_ws_bytes(rows, cols);
  if (need == 0)   // no exchange for this shape: exactly quake_softmax
    return softmax_entry<true, false>(x, y, rows, cols, ldx, ldy, dtype, mode, t, 0, 0, 1,
                                      nullptr, 0, stream);
  if (need > kScratchBytes) return QUAKE_ENOSCRATCH;
  char* ws = nullptr;
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = scratch_on_current_device(s, &ws);
  if (st != QUAKE_OK) return st;
  return softmax_entry<true, false>(x, y, rows, cols, ldx, ldy, dtype, mode, t, 0, 0, 1, ws,
                                    kScratchBytes, stream);
}

extern "C" quake_status quake_softmax(const void* x, void* y, int64_t rows, int64_t cols,
                                      int64_t ldx, int64_t ldy, quake_dtype dtype,
                                      quake_mode mode, float t, void* stream) {
  return softmax_entry<true, false>(x, y, rows, cols, ldx, ldy, dtype, mode, t, 0, 0, 1, nullptr,
                                    0, stream);
}

extern "C" quake_status quake_softmax_workspace_size(int64_t rows, int64_t cols,
                                                     quake_dtype dtype, int64_t* bytes) {
  if (bytes == nullptr) return QUAKE_EINVAL;
  *bytes = 0;
  if (!valid_dtype(dtype)) return QUAKE_EDTYPE;
  if (rows < 0 || cols < 0) return QUAKE_EINVAL;
  *bytes = split_ws_bytes(rows, cols);
  return QUAKE_OK;
}

extern "C" quake_status quake_softmax_ws(const void* x, void* y, int64_t rows, int64_t cols,
                                         int64_t ldx, int64_t ldy, quake_dtype dtype,
                                         quake_mode mode, float t, void* workspace,
                                         int64_t workspace_bytes, void* stream) {
  return softmax_entry<true, false>(x, y, rows, cols, ldx, ldy, dtype, mode, t, 0, 0, 1,
                                    workspace, workspace_bytes, stream);
}

extern "C" quake_status quake_softmax_unfused(const void* x, void* y, int64_t rows, int64_t cols,
                                              int64_t ldx, int64_t ldy, quake_dtype dtype,
                                              quake_mode mode, float t, void* stream) {
  return softmax_entry<false, false>(x, y, rows, cols, ldx, ldy, dtype, mode, t, 0, 0, 1, nullptr,
                                     0, stream);
}

extern "C" quake_status quake_softmax_causal(const void* x, void* y, int64_t rows, int64_t cols,
                                             int64_t ldx, int64_t ldy, int64_t period,
                                             int64_t shift, int write_masked, quake_dtype dtype,
                                             quake_mode mode, float t, void* stream) {
  return softmax_entry<true, true>(x, y, rows, cols, ldx, ldy, dtype, mode, t, period, shift,
                                   write_masked, nullptr, 0, stream);
}
