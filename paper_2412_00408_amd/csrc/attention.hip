// attention.hip — quake_attention: O = softmax(t Q K^T) V per head (optionally
// causal), bfloat16 or binary16, with the softmax of Algorithm 2
// (arXiv:2412.00408, Sec. III-C) taken against each query's final row max.
// Every exponential of a query waits for the max of its whole row, so there is
// no online rescaling: QuAKE is not multiplicative (Q(a) Q(b) != Q(a + b)), and
// a flash-style running max would change the results Algorithm 2 defines. Up
// to 1024 keys the scores of a query stay in registers (attn_kernel, four
// waves up to 512 keys, eight beyond); longer sequences compute them twice,
// once for the max and once for the exponentials (attn_long_kernel).
//
// One workgroup = 32 queries of one head, W waves; wave w takes the 32-key
// blocks w, w + W, w + 2 W, ... (interleaved, so causal work stays balanced).
// The scores are computed transposed, S^T = K Q^T, on the matrix cores
// (v_mfma_f32_32x32x16_bf16 / _f16; A = 32 keys x 16 dims of K, staged through
// LDS as described below, B = the 32 queries' dims read straight from Q's
// rows), so that lane l holds one query (l mod 32) and keys
// 8 g + 4 (l / 32) + i, g, i < 4, of each block:
//   * the row max and the row sum reduce the lane's own values, exchange once
//     with lane l xor 32 (v_permlane32_swap) and once across waves through LDS;
//   * the exponentials, rounded to the 16-bit format, become the B operand of
//     the second product O^T = V^T P after one v_permlane32_swap per dword pair
//     (lane l < 32 takes keys 4-7 from its partner and gives it keys 8-11),
//     without a trip through LDS. V is passed transposed ([head, dim, key]), so
//     the A operand (32 dims x 16 keys) is 16 contiguous bytes of a row of V^T.
// Causal key blocks above a query block's diagonal are neither loaded nor
// multiplied. The W partial O^T meet in LDS; each wave adds up, normalises by
// 1 / sum and stores 1 / W of the 32 x 64 output tile.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kAttnD = 64;              // head dimension
constexpr int kAttnBlk = 4;             // key blocks of 32 per wave, one pass
constexpr int kAttnMaxWaves = 8;        // waves of the largest one-pass workgroup
constexpr int kAttnMaxS = 32 * kAttnBlk * kAttnMaxWaves;   // longest one-pass sequence: 1024
constexpr int kAttnLongMaxS = 131072;   // longest sequence (two-pass kernel)
constexpr int kAttnQ = 32;              // queries per workgroup
constexpr int kAttnWaves = 4;           // waves of the two-pass workgroup
constexpr int kAttnThreads = 64 * kAttnWaves;
// Two-pass workgroups take two groups of 32 queries from this many such
// tiles on (two workgroups per CU of 256 without the mask; with it four, as
// the longest causal tiles then take twice as long and the launch's tail
// grows), else one group.
constexpr int kAttnLongQGMinTiles = 512, kAttnLongQGMinTilesCausal = 1024;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* vt;
  uint16_t* o;
  int32_t s;         // sequence length, 1 .. 131072
  int32_t ldv;       // row stride of V^T in elements, >= s
  int32_t qtiles;    // query tiles of the launched kernel: ceil(s / 32), two-pass ceil(s / 64)
  float c0;          // Algorithm 2: 2^23 t / ln2 (EXACT: t / ln2)
  uint32_t causal;
  uint32_t xcd_heads;   // heads a multiple of 8: heads per XCD, else 0
};

__device__ __forceinline__ u32x4_t ld16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

// One 32x32x16 matrix-core step on raw 16-bit operands of format DT
// (bfloat16 or binary16), and two binary32 values rounded to a DT pair.
template <int DT>
__device__ __forceinline__ f32x16_t mma(u32x4_t a, u32x4_t b, f32x16_t c) {
  if constexpr (DT == BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                  __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}
template <int DT>
__device__ __forceinline__ uint32_t pack16(float a, float b) {
  if constexpr (DT == BF16)
    return pack_bf16(a, b);
  else
    return pack_f16(a, b);
}

// the value held by lane l xor 32
__device__ __forceinline__ float xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(as_u(v), as_u(v), false, false);
  return as_f((threadIdx.x & 32) ? r[0] : r[1]);
}

// Operand staging. The matrix cores want lane (r, h) = (lane mod 32, lane / 32)
// to hold 16 bytes of row r of a 32-row block; loaded straight from global
// memory that is 32 rows per instruction. Instead each block is read with
// whole rows per instruction (coalesced), written to the wave's own LDS slots
// and read back in operand layout; 16-byte slots are XOR-swizzled so that
// both the writes and the operand reads are free of bank conflicts (whether
// the LDS serves 8 lanes of a 16-byte access per clock over 32 banks or 16
// lanes over 64 banks). A wave
// writes a block, reads it back and only then writes the next one, so one
// buffer per wave suffices (LDS operations of a wave complete in order).
//
// K block: 32 keys x 128 B. Slot of (row r, chunk c): 8 r + (c ^ fk(r)) with
// fk(r) = (r mod 8) ^ ((r / 8) mod 2).
// Load j of 4 covers rows 8 j .. 8 j + 7; lane l takes row 8 j + l / 8,
// chunk l mod 8, at byte koff = 128 (l / 8) + 16 (l mod 8) + 1024 j from the
// block's first row (a uniform base, so only koff lives in a vector register).
// In a block that reaches past s, rows past s are clamped to row s - 1 (their
// scores are masked afterwards).
__device__ __forceinline__ uint32_t kblock_lane_offset(int lane) {
  return (uint32_t)(128 * (lane >> 3) + 16 * (lane & 7));
}
__device__ __forceinline__ void kblock_load(const uint16_t* k, int kbase, int s, int lane,
                                            uint32_t koff, u32x4_t (&g)[4]) {
  if (kbase + 32 <= s) {
    const char* base = reinterpret_cast<const char*>(k + (int64_t)kbase * kAttnD);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      g[j] = *reinterpret_cast<const u32x4_t*>(base + koff + 1024 * j);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = min(kbase + 8 * j + (lane >> 3), s - 1);
      g[j] = ld16(k + (int64_t)row * kAttnD + 8 * (lane & 7));
    }
  }
}
__device__ __forceinline__ int kswz(int r) { return (r & 7) ^ ((r >> 3) & 1); }
__device__ __forceinline__ void kblock_store(u32x4_t* buf, int lane, const u32x4_t (&g)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = 8 * j + (lane >> 3);
    buf[8 * r + ((lane & 7) ^ kswz(r))] = g[j];
  }
}
// A operands of S^T = K Q^T: 16-dim step ks, dims 16 ks + 8 h .. + 7 of key fr
__device__ __forceinline__ void kblock_read(const u32x4_t* buf, int fr, int h, u32x4_t (&a)[4]) {
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
    a[ks] = buf[8 * fr + ((2 * ks + h) ^ kswz(fr))];
}

// Layouts of V^T the kernel is built for: sequence a multiple of 32 with
// 16-byte rows (no block reaches past s), any sequence with 16-byte rows, and
// any sequence with rows of any alignment.
enum VtKind { kVtFull = 0, kVtRagged = 1, kVtScalar = 2 };

// V^T block: 64 dims x 32 keys (64 B). Slot of (row d, chunk c):
// 4 d + (c ^ fv(d)) with fv(d) = ((d / 2) ^ (d / 4)) mod 4. Load j of 4 covers
// rows 16 j .. 16 j + 15; lane l takes row 16 j + l / 4, keys kbase + 8 (l mod 4)
// .. + 7, at byte voff[j] = 2 ((16 j + l / 4) ldv + 8 (l mod 4)) from key
// kbase of row 0 (a uniform base). In a block that reaches past s (`tail`,
// uniform) keys at or past s read as zero without leaving the row: their
// probabilities are zero, and the padding of the row may hold anything.
__device__ __forceinline__ void vblock_lane_offsets(int lane, int ldv, uint32_t (&voff)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
    voff[j] = 2u * ((uint32_t)(16 * j + (lane >> 2)) * (uint32_t)ldv + 8u * (uint32_t)(lane & 3));
}
template <int VK>
__device__ __forceinline__ void vblock_load(const uint16_t* vt, int ldv, int kbase, int s,
                                            bool tail, int lane, const uint32_t (&voff)[4],
                                            u32x4_t (&g)[4]) {
  if (VK != kVtScalar && !tail) {
    const char* base = reinterpret_cast<const char*>(vt + kbase);
#pragma unroll
    for (int j = 0; j < 4; ++j) g[j] = *reinterpret_cast<const u32x4_t*>(base + voff[j]);
    return;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint16_t* row = vt + (int64_t)(16 * j + (lane >> 2)) * ldv;
    const int key0 = kbase + 8 * (lane & 3);
    u32x4_t v;
    if constexpr (VK != kVtScalar) {
      const int nv = s - key0;
      v = ld16(row + (nv > 0 ? key0 : 0));
#pragma unroll
      for (int i = 0; i < 4; ++i)
        v[i] = (2 * i + 1 < nv) ? v[i] : ((2 * i < nv) ? (v[i] & 0xFFFFu) : 0u);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k0 = key0 + 2 * i, k1 = k0 + 1;
        const uint32_t lo = (!tail || k0 < s) ? row[(!tail || k0 < s) ? k0 : 0] : 0u;
        const uint32_t hi = (!tail || k1 < s) ? row[(!tail || k1 < s) ? k1 : 0] : 0u;
        v[i] = lo | (hi << 16);
      }
    }
    g[j] = v;
  }
}
__device__ __forceinline__ int vswz(int d) { return ((d >> 1) ^ (d >> 2)) & 3; }
__device__ __forceinline__ void vblock_store(u32x4_t* buf, int lane, const u32x4_t (&g)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int d = 16 * j + (lane >> 2);
    buf[4 * d + ((lane & 3) ^ vswz(d))] = g[j];
  }
}
// A operands of O^T = V^T P: 16-key step ks, 32-dim half db; keys
// 16 ks + 8 h .. + 7 of dim 32 db + fr
__device__ __forceinline__ void vblock_read(const u32x4_t* buf, int fr, int h,
                                            u32x4_t (&a)[2][2]) {
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int db = 0; db < 2; ++db) {
      const int d = 32 * db + fr;
      a[ks][db] = buf[4 * d + ((2 * ks + h) ^ vswz(d))];
    }
}

// Sum of the N values v[LO .. LO + N) in a fixed pairwise order:
// ((v0 + v1) + (v2 + v3)) + ...
template <int LO, int N, int TOTAL>
__device__ __forceinline__ float tree_sum(const float (&v)[TOTAL]) {
  if constexpr (N == 1)
    return v[LO];
  else
    return tree_sum<LO, N / 2, TOTAL>(v) + tree_sum<LO + N / 2, N / 2, TOTAL>(v);
}

// End of a tile of W waves and QG groups of 32 queries: the row sums over the
// waves, the W partial O^T through LDS (each wave's own 8 KB region, its
// staging reads done; one group after the other), and the output. Accumulator
// register r of oacc[c][db] in lane l holds dim 32 db + 8 (r / 4) + 4 (l / 32) +
// r mod 4 of query 32 c + l mod 32 of the tile; call j = 16 db + r its row.
// Wave w adds rows R w .. R w + R - 1 (R = 32 / W) over the waves in a fixed
// order, normalises them by 1 / sum and stores them, four consecutive dims
// (8 bytes) at a time. Every wave reaches every barrier: lanes of queries past
// s only skip their stores.
template <int DT, int W, int QG>
__device__ __forceinline__ void attn_finish(u32x4_t (*s_buf)[512], float* s_sum,
                                            const f32x16_t (&oacc)[QG][2], const float (&part)[QG],
                                            const float (&m)[QG], int wave, int lane, int q0,
                                            int S, uint16_t* ohead) {
  constexpr int R = 32 / W;
  static_assert(W == 4 || W == 8, "four or eight waves");
  const int fr = lane & 31;
#pragma unroll
  for (int c = 0; c < QG; ++c) {
    const float p = part[c] + xor32(part[c]);
    if (lane < 32) s_sum[(wave * QG + c) * 32 + lane] = p;
  }
#pragma unroll
  for (int c = 0; c < QG; ++c) {
    if (c > 0) __syncthreads();   // every wave has read the previous group's partials
    __builtin_amdgcn_wave_barrier();
    float* po = reinterpret_cast<float*>(s_buf[wave]);
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) po[(db * 16 + r) * 64 + lane] = oacc[c][db][r];
    __syncthreads();
    const int query = q0 + 32 * c + fr;
    if (query < S) {
      float sums[W];
#pragma unroll
      for (int w = 0; w < W; ++w) sums[w] = s_sum[(w * QG + c) * 32 + fr];
      const float total = tree_sum<0, W, W>(sums);
      const float inv = (m[c] == -INFINITY || !(total > 0.0f)) ? 0.0f : 1.0f / total;
      float v[R];
#pragma unroll
      for (int i = 0; i < R; ++i) {
        const int idx = (R * wave + i) * 64 + lane;
        float parts[W];
#pragma unroll
        for (int w = 0; w < W; ++w) parts[w] = reinterpret_cast<const float*>(s_buf[w])[idx];
        v[i] = tree_sum<0, W, W>(parts) * inv;
      }
      uint16_t* orow = ohead + (int64_t)query * kAttnD;
      // row R wave + i: db = that / 16, r = that mod 16; four dims per store
#pragma unroll
      for (int i = 0; i < R; i += 4) {
        const int j = R * wave + i, db = j >> 4, r = j & 15;
        uint2 w2;
        w2.x = pack16<DT>(v[i], v[i + 1]);
        w2.y = pack16<DT>(v[i + 2], v[i + 3]);
        *reinterpret_cast<uint2*>(orow + 32 * db + 8 * (r >> 2) + 4 * (lane >> 5)) = w2;
      }
    }
  }
}

// One pass, up to 128 W keys (W = 4 or 8 waves): every score of the tile
// stays in registers, four key blocks per wave at most. With 8 waves (513 to
// 1024 keys) two workgroups share a CU (66 KB of LDS each); a 16-wave
// workgroup (one per CU) for 2048 keys was measured slower than two passes
// with the mask and no faster without it.
template <int DT, int MODE, int VK, int W>
__global__ __launch_bounds__(64 * W, W == 4 ? 4 : 1) void attn_kernel(AttnArgs g) {
  __shared__ float s_max[W][kAttnQ];
  __shared__ float s_sum[W][kAttnQ];
  // per wave: operand staging (4 KB), then its partial O^T (8 KB)
  __shared__ u32x4_t s_buf[W][512];

  const int lane = threadIdx.x & 63;
  // uniform across the wave: every condition below that depends on it is a
  // scalar branch
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // Tile order. blockIdx round-robins over the 8 XCDs; with the heads a
  // multiple of 8, XCD x takes heads x H8 .. x H8 + H8 - 1 (H8 = heads / 8), so
  // their K and V stay in that XCD's L2, and it starts its tiles longest causal
  // rows first across all its heads (query tile qtiles - 1 of every head, then
  // qtiles - 2, ...), which keeps the end of the launch from waiting on a few
  // long tiles started late.
  int bh, qb;
  if (g.xcd_heads) {
    const uint32_t x = blockIdx.x & 7u, slot = blockIdx.x >> 3;
    bh = (int)(x * g.xcd_heads + slot % g.xcd_heads);
    qb = g.qtiles - 1 - (int)(slot / g.xcd_heads);
  } else {
    bh = (int)(blockIdx.x / (uint32_t)g.qtiles);
    qb = g.qtiles - 1 - (int)(blockIdx.x % (uint32_t)g.qtiles);
  }
  const int S = g.s;
  const int q0 = qb * kAttnQ;
  const int kblocks = (S + 31) >> 5;
  const int nkb = g.causal ? min(kblocks, qb + 1) : kblocks;   // live key blocks of the tile
  // this wave's blocks are w, w + W, ...: the first nlive of them are live
  const int nlive = max(0, (nkb - wave + W - 1) / W);
  const int fr = lane & 31, fk = 8 * (lane >> 5);
  const int query = q0 + fr;
  const uint16_t* Q = g.q + (int64_t)bh * S * kAttnD;
  const uint16_t* K = g.k + (int64_t)bh * S * kAttnD;
  const uint16_t* Vt = g.vt + (int64_t)bh * kAttnD * g.ldv;

  // S^T = K Q^T over the live key blocks, the next block's K in flight
  u32x4_t qf[4];
  {
    const uint16_t* qr = Q + (int64_t)min(query, S - 1) * kAttnD + fk;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qf[ks] = ld16(qr + 16 * ks);
  }
  u32x4_t* stage = s_buf[wave];
  const int h = lane >> 5;
  const uint32_t koff = kblock_lane_offset(lane);
  uint32_t voff[4];
  vblock_lane_offsets(lane, g.ldv, voff);
  u32x4_t gk[4];
  if (nlive > 0) kblock_load(K, 32 * wave, S, lane, koff, gk);
  f32x16_t sacc[kAttnBlk];
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < kAttnBlk; ++i) {
    if (i < nlive) {
      const int kbg = W * i + wave;
      kblock_store(stage, lane, gk);
      if (i + 1 < nlive) kblock_load(K, 32 * (kbg + W), S, lane, koff, gk);
      __builtin_amdgcn_wave_barrier();   // lanes read what other lanes wrote
      u32x4_t ka[4];
      kblock_read(stage, fr, h, ka);
      __builtin_amdgcn_wave_barrier();   // before the slots are written again
      const f32x16_t zero = {};
      sacc[i] = mma<DT>(ka[0], qf[0], zero);
#pragma unroll
      for (int ks = 1; ks < 4; ++ks)
        sacc[i] = mma<DT>(ka[ks], qf[ks], sacc[i]);
      const bool diag = g.causal && kbg == qb;
      if (diag || (VK != kVtFull && 32 * kbg + 32 > S)) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * kbg + 8 * (r >> 2) + 4 * h + (r & 3);
          if (key >= S || (diag && key > query)) sacc[i][r] = -INFINITY;
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) m = fmaxf(m, sacc[i][r]);
    }
  }
  // the first block of V^T in flight across the reductions
  u32x4_t gv[4];
  if (nlive > 0)
    vblock_load<VK>(Vt, g.ldv, 32 * wave, S, VK != kVtFull && 32 * wave + 32 > S, lane, voff, gv);

  // row (query) max: the lane's own values, lane l xor 32, the other waves
  m = fmaxf(m, xor32(m));
  if (lane < 32) s_max[wave][lane] = m;
  __syncthreads();
  m = s_max[0][fr];
#pragma unroll
  for (int w = 1; w < W; ++w) m = fmaxf(m, s_max[w][fr]);

  // Algorithm 2: exponentials against the row max (c1 folds it in) and their
  // sum, every block's before the second product, so that the binary32
  // scores are dead before its accumulators and operands are live; the
  // probabilities rounded to 16-bit pairs (keys 8 gi + 4 (lane / 32) + 0..3 of
  // each block)
  const float c1 = (m == -INFINITY) ? 0.0f : __builtin_fmaf(-g.c0, m, MODE == EXACT ? 0.0f : kK127);
  float part = 0.0f;
  uint32_t pk[kAttnBlk][4][2];
  // the folded clamp (qexp_row) where registers allow a second copy of the
  // loop: with four waves the kernel is held to 128 VGPRs
  const bool below = W == 8 && row_c1_below(c1);
#pragma unroll
  for (int i = 0; i < kAttnBlk; ++i) {
    if (i < nlive) {
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        float e[4];
        if (W == 8 && below) {
#pragma unroll
          for (int j = 0; j < 4; ++j) e[j] = qexp_row<MODE, true>(sacc[i][4 * gi + j], g.c0, c1);
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) e[j] = qexp<MODE>(sacc[i][4 * gi + j], g.c0, c1);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) part += e[j];
        pk[i][gi][0] = pack16<DT>(e[0], e[1]);
        pk[i][gi][1] = pack16<DT>(e[2], e[3]);
      }
    }
  }

  // O^T = V^T P over this wave's live keys, the next block's V in flight
  f32x16_t oacc[2] = {};
#pragma unroll
  for (int i = 0; i < kAttnBlk; ++i) {
    if (i < nlive) {
      const int kbg = W * i + wave;
      vblock_store(stage, lane, gv);
      if (i + 1 < nlive) {
        const int nb = 32 * (kbg + W);
        vblock_load<VK>(Vt, g.ldv, nb, S, VK != kVtFull && nb + 32 > S, lane, voff, gv);
      }
      __builtin_amdgcn_wave_barrier();
      u32x4_t va[2][2];
      vblock_read(stage, fr, h, va);
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        // lanes < 32 end with keys 16 ks + 0..7, lanes >= 32 with 16 ks + 8..15
        const auto s0 = __builtin_amdgcn_permlane32_swap(pk[i][2 * ks][0], pk[i][2 * ks + 1][0],
                                                         false, false);
        const auto s1 = __builtin_amdgcn_permlane32_swap(pk[i][2 * ks][1], pk[i][2 * ks + 1][1],
                                                         false, false);
        const u32x4_t bv = {s0[0], s1[0], s0[1], s1[1]};
#pragma unroll
        for (int db = 0; db < 2; ++db)
          oacc[db] = mma<DT>(va[ks][db], bv, oacc[db]);
      }
    }
  }

  const f32x16_t oacc1[1][2] = {{oacc[0], oacc[1]}};
  const float part1[1] = {part}, m1[1] = {m};
  attn_finish<DT, W, 1>(s_buf, &s_sum[0][0], oacc1, part1, m1, wave, lane, q0, S,
                        g.o + (int64_t)bh * S * kAttnD);
}

// Sequences longer than 1024 keys: four waves and the same staging, but the
// scores are not kept. Pass 1 computes them to find each query's row max;
// pass 2 computes them again, block by block, and takes the exponentials
// against that max (Algorithm 2 needs the final max before any exponential),
// their sum and the second product. A workgroup takes QG groups of 32
// queries: every key and value block a wave stages serves all groups (one
// load and one trip through LDS for 32 QG queries), and the groups' products
// and exponentials are independent chains. Per query the scores, the max,
// the exponentials, the sums and the products are computed by the same
// instructions in the same order as in the one-pass kernel, so both give
// identical results. With the mask, the key block past group 0's diagonal
// (group 1's diagonal block) is skipped for group 0, as in the one-pass kernel.
template <int DT, int MODE, int VK, int QG>
__global__ __launch_bounds__(kAttnThreads, QG == 1 ? 3 : 2) void attn_long_kernel(AttnArgs g) {
  __shared__ float s_max[kAttnWaves][QG * kAttnQ];
  __shared__ float s_sum[kAttnWaves * QG * kAttnQ];
  __shared__ u32x4_t s_buf[kAttnWaves][512];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int bh, qt;
  if (g.xcd_heads) {
    const uint32_t x = blockIdx.x & 7u, slot = blockIdx.x >> 3;
    bh = (int)(x * g.xcd_heads + slot % g.xcd_heads);
    qt = g.qtiles - 1 - (int)(slot / g.xcd_heads);
  } else {
    bh = (int)(blockIdx.x / (uint32_t)g.qtiles);
    qt = g.qtiles - 1 - (int)(blockIdx.x % (uint32_t)g.qtiles);
  }
  const int S = g.s;
  const int q0 = qt * QG * kAttnQ;
  const int kblocks = (S + 31) >> 5;
  // group c (queries q0 + 32 c ..) has its diagonal in key block QG qt + c and
  // needs the key blocks before nkbc[c]; the last group needs the most
  int nkbc[QG];
#pragma unroll
  for (int c = 0; c < QG; ++c) nkbc[c] = g.causal ? min(kblocks, QG * qt + c + 1) : kblocks;
  const int nkb = nkbc[QG - 1];
  const int nlive = max(0, (nkb - wave + kAttnWaves - 1) / kAttnWaves);
  const int fr = lane & 31, fk = 8 * (lane >> 5), h = lane >> 5;
  const uint16_t* Q = g.q + (int64_t)bh * S * kAttnD;
  const uint16_t* K = g.k + (int64_t)bh * S * kAttnD;
  const uint16_t* Vt = g.vt + (int64_t)bh * kAttnD * g.ldv;
  u32x4_t* stage = s_buf[wave];
  const uint32_t koff = kblock_lane_offset(lane);
  uint32_t voff[4];
  vblock_lane_offsets(lane, g.ldv, voff);

  u32x4_t qf[QG][4];
#pragma unroll
  for (int c = 0; c < QG; ++c) {
    const uint16_t* qr = Q + (int64_t)min(q0 + 32 * c + fr, S - 1) * kAttnD + fk;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qf[c][ks] = ld16(qr + 16 * ks);
  }
  // K block kbg: gk is written to the staging slots and then refilled with the
  // block `next` (if any); the A operands are read back into ka
  u32x4_t gk[4], gv[4];
  auto stage_k = [&](int next, u32x4_t (&ka)[4]) {
    kblock_store(stage, lane, gk);
    if (next >= 0) kblock_load(K, 32 * next, S, lane, koff, gk);
    __builtin_amdgcn_wave_barrier();   // lanes read what other lanes wrote
    kblock_read(stage, fr, h, ka);
    __builtin_amdgcn_wave_barrier();   // before the slots are written again
  };
  // group c's block of S^T = K Q^T; with `masked`, keys past s and, on the
  // group's diagonal, keys above it are set to -inf
  auto scores = [&](const u32x4_t (&ka)[4], int c, int kbg, bool masked) {
    const f32x16_t zero = {};
    f32x16_t sacc = mma<DT>(ka[0], qf[c][0], zero);
#pragma unroll
    for (int ks = 1; ks < 4; ++ks)
      sacc = mma<DT>(ka[ks], qf[c][ks], sacc);
    const bool diag = g.causal && kbg == QG * qt + c;
    if (masked && (diag || (VK != kVtFull && 32 * kbg + 32 > S))) {
      const int query = q0 + 32 * c + fr;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * kbg + 8 * (r >> 2) + 4 * h + (r & 3);
        if (key >= S || (diag && key > query)) sacc[r] = -INFINITY;
      }
    }
    return sacc;
  };
  // A block is plain when every group needs it and none masks it: no key past
  // s, no group's diagonal. Its groups then run as one branch-free stretch, so
  // the scheduler can overlap one group's products with another's VALU work.
  auto plain_block = [&](int kbg) {
    return kbg < nkbc[0] && !(g.causal && kbg >= QG * qt) &&
           !(VK != kVtFull && 32 * kbg + 32 > S);
  };

  // pass 1: the row max
  if (nlive > 0) kblock_load(K, 32 * wave, S, lane, koff, gk);
  float m[QG];
#pragma unroll
  for (int c = 0; c < QG; ++c) m[c] = -INFINITY;
  for (int i = 0; i < nlive; ++i) {
    const int kbg = kAttnWaves * i + wave;
    u32x4_t ka[4];
    stage_k(i + 1 < nlive ? kbg + kAttnWaves : -1, ka);
    if (plain_block(kbg)) {
      f32x16_t sacc[QG];
#pragma unroll
      for (int c = 0; c < QG; ++c) sacc[c] = scores(ka, c, kbg, false);
#pragma unroll
      for (int c = 0; c < QG; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) m[c] = fmaxf(m[c], sacc[c][r]);
    } else {
#pragma unroll
      for (int c = 0; c < QG; ++c) {
        if (kbg < nkbc[c]) {
          const f32x16_t sacc = scores(ka, c, kbg, true);
#pragma unroll
          for (int r = 0; r < 16; ++r) m[c] = fmaxf(m[c], sacc[r]);
        }
      }
    }
  }
  if (nlive > 0) {
    kblock_load(K, 32 * wave, S, lane, koff, gk);
    vblock_load<VK>(Vt, g.ldv, 32 * wave, S, VK != kVtFull && 32 * wave + 32 > S, lane, voff, gv);
  }
#pragma unroll
  for (int c = 0; c < QG; ++c) {
    m[c] = fmaxf(m[c], xor32(m[c]));
    if (lane < 32) s_max[wave][32 * c + lane] = m[c];
  }
  __syncthreads();
  float c1[QG];
#pragma unroll
  for (int c = 0; c < QG; ++c) {
    const int j = 32 * c + fr;
    m[c] = fmaxf(fmaxf(s_max[0][j], s_max[1][j]), fmaxf(s_max[2][j], s_max[3][j]));
    c1[c] = (m[c] == -INFINITY) ? 0.0f
                                : __builtin_fmaf(-g.c0, m[c], MODE == EXACT ? 0.0f : kK127);
  }
  bool below = true;
#pragma unroll
  for (int c = 0; c < QG; ++c) below = below && row_c1_below(c1[c]);

  // pass 2: the scores again, their exponentials, the sums and O^T = V^T P
  float part[QG];
  f32x16_t oacc[QG][2];
#pragma unroll
  for (int c = 0; c < QG; ++c) {
    part[c] = 0.0f;
    oacc[c][0] = f32x16_t{};
    oacc[c][1] = f32x16_t{};
  }
  for (int i = 0; i < nlive; ++i) {
    const int kbg = kAttnWaves * i + wave;
    const int nb = kbg + kAttnWaves;
    u32x4_t ka[4];
    stage_k(i + 1 < nlive ? nb : -1, ka);
    uint32_t pk[QG][4][2];
    auto exps = [&](const f32x16_t& sacc, int c, auto below) {
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        float e[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          e[j] = qexp_row<MODE, decltype(below)::value>(sacc[4 * gi + j], g.c0, c1[c]);
          part[c] += e[j];
        }
        pk[c][gi][0] = pack16<DT>(e[0], e[1]);
        pk[c][gi][1] = pack16<DT>(e[2], e[3]);
      }
    };
#pragma unroll
    for (int c = 0; c < QG; ++c) {
      if (kbg < nkbc[c]) {
        const f32x16_t sacc = scores(ka, c, kbg, true);
        if (below)
          exps(sacc, c, std::true_type{});
        else
          exps(sacc, c, std::false_type{});
      }
    }
    vblock_store(stage, lane, gv);
    if (i + 1 < nlive)
      vblock_load<VK>(Vt, g.ldv, 32 * nb, S, VK != kVtFull && 32 * nb + 32 > S, lane, voff, gv);
    __builtin_amdgcn_wave_barrier();
    u32x4_t va[2][2];
    vblock_read(stage, fr, h, va);
    __builtin_amdgcn_wave_barrier();
    auto pv = [&](int c) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const auto s0 = __builtin_amdgcn_permlane32_swap(pk[c][2 * ks][0], pk[c][2 * ks + 1][0],
                                                         false, false);
        const auto s1 = __builtin_amdgcn_permlane32_swap(pk[c][2 * ks][1], pk[c][2 * ks + 1][1],
                                                         false, false);
        const u32x4_t bv = {s0[0], s1[0], s0[1], s1[1]};
#pragma unroll
        for (int db = 0; db < 2; ++db)
          oacc[c][db] = mma<DT>(va[ks][db], bv, oacc[c][db]);
      }
    };
#pragma unroll
    for (int c = 0; c < QG; ++c)
      if (kbg < nkbc[c]) pv(c);
  }

  attn_finish<DT, kAttnWaves, QG>(s_buf, s_sum, oacc, part, m, wave, lane, q0, S,
                                  g.o + (int64_t)bh * S * kAttnD);
}

// waves = 4, 8: the one-pass kernel with that many waves; 0: two passes with
// qg groups of 32 queries per workgroup
template <int DT, int MODE, int VK>
void launch_attn_vk(int waves, int qg, dim3 grid, hipStream_t s, const AttnArgs& g) {
  if (waves == 4)
    hipLaunchKernelGGL((attn_kernel<DT, MODE, VK, 4>), grid, dim3(64 * 4), 0, s, g);
  else if (waves == 8)
    hipLaunchKernelGGL((attn_kernel<DT, MODE, VK, 8>), grid, dim3(64 * 8), 0, s, g);
  else if (qg == 2)
    hipLaunchKernelGGL((attn_long_kernel<DT, MODE, VK, 2>), grid, dim3(kAttnThreads), 0, s, g);
  else
    hipLaunchKernelGGL((attn_long_kernel<DT, MODE, VK, 1>), grid, dim3(kAttnThreads), 0, s, g);
}

template <int DT, int MODE>
void launch_attn_mode(int vk, int waves, int qg, dim3 grid, hipStream_t s, const AttnArgs& g) {
  if (vk == kVtFull)
    launch_attn_vk<DT, MODE, kVtFull>(waves, qg, grid, s, g);
  else if (vk == kVtRagged)
    launch_attn_vk<DT, MODE, kVtRagged>(waves, qg, grid, s, g);
  else
    launch_attn_vk<DT, MODE, kVtScalar>(waves, qg, grid, s, g);
}

template <int DT>
void launch_attn(int mode, int vk, int waves, int qg, dim3 grid, hipStream_t s,
                 const AttnArgs& g) {
  switch (mode) {
    case QUAKE_EXACT: launch_attn_mode<DT, EXACT>(vk, waves, qg, grid, s, g); break;
    case QUAKE_1: launch_attn_mode<DT, Q1>(vk, waves, qg, grid, s, g); break;
    case QUAKE_2: launch_attn_mode<DT, Q2>(vk, waves, qg, grid, s, g); break;
    default: launch_attn_mode<DT, Q2M>(vk, waves, qg, grid, s, g); break;
  }
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_attention(const void* q, const void* k, const void* vt, void* o,
                                        int64_t heads, int64_t seq, int64_t dim, int64_t ldv,
                                        quake_dtype dtype, quake_mode mode, float t, int causal,
                                        void* stream) {
  if (dtype != QUAKE_BF16 && dtype != QUAKE_F16) return QUAKE_EDTYPE;
  if (!valid_mode(mode)) return QUAKE_EMODE;
  if (heads < 0 || seq < 0 || dim != kAttnD || seq > kAttnLongMaxS) return QUAKE_EINVAL;
  if (ldv < seq || ldv > INT32_MAX) return QUAKE_EINVAL;
  if (!std::isfinite(t) || !(t > 0.0f)) return QUAKE_EINVAL;
  const float c0 = softmax_c0(t, mode);
  if (!std::isfinite(c0) || c0 == 0.0f) return QUAKE_EINVAL;
  if (heads == 0 || seq == 0) return QUAKE_OK;
  if (q == nullptr || k == nullptr || vt == nullptr || o == nullptr) return QUAKE_EINVAL;
  if (!aligned16(q) || !aligned16(k) || ((uintptr_t)vt & 1u) != 0 || ((uintptr_t)o & 7u) != 0)
    return QUAKE_EINVAL;
  // one pass with 4 key blocks per wave (128 keys), else two passes
  const int waves = seq <= 512 ? 4 : seq <= kAttnMaxS ? 8 : 0;
  const int64_t tiles2 = (seq + 2 * kAttnQ - 1) / (2 * kAttnQ);   // per head, with two groups
  const int64_t min_tiles = causal ? kAttnLongQGMinTilesCausal : kAttnLongQGMinTiles;
  const int qg = (waves == 0 && heads >= (min_tiles + tiles2 - 1) / tiles2) ? 2 : 1;
  const int64_t tile = kAttnQ * qg;   // queries per workgroup
  const int64_t qtiles = (seq + tile - 1) / tile;
  if (heads > INT32_MAX / qtiles || heads * ldv * kAttnD > INT64_MAX / 4) return QUAKE_EINVAL;
  const AttnArgs g{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(vt), static_cast<uint16_t*>(o), (int32_t)seq,
                   (int32_t)ldv, (int32_t)qtiles, c0, (uint32_t)(causal != 0),
                   (uint32_t)(heads % 8 == 0 ? heads / 8 : 0)};
  const dim3 grid((uint32_t)(heads * qtiles));
  const hipStream_t s = static_cast<hipStream_t>(stream);
  // 16-byte rows, and byte offsets within a 64-row block of V^T that fit 32 bits
  const bool vec = aligned16(vt) && ldv % 8 == 0 && ldv <= (1 << 24);
  const int vk = !vec ? kVtScalar : (seq % 32 == 0 ? kVtFull : kVtRagged);
  if (dtype == QUAKE_BF16)
    launch_attn<BF16>(mode, vk, waves, qg, grid, s, g);
  else
    launch_attn<F16>(mode, vk, waves, qg, grid, s, g);
  return launch_status();
}
