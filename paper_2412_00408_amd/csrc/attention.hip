// attention.hip — quake_attention: O = softmax(t Q K^T) V per head (optionally
// causal), with the softmax of Algorithm 2 (arXiv:2412.00408, Sec. III-C) taken
// against each query's final row max. All scores of a query are in registers
// before any exponential is taken, so there is no online rescaling: QuAKE is
// not multiplicative (Q(a) Q(b) != Q(a + b)), and a flash-style running max
// would change the results Algorithm 2 defines.
//
// One workgroup = 32 queries of one head, four waves; wave w takes the 32-key
// blocks w, w + 4, w + 8, w + 12 (interleaved, so causal work stays balanced).
// The scores are computed transposed, S^T = K Q^T, on the matrix cores
// (v_mfma_f32_32x32x16_bf16; A = 32 keys x 16 dims straight from K's rows,
// B = the 32 queries' dims straight from Q's rows), so that lane l holds one
// query (l mod 32) and keys 8 g + 4 (l / 32) + i, g, i < 4, of each block:
//   * the row max and the row sum reduce the lane's own values, exchange once
//     with lane l xor 32 (v_permlane32_swap) and once across waves through LDS;
//   * the exponentials, rounded to bfloat16, become the B operand of the second
//     product O^T = V^T P after one v_permlane32_swap per dword pair (lane
//     l < 32 takes keys 4-7 from its partner and gives it keys 8-11), without a
//     trip through LDS. V is passed transposed ([head, dim, key]), so the A
//     operand (32 dims x 16 keys) is 16 contiguous bytes per lane.
// Causal key blocks above a query block's diagonal are neither loaded nor
// multiplied. The four partial O^T meet in LDS; wave w adds up, normalises by
// 1 / sum and stores one quarter of the 32 x 64 output tile as bfloat16.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "quake_device.hpp"
#include "quake_host.hpp"

namespace qk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kAttnD = 64;                     // head dimension
constexpr int kAttnMaxS = 512;                 // longest sequence: 16 key blocks
constexpr int kAttnQ = 32;                     // queries per workgroup
constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = 64 * kAttnWaves;
constexpr int kAttnBlk = kAttnMaxS / 32 / kAttnWaves;   // key blocks per wave

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* vt;
  uint16_t* o;
  int32_t s;         // sequence length, 1 .. 512
  int32_t ldv;       // row stride of V^T in elements, >= s
  int32_t qblocks;   // ceil(s / 32)
  float c0;          // Algorithm 2: 2^23 t / ln2 (EXACT: t / ln2)
  uint32_t causal;
};

__device__ __forceinline__ u32x4_t ld16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

// the value held by lane l xor 32
__device__ __forceinline__ float xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(as_u(v), as_u(v), false, false);
  return as_f((threadIdx.x & 32) ? r[0] : r[1]);
}

// 8 keys key0 .. key0 + 7 of one V^T row; keys at or past s read as zero (their
// probabilities are zero, and the padding of the row may hold anything).
// VEC: rows 16-byte aligned (ldv a multiple of 8), one 16-byte load; else eight
// 2-byte loads.
template <bool VEC>
__device__ __forceinline__ bf16x8_t load_v(const uint16_t* row, int key0, int s, bool tail) {
  if constexpr (VEC) {
    if (!tail) return __builtin_bit_cast(bf16x8_t, ld16(row + key0));
    u32x4_t v = {0u, 0u, 0u, 0u};
    const int nv = s - key0;
    if (nv > 0) {
      v = ld16(row + key0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (2 * i >= nv) v[i] = 0u;
        else if (2 * i + 1 >= nv) v[i] &= 0xFFFFu;
      }
    }
    return __builtin_bit_cast(bf16x8_t, v);
  } else {
    uint16_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = (!tail || key0 + i < s) ? row[key0 + i] : (uint16_t)0;
    u32x4_t v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (uint32_t)e[2 * i] | ((uint32_t)e[2 * i + 1] << 16);
    return __builtin_bit_cast(bf16x8_t, v);
  }
}

template <int MODE, bool VEC>
__global__ __launch_bounds__(kAttnThreads) void attn_kernel(AttnArgs g) {
  __shared__ float s_max[kAttnWaves][kAttnQ];
  __shared__ float s_sum[kAttnWaves][kAttnQ];
  __shared__ float s_o[kAttnWaves][32 * 64];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int bh = (int)(blockIdx.x / (uint32_t)g.qblocks);
  const int qb = (int)(blockIdx.x % (uint32_t)g.qblocks);
  const int S = g.s;
  const int q0 = qb * kAttnQ;
  const int kblocks = (S + 31) >> 5;
  const int nkb = g.causal ? min(kblocks, qb + 1) : kblocks;   // live key blocks of the tile
  const int fr = lane & 31, fk = 8 * (lane >> 5);
  const int query = q0 + fr;
  const uint16_t* Q = g.q + (int64_t)bh * S * kAttnD;
  const uint16_t* K = g.k + (int64_t)bh * S * kAttnD;
  const uint16_t* Vt = g.vt + (int64_t)bh * kAttnD * g.ldv;

  // S^T = K Q^T over the live key blocks of this wave
  bf16x8_t qf[4];
  {
    const uint16_t* qr = Q + (int64_t)min(query, S - 1) * kAttnD + fk;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qf[ks] = __builtin_bit_cast(bf16x8_t, ld16(qr + 16 * ks));
  }
  f32x16_t sacc[kAttnBlk];
#pragma unroll
  for (int i = 0; i < kAttnBlk; ++i) {
    const int kbg = kAttnWaves * i + wave;
#pragma unroll
    for (int r = 0; r < 16; ++r) sacc[i][r] = -INFINITY;
    if (kbg < nkb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[i][r] = 0.0f;
      const uint16_t* kr = K + (int64_t)min(32 * kbg + fr, S - 1) * kAttnD + fk;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        sacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, ld16(kr + 16 * ks)), qf[ks], sacc[i], 0, 0, 0);
      const bool diag = g.causal && kbg == qb;
      if (diag || 32 * kbg + 32 > S) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * kbg + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (key >= S || (diag && key > query)) sacc[i][r] = -INFINITY;
        }
      }
    }
  }

  // row (query) max: the lane's own values, lane l xor 32, the other waves
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < kAttnBlk; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) m = fmaxf(m, sacc[i][r]);
  m = fmaxf(m, xor32(m));
  if (lane < 32) s_max[wave][lane] = m;
  __syncthreads();
  m = fmaxf(fmaxf(s_max[0][fr], s_max[1][fr]), fmaxf(s_max[2][fr], s_max[3][fr]));

  // Algorithm 2: exponentials against the row max (c1 folds it in), their sum
  const float c1 = (m == -INFINITY) ? 0.0f : __builtin_fmaf(-g.c0, m, MODE == EXACT ? 0.0f : kK127);
  float part = 0.0f;
#pragma unroll
  for (int i = 0; i < kAttnBlk; ++i) {
    if (kAttnWaves * i + wave < nkb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sacc[i][r] = qexp<MODE>(sacc[i][r], g.c0, c1);
        part += sacc[i][r];
      }
    }
  }
  part += xor32(part);
  if (lane < 32) s_sum[wave][lane] = part;

  // O^T = V^T P over this wave's live keys
  f32x16_t oacc[2];
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;
#pragma unroll
  for (int i = 0; i < kAttnBlk; ++i) {
    const int kbg = kAttnWaves * i + wave;
    if (kbg < nkb) {
      const bool tail = 32 * kbg + 32 > S;
      uint32_t gp[4][2];   // keys 8 gi + 4 (lane / 32) + 0..3 as two bfloat16 pairs
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        gp[gi][0] = pack_bf16(sacc[i][4 * gi + 0], sacc[i][4 * gi + 1]);
        gp[gi][1] = pack_bf16(sacc[i][4 * gi + 2], sacc[i][4 * gi + 3]);
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        // lanes < 32 end with keys 16 ks + 0..7, lanes >= 32 with 16 ks + 8..15
        const auto s0 = __builtin_amdgcn_permlane32_swap(gp[2 * ks][0], gp[2 * ks + 1][0], false, false);
        const auto s1 = __builtin_amdgcn_permlane32_swap(gp[2 * ks][1], gp[2 * ks + 1][1], false, false);
        const u32x4_t bv = {s0[0], s1[0], s0[1], s1[1]};
        const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, bv);
        const int key0 = 32 * kbg + 16 * ks + fk;
#pragma unroll
        for (int db = 0; db < 2; ++db) {
          const bf16x8_t vf = load_v<VEC>(Vt + (int64_t)(32 * db + fr) * g.ldv, key0, S, tail);
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, oacc[db], 0, 0, 0);
        }
      }
    }
  }

  // the four partial O^T through LDS; wave w finishes dims 8 w + 4 (lane / 32)
  // + 0..3 of both 32-dim halves
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) s_o[wave][(db * 16 + r) * 64 + lane] = oacc[db][r];
  __syncthreads();
  if (query < S) {
    const float total = (s_sum[0][fr] + s_sum[1][fr]) + (s_sum[2][fr] + s_sum[3][fr]);
    const float inv = (m == -INFINITY || !(total > 0.0f)) ? 0.0f : 1.0f / total;
    uint16_t* orow = g.o + ((int64_t)bh * S + query) * kAttnD;
#pragma unroll
    for (int db = 0; db < 2; ++db) {
      float v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int idx = (db * 16 + 4 * wave + j) * 64 + lane;
        v[j] = ((s_o[0][idx] + s_o[1][idx]) + (s_o[2][idx] + s_o[3][idx])) * inv;
      }
      uint2 w;
      w.x = pack_bf16(v[0], v[1]);
      w.y = pack_bf16(v[2], v[3]);
      *reinterpret_cast<uint2*>(orow + 32 * db + 8 * wave + 4 * (lane >> 5)) = w;
    }
  }
}

template <int MODE>
void launch_attn(bool vec, dim3 grid, hipStream_t s, const AttnArgs& g) {
  if (vec)
    hipLaunchKernelGGL((attn_kernel<MODE, true>), grid, dim3(kAttnThreads), 0, s, g);
  else
    hipLaunchKernelGGL((attn_kernel<MODE, false>), grid, dim3(kAttnThreads), 0, s, g);
}

}  // namespace qk

using namespace qk;

extern "C" quake_status quake_attention(const void* q, const void* k, const void* vt, void* o,
                                        int64_t heads, int64_t seq, int64_t dim, int64_t ldv,
                                        quake_dtype dtype, quake_mode mode, float t, int causal,
                                        void* stream) {
  if (dtype != QUAKE_BF16) return QUAKE_EDTYPE;
  if (!valid_mode(mode)) return QUAKE_EMODE;
  if (heads < 0 || seq < 0 || dim != kAttnD || seq > kAttnMaxS) return QUAKE_EINVAL;
  if (ldv < seq || ldv > INT32_MAX) return QUAKE_EINVAL;
  if (!std::isfinite(t) || !(t > 0.0f)) return QUAKE_EINVAL;
  const float c0 = softmax_c0(t, mode);
  if (!std::isfinite(c0) || c0 == 0.0f) return QUAKE_EINVAL;
  if (heads == 0 || seq == 0) return QUAKE_OK;
  if (q == nullptr || k == nullptr || vt == nullptr || o == nullptr) return QUAKE_EINVAL;
  if (!aligned16(q) || !aligned16(k) || ((uintptr_t)vt & 1u) != 0 || ((uintptr_t)o & 7u) != 0)
    return QUAKE_EINVAL;
  const int64_t qblocks = (seq + kAttnQ - 1) / kAttnQ;
  if (heads > INT32_MAX / qblocks || heads * ldv * kAttnD > INT64_MAX / 4) return QUAKE_EINVAL;
  const AttnArgs g{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(vt), static_cast<uint16_t*>(o), (int32_t)seq,
                   (int32_t)ldv, (int32_t)qblocks, c0, (uint32_t)(causal != 0)};
  const dim3 grid((uint32_t)(heads * qblocks));
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const bool vec = aligned16(vt) && ldv % 8 == 0;
  switch (mode) {
    case QUAKE_EXACT: launch_attn<EXACT>(vec, grid, s, g); break;
    case QUAKE_1: launch_attn<Q1>(vec, grid, s, g); break;
    case QUAKE_2: launch_attn<Q2>(vec, grid, s, g); break;
    default: launch_attn<Q2M>(vec, grid, s, g); break;
  }
  return launch_status();
}
