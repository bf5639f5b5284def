// Head-collapsed indexer scores on bf16 MFMA (Section 6.3; Algorithm 2 step 4).
//
//   z[t,s] = ReLU(iscale * <q_idx[t], k_idx[s]>),  s <= t
//
// Two kernels share one structure: a workgroup owns a range of queries
// (64 per wave, resident in registers as MFMA operands) and a chunk of up to
// 1024 keys, which it streams through double-buffered LDS tiles. Each key
// tile is read from L2 once per workgroup and reused by every wave. Only key
// tiles at or below a wave's last query are multiplied (causal skipping).
//
// * indexer_block_kernel (b in {16, 32, 64, 128}): the epilogue scales,
//   applies the ReLU and the per-pair causal mask (t >= s, Section 4.2) and
//   reduces over the b queries of each selection block (max or sum) before
//   anything leaves the chip; one float per (block, key) is stored.
// * indexer_rows_kernel (b = 1): every causal score is stored. The MFMA is
//   issued with keys as rows (scores transposed) so that each lane holds
//   four consecutive keys of one query and writes them as one 16-byte store.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"

namespace sp {
namespace {

constexpr int kQW = 64;     // queries per wave
constexpr int kKC = 1024;   // keys per workgroup chunk

template <int DI>
struct Tile {
  static constexpr int KT = DI <= 128 ? 64 : 32;   // keys per LDS tile
  static constexpr int RB = DI * 2 + 16;           // padded row bytes (bank spread)
  static constexpr int BYTES = KT * RB;
  static constexpr int CHUNKS = KT * DI / 8;       // 16-byte pieces per tile
  static constexpr int KS = DI / 32;               // MFMA k-steps
};

// Global -> registers -> LDS staging of one key tile, rows clamped to S-1.
template <int DI, int NT>
struct KeyStage {
  static constexpr int PER = (Tile<DI>::CHUNKS + NT - 1) / NT;
  uint4 reg[PER];
  __device__ __forceinline__ void load(const uint16_t *__restrict__ ki, int S, int k0, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < Tile<DI>::CHUNKS) {
        const int row = c / (DI / 8), col = c % (DI / 8);
        const int s = min(k0 + row, S - 1);
        reg[i] = ldg16(ki + (size_t)s * DI + col * 8);
      }
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < Tile<DI>::CHUNKS) {
        const int row = c / (DI / 8), col = c % (DI / 8);
        sts16(lds + row * Tile<DI>::RB + col * 16, reg[i]);
      }
    }
  }
};

__device__ __forceinline__ float agg2(int agg, float a, float b) {
  return agg == SP_AGG_MAX ? fmaxf(a, b) : a + b;
}

__device__ __forceinline__ float as_f(uint32_t x) { return __uint_as_float(x); }
__device__ __forceinline__ uint32_t as_u(float x) { return __float_as_uint(x); }

// Reduce-scatter across the four 16-lane groups of a wave. Every lane holds
// one partial per column tile; afterwards lane (g, c) holds the reduction over
// the four groups of column tile owned_ct(g) at column c. Two half-wave swaps
// and one row swap (gfx950 v_permlane32_swap / v_permlane16_swap) replace the
// eight cross-lane shuffles a per-tile butterfly would take.
template <int NCT>
__device__ __forceinline__ int owned_ct(int g) {
  return NCT == 4 ? ((g & 1) << 1) | (g >> 1) : g >> 1;
}

template <class Op>
__device__ __forceinline__ float reduce_scatter(const float (&v)[4], Op op) {
  const auto a = __builtin_amdgcn_permlane32_swap(as_u(v[0]), as_u(v[1]), false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(as_u(v[2]), as_u(v[3]), false, false);
  const float m01 = op(as_f(a[0]), as_f(a[1]));   // rows 0,1: tile 0; rows 2,3: tile 1
  const float m23 = op(as_f(b[0]), as_f(b[1]));   // rows 0,1: tile 2; rows 2,3: tile 3
  const auto c = __builtin_amdgcn_permlane16_swap(as_u(m01), as_u(m23), false, false);
  return op(as_f(c[0]), as_f(c[1]));
}

template <class Op>
__device__ __forceinline__ float reduce_scatter(const float (&v)[2], Op op) {
  const auto a = __builtin_amdgcn_permlane32_swap(as_u(v[0]), as_u(v[1]), false, false);
  const float m = op(as_f(a[0]), as_f(a[1]));     // rows 0,1: tile 0; rows 2,3: tile 1
  const auto c = __builtin_amdgcn_permlane16_swap(as_u(m), as_u(m), false, false);
  return op(as_f(c[0]), as_f(c[1]));
}

// MAXPOS: aggregation is max and the scale is non-negative, so scale and
// ReLU commute with the max: rows are reduced on raw MFMA outputs and only
// the reduced value is scaled; tiles entirely below a wave's first query
// skip the causal test.
template <int DI, int BQ, bool MAXPOS>
__global__ __launch_bounds__(512) void indexer_block_kernel(int S, int agg, int relu,
                                                            float scale,
                                                            const uint16_t *__restrict__ qi,
                                                            const uint16_t *__restrict__ ki,
                                                            float *__restrict__ Y) {
  constexpr int NT = 512, NW = 8;
  constexpr int KT = Tile<DI>::KT, RB = Tile<DI>::RB, KS = Tile<DI>::KS;
  constexpr int NCT = KT / 16;
  constexpr int QG = NW * kQW;
  __shared__ __align__(16) char lds[2][Tile<DI>::BYTES];
  __shared__ float red[NW / 2][KT];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  const int q0 = blockIdx.x * QG;
  const int k_begin = blockIdx.y * kKC;
  const int q_last = min(q0 + QG, S) - 1;
  if (k_begin > q_last) return;
  const int k_end = min(k_begin + kKC, q_last + 1);
  const int ntiles = (k_end - k_begin + KT - 1) / KT;
  const int qw0 = q0 + wave * kQW;
  const int qw_last = min(qw0 + kQW, S) - 1;  // < qw0 when the wave is past the end
  // key column this lane holds after the reduce-scatter (relative to the tile)
  const int my_col = owned_ct<NCT>(g) * 16 + c16;
  const bool col_writer = NCT == 4 || (g & 1) == 0;

  bf16x8 a[4][KS];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    const int row = min(qw0 + rt * 16 + c16, S - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      a[rt][ks] = as_bf16x8(ldg16(qi + (size_t)row * DI + ks * 32 + g * 8));
  }

  KeyStage<DI, NT> stage;
  stage.load(ki, S, k_begin, tid);
  stage.store(lds[0], tid);
  __syncthreads();

  const float neutral = agg == SP_AGG_MAX ? -INFINITY : 0.f;
  auto op = [agg](float x, float y) { return MAXPOS ? fmaxf(x, y) : agg2(agg, x, y); };
  constexpr int BPW = BQ >= kQW ? 1 : kQW / BQ;   // blocks per wave
  constexpr int RPB = BQ >= kQW ? 4 : BQ / 16;    // row tiles per block
  for (int it = 0; it < ntiles; ++it) {
    const int kt0 = k_begin + it * KT;
    const bool more = it + 1 < ntiles;
    if (more) stage.load(ki, S, kt0 + KT, tid);
    const char *cur = lds[it & 1];
    const bool active = kt0 <= qw_last;
    // full: every (query, key) pair of the wave and tile is causal and valid
    const bool full = kt0 + KT - 1 <= qw0 && qw0 + kQW - 1 <= qw_last;
    // out[bb]: aggregate over the queries of block bb, for key column my_col
    float out[BPW];
#pragma unroll
    for (int bb = 0; bb < BPW; ++bb) out[bb] = neutral;
    if (active) {
      float part[BPW][NCT];
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
        const int s = kt0 + ct * 16 + c16;
        f32x4 acc[4];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 b = as_bf16x8(lds16(cur + (ct * 16 + c16) * RB + ks * 64 + g * 16));
#pragma unroll
          for (int rt = 0; rt < 4; ++rt) acc[rt] = mfma16(a[rt][ks], b, acc[rt]);
        }
#pragma unroll
        for (int bb = 0; bb < BPW; ++bb) part[bb][ct] = neutral;
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
          float x[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            x[r] = acc[rt][r];
            if constexpr (!MAXPOS) {
              x[r] *= scale;
              if (relu) x[r] = fmaxf(x[r], 0.f);
            }
          }
          if (!full) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int t = qw0 + rt * 16 + g * 4 + r;
              if (!(t <= qw_last && s <= t)) x[r] = neutral;
            }
          }
          const float m = op(op(x[0], x[1]), op(x[2], x[3]));
          part[rt / RPB][ct] = op(part[rt / RPB][ct], m);
        }
      }
#pragma unroll
      for (int bb = 0; bb < BPW; ++bb) {
        float m = reduce_scatter(part[bb], op);
        if constexpr (MAXPOS) {
          m *= scale;
          if (relu) m = fmaxf(m, 0.f);   // -inf (no causal row) becomes 0; never stored
        }
        out[bb] = m;
      }
    }
    const int s = kt0 + my_col;
    if constexpr (BQ <= kQW) {
#pragma unroll
      for (int bb = 0; bb < BPW; ++bb) {
        const int tb0 = qw0 + bb * BQ;                  // first query of the block
        const int tb1 = min(tb0 + BQ, S) - 1;
        if (col_writer && tb0 < S && s <= tb1) Y[(size_t)(tb0 / BQ) * S + s] = out[bb];
      }
    } else {
      // BQ = 128: waves 2i and 2i+1 hold the two halves of one block.
      if (wave & 1) red[wave >> 1][my_col] = out[0];
      __syncthreads();
      if (!(wave & 1)) {
        const int tb0 = qw0;
        const int tb1 = min(tb0 + BQ, S) - 1;
        const float m = op(out[0], red[wave >> 1][my_col]);
        if (col_writer && tb0 < S && s <= tb1) Y[(size_t)(tb0 / BQ) * S + s] = m;
      }
    }
    if (more) stage.store(lds[(it + 1) & 1], tid);
    __syncthreads();
  }
}

template <int DI, bool VEC>
__global__ __launch_bounds__(256) void indexer_rows_kernel(int S, int relu, float scale,
                                                           const uint16_t *__restrict__ qi,
                                                           const uint16_t *__restrict__ ki,
                                                           float *__restrict__ Z) {
  constexpr int NT = 256, NW = 4;
  constexpr int KT = Tile<DI>::KT, RB = Tile<DI>::RB, KS = Tile<DI>::KS;
  constexpr int QG = NW * kQW;
  __shared__ __align__(16) char lds[2][Tile<DI>::BYTES];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  const int q0 = blockIdx.x * QG;
  const int k_begin = blockIdx.y * kKC;
  const int q_last = min(q0 + QG, S) - 1;
  if (k_begin > q_last) return;
  const int k_end = min(k_begin + kKC, q_last + 1);
  const int ntiles = (k_end - k_begin + KT - 1) / KT;
  const int qw0 = q0 + wave * kQW;
  const int qw_last = min(qw0 + kQW, S) - 1;

  // Queries are the B operand: lane holds query column c16 of tile qc.
  bf16x8 bq[4][KS];
#pragma unroll
  for (int qc = 0; qc < 4; ++qc) {
    const int row = min(qw0 + qc * 16 + c16, S - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      bq[qc][ks] = as_bf16x8(ldg16(qi + (size_t)row * DI + ks * 32 + g * 8));
  }

  KeyStage<DI, NT> stage;
  stage.load(ki, S, k_begin, tid);
  stage.store(lds[0], tid);
  __syncthreads();

  for (int it = 0; it < ntiles; ++it) {
    const int kt0 = k_begin + it * KT;
    const bool more = it + 1 < ntiles;
    if (more) stage.load(ki, S, kt0 + KT, tid);
    const char *cur = lds[it & 1];
    if (kt0 <= qw_last) {
#pragma unroll
      for (int kr = 0; kr < KT / 16; ++kr) {
        f32x4 acc[4];
#pragma unroll
        for (int qc = 0; qc < 4; ++qc) acc[qc] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 a = as_bf16x8(lds16(cur + (kr * 16 + c16) * RB + ks * 64 + g * 16));
#pragma unroll
          for (int qc = 0; qc < 4; ++qc) acc[qc] = mfma16(a, bq[qc][ks], acc[qc]);
        }
        const int s0 = kt0 + kr * 16 + g * 4;  // this lane's four consecutive keys
#pragma unroll
        for (int qc = 0; qc < 4; ++qc) {
          const int t = qw0 + qc * 16 + c16;
          if (t > qw_last || s0 > t) continue;
          float x[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            x[r] = acc[qc][r] * scale;
            if (relu) x[r] = x[r] > 0.f ? x[r] : 0.f;
          }
          float *dst = Z + (size_t)t * S + s0;
          if (s0 + 3 <= t) {
            if constexpr (VEC) {
              *reinterpret_cast<float4 *>(dst) = make_float4(x[0], x[1], x[2], x[3]);
            } else {
#pragma unroll
              for (int r = 0; r < 4; ++r) dst[r] = x[r];
            }
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (s0 + r <= t) dst[r] = x[r];
          }
        }
      }
    }
    if (more) stage.store(lds[(it + 1) & 1], tid);
    __syncthreads();
  }
}

template <int DI>
hipError_t launch_di(const Prob &p, const void *qi, const void *ki, float *scores,
                     hipStream_t st) {
  const uint16_t *q = (const uint16_t *)qi, *k = (const uint16_t *)ki;
  if (p.b == 1) {
    dim3 grid((p.S + 255) / 256, (p.S + kKC - 1) / kKC);
    if (p.S % 4 == 0)
      hipLaunchKernelGGL((indexer_rows_kernel<DI, true>), grid, dim3(256), 0, st, p.S, p.relu,
                         p.iscale, q, k, scores);
    else
      hipLaunchKernelGGL((indexer_rows_kernel<DI, false>), grid, dim3(256), 0, st, p.S, p.relu,
                         p.iscale, q, k, scores);
    return hipGetLastError();
  }
  dim3 grid((p.S + 511) / 512, (p.S + kKC - 1) / kKC);
  const bool maxpos = p.agg == SP_AGG_MAX && p.iscale >= 0.f;
#define SP_BLK(BQ)                                                                           \
  if (maxpos)                                                                                \
    hipLaunchKernelGGL((indexer_block_kernel<DI, BQ, true>), grid, dim3(512), 0, st, p.S,    \
                       p.agg, p.relu, p.iscale, q, k, scores);                               \
  else                                                                                       \
    hipLaunchKernelGGL((indexer_block_kernel<DI, BQ, false>), grid, dim3(512), 0, st, p.S,   \
                       p.agg, p.relu, p.iscale, q, k, scores)
  switch (p.b) {
    case 16: SP_BLK(16); break;
    case 32: SP_BLK(32); break;
    case 64: SP_BLK(64); break;
    default: SP_BLK(128); break;
  }
#undef SP_BLK
  return hipGetLastError();
}

}  // namespace

bool indexer_mfma_supported(const Prob &p) {
  return p.dtype == SP_DTYPE_BF16 && (p.di == 64 || p.di == 128 || p.di == 256) &&
         (p.b == 1 || p.b == 16 || p.b == 32 || p.b == 64 || p.b == 128);
}

hipError_t launch_indexer_mfma(const Prob &p, const void *qi, const void *ki, float *scores,
                               hipStream_t st) {
  if (p.di == 64) return launch_di<64>(p, qi, ki, scores, st);
  if (p.di == 128) return launch_di<128>(p, qi, ki, scores, st);
  return launch_di<256>(p, qi, ki, scores, st);
}

}  // namespace sp
