// Column-parallel support scores with selection-block aggregation, for any
// shape and dtype (the MFMA kernels cover the large bf16 shapes).
//
// Oracle mass (Section 4.1, 4.2; Algorithm 1, head-averaged probabilities):
//   P_t(s) = (1/Hq) sum_h exp(scale <q[t,h],k[s,g(h)]> - lse[t,h]),  s <= t
// or, for the per-KV-group support of the head axis (Section 3), the same
// average over the G heads of one KV group, one table per group.
// Indexer score (Section 6.3; Algorithm 2, candidate scoring):
//   z[t,s] = ReLU(iscale <q_idx[t], k_idx[s]>),  s <= t
// Block aggregate (Section 4.2): Y[r,s] = AGG_{t in block r, t >= s} X[t,s].
//
// One workgroup of 256 threads per (block r, 256 consecutive columns s).
// The queries of the block are visited in order; the current query's
// vectors are staged in LDS and broadcast to every thread, and each thread
// owns one column s and accumulates its aggregate in a register.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

constexpr int kCols = 256;

template <typename T, int D>
__global__ __launch_bounds__(kCols) void mass_rowwise_kernel(
    int S, int Hq, int Hkv, int G, int b, int agg, int per_group, float scale_log2,
    const T *__restrict__ q, const T *__restrict__ k, const float *__restrict__ lse,
    float *__restrict__ mass) {
  extern __shared__ float smem[];
  float *qs = smem;            // [Hq, D], pre-scaled by scale*log2(e)
  float *ls = smem + Hq * D;   // [Hq], lse*log2(e)
  const int r = blockIdx.x;
  const int t0 = r * b;
  const int t1 = min(t0 + b, S) - 1;
  const int c0 = blockIdx.y * kCols;
  if (c0 > t1) return;  // uniform over the workgroup
  const int s = c0 + threadIdx.x;
  // KV groups averaged: all of them, or group blockIdx.z (per-group support)
  const int j0 = per_group ? (int)blockIdx.z : 0, nj = per_group ? 1 : Hkv;
  mass += (size_t)blockIdx.z * gridDim.x * S;
  const float invH = 1.f / (float)(nj * G);
  float y = 0.f;
  bool have = false;
  for (int t = t0; t <= t1; ++t) {
    __syncthreads();
    for (int i = threadIdx.x; i < Hq * D; i += kCols)
      qs[i] = to_float(q[(size_t)t * Hq * D + i]) * scale_log2;
    for (int i = threadIdx.x; i < Hq; i += kCols) ls[i] = lse[(size_t)t * Hq + i] * kLog2e;
    __syncthreads();
    if (s <= t) {
      float pt = 0.f;
      for (int j = j0; j < j0 + nj; ++j) {
        // the key row in chunks of at most 128 (bounded registers at d = 256)
        constexpr int CH = D < 128 ? D : 128;
        for (int hh = 0; hh < G; ++hh) {
          const int h = j * G + hh;
          float dot = 0.f;
          for (int c = 0; c < D; c += CH) {
            float kr[CH];
            load_row<CH>(k + ((size_t)s * Hkv + j) * D + c, kr);
#pragma unroll
            for (int e = 0; e < CH; ++e) dot = fmaf(qs[h * D + c + e], kr[e], dot);
          }
          pt += exp2f(dot - ls[h]);
        }
      }
      pt *= invH;
      if (!have) {
        y = pt;
        have = true;
      } else {
        y = (agg == SP_AGG_MAX) ? fmaxf(y, pt) : y + pt;
      }
    }
  }
  if (s <= t1) mass[(size_t)r * S + s] = y;
}

template <typename T, int DI>
__global__ __launch_bounds__(kCols) void indexer_rowwise_kernel(
    int S, int qo, int b, int agg, int relu, float iscale, const T *__restrict__ qi,
    const T *__restrict__ ki, float *__restrict__ scores) {
  // qi is addressed by position (shifted back by qo rows by the host); rows of
  // scores count blocks from the chunk start qo
  __shared__ float qs[DI];
  const int r = blockIdx.x;
  const int t0 = qo + r * b;
  const int t1 = min(t0 + b, S) - 1;
  const int c0 = blockIdx.y * kCols;
  if (c0 > t1) return;
  const int s = c0 + threadIdx.x;
  const int sl = s <= t1 ? s : t1;  // clamp so every load stays in bounds
  constexpr int CH = DI < 128 ? DI : 128;
  float y = 0.f;
  bool have = false;
  for (int t = t0; t <= t1; ++t) {
    __syncthreads();
    for (int i = threadIdx.x; i < DI; i += kCols) qs[i] = to_float(qi[(size_t)t * DI + i]);
    __syncthreads();
    if (s <= t) {
      float dot = 0.f;
#pragma unroll
      for (int c = 0; c < DI; c += CH) {
        float kr[CH];
        load_row<CH>(ki + (size_t)sl * DI + c, kr);
#pragma unroll
        for (int e = 0; e < CH; ++e) dot = fmaf(qs[c + e], kr[e], dot);
      }
      float z = dot * iscale;
      if (relu) z = z > 0.f ? z : 0.f;
      if (!have) {
        y = z;
        have = true;
      } else {
        y = (agg == SP_AGG_MAX) ? fmaxf(y, z) : y + z;
      }
    }
  }
  if (s <= t1) scores[(size_t)r * S + s] = y;
}

// Blocks r x column tiles; tiles past a block's last query exit at once.
dim3 grid_for(const Prob &p) { return dim3(p.R, (p.S + kCols - 1) / kCols); }

}  // namespace

hipError_t launch_mass_rowwise(const Prob &p, const void *q, const void *k, const float *lse,
                               float *mass, hipStream_t st) {
  const size_t lds = sizeof(float) * (size_t)p.Hq * (p.d + 1);
  const float sl2 = p.scale * kLog2e;
  dim3 grid = grid_for(p);
  grid.z = p.ha ? p.Hkv : 1;   // per-group support: one mass table per KV group
#define SP_MASS(T, D)                                                                        \
  hipLaunchKernelGGL((mass_rowwise_kernel<T, D>), grid, dim3(kCols), lds, st, p.S, p.Hq,    \
                     p.Hkv, p.G, p.b, p.agg, p.ha, sl2, (const T *)q, (const T *)k, lse, mass)
  if (p.dtype == SP_DTYPE_BF16) {
    if (p.d == 64) SP_MASS(bf16, 64);
    else if (p.d == 128) SP_MASS(bf16, 128);
    else SP_MASS(bf16, 256);
  } else {
    if (p.d == 64) SP_MASS(float, 64);
    else if (p.d == 128) SP_MASS(float, 128);
    else SP_MASS(float, 256);
  }
#undef SP_MASS
  return hipGetLastError();
}

hipError_t launch_indexer_rowwise(const Prob &p, const void *qi, const void *ki, float *scores,
                                  hipStream_t st) {
  const dim3 grid = grid_for(p);
#define SP_IDX(T, DI)                                                                        \
  hipLaunchKernelGGL((indexer_rowwise_kernel<T, DI>), grid, dim3(kCols), 0, st, p.S, p.qo,   \
                     p.b, p.agg, p.relu, p.iscale, (const T *)qi - (size_t)p.qo * DI,        \
                     (const T *)ki, scores)
  if (p.dtype == SP_DTYPE_BF16) {
    if (p.di == 64) SP_IDX(bf16, 64);
    else if (p.di == 128) SP_IDX(bf16, 128);
    else SP_IDX(bf16, 256);
  } else {
    if (p.di == 64) SP_IDX(float, 64);
    else if (p.di == 128) SP_IDX(float, 128);
    else SP_IDX(float, 256);
  }
#undef SP_IDX
  return hipGetLastError();
}

}  // namespace sp
