// Attention-mass oracle scores on bf16 MFMA (Section 4.1 head-averaged mass;
// Section 4.2 block aggregation; Algorithm 1, head-averaged probabilities):
//
//   P_t(s)    = (1/Hq) sum_h exp(scale <q[t,h], k[s,g(h)]> - lse[t,h]),  s <= t
//   mass[r,s] = AGG_{t in block r, t >= s} P_t(s)
//
// The sum runs over every query head, so one workgroup owns all Hq heads of
// 16 queries at a time: wave w (of 8) holds the Q fragments of heads
// w, w+8, ... for those queries in registers. A tile of 32 keys of every KV
// head (contiguous in memory) is staged in LDS; each wave forms its heads'
// transposed scores S^T = K Q^T with MFMA, exponentiates against the
// normaliser and sums over its heads in registers. The eight per-wave partial
// sums are then added in LDS, masked causally and scaled by 1/Hq.
//
// b = 1: the workgroup covers 16 queries and one chunk of keys and stores
// P rows directly. b a multiple of 16: the workgroup covers one selection
// block (b/16 groups of 16 queries, in turn) and one chunk of keys, and keeps
// the block aggregate of the chunk in LDS until it is stored.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"

namespace sp {
namespace {

constexpr int kNW = 8;          // waves; wave w takes heads w, w+8, ...
constexpr int kTK = 32;         // keys per tile
constexpr int kKC = 512;        // keys per workgroup chunk
constexpr int kRedStride = 17;  // padded row of the cross-wave reduction buffer

template <int D>
struct MassLayout {
  static constexpr int KRB = D * 2 + 16;
  static constexpr int KS = D / 32;
};

template <int D, int HPW, int HKV>
__global__ __launch_bounds__(kNW * 64) void mass_kernel(
    int S, int Hq, int G, int b, int agg, float scale_log2, const uint16_t *__restrict__ q,
    const uint16_t *__restrict__ k, const float *__restrict__ lse, float *__restrict__ mass) {
  constexpr int NT = kNW * 64;
  constexpr int KRB = MassLayout<D>::KRB, KS = MassLayout<D>::KS;
  constexpr int TILE_BYTES = kTK * HKV * KRB;
  constexpr int PIECES = kTK * HKV * D / 8;
  constexpr int PER = (PIECES + NT - 1) / NT;
  __shared__ __align__(16) char ktile[TILE_BYTES];
  __shared__ float red[kNW][kTK][kRedStride];
  __shared__ float yagg[kKC];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  const int k_begin = blockIdx.y * kKC;
  // Query range of the workgroup: a selection block (b > 1) or 16 queries.
  const int bq = b > 1 ? b : 16;
  const int tq0 = blockIdx.x * bq;
  const int tq1 = min(tq0 + bq, S) - 1;
  if (k_begin > tq1) return;
  const int k_end = min(k_begin + kKC, tq1 + 1);
  const float neutral = agg == SP_AGG_MAX ? -INFINITY : 0.f;
  const float invH = 1.f / (float)Hq;
  if (b > 1)
    for (int i = tid; i < kKC; i += NT) yagg[i] = neutral;

  uint4 kreg[PER];
  auto load_tile = [&](int base) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < PIECES) {
        const int key = c / (HKV * D / 8), rem = c % (HKV * D / 8);
        const int s = min(base + key, S - 1);
        kreg[i] = ldg16(k + (size_t)s * HKV * D + rem * 8);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < PIECES) {
        const int key = c / (HKV * D / 8), rem = c % (HKV * D / 8);
        const int jj = rem / (D / 8), col = rem % (D / 8);
        sts16(ktile + (jj * kTK + key) * KRB + col * 16, kreg[i]);
      }
    }
  };

  for (int sq0 = tq0; sq0 <= tq1; sq0 += 16) {
    const int sq1 = min(sq0 + 16, S) - 1;   // this group's last query
    const int kend = min(k_end, sq1 + 1);
    if (k_begin >= kend) continue;            // uniform: no key of the chunk is causal here
    const int ntiles = (kend - k_begin + kTK - 1) / kTK;
    // Q fragments and normalisers of this wave's heads for query sq0 + c16.
    const int tq = min(sq0 + c16, S - 1);
    bf16x8 bqf[HPW][KS];
    float lse2[HPW];
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      const int h = wave + hh * kNW;
      const uint16_t *qp = q + ((size_t)tq * Hq + h) * D;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) bqf[hh][ks] = as_bf16x8(ldg16(qp + ks * 32 + g * 8));
      lse2[hh] = lse[(size_t)tq * Hq + h] * kLog2e;
    }
    load_tile(k_begin);
    for (int it = 0; it < ntiles; ++it) {
      const int base = k_begin + it * kTK;
      __syncthreads();                 // previous tile fully consumed
      store_tile();
      __syncthreads();
      if (it + 1 < ntiles) load_tile(base + kTK);
      // Partial mass of this wave's heads: lane = query c16, keys 16*ks2 + 4g + r.
      float part[2][4];
#pragma unroll
      for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
        for (int r = 0; r < 4; ++r) part[ks2][r] = 0.f;
#pragma unroll
      for (int hh = 0; hh < HPW; ++hh) {
        const int jj = (wave + hh * kNW) / G;
#pragma unroll
        for (int ks2 = 0; ks2 < 2; ++ks2) {
          f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 a =
                as_bf16x8(lds16(ktile + (jj * kTK + ks2 * 16 + c16) * KRB + ks * 64 + g * 16));
            acc = mfma16(a, bqf[hh][ks], acc);
          }
#pragma unroll
          for (int r = 0; r < 4; ++r)
            part[ks2][r] += __builtin_amdgcn_exp2f(fmaf(acc[r], scale_log2, -lse2[hh]));
        }
      }
#pragma unroll
      for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][ks2 * 16 + g * 4 + r][c16] = part[ks2][r];
      __syncthreads();
      // Sum over the waves: thread -> (query tq16 = tid / 32, key kk = tid % 32).
      const int kk = tid & 31, t16 = tid >> 5;
      const int s = base + kk, t = sq0 + t16;
      float p = 0.f;
#pragma unroll
      for (int w = 0; w < kNW; ++w) p += red[w][kk][t16];
      p *= invH;
      const bool ok = t <= sq1 && s <= t;
      if (b == 1) {
        if (ok) mass[(size_t)t * S + s] = p;
      } else {
        // reuse red[0] for the per-query values, then reduce over the 16 queries
        __syncthreads();
        red[0][kk][t16] = ok ? p : neutral;
        __syncthreads();
        if (tid < kTK) {
          float y = yagg[base - k_begin + tid];
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float x = red[0][tid][i];
            y = agg == SP_AGG_MAX ? fmaxf(y, x) : y + x;
          }
          yagg[base - k_begin + tid] = y;
        }
      }
    }
    __syncthreads();
  }
  if (b > 1) {
    __syncthreads();
    for (int i = tid; i < k_end - k_begin; i += NT)
      mass[(size_t)blockIdx.x * S + k_begin + i] = yagg[i];
  }
}

template <int D, int HPW, int HKV>
hipError_t launch_t(const Prob &p, const void *q, const void *k, const float *lse, float *mass,
                    hipStream_t st) {
  const int bq = p.b > 1 ? p.b : 16;
  dim3 grid((p.S + bq - 1) / bq, (p.S + kKC - 1) / kKC);
  hipLaunchKernelGGL((mass_kernel<D, HPW, HKV>), grid, dim3(kNW * 64), 0, st, p.S, p.Hq, p.G,
                     p.b, p.agg, p.scale * kLog2e, (const uint16_t *)q, (const uint16_t *)k, lse,
                     mass);
  return hipGetLastError();
}

template <int D, int HKV>
hipError_t launch_h(const Prob &p, const void *q, const void *k, const float *lse, float *mass,
                    hipStream_t st) {
  switch (p.Hq / kNW) {
    case 1: return launch_t<D, 1, HKV>(p, q, k, lse, mass, st);
    case 2: return launch_t<D, 2, HKV>(p, q, k, lse, mass, st);
    case 4: return launch_t<D, 4, HKV>(p, q, k, lse, mass, st);
    default: return launch_t<D, 8, HKV>(p, q, k, lse, mass, st);
  }
}

template <int D>
hipError_t launch_d(const Prob &p, const void *q, const void *k, const float *lse, float *mass,
                    hipStream_t st) {
  switch (p.Hkv) {
    case 1: return launch_h<D, 1>(p, q, k, lse, mass, st);
    case 2: return launch_h<D, 2>(p, q, k, lse, mass, st);
    case 4: return launch_h<D, 4>(p, q, k, lse, mass, st);
    default: return launch_h<D, 8>(p, q, k, lse, mass, st);
  }
}

}  // namespace

bool mass_mfma_supported(const Prob &p) {
  const int hpw = p.Hq / kNW;
  return p.dtype == SP_DTYPE_BF16 && (p.d == 64 || p.d == 128) && p.Hq % kNW == 0 &&
         (hpw == 1 || hpw == 2 || hpw == 4 || hpw == 8) &&
         (p.Hkv == 1 || p.Hkv == 2 || p.Hkv == 4 || p.Hkv == 8) &&
         (p.b == 1 || (p.b % 16 == 0 && p.b <= 1024));
}

hipError_t launch_mass_mfma(const Prob &p, const void *q, const void *k, const float *lse,
                            float *mass, hipStream_t st) {
  if (p.d == 64) return launch_d<64>(p, q, k, lse, mass, st);
  return launch_d<128>(p, q, k, lse, mass, st);
}

}  // namespace sp
