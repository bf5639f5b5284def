// Attention-mass oracle scores on bf16 MFMA (Section 4.1 head-averaged mass;
// Section 4.2 block aggregation; Algorithm 1, head-averaged probabilities):
//
//   P_t(s)    = (1/Hq) sum_h exp(scale <q[t,h], k[s,g(h)]> - lse[t,h]),  s <= t
//   mass[r,s] = AGG_{t in block r, t >= s} P_t(s)
//
// The sum runs over every query head, so a workgroup owns all Hq heads of its
// queries; each wave holds the query operands of Hq/8 heads in registers and
// sums its heads in registers, and the eight per-wave partial sums are added
// in LDS.
//
// mass32_kernel (b = 1, or b a multiple of 32; the heads of a wave share one
// KV head): a workgroup covers 32 queries (or the b queries of one block, 32
// at a time) and a chunk of 1024 keys. Scores are formed transposed on
// v_mfma_f32_32x32x16_bf16, S^T = K Q^T with keys as rows: a lane then holds
// one query and 16 keys of a 32-key tile, so its normaliser is one register
// per head and the head sum is lane-local. The 32-key tile of every KV head
// is loaded straight into LDS (padded rows); the next tile's loads are issued
// as soon as the current one is in registers and run under the exponentials.
//
// mass_kernel (the other shapes, and every shape at head_dim 256, whose
// 32-key tiles of eight KV heads would not fit LDS twice): 16 queries per
// workgroup on v_mfma_f32_16x16x32_bf16, K staged through registers.
//
// b = 1 stores P rows directly. b > 1 keeps the block aggregate of the key
// chunk in LDS until it is stored.
#include <math.h>

#include "attn_tile.hpp"
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
    default:
      if constexpr (D == 256)
        return hipErrorInvalidValue;   // not dispatched here
      else
        return launch_t<D, 8, HKV>(p, q, k, lse, mass, st);
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


// ---------------------------------------------------------------- mass32_kernel
constexpr int kMT = 32;       // keys per tile; queries per query tile
// keys per workgroup chunk (block rows keep the chunk's aggregate in LDS):
// a query tile is re-read once per chunk, and chunks of 2048 measured a few
// percent faster than 1024, 4096 or 8192
template <bool ROWS>
constexpr int mass_chunk() { return 2048; }
constexpr int kRS = 36;       // row stride (floats) of the partial-sum buffer (bank spread)
constexpr int kMaxHkv = 8;

template <int D>
struct Mass32 {
  static constexpr int KRB = D * 2 + 16;     // padded LDS row of one key of one KV head
  static constexpr int SLOTS = D / 8 + 1;    // 16-byte slots per row (the last is padding)
  static constexpr int KS = D / 16;          // k-steps of the 32x32x16 product
  static constexpr int KBYTES = kMaxHkv * kMT * KRB;
};

constexpr int kPartBytes = kMT * kRS * 4;
// Sums over the eight partials at LDS byte addresses a0, a0 + kPartBytes, ...
// and a1, a1 + kPartBytes, ..., each in that order, with one wait. Inline
// reads: the compiler would otherwise wait for every direct-to-LDS tile load
// in flight before an LDS read. The outputs are early-clobber: a read's data
// may land while later reads of the block still need the address registers.
__device__ __forceinline__ void sum_partials2(uint32_t a0, uint32_t a1, float &v0, float &v1) {
  float x[kNW], y[kNW];
  asm volatile(
      "ds_read_b32 %0, %16\n\tds_read_b32 %1, %16 offset:%18\n\t"
      "ds_read_b32 %2, %16 offset:%19\n\tds_read_b32 %3, %16 offset:%20\n\t"
      "ds_read_b32 %4, %16 offset:%21\n\tds_read_b32 %5, %16 offset:%22\n\t"
      "ds_read_b32 %6, %16 offset:%23\n\tds_read_b32 %7, %16 offset:%24\n\t"
      "ds_read_b32 %8, %17\n\tds_read_b32 %9, %17 offset:%18\n\t"
      "ds_read_b32 %10, %17 offset:%19\n\tds_read_b32 %11, %17 offset:%20\n\t"
      "ds_read_b32 %12, %17 offset:%21\n\tds_read_b32 %13, %17 offset:%22\n\t"
      "ds_read_b32 %14, %17 offset:%23\n\tds_read_b32 %15, %17 offset:%24\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3]), "=&v"(x[4]), "=&v"(x[5]),
        "=&v"(x[6]), "=&v"(x[7]), "=&v"(y[0]), "=&v"(y[1]), "=&v"(y[2]), "=&v"(y[3]),
        "=&v"(y[4]), "=&v"(y[5]), "=&v"(y[6]), "=&v"(y[7])
      : "v"(a0), "v"(a1), "i"(kPartBytes), "i"(2 * kPartBytes), "i"(3 * kPartBytes),
        "i"(4 * kPartBytes), "i"(5 * kPartBytes), "i"(6 * kPartBytes), "i"(7 * kPartBytes)
      : "memory");
  v0 = 0.f;
  v1 = 0.f;
#pragma unroll
  for (int p = 0; p < kNW; ++p) {
    v0 += x[p];
    v1 += y[p];
  }
}
__device__ __forceinline__ float lds_read_f32(uint32_t a) {
  float x;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(x) : "v"(a) : "memory");
  return x;
}
__device__ __forceinline__ void lds_write_f32(uint32_t a, float x) {
  asm volatile("ds_write_b32 %0, %1" : : "v"(a), "v"(x) : "memory");
}

template <int D, int HPW, bool ROWS>
__global__ __launch_bounds__(kNW * 64) void mass32_kernel(
    int S, int Hq, int Hkv, int G, int b, int agg, float scale_log2,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const float *__restrict__ lse, float *__restrict__ mass) {
  using T = Mass32<D>;
  constexpr int KRB = T::KRB, SLOTS = T::SLOTS, KS = T::KS;
  __shared__ __align__(16) char ktile[T::KBYTES];
  __shared__ __align__(16) float red[2][kNW][kMT][kRS];
  constexpr int kMKC = mass_chunk<ROWS>();
  __shared__ float yagg[ROWS ? 1 : kMKC];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, half = lane >> 5;
  const int span = ROWS ? kMT : b;
  const int tq0 = blockIdx.x * span;
  const int tq_last = min(tq0 + span, S) - 1;
  const int k_begin = blockIdx.y * kMKC;
  if (k_begin > tq_last) return;   // the whole workgroup
  const int k_end = min(k_begin + kMKC, tq_last + 1);
  const int h0 = wave * HPW;       // the wave's heads h0 .. h0 + HPW - 1
  const int jj = h0 / G;           // their KV head
  const float neutral = agg == SP_AGG_MAX ? -INFINITY : 0.f;
  const float invH = 1.f / (float)Hq;
  auto op = [agg](float x, float y) { return agg == SP_AGG_MAX ? fmaxf(x, y) : x + y; };
  if constexpr (!ROWS)
    for (int i = tid; i < kMKC; i += kNW * 64) yagg[i] = neutral;

  // K tile: row jj * 32 + key, slot c of a row at byte (row * SLOTS + c) * 16,
  // so chunk c of 64 slots is 1 KiB at c * 1024. A lane's byte offset within
  // a tile of keys k0 .. is fixed (kept in registers, ~0 for lanes on padding
  // slots or past the last row, which load nothing). Keys past S - 1 fall
  // outside the buffer and load zeros (they are masked).
  constexpr int kMaxChunks = (kMaxHkv * kMT * SLOTS + 63) / 64;
  constexpr int kCPW = (kMaxChunks + kNW - 1) / kNW;   // chunks per wave, at most
  const int rows = Hkv * kMT, chunks = (rows * SLOTS + 63) / 64;
  const uint32_t key_bytes = (uint32_t)Hkv * D * 2;
  const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(k), (short)0,
                                                    (uint32_t)S * key_bytes, kBufferDword3);
  const uint32_t kt = (uint32_t)(size_t)(__attribute__((address_space(3))) char *)ktile;
  auto lane_offset = [&](int i) {
    const int slot = (wave + i * kNW) * 64 + lane;
    const int row = slot / SLOTS, col = slot % SLOTS;
    return (row < rows && col < SLOTS - 1)
               ? (uint32_t)(row % kMT) * key_bytes + (uint32_t)((row / kMT) * D + col * 8) * 2
               : ~0u;
  };
  // per-query rows keep the offsets in registers; block aggregation (more
  // live state) recomputes them per tile
  uint32_t koff[ROWS ? kCPW : 1];
  if constexpr (ROWS) {
#pragma unroll
    for (int i = 0; i < kCPW; ++i) koff[i] = lane_offset(i);
  }
  auto issue_k = [&](int k0) {
    const uint32_t sb = (uint32_t)k0 * key_bytes;
#pragma unroll
    for (int i = 0; i < kCPW; ++i) {
      const int c = wave + i * kNW;
      uint32_t off;
      if constexpr (ROWS) off = koff[i];
      else off = lane_offset(i);
      if (c < chunks && off != ~0u)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs, (__attribute__((address_space(3))) void *)(size_t)(kt + c * 1024), 16, off + sb,
            0, 0, 0);
    }
  };

  // B operands of the wave's heads for query tqt + n: dims 16 ks + 8 half ..
  bf16x8 qf[HPW][KS];
  float lse2[HPW];
  auto load_q = [&](int tqt) {
    const int t = min(tqt + n, S - 1);
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      const uint16_t *qp = q + ((size_t)t * Hq + h0 + hh) * D + half * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[hh][ks] = as_bf16x8(ldg16(qp + ks * 16));
      lse2[hh] = lse[(size_t)t * Hq + h0 + hh] * kLog2e;
    }
  };

  // Sum of the eight partials of tile (buffer rb, keys k0 .., queries tqt ..)
  // in wave order, scaled by 1/Hq; masked causally. b = 1: lane -> key
  // lane % 32, rows 4 wave + 2 half + e, stored. b > 1: lane -> key
  // (64 wave + lane) / 16, rows 2 (lane % 16) + e; the block aggregate over
  // the tile's rows goes into yagg.
  const uint32_t red_a = (uint32_t)(size_t)(__attribute__((address_space(3))) float *)&red[0][0][0][0];
  const uint32_t yagg_a = (uint32_t)(size_t)(__attribute__((address_space(3))) float *)yagg;
  auto reduce = [&](int rb, int k0, int tqt) {
    const uint32_t base = red_a + rb * (kNW * kPartBytes);
    if constexpr (ROWS) {
      const int kk = lane & 31, s = k0 + kk, row = 4 * wave + 2 * half;
      float v[2];
      sum_partials2(base + (row * kRS + kk) * 4, base + ((row + 1) * kRS + kk) * 4, v[0], v[1]);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int t = tqt + row + e;
        if (t <= tq_last && s <= t) mass[(size_t)t * S + s] = v[e] * invH;
      }
    } else {
      const int kk = (wave * 64 + lane) >> 4, r2 = lane & 15, s = k0 + kk, row = 2 * r2;
      float v[2];
      sum_partials2(base + (row * kRS + kk) * 4, base + ((row + 1) * kRS + kk) * 4, v[0], v[1]);
      float x = neutral;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int t = tqt + row + e;
        if (t <= tq_last && s <= t) x = op(x, v[e] * invH);
      }
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) x = op(x, __shfl_xor(x, off, 16));
      if (r2 == 0 && s < k_end) {
        const uint32_t ya = yagg_a + (s - k_begin) * 4;
        lds_write_f32(ya, op(lds_read_f32(ya), x));
      }
    }
  };

  const char *krow = ktile + (jj * kMT + n) * KRB + half * 16;
  int rb = 0;
  for (int tqt = tq0; tqt <= tq_last; tqt += kMT) {   // query tiles (one when b = 1)
    const int t_hi = min(tqt + kMT, S) - 1;
    const int ke = min(k_end, t_hi + 1);
    if (k_begin >= ke) continue;   // uniform
    const int ntiles = (ke - k_begin + kMT - 1) / kMT;
    load_q(tqt);
    __syncthreads();   // the previous query tile's K tile and partials are consumed
    issue_k(k_begin);
    for (int it = 0; it < ntiles; ++it) {
      const int k0 = k_begin + it * kMT;
      wait_loads<0>();
      __syncthreads();   // K tile it in LDS
      bf16x8 kf[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kf[ks] = as_bf16x8(lds16(krow + ks * 32));
      __syncthreads();   // every wave holds its K operands: the buffer is free
      if (it + 1 < ntiles) issue_k(k0 + kMT);
      // rows of the previous key tile (their stores complete under this tile)
      if (it > 0) reduce(rb ^ 1, k0 - kMT, tqt);
      // Heads are pipelined: the products of head hh + 1 issue between the
      // exponentials of head hh (one MFMA, then its share of the vector work),
      // so the matrix core runs while the wave exponentiates.
      f32x16 psum;
#pragma unroll
      for (int e = 0; e < 16; ++e) psum[e] = 0.f;
      f32x16 acc[2];
      auto products = [&](int hh, f32x16 &c) {
#pragma unroll
        for (int e = 0; e < 16; ++e) c[e] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) c = mfma32(kf[ks], qf[hh][ks], c);
      };
      auto exponentials = [&](int hh, const f32x16 &c) {
#pragma unroll
        for (int e = 0; e < 16; ++e)
          psum[e] += __builtin_amdgcn_exp2f(fmaf(c[e], scale_log2, -lse2[hh]));
      };
      products(0, acc[0]);
#pragma unroll
      for (int hh = 1; hh < HPW; ++hh) {
        products(hh, acc[hh & 1]);
        exponentials(hh - 1, acc[(hh - 1) & 1]);
        // 48 vector instructions over the KS products: one MFMA, then 48 / KS
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 48 / KS, 0);
        }
      }
      exponentials(HPW - 1, acc[(HPW - 1) & 1]);
      // lane (n, half) holds query n, keys 8i + 4 half + r: element 4i + r
      float *rw = &red[rb][wave][n][half * 4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<float4 *>(rw + 8 * i) =
            make_float4(psum[4 * i], psum[4 * i + 1], psum[4 * i + 2], psum[4 * i + 3]);
      // the next tile's first barrier publishes these partials to its reduce
      rb ^= 1;
    }
    __syncthreads();   // partials of the last tile complete
    reduce(rb ^ 1, k_begin + (ntiles - 1) * kMT, tqt);
  }
  if constexpr (!ROWS) {
    __syncthreads();
    for (int i = tid; i < k_end - k_begin; i += kNW * 64)
      mass[(size_t)blockIdx.x * S + k_begin + i] = yagg[i];
  }
}

template <int D, int HPW>
hipError_t launch32_t(const Prob &p, const void *q, const void *k, const float *lse,
                      float *mass, hipStream_t st) {
  const bool rows = p.b == 1;
  const int span = rows ? kMT : p.b;
  const int chunk = rows ? mass_chunk<true>() : mass_chunk<false>();
  dim3 grid((p.S + span - 1) / span, (p.S + chunk - 1) / chunk);
  if (rows)
    hipLaunchKernelGGL((mass32_kernel<D, HPW, true>), grid, dim3(kNW * 64), 0, st, p.S, p.Hq,
                       p.Hkv, p.G, p.b, p.agg, p.scale * kLog2e, (const uint16_t *)q,
                       (const uint16_t *)k, lse, mass);
  else
    hipLaunchKernelGGL((mass32_kernel<D, HPW, false>), grid, dim3(kNW * 64), 0, st, p.S, p.Hq,
                       p.Hkv, p.G, p.b, p.agg, p.scale * kLog2e, (const uint16_t *)q,
                       (const uint16_t *)k, lse, mass);
  return hipGetLastError();
}

bool mass32_supported(const Prob &p) {
  const int hpw = p.Hq / kNW;
  return p.Hq % kNW == 0 && (hpw == 1 || hpw == 2 || hpw == 4 || (hpw == 8 && p.d == 64)) &&
         p.G % hpw == 0 && p.Hkv <= kMaxHkv && (p.b == 1 || p.b % kMT == 0);
}

template <int D>
hipError_t launch32_d(const Prob &p, const void *q, const void *k, const float *lse,
                      float *mass, hipStream_t st) {
  switch (p.Hq / kNW) {
    case 1: return launch32_t<D, 1>(p, q, k, lse, mass, st);
    case 2: return launch32_t<D, 2>(p, q, k, lse, mass, st);
    case 4: return launch32_t<D, 4>(p, q, k, lse, mass, st);
    default:
      if constexpr (D == 64) return launch32_t<D, 8>(p, q, k, lse, mass, st);
      return hipErrorInvalidValue;
  }
}

}  // namespace

bool mass_mfma_supported(const Prob &p) {
  const int hpw = p.Hq / kNW;
  // at d = 256 the 16-query kernel holds 32 registers of query operands per
  // head: up to four heads a wave (Hq <= 32)
  return p.dtype == SP_DTYPE_BF16 && (p.d == 64 || p.d == 128 || (p.d == 256 && hpw <= 4)) &&
         p.Hq % kNW == 0 && (hpw == 1 || hpw == 2 || hpw == 4 || hpw == 8) &&
         (p.Hkv == 1 || p.Hkv == 2 || p.Hkv == 4 || p.Hkv == 8) &&
         (p.b == 1 || (p.b % 16 == 0 && p.b <= 1024));
}

hipError_t launch_mass_mfma(const Prob &p, const void *q, const void *k, const float *lse,
                            float *mass, hipStream_t st) {
  if (p.d != 256 && mass32_supported(p)) {
    if (p.d == 64) return launch32_d<64>(p, q, k, lse, mass, st);
    return launch32_d<128>(p, q, k, lse, mass, st);
  }
  if (p.d == 64) return launch_d<64>(p, q, k, lse, mass, st);
  if (p.d == 256) return launch_d<256>(p, q, k, lse, mass, st);
  return launch_d<128>(p, q, k, lse, mass, st);
}

}  // namespace sp
