// Selection-block-shared sparse GQA attention on bf16 MFMA (Section 3 restricted
// attention; Section 4.2 per-query causal mask; Algorithm 1 step 5 and
// Algorithm 2 step 5: one support per block, replicated over KV heads).
//
// One workgroup per (selection block r, KV head j, chunk of up to 256 query
// rows). A query row is a (query t, head h) pair with g(h) = j; there are
// b*G of them per (r, j), ordered query-major. The support idx[r] is walked
// in tiles of 64 positions. For each tile the workgroup gathers the 64
// selected K rows (row-major) and V rows (transposed, d-major) of head j
// into LDS once; every wave then reuses them for its 32 query rows. This is
// the only HBM traffic that grows with k: each selected row is read once per
// (block, KV head), not once per query.
//
// Scores are computed transposed (S^T = K Q^T) so that each lane owns one
// query row: the row max, the exponentials, the row sum and the rescale of
// the output (also kept transposed, O^T = V^T P^T) never leave the lane,
// except for one pair of shuffles per tile for the max. Keys with s > t (the
// query's own causal mask), negative sentinels and s >= S contribute nothing.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"

namespace sp {
namespace {

constexpr int kKT = 64;   // support positions per tile
constexpr int kQPW = 32;  // query rows per wave

template <int D>
struct SLayout {
  static constexpr int KRB = D * 2 + 16;        // K tile row bytes (padded)
  static constexpr int VTS = 72;                // V^T row stride in elements (64 + pad)
  static constexpr int KBYTES = kKT * KRB;
  static constexpr int VBYTES = D * VTS * 2;
  static constexpr int BUF = KBYTES + VBYTES + kKT * 4;   // + positions
  static constexpr int KS = D / 32;             // k-steps of Q K^T
  static constexpr int DT = D / 16;             // 16-row tiles of O^T
};

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void sparse_block_kernel(
    int S, int Hq, int Hkv, int G, int b, int kk, float scale_log2,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, const int32_t *__restrict__ idx,
    uint16_t *__restrict__ o) {
  using L = SLayout<D>;
  constexpr int NT = NW * 64;
  constexpr int KS = L::KS, DT = L::DT;
  __shared__ __align__(16) char lds[2][L::BUF];
  __shared__ int red_last[NW];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  const int r = blockIdx.x, j = blockIdx.y;
  const int t0 = r * b;
  const int t1 = min(t0 + b, S) - 1;
  const int nrows = (t1 - t0 + 1) * G;                    // valid query rows of (r, j)
  const int row0 = blockIdx.z * (NW * kQPW) + wave * kQPW; // this wave's first row
  const int32_t *ir = idx + (size_t)r * kk;

  // Last support entry that any query of the block can use, over any order.
  int last = -1;
  for (int c = tid; c < kk; c += NT) {
    const int s = ir[c];
    if (s >= 0 && s <= t1) last = c;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) last = max(last, __shfl_xor(last, off, 64));
  if (lane == 0) red_last[wave] = last;
  __syncthreads();
  last = -1;
#pragma unroll
  for (int w = 0; w < NW; ++w) last = max(last, red_last[w]);
  const int ntiles = (last + kKT) / kKT;  // 0 when nothing is usable

  // This lane's query rows (one per 16-row tile qc) and their Q fragments.
  int qt[2];
  bool qvalid[2];
  bf16x8 bq[2][KS];
#pragma unroll
  for (int qc = 0; qc < 2; ++qc) {
    const int m = row0 + qc * 16 + c16;
    qvalid[qc] = m < nrows;
    const int mm = qvalid[qc] ? m : 0;
    qt[qc] = t0 + mm / G;
    const int h = j * G + mm % G;
    const uint16_t *qp = q + ((size_t)qt[qc] * Hq + h) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) bq[qc][ks] = as_bf16x8(ldg16(qp + ks * 32 + g * 8));
  }

  // Gather assignment. K: 16-byte pieces c = tid + i*NT (key c / (D/8)).
  // V: thread -> (key quad, 4 consecutive d) when the tile has enough quads.
  constexpr int KPIECES = kKT * D / 8;
  constexpr int KPER = (KPIECES + NT - 1) / NT;
  constexpr int VUNITS = (kKT / 4) * (D / 4);   // (key quad, d quad) units
  constexpr int VPER = (VUNITS + NT - 1) / NT;
  uint4 kreg[KPER];
  uint2 vreg[VPER][4];
  int spos = -1;

  auto gather = [&](int c0) {
#pragma unroll
    for (int i = 0; i < KPER; ++i) {
      const int c = tid + i * NT;
      if (c < KPIECES) {
        const int key = c / (D / 8), col = c % (D / 8);
        const int e = c0 + key;
        int s = e < kk ? ir[e] : -1;
        s = (s >= 0 && s < S) ? s : 0;
        kreg[i] = ldg16(k + ((size_t)s * Hkv + j) * D + col * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < VPER; ++i) {
      const int u = tid + i * NT;
      if (u < VUNITS) {
        const int kq = u / (D / 4), dq = u % (D / 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int c = c0 + kq * 4 + e;
          int s = c < kk ? ir[c] : -1;
          s = (s >= 0 && s < S) ? s : 0;
          vreg[i][e] = *reinterpret_cast<const uint2 *>(v + ((size_t)s * Hkv + j) * D + dq * 4);
        }
      }
    }
    if (tid < kKT) {
      const int c = c0 + tid;
      spos = c < kk ? ir[c] : -1;
    }
  };
  auto stage = [&](char *buf) {
    char *kl = buf;
    uint16_t *vt = reinterpret_cast<uint16_t *>(buf + L::KBYTES);
    int *sl = reinterpret_cast<int *>(buf + L::KBYTES + L::VBYTES);
#pragma unroll
    for (int i = 0; i < KPER; ++i) {
      const int c = tid + i * NT;
      if (c < KPIECES) {
        const int key = c / (D / 8), col = c % (D / 8);
        sts16(kl + key * L::KRB + col * 16, kreg[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < VPER; ++i) {
      const int u = tid + i * NT;
      if (u < VUNITS) {
        const int kq = u / (D / 4), dq = u % (D / 4);
        // vreg[i][e] holds d = 4dq..4dq+3 of key 4kq+e; write column-wise.
#pragma unroll
        for (int dd = 0; dd < 4; ++dd) {
          uint32_t w[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t word = (dd < 2) ? vreg[i][e].x : vreg[i][e].y;
            w[e] = (dd & 1) ? (word >> 16) : (word & 0xffffu);
          }
          uint2 packed;
          packed.x = w[0] | (w[1] << 16);
          packed.y = w[2] | (w[3] << 16);
          *reinterpret_cast<uint2 *>(vt + (dq * 4 + dd) * L::VTS + kq * 4) = packed;
        }
      }
    }
    if (tid < kKT) sl[tid] = spos;
  };

  f32x4 oacc[DT][2];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int qc = 0; qc < 2; ++qc) oacc[dt][qc] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow[2] = {-INFINITY, -INFINITY};
  float lrow[2] = {0.f, 0.f};   // this lane's share of the row sum

  if (ntiles > 0) {
    gather(0);
    stage(lds[0]);
  }
  __syncthreads();
  const bool wave_live = row0 < nrows;
  for (int it = 0; it < ntiles; ++it) {
    const bool more = it + 1 < ntiles;
    if (more) gather((it + 1) * kKT);
    const char *cur = lds[it & 1];
    if (wave_live) {
      const char *kl = cur;
      const uint16_t *vt = reinterpret_cast<const uint16_t *>(cur + L::KBYTES);
      const int *sl = reinterpret_cast<const int *>(cur + L::KBYTES + L::VBYTES);
      // S^T = K Q^T for 4 key tiles of 16 x 2 query tiles of 16.
      f32x4 sacc[4][2];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
        for (int qc = 0; qc < 2; ++qc) sacc[kt][qc] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 a = as_bf16x8(lds16(kl + (kt * 16 + c16) * L::KRB + ks * 64 + g * 16));
#pragma unroll
          for (int qc = 0; qc < 2; ++qc) sacc[kt][qc] = mfma16(a, bq[qc][ks], sacc[kt][qc]);
        }
      }
      // Online softmax, per lane (query row) and tile.
      bf16x8 pfrag[2][2];   // [qc][32-key half]
#pragma unroll
      for (int qc = 0; qc < 2; ++qc) {
        float x[4][4];
        float tmax = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          const int4 s4 = *reinterpret_cast<const int4 *>(sl + kt * 16 + g * 4);
          const int sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const bool ok = sv[rr] >= 0 && sv[rr] <= qt[qc] && sv[rr] < S;
            x[kt][rr] = ok ? sacc[kt][qc][rr] * scale_log2 : -INFINITY;
            tmax = fmaxf(tmax, x[kt][rr]);
          }
        }
        tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
        const float mnew = fmaxf(mrow[qc], tmax);
        const float mref = mnew == -INFINITY ? 0.f : mnew;
        const float corr = exp2f(mrow[qc] - mref);
        mrow[qc] = mnew;
        float psum = 0.f;
        float pv[4][4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            pv[kt][rr] = exp2f(x[kt][rr] - mref);
            psum += pv[kt][rr];
          }
        lrow[qc] = lrow[qc] * corr + psum;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) oacc[dt][qc][rr] *= corr;
#pragma unroll
        for (int f = 0; f < 2; ++f) {
          bf16x8 pf;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            pf[e] = (__bf16)pv[2 * f][e];
            pf[4 + e] = (__bf16)pv[2 * f + 1][e];
          }
          pfrag[qc][f] = pf;
        }
      }
      // O^T += V^T P^T over the tile's two 32-key halves.
#pragma unroll
      for (int f = 0; f < 2; ++f) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const uint16_t *vrow = vt + (dt * 16 + c16) * L::VTS + f * 32 + g * 4;
          const uint2 lo = *reinterpret_cast<const uint2 *>(vrow);
          const uint2 hi = *reinterpret_cast<const uint2 *>(vrow + 16);
          uint4 u;
          u.x = lo.x; u.y = lo.y; u.z = hi.x; u.w = hi.y;
          const bf16x8 a = as_bf16x8(u);
#pragma unroll
          for (int qc = 0; qc < 2; ++qc) oacc[dt][qc] = mfma16(a, pfrag[qc][f], oacc[dt][qc]);
        }
      }
    }
    if (more) stage(lds[(it + 1) & 1]);
    __syncthreads();
  }

  if (!wave_live) return;
#pragma unroll
  for (int qc = 0; qc < 2; ++qc) {
    float l = lrow[qc];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (!qvalid[qc]) continue;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const int m = row0 + qc * 16 + c16;
    const int h = j * G + m % G;
    uint16_t *op = o + ((size_t)qt[qc] * Hq + h) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      uint2 w;
      w.x = (uint32_t)float_to_bf16(oacc[dt][qc][0] * inv) |
            ((uint32_t)float_to_bf16(oacc[dt][qc][1] * inv) << 16);
      w.y = (uint32_t)float_to_bf16(oacc[dt][qc][2] * inv) |
            ((uint32_t)float_to_bf16(oacc[dt][qc][3] * inv) << 16);
      *reinterpret_cast<uint2 *>(op + dt * 16 + g * 4) = w;
    }
  }
}

template <int D>
hipError_t launch_d(const Prob &p, const void *q, const void *k, const void *v,
                    const int32_t *idx, void *o, hipStream_t st) {
  const int rows = p.b * p.G;
  int nw = (rows + kQPW - 1) / kQPW;
  nw = nw <= 1 ? 1 : nw <= 2 ? 2 : nw <= 4 ? 4 : 8;
  const int chunks = (rows + nw * kQPW - 1) / (nw * kQPW);
  dim3 grid(p.R, p.Hkv, chunks);
  const float sl2 = p.scale * kLog2e;
#define SP_SB(NW)                                                                            \
  hipLaunchKernelGGL((sparse_block_kernel<D, NW>), grid, dim3(NW * 64), 0, st, p.S, p.Hq,    \
                     p.Hkv, p.G, p.b, p.k, sl2, (const uint16_t *)q, (const uint16_t *)k,     \
                     (const uint16_t *)v, idx, (uint16_t *)o)
  switch (nw) {
    case 1: SP_SB(1); break;
    case 2: SP_SB(2); break;
    case 4: SP_SB(4); break;
    default: SP_SB(8); break;
  }
#undef SP_SB
  return hipGetLastError();
}

}  // namespace

bool sparse_block_mfma_supported(const Prob &p) {
  return p.dtype == SP_DTYPE_BF16 && (p.d == 64 || p.d == 128) && p.b >= 16;
}

hipError_t launch_sparse_block_mfma(const Prob &p, const void *q, const void *k, const void *v,
                                    const int32_t *idx, void *o, hipStream_t st) {
  if (p.d == 64) return launch_d<64>(p, q, k, v, idx, o, st);
  return launch_d<128>(p, q, k, v, idx, o, st);
}

}  // namespace sp
