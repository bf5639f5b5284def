// Attention tile machinery shared by the MFMA attention kernels.
//
// A workgroup owns up to 256 query rows ((query, head) pairs of one KV head,
// 32 per wave) and walks a list of key positions in tiles of 64. For each
// tile it stages K (row-major, padded rows) and V (transposed, d-major) of
// the KV head in LDS, plus the tile's positions. attn_tile() then updates
// each lane's online-softmax state: scores are computed transposed,
// S^T = K Q^T, so lane (g, c16) owns query row c16 of each 16-row tile and
// holds keys 16*kt + 4g + r; the output is kept transposed too,
// O^T = V^T P^T, so the per-row rescale stays in the lane.
//
// A key at position s contributes to a row of query t only if
// 0 <= s <= t and s < S (the causal mask of Section 3, applied per query as
// in Section 4.2); any other position (e.g. a -1 sentinel) contributes
// nothing.
#pragma once

#include <math.h>

#include "common.hpp"
#include "mfma.hpp"

namespace sp {

constexpr int kAttnKT = 64;    // key positions per tile
constexpr int kAttnQPW = 32;   // query rows per wave

template <int D>
struct AttnLayout {
  static constexpr int KRB = D * 2 + 16;   // K row bytes, padded: 16 lanes hit distinct banks
  static constexpr int VTS = 72;           // V^T row stride (elements): conflict-free b64 reads
  static constexpr int KBYTES = kAttnKT * KRB;
  static constexpr int VBYTES = D * VTS * 2;
  static constexpr int BUF = KBYTES + VBYTES + kAttnKT * 4;
  static constexpr int KS = D / 32;        // k-steps of K Q^T
  static constexpr int DT = D / 16;        // 16-row tiles of O^T
};

// Global -> registers -> LDS staging of one tile of K, V^T and positions.
// POS(c) gives the position of tile entry c (0..63), or a negative value.
template <int D, int NT, bool WANT_V>
struct KVStage {
  using L = AttnLayout<D>;
  static constexpr int KPIECES = kAttnKT * D / 8;
  static constexpr int KPER = (KPIECES + NT - 1) / NT;
  static constexpr int VUNITS = (kAttnKT / 4) * (D / 4);
  static constexpr int VPER = WANT_V ? (VUNITS + NT - 1) / NT : 0;
  uint4 kreg[KPER];
  uint2 vreg[VPER > 0 ? VPER : 1][4];
  int spos;

  template <typename POS>
  __device__ __forceinline__ void load(const uint16_t *__restrict__ k,
                                       const uint16_t *__restrict__ v, int S, int Hkv, int j,
                                       int tid, POS pos) {
#pragma unroll
    for (int i = 0; i < KPER; ++i) {
      const int c = tid + i * NT;
      if (c < KPIECES) {
        const int key = c / (D / 8), col = c % (D / 8);
        int s = pos(key);
        s = (s >= 0 && s < S) ? s : 0;
        kreg[i] = ldg16(k + ((size_t)s * Hkv + j) * D + col * 8);
      }
    }
    if constexpr (WANT_V) {
#pragma unroll
      for (int i = 0; i < VPER; ++i) {
        const int u = tid + i * NT;
        if (u < VUNITS) {
          const int kq = u / (D / 4), dq = u % (D / 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            int s = pos(kq * 4 + e);
            s = (s >= 0 && s < S) ? s : 0;
            vreg[i][e] = *reinterpret_cast<const uint2 *>(v + ((size_t)s * Hkv + j) * D + dq * 4);
          }
        }
      }
    }
    if (tid < kAttnKT) spos = pos(tid);
  }

  __device__ __forceinline__ void store(char *buf, int tid) const {
    char *kl = buf;
#pragma unroll
    for (int i = 0; i < KPER; ++i) {
      const int c = tid + i * NT;
      if (c < KPIECES) {
        const int key = c / (D / 8), col = c % (D / 8);
        sts16(kl + key * L::KRB + col * 16, kreg[i]);
      }
    }
    if constexpr (WANT_V) {
      uint16_t *vt = reinterpret_cast<uint16_t *>(buf + L::KBYTES);
#pragma unroll
      for (int i = 0; i < VPER; ++i) {
        const int u = tid + i * NT;
        if (u < VUNITS) {
          const int kq = u / (D / 4), dq = u % (D / 4);
          // vreg[i][e] holds d = 4dq..4dq+3 of key 4kq+e; write one d row at a time.
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
    }
    if (tid < kAttnKT) reinterpret_cast<int *>(buf + L::KBYTES + L::VBYTES)[tid] = spos;
  }
};

// Per-wave online-softmax state for 2 x 16 query rows.
template <int D>
struct AttnState {
  f32x4 oacc[AttnLayout<D>::DT][2];
  float m[2];
  float l[2];   // this lane's share of the row sum (reduce over g at the end)
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int dt = 0; dt < AttnLayout<D>::DT; ++dt)
#pragma unroll
      for (int qc = 0; qc < 2; ++qc) oacc[dt][qc] = f32x4{0.f, 0.f, 0.f, 0.f};
    m[0] = m[1] = -INFINITY;
    l[0] = l[1] = 0.f;
  }
};

// One tile: scores, mask, online softmax, and (WANT_O) the P V product.
// mask = false promises every staged position p satisfies 0 <= p <= qt.
template <int D, bool WANT_O>
__device__ __forceinline__ void attn_tile(const char *buf, const bf16x8 (&bq)[2][AttnLayout<D>::KS],
                                          const int (&qt)[2], float scale_log2, bool mask,
                                          AttnState<D> &st, int g, int c16) {
  using L = AttnLayout<D>;
  constexpr int KS = L::KS, DT = L::DT;
  const char *kl = buf;
  const uint16_t *vt = reinterpret_cast<const uint16_t *>(buf + L::KBYTES);
  const int *sl = reinterpret_cast<const int *>(buf + L::KBYTES + L::VBYTES);
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
  bf16x8 pfrag[2][2];
#pragma unroll
  for (int qc = 0; qc < 2; ++qc) {
    float x[4][4];
    float tmax = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      int4 s4 = make_int4(0, 0, 0, 0);
      if (mask) s4 = *reinterpret_cast<const int4 *>(sl + kt * 16 + g * 4);
      const int sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const bool ok = !mask || (sv[rr] >= 0 && sv[rr] <= qt[qc]);
        x[kt][rr] = ok ? sacc[kt][qc][rr] * scale_log2 : -INFINITY;
        tmax = fmaxf(tmax, x[kt][rr]);
      }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(st.m[qc], tmax);
    const float mref = mnew == -INFINITY ? 0.f : mnew;
    const float corr = exp2f(st.m[qc] - mref);
    st.m[qc] = mnew;
    float psum = 0.f;
    float pv[4][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        pv[kt][rr] = exp2f(x[kt][rr] - mref);
        psum += pv[kt][rr];
      }
    st.l[qc] = st.l[qc] * corr + psum;
    if constexpr (WANT_O) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) st.oacc[dt][qc][rr] *= corr;
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
  }
  if constexpr (WANT_O) {
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
        for (int qc = 0; qc < 2; ++qc) st.oacc[dt][qc] = mfma16(a, pfrag[qc][f], st.oacc[dt][qc]);
      }
    }
  }
}

// Q fragments (B operand of K Q^T) for this lane's two query rows.
// Row m (query-major within the workgroup's rows) is query t0 + m/G, head j*G + m%G.
template <int D>
__device__ __forceinline__ void load_q_rows(const uint16_t *__restrict__ q, int Hq, int G, int j,
                                            int t0, int row0, int nrows, int g, int c16,
                                            bf16x8 (&bq)[2][AttnLayout<D>::KS], int (&qt)[2],
                                            int (&qh)[2], bool (&qvalid)[2]) {
#pragma unroll
  for (int qc = 0; qc < 2; ++qc) {
    const int m = row0 + qc * 16 + c16;
    qvalid[qc] = m < nrows;
    const int mm = qvalid[qc] ? m : 0;
    qt[qc] = t0 + mm / G;
    qh[qc] = j * G + mm % G;
    const uint16_t *qp = q + ((size_t)qt[qc] * Hq + qh[qc]) * D;
#pragma unroll
    for (int ks = 0; ks < AttnLayout<D>::KS; ++ks)
      bq[qc][ks] = as_bf16x8(ldg16(qp + ks * 32 + g * 8));
  }
}

// Final normalisation: writes o (bf16, if non-null) and lse (natural log, if
// non-null) for this lane's valid rows. Rows with no usable key get o = 0
// and lse = -inf.
template <int D>
__device__ __forceinline__ void attn_finish(AttnState<D> &st, const int (&qt)[2],
                                            const int (&qh)[2], const bool (&qvalid)[2], int Hq,
                                            uint16_t *__restrict__ o, float *__restrict__ lse,
                                            int g) {
#pragma unroll
  for (int qc = 0; qc < 2; ++qc) {
    float l = st.l[qc];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (!qvalid[qc]) continue;
    if (lse && g == 0)
      lse[(size_t)qt[qc] * Hq + qh[qc]] = l > 0.f ? (st.m[qc] + log2f(l)) * kLn2 : -INFINITY;
    if (o) {
      const float inv = l > 0.f ? 1.f / l : 0.f;
      uint16_t *op = o + ((size_t)qt[qc] * Hq + qh[qc]) * D;
#pragma unroll
      for (int dt = 0; dt < AttnLayout<D>::DT; ++dt) {
        uint2 w;
        w.x = (uint32_t)float_to_bf16(st.oacc[dt][qc][0] * inv) |
              ((uint32_t)float_to_bf16(st.oacc[dt][qc][1] * inv) << 16);
        w.y = (uint32_t)float_to_bf16(st.oacc[dt][qc][2] * inv) |
              ((uint32_t)float_to_bf16(st.oacc[dt][qc][3] * inv) << 16);
        *reinterpret_cast<uint2 *>(op + dt * 16 + g * 4) = w;
      }
    }
  }
}

}  // namespace sp
