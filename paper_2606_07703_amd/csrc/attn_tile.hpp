// Attention tile machinery shared by the MFMA attention kernels.
//
// A workgroup owns up to 256 query rows ((query, head) pairs of one KV head,
// 32 per wave) and walks a list of key positions in tiles of 64. For each
// tile it stages K and V of the KV head in LDS (both row-major, padded rows),
// plus the tile's positions and their min/max. attn_tile() then updates each
// lane's online-softmax state: scores are computed transposed, S^T = K Q^T,
// so lane (g, c16) owns query row c16 of each 16-row tile and holds keys
// 16*kt + 4g + r; the output is kept transposed too, O^T = V^T P^T, with the
// V^T operand read straight from the row-major V tile by the gfx950 LDS
// transpose read (ds_read_b64_tr_b16), so the per-row rescale stays in the
// lane and no transposed copy of V is ever written.
//
// A key at position s contributes to a row of query t only if
// 0 <= s <= t (the causal mask of Section 3, applied per query as in
// Section 4.2); any other position (e.g. a -1 sentinel) contributes nothing.
// A wave skips the mask test on tiles whose positions all lie in
// [0, first query of the wave].
//
// The running row maximum is raised only when a tile's maximum exceeds it by
// more than 2^kLazy in the exponent base-2 domain; until then the stale
// maximum is kept (probabilities up to 2^kLazy are exact in fp32 and bf16
// range), so the output accumulators are rescaled only when it moves.
#pragma once

#include <math.h>

#include "common.hpp"
#include "mfma.hpp"

namespace sp {

constexpr int kAttnKT = 64;      // key positions per tile
constexpr int kAttnQPW = 32;     // query rows per wave
constexpr float kLazy = 8.f;     // max may lag by up to 8 (factor 256)
// Word 3 of a raw buffer resource on gfx950: 32-bit data format, no swizzle.
constexpr int kBufferDword3 = 0x00020000;

typedef short v4i16 __attribute__((ext_vector_type(4)));

template <int D>
struct AttnLayout {
  static constexpr int KRB = D * 2 + 16;   // K row bytes: 16 lanes x 16 B on distinct banks
  static constexpr int VRB = D * 2 + 32;   // V row bytes: conflict-free transpose reads
  static constexpr int KBYTES = kAttnKT * KRB;
  static constexpr int VBYTES = kAttnKT * VRB;
  static constexpr int POS = KBYTES + VBYTES;          // int positions[64], then min, max
  static constexpr int BUF = POS + kAttnKT * 4 + 16;
  static constexpr int KS = D / 32;        // k-steps of K Q^T
  static constexpr int DT = D / 16;        // 16-row tiles of O^T
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Wait for every outstanding memory operation of this wave. Issued once
// before a tile loop, it tells the compiler that loads made before the loop
// (Q fragments, the first tile) are complete, so no wait on them is placed
// inside the loop, where it would also stall on the next tile's prefetch.
__device__ __forceinline__ void drain_memory() { __builtin_amdgcn_s_waitcnt(0); }

// Global -> registers -> LDS staging of one tile of K, V and positions.
// pos(e) gives the position of tile entry e (0..63), or a negative value.
template <int D, int NT, bool WANT_V>
struct KVStage {
  using L = AttnLayout<D>;
  static constexpr int PIECES = kAttnKT * D / 8;    // 16-byte pieces of one tile
  static constexpr int PER = (PIECES + NT - 1) / NT;
  uint4 kreg[PER];
  uint4 vreg[WANT_V ? PER : 1];
  int spos;

  // All positions are resolved before any row load is issued, so the row
  // loads of a tile go out back to back.
  template <typename POS>
  __device__ __forceinline__ void load(const uint16_t *__restrict__ k,
                                       const uint16_t *__restrict__ v, int S, int Hkv, int j,
                                       int tid, POS pos) {
    load_rows(k, v, S, Hkv, j, tid, pos, pos);
  }

  // As load, with the K/V row of tile entry e given by row(e) (a paged
  // cache) while pos(e) stays the token position the mask uses; k and v
  // hold nrows rows of Hkv heads.
  template <typename POS, typename ROW>
  __device__ __forceinline__ void load_rows(const uint16_t *__restrict__ k,
                                            const uint16_t *__restrict__ v, int nrows, int Hkv,
                                            int j, int tid, POS pos, ROW row) {
    // Rows are fetched through buffer resources (base and size in SGPRs,
    // 32-bit byte offsets per lane): one multiply-add per piece instead of
    // 64-bit address arithmetic. The API keeps k and v below 4 GiB.
    const uint32_t nbytes = (uint32_t)nrows * Hkv * D * 2;
    const auto krs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(k), (short)0,
                                                       nbytes, kBufferDword3);
    const auto vrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(v), (short)0,
                                                       nbytes, kBufferDword3);
    uint32_t off[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      const int key = c / (D / 8), col = c % (D / 8);
      int s = c < PIECES ? row(key) : 0;
      s = (s >= 0 && s < nrows) ? s : 0;
      off[i] = ((uint32_t)s * Hkv + j) * (D * 2) + col * 16;
    }
    if (tid < kAttnKT) spos = pos(tid);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (tid + i * NT < PIECES) {
        kreg[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(krs, off[i], 0, 0));
        if constexpr (WANT_V)
          vreg[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(vrs, off[i], 0, 0));
      }
    }
  }

  // Also publishes min and max of the tile's positions (wave 0 holds them).
  __device__ __forceinline__ void store(char *buf, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < PIECES) {
        const int key = c / (D / 8), col = c % (D / 8);
        sts16(buf + key * L::KRB + col * 16, kreg[i]);
        if constexpr (WANT_V) sts16(buf + L::KBYTES + key * L::VRB + col * 16, vreg[i]);
      }
    }
    if (tid < kAttnKT) {
      int *pl = reinterpret_cast<int *>(buf + L::POS);
      pl[tid] = spos;
      int mn = spos, mx = spos;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        mn = min(mn, __shfl_xor(mn, off, 64));
        mx = max(mx, __shfl_xor(mx, off, 64));
      }
      if (tid == 0) {
        pl[kAttnKT] = mn;
        pl[kAttnKT + 1] = mx;
      }
    }
  }
};

// Per-wave online-softmax state for 2 x 16 query rows.
template <int D>
struct AttnState {
  f32x4 oacc[AttnLayout<D>::DT][2];
  float m[2];   // running max (base-2 scaled logits), possibly lagging by < kLazy
  float l[2];   // this lane's share of the row sum (reduce over g at the end)
  // Row sums taken on the matrix cores (attn_tile MFMA_SUM): a ones A
  // operand times P^T puts each row's sum in every C row.
  f32x4 lsum[2];
  __device__ __forceinline__ void init() {
    lsum[0] = lsum[1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < AttnLayout<D>::DT; ++dt)
#pragma unroll
      for (int qc = 0; qc < 2; ++qc) oacc[dt][qc] = f32x4{0.f, 0.f, 0.f, 0.f};
    m[0] = m[1] = -INFINITY;
    l[0] = l[1] = 0.f;
  }
};

// One tile: scores, mask, online softmax, and (WANT_O) the P V product.
// wave_tmin is the smallest query of the wave's valid rows. MFMA_SUM (with
// WANT_O) takes the row sums from the matrix cores, over the same bf16
// probabilities that weight V; otherwise they are fp32 vector sums (kept
// where the log-sum-exp is an output).
template <int D, bool WANT_O, bool MFMA_SUM = false>
__device__ __forceinline__ void attn_tile(const char *buf, const bf16x8 (&bq)[2][AttnLayout<D>::KS],
                                          const int (&qt)[2], float scale_log2, int wave_tmin,
                                          AttnState<D> &st, int g, int c16) {
  using L = AttnLayout<D>;
  constexpr int KS = L::KS, DT = L::DT;
  const char *kl = buf;
  const char *vl = buf + L::KBYTES;
  const int *sl = reinterpret_cast<const int *>(buf + L::POS);
  const bool mask = !(sl[kAttnKT] >= 0 && sl[kAttnKT + 1] <= wave_tmin);
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
  if (mask) {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const int4 s4 = *reinterpret_cast<const int4 *>(sl + kt * 16 + g * 4);
      const int sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
      for (int qc = 0; qc < 2; ++qc)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
          if (!(sv[rr] >= 0 && sv[rr] <= qt[qc])) sacc[kt][qc][rr] = -INFINITY;
    }
  }
  bf16x8 pfrag[2][2];
  bool grew_any = false;
  float corr[2];
#pragma unroll
  for (int qc = 0; qc < 2; ++qc) {
    float tmax = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) tmax = fmaxf(tmax, sacc[kt][qc][rr]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    tmax *= scale_log2;   // scale > 0 commutes with max
    const float mold = st.m[qc];
    const bool grow = tmax > mold + kLazy;
    const float mnew = grow ? tmax : mold;
    grew_any |= grow;
    const float mref = mnew == -INFINITY ? 0.f : mnew;
    corr[qc] = fast_exp2(mold - mref);   // mold = -inf gives 0; unchanged gives 1
    st.m[qc] = mnew;
    float psum = 0.f;
    float pv[4][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        pv[kt][rr] = fast_exp2(fmaf(sacc[kt][qc][rr], scale_log2, -mref));
        if constexpr (!MFMA_SUM) psum += pv[kt][rr];
      }
    if constexpr (!MFMA_SUM) st.l[qc] = st.l[qc] * corr[qc] + psum;
    if constexpr (WANT_O) {
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
    if (__any(grew_any)) {
#pragma unroll
      for (int qc = 0; qc < 2; ++qc)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) st.oacc[dt][qc][rr] *= corr[qc];
      if constexpr (MFMA_SUM) {
#pragma unroll
        for (int qc = 0; qc < 2; ++qc)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) st.lsum[qc][rr] *= corr[qc];
      }
    }
    if constexpr (MFMA_SUM) {
      // one MFMA per 32 keys and 16 rows instead of 32 vector adds per tile
      bf16x8 ones;
#pragma unroll
      for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;
#pragma unroll
      for (int qc = 0; qc < 2; ++qc)
#pragma unroll
        for (int f = 0; f < 2; ++f) st.lsum[qc] = mfma16(ones, pfrag[qc][f], st.lsum[qc]);
    }
    // O^T += V^T P^T. Lane (g, c16) of the V^T fragment needs d = 16dt + c16
    // and keys 32f + 4g + {0..3} (then +16): each transpose read has the 16
    // lanes of group g point at rows 32f + 4g + c16/4 (+16), d = 16dt + 4(c16%4).
    const char *vbase = vl + (g * 4 + (c16 >> 2)) * L::VRB + (c16 & 3) * 8;
#pragma unroll
    for (int f = 0; f < 2; ++f) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const char *p0 = vbase + (f * 32) * L::VRB + dt * 32;
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16 *)(size_t)(p0));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16 *)(size_t)(p0 + 16 * L::VRB));
        bf16x8 a;
        __builtin_memcpy(&a, &lo, 8);
        __builtin_memcpy(reinterpret_cast<char *>(&a) + 8, &hi, 8);
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
    l += st.lsum[qc][0];
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
