// Sparse GQA attention for per-query (or small-block) supports on bf16 MFMA
// (Section 3 restricted attention; Section 4.2 per-query causal mask;
// Algorithm 2, selection and sparse GQA prefill with b_sel = 1).
//
// Each query owns its support, so there is nothing to share between queries:
// one wave handles one (query t, KV head j) pair and the G query heads of
// that group. Per 32-entry tile of the support row it
//   * gathers the 32 selected K rows straight into MFMA A operands and
//     computes S^T = K Q^T (keys x heads; the G heads fill G of the 16 MFMA
//     columns),
//   * runs the online softmax with each lane holding 8 keys of one head
//     column,
//   * stages the 32 V rows in a wave-private LDS slot and forms
//     O^T += V^T P^T, reading V^T with the gfx950 transpose read.
// The support row itself is copied once into the wave's LDS slot so the
// gather addresses of the next tile are an LDS read away. Work items are laid
// out so that workgroup i (which runs on XCD i % 8) holds KV head i % Hkv: with
// 8 KV heads each XCD's L2 serves the gathers of one head.
//
// Tile entries: MFMA row m of key-tile kt (0..1) is tile entry
// 8(m/4) + 4kt + m%4, so the lane (g, c) that holds rows 4g..4g+3 of both
// key-tiles holds tile entries 8g..8g+7: the same 8 entries whose V rows it
// stages, whose positions it masks with, and whose probabilities form its B
// operand of the P V product.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"

namespace sp {
namespace {

constexpr int kQT = 32;         // support entries per tile
constexpr int kPosChunk = 2048; // support entries held in LDS at a time
constexpr float kLazyQ = 8.f;   // running max may lag by up to 2^8

typedef short v4i16 __attribute__((ext_vector_type(4)));

template <int NW, int D>
struct QuerySlots {
  static constexpr int VRB = 2 * D + 32;   // V row bytes: conflict-free transpose reads
  static constexpr int KRB = 2 * D + 16;   // K row bytes: conflict-free operand reads
  int pos[NW][kPosChunk];
  // one slot per wave: a tile's K rows, then (once its products have read
  // them) the same tile's V rows
  char slot[NW][kQT * (VRB > KRB ? VRB : KRB)];
};

template <class Op>
__device__ __forceinline__ float reduce4(float x, Op op) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  const float y = op(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto c = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false,
                                                  false);
  return op(__uint_as_float(c[0]), __uint_as_float(c[1]));
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void sparse_query_kernel(
    int S, int Hq, int Hkv, int G, int b, int kk, size_t gstride, int n_groups, float scale_log2,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, const int32_t *__restrict__ idx,
    uint16_t *__restrict__ o, KvPages pages, int qo) {
  // q and o are addressed by position: the host shifts them back by qo rows
  constexpr int KS = D / 32, DT = D / 16;
  constexpr int PPR = D / 8;         // 16-byte pieces per K/V row
  constexpr int RPL = PPR / 2;       // V pieces per lane per tile (8 rows x PPR / 16 lanes)
  using Slots = QuerySlots<NW, D>;
  constexpr int VRB = Slots::VRB, KRB = Slots::KRB;
  __shared__ __align__(16) Slots sh;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 4, c16 = lane & 15;

  const int j = blockIdx.x % Hkv;
  const int grp = n_groups - 1 - blockIdx.x / Hkv;   // longest queries first
  const int t = qo + grp * NW + wave;
  if (t >= S) return;   // no workgroup barrier below: waves are independent
  const int32_t *row = idx + (size_t)j * gstride + (size_t)((t - qo) / b) * kk;
  int *ipos = sh.pos[wave];
  char *vb = sh.slot[wave];
  char *kbs = sh.slot[wave];

  // Q as the B operand of S^T = K Q^T: column c16 is head j*G + c16.
  const bool hcol = c16 < G;
  const int h = j * G + (hcol ? c16 : 0);
  bf16x8 qb[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const uint4 u = ldg16(q + ((size_t)t * Hq + h) * D + ks * 32 + g * 8);
    qb[ks] = as_bf16x8(hcol ? u : make_uint4(0, 0, 0, 0));
  }

  f32x4 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const size_t kv_head = (size_t)j * D;
  const size_t kv_row = (size_t)Hkv * D;

  for (int c0 = 0; c0 < kk; c0 += kPosChunk) {
    const int n = min(kPosChunk, kk - c0);
    // Copy the chunk of the support row into the wave's slot as K/V rows;
    // entries that cannot contribute (sentinel, out of range, after t, a
    // page outside the cache) become -1. The tile loop ends after the last
    // usable entry.
    int last = -1;
    for (int e = lane; e < kPosChunk; e += 64) {
      int s = e < n ? row[c0 + e] : -1;
      s = (s >= 0 && s <= t) ? pages.row(s) : -1;
      ipos[e] = s;
      if (s >= 0) last = e;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) last = max(last, __shfl_xor(last, off, 64));
    const int ntiles = (last + kQT) / kQT;
    if (ntiles == 0) continue;

    // Gather of tile it into registers, K and V alike: the 8 rows of group g
    // are 8 PPR 16-byte pieces; lane (g, c16) takes pieces c16 + 16e, e <
    // RPL, that is piece (c16 + 16e) % PPR of row 8g + (c16 + 16e) / PPR (at
    // d = 128 its own 8 entries, whole). A gather instruction then covers 4
    // whole rows: the address unit serves that shape at more than twice the
    // rate of 16 rows x 64 bytes (the MFMA operand layout, which K is read
    // in from the wave's LDS slot instead).
    uint4 kreg[RPL], vreg[RPL];
    // tile entry (within the group's 8) and piece of the lane's V piece e:
    // compile-time where PPR >= 16, else the lane's half picks the entry
    auto ventry = [&](int e) { return PPR >= 16 ? 16 * e / PPR : (c16 + 16 * e) / PPR; };
    auto vpiece = [&](int e) { return (c16 + 16 * e) % PPR; };
    auto issue = [&](int it) {
      const int e0 = it * kQT;
      const int4 pa = *reinterpret_cast<const int4 *>(ipos + e0 + 8 * g);
      const int4 pb = *reinterpret_cast<const int4 *>(ipos + e0 + 8 * g + 4);
      const int ps[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
#pragma unroll
      for (int e = 0; e < RPL; ++e) {
        int s;
        if constexpr (PPR >= 16) {
          s = ps[16 * e / PPR];
        } else {   // entries 2e (lanes c16 < 8) and 2e + 1 (c16 >= 8) at d = 64
          static_assert(PPR == 8, "d = 64, 128 or 256");
          s = c16 >= 8 ? ps[2 * e + 1] : ps[2 * e];
        }
        const size_t rb = (size_t)max(s, 0) * kv_row + kv_head + vpiece(e) * 8;
        kreg[e] = ldg16(k + rb);
        vreg[e] = ldg16(v + rb);
      }
    };
    issue(0);
    for (int it = 0; it < ntiles; ++it) {
      // K rows of this tile -> the wave's slot (after the previous tile's V
      // reads), products S^T = K Q^T, then V rows over them
#pragma unroll
      for (int e = 0; e < RPL; ++e)
        sts16(kbs + (8 * g + ventry(e)) * KRB + vpiece(e) * 16, kreg[e]);
      f32x4 sacc[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        sacc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
        // A operand: MFMA row c16 of key-tile kt is tile entry 8(c16/4) + 4kt + c16%4
        const char *krow = kbs + (8 * (c16 >> 2) + 4 * kt + (c16 & 3)) * KRB + g * 16;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          sacc[kt] = mfma16(as_bf16x8(lds16(krow + ks * 64)), qb[ks], sacc[kt]);
      }
      // the K operand reads have returned (the products consumed them); LDS
      // operations of one wave complete in order
#pragma unroll
      for (int e = 0; e < RPL; ++e)
        sts16(vb + (8 * g + ventry(e)) * VRB + vpiece(e) * 16, vreg[e]);
      const int e0 = it * kQT;
      const int4 pa = *reinterpret_cast<const int4 *>(ipos + e0 + 8 * g);
      const int4 pb = *reinterpret_cast<const int4 *>(ipos + e0 + 8 * g + 4);
      if (it + 1 < ntiles) issue(it + 1);
      // mask: entry 8g + 4kt + r of the tile
      const int ps[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
      float x[8];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) x[4 * kt + r] = ps[4 * kt + r] >= 0 ? sacc[kt][r] : -INFINITY;
      float tmax = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
                         fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
      tmax = reduce4(tmax, [](float a, float c) { return fmaxf(a, c); }) * scale_log2;
      // The running max moves only when the tile max exceeds it by 2^kLazyQ.
      const bool grow = tmax > m_run + kLazyQ;
      const float mnew = grow ? tmax : m_run;
      const float mref = mnew == -INFINITY ? 0.f : mnew;
      if (__any(grow)) {
        const float corr = __builtin_amdgcn_exp2f(m_run - mref);   // -inf -> 0
        l_run *= corr;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 4; ++r) oacc[dt][r] *= corr;
      }
      m_run = mnew;
      float p[8], psum = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = __builtin_amdgcn_exp2f(fmaf(x[e], scale_log2, -mref));
        psum += p[e];
      }
      l_run += psum;
      bf16x8 pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = (__bf16)p[e];
      // O^T += V^T P^T: lane (g, c16) needs d = 16dt + c16 for entries
      // 8g..8g+3 (lo) and 8g+4..8g+7 (hi); the 16 lanes of group g point at
      // rows 8g + c16/4 (+4), d = 16dt + 4(c16%4).
      const char *vbase = vb + (8 * g + (c16 >> 2)) * VRB + (c16 & 3) * 8;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const char *p0 = vbase + dt * 32;
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16 *)(size_t)(p0));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16 *)(size_t)(p0 + 4 * VRB));
        bf16x8 a;
        __builtin_memcpy(&a, &lo, 8);
        __builtin_memcpy(reinterpret_cast<char *>(&a) + 8, &hi, 8);
        oacc[dt] = mfma16(a, pf, oacc[dt]);
      }
    }
  }

  const float l = reduce4(l_run, [](float a, float c) { return a + c; });
  if (!hcol) return;
  const float inv = l > 0.f ? 1.f / l : 0.f;
  uint16_t *op = o + ((size_t)t * Hq + h) * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    uint2 w;
    w.x = pack_bf16x2(oacc[dt][0] * inv, oacc[dt][1] * inv);
    w.y = pack_bf16x2(oacc[dt][2] * inv, oacc[dt][3] * inv);
    *reinterpret_cast<uint2 *>(op + dt * 16 + g * 4) = w;
  }
}

template <int D>
hipError_t launch_d(const Prob &p, const void *q, const void *k, const void *v,
                    const int32_t *idx, void *o, hipStream_t st, KvPages pages) {
  // waves are independent; at d = 256 two per workgroup keep three
  // workgroups' LDS slots on a CU
  constexpr int NW = D == 256 ? 2 : 4;
  const int n_groups = (p.nq + NW - 1) / NW;
  const size_t shift = (size_t)p.qo * p.Hq * D;   // chunk rows addressed by position
  hipLaunchKernelGGL((sparse_query_kernel<D, NW>), dim3(n_groups * p.Hkv), dim3(NW * 64), 0, st,
                     p.S, p.Hq, p.Hkv, p.G, p.b, p.k, p.idx_group_stride(), n_groups,
                     p.scale * kLog2e,
                     (const uint16_t *)q - shift, (const uint16_t *)k, (const uint16_t *)v, idx,
                     (uint16_t *)o - shift, pages, p.qo);
  return hipGetLastError();
}

}  // namespace

bool sparse_query_mfma_supported(const Prob &p) {
  return p.dtype == SP_DTYPE_BF16 && (p.d == 64 || p.d == 128 || p.d == 256) && p.G <= 16;
}

hipError_t launch_sparse_query_mfma(const Prob &p, const void *q, const void *k, const void *v,
                                    const int32_t *idx, void *o, hipStream_t st, KvPages pages) {
  if (p.d == 64) return launch_d<64>(p, q, k, v, idx, o, st, pages);
  if (p.d == 256) return launch_d<256>(p, q, k, v, idx, o, st, pages);
  return launch_d<128>(p, q, k, v, idx, o, st, pages);
}

}  // namespace sp
