// Row-wise causal GQA attention, dense or restricted to a shared support.
//
// Dense:  o[t,h] = sum_{s<=t} softmax(scale <q[t,h],k[s,g(h)]>) v[s,g(h)]   (Section 3)
// Sparse: the same softmax over U = { s in idx[t/b] : 0 <= s <= t }        (Section 3, 4.2)
//
// One wave64 per (query t, chunk of HPW query heads of one KV group). The
// wave is split into four 16-lane groups; each group walks every fourth key
// of the list and keeps its own online-softmax state, with each lane holding
// d/16 contiguous elements of the head dimension. A key row k[s,g,:] is read
// by one group as a single coalesced segment (256 B for bf16 at d=128), and
// the HPW heads of the chunk reuse it from registers. The four partial
// states are merged with cross-group shuffles at the end.
//
// This path serves every shape and dtype; it is also the per-query sparse
// path, where each query owns its support and there is nothing to share
// between queries.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

constexpr float kLazy = 8.f;

template <typename T, int D, int HPW, bool SPARSE>
__global__ __launch_bounds__(64) void attn_rowwise_kernel(
    int S, int Hq, int Hkv, int G, float scale_log2, const T *__restrict__ q,
    const T *__restrict__ k, const T *__restrict__ v, const int32_t *__restrict__ idx, int kk,
    int b, size_t gstride, T *__restrict__ o, float *__restrict__ lse, KvPages pages, int qo) {
  // q, o and lse are addressed by position: the host shifts them back by qo rows
  constexpr int EPL = D / 16;
  const int t = qo + blockIdx.x;
  const int h0 = blockIdx.y * HPW;
  const int j = h0 / G;
  const int lane = threadIdx.x;
  const int grp = lane >> 4;
  const int sub = lane & 15;

  float qr[HPW][EPL];
#pragma unroll
  for (int hh = 0; hh < HPW; ++hh) {
    load_row<EPL>(q + ((size_t)t * Hq + h0 + hh) * D + sub * EPL, qr[hh]);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qr[hh][e] *= scale_log2;
  }
  float m[HPW], l[HPW], acc[HPW][EPL];
#pragma unroll
  for (int hh = 0; hh < HPW; ++hh) {
    m[hh] = -INFINITY;
    l[hh] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[hh][e] = 0.f;
  }

  const int n = SPARSE ? kk : t + 1;
  const int32_t *ir = SPARSE ? idx + (size_t)j * gstride + (size_t)((t - qo) / b) * kk : nullptr;
  for (int base = 0; base < n; base += 4) {
    const int i = base + grp;
    int s = i;
    bool valid = i < n;
    if (SPARSE) {
      s = valid ? ir[i] : -1;
      valid = valid && s >= 0 && s <= t && s < S;
      if (valid) {
        s = pages.row(s);   // the K/V row (identity unless the cache is paged)
        valid = s >= 0;
      }
    }
    if (!valid) s = 0;
    float kf[EPL], vf[EPL];
    load_row<EPL>(k + ((size_t)s * Hkv + j) * D + sub * EPL, kf);
    load_row<EPL>(v + ((size_t)s * Hkv + j) * D + sub * EPL, vf);
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      float part = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) part = fmaf(qr[hh][e], kf[e], part);
      const float x = row16_sum(part);
      if (valid) {
        // The running max moves only when a logit exceeds it by 2^kLazy, so
        // the accumulator is rescaled rarely (probabilities stay <= 2^kLazy).
        if (x > m[hh] + kLazy) {
          const float corr = __builtin_amdgcn_exp2f(m[hh] - x);  // m = -inf gives 0
          l[hh] *= corr;
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc[hh][e] *= corr;
          m[hh] = x;
        }
        const float pr = __builtin_amdgcn_exp2f(x - m[hh]);
        l[hh] += pr;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[hh][e] = fmaf(pr, vf[e], acc[hh][e]);
      }
    }
  }

  // Merge the four groups' states (lanes sub, sub+16, sub+32, sub+48).
#pragma unroll
  for (int hh = 0; hh < HPW; ++hh) {
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float mo = __shfl_xor(m[hh], off, 64);
      const float lo = __shfl_xor(l[hh], off, 64);
      const float mn = fmaxf(m[hh], mo);
      const float c1 = (m[hh] == -INFINITY) ? 0.f : exp2f(m[hh] - mn);
      const float c2 = (mo == -INFINITY) ? 0.f : exp2f(mo - mn);
      l[hh] = l[hh] * c1 + lo * c2;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float ao = __shfl_xor(acc[hh][e], off, 64);
        acc[hh][e] = acc[hh][e] * c1 + ao * c2;
      }
      m[hh] = mn;
    }
  }
  if (grp == 0) {
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      const float inv = l[hh] > 0.f ? 1.f / l[hh] : 0.f;
      float out[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) out[e] = acc[hh][e] * inv;
      if (o) store_row<EPL>(o + ((size_t)t * Hq + h0 + hh) * D + sub * EPL, out);
      if (lse && sub == 0)
        lse[(size_t)t * Hq + h0 + hh] = l[hh] > 0.f ? (m[hh] + log2f(l[hh])) * kLn2 : -INFINITY;
    }
  }
}

template <typename T, int D, int HPW>
hipError_t launch_t(const Prob &p, const void *q, const void *k, const void *v,
                    const int32_t *idx, void *o, float *lse, hipStream_t st, KvPages pages) {
  dim3 grid(p.nq, p.Hq / HPW);
  const float sl2 = p.scale * kLog2e;
  // chunk rows are addressed by position
  const size_t shift = (size_t)p.qo * p.Hq;
  const T *qs = (const T *)q - shift * D;
  T *os = o ? (T *)o - shift * D : nullptr;
  float *ls = lse ? lse - shift : nullptr;
  if (idx)
    hipLaunchKernelGGL((attn_rowwise_kernel<T, D, HPW, true>), grid, dim3(64), 0, st, p.S,
                       p.Hq, p.Hkv, p.G, sl2, qs, (const T *)k, (const T *)v, idx, p.k, p.b,
                       p.idx_group_stride(), os, ls, pages, p.qo);
  else
    hipLaunchKernelGGL((attn_rowwise_kernel<T, D, HPW, false>), grid, dim3(64), 0, st, p.S,
                       p.Hq, p.Hkv, p.G, sl2, qs, (const T *)k, (const T *)v, nullptr, 0, 1,
                       (size_t)0, os, ls, KvPages(), p.qo);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_d(const Prob &p, const void *q, const void *k, const void *v,
                    const int32_t *idx, void *o, float *lse, hipStream_t st, KvPages pages) {
  if (p.G % 4 == 0) return launch_t<T, D, 4>(p, q, k, v, idx, o, lse, st, pages);
  if (p.G % 2 == 0) return launch_t<T, D, 2>(p, q, k, v, idx, o, lse, st, pages);
  return launch_t<T, D, 1>(p, q, k, v, idx, o, lse, st, pages);
}

}  // namespace

hipError_t launch_attn_rowwise(const Prob &p, const void *q, const void *k, const void *v,
                               const int32_t *idx, void *o, float *lse, hipStream_t st,
                               KvPages pages) {
  if (p.dtype == SP_DTYPE_BF16) {
    if (p.d == 64) return launch_d<bf16, 64>(p, q, k, v, idx, o, lse, st, pages);
    if (p.d == 128) return launch_d<bf16, 128>(p, q, k, v, idx, o, lse, st, pages);
    return launch_d<bf16, 256>(p, q, k, v, idx, o, lse, st, pages);
  }
  if (p.d == 64) return launch_d<float, 64>(p, q, k, v, idx, o, lse, st, pages);
  if (p.d == 128) return launch_d<float, 128>(p, q, k, v, idx, o, lse, st, pages);
  return launch_d<float, 256>(p, q, k, v, idx, o, lse, st, pages);
}

}  // namespace sp
