// Selection-block-shared sparse GQA attention on bf16 MFMA (Section 3
// restricted attention; Section 4.2 per-query causal mask; Algorithm 1 step 5
// and Algorithm 2 step 5: one support per block, replicated over KV heads).
//
// One workgroup per (selection block r, KV head j, chunk of up to 256 query
// rows). A query row is a (query t, head h) pair with g(h) = j; there are
// b*G of them per (r, j), ordered query-major. The support idx[r] is walked
// in tiles of 64 entries: the workgroup gathers the 64 selected K rows and
// V rows of head j into LDS once, and every wave reuses them for its 32 query
// rows. Each selected row therefore leaves HBM once per (block, KV head),
// not once per query. Every query applies its own causal mask to the shared
// support; sentinels and out-of-range entries contribute nothing, and the
// order of a support row does not matter.
#include "attn_tile.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

constexpr int kMaxSupport = 4096;   // support row cached in LDS

template <int D, int NW, bool PAGED>
__global__ __launch_bounds__(NW * 64) void sparse_block_kernel(
    int S, int Hq, int Hkv, int G, int b, int kk, size_t gstride, float scale_log2,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, const int32_t *__restrict__ idx,
    uint16_t *__restrict__ o, KvPages pages, int qo) {
  // q and o are addressed by position: the host shifts them back by qo rows
  using L = AttnLayout<D>;
  constexpr int NT = NW * 64;
  __shared__ __align__(16) char lds[2][L::BUF];
  __shared__ int red_last[NW];
  __shared__ int ir[kMaxSupport];
  // paged cache: the K/V row of each support entry (ir keeps the position)
  __shared__ int irp[PAGED ? kMaxSupport : 1];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  const int r = blockIdx.x, j = blockIdx.y;   // r counts blocks from the chunk start
  const int t0 = qo + r * b;
  const int t1 = min(t0 + b, S) - 1;
  const int nrows = (t1 - t0 + 1) * G;
  const int row0 = blockIdx.z * (NW * kAttnQPW) + wave * kAttnQPW;

  // Cache the support row; tiles end after the last entry any query of the
  // block can use (any order).
  int last = -1;
  for (int c = tid; c < kk; c += NT) {
    int s = idx[(size_t)j * gstride + (size_t)r * kk + c];
    if constexpr (PAGED) {
      const int row = (s >= 0 && s < S) ? pages.row(s) : -1;
      if (row < 0) s = -1;   // sentinel, or a page outside the cache: skipped
      irp[c] = row;
    }
    ir[c] = s;
    if (s >= 0 && s <= t1) last = c;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) last = max(last, __shfl_xor(last, off, 64));
  if (lane == 0) red_last[wave] = last;
  __syncthreads();
  last = -1;
#pragma unroll
  for (int w = 0; w < NW; ++w) last = max(last, red_last[w]);
  const int ntiles = (last + kAttnKT) / kAttnKT;

  bf16x8 bq[2][L::KS];
  int qt[2], qh[2];
  bool qvalid[2];
  load_q_rows<D>(q, Hq, G, j, t0, row0, nrows, g, c16, bq, qt, qh, qvalid);

  AttnState<D> st;
  st.init();
  KVStage<D, NT, true> stage;
  auto pos_of = [&](int c0) {
    return [=](int e) { return c0 + e < kk ? ir[c0 + e] : -1; };
  };
  auto row_of = [&](int c0) {
    return [=](int e) { return c0 + e < kk ? (PAGED ? irp[c0 + e] : ir[c0 + e]) : -1; };
  };
  const int kv_rows = PAGED ? pages.num_pages * pages.page_size : S;
  if (ntiles > 0) {
    stage.load_rows(k, v, kv_rows, Hkv, j, tid, pos_of(0), row_of(0));
    stage.store(lds[0], tid);
  }
  drain_memory();
  __syncthreads();
  const bool live = row0 < nrows;
  const int wave_tmin = t0 + row0 / G;
  for (int it = 0; it < ntiles; ++it) {
    const bool more = it + 1 < ntiles;
    if (more)
      stage.load_rows(k, v, kv_rows, Hkv, j, tid, pos_of((it + 1) * kAttnKT),
                      row_of((it + 1) * kAttnKT));
    if (live) attn_tile<D, true, true>(lds[it & 1], bq, qt, scale_log2, wave_tmin, st, g, c16);
    if (more) stage.store(lds[(it + 1) & 1], tid);
    __syncthreads();
  }
  if (live) attn_finish<D>(st, qt, qh, qvalid, Hq, o, nullptr, g);
}

template <int D, bool PAGED>
hipError_t launch_d(const Prob &p, const void *q, const void *k, const void *v,
                    const int32_t *idx, void *o, hipStream_t st, KvPages pages) {
  const int rows = p.b * p.G;
  int nw = (rows + kAttnQPW - 1) / kAttnQPW;
  nw = nw <= 1 ? 1 : nw <= 2 ? 2 : nw <= 4 ? 4 : 8;
  const int chunks = (rows + nw * kAttnQPW - 1) / (nw * kAttnQPW);
  dim3 grid(p.R, p.Hkv, chunks);
  const float sl2 = p.scale * kLog2e;
  const size_t shift = (size_t)p.qo * p.Hq * D;   // chunk rows addressed by position
  const uint16_t *qs = (const uint16_t *)q - shift;
  uint16_t *os = (uint16_t *)o - shift;
#define SP_SB(NW)                                                                            \
  hipLaunchKernelGGL((sparse_block_kernel<D, NW, PAGED>), grid, dim3(NW * 64), 0, st, p.S,  \
                     p.Hq, p.Hkv, p.G, p.b, p.k, p.idx_group_stride(), sl2,                   \
                     qs, (const uint16_t *)k, (const uint16_t *)v, idx, os, pages, p.qo)
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
  return p.dtype == SP_DTYPE_BF16 && (p.d == 64 || p.d == 128) && p.b >= 16 &&
         p.k <= kMaxSupport;
}

hipError_t launch_sparse_block_mfma(const Prob &p, const void *q, const void *k, const void *v,
                                    const int32_t *idx, void *o, hipStream_t st, KvPages pages) {
  if (pages.table) {
    if (p.d == 64) return launch_d<64, true>(p, q, k, v, idx, o, st, pages);
    return launch_d<128, true>(p, q, k, v, idx, o, st, pages);
  }
  if (p.d == 64) return launch_d<64, false>(p, q, k, v, idx, o, st, pages);
  return launch_d<128, false>(p, q, k, v, idx, o, st, pages);
}

}  // namespace sp
