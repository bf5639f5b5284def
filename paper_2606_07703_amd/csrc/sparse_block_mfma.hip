// Selection-block-shared sparse GQA attention on bf16 MFMA (Section 3
// restricted attention; Section 4.2 per-query causal mask; Algorithm 1, restricted recomputation
// and Algorithm 2, selection and sparse GQA prefill: one support per block, replicated over KV heads).
//
// One workgroup per (selection block r, KV head j, chunk of up to 256 query
// rows; 128 at head_dim 256). A query row is a (query t, head h) pair with g(h) = j; there are
// b*G of them per (r, j), ordered query-major. The support idx[r] is walked
// in tiles of 64 entries: the workgroup gathers the 64 selected K rows and
// V rows of head j into LDS once, and every wave reuses them for its 32 query
// rows. Each selected row therefore leaves HBM once per (block, KV head),
// not once per query. Every query applies its own causal mask to the shared
// support; sentinels and out-of-range entries contribute nothing, and the
// order of a support row does not matter.
//
// Workgroups are numbered with the KV head fastest: consecutive workgroups go
// to different XCDs, so with Hkv = 8 each XCD's L2 holds the K/V rows of one
// head only. Blocks are dispatched from the last to the first.
#include <limits.h>

#include "attn_tile.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

// Support entries cached in LDS (a multiple of the tile): 4096, except for
// the paged cache at head_dim 256, whose K/V tiles and second row table leave
// room for 2048.
constexpr int max_support(int D, bool paged) { return D == 256 && paged ? 2048 : 4096; }
constexpr int kMaxTiles = 4096 / kAttnKT;

// The usable support entries in LDS: positions (pos), K/V rows (row: the
// position, or its paged-cache row), and which tiles need the causal mask
// for this wave (a bit per tile, kept in registers so the softmax phase reads
// no LDS).
struct SupportKeys {
  static constexpr bool kLookup = true;   // rows are read from the LDS support cache
  int ntiles;
  const int *pos;
  const int *rows;
  uint64_t mask_bits;   // bit t: tile t holds a position past the wave's first query or padding
  __device__ __forceinline__ int row(int tile, int e) const { return rows[tile * kAttnKT + e]; }
  __device__ __forceinline__ bool needs_mask(int tile, int) const {
    return (mask_bits >> tile) & 1;
  }
  __device__ __forceinline__ int4 pos4(int tile, int e0) const {
    // read past the direct-to-LDS tile loads in flight (they never write pos)
    const uint32_t a = (uint32_t)(size_t)(const __attribute__((address_space(3))) int *)pos;
    return lds_read_i32x4(a + (tile * kAttnKT + e0) * 4);
  }
};

template <int D, int NW, bool PAGED>
__global__ __launch_bounds__(NW * 64) SP_ATTN_OCCUPANCY(D) void sparse_block_kernel(
    int S, int Hq, int Hkv, int G, int b, int kk, int nchunks, size_t gstride, float scale_log2,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, const int32_t *__restrict__ idx,
    uint16_t *__restrict__ o, KvPages pages, int qo) {
  // q and o are addressed by position: the host shifts them back by qo rows
  using L = AttnLayout<D>;
  constexpr int NT = NW * 64;
  constexpr int kMaxSupport = max_support(D, PAGED);
  __shared__ __align__(16) char lds[L::lds_bytes(true, NW)];
  __shared__ int red_cnt[2][NW];
  __shared__ __align__(16) int ir[kMaxSupport];
  // paged cache: the K/V row of each support entry (ir keeps the position)
  __shared__ __align__(16) int irp[PAGED ? kMaxSupport : 1];
  __shared__ int tkey[kMaxTiles];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, n = lane & 31;
  // the row chunks of one (block, KV head) are Hkv workgroups apart: the same
  // XCD, dispatched together, so the second gathers its rows from that L2
  const int j = (int)blockIdx.x % Hkv;
  const int rest = (int)blockIdx.x / Hkv;
  const int chunk = rest % nchunks;
  // blocks run last to first: the supports of the first blocks are cut short
  // by the causal limit, and those small workgroups then fill the end of the
  // launch instead of its start
  const int nblocks = (int)gridDim.x / (Hkv * nchunks);
  const int r = nblocks - 1 - rest / nchunks;   // counts blocks from the chunk start
  const int t0 = qo + r * b;
  const int t1 = min(t0 + b, S) - 1;
  const int nrows = (t1 - t0 + 1) * G;
  const int row0 = chunk * (NW * kAttnQPW) + wave * kAttnQPW;

  QRow<D> qr;
  load_q_row<D>(q, Hq, G, j, t0, row0 + n, nrows, h, qr);

  // Cache the usable entries of the support row (positions 0 <= s <= t1,
  // on a page inside the cache), compacted to the front in their original
  // order; sentinels and later positions contribute to no query of the block.
  // Positions in a row are distinct, so at most t1 + 1 entries remain. Each
  // thread takes kEPT consecutive entries per pass (one pass when kk <= 8 NT):
  // all its loads are in flight together, a wave scan of the per-thread
  // counts (bit-sliced ballots: no LDS round trips) gives the write offsets,
  // and one barrier per pass publishes the wave totals (double-buffered, so
  // passes need no second barrier). Each tile's largest position (tkey; the
  // tile needs the causal mask for queries below it) is raised with LDS
  // atomics as the entries are written.
  constexpr int kEPT = 8;
  for (int i = tid; i < kMaxTiles; i += NT) tkey[i] = INT_MIN;
  int nv = 0;
  for (int c0 = 0, pass = 0; c0 < kk; c0 += NT * kEPT, ++pass) {
    const int cb = c0 + tid * kEPT;
    const int32_t *row = idx + (size_t)j * gstride + (size_t)r * kk;
    int sv[kEPT], pr[kEPT];
    if (cb + kEPT <= kk && (((uintptr_t)(row + cb)) & 15) == 0) {
      const int4 a = *reinterpret_cast<const int4 *>(row + cb);
      const int4 c = *reinterpret_cast<const int4 *>(row + cb + 4);
      sv[0] = a.x; sv[1] = a.y; sv[2] = a.z; sv[3] = a.w;
      sv[4] = c.x; sv[5] = c.y; sv[6] = c.z; sv[7] = c.w;
    } else {
#pragma unroll
      for (int e = 0; e < kEPT; ++e) sv[e] = cb + e < kk ? row[cb + e] : -1;
    }
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < kEPT; ++e) {
      pr[e] = sv[e];
      if constexpr (PAGED) pr[e] = (sv[e] >= 0 && sv[e] <= t1) ? pages.row(sv[e]) : -1;
      cnt += (sv[e] >= 0 && sv[e] <= t1 && pr[e] >= 0);
    }
    // exclusive prefix of cnt (0 .. 8, four bits) over the wave, and its total
    int excl = 0, wtot = 0;
#pragma unroll
    for (int bit = 0; bit < 4; ++bit) {
      const uint64_t m = __ballot((cnt >> bit) & 1);
      const uint32_t below = __builtin_amdgcn_mbcnt_hi(
          (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      excl += (int)below << bit;
      wtot += __popcll(m) << bit;
    }
    if (lane == 0) red_cnt[pass & 1][wave] = wtot;
    __syncthreads();
    int pos = nv + excl;
    for (int w = 0; w < NW; ++w) {
      const int tw = red_cnt[pass & 1][w];
      if (w < wave) pos += tw;
      nv += tw;
    }
#pragma unroll
    for (int e = 0; e < kEPT; ++e)
      if (sv[e] >= 0 && sv[e] <= t1 && pr[e] >= 0) {
        ir[pos] = sv[e];
        if constexpr (PAGED) irp[pos] = pr[e];
        atomicMax(&tkey[pos / kAttnKT], sv[e]);
        ++pos;
      }
  }
  const int ntiles = min((t1 + kAttnKT) / kAttnKT, (nv + kAttnKT - 1) / kAttnKT);
  for (int c = nv + tid; c < ntiles * kAttnKT; c += NT) {
    ir[c] = -1;
    if constexpr (PAGED) irp[c] = -1;
  }
  // a tile that holds padding is masked for every query
  if (tid == 0 && ntiles * kAttnKT > nv) atomicMax(&tkey[ntiles - 1], INT_MAX);
  __syncthreads();

  AttnState<D> st;
  const int kv_rows = PAGED ? pages.num_pages * pages.page_size : S;
  const int wave_tmin = t0 + min(row0, nrows - 1) / G;
  // bit t: tile t needs the causal mask for this wave (ntiles <= 64)
  const uint64_t mask_bits = __ballot(lane < ntiles && tkey[lane < ntiles ? lane : 0] > wave_tmin);
  const SupportKeys keys{ntiles, ir, PAGED ? irp : ir, mask_bits};
  AttnPipe<D, NW, true, SupportKeys> pipe(lds, keys, k, v, kv_rows, Hkv, j, scale_log2, wave_tmin,
                                          qr, st);
  pipe.run();
  attn_finish<D>(st, qr, Hq, o, nullptr, h, lds);
}

template <int D, bool PAGED>
hipError_t launch_d(const Prob &p, const void *q, const void *k, const void *v,
                    const int32_t *idx, void *o, hipStream_t st, KvPages pages) {
  const int rows = p.b * p.G;
  int nw = (rows + kAttnQPW - 1) / kAttnQPW;
  nw = nw <= 1 ? 1 : nw <= 2 ? 2 : nw <= 4 ? 4 : attn_max_waves<D>();
  // at head_dim 256 a wave's share of the tile loads grows with fewer waves
  // (69 chunks for one) and its row registers no longer fit: always four
  if (D == 256) nw = 4;
  const int chunks = (rows + nw * kAttnQPW - 1) / (nw * kAttnQPW);
  dim3 grid(p.R * p.Hkv * chunks);
  const float sl2 = p.scale * kLog2e;
  const size_t shift = (size_t)p.qo * p.Hq * D;   // chunk rows addressed by position
  const uint16_t *qs = (const uint16_t *)q - shift;
  uint16_t *os = (uint16_t *)o - shift;
#define SP_SB(NW)                                                                            \
  hipLaunchKernelGGL((sparse_block_kernel<D, NW, PAGED>), grid, dim3(NW * 64), 0, st, p.S,  \
                     p.Hq, p.Hkv, p.G, p.b, p.k, chunks, p.idx_group_stride(), sl2,           \
                     qs, (const uint16_t *)k, (const uint16_t *)v, idx, os, pages, p.qo)
  if constexpr (D == 256) {
    SP_SB(4);
  } else {
    switch (nw) {
      case 1: SP_SB(1); break;
      case 2: SP_SB(2); break;
      case 4: SP_SB(4); break;
      default: SP_SB(8); break;
    }
  }
#undef SP_SB
  return hipGetLastError();
}

}  // namespace

bool sparse_block_mfma_supported(const Prob &p, bool paged) {
  return p.dtype == SP_DTYPE_BF16 && (p.d == 64 || p.d == 128 || p.d == 256) && p.b >= 16 &&
         p.k <= max_support(p.d, paged);
}

hipError_t launch_sparse_block_mfma(const Prob &p, const void *q, const void *k, const void *v,
                                    const int32_t *idx, void *o, hipStream_t st, KvPages pages) {
  if (pages.table) {
    if (p.d == 64) return launch_d<64, true>(p, q, k, v, idx, o, st, pages);
    if (p.d == 256) return launch_d<256, true>(p, q, k, v, idx, o, st, pages);
    return launch_d<128, true>(p, q, k, v, idx, o, st, pages);
  }
  if (p.d == 64) return launch_d<64, false>(p, q, k, v, idx, o, st, pages);
  if (p.d == 256) return launch_d<256, false>(p, q, k, v, idx, o, st, pages);
  return launch_d<128, false>(p, q, k, v, idx, o, st, pages);
}

}  // namespace sp
