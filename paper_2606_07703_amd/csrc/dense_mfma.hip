// Dense causal GQA attention on bf16 MFMA (Section 3, first equation;
// Algorithm 1 step 2): a flash-attention forward that also returns the
// softmax normaliser lse[t,h] = log sum_{s<=t} exp(scale <q[t,h], k[s,g(h)]>).
//
// One workgroup per (tile of 256/G queries, KV head j): its 256 query rows are
// every (query, head) pair of the tile with g(h) = j, so each K/V tile staged
// in LDS serves all G heads of the group. Key tiles below a wave's first
// query need no mask; only tiles reaching the diagonal apply s <= t.
// Query tiles are scheduled longest first (the causal work of tile i grows
// with i), which shortens the tail of the launch.
//
// With o == nullptr only the normalisers are produced: the P V product and
// the V traffic are skipped (the oracle's first pass needs nothing else).
#include "attn_tile.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

constexpr int kNW = 8;

template <int D, bool WANT_O>
__global__ __launch_bounds__(kNW * 64) void dense_fwd_kernel(
    int S, int Hq, int Hkv, int G, int TQ, int nqt, float scale_log2,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, uint16_t *__restrict__ o, float *__restrict__ lse) {
  using L = AttnLayout<D>;
  constexpr int NT = kNW * 64;
  __shared__ __align__(16) char lds[2][L::BUF];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  const int qi = nqt - 1 - (int)blockIdx.x;
  const int j = blockIdx.y;
  const int t0 = qi * TQ;
  const int tl = min(t0 + TQ, S) - 1;
  const int nrows = (tl - t0 + 1) * G;
  const int row0 = wave * kAttnQPW;

  bf16x8 bq[2][L::KS];
  int qt[2], qh[2];
  bool qvalid[2];
  load_q_rows<D>(q, Hq, G, j, t0, row0, nrows, g, c16, bq, qt, qh, qvalid);

  AttnState<D> st;
  st.init();
  KVStage<D, NT, WANT_O> stage;
  const int ntiles = tl / kAttnKT + 1;
  auto pos_of = [&](int base) {
    return [=](int e) { return base + e < S ? base + e : -1; };
  };
  stage.load(k, v, S, Hkv, j, tid, pos_of(0));
  stage.store(lds[0], tid);
  drain_memory();
  __syncthreads();
  const bool live = row0 < nrows;
  const int wave_tmin = t0 + row0 / G;
  for (int it = 0; it < ntiles; ++it) {
    const bool more = it + 1 < ntiles;
    if (more) stage.load(k, v, S, Hkv, j, tid, pos_of((it + 1) * kAttnKT));
    if (live) attn_tile<D, WANT_O>(lds[it & 1], bq, qt, scale_log2, wave_tmin, st, g, c16);
    if (more) stage.store(lds[(it + 1) & 1], tid);
    __syncthreads();
  }
  if (live) attn_finish<D>(st, qt, qh, qvalid, Hq, WANT_O ? o : nullptr, lse, g);
}

template <int D>
hipError_t launch_d(const Prob &p, const void *q, const void *k, const void *v, void *o,
                    float *lse, hipStream_t st) {
  const int TQ = (kNW * kAttnQPW) / p.G;
  const int nqt = (p.S + TQ - 1) / TQ;
  dim3 grid(nqt, p.Hkv);
  const float sl2 = p.scale * kLog2e;
  if (o)
    hipLaunchKernelGGL((dense_fwd_kernel<D, true>), grid, dim3(kNW * 64), 0, st, p.S, p.Hq,
                       p.Hkv, p.G, TQ, nqt, sl2, (const uint16_t *)q, (const uint16_t *)k,
                       (const uint16_t *)v, (uint16_t *)o, lse);
  else
    hipLaunchKernelGGL((dense_fwd_kernel<D, false>), grid, dim3(kNW * 64), 0, st, p.S, p.Hq,
                       p.Hkv, p.G, TQ, nqt, sl2, (const uint16_t *)q, (const uint16_t *)k,
                       (const uint16_t *)v, nullptr, lse);
  return hipGetLastError();
}

}  // namespace

bool dense_mfma_supported(const Prob &p) {
  return p.dtype == SP_DTYPE_BF16 && (p.d == 64 || p.d == 128) && p.G <= kNW * kAttnQPW;
}

hipError_t launch_dense_mfma(const Prob &p, const void *q, const void *k, const void *v,
                             void *o, float *lse, hipStream_t st) {
  if (p.d == 64) return launch_d<64>(p, q, k, v, o, lse, st);
  return launch_d<128>(p, q, k, v, o, lse, st);
}

}  // namespace sp
