// Dense causal GQA attention on bf16 MFMA (Section 3, first equation;
// Algorithm 1, dense scores and normalisers): a flash-attention forward that also returns the
// softmax normaliser lse[t,h] = log sum_{s<=t} exp(scale <q[t,h], k[s,g(h)]>).
//
// One workgroup per (tile of 256/G queries, KV head j; 128/G at head_dim
// 256): its 256 (128) query rows are every (query, head) pair of the tile
// with g(h) = j, so each K/V tile staged in LDS serves all G heads of the
// group. Key tiles below a wave's first
// query need no mask; only tiles reaching the diagonal apply s <= t.
// Workgroups are numbered with the KV head fastest, so consecutive
// workgroups (which the dispatcher spreads over the XCDs) keep one head per
// XCD when Hkv is 8, and query tiles are scheduled longest first (the causal
// work of tile i grows with i), which shortens the tail of the launch.
//
// With o == nullptr only the normalisers are produced: the P V product and
// the V traffic are skipped (the oracle's first pass needs nothing else).
#include "attn_tile.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

struct DenseKeys {
  static constexpr bool kLookup = false;   // rows are arithmetic
  int ntiles, S;
  __device__ __forceinline__ int row(int tile, int e) const { return tile * kAttnKT + e; }
  __device__ __forceinline__ bool needs_mask(int tile, int wave_tmin) const {
    return tile * kAttnKT + kAttnKT - 1 > wave_tmin;
  }
  __device__ __forceinline__ int4 pos4(int tile, int e0) const {
    const int s = tile * kAttnKT + e0;
    return int4{s, s + 1, s + 2, s + 3};
  }
};

template <int D, bool WANT_O>
__global__ __launch_bounds__(attn_max_waves<D>() * 64) SP_ATTN_OCCUPANCY(D) void dense_fwd_kernel(
    int S, int Hq, int Hkv, int G, int TQ, int nqt, float scale_log2,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, uint16_t *__restrict__ o, float *__restrict__ lse) {
  using L = AttnLayout<D>;
  constexpr int kNW = attn_max_waves<D>();
  __shared__ __align__(16) char lds[L::lds_bytes(WANT_O, kNW)];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, n = lane & 31;
  const int j = (int)blockIdx.x % Hkv;
  const int qi = nqt - 1 - (int)blockIdx.x / Hkv;
  const int t0 = qi * TQ;
  const int tl = min(t0 + TQ, S) - 1;
  const int nrows = (tl - t0 + 1) * G;
  const int row0 = wave * kAttnQPW;

  QRow<D> qr;
  load_q_row<D>(q, Hq, G, j, t0, row0 + n, nrows, h, qr);
  AttnState<D> st;
  const DenseKeys keys{tl / kAttnKT + 1, S};
  const int wave_tmin = t0 + min(row0, nrows - 1) / G;
  AttnPipe<D, kNW, WANT_O, DenseKeys> pipe(lds, keys, k, v, S, Hkv, j, scale_log2, wave_tmin, qr,
                                           st);
  pipe.run();
  attn_finish<D>(st, qr, Hq, WANT_O ? o : nullptr, lse, h, lds);
}

template <int D>
hipError_t launch_d(const Prob &p, const void *q, const void *k, const void *v, void *o,
                    float *lse, hipStream_t st) {
  constexpr int kNW = attn_max_waves<D>();
  const int TQ = (kNW * kAttnQPW) / p.G;
  const int nqt = (p.S + TQ - 1) / TQ;
  dim3 grid(nqt * p.Hkv);
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
  return p.dtype == SP_DTYPE_BF16 && (p.d == 64 || p.d == 128 || p.d == 256) &&
         p.G <= (p.d == 256 ? attn_max_waves<256>() : attn_max_waves<128>()) * kAttnQPW;
}

hipError_t launch_dense_mfma(const Prob &p, const void *q, const void *k, const void *v,
                             void *o, float *lse, hipStream_t st) {
  if (p.d == 64) return launch_d<64>(p, q, k, v, o, lse, st);
  if (p.d == 256) return launch_d<256>(p, q, k, v, o, lse, st);
  return launch_d<128>(p, q, k, v, o, lse, st);
}

}  // namespace sp
