// Fused per-query indexer scoring and top-k selection (Section 6.3 score;
// Section 6.4 and Algorithm 2, scoring, selection and sparse prefill with b_sel = 1; Section 4.1 TopK):
// the top-k of z[t, s] = ReLU(scale <q_idx[t], k_idx[s]>) over s <= t, for
// every query t, without ever storing the S x S score matrix.
//
// Selection is the same as sp_topk_select on the stored scores: for a row
// with L = t+1 > k positions, the Wf = min(W, k) most recent positions are
// forced and k' = k - Wf are taken from [0, L - Wf) in the order (score
// descending, position ascending); output rows are ascending, -1 padded.
//
// Scores are recomputed on the matrix cores in every pass of a radix select
// over the order-preserving uint32 keys of the fp32 scores, 8 bits per pass:
//   * hist pass p (p = 0..3): work items are (64-query group, 4096-key
//     chunk) pairs; each item histograms the keys of its rows that still
//     match the row's prefix, in LDS with 16-bit counters, and writes its
//     partial histograms to the workspace;
//   * resolve pass p: one wave per row sums the partials, picks the digit
//     holding the k'-th largest key, extends the prefix, and records per
//     chunk how many keys fell above it (and, last, how many sit exactly on
//     it). A row whose chosen bin holds exactly the keys still needed is
//     settled: every key with that prefix is taken and later passes skip it.
//   * emit: items recompute their scores once more and write the chosen
//     positions in position order; each chunk's starting offset comes from
//     the per-chunk counts, so the rows come out ascending with no sort.
// The score of a (query, key) pair is bit-identical in every pass (the same
// MFMA chain and epilogue), which keeps the passes consistent.
#include <math.h>

#include <atomic>

#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"

namespace sp {
namespace {

constexpr int kFQ = 64;          // queries per work item (4 waves x 16)
constexpr int kFW = 4;           // waves per work item
constexpr int kFC = 4096;        // keys per chunk
constexpr int kFKT = 64;         // keys per LDS tile
constexpr int kFBins = 256;      // 8-bit digits
constexpr int kFMaxChunks = 16;  // S <= 65535
constexpr uint32_t kFZero = 0x80000000u;   // float_key(+0.0f)

enum : uint32_t { kRowSettled = 1u, kRowDirect = 2u };

struct RowState {
  uint32_t prefix;      // fixed high bits of the threshold key
  uint32_t pmask;       // which bits are fixed
  uint32_t remaining;   // keys still to take among those matching prefix
  uint32_t flags;
};

// Workspace layout (all counts per row are over the row's candidates).
struct FzWs {
  RowState *state;     // [S]
  uint16_t *hist;      // [chunks][S][kFBins] partial histograms of a pass
  uint32_t *gt;        // [S][kFMaxChunks] keys above the threshold prefix, per chunk
  uint32_t *eq;        // [S][kFMaxChunks] keys matching the final prefix, per chunk
};

int fz_chunks(int S) { return (S + kFC - 1) / kFC; }

size_t fz_bytes(int S) {
  auto al = [](size_t b) { return (b + 255) & ~size_t(255); };
  return al(sizeof(RowState) * S) + al(sizeof(uint16_t) * (size_t)fz_chunks(S) * S * kFBins) +
         2 * al(sizeof(uint32_t) * (size_t)S * kFMaxChunks);
}

FzWs fz_carve(void *ws, int S) {
  auto al = [](size_t b) { return (b + 255) & ~size_t(255); };
  char *p = static_cast<char *>(ws);
  FzWs w;
  w.state = reinterpret_cast<RowState *>(p);
  p += al(sizeof(RowState) * S);
  w.hist = reinterpret_cast<uint16_t *>(p);
  p += al(sizeof(uint16_t) * (size_t)fz_chunks(S) * S * kFBins);
  w.gt = reinterpret_cast<uint32_t *>(p);
  p += al(sizeof(uint32_t) * (size_t)S * kFMaxChunks);
  w.eq = reinterpret_cast<uint32_t *>(p);
  return w;
}

struct FzProb {
  int S, k, Wf, relu;
  float scale;
};

__host__ __device__ __forceinline__ int fz_nc(const FzProb &f, int t) { return t + 1 - f.Wf; }
__host__ __device__ __forceinline__ int fz_ngroups(int S) { return (S + kFQ - 1) / kFQ; }
// candidates of the group's last row (the largest in the group)
__host__ __device__ __forceinline__ int fz_group_nc(const FzProb &f, int grp) {
  return fz_nc(f, min((grp + 1) * kFQ, f.S) - 1);
}
// chunks holding candidates of some non-direct row of the group
__host__ __device__ __forceinline__ int fz_group_chunks(const FzProb &f, int grp) {
  const int t_last = min((grp + 1) * kFQ, f.S) - 1;
  if (t_last + 1 <= f.k) return 0;   // every row of the group is direct
  return (fz_group_nc(f, grp) + kFC - 1) / kFC;
}

// Item i -> (group, chunk), items ordered by chunk then group.
__device__ __forceinline__ void fz_decode(const FzProb &f, int i, int &grp, int &chunk) {
  const int ng = fz_ngroups(f.S);
  for (int c = 0;; ++c) {
    // groups needing chunk c are a suffix [g0, ng) (fz_group_chunks grows with grp)
    int g0 = ng;
    int lo = 0, hi = ng;
    while (lo < hi) {
      const int mid = (lo + hi) / 2;
      if (fz_group_chunks(f, mid) > c) hi = mid; else lo = mid + 1;
    }
    g0 = lo;
    const int cnt = ng - g0;
    if (i < cnt) {
      grp = g0 + i;
      chunk = c;
      return;
    }
    i -= cnt;
  }
}

int fz_items(const FzProb &f) {
  int n = 0;
  for (int g = 0; g < fz_ngroups(f.S); ++g) n += fz_group_chunks(f, g);
  return n;
}

template <int DI>
struct FzTile {
  static constexpr int RB = DI * 2 + 16;      // padded LDS row bytes
  static constexpr int BYTES = kFKT * RB;
  static constexpr int KS = DI / 32;
  static constexpr int PIECES = kFKT * DI / 8;
  static constexpr int PER = (PIECES + kFW * 64 - 1) / (kFW * 64);
};

// Register-staged copy of one 64-key tile (rows past S-1 repeat S-1).
template <int DI>
struct FzStage {
  uint4 reg[FzTile<DI>::PER];
  __device__ __forceinline__ void load(const uint16_t *__restrict__ ki, int S, int k0, int tid) {
#pragma unroll
    for (int i = 0; i < FzTile<DI>::PER; ++i) {
      const int c = tid + i * kFW * 64;
      if (c < FzTile<DI>::PIECES) {
        const int row = c / (DI / 8), col = c % (DI / 8);
        reg[i] = ldg16(ki + (size_t)min(k0 + row, S - 1) * DI + col * 8);
      }
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < FzTile<DI>::PER; ++i) {
      const int c = tid + i * kFW * 64;
      if (c < FzTile<DI>::PIECES)
        sts16(lds + (c / (DI / 8)) * FzTile<DI>::RB + (c % (DI / 8)) * 16, reg[i]);
    }
  }
};

// Walk ntiles 64-key tiles from k_begin through two LDS buffers, with tile
// it+2 already in flight (registers) while tile it is used: body(it, tile).
// Contains barriers: every thread of the workgroup calls it.
template <int DI, class Body>
__device__ __forceinline__ void fz_walk(const uint16_t *__restrict__ ki, int S, int k_begin,
                                        int ntiles, int tid, char (*lds)[FzTile<DI>::BYTES],
                                        Body body) {
  FzStage<DI> sa, sb;
  sa.load(ki, S, k_begin, tid);
  if (ntiles > 1) sb.load(ki, S, k_begin + kFKT, tid);
  sa.store(lds[0], tid);
  __syncthreads();
  for (int it = 0; it < ntiles; it += 2) {
    if (it + 2 < ntiles) sa.load(ki, S, k_begin + (it + 2) * kFKT, tid);
    body(it, lds[0]);
    if (it + 1 < ntiles) sb.store(lds[1], tid);
    __syncthreads();
    if (it + 1 < ntiles) {
      if (it + 3 < ntiles) sb.load(ki, S, k_begin + (it + 3) * kFKT, tid);
      body(it + 1, lds[1]);
      if (it + 2 < ntiles) sa.store(lds[0], tid);
      __syncthreads();
    }
  }
}

// Keys of a 16-key row tile for this lane's query: sacc = S^T with lane
// (g, c16) holding keys 16kt + 4g + r of query column c16. The same code
// runs in every pass, so a pair's key never changes between passes.
template <int DI>
__device__ __forceinline__ void fz_keys(const char *tile, int kt, const bf16x8 (&qb)[DI / 32],
                                        const FzProb &f, int g, int c16, uint32_t (&key)[4]) {
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < DI / 32; ++ks)
    acc = mfma16(as_bf16x8(lds16(tile + (kt * 16 + c16) * FzTile<DI>::RB + ks * 64 + g * 16)),
                 qb[ks], acc);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float z = acc[r] * f.scale;
    if (f.relu) z = fmaxf(z, 0.f);
    key[r] = float_key(z);
  }
}

template <int DI>
__device__ __forceinline__ void fz_load_q(const uint16_t *__restrict__ qi, int S, int t,
                                          int g, bf16x8 (&qb)[DI / 32]) {
  const int tq = min(t, S - 1);
#pragma unroll
  for (int ks = 0; ks < DI / 32; ++ks)
    qb[ks] = as_bf16x8(ldg16(qi + (size_t)tq * DI + ks * 32 + g * 8));
}

// ----------------------------------------------------------------- init
__global__ __launch_bounds__(256) void fz_init_kernel(FzProb f, FzWs w, int32_t *__restrict__ idx) {
  const int t = blockIdx.x, tid = threadIdx.x;
  const int L = t + 1;
  int32_t *out = idx + (size_t)t * f.k;
  if (L <= f.k) {
    for (int c = tid; c < f.k; c += 256) out[c] = c < L ? c : -1;
    if (tid == 0) w.state[t] = RowState{0u, 0u, 0u, kRowSettled | kRowDirect};
    return;
  }
  const int nc = L - f.Wf;
  const int kp = f.k - f.Wf;
  for (int c = tid; c < f.Wf; c += 256) out[kp + c] = nc + c;
  if (tid < kFMaxChunks) {
    w.gt[(size_t)t * kFMaxChunks + tid] = 0u;
    w.eq[(size_t)t * kFMaxChunks + tid] = 0u;
  }
  if (tid == 0) {
    // k' = 0: nothing to choose; a prefix no key can exceed or match
    w.state[t] = kp == 0 ? RowState{0xffffffffu, 0xffffffffu, 0u, kRowSettled}
                         : RowState{0u, 0u, (uint32_t)kp, 0u};
  }
}

// ----------------------------------------------------------------- hist
template <int DI>
__global__ __launch_bounds__(kFW * 64) void fz_hist_kernel(FzProb f, FzWs w, int pass,
                                                           const uint16_t *__restrict__ qi,
                                                           const uint16_t *__restrict__ ki) {
  using T = FzTile<DI>;
  __shared__ __align__(16) char lds[2][T::BYTES];
  // two 16-bit counters per word; rows padded by a word so the 16 rows of a
  // wave land on different banks
  __shared__ uint32_t hist[kFQ][kFBins / 2 + 1];
  __shared__ int any_active;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  int grp, chunk;
  fz_decode(f, blockIdx.x, grp, chunk);
  const int rl = wave * 16 + c16;          // this lane's row within the group
  const int t = grp * kFQ + rl;
  RowState st{0u, 0u, 0u, kRowSettled};
  if (t < f.S) st = w.state[t];
  const bool active = !(st.flags & kRowSettled);
  if (tid == 0) any_active = 0;
  for (int i = tid; i < kFQ * (kFBins / 2 + 1); i += kFW * 64) (&hist[0][0])[i] = 0u;
  __syncthreads();
  if (active) any_active = 1;
  __syncthreads();
  if (!any_active) return;   // every row settled: its partials are never read

  bf16x8 qb[DI / 32];
  fz_load_q<DI>(qi, f.S, t, g, qb);
  const int nc = active ? fz_nc(f, t) : 0;
  const int shift = 24 - 8 * pass;
  const int k_begin = chunk * kFC;
  const int k_end = min(k_begin + kFC, fz_group_nc(f, grp));
  const int ntiles = (k_end - k_begin + kFKT - 1) / kFKT;
  uint32_t zeros = 0;
  const bool zero_matches = active && ((kFZero & st.pmask) == st.prefix);
  fz_walk<DI>(ki, f.S, k_begin, ntiles, tid, lds, [&](int it, const char *tile) __attribute__((always_inline)) {
    const int kt0 = k_begin + it * kFKT;
    // the MFMA needs every lane's operands: branch on the wave, mask per lane
    if (!__any(active && kt0 < nc)) return;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      uint32_t key[4];
      fz_keys<DI>(tile, kt, qb, f, g, c16, key);
      // Branch-free per key: zero keys (ReLU makes many) go to a register
      // count; a lane's equal neighbouring digits are merged; then, if any
      // lane of the wave counts anything, four unconditional LDS atomics
      // (a zero increment for the rest).
      uint32_t dig[4], inc[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int s = kt0 + kt * 16 + g * 4 + r;
        const bool m = active & (s < nc) & ((key[r] & st.pmask) == st.prefix);
        const bool z = key[r] == kFZero;
        zeros += (uint32_t)(m & z);
        dig[r] = (key[r] >> shift) & 0xffu;
        inc[r] = (uint32_t)(m & !z);
      }
#pragma unroll
      for (int r = 3; r > 0; --r) {
        const bool mg = (inc[r] != 0u) & (inc[r - 1] != 0u) & (dig[r] == dig[r - 1]);
        inc[r - 1] += mg ? inc[r] : 0u;
        inc[r] = mg ? 0u : inc[r];
      }
      if (__any(inc[0] | inc[1] | inc[2] | inc[3])) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          atomicAdd(&hist[rl][dig[r] >> 1], inc[r] << ((dig[r] & 1u) * 16));
      }
    }
  });
  // zero keys of a column: lanes c16, c16+16, c16+32, c16+48
  zeros += __shfl_xor(zeros, 16, 64);
  zeros += __shfl_xor(zeros, 32, 64);
  if (zero_matches && g == 0 && zeros) {
    const uint32_t d = (kFZero >> shift) & 0xffu;
    atomicAdd(&hist[rl][d >> 1], zeros << ((d & 1u) * 16));
  }
  __syncthreads();
  for (int i = tid; i < kFQ * kFBins / 2; i += kFW * 64) {
    const int r = i / (kFBins / 2), b2 = i % (kFBins / 2);
    const int tr = grp * kFQ + r;
    if (tr < f.S)
      reinterpret_cast<uint32_t *>(w.hist + ((size_t)chunk * f.S + tr) * kFBins)[b2] =
          hist[r][b2];
  }
}

// ---------------------------------------------------------------- resolve
// One wave per row; lane l owns bins 4l..4l+3.
__global__ __launch_bounds__(256) void fz_resolve_kernel(FzProb f, FzWs w, int pass) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= f.S) return;
  RowState st = w.state[t];
  if (st.flags & kRowSettled) return;
  const int nch = (fz_nc(f, t) + kFC - 1) / kFC;
  uint32_t part[kFMaxChunks][4];
  uint32_t cnt[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int c = 0; c < kFMaxChunks; ++c) {
    if (c < nch) {
      const uint2 h = *reinterpret_cast<const uint2 *>(w.hist + ((size_t)c * f.S + t) * kFBins +
                                                        lane * 4);
      part[c][0] = h.x & 0xffffu;
      part[c][1] = h.x >> 16;
      part[c][2] = h.y & 0xffffu;
      part[c][3] = h.y >> 16;
    } else {
      part[c][0] = part[c][1] = part[c][2] = part[c][3] = 0u;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) cnt[e] += part[c][e];
  }
  // keys above this lane's bins: sum over lanes with higher bins
  const uint32_t mine = cnt[0] + cnt[1] + cnt[2] + cnt[3];
  uint32_t incl = mine;   // inclusive suffix sum over lanes >= lane
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_down(incl, off, 64);
    if (lane + off < 64) incl += o;
  }
  const uint32_t above = incl - mine;
  const uint32_t need = st.remaining;
  // the lane whose bins contain the need-th largest key
  const bool here = above < need && above + mine >= need;
  const uint64_t bal = __ballot(here);
  if (bal == 0) {   // fewer matching keys than needed: cannot happen for consistent passes
    if (lane == 0) w.state[t].flags = st.flags | kRowSettled;
    return;
  }
  const int owner = __ffsll((unsigned long long)bal) - 1;
  int bin = 0;
  uint32_t above_bin = 0, in_bin = 0;
  if (lane == owner) {
    uint32_t acc = above;
    for (int e = 3; e >= 0; --e) {
      if (acc + cnt[e] >= need) {
        bin = lane * 4 + e;
        above_bin = acc;
        in_bin = cnt[e];
        break;
      }
      acc += cnt[e];
    }
  }
  bin = __shfl(bin, owner, 64);
  above_bin = __shfl(above_bin, owner, 64);
  in_bin = __shfl(in_bin, owner, 64);
  // per-chunk keys above the chosen bin, and on it
#pragma unroll
  for (int c = 0; c < kFMaxChunks; ++c) {
    if (c >= nch) continue;   // uniform
    uint32_t gtc = 0, eqc = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int b = lane * 4 + e;
      gtc += b > bin ? part[c][e] : 0u;
      eqc += b == bin ? part[c][e] : 0u;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      gtc += __shfl_xor(gtc, off, 64);
      eqc += __shfl_xor(eqc, off, 64);
    }
    if (lane == 0) {
      w.gt[(size_t)t * kFMaxChunks + c] += gtc;
      w.eq[(size_t)t * kFMaxChunks + c] = eqc;
    }
  }
  if (lane == 0) {
    const int shift = 24 - 8 * pass;
    st.prefix |= (uint32_t)bin << shift;
    st.pmask |= 0xffu << shift;
    st.remaining = need - above_bin;
    if (st.remaining == in_bin || pass == 3) st.flags |= kRowSettled;
    w.state[t] = st;
  }
}

// ------------------------------------------------------------------- emit
template <int DI>
__global__ __launch_bounds__(kFW * 64) void fz_emit_kernel(FzProb f, FzWs w,
                                                           const uint16_t *__restrict__ qi,
                                                           const uint16_t *__restrict__ ki,
                                                           int32_t *__restrict__ idx) {
  using T = FzTile<DI>;
  __shared__ __align__(16) char lds[2][T::BYTES];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  int grp, chunk;
  fz_decode(f, blockIdx.x, grp, chunk);
  const int t = grp * kFQ + wave * 16 + c16;
  RowState st{0u, 0u, 0u, kRowDirect};
  if (t < f.S) st = w.state[t];
  const bool live = t < f.S && !(st.flags & kRowDirect);
  const int nc = live ? fz_nc(f, t) : 0;
  const int kp = f.k - f.Wf;
  // offsets of this chunk: keys taken in earlier chunks
  uint32_t gt_before = 0, eq_before = 0;
  if (live) {
    for (int c = 0; c < chunk; ++c) {
      gt_before += w.gt[(size_t)t * kFMaxChunks + c];
      eq_before += w.eq[(size_t)t * kFMaxChunks + c];
    }
  }
  int32_t *out = idx + (size_t)min(t, f.S - 1) * f.k;

  bf16x8 qb[DI / 32];
  fz_load_q<DI>(qi, f.S, t, g, qb);
  const int k_begin = chunk * kFC;
  const int k_end = min(k_begin + kFC, fz_group_nc(f, grp));
  const int ntiles = (k_end - k_begin + kFKT - 1) / kFKT;
  fz_walk<DI>(ki, f.S, k_begin, ntiles, tid, lds, [&](int it, const char *tile) __attribute__((always_inline)) {
    const int kt0 = k_begin + it * kFKT;
    // the MFMA needs every lane's operands: branch on the wave, mask per lane
    if (__any(live && kt0 < nc)) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        uint32_t key[4];
        fz_keys<DI>(tile, kt, qb, f, g, c16, key);
        uint32_t cg = 0, ce = 0;
        bool isg[4], ise[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = kt0 + kt * 16 + g * 4 + r;
          const uint32_t m = key[r] & st.pmask;
          isg[r] = live && s < nc && m > st.prefix;
          ise[r] = live && s < nc && m == st.prefix;
          cg += isg[r];
          ce += ise[r];
        }
        // exclusive scan over the four lane groups of this column (keys in
        // position order: group g holds keys 4g..4g+3 of the 16)
        const uint32_t v = (cg << 16) | ce;
        uint32_t incl = v;
        uint32_t o = __shfl_up(incl, 16, 64);
        if (g >= 1) incl += o;
        o = __shfl_up(incl, 32, 64);
        if (g >= 2) incl += o;
        const uint32_t total = __shfl(incl, 48 + c16, 64);
        const uint32_t ex = incl - v;
        uint32_t my_gt = gt_before + (ex >> 16);
        uint32_t my_eq = eq_before + (ex & 0xffffu);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          bool take = isg[r];
          if (ise[r]) {
            take = my_eq < st.remaining;
            ++my_eq;
          }
          if (take) {
            const uint32_t pos = my_gt + min(my_eq - (ise[r] ? 1u : 0u), st.remaining);
            if (pos < (uint32_t)kp) out[pos] = kt0 + kt * 16 + g * 4 + r;
          }
          if (isg[r]) ++my_gt;
        }
        gt_before += total >> 16;
        eq_before += total & 0xffffu;
      }
    }
  });
}

template <int DI>
hipError_t launch_di(const FzProb &f, const void *qi, const void *ki, int32_t *idx, void *ws,
                     hipStream_t st) {
  const FzWs w = fz_carve(ws, f.S);
  const uint16_t *q = (const uint16_t *)qi, *k = (const uint16_t *)ki;
  hipLaunchKernelGGL(fz_init_kernel, dim3(f.S), dim3(256), 0, st, f, w, idx);
  const int items = fz_items(f);
  if (items > 0) {
    for (int pass = 0; pass < 4; ++pass) {
      hipLaunchKernelGGL((fz_hist_kernel<DI>), dim3(items), dim3(kFW * 64), 0, st, f, w, pass,
                         q, k);
      hipLaunchKernelGGL(fz_resolve_kernel, dim3((f.S + 3) / 4), dim3(256), 0, st, f, w, pass);
    }
    hipLaunchKernelGGL((fz_emit_kernel<DI>), dim3(items), dim3(kFW * 64), 0, st, f, w, q, k, idx);
  }
  return hipGetLastError();
}

// Scratch of the allocation-free entry point: one array per GPU the library
// runs on, held until the process ends. Every call on a GPU shares it.
static __device__ __align__(256) char scratch[kIndexerTopkStaticBytes];

// Device address of this device's copy of `scratch`, looked up once per
// device (with that device current) and kept. In host code the array's name
// is only a stand-in for the symbol, never an address a kernel may use.
constexpr int kScratchDevices = 64;
std::atomic<void *> g_scratch[kScratchDevices];

hipError_t static_scratch(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  void *ptr = g_scratch[dev].load(std::memory_order_acquire);
  if (!ptr) {
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch[dev].store(ptr, std::memory_order_release);
  }
  *out = ptr;
  return hipSuccess;
}

}  // namespace

size_t indexer_topk_workspace(const Prob &p) { return fz_bytes(p.S); }

hipError_t launch_indexer_topk_static(const Prob &p, const void *qi, const void *ki,
                                      int32_t *idx, hipStream_t st) {
  if (fz_bytes(p.S) > kIndexerTopkStaticBytes) return hipErrorInvalidValue;   // checked by the API
  void *ws = nullptr;
  const hipError_t e = static_scratch(&ws);
  if (e != hipSuccess) return e;
  // every partial the passes read is written by an earlier pass of the same
  // call (fz_init_kernel resets the per-row state), so no clearing is needed
  return launch_indexer_topk(p, qi, ki, idx, ws, st);
}

bool indexer_topk_supported(const Prob &p) {
  return p.dtype == SP_DTYPE_BF16 && (p.di == 64 || p.di == 128 || p.di == 256) && p.b == 1 &&
         p.S <= kFMaxChunks * kFC - 1 && p.S <= 65535 && p.iscale >= 0.f;
}

hipError_t launch_indexer_topk(const Prob &p, const void *qi, const void *ki, int32_t *idx,
                               void *ws, hipStream_t st) {
  FzProb f{p.S, p.k, p.W < p.k ? p.W : p.k, p.relu, p.iscale};
  if (p.di == 64) return launch_di<64>(f, qi, ki, idx, ws, st);
  if (p.di == 128) return launch_di<128>(f, qi, ki, idx, ws, st);
  return launch_di<256>(f, qi, ki, idx, ws, st);
}

}  // namespace sp
