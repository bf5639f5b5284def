// Attention tile pipeline shared by the MFMA attention kernels (dense causal
// flash attention, Section 3; selection-block-shared sparse attention,
// Sections 3 and 4.2).
//
// A workgroup owns up to NW*32 query rows ((query, head) pairs of one KV
// head, 32 per wave) and walks a list of key positions in tiles of 64. Scores
// are computed transposed, S^T = K Q^T, on v_mfma_f32_32x32x16_bf16: lane
// (n, h) = (l%32, l/32) owns query row n of its wave and holds 32 of the 64
// keys of a tile (keys 32kb + 8i + 4h + r), so the row max and row sum need
// one half-wave swap. The output is kept transposed too, O^T = V^T P^T: the
// score accumulators, rounded to bf16, are already the B operand of that
// product, and the V^T operand is read straight from the row-major V tile by
// the gfx950 LDS transpose read (ds_read_b64_tr_b16).
//
// Two-phase schedule. For key tile n a wave runs
//   M_n (matrix cores): S_n = K_n Q^T, and O += V_{n-1}^T P_{n-1}^T;
//   V_n (vector units): mask and row maxima of S_n, rescale of O when a row
//        maximum rises, P_n = exp2(S_n - m) with its row sums, bf16 P_n.
// The eight waves of a workgroup form two groups with one wave of each on
// every SIMD; group 1 runs half a step behind group 0, so while one wave of
// a SIMD issues matrix instructions its partner issues the softmax, and the
// two pipes overlap without fine-grained interleaving inside a wave. Each
// half step ends with one workgroup barrier. K tile n and V tile n - 1 stay
// in LDS for the two half steps in which the groups run M_n; meanwhile every
// wave loads its share of the next step's tiles straight into the other
// buffers. Smaller workgroups run M_n and V_n back to back.
//
// A key at position s contributes to a row of query t only if 0 <= s <= t
// (the causal mask of Section 3, applied per query as in Section 4.2); any
// other position (a -1 sentinel) contributes nothing. Tiles whose positions
// all lie in [0, first query of the wave] skip the mask.
//
// The running row maximum is raised only when a tile's maximum exceeds it by
// more than 2^kLazy in the exponent base-2 domain; until then the stale
// maximum is kept (probabilities up to 2^kLazy are exact in fp32 and within
// bf16 range), so the accumulators are rescaled only when it moves.
#pragma once

#include <math.h>

#include "common.hpp"
#include "mfma.hpp"

namespace sp {

// The attention workgroups fill most of a CU's LDS, so at most two waves
// share a SIMD; telling the compiler so lets it spend up to 256 registers a
// wave on operand prefetch instead of trimming for an occupancy it cannot
// reach. At head_dim 256 a wave's accumulators and query operands alone take
// 192 registers: those workgroups run one wave per SIMD (up to 512).
#define SP_ATTN_OCCUPANCY(D) __attribute__((amdgpu_waves_per_eu(1, (D) == 256 ? 1 : 2)))

// Waves per attention workgroup at head dimension D: two groups of four
// (one wave of each per SIMD) up to 128, one group at 256.
template <int D>
constexpr int attn_max_waves() {
  return D == 256 ? 4 : 8;
}

// Operand pairs of the matrix phase read ahead of the products.
constexpr int kMPrefetch = 2;

constexpr int kAttnKT = 64;      // key positions per tile
constexpr int kAttnQPW = 32;     // query rows per wave
constexpr float kLazy = 8.f;     // max may lag by up to 8 (factor 256)
// Word 3 of a raw buffer resource on gfx950: 32-bit data format, no swizzle.
constexpr int kBufferDword3 = 0x00020000;

typedef short v4i16 __attribute__((ext_vector_type(4)));

template <int D>
struct AttnLayout {
  // K and V tiles (64 rows of D bf16) are row-major with unpadded rows, and
  // the pieces of each row are permuted by row so that operand reads hit
  // distinct banks: 16-byte slot c of K row r is stored at c ^ kswz(r) (the
  // 16 rows of a b128 read phase, same slot, then fall on 16 different
  // slots), and 64-byte group g of V row r at g ^ vswz(r) (the 4 rows a
  // transpose-read phase touches fall on 4 different 16-bank groups). Both
  // depend only on r mod 16, so a K read is one base per k-step, and a V read
  // one base per 32-dim block, plus an immediate offset. A tile is a whole
  // number of 1 KiB chunks (the unit of a direct-to-LDS load).
  static constexpr int RB = D * 2;            // bytes of one row in HBM
  static constexpr int C = D / 8;             // 16-byte columns of a row
  static constexpr int KSLOTS = C;            // 16-byte slots of a K row
  static constexpr int VSLOTS = C;            // 16-byte slots of a V row
  static constexpr int KRB = 16 * KSLOTS;
  static constexpr int VRB = 16 * VSLOTS;
  static constexpr int KTILE = kAttnKT * KRB;
  static constexpr int VTILE = kAttnKT * VRB;
  static_assert(KTILE % 1024 == 0 && VTILE % 1024 == 0, "tiles are whole chunks");
  static constexpr int KS = D / 16;   // k-steps of K Q^T
  static constexpr int DT = D / 32;   // 32-row blocks of O^T (64-byte groups of a V row)
  __host__ __device__ static constexpr int vswz(int r) { return DT >= 4 ? (r & 3) : ((r >> 1) & 1); }
  // K: 16-byte slot c of row r stored at c ^ kswz(r), so the 16 rows of a
  // b128 operand-read phase (same slot) land on distinct banks
  __host__ __device__ static constexpr int kswz(int r) { return D == 64 ? ((r >> 1) & 7) : (r & 15); }
  // two K buffers, then (when the output is wanted) two V buffers
  static constexpr int bytes(bool want_v) { return 2 * KTILE + (want_v ? 2 * VTILE : 0); }
  // the output staging of attn_finish reuses the tiles: 32 rows per wave at
  // a stride of RB + 16 bytes
  static constexpr int FINISH_OS = RB + 16;
  static constexpr int lds_bytes(bool want_v, int nw) {
    return want_v && nw * kAttnQPW * FINISH_OS > bytes(true) ? nw * kAttnQPW * FINISH_OS
                                                             : bytes(want_v);
  }
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Wait for every outstanding memory operation of this wave. Issued once
// before the tile loop, it tells the compiler that loads made before the
// loop (Q fragments, the first tile) are complete, so no wait on them is
// placed inside the loop, where it would also stall on the next prefetch.
__device__ __forceinline__ void drain_memory() { __builtin_amdgcn_s_waitcnt(0); }

// Ends a phase for v: v is computed before this point and not moved past
// it. Matrix and vector arithmetic has no memory effects, so without this the
// compiler may sink a phase's products past the barrier that ends the phase
// (to their first use in the next one), which breaks the two-group schedule.
template <class T>
__device__ __forceinline__ void settle(T &v) {
  asm volatile("" : "+v"(v));
}

// Combine lane l with lane l ^ 32 (the other half of a query column).
__device__ __forceinline__ float half_max(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
}
__device__ __forceinline__ float half_sum(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}

// LDS read of four ints at LDS byte address a, by inline assembly: the
// compiler would otherwise wait for every outstanding direct-to-LDS tile
// load first, although those never write the arrays read this way.
__device__ __forceinline__ int4 lds_read_i32x4(uint32_t a) {
  int4 r;
  asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(r) : "v"(a) : "memory");
  return r;
}

// Global -> LDS staging of one tile of K or V rows of KV head j, with no
// register round trip: a load instruction fills one 1 KiB chunk of the tile
// (buffer_load_dwordx4 ... lds puts lane L's 16 bytes at byte 16L of it).
// Lane L of chunk q holds 16-byte slot 64q + L of the tile, that is row
// (64q + L) / SLOTS, stored column (64q + L) % SLOTS, and fetches the column
// whose permuted place that slot is. The chunks of a tile go to the waves in
// turn.
template <int D, int NW, bool IS_V>
struct TileLoader {
  using L = AttnLayout<D>;
  static constexpr int SLOTS = IS_V ? L::VSLOTS : L::KSLOTS;
  static constexpr int CHUNKS = (IS_V ? L::VTILE : L::KTILE) / 1024;
  static constexpr int PER = (CHUNKS + NW - 1) / NW;

  // rows() resolves the row of every chunk this lane loads (row(e) gives the
  // row of tile entry e; padding slots take entry 0), issue() then fetches
  // them. Split so that a pipeline can resolve the rows of its next loads
  // (an LDS lookup for gathered tiles) a step ahead of issuing them.
  template <typename ROW>
  __device__ __forceinline__ static void rows(int wave, int lane, ROW row, int (&out)[PER]) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int q = wave + p * NW;
      const int slot = (q < CHUNKS ? q : 0) * 64 + lane;
      const int r = slot / SLOTS, c = slot % SLOTS;
      out[p] = row(c < L::C ? r : 0);
    }
  }

  // Rows outside [0, nrows) read row 0; their keys are masked. No lane of a
  // chunk is masked (the rows have no padding slots). Rows are fetched
  // through a buffer resource (base and size in SGPRs, 32-bit byte offsets
  // per lane); the API keeps k and v below 4 GiB.
  __device__ __forceinline__ static void issue(uint32_t tile, const uint16_t *base, int nrows,
                                               int Hkv, int j, int wave, int lane,
                                               const int (&rw)[PER]) {
    const uint32_t row_bytes = (uint32_t)Hkv * L::RB;
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(base), (short)0,
                                                      (uint32_t)nrows * row_bytes, kBufferDword3);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int q = wave + p * NW;
      const int slot = (q < CHUNKS ? q : 0) * 64 + lane;
      int c = slot % SLOTS;
      if constexpr (IS_V) c ^= 4 * L::vswz(slot / SLOTS);
      else c ^= L::kswz(slot / SLOTS);
      const uint32_t s = (rw[p] >= 0 && rw[p] < nrows) ? (uint32_t)rw[p] : 0u;
      const uint32_t off = s * row_bytes + (uint32_t)(j * L::RB + (c < L::C ? c : 0) * 16);
      if (CHUNKS % NW == 0 || q < CHUNKS)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs, (__attribute__((address_space(3))) void *)(size_t)(tile + q * 1024), 16, off,
            0, 0, 0);
    }
  }

  template <typename ROW>
  __device__ __forceinline__ static void load(uint32_t tile, const uint16_t *base, int nrows,
                                              int Hkv, int j, int wave, int lane, ROW row) {
    int rw[PER];
    rows(wave, lane, row, rw);
    issue(tile, base, nrows, Hkv, j, wave, lane, rw);
  }
};

// Wait until at most N of this wave's global loads (the direct-to-LDS tile
// loads, which complete in issue order) are outstanding; a barrier after it
// publishes the older tiles to the workgroup. expcnt and lgkmcnt are left at
// their maxima.
template <int N>
__device__ __forceinline__ void wait_loads() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// This lane's query row: Q fragments (B operand of K Q^T), position, head.
template <int D>
struct QRow {
  bf16x8 bq[AttnLayout<D>::KS];
  int t, head;
  bool valid;
};

// Row m of a workgroup (query-major) is query t0 + m/G, head j*G + m%G. Rows
// past nrows load row 0 of the workgroup and are never written.
template <int D>
__device__ __forceinline__ void load_q_row(const uint16_t *__restrict__ q, int Hq, int G, int j,
                                           int t0, int m, int nrows, int h, QRow<D> &qr) {
  qr.valid = m < nrows;
  const int mm = qr.valid ? m : 0;
  qr.t = t0 + mm / G;
  qr.head = j * G + mm % G;
  const uint16_t *qp = q + ((size_t)qr.t * Hq + qr.head) * D + 8 * h;
#pragma unroll
  for (int ks = 0; ks < AttnLayout<D>::KS; ++ks) qr.bq[ks] = as_bf16x8(ldg16(qp + 16 * ks));
}

// Per-wave online-softmax state for 32 query rows.
template <int D>
struct AttnState {
  f32x16 o[AttnLayout<D>::DT];   // O^T, rows d = 32dt + 8i + 4h + r
  bf16x8 p[4];                   // P^T of the last softmaxed tile, k-step f: keys 16f..16f+15
  float m;                       // running max (base-2 scaled logits), may lag by < kLazy
  float l;                       // this lane's part of the row sum
};

// This lane's read offsets into a K tile and a V tile. K fragment (kb, ks)
// of lane (n, h) is row 32kb + n, slot 2ks + h, stored at (2ks + h) ^
// kswz(n): one base per k-step. V^T fragment (f, dt) of
// lane (grp, c16) reads, by transpose, rows 16f + 4h + c16/4 (then +8),
// d = 32dt + 16(grp%2) + 4(c16%4) onwards, whose 64-byte group dt is stored
// at dt ^ vswz(row): one base per d-block dt (the same for all the rows this
// lane reads). The parts that depend on kb and f are immediate offsets.
template <int D>
struct TileOffsets {
  using L = AttnLayout<D>;
  uint32_t k[L::KS], v[L::DT];
  __device__ __forceinline__ void init(int lane) {
    const int n = lane & 31, h = lane >> 5, c16 = lane & 15, grp = lane >> 4;
#pragma unroll
    for (int ks = 0; ks < L::KS; ++ks) k[ks] = n * L::KRB + ((2 * ks + h) ^ L::kswz(n)) * 16;
    const int r0 = 4 * h + (c16 >> 2);
#pragma unroll
    for (int dt = 0; dt < L::DT; ++dt)
      v[dt] = r0 * L::VRB + 64 * (dt ^ L::vswz(r0)) + 32 * (grp & 1) + 8 * (c16 & 3);
  }
};

// Masks scores whose position fails 0 <= s <= t; pos4(e0) returns the
// positions of tile entries e0..e0+3.
template <class POS4>
__device__ __forceinline__ void mask_tile(f32x16 (&s)[2], int t, int h, POS4 pos4) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int4 p = pos4(32 * kb + 8 * i + 4 * h);
      const int pv[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (!(pv[r] >= 0 && pv[r] <= t)) s[kb][4 * i + r] = -INFINITY;
    }
}

// Row maximum over the lane's 32 keys (a balanced tree: the softmax phase
// runs with no other vector wave on its SIMD to hide dependent latencies),
// then across the two half-waves.
__device__ __forceinline__ float tile_max(const f32x16 (&s)[2]) {
  float m[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) m[e] = fmaxf(s[0][e], s[1][e]);
#pragma unroll
  for (int w = 8; w > 0; w >>= 1)
#pragma unroll
    for (int e = 0; e < w; ++e) m[e] = fmaxf(m[e], m[e + w]);
  return half_max(m[0]);
}

// P_i = exp2(scale_log2 * S_i - mref), summed into l; WANT_P keeps it in
// bf16 as the B operand of the next P V product.
// The row sum keeps four partial sums (one per k-step) so that its additions
// do not form one dependent chain.
template <int D, bool WANT_P>
__device__ __forceinline__ void exp_tile(const f32x16 (&s)[2], float scale_log2, float mref,
                                         AttnState<D> &st) {
  float sum[4];
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    bf16x8 pf;
    sum[f] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float pv = fast_exp2(fmaf(s[f >> 1][8 * (f & 1) + e], scale_log2, -mref));
      sum[f] += pv;
      pf[e] = (__bf16)pv;
    }
    if constexpr (WANT_P) st.p[f] = pf;
  }
  st.l += (sum[0] + sum[1]) + (sum[2] + sum[3]);
}

// Operand reads of pair IT of m_tile, issued by inline assembly: each
// product then waits with its own lgkmcnt for exactly the reads it needs (LDS
// reads complete in order). The compiler cannot prove that these reads miss
// the tiles the direct-to-LDS loads are filling, and would otherwise wait for
// every outstanding load before the first read.
template <int D, int IT>
__device__ __forceinline__ void m_kread(const uint32_t (&kas)[AttnLayout<D>::KS],
                                        bf16x8 &r) {   // k-step IT/2, key half IT%2
  using L = AttnLayout<D>;
  asm volatile("ds_read_b128 %0, %1 offset:%2"
               : "=v"(r)
               : "v"(kas[IT >> 1]), "i"((IT & 1) * 32 * L::KRB));
}
template <int D, int IT>
__device__ __forceinline__ void m_vread(const uint32_t (&vas)[AttnLayout<D>::DT],
                                        bf16x8 &r) {   // k-step IT/DT, d-block IT%DT
  using L = AttnLayout<D>;
  const uint32_t va = vas[IT % L::DT];
  constexpr int off = (IT / L::DT) * 16 * L::VRB;
  uint2 lo, hi;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(lo) : "v"(va), "i"(off));
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(hi) : "v"(va), "i"(off + 8 * L::VRB));
  __builtin_memcpy(&r, &lo, 8);
  __builtin_memcpy(reinterpret_cast<char *>(&r) + 8, &hi, 8);
}

// M_n for one wave: S = K_n Q^T (QK) and O += V_{n-1}^T P^T (PV), as one
// sequence of D/8 (QK, PV) pairs of matrix instructions: 2 KS = 4 DT = D/8,
// so pair it is QK k-step it/2 of key half it%2 and PV k-step it/DT of
// d-block it%DT. Alternating the two products keeps six accumulators in
// flight, and the operand reads run kMPrefetch pairs ahead of the products.
template <int D, bool QK, bool PV>
__device__ __forceinline__ void m_tile(uint32_t kt, uint32_t vt, const TileOffsets<D> &to,
                                       const bf16x8 (&bq)[AttnLayout<D>::KS], f32x16 (&s)[2],
                                       AttnState<D> &st) {
  using L = AttnLayout<D>;
  constexpr int NP = D / 8;
  if constexpr (QK) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[kb][e] = 0.f;
  }
  uint32_t ka[L::KS], va[L::DT];
#pragma unroll
  for (int ks = 0; ks < L::KS; ++ks) ka[ks] = kt + to.k[ks];
#pragma unroll
  for (int dt = 0; dt < L::DT; ++dt) va[dt] = vt + to.v[dt];
  // The counts below assume only these reads are outstanding on the LGKM
  // counter (scalar loads return out of order): drain it first.
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  // LDS reads per pair: QK 1, PV 2; operands of the next PF pairs are in
  // flight while a pair's products issue
  constexpr int RV = PV ? 2 : 0, RP = (QK ? 1 : 0) + RV;
  constexpr int PF = kMPrefetch;
  constexpr int NB = PF + 1;
  bf16x8 kf[NB], vf[NB];
  static_for<0, PF>([&](auto I) {
    constexpr int it = decltype(I)::value;
    if constexpr (QK) m_kread<D, it>(ka, kf[it]);
    if constexpr (PV) m_vread<D, it>(va, vf[it]);
  });
  static_for<0, NP>([&](auto I) {
    constexpr int it = decltype(I)::value;
    constexpr int nx = it + PF;   // pair whose reads are issued now
    if constexpr (nx < NP) {
      if constexpr (QK) m_kread<D, (nx < NP ? nx : 0)>(ka, kf[nx % NB]);
      if constexpr (PV) m_vread<D, (nx < NP ? nx : 0)>(va, vf[nx % NB]);
    }
    // reads issued after this pair's: those of the next min(PF, NP-1-it) pairs
    constexpr int later = (NP - 1 - it < PF ? NP - 1 - it : PF) * RP;
    if constexpr (QK) {
      asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(kf[it % NB]) : "i"(RV + later));
      s[it & 1] = mfma32(kf[it % NB], bq[it >> 1], s[it & 1]);
    }
    if constexpr (PV) {
      asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(vf[it % NB]) : "i"(later));
      st.o[it % L::DT] = mfma32(vf[it % NB], st.p[it / L::DT], st.o[it % L::DT]);
    }
  });
}

template <int D, int NW, bool WANT_O, class Src>
struct AttnPipe {
  using L = AttnLayout<D>;
  // two groups of four waves; wave w runs on SIMD w % 4
  static constexpr bool kPaired = NW == 8;
  const Src &src;
  const uint16_t *k, *v;
  int kv_rows, Hkv, j, wave, lane, h, wave_tmin, nt, group;
  float scale_log2;
  uint32_t lds;   // K tile i at lds + (i % 2) KTILE, V tile i after the two K buffers
  TileOffsets<D> to;
  const QRow<D> &qr;
  AttnState<D> &st;
  f32x16 s[2];    // S_n between M_n and V_n

  __device__ __forceinline__ AttnPipe(char *lds_, const Src &src_, const uint16_t *k_,
                                      const uint16_t *v_, int kv_rows_, int Hkv_, int j_,
                                      float sl2, int wave_tmin_, const QRow<D> &qr_,
                                      AttnState<D> &st_)
      : src(src_), k(k_), v(v_), kv_rows(kv_rows_), Hkv(Hkv_), j(j_), wave_tmin(wave_tmin_),
        nt(__builtin_amdgcn_readfirstlane(src_.ntiles)), scale_log2(sl2), qr(qr_), st(st_) {
    // wave-uniform values in scalar registers: the loop and the group
    // branches are then scalar branches
    wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    lane = threadIdx.x & 63;
    h = lane >> 5;
    group = kPaired ? wave >> 2 : 0;
    lds = (uint32_t)(size_t)(__attribute__((address_space(3))) char *)lds_;
    to.init(lane);
  }

  __device__ __forceinline__ uint32_t ktile(int i) const { return lds + (i & 1) * L::KTILE; }
  __device__ __forceinline__ uint32_t vtile(int i) const {
    return lds + 2 * L::KTILE + (i & 1) * L::VTILE;
  }

  // Rows of the chunks the next load_next issues: K_{n+1} and V_n. A source
  // whose rows are an LDS lookup (Src::kLookup) resolves them a step ahead;
  // one whose rows are arithmetic resolves them at issue.
  using KLoader = TileLoader<D, NW, false>;
  using VLoader = TileLoader<D, NW, true>;
  int krows[KLoader::PER], vrows[VLoader::PER];
  __device__ __forceinline__ void fetch_rows(int n) {
    if (n + 1 < nt) KLoader::rows(wave, lane, [&](int e) { return src.row(n + 1, e); }, krows);
    if constexpr (WANT_O)
      if (n < nt) VLoader::rows(wave, lane, [&](int e) { return src.row(n, e); }, vrows);
  }

  // Tiles of step n + 1: K_{n+1} and V_n, each wave its share of the chunks.
  // Their buffers held K_{n-1} and V_{n-2}, last read in M_{n-1}, before the
  // barrier that opened step n. Issued at the top of the step; looked-up rows
  // were resolved during the previous step (lookup_next).
  __device__ __forceinline__ void load_next(int n) {
    if constexpr (!Src::kLookup) fetch_rows(n);
    if (n + 1 < nt) KLoader::issue(ktile(n + 1), k, kv_rows, Hkv, j, wave, lane, krows);
    if constexpr (WANT_O)
      if (n < nt) VLoader::issue(vtile(n), v, kv_rows, Hkv, j, wave, lane, vrows);
  }
  // Looks up the rows of step n + 1's loads. Called just before a barrier:
  // the barrier's wait for LDS reads then falls in time the wave would spend
  // waiting there anyway, not at the start of an MFMA phase.
  __device__ __forceinline__ void lookup_next(int n) {
    if constexpr (Src::kLookup) fetch_rows(n + 1);
  }

  // M_n: QK (n < nt) and PV (n >= 1)
  template <bool QK, bool PV>
  __device__ __forceinline__ void phase_m(int n) {
    m_tile<D, QK, PV && WANT_O>(QK ? ktile(n) : 0, PV ? vtile(n - 1) : 0, to, qr.bq, s, st);
    if constexpr (QK) {
      settle(s[0]);
      settle(s[1]);
    }
    if constexpr (PV && WANT_O) {
#pragma unroll
      for (int dt = 0; dt < L::DT; ++dt) settle(st.o[dt]);
    }
  }

  // V_n, for 0 <= n < nt
  __device__ __forceinline__ void phase_v(int n) {
    if (src.needs_mask(n, wave_tmin))
      mask_tile(s, qr.t, h, [&](int e0) { return src.pos4(n, e0); });
    const float mx = tile_max(s) * scale_log2;   // scale > 0 commutes with max
    const float mold = st.m;
    const bool raised = mx > mold + kLazy;
    const float mnew = raised ? mx : mold;
    const float mref = mnew == -INFINITY ? 0.f : mnew;
    st.m = mnew;
    // Rows whose maximum was raised rescale l and O (rare after the first
    // tile). The branch is per lane: lanes that do not take it are masked,
    // so O is updated in place on both paths.
    if (raised) {
      const float corr = fast_exp2(mold - mref);   // mold = -inf gives 0
      st.l *= corr;
      if constexpr (WANT_O) {
#pragma unroll
        for (int dt = 0; dt < L::DT; ++dt)
#pragma unroll
          for (int e = 0; e < 16; ++e) st.o[dt][e] *= corr;
      }
    }
    exp_tile<D, WANT_O>(s, scale_log2, mref, st);
    if constexpr (WANT_O) {
#pragma unroll
      for (int f = 0; f < 4; ++f) settle(st.p[f]);
    }
    settle(st.l);
    settle(st.m);
  }

  __device__ __forceinline__ void end_step() {
    wait_loads<0>();
    __syncthreads();
  }

  __device__ __forceinline__ void run() {
#pragma unroll
    for (int dt = 0; dt < L::DT; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) st.o[dt][e] = 0.f;
    st.m = -INFINITY;
    st.l = 0.f;
    if (nt <= 0) return;
    TileLoader<D, NW, false>::load(ktile(0), k, kv_rows, Hkv, j, wave, lane,
                                   [&](int e) { return src.row(0, e); });
    if constexpr (Src::kLookup) fetch_rows(0);
    drain_memory();
    __syncthreads();
    // Every step: all waves issue the next step's loads, run their phases
    // (group 1 half a step behind group 0) and wait for their loads before
    // the step's last barrier. The first and last steps are peeled so the
    // loop body has no phase conditions, and each group runs a loop of its
    // own (same barriers).
    if (!kPaired) {
      load_next(0);
      phase_m<true, false>(0);
      phase_v(0);
      lookup_next(0);
      end_step();
#pragma unroll 1
      for (int n = 1; n < nt; ++n) {
        load_next(n);
        phase_m<true, true>(n);
        phase_v(n);
        lookup_next(n);
        end_step();
      }
      phase_m<false, true>(nt);
    } else if (group == 0) {
      load_next(0);
      phase_m<true, false>(0);
      lookup_next(0);
      __syncthreads();
      phase_v(0);
      end_step();
#pragma unroll 1
      for (int n = 1; n < nt; ++n) {
        load_next(n);
        phase_m<true, true>(n);
        lookup_next(n);
        __syncthreads();
        phase_v(n);
        end_step();
      }
      phase_m<false, true>(nt);
      __syncthreads();
      __syncthreads();
    } else {
      load_next(0);
      lookup_next(0);
      __syncthreads();
      phase_m<true, false>(0);
      end_step();
#pragma unroll 1
      for (int n = 1; n < nt; ++n) {
        load_next(n);
        phase_v(n - 1);
        lookup_next(n);
        __syncthreads();
        phase_m<true, true>(n);
        end_step();
      }
      phase_v(nt - 1);
      __syncthreads();
      phase_m<false, true>(nt);
      __syncthreads();
    }
  }
};

// Final normalisation: writes o (bf16, if non-null) and lse (natural log, if
// non-null) for this wave's valid rows. Rows with no usable key get o = 0 and
// lse = -inf.
//
// O is held transposed (lane (n, h) has 8-byte pieces of row n), and stored
// from there each instruction would scatter 16 bytes over 32 rows. Instead
// every wave writes its 32 normalised rows into a private slice of the tile
// buffers (idle once every wave has left the pipeline), reads them back
// row-major and stores whole rows: 1 KiB of consecutive rows per
// instruction. A row's destination comes from the lane that owns it by a
// lane shuffle. Every wave of the workgroup calls this (when o is given, it
// waits at a workgroup barrier before touching the tiles); lds is the
// pipeline's tile storage.
template <int D>
__device__ __forceinline__ void attn_finish(const AttnState<D> &st, const QRow<D> &qr, int Hq,
                                            uint16_t *__restrict__ o, float *__restrict__ lse,
                                            int h, char *lds) {
  using L = AttnLayout<D>;
  const float l = half_sum(st.l);
  if (lse && h == 0 && qr.valid)
    lse[(size_t)qr.t * Hq + qr.head] = l > 0.f ? (st.m + log2f(l)) * kLn2 : -INFINITY;
  if (!o) return;
  // slice row stride: 16 rows of a 64-lane write land on distinct bank pairs
  constexpr int OS = L::FINISH_OS;
  static_assert(kAttnQPW * OS * attn_max_waves<D>() <= L::lds_bytes(true, attn_max_waves<D>()),
                "slices fit the tile storage");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  char *slice = lds + wave * kAttnQPW * OS;
  const float inv = l > 0.f ? 1.f / l : 0.f;
  __syncthreads();
  char *wr = slice + (lane & 31) * OS + 8 * h;
#pragma unroll
  for (int dt = 0; dt < L::DT; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint2 w;
      w.x = pack_bf16x2(st.o[dt][4 * i] * inv, st.o[dt][4 * i + 1] * inv);
      w.y = pack_bf16x2(st.o[dt][4 * i + 2] * inv, st.o[dt][4 * i + 3] * inv);
      *reinterpret_cast<uint2 *>(wr + 64 * dt + 16 * i) = w;
    }
  // the reads below take other lanes' rows
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  constexpr int LPR = L::RB / 16;   // lanes per row
  constexpr int RPI = 64 / LPR;     // rows per store instruction
  const int rr = lane / LPR, cc = lane % LPR;
  const int my_t = qr.valid ? qr.t : -1;
#pragma unroll
  for (int it = 0; it < kAttnQPW / RPI; ++it) {
    const int m = it * RPI + rr;
    const int t = __shfl(my_t, m, 64);
    const int head = __shfl(qr.head, m, 64);
    const int4 val = *reinterpret_cast<const int4 *>(slice + m * OS + cc * 16);
    if (t >= 0)
      *reinterpret_cast<int4 *>(o + ((size_t)t * Hq + head) * D + cc * 8) = val;
  }
}

}  // namespace sp
