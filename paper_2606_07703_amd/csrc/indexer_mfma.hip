// Head-collapsed indexer scores on bf16 MFMA (Section 6.3; Algorithm 2, candidate scoring).
//
//   z[t,s] = ReLU(iscale * <q_idx[t], k_idx[s]>),  s <= t
//
// Two kernels share one structure: a workgroup owns a range of queries
// (64 per wave, resident in registers as MFMA operands) and streams key
// tiles through double-buffered LDS. Each key tile is read from L2 once per
// workgroup and reused by every wave. Only key tiles at or below a wave's
// last query are multiplied (causal skipping). The rows kernel gives each
// workgroup a chunk of up to 1024 keys; the block kernel runs a persistent
// grid over (query group, key tile) units, split evenly between workgroups.
//
// * indexer_block_kernel (b in {16, 32, 64, 128}): the epilogue scales,
//   applies the ReLU and the per-pair causal mask (t >= s, Section 4.2) and
//   reduces over the b queries of each selection block (max or sum) before
//   anything leaves the chip; one float per (block, key) is stored.
// * indexer_rows_kernel (b = 1): every causal score is stored. The MFMA is
//   issued with keys as rows (scores transposed), so a lane holds runs of
//   four consecutive keys of one query; each wave passes a tile's scores
//   through a few LDS rows so that a store instruction writes whole row
//   segments of 4 (or 8) queries instead of 64 bytes of 16 queries.
#include <math.h>

#include <atomic>
#include <climits>

#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"
#include "persistent_units.hpp"

namespace sp {
namespace {

constexpr int kQW = 64;     // queries per wave
constexpr int kKC = 1024;   // keys per workgroup chunk (rows kernel)
constexpr int kIdxBufferDword3 = 0x00020000;   // raw buffer resource: 32-bit data format
// Waits until this wave's vector memory operations (direct-to-LDS key tile
// loads and stores) have completed; LDS and scalar counters are not checked.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

template <int DI>
struct Tile {
  static constexpr int KT = DI <= 128 ? 64 : 32;   // keys per LDS tile
  static constexpr int RB = DI * 2 + 16;           // padded row bytes (bank spread)
  static constexpr int BYTES = KT * RB;
  static constexpr int CHUNKS = KT * DI / 8;       // 16-byte pieces per tile
  static constexpr int KS = DI / 32;               // MFMA k-steps
};

// Global -> registers -> LDS staging of one key tile, rows clamped to S-1.
template <int DI, int NT>
struct KeyStage {
  static constexpr int PER = (Tile<DI>::CHUNKS + NT - 1) / NT;
  uint4 reg[PER];
  __device__ __forceinline__ void load(const uint16_t *__restrict__ ki, int S, int k0, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < Tile<DI>::CHUNKS) {
        const int row = c / (DI / 8), col = c % (DI / 8);
        const int s = min(k0 + row, S - 1);
        reg[i] = ldg16(ki + (size_t)s * DI + col * 8);
      }
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < Tile<DI>::CHUNKS) {
        const int row = c / (DI / 8), col = c % (DI / 8);
        sts16(lds + row * Tile<DI>::RB + col * 16, reg[i]);
      }
    }
  }
};

__device__ __forceinline__ float agg2(int agg, float a, float b) {
  return agg == SP_AGG_MAX ? fmaxf(a, b) : a + b;
}

__device__ __forceinline__ float as_f(uint32_t x) { return __uint_as_float(x); }
__device__ __forceinline__ uint32_t as_u(float x) { return __float_as_uint(x); }

// MAXPOS: aggregation is max and the scale is non-negative, so scale and
// ReLU commute with the max: rows are reduced on raw MFMA outputs and only
// the reduced value is scaled; tiles entirely below a wave's first query
// skip the causal test. The kernel's split of (query group, key tile) units
// over its persistent grid is in persistent_units.hpp.

// Key tiles of the block kernel: NSUB sub-tiles of 64 keys, staged one tile
// ahead through registers into double-buffered LDS.
template <int DI>
struct BlockTile {
  static constexpr int NSUB = DI <= 128 ? 2 : 1;
  static constexpr int KT = 64 * NSUB;
  static constexpr int RB = DI * 2 + 16;
  static constexpr int BYTES = KT * RB;
};

template <int DI, int KT, int RB, int NT>
struct KeyStageT {
  static constexpr int CHUNKS = KT * DI / 8;
  static constexpr int PER = (CHUNKS + NT - 1) / NT;
  uint4 reg[PER];
  __device__ __forceinline__ void load(const uint16_t *__restrict__ ki, int S, int k0, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < CHUNKS) {
        const int row = c / (DI / 8), col = c % (DI / 8);
        const int s = min(k0 + row, S - 1);
        reg[i] = ldg16(ki + (size_t)s * DI + col * 8);
      }
    }
  }
  __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c < CHUNKS) {
        const int row = c / (DI / 8), col = c % (DI / 8);
        sts16(lds + row * RB + col * 16, reg[i]);
      }
    }
  }
};

// Direct-to-LDS loads of one key tile of the block kernel: slot c of padded
// row r at byte (r * SLOTS + c) * 16, so chunk q of 64 slots is 1 KiB at
// q * 1024, and wave w issues chunks w, w + NW, ... A lane's offset within a
// tile is fixed (kept in registers); lanes on the padding slot load the
// row's first 16 bytes into it (nothing reads it). Keys past S - 1 fall
// outside the buffer and load zeros (they are always masked).
template <int DI, int KT, int RB, int NW>
struct KeyTileDma {
  static constexpr int SLOTS = DI / 8 + 1, CHUNKS = KT * SLOTS / 64;
  static constexpr int CPW = (CHUNKS + NW - 1) / NW;
  static_assert(KT * SLOTS % 64 == 0 && SLOTS * 16 == RB, "whole chunks of padded rows");
  __device__ __forceinline__ static void offsets(int wave, int lane, uint32_t (&koff)[CPW]) {
#pragma unroll
    for (int p = 0; p < CPW; ++p) {
      const int slot = (wave + p * NW) * 64 + lane;
      const int row = slot / SLOTS, col = slot % SLOTS;
      koff[p] = (uint32_t)row * (DI * 2) + (uint32_t)(col < SLOTS - 1 ? col : 0) * 16;
    }
  }
  __device__ __forceinline__ static void issue(uint32_t base, const uint16_t *ki, int S, int k0,
                                               int wave, const uint32_t (&koff)[CPW]) {
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(ki), (short)0,
                                                      (uint32_t)S * (DI * 2), kIdxBufferDword3);
    const uint32_t sb = (uint32_t)k0 * (DI * 2);
#pragma unroll
    for (int p = 0; p < CPW; ++p) {
      const int q = wave + p * NW;
      if (CHUNKS % NW == 0 || q < CHUNKS)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs, (__attribute__((address_space(3))) void *)(size_t)(base + q * 1024), 16,
            koff[p] + sb, 0, 0, 0);
    }
  }
};

// Half-wave combine on 32x32 MFMA outputs: lane l with lane l ^ 32.
template <class Op>
__device__ __forceinline__ float half_combine(float x, Op op) {
  const auto a = __builtin_amdgcn_permlane32_swap(as_u(x), as_u(x), false, false);
  return op(as_f(a[0]), as_f(a[1]));
}

// The block kernel runs on v_mfma_f32_32x32x16_bf16 with queries as rows:
// A = 32 queries x 16 dims (resident in registers), B = 16 dims x 32 keys
// (a key row read from LDS), so lane (n, h) of a 32x32 score tile holds key
// column n for queries 8i + 4h + r. A selection block's aggregate is then a
// lane-local reduction plus one half-wave combine, and the half index h picks
// which key tile or block a lane stores, so every store row is contiguous.
template <int DI, int BQ, bool MAXPOS, int NW>
__global__ __launch_bounds__(NW * 64) void indexer_block_kernel(int S, int g0, int n_units,
                                                                int agg, int relu, float scale,
                                                                const uint16_t *__restrict__ qi,
                                                                const uint16_t *__restrict__ ki,
                                                                float *__restrict__ Y) {
  using T = BlockTile<DI>;
  constexpr int NT = NW * 64;
  constexpr int KT = T::KT, RB = T::RB, KS = DI / 16, NSUB = T::NSUB;
  constexpr int QG = NW * kQW;
  static_assert(QG % KT == 0, "query groups hold whole key tiles");
  __shared__ __align__(16) char lds[2][T::BYTES];
  __shared__ float red[NW / 2][KT];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, h = lane >> 5;
  const int run = xcd_run(blockIdx.x, gridDim.x);
  int u0, u1;
  run_units(n_units, run, gridDim.x, u0, u1);
  if (u0 == u1) return;
  UnitCursor<QG, KT> uc;
  uc.S = S;
  uc.seek(g0, u0);

  // A operands of the current group: query tile qt (32 queries), k-step ks:
  // row qw0 + 32qt + n, dims 16ks + 8h .. + 7
  int qw0 = 0, qw_last = -1;   // qw_last < qw0 when the wave is past the end
  bf16x8 a[2][KS];

  using Dma = KeyTileDma<DI, KT, RB, NW>;
  uint32_t koff[Dma::CPW];
  Dma::offsets(wave, lane, koff);
  const uint32_t lds_base = (uint32_t)(size_t)(__attribute__((address_space(3))) char *)&lds[0][0];
  auto issue_keys = [&](int b, int k0) {   // into buffer b
    Dma::issue(lds_base + b * T::BYTES, ki, S, k0, wave, koff);
  };
  issue_keys(0, uc.t * KT);
  wait_vmem();
  __syncthreads();

  const float neutral = agg == SP_AGG_MAX ? -INFINITY : 0.f;
  auto op = [agg](float x, float y) { return MAXPOS ? fmaxf(x, y) : agg2(agg, x, y); };
  constexpr int BPW = BQ >= kQW ? 1 : kQW / BQ;   // blocks per wave
  // values a lane keeps per 64-key sub-tile: BPW = 1: the key tile ct = h;
  // BPW >= 2: for each key tile, the blocks bb = h, h + 2, ...
  constexpr int NV = BPW == 1 ? 1 : BPW;

  // One 64-key sub-tile (key tiles ct = 0, 1 of 32 keys): scores of the
  // wave's 64 queries, masked unless FULL (every pair causal and valid),
  // aggregated per selection block. out[v] is the value for key
  // ks0 + 32 ct(v) + n of block bb(v).
  auto subtile = [&](const char *cur, int sb, int ks0, float (&out)[NV], auto full_) {
    constexpr bool FULL = decltype(full_)::value;
    f32x16 acc[2][2];
    // aggregate of key tile ct per selection block, kept in out[] (see above)
    auto reduce_key_tile = [&](int ct) {
      const int s = ks0 + ct * 32 + n;
      float vals[BPW];
#pragma unroll
      for (int bb = 0; bb < BPW; ++bb) vals[bb] = neutral;
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float x[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            x[r] = acc[ct][qt][4 * i + r];
            if constexpr (!MAXPOS) {
              x[r] *= scale;
              if (relu) x[r] = fmaxf(x[r], 0.f);
            }
            if constexpr (!FULL) {
              const int t = qw0 + qt * 32 + i * 8 + h * 4 + r;
              if (!(t <= qw_last && s <= t)) x[r] = neutral;
            }
          }
          // block of query rows 32qt + 8i + 4h + r (a block never splits an 8-row group)
          const int bb = BPW == 1 ? 0 : (qt * 32 + i * 8) / BQ;
          vals[bb] = op(vals[bb], op(op(x[0], x[1]), op(x[2], x[3])));
        }
#pragma unroll
      for (int bb = 0; bb < BPW; ++bb) {
        float m = half_combine(vals[bb], op);
        if constexpr (MAXPOS) {
          m *= scale;
          if (relu) m = fmaxf(m, 0.f);   // -inf (no causal row) becomes 0; never stored
        }
        vals[bb] = m;
      }
      if constexpr (BPW == 1) {
        if (ct == 0) out[0] = vals[0];
        else out[0] = h ? vals[0] : out[0];
      } else {
#pragma unroll
        for (int m = 0; m < BPW / 2; ++m) out[ct * (BPW / 2) + m] = h ? vals[2 * m + 1] : vals[2 * m];
      }
    };
    // key tiles multiplied together: both (four accumulator chains), or one
    // at a time when the 256-dim query operands leave no room
    constexpr int CTP = DI <= 128 ? 2 : 1;
    const char *krow = cur + (sb * 64 + n) * RB + h * 16;
#pragma unroll
    for (int c0 = 0; c0 < 2; c0 += CTP) {
#pragma unroll
      for (int ct = c0; ct < c0 + CTP; ++ct)
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[ct][qt][e] = 0.f;
      // reads of key fragment (ks, ct) run two steps ahead of its products
      // (inline reads with their own lgkmcnt waits; LDS reads complete in order)
      constexpr int NR = KS * CTP, PF = 2, NBF = PF + 1;
      bf16x8 kb[NBF];
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      static_for<0, NR + PF>([&](auto I) {
        constexpr int x = decltype(I)::value;
        if constexpr (x < NR) {   // issue read x
          constexpr int ks = x / CTP, cc = x % CTP;
          asm volatile("ds_read_b128 %0, %1 offset:%2"
                       : "=v"(kb[x % NBF])
                       : "v"((uint32_t)(size_t)(const __attribute__((address_space(3))) char *)krow),
                         "i"((c0 + cc) * 32 * RB + ks * 32));
        }
        if constexpr (x >= PF) {   // products of read x - PF
          constexpr int y = x - PF, ks = y / CTP, ct = y % CTP;
          constexpr int later = (NR - 1 - y < PF ? NR - 1 - y : PF);
          asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(kb[y % NBF]) : "i"(later));
#pragma unroll
          for (int qt = 0; qt < 2; ++qt)
            acc[c0 + ct][qt] = mfma32(a[qt][ks], kb[y % NBF], acc[c0 + ct][qt]);
        }
      });
      if constexpr (CTP == 1) reduce_key_tile(c0);
    }
    if constexpr (CTP == 2) {
      reduce_key_tile(0);
      reduce_key_tile(1);
    }
  };
  // key (within a 64-key sub-tile) and block of kept value v
  auto v_key = [&](int v) { return BPW == 1 ? 32 * h + n : 32 * (v / (BPW / 2)) + n; };
  auto v_block = [&](int v) { return BPW == 1 ? 0 : 2 * (v % (BPW / 2)) + h; };

  // Stores of a tile's block values (b <= 64); issued one tile late so that
  // the wait for the next key tile's loads does not wait for them.
  auto store_tile = [&](const float (&o)[NSUB][NV], int kt0, int qw0_) {
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int s = kt0 + sb * 64 + v_key(v);
        const int tb0 = qw0_ + v_block(v) * BQ;          // first query of the block
        const int tb1 = min(tb0 + BQ, S) - 1;
        if (tb0 < S && s <= tb1) Y[(size_t)(tb0 / BQ) * S + s] = o[sb][v];
      }
  };
  // Tile wholly below the wave's first query (no masks): its 2 NSUB chains of
  // 32 keys (sub-tile sb, key tile ct) form one stream of operand reads and
  // products, and the reduction of each chain runs interleaved with the
  // products of the next, one (query tile, row group) step per operand read,
  // so the vector work issues while the matrix core runs. With DEFER (b <= 64)
  // the last chain's reduction is carried into the next such tile's first
  // chain (the tile-end barrier then does not wait for it); otherwise it
  // follows the products.
  constexpr int NCH = 2 * NSUB, STEPS = 8;
  f32x16 facc[2][2] = {};   // accumulators of chains of even / odd index
  float fvals[2][BPW];    // their block values
  // step st of chain pc's reduction: query tile st / 4, row group st % 4
  auto red_step = [&](auto pc_, auto st_) {
    constexpr int pc = decltype(pc_)::value, st = decltype(st_)::value;
    constexpr int c = pc & 1, qt = st >> 2, i = st & 3;
    if constexpr (st == 0) {
#pragma unroll
      for (int bb = 0; bb < BPW; ++bb) fvals[c][bb] = neutral;
    }
    float x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      x[r] = facc[c][qt][4 * i + r];
      if constexpr (!MAXPOS) {
        x[r] *= scale;
        if (relu) x[r] = fmaxf(x[r], 0.f);
      }
    }
    constexpr int bb = BPW == 1 ? 0 : (qt * 32 + i * 8) / BQ;
    fvals[c][bb] = op(fvals[c][bb], op(op(x[0], x[1]), op(x[2], x[3])));
  };
  // chain pc done: combine the half-waves and keep this lane's values in o
  auto finalize = [&](auto pc_, float (&o)[NSUB][NV]) {
    constexpr int pc = decltype(pc_)::value, c = pc & 1, sb = pc >> 1, ct = pc & 1;
#pragma unroll
    for (int bb = 0; bb < BPW; ++bb) {
      float m = half_combine(fvals[c][bb], op);
      if constexpr (MAXPOS) {
        m *= scale;
        if (relu) m = fmaxf(m, 0.f);
      }
      fvals[c][bb] = m;
    }
    if constexpr (BPW == 1) {
      if constexpr (ct == 0) o[sb][0] = fvals[c][0];
      else o[sb][0] = h ? fvals[c][0] : o[sb][0];
    } else {
#pragma unroll
      for (int m = 0; m < BPW / 2; ++m)
        o[sb][ct * (BPW / 2) + m] = h ? fvals[c][2 * m + 1] : fvals[c][2 * m];
    }
  };
  using LastChain = std::integral_constant<int, NCH - 1>;
  // the carried reduction, on its own (before a masked tile, at the end)
  auto flush = [&](float (&o)[NSUB][NV]) {
    static_for<0, STEPS>([&](auto S_) { red_step(LastChain{}, S_); });
    finalize(LastChain{}, o);
  };
  int pend_kt0 = -1, pend_qw0 = 0;   // tile and query base of the values in pend
  auto full_tile = [&](const char *cur, float (&out)[NSUB][NV], float (&prev)[NSUB][NV],
                       bool carry, auto defer_) {
    constexpr bool DEFER = decltype(defer_)::value;
    constexpr int NR = NCH * KS, PF = 2, NBF = PF + 1;
    bf16x8 kb[NBF];
    const uint32_t kbase =
        (uint32_t)(size_t)(const __attribute__((address_space(3))) char *)(cur + n * RB + h * 16);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    static_for<0, NR + PF>([&](auto I) {
      constexpr int x = decltype(I)::value;
      if constexpr (x < NR) {   // issue read x: chain x / KS, k-step x % KS
        constexpr int ch = x / KS, ks = x % KS;
        constexpr int off = (ch >> 1) * 64 * RB + (ch & 1) * 32 * RB + ks * 32;
        asm volatile("ds_read_b128 %0, %1 offset:%2"
                     : "=v"(kb[x % NBF])
                     : "v"(kbase), "i"(off));
      }
      if constexpr (x >= PF) {   // products of read x - PF, then reduction steps of the previous chain
        constexpr int y = x - PF, ch = y / KS, ks = y % KS, c = ch & 1;
        constexpr int later = (NR - 1 - y < PF ? NR - 1 - y : PF);
        asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(kb[y % NBF]) : "i"(later));
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
          facc[c][qt] = mfma32(a[qt][ks], kb[y % NBF], ks == 0 ? f32x16{} : facc[c][qt]);
        if constexpr (ch >= 1) {
          static_for<ks * STEPS / KS, (ks + 1) * STEPS / KS>(
              [&](auto S_) { red_step(std::integral_constant<int, ch - 1>{}, S_); });
          if constexpr (ks == KS - 1) finalize(std::integral_constant<int, ch - 1>{}, out);
        } else if constexpr (DEFER) {
          // the previous tile's last chain (odd accumulators): reduced here
          // whether or not it is pending, stored only if it is
          static_for<ks * STEPS / KS, (ks + 1) * STEPS / KS>(
              [&](auto S_) { red_step(LastChain{}, S_); });
          if constexpr (ks == KS - 1) {
            finalize(LastChain{}, prev);
            if (carry) store_tile(prev, pend_kt0, pend_qw0);
          }
        }
      }
    });
    if constexpr (!DEFER) flush(out);
  };

  // One key tile; prev holds the values of the tile before (b <= 64: stored
  // here, after its carried chain is reduced if carry). Returns whether this
  // tile's last chain is carried.
  auto tile = [&](int kt0, const char *cur, float (&out)[NSUB][NV], float (&prev)[NSUB][NV],
                  bool carry) -> bool {
    // (DI = 256 keeps one code path: its 128 query registers leave no room
    // for two instantiations of the sub-tile)
    const bool full = DI <= 128 && kt0 + KT - 1 <= qw0 && qw0 + kQW - 1 <= qw_last;
    if (full) {
      if constexpr (DI <= 128) {
        if constexpr (BQ <= kQW) {
          if (!carry && pend_kt0 >= 0) store_tile(prev, pend_kt0, pend_qw0);
          full_tile(cur, out, prev, carry, std::true_type{});
        } else {
          full_tile(cur, out, prev, false, std::false_type{});
        }
      }
    } else {
      if constexpr (BQ <= kQW) {
        if constexpr (DI <= 128)
          if (carry) flush(prev);
        if (pend_kt0 >= 0) store_tile(prev, pend_kt0, pend_qw0);
      }
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb) {
        const int ks0 = kt0 + sb * 64;
#pragma unroll
        for (int v = 0; v < NV; ++v) out[sb][v] = neutral;
        if (ks0 <= qw_last) subtile(cur, sb, ks0, out[sb], std::false_type{});
      }
    }
    if constexpr (BQ > kQW) {
      // BQ = 128: waves 2i and 2i+1 hold the two halves of one block.
      if (wave & 1) {
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb) red[wave >> 1][sb * 64 + v_key(0)] = out[sb][0];
      }
      __syncthreads();
      if (!(wave & 1)) {
        const int tb0 = qw0;
        const int tb1 = min(tb0 + BQ, S) - 1;
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb) {
          const int s = kt0 + sb * 64 + v_key(0);
          const float m = op(out[sb][0], red[wave >> 1][sb * 64 + v_key(0)]);
          if (tb0 < S && s <= tb1) Y[(size_t)(tb0 / BQ) * S + s] = m;
        }
      }
    }
    return BQ <= kQW && full;
  };
  float pend[NSUB][NV];   // block values of the last tile, stored one tile late (b <= 64)
  bool carry = false;     // its last chain's reduction is still pending
  // groups of the run; the key pipeline runs on across group boundaries
  for (int u = u0; u < u1;) {
    const int group = uc.qg, nt = uc.nt;
    qw0 = group * QG + wave * kQW;
    qw_last = min(qw0 + kQW, S) - 1;
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      const int row = min(qw0 + qt * 32 + n, S - 1);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        a[qt][ks] = as_bf16x8(ldg16(qi + (size_t)row * DI + ks * 16 + h * 8));
    }
    const int t_end = min(nt, uc.t + (u1 - u));
    for (int t = uc.t; t < t_end; ++t, ++u) {
      if (u + 1 < u1) issue_keys((u - u0 + 1) & 1, t + 1 < nt ? (t + 1) * KT : 0);
      float out[NSUB][NV];
      carry = tile(t * KT, lds[(u - u0) & 1], out, pend, carry);
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
        for (int v = 0; v < NV; ++v) pend[sb][v] = out[sb][v];
      pend_kt0 = t * KT;
      pend_qw0 = qw0;
      // the next tile's keys (and the stores of the tile before) have landed
      wait_vmem();
      __syncthreads();
    }
    uc.next_group();
  }
  if constexpr (BQ <= kQW) {
    if constexpr (DI <= 128)
      if (carry) flush(pend);
    store_tile(pend, pend_kt0, pend_qw0);
  }
}

template <int DI, bool VEC>
__global__ __launch_bounds__(256) void indexer_rows_kernel(int S, int qo, int relu, float scale,
                                                           const uint16_t *__restrict__ qi,
                                                           const uint16_t *__restrict__ ki,
                                                           float *__restrict__ Z) {
  constexpr int NT = 256, NW = 4;
  constexpr int KT = Tile<DI>::KT, RB = Tile<DI>::RB, KS = Tile<DI>::KS;
  constexpr int QG = NW * kQW;
  constexpr int KR = KT / 16;          // 16-key row tiles of a key tile
  constexpr int SRB = KT * 4 + 16;     // staging row stride: 16 rows of a 16-byte write on distinct banks
  constexpr int LPR = KT * 4 / 16;     // lanes per staged row
  constexpr int RPI = 64 / LPR;        // rows per store instruction
  __shared__ __align__(16) char lds[2][Tile<DI>::BYTES];
  __shared__ __align__(16) char stage_rows[NW][16 * SRB];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  char *stg = stage_rows[wave];
  const int q0 = qo + blockIdx.x * QG;   // qi and Z are addressed by position
  const int k_begin = blockIdx.y * kKC;
  const int q_last = min(q0 + QG, S) - 1;
  if (k_begin > q_last) return;
  const int k_end = min(k_begin + kKC, q_last + 1);
  const int ntiles = (k_end - k_begin + KT - 1) / KT;
  const int qw0 = q0 + wave * kQW;
  const int qw_last = min(qw0 + kQW, S) - 1;

  // Queries are the B operand: lane holds query column c16 of tile qc.
  bf16x8 bq[4][KS];
#pragma unroll
  for (int qc = 0; qc < 4; ++qc) {
    const int row = min(qw0 + qc * 16 + c16, S - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      bq[qc][ks] = as_bf16x8(ldg16(qi + (size_t)row * DI + ks * 32 + g * 8));
  }

  KeyStage<DI, NT> stage;
  stage.load(ki, S, k_begin, tid);
  stage.store(lds[0], tid);
  __syncthreads();

  for (int it = 0; it < ntiles; ++it) {
    const int kt0 = k_begin + it * KT;
    const bool more = it + 1 < ntiles;
    if (more) stage.load(ki, S, kt0 + KT, tid);
    const char *cur = lds[it & 1];
    if (kt0 <= qw_last) {
      // One 16-query piece at a time (K fragments are re-read from LDS per
      // piece; this kernel is bound by its stores): acc[kr] holds keys
      // kt0 + 16kr + 4g .. +3 of query qw0 + 16qc + c16. The scaled scores
      // go to the wave's staging rows (row c16, keys 16kr + 4g .. +3), are
      // read back one row segment per LPR lanes and stored as whole rows of
      // the tile: RPI query rows of KT consecutive keys per instruction,
      // where a store straight from the MFMA layout would touch 16 rows.
#pragma unroll
      for (int qc = 0; qc < 4; ++qc) {
        const int tq0 = qw0 + qc * 16;
        if (tq0 > qw_last || kt0 > tq0 + 15) continue;   // no causal pair (wave-uniform)
        f32x4 acc[KR];
#pragma unroll
        for (int kr = 0; kr < KR; ++kr) {
          acc[kr] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            acc[kr] = mfma16(as_bf16x8(lds16(cur + (kr * 16 + c16) * RB + ks * 64 + g * 16)),
                             bq[qc][ks], acc[kr]);
        }
#pragma unroll
        for (int kr = 0; kr < KR; ++kr) {
          float4 x;
          x.x = acc[kr][0] * scale;
          x.y = acc[kr][1] * scale;
          x.z = acc[kr][2] * scale;
          x.w = acc[kr][3] * scale;
          if (relu) {
            x.x = x.x > 0.f ? x.x : 0.f;
            x.y = x.y > 0.f ? x.y : 0.f;
            x.z = x.z > 0.f ? x.z : 0.f;
            x.w = x.w > 0.f ? x.w : 0.f;
          }
          *reinterpret_cast<float4 *>(stg + c16 * SRB + kr * 64 + g * 16) = x;
        }
        // the reads below take other lanes' rows
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int j = 0; j < 16 / RPI; ++j) {
          const int rr = j * RPI + lane / LPR, cc = lane % LPR;
          const float4 x = *reinterpret_cast<const float4 *>(stg + rr * SRB + cc * 16);
          const int t = tq0 + rr, s0 = kt0 + cc * 4;
          float *dst = Z + (size_t)t * S + s0;
          if (t > qw_last || s0 > t) continue;
          if (s0 + 3 <= t) {
            if constexpr (VEC) {
              *reinterpret_cast<float4 *>(dst) = x;
            } else {
              dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w;
            }
          } else {
            // the diagonal: a loop, so that its first store is not merged
            // with the 16-byte store above (which would split that store)
#pragma unroll 1
            for (int r = 0; s0 + r <= t; ++r)
              dst[r] = r == 0 ? x.x : (r == 1 ? x.y : x.z);
          }
        }
        // the next piece's writes reuse the rows just read
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    }
    if (more) stage.store(lds[(it + 1) & 1], tid);
    __syncthreads();
  }
}

// Per-device caches of the persistent launch: compute units per device, and
// resident workgroups per CU for each kernel instance K (instances differ in
// LDS and registers, so each has its own entry).
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];
template <auto K>
struct Residency {
  static inline std::atomic<int> per_cu[kMaxDevices];
};

// Launches kernel K as a persistent grid: as many workgroups as are resident
// on the current device at once (CUs times K's occupancy), at most one per
// unit of work.
template <auto K, class... Args>
hipError_t launch_persistent(int threads, int n_units, hipStream_t st, Args... args) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  int c = g_cus[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    e = hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    g_cus[dev].store(c, std::memory_order_relaxed);
  }
  int w = Residency<K>::per_cu[dev].load(std::memory_order_relaxed);
  if (w == 0) {
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&w, K, threads, 0);
    if (e != hipSuccess) return e;
    w = w < 1 ? 1 : w;
    Residency<K>::per_cu[dev].store(w, std::memory_order_relaxed);
  }
  const int grid = n_units < c * w ? n_units : c * w;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(K, dim3(grid), dim3(threads), 0, st, args...);
  return hipGetLastError();
}

template <int DI>
hipError_t launch_di(const Prob &p, const void *qi, const void *ki, float *scores,
                     hipStream_t st) {
  // chunk rows (a call starting at position qo) are addressed by position:
  // q_idx and per-query scores are shifted back by qo rows, block scores by
  // qo / b rows
  const uint16_t *q = (const uint16_t *)qi - (size_t)p.qo * DI, *k = (const uint16_t *)ki;
  if (p.b == 1) {
    float *z = scores - (size_t)p.qo * p.S;
    dim3 grid((p.nq + 255) / 256, (p.S + kKC - 1) / kKC);
    if (p.S % 4 == 0)
      hipLaunchKernelGGL((indexer_rows_kernel<DI, true>), grid, dim3(256), 0, st, p.S, p.qo,
                         p.relu, p.iscale, q, k, z);
    else
      hipLaunchKernelGGL((indexer_rows_kernel<DI, false>), grid, dim3(256), 0, st, p.S, p.qo,
                         p.relu, p.iscale, q, k, z);
    return hipGetLastError();
  }
  constexpr int NW = 8, QG = NW * kQW;
  const int g0 = p.qo / QG;   // a multiple of the query group (checked)
  float *y = scores - (size_t)(p.qo / p.b) * p.S;
  const long long units = count_units<QG, BlockTile<DI>::KT>(p.S, g0);
  if (units > INT_MAX) return hipErrorInvalidValue;
  const int n_units = (int)units;
  const bool maxpos = p.agg == SP_AGG_MAX && p.iscale >= 0.f;
#define SP_BLK(BQ)                                                                           \
  if (maxpos)                                                                                \
    err = launch_persistent<indexer_block_kernel<DI, BQ, true, NW>>(                         \
        NW * 64, n_units, st, p.S, g0, n_units, p.agg, p.relu, p.iscale, q, k, y);           \
  else                                                                                       \
    err = launch_persistent<indexer_block_kernel<DI, BQ, false, NW>>(                        \
        NW * 64, n_units, st, p.S, g0, n_units, p.agg, p.relu, p.iscale, q, k, y)
  hipError_t err;
  switch (p.b) {
    case 16: SP_BLK(16); break;
    case 32: SP_BLK(32); break;
    case 64: SP_BLK(64); break;
    default: SP_BLK(128); break;
  }
#undef SP_BLK
  return err;
}

}  // namespace

bool indexer_mfma_supported(const Prob &p) {
  // a chunked call of the block kernel starts on one of its 512-query groups
  return p.dtype == SP_DTYPE_BF16 && (p.di == 64 || p.di == 128 || p.di == 256) &&
         (p.b == 1 ||
          ((p.b == 16 || p.b == 32 || p.b == 64 || p.b == 128) && p.qo % 512 == 0));
}

hipError_t launch_indexer_mfma(const Prob &p, const void *qi, const void *ki, float *scores,
                               hipStream_t st) {
  if (p.di == 64) return launch_di<64>(p, qi, ki, scores, st);
  if (p.di == 128) return launch_di<128>(p, qi, ki, scores, st);
  return launch_di<256>(p, qi, ki, scores, st);
}

}  // namespace sp
