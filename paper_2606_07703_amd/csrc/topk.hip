// Top-k support selection per score row (Section 4.1 TopK; Section 4.2;
// Algorithm 1, selection and restricted recomputation; Algorithm 2, selection and sparse GQA prefill).
//
// Row r has L = t1_r+1 causal positions. If L <= k every position is taken.
// Otherwise the Wf = min(W, k) most recent positions are forced and the
// other k' = k-Wf are chosen among positions [0, L-Wf) in the order
// (score descending, position ascending).
//
// Keys are the order-preserving uint32 images of the fp32 scores (-0 and +0
// share one key). One workgroup per row finds the exact k'-th largest key T
// with three radix passes over LDS histograms (11, 11 and 10 bits; each pass
// counts only keys sharing the prefix fixed so far). The chosen set is then
// {key > T} plus the first (k' - #{key > T}) positions with key == T, and a
// final ordered pass compacts the chosen positions with block-wide prefix
// sums, so every output row comes out ascending without a sort.
//
// topk_reg_kernel keeps the row in registers (each thread owns runs of 16
// consecutive positions) for rows of up to 32768 candidates; the exact zero
// keys that ReLU produces in bulk are counted by wave ballots instead of
// contended LDS atomics, and when few keys share the threshold's top 22 bits
// they are ranked directly instead of by the third pass. topk_rows_kernel
// streams longer rows from memory on every pass, 512 threads a row.
#include "common.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

constexpr uint32_t kZeroKey = 0x80000000u;   // float_key(+0.0f)
// Word 3 of a raw buffer resource on gfx950: 32-bit data format, no swizzle.
constexpr int kTopkBufferDword3 = 0x00020000;

__device__ __forceinline__ int digit_shift(int pass) { return pass == 0 ? 21 : (pass == 1 ? 10 : 0); }
__device__ __forceinline__ int digit_bits(int pass) { return pass == 2 ? 10 : 11; }

// Exclusive prefix over a block of NT threads of per-thread values whose set
// bits all lie in MASK, and the block total: bit-sliced wave ballots (no LDS
// round trips inside a wave), then one barrier to combine the wave totals.
// `row` selects a scratch row: consecutive scans must alternate rows (a row
// is written again only after the barrier of the scan in between).
template <int NT, uint32_t MASK>
__device__ __forceinline__ uint32_t scan_bits(uint32_t v, uint32_t (*scratch)[NT / 64], int row,
                                              uint32_t *total) {
  constexpr int NW = NT / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t excl = 0, wtot = 0;
#pragma unroll
  for (int bit = 0; bit < 32; ++bit) {
    if (!((MASK >> bit) & 1u)) continue;
    const uint64_t m = __ballot((v >> bit) & 1u);
    excl += __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                      __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u)) << bit;
    wtot += (uint32_t)__popcll(m) << bit;
  }
  if (lane == 0) scratch[row][wave] = wtot;
  __syncthreads();
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const uint32_t t = scratch[row][w];
    base += w < wave ? t : 0u;
    tot += t;
  }
  *total = tot;
  return base + excl;
}

// Given NC interleaved copies of a filled histogram of nb bins (bin i of
// copy c at hist[i*NC + c]), less subcnt in bin subbin (padding keys counted
// there), find the bin holding the `remaining`-th largest key; writes (bin,
// rank within bin) to sel. CMASK covers the bits of a thread's count (the
// keys of its bins). Every thread must call it (it contains barriers).
template <int NT, uint32_t CMASK, int NC = 1>
__device__ __forceinline__ void find_digit(const uint32_t *hist, int nb, uint32_t remaining,
                                           uint32_t (*scratch)[NT / 64], int row,
                                           uint32_t *sel, int subbin = 0, uint32_t subcnt = 0) {
  const int tid = threadIdx.x;
  const int per = nb / NT;            // nb is a multiple of NT
  const int hi = nb - tid * per;      // thread 0 owns the highest bins
  auto bin = [&](int i) {
    uint32_t c = 0;
#pragma unroll
    for (int x = 0; x < NC; ++x) c += hist[i * NC + x];
    return i == subbin ? c - subcnt : c;
  };
  uint32_t mine = 0;
  for (int i = hi - per; i < hi; ++i) mine += bin(i);
  uint32_t total;
  const uint32_t above = scan_bits<NT, CMASK>(mine, scratch, row, &total);
  if (above < remaining && above + mine >= remaining) {
    uint32_t acc = above;
    for (int i = hi - 1; i >= hi - per; --i) {
      const uint32_t c = bin(i);
      if (acc + c >= remaining) {
        sel[0] = (uint32_t)i;
        sel[1] = remaining - acc;
        break;
      }
      acc += c;
    }
  }
  __syncthreads();
}

// Row of workgroup i of n. Row r has (r + 1) b candidates, so the first half
// of the grid takes the rows from the longest down and the second half from
// the shortest up: workgroups i and i + n/2, which the dispatcher places on
// one CU when the grid is two workgroups per CU, then hold rows of equal
// total length, and a longer grid starts its longest rows first.
__device__ __forceinline__ int row_of(int i, int n) {
  const int half = (n + 1) / 2;
  return i < half ? n - 1 - i : i - half;
}

// ------------------------------------------------------------ register rows
constexpr int kRegNT = 512;
constexpr int kRun = 16;                      // consecutive positions per run
constexpr int kRegSub = 4;                    // runs per thread
constexpr int kRegCap = kRegNT * kRun * kRegSub;   // 32768 candidates
// The first digit's histogram has kCopies interleaved copies, lane l counting
// into copy l % kCopies: block-aggregated scores crowd into a few top bins,
// and the copies (adjacent words, so different banks) cut the conflicts of
// one wave's atomics on them; the later digits, over keys sharing the first,
// spread out and use one copy.
constexpr int kCopies = 4;
// Keys sharing the 22-bit prefix of T gathered for a direct search (at most
// one per thread) instead of the third histogram pass.
constexpr int kCand = 256;

// Two workgroups per CU (16 waves: at most 128 registers a wave), so that a
// long row and a short one share each CU (see row_of).
//
// PACKED (every row starts 16-byte aligned): the row is read by 16-byte
// loads through a buffer resource whose range ends at the row's last
// candidate. Raw buffer loads check that range per dword: the dwords past it
// read as zeros without touching memory, also inside a load that straddles
// it, so no position is tested and no load is guarded; those npad padding
// positions are zero keys, taken out of the zero key's bin. The loads hold
// raw fp32 bits until the first pass forms each run's keys and counts them
// in load order, so its LDS atomics overlap the loads still in flight (the
// row load is the largest single cost of a long row). Otherwise each
// position is tested at load time and padding holds key 0, taken out of
// bin 0 while every digit fixed so far is 0.
template <bool PACKED>
__global__ __launch_bounds__(kRegNT) __attribute__((amdgpu_waves_per_eu(4, 4))) void
topk_reg_kernel(int S, int qo, int b, int k, int W, const float *__restrict__ scores,
                int32_t *__restrict__ idx) {
  constexpr int NT = kRegNT;
  constexpr int kHist = kCopies * 2048;
  // histogram copies, then one discard word per lane (counts of keys outside
  // the digit's prefix go there, so every key costs one unconditional
  // atomic and no branch); after the passes, the output row is staged here
  __shared__ uint32_t hist[kHist + 64];
  __shared__ uint32_t scratch[2][NT / 64];
  __shared__ uint32_t sel[3];

  const int r = row_of((int)blockIdx.x, (int)gridDim.x);
  const int tid = threadIdx.x, lane = tid & 63;
  const int t1 = min(qo + r * b + b, S) - 1;   // rows count blocks from the chunk start
  const int L = t1 + 1;
  // blockIdx.y: the KV group of a per-group table (0 for a shared one)
  const size_t row_id = (size_t)blockIdx.y * gridDim.x + r;
  int32_t *out = idx + row_id * k;
  const float *row = scores + row_id * S;
  if (L <= k) {
    for (int c = tid; c < k; c += NT) out[c] = c < L ? c : -1;
    return;
  }
  const int Wf = min(W, k);
  const int nc = L - Wf;
  const int kp = k - Wf;
  const int nsub = (nc + NT * kRun - 1) / (NT * kRun);   // runs in use (<= kRegSub)

  // Run j of thread t covers positions [kRun*(t + NT*j), +kRun); npad
  // positions of the runs in use lie at or past nc.
  constexpr uint32_t kPadKey = 0u;   // padding key when !PACKED
  const uint32_t npad = (uint32_t)(nsub * NT * kRun - nc);
  uint32_t key[kRegSub][kRun];
  if constexpr (PACKED) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(row), (short)0,
                                                      (uint32_t)nc * 4u, kTopkBufferDword3);
#pragma unroll
    for (int j = 0; j < kRegSub; ++j) {
      const uint32_t off = (uint32_t)(kRun * (tid + NT * j)) * 4u;
#pragma unroll
      for (int i = 0; i < kRun; i += 4) {
        // unconditional: a run past nc reads zeros without touching memory,
        // and the waits of the first pass then count loads exactly
        const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(rs, off + i * 4, 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) key[j][i + e] = x[e];
      }
    }
  } else {
    const bool vec = (((row_id * S) & 3) == 0);   // row start 16-byte aligned
#pragma unroll
    for (int j = 0; j < kRegSub; ++j) {
      const int p0 = kRun * (tid + NT * j);
#pragma unroll
      for (int i = 0; i < kRun; i += 4) {
        float f[4] = {0.f, 0.f, 0.f, 0.f};
        if (j < nsub) {
          if (vec && p0 + i + 3 < nc) {
            const float4 x = *reinterpret_cast<const float4 *>(row + p0 + i);
            f[0] = x.x; f[1] = x.y; f[2] = x.z; f[3] = x.w;
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (p0 + i + e < nc) f[e] = row[p0 + i + e];
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          key[j][i + e] = p0 + i + e < nc ? float_key(f[e]) : kPadKey;
      }
    }
  }
  // bin of digit `shift` that the padding keys fall in, if they share `prefix`
  auto pad_bin = [&](int shift, uint32_t dmask, uint32_t prefix, uint32_t pmask) -> int {
    const uint32_t pk = PACKED ? kZeroKey : kPadKey;
    return (pk & pmask) == prefix ? (int)((pk >> shift) & dmask) : -1;
  };

  uint32_t T = 0xffffffffu, remaining = 0;
  uint32_t ties = 0;   // candidates whose key equals T
  if (kp > 0) {
    uint32_t prefix = 0, pmask = 0;
    remaining = (uint32_t)kp;
    uint32_t *discard = hist + kHist + lane;
    // one radix pass; FIRST: the first digit, whose pass also forms the keys
    // when PACKED
    auto run_pass = [&](int pass, auto first_) {
      constexpr bool FORM = PACKED && decltype(first_)::value;
      const int shift = digit_shift(pass), nb = 1 << digit_bits(pass);
      const uint32_t dmask = (uint32_t)nb - 1u;
      const int nco = pass == 0 ? kCopies : 1;   // histogram copies of this digit
      uint32_t *hc = hist + (pass == 0 ? lane % kCopies : 0);
      for (int i = tid; i < nb * nco; i += NT) hist[i] = 0;
      if constexpr (FORM) {
        // LDS-only barrier: the clears are visible, the row loads stay in flight
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
      } else {
        __syncthreads();
      }
      uint32_t zc = 0;
      // opaque to the compiler, so the per-key zero tests stay inside the
      // pass instead of being hoisted out as 64 saved lane masks
      uint32_t zkey = kZeroKey;
      asm volatile("" : "+s"(zkey));
#pragma unroll
      for (int j = 0; j < kRegSub; ++j) {
        if (j >= nsub) continue;   // uniform
#pragma unroll
        for (int i = 0; i < kRun; ++i) {
          uint32_t kv = key[j][i];
          if constexpr (FORM) {
            kv = float_key(__uint_as_float(kv));
            key[j][i] = kv;
          }
          const bool in = (kv & pmask) == prefix;
          const bool zero = kv == zkey;
          zc += (in && zero) ? 1u : 0u;
          atomicAdd(in && !zero ? &hc[((kv >> shift) & dmask) * nco] : discard, 1u);
        }
      }
      if ((kZeroKey & pmask) == prefix) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) zc += __shfl_xor(zc, off, 64);
        if (lane == 0 && zc) atomicAdd(&hist[((kZeroKey >> shift) & dmask) * nco], zc);
      }
      __syncthreads();
      const int pb = pad_bin(shift, dmask, prefix, pmask);
      const uint32_t pc = pb >= 0 ? npad : 0u;
      if (pass == 0)
        find_digit<NT, 0xffffu, kCopies>(hist, nb, remaining, scratch, 0, sel, pb, pc);
      else
        find_digit<NT, 0xffffu>(hist, nb, remaining, scratch, pass & 1, sel, pb, pc);
      // the chosen bin's keys: after the second digit, the candidates of the
      // third; after the last digit, exactly the keys equal to T
      if (pass >= 1) ties = hist[sel[0]] - (pb == (int)sel[0] ? npad : 0u);
      prefix |= sel[0] << shift;
      pmask |= dmask << shift;
      remaining = sel[1];
      __syncthreads();
    };
    run_pass(0, std::true_type{});
    run_pass(1, std::false_type{});
    // Third digit. When few keys share the 22-bit prefix (and no zero or
    // padding key does), they are gathered into LDS and T is found among
    // them directly: each gathered key counts the gathered keys above it
    // and equal to it. Otherwise a third histogram pass.
    const uint32_t pad_key = PACKED ? kZeroKey : kPadKey;
    if (ties <= kCand && (kZeroKey & pmask) != prefix && (pad_key & pmask) != prefix) {
      const uint32_t n1 = ties;
      uint32_t *cnt = hist + kHist;   // a discard word, free after the passes
      if (tid == 0) *cnt = 0u;
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kRegSub; ++j) {
        if (j >= nsub) continue;   // uniform
#pragma unroll
        for (int i = 0; i < kRun; ++i) {
          const uint32_t kv = key[j][i];
          if ((kv & pmask) == prefix) hist[atomicAdd(cnt, 1u)] = kv;
        }
      }
      __syncthreads();
      if (tid < (int)n1) {
        const uint32_t v = hist[tid];
        uint32_t above = 0, same = 0;
        for (uint32_t c = 0; c < n1; ++c) {
          const uint32_t u = hist[c];
          above += u > v ? 1u : 0u;
          same += u == v ? 1u : 0u;
        }
        // v is T: the remaining-th largest of the gathered keys (equal keys
        // write the same values)
        if (above < remaining && remaining <= above + same) {
          sel[0] = v;
          sel[1] = remaining - above;
          sel[2] = same;
        }
      }
      __syncthreads();
      T = sel[0];
      remaining = sel[1];
      ties = sel[2];
    } else {
      run_pass(2, std::false_type{});
      T = prefix;
    }
  }
  // (kp = 0: nothing is chosen; unformed PACKED keys are never read)

  // Ordered emission, one run index j at a time (runs of index j, in thread
  // order, cover positions [kRun*NT*j, kRun*NT*(j+1)) in order). Chosen
  // positions are written to their output slot in LDS (hist, free after the
  // passes) when the row fits, then copied out with coalesced stores.
  //
  // When every key equal to T is taken (the usual case: T is one key), the
  // chosen set is {key >= T}: one mask and one count per run.
  auto emit_all = [&](auto staged_tag) {
    constexpr bool STAGED = decltype(staged_tag)::value;
    uint32_t before = 0;
#pragma unroll
    for (int j = 0; j < kRegSub; ++j) {
      if (j >= nsub) break;   // uniform
      const int p0 = kRun * (tid + NT * j);
      const int nv = min(max(nc - p0, 0), kRun);   // this run's real positions
      uint32_t take = 0;
#pragma unroll
      for (int i = 0; i < kRun; ++i) take |= key[j][i] >= T ? 1u << i : 0u;
      take &= (1u << nv) - 1u;   // nv <= 16
      uint32_t total;
      const uint32_t ex =
          scan_bits<NT, 0x1fu>((uint32_t)__popc(take), scratch, (j + 1) & 1, &total);
      uint32_t pos = before + ex;
      while (take) {
        const int i = __builtin_ctz(take);
        take &= take - 1u;
        if constexpr (STAGED)
          hist[pos] = (uint32_t)(p0 + i);
        else if (pos < (uint32_t)kp)   // always true for consistent counts
          out[pos] = p0 + i;
        ++pos;
      }
      before += total;
    }
  };
  auto emit = [&](auto staged_tag) {
    constexpr bool STAGED = decltype(staged_tag)::value;
    uint32_t gt_before = 0, eq_before = 0;
#pragma unroll
    for (int j = 0; j < kRegSub; ++j) {
      if (j >= nsub) break;   // uniform
      const int p0 = kRun * (tid + NT * j);
      const int nv = min(max(nc - p0, 0), kRun);   // this run's real positions
      // bit i: key i of the run is above T / equal to T
      uint32_t gtm = 0, eqm = 0;
#pragma unroll
      for (int i = 0; i < kRun; ++i) {
        gtm |= key[j][i] > T ? 1u << i : 0u;
        eqm |= key[j][i] == T ? 1u << i : 0u;
      }
      const uint32_t vmask = (1u << nv) - 1u;   // nv <= 16
      gtm &= vmask;
      eqm &= vmask;
      const uint32_t cgt = (uint32_t)__popc(gtm), ceq = (uint32_t)__popc(eqm);
      uint32_t total;
      // counts of at most 16 each: bits 0..4 and 16..20
      const uint32_t ex =
          scan_bits<NT, 0x1f001fu>((cgt << 16) | ceq, scratch, (j + 1) & 1, &total);
      const uint32_t my_gt = gt_before + (ex >> 16);
      const uint32_t my_eq = eq_before + (ex & 0xffffu);
      // chosen: every key above T, and the first (remaining - my_eq) of the
      // run's keys equal to T (none once my_eq reaches remaining; written
      // without a wrapping subtraction)
      const uint32_t used = min(my_eq, remaining);
      uint32_t neq = min(remaining - used, ceq);
      uint32_t take = gtm, e = eqm;
      for (; neq > 0; --neq) {
        const uint32_t low = e & (0u - e);
        take |= low;
        e ^= low;
      }
      // chosen positions in order, from this run's first output slot
      uint32_t pos = my_gt + used;
      while (take) {
        const int i = __builtin_ctz(take);
        take &= take - 1u;
        if constexpr (STAGED)
          hist[pos] = (uint32_t)(p0 + i);
        else if (pos < (uint32_t)kp)   // always true for consistent counts
          out[pos] = p0 + i;
        ++pos;
      }
      gt_before += total >> 16;
      eq_before += total & 0xffffu;
    }
  };
  if (kp > 0) {
    const bool all = ties == remaining;   // uniform
    if (kp <= kHist) {
      if (all)
        emit_all(std::true_type{});
      else
        emit(std::true_type{});
      __syncthreads();
      for (int c = tid; c < kp; c += NT) out[c] = (int32_t)hist[c];
    } else if (all) {
      emit_all(std::false_type{});
    } else {
      emit(std::false_type{});
    }
  }
  for (int c = tid; c < Wf; c += NT) out[kp + c] = nc + c;
}

// -------------------------------------------------------------- streamed rows
constexpr int kNT = 512;
constexpr int kEmitPer = 16;
constexpr int kEmitChunk = kNT * kEmitPer;
constexpr int kEmitStride = kNT + 4;   // LDS column stride: conflict-free writes and reads

// VEC: every row starts 16-byte aligned and S % 4 == 0, so the passes read
// four keys per load through range-checked buffer loads, the next step's in
// flight while a step is counted; otherwise one key per load, and the
// emission stages its keys in LDS.
template <bool VEC>
__global__ __launch_bounds__(kNT) void topk_rows_kernel(int S, int qo, int b, int k, int W,
                                                        const float *__restrict__ scores,
                                                        int32_t *__restrict__ idx) {
  __shared__ uint32_t hist[2048];
  __shared__ uint32_t scratch[2][kNT / 64];
  __shared__ uint32_t sel[2];

  const int r = row_of((int)blockIdx.x, (int)gridDim.x);
  const int tid = threadIdx.x, lane = tid & 63;
  const int t1 = min(qo + r * b + b, S) - 1;   // rows count blocks from the chunk start
  const int L = t1 + 1;
  // blockIdx.y: the KV group of a per-group table (0 for a shared one)
  const size_t row_id = (size_t)blockIdx.y * gridDim.x + r;
  int32_t *out = idx + row_id * k;
  const float *row = scores + row_id * S;

  if (L <= k) {
    for (int c = tid; c < k; c += kNT) out[c] = c < L ? c : -1;
    return;
  }
  const int Wf = min(W, k);
  const int nc = L - Wf;
  const int kp = k - Wf;

  uint32_t T = 0xffffffffu;
  uint32_t remaining = 0;
  if (kp > 0) {
    uint32_t prefix = 0, pmask = 0;
    remaining = (uint32_t)kp;
#pragma unroll 1
    for (int pass = 0; pass < 3; ++pass) {
      const int shift = digit_shift(pass), nb = 1 << digit_bits(pass);
      const uint32_t dmask = (uint32_t)nb - 1u;
      for (int i = tid; i < nb; i += kNT) hist[i] = 0;
      __syncthreads();
      uint32_t zc = 0;
      auto count = [&](uint32_t kv) {
        if ((kv & pmask) == prefix) {
          if (kv == kZeroKey) ++zc;
          else atomicAdd(&hist[(kv >> shift) & dmask], 1u);
        }
      };
      if constexpr (VEC) {
        // A step covers 16 NT positions: thread tid reads positions
        // 4(tid + NT u) .. +3 for u < 4, through a buffer resource ranged to
        // the nc candidates (reads past them return zeros, which are not
        // counted). The loads are unconditional, so the next step's are in
        // flight while this step is counted.
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(row), (short)0,
                                                          (uint32_t)nc * 4u, kTopkBufferDword3);
        constexpr int kStep = 16 * kNT;
        auto load = [&](u32x4 (&x)[4], int base) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            x[u] = __builtin_amdgcn_raw_buffer_load_b128(
                rs, (uint32_t)(base + 4 * (tid + kNT * u)) * 4u, 0, 0);
        };
        auto counts = [&](const u32x4 (&x)[4], int base) {
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int p0 = base + 4 * (tid + kNT * u);
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (p0 + e < nc) count(float_key(__uint_as_float(x[u][e])));
          }
        };
        u32x4 xa[4], xb[4];
        load(xa, 0);
        for (int base = 0; base < nc; base += 2 * kStep) {
          load(xb, base + kStep);
          counts(xa, base);
          load(xa, base + 2 * kStep);
          counts(xb, base + kStep);
        }
      } else {
        for (int i = tid; i < nc; i += kNT) count(float_key(row[i]));
      }
      if ((kZeroKey & pmask) == prefix) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) zc += __shfl_xor(zc, off, 64);
        if (lane == 0 && zc) atomicAdd(&hist[(kZeroKey >> shift) & dmask], zc);
      }
      __syncthreads();
      // a thread's bins can hold more than 65535 of a long row's keys
      find_digit<kNT, 0xffffffffu>(hist, nb, remaining, scratch, pass & 1, sel);
      prefix |= sel[0] << shift;
      pmask |= dmask << shift;
      remaining = sel[1];
      __syncthreads();
    }
    T = prefix;
  }

  // Ordered emission over candidates in chunks of kEmitChunk positions;
  // thread tid takes the kEmitPer consecutive positions from kEmitPer * tid.
  uint32_t gt_before = 0, eq_before = 0;
  int srow = 1;
  // Counts a chunk's keys above and on the threshold, scans them over the
  // block and writes the chosen positions (key(e) is the key at lo + e).
  auto emit_chunk = [&](int base, auto key) {
    const int lo = base + tid * kEmitPer;
    uint32_t cgt = 0, ceq = 0;
#pragma unroll
    for (int e = 0; e < kEmitPer; ++e) {
      if (lo + e < nc) {
        const uint32_t kv = key(e);
        cgt += kv > T;
        ceq += kv == T;
      }
    }
    uint32_t total;
    const uint32_t ex = scan_bits<kNT, 0x1f001fu>((cgt << 16) | ceq, scratch, srow, &total);
    srow ^= 1;
    uint32_t my_gt = gt_before + (ex >> 16);
    uint32_t my_eq = eq_before + (ex & 0xffffu);
    uint32_t pos = my_gt + min(my_eq, remaining);
#pragma unroll
    for (int e = 0; e < kEmitPer; ++e) {
      if (lo + e < nc) {
        const uint32_t kv = key(e);
        bool take = kv > T;
        if (kv == T) {
          take = my_eq < remaining;
          ++my_eq;
        }
        if (take) {
          if (pos < (uint32_t)kp) out[pos] = lo + e;   // always true for consistent counts
          ++pos;
        }
      }
    }
    gt_before += total >> 16;
    eq_before += total & 0xffffu;
  };
  if constexpr (VEC) {
    // Each thread's 16 positions are four 16-byte loads through a buffer
    // resource ranged to the candidates (zeros past nc, not counted); the
    // next chunk's loads are in flight while a chunk is counted and emitted.
    // No LDS staging: scan_bits alternates its two scratch rows, so one
    // barrier per chunk (inside the scan) suffices.
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(row), (short)0,
                                                      (uint32_t)nc * 4u, kTopkBufferDword3);
    auto load = [&](u32x4 (&x)[4], int base) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
        x[u] = __builtin_amdgcn_raw_buffer_load_b128(
            rs, (uint32_t)(base + tid * kEmitPer + 4 * u) * 4u, 0, 0);
    };
    u32x4 xa[4], xb[4];
    load(xa, 0);
    for (int base = 0; base < nc; base += 2 * kEmitChunk) {
      load(xb, base + kEmitChunk);
      emit_chunk(base, [&](int e) { return float_key(__uint_as_float(xa[e >> 2][e & 3])); });
      load(xa, base + 2 * kEmitChunk);
      if (base + kEmitChunk < nc)
        emit_chunk(base + kEmitChunk,
                   [&](int e) { return float_key(__uint_as_float(xb[e >> 2][e & 3])); });
    }
  } else {
    // Keys pass through LDS: position q of a chunk sits at
    // (q % kEmitPer) * kEmitStride + q / kEmitPer.
    __shared__ uint32_t keys[kEmitPer * kEmitStride];
    for (int base = 0; base < nc; base += kEmitChunk) {
      const int n = min(kEmitChunk, nc - base);
      for (int i = tid; i < kEmitChunk; i += kNT)
        keys[(i % kEmitPer) * kEmitStride + i / kEmitPer] = i < n ? float_key(row[base + i]) : 0u;
      __syncthreads();
      emit_chunk(base, [&](int e) { return keys[e * kEmitStride + tid]; });
      __syncthreads();
    }
  }
  for (int c = tid; c < Wf; c += kNT) out[kp + c] = nc + c;
}

}  // namespace

hipError_t launch_topk(const Prob &p, const float *scores, int32_t *idx, hipStream_t st) {
  // Longest candidate range of any row: the last block's causal length minus the window.
  const int Lmax = min(p.qo + p.R * p.b, p.S);
  const int ncmax = Lmax - min(p.W, p.k);
  // every row starts 16-byte aligned
  const bool packed = ((uintptr_t)scores & 15) == 0 && p.S % 4 == 0;
  if (ncmax <= kRegCap && packed)
    hipLaunchKernelGGL(topk_reg_kernel<true>, dim3(p.R, p.ha ? p.Hkv : 1), dim3(kRegNT), 0, st,
                       p.S, p.qo, p.b, p.k, p.W, scores, idx);
  else if (ncmax <= kRegCap)
    hipLaunchKernelGGL(topk_reg_kernel<false>, dim3(p.R, p.ha ? p.Hkv : 1), dim3(kRegNT), 0, st,
                       p.S, p.qo, p.b, p.k, p.W, scores, idx);
  else if (packed)
    hipLaunchKernelGGL(topk_rows_kernel<true>, dim3(p.R, p.ha ? p.Hkv : 1), dim3(kNT), 0, st,
                       p.S, p.qo, p.b, p.k, p.W, scores, idx);
  else
    hipLaunchKernelGGL(topk_rows_kernel<false>, dim3(p.R, p.ha ? p.Hkv : 1), dim3(kNT), 0, st,
                       p.S, p.qo, p.b, p.k, p.W, scores, idx);
  return hipGetLastError();
}

}  // namespace sp
