// Top-k support selection per score row (Section 4.1 TopK; Section 4.2;
// Algorithm 1 steps 4-5; Algorithm 2 step 5).
//
// Row r has L = t1_r+1 causal positions. If L <= k every position is taken.
// Otherwise the Wf = min(W, k) most recent positions are forced and the
// other k' = k-Wf are chosen among positions [0, L-Wf) in the order
// (score descending, position ascending).
//
// Keys are the order-preserving uint32 images of the fp32 scores. One
// workgroup per row finds the exact k'-th largest key T with three radix
// passes (12, 12 and 8 bits; LDS histograms; each pass counts only keys that
// share the prefix fixed so far). The chosen set is then {key > T} plus the
// first (k' - #{key > T}) positions with key == T. A final pass visits the
// row in position order and compacts the chosen positions with block-wide
// prefix sums, so every output row comes out ascending without a sort.
#include "common.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

constexpr int kNT = 256;         // threads per workgroup
constexpr int kEmitPer = 16;     // consecutive elements per thread in the emit pass
constexpr int kEmitChunk = kNT * kEmitPer;

__global__ __launch_bounds__(kNT) void topk_rows_kernel(int S, int b, int k, int W,
                                                        const float *__restrict__ scores,
                                                        int32_t *__restrict__ idx) {
  __shared__ uint32_t hist[4096];
  __shared__ uint32_t scan_scratch[kNT / 64 + 1];
  __shared__ uint32_t sel[2];
  __shared__ uint32_t keys[kEmitChunk];

  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int t1 = min(r * b + b, S) - 1;
  const int L = t1 + 1;
  int32_t *out = idx + (size_t)r * k;
  const float *row = scores + (size_t)r * S;

  if (L <= k) {
    for (int c = tid; c < k; c += kNT) out[c] = c < L ? c : -1;
    return;
  }
  const int Wf = min(W, k);
  const int nc = L - Wf;  // candidate positions [0, nc)
  const int kp = k - Wf;  // how many candidates to choose (nc > kp)

  uint32_t T = 0xffffffffu;
  uint32_t remaining = 0;  // how many keys equal to T are taken
  if (kp > 0) {
    uint32_t prefix = 0, pmask = 0;
    remaining = (uint32_t)kp;
#pragma unroll 1
    for (int pass = 0; pass < 3; ++pass) {
      const int shift = pass == 0 ? 20 : (pass == 1 ? 8 : 0);
      const int nbits = pass == 2 ? 8 : 12;
      const int nb = 1 << nbits;
      const uint32_t dmask = (uint32_t)nb - 1u;
      for (int i = tid; i < nb; i += kNT) hist[i] = 0;
      __syncthreads();
      for (int i = tid; i < nc; i += kNT) {
        const uint32_t key = float_key(row[i]);
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1u);
      }
      __syncthreads();
      // Thread `tid` owns bins [nb - (tid+1)*per, nb - tid*per): thread 0 the
      // highest. An exclusive scan of the per-thread sums gives, for each
      // thread, the number of keys in bins above its range.
      const int per = nb / kNT;
      const int hi = nb - tid * per;  // exclusive upper bin
      uint32_t mine = 0;
      for (int i = hi - per; i < hi; ++i) mine += hist[i];
      uint32_t total;
      const uint32_t above = block_exclusive_scan<kNT>(mine, scan_scratch, &total);
      if (above < remaining && above + mine >= remaining) {
        uint32_t acc = above;
        for (int i = hi - 1; i >= hi - per; --i) {
          const uint32_t c = hist[i];
          if (acc + c >= remaining) {
            sel[0] = (uint32_t)i;
            sel[1] = remaining - acc;
            break;
          }
          acc += c;
        }
      }
      __syncthreads();
      prefix |= sel[0] << shift;
      pmask |= dmask << shift;
      remaining = sel[1];
      __syncthreads();
    }
    T = prefix;
  }

  // Ordered emission over candidates: selected = key > T, or key == T among
  // the first `remaining` such positions.
  uint32_t gt_before = 0, eq_before = 0;
  for (int base = 0; base < nc; base += kEmitChunk) {
    const int n = min(kEmitChunk, nc - base);
    for (int i = tid; i < n; i += kNT) keys[i] = float_key(row[base + i]);
    __syncthreads();
    const int lo = tid * kEmitPer;
    uint32_t cgt = 0, ceq = 0;
#pragma unroll
    for (int e = 0; e < kEmitPer; ++e) {
      if (lo + e < n) {
        const uint32_t key = keys[lo + e];
        cgt += key > T;
        ceq += key == T;
      }
    }
    uint32_t total;
    const uint32_t ex = block_exclusive_scan<kNT>((cgt << 16) | ceq, scan_scratch, &total);
    uint32_t my_gt = gt_before + (ex >> 16);
    uint32_t my_eq = eq_before + (ex & 0xffffu);
    uint32_t pos = my_gt + min(my_eq, remaining);
#pragma unroll
    for (int e = 0; e < kEmitPer; ++e) {
      if (lo + e < n) {
        const uint32_t key = keys[lo + e];
        // pos < kp always holds when the counts above are consistent; the
        // test keeps every store inside the row regardless.
        if (key > T) {
          if (pos < (uint32_t)kp) out[pos] = base + lo + e;
          ++pos;
        } else if (key == T) {
          if (my_eq < remaining) {
            if (pos < (uint32_t)kp) out[pos] = base + lo + e;
            ++pos;
          }
          ++my_eq;
        }
      }
    }
    gt_before += total >> 16;
    eq_before += total & 0xffffu;
    __syncthreads();
  }
  for (int c = tid; c < Wf; c += kNT) out[kp + c] = nc + c;
}

}  // namespace

hipError_t launch_topk(const Prob &p, const float *scores, int32_t *idx, hipStream_t st) {
  hipLaunchKernelGGL(topk_rows_kernel, dim3(p.R), dim3(kNT), 0, st, p.S, p.b, p.k, p.W, scores,
                     idx);
  return hipGetLastError();
}

}  // namespace sp
