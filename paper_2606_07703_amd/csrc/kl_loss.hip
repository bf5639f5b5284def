// KL distillation objective of the indexer and its gradient (Section 6.2):
//
//   kl_i = KL(P_i || softmax(z_i)) = sum_{s<=t_i} P_i(s) (log P_i(s) - z_i(s)) + LSE_i sum P_i
//   LSE_i = log sum_{s<=t_i} exp z_i(s),       loss = (1/n) sum_i kl_i
//   d loss / d z_i(s) = (exp(z_i(s) - LSE_i) sum P_i - P_i(s)) / n   (s <= t_i), 0 after t_i
//
// One 1024-thread workgroup per supervised row; HBM-bound. Rows of up to
// 32768 valid keys stay in registers between the statistics pass and the
// gradient pass, so each input element is read once; longer rows stream
// twice. The exp-sum is kept online per thread (running max, rescaled sum) and
// merged across the workgroup; the P log P - P z sum and sum P accumulate in
// fp64, since the KL of a good student is a small difference of large terms.
// The mean over rows is a second, single-workgroup pass in a fixed order, so
// the loss is deterministic.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace sp {
namespace {

constexpr int kKlThreads = 1024;
constexpr int kKlResident = 32;   // elements per thread kept in registers

struct KlStats {
  float m;     // running max of z
  float se;    // sum exp(z - m)
  double a;    // sum P (log P - z)
  double sp;   // sum P
};

__device__ __forceinline__ void kl_add(KlStats &st, float zv, float pv) {
  if (zv > st.m) {
    st.se = st.se * __expf(st.m - zv) + 1.f;   // m = -inf gives 0 * ... = 0
    st.m = zv;
  } else {
    st.se += __expf(zv - st.m);
  }
  if (pv > 0.f) st.a += (double)(pv * (__logf(pv) - zv));
  st.sp += (double)pv;
}

__device__ __forceinline__ KlStats kl_merge(KlStats x, KlStats y) {
  const float m = fmaxf(x.m, y.m);
  KlStats r;
  r.m = m;
  r.se = (x.m == -INFINITY ? 0.f : x.se * __expf(x.m - m)) +
         (y.m == -INFINITY ? 0.f : y.se * __expf(y.m - m));
  r.a = x.a + y.a;
  r.sp = x.sp + y.sp;
  return r;
}

__device__ __forceinline__ KlStats kl_shfl(const KlStats &x, int off) {
  KlStats y;
  y.m = __shfl_xor(x.m, off, 64);
  y.se = __shfl_xor(x.se, off, 64);
  y.a = __shfl_xor(x.a, off, 64);
  y.sp = __shfl_xor(x.sp, off, 64);
  return y;
}

__global__ __launch_bounds__(kKlThreads) void kl_rows_kernel(int S, int n,
                                                             const int32_t *__restrict__ rows,
                                                             const float *__restrict__ P,
                                                             const float *__restrict__ z,
                                                             float *__restrict__ kl,
                                                             float *__restrict__ grad) {
  constexpr int NT = kKlThreads, E = kKlResident, NW = NT / 64;
  __shared__ KlStats red[NW];
  __shared__ KlStats total;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = blockIdx.x;
  const int t = rows[i];
  const size_t base = (size_t)i * S;
  float *gi = grad ? grad + base : nullptr;
  if (t < 0 || t >= S) {
    if (kl && tid == 0) kl[i] = 0.f;
    if (gi)
      for (int s = tid; s < S; s += NT) gi[s] = 0.f;
    return;
  }
  const int L = t + 1;
  const bool resident = L <= NT * E;
  const float *Pi = P + base;
  const float *zi = z + base;

  KlStats st{-INFINITY, 0.f, 0.0, 0.0};
  float zr[E], pr[E];
  if (resident) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int s = tid + e * NT;
      zr[e] = s < L ? zi[s] : -INFINITY;
      pr[e] = s < L ? Pi[s] : 0.f;
    }
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (tid + e * NT < L) kl_add(st, zr[e], pr[e]);
  } else {
    for (int s = tid; s < L; s += NT) kl_add(st, zi[s], Pi[s]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) st = kl_merge(st, kl_shfl(st, off));
  if (lane == 0) red[wave] = st;
  __syncthreads();
  if (tid == 0) {
    KlStats acc = red[0];
    for (int w = 1; w < NW; ++w) acc = kl_merge(acc, red[w]);
    total = acc;
  }
  __syncthreads();
  const KlStats tot = total;
  const double lse = (double)tot.m + log((double)tot.se);
  if (kl && tid == 0) kl[i] = (float)(tot.a + lse * tot.sp);
  if (!gi) return;
  const float lsef = (float)lse;
  const float spn = (float)(tot.sp / n), inv_n = 1.f / n;
  if (resident) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int s = tid + e * NT;
      if (s < L) gi[s] = __expf(zr[e] - lsef) * spn - pr[e] * inv_n;
    }
  } else {
    for (int s = tid; s < L; s += NT) gi[s] = __expf(zi[s] - lsef) * spn - Pi[s] * inv_n;
  }
  for (int s = L + tid; s < S; s += NT) gi[s] = 0.f;
}

// loss = (1/n) sum_i kl_i, summed in fp64 in a fixed order.
__global__ __launch_bounds__(kKlThreads) void kl_mean_kernel(int n, const float *__restrict__ kl,
                                                             float *__restrict__ loss) {
  constexpr int NT = kKlThreads, NW = NT / 64;
  __shared__ double red[NW];
  const int tid = threadIdx.x;
  double acc = 0.0;
  for (int i = tid; i < n; i += NT) acc += (double)kl[i];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if ((tid & 63) == 0) red[tid >> 6] = acc;
  __syncthreads();
  if (tid == 0) {
    double s = 0.0;
    for (int w = 0; w < NW; ++w) s += red[w];
    loss[0] = (float)(s / n);
  }
}

}  // namespace

hipError_t launch_kl_loss(int S, int n, const int32_t *rows, const float *P, const float *z,
                          float *kl, float *loss, float *grad, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(kl_rows_kernel, dim3(n), dim3(kKlThreads), 0, st, S, n, rows, P, z, kl,
                     grad);
  if (loss) hipLaunchKernelGGL(kl_mean_kernel, dim3(1), dim3(kKlThreads), 0, st, n, kl, loss);
  return hipGetLastError();
}

}  // namespace sp
