// Head-collapsed indexer front end on bf16 MFMA (Section 6.3, projection and
// score equations; Algorithm 2, indexer projection and its key normalisation, RoPE and query scale):
//
//   q_idx[t] = RoPE(W_Q x_t, pos0 + t)
//   k_idx[t] = RoPE(LN(W_K x_t), pos0 + t),  LN over d_idx with gamma, beta
//   RoPE(a, p): the pair (a[c], a[c + d_idx/2]) turns by p * theta^(-2c/d_idx)
//
// One workgroup per 64 tokens computes both projections at once, C = x W^T
// with W = [W_Q; W_K] ([2 d_idx, d_model]): x and W tiles of 64 model
// columns go through double-buffered LDS (register staged), eight waves each
// own 2 d_idx / 8 output columns of all 64 tokens. The fp32 C tile is then
// parked in LDS and the epilogue works a token row at a time: each lane
// holds one rotation pair, takes the LayerNorm statistics of the key row
// with a wave reduction, rotates, and writes bf16. Angles are formed and
// range-reduced in fp64 (positions reach 1e5 and beyond) before a float
// sincos.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"

namespace sp {
namespace {

constexpr int kPT = 64;    // tokens per workgroup
constexpr int kPW = 8;     // waves

template <int DI>
struct ProjLayout {
  static constexpr int KPK = DI == 256 ? 32 : 64;    // model columns per k-chunk (LDS fit)
  static constexpr int N = 2 * DI;                    // output columns (q then k)
  static constexpr int RB = KPK * 2 + 16;             // padded row bytes of an LDS tile
  static constexpr int XBYTES = kPT * RB;
  static constexpr int WBYTES = N * RB;
  static constexpr int BUF = XBYTES + WBYTES;
  static constexpr int CT = N / kPW / 16;             // 16-column tiles per wave
  static constexpr int CSTRIDE = N + 4;               // floats per token row of the C tile
  static constexpr int CBYTES = kPT * CSTRIDE * 4;
  static constexpr int LDS = (2 * BUF > CBYTES ? 2 * BUF : CBYTES);
};

template <int DI>
__global__ __launch_bounds__(kPW * 64) void project_kernel(
    int S, int dm, int pos0, float theta, float eps, const uint16_t *__restrict__ x,
    const uint16_t *__restrict__ wq, const uint16_t *__restrict__ wk,
    const float *__restrict__ gamma, const float *__restrict__ beta, uint16_t *__restrict__ qo,
    uint16_t *__restrict__ ko) {
  using L = ProjLayout<DI>;
  constexpr int NT = kPW * 64, N = L::N, RB = L::RB, CT = L::CT, kPK = L::KPK;
  constexpr int XP = kPT * kPK / 8;     // 16-byte pieces of an x tile
  constexpr int WP = N * kPK / 8;       // ... of a W tile
  constexpr int XPER = (XP + NT - 1) / NT, WPER = (WP + NT - 1) / NT;
  __shared__ __align__(16) char lds[L::LDS];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c16 = lane & 15;
  const int t0 = blockIdx.x * kPT;

  uint4 xs[XPER], ws[WPER];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < XPER; ++i) {
      const int c = tid + i * NT;
      if (c < XP) {
        const int row = c / (kPK / 8), col = c % (kPK / 8);
        const int t = min(t0 + row, S - 1);
        xs[i] = ldg16(x + (size_t)t * dm + k0 + col * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < WPER; ++i) {
      const int c = tid + i * NT;
      if (c < WP) {
        const int row = c / (kPK / 8), col = c % (kPK / 8);
        const uint16_t *w = row < DI ? wq + (size_t)row * dm : wk + (size_t)(row - DI) * dm;
        ws[i] = ldg16(w + k0 + col * 8);
      }
    }
  };
  auto store = [&](char *buf) {
#pragma unroll
    for (int i = 0; i < XPER; ++i) {
      const int c = tid + i * NT;
      if (c < XP) sts16(buf + (c / (kPK / 8)) * RB + (c % (kPK / 8)) * 16, xs[i]);
    }
#pragma unroll
    for (int i = 0; i < WPER; ++i) {
      const int c = tid + i * NT;
      if (c < WP)
        sts16(buf + L::XBYTES + (c / (kPK / 8)) * RB + (c % (kPK / 8)) * 16, ws[i]);
    }
  };

  f32x4 acc[4][CT];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = dm / kPK;
  load(0);
  store(lds);
  __syncthreads();
  for (int it = 0; it < nk; ++it) {
    const bool more = it + 1 < nk;
    if (more) load((it + 1) * kPK);
    const char *buf = lds + (it & 1) * L::BUF;
#pragma unroll
    for (int ks = 0; ks < kPK / 32; ++ks) {
      bf16x8 a[4], b[CT];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
        a[rt] = as_bf16x8(lds16(buf + (rt * 16 + c16) * RB + ks * 64 + g * 16));
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
        b[ct] = as_bf16x8(lds16(buf + L::XBYTES + ((wave * CT + ct) * 16 + c16) * RB +
                                ks * 64 + g * 16));
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = mfma16(a[rt], b[ct], acc[rt][ct]);
    }
    if (more) store(lds + ((it + 1) & 1) * L::BUF);
    __syncthreads();
  }

  // Park C (token-major, fp32) in LDS: lane (g, c16) holds tokens
  // 16rt + 4g + r of column (wave*CT + ct)*16 + c16.
  float *cl = reinterpret_cast<float *>(lds);
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        cl[(rt * 16 + g * 4 + r) * L::CSTRIDE + (wave * CT + ct) * 16 + c16] = acc[rt][ct][r];
  __syncthreads();

  // Epilogue: one (token, q or k) row per wave step; lane pairs c, c + DI/2.
  constexpr int H = DI / 2;
  constexpr int PPL = (H + 63) / 64;   // pairs per lane
  double inv_freq[PPL];
  float gam[PPL][2], bet[PPL][2];
#pragma unroll
  for (int u = 0; u < PPL; ++u) {
    const int c = lane + u * 64;
    inv_freq[u] = exp2(-(2.0 * c / DI) * log2((double)theta));
    gam[u][0] = c < H ? gamma[c] : 0.f;
    gam[u][1] = c < H ? gamma[c + H] : 0.f;
    bet[u][0] = c < H ? beta[c] : 0.f;
    bet[u][1] = c < H ? beta[c + H] : 0.f;
  }
  const double two_pi = 6.283185307179586;
  for (int row = wave; row < 2 * kPT; row += kPW) {
    const int tl = row >> 1, is_k = row & 1;
    const int t = t0 + tl;
    if (t >= S) continue;   // wave-uniform
    const float *cr = cl + tl * L::CSTRIDE + is_k * DI;
    float lo[PPL], hi[PPL];
#pragma unroll
    for (int u = 0; u < PPL; ++u) {
      const int c = lane + u * 64;
      lo[u] = c < H ? cr[c] : 0.f;
      hi[u] = c < H ? cr[c + H] : 0.f;
    }
    if (is_k) {
      float s = 0.f;
#pragma unroll
      for (int u = 0; u < PPL; ++u) s += lo[u] + hi[u];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
      const float mean = s / DI;
      float v = 0.f;
#pragma unroll
      for (int u = 0; u < PPL; ++u) {
        const int c = lane + u * 64;
        if (c < H) {
          v += (lo[u] - mean) * (lo[u] - mean);
          v += (hi[u] - mean) * (hi[u] - mean);
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
      const float inv = 1.f / sqrtf(v / DI + eps);
#pragma unroll
      for (int u = 0; u < PPL; ++u) {
        lo[u] = (lo[u] - mean) * inv * gam[u][0] + bet[u][0];
        hi[u] = (hi[u] - mean) * inv * gam[u][1] + bet[u][1];
      }
    }
    uint16_t *out = (is_k ? ko : qo) + (size_t)t * DI;
    const double p = (double)pos0 + t;
#pragma unroll
    for (int u = 0; u < PPL; ++u) {
      const int c = lane + u * 64;
      if (c >= H) continue;
      double ang = p * inv_freq[u];
      ang -= two_pi * rint(ang / two_pi);
      float sn, cs;
      sincosf((float)ang, &sn, &cs);
      out[c] = float_to_bf16(lo[u] * cs - hi[u] * sn);
      out[c + H] = float_to_bf16(hi[u] * cs + lo[u] * sn);
    }
  }
}

template <int DI>
hipError_t launch_di(int S, int dm, int pos0, float theta, float eps, const void *x,
                     const void *wq, const void *wk, const float *gamma, const float *beta,
                     void *qo, void *ko, hipStream_t st) {
  hipLaunchKernelGGL((project_kernel<DI>), dim3((S + kPT - 1) / kPT), dim3(kPW * 64), 0, st, S,
                     dm, pos0, theta, eps, (const uint16_t *)x, (const uint16_t *)wq,
                     (const uint16_t *)wk, gamma, beta, (uint16_t *)qo, (uint16_t *)ko);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_indexer_project(int S, int di, int dm, int pos0, float theta, float eps,
                                  const void *x, const void *wq, const void *wk,
                                  const float *gamma, const float *beta, void *qo, void *ko,
                                  hipStream_t st) {
  if (di == 64) return launch_di<64>(S, dm, pos0, theta, eps, x, wq, wk, gamma, beta, qo, ko, st);
  if (di == 128)
    return launch_di<128>(S, dm, pos0, theta, eps, x, wq, wk, gamma, beta, qo, ko, st);
  return launch_di<256>(S, dm, pos0, theta, eps, x, wq, wk, gamma, beta, qo, ko, st);
}

}  // namespace sp
