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

// Epilogue on the fp32 C tile parked in LDS (token-major, cstride floats per
// token, columns q then k): one (token, q or k) row per wave step, lane pairs
// c, c + DI/2.
template <int DI, int TOK, int NWAVE>
__device__ __forceinline__ void project_epilogue(const float *cl, int cstride, int S, int t0,
                                                 int pos0, float theta, float eps,
                                                 const float *__restrict__ gamma,
                                                 const float *__restrict__ beta,
                                                 uint16_t *__restrict__ qo,
                                                 uint16_t *__restrict__ ko, int wave, int lane) {
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
  for (int row = wave; row < 2 * TOK; row += NWAVE) {
    const int tl = row >> 1, is_k = row & 1;
    const int t = t0 + tl;
    if (t >= S) continue;   // wave-uniform
    const float *cr = cl + tl * cstride + is_k * DI;
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

  project_epilogue<DI, kPT, kPW>(cl, L::CSTRIDE, S, t0, pos0, theta, eps, gamma, beta, qo, ko,
                                  wave, lane);
}

// Wide kernel for d_idx <= 128: 128 tokens per workgroup, so at 32K tokens
// one round of 256 workgroups covers the chip and each W tile read from L2
// serves twice the tokens. x, W_Q and W_K tiles of 32 model columns go
// straight from memory into LDS rows of four 16-byte slots, stored at slot
// c ^ ((row >> 1) & 3) so that eight consecutive rows read at one slot hit
// distinct banks, in a ring of kWStages stages, kWStages - 2 of them in
// flight behind the one being multiplied. Eight waves (two token halves by four
// output quarters) run v_mfma_f32_32x32x16_bf16 with tokens as A rows and
// output columns as B rows; the operand reads are inline so the compiler
// adds no wait for the direct loads still in flight.
constexpr int kWT = 128;        // tokens per workgroup
constexpr int kWK = 32;         // model columns per stage
constexpr int kWW = 8;          // waves
constexpr int kWStages = 6;
constexpr int kProjBufferDword3 = 0x00020000;   // raw buffer resource: 32-bit data format

template <int DI>
struct WideLayout {
  static constexpr int N = 2 * DI;                   // output columns (q then k)
  static constexpr int SLOTS = kWK / 8;              // 16-byte slots per row
  static constexpr int RB = SLOTS * 16;              // row bytes (64)
  static constexpr int XCH = kWT * SLOTS / 64;       // 1 KiB direct loads per stage: x
  static constexpr int QCH = DI * SLOTS / 64;        // ... W_Q (and as many for W_K)
  static constexpr int CH = XCH + 2 * QCH;
  static constexpr int CPW = (CH + kWW - 1) / kWW;   // per wave; surplus ones repeat a chunk
  static_assert(SLOTS == 4, "the swizzle permutes four slots");
  static constexpr int XBYTES = kWT * RB;
  static constexpr int STAGE = (kWT + N) * RB;
  static constexpr int NB = N / 4 / 32;              // 32-column output blocks per wave
  static constexpr int KS = kWK / 16;                // k-steps per stage
  static constexpr int CSTRIDE = N + 4;              // floats per token row of the C tile
  static constexpr int CBYTES = kWT * CSTRIDE * 4;
  static constexpr int LDS = kWStages * STAGE > CBYTES ? kWStages * STAGE : CBYTES;
  static_assert(kWT * SLOTS % 64 == 0 && DI * SLOTS % 64 == 0, "whole 1 KiB chunks");
  static_assert(LDS <= 160 * 1024, "fits the LDS of a CU");
};

// vmcnt(n) alone (expcnt and lgkmcnt left at their maxima)
constexpr int vm_wait_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Direct loads of one stage. Chunk q of a stage covers 64 consecutive slots
// of one array's rows; lane l of chunk q writes LDS bytes [1024 q + 16 l,
// + 16), which hold row (64 q + l) / 4 at column slot ((64 q + l) % 4) ^
// swizzle(row). Token rows past the sequence end read the last row (their
// outputs are not written).
template <int DI>
struct WideDma {
  using L = WideLayout<DI>;
  __device__ __forceinline__ static int chunk(int wave, int p) { return (wave + p * kWW) % L::CH; }
  __device__ __forceinline__ static void offsets(int S, int dm, int t0, int wave, int lane,
                                                 uint32_t (&off)[L::CPW]) {
#pragma unroll
    for (int p = 0; p < L::CPW; ++p) {
      const int q = chunk(wave, p);
      const int q0 = q < L::XCH ? q : (q - L::XCH) % L::QCH;
      const int slot = q0 * 64 + lane, row = slot / L::SLOTS;
      const uint32_t cb = (uint32_t)((slot % L::SLOTS) ^ ((row >> 1) & 3)) * 16;
      const int r = q < L::XCH ? min(t0 + row, S - 1) : row;
      off[p] = (uint32_t)r * (uint32_t)dm * 2u + cb;
    }
  }
  __device__ __forceinline__ static void issue(uint32_t stage, int k0, int S, int dm,
                                               const uint16_t *x, const uint16_t *wq,
                                               const uint16_t *wk, int wave,
                                               const uint32_t (&off)[L::CPW]) {
    const uint32_t kb = (uint32_t)k0 * 2u;
#pragma unroll
    for (int p = 0; p < L::CPW; ++p) {
      const int q = chunk(wave, p);
      const uint16_t *base = q < L::XCH ? x : q < L::XCH + L::QCH ? wq : wk;
      const uint32_t bytes = (uint32_t)(q < L::XCH ? S : DI) * (uint32_t)dm * 2u;
      const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(base), (short)0,
                                                        bytes, kProjBufferDword3);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void *)(size_t)(stage + q * 1024), 16,
          off[p] + kb, 0, 0, 0);
    }
  }
};

template <int DI>
__global__ __launch_bounds__(kWW * 64) void project_wide_kernel(
    int S, int dm, int pos0, float theta, float eps, const uint16_t *__restrict__ x,
    const uint16_t *__restrict__ wq, const uint16_t *__restrict__ wk,
    const float *__restrict__ gamma, const float *__restrict__ beta, uint16_t *__restrict__ qo,
    uint16_t *__restrict__ ko) {
  using L = WideLayout<DI>;
  using Dma = WideDma<DI>;
  constexpr int NB = L::NB, KS = L::KS, RB = L::RB, NS = kWStages;
  __shared__ __align__(16) char lds[L::LDS];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, h = lane >> 5;
  const int wt = wave >> 2, wo = wave & 3;   // token half, output quarter
  const int t0 = blockIdx.x * kWT;
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) char *)&lds[0];

  uint32_t off[L::CPW];
  Dma::offsets(S, dm, t0, wave, lane, off);
  const int nk = dm / kWK;
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < nk) Dma::issue(lds0 + st * L::STAGE, st * kWK, S, dm, x, wq, wk, wave, off);

  f32x16 acc[2][NB];
#pragma unroll
  for (int bt = 0; bt < 2; ++bt)
#pragma unroll
    for (int bo = 0; bo < NB; ++bo) acc[bt][bo] = f32x16{};
  // per-lane LDS offsets within a stage: A rows (tokens), B rows (outputs);
  // row bases are multiples of 32, so a lane's swizzle is (n >> 1) & 3, and
  // k-step ks reads column slot 2 ks + h
  const uint32_t sw = (uint32_t)((n >> 1) & 3);
  const uint32_t xrow = (uint32_t)(wt * 64 + n) * RB;
  const uint32_t wrow = (uint32_t)L::XBYTES + (uint32_t)(wo * NB * 32 + n) * RB;
  const uint32_t kso[2] = {((uint32_t)h ^ sw) * 16, (((uint32_t)h + 2) ^ sw) * 16};
  for (int it = 0; it < nk; ++it) {
    // this wave's loads of stage it have landed (later stages may still fly)
    if (it + NS - 2 < nk)
      __builtin_amdgcn_s_waitcnt(vm_wait_imm((NS - 2) * L::CPW));
    else
      __builtin_amdgcn_s_waitcnt(vm_wait_imm(0));
    // every wave's loads of stage it have landed and stage it - 1 is fully
    // read (each wave waited for its own reads before its products): a bare
    // barrier, as the fence of a full one would also wait for the loads of
    // the later stages
    __builtin_amdgcn_s_barrier();
    if (it + NS - 1 < nk)
      Dma::issue(lds0 + ((it + NS - 1) % NS) * L::STAGE, (it + NS - 1) * kWK, S, dm, x, wq, wk,
                 wave, off);
    const uint32_t sbase = lds0 + (it % NS) * L::STAGE;
    bf16x8 fa[KS][2], fb[KS][NB];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint32_t xa = sbase + xrow + kso[ks], wa = sbase + wrow + kso[ks];
#pragma unroll
      for (int bt = 0; bt < 2; ++bt)
        asm volatile("ds_read_b128 %0, %1 offset:%2"
                     : "=v"(fa[ks][bt])
                     : "v"(xa), "i"(bt * 32 * RB));
#pragma unroll
      for (int bo = 0; bo < NB; ++bo)
        asm volatile("ds_read_b128 %0, %1 offset:%2"
                     : "=v"(fb[ks][bo])
                     : "v"(wa), "i"(bo * 32 * RB));
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      // reads complete in order: k-step ks needs all but the later k-steps' reads
      if (ks == 0) {
        asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(fa[0][0]), "+v"(fa[0][1]) : "i"((KS - 1) * (2 + NB)));
#pragma unroll
        for (int bo = 0; bo < NB; ++bo) asm volatile("" : "+v"(fb[0][bo]));
      } else {
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fa[ks][0]), "+v"(fa[ks][1]));
#pragma unroll
        for (int bo = 0; bo < NB; ++bo) asm volatile("" : "+v"(fb[ks][bo]));
      }
#pragma unroll
      for (int bt = 0; bt < 2; ++bt)
#pragma unroll
        for (int bo = 0; bo < NB; ++bo) acc[bt][bo] = mfma32(fa[ks][bt], fb[ks][bo], acc[bt][bo]);
    }
  }
  __builtin_amdgcn_s_waitcnt(vm_wait_imm(0));
  __syncthreads();   // the ring is free: park C (token-major, fp32)
  float *cl = reinterpret_cast<float *>(lds);
#pragma unroll
  for (int bt = 0; bt < 2; ++bt)
#pragma unroll
    for (int bo = 0; bo < NB; ++bo)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int tl = wt * 64 + bt * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
        cl[tl * L::CSTRIDE + wo * NB * 32 + bo * 32 + n] = acc[bt][bo][e];
      }
  __syncthreads();
  project_epilogue<DI, kWT, kWW>(cl, L::CSTRIDE, S, t0, pos0, theta, eps, gamma, beta, qo, ko,
                                 wave, lane);
}

template <int DI>
hipError_t launch_di(int S, int dm, int pos0, float theta, float eps, const void *x,
                     const void *wq, const void *wk, const float *gamma, const float *beta,
                     void *qo, void *ko, hipStream_t st) {
  if constexpr (DI <= 128) {
    // the wide kernel's buffer offsets are 32-bit
    if ((uint64_t)S * (uint64_t)dm * 2u < (1ull << 32) && dm % kWK == 0) {
      hipLaunchKernelGGL((project_wide_kernel<DI>), dim3((S + kWT - 1) / kWT), dim3(kWW * 64), 0,
                         st, S, dm, pos0, theta, eps, (const uint16_t *)x, (const uint16_t *)wq,
                         (const uint16_t *)wk, gamma, beta, (uint16_t *)qo, (uint16_t *)ko);
      return hipGetLastError();
    }
  }
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
