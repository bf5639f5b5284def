// Device helpers shared by the gfx950 kernels: element conversion, vector
// loads, wave64 reductions and block scans.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace sp {

// Compile-time loop: f(std::integral_constant<int, I>{}) for I in [B, E).
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// bf16 is stored as raw 16-bit patterns; float <-> bf16 by bit manipulation.
struct bf16 {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_float(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Two floats -> two bf16 in one word (a low, b high), round to nearest even,
// by the hardware packed conversion.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Round-to-nearest-even float -> bf16 (NaN kept quiet).
__device__ __forceinline__ uint16_t float_to_bf16(float f) {
  uint32_t x = __float_as_uint(f);
  if ((x & 0x7f800000u) == 0x7f800000u && (x & 0x007fffffu)) return 0x7fc0;
  x += 0x7fffu + ((x >> 16) & 1u);
  return static_cast<uint16_t>(x >> 16);
}

// Load N consecutive elements starting at p (16-byte friendly when N*size is
// a multiple of 16 and p is aligned accordingly) and widen to float.
template <int N>
__device__ __forceinline__ void load_row(const float *p, float (&out)[N]) {
  static_assert(N % 4 == 0, "N must be a multiple of 4");
#pragma unroll
  for (int i = 0; i < N; i += 4) {
    float4 x = *reinterpret_cast<const float4 *>(p + i);
    out[i] = x.x; out[i + 1] = x.y; out[i + 2] = x.z; out[i + 3] = x.w;
  }
}

template <int N>
__device__ __forceinline__ void load_row(const bf16 *p, float (&out)[N]) {
  static_assert(N % 4 == 0, "N must be a multiple of 4");
  const uint16_t *u = reinterpret_cast<const uint16_t *>(p);
  if constexpr (N % 8 == 0) {
#pragma unroll
    for (int i = 0; i < N; i += 8) {
      uint4 x = *reinterpret_cast<const uint4 *>(u + i);
      uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        out[i + 2 * j] = __uint_as_float(w[j] << 16);
        out[i + 2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < N; i += 4) {
      uint2 x = *reinterpret_cast<const uint2 *>(u + i);
      out[i] = __uint_as_float(x.x << 16);
      out[i + 1] = __uint_as_float(x.x & 0xffff0000u);
      out[i + 2] = __uint_as_float(x.y << 16);
      out[i + 3] = __uint_as_float(x.y & 0xffff0000u);
    }
  }
}

template <int N>
__device__ __forceinline__ void store_row(float *p, const float (&in)[N]) {
#pragma unroll
  for (int i = 0; i < N; i += 4)
    *reinterpret_cast<float4 *>(p + i) = make_float4(in[i], in[i + 1], in[i + 2], in[i + 3]);
}

template <int N>
__device__ __forceinline__ void store_row(bf16 *p, const float (&in)[N]) {
  uint16_t *u = reinterpret_cast<uint16_t *>(p);
#pragma unroll
  for (int i = 0; i < N; i += 4) {
    uint2 x;
    x.x = static_cast<uint32_t>(float_to_bf16(in[i])) |
          (static_cast<uint32_t>(float_to_bf16(in[i + 1])) << 16);
    x.y = static_cast<uint32_t>(float_to_bf16(in[i + 2])) |
          (static_cast<uint32_t>(float_to_bf16(in[i + 3])) << 16);
    *reinterpret_cast<uint2 *>(u + i) = x;
  }
}

__device__ __forceinline__ float to_float(float x) { return x; }
__device__ __forceinline__ float to_float(bf16 x) { return bf16_to_float(x.bits); }

// Sum over aligned groups of W lanes (W a power of two <= 64).
template <int W>
__device__ __forceinline__ float group_sum(float x) {
#pragma unroll
  for (int off = W / 2; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// Sum over each 16-lane row with DPP lane moves (no LDS traffic): swap
// neighbours, swap pairs, then rotate the row by 4 and by 8; every lane ends
// with its row's total.
__device__ __forceinline__ float row16_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false));
  return x;
}

// Order-preserving map float -> uint32 (larger float, larger key); -0.0 and
// +0.0 share one key.
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u << 1) == 0u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over a block of NT threads (NT a multiple of 64).
// `scratch` must hold NT/64 + 1 words. Returns the exclusive prefix; *total
// receives the block total. Contains barriers: call from every thread.
template <int NT>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t *scratch,
                                                         uint32_t *total) {
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    uint32_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) scratch[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t acc = 0;
    for (int w = 0; w < NT / 64; ++w) {
      uint32_t c = scratch[w];
      scratch[w] = acc;
      acc += c;
    }
    scratch[NT / 64] = acc;
  }
  __syncthreads();
  uint32_t ex = scratch[wid] + x - v;
  *total = scratch[NT / 64];
  __syncthreads();
  return ex;
}

}  // namespace sp
