// Row-wise helpers shared by the per-token kernels of the denoiser
// (denoise.hip) and the input encoder (encode.hip): 16-byte loads and stores of
// eight elements, round-to-nearest-even bfloat16, and a LayerNorm of a row
// held by one wave.
#pragma once

#include "sp_internal.h"

namespace sp {
namespace {

constexpr int kRowWaves = 4;
constexpr int kMaxChunks = 8;       // 8-element chunks per lane: d <= 4096

__device__ __forceinline__ float wave_sum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Eight consecutive elements: bfloat16 in 16 bytes, float32 in 32 bytes.
__device__ __forceinline__ void load8(const uint16_t* p, float (&v)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = __uint_as_float(w[k] << 16);
    v[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void store8(uint16_t* p, const float (&v)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
    w[k] = (uint32_t)f32_to_bf16(v[2 * k]) | ((uint32_t)f32_to_bf16(v[2 * k + 1]) << 16);
  *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ void store8(float* p, const float (&v)[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}

// LayerNorm of a row held as chunks v[i] (elements 8 (lane + 64 i) ..), scaled
// by g and shifted by b, written as bfloat16.
__device__ __forceinline__ void ln_store(const float (&v)[kMaxChunks][8], int nch, int d,
                                         int lane, const float* __restrict__ g,
                                         const float* __restrict__ b, uint16_t* __restrict__ z) {
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i)
    if (lane + 64 * i < nch)
#pragma unroll
      for (int k = 0; k < 8; ++k) s += v[i][k];
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i)
    if (lane + 64 * i < nch)
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float t = v[i][k] - mean;
        q = fmaf(t, t, q);
      }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + kBlockLnEps);
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    const int c = 8 * (lane + 64 * i);
    if (c >= d) break;
    float gg[8], bb[8], o[8];
    load8(g + c, gg);
    load8(b + c, bb);
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = fmaf((v[i][k] - mean) * rstd, gg[k], bb[k]);
    store8(z + c, o);
  }
}

}  // namespace
}  // namespace sp
