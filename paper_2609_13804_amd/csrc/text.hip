// Text context of Algorithm 1 step 1 (Section "Conditional Sequential Pointer
// Policy": text projection, LayerNorm, gain g_text), reduced to the pointer
// query space:  c_b = g_text * mean_l LN(E_{b,l} W_text^T).
//
// The projection itself is a dense contraction (gemm.hip, float32 output,
// split over K into `split` partial products).  Two kernels follow it, both
// with a fixed summation order:
//   * text_norm_kernel: one wave per text row adds the row's partial products
//     in split order, normalises it (no affine parameters, biased variance,
//     eps) and writes it over partial product 0;
//   * text_mean_kernel: one thread per (image, column) averages the image's
//     normalised rows in row order and applies the gain.
#include "sp_internal.h"

namespace sp {
namespace {

constexpr int kNormWaves = 4;

__device__ inline float wsum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

template <int SPLIT>
__global__ __launch_bounds__(kNormWaves * 64) void text_norm_kernel(float* __restrict__ T,
                                                                    int64_t T_txt, int h,
                                                                    float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kNormWaves + (threadIdx.x >> 6);
  if (r >= T_txt) return;
  const int per = h / 64;
  float* row = T + r * h;
  float xp[SPLIT][16];
#pragma unroll
  for (int p = 0; p < SPLIT; ++p)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      xp[p][i] = i < per ? row[(int64_t)p * T_txt * h + lane + 64 * i] : 0.0f;
  float x[16];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    x[i] = xp[0][i];
#pragma unroll
    for (int p = 1; p < SPLIT; ++p) x[i] += xp[p][i];
    s += x[i];
  }
  const float mean = wsum(s) / (float)h;
  float q = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < per) {
      const float dlt = x[i] - mean;
      q = fmaf(dlt, dlt, q);
    }
  const float inv = 1.0f / sqrtf(wsum(q) / (float)h + eps);
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < per) row[lane + 64 * i] = (x[i] - mean) * inv;
}

// grid (B, ceil(h / 256)): thread t of block (b, y) owns column 256 y + t.
__global__ __launch_bounds__(256) void text_mean_kernel(const float* __restrict__ T,
                                                        const int32_t* __restrict__ text_off,
                                                        int64_t T_txt, int h, float g_text,
                                                        float* __restrict__ ctx, int32_t* err) {
  const int b = blockIdx.x;
  const int c = blockIdx.y * 256 + threadIdx.x;
  const int64_t r0 = text_off[b], r1 = text_off[b + 1];
  if (r0 < 0 || r1 < r0 || r1 > T_txt) {
    if (blockIdx.y == 0 && threadIdx.x == 0) set_device_error(err, SP_DEV_BAD_OFFSETS);
    if (c < h) ctx[(int64_t)b * h + c] = 0.0f;
    return;
  }
  if (c >= h) return;
  const float* col = T + c;
  float s = 0.0f;
  int64_t r = r0;
  for (; r + 8 <= r1; r += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = col[(r + u) * h];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  for (; r < r1; ++r) s += col[r * h];
  const int64_t L = r1 - r0;
  ctx[(int64_t)b * h + c] = L > 0 ? g_text * (s / (float)L) : 0.0f;
}

}  // namespace

hipError_t launch_text_pool(float* T, int split, const int32_t* text_off, int B, int64_t T_txt,
                            int h, float g_text, float ln_eps, float* ctx, int32_t* err,
                            hipStream_t stream) {
  if (B == 0) return hipSuccess;
  if (T_txt > 0) {
    const dim3 grid((unsigned)((T_txt + kNormWaves - 1) / kNormWaves)), block(kNormWaves * 64);
    switch (split) {
      case 1: hipLaunchKernelGGL(text_norm_kernel<1>, grid, block, 0, stream, T, T_txt, h, ln_eps); break;
      case 2: hipLaunchKernelGGL(text_norm_kernel<2>, grid, block, 0, stream, T, T_txt, h, ln_eps); break;
      case 4: hipLaunchKernelGGL(text_norm_kernel<4>, grid, block, 0, stream, T, T_txt, h, ln_eps); break;
      case 8: hipLaunchKernelGGL(text_norm_kernel<8>, grid, block, 0, stream, T, T_txt, h, ln_eps); break;
      default: return hipErrorInvalidValue;
    }
  }
  hipLaunchKernelGGL(text_mean_kernel, dim3(B, (h + 255) / 256), dim3(256), 0, stream, T,
                     text_off, T_txt, h, g_text, ctx, err);
  return hipGetLastError();
}

}  // namespace sp
