// Text context of Algorithm 1 step 1 (Section "Conditional Sequential Pointer
// Policy": text projection, LayerNorm, gain g_text), reduced to the pointer
// query space:  c_b = g_text * mean_l LN(E_{b,l} W_text^T).
//
// The projection itself is a dense contraction (gemm.hip, float32 output,
// split over K into `split` partial products that are added here in a fixed
// order); this kernel normalises each projected row (no affine parameters,
// biased variance, eps) and averages the rows of an image.  One workgroup per image;
// each wave normalises whole rows with wave-level reductions and keeps a
// private running sum, and the waves' sums are combined in a fixed order.
#include "sp_internal.h"

namespace sp {
namespace {

constexpr int kPoolWaves = 8;

__device__ inline float wsum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

template <int SPLIT>
__global__ __launch_bounds__(kPoolWaves * 64) void text_pool_kernel(
    const float* __restrict__ T, const int32_t* __restrict__ text_off, int64_t T_txt, int h,
    float g_text, float eps, float* __restrict__ ctx, int32_t* err) {
  __shared__ float part[kPoolWaves][1024];
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t r0 = text_off[b], r1 = text_off[b + 1];
  const int per = h / 64;
  if (r0 < 0 || r1 < r0 || r1 > T_txt) {
    if (threadIdx.x == 0) set_device_error(err, SP_DEV_BAD_OFFSETS);
    for (int c = threadIdx.x; c < h; c += blockDim.x) ctx[(int64_t)b * h + c] = 0.0f;
    return;
  }
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
  for (int64_t r = r0 + wave; r < r1; r += kPoolWaves) {
    // The K-split partial products of this row, all loads in flight at once,
    // added in split order.
    const float* row = T + r * h;
    float xp[SPLIT][16];
#pragma unroll
    for (int p = 0; p < SPLIT; ++p)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        xp[p][i] = i < per ? row[(int64_t)p * T_txt * h + lane + 64 * i] : 0.0f;
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      x[i] = xp[0][i];
#pragma unroll
      for (int p = 1; p < SPLIT; ++p) x[i] += xp[p][i];
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += x[i];
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
      if (i < per) acc[i] += (x[i] - mean) * inv;
  }
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < per) part[wave][lane + 64 * i] = acc[i];
  __syncthreads();
  const int64_t L = r1 - r0;
  for (int c = threadIdx.x; c < h; c += blockDim.x) {
    float s = 0.0f;
    for (int w = 0; w < kPoolWaves; ++w) s += part[w][c];
    ctx[(int64_t)b * h + c] = L > 0 ? g_text * (s / (float)L) : 0.0f;
  }
}

}  // namespace

hipError_t launch_text_pool(const float* T, int split, const int32_t* text_off, int B,
                            int64_t T_txt, int h, float g_text, float ln_eps, float* ctx,
                            int32_t* err, hipStream_t stream) {
  if (B == 0) return hipSuccess;
  const dim3 grid(B), block(kPoolWaves * 64);
  switch (split) {
    case 1: hipLaunchKernelGGL(text_pool_kernel<1>, grid, block, 0, stream, T, text_off, T_txt, h,
                               g_text, ln_eps, ctx, err); break;
    case 2: hipLaunchKernelGGL(text_pool_kernel<2>, grid, block, 0, stream, T, text_off, T_txt, h,
                               g_text, ln_eps, ctx, err); break;
    case 4: hipLaunchKernelGGL(text_pool_kernel<4>, grid, block, 0, stream, T, text_off, T_txt, h,
                               g_text, ln_eps, ctx, err); break;
    case 8: hipLaunchKernelGGL(text_pool_kernel<8>, grid, block, 0, stream, T, text_off, T_txt, h,
                               g_text, ln_eps, ctx, err); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sp
