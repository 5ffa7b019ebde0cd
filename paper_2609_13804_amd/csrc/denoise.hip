// The training pathway's noise gate and locally masked denoiser (Section
// "Trajectory-Aware Differentiable Optimization": the variance-preserving
// gate of Eq. 9 and the denoiser block after it).
//
//   x~ = sqrt(a) x + sqrt(1 - a) eps                         (per token)
//   h  = x~ + W_O (W_V LN1(x~) + b_V) + b_O                  (diagonal attention)
//   X^ = h + W_2 GELU(W_1 LN2(h) + b_1) + b_2
//
// Restricting the block's self-attention to the diagonal gives every token a
// single key, its own, so the softmax weight is 1 and the attention output is
// the value projection; the block is per-token work: four dense products on
// the matrix cores (gemm.hip) and five row kernels here.  The residual stream
// (x~, then h) stays float32; every product operand and result is bfloat16,
// rounded once to nearest-even.
//
// Row kernels: 16-byte accesses (8 bfloat16 or 4 float32 elements); the
// LayerNorm kernels run one wave per token row and sum in a fixed order
// (per-lane partial sums, then a butterfly), so results are deterministic.
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
  const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + kDenoiseLnEps);
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

// x~ = sqrt(a) x + sqrt(1 - a) eps into xt (float32), and LN1(x~) into z.
// One wave per row.
__global__ __launch_bounds__(64 * kRowWaves) void gate_ln_kernel(
    const uint16_t* __restrict__ X, const float* __restrict__ alpha,
    const uint16_t* __restrict__ eps, int64_t T, int d, const float* __restrict__ g,
    const float* __restrict__ b, float* __restrict__ xt, uint16_t* __restrict__ z) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6);
  if (r >= T) return;
  const int nch = d / 8;
  const float a = alpha[r];
  const float sa = sqrtf(a), sb = sqrtf(1.0f - a);
  float v[kMaxChunks][8];
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    if (lane + 64 * i >= nch) break;
    const int64_t o = r * d + 8 * (lane + 64 * i);
    float x[8], e[8];
    load8(X + o, x);
    load8(eps + o, e);
#pragma unroll
    for (int k = 0; k < 8; ++k) v[i][k] = fmaf(sb, e[k], sa * x[k]);
    store8(xt + o, v[i]);
  }
  ln_store(v, nch, d, lane, g, b, z + r * d);
}

// h = (x~ + t) + b_O in place over xt, and LN2(h) into z.  One wave per row.
__global__ __launch_bounds__(64 * kRowWaves) void resid_ln_kernel(
    float* __restrict__ xt, const uint16_t* __restrict__ t, const float* __restrict__ bias,
    int64_t T, int d, const float* __restrict__ g, const float* __restrict__ b,
    uint16_t* __restrict__ z) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6);
  if (r >= T) return;
  const int nch = d / 8;
  float v[kMaxChunks][8];
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    if (lane + 64 * i >= nch) break;
    const int c = 8 * (lane + 64 * i);
    const int64_t o = r * d + c;
    float x[8], y[8], bb[8];
    load8(xt + o, x);
    load8(t + o, y);
    load8(bias + c, bb);
#pragma unroll
    for (int k = 0; k < 8; ++k) v[i][k] = (x[k] + y[k]) + bb[k];
    store8(xt + o, v[i]);
  }
  ln_store(v, nch, d, lane, g, b, z + r * d);
}

// The flat passes: one workgroup per row of width n (a multiple of 8), each
// thread taking 8-element chunks.
//   P = bf16(P + bias)
__global__ __launch_bounds__(256) void bias_kernel(uint16_t* __restrict__ P, int n,
                                                   const float* __restrict__ bias) {
  uint16_t* row = P + (int64_t)blockIdx.x * n;
  for (int c = 8 * threadIdx.x; c < n; c += 8 * 256) {
    float x[8], bb[8];
    load8(row + c, x);
    load8(bias + c, bb);
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] += bb[k];
    store8(row + c, x);
  }
}

//   H = bf16(GELU(H + b_1)), the exact GELU x Phi(x)
__global__ __launch_bounds__(256) void bias_gelu_kernel(uint16_t* __restrict__ H, int n,
                                                        const float* __restrict__ bias) {
  uint16_t* row = H + (int64_t)blockIdx.x * n;
  for (int c = 8 * threadIdx.x; c < n; c += 8 * 256) {
    float x[8], bb[8];
    load8(row + c, x);
    load8(bias + c, bb);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float y = x[k] + bb[k];
      x[k] = 0.5f * y * (1.0f + erff(y * 0.70710678118654752f));
    }
    store8(row + c, x);
  }
}

//   out = bf16((h + t) + b_2)
__global__ __launch_bounds__(256) void out_kernel(const float* __restrict__ h,
                                                  const uint16_t* __restrict__ t, int d,
                                                  const float* __restrict__ bias,
                                                  uint16_t* __restrict__ out) {
  const int64_t o = (int64_t)blockIdx.x * d;
  for (int c = 8 * threadIdx.x; c < d; c += 8 * 256) {
    float x[8], y[8], bb[8];
    load8(h + o + c, x);
    load8(t + o + c, y);
    load8(bias + c, bb);
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = (x[k] + y[k]) + bb[k];
    store8(out + o + c, x);
  }
}

}  // namespace

hipError_t launch_gate_denoise(const DenoiseArgs& a, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  const int d = a.d;
  const int64_t T = a.T;
  const unsigned rows = (unsigned)((T + kRowWaves - 1) / kRowWaves);
  uint16_t* P = a.buf_p;   // [T, d] bfloat16
  uint16_t* Q = a.buf_q;   // [T, d] bfloat16
  hipError_t e;
  hipLaunchKernelGGL(gate_ln_kernel, dim3(rows), dim3(64 * kRowWaves), 0, stream, a.X, a.alpha,
                     a.eps, T, d, a.ln1_g, a.ln1_b, a.xt, P);
  if ((e = launch_dense_bf16(P, a.W_v, T, d, d, Q, stream)) != hipSuccess) return e;     // W_V z
  hipLaunchKernelGGL(bias_kernel, dim3((unsigned)T), dim3(256), 0, stream, Q, d, a.b_v);
  if ((e = launch_dense_bf16(Q, a.W_o, T, d, d, P, stream)) != hipSuccess) return e;     // W_O u
  hipLaunchKernelGGL(resid_ln_kernel, dim3(rows), dim3(64 * kRowWaves), 0, stream, a.xt, P,
                     a.b_o, T, d, a.ln2_g, a.ln2_b, Q);
  if ((e = launch_dense_bf16(Q, a.W_1, T, 4 * (int64_t)d, d, a.hid, stream)) != hipSuccess)
    return e;                                                                             // W_1 z
  hipLaunchKernelGGL(bias_gelu_kernel, dim3((unsigned)T), dim3(256), 0, stream, a.hid, 4 * d,
                     a.b_1);
  if ((e = launch_dense_bf16(a.hid, a.W_2, T, d, 4 * d, P, stream)) != hipSuccess) return e;  // W_2 a
  hipLaunchKernelGGL(out_kernel, dim3((unsigned)T), dim3(256), 0, stream, a.xt, P, d, a.b_2,
                     a.out);
  return hipGetLastError();
}

}  // namespace sp
