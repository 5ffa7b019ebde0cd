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
// Row kernels: one wave per token row, 64 lanes striding the row, sums in a
// fixed order (lane-strided partial sums, then a butterfly), so results are
// deterministic.
#include "sp_internal.h"

namespace sp {
namespace {

constexpr int kRowWaves = 4;
constexpr int kMaxPer = 64;         // row elements per lane: d <= 4096

__device__ __forceinline__ float wave_sum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// LayerNorm of the row held in v[0 .. per) (element lane + 64 i), scaled by g
// and shifted by b, written as bfloat16.
__device__ __forceinline__ void ln_store(const float (&v)[kMaxPer], int per, int d, int lane,
                                         const float* __restrict__ g,
                                         const float* __restrict__ b, uint16_t* __restrict__ z) {
  float s = 0.0f;
  for (int i = 0; i < per; ++i) s += v[i];
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
  for (int i = 0; i < per; ++i) {
    const float t = v[i] - mean;
    q = fmaf(t, t, q);
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + kDenoiseLnEps);
  for (int i = 0; i < per; ++i) {
    const int c = lane + 64 * i;
    z[c] = f32_to_bf16(fmaf((v[i] - mean) * rstd, g[c], b[c]));
  }
}

// x~ = sqrt(a) x + sqrt(1 - a) eps into xt (float32), and LN1(x~) into z.
__global__ __launch_bounds__(64 * kRowWaves) void gate_ln_kernel(
    const uint16_t* __restrict__ X, const float* __restrict__ alpha,
    const uint16_t* __restrict__ eps, int64_t T, int d, const float* __restrict__ g,
    const float* __restrict__ b, float* __restrict__ xt, uint16_t* __restrict__ z) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6);
  if (r >= T) return;
  const int per = d / 64;
  const float a = alpha[r];
  const float sa = sqrtf(a), sb = sqrtf(1.0f - a);
  float v[kMaxPer];
  for (int i = 0; i < per; ++i) {
    const int64_t o = r * d + lane + 64 * i;
    v[i] = fmaf(sb, bf16_to_f32(eps[o]), sa * bf16_to_f32(X[o]));
    xt[o] = v[i];
  }
  ln_store(v, per, d, lane, g, b, z + r * d);
}

// P = bf16(P + bias) over rows of width n.
__global__ __launch_bounds__(256) void bias_kernel(uint16_t* __restrict__ P, int64_t T, int n,
                                                   const float* __restrict__ bias) {
  const int64_t total = T * n;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256)
    P[i] = f32_to_bf16(bf16_to_f32(P[i]) + bias[i % n]);
}

// h = (x~ + t) + b_O in place over xt, and LN2(h) into z.
__global__ __launch_bounds__(64 * kRowWaves) void resid_ln_kernel(
    float* __restrict__ xt, const uint16_t* __restrict__ t, const float* __restrict__ bias,
    int64_t T, int d, const float* __restrict__ g, const float* __restrict__ b,
    uint16_t* __restrict__ z) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6);
  if (r >= T) return;
  const int per = d / 64;
  float v[kMaxPer];
  for (int i = 0; i < per; ++i) {
    const int c = lane + 64 * i;
    const int64_t o = r * d + c;
    v[i] = (xt[o] + bf16_to_f32(t[o])) + bias[c];
    xt[o] = v[i];
  }
  ln_store(v, per, d, lane, g, b, z + r * d);
}

// H = bf16(GELU(H + b_1)), the exact GELU x Phi(x), over rows of width n.
__global__ __launch_bounds__(256) void bias_gelu_kernel(uint16_t* __restrict__ H, int64_t T, int n,
                                                        const float* __restrict__ bias) {
  const int64_t total = T * n;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const float x = bf16_to_f32(H[i]) + bias[i % n];
    H[i] = f32_to_bf16(0.5f * x * (1.0f + erff(x * 0.70710678118654752f)));
  }
}

// out = bf16((h + t) + b_2).
__global__ __launch_bounds__(256) void out_kernel(const float* __restrict__ h,
                                                  const uint16_t* __restrict__ t, int64_t T, int d,
                                                  const float* __restrict__ bias,
                                                  uint16_t* __restrict__ out) {
  const int64_t total = T * d;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256)
    out[i] = f32_to_bf16((h[i] + bf16_to_f32(t[i])) + bias[i % d]);
}

unsigned grid_for(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (unsigned)(b < 8192 ? (b > 0 ? b : 1) : 8192);
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
  hipLaunchKernelGGL(bias_kernel, dim3(grid_for(T * d)), dim3(256), 0, stream, Q, T, d, a.b_v);
  if ((e = launch_dense_bf16(Q, a.W_o, T, d, d, P, stream)) != hipSuccess) return e;     // W_O u
  hipLaunchKernelGGL(resid_ln_kernel, dim3(rows), dim3(64 * kRowWaves), 0, stream, a.xt, P,
                     a.b_o, T, d, a.ln2_g, a.ln2_b, Q);
  if ((e = launch_dense_bf16(Q, a.W_1, T, 4 * (int64_t)d, d, a.hid, stream)) != hipSuccess)
    return e;                                                                             // W_1 z
  hipLaunchKernelGGL(bias_gelu_kernel, dim3(grid_for(T * 4 * d)), dim3(256), 0, stream, a.hid, T,
                     4 * d, a.b_1);
  if ((e = launch_dense_bf16(a.hid, a.W_2, T, d, 4 * d, P, stream)) != hipSuccess) return e;  // W_2 a
  hipLaunchKernelGGL(out_kernel, dim3(grid_for(T * d)), dim3(256), 0, stream, a.xt, P, T, d,
                     a.b_2, a.out);
  return hipGetLastError();
}

}  // namespace sp
