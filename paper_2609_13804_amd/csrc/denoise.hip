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
// the matrix cores (gemm.hip; the value bias and the MLP's bias and GELU run
// in their epilogues) and three row kernels here.  The residual stream
// (x~, then h) stays float32; every product operand and result is bfloat16,
// rounded once to nearest-even.
//
// Row kernels (row_ops.h for the shared pieces): 16-byte accesses (8 bfloat16
// or 4 float32 elements); the LayerNorm kernels run one wave per token row and
// sum in a fixed order (per-lane partial sums, then a butterfly), so results
// are deterministic.  The residual + LayerNorm kernel serves the input
// encoder too (launcher below).
#include "sp_internal.h"
#include "row_ops.h"

namespace sp {
namespace {

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

// The flat pass: one workgroup per row of width d (a multiple of 8), each
// thread taking 8-element chunks.
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

hipError_t launch_resid_ln(float* xt, const uint16_t* t, const float* bias, int64_t T, int d,
                           const float* g, const float* b, uint16_t* z, hipStream_t stream) {
  if (T > 0)
    hipLaunchKernelGGL(resid_ln_kernel, dim3((unsigned)((T + kRowWaves - 1) / kRowWaves)),
                       dim3(64 * kRowWaves), 0, stream, xt, t, bias, T, d, g, b, z);
  return hipGetLastError();
}

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
  if ((e = launch_dense_bf16(P, a.W_v, T, d, d, Q, stream, a.b_v)) != hipSuccess) return e;  // W_V z + b_V
  if ((e = launch_dense_bf16(Q, a.W_o, T, d, d, P, stream)) != hipSuccess) return e;     // W_O u
  hipLaunchKernelGGL(resid_ln_kernel, dim3(rows), dim3(64 * kRowWaves), 0, stream, a.xt, P,
                     a.b_o, T, d, a.ln2_g, a.ln2_b, Q);
  if ((e = launch_dense_bf16(Q, a.W_1, T, 4 * (int64_t)d, d, a.hid, stream, a.b_1, true)) !=
      hipSuccess)
    return e;                                                                  // GELU(W_1 z + b_1)
  if ((e = launch_dense_bf16(a.hid, a.W_2, T, d, 4 * d, P, stream)) != hipSuccess) return e;  // W_2 a
  hipLaunchKernelGGL(out_kernel, dim3((unsigned)T), dim3(256), 0, stream, a.xt, P, d, a.b_2,
                     a.out);
  return hipGetLastError();
}

}  // namespace sp
