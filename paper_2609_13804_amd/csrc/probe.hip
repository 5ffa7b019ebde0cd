// LDS read bandwidth probe for gfx950 (libstepprune_probe.so; the benchmark
// loads it to measure the LDS peak it prices the selector's key scan with).
//
// Every workgroup fills 64 KB of LDS, then each thread reads 16-byte chunks
// (ds_read_b128) for `iters` rounds of eight reads, a wave reading 1 KB of
// consecutive chunks per read (no bank conflicts); one store per thread ends
// the kernel.  Two workgroups of
// 512 threads fit a compute unit's 160 KB of LDS.  Bytes read per launch:
// blocks * 512 * iters * 8 * 16.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 512;
constexpr int kChunks = 64 * 1024 / 16;   // 16-byte chunks of LDS per workgroup

__global__ __launch_bounds__(kThreads) void lds_read_probe_kernel(uint32_t* out, int iters) {
  __shared__ uint4 buf[kChunks];
  const int tid = threadIdx.x;
  for (int i = tid; i < kChunks; i += kThreads)
    buf[i] = make_uint4(i, 3u * i, 5u * i, 7u * i);
  __syncthreads();
  // Read k of a round is chunk base + 512 k (base < 512, so the eight reads
  // share one address and take immediate offsets of k * 8 KB).  The values
  // are consumed by empty asm statements: the loop does no ALU work besides
  // the address update.
  int base = tid;
  for (int it = 0; it < iters; ++it) {
    uint4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = buf[base + k * kThreads];
#pragma unroll
    for (int k = 0; k < 8; ++k) asm volatile("" ::"v"(v[k].x), "v"(v[k].y), "v"(v[k].z), "v"(v[k].w));
    base = (base + 64) & (kThreads - 1);
  }
  out[(int64_t)blockIdx.x * kThreads + tid] = (uint32_t)base;
}

}  // namespace

extern "C" {

// Launches the probe on `stream`: `blocks` workgroups of 512 threads, `iters`
// rounds each.  out: device buffer of blocks * 512 uint32.  Returns the launch
// status (hipErrorInvalidValue for a null buffer or non-positive sizes).
hipError_t stepprune_probe_lds(uint32_t* out, int blocks, int iters, hipStream_t stream) {
  if (!out || blocks <= 0 || iters <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lds_read_probe_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, out,
                     iters);
  return hipGetLastError();
}

// Threads per workgroup of the probe (bytes per launch use it).
int stepprune_probe_lds_threads(void) { return kThreads; }

}  // extern "C"
