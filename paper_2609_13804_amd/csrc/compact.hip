// Algorithm 1 step 5: physically gather the kept visual tokens (native order)
// ahead of the prompt rows (Section "Train-Inference Alignment").
//
// Pure data movement, bound by HBM bandwidth: every kept row and every text
// row is read once and written once with 16-byte vector accesses, one wave per
// row, all of a row's loads in flight before its stores.  Grid: (row blocks, image).  For the packed layout each workgroup
// derives its image's start row from the kept counts of the earlier images
// (cu[b] = text_off[b] - text_off[0] + sum_{b' < b} K_b'), so no separate
// scan kernel is needed; the first workgroup of each image writes its
// sequence length entry.
#include "sp_internal.h"

namespace sp {
namespace {

constexpr int kCompactWaves = 4;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kCompactWaves * 64) void compact_kernel(CompactArgs p) {
  __shared__ int64_t red[kCompactWaves * 64];
  const int b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t t0 = p.text_off[b], t1 = p.text_off[b + 1];
  const int64_t i0 = p.img_off[b], i1 = p.img_off[b + 1];
  const int64_t k0 = p.kept_off[b], k1 = p.kept_off[b + 1];
  const int64_t K = p.kept_cnt[b];
  if (t1 < t0 || i1 < i0 || k1 < k0 || k0 < 0 || K < 0 || K > k1 - k0) {
    if (tid == 0) set_device_error(p.err, SP_DEV_BAD_OFFSETS);
    return;
  }
  const int64_t L = t1 - t0;
  int64_t base;
  if (p.layout == SP_LAYOUT_PADDED) {
    base = (int64_t)b * p.rows_per_image;
    if (K + L > p.rows_per_image) {
      if (tid == 0) set_device_error(p.err, SP_DEV_OUTPUT_OVERFLOW);
      return;
    }
    if (blockIdx.x == 0 && tid == 0) p.seq_info[b] = (int32_t)(K + L);
  } else {
    int64_t s = 0;
    for (int i = tid; i < b; i += blockDim.x) s += p.kept_cnt[i];
    red[tid] = s;
    __syncthreads();
    for (int w = blockDim.x / 2; w > 0; w >>= 1) {
      if (tid < w) red[tid] += red[tid + w];
      __syncthreads();
    }
    base = red[0] + (t0 - p.text_off[0]);
    if (blockIdx.x == 0 && tid == 0) {
      p.seq_info[b + 1] = (int32_t)(base + K + L);
      if (b == 0) p.seq_info[0] = 0;
    }
  }
  if (base + K + L > p.out_rows) {
    if (tid == 0) set_device_error(p.err, SP_DEV_OUTPUT_OVERFLOW);
    return;
  }
  const int64_t row_bytes = (int64_t)p.d * p.elem_bytes;
  const int chunks = (int)(row_bytes / 16);
  const char* X = static_cast<const char*>(p.X);
  const char* E = static_cast<const char*>(p.E);
  char* out = static_cast<char*>(p.out);
  const int64_t stride = (int64_t)gridDim.x * kCompactWaves;
  for (int64_t r = (int64_t)blockIdx.x * kCompactWaves + wave; r < K + L; r += stride) {
    const char* src;
    if (r < K) {
      const int64_t idx = p.kept_idx[k0 + r];
      if (idx < 0 || idx >= i1 - i0) {
        if (lane == 0) set_device_error(p.err, SP_DEV_BAD_OFFSETS);
        continue;
      }
      src = X + (i0 + idx) * row_bytes;
    } else {
      src = E + (t0 + r - K) * row_bytes;
    }
    char* dst = out + (base + r) * row_bytes;
    // A row's loads are all issued before its stores (eight 16-byte chunks per
    // lane at a time, 8 KB per wave in flight); load-store pairs through
    // possibly aliasing pointers would each wait for their own load.  Chunk
    // indices past the row are clamped to its last chunk rather than skipped:
    // those lanes copy that chunk again (the same bytes to the same place), and
    // the loop stays free of branches, whose joins would make the compiler wait
    // for every access before the next.
    const u32x4_t* s16 = reinterpret_cast<const u32x4_t*>(src);
    u32x4_t* d16 = reinterpret_cast<u32x4_t*>(dst);
    for (int c0 = 0; c0 < chunks; c0 += 8 * 64) {
      u32x4_t v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int c = c0 + lane + 64 * k;
        v[k] = s16[c < chunks ? c : chunks - 1];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int c = c0 + lane + 64 * k;
        d16[c < chunks ? c : chunks - 1] = v[k];
      }
    }
  }
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, hipStream_t stream) {
  if (a.B == 0) return hipSuccess;
  int64_t per_image = a.layout == SP_LAYOUT_PADDED ? a.rows_per_image : a.out_rows / a.B + 1;
  int64_t y = (per_image + kCompactWaves - 1) / kCompactWaves;
  if (y < 1) y = 1;
  if (y > 256) y = 256;
  hipLaunchKernelGGL(compact_kernel, dim3((unsigned)y, (unsigned)a.B), dim3(kCompactWaves * 64), 0,
                     stream, a);
  return hipGetLastError();
}

}  // namespace sp
