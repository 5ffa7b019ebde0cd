// Algorithm 1 steps 2-4 on gfx950: the sequential pointer selection with STOP.
//
// For one group (episode) with tokens 0..n-1 the pointer step of Eq. 4 under
// the one-layer reading is
//     u_t     = c + q_e + sum_tau alpha_tau v_tau,
//     alpha   = softmax_tau(sigma <q_e, k_tau>)          over the history,
//     l_t(j)  = sigma <u_t, k_j>,   l_t(STOP) = sigma <u_t, k_stop> + b_stop.
// By linearity l_t(j) = sigma (cK[j] + A[e, j] + sum_tau alpha_tau B[tau, j]) with
//     A = [Q; q_start] [K; k_stop; k_start]^T,  B = [V; v_start] [K; k_stop]^T,
//     cK = c [K; k_stop]^T,
// and the history scores are sigma A[e, col(tau)].  A and B are dense
// contractions computed once per group on the matrix cores (gemm.hip), so a
// step needs only the rows A[e, :] and B[e, :] of the newest history entry e:
// one dependent load, then O(t * n) float32 FMAs over history rows kept in
// LDS.  One workgroup runs one episode end to end, thread j owning candidate
// column j (j = n is STOP), so no step ever leaves the compute unit.
//
// Gram layout per group (float32, row stride ld): rows [0, n) A rows of the
// tokens, row n the A row of START, rows [n+1, 2n+1) B rows of the tokens,
// row 2n+1 the B row of START; columns [0, n) tokens, n STOP, n+1 START.
#include "sp_internal.h"

namespace sp {
namespace {

constexpr int kMaxWaves = 16;

// Dynamic LDS of the selection kernel (byte offsets), shared by host and device.
struct SelLds {
  int hist, arow, hrow, alpha, red, stop, total;
  __host__ __device__ SelLds(int rows, int hist_ld, int max_cap) {
    hist = 0;
    arow = hist + rows * hist_ld * 4;
    hrow = arow + (hist_ld + 4) * 4;
    alpha = hrow + (max_cap + 1) * 4;
    red = (alpha + (max_cap + 1) * 4 + 15) & ~15;
    stop = red + 2 * kMaxWaves * 8;
    total = stop + 16;
  }
};

// Order-preserving key: larger value wins, equal values go to the lower index.
__device__ inline uint64_t make_key(float v, int idx) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint32_t)(~(uint32_t)idx);
}
__device__ inline int key_index(uint64_t k) { return (int)(~(uint32_t)(k & 0xffffffffu)); }
__device__ inline float key_value(uint64_t k) {
  uint32_t u = (uint32_t)(k >> 32);
  u = (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u;
  return __uint_as_float(u);
}

__device__ inline uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = __shfl_xor((uint32_t)v, m, 64);
  uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m, 64);
  return ((uint64_t)hi << 32) | lo;
}

// Keys are unique (they carry the index) or zero (no candidate).
__device__ inline void top2_merge(uint64_t& a1, uint64_t& a2, uint64_t b1, uint64_t b2) {
  const uint64_t hi = a1 > b1 ? a1 : b1;
  const uint64_t lo = a1 > b1 ? b1 : a1;
  uint64_t second = lo > a2 ? lo : a2;
  second = second > b2 ? second : b2;
  a1 = hi;
  a2 = second;
}

__device__ inline float wave_max(float v) {
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}
__device__ inline float wave_sum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// ------------------------------------------------------------------ c . K

// cK[g, j] = c_b . K_j for the group's tokens and STOP, float32 accumulation.
// One wave per column; lane l covers elements l, l+64, ...
template <typename T>
__global__ __launch_bounds__(256) void ck_kernel(const T* __restrict__ KQV, int64_t T_vis, int h,
                                                 const float* __restrict__ ctx,
                                                 const int32_t* __restrict__ grp_off,
                                                 const int32_t* __restrict__ grp_img, int B,
                                                 int max_group, float* __restrict__ cK, int ck_ld,
                                                 int cols_per_block) {
  const int g = blockIdx.y;
  const int64_t g0 = grp_off[g], n = grp_off[g + 1] - g0;
  const int b = grp_img[g];
  if (g0 < 0 || n < 0 || n > max_group || g0 + n > T_vis || b < 0 || b >= B) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int per = h / 64;
  float c[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) c[i] = i < per ? ctx[(int64_t)b * h + lane + 64 * i] : 0.0f;
  const int64_t ld = 3 * (int64_t)h;
  const int j0 = blockIdx.x * cols_per_block;
  for (int j = j0 + wave; j < j0 + cols_per_block && j <= n; j += 4) {
    const T* krow = KQV + (j < n ? (g0 + j) : (T_vis + 1)) * ld;
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < per) s = fmaf(c[i], (float)krow[lane + 64 * i], s);
    s = wave_sum(s);
    if (lane == 0) cK[(int64_t)g * ck_ld + j] = s;
  }
}

// ------------------------------------------------------------------ the recurrence

struct SelParams {
  const float* gram;
  int64_t gstride;
  int ld;
  const float* cK;
  int ck_ld;
  const int32_t* img_off;
  int B;
  const int32_t* grp_off;
  const int32_t* grp_img;
  const int32_t* grp_cap;
  int64_t T_vis;
  int max_group;
  int max_cap;
  int hist_lds_rows;   // history rows held in LDS; older ones read from the Gram buffer
  int hist_ld;         // LDS row stride (floats)
  float sigma;
  float b_stop;
  uint32_t flags;
  int32_t* grp_kept;   // [G, max_cap] group-local kept indices, ascending
  int32_t* grp_count;  // [G]
  int32_t* grp_cnt_out;
  float* trace;
  int trace_steps;
  int32_t* err;
};

template <bool TRACE>
__global__ __launch_bounds__(1024) void select_kernel(SelParams p) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int g = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int nwaves = blockDim.x >> 6;

  const int64_t g0 = p.grp_off[g], g1 = p.grp_off[g + 1];
  const int n = (int)(g1 - g0);
  const int cap = p.grp_cap[g];
  const int b = p.grp_img[g];
  {
    int code = 0;
    if (g0 < 0 || g1 < g0 || g1 > p.T_vis || b < 0 || b >= p.B) code = SP_DEV_BAD_OFFSETS;
    else if (n > p.max_group) code = SP_DEV_GROUP_TOO_LARGE;
    else if (cap < 0 || (cap < n ? cap : n) > p.max_cap) code = SP_DEV_BAD_CAP;
    else if (g0 < p.img_off[b] || g1 > p.img_off[b + 1]) code = SP_DEV_BAD_OFFSETS;
    if (code) {
      if (tid == 0) {
        set_device_error(p.err, code);
        p.grp_count[g] = 0;
        if (p.grp_cnt_out) p.grp_cnt_out[g] = 0;
      }
      return;
    }
  }
  const bool no_history = (p.flags & SP_NO_HISTORY) != 0;
  const int R = p.hist_lds_rows;
  const int HL = p.hist_ld;

  const SelLds L(R, HL, p.max_cap);
  float* hist = reinterpret_cast<float*>(smem + L.hist);        // [R][HL] history B rows
  float* arow = reinterpret_cast<float*>(smem + L.arow);        // [HL + 4] A row of newest entry
  int* hrow = reinterpret_cast<int*>(smem + L.hrow);            // [max_cap + 1] history rows
  float* alpha = reinterpret_cast<float*>(smem + L.alpha);      // [max_cap + 1] softmax weights
  uint64_t* red = reinterpret_cast<uint64_t*>(smem + L.red);    // [2][kMaxWaves] wave maxima
  float* stop_sh = reinterpret_cast<float*>(smem + L.stop);     // STOP logit (trace)

  const float* A = p.gram + (int64_t)g * p.gstride;        // A row r: A + r * ld
  const float* Bm = A + (int64_t)(n + 1) * p.ld;           // B row r: Bm + r * ld
  const int j = tid;
  const bool col = j <= n;                                 // owns a candidate column
  const float ck = col ? p.cK[(int64_t)g * p.ck_ld + j] : 0.0f;

  // History entry 0 is START (row n of A and B, column n + 1 of A).
  if (j <= n + 1) arow[j] = A[(int64_t)n * p.ld + j];
  if (col) {
    const float bv = Bm[(int64_t)n * p.ld + j];
    if (R > 0) hist[j] = bv;
  }
  if (tid == 0) hrow[0] = n;
  bool selected = false;
  int hlen = 1;
  int kept = 0;
  __syncthreads();

  for (int t = 1; t <= cap; ++t) {
    // Softmax weights of the history (one wave).
    if (wave == 0) {
      float m = -INFINITY;
      for (int tau = lane; tau < hlen; tau += 64) {
        const int r = hrow[tau];
        const float s = p.sigma * arow[r == n ? n + 1 : r];
        alpha[tau] = s;
        m = fmaxf(m, s);
      }
      m = wave_max(m);
      float sum = 0.0f;
      for (int tau = lane; tau < hlen; tau += 64) {
        const float e = expf(alpha[tau] - m);
        alpha[tau] = e;
        sum += e;
      }
      sum = wave_sum(sum);
      for (int tau = lane; tau < hlen; tau += 64) alpha[tau] = alpha[tau] / sum;
    }
    __syncthreads();

    // Pointer logits of this thread's candidate.
    uint64_t k1 = 0, k2 = 0;
    float lj = 0.0f;
    if (col && !selected) {
      float acc = ck + arow[j];
      const int nl = hlen < R ? hlen : R;
      for (int tau = 0; tau < nl; ++tau) acc = fmaf(alpha[tau], hist[tau * HL + j], acc);
      for (int tau = nl; tau < hlen; ++tau)
        acc = fmaf(alpha[tau], Bm[(int64_t)hrow[tau] * p.ld + j], acc);
      lj = p.sigma * acc;
      if (j == n) {
        lj += p.b_stop;
        if (TRACE) *stop_sh = lj;
      }
      k1 = make_key(lj, j);
    }
    // First maximal candidate over the group (STOP has the largest index, so
    // it loses exact ties).
    for (int m = 32; m >= 1; m >>= 1) {
      const uint64_t o1 = shfl_xor_u64(k1, m);
      if (TRACE) {
        const uint64_t o2 = shfl_xor_u64(k2, m);
        top2_merge(k1, k2, o1, o2);
      } else {
        k1 = k1 > o1 ? k1 : o1;
      }
    }
    if (lane == 0) {
      red[wave] = k1;
      if (TRACE) red[kMaxWaves + wave] = k2;
    }
    __syncthreads();
    uint64_t best = 0, second = 0;
    for (int w = 0; w < nwaves; ++w) {
      if (TRACE) top2_merge(best, second, red[w], red[kMaxWaves + w]);
      else best = best > red[w] ? best : red[w];
    }
    const int a = key_index(best);       // best != 0: STOP always competes
    if (TRACE && tid == 0 && t <= p.trace_steps) {
      float* rec = p.trace + ((int64_t)g * p.trace_steps + (t - 1)) * 4;
      rec[0] = __int_as_float(a == n ? -1 : a);
      rec[1] = key_value(best);
      rec[2] = second ? key_value(second) : -INFINITY;
      rec[3] = *stop_sh;
    }
    if (a == n) break;
    ++kept;
    if (j == a) selected = true;
    if (!no_history) {
      // Append a to the history: its A row becomes the current row, its B row
      // the newest history row.
      if (tid == 0) hrow[hlen] = a;
      if (j <= n + 1) arow[j] = A[(int64_t)a * p.ld + j];
      if (col && hlen < R) hist[hlen * HL + j] = Bm[(int64_t)a * p.ld + j];
      ++hlen;
    }
    __syncthreads();
  }

  // Native order (Algorithm 1 step 4): kept positions are the set bits of the
  // selection mask, counted in ascending index order.
  __syncthreads();
  int32_t* red32 = reinterpret_cast<int32_t*>(red);
  const uint64_t ballot = __ballot(j < n && selected);
  if (lane == 0) red32[wave] = __popcll(ballot);
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wave; ++w) before += red32[w];
  if (j < n && selected) {
    const int pos = before + __popcll(ballot & ((1ull << lane) - 1ull));
    p.grp_kept[(int64_t)g * p.max_cap + pos] = j;
  }
  if (tid == 0) {
    p.grp_count[g] = kept;
    if (p.grp_cnt_out) p.grp_cnt_out[g] = kept;
  }
}

// Trace records past an episode's end carry taken = -2.
__global__ void trace_fill_kernel(float* trace, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) {
    float* rec = trace + i * 4;
    rec[0] = __int_as_float(-2);
    rec[1] = rec[2] = rec[3] = 0.0f;
  }
}

// Per image: concatenate its groups' kept lists in group order, offset to
// image-local indices.
__global__ __launch_bounds__(256) void finalize_kernel(const int32_t* __restrict__ img_off, int B,
                                                       const int32_t* __restrict__ grp_off,
                                                       const int32_t* __restrict__ grp_img, int G,
                                                       const int32_t* __restrict__ grp_kept,
                                                       const int32_t* __restrict__ grp_count,
                                                       int max_cap,
                                                       const int32_t* __restrict__ kept_off,
                                                       int32_t* __restrict__ kept_idx,
                                                       int32_t* __restrict__ kept_cnt,
                                                       int32_t* err) {
  const int b = blockIdx.x;
  const int64_t base = kept_off[b];
  const int64_t room = (int64_t)kept_off[b + 1] - base;
  if (base < 0 || room < 0) {
    if (threadIdx.x == 0) {
      set_device_error(err, SP_DEV_BAD_OFFSETS);
      kept_cnt[b] = 0;
    }
    return;
  }
  int64_t filled = 0;
  for (int g = 0; g < G; ++g) {
    if (grp_img[g] != b) continue;
    const int cnt = grp_count[g];
    const int off = grp_off[g] - img_off[b];
    if (filled + cnt > room) {
      if (threadIdx.x == 0) set_device_error(err, SP_DEV_OUTPUT_OVERFLOW);
      break;
    }
    for (int i = threadIdx.x; i < cnt; i += blockDim.x)
      kept_idx[base + filled + i] = off + grp_kept[(int64_t)g * max_cap + i];
    filled += cnt;
  }
  if (threadIdx.x == 0) kept_cnt[b] = (int32_t)filled;
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  if (a.G == 0) {
    if (a.B > 0)
      hipLaunchKernelGGL(finalize_kernel, dim3(a.B), dim3(256), 0, stream, a.img_off, a.B,
                         a.grp_off, a.grp_img, a.G, a.grp_kept, a.grp_count, a.max_cap, a.kept_off,
                         a.kept_idx, a.kept_cnt, a.err);
    return hipGetLastError();
  }
  hipError_t e = launch_gram_gemm(a.dtype, a.KQV, a.T_vis, a.h, a.grp_off, a.G, a.max_group,
                                  a.gram, a.gram_group_stride, a.gram_ld, a.err, stream);
  if (e != hipSuccess) return e;

  const int cols_per_block = 32;
  const dim3 ck_grid((a.max_group + 1 + cols_per_block - 1) / cols_per_block, a.G);
  if (a.dtype == SP_BF16)
    hipLaunchKernelGGL(ck_kernel<__bf16>, ck_grid, dim3(256), 0, stream, (const __bf16*)a.KQV,
                       a.T_vis, a.h, a.ctx, a.grp_off, a.grp_img, a.B, a.max_group, a.cK, a.ck_ld,
                       cols_per_block);
  else
    hipLaunchKernelGGL(ck_kernel<float>, ck_grid, dim3(256), 0, stream, (const float*)a.KQV,
                       a.T_vis, a.h, a.ctx, a.grp_off, a.grp_img, a.B, a.max_group, a.cK, a.ck_ld,
                       cols_per_block);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  const bool trace = (a.flags & SP_TRACE) && a.trace && a.trace_steps > 0;
  if (trace) {
    const int64_t count = (int64_t)a.G * a.trace_steps;
    hipLaunchKernelGGL(trace_fill_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0,
                       stream, a.trace, count);
  }

  SelParams p;
  p.gram = a.gram;
  p.gstride = a.gram_group_stride;
  p.ld = a.gram_ld;
  p.cK = a.cK;
  p.ck_ld = a.ck_ld;
  p.img_off = a.img_off;
  p.B = a.B;
  p.grp_off = a.grp_off;
  p.grp_img = a.grp_img;
  p.grp_cap = a.grp_cap;
  p.T_vis = a.T_vis;
  p.max_group = a.max_group;
  p.max_cap = a.max_cap;
  p.sigma = 1.0f / sqrtf((float)a.h);
  p.b_stop = a.b_stop;
  p.flags = a.flags;
  p.grp_kept = a.grp_kept;
  p.grp_count = a.grp_count;
  p.grp_cnt_out = a.grp_cnt;
  p.trace = trace ? a.trace : nullptr;
  p.trace_steps = trace ? a.trace_steps : 0;
  p.err = a.err;

  const int threads = (a.max_group + 2 + 63) / 64 * 64;
  p.hist_ld = (int)align_up((size_t)a.max_group + 1, 4);
  const size_t fixed = (size_t)SelLds(0, p.hist_ld, a.max_cap).total;
  const size_t row_bytes = (size_t)p.hist_ld * 4;
  size_t rows = fixed < (size_t)kLdsBytes ? ((size_t)kLdsBytes - fixed) / row_bytes : 0;
  const size_t want = (size_t)a.max_cap + 1;
  if (rows > want) rows = want;
  p.hist_lds_rows = (int)rows;
  const size_t lds = (size_t)SelLds((int)rows, p.hist_ld, a.max_cap).total;

  if (trace) {
    hipFuncSetAttribute((const void*)select_kernel<true>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(select_kernel<true>, dim3(a.G), dim3(threads), lds, stream, p);
  } else {
    hipFuncSetAttribute((const void*)select_kernel<false>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(select_kernel<false>, dim3(a.G), dim3(threads), lds, stream, p);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;

  hipLaunchKernelGGL(finalize_kernel, dim3(a.B), dim3(256), 0, stream, a.img_off, a.B, a.grp_off,
                     a.grp_img, a.G, a.grp_kept, a.grp_count, a.max_cap, a.kept_off, a.kept_idx,
                     a.kept_cnt, a.err);
  return hipGetLastError();
}

}  // namespace sp
