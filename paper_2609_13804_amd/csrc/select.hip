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
// and the history scores are sigma A[e, col(tau)].  A, B and cK are dense
// contractions computed once per group on the matrix cores (gemm.hip), so a
// step needs only the rows A[e, :] and B[e, :] of the newest history entry e:
// one dependent load, then O(t * n) float32 FMAs.  One workgroup runs one
// episode end to end, thread j owning candidate column j (j = n is STOP), so
// no step ever leaves the compute unit: each thread keeps its column of the
// history B rows in registers (LDS past RREG entries), every wave computes the
// history softmax itself, reductions use DPP, and a step costs two barriers.
//
// Gram layout per group (float32, row stride ld): rows [0, n) A rows of the
// tokens, row n the A row of START, rows [n+1, 2n+1) B rows of the tokens,
// row 2n+1 the B row of START, rows 2n+2 .. 2n+4 three parts of cK whose sum
// is cK (the context enters the products as three rows of the working dtype);
// columns [0, n) tokens, n STOP, n+1 START.
#include "sp_internal.h"

namespace sp {
namespace {

constexpr int kMaxWaves = 16;

// ------------------------------------------------------------------ the recurrence

typedef float f32x32_t __attribute__((ext_vector_type(32)));

struct SelParams {
  const float* gram;
  int64_t gstride;
  int ld;
  const int32_t* img_off;
  int B;
  const int32_t* grp_off;
  const int32_t* grp_img;
  const int32_t* grp_cap;
  int64_t T_vis;
  int max_group;
  int max_cap;
  int lds_tier;        // history entries per column held in LDS after the registers
  int alpha_ld;        // softmax weight array length (floats, multiple of 16)
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

// Dynamic LDS of the recurrence (byte offsets), shared by host and device.
// The LDS history tier is column-major, [column][lds_tier], so one 16-byte
// read gives a thread four consecutive history entries of its column.
struct SelLds {
  int hist, arow, hcol, alpha, red, stop, total;
  __host__ __device__ SelLds(int lds_tier, int max_group, int max_cap, int alpha_ld) {
    hist = 0;
    arow = hist + (max_group + 1) * lds_tier * 4;
    hcol = arow + ((max_group + 2 + 3) & ~3) * 4;
    alpha = (hcol + (max_cap + 2) * 4 + 15) & ~15;
    red = alpha + alpha_ld * 4;
    stop = red + kMaxWaves * 16;
    total = stop + 16;
  }
};

// One workgroup runs one episode.  Thread j owns candidate column j (j = n is
// STOP, j = n + 1 only loads the START column of A rows).  History B values of
// its column: the first RREG in registers, the next lds_tier in LDS, any
// further ones re-read from the Gram buffer in batches.
template <int NT, int RREG, bool TRACE>
__global__ __launch_bounds__(NT) void select_kernel(SelParams p) {
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
  const int LT = p.lds_tier;
  const SelLds L(LT, p.max_group, p.max_cap, p.alpha_ld);
  float* hist = reinterpret_cast<float*>(smem + L.hist);      // [max_group + 1][LT]
  float* arow = reinterpret_cast<float*>(smem + L.arow);      // A row of the newest entry
  int* hcol = reinterpret_cast<int*>(smem + L.hcol);          // A column of each history entry
  float* alpha = reinterpret_cast<float*>(smem + L.alpha);    // softmax weights (zero padded)
  float4* red = reinterpret_cast<float4*>(smem + L.red);      // per wave {v1, i1, v2, i2}
  float* stop_sh = reinterpret_cast<float*>(smem + L.stop);

  const float* A = p.gram + (int64_t)g * p.gstride;           // A row r at A + r * ld
  const float* Bm = A + (int64_t)(n + 1) * p.ld;              // B row r at Bm + r * ld
  const int j = tid;
  const bool col = j <= n;
  const float* ckp = A + (int64_t)(2 * n + 2) * p.ld + j;   // the three parts of cK[j]
  const float ck = col ? (ckp[0] + ckp[p.ld]) + ckp[2 * p.ld] : 0.0f;
  const float sigma = p.sigma;
  float* hist_j = hist + (col ? j : 0) * LT;

  // Register-resident history of this column: up to 128 values in four
  // separate 32-wide vector registers.  Reads use constant slots after
  // unrolling; a write picks the vector with a uniform branch and the element
  // with an indexed register move.  Separate variables rather than an array,
  // and conditions the optimiser cannot prove exclusive, keep every access a
  // register operation (an aggregate written at a dynamic index would be
  // placed in scratch memory).
  static_assert(RREG % 32 == 0 && RREG <= 128, "history registers come in 32-wide vectors");
  constexpr int NV = RREG / 32;
  f32x32_t h0{}, h1{}, h2{}, h3{};
  auto hget = [&](int i) -> float {
    return i < 32 ? h0[i & 31] : i < 64 ? h1[i & 31] : i < 96 ? h2[i & 31] : h3[i & 31];
  };
  auto hput = [&](int pos, float x) {
    const int e = pos & 31;
    const int k = pos >> 5;
    if (__builtin_amdgcn_readfirstlane(k == 0)) h0[e] = x;
    if (NV > 1 && __builtin_amdgcn_readfirstlane(k == 1)) h1[e] = x;
    if (NV > 2 && __builtin_amdgcn_readfirstlane(k == 2)) h2[e] = x;
    if (NV > 3 && __builtin_amdgcn_readfirstlane(k == 3)) h3[e] = x;
  };
  // A column of history entry lane + 64 k, for the first 256 entries.
  int hc0 = lane == 0 ? n + 1 : 0, hc1 = 0, hc2 = 0, hc3 = 0;

  // History entry 0 is START: row n of A and B, column n + 1 of A.
  if (j <= n + 1) arow[j] = A[(int64_t)n * p.ld + j];
  h0[0] = col ? Bm[(int64_t)n * p.ld + j] : 0.0f;
  if (tid == 0) hcol[0] = n + 1;
  bool selected = false;
  int hl = 1;       // history length
  int kept = 0;
  __syncthreads();

  for (int t = 1; t <= cap; ++t) {
    // ---- softmax of sigma * A[e, history]; every wave computes the same
    // weights and writes the same values to the shared array, reading back only
    // what it wrote itself.
    const int hpad = (hl + 15) & ~15;
    if (hl <= 256) {
      float sv[4];
      float m = -INFINITY;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        sv[k] = -INFINITY;
        if (64 * k < hl) {
          const int hc = k == 0 ? hc0 : k == 1 ? hc1 : k == 2 ? hc2 : hc3;
          if (lane + 64 * k < hl) sv[k] = sigma * arow[hc];
          m = fmaxf(m, sv[k]);
        }
      }
      m = wave_max_dpp(m);
      float sum = 0.0f;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (64 * k < hl) {
          sv[k] = lane + 64 * k < hl ? expf(sv[k] - m) : 0.0f;
          sum += sv[k];
        }
      }
      sum = wave_sum_dpp(sum);
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (lane + 64 * k < hpad) alpha[lane + 64 * k] = sv[k] / sum;
    } else {
      // Longer histories: scores are recomputed in each pass so that only
      // final weights (identical in every wave) are ever written.
      float m = -INFINITY;
      for (int tau = lane; tau < hl; tau += 64) m = fmaxf(m, sigma * arow[hcol[tau]]);
      m = wave_max_dpp(m);
      float sum = 0.0f;
      for (int tau = lane; tau < hl; tau += 64) sum += expf(sigma * arow[hcol[tau]] - m);
      sum = wave_sum_dpp(sum);
      for (int tau = lane; tau < hl; tau += 64) alpha[tau] = expf(sigma * arow[hcol[tau]] - m) / sum;
      if (hl + lane < hpad) alpha[hl + lane] = 0.0f;
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();

    // ---- pointer logit of this thread's candidate
    float acc = col ? ck + arow[j] : 0.0f;
#pragma unroll
    for (int blk = 0; blk < RREG; blk += 16) {
      if (blk < hl) {
        const float4* a4 = reinterpret_cast<const float4*>(alpha + blk);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 x = a4[q];
          acc = fmaf(x.x, hget(blk + 4 * q + 0), acc);
          acc = fmaf(x.y, hget(blk + 4 * q + 1), acc);
          acc = fmaf(x.z, hget(blk + 4 * q + 2), acc);
          acc = fmaf(x.w, hget(blk + 4 * q + 3), acc);
        }
      }
    }
    if (hl > RREG) {
      const int lds_end = hl < RREG + LT ? hl : RREG + LT;
      int tau = RREG;
      for (; tau + 4 <= lds_end; tau += 4) {
        const float4 x = *reinterpret_cast<const float4*>(alpha + tau);
        const float4 y = col ? *reinterpret_cast<const float4*>(hist_j + (tau - RREG))
                             : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        acc = fmaf(x.x, y.x, acc);
        acc = fmaf(x.y, y.y, acc);
        acc = fmaf(x.z, y.z, acc);
        acc = fmaf(x.w, y.w, acc);
      }
      for (; tau < lds_end; ++tau) acc = fmaf(alpha[tau], col ? hist_j[tau - RREG] : 0.0f, acc);
      for (; tau < hl; tau += 8) {
        float hv[8], av[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          hv[u] = 0.0f;
          av[u] = 0.0f;
          if (tau + u < hl) {
            const int c = hcol[tau + u];
            const int r = c == n + 1 ? n : c;
            av[u] = alpha[tau + u];
            if (col) hv[u] = Bm[(int64_t)r * p.ld + j];
          }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = fmaf(av[u], hv[u], acc);
      }
    }
    float lj = sigma * acc;
    if (j == n) {
      lj += p.b_stop;
      if (TRACE) *stop_sh = lj;
    }
    const bool valid = col && !selected;

    // ---- first maximal candidate of this wave (lowest index on ties)
    const float v = valid ? lj : -INFINITY;
    const float vmax = wave_max_dpp(v);
    const uint64_t mask = __ballot(valid && v == vmax);
    const int i1 = mask ? wave * 64 + __ffsll((unsigned long long)mask) - 1 : -1;
    float v2 = -INFINITY;
    int i2 = -1;
    if (TRACE) {
      const bool keep = valid && j != i1;
      const float w2 = keep ? lj : -INFINITY;
      v2 = wave_max_dpp(w2);
      const uint64_t mask2 = __ballot(keep && w2 == v2);
      i2 = mask2 ? wave * 64 + __ffsll((unsigned long long)mask2) - 1 : -1;
    }
    if (lane == 0) red[wave] = make_float4(vmax, __int_as_float(i1), v2, __int_as_float(i2));
    __syncthreads();

    // ---- merge the waves' candidates with one wave-wide reduction: lane w
    // holds wave w's best (lanes 16 + w its runner-up); largest value, then
    // lowest index.
    float cv = -INFINITY;
    int ci = -1;
    if (lane < nwaves) {
      const float4 r = red[lane];
      cv = r.x;
      ci = __float_as_int(r.y);
    } else if (TRACE && lane >= 16 && lane < 16 + nwaves) {
      const float4 r = red[lane - 16];
      cv = r.z;
      ci = __float_as_int(r.w);
    }
    const float bv = wave_max_dpp(ci >= 0 ? cv : -INFINITY);
    const int a = wave_min_dpp(ci >= 0 && cv == bv ? ci : INT_MAX);   // STOP always competes
    if (TRACE) {
      // Runner-up over the same lanes (whole wave active for the reductions).
      const bool rest = ci >= 0 && ci != a;
      const float sv2 = wave_max_dpp(rest ? cv : -INFINITY);
      const int si2 = wave_min_dpp(rest && cv == sv2 ? ci : INT_MAX);
      if (tid == 0 && t <= p.trace_steps) {
      float* rec = p.trace + ((int64_t)g * p.trace_steps + (t - 1)) * 4;
      rec[0] = __int_as_float(a == n ? -1 : a);
      rec[1] = bv;
      rec[2] = si2 != INT_MAX ? sv2 : -INFINITY;
      rec[3] = *stop_sh;
      }
    }
    if (a == n) break;
    ++kept;
    if (j == a) selected = true;
    if (!no_history) {
      // Append a: its A row becomes the current row, its B row the newest
      // history entry of every column.
      if (tid == 0) hcol[hl] = a;
      {
        const int k = hl >> 6;
        const bool mine = lane == (hl & 63);
        if (__builtin_amdgcn_readfirstlane(k == 0) && mine) hc0 = a;
        if (__builtin_amdgcn_readfirstlane(k == 1) && mine) hc1 = a;
        if (__builtin_amdgcn_readfirstlane(k == 2) && mine) hc2 = a;
        if (__builtin_amdgcn_readfirstlane(k == 3) && mine) hc3 = a;
      }
      if (j <= n + 1) arow[j] = A[(int64_t)a * p.ld + j];
      const float bv_new = col ? Bm[(int64_t)a * p.ld + j] : 0.0f;
      if (hl < RREG) hput(hl, bv_new);
      else if (hl < RREG + LT && col) hist_j[hl - RREG] = bv_new;
      ++hl;
    }
    __syncthreads();
  }

  // ---- native order (Algorithm 1 step 4): ascending positions of the set bits
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
  record_event(a.events, 0, stream);
  GramArgs ga;
  ga.dtype = a.dtype;
  ga.KQV = a.KQV;
  ga.T_vis = a.T_vis;
  ga.h = a.h;
  ga.ctx = a.ctx;
  ga.B = a.B;
  ga.grp_off = a.grp_off;
  ga.grp_img = a.grp_img;
  ga.G = a.G;
  ga.max_group = a.max_group;
  ga.csplit = a.csplit;
  ga.gram = a.gram;
  ga.gram_group_stride = a.gram_group_stride;
  ga.gram_ld = a.gram_ld;
  ga.err = a.err;
  hipError_t e = launch_gram_gemm(ga, stream);
  if (e != hipSuccess) return e;
  record_event(a.events, 1, stream);

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
  const int nt_class = threads <= 320 ? 320 : threads <= 640 ? 640 : 1024;
  const int need = a.max_cap + 1;                       // longest possible history
  // History registers per thread: the VGPR budget is 512 / (waves per SIMD),
  // so 16 waves allow 64 values, 10 waves 96 and 5 waves 128.
  const int rmax = nt_class == 1024 ? 64 : nt_class == 640 ? 96 : 128;
  int rreg = (need + 31) / 32 * 32;
  if (rreg > rmax) rreg = rmax;
  p.alpha_ld = (int)align_up((size_t)a.max_cap + 2, 16);
  const size_t fixed = (size_t)SelLds(0, a.max_group, a.max_cap, p.alpha_ld).total;
  const size_t per_entry = (size_t)(a.max_group + 1) * 4;   // one LDS history entry, all columns
  size_t lt_max = fixed < (size_t)kLdsBytes ? ((size_t)kLdsBytes - fixed) / per_entry : 0;
  // Column stride of 8k + 4 floats keeps the 16-byte reads of eight
  // consecutive columns on distinct banks.
  lt_max = lt_max >= 4 ? (lt_max - 4) / 8 * 8 + 4 : 0;
  size_t lt = 0;
  if (need > rreg) {
    lt = (size_t)(need - rreg + 3) / 8 * 8 + 4;   // smallest 8k + 4 >= the entries needed
    if (lt > lt_max) lt = lt_max;
  }
  p.lds_tier = (int)lt;
  const size_t lds = (size_t)SelLds((int)lt, a.max_group, a.max_cap, p.alpha_ld).total;

  const void* fn = nullptr;
#define SP_PICK(NT, RR)                                                             \
  if (nt_class == NT && rreg == RR)                                                 \
    fn = trace ? (const void*)select_kernel<NT, RR, true> : (const void*)select_kernel<NT, RR, false>;
  SP_PICK(320, 32) SP_PICK(320, 64) SP_PICK(320, 96) SP_PICK(320, 128)
  SP_PICK(640, 32) SP_PICK(640, 64) SP_PICK(640, 96)
  SP_PICK(1024, 32) SP_PICK(1024, 64)
#undef SP_PICK
  if (!fn) return hipErrorInvalidValue;
  record_event(a.events, 2, stream);
  if ((e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) != hipSuccess)
    return e;
  void* kargs[] = {&p};
  if ((e = hipLaunchKernel(fn, dim3(a.G), dim3(threads), kargs, lds, stream)) != hipSuccess) return e;
  record_event(a.events, 3, stream);

  hipLaunchKernelGGL(finalize_kernel, dim3(a.B), dim3(256), 0, stream, a.img_off, a.B, a.grp_off,
                     a.grp_img, a.G, a.grp_kept, a.grp_count, a.max_cap, a.kept_off, a.kept_idx,
                     a.kept_cnt, a.err);
  return hipGetLastError();
}

}  // namespace sp
