// Dense contractions of the selection path on gfx950 matrix cores.
//
//   C[m, n] = sum_k A[m, k] * B[n, k]      (both operands K-contiguous)
//
// bfloat16 operands use v_mfma_f32_32x32x16_bf16, float32 operands
// v_mfma_f32_32x32x2_f32; accumulation is float32 and the result is stored
// once (bfloat16 rounded to nearest-even, or float32).  A workgroup of four
// waves owns a BM x BN tile; each wave owns a (BM/2) x (BN/2) quadrant made
// of 32 x 32 MFMA tiles.  K is walked in BK-wide stages through two LDS
// buffers: the next stage is fetched into registers while the current one
// feeds the matrix cores, then written to the other buffer, so one barrier
// per stage suffices.
//
// Three users:
//  * the projection of Algorithm 1 step 1: A = [X; s_start; s_stop], B = W_kqv;
//  * the text projection W_text E_text^T (float32 output for the LayerNorm);
//  * per-group Gram products of the projected rows used by the selection
//    recurrence (select.hip): rows [Q_g; q_start; V_g; v_start] against
//    columns [K_g; k_stop; k_start].
#include "sp_internal.h"

namespace sp {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

__device__ inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename OutT>
__device__ inline OutT store_cvt(float v);
template <>
__device__ inline float store_cvt<float>(float v) { return v; }
template <>
__device__ inline uint16_t store_cvt<uint16_t>(float v) { return f32_to_bf16_rne(v); }

template <typename T, int BM, int BN, int BK>
struct Tile {
  static constexpr int VEC = 16 / (int)sizeof(T);      // elements per 16-byte chunk
  static constexpr bool BF16 = sizeof(T) == 2;
  static constexpr int KM = BF16 ? 16 : 2;              // K of one MFMA
  static constexpr int LDK = BK + VEC;                  // padded LDS row, elements
  static constexpr int CPR = BK / VEC;                  // chunks per tile row
  static constexpr int CH_A = BM * CPR / kThreads;      // chunks per thread per stage
  static constexpr int CH_B = BN * CPR / kThreads;
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int LDS_BYTES = 2 * (BM + BN) * LDK * (int)sizeof(T);
  static_assert(BM * CPR % kThreads == 0 && BN * CPR % kThreads == 0, "tile/thread mismatch");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be a multiple of 32");
};

// One BM x BN output tile.  ARows/BRows map a row index to its K-contiguous
// storage; rows at or past M (N) read as zero and are not stored.
template <typename T, typename OutT, int BM, int BN, int BK, class ARows, class BRows>
__device__ __forceinline__ void gemm_block(const ARows& ar, const BRows& br, int64_t M, int64_t N,
                                           int K, OutT* __restrict__ C, int64_t ldc, int64_t m0,
                                           int64_t n0, char* smem) {
  using G = Tile<T, BM, BN, BK>;
  T* As = reinterpret_cast<T*>(smem);
  T* Bs = As + 2 * BM * G::LDK;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const T* pa[G::CH_A];
  const T* pb[G::CH_B];
  int la[G::CH_A], lb[G::CH_B];
#pragma unroll
  for (int i = 0; i < G::CH_A; ++i) {
    const int c = tid + i * kThreads;
    const int row = c / G::CPR, kc = c % G::CPR;
    const int64_t gm = m0 + row;
    pa[i] = gm < M ? ar.row(gm) + kc * G::VEC : nullptr;
    la[i] = row * G::LDK + kc * G::VEC;
  }
#pragma unroll
  for (int i = 0; i < G::CH_B; ++i) {
    const int c = tid + i * kThreads;
    const int row = c / G::CPR, kc = c % G::CPR;
    const int64_t gn = n0 + row;
    pb[i] = gn < N ? br.row(gn) + kc * G::VEC : nullptr;
    lb[i] = row * G::LDK + kc * G::VEC;
  }

  u32x4_t va[G::CH_A], vb[G::CH_B];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < G::CH_A; ++i)
      va[i] = pa[i] ? *reinterpret_cast<const u32x4_t*>(pa[i] + k0) : u32x4_t{0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < G::CH_B; ++i)
      vb[i] = pb[i] ? *reinterpret_cast<const u32x4_t*>(pb[i] + k0) : u32x4_t{0, 0, 0, 0};
  };
  auto lstore = [&](int buf) {
    T* a = As + buf * BM * G::LDK;
    T* b = Bs + buf * BN * G::LDK;
#pragma unroll
    for (int i = 0; i < G::CH_A; ++i) *reinterpret_cast<u32x4_t*>(a + la[i]) = va[i];
#pragma unroll
    for (int i = 0; i < G::CH_B; ++i) *reinterpret_cast<u32x4_t*>(b + lb[i]) = vb[i];
  };

  f32x16_t acc[G::TM][G::TN];
#pragma unroll
  for (int i = 0; i < G::TM; ++i)
#pragma unroll
    for (int j = 0; j < G::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int KT = K / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  const int arow = wm * G::WM + (lane & 31);
  const int brow = wn * G::WN + (lane & 31);
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) gload((kt + 1) * BK);
    const T* Ab = As + buf * BM * G::LDK;
    const T* Bb = Bs + buf * BN * G::LDK;
#pragma unroll
    for (int ks = 0; ks < BK; ks += G::KM) {
      if constexpr (G::BF16) {
        bf16x8_t a[G::TM], b[G::TN];
        const int koff = ks + (lane >> 5) * 8;
#pragma unroll
        for (int i = 0; i < G::TM; ++i)
          a[i] = *reinterpret_cast<const bf16x8_t*>(Ab + (arow + i * 32) * G::LDK + koff);
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
          b[j] = *reinterpret_cast<const bf16x8_t*>(Bb + (brow + j * 32) * G::LDK + koff);
#pragma unroll
        for (int i = 0; i < G::TM; ++i)
#pragma unroll
          for (int j = 0; j < G::TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      } else {
        float a[G::TM], b[G::TN];
        const int koff = ks + (lane >> 5);
#pragma unroll
        for (int i = 0; i < G::TM; ++i) a[i] = Ab[(arow + i * 32) * G::LDK + koff];
#pragma unroll
        for (int j = 0; j < G::TN; ++j) b[j] = Bb[(brow + j * 32) * G::LDK + koff];
#pragma unroll
        for (int i = 0; i < G::TM; ++i)
#pragma unroll
          for (int j = 0; j < G::TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
      }
    }
    if (kt + 1 < KT) lstore(buf ^ 1);
    __syncthreads();
  }

  // 32x32 MFMA result layout: lane l, register r holds
  // row 8*(r/4) + 4*(l/32) + r%4, column l%32.
#pragma unroll
  for (int i = 0; i < G::TM; ++i)
#pragma unroll
    for (int j = 0; j < G::TN; ++j) {
      const int64_t col = n0 + wn * G::WN + j * 32 + (lane & 31);
      if (col >= N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * G::WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < M) C[row * ldc + col] = store_cvt<OutT>(acc[i][j][r]);
      }
    }
}

// ------------------------------------------------------------------ row maps

template <typename T>
struct ProjRows {
  const T* X;
  int64_t T_vis;
  const T* s_start;
  const T* s_stop;
  int ld;
  __device__ const T* row(int64_t m) const {
    if (m < T_vis) return X + m * ld;
    return m == T_vis ? s_start : s_stop;
  }
};

template <typename T>
struct DenseRows {
  const T* base;
  int64_t ld;
  __device__ const T* row(int64_t m) const { return base + m * ld; }
};

// Gram operand rows of one group with tokens [g0, g0 + n): A side is
// [Q tokens; q_start; V tokens; v_start], B side is [K tokens; k_stop; k_start].
template <typename T>
struct GramARows {
  const T* KQV;
  int64_t g0, n, start_row;
  int h;
  __device__ const T* row(int64_t r) const {
    const int64_t ld = 3 * (int64_t)h;
    if (r < n) return KQV + (g0 + r) * ld + h;
    if (r == n) return KQV + start_row * ld + h;
    if (r < 2 * n + 1) return KQV + (g0 + r - n - 1) * ld + 2 * h;
    return KQV + start_row * ld + 2 * h;
  }
};

template <typename T>
struct GramBRows {
  const T* KQV;
  int64_t g0, n, start_row;
  int h;
  __device__ const T* row(int64_t c) const {
    const int64_t ld = 3 * (int64_t)h;
    if (c < n) return KQV + (g0 + c) * ld;
    if (c == n) return KQV + (start_row + 1) * ld;   // STOP key
    return KQV + start_row * ld;                      // START key
  }
};

// ------------------------------------------------------------------ kernels

template <typename T, typename OutT, int BM, int BN, int BK>
__global__ __launch_bounds__(kThreads) void project_gemm_kernel(ProjRows<T> ar, DenseRows<T> br,
                                                                int64_t M, int64_t N, int K,
                                                                OutT* C) {
  __shared__ __attribute__((aligned(16))) char smem[Tile<T, BM, BN, BK>::LDS_BYTES];
  const int64_t nt = (N + BN - 1) / BN;
  const int64_t t = blockIdx.x;
  gemm_block<T, OutT, BM, BN, BK>(ar, br, M, N, K, C, N, (t / nt) * BM, (t % nt) * BN, smem);
}

template <typename T, int BM, int BN, int BK>
__global__ __launch_bounds__(kThreads) void dense_gemm_kernel(DenseRows<T> ar, DenseRows<T> br,
                                                              int64_t M, int64_t N, int K,
                                                              float* C) {
  __shared__ __attribute__((aligned(16))) char smem[Tile<T, BM, BN, BK>::LDS_BYTES];
  const int64_t nt = (N + BN - 1) / BN;
  const int64_t t = blockIdx.x;
  gemm_block<T, float, BM, BN, BK>(ar, br, M, N, K, C, N, (t / nt) * BM, (t % nt) * BN, smem);
}

// grid.x: tiles of the largest group, grid.y: group.
template <typename T, int BM, int BN, int BK>
__global__ __launch_bounds__(kThreads) void gram_gemm_kernel(const T* KQV, int64_t T_vis, int h,
                                                             const int32_t* grp_off, int max_group,
                                                             float* gram, int64_t gstride, int ld,
                                                             int32_t* err) {
  __shared__ __attribute__((aligned(16))) char smem[Tile<T, BM, BN, BK>::LDS_BYTES];
  const int g = blockIdx.y;
  const int64_t g0 = grp_off[g], g1 = grp_off[g + 1];
  const int64_t n = g1 - g0;
  if (g0 < 0 || g1 > T_vis || n < 0 || n > max_group) {
    if (blockIdx.x == 0 && threadIdx.x == 0)
      set_device_error(err, n > max_group ? SP_DEV_GROUP_TOO_LARGE : SP_DEV_BAD_OFFSETS);
    return;
  }
  const int64_t M = 2 * (n + 1), N = n + 2;
  const int64_t nt = (N + BN - 1) / BN;
  const int64_t t = blockIdx.x;
  const int64_t m0 = (t / nt) * BM, n0 = (t % nt) * BN;
  if (m0 >= M) return;   // whole block idle for this (smaller) group
  GramARows<T> ar{KQV, g0, n, T_vis, h};
  GramBRows<T> br{KQV, g0, n, T_vis, h};
  gemm_block<T, float, BM, BN, BK>(ar, br, M, N, h, gram + g * gstride, ld, m0, n0, smem);
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

hipError_t launch_project_gemm(int dtype, const void* X, int64_t T_vis, const void* s_start,
                               const void* s_stop, const void* W, int d, int n_out, void* out,
                               hipStream_t stream) {
  const int64_t M = T_vis + 2, N = n_out;
  if (dtype == SP_BF16) {
    constexpr int BM = 256, BN = 256, BK = 64;
    using T = uint16_t;
    ProjRows<__bf16> ar{(const __bf16*)X, T_vis, (const __bf16*)s_start, (const __bf16*)s_stop, d};
    DenseRows<__bf16> br{(const __bf16*)W, d};
    (void)sizeof(T);
    hipLaunchKernelGGL((project_gemm_kernel<__bf16, uint16_t, BM, BN, BK>),
                       dim3((unsigned)(ceil_div(M, BM) * ceil_div(N, BN))), dim3(kThreads), 0, stream,
                       ar, br, M, N, d, (uint16_t*)out);
  } else {
    constexpr int BM = 128, BN = 128, BK = 32;
    ProjRows<float> ar{(const float*)X, T_vis, (const float*)s_start, (const float*)s_stop, d};
    DenseRows<float> br{(const float*)W, d};
    hipLaunchKernelGGL((project_gemm_kernel<float, float, BM, BN, BK>),
                       dim3((unsigned)(ceil_div(M, BM) * ceil_div(N, BN))), dim3(kThreads), 0, stream,
                       ar, br, M, N, d, (float*)out);
  }
  return hipGetLastError();
}

hipError_t launch_text_gemm(int dtype, const void* E, int64_t T_txt, const void* W, int d_text,
                            int h, float* out, hipStream_t stream) {
  if (T_txt == 0) return hipSuccess;
  if (dtype == SP_BF16) {
    constexpr int BM = 128, BN = 128, BK = 64;
    DenseRows<__bf16> ar{(const __bf16*)E, d_text};
    DenseRows<__bf16> br{(const __bf16*)W, d_text};
    hipLaunchKernelGGL((dense_gemm_kernel<__bf16, BM, BN, BK>),
                       dim3((unsigned)(ceil_div(T_txt, BM) * ceil_div(h, BN))), dim3(kThreads), 0,
                       stream, ar, br, T_txt, (int64_t)h, d_text, out);
  } else {
    constexpr int BM = 128, BN = 128, BK = 32;
    DenseRows<float> ar{(const float*)E, d_text};
    DenseRows<float> br{(const float*)W, d_text};
    hipLaunchKernelGGL((dense_gemm_kernel<float, BM, BN, BK>),
                       dim3((unsigned)(ceil_div(T_txt, BM) * ceil_div(h, BN))), dim3(kThreads), 0,
                       stream, ar, br, T_txt, (int64_t)h, d_text, out);
  }
  return hipGetLastError();
}

hipError_t launch_gram_gemm(int dtype, const void* KQV, int64_t T_vis, int h,
                            const int32_t* grp_off, int G, int max_group, float* gram,
                            int64_t gram_group_stride, int gram_ld, int32_t* err,
                            hipStream_t stream) {
  if (G == 0) return hipSuccess;
  const int64_t M = 2 * ((int64_t)max_group + 1), N = max_group + 2;
  if (dtype == SP_BF16) {
    constexpr int BM = 128, BN = 128, BK = 64;
    hipLaunchKernelGGL((gram_gemm_kernel<__bf16, BM, BN, BK>),
                       dim3((unsigned)(ceil_div(M, BM) * ceil_div(N, BN)), (unsigned)G),
                       dim3(kThreads), 0, stream, (const __bf16*)KQV, T_vis, h, grp_off, max_group,
                       gram, gram_group_stride, gram_ld, err);
  } else {
    constexpr int BM = 128, BN = 128, BK = 32;
    hipLaunchKernelGGL((gram_gemm_kernel<float, BM, BN, BK>),
                       dim3((unsigned)(ceil_div(M, BM) * ceil_div(N, BN)), (unsigned)G),
                       dim3(kThreads), 0, stream, (const float*)KQV, T_vis, h, grp_off, max_group,
                       gram, gram_group_stride, gram_ld, err);
  }
  return hipGetLastError();
}

}  // namespace sp
