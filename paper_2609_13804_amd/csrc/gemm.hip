// Dense contractions of the selection path on gfx950 matrix cores.
//
//   C[m, n] = sum_k A[m, k] * B[n, k]      (both operands K-contiguous)
//
// Accumulation is float32 and the result is stored once (bfloat16 rounded to
// nearest-even, or float32).  Two cores:
//  * bfloat16, gemm_bf16_256: 256 x 256 tiles of eight waves, each wave owning
//    128 x 64 as 32 x 32 tiles of v_mfma_f32_32x32x16_bf16; K in 32-wide
//    stages through a four-deep LDS ring filled straight from global memory.
//  * float32, gemm_block: BM x BN tiles of four waves, each owning a
//    (BM/2) x (BN/2) quadrant of 32 x 32 tiles of v_mfma_f32_32x32x2_f32; K in
//    BK-wide stages through two LDS buffers, the next stage fetched into
//    registers while the current one feeds the matrix cores.
//
// Three users:
//  * the projection of Algorithm 1 step 1: A = [X; s_start; s_stop], B = W_kqv;
//  * the text projection W_text E_text^T (float32 output for the LayerNorm);
//  * per-group Gram products of the projected rows used by the selection
//    recurrence (select.hip): rows [Q_g; q_start; V_g; v_start; context split]
//    against columns [K_g; k_stop; k_start].
#include <type_traits>

#include "sp_internal.h"
#include "lds_dma.h"

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

// Geometry of the float32 core's tiles.
template <typename T, int BM, int BN, int BK>
struct Tile {
  static_assert(sizeof(T) == 4, "the register-staged core is float32 only");
  static constexpr int VEC = 16 / (int)sizeof(T);      // elements per 16-byte chunk
  static constexpr int KM = 2;                          // K of one MFMA
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

// ------------------------------------------------------------------ bf16, 256 x 256 tiles
//
// Large bfloat16 GEMMs: a 256 x 256 output tile per workgroup of four or
// eight waves (MFMA 32x32x16 tiles, accumulators in AGPRs), K in 32-wide
// stages.  Operand tiles go straight from global memory into LDS
// (global_load_lds_dwordx4: one wave instruction fills 1 KiB = 16 rows x 64
// bytes) through a ring of S stage buffers, loads running S - 1 stages ahead
// of the matrix cores.  Each stage's loads are issued a few at a time between
// matrix-core instructions rather than in one burst.  Within a 64-byte row
// the four 16-byte chunks are stored XOR-swizzled (chunk c of row r at slot
// c ^ ((r >> 2) & 3)), which the load realises by choosing each lane's source
// address: a 16-byte fragment read serves 16 lanes (16 consecutive rows, 4 rows
// per 256-byte pass over the 64 banks) at a time, and rows 4 apart take
// different slots, so no two lanes of a pass share a bank.  Rows past M (N)
// are clamped to the last valid row and their results are not stored.
constexpr int kBM = 256, kBN = 256, kBK = 32, kStages = 4;
constexpr int kOpBytes = kBM * kBK * 2;                // one operand tile, 16 KiB
constexpr int kStageBytes = 2 * kOpBytes;              // A and B, 32 KiB

// Byte offset of (row, 16-byte chunk) in a swizzled operand tile (64-byte rows).
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * 64 + ((chunk ^ ((row >> 2) & 3)) << 4);
}

// WAVES = 4: each wave owns a 128 x 128 quadrant (one wave per SIMD).
// WAVES = 8: each wave owns 128 x 64 (two waves per SIMD, so one wave's
// matrix-core work covers the other's waits at barriers and loads).
// Output epilogue of the bfloat16 core: the product as it is, or (bfloat16
// output only) the product rounded to bfloat16, plus a per-column float32 bias,
// optionally through the exact GELU, rounded again: the same values as storing
// the product and then running a bias (+ GELU) pass over it.
constexpr int kEpiNone = 0, kEpiBias = 1, kEpiBiasGelu = 2;

template <int WAVES, typename OutT, class ARows, class BRows, int EPI = kEpiNone>
__device__ __forceinline__ void gemm_bf16_256(const ARows& ar, const BRows& br, int64_t M,
                                              int64_t N, int K, OutT* __restrict__ C, int64_t ldc,
                                              int64_t m0, int64_t n0, char* smem,
                                              const float* __restrict__ bias = nullptr) {
  static_assert(WAVES == 4 || WAVES == 8, "four or eight waves");
  static_assert(EPI == kEpiNone || sizeof(OutT) == 2, "bias epilogues write bfloat16");
  constexpr int GPW = 16 / WAVES;            // 16-row groups per operand per wave
  constexpr int LPW = 2 * GPW;               // DMA instructions per wave per stage
  constexpr int WGN = WAVES / 2;             // waves along N (two along M)
  constexpr int TN = 8 / WGN;                // 32-column MFMA tiles per wave along N
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;

  // This wave loads 16-row groups wave + WAVES i (i < GPW) of both operand
  // tiles; lane (rl = lane / 4, slot = lane % 4) fetches chunk
  // slot ^ ((rl >> 2) & 3) of row rl.
  const int rl = lane >> 2;
  const int chunk = (lane & 3) ^ ((rl >> 2) & 3);
  const __bf16* pa[GPW];
  const __bf16* pb[GPW];
#pragma unroll
  for (int i = 0; i < GPW; ++i) {
    const int r = 16 * (wave + WAVES * i) + rl;
    const int64_t gm = m0 + r < M ? m0 + r : M - 1;
    const int64_t gn = n0 + r < N ? n0 + r : N - 1;
    pa[i] = ar.row(gm) + chunk * 8;
    pb[i] = br.row(gn) + chunk * 8;
  }
  auto issue = [&](int buf, int k0) {
    char* a = smem + buf * kStageBytes;
    char* b = a + kOpBytes;
#pragma unroll
    for (int i = 0; i < GPW; ++i) lds_dma16(pa[i] + k0, a + (wave + WAVES * i) * 1024);
#pragma unroll
    for (int i = 0; i < GPW; ++i) lds_dma16(pb[i] + k0, b + (wave + WAVES * i) * 1024);
  };

  f32x16_t acc[4][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int arow0 = wm * 128 + (lane & 31);
  const int brow0 = wn * (32 * TN) + (lane & 31);
  const int khalf = lane >> 5;
  auto load_frags = [&](const char* As, const char* Bs, int ks, bf16x8_t (&a)[4], bf16x8_t (&b)[TN]) {
    const int c = ks * 2 + khalf;
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const bf16x8_t*>(As + swz(arow0 + 32 * i, c));
#pragma unroll
    for (int j = 0; j < TN; ++j) b[j] = *reinterpret_cast<const bf16x8_t*>(Bs + swz(brow0 + 32 * j, c));
  };

  // Software pipeline over K stages.  Iteration kt multiplies stage kt in two
  // halves (16 k each); between them it waits for stage kt + 1, passes the
  // workgroup barrier, refills the ring with stage kt + S - 1 and starts
  // reading stage kt + 1's fragments, so the barrier and the LDS latency hide
  // behind matrix-core work.
  const int KT = K / kBK;
#pragma unroll
  for (int s = 0; s < kStages - 1; ++s)
    if (s < KT) issue(s, s * kBK);
  if (KT > kStages - 2) wait_vmcnt<(kStages - 2) * LPW>();
  else wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  // Two fragment sets used in turn (the loop is unrolled by two), so the
  // next stage's fragments land in registers no copy has to wait for.
  struct Frags {
    bf16x8_t a0[4], b0[TN], a1[4], b1[TN];
  };
  Frags f0, f1;
  load_frags(smem, smem + kOpBytes, 0, f0.a0, f0.b0);
  load_frags(smem, smem + kOpBytes, 1, f0.a1, f0.b1);
  // DMA instruction q of a stage: the first GPW fill A's row groups, the rest B's.
  auto issue_one = [&](int buf, int k0, int q) {
    char* a = smem + buf * kStageBytes;
    if (q < GPW) lds_dma16(pa[q] + k0, a + (wave + WAVES * q) * 1024);
    else lds_dma16(pb[q - GPW] + k0, a + kOpBytes + (wave + WAVES * (q - GPW)) * 1024);
  };
  // MORE / REFILL: 1 means always, -1 decided at run time.  The steady-state
  // loop instantiates both as 1, so its body has no branches: at a join of
  // branches the compiler's wait counting falls back to waiting for every
  // outstanding LDS read, and each half-step would then stall on the
  // fragment reads it has just issued.
  auto step = [&](int kt, Frags& cur, Frags& nxt, auto more_c, auto refill_c) {
    constexpr int MORE = decltype(more_c)::value, REFILL = decltype(refill_c)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.a0[i], cur.b0[j], acc[i][j], 0, 0, 0);
    const bool more = MORE == 1 || kt + 1 < KT;
    const bool refill = REFILL == 1 || kt + kStages - 1 < KT;
    if (more) {
      // Stage kt + 1 has landed once at most (stages issued after it) x loads
      // of this wave remain.  The buffer refilled below held stage kt - 1,
      // whose fragments every wave consumed before this barrier.
      if (refill) wait_vmcnt<(kStages - 3) * LPW>();
      else wait_vmcnt<0>();
      // Bare s_barrier (no fence): a workgroup fence would wait for every load
      // still in flight and collapse the ring to a single stage.
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      const char* As = smem + ((kt + 1) % kStages) * kStageBytes;
      load_frags(As, As + kOpBytes, 0, nxt.a0, nxt.b0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // The refill of stage kt + S - 1 is spread over this half's matrix-core
    // work: issued in one burst, the loads would stall this wave's issue until
    // the memory pipeline drained them, and the matrix cores with it.
    const int rbuf = (kt + kStages - 1) % kStages, rk0 = (kt + kStages - 1) * kBK;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.a1[i], cur.b1[j], acc[i][j], 0, 0, 0);
      if (refill) {
#pragma unroll
        for (int u = 0; u < LPW / 4; ++u) issue_one(rbuf, rk0, i * (LPW / 4) + u);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (more) {
      const char* As = smem + ((kt + 1) % kStages) * kStageBytes;
      load_frags(As, As + kOpBytes, 1, nxt.a1, nxt.b1);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  using Always = std::integral_constant<int, 1>;
  using Checked = std::integral_constant<int, -1>;
  int kt = 0;
  // Steady state: both steps of a pair have a next stage and a refill.
  for (; kt + kStages < KT; kt += 2) {
    step(kt, f0, f1, Always{}, Always{});
    step(kt + 1, f1, f0, Always{}, Always{});
  }
  for (; kt + 1 < KT; kt += 2) {
    step(kt, f0, f1, Checked{}, Checked{});
    step(kt + 1, f1, f0, Checked{}, Checked{});
  }
  if (kt < KT) step(kt, f0, f1, Checked{}, Checked{});

  // Epilogue through LDS: once every wave is past the K loop the operand ring
  // is free, so the tile is staged there in row-major order and leaves as
  // 16-byte row chunks (whole cache lines, an eighth or a quarter of the store
  // instructions of storing the MFMA layout directly).  A float32 tile needs
  // twice the ring, so it is staged in two passes of 128 rows (the waves with
  // wm = 0, then wm = 1).  Chunks of rows with bit 2 set are XOR-ed by half a
  // row of banks: the two rows one write instruction covers (r and r + 4)
  // then hit different banks.
  constexpr int E = (int)sizeof(OutT);
  constexpr int EPC = 16 / E;                              // elements per 16-byte chunk
  constexpr int CPR = kBN / EPC;                           // chunks per staged row
  constexpr int ROWS = kStages * kStageBytes / (kBN * E);  // rows staged per pass
  constexpr int PASSES = kBM / ROWS;
  constexpr int XS = CPR / 8;
  constexpr int THREADS = 64 * WAVES;
  static_assert(ROWS == 128 || ROWS == 256, "one or two staging passes");
  static_assert(ROWS * CPR % THREADS == 0, "whole chunks per thread");
  auto sw = [](int lr) { return ((lr >> 2) & 1) * XS; };
  const bool vec = ((uintptr_t)C % 16 == 0) && ((int64_t)ldc * E % 16 == 0);
  OutT* T = reinterpret_cast<OutT*>(smem);
  __syncthreads();
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    if (PASSES == 1 || wm == p) {
      // 32x32 MFMA result layout: lane l, register r holds
      // row 8*(r/4) + 4*(l/32) + r%4, column l%32.
      float bj[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int64_t col = n0 + wn * (32 * TN) + j * 32 + (lane & 31);
        bj[j] = EPI != kEpiNone && col < N ? bias[col] : 0.0f;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int lr = wm * 128 - p * ROWS + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            const int lc = wn * (32 * TN) + j * 32 + (lane & 31);
            OutT v;
            if constexpr (EPI == kEpiNone) {
              v = store_cvt<OutT>(acc[i][j][r]);
            } else {
              float y = __uint_as_float((uint32_t)f32_to_bf16_rne(acc[i][j][r]) << 16) + bj[j];
              if constexpr (EPI == kEpiBiasGelu) y = 0.5f * y * (1.0f + erff(y * 0.70710678118654752f));
              v = f32_to_bf16_rne(y);
            }
            T[lr * kBN + ((lc / EPC) ^ sw(lr)) * EPC + lc % EPC] = v;
          }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < ROWS * CPR / THREADS; ++q) {
      const int c = tid + THREADS * q, lr = c / CPR, ch = c % CPR;
      const int64_t row = m0 + p * ROWS + lr, col = n0 + (int64_t)ch * EPC;
      if (row >= M || col >= N) continue;
      const OutT* src = T + lr * kBN + (ch ^ sw(lr)) * EPC;
      OutT* dst = C + row * ldc + col;
      if (vec && col + EPC <= N) {
        *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
      } else {
        for (int e = 0; e < EPC && col + e < N; ++e) dst[e] = src[e];
      }
    }
    if (p + 1 < PASSES) __syncthreads();
  }
}

// Workgroup w runs on XCD w % 8, which takes a contiguous run of the tiles in
// banded order: bands of kBand row panels, each band walked column by column
// (the last band as tall as the rows left).  The 32 tiles one XCD runs at a
// time then cover about kBand row panels and 32 / kBand column panels, so they
// share about 12 operand panels in that XCD's L2 (a row-major run of 32 tiles
// spans all the column panels of a wide product).  Returns -1 for the padding
// workgroups of the last run.
constexpr int64_t kBand = 4;

__device__ __forceinline__ int64_t xcd_tile(int64_t w, int64_t mt, int64_t nt) {
  const int64_t tiles = mt * nt;
  const int64_t per = (tiles + 7) / 8;
  const int64_t i = (w % 8) * per + w / 8;
  if (i >= tiles) return -1;
  const int64_t band = i / (kBand * nt), o = i % (kBand * nt);
  const int64_t rows = mt - band * kBand < kBand ? mt - band * kBand : kBand;
  return (band * kBand + o % rows) * nt + o / rows;
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
// [Q tokens; q_start; V tokens; v_start; c_hi; c_mid; c_lo] (the last three
// from the image's context split), B side is [K tokens; k_stop; k_start].
template <typename T>
struct GramARows {
  const T* KQV;
  int64_t g0, n, start_row;
  int h;
  const T* csplit;     // the image's three context rows
  __device__ const T* row(int64_t r) const {
    const int64_t ld = 3 * (int64_t)h;
    if (r < n) return KQV + (g0 + r) * ld + h;
    if (r == n) return KQV + start_row * ld + h;
    if (r < 2 * n + 1) return KQV + (g0 + r - n - 1) * ld + 2 * h;
    if (r == 2 * n + 1) return KQV + start_row * ld + 2 * h;
    return csplit + (r - 2 * n - 2) * h;
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

constexpr int kProjWaves = 8;

// Blocks [0, proj_blocks) take the projection's tiles in XCD-grouped order
// (bfloat16 output); the blocks after them take the text projection's tiles
// (float32 output).  The text tiles are dispatched last, onto the compute
// units the projection's last round leaves idle.
__global__ __launch_bounds__(64 * kProjWaves) void project_gemm_bf16_kernel(
    ProjRows<__bf16> ar, DenseRows<__bf16> br, int64_t M, int64_t N, int K, uint16_t* C,
    int64_t proj_blocks, DenseRows<__bf16> er, DenseRows<__bf16> wr, int64_t M2, int64_t N2, int K2,
    float* C2) {
  __shared__ __attribute__((aligned(1024))) char smem[kStages * kStageBytes];
  if ((int64_t)blockIdx.x < proj_blocks) {
    const int64_t nt = (N + kBN - 1) / kBN;
    const int64_t t = xcd_tile(blockIdx.x, (M + kBM - 1) / kBM, nt);
    if (t < 0) return;
    gemm_bf16_256<kProjWaves, uint16_t>(ar, br, M, N, K, C, N, (t / nt) * kBM, (t % nt) * kBN, smem);
  } else {
    const int64_t nt = (N2 + kBN - 1) / kBN;
    const int64_t t = (int64_t)blockIdx.x - proj_blocks;
    gemm_bf16_256<kProjWaves, float>(er, wr, M2, N2, K2, C2, N2, (t / nt) * kBM, (t % nt) * kBN,
                                     smem);
  }
}

// A bfloat16 product C = A B^T (bfloat16 out) on the 256 x 256 core, tiles in
// XCD-grouped order, with an optional bias (+ GELU) epilogue.
template <int EPI>
__global__ __launch_bounds__(64 * kProjWaves) void dense_bf16_kernel(DenseRows<__bf16> ar,
                                                                    DenseRows<__bf16> br,
                                                                    int64_t M, int64_t N, int K,
                                                                    uint16_t* C, const float* bias) {
  __shared__ __attribute__((aligned(1024))) char smem[kStages * kStageBytes];
  const int64_t nt = (N + kBN - 1) / kBN;
  const int64_t t = xcd_tile(blockIdx.x, (M + kBM - 1) / kBM, nt);
  if (t < 0) return;
  gemm_bf16_256<kProjWaves, uint16_t, DenseRows<__bf16>, DenseRows<__bf16>, EPI>(
      ar, br, M, N, K, C, N, (t / nt) * kBM, (t % nt) * kBN, smem, bias);
}

// grid.x: output tiles, grid.y: K split p, which covers k in [p K, (p + 1) K)
// and writes partial product p at C + p M N.
template <typename T, int BM, int BN, int BK>
__global__ __launch_bounds__(kThreads) void dense_gemm_kernel(DenseRows<T> ar, DenseRows<T> br,
                                                              int64_t M, int64_t N, int K,
                                                              float* C) {
  __shared__ __attribute__((aligned(16))) char smem[Tile<T, BM, BN, BK>::LDS_BYTES];
  const int64_t nt = (N + BN - 1) / BN;
  const int64_t t = blockIdx.x;
  const int64_t k0 = (int64_t)blockIdx.y * K;
  DenseRows<T> a{ar.base + k0, ar.ld}, b{br.base + k0, br.ld};
  gemm_block<T, float, BM, BN, BK>(a, b, M, N, K, C + blockIdx.y * M * N, N, (t / nt) * BM,
                                   (t % nt) * BN, smem);
}

// The context of image b as three rows of the working dtype whose sum is the
// float32 value exactly (bfloat16: successive round-to-nearest-even residuals,
// 3 x 8 significant bits; float32: the value and two zero rows).
template <typename T>
__global__ __launch_bounds__(256) void ctx_split_kernel(const float* __restrict__ ctx, int h,
                                                        T* __restrict__ csplit) {
  const int b = blockIdx.x;
  for (int i = threadIdx.x; i < h; i += blockDim.x) {
    const float c = ctx[(int64_t)b * h + i];
    T* out = csplit + (int64_t)b * kGramExtraRows * h + i;
    if constexpr (sizeof(T) == 2) {
      const uint16_t hi = f32_to_bf16_rne(c);
      const float r1 = c - __uint_as_float((uint32_t)hi << 16);
      const uint16_t mid = f32_to_bf16_rne(r1);
      const float r2 = r1 - __uint_as_float((uint32_t)mid << 16);
      const uint16_t lo = f32_to_bf16_rne(r2);
      reinterpret_cast<uint16_t*>(out)[0] = hi;
      reinterpret_cast<uint16_t*>(out)[h] = mid;
      reinterpret_cast<uint16_t*>(out)[2 * h] = lo;
    } else {
      out[0] = c;
      out[h] = 0.0f;
      out[2 * h] = 0.0f;
    }
  }
}

// Workgroup w runs on XCD w % 8.  With at least eight groups, all tiles of a
// group are placed on one XCD (group x + 8 k on XCD x) so that the group's
// rows are fetched into one L2.
__device__ __forceinline__ bool gram_tile(int64_t w, int per_group, int G, int xcd_grouped,
                                          int64_t& g, int64_t& t) {
  if (xcd_grouped) {
    const int64_t i = w / 8;
    g = w % 8 + 8 * (i / per_group);
    t = i % per_group;
  } else {
    g = w / per_group;
    t = w % per_group;
  }
  return g < G;
}

// Validates group g; on inconsistent offsets one workgroup records the error.
__device__ __forceinline__ bool gram_group_ok(const GramArgs& a, int64_t g, int64_t t, int64_t& g0,
                                              int64_t& n, int& b) {
  g0 = a.grp_off[g];
  const int64_t g1 = a.grp_off[g + 1];
  n = g1 - g0;
  b = a.grp_img[g];
  if (g0 < 0 || g1 > a.T_vis || n < 0 || n > a.max_group || b < 0 || b >= a.B) {
    if (t == 0 && threadIdx.x == 0)
      set_device_error(a.err, n > a.max_group ? SP_DEV_GROUP_TOO_LARGE : SP_DEV_BAD_OFFSETS);
    return false;
  }
  return true;
}

// The Gram entries that involve START, STOP or the context split, for the
// `edge` layout: item j of a group (a token, or j = n for the corner, where
// q_start, v_start and k_stop stand in for q_j, v_j and k_j) gives
//   A[j][n] = q_j . k_stop    A[j][n + 1] = q_j . k_start    B[j][n] = v_j . k_stop
//   A[n][j] = q_start . k_j   B[n][j] = v_start . k_j        CK[s][j] = c_s . k_j
// as float32 sums of exact bfloat16 products, one wave per item.
// The eight sums are reduced together: each shuffle step halves the values
// a lane carries, and lane 8 k ends with value k.
constexpr int kEdgeItems = 8;   // items per wave, four waves per workgroup

// Grid (G, ceil((max_group + 1) / 32)): workgroup (g, y) of four waves takes
// items [32 y, 32 y + 32) of group g.
__global__ __launch_bounds__(256) void gram_edge_kernel(GramArgs a) {
  const int64_t g = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t g0 = a.grp_off[g], g1 = a.grp_off[g + 1];
  const int64_t n = g1 - g0;
  const int b = a.grp_img[g];
  if (g0 < 0 || g1 > a.T_vis || n < 0 || n > a.max_group || b < 0 || b >= a.B) return;
  const int h = a.h;
  const int64_t ld3 = 3 * (int64_t)h, ld = a.gram_ld;
  const __bf16* KQV = static_cast<const __bf16*>(a.KQV);
  const __bf16* kst = KQV + a.T_vis * ld3;              // START: k, q, v
  const __bf16* kstop = KQV + (a.T_vis + 1) * ld3;      // STOP key
  const __bf16* cs = static_cast<const __bf16*>(a.csplit) + (int64_t)b * kGramExtraRows * h;
  float* A = a.gram + g * a.gram_group_stride;
  float* Bm = A + (n + 1) * ld;
  float* CK = A + (2 * n + 2) * ld;
  // this lane's eight-element slices (at most two: h <= 1024) of the shared vectors
  typedef uint32_t u4 __attribute__((ext_vector_type(4)));
  auto ld16 = [&](const __bf16* p, int c) -> u4 {
    const int e = 8 * lane + 512 * c;
    return e < h ? *reinterpret_cast<const u4*>(p + e) : u4{0, 0, 0, 0};
  };
  // the two bfloat16 values of word i, widened exactly to float32
  auto lo = [](u4 x, int i) { return __uint_as_float(x[i] << 16); };
  auto hi = [](u4 x, int i) { return __uint_as_float(x[i] & 0xffff0000u); };
  // this lane's eight-element slices of the shared vectors (packed)
  u4 sv[7][2];
  const __bf16* shared_rows[7] = {kstop, kst, kst + h, kst + 2 * h, cs, cs + h, cs + 2 * h};
#pragma unroll
  for (int v = 0; v < 7; ++v)
#pragma unroll
    for (int c = 0; c < 2; ++c) sv[v][c] = ld16(shared_rows[v], c);
  // item i's rows: its token's [k | q | v], or k_stop, q_start, v_start (j = n)
  auto load_item = [&](int64_t j, u4 (&q)[2], u4 (&v)[2], u4 (&k)[2]) {
    const __bf16* krow = j < n ? KQV + (g0 + j) * ld3 : kstop;
    const __bf16* qrow = j < n ? krow + h : kst + h;
    const __bf16* vrow = j < n ? krow + 2 * h : kst + 2 * h;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      q[c] = ld16(qrow, c);
      v[c] = ld16(vrow, c);
      k[c] = ld16(krow, c);
    }
  };
  const int64_t j0 = (int64_t)blockIdx.y * 4 * kEdgeItems + wave;
  u4 qn[2], vn[2], kn[2];     // the next item's rows, requested one item ahead
  if (j0 <= n) load_item(j0, qn, vn, kn);
  for (int i = 0; i < kEdgeItems; ++i) {
    const int64_t j = j0 + 4 * i;
    if (j > n) break;
    u4 q[2], v[2], k[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      q[c] = qn[c];
      v[c] = vn[c];
      k[c] = kn[c];
    }
    if (i + 1 < kEdgeItems && j + 4 <= n) load_item(j + 4, qn, vn, kn);
    float d[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          auto f = [&](u4 x) { return half ? hi(x, p) : lo(x, p); };
          const float qv = f(q[c]), vv = f(v[c]), kv = f(k[c]);
          d[0] = fmaf(qv, f(sv[0][c]), d[0]);
          d[1] = fmaf(qv, f(sv[1][c]), d[1]);
          d[2] = fmaf(vv, f(sv[0][c]), d[2]);
          d[3] = fmaf(f(sv[2][c]), kv, d[3]);
          d[4] = fmaf(f(sv[3][c]), kv, d[4]);
          d[5] = fmaf(f(sv[4][c]), kv, d[5]);
          d[6] = fmaf(f(sv[5][c]), kv, d[6]);
          d[7] = fmaf(f(sv[6][c]), kv, d[7]);
        }
    // 8 values -> 4 (xor 32) -> 2 (xor 16) -> 1 (xor 8), then xor 4, 2, 1
    const bool h32 = lane & 32, h16 = lane & 16, h8 = lane & 8;
    float r4[4], r2[2];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      r4[k] = (h32 ? d[k + 4] : d[k]) + __shfl_xor(h32 ? d[k] : d[k + 4], 32, 64);
#pragma unroll
    for (int k = 0; k < 2; ++k)
      r2[k] = (h16 ? r4[k + 2] : r4[k]) + __shfl_xor(h16 ? r4[k] : r4[k + 2], 16, 64);
    float r = (h8 ? r2[1] : r2[0]) + __shfl_xor(h8 ? r2[0] : r2[1], 8, 64);
    r += __shfl_xor(r, 4, 64);
    r += __shfl_xor(r, 2, 64);
    r += __shfl_xor(r, 1, 64);
    if ((lane & 7) == 0) {
      const int k = (h32 ? 4 : 0) + (h16 ? 2 : 0) + (h8 ? 1 : 0);
      float* dst = k == 0 ? A + j * ld + n
                 : k == 1 ? A + j * ld + n + 1
                 : k == 2 ? Bm + j * ld + n
                 : k == 3 ? A + n * ld + j
                 : k == 4 ? Bm + n * ld + j
                          : CK + (k - 5) * ld + j;
      *dst = r;
    }
  }
}

// bfloat16 Gram products on the 256 x 256 direct-to-LDS core: 15 tiles per
// 576-token group, one round for 16 groups.  With `edge` the tiles cover the
// token blocks only, [Q] x [K] into A's rows 0..n-1 and [V] x [K] into B's
// rows 0..n-1 (tq x tq tiles each), and gram_edge_kernel computes the rows
// and columns of START, STOP and the context split.
constexpr int kGramWaves = 8;

__global__ __launch_bounds__(64 * kGramWaves) void gram_gemm_bf16_kernel(GramArgs a, int per_group,
                                                                 int xcd_grouped, int edge) {
  __shared__ __attribute__((aligned(1024))) char smem[kStages * kStageBytes];
  int64_t g, t, g0, n;
  int b;
  if (!gram_tile(blockIdx.x, per_group, a.G, xcd_grouped, g, t)) return;
  if (!gram_group_ok(a, g, t, g0, n, b)) return;
  const __bf16* KQV = static_cast<const __bf16*>(a.KQV);
  if (edge) {
    const int64_t tq = (a.max_group + kBN - 1) / kBN;
    const int64_t sub = t / (tq * tq), tt = t % (tq * tq);
    const int64_t m0 = (tt / tq) * kBM, n0 = (tt % tq) * kBN;
    if (m0 >= n || n0 >= n) return;   // tile outside this (smaller) group
    const int64_t ld3 = 3 * (int64_t)a.h;
    DenseRows<__bf16> ar{KQV + g0 * ld3 + (sub == 0 ? a.h : 2 * a.h), ld3};   // Q or V rows
    DenseRows<__bf16> br{KQV + g0 * ld3, ld3};                               // K rows
    float* C = a.gram + g * a.gram_group_stride + (sub == 0 ? 0 : (n + 1) * a.gram_ld);
    gemm_bf16_256<kGramWaves, float>(ar, br, n, n, a.h, C, a.gram_ld, m0, n0, smem);
    return;
  }
  const __bf16* cs = static_cast<const __bf16*>(a.csplit) + (int64_t)b * kGramExtraRows * a.h;
  const int64_t M = 2 * (n + 1) + kGramExtraRows, N = n + 2;
  const int64_t nt = (a.max_group + 2 + kBN - 1) / kBN;
  const int64_t m0 = (t / nt) * kBM, n0 = (t % nt) * kBN;
  if (m0 >= M || n0 >= N) return;   // tile outside this (smaller) group
  GramARows<__bf16> ar{KQV, g0, n, a.T_vis, a.h, cs};
  GramBRows<__bf16> br{KQV, g0, n, a.T_vis, a.h};
  gemm_bf16_256<kGramWaves, float>(ar, br, M, N, a.h, a.gram + g * a.gram_group_stride, a.gram_ld, m0, n0,
                       smem);
}

// float32 Gram products on the register-staged core, BM x BN tiles.
template <int BM, int BN>
__global__ __launch_bounds__(kThreads) void gram_gemm_f32_kernel(GramArgs a, int per_group,
                                                                int xcd_grouped) {
  constexpr int BK = 32;
  __shared__ __attribute__((aligned(16))) char smem[Tile<float, BM, BN, BK>::LDS_BYTES];
  int64_t g, t, g0, n;
  int b;
  if (!gram_tile(blockIdx.x, per_group, a.G, xcd_grouped, g, t)) return;
  if (!gram_group_ok(a, g, t, g0, n, b)) return;
  const float* KQV = static_cast<const float*>(a.KQV);
  const float* cs = static_cast<const float*>(a.csplit) + (int64_t)b * kGramExtraRows * a.h;
  const int64_t M = 2 * (n + 1) + kGramExtraRows, N = n + 2;
  const int64_t nt = (a.max_group + 2 + BN - 1) / BN;
  const int64_t m0 = (t / nt) * BM, n0 = (t % nt) * BN;
  if (m0 >= M || n0 >= N) return;
  GramARows<float> ar{KQV, g0, n, a.T_vis, a.h, cs};
  GramBRows<float> br{KQV, g0, n, a.T_vis, a.h};
  gemm_block<float, float, BM, BN, BK>(ar, br, M, N, a.h, a.gram + g * a.gram_group_stride,
                                       a.gram_ld, m0, n0, smem);
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// The float32 paths serve small batches (one image of a few hundred tokens):
// 128 x 128 tiles would leave most compute units idle, so 64 x 64 tiles are
// taken while the 128 x 128 ones would not fill the chip once.  Each output
// accumulates its K in the same order either way.
inline bool small_f32_tiles(int64_t M, int64_t N) { return ceil_div(M, 128) * ceil_div(N, 128) < 256; }

}  // namespace

int text_split(int dtype, int64_t T_txt, int h, int d_text) {
  if (dtype == SP_BF16) return 1;   // computed beside the projection, whole K
  // Enough workgroups to cover the chip: split K while the tiles are fewer
  // than 512, up to 8 ways, keeping each part a whole number of 64-wide stages.
  const int64_t tiles = ceil_div(T_txt, 128) * ceil_div(h, 128);
  int s = 1;
  while (s < 8 && tiles * s < 512 && d_text % (2 * s * 64) == 0) s *= 2;
  return s;
}

namespace {

hipError_t launch_text_gemm_f32(const void* E, int64_t T_txt, const void* W, int d_text, int h,
                                float* out, hipStream_t stream) {
  if (T_txt == 0) return hipSuccess;
  const int split = text_split(SP_F32, T_txt, h, d_text);
  const int kpart = d_text / split;
  const dim3 grid((unsigned)(ceil_div(T_txt, 128) * ceil_div(h, 128)), (unsigned)split);
  DenseRows<float> ar{(const float*)E, d_text};
  DenseRows<float> br{(const float*)W, d_text};
  hipLaunchKernelGGL((dense_gemm_kernel<float, 128, 128, 32>), grid, dim3(kThreads), 0, stream,
                     ar, br, T_txt, (int64_t)h, kpart, out);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_project_gemm(int dtype, const void* X, int64_t T_vis, const void* s_start,
                               const void* s_stop, const void* W, int d, int n_out, void* out,
                               const void* E, int64_t T_txt, const void* W_text, int d_text, int h,
                               float* tproj, hipStream_t stream) {
  const int64_t M = T_vis + 2, N = n_out;
  if (dtype == SP_BF16) {
    ProjRows<__bf16> ar{(const __bf16*)X, T_vis, (const __bf16*)s_start, (const __bf16*)s_stop, d};
    DenseRows<__bf16> br{(const __bf16*)W, d};
    DenseRows<__bf16> er{(const __bf16*)E, d_text};
    DenseRows<__bf16> wr{(const __bf16*)W_text, d_text};
    const int64_t proj_blocks = ceil_div(ceil_div(M, kBM) * ceil_div(N, kBN), 8) * 8;
    const int64_t text_blocks = T_txt > 0 ? ceil_div(T_txt, kBM) * ceil_div(h, kBN) : 0;
    hipLaunchKernelGGL(project_gemm_bf16_kernel, dim3((unsigned)(proj_blocks + text_blocks)),
                       dim3(64 * kProjWaves), 0, stream, ar, br, M, N, d, (uint16_t*)out,
                       proj_blocks, er, wr, T_txt, (int64_t)h, d_text, tproj);
    return hipGetLastError();
  }
  ProjRows<float> ar{(const float*)X, T_vis, (const float*)s_start, (const float*)s_stop, d};
  DenseRows<float> br{(const float*)W, d};
  if (small_f32_tiles(M, N))
    hipLaunchKernelGGL((project_gemm_kernel<float, float, 64, 64, 32>),
                       dim3((unsigned)(ceil_div(M, 64) * ceil_div(N, 64))), dim3(kThreads), 0, stream,
                       ar, br, M, N, d, (float*)out);
  else
    hipLaunchKernelGGL((project_gemm_kernel<float, float, 128, 128, 32>),
                       dim3((unsigned)(ceil_div(M, 128) * ceil_div(N, 128))), dim3(kThreads), 0,
                       stream, ar, br, M, N, d, (float*)out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_text_gemm_f32(E, T_txt, W_text, d_text, h, tproj, stream);
}

hipError_t launch_gram_gemm(const GramArgs& a, hipStream_t stream) {
  if (a.G == 0) return hipSuccess;
  const int64_t M = 2 * ((int64_t)a.max_group + 1) + kGramExtraRows, N = a.max_group + 2;
  const int xcd_grouped = a.G >= 8;
  if (a.dtype == SP_BF16) {
    hipLaunchKernelGGL(ctx_split_kernel<__bf16>, dim3(a.B), dim3(256), 0, stream, a.ctx, a.h,
                       (__bf16*)a.csplit);
    // The token blocks alone take fewer tiles when the group size sits just
    // below a multiple of 256 (256-token groups: 2 tiles instead of 6); then
    // the START / STOP / context entries come from gram_edge_kernel.  (It
    // re-reads the group's rows: at 256-token groups it takes about 300 us
    // on the 64 x 3328 batch against 450 us for the two tiles a group.)
    const int64_t tq = ceil_div((int64_t)a.max_group, kBN);
    const int64_t full = ceil_div(M, kBM) * ceil_div(N, kBN);
    const int edge = a.max_group > 0 && 2 * tq * tq < full;
    const int per_group = (int)(edge ? 2 * tq * tq : full);
    const int64_t blocks =
        xcd_grouped ? 8 * ceil_div(a.G, 8) * per_group : (int64_t)a.G * per_group;
    hipLaunchKernelGGL(gram_gemm_bf16_kernel, dim3((unsigned)blocks), dim3(64 * kGramWaves), 0, stream, a,
                       per_group, xcd_grouped, edge);
    if (edge)
      hipLaunchKernelGGL(gram_edge_kernel,
                         dim3((unsigned)a.G, (unsigned)ceil_div((int64_t)a.max_group + 1, 4 * kEdgeItems)),
                         dim3(256), 0, stream, a);
  } else {
    hipLaunchKernelGGL(ctx_split_kernel<float>, dim3(a.B), dim3(256), 0, stream, a.ctx, a.h,
                       (float*)a.csplit);
    const bool small = small_f32_tiles(M * a.G, N);
    const int T = small ? 64 : 128;
    const int per_group = (int)(ceil_div(M, T) * ceil_div(N, T));
    const int64_t blocks =
        xcd_grouped ? 8 * ceil_div(a.G, 8) * per_group : (int64_t)a.G * per_group;
    if (small)
      hipLaunchKernelGGL((gram_gemm_f32_kernel<64, 64>), dim3((unsigned)blocks), dim3(kThreads), 0,
                         stream, a, per_group, xcd_grouped);
    else
      hipLaunchKernelGGL((gram_gemm_f32_kernel<128, 128>), dim3((unsigned)blocks), dim3(kThreads), 0,
                         stream, a, per_group, xcd_grouped);
  }
  return hipGetLastError();
}

hipError_t launch_dense_bf16(const void* A, const void* B, int64_t M, int64_t N, int K, void* C,
                             hipStream_t stream, const float* bias, bool gelu) {
  if (M == 0 || N == 0) return hipSuccess;
  DenseRows<__bf16> ar{(const __bf16*)A, K};
  DenseRows<__bf16> br{(const __bf16*)B, K};
  const dim3 grid((unsigned)(ceil_div(ceil_div(M, kBM) * ceil_div(N, kBN), 8) * 8));
  const dim3 block(64 * kProjWaves);
  uint16_t* out = (uint16_t*)C;
  if (!bias)
    hipLaunchKernelGGL(dense_bf16_kernel<kEpiNone>, grid, block, 0, stream, ar, br, M, N, K, out, bias);
  else if (!gelu)
    hipLaunchKernelGGL(dense_bf16_kernel<kEpiBias>, grid, block, 0, stream, ar, br, M, N, K, out, bias);
  else
    hipLaunchKernelGGL(dense_bf16_kernel<kEpiBiasGelu>, grid, block, 0, stream, ar, br, M, N, K, out,
                       bias);
  return hipGetLastError();
}

}  // namespace sp
