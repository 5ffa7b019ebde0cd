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
// step needs only the row A[e, :] and the column values B[e, j] of the newest
// history entry e: one dependent load, then O(t * n) float32 FMAs.  One
// workgroup runs one episode end to end (select_kernel below), so no step
// ever leaves the compute unit.
//
// Gram layout per group (float32, row stride ld): rows [0, n) A rows of the
// tokens, row n the A row of START, rows [n+1, 2n+1) B rows of the tokens,
// row 2n+1 the B row of START, rows 2n+2 .. 2n+4 three parts of cK whose sum
// is cK (the context enters the products as three rows of the working dtype);
// columns [0, n) tokens, n STOP, n+1 START.
#include "sp_internal.h"

namespace sp {
namespace {

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
  int W;               // waves per workgroup; lane-owned columns [0, 64 W)
  int lt;              // lane-owned history entries per thread in LDS after the registers
  int ks;              // second-column history entries in LDS (multiple of 64)
  int alpha_ld;        // softmax weight array length (floats, multiple of 16)
  int hcap;            // history capacity of the LDS index arrays (>= max_cap + 1)
  float sigma;
  float c1;            // sigma * log2(e)
  float b_stop;
  int g;               // tokens kept per round (grouped kernels; 1 otherwise)
  uint32_t flags;
  int32_t* grp_kept;   // [G, max_cap] group-local kept indices, ascending
  int32_t* grp_count;  // [G]
  int32_t* grp_cnt_out;
  float* trace;
  int trace_steps;
  int trace_w;         // floats per trace record
  int logit_off;       // SP_LOGITS: offset of the logit vector in a record
  int logit_n;         // SP_LOGITS: token slots of that vector (max_group; 0 = no dump)
  // trajectory sums (Eqs. 5-7; g = 1 kernels instantiated with TRAJ)
  float* traj_s;
  float* traj_kbar;
  float* traj_pstop;
  int traj_pstop_steps;
  float traj_c;        // log2(e) / tau
  float traj_beta;
  int32_t* err;
};

// Dynamic LDS of the recurrence (byte offsets), shared by host and device.
//   hmain [64 W][lt]        lane-owned history past the registers (column-major)
//   hsec  [ks / 16][64][4][4]  history of the second columns: entry 16 k + 4 q + e of
//                           column 512 + c at [k][c][q][e] (quarter q of each block)
//   alpha [copies][alpha_ld] softmax weights (unnormalised), zero past the current
//                           history: g = 1, one copy per wave, written and read by
//                           that wave alone; grouped rounds, one copy written by
//                           wave 0
//   sm    [4]               grouped rounds: 1 / softmax sum, STOP term of the older
//                           entries
//   hcol  [hcap]            history columns (START = n + 1)
//   shist [hcap]            STOP column of the history B rows
//   key   [2][16]           g = 1: each wave's decision key, by step parity
//   red   [2][16]           per-wave best and runner-up (tracing), by step parity
//   cnt   [16]              end-of-episode counts
//   ckeys [16][kGMax + 1]   grouped rounds: each wave's best keys, descending (slots
//                           a launch never writes stay zero)
//   ranked [16][kGMax + 1]  grouped rounds: each wave's copy of the merged ranks
//   zpart [2][16]           trajectory sums: per-wave partial softmax sums by step parity
struct SelLds {
  int hmain, hsec, alpha, sm, hcol, shist, key, red, cnt, ckeys, ranked, zpart, total;
  __host__ __device__ SelLds(int W, int lt, int ks, int alpha_ld, int hcap, int copies) {
    hmain = 0;
    hsec = hmain + 64 * W * lt * 4;
    alpha = hsec + ks * 64 * 4;
    sm = alpha + copies * alpha_ld * 4;
    hcol = sm + 16;
    shist = (hcol + hcap * 4 + 15) & ~15;
    key = (shist + hcap * 4 + 15) & ~15;
    red = key + 2 * 16 * 8;
    cnt = red + 2 * 16 * 16;
    ckeys = cnt + 16 * 4;
    ranked = ckeys + 16 * (kGMax + 1) * 8;
    zpart = ranked + 16 * (kGMax + 1) * 8;
    total = zpart + 2 * 16 * 4;
  }
};

// The value, recomputed where it is used: keeps rarely used addresses out of
// the registers that hold the history across the step loop.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Workgroup barrier that orders LDS accesses only: outstanding global loads
// stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wave-wide max / sum, one fused DPP operation per stage: row shifts 1, 2, 4,
// 8, then row broadcasts 15 and 31 (lanes without a source keep their value);
// lane 63 ends with the result, returned to every lane.  A fixed combination
// order, so results are deterministic.  The nops cover the VALU-write to DPP-
// read hazard between stages.
__device__ __forceinline__ float wave_max_fused(float v) {
  asm volatile(
      "s_nop 1\n\tv_max_f32_dpp %0, %0, %0 row_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_max_f32_dpp %0, %0, %0 row_shr:2 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_max_f32_dpp %0, %0, %0 row_shr:4 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_max_f32_dpp %0, %0, %0 row_shr:8 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_max_f32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
      "s_nop 1\n\tv_max_f32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
      "s_nop 1"
      : "+v"(v));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ __forceinline__ float wave_sum_fused(float v) {
  asm volatile(
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_shr:2 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_shr:4 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_shr:8 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
      "s_nop 1"
      : "+v"(v));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Two wave-wide sums in one DPP chain (independent stages interleaved).
__device__ __forceinline__ void wave_sum2_fused(float& a, float& b) {
  asm volatile(
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32_dpp %1, %1, %1 row_shr:1 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_shr:2 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32_dpp %1, %1, %1 row_shr:2 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_shr:4 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32_dpp %1, %1, %1 row_shr:4 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_shr:8 row_mask:0xf bank_mask:0xf\n\t"
      "v_add_f32_dpp %1, %1, %1 row_shr:8 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
      "v_add_f32_dpp %1, %1, %1 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
      "s_nop 1\n\tv_add_f32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
      "v_add_f32_dpp %1, %1, %1 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
      "s_nop 1"
      : "+v"(a), "+v"(b));
  a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(a), 63));
  b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(b), 63));
}

// Decision key: larger value first, then lower index (64-bit unsigned max).
__device__ __forceinline__ uint64_t cand_key(float v, int idx) {
  const uint32_t u = __float_as_uint(v);
  const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)ord << 32) | (uint32_t)(0xffffffffu - (uint32_t)idx);
}
__device__ __forceinline__ float key_value(uint64_t k) {
  const uint32_t ord = (uint32_t)(k >> 32);
  return __uint_as_float((ord & 0x80000000u) ? (ord & 0x7fffffffu) : ~ord);
}
__device__ __forceinline__ int key_index(uint64_t k) {
  return (int)(0xffffffffu - (uint32_t)k);
}

// One workgroup runs one episode with W waves.  Thread j < 64 W owns
// candidate column j: its history B values are in registers (the first RREG
// entries), then in LDS (lt entries), then re-read from the Gram buffer.
// With SEC (W = 8, 513-576 tokens) waves 0-3 (one per SIMD) also own the
// columns 512-575: lane 4 c + q of wave w sums quarter q of every 16-entry
// block of the history of column 512 + 16 w + c (history in LDS), and a quad
// reduction combines the four quarters.  Each SIMD then carries the same
// share of the step's FMAs.  STOP is not a column: its history term is a dot
// product of the weights with the STOP column of the history rows, reduced
// inside the softmax.
//
// A step: every wave computes its columns' logits from the softmax weights in
// LDS and folds its best candidate into the step's decision key (a 64-bit LDS
// atomic max of value bits and inverted index, so ties go to the lower index
// and STOP, index n, loses them); barrier; every wave reads the same decision;
// each thread loads the chosen row's A and B values of its columns, and wave
// 0 gathers the history scores from the chosen A row and writes the next
// softmax into LDS; barrier.  The B values are first needed at the end of the
// next step's logits, after the older history terms.
//
// Grouped kernels (GMAX > 1, Eq. 11) keep g tokens per round: the newest
// history entries are a group of ng tokens whose mean query row drives the
// next round (its A row is the mean of the members' A rows, so the history
// scores and the A term of the logits are means too); each wave then finds
// its g best candidates, writes their keys to LDS, and after the barrier
// every wave ranks all of them the same way, stops if STOP's key beats the
// best, and otherwise takes the g best as the round's group.
template <int RREG, bool SEC, bool TRACE, int MAXT, int GMAX, bool TRAJ>
__global__ __launch_bounds__(MAXT) void select_kernel(SelParams p) {
  constexpr bool GROUPED = GMAX > 1;
  static_assert(GMAX >= 1 && GMAX <= kGMax, "group size");
  static_assert(!(SEC && MAXT == 1024), "second columns only in 8-wave groups");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int g = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int W = SEC ? 8 : p.W;

  const int64_t g0 = p.grp_off[g], g1 = p.grp_off[g + 1];
  const int n = (int)(g1 - g0);
  const int cap = p.grp_cap[g];
  const int b = p.grp_img[g];
  {
    int code = 0;
    if (g0 < 0 || g1 < g0 || g1 > p.T_vis || b < 0 || b >= p.B) code = SP_DEV_BAD_OFFSETS;
    else if (n > p.max_group) code = SP_DEV_GROUP_TOO_LARGE;
    else if (cap < 0 || (int64_t)p.max_cap <
                          ((int64_t)cap * (GROUPED ? p.g : 1) < n ? (int64_t)cap * (GROUPED ? p.g : 1) : n))
      code = SP_DEV_BAD_CAP;
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
  const bool full = (p.flags & SP_FULL_ROLLOUT) != 0;   // STOP scored, never taken while tokens remain
  const int lt = p.lt, ks = p.ks;
  const SelLds L(W, lt, ks, p.alpha_ld, p.hcap, GROUPED ? 1 : W);
  float* hmain = reinterpret_cast<float*>(smem + L.hmain);
  float* hsec = reinterpret_cast<float*>(smem + L.hsec);
  float* alpha = reinterpret_cast<float*>(smem + L.alpha);
  // this wave's copy of the history weights (g = 1), the shared one otherwise
  float* alphaw = alpha + (GROUPED ? 0 : wave * p.alpha_ld);
  float* sm = reinterpret_cast<float*>(smem + L.sm);
  int* hcol = reinterpret_cast<int*>(smem + L.hcol);
  float* shist = reinterpret_cast<float*>(smem + L.shist);
  unsigned long long* key = reinterpret_cast<unsigned long long*>(smem + L.key);
  unsigned long long* ckeys = reinterpret_cast<unsigned long long*>(smem + L.ckeys);
  unsigned long long* ranked = reinterpret_cast<unsigned long long*>(smem + L.ranked);
  float* zpart = reinterpret_cast<float*>(smem + L.zpart);
  float4* red = reinterpret_cast<float4*>(smem + L.red);
  int* cnt = reinterpret_cast<int*>(smem + L.cnt);

  const int ld = p.ld;
  const float* A = p.gram + (int64_t)g * p.gstride;          // A row r at A + r * ld
  const float* Bm = A + (int64_t)(n + 1) * ld;               // B row r at Bm + r * ld
  const float* CK = A + (int64_t)(2 * n + 2) * ld;           // the three parts of cK
  const int j = tid;
  const bool mcol = j < n;
  const int sq = lane & 3;                                   // history quarter (second columns)
  const int scl = (wave << 4) | (lane >> 2);                 // second column - 512
  const int js = 512 + scl;
  const bool swave = SEC && wave < 4;
  const bool scol = swave && js < n;
  const int jc = mcol ? j : 0, jsc = scol ? js : 0;   // columns a lane reads (0 when it has none)
  const float sigma = p.sigma, c1 = p.c1;

  auto ckv = [&](int c) { return (CK[c] + CK[ld + c]) + CK[2 * ld + c]; };
  const float ck_main = mcol ? ckv(j) : 0.0f;
  const float ck_sec = scol ? ckv(js) : 0.0f;
  const float ck_stop = ckv(n);

  for (int i = 0; i < lt; ++i) hmain[j * lt + i] = 0.0f;
  if (SEC)
    for (int i = tid; i < ks * 16; i += 64 * W)
      reinterpret_cast<float4*>(hsec)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  // the weights past the history stay zero: each copy's only writer clears it
  // before its first softmax
  if (!GROUPED || wave == 0)
    for (int i = lane; i < p.alpha_ld; i += 64) alphaw[i] = 0.0f;
  if (GROUPED)
    for (int i = tid; i < 16 * (kGMax + 1); i += 64 * W) ckeys[i] = 0ull;

  // Lane-owned history values in 32-wide vector registers.  Reads use
  // constant slots after unrolling; a write picks the vector with a uniform
  // branch and the element with an indexed register move.  Separate variables
  // and conditions the optimiser cannot prove exclusive keep every access a
  // register operation.
  static_assert(RREG % 32 == 0 && RREG <= 160, "history registers come in 32-wide vectors");
  constexpr int NV = RREG / 32;
  f32x32_t h0{}, h1{}, h2{}, h3{}, h4{};
  auto hget = [&](int i) -> float {
    return i < 32 ? h0[i & 31] : i < 64 ? h1[i & 31] : i < 96 ? h2[i & 31]
         : i < 128 ? h3[i & 31] : h4[i & 31];
  };
  auto hput = [&](int pos, float x) {
    const int e = __builtin_amdgcn_readfirstlane(pos & 31);   // uniform: one indexed move
    const int k = __builtin_amdgcn_readfirstlane(pos >> 5);
    // one opaque scalar copy of k per test: scalar compares and branches
    int k0 = k, k1 = k, k2 = k, k3 = k, k4 = k;
    asm volatile("" : "+s"(k0), "+s"(k1), "+s"(k2), "+s"(k3), "+s"(k4));
    if (k0 == 0) h0[e] = x;
    if (NV > 1 && k1 == 1) h1[e] = x;
    if (NV > 2 && k2 == 2) h2[e] = x;
    if (NV > 3 && k3 == 3) h3[e] = x;
    if (NV > 4 && k4 == 4) h4[e] = x;
  };
  // Slot pos of a four-register, 256-entry history array (entry lane + 64 k
  // in register k): the owning lane takes v.  The register is chosen with a
  // scalar comparison, the lane with a select.
  auto put4 = [&](auto& r0, auto& r1, auto& r2, auto& r3, int pos, auto v) {
    const int k = __builtin_amdgcn_readfirstlane(pos >> 6);
    const bool mine = lane == (pos & 63);
    r0 = mine && k == 0 ? v : r0;
    r1 = mine && k == 1 ? v : r1;
    r2 = mine && k == 2 ? v : r2;
    r3 = mine && k == 3 ? v : r3;
  };
  // History column of entry lane + 64 k, for the first 256 entries.
  int hc0 = 0, hc1 = 0, hc2 = 0, hc3 = 0;
  // The STOP column of the history's B rows, entry lane + 64 k in slot k (also
  // kept in LDS for histories past 256 entries): every wave keeps it for
  // g = 1, wave 0 for grouped rounds.
  float sh0 = 0.0f, sh1 = 0.0f, sh2 = 0.0f, sh3 = 0.0f;

  // The newest history entry (position hl - 1): its column, its A values, and
  // its B values, which are stored into the history one step later.
  int ecol = n + 1;
  float a_main = 0.0f, a_sec = 0.0f, a_stop = 0.0f;
  float b_main = 0.0f, b_sec = 0.0f, b_stop = 0.0f;
  int hl = 0;
  // g = 1: this wave's softmax of the newest entry: the reciprocal of the
  // weights' sum, the STOP term of the older entries and the newest weight.
  float s_inv = 0.0f, s_st = 0.0f, s_enew = 0.0f;
  // Grouped rounds: the newest group (ng entries at the end of the history),
  // its rows, and its B values, stored into the history at the next decision.
  const int gsz = GROUPED ? p.g : 1;
  int ng = 1;
  [[maybe_unused]] int grow[GMAX];
  [[maybe_unused]] float bg[GMAX], bgs[GMAX], bst[GMAX];
#pragma unroll
  for (int i = 0; i < GMAX; ++i) {
    grow[i] = n;
    bg[i] = bgs[i] = bst[i] = 0.0f;
  }

  // g = 1: history softmax of the newest entry e (its A row Ar), run by every
  // wave into its own weights: e_tau = exp(sigma (A[e, col(tau)] - max)), the
  // reciprocal of their sum, the STOP term of the older entries (sum e_tau
  // B[tau, STOP]) and the newest entry's own weight.  r0..r3 are the scores
  // gathered at the history columns before the newest entry's column was set
  // (its slot takes r_new, its own score); bst_prev is the STOP value of the
  // entry stored into the history this step.
  auto softmax_all = [&](const float* Ar, float r0, float r1, float r2, float r3, float r_new,
                         float bst_prev) {
    const int hpad = (hl + 15) & ~15;
    const int pos = hl - 1;
    float m, sum = 0.0f, s2 = 0.0f;
    if (hl <= 256) {
      put4(r0, r1, r2, r3, pos, r_new);
      const float x0 = lane < hl ? r0 * c1 : -INFINITY;
      const float x1 = lane + 64 < hl ? r1 * c1 : -INFINITY;
      const float x2 = lane + 128 < hl ? r2 * c1 : -INFINITY;
      const float x3 = lane + 192 < hl ? r3 * c1 : -INFINITY;
      m = wave_max_fused(fmaxf(fmaxf(x0, x1), fmaxf(x2, x3)));
      auto one = [&](int k, float x, float sh) {
        const int tau = lane + 64 * k;
        const float e = tau < hl ? __builtin_amdgcn_exp2f(x - m) : 0.0f;
        sum += e;
        s2 = fmaf(e, tau < hl - 1 ? sh : 0.0f, s2);
        if (tau < hpad) alphaw[opaque(tau)] = e;
      };
      one(0, x0, sh0);
      if (64 < hpad) one(1, x1, sh1);
      if (128 < hpad) one(2, x2, sh2);
      if (192 < hpad) one(3, x3, sh3);
    } else {
      // longer histories: the scores are gathered again in each pass; the
      // newest column and the STOP value stored this step come from registers
      // (other waves' writes of this step need not be visible yet)
      auto col = [&](int tau) { return tau == pos ? ecol : hcol[tau]; };
      m = -INFINITY;
      for (int tau = lane; tau < hl; tau += 64) m = fmaxf(m, Ar[col(tau)] * c1);
      m = wave_max_fused(m);
      for (int tau = lane; tau < hpad; tau += 64) {
        const float e = tau < hl ? __builtin_amdgcn_exp2f(Ar[col(tau)] * c1 - m) : 0.0f;
        sum += e;
        const float sv = tau < pos - 1 ? shist[tau] : tau == pos - 1 ? bst_prev : 0.0f;
        s2 = fmaf(e, sv, s2);
        alphaw[tau] = e;
      }
    }
    wave_sum2_fused(sum, s2);
    s_inv = __builtin_amdgcn_rcpf(sum);
    s_st = s2;
    s_enew = __builtin_amdgcn_exp2f(r_new * c1 - m);
  };

  // g = 1: store the newest entry's B values into the history (before the
  // next entry replaces them).
  auto store_entry = [&]() {
    const int pos = hl - 1;
    if (pos < RREG) hput(pos, b_main);
    else if (pos < RREG + lt) hmain[opaque(j) * lt + (pos - RREG)] = b_main;
    // waves 0-3: 4 scl + sq is the thread index
    if (swave && pos < ks && sq == ((pos >> 2) & 3))
      hsec[(((pos >> 4) * 256 + opaque(tid)) << 2) + (pos & 3)] = b_sec;
    if (tid == 0) shist[pos] = b_stop;
    put4(sh0, sh1, sh2, sh3, pos, b_stop);
  };

  // g = 1: entry (row r, column c) becomes the newest.  Every load of the step
  // is issued first, so they share one memory round trip: this thread's A and
  // B values of the new row (columns without a candidate read column 0 and
  // are never used), the STOP column, and the history scores gathered from the
  // new row at the history columns (slots past the history read a valid
  // column and are masked).  The bookkeeping runs while they are in flight;
  // then every wave computes the history softmax.
  auto advance = [&](int r, int c) {
    const float* Ar = A + (int64_t)r * ld;
    const float* Br = Bm + (int64_t)r * ld;
    const float na = Ar[jc], nb = Br[jc];
    float nas = 0.0f, nbs = 0.0f;
    if (SEC) {
      nas = Ar[jsc];
      nbs = Br[jsc];
    }
    const float na_stop = Ar[n], nb_stop = Br[n];
    const float r_new = Ar[c];
    float r0 = 0.0f, r1 = 0.0f, r2 = 0.0f, r3 = 0.0f;
    if (hl < 256) {
      r0 = Ar[hc0];
      r1 = Ar[hc1];
      r2 = Ar[hc2];
      r3 = Ar[hc3];
    }
    const float bst_prev = b_stop;
    const int pos = hl;
    if (pos > 0) store_entry();
    put4(hc0, hc1, hc2, hc3, pos, c);
    if (tid == 0) hcol[pos] = c;
    ecol = c;
    hl = pos + 1;
    a_main = na;
    b_main = nb;
    a_sec = nas;
    b_sec = nbs;
    a_stop = na_stop;
    b_stop = nb_stop;
    softmax_all(Ar, r0, r1, r2, r3, r_new, bst_prev);
  };

  // Grouped rounds: history softmax for the mean query of the newest group,
  // x_tau = sigma mean_i A[row_i, col(tau)]; the newest group's own weights
  // stay in alpha (their B values are added separately), sm[1] is the STOP
  // term of the entries before it.  Wave 0 only.
  auto softmax_group = [&]() {
    const int hpad = (hl + 15) & ~15;
    const int old = hl - ng;
    const float cm = c1 / (float)ng;
    float m, sum = 0.0f, s2 = 0.0f;
    if (hl <= 256) {
      // every member slot's scores requested together (slots past the group
      // hold a valid row and are masked out of the sums)
      float y[GMAX][4];
#pragma unroll
      for (int i = 0; i < GMAX; ++i) {
        const float* Ar = A + (int64_t)grow[i] * ld;
        y[i][0] = Ar[hc0];
        y[i][1] = Ar[hc1];
        y[i][2] = Ar[hc2];
        y[i][3] = Ar[hc3];
      }
      // all requested before any is used (one round trip)
#pragma unroll
      for (int i = 0; i < GMAX; ++i)
        asm volatile("" : "+v"(y[i][0]), "+v"(y[i][1]), "+v"(y[i][2]), "+v"(y[i][3]));
      float r0 = 0.0f, r1 = 0.0f, r2 = 0.0f, r3 = 0.0f;
#pragma unroll
      for (int i = 0; i < GMAX; ++i) {
        const bool in = i < ng;
        r0 += in ? y[i][0] : 0.0f;
        r1 += in ? y[i][1] : 0.0f;
        r2 += in ? y[i][2] : 0.0f;
        r3 += in ? y[i][3] : 0.0f;
      }
      const float x0 = lane < hl ? r0 * cm : -INFINITY;
      const float x1 = lane + 64 < hl ? r1 * cm : -INFINITY;
      const float x2 = lane + 128 < hl ? r2 * cm : -INFINITY;
      const float x3 = lane + 192 < hl ? r3 * cm : -INFINITY;
      m = wave_max_fused(fmaxf(fmaxf(x0, x1), fmaxf(x2, x3)));
      auto one = [&](int k, float x, float sh) {
        const int tau = lane + 64 * k;
        const float e = tau < hl ? __builtin_amdgcn_exp2f(x - m) : 0.0f;
        sum += e;
        s2 = fmaf(e, tau < old ? sh : 0.0f, s2);
        if (tau < hpad) alpha[opaque(tau)] = e;
      };
      one(0, x0, sh0);
      if (64 < hpad) one(1, x1, sh1);
      if (128 < hpad) one(2, x2, sh2);
      if (192 < hpad) one(3, x3, sh3);
    } else {
      // longer histories: the scores are gathered again in each pass
      auto score = [&](int tau) {
        const int c = hcol[tau];
        float y[GMAX];
#pragma unroll
        for (int i = 0; i < GMAX; ++i) y[i] = A[(int64_t)grow[i] * ld + c];
        float r = 0.0f;
#pragma unroll
        for (int i = 0; i < GMAX; ++i) r += i < ng ? y[i] : 0.0f;
        return r * cm;
      };
      m = -INFINITY;
      for (int tau = lane; tau < hl; tau += 64) m = fmaxf(m, score(tau));
      m = wave_max_fused(m);
      for (int tau = lane; tau < hpad; tau += 64) {
        const float e = tau < hl ? __builtin_amdgcn_exp2f(score(tau) - m) : 0.0f;
        sum += e;
        s2 = fmaf(e, tau < old ? shist[tau < old ? tau : 0] : 0.0f, s2);
        alpha[tau] = e;
      }
    }
    wave_sum2_fused(sum, s2);
    if (lane == 0) {
      sm[0] = __builtin_amdgcn_rcpf(sum);
      sm[1] = s2;
    }
  };
  // Grouped rounds: load a group of cnt members (rows, columns) as the newest
  // entries: this thread's mean A value over the members and each member's B
  // values of its columns (left in flight); wave 0 computes the next softmax.
  // Every member slot's loads are issued together (slots past cnt hold a
  // valid row, columns without a candidate read column 0, and both are masked
  // out), so they share one memory round trip; 16-wave groups load one
  // member at a time.
  auto load_group = [&](const int (&rows)[GMAX], const int (&cols)[GMAX], int cnt) {
    float am = 0.0f, as2 = 0.0f, ast = 0.0f;
    [[maybe_unused]] float av[GMAX], asv[GMAX], atv[GMAX];
    if constexpr (MAXT == 1024) {
      // 16-wave groups (128 registers a lane): one member at a time, which
      // keeps fewer values live across the round
#pragma unroll
      for (int i = 0; i < GMAX; ++i) {
        if (i < cnt) {
          const float* Ar = A + (int64_t)rows[i] * ld;
          const float* Br = Bm + (int64_t)rows[i] * ld;
          am += mcol ? Ar[j] : 0.0f;
          bg[i] = mcol ? Br[j] : 0.0f;
          ast += Ar[n];
          bst[i] = Br[n];
          grow[i] = rows[i];
        }
      }
    } else {
      const int jc = mcol ? j : 0;
      const int jsc = scol ? js : 0;
#pragma unroll
      for (int i = 0; i < GMAX; ++i) {
        const float* Ar = A + (int64_t)rows[i] * ld;
        const float* Br = Bm + (int64_t)rows[i] * ld;
        av[i] = Ar[jc];
        bg[i] = Br[jc];
        asv[i] = 0.0f;
        if (SEC) {
          asv[i] = Ar[jsc];
          bgs[i] = Br[jsc];
        }
        atv[i] = Ar[n];
        bst[i] = Br[n];
        grow[i] = rows[i];
      }
    }
#pragma unroll
    for (int i = 0; i < GMAX; ++i) {
      if (i < cnt) {
        const int pos = hl + i;
        const int k = pos >> 6;
        const bool mine = lane == (pos & 63);
        if (__builtin_amdgcn_readfirstlane(k == 0) && mine) hc0 = cols[i];
        if (__builtin_amdgcn_readfirstlane(k == 1) && mine) hc1 = cols[i];
        if (__builtin_amdgcn_readfirstlane(k == 2) && mine) hc2 = cols[i];
        if (__builtin_amdgcn_readfirstlane(k == 3) && mine) hc3 = cols[i];
        if (tid == 0) hcol[pos] = cols[i];
      }
    }
    hl += cnt;
    ng = cnt;
    if (wave == 0) softmax_group();
    // the members' A values are summed only now, so wave 0's softmax gathers
    // went out while they were still in flight
    if constexpr (MAXT != 1024) {
#pragma unroll
      for (int i = 0; i < GMAX; ++i) {
        const bool in = i < cnt;
        am += in ? av[i] : 0.0f;
        as2 += in ? asv[i] : 0.0f;
        ast += in ? atv[i] : 0.0f;
      }
    }
    a_main = mcol ? am / (float)cnt : 0.0f;
    a_sec = scol ? as2 / (float)cnt : 0.0f;
    a_stop = ast / (float)cnt;
  };
  // Grouped rounds: store the newest group's B values into the history.
  auto store_group = [&]() {
#pragma unroll
    for (int i = 0; i < GMAX; ++i) {
      if (i < ng) {
        const int pos = hl - ng + i;
        if (pos < RREG) hput(pos, bg[i]);
        else if (pos < RREG + lt) hmain[opaque(j) * lt + (pos - RREG)] = bg[i];
        if (swave && pos < ks && sq == ((pos >> 2) & 3))
          hsec[(((pos >> 4) * 256 + opaque(tid)) << 2) + (pos & 3)] = bgs[i];
        if (tid == 0) shist[pos] = bst[i];
        if (wave == 0) {
          const int k = pos >> 6;
          const bool mine = lane == (pos & 63);
          if (__builtin_amdgcn_readfirstlane(k == 0) && mine) sh0 = bst[i];
          if (__builtin_amdgcn_readfirstlane(k == 1) && mine) sh1 = bst[i];
          if (__builtin_amdgcn_readfirstlane(k == 2) && mine) sh2 = bst[i];
          if (__builtin_amdgcn_readfirstlane(k == 3) && mine) sh3 = bst[i];
        }
      }
    }
  };

  if constexpr (GROUPED) {
    // history entry 0 is START: row n of A and B, column n + 1
    int rows[GMAX], cols[GMAX];
#pragma unroll
    for (int i = 0; i < GMAX; ++i) rows[i] = cols[i] = 0;
    rows[0] = n;
    cols[0] = n + 1;
    load_group(rows, cols, 1);
  } else {
    advance(n, n + 1);   // history entry 0 is START: row n of A and B, column n + 1
    // Consume START's loaded values here: a load still pending at the loop's
    // entry would make every step wait for its first load before the history
    // bookkeeping.
    asm volatile("" ::"v"(a_main), "v"(b_main), "v"(a_sec), "v"(b_sec), "v"(a_stop), "v"(b_stop));
  }
  lds_barrier();
  bool selected = false, sel_sec = false;
  int kept = 0;

  // Trajectory sums (g = 1, TRAJ kernels): step t's unnormalised candidate
  // weights e = exp((l - max) / tau) stay in registers while the per-wave
  // partial sums cross the step's closing barrier; at the top of step t + 1
  // every lane adds the partials in wave order, and with p_t = e / Z updates
  // s (its columns), K_bar and A.  Uniform values are kept in every lane.
  const bool traj = TRAJ && !GROUPED && p.traj_s != nullptr;
  float tj_A = 1.0f, tj_bt = 1.0f, tj_kbar = 0.0f, tj_s = 0.0f, tj_s2 = 0.0f;
  float tj_e = 0.0f, tj_e2 = 0.0f, tj_estop = 0.0f;
  int tj_t = 0;
  bool tj_pending = false;
  auto traj_finish = [&]() {
    const int pp = tj_t & 1;
    float Z = tj_estop;
    for (int w = 0; w < W; ++w) Z += zpart[pp * 16 + w];
    const float inv = Z > 0.0f ? 1.0f / Z : 0.0f;
    const float pst = Z > 0.0f ? tj_estop * inv : 1.0f;   // no finite candidate: p(STOP) = 1
    tj_bt *= p.traj_beta;                                   // beta^t
    const float wgt = tj_A * tj_bt * inv;
    tj_s = fmaf(wgt, tj_e, tj_s);
    tj_s2 = fmaf(wgt, tj_e2, tj_s2);
    tj_kbar = fmaf(tj_A, 1.0f - pst, tj_kbar);
    if (tid == 0 && p.traj_pstop && tj_t <= p.traj_pstop_steps)
      p.traj_pstop[(int64_t)g * p.traj_pstop_steps + (tj_t - 1)] = pst;
    tj_A *= 1.0f - pst;
    tj_pending = false;
  };

  for (int t = 1; t <= cap; ++t) {
    const int par = t & 1;
    if (traj && tj_pending) traj_finish();
    const float inv = GROUPED ? sm[0] : s_inv, st = GROUPED ? sm[1] : s_st;
    const float e_new = GROUPED ? 0.0f : s_enew;

    // ---- second columns (waves 0-3), older entries: each lane sums its
    // quarter of every 16-entry block, 64 entries per pass with all eight
    // reads issued first, and a quad sum combines the quarters.  Entries past
    // the newest are zero in LDS and alpha is zero past the history, so whole
    // passes need no masking.  This runs before the lane-owned logits: its LDS
    // round trips then overlap the other wave of the SIMD (waves 4-7 have no
    // second columns) instead of holding the step's decision after it.
    float qs = 0.0f;
    if (swave) {
      float acc2 = 0.0f, acc2b = 0.0f;
      const int last = hl - ng;                // the newest entries are added after the logits
      const int lend = last < ks ? last : ks;
      const int st4 = opaque(tid);                 // 4 scl + sq in waves 0-3
      const float* as = alphaw + 4 * (st4 & 3);
      const float* hs = hsec + st4 * 4;
      for (int k0 = 0; 16 * k0 < lend; k0 += 4) {
        float4 av[4], hv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          av[u] = *reinterpret_cast<const float4*>(as + 16 * (k0 + u));
          hv[u] = *reinterpret_cast<const float4*>(hs + (k0 + u) * 1024);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          acc2 = fmaf(av[u].x, hv[u].x, acc2);
          acc2b = fmaf(av[u].y, hv[u].y, acc2b);
          acc2 = fmaf(av[u].z, hv[u].z, acc2);
          acc2b = fmaf(av[u].w, hv[u].w, acc2b);
        }
      }
      // entries past the LDS tier: read again from the Gram buffer, every
      // fourth one per lane
      for (int tau = ks + sq; tau < last; tau += 4) {
        const int c = hcol[tau];
        const float hv = scol ? Bm[(int64_t)(c == n + 1 ? n : c) * ld + js] : 0.0f;
        acc2 = fmaf(alphaw[tau], hv, acc2);
      }
      // quad sum of the four quarters: (q0 + q1) + (q2 + q3) in every lane of
      // the quad (each addition is commutative, so all four agree bit for bit)
      qs = acc2 + acc2b;
      qs += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(qs), 0xB1, 0xF, 0xF, true));
      qs += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(qs), 0x4E, 0xF, 0xF, true));
    }

    // ---- logits of the lane-owned columns: older entries from the history
    // tiers (the newest entry's slots still hold zero), then the newest.
    float acc = 0.0f, accb = 0.0f;   // two independent chains (even, odd entries)
    {
      // Weights come from LDS 16 at a time, the next 16 requested before the
      // current 16 are used (alternating register sets, no copies).
      const float4* a4 = reinterpret_cast<const float4*>(alphaw);
      float4 xa[2][4];
      xa[0][0] = a4[0]; xa[0][1] = a4[1]; xa[0][2] = a4[2]; xa[0][3] = a4[3];
#pragma unroll
      for (int bi = 0; bi < RREG / 16; ++bi) {
        const int blk = bi * 16;
        if (blk < hl) {
          const int cur = bi & 1, nxt = cur ^ 1;
          if (blk + 16 < RREG) {   // unconditional: a uniform skip would make every wait conservative
            xa[nxt][0] = a4[(blk + 16) / 4 + 0];
            xa[nxt][1] = a4[(blk + 16) / 4 + 1];
            xa[nxt][2] = a4[(blk + 16) / 4 + 2];
            xa[nxt][3] = a4[(blk + 16) / 4 + 3];
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc = fmaf(xa[cur][q].x, hget(blk + 4 * q + 0), acc);
            accb = fmaf(xa[cur][q].y, hget(blk + 4 * q + 1), accb);
            acc = fmaf(xa[cur][q].z, hget(blk + 4 * q + 2), acc);
            accb = fmaf(xa[cur][q].w, hget(blk + 4 * q + 3), accb);
          }
        }
      }
    }
    if (hl > RREG) {
      const int lend = hl < RREG + lt ? hl : RREG + lt;
      const float* hj = hmain + opaque(j) * lt - RREG;
      int tau = RREG;
      for (; tau + 16 <= lend; tau += 16) {
        float4 av[4], hv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          av[u] = *reinterpret_cast<const float4*>(alphaw + tau + 4 * u);
          hv[u] = *reinterpret_cast<const float4*>(hj + tau + 4 * u);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          acc = fmaf(av[u].x, hv[u].x, acc);
          accb = fmaf(av[u].y, hv[u].y, accb);
          acc = fmaf(av[u].z, hv[u].z, acc);
          accb = fmaf(av[u].w, hv[u].w, accb);
        }
      }
      for (; tau < lend; tau += 4) {
        const float4 av = *reinterpret_cast<const float4*>(alphaw + tau);
        const float4 hv = *reinterpret_cast<const float4*>(hj + tau);
        acc = fmaf(av.x, hv.x, acc);
        accb = fmaf(av.y, hv.y, accb);
        acc = fmaf(av.z, hv.z, acc);
        accb = fmaf(av.w, hv.w, accb);
      }
      for (tau = RREG + lt; tau < hl - ng; tau += 8) {
        float hv[8], av[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          hv[u] = 0.0f;
          av[u] = 0.0f;
          if (tau + u < hl - ng) {
            const int c = hcol[tau + u];
            av[u] = alphaw[tau + u];
            if (mcol) hv[u] = Bm[(int64_t)(c == n + 1 ? n : c) * ld + j];
          }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = fmaf(av[u], hv[u], acc);
      }
    }
    float sp;
    [[maybe_unused]] float wg[GMAX];     // grouped: the newest group's weights
    if constexpr (GROUPED) {
#pragma unroll
      for (int i = 0; i < GMAX; ++i) wg[i] = i < ng ? alpha[hl - ng + i] : 0.0f;
      acc += accb;
      sp = st;
#pragma unroll
      for (int i = 0; i < GMAX; ++i) {
        if (i < ng) {
          acc = fmaf(wg[i], bg[i], acc);
          sp = fmaf(wg[i], bst[i], sp);
        }
      }
    } else {
      acc = fmaf(e_new, b_main, acc + accb);
      sp = fmaf(e_new, b_stop, st);
    }
    const float lj = sigma * (ck_main + a_main + acc * inv);
    const float l_stop = sigma * (ck_stop + a_stop + sp * inv) + p.b_stop;

    // ---- second columns: the newest entries, then the logit
    float ls = -INFINITY;
    if (swave) {
      if constexpr (GROUPED) {
#pragma unroll
        for (int i = 0; i < GMAX; ++i)
          if (i < ng) qs = fmaf(wg[i], bgs[i], qs);
      } else {
        qs = fmaf(e_new, b_sec, qs);
      }
      ls = scol && !sel_sec ? sigma * (ck_sec + a_sec + qs * inv) : -INFINITY;
    }

    if (TRACE && p.logit_n > 0 && t <= p.trace_steps) {
      // SP_LOGITS: the step's whole logit vector after its record (token slots
      // of masked tokens and past the group keep -inf), STOP last
      float* lrec = p.trace + ((int64_t)g * p.trace_steps + (t - 1)) * p.trace_w + p.logit_off;
      if (mcol) lrec[j] = selected ? -INFINITY : lj;
      if (SEC && scol && sq == 0) lrec[js] = ls;
      if (tid == 0) lrec[p.logit_n] = l_stop;
    }

    if constexpr (GROUPED) {
      // ---- this wave's best gl candidates, descending (lowest index on ties)
      const int gl = gsz + (TRACE ? 1 : 0);
      const bool valid = mcol && !selected;
      float v1 = valid ? lj : -INFINITY;
      float ls1 = ls;
      unsigned long long* ck = ckeys + wave * (kGMax + 1);
#pragma unroll
      for (int r = 0; r <= GMAX; ++r) {
        if (r < gl) {
          const float vm = wave_max_fused(swave ? fmaxf(v1, ls1) : v1);
          unsigned long long kr = 0ull;
          if (vm > -INFINITY) {
            const uint64_t m1 = __ballot(v1 == vm);
            int idx;
            if (m1) idx = wave * 64 + __ffsll((unsigned long long)m1) - 1;
            else idx = 512 + (wave << 4) + ((__ffsll((unsigned long long)__ballot(ls1 == vm)) - 1) >> 2);
            kr = cand_key(vm, idx);
            if (j == idx) v1 = -INFINITY;
            if (SEC && js == idx) ls1 = -INFINITY;
          }
          if (lane == 0) ck[r] = kr;
        }
      }
      lds_barrier();

      // ---- the decision: every wave ranks all keys the same way (valid keys
      // are distinct, having distinct indices; empty slots hold 0 and rank
      // below them), files the first GMAX + 1 by rank into its own list and
      // reads them back.  The slot count is fixed by the launch shape, so the
      // reads of the counting pass are independent and overlap.
      constexpr int NS = (MAXT / 64) * (kGMax + 1);
      constexpr int NQ = (NS + 63) / 64;
      static_assert(NS % 8 == 0, "key slots are read eight at a time");
      unsigned long long kv[NQ];
      int rk[NQ];
      int nvalid = 0;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int i = lane + 64 * q;
        kv[q] = i < NS ? ckeys[i] : 0ull;
        rk[q] = 0;
        nvalid += __popcll(__ballot(kv[q] != 0ull));
      }
      const ulonglong2* ck2 = reinterpret_cast<const ulonglong2*>(ckeys);
#pragma unroll(MAXT == 1024 ? 1 : NS / 8)
      for (int s0 = 0; s0 < NS / 2; s0 += 4) {
        ulonglong2 o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) o[u] = ck2[s0 + u];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int q = 0; q < NQ; ++q) rk[q] += (o[u].x > kv[q] ? 1 : 0) + (o[u].y > kv[q] ? 1 : 0);
      }
      unsigned long long* rl = ranked + wave * (kGMax + 1);
#pragma unroll
      for (int q = 0; q < NQ; ++q)
        if (kv[q] != 0ull && rk[q] <= GMAX) rl[rk[q]] = kv[q];
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // the key of rank r among the valid keys (0 if there is none)
      auto rank_key = [&](int r) -> unsigned long long { return r < nvalid ? rl[r] : 0ull; };
      // Valid keys hold ranks 0 .. valid - 1, so the group is ranks < min(g, valid).
      int gi[GMAX];
      int cnt = 0;
      float top_v = -INFINITY, gmin = -INFINITY, ru = -INFINITY;
      unsigned long long top0 = 0ull;
#pragma unroll
      for (int r = 0; r <= GMAX; ++r) {
        const unsigned long long kr = r < gl ? rank_key(r) : 0ull;
        if (r == 0) {
          top0 = kr;
          top_v = kr ? key_value(kr) : -INFINITY;
        }
        if (r < GMAX) gi[r] = kr != 0ull && r < gsz ? key_index(kr) : n;
        if (r < gsz && kr != 0ull) {
          ++cnt;
          gmin = key_value(kr);
        }
        if (TRACE && r == gsz && kr != 0ull) ru = key_value(kr);
      }
      // STOP ends the episode only as the round's largest logit (it loses ties)
      const unsigned long long stop_key = l_stop > -INFINITY ? cand_key(l_stop, n) : 0ull;
      const bool stop = top0 == 0ull || (!full && stop_key > top0);
      if (TRACE && tid == 0 && t <= p.trace_steps) {
        float* rec = p.trace + ((int64_t)g * p.trace_steps + (t - 1)) * p.trace_w;
#pragma unroll
        for (int r = 0; r < GMAX; ++r)
          if (r < gsz) rec[r] = __int_as_float(stop ? (r == 0 ? -1 : -3) : (r < cnt ? gi[r] : -3));
        rec[gsz] = stop ? l_stop : gmin;
        rec[gsz + 1] = stop ? top_v : fmaxf(ru, l_stop);
        rec[gsz + 2] = l_stop;
      }
      if (stop) break;
      kept += cnt;
#pragma unroll
      for (int r = 0; r < GMAX; ++r) {
        if (r < cnt) {
          if (j == gi[r]) selected = true;
          if (SEC && js == gi[r]) sel_sec = true;
        }
      }
      if (!no_history) {
        store_group();
        load_group(gi, gi, cnt);
      }
      lds_barrier();     // the next softmax is in LDS
    } else {
      // ---- this wave's best candidate (lowest index on ties) as its key in
      // the step's slots (wave 0 folds STOP in); the slots of this parity are
      // written again two steps on, after every wave has read them and passed
      // the next barrier
      const bool valid = mcol && !selected;
      const float v = valid ? lj : -INFINITY;
      const float vmax = wave_max_fused(swave ? fmaxf(v, ls) : v);
      int i1 = -1;
      unsigned long long wkey = 0ull;
      if (vmax > -INFINITY) {
        const uint64_t m1 = __ballot(valid && v == vmax);
        if (m1) i1 = wave * 64 + __ffsll((unsigned long long)m1) - 1;
        else if (SEC) i1 = 512 + (wave << 4) + ((__ffsll((unsigned long long)__ballot(ls == vmax)) - 1) >> 2);
        wkey = cand_key(vmax, i1);
      }
      if (wave == 0 && l_stop > -INFINITY && !full) {
        const unsigned long long sk = cand_key(l_stop, n);
        wkey = sk > wkey ? sk : wkey;
      }
      unsigned long long* kp = key + par * 16;
      if (lane == 0) kp[wave] = wkey;
      if (TRACE) {
        // runner-up of this wave: the best candidate other than i1
        const float w1 = valid && j != i1 ? lj : -INFINITY;
        const float w2 = SEC && js != i1 ? ls : -INFINITY;
        const float v2 = wave_max_fused(fmaxf(w1, w2));
        if (lane == 0) red[par * 16 + wave] = make_float4(vmax, __int_as_float(i1), v2, 0.0f);
      }
      lds_barrier();

      // ---- the decision: the largest key of the step (every wave reads them all)
      unsigned long long kk = 0ull;
      for (int w = 0; w < W; ++w) {
        const unsigned long long kw = kp[w];
        kk = kw > kk ? kw : kk;
      }
      // uniform: into scalar registers, so the row addresses are scalar work
      kk = ((unsigned long long)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(kk >> 32)) << 32) |
           (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)kk);
      const int a = kk ? key_index(kk) : n;       // no finite candidate: STOP
      if (TRACE && tid == 0 && t <= p.trace_steps) {
        // runner-up: the largest value among the candidates other than a
        float r2 = a == n ? -INFINITY : l_stop;
        for (int w = 0; w < W; ++w) {
          const float4 r = red[par * 16 + w];
          r2 = fmaxf(r2, __float_as_int(r.y) == a ? r.z : r.x);
        }
        float* rec = p.trace + ((int64_t)g * p.trace_steps + (t - 1)) * p.trace_w;
        rec[0] = __int_as_float(a == n ? -1 : a);
        rec[1] = kk ? key_value(kk) : l_stop;
        rec[2] = r2;
        rec[3] = l_stop;
      }
      if (traj) {
        // this step's candidate weights (the taken token is still a candidate)
        const float top = kk ? key_value(kk) : -INFINITY;
        const float M = top > l_stop ? top : l_stop;
        const bool any = M > -INFINITY;
        tj_e = any && mcol && !selected ? __builtin_amdgcn_exp2f((lj - M) * p.traj_c) : 0.0f;
        tj_e2 = any && ls > -INFINITY && sq == 0 ? __builtin_amdgcn_exp2f((ls - M) * p.traj_c) : 0.0f;
        tj_estop = any && l_stop > -INFINITY ? __builtin_amdgcn_exp2f((l_stop - M) * p.traj_c) : 0.0f;
        const float part = wave_sum_fused(tj_e + tj_e2);
        if (lane == 0) zpart[par * 16 + wave] = part;
        tj_t = t;
        tj_pending = true;
      }
      if (a == n) break;
      ++kept;
      if (j == a) selected = true;
      if (SEC && js == a) sel_sec = true;
      // the next step's weights: every wave computes its own, so no second
      // barrier is needed
      if (!no_history) advance(a, a);
    }
  }

  // ---- native order (Algorithm 1 step 4): ascending positions of the set
  // bits, lane-owned columns first, then the second columns (one lane of each
  // quad reports; waves 0-3 hold them in ascending order).
  __syncthreads();
  if (traj) {
    if (tj_pending) traj_finish();
    if (mcol) p.traj_s[g0 + j] = tj_s;
    if (SEC && scol && sq == 0) p.traj_s[g0 + js] = tj_s2;
    if (tid == 0) p.traj_kbar[g] = tj_kbar;
  }
  const uint64_t ballot = __ballot(mcol && selected);
  const uint64_t sb = __ballot(scol && sel_sec && sq == 0);
  if (lane == 0) {
    cnt[wave] = __popcll(ballot);
    if (SEC && wave < 4) cnt[8 + wave] = __popcll(sb);
  }
  __syncthreads();
  int before = 0, total = 0, before2 = 0;
  for (int w = 0; w < W; ++w) {
    if (w < wave) before += cnt[w];
    total += cnt[w];
  }
  if (SEC)
    for (int w = 0; w < wave && w < 4; ++w) before2 += cnt[8 + w];
  if (mcol && selected) {
    const int pos = before + __popcll(ballot & ((1ull << lane) - 1ull));
    p.grp_kept[(int64_t)g * p.max_cap + pos] = j;
  }
  if (scol && sel_sec && sq == 0) {
    const int pos = total + before2 + __popcll(sb & ((1ull << lane) - 1ull));
    p.grp_kept[(int64_t)g * p.max_cap + pos] = js;
  }
  if (tid == 0) {
    p.grp_count[g] = kept;
    if (p.grp_cnt_out) p.grp_cnt_out[g] = kept;
  }
}

// p_t(STOP) records past an episode's end hold NaN.
__global__ void fill_nan_kernel(float* x, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) x[i] = __int_as_float(0x7fc00000);
}

// Trace records (width floats) past an episode's end carry taken = -2; the
// logit vectors of SP_LOGITS (from float lo on) start at -inf.
__global__ void trace_fill_kernel(float* trace, int64_t count, int width, int lo) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) {
    float* rec = trace + i * width;
    rec[0] = __int_as_float(-2);
    for (int k = 1; k < lo; ++k) rec[k] = 0.0f;
    for (int k = lo; k < width; ++k) rec[k] = -INFINITY;
  }
}

// Per group (one wave each): copy its kept list into its image's slice of
// kept_idx, after the kept lists of the image's earlier groups, offset to
// image-local indices.  The groups of an image are contiguous and images come
// in order, so a group finds its place by summing the counts of the run of
// same-image groups just before it (64 at a time, one load per lane).  The
// image's last group writes the image's count; each group zeroes the counts
// of the images between the previous group's image and its own (the last
// group also those after its own), which have no group.  On an overflow of
// the image's slice the image's count is 0 (and the error word says why).
__global__ __launch_bounds__(64) void finalize_kernel(const int32_t* __restrict__ img_off, int B,
                                                      const int32_t* __restrict__ grp_off,
                                                      const int32_t* __restrict__ grp_img, int G,
                                                      const int32_t* __restrict__ grp_kept,
                                                      const int32_t* __restrict__ grp_count,
                                                      int max_cap,
                                                      const int32_t* __restrict__ kept_off,
                                                      int32_t* __restrict__ kept_idx,
                                                      int32_t* __restrict__ kept_cnt,
                                                      int32_t* err) {
  const int lane = threadIdx.x;
  if (G == 0) {
    for (int b = lane; b < B; b += 64) kept_cnt[b] = 0;
    return;
  }
  const int g = blockIdx.x;
  const int b = grp_img[g];
  const int prev = g > 0 ? grp_img[g - 1] : -1;
  const int next = g + 1 < G ? grp_img[g + 1] : B;
  if (b < 0 || b >= B || prev > b || next < b) {
    if (lane == 0) set_device_error(err, SP_DEV_BAD_OFFSETS);
    return;
  }
  // images strictly between the previous group's and this one have no group,
  // nor have those after the last group's
  for (int i = prev + 1 + lane; i < b; i += 64) kept_cnt[i] = 0;
  if (g == G - 1)
    for (int i = b + 1 + lane; i < B; i += 64) kept_cnt[i] = 0;

  // counts of the run of this image's groups before g
  int before = 0;
  for (int top = g - 1; top >= 0; top -= 64) {
    const int q = top - lane;
    const bool same = q >= 0 && grp_img[q] == b;
    const int c = same ? grp_count[q] : 0;
    const uint64_t other = __ballot(!same);
    const int run = other ? __ffsll((unsigned long long)other) - 1 : 64;
    int v = lane < run ? c : 0;
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    before += v;
    if (run < 64) break;
  }
  const int cnt = grp_count[g];
  const int64_t base = kept_off[b];
  const int64_t room = (int64_t)kept_off[b + 1] - base;
  if (base < 0 || room < 0) {
    if (lane == 0) set_device_error(err, SP_DEV_BAD_OFFSETS);
    return;
  }
  // every group of the image tests the image's total, so a slice that
  // overflows anywhere receives nothing
  int total = 0;
  {
    // the image's groups after g, counted the same way
    int after = 0;
    for (int bot = g + 1; bot < G; bot += 64) {
      const int q = bot + lane;
      const bool same = q < G && grp_img[q] == b;
      const int c = same ? grp_count[q] : 0;
      const uint64_t other = __ballot(!same);
      const int run = other ? __ffsll((unsigned long long)other) - 1 : 64;
      int v = lane < run ? c : 0;
      for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
      after += v;
      if (run < 64) break;
    }
    total = before + cnt + after;
  }
  if (total > room) {
    if (lane == 0) {
      set_device_error(err, SP_DEV_OUTPUT_OVERFLOW);
      if (next > b) kept_cnt[b] = 0;
    }
    return;
  }
  const int off = grp_off[g] - img_off[b];
  for (int i = lane; i < cnt; i += 64)
    kept_idx[base + before + i] = off + grp_kept[(int64_t)g * max_cap + i];
  if (lane == 0 && next > b) kept_cnt[b] = total;
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  const bool gram_only = (a.flags & SP_GRAM_ONLY) != 0;
  const bool reuse_gram = (a.flags & SP_REUSE_GRAM) != 0;
  if (a.G == 0) {
    if (gram_only) return hipSuccess;
    if (a.B > 0)
      hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(64), 0, stream, a.img_off, a.B,
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
  // the Gram products, unless a previous SP_GRAM_ONLY call left them in ws
  hipError_t e = reuse_gram ? hipSuccess : launch_gram_gemm(ga, stream);
  if (e != hipSuccess) return e;
  record_event(a.events, 1, stream);
  if (gram_only) return hipGetLastError();

  const bool trace = (a.flags & SP_TRACE) && a.trace && a.trace_steps > 0;
  const int rec_base = a.g > 1 ? a.g + 3 : 4;
  const int logit_n = trace && (a.flags & SP_LOGITS) ? a.max_group : 0;
  const int trace_w = rec_base + (logit_n > 0 ? logit_n + 1 : 0);
  if (trace) {
    const int64_t count = (int64_t)a.G * a.trace_steps;
    hipLaunchKernelGGL(trace_fill_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0,
                       stream, a.trace, count, trace_w, rec_base);
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
  p.b_stop = a.b_stop;
  p.g = a.g;
  p.flags = a.flags;
  p.grp_kept = a.grp_kept;
  p.grp_count = a.grp_count;
  p.grp_cnt_out = a.grp_cnt;
  p.trace = trace ? a.trace : nullptr;
  p.trace_steps = trace ? a.trace_steps : 0;
  p.trace_w = trace_w;
  p.logit_off = rec_base;
  p.logit_n = logit_n;
  const bool traj = a.traj_s != nullptr;
  p.traj_s = a.traj_s;
  p.traj_kbar = a.traj_kbar;
  p.traj_pstop = a.traj_pstop;
  p.traj_pstop_steps = a.traj_pstop ? a.traj_pstop_steps : 0;
  p.traj_c = traj ? 1.4426950408889634f / a.traj_tau : 0.0f;
  p.traj_beta = a.traj_beta;
  if (traj && p.traj_pstop_steps > 0) {
    const int64_t count = (int64_t)a.G * p.traj_pstop_steps;
    hipLaunchKernelGGL(fill_nan_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, stream,
                       p.traj_pstop, count);
  }
  p.err = a.err;

  // Waves: one lane per token column up to 512 columns (2 waves per SIMD, 256
  // registers each); 513-576 columns keep 8 waves and give wave 0 a second
  // column per lane; larger groups take 16 waves (128 registers each).
  const int mg = a.max_group > 0 ? a.max_group : 1;
  int W;
  bool sec = false;
  if (mg <= 512) {
    W = (mg + 63) / 64;
  } else if (mg <= 576) {
    W = 8;
    sec = true;
  } else {
    W = (mg + 63) / 64;
  }
  const bool wide = W > 8;
  const int need = a.max_cap + 1;                       // longest possible history
  const bool grouped = a.g > 1;
  // grouped kernels hold the newest group's values too, and their histories
  // grow g entries a round: 64 history registers, then the LDS tier
  int rreg = wide ? 32 : need <= 64 || grouped ? 64 : need <= 128 ? 128 : 160;
  // the trajectory sums take registers too: at most 128 history registers
  if (a.traj_s && rreg > 128) rreg = 128;
  p.W = W;
  p.hcap = (int)align_up((size_t)need + 1, 4);
  // alpha covers the register blocks' prefetch (up to rreg) and the second
  // columns' 64-entry passes.
  p.alpha_ld = (int)align_up((size_t)(need > rreg ? need : rreg), sec ? 64 : 16);
  p.sigma = 1.0f / sqrtf((float)a.h);
  p.c1 = p.sigma * 1.4426950408889634f;
  // LDS: fixed arrays, then wave 0's second-column history (all of it if it
  // fits), then the lane-owned tier past the registers; entries beyond either
  // are read again from the Gram buffer.
  const int copies = grouped ? 1 : W;              // softmax weight copies
  const size_t fixed = (size_t)SelLds(W, 0, 0, p.alpha_ld, p.hcap, copies).total;
  size_t room = fixed < (size_t)kLdsBytes ? (size_t)kLdsBytes - fixed : 0;
  int ks = 0;
  if (sec) {
    ks = (need + 63) / 64 * 64;                         // whole 64-entry passes
    const size_t per = 64 * 4;
    if ((size_t)ks * per > room) ks = (int)(room / per) / 64 * 64;
    room -= (size_t)ks * per;
  }
  int lt = 0;
  if (need > rreg) {
    lt = (need - rreg + 3) / 8 * 8 + 4;                 // smallest 8k + 4 >= the entries needed
    const size_t per = (size_t)64 * W * 4;
    size_t lt_max = room / per;
    // Column stride of 8k + 4 floats keeps the 16-byte reads of eight
    // consecutive columns on distinct banks.
    lt_max = lt_max >= 4 ? (lt_max - 4) / 8 * 8 + 4 : 0;
    if ((size_t)lt > lt_max) lt = (int)lt_max;
  }
  p.lt = lt;
  p.ks = ks;
  const size_t lds = (size_t)SelLds(W, lt, ks, p.alpha_ld, p.hcap, copies).total;
  if (lds > (size_t)kLdsBytes) return hipErrorInvalidValue;

  const void* fn = nullptr;
#define SP_PICK(RR, SEC, MAXT)                                                           \
  if (!grouped && rreg == RR && sec == SEC && (MAXT == 1024) == wide) {                  \
    if (traj)                                                                            \
      fn = trace ? (const void*)select_kernel<RR, SEC, true, MAXT, 1, true>              \
                 : (const void*)select_kernel<RR, SEC, false, MAXT, 1, true>;            \
    else                                                                                 \
      fn = trace ? (const void*)select_kernel<RR, SEC, true, MAXT, 1, false>             \
                 : (const void*)select_kernel<RR, SEC, false, MAXT, 1, false>;           \
  }
#define SP_PICK_NT(RR, SEC, MAXT)                                                        \
  if (!grouped && rreg == RR && sec == SEC && (MAXT == 1024) == wide && !traj)           \
    fn = trace ? (const void*)select_kernel<RR, SEC, true, MAXT, 1, false>               \
               : (const void*)select_kernel<RR, SEC, false, MAXT, 1, false>;
  SP_PICK(64, false, 512) SP_PICK(128, false, 512) SP_PICK_NT(160, false, 512)
  SP_PICK(64, true, 512) SP_PICK(128, true, 512) SP_PICK_NT(160, true, 512)
  SP_PICK(32, false, 1024)
#undef SP_PICK
#undef SP_PICK_NT
#define SP_PICK_G(RR, SEC, MAXT)                                                         \
  if (grouped && rreg == RR && sec == SEC && (MAXT == 1024) == wide)                     \
    fn = trace ? (const void*)select_kernel<RR, SEC, true, MAXT, kGMax, false>           \
               : (const void*)select_kernel<RR, SEC, false, MAXT, kGMax, false>;
  SP_PICK_G(64, false, 512) SP_PICK_G(64, true, 512) SP_PICK_G(32, false, 1024)
#undef SP_PICK_G
  if (!fn) return hipErrorInvalidValue;
  record_event(a.events, 2, stream);
  if ((e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds)) != hipSuccess)
    return e;
  void* kargs[] = {&p};
  if ((e = hipLaunchKernel(fn, dim3(a.G), dim3(64 * W), kargs, lds, stream)) != hipSuccess) return e;
  record_event(a.events, 3, stream);

  hipLaunchKernelGGL(finalize_kernel, dim3(a.G), dim3(64), 0, stream, a.img_off, a.B, a.grp_off,
                     a.grp_img, a.G, a.grp_kept, a.grp_count, a.max_cap, a.kept_off, a.kept_idx,
                     a.kept_cnt, a.err);
  return hipGetLastError();
}

}  // namespace sp
