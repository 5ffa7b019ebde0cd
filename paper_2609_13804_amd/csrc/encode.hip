// Eq. 3 on gfx950: the cross-modal input encoder.
//
//   E~ = g LN(E_text W_p^T)                  text projected into R^d (LayerNorm
//                                            without scale or shift, eps 1e-5)
//   H  = Enc([X_b; E~_b])[first N_b rows]    per image b
//
// Enc is two pre-norm transformer blocks of width d: multi-head attention with
// heads of width 128 over the image's whole sequence (bidirectional, or causal
// on request), and an MLP 4d wide with the exact GELU.  Every linear map runs
// on the matrix cores (gemm.hip's bfloat16 core), the q/k/v bias and the MLP's
// bias and GELU in the products' epilogues; the residual + LayerNorm steps are
// row kernels (denoise.hip), the rest is here.
//
// Sequence layout: image b's sequence occupies rows [so_b, so_b + S_b) of the
// workspace buffers, so_b = img_off[b] + text_off[b], S_b = N_b + L_b, its
// visual tokens first (visual row i of image b is sequence row
// i + text_off[b]) and its text tokens after them (text row t of image b is
// sequence row img_off[b + 1] + t).
//
// The residual stream R is float32.  The text product, the LayerNorm outputs,
// every product's result, the biased q/k/v, the probabilities that weight the
// values, each head's output, the GELU output and H are bfloat16, rounded
// once to nearest-even.
#include "sp_internal.h"
#include "lds_dma.h"
#include "row_ops.h"

namespace sp {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kHead = 128;                  // head width
constexpr int kQPerWave = 32;               // queries of one wave (one 32 x 32 MFMA tile)
constexpr int kAttnWaves = 4;               // 128 queries per workgroup
constexpr int kKeyBlock = 32;               // keys per online-softmax step
constexpr int kKeyTile = 64;                // keys per LDS tile of K and V^T
constexpr int kVtKeys = 64;                 // keys per transpose tile
constexpr float kTextLnEps = 1e-5f;

// The image owning row r of a packed array with offsets off[0..B]: the last
// image whose range starts at or before r (empty images are skipped).
__device__ __forceinline__ int owner(const int32_t* __restrict__ off, int B, int64_t r) {
  int lo = 0, hi = B;                       // off[lo] <= r < off[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (off[mid] <= r) lo = mid;
    else hi = mid;
  }
  return lo;
}

// Image b's sequence offset and length, or false (with the error word set)
// when its offsets are inconsistent or its length exceeds max_seq.
__device__ __forceinline__ bool sequence_of(const int32_t* __restrict__ img_off,
                                            const int32_t* __restrict__ text_off, int b,
                                            int max_seq, int64_t S_total, int64_t& so, int& S,
                                            int32_t* err, bool report) {
  const int n = img_off[b + 1] - img_off[b], L = text_off[b + 1] - text_off[b];
  so = (int64_t)img_off[b] + text_off[b];
  S = n + L;
  if (n < 0 || L < 0 || so < 0 || so + S > S_total) {
    if (report) set_device_error(err, SP_DEV_BAD_OFFSETS);
    return false;
  }
  if (S > max_seq) {
    if (report) set_device_error(err, SP_DEV_GROUP_TOO_LARGE);
    return false;
  }
  return true;
}

// ---------------------------------------------------------------- row kernels

// R[i + text_off[b]] = X[i], one workgroup per visual row.
__global__ __launch_bounds__(256) void enc_visual_kernel(
    const uint16_t* __restrict__ X, int d, const int32_t* __restrict__ img_off,
    const int32_t* __restrict__ text_off, int B, int64_t S_total, float* __restrict__ R,
    int32_t* err) {
  const int64_t i = blockIdx.x;
  const int b = owner(img_off, B, i);
  const int64_t s = i + text_off[b];
  if (s < 0 || s >= S_total) {
    if (threadIdx.x == 0) set_device_error(err, SP_DEV_BAD_OFFSETS);
    return;
  }
  for (int c = 8 * threadIdx.x; c < d; c += 8 * 256) {
    float v[8];
    load8(X + i * d + c, v);
    store8(R + s * d + c, v);
  }
}

// R[img_off[b + 1] + t] = g LN(P[t]) for text row t (LayerNorm without scale
// or shift, biased variance, eps 1e-5).  One wave per row.
__global__ __launch_bounds__(64 * kRowWaves) void enc_text_kernel(
    const uint16_t* __restrict__ P, int64_t T_txt, int d, const int32_t* __restrict__ img_off,
    const int32_t* __restrict__ text_off, int B, int64_t S_total, float g, float* __restrict__ R,
    int32_t* err) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6);
  if (t >= T_txt) return;
  const int b = owner(text_off, B, t);
  const int64_t s = (int64_t)img_off[b + 1] + t;
  if (s < 0 || s >= S_total) {
    if (lane == 0) set_device_error(err, SP_DEV_BAD_OFFSETS);
    return;
  }
  const int nch = d / 8;
  float v[kMaxChunks][8];
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    if (lane + 64 * i >= nch) break;
    load8(P + t * d + 8 * (lane + 64 * i), v[i]);
#pragma unroll
    for (int k = 0; k < 8; ++k) sum += v[i][k];
  }
  const float mean = wave_sum(sum) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    if (lane + 64 * i >= nch) break;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float u = v[i][k] - mean;
      q = fmaf(u, u, q);
    }
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + kTextLnEps);
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    if (lane + 64 * i >= nch) break;
    float o[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = g * ((v[i][k] - mean) * rstd);
    store8(R + s * d + 8 * (lane + 64 * i), o);
  }
}

// Z = LN(R) with scale g and shift b (the first block's LN1).  One wave per row.
__global__ __launch_bounds__(64 * kRowWaves) void enc_ln_kernel(
    const float* __restrict__ R, int64_t S, int d, const float* __restrict__ g,
    const float* __restrict__ b, uint16_t* __restrict__ Z) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6);
  if (r >= S) return;
  const int nch = d / 8;
  float v[kMaxChunks][8];
#pragma unroll
  for (int i = 0; i < kMaxChunks; ++i) {
    if (lane + 64 * i >= nch) break;
    load8(R + r * d + 8 * (lane + 64 * i), v[i]);
  }
  ln_store(v, nch, d, lane, g, b, Z + r * d);
}

// H[i] = bf16((R[s] + T[s]) + bias) for visual row i (s = i + text_off[b]):
// the last block's residual, visual positions only.  One workgroup per row.
__global__ __launch_bounds__(256) void enc_out_kernel(
    const float* __restrict__ R, const uint16_t* __restrict__ T, const float* __restrict__ bias,
    int d, const int32_t* __restrict__ img_off, const int32_t* __restrict__ text_off, int B,
    int64_t S_total, uint16_t* __restrict__ H, int32_t* err) {
  const int64_t i = blockIdx.x;
  const int b = owner(img_off, B, i);
  const int64_t s = i + text_off[b];
  if (s < 0 || s >= S_total) {
    if (threadIdx.x == 0) set_device_error(err, SP_DEV_BAD_OFFSETS);
    return;
  }
  for (int c = 8 * threadIdx.x; c < d; c += 8 * 256) {
    float x[8], y[8], bb[8];
    load8(R + s * d + c, x);
    load8(T + s * d + c, y);
    load8(bias + c, bb);
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = (x[k] + y[k]) + bb[k];
    store8(H + i * d + c, x);
  }
}

// ---------------------------------------------------------------- attention

// Vt[b][head][e][p] = V[so_b + k][128 head + e] for k < S_b, 0 up to smax_pad:
// each head's values transposed, keys contiguous except that the middle two
// 4-key quarters of every 16 keys trade places (position p of key k: quarter
// order 0, 2, 1, 3).  The attention's value operand for a lane half is then
// one 16-byte chunk (see attn_kernel).  One workgroup per 64 keys x 128.
__global__ __launch_bounds__(256) void vt_kernel(
    const uint16_t* __restrict__ QKV, int d, int smax_pad, const int32_t* __restrict__ img_off,
    const int32_t* __restrict__ text_off, int max_seq, int64_t S_total, uint16_t* __restrict__ Vt,
    int32_t* err) {
  const int b = blockIdx.z, hd = blockIdx.y, heads = gridDim.y;
  const int k0 = blockIdx.x * kVtKeys;
  int64_t so;
  int S;
  if (!sequence_of(img_off, text_off, b, max_seq, S_total, so, S, err, false)) return;
  __shared__ __attribute__((aligned(16))) uint16_t tile[kVtKeys][kHead + 8];
  const int tid = threadIdx.x;
  const int64_t ld = 3 * (int64_t)d;
  for (int i = tid; i < kVtKeys * (kHead / 8); i += 256) {
    const int r = i / (kHead / 8), ch = i % (kHead / 8);
    const int k = k0 + r;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (k < S) v = *reinterpret_cast<const uint4*>(QKV + (so + k) * ld + 2 * d + hd * kHead + 8 * ch);
    *reinterpret_cast<uint4*>(&tile[r][8 * ch]) = v;
  }
  __syncthreads();
  const int e = tid >> 1, kh = tid & 1;
  uint16_t* dst = Vt + (((int64_t)b * heads + hd) * kHead + e) * smax_pad + k0 + 32 * kh;
#pragma unroll
  for (int j = 0; j < 32; j += 16) {
    const uint16_t* c = &tile[32 * kh + j][e];
    auto two = [&](int k) {
      return (uint32_t)c[k * (kHead + 8)] | ((uint32_t)c[(k + 1) * (kHead + 8)] << 16);
    };
    // positions 0-7: keys 0-3, 8-11; positions 8-15: keys 4-7, 12-15
    *reinterpret_cast<uint4*>(dst + j) = make_uint4(two(0), two(2), two(8), two(10));
    *reinterpret_cast<uint4*>(dst + j + 8) = make_uint4(two(4), two(6), two(12), two(14));
  }
}

__device__ __forceinline__ bf16x8_t ld16(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(p));
}
__device__ __forceinline__ bf16x8_t pack8(const float* v) {
  uint4 u;
  u.x = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
  u.y = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
  u.z = (uint32_t)f32_to_bf16(v[4]) | ((uint32_t)f32_to_bf16(v[5]) << 16);
  u.w = (uint32_t)f32_to_bf16(v[6]) | ((uint32_t)f32_to_bf16(v[7]) << 16);
  return __builtin_bit_cast(bf16x8_t, u);
}

// Multi-head attention of every image's sequence: O[so + q][128 h + e] =
// sum_k softmax_k(q . k / sqrt(128)) v[k][e], over the image's keys (causal:
// keys k <= q).  Grid (query blocks of 128, heads, images); a wave takes 32
// queries and walks the keys 32 at a time with an online softmax:
//   S^T = K Q^T on the matrix cores (v_mfma_f32_32x32x16_bf16: K as the row
//   operand, Q as the column operand), so lane l holds query q0 + l % 32 and
//   16 of the block's 32 keys (key 8 (r / 4) + 4 (l / 32) + r % 4 in register
//   r); a query's maximum and sum need its lane and the lane 32 away;
//   O^T += V^T P: the probabilities a lane holds are its half of the
//   operand's k slots as they stand (slot 8 (l / 32) + j is key 4 (l / 32) + j
//   for j < 4 and 8 + 4 (l / 32) + j - 4 for j >= 4, plus 16 for the second
//   16 keys), which is the order vt_kernel stores the values in.
// The workgroup's four waves share the keys and values: 64-key tiles of K
// (64 x 128) and V^T (128 x 64) pass through LDS, two tiles deep, the next
// tile loading straight into LDS while the current one is used.
// LDS rows are 16-byte chunks XOR-swizzled so that each 16-lane pass of a
// fragment read touches every bank once.
// Probabilities enter the products rounded to bfloat16; the running maximum
// rescales the partial sums in float32.
__global__ __launch_bounds__(64 * kAttnWaves) void attn_kernel(
    const uint16_t* __restrict__ QKV, const uint16_t* __restrict__ Vt, int d, int smax_pad,
    const int32_t* __restrict__ img_off, const int32_t* __restrict__ text_off, int max_seq,
    int64_t S_total, int causal, float c2, uint16_t* __restrict__ O, int32_t* err) {
  constexpr int kTileBytes = kKeyTile * kHead * 2;                 // one K or V^T tile, 16 KB
  __shared__ __attribute__((aligned(16))) char smem[2][2][kTileBytes];   // [buffer][K, V^T]
  const int b = blockIdx.z, hd = blockIdx.y, heads = gridDim.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int64_t so;
  int S;
  const bool report = tid == 0 && blockIdx.x == 0 && hd == 0;
  if (!sequence_of(img_off, text_off, b, max_seq, S_total, so, S, err, report)) return;
  const int qw = blockIdx.x * (kQPerWave * kAttnWaves);            // the workgroup's first query
  if (qw >= S) return;
  const int q0 = qw + wave * kQPerWave;                             // this wave's (may be past S)
  const int ql = lane & 31, half = lane >> 5;
  const int64_t ld = 3 * (int64_t)d;
  const uint16_t* Qb = QKV + so * ld + hd * kHead;
  const uint16_t* Kb = Qb + d;
  const uint16_t* Vb = Vt + ((int64_t)b * heads + hd) * kHead * (int64_t)smax_pad;
  const int q = q0 + ql;
  const int qr = q < S ? q : S - 1;           // queries past the sequence compute on its last row
  bf16x8_t qf[kHead / 16];
#pragma unroll
  for (int s = 0; s < kHead / 16; ++s) qf[s] = ld16(Qb + qr * ld + 16 * s + 8 * half);

  // keys the workgroup needs, and this wave's own limit
  const int kend_wg = causal ? (S < qw + kQPerWave * kAttnWaves ? S : qw + kQPerWave * kAttnWaves) : S;
  // (a wave past the sequence only helps load the tiles)
  const int kend = q0 >= S ? 0 : causal ? (S < q0 + kQPerWave ? S : q0 + kQPerWave) : S;
  const int tiles = (kend_wg + kKeyTile - 1) / kKeyTile;

  // Tile loads, straight into LDS: a load instruction fills 1 KB, 4 rows of
  // the K tile (row group w + 4 i of wave w) or 8 rows of the V^T tile; lane
  // i lands on chunk i % 16 (i % 8) of its row, so it fetches the logical
  // chunk that the swizzle puts there.  K rows past the sequence read its last
  // key (masked below); V^T keys past the sequence are zero in Vt up to
  // smax_pad.
  static_assert(kKeyTile * kHead * 2 / 1024 == 4 * kAttnWaves, "four row groups per wave");
  static_assert(kVtKeys % kKeyTile == 0, "V^T rows are padded to whole key tiles");
  auto issue_tile = [&](int kt, int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int grp = wave + kAttnWaves * i;
      const int r = 4 * grp + (lane >> 4), ch = (lane & 15) ^ (r & 15);
      const int k = kt * kKeyTile + r;
      lds_dma16(Kb + (int64_t)(k < S ? k : S - 1) * ld + 8 * ch, smem[buf][0] + grp * 1024);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int grp = wave + kAttnWaves * i;
      const int e = 8 * grp + (lane >> 3), ch = (lane & 7) ^ ((e >> 1) & 7);
      lds_dma16(Vb + (int64_t)e * smax_pad + kt * kKeyTile + 8 * ch, smem[buf][1] + grp * 1024);
    }
  };
  // fragment reads: K rows of key block kb (32 keys) in e-slice s; V^T rows of
  // e-tile t at the 16-key group g of the tile
  auto kfrag = [&](int buf, int r, int s) {
    const int ch = 2 * s + half;
    return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(smem[buf][0] + r * 256 + ((ch ^ (r & 15)) << 4)));
  };
  auto vfrag = [&](int buf, int e, int grp) {
    const int ch = 2 * grp + half;
    return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(smem[buf][1] + e * 128 + ((ch ^ ((e >> 1) & 7)) << 4)));
  };

  f32x16_t o[kHead / 32];
#pragma unroll
  for (int t = 0; t < kHead / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;

  issue_tile(0, 0);
  wait_vmcnt<0>();
  __syncthreads();
  for (int kt = 0; kt < tiles; ++kt) {
    const int buf = kt & 1;
    // the other buffer was last read before the previous barrier
    if (kt + 1 < tiles) issue_tile(kt + 1, buf ^ 1);
#pragma unroll
    for (int sb = 0; sb < kKeyTile / kKeyBlock; ++sb) {
      const int kb = kt * kKeyTile + sb * kKeyBlock;
      if (kb >= kend) break;                  // uniform in the wave
      f32x16_t st;
#pragma unroll
      for (int r = 0; r < 16; ++r) st[r] = 0.0f;
#pragma unroll
      for (int s = 0; s < kHead / 16; ++s)
        st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kfrag(buf, sb * kKeyBlock + ql, s), qf[s], st,
                                                     0, 0, 0);
      // Key kb is visible to every query of the wave (kb < S, and kb <= q0 when
      // causal), so the block maximum is finite.
      float x[16], bm = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb + 8 * (r >> 2) + 4 * half + (r & 3);
        const bool ok = key < S && (!causal || key <= q);
        x[r] = ok ? st[r] * c2 : -INFINITY;
        bm = fmaxf(bm, x[r]);
      }
      bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
      const float mn = fmaxf(m, bm);
      const float sc = __builtin_amdgcn_exp2f(m - mn);     // 0 on the first block
      float p[16], ls = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[r] = __builtin_amdgcn_exp2f(x[r] - mn);
        ls += p[r];
      }
      ls += __shfl_xor(ls, 32, 64);
      l = fmaf(l, sc, ls);
      m = mn;
#pragma unroll
      for (int t = 0; t < kHead / 32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] *= sc;
      const bf16x8_t pb0 = pack8(p), pb1 = pack8(p + 8);
#pragma unroll
      for (int t = 0; t < kHead / 32; ++t) {
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(buf, 32 * t + ql, 2 * sb), pb0, o[t], 0, 0, 0);
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(buf, 32 * t + ql, 2 * sb + 1), pb1, o[t], 0, 0, 0);
      }
    }
    wait_vmcnt<0>();                         // this wave's loads of the next tile
    __syncthreads();
  }
  if (q >= S) return;
  // O^T[e][q] in o[t][r]: e = 32 t + 8 (r / 4) + 4 (l / 32) + r % 4
  const float inv = 1.0f / l;
  uint16_t* orow = O + (so + q) * d + hd * kHead;
#pragma unroll
  for (int t = 0; t < kHead / 32; ++t)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const float v0 = o[t][4 * g4] * inv, v1 = o[t][4 * g4 + 1] * inv;
      const float v2 = o[t][4 * g4 + 2] * inv, v3 = o[t][4 * g4 + 3] * inv;
      uint2 w;
      w.x = (uint32_t)f32_to_bf16(v0) | ((uint32_t)f32_to_bf16(v1) << 16);
      w.y = (uint32_t)f32_to_bf16(v2) | ((uint32_t)f32_to_bf16(v3) << 16);
      *reinterpret_cast<uint2*>(orow + 32 * t + 8 * g4 + 4 * half) = w;
    }
}

}  // namespace

size_t encode_smax_pad(int max_seq) { return align_up((size_t)(max_seq > 0 ? max_seq : 1), kVtKeys); }

hipError_t launch_encode(const EncodeArgs& a, hipStream_t stream) {
  if (a.T_vis == 0) return hipSuccess;             // no visual rows: nothing to output
  const int d = a.d;
  const int64_t S = a.T_vis + a.T_txt;
  const int heads = d / kHead;
  const int smax_pad = (int)encode_smax_pad(a.max_seq);
  const unsigned row_blocks = (unsigned)((S + kRowWaves - 1) / kRowWaves);
  hipError_t e;
  // the sequences: visual rows, then the projected text rows
  if (a.T_txt > 0) {
    if ((e = launch_dense_bf16(a.E, a.W_p, a.T_txt, d, a.d_text, a.HID, stream)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(enc_text_kernel, dim3((unsigned)((a.T_txt + kRowWaves - 1) / kRowWaves)),
                       dim3(64 * kRowWaves), 0, stream, a.HID, a.T_txt, d, a.img_off, a.text_off,
                       a.B, S, a.g_text, a.R, a.err);
  }
  hipLaunchKernelGGL(enc_visual_kernel, dim3((unsigned)a.T_vis), dim3(256), 0, stream, a.X, d,
                     a.img_off, a.text_off, a.B, S, a.R, a.err);
  hipLaunchKernelGGL(enc_ln_kernel, dim3(row_blocks), dim3(64 * kRowWaves), 0, stream, a.R, S, d,
                     a.blk[0].ln1_g, a.blk[0].ln1_b, a.L);
  const float c2 = 1.4426950408889634f / sqrtf((float)kHead);
  const dim3 attn_grid((unsigned)((a.max_seq + kQPerWave * kAttnWaves - 1) / (kQPerWave * kAttnWaves)),
                       (unsigned)heads, (unsigned)a.B);
  const dim3 vt_grid((unsigned)(smax_pad / kVtKeys), (unsigned)heads, (unsigned)a.B);
  for (int k = 0; k < kEncoderBlocks; ++k) {
    const EncoderBlockArgs& p = a.blk[k];
    // q, k, v of LN1(R) (in L), biased in the product's epilogue
    if ((e = launch_dense_bf16(a.L, p.W_qkv, S, 3 * (int64_t)d, d, a.QKV, stream, p.b_qkv)) !=
        hipSuccess)
      return e;
    hipLaunchKernelGGL(vt_kernel, vt_grid, dim3(256), 0, stream, a.QKV, d, smax_pad, a.img_off,
                       a.text_off, a.max_seq, S, a.Vt, a.err);
    hipLaunchKernelGGL(attn_kernel, attn_grid, dim3(64 * kAttnWaves), 0, stream, a.QKV, a.Vt, d,
                       smax_pad, a.img_off, a.text_off, a.max_seq, S, a.causal ? 1 : 0, c2, a.A,
                       a.err);
    // R += A W_o^T + b_o; LN2 into A
    if ((e = launch_dense_bf16(a.A, p.W_o, S, d, d, a.L, stream)) != hipSuccess) return e;
    if ((e = launch_resid_ln(a.R, a.L, p.b_o, S, d, p.ln2_g, p.ln2_b, a.A, stream)) != hipSuccess)
      return e;
    // the MLP
    if ((e = launch_dense_bf16(a.A, p.W_1, S, 4 * (int64_t)d, d, a.HID, stream, p.b_1, true)) !=
        hipSuccess)
      return e;
    if ((e = launch_dense_bf16(a.HID, p.W_2, S, d, 4 * d, a.L, stream)) != hipSuccess) return e;
    if (k + 1 < kEncoderBlocks) {
      // R += L + b_2, and the next block's LN1 into L (in place, row by row)
      if ((e = launch_resid_ln(a.R, a.L, p.b_2, S, d, a.blk[k + 1].ln1_g, a.blk[k + 1].ln1_b, a.L,
                               stream)) != hipSuccess)
        return e;
    } else {
      hipLaunchKernelGGL(enc_out_kernel, dim3((unsigned)a.T_vis), dim3(256), 0, stream, a.R, a.L,
                         p.b_2, d, a.img_off, a.text_off, a.B, S, a.H, a.err);
    }
  }
  return hipGetLastError();
}

}  // namespace sp
