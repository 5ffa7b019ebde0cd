// Internal declarations shared by the HIP translation units of libstepprune.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>
#include <stddef.h>
#include <limits.h>
#include <math.h>

#include "stepprune.h"

namespace sp {

// Workspace header: the first 256 bytes of every workspace.
struct WsHeader {
  int32_t error;       // SP_DEV_* code, first error wins (atomicCAS from 0)
  int32_t pad[63];
};
constexpr size_t kWsHeaderBytes = 256;

constexpr int kMaxGroup = 1022;        // largest group the selection kernel takes
constexpr int kLdsBytes = 160 * 1024;  // LDS per workgroup on gfx950

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Records events[i] on the stream when the caller supplied it.
inline void record_event(const hipEvent_t* events, int i, hipStream_t stream) {
  if (events && events[i]) (void)hipEventRecord(events[i], stream);
}

// The first error wins and stays until stepprune_read_device_error clears it.
__device__ inline void set_device_error(int32_t* err, int32_t code) {
  atomicCAS(err, 0, code);
}

// ---------------------------------------------------------------- GEMM launchers
// C[m, n] = sum_k A[m, k] * B[n, k]  (both operands K-contiguous), fp32 accumulate.

// Projection: A rows are X rows 0..T_vis-1, then s_start, then s_stop; and
// the text projection: A = E_text [T_txt, d_text], B = W_text [h, d_text],
// float32 output split over K into text_split() partial products
// [split][T_txt][h], which launch_text_pool adds in a fixed order.  For
// bfloat16 both products run in one launch (the text tiles fill the compute
// units the projection's last round leaves idle) and the text product is not
// split.
int text_split(int dtype, int64_t T_txt, int h, int d_text);
hipError_t launch_project_gemm(int dtype, const void* X, int64_t T_vis, const void* s_start,
                               const void* s_stop, const void* W, int d, int n_out, void* out,
                               const void* E, int64_t T_txt, const void* W_text, int d_text, int h,
                               float* tproj, hipStream_t stream);
// Per-group Gram products of the projected rows (see select.hip for the
// layout).  The text context of each image is first written as three rows of
// the working dtype whose sum is exactly the float32 context (csplit,
// [B][3][h]); they are the last three A-side rows of every group, so the
// matrix cores also produce the three parts of cK = c [K; k_stop]^T.
struct GramArgs {
  int dtype;
  const void* KQV;
  int64_t T_vis;
  int h;
  const float* ctx;
  int B;
  const int32_t* grp_off;
  const int32_t* grp_img;
  int G;
  int max_group;
  void* csplit;
  float* gram;
  int64_t gram_group_stride;
  int gram_ld;
  int32_t* err;
};
constexpr int kGramExtraRows = 3;      // A-side rows of the context split
hipError_t launch_gram_gemm(const GramArgs& a, hipStream_t stream);

// ---------------------------------------------------------------- other launchers
// LayerNorm of every projected text row (in place over partial product 0)
// and the per-image mean with gain: ctx[b] = g_text * mean_l LN(T_l).
hipError_t launch_text_pool(float* T, int split, const int32_t* text_off, int B, int64_t T_txt,
                            int h, float g_text, float ln_eps, float* ctx, int32_t* err,
                            hipStream_t stream);

// Largest number of tokens kept per round (Eq. 11's group size g; the paper's
// high-resolution setting uses 5).
constexpr int kGMax = 5;

struct SelectArgs {
  int dtype;
  const void* KQV;
  const float* ctx;
  int64_t T_vis;
  int h;
  const int32_t* img_off;
  int B;
  const int32_t* grp_off;
  const int32_t* grp_img;
  const int32_t* grp_cap;
  int G;
  int max_group;
  int max_cap;
  const int32_t* kept_off;
  float b_stop;
  int g;                 // tokens per round, 1..kGMax
  uint32_t flags;
  int32_t* kept_idx;
  int32_t* kept_cnt;
  int32_t* grp_cnt;
  float* trace;
  int trace_steps;
  // trajectory sums (Eqs. 5-7), all null / zero when not requested
  float traj_tau;
  float traj_beta;
  float* traj_s;         // [T_vis]
  float* traj_kbar;      // [G]
  float* traj_pstop;     // [G, traj_pstop_steps] or null
  int traj_pstop_steps;
  // workspace pieces
  float* gram;
  int64_t gram_group_stride;
  int gram_ld;
  void* csplit;          // [B][3][h] of the working dtype
  int32_t* grp_kept;     // [G, max_cap]
  int32_t* grp_count;    // [G]
  int32_t* err;
  const hipEvent_t* events;
};
hipError_t launch_select(const SelectArgs& a, hipStream_t stream);

struct CompactArgs {
  int elem_bytes;
  int d;
  const void* X;
  const int32_t* img_off;
  const void* E;
  const int32_t* text_off;
  const int32_t* kept_idx;
  const int32_t* kept_off;
  const int32_t* kept_cnt;
  int B;
  int layout;
  int rows_per_image;
  int64_t out_rows;
  void* out;
  int32_t* seq_info;
  int32_t* err;
};
hipError_t launch_compact(const CompactArgs& a, hipStream_t stream);

// C = A B^T for bfloat16 A [M, K] and B [N, K] (rows K-contiguous), bfloat16
// C [M, N]; K a multiple of 32.  With bias [N] (float32) each element is
// bf16(bf16(product) + bias), or bf16(GELU(bf16(product) + bias)) with gelu:
// what a separate bias (+ GELU) pass over the stored product gives.
hipError_t launch_dense_bf16(const void* A, const void* B, int64_t M, int64_t N, int K, void* C,
                             hipStream_t stream, const float* bias = nullptr, bool gelu = false);

// Noise gate and locally masked denoiser (denoise.hip).  Workspace buffers:
// xt float32 [T, d] (the residual stream), buf_p and buf_q bfloat16 [T, d],
// hid bfloat16 [T, 4d].
// LayerNorm eps of the transformer blocks (the denoiser's and the encoder's).
constexpr float kBlockLnEps = 1e-6f;
struct DenoiseArgs {
  int64_t T;
  int d;
  const uint16_t* X;
  const float* alpha;
  const uint16_t* eps;
  const float* ln1_g;
  const float* ln1_b;
  const uint16_t* W_v;
  const float* b_v;
  const uint16_t* W_o;
  const float* b_o;
  const float* ln2_g;
  const float* ln2_b;
  const uint16_t* W_1;
  const float* b_1;
  const uint16_t* W_2;
  const float* b_2;
  uint16_t* out;
  float* xt;
  uint16_t* buf_p;
  uint16_t* buf_q;
  uint16_t* hid;
};
hipError_t launch_gate_denoise(const DenoiseArgs& a, hipStream_t stream);

// Row kernel of denoise.hip, shared with the encoder: xt = (xt + t) + bias in
// place and z = LN(xt) (scale g, shift b) over rows of width d (d <= 4096).
hipError_t launch_resid_ln(float* xt, const uint16_t* t, const float* bias, int64_t T, int d,
                           const float* g, const float* b, uint16_t* z, hipStream_t stream);

// Cross-modal input encoder (encode.hip, Eq. 3): two pre-norm transformer
// blocks over every image's [X_b; g LN(E_b W_p^T)] sequence.  Weights are
// bfloat16 [out, in]; vectors float32.  Workspace buffers (rows of the
// S = T_vis + T_txt sequence rows): R float32 [S, d] (the residual stream),
// L and A bfloat16 [S, d], QKV bfloat16 [S, 3d], HID bfloat16 [S, 4d] (also the
// text product [T_txt, d]), Vt bfloat16 [B, d, encode_smax_pad(max_seq)].
constexpr int kEncoderBlocks = 2;
struct EncoderBlockArgs {
  const float* ln1_g;
  const float* ln1_b;
  const uint16_t* W_qkv;
  const float* b_qkv;
  const uint16_t* W_o;
  const float* b_o;
  const float* ln2_g;
  const float* ln2_b;
  const uint16_t* W_1;
  const float* b_1;
  const uint16_t* W_2;
  const float* b_2;
};
struct EncodeArgs {
  int d, d_text;
  int64_t T_vis, T_txt;
  int B;
  int max_seq;
  bool causal;
  float g_text;
  const uint16_t* X;
  const int32_t* img_off;
  const uint16_t* E;
  const int32_t* text_off;
  const uint16_t* W_p;
  EncoderBlockArgs blk[kEncoderBlocks];
  uint16_t* H;
  float* R;
  uint16_t* L;
  uint16_t* A;
  uint16_t* QKV;
  uint16_t* HID;
  uint16_t* Vt;
  int32_t* err;
};
// Keys per image row of Vt: max_seq rounded up to the transpose tile.
size_t encode_smax_pad(int max_seq);
hipError_t launch_encode(const EncodeArgs& a, hipStream_t stream);

}  // namespace sp
