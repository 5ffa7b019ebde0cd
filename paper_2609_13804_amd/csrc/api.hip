// C ABI of libstepprune (include/stepprune.h): host-side validation, workspace
// layout and launch order.  Every entry point validates its arguments before
// touching the device and never throws.
#include <string.h>

#include <mutex>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "sp_internal.h"

using namespace sp;

namespace {

// A roctx range named after the entry point around each call (host-side
// enqueue), so a marker trace shows the three stages of Algorithm 1.
struct TraceRange {
  explicit TraceRange(const char* name) { roctxRangePushA(name); }
  ~TraceRange() { roctxRangePop(); }
  TraceRange(const TraceRange&) = delete;
  TraceRange& operator=(const TraceRange&) = delete;
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

sp_status check_dims(const sp_dims* d) {
  if (!d) return SP_EINVAL;
  if (d->d <= 0 || d->d_text <= 0 || d->h <= 0) return SP_EINVAL;
  if (d->d % 64 || d->d_text % 64 || d->h % 64) return SP_EINVAL;
  if (d->dtype != SP_F32 && d->dtype != SP_BF16) return SP_EUNSUPPORTED;
  if (d->h > 1024) return SP_EUNSUPPORTED;
  if (d->dtype == SP_F32 && d->h > 512) return SP_EUNSUPPORTED;
  return SP_OK;
}

int elem_bytes(const sp_dims* d) { return d->dtype == SP_F32 ? 4 : 2; }

struct SelectWs {
  size_t gram, csplit, kept, count, total;
  int64_t gstride;
  int gram_ld;
};

// Header; Gram blocks [G][2 (max_group + 1) + 3][ld] float32; context split
// [B][3][h] in the working dtype; group-local kept lists; group counts.
SelectWs select_ws_layout(const sp_dims* d, int B, int G, int max_group, int max_cap) {
  SelectWs w;
  w.gram_ld = (int)align_up((size_t)max_group + 2, 4);
  w.gstride = (int64_t)(2 * (max_group + 1) + kGramExtraRows) * w.gram_ld;
  size_t off = kWsHeaderBytes;
  w.gram = off;
  off = align_up(off + (size_t)G * w.gstride * 4, 256);
  w.csplit = off;
  off = align_up(off + (size_t)B * kGramExtraRows * d->h * elem_bytes(d), 256);
  w.kept = off;
  off = align_up(off + (size_t)G * (max_cap > 0 ? max_cap : 1) * 4, 256);
  w.count = off;
  off = align_up(off + (size_t)G * 4, 256);
  w.total = off;
  return w;
}

// Header, then the text projection's K-split partial products [split][T_txt][h].
size_t project_ws_bytes(const sp_dims* d, int64_t T_txt) {
  const size_t split = (size_t)text_split(d->dtype, T_txt, d->h, d->d_text);
  return kWsHeaderBytes + align_up(split * (size_t)T_txt * d->h * 4, 256);
}

sp_status hip_status(hipError_t e) { return e == hipSuccess ? SP_OK : SP_EHIP; }

// Header, then the gate and denoiser's intermediates: x~ / h float32 [T, d],
// two bfloat16 [T, d] buffers and the bfloat16 [T, 4d] hidden activations.
struct GateWs {
  size_t xt, p, q, hid, total;
};
GateWs gate_ws_layout(const sp_dims* d, int64_t T) {
  GateWs w;
  const size_t td = (size_t)T * d->d;
  w.xt = kWsHeaderBytes;
  w.p = align_up(w.xt + td * 4, 256);
  w.q = align_up(w.p + td * 2, 256);
  w.hid = align_up(w.q + td * 2, 256);
  w.total = align_up(w.hid + td * 4 * 2, 256);
  return w;
}

// Header, then the encoder's buffers (sp_internal.h, EncodeArgs).
struct EncodeWs {
  size_t R, L, A, QKV, HID, Vt, total;
};
EncodeWs encode_ws_layout(const sp_dims* d, int64_t T_vis, int64_t T_txt, int B, int max_seq) {
  EncodeWs w;
  const size_t S = (size_t)(T_vis + T_txt), dd = (size_t)d->d;
  w.R = kWsHeaderBytes;
  w.L = align_up(w.R + S * dd * 4, 256);
  w.A = align_up(w.L + S * dd * 2, 256);
  w.QKV = align_up(w.A + S * dd * 2, 256);
  w.HID = align_up(w.QKV + S * dd * 3 * 2, 256);
  w.Vt = align_up(w.HID + S * dd * 4 * 2, 256);
  w.total = align_up(w.Vt + (size_t)B * dd * encode_smax_pad(max_seq) * 2, 256);
  return w;
}

// The encoder takes bfloat16, d a multiple of 128 (heads of width 128) up to
// 4096 (the row kernels keep a row in one wave's registers).
sp_status check_encode_dims(const sp_dims* d) {
  sp_status st = check_dims(d);
  if (st != SP_OK) return st;
  if (d->dtype != SP_BF16 || d->d % 128 || d->d > 4096) return SP_EUNSUPPORTED;
  return SP_OK;
}

}  // namespace

extern "C" {

const char* stepprune_status_string(sp_status s) {
  // A C caller may pass any int: read its bytes, since loading an enumeration
  // outside its enumerators' range is undefined in C++.
  static_assert(sizeof(sp_status) == sizeof(int32_t), "sp_status is int-sized");
  int32_t v;
  memcpy(&v, &s, sizeof(v));
  switch (v) {
    case SP_OK: return "ok";
    case SP_EINVAL: return "invalid argument";
    case SP_EUNSUPPORTED: return "unsupported argument";
    case SP_EWORKSPACE: return "workspace too small";
    case SP_EHIP: return "HIP runtime error";
    case SP_EDEVICE: return "device-side error (see stepprune_read_device_error)";
  }
  return "unknown status";
}

size_t stepprune_workspace_bytes(int32_t which, const sp_dims* dims, int64_t T_vis, int64_t T_txt,
                                 int32_t B, int32_t G, int32_t max_group, int32_t max_cap) {
  if (check_dims(dims) != SP_OK || T_vis < 0 || T_txt < 0 || B < 0 || G < 0) return 0;
  switch (which) {
    case 0: return project_ws_bytes(dims, T_txt);
    case 1:
      if (max_group < 0 || max_group > kMaxGroup || max_cap < 0) return 0;
      return select_ws_layout(dims, B, G, max_group, max_cap).total;
    case 2: return kWsHeaderBytes;
    case 3:
      if (dims->dtype != SP_BF16 || dims->d > 4096) return 0;
      return gate_ws_layout(dims, T_vis).total;
    case 4:
      if (check_encode_dims(dims) != SP_OK || B < 1 || max_group < 1) return 0;
      return encode_ws_layout(dims, T_vis, T_txt, B, max_group).total;
  }
  return 0;
}

sp_status stepprune_project(const sp_dims* dims, const void* X, int64_t T_vis, const void* s_start,
                            const void* s_stop, const void* W_kqv, const void* E_text,
                            const int32_t* text_off, int32_t B, int64_t T_txt, const void* W_text,
                            float g_text, float ln_eps, void* KQV, float* ctx, void* ws,
                            size_t ws_bytes, const hipEvent_t* events, hipStream_t stream) {
  const TraceRange range("stepprune_project");
  sp_status st = check_dims(dims);
  if (st != SP_OK) return st;
  if (T_vis < 0 || T_txt < 0 || B < 1) return SP_EINVAL;
  if (!s_start || !s_stop || !W_kqv || !KQV || !ctx || !text_off || !W_text || !ws) return SP_EINVAL;
  if ((T_vis > 0 && !X) || (T_txt > 0 && !E_text)) return SP_EINVAL;
  if (!aligned16(X) || !aligned16(s_start) || !aligned16(s_stop) || !aligned16(W_kqv) ||
      !aligned16(E_text) || !aligned16(W_text) || !aligned16(KQV) || !aligned16(ctx) ||
      !aligned16(ws))
    return SP_EINVAL;
  if (!(ln_eps >= 0.0f)) return SP_EINVAL;
  if (ws_bytes < project_ws_bytes(dims, T_txt)) return SP_EWORKSPACE;

  int32_t* err = reinterpret_cast<int32_t*>(ws);
  float* tproj = reinterpret_cast<float*>(static_cast<char*>(ws) + kWsHeaderBytes);
  record_event(events, 0, stream);
  hipError_t e = launch_project_gemm(dims->dtype, X, T_vis, s_start, s_stop, W_kqv, dims->d,
                                     3 * dims->h, KQV, E_text, T_txt, W_text, dims->d_text,
                                     dims->h, tproj, stream);
  record_event(events, 1, stream);
  if (e == hipSuccess)
    e = launch_text_pool(tproj, text_split(dims->dtype, T_txt, dims->h, dims->d_text), text_off, B,
                         T_txt, dims->h, g_text, ln_eps, ctx, err, stream);
  return hip_status(e);
}

}  // extern "C"

namespace {

// ------------------------------------------------------------ fixed scratch
// The scratch of stepprune_select_noalloc: one array in device memory, a copy
// per GPU, held until the process ends.  In host code the array's name is a
// stand-in, not a device address: host code uses only the address that
// hipGetSymbolAddress returns for the current device, fetched once per device
// and kept in scratch_ptr.
static __device__ __align__(256) char scratch[STEPPRUNE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices];

// The scratch address on the device that owns `stream` (it must be the
// current device: the symbol is looked up with that device current).
sp_status device_scratch(hipStream_t stream, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SP_EHIP;
  if (stream) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return SP_EHIP;
    if (sdev != dev) return SP_EINVAL;
  }
  if (dev < 0 || dev >= kMaxDevices) return SP_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SP_EHIP;
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return SP_OK;
}

// Shared body of stepprune_select, stepprune_select_trajectory (traj may be
// null for the others) and stepprune_select_noalloc (use_scratch: the
// workspace is the device's fixed scratch and the error word is err_word).
sp_status select_impl(const sp_dims* dims, const void* KQV, const float* ctx, int64_t T_vis,
                      const int32_t* img_off, int32_t B, const int32_t* grp_off,
                      const int32_t* grp_img, const int32_t* grp_cap, int32_t G,
                      int32_t max_group, int32_t max_cap, const int32_t* kept_off, float b_stop,
                      int32_t g, uint32_t flags, int32_t* kept_idx, int32_t* kept_cnt,
                      int32_t* grp_cnt, float* trace, int32_t trace_steps,
                      const sp_trajectory* traj, void* ws, size_t ws_bytes,
                      const hipEvent_t* events, hipStream_t stream,
                      bool use_scratch = false, int32_t* err_word = nullptr) {
  sp_status st = check_dims(dims);
  if (st != SP_OK) return st;
  if (T_vis < 0 || B < 1 || G < 0 || max_group < 0 || max_cap < 0 || trace_steps < 0)
    return SP_EINVAL;
  if (g < 1) return SP_EINVAL;
  if (g > kGMax) return SP_EUNSUPPORTED;
  if (max_group > kMaxGroup) return SP_EUNSUPPORTED;
  if (flags & ~(uint32_t)(SP_TRACE | SP_NO_HISTORY | SP_FULL_ROLLOUT | SP_GRAM_ONLY | SP_REUSE_GRAM |
                          SP_LOGITS))
    return SP_EINVAL;
  if ((flags & SP_LOGITS) && !(flags & SP_TRACE)) return SP_EINVAL;
  if ((flags & SP_GRAM_ONLY) && (flags & SP_REUSE_GRAM)) return SP_EINVAL;
  if ((flags & SP_GRAM_ONLY) && traj) return SP_EINVAL;
  if (!KQV || !ctx || !img_off || !kept_off || !kept_cnt) return SP_EINVAL;
  if (use_scratch ? !err_word || (reinterpret_cast<uintptr_t>(err_word) & 3u) : !ws)
    return SP_EINVAL;
  if (G > 0 && (!grp_off || !grp_img || !grp_cap || !kept_idx)) return SP_EINVAL;
  if ((flags & SP_TRACE) && trace_steps > 0 && !trace) return SP_EINVAL;
  if (b_stop != b_stop) return SP_EINVAL;   // NaN
  if (traj) {
    if (!(traj->tau > 0.0f) || !(traj->beta > 0.0f && traj->beta <= 1.0f)) return SP_EINVAL;
    if (traj->pstop_steps < 0 || (traj->pstop_steps > 0 && !traj->pstop)) return SP_EINVAL;
    if ((G > 0 && !traj->kbar) || (T_vis > 0 && !traj->s)) return SP_EINVAL;
    if (g != 1) return SP_EUNSUPPORTED;
  }
  if (!aligned16(KQV) || !aligned16(ctx) || (!use_scratch && !aligned16(ws))) return SP_EINVAL;
  const SelectWs lay = select_ws_layout(dims, B, G, max_group, max_cap);
  if (use_scratch) {
    if (lay.total > (size_t)STEPPRUNE_NOALLOC_SCRATCH_BYTES) return SP_EWORKSPACE;
    const sp_status sst = device_scratch(stream, &ws);
    if (sst != SP_OK) return sst;
    ws_bytes = STEPPRUNE_NOALLOC_SCRATCH_BYTES;
  }
  if (ws_bytes < lay.total) return SP_EWORKSPACE;

  char* wsb = static_cast<char*>(ws);
  SelectArgs a;
  a.dtype = dims->dtype;
  a.KQV = KQV;
  a.ctx = ctx;
  a.T_vis = T_vis;
  a.h = dims->h;
  a.img_off = img_off;
  a.B = B;
  a.grp_off = grp_off;
  a.grp_img = grp_img;
  a.grp_cap = grp_cap;
  a.G = G;
  a.max_group = max_group;
  a.max_cap = max_cap > 0 ? max_cap : 1;
  a.kept_off = kept_off;
  a.b_stop = b_stop;
  a.g = g;
  a.flags = flags;
  a.kept_idx = kept_idx;
  a.kept_cnt = kept_cnt;
  a.grp_cnt = grp_cnt;
  a.trace = trace;
  a.trace_steps = trace_steps;
  a.traj_tau = traj ? traj->tau : 0.0f;
  a.traj_beta = traj ? traj->beta : 0.0f;
  a.traj_s = traj ? traj->s : nullptr;
  a.traj_kbar = traj ? traj->kbar : nullptr;
  a.traj_pstop = traj && traj->pstop_steps > 0 ? traj->pstop : nullptr;
  a.traj_pstop_steps = traj && traj->pstop ? traj->pstop_steps : 0;
  a.gram = reinterpret_cast<float*>(wsb + lay.gram);
  a.gram_group_stride = lay.gstride;
  a.gram_ld = lay.gram_ld;
  a.csplit = wsb + lay.csplit;
  a.grp_kept = reinterpret_cast<int32_t*>(wsb + lay.kept);
  a.grp_count = reinterpret_cast<int32_t*>(wsb + lay.count);
  a.err = use_scratch ? err_word : reinterpret_cast<int32_t*>(wsb);
  a.events = events;
  return hip_status(launch_select(a, stream));
}

}  // namespace

extern "C" {

sp_status stepprune_select(const sp_dims* dims, const void* KQV, const float* ctx, int64_t T_vis,
                           const int32_t* img_off, int32_t B, const int32_t* grp_off,
                           const int32_t* grp_img, const int32_t* grp_cap, int32_t G,
                           int32_t max_group, int32_t max_cap, const int32_t* kept_off,
                           float b_stop, int32_t g, uint32_t flags, int32_t* kept_idx,
                           int32_t* kept_cnt, int32_t* grp_cnt, float* trace, int32_t trace_steps,
                           void* ws, size_t ws_bytes, const hipEvent_t* events,
                           hipStream_t stream) {
  const TraceRange range("stepprune_select");
  return select_impl(dims, KQV, ctx, T_vis, img_off, B, grp_off, grp_img, grp_cap, G, max_group,
                     max_cap, kept_off, b_stop, g, flags, kept_idx, kept_cnt, grp_cnt, trace,
                     trace_steps, nullptr, ws, ws_bytes, events, stream);
}

sp_status stepprune_select_trajectory(const sp_dims* dims, const void* KQV, const float* ctx,
                                      int64_t T_vis, const int32_t* img_off, int32_t B,
                                      const int32_t* grp_off, const int32_t* grp_img,
                                      const int32_t* grp_cap, int32_t G, int32_t max_group,
                                      int32_t max_cap, const int32_t* kept_off, float b_stop,
                                      int32_t g, uint32_t flags, int32_t* kept_idx,
                                      int32_t* kept_cnt, int32_t* grp_cnt, float* trace,
                                      int32_t trace_steps, const sp_trajectory* traj, void* ws,
                                      size_t ws_bytes, const hipEvent_t* events,
                                      hipStream_t stream) {
  const TraceRange range("stepprune_select_trajectory");
  if (!traj) return SP_EINVAL;
  return select_impl(dims, KQV, ctx, T_vis, img_off, B, grp_off, grp_img, grp_cap, G, max_group,
                     max_cap, kept_off, b_stop, g, flags, kept_idx, kept_cnt, grp_cnt, trace,
                     trace_steps, traj, ws, ws_bytes, events, stream);
}

sp_status stepprune_select_noalloc(const sp_dims* dims, const void* KQV, const float* ctx,
                                   int64_t T_vis, const int32_t* img_off, int32_t B,
                                   const int32_t* grp_off, const int32_t* grp_img,
                                   const int32_t* grp_cap, int32_t G, int32_t max_group,
                                   int32_t max_cap, const int32_t* kept_off, float b_stop,
                                   int32_t g, uint32_t flags, int32_t* kept_idx,
                                   int32_t* kept_cnt, int32_t* grp_cnt, float* trace,
                                   int32_t trace_steps, int32_t* err,
                                   const hipEvent_t* events, hipStream_t stream) {
  const TraceRange range("stepprune_select_noalloc");
  return select_impl(dims, KQV, ctx, T_vis, img_off, B, grp_off, grp_img, grp_cap, G, max_group,
                     max_cap, kept_off, b_stop, g, flags, kept_idx, kept_cnt, grp_cnt, trace,
                     trace_steps, nullptr, nullptr, 0, events, stream, true, err);
}

sp_status stepprune_compact(const sp_dims* dims, const void* X, const int32_t* img_off,
                            const void* E_text, const int32_t* text_off, const int32_t* kept_idx,
                            const int32_t* kept_off, const int32_t* kept_cnt, int32_t B,
                            int32_t layout, int32_t rows_per_image, int64_t out_rows, void* out,
                            int32_t* seq_info, void* ws, size_t ws_bytes,
                            const hipEvent_t* events, hipStream_t stream) {
  const TraceRange range("stepprune_compact");
  sp_status st = check_dims(dims);
  if (st != SP_OK) return st;
  if (dims->d_text != dims->d) return SP_EUNSUPPORTED;
  if (B < 1 || out_rows < 0) return SP_EINVAL;
  if (layout != SP_LAYOUT_PADDED && layout != SP_LAYOUT_PACKED) return SP_EINVAL;
  if (layout == SP_LAYOUT_PADDED && (rows_per_image < 0 || (int64_t)rows_per_image * B > out_rows))
    return SP_EINVAL;
  if (!X || !img_off || !E_text || !text_off || !kept_idx || !kept_off || !kept_cnt || !out ||
      !seq_info || !ws)
    return SP_EINVAL;
  if (!aligned16(X) || !aligned16(E_text) || !aligned16(out) || !aligned16(ws)) return SP_EINVAL;
  if (ws_bytes < kWsHeaderBytes) return SP_EWORKSPACE;
  CompactArgs a;
  a.elem_bytes = elem_bytes(dims);
  a.d = dims->d;
  a.X = X;
  a.img_off = img_off;
  a.E = E_text;
  a.text_off = text_off;
  a.kept_idx = kept_idx;
  a.kept_off = kept_off;
  a.kept_cnt = kept_cnt;
  a.B = B;
  a.layout = layout;
  a.rows_per_image = rows_per_image;
  a.out_rows = out_rows;
  a.out = out;
  a.seq_info = seq_info;
  a.err = reinterpret_cast<int32_t*>(ws);
  record_event(events, 0, stream);
  hipError_t e = launch_compact(a, stream);
  record_event(events, 1, stream);
  return hip_status(e);
}

sp_status stepprune_read_device_error(void* ws, hipStream_t stream, int32_t* code) {
  if (!ws || !code) return SP_EINVAL;
  if (hipStreamSynchronize(stream) != hipSuccess) return SP_EHIP;
  int32_t v = 0;
  if (hipMemcpy(&v, ws, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return SP_EHIP;
  *code = v;
  if (v != 0) {
    const int32_t zero = 0;
    if (hipMemcpy(ws, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess) return SP_EHIP;
    return SP_EDEVICE;
  }
  return SP_OK;
}

sp_status stepprune_encode(const sp_dims* dims, const void* X, int64_t T_vis,
                           const int32_t* img_off, int32_t B, const void* E_text,
                           const int32_t* text_off, int64_t T_txt, const void* W_p, float g_text,
                           const sp_encoder_block* blocks, int32_t max_seq, uint32_t flags,
                           void* H, void* ws, size_t ws_bytes, const hipEvent_t* events,
                           hipStream_t stream) {
  const TraceRange range("stepprune_encode");
  sp_status st = check_encode_dims(dims);
  if (st != SP_OK) return st;
  if (T_vis < 0 || T_txt < 0 || B < 1 || max_seq < 1 || !blocks) return SP_EINVAL;
  if (flags & ~(uint32_t)SP_ENC_CAUSAL) return SP_EINVAL;
  if (!img_off || !text_off || !W_p || !ws || (T_vis > 0 && (!X || !H)) || (T_txt > 0 && !E_text))
    return SP_EINVAL;
  if (!aligned16(X) || !aligned16(E_text) || !aligned16(W_p) || !aligned16(H) || !aligned16(ws))
    return SP_EINVAL;
  if (!(g_text == g_text)) return SP_EINVAL;   // NaN
  for (int k = 0; k < kEncoderBlocks; ++k) {
    const sp_encoder_block& p = blocks[k];
    const void* ptrs[] = {p.ln1_g, p.ln1_b, p.W_qkv, p.b_qkv, p.W_o, p.b_o,
                          p.ln2_g, p.ln2_b, p.W_1, p.b_1, p.W_2, p.b_2};
    for (const void* q : ptrs)
      if (!q || !aligned16(q)) return SP_EINVAL;
  }
  const EncodeWs w = encode_ws_layout(dims, T_vis, T_txt, B, max_seq);
  if (ws_bytes < w.total) return SP_EWORKSPACE;
  char* base = static_cast<char*>(ws);
  EncodeArgs a;
  a.d = dims->d;
  a.d_text = dims->d_text;
  a.T_vis = T_vis;
  a.T_txt = T_txt;
  a.B = B;
  a.max_seq = max_seq;
  a.causal = (flags & SP_ENC_CAUSAL) != 0;
  a.g_text = g_text;
  a.X = static_cast<const uint16_t*>(X);
  a.img_off = img_off;
  a.E = static_cast<const uint16_t*>(E_text);
  a.text_off = text_off;
  a.W_p = static_cast<const uint16_t*>(W_p);
  for (int k = 0; k < kEncoderBlocks; ++k) {
    const sp_encoder_block& p = blocks[k];
    EncoderBlockArgs& q = a.blk[k];
    q.ln1_g = p.ln1_g;
    q.ln1_b = p.ln1_b;
    q.W_qkv = static_cast<const uint16_t*>(p.W_qkv);
    q.b_qkv = p.b_qkv;
    q.W_o = static_cast<const uint16_t*>(p.W_o);
    q.b_o = p.b_o;
    q.ln2_g = p.ln2_g;
    q.ln2_b = p.ln2_b;
    q.W_1 = static_cast<const uint16_t*>(p.W_1);
    q.b_1 = p.b_1;
    q.W_2 = static_cast<const uint16_t*>(p.W_2);
    q.b_2 = p.b_2;
  }
  a.H = static_cast<uint16_t*>(H);
  a.R = reinterpret_cast<float*>(base + w.R);
  a.L = reinterpret_cast<uint16_t*>(base + w.L);
  a.A = reinterpret_cast<uint16_t*>(base + w.A);
  a.QKV = reinterpret_cast<uint16_t*>(base + w.QKV);
  a.HID = reinterpret_cast<uint16_t*>(base + w.HID);
  a.Vt = reinterpret_cast<uint16_t*>(base + w.Vt);
  a.err = reinterpret_cast<int32_t*>(base);
  record_event(events, 0, stream);
  const hipError_t e = launch_encode(a, stream);
  record_event(events, 1, stream);
  return hip_status(e);
}

sp_status stepprune_gate_denoise(const sp_dims* dims, const void* X, int64_t T,
                                 const float* alpha, const void* eps, const sp_denoiser* p,
                                 void* out, void* ws, size_t ws_bytes,
                                 const hipEvent_t* events, hipStream_t stream) {
  const TraceRange range("stepprune_gate_denoise");
  sp_status st = check_dims(dims);
  if (st != SP_OK) return st;
  if (dims->dtype != SP_BF16 || dims->d > 4096) return SP_EUNSUPPORTED;
  if (T < 0 || !p || !out || !ws) return SP_EINVAL;
  if (T > 0 && (!X || !alpha || !eps)) return SP_EINVAL;
  if (!p->ln1_g || !p->ln1_b || !p->W_v || !p->b_v || !p->W_o || !p->b_o || !p->ln2_g ||
      !p->ln2_b || !p->W_1 || !p->b_1 || !p->W_2 || !p->b_2)
    return SP_EINVAL;
  if (!aligned16(X) || !aligned16(eps) || !aligned16(out) || !aligned16(ws) ||
      !aligned16(p->W_v) || !aligned16(p->W_o) || !aligned16(p->W_1) || !aligned16(p->W_2) ||
      !aligned16(p->ln1_g) || !aligned16(p->ln1_b) || !aligned16(p->b_v) || !aligned16(p->b_o) ||
      !aligned16(p->ln2_g) || !aligned16(p->ln2_b) || !aligned16(p->b_1) || !aligned16(p->b_2))
    return SP_EINVAL;
  if (out == X || out == eps) return SP_EINVAL;
  const GateWs w = gate_ws_layout(dims, T);
  if (ws_bytes < w.total) return SP_EWORKSPACE;
  char* base = static_cast<char*>(ws);
  DenoiseArgs a;
  a.T = T;
  a.d = dims->d;
  a.X = static_cast<const uint16_t*>(X);
  a.alpha = alpha;
  a.eps = static_cast<const uint16_t*>(eps);
  a.ln1_g = p->ln1_g;
  a.ln1_b = p->ln1_b;
  a.W_v = static_cast<const uint16_t*>(p->W_v);
  a.b_v = p->b_v;
  a.W_o = static_cast<const uint16_t*>(p->W_o);
  a.b_o = p->b_o;
  a.ln2_g = p->ln2_g;
  a.ln2_b = p->ln2_b;
  a.W_1 = static_cast<const uint16_t*>(p->W_1);
  a.b_1 = p->b_1;
  a.W_2 = static_cast<const uint16_t*>(p->W_2);
  a.b_2 = p->b_2;
  a.out = static_cast<uint16_t*>(out);
  a.xt = reinterpret_cast<float*>(base + w.xt);
  a.buf_p = reinterpret_cast<uint16_t*>(base + w.p);
  a.buf_q = reinterpret_cast<uint16_t*>(base + w.q);
  a.hid = reinterpret_cast<uint16_t*>(base + w.hid);
  record_event(events, 0, stream);
  const hipError_t e = launch_gate_denoise(a, stream);
  record_event(events, 1, stream);
  return hip_status(e);
}

}  // extern "C"
