/*
 * Host-validation driver for the sanitizer build of the C ABI
 * (tests/test_asan_host.py): every entry point is called with arguments its
 * host-side validation refuses, so nothing reaches the device, and each
 * returned status is checked.  The ABI source is compiled with AddressSanitizer
 * and UndefinedBehaviorSanitizer on the host, so an out-of-bounds read, an
 * overflow or a misaligned access in the validation code stops the program.
 * Pointers are fake (never dereferenced); the stream is 0.
 */
#include <stdint.h>
#include <stdio.h>

#include "stepprune.h"

#define FAKE ((void*)0x10000)
#define FAKE_OUT ((void*)0x110000)
#define MISALIGNED ((void*)0x10008)

static int failures = 0;

static void expect(const char* what, sp_status got, sp_status want) {
  if (got != want) {
    printf("FAIL %s: got %d (%s), want %d\n", what, (int)got, stepprune_status_string(got), (int)want);
    ++failures;
  }
}

static sp_status project(sp_dims d, const void* X, int32_t B, float ln_eps, size_t ws_bytes) {
  return stepprune_project(&d, X, 10, FAKE, FAKE, FAKE, FAKE, (const int32_t*)FAKE, B, 4, FAKE,
                           1.0f, ln_eps, FAKE, (float*)FAKE, FAKE, ws_bytes, NULL, 0);
}

static sp_status select_(sp_dims d, int32_t g, int32_t max_group, uint32_t flags, float b_stop) {
  return stepprune_select(&d, FAKE, (const float*)FAKE, 10, (const int32_t*)FAKE, 1,
                          (const int32_t*)FAKE, (const int32_t*)FAKE, (const int32_t*)FAKE, 1,
                          max_group, 4, (const int32_t*)FAKE, b_stop, g, flags, (int32_t*)FAKE,
                          (int32_t*)FAKE, NULL, NULL, 0, FAKE, 0, NULL, 0);
}

static sp_status noalloc(sp_dims d, int32_t G, int32_t max_group, void* err) {
  return stepprune_select_noalloc(&d, FAKE, (const float*)FAKE, 9000, (const int32_t*)FAKE, 1,
                                  (const int32_t*)FAKE, (const int32_t*)FAKE, (const int32_t*)FAKE,
                                  G, max_group, 8, (const int32_t*)FAKE, 0.0f, 1, 0, (int32_t*)FAKE,
                                  (int32_t*)FAKE, NULL, NULL, 0, (int32_t*)err, NULL, 0);
}

static sp_status compact(sp_dims d, int32_t layout, int32_t rows_per_image, void* out) {
  return stepprune_compact(&d, FAKE, (const int32_t*)FAKE, FAKE, (const int32_t*)FAKE,
                           (const int32_t*)FAKE, (const int32_t*)FAKE, (const int32_t*)FAKE, 2,
                           layout, rows_per_image, 16, out, (int32_t*)FAKE, FAKE, 0, NULL, 0);
}

static sp_status encode(sp_dims d, const sp_encoder_block* blocks, int32_t max_seq, uint32_t flags,
                        size_t ws_bytes) {
  return stepprune_encode(&d, FAKE, 10, (const int32_t*)FAKE, 1, FAKE, (const int32_t*)FAKE, 4,
                          FAKE, 1.0f, blocks, max_seq, flags, FAKE_OUT, FAKE, ws_bytes, NULL, 0);
}

int main(void) {
  const sp_dims bf = {256, 256, 128, SP_BF16};
  sp_dims d;
  for (int s = SP_OK; s <= SP_EDEVICE; ++s) (void)stepprune_status_string((sp_status)s);
  (void)stepprune_status_string((sp_status)99);

  /* workspace sizes, every stage and invalid ones */
  if (stepprune_workspace_bytes(1, &bf, 100, 10, 2, 3, 50, 10) == 0) { puts("FAIL ws 1"); ++failures; }
  if (stepprune_workspace_bytes(1, &bf, 100, 10, 2, 3, 5000, 10) != 0) { puts("FAIL ws big"); ++failures; }
  if (stepprune_workspace_bytes(9, &bf, 100, 10, 2, 3, 50, 10) != 0) { puts("FAIL ws 9"); ++failures; }
  if (stepprune_workspace_bytes(1, NULL, 100, 10, 2, 3, 50, 10) != 0) { puts("FAIL ws null"); ++failures; }
  for (int which = 0; which <= 4; ++which) (void)stepprune_workspace_bytes(which, &bf, 1000, 64, 4, 4, 300, 64);

  /* project */
  d = bf; d.h = 96; expect("project h % 64", project(d, FAKE, 1, 1e-5f, 0), SP_EINVAL);
  d = bf; d.dtype = 7; expect("project dtype", project(d, FAKE, 1, 1e-5f, 0), SP_EUNSUPPORTED);
  d = bf; d.dtype = SP_F32; d.h = 576; expect("project f32 h", project(d, FAKE, 1, 1e-5f, 0), SP_EUNSUPPORTED);
  expect("project X null", project(bf, NULL, 1, 1e-5f, 0), SP_EINVAL);
  expect("project B 0", project(bf, FAKE, 0, 1e-5f, 0), SP_EINVAL);
  expect("project eps", project(bf, FAKE, 1, -1.0f, 0), SP_EINVAL);
  expect("project misaligned", project(bf, MISALIGNED, 1, 1e-5f, 0), SP_EINVAL);
  expect("project ws", project(bf, FAKE, 1, 1e-5f, 0), SP_EWORKSPACE);
  expect("project dims null", stepprune_project(NULL, NULL, 0, NULL, NULL, NULL, NULL, NULL, 1, 0,
                                                NULL, 1.0f, 1e-5f, NULL, NULL, NULL, 0, NULL, 0),
         SP_EINVAL);

  /* select and its variants */
  expect("select g 0", select_(bf, 0, 10, 0, 0.0f), SP_EINVAL);
  expect("select g 6", select_(bf, 6, 10, 0, 0.0f), SP_EUNSUPPORTED);
  expect("select group", select_(bf, 1, 1023, 0, 0.0f), SP_EUNSUPPORTED);
  expect("select flags", select_(bf, 1, 10, 64, 0.0f), SP_EINVAL);
  expect("select logits without trace", select_(bf, 1, 10, SP_LOGITS, 0.0f), SP_EINVAL);
  expect("select two phases", select_(bf, 1, 10, SP_GRAM_ONLY | SP_REUSE_GRAM, 0.0f), SP_EINVAL);
  expect("select nan", select_(bf, 1, 10, 0, 0.0f / 0.0f), SP_EINVAL);
  expect("select ws", select_(bf, 1, 10, 0, 0.0f), SP_EWORKSPACE);
  expect("noalloc err", noalloc(bf, 1, 10, NULL), SP_EINVAL);
  expect("noalloc misaligned err", noalloc(bf, 1, 10, (char*)FAKE + 2), SP_EINVAL);
  expect("noalloc beyond scratch", noalloc(bf, 9, 1000, FAKE), SP_EWORKSPACE);
  {
    sp_trajectory tj = {0.0f, 0.9f, (float*)FAKE, (float*)FAKE, NULL, 0};
    expect("trajectory tau", stepprune_select_trajectory(
        &bf, FAKE, (const float*)FAKE, 10, (const int32_t*)FAKE, 1, (const int32_t*)FAKE,
        (const int32_t*)FAKE, (const int32_t*)FAKE, 1, 10, 4, (const int32_t*)FAKE, 0.0f, 1, 0,
        (int32_t*)FAKE, (int32_t*)FAKE, NULL, NULL, 0, &tj, FAKE, 0, NULL, 0), SP_EINVAL);
    tj.tau = 1.0f;
    expect("trajectory ws", stepprune_select_trajectory(
        &bf, FAKE, (const float*)FAKE, 10, (const int32_t*)FAKE, 1, (const int32_t*)FAKE,
        (const int32_t*)FAKE, (const int32_t*)FAKE, 1, 10, 4, (const int32_t*)FAKE, 0.0f, 1, 0,
        (int32_t*)FAKE, (int32_t*)FAKE, NULL, NULL, 0, &tj, FAKE, 0, NULL, 0), SP_EWORKSPACE);
  }

  /* compact */
  d = bf; d.d_text = 128; expect("compact d_text", compact(d, SP_LAYOUT_PADDED, 8, FAKE_OUT), SP_EUNSUPPORTED);
  expect("compact layout", compact(bf, 7, 8, FAKE_OUT), SP_EINVAL);
  expect("compact rows", compact(bf, SP_LAYOUT_PADDED, 9, FAKE_OUT), SP_EINVAL);
  expect("compact out", compact(bf, SP_LAYOUT_PADDED, 8, MISALIGNED), SP_EINVAL);
  expect("compact ws", compact(bf, SP_LAYOUT_PADDED, 8, FAKE_OUT), SP_EWORKSPACE);

  /* encode */
  {
    sp_encoder_block blocks[2];
    const void** f = (const void**)blocks;
    for (size_t i = 0; i < sizeof(blocks) / sizeof(void*); ++i) f[i] = FAKE;
    expect("encode ws", encode(bf, blocks, 64, 0, 0), SP_EWORKSPACE);
    d = bf; d.d = 320; expect("encode heads", encode(d, blocks, 64, 0, 0), SP_EUNSUPPORTED);
    expect("encode max_seq", encode(bf, blocks, 0, 0, 0), SP_EINVAL);
    expect("encode flags", encode(bf, blocks, 64, 2, 0), SP_EINVAL);
    expect("encode blocks", encode(bf, NULL, 64, 0, 0), SP_EINVAL);
    f[sizeof(blocks) / sizeof(void*) - 1] = NULL;
    expect("encode null b_2", encode(bf, blocks, 64, 0, 0), SP_EINVAL);
  }

  /* gate and denoiser */
  {
    sp_denoiser p;
    const void** f = (const void**)&p;
    for (size_t i = 0; i < sizeof(p) / sizeof(void*); ++i) f[i] = FAKE;
    d = bf; d.dtype = SP_F32;
    expect("denoise dtype", stepprune_gate_denoise(&d, FAKE, 10, (const float*)FAKE, FAKE, &p,
                                                   FAKE_OUT, FAKE, 0, NULL, 0), SP_EUNSUPPORTED);
    expect("denoise alias", stepprune_gate_denoise(&bf, FAKE, 10, (const float*)FAKE, FAKE, &p,
                                                   FAKE, FAKE, 0, NULL, 0), SP_EINVAL);
    expect("denoise ws", stepprune_gate_denoise(&bf, FAKE, 10, (const float*)FAKE, FAKE, &p,
                                                FAKE_OUT, FAKE, 0, NULL, 0), SP_EWORKSPACE);
  }

  {
    int32_t code = 0;
    expect("read error null", stepprune_read_device_error(NULL, 0, &code), SP_EINVAL);
  }
  printf("%s: %d failure(s)\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
