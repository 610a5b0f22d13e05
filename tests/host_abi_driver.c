/* Drives the C ABI's host-side validation and error paths of a library
 * built with AddressSanitizer + UndefinedBehaviorSanitizer on its host code
 * (paper_2405_14105_amd/build.py, build_host_sanitized).  Needs no GPU:
 * every call either fails validation before touching the device or fails
 * on the first HIP call (no device), which exercises the clean-up paths.
 * Exits 0 when every status is the expected one. */
#include <stdio.h>
#include <string.h>

#include "dsi.h"

static int failures = 0;

static void expect(const char* what, dsi_status got, dsi_status want) {
  if (got != want) {
    printf("FAIL %s: status %d, expected %d (%s)\n", what, (int)got, (int)want, dsi_last_error());
    ++failures;
  }
}

static void expect_error(const char* what, dsi_status got) {
  if (got == DSI_OK) {
    printf("FAIL %s: succeeded without a device\n", what);
    ++failures;
  }
  const char* msg = dsi_last_error();
  if (!msg || !msg[0]) {
    printf("FAIL %s: no error message\n", what);
    ++failures;
  }
}

static dsi_config cfg(int layers, int d, int heads, int kv, int hd, int ff, int vocab) {
  dsi_config c;
  memset(&c, 0, sizeof c);
  c.n_layers = layers;
  c.d_model = d;
  c.n_heads = heads;
  c.n_kv_heads = kv;
  c.head_dim = hd;
  c.d_ff = ff;
  c.vocab = vocab;
  c.rope_base = 10000.f;
  c.rms_eps = 1e-5f;
  c.wdtype = DSI_BF16;
  c.kvdtype = DSI_BF16;
  return c;
}

int main(void) {
  dsi_model* m = NULL;
  dsi_kv* kv = NULL;
  int dummy[64];
  float fdummy[64];
  void* P = dummy;

  /* model creation: argument and shape validation */
  dsi_config c = cfg(2, 128, 4, 2, 32, 256, 1000);
  expect("create null cfg", dsi_model_create(NULL, NULL, &m), DSI_EINVAL);
  expect("create null out", dsi_model_create(&c, NULL, NULL), DSI_EINVAL);
  dsi_config bad = cfg(2, 100, 4, 2, 32, 256, 1000);
  expect("create d_model % 32", dsi_model_create(&bad, NULL, &m), DSI_EINVAL);
  bad = cfg(2, 128, 3, 2, 32, 256, 1000);
  expect("create heads % kv", dsi_model_create(&bad, NULL, &m), DSI_EINVAL);
  bad = cfg(2, 128, 4, 2, 48, 256, 1000);
  expect("create head_dim", dsi_model_create(&bad, NULL, &m), DSI_EINVAL);
  bad = cfg(0, 128, 4, 2, 32, 256, 1000);
  expect("create zero layers", dsi_model_create(&bad, NULL, &m), DSI_EINVAL);
  bad = cfg(2, 128, 4, 2, 32, 256, 0);
  expect("create zero vocab", dsi_model_create(&bad, NULL, &m), DSI_EINVAL);
  bad = cfg(2, 128, 4, 2, 32, 256, 1000);
  bad.wdtype = 7;
  expect("create bad dtype", dsi_model_create(&bad, NULL, &m), DSI_EINVAL);
  bad = cfg(2, 128, 4, 2, 32, 256, 1000);
  bad.rms_eps = -1.f;
  expect("create bad eps", dsi_model_create(&bad, NULL, &m), DSI_EINVAL);
  bad = cfg(2, 16384, 4, 2, 32, 256, 1000);
  expect("create d_model too large", dsi_model_create(&bad, NULL, &m), DSI_EINVAL);
  /* a valid shape: the allocation fails without a device, the partial
     model is released */
  expect_error("create valid shape without device", dsi_model_create(&c, NULL, &m));

  /* null handles */
  expect("destroy null model", dsi_model_destroy(NULL), DSI_OK);
  expect("destroy null kv", dsi_kv_destroy(NULL), DSI_OK);
  expect("set_tensor null", dsi_model_set_tensor(NULL, 0, DSI_T_WQ, P, 4, 0), DSI_EINVAL);
  expect("kv_create null", dsi_kv_create(NULL, 1, 16, &kv), DSI_EINVAL);
  expect("prefill null", dsi_prefill(NULL, NULL, 0, dummy, 1, NULL), DSI_EINVAL);
  dsi_verify_args va;
  memset(&va, 0, sizeof va);
  va.n_windows = 1;
  va.k = 3;
  va.d_tokens = dummy;
  va.temperature = 1.f;
  expect("verify null", dsi_verify(NULL, NULL, &va, dummy, dummy), DSI_EINVAL);
  expect("verify null args", dsi_verify(NULL, NULL, NULL, NULL, NULL), DSI_EINVAL);
  dsi_tree_args ta;
  memset(&ta, 0, sizeof ta);
  expect("tree null", dsi_verify_tree(NULL, NULL, &ta, dummy, dummy, dummy), DSI_EINVAL);
  expect("rollback null", dsi_kv_rollback(NULL, 0, 0), DSI_EINVAL);
  expect("poison null", dsi_kv_poison(NULL, 0), DSI_EINVAL);
  int32_t len = 0;
  expect("length null", dsi_kv_length(NULL, 0, &len), DSI_EINVAL);
  expect("sync null", dsi_sync(NULL), DSI_EINVAL);
  expect("export null", dsi_kv_export(NULL, 0, 0, 1, P, P), DSI_EINVAL);
  expect("import null", dsi_kv_import(NULL, 0, 0, 1, P, P), DSI_EINVAL);
  expect("set_length null", dsi_kv_set_length(NULL, 0, 1), DSI_EINVAL);
  expect("profile_begin null", dsi_profile_begin(NULL, DSI_K_QKV), DSI_EINVAL);
  int32_t launches = 0;
  double ms = 0.0;
  expect("profile_end null", dsi_profile_end(NULL, &launches, &ms), DSI_EINVAL);
  expect("profile_kernel null", dsi_profile_kernel(NULL, NULL, DSI_K_QKV, 1, &launches, &ms), DSI_EINVAL);
  uint64_t nb = 0;
  expect("profile_stream null buffer", dsi_profile_stream(NULL, 1 << 30, 1, 0, 0, 1, P, &nb, &ms), DSI_EINVAL);
  expect("profile_stream misaligned", dsi_profile_stream((const char*)P + 4, 1 << 30, 1, 0, 0, 1, P, &nb, &ms),
         DSI_EINVAL);
  expect("profile_stream small slices", dsi_profile_stream(P, 32 << 20, 4, 0, 0, 1, P, &nb, &ms), DSI_EINVAL);
  expect("profile_stream zero rounds", dsi_profile_stream(P, 1 << 30, 1, 0, 0, 0, P, &nb, &ms), DSI_EINVAL);
  expect("profile_stream negative workgroups", dsi_profile_stream(P, 1 << 30, 1, 0, -1, 1, P, &nb, &ms),
         DSI_EINVAL);
  expect("profile_stream too many workgroups", dsi_profile_stream(P, 1 << 30, 1, 0, 4097, 1, P, &nb, &ms),
         DSI_EINVAL);

  /* accept/reject: host validation of the batch shape and arguments */
  expect("accept zero windows", dsi_accept(NULL, 0, 3, 100, fdummy, dummy, fdummy, fdummy, 1.f, 0, dummy, dummy),
         DSI_EINVAL);
  expect("accept too many rows", dsi_accept(NULL, 9, 7, 100, fdummy, dummy, fdummy, fdummy, 1.f, 0, dummy, dummy),
         DSI_EINVAL);
  expect("accept missing q", dsi_accept(NULL, 1, 3, 100, fdummy, dummy, NULL, fdummy, 1.f, 0, dummy, dummy),
         DSI_EINVAL);
  expect("accept T <= 0", dsi_accept(NULL, 1, 3, 100, fdummy, dummy, fdummy, fdummy, 0.f, 0, dummy, dummy),
         DSI_EINVAL);
  expect("accept bad mode", dsi_accept(NULL, 1, 3, 100, fdummy, dummy, fdummy, fdummy, 1.f, 7, dummy, dummy),
         DSI_EINVAL);
  expect("accept_noalloc too many rows",
         dsi_accept_noalloc(NULL, 9, 7, 100, fdummy, dummy, fdummy, fdummy, 1.f, 0, dummy, dummy), DSI_EINVAL);
  expect("accept_noalloc workspace too small",
         dsi_accept_noalloc(NULL, 1, 3, 1 << 30, fdummy, dummy, fdummy, fdummy, 1.f, 0, dummy, dummy),
         DSI_ECAPACITY);
  /* valid arguments: fails on the first HIP call */
  expect_error("accept valid without device",
               dsi_accept(NULL, 1, 3, 100, fdummy, dummy, fdummy, fdummy, 1.f, 0, dummy, dummy));
  expect_error("accept_noalloc valid without device",
               dsi_accept_noalloc(NULL, 1, 3, 100, fdummy, dummy, fdummy, fdummy, 1.f, 0, dummy, dummy));
  expect("draft null", dsi_draft(NULL, NULL, 0, dummy, 1, 3, fdummy, 1.f, dummy, fdummy), DSI_EINVAL);

  if (failures) {
    printf("%d failure(s)\n", failures);
    return 1;
  }
  printf("host ABI paths ok\n");
  return 0;
}
