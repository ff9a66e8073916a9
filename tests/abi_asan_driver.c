/* Host-side driver of the C ABI, built with AddressSanitizer together with the
 * library's host code: every size query, view query and argument-error path of
 * every entry point, the trace API and the thread-local error strings.  No
 * call here reaches a device launch unless argv[1] is "launch" (a machine with
 * no GPU: the launch is refused and must come back as MOE_ERR_HIP).
 *
 * Exit status 0 when every checked return value is the expected one; each
 * mismatch prints one line.  AddressSanitizer aborts the run on any invalid
 * host memory access. */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "moe.h"

static int failures = 0;

#define EXPECT(cond)                                                \
  do {                                                              \
    if (!(cond)) {                                                  \
      fprintf(stderr, "FAIL line %d: %s\n", __LINE__, #cond);       \
      ++failures;                                                   \
    }                                                               \
  } while (0)

/* The error string must be readable in full (ASan checks every byte). */
static size_t last_error_len(void) {
  const char* s = moe_last_error();
  return s ? strlen(s) : 0;
}

#define FAKE ((void*)(uintptr_t)(1u << 20)) /* 16-byte aligned, never dereferenced */
#define MIS ((void*)(uintptr_t)((1u << 20) + 8))

static moe_dims dims(int T, int H, int E, int F, int k) {
  moe_dims d;
  memset(&d, 0, sizeof d);
  d.T = T, d.H = H, d.E = E, d.F = F, d.top_k = k;
  return d;
}

static int fwd(const moe_dims* d, const void* x, const void* w_down, size_t ws) {
  return moe_fwd(d, x, FAKE, FAKE, FAKE, w_down, NULL, FAKE, FAKE, FAKE, ws, NULL);
}

static int bwd(const moe_dims* d, const void* dy, void* dw_r, size_t ws) {
  return moe_bwd(d, FAKE, FAKE, FAKE, FAKE, FAKE, dy, FAKE, FAKE, dw_r, FAKE, FAKE, FAKE, FAKE, ws, NULL);
}

static void sizes(void) {
  moe_dims d = dims(256, 128, 8, 256, 2);
  size_t saved = moe_saved_bytes(&d);
  EXPECT(saved > 0);
  EXPECT(moe_fwd_workspace_bytes(&d) > 0);
  EXPECT(moe_bwd_workspace_bytes(&d) > 0);
  EXPECT(moe_infer_workspace_bytes(&d) > 0);
  EXPECT(moe_lora_saved_bytes(&d, 16) > saved);
  EXPECT(moe_lora_workspace_bytes(&d, 64) > 0);
  EXPECT(moe_lora_saved_bytes(&d, 24) == 0);
  moe_dims bad = dims(256, 100, 8, 256, 2);
  EXPECT(moe_saved_bytes(&bad) == 0 && moe_fwd_workspace_bytes(&bad) == 0 && moe_bwd_workspace_bytes(&bad) == 0);
  EXPECT(moe_saved_bytes(NULL) == 0 && moe_infer_workspace_bytes(NULL) == 0);
  /* the largest expert count and top-k the limits allow */
  moe_dims wide = dims(4096, 2048, MOE_MAX_EXPERTS, 768, MOE_MAX_TOPK);
  EXPECT(moe_saved_bytes(&wide) > 0 && moe_bwd_workspace_bytes(&wide) > 0);
  moe_dims over = dims(4096, 2048, MOE_MAX_EXPERTS + 8, 768, 8);
  EXPECT(moe_saved_bytes(&over) == 0);

  moe_saved_view v;
  EXPECT(moe_saved_views(&d, FAKE, &v) == MOE_OK);
  EXPECT(v.logits != NULL && v.xp != NULL && v.g != NULL && v.o != NULL);
  EXPECT(moe_saved_views(&bad, FAKE, &v) == MOE_ERR_SHAPE || moe_saved_views(&bad, FAKE, &v) == MOE_ERR_ARG);
  EXPECT(moe_saved_views(&d, FAKE, NULL) == MOE_ERR_ARG);
  moe_dims rc = d;
  rc.flags = MOE_F_RECOMPUTE;
  EXPECT(moe_saved_views(&rc, FAKE, &v) == MOE_OK && v.g == NULL && v.u == NULL);

  moe_experts_dims ed = {1000, 256, 4, 128, 0};
  EXPECT(moe_experts_saved_bytes(&ed) > 0 && moe_experts_workspace_bytes(&ed) > 0);
  moe_experts_saved_view ev;
  EXPECT(moe_experts_saved_views(&ed, FAKE, &ev) == MOE_OK && ev.offsets != NULL && ev.a != NULL);
  moe_experts_dims edb = {1000, 256, 4, 100, 0};
  EXPECT(moe_experts_saved_bytes(&edb) == 0);
  EXPECT(moe_version() >= 100);
}

static void errors(void) {
  moe_dims d = dims(256, 128, 8, 256, 2);
  const size_t ws = (size_t)1 << 40;
  /* dims */
  moe_dims b;
  b = dims(0, 128, 8, 256, 2);
  EXPECT(fwd(&b, FAKE, FAKE, ws) == MOE_ERR_ARG && last_error_len() > 0);
  b = dims(256, 128, 8, 256, 0);
  EXPECT(fwd(&b, FAKE, FAKE, ws) == MOE_ERR_ARG && last_error_len() > 0);
  b = dims(256, 128, 8, 256, 9);
  EXPECT(bwd(&b, FAKE, FAKE, ws) == MOE_ERR_ARG && last_error_len() > 0);
  b = dims(256, 100, 8, 256, 2);
  EXPECT(fwd(&b, FAKE, FAKE, ws) == MOE_ERR_SHAPE && last_error_len() > 0);
  b = dims(256, 128, 12, 256, 2);
  EXPECT(bwd(&b, FAKE, FAKE, ws) == MOE_ERR_SHAPE && last_error_len() > 0);
  b = d;
  b.flags = 8u;
  EXPECT(fwd(&b, FAKE, FAKE, ws) == MOE_ERR_ARG);
  b = d;
  b.aux_loss_coef = -0.5f;
  EXPECT(fwd(&b, FAKE, FAKE, ws) == MOE_ERR_ARG);
  b = d;
  b.z_loss_coef = NAN;
  EXPECT(bwd(&b, FAKE, FAKE, ws) == MOE_ERR_ARG);
  EXPECT(fwd(NULL, FAKE, FAKE, ws) == MOE_ERR_ARG);
  /* pointers, alignment, workspace */
  EXPECT(fwd(&d, NULL, FAKE, ws) == MOE_ERR_ARG && strstr(moe_last_error(), "x") != NULL);
  EXPECT(fwd(&d, FAKE, MIS, ws) == MOE_ERR_ALIGN);
  EXPECT(fwd(&d, FAKE, FAKE, 0) == MOE_ERR_WORKSPACE);
  b = d;
  b.flags = MOE_F_MASK; /* mask flag without a mask */
  EXPECT(fwd(&b, FAKE, FAKE, ws) == MOE_ERR_ARG);
  EXPECT(bwd(&d, NULL, FAKE, ws) == MOE_ERR_ARG);
  EXPECT(bwd(&d, FAKE, MIS, ws) == MOE_ERR_ALIGN);
  EXPECT(bwd(&d, FAKE, FAKE, 1024) == MOE_ERR_WORKSPACE);
  /* forward-only */
  EXPECT(moe_infer(&d, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, NULL, FAKE, ws, NULL) == MOE_ERR_ARG);
  EXPECT(moe_infer(&d, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, FAKE, FAKE, 16, NULL) == MOE_ERR_WORKSPACE);
  /* allocation-free forward: too large for its static array */
  moe_dims big = dims(65536, 2048, 128, 768, 8);
  EXPECT(moe_fwd_noalloc(&big, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, FAKE, FAKE, NULL) == MOE_ERR_WORKSPACE);
  EXPECT(moe_fwd_noalloc(&d, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, FAKE, NULL, NULL) == MOE_ERR_ARG);
  /* LoRA */
  moe_lora lo = {16, 2.0f, FAKE, FAKE, FAKE, FAKE, FAKE};
  EXPECT(moe_lora_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, NULL, FAKE, FAKE, FAKE, ws, NULL) == MOE_ERR_ARG);
  moe_lora lb = lo;
  lb.rank = 24;
  EXPECT(moe_lora_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, &lb, NULL, FAKE, FAKE, FAKE, ws, NULL) == MOE_ERR_SHAPE);
  lb = lo;
  lb.scale = INFINITY;
  EXPECT(moe_lora_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, &lb, NULL, FAKE, FAKE, FAKE, ws, NULL) == MOE_ERR_ARG);
  lb = lo;
  lb.a2 = MIS;
  EXPECT(moe_lora_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, &lb, NULL, FAKE, FAKE, FAKE, ws, NULL) == MOE_ERR_ALIGN);
  EXPECT(moe_lora_bwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, &lo, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                      16, NULL) == MOE_ERR_WORKSPACE);
  /* one expert-parallel rank's share */
  moe_experts_dims ed = {100, 128, 4, 128, 0};
  EXPECT(moe_experts_fwd(&ed, FAKE, NULL, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, 0, NULL) == MOE_ERR_ARG);
  moe_experts_dims edb = {100, 128, 4, 100, 0};
  EXPECT(moe_experts_fwd(&edb, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, 0, NULL) == MOE_ERR_SHAPE);
  EXPECT(moe_experts_bwd(&ed, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16, NULL) ==
         MOE_ERR_WORKSPACE);
}

static void trace_api(void) {
  EXPECT(moe_trace_enable(0) == 0);
  int n = moe_trace_read(NULL, NULL, 0);
  EXPECT(n >= 17);
  double ms[64];
  int32_t launches[64];
  EXPECT(moe_trace_read(ms, launches, n < 64 ? n : 64) == n);
  for (int i = 0; i < n; ++i) {
    const char* s = moe_trace_name(i);
    EXPECT(s != NULL && strlen(s) > 0);
  }
  EXPECT(strlen(moe_trace_name(-1)) == 0 && strlen(moe_trace_name(n)) == 0);
}

/* moe_last_error is per thread: each thread sees the message of its own
 * last failing call. */
static void* thread_errors(void* arg) {
  const int which = *(const int*)arg;
  moe_dims d = dims(256, 128, 8, 256, 2);
  int ok = 1;
  for (int i = 0; i < 200; ++i) {
    if (which == 0) {
      ok &= fwd(&d, NULL, FAKE, (size_t)1 << 40) == MOE_ERR_ARG;
      ok &= strstr(moe_last_error(), "x") != NULL;
    } else {
      ok &= fwd(&d, FAKE, FAKE, 0) == MOE_ERR_WORKSPACE;
      ok &= strstr(moe_last_error(), "orkspace") != NULL;
    }
  }
  return ok ? (void*)1 : NULL;
}

static void threads(void) {
  pthread_t th[2];
  int ids[2] = {0, 1};
  for (int i = 0; i < 2; ++i) EXPECT(pthread_create(&th[i], NULL, thread_errors, &ids[i]) == 0);
  for (int i = 0; i < 2; ++i) {
    void* r = NULL;
    EXPECT(pthread_join(th[i], &r) == 0);
    EXPECT(r == (void*)1);
  }
}

int main(int argc, char** argv) {
  sizes();
  errors();
  trace_api();
  threads();
  if (argc > 1 && strcmp(argv[1], "launch") == 0) {
    /* no GPU in the machine: valid arguments, the launch is refused */
    moe_dims d = dims(256, 128, 8, 256, 2);
    EXPECT(fwd(&d, FAKE, FAKE, (size_t)1 << 30) == MOE_ERR_HIP && last_error_len() > 0);
  }
  printf("abi driver: %d failure(s)\n", failures);
  return failures ? 1 : 0;
}
