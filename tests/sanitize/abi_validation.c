/* Host-side checks of the C ABI in include/tls.h, written in C and built
 * with AddressSanitizer and UndefinedBehaviorSanitizer over a host-only
 * build of the library (no device code, no GPU).  Every call here either is
 * a pure host function (version, status strings, workspace sizing) or is
 * rejected by host validation before anything is enqueued, so the program
 * runs without a device; the sanitizers check the validation and sizing
 * arithmetic itself (out-of-bounds reads of the argument structs, signed
 * overflow in size products, misaligned or null dereferences).
 * Exit status 0 when every expectation holds; the first failed one is
 * printed with its line. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "tls.h"

static int g_failures = 0;

#define EXPECT(cond)                                              \
  do {                                                            \
    if (!(cond)) {                                                \
      fprintf(stderr, "abi_validation.c:%d: %s\n", __LINE__, #cond); \
      ++g_failures;                                               \
    }                                                             \
  } while (0)

static tls_layout gqa(int32_t b, int32_t T) {
  tls_layout L;
  memset(&L, 0, sizeof L);
  L.batch = b;
  L.num_q_heads = 32;
  L.num_kv_heads = 8;
  L.head_dim_qk = 128;
  L.head_dim_v = 128;
  L.block_size = 64;
  L.index_channels = 32;
  L.max_ctx = T;
  L.dtype = TLS_DTYPE_BF16;
  return L;
}

static tls_layout mla(int32_t b, int32_t T) {
  tls_layout L = gqa(b, T);
  L.num_q_heads = 16;
  L.num_kv_heads = 1;
  L.head_dim_qk = 576;
  L.head_dim_v = 512;
  L.index_channels = 128;
  L.mla_shared_kv = 1;
  return L;
}

/* A pointer value validation may test for NULL but never dereferences. */
static void* const D = (void*)(uintptr_t)0x1000;

static void strings(void) {
  const char* v = tls_version();
  EXPECT(v != NULL && strstr(v, "gfx950") != NULL);
  for (int s = -4; s <= 12; ++s) {
    const char* n = tls_status_string(s);
    EXPECT(n != NULL && strlen(n) > 0);
  }
  EXPECT(strcmp(tls_status_string(TLS_OK), "TLS_OK") == 0);
}

static void workspace_sizes(void) {
  size_t a = 0, b = 0, c = 0;
  tls_layout L = gqa(2, 4096);
  EXPECT(tls_workspace_size(&L, 8, 128, &a) == TLS_OK);
  EXPECT(tls_workspace_size(&L, 64, 2048, &b) == TLS_OK);
  EXPECT(a > 0 && b > a);
  /* the largest shapes the library takes: sizes must not wrap */
  tls_layout big = gqa(8191, 64 * 12288); /* 65528 units, 12288 blocks each */
  EXPECT(tls_workspace_size(&big, 128, 8192, &c) == TLS_OK);
  EXPECT(c > b);
  big.max_ctx = 64 * 12288 + 1; /* one block past the top-k capacity */
  EXPECT(tls_workspace_size(&big, 128, 8192, &c) == TLS_ERR_UNSUPPORTED);
  big = gqa(8192, 4096); /* 65536 units: past the grid limit */
  EXPECT(tls_workspace_size(&big, 8, 128, &c) == TLS_ERR_UNSUPPORTED);
  tls_layout m = mla(8, 65536);
  EXPECT(tls_workspace_size(&m, 128, 2048, &c) == TLS_OK && c > 0);
  /* a sweep of budgets and lengths through the host planner */
  for (int32_t T = 64; T <= 64 * 16384; T *= 4)
    for (int32_t kb = 1; kb <= 256; kb *= 2)
      for (int32_t kt = 1; kt <= 16384; kt *= 8) {
        tls_layout S = gqa(3, T + 17);
        size_t bytes = 0;
        const tls_status st = tls_workspace_size(&S, kb, kt, &bytes);
        EXPECT(st == TLS_OK || st == TLS_ERR_UNSUPPORTED || st == TLS_ERR_INVALID_ARGUMENT);
        if (st == TLS_OK) EXPECT(bytes > 0);
      }
  /* bad layouts and budgets */
  tls_layout bad = gqa(2, 4096);
  bad.num_q_heads = 30;
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) == TLS_ERR_INVALID_ARGUMENT);
  bad = gqa(2, 4096);
  bad.index_channels = 48;
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) == TLS_ERR_INVALID_ARGUMENT);
  bad = gqa(2, 4096);
  bad.dtype = 7;
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) == TLS_ERR_INVALID_ARGUMENT);
  bad = gqa(-1, 4096);
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) == TLS_ERR_INVALID_ARGUMENT);
  bad = gqa(2, -64);
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) == TLS_ERR_INVALID_ARGUMENT);
  bad = gqa(2, 4096);
  bad.block_size = 0;
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) != TLS_OK);
  bad = gqa(2, 4096);
  bad.num_kv_heads = 0;
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) == TLS_ERR_INVALID_ARGUMENT);
  bad = gqa(2, 4096);
  bad.head_dim_qk = 100;
  bad.head_dim_v = 100;
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) == TLS_ERR_UNSUPPORTED);
  bad = gqa(2, 4096);
  bad.max_ctx = 2147483647;
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) != TLS_OK);
  bad = gqa(2147483647, 4096);
  EXPECT(tls_workspace_size(&bad, 8, 128, &a) != TLS_OK);
  L = gqa(2, 4096);
  EXPECT(tls_workspace_size(&L, 0, 128, &a) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_workspace_size(&L, 8, 0, &a) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_workspace_size(&L, 8, -5, &a) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_workspace_size(&L, 300, 128, &a) == TLS_ERR_UNSUPPORTED);
  EXPECT(tls_workspace_size(&L, 2147483647, 2147483647, &a) != TLS_OK);
  EXPECT(tls_workspace_size(NULL, 8, 128, &a) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_workspace_size(&L, 8, 128, NULL) == TLS_ERR_INVALID_ARGUMENT);
}

static tls_status decode(const tls_layout* L, const tls_kv_view* kv, int32_t K_b, int32_t K_t, const void* bin,
                         const void* tin, void* bout, void* tout, size_t ws_bytes, const tls_decode_opts* o) {
  return tls_sparse_decode(L, D, kv, D, D, D, D, D, D, K_b, K_t, bin, tin, D, NULL, bout, tout, D, ws_bytes, o,
                           NULL);
}

static void decode_validation(void) {
  const tls_layout L = gqa(2, 4096);
  const tls_layout M = mla(2, 4096);
  tls_kv_view kv = {D, D, NULL, 0};
  tls_kv_view k_only = {D, NULL, NULL, 0};
  tls_decode_opts o;
  memset(&o, 0, sizeof o);
  const size_t huge = (size_t)1 << 40;
  EXPECT(decode(NULL, &kv, 8, 128, NULL, NULL, NULL, NULL, huge, &o) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, NULL, 8, 128, NULL, NULL, NULL, NULL, huge, &o) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &k_only, 8, 128, NULL, NULL, NULL, NULL, huge, &o) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&M, &kv, 8, 128, NULL, NULL, NULL, NULL, huge, &o) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 0, 128, NULL, NULL, NULL, NULL, huge, &o) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 0, NULL, NULL, NULL, NULL, huge, &o) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, NULL, NULL, 16, &o) == TLS_ERR_WORKSPACE_TOO_SMALL);
  for (int i = 0; i < 6; ++i) {
    tls_decode_opts r = o;
    r.reserved[i] = 1;
    EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, NULL, NULL, huge, &r) == TLS_ERR_INVALID_ARGUMENT);
  }
  tls_decode_opts m = o;
  m.mode = 4;
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, NULL, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  m.mode = -1;
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, NULL, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  m.mode = TLS_MODE_DENSE;
  EXPECT(decode(&L, &kv, 8, 128, D, NULL, NULL, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, NULL, D, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  m.mode = TLS_MODE_TOKEN_SPARSE;
  EXPECT(decode(&L, &kv, 8, 128, NULL, D, NULL, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, D, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  m.mode = TLS_MODE_BLOCK_SPARSE;
  EXPECT(decode(&L, &kv, 8, 128, NULL, D, NULL, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, NULL, D, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  /* the lagged operator: both block lists, not overlapping, no given tokens */
  m.mode = TLS_MODE_LAGGED;
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, NULL, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, D, NULL, NULL, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, D, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, D, NULL, D, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, D, NULL, (char*)D + 4, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(decode(&L, &kv, 8, 128, D, D, (char*)D + (1 << 20), NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  m.mode = 5;
  EXPECT(decode(&L, &kv, 8, 128, NULL, NULL, NULL, NULL, huge, &m) == TLS_ERR_INVALID_ARGUMENT);
  /* pooled view: slot map without slots */
  tls_kv_view pool = {D, D, (const int32_t*)D, 0};
  EXPECT(decode(&L, &pool, 8, 128, NULL, NULL, NULL, NULL, huge, &o) == TLS_ERR_INVALID_ARGUMENT);
  /* the allocation-free variant rejects the same arguments, and a route
   * whose scratch exceeds its buffer, before touching a device */
  EXPECT(tls_sparse_decode_noalloc(&L, D, &k_only, D, D, D, D, D, D, 8, 128, NULL, NULL, D, NULL, NULL, NULL, NULL,
                                   &o, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_sparse_decode_noalloc(&L, D, &kv, D, D, D, D, D, D, 0, 128, NULL, NULL, D, NULL, NULL, NULL, NULL, &o,
                                   NULL) == TLS_ERR_INVALID_ARGUMENT);
  tls_decode_opts t = o;
  t.mode = TLS_MODE_TOKEN_SPARSE;
  const tls_layout wide = gqa(256, 65600);
  EXPECT(tls_sparse_decode_noalloc(&wide, D, &kv, D, D, D, D, D, D, 8, 128, NULL, NULL, D, NULL, NULL, NULL, NULL,
                                   &t, NULL) == TLS_ERR_WORKSPACE_TOO_SMALL);
}

static void selection_and_index_validation(void) {
  const tls_layout L = gqa(2, 4096);
  const tls_layout M = mla(2, 4096);
  EXPECT(tls_select_blocks(&L, D, D, D, D, 8, D, NULL, D, 16, NULL) == TLS_ERR_WORKSPACE_TOO_SMALL);
  EXPECT(tls_select_blocks(&L, NULL, D, D, D, 8, D, NULL, D, (size_t)1 << 40, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_select_blocks(&L, D, D, D, D, 0, D, NULL, D, (size_t)1 << 40, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_select_tokens(&L, D, D, D, D, D, 8, D, 0, D, NULL, D, (size_t)1 << 40, NULL) ==
         TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_select_tokens(&L, D, NULL, D, D, D, 8, D, 128, D, NULL, D, (size_t)1 << 40, NULL) ==
         TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_build_block_index(&L, NULL, D, 0, 64, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_build_block_index(&L, D, D, 0, 5000, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_build_block_index(&L, D, D, -1, 64, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_build_token_index(&L, D, D, NULL, 0, 64, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_build_token_index(&L, D, D, D, 64, 0, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_prefill_kv(&L, NULL, D, D, D, 0, 64, D, D, D, D, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_prefill_kv(&L, D, NULL, D, D, 0, 64, D, D, D, D, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_prefill_kv(&M, D, D, D, D, 0, 64, D, D, D, D, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_prefill_kv(&L, D, D, D, D, 0, 4097, D, D, D, D, D, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_prefill_kv(&L, D, D, D, D, 64, 64, D, D, D, D, D, D, NULL) == TLS_OK); /* empty range */
  EXPECT(tls_calibrate_absmax(&L, D, D, -1, D, D, 0, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_calibrate_absmax(&L, D, D, 16, D, D, 2, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_calibrate_channels(&L, D, D, NULL, NULL, NULL) == TLS_ERR_INVALID_ARGUMENT);
}

static void offload_validation(void) {
  const tls_layout L = gqa(2, 4096);
  const tls_layout M = mla(2, 4096);
  const size_t huge = (size_t)1 << 40;
  EXPECT(tls_prefetch_blocks(&L, D, D, D, D, D, 8, D, D, 10, D, D, NULL, D, huge, NULL) ==
         TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_prefetch_blocks(&L, D, D, D, D, NULL, 8, D, D, 4, D, D, NULL, D, huge, NULL) ==
         TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_prefetch_blocks(&L, D, D, D, D, D, 0, D, D, 64, D, D, NULL, D, huge, NULL) ==
         TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_offload_kv(&L, D, D, D, 0, 64, NULL, D, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_offload_kv(&M, D, D, D, 0, 64, D, NULL, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_init_residency(&L, D, D, D, D, 0, D, D, 16, D, D, D, huge, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_init_residency(&L, D, D, D, D, 8, D, D, 4, D, D, D, huge, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_init_residency(&M, D, D, D, D, 8, D, D, 16, D, D, D, huge, NULL) == TLS_ERR_INVALID_ARGUMENT);
  tls_kv_view bad_pool = {D, D, NULL, 16};
  EXPECT(tls_append_tokens(&L, D, D, D, D, D, D, D, D, D, D, &bad_pool, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_append_tokens(&L, NULL, D, D, D, D, D, D, D, D, D, NULL, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_append_tokens(&M, D, D, D, D, D, D, D, D, D, D, NULL, NULL) == TLS_ERR_INVALID_ARGUMENT);
  int32_t flags = 0;
  EXPECT(tls_check_device_error(NULL, 0, 0, &flags, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_check_device_error(D, huge, 0, NULL, NULL) == TLS_ERR_INVALID_ARGUMENT);
  EXPECT(tls_workspace_init(NULL, 0, NULL) == TLS_ERR_INVALID_ARGUMENT);
}

int main(void) {
  strings();
  workspace_sizes();
  decode_validation();
  selection_and_index_validation();
  offload_validation();
  if (g_failures) {
    fprintf(stderr, "%d expectation(s) failed\n", g_failures);
    return 1;
  }
  printf("abi_validation: all host-side checks passed\n");
  return 0;
}
