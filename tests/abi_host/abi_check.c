/* Host-only check of the C ABI's argument handling, compiled as C99 and linked with the
 * library's host layer built under AddressSanitizer and UndefinedBehaviorSanitizer.
 *
 * Runs only where no GPU is present.  Device pointers are fake addresses (aligned or
 * deliberately misaligned) that the library never dereferences: every call below is
 * rejected during validation, is an empty layer, or -- in the last group -- passes
 * validation and must then report the failed launch as CRISP_EHIP.
 * Exit status 0 iff every expectation held. */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "crisp.h"

static int failures;
static int checks;

#define EXPECT(cond, ...)                                         \
  do {                                                            \
    ++checks;                                                     \
    if (!(cond)) {                                                \
      ++failures;                                                 \
      fprintf(stderr, "FAIL line %d: ", __LINE__);                \
      fprintf(stderr, __VA_ARGS__);                               \
      fprintf(stderr, " [last error: %s]\n", crisp_last_error()); \
    }                                                             \
  } while (0)

#define DEV(addr) ((void*)(uintptr_t)(addr))

static void* const P256 = DEV(0x7f0000100000ull); /* 256-byte aligned */
static void* const P8 = DEV(0x7f0000100008ull);   /* 8- but not 16-byte aligned */
static void* const P16 = DEV(0x7f0000100010ull);  /* 16- but not 256-byte aligned */
static void* const P2 = DEV(0x7f0000100002ull);   /* 2- but not 4-byte aligned */

static crisp_shape shape(int hq, int hkv, int n, int d, int b) {
  crisp_shape s;
  s.n_q_heads = hq;
  s.n_kv_heads = hkv;
  s.seq_len = n;
  s.head_dim = d;
  s.block = b;
  return s;
}

/* Every compute entry point with otherwise valid arguments for shape s and params p
 * (workspace big enough for s when s is valid); returns the statuses in st[6]. */
static void call_all(const crisp_shape* s, const crisp_params* p, crisp_status st[6]) {
  size_t ws = (size_t)1 << 40;
  int64_t cap = (int64_t)1 << 40;
  st[0] = crisp_estimate(s, p, P256, P256, P256, P256, P256, P256, ws, NULL);
  st[1] = crisp_jsd(s, p, P256, P256, P256, P256, P256, ws, NULL);
  st[2] = crisp_route_select(s, p, P256, P256, P256, P256, P256, P256, P256, P256, cap, NULL, P256, ws, NULL);
  st[3] = crisp_sparse_attn(s, 0.f, P256, P256, P256, P256, P256, cap, P256, NULL, 0, NULL);
  st[4] = crisp_prefill_attn(s, p, P256, P256, P256, P256, NULL, NULL, NULL, P256, ws, NULL);
  st[5] = crisp_dense_attn(s, 0.f, P256, P256, P256, P256, NULL);
}

static void check_defaults(void) {
  crisp_params p;
  memset(&p, 0xff, sizeof(p));
  crisp_params_default(&p);
  EXPECT(p.alpha == 1.0f && p.tau_proxy == 0.2f && p.gamma == 0.95f, "paper defaults alpha/tau/gamma");
  EXPECT(p.w_sink == 128 && p.w_local == 128 && p.k_min_blocks == 0 && p.softmax_scale == 0.0f, "anchor defaults");
  EXPECT(p.route_mode == CRISP_ROUTE_BY_CSTRUCT && p.vs_mode == CRISP_VS_FLOOR && p.floor_mode == CRISP_FLOOR_MEAN,
         "mode defaults");
  EXPECT(p.tau_jsd == 0.1f && p.dense_below_len == 0, "comparator defaults");
  crisp_params_default(NULL); /* ignored */
}

static void check_sizes(void) {
  crisp_shape s = shape(32, 8, 131072, 128, 128);
  EXPECT(crisp_col_capacity(&s) == 1024LL * 1025 / 2, "capacity at 128k");
  crisp_shape bad = shape(3, 2, 4096, 128, 128);
  EXPECT(crisp_col_capacity(&bad) == -1, "capacity of a bad shape");
  EXPECT(crisp_col_capacity(NULL) == -1, "capacity of a null shape");
  size_t a = 0, b = 0, c = 0;
  EXPECT(crisp_workspace_size(&s, &a) == CRISP_OK && a > 0 && a % 256 == 0, "workspace size %zu", a);
  EXPECT(crisp_prefill_workspace_size(&s, &b) == CRISP_OK && b > a, "prefill workspace %zu > %zu", b, a);
  EXPECT(crisp_sparse_workspace_size(&s, &c) == CRISP_OK && c > 0 && c % 256 == 0, "sparse workspace %zu", c);
  EXPECT(crisp_workspace_size(&s, NULL) == CRISP_EINVAL, "null bytes");
  EXPECT(crisp_prefill_workspace_size(&s, NULL) == CRISP_EINVAL, "null bytes (prefill)");
  EXPECT(crisp_sparse_workspace_size(&s, NULL) == CRISP_EINVAL, "null bytes (sparse)");
  EXPECT(crisp_workspace_size(&bad, &a) == CRISP_EINVAL, "workspace of a bad shape");
  crisp_shape big = shape(17, 1, 1 << 21, 128, 64);
  EXPECT(crisp_workspace_size(&big, &a) == CRISP_OK && a > ((size_t)1 << 31), "longest layer workspace %zu", a);
  EXPECT(crisp_prefill_workspace_size(&big, &b) == CRISP_OK && b > a, "longest layer prefill workspace");
  crisp_shape empty = shape(4, 2, 0, 128, 128);
  EXPECT(crisp_workspace_size(&empty, &a) == CRISP_OK, "empty layer workspace");
}

static void check_shapes(void) {
  crisp_params p;
  crisp_params_default(&p);
  struct {
    crisp_shape s;
    crisp_status want;
  } cases[] = {
      {{3, 2, 4096, 128, 128}, CRISP_EINVAL},        /* H_q not a multiple of H_kv */
      {{4, 0, 4096, 128, 128}, CRISP_EINVAL},        /* no KV head */
      {{-4, 2, 4096, 128, 128}, CRISP_EINVAL},       /* negative heads */
      {{4, 2, -128, 128, 128}, CRISP_EINVAL},        /* negative length */
      {{4, 2, 4096, 64, 128}, CRISP_EUNSUPPORTED},   /* head_dim */
      {{4, 2, 4096, 256, 128}, CRISP_EUNSUPPORTED},  /* head_dim */
      {{4, 2, 4096, 128, 32}, CRISP_EUNSUPPORTED},   /* block */
      {{4, 2, 4096, 128, 256}, CRISP_EUNSUPPORTED},  /* block */
      {{4, 2, (1 << 21) + 128, 128, 128}, CRISP_EUNSUPPORTED}, /* above the longest layer */
  };
  for (size_t i = 0; i < sizeof(cases) / sizeof(cases[0]); ++i) {
    crisp_status st[6];
    call_all(&cases[i].s, &p, st);
    for (int e = 0; e < 6; ++e)
      EXPECT(st[e] == cases[i].want && crisp_last_error()[0] != '\0', "shape case %zu entry %d: %s", i, e,
             crisp_status_string(st[e]));
  }
  crisp_status st[6];
  call_all(NULL, &p, st);
  for (int e = 0; e < 6; ++e) EXPECT(st[e] == CRISP_EINVAL, "null shape entry %d", e);
}

static void check_params(void) {
  crisp_shape s = shape(4, 2, 4096, 128, 128);
  crisp_params base;
  crisp_params_default(&base);
  for (int c = 0; c < 14; ++c) {
    crisp_params p = base;
    switch (c) {
      case 0: p.alpha = -0.5f; break;
      case 1: p.alpha = NAN; break;
      case 2: p.alpha = INFINITY; break;
      case 3: p.gamma = 0.f; break;
      case 4: p.gamma = 1.5f; break;
      case 5: p.tau_proxy = NAN; break;
      case 6: p.w_sink = -1; break;
      case 7: p.w_local = -1; break;
      case 8: p.k_min_blocks = -2; break;
      case 9: p.softmax_scale = -1.f; break;
      case 10: p.route_mode = 7; break;
      case 11: p.vs_mode = -1; break;
      case 12: p.tau_jsd = INFINITY; break;
      case 13: p.floor_mode = 2; break;
    }
    crisp_status st[6];
    call_all(&s, &p, st);
    EXPECT(st[0] == CRISP_EINVAL && st[1] == CRISP_EINVAL && st[2] == CRISP_EINVAL && st[4] == CRISP_EINVAL,
           "param case %d: %d %d %d %d", c, st[0], st[1], st[2], st[4]);
    crisp_params q = base;
    q.dense_below_len = -1;
    EXPECT(crisp_prefill_attn(&s, &q, P256, P256, P256, P256, NULL, NULL, NULL, P256, (size_t)1 << 40, NULL) ==
               CRISP_EINVAL, "negative gate");
  }
  crisp_status st[6];
  call_all(&s, NULL, st);
  EXPECT(st[0] == CRISP_EINVAL && st[1] == CRISP_EINVAL && st[2] == CRISP_EINVAL && st[4] == CRISP_EINVAL,
         "null params");
  EXPECT(crisp_sparse_attn(&s, NAN, P256, P256, P256, P256, P256, 1 << 20, P256, NULL, 0, NULL) == CRISP_EINVAL,
         "NaN scale (sparse)");
  EXPECT(crisp_dense_attn(&s, -1.f, P256, P256, P256, P256, NULL) == CRISP_EINVAL, "negative scale (dense)");
}

static void check_pointers(void) {
  crisp_shape s = shape(4, 2, 4096, 128, 128);
  crisp_params p;
  crisp_params_default(&p);
  size_t ws = 0, pws = 0, sws = 0;
  crisp_workspace_size(&s, &ws);
  crisp_prefill_workspace_size(&s, &pws);
  crisp_sparse_workspace_size(&s, &sws);
  const int64_t cap = crisp_col_capacity(&s);

  EXPECT(crisp_estimate(&s, &p, NULL, P256, P256, P256, P256, P256, ws, NULL) == CRISP_EINVAL &&
             strstr(crisp_last_error(), "q") != NULL, "null q");
  EXPECT(crisp_estimate(&s, &p, P8, P256, P256, P256, P256, P256, ws, NULL) == CRISP_EINVAL, "misaligned q");
  EXPECT(crisp_estimate(&s, &p, P256, P256, P2, P256, P256, P256, ws, NULL) == CRISP_EINVAL, "misaligned c_struct");
  EXPECT(crisp_estimate(&s, &p, P256, P256, P256, P256, P256, P16, ws, NULL) == CRISP_EINVAL,
         "workspace not 256-aligned");
  /* crisp_workspace_size covers the largest of three entry points; 256 bytes fit none */
  EXPECT(crisp_estimate(&s, &p, P256, P256, P256, P256, P256, P256, 256, NULL) == CRISP_EINVAL &&
             strstr(crisp_last_error(), "workspace") != NULL, "small workspace");
  EXPECT(crisp_jsd(&s, &p, P256, P256, NULL, P256, P256, ws, NULL) == CRISP_EINVAL, "null p_v (jsd)");
  EXPECT(crisp_jsd(&s, &p, P256, P256, P256, P256, P256, 256, NULL) == CRISP_EINVAL, "small workspace (jsd)");
  EXPECT(crisp_route_select(&s, &p, P256, P256, P256, P256, P256, P256, P256, P256, cap - 1, NULL, P256, ws, NULL) ==
             CRISP_EINVAL, "col capacity one short");
  EXPECT(crisp_route_select(&s, &p, P256, P256, P256, P256, P256, NULL, P256, P256, cap, NULL, P256, ws, NULL) ==
             CRISP_EINVAL, "null route");
  EXPECT(crisp_route_select(&s, &p, P256, P256, P256, P256, P256, P256, P2, P256, cap, NULL, P256, ws, NULL) ==
             CRISP_EINVAL, "misaligned row_ptr");
  EXPECT(crisp_route_select(&s, &p, P256, P256, P256, P256, P256, P256, P256, P256, cap, NULL, P256, 256, NULL) ==
             CRISP_EINVAL, "small workspace (select)");
  EXPECT(crisp_sparse_attn(&s, 0.f, P256, P256, P8, P256, P256, cap, P256, NULL, 0, NULL) == CRISP_EINVAL,
         "misaligned v");
  EXPECT(crisp_sparse_attn(&s, 0.f, P256, P256, P256, P256, P256, -1, P256, NULL, 0, NULL) == CRISP_EINVAL,
         "negative capacity");
  EXPECT(crisp_sparse_attn(&s, 0.f, P256, P256, P256, P256, P256, cap, P256, P256, sws - 1, NULL) == CRISP_EINVAL,
         "small sparse workspace");
  EXPECT(crisp_sparse_attn(&s, 0.f, P256, P256, P256, P256, P256, cap, P256, P16, sws, NULL) == CRISP_EINVAL,
         "sparse workspace not 256-aligned");
  EXPECT(crisp_sparse_attn_noalloc(&s, 0.f, P256, P256, P8, P256, P256, cap, P256, NULL) == CRISP_EINVAL,
         "misaligned v (no-alloc)");
  EXPECT(crisp_sparse_attn_noalloc(&s, 0.f, P256, P256, P256, NULL, P256, cap, P256, NULL) == CRISP_EINVAL,
         "null row_ptr (no-alloc)");
  EXPECT(crisp_sparse_attn_noalloc(&s, 0.f, P256, P256, P256, P256, P256, -1, P256, NULL) == CRISP_EINVAL,
         "negative capacity (no-alloc)");
  EXPECT(crisp_sparse_attn_noalloc(&s, NAN, P256, P256, P256, P256, P256, cap, P256, NULL) == CRISP_EINVAL,
         "NaN scale (no-alloc)");
  {
    /* 128 heads x 32768 blocks: the work list alone is one int past the static area */
    crisp_shape big = shape(128, 1, 1 << 21, 128, 64);
    EXPECT(crisp_sparse_attn_noalloc(&big, 0.f, P256, P256, P256, P256, P256, (int64_t)1 << 40, P256, NULL) ==
               CRISP_EINVAL && strstr(crisp_last_error(), "static area") != NULL,
           "layer too large for the static schedule area");
  }
  EXPECT(crisp_dense_attn(&s, 0.f, P256, P256, P256, NULL, NULL) == CRISP_EINVAL, "null o (dense)");
  EXPECT(crisp_prefill_attn(&s, &p, P256, P256, P256, P256, P256, NULL, P256, P256, pws, NULL) == CRISP_EINVAL,
         "lists partly given");
  EXPECT(crisp_prefill_attn(&s, &p, P256, P256, P256, P256, NULL, NULL, NULL, P256, pws - 1, NULL) == CRISP_EINVAL,
         "prefill workspace one short");
  EXPECT(crisp_prefill_attn(&s, &p, P256, P256, P256, P256, P256, P256, P256, P256, ws - 1, NULL) == CRISP_EINVAL,
         "workspace one short with lists given");
  EXPECT(crisp_prefill_attn(&s, &p, P256, P256, P256, P256, P256, P2, P256, P256, pws, NULL) == CRISP_EINVAL,
         "misaligned row_ptr (prefill)");
}

static void check_empty(void) {
  crisp_params p;
  crisp_params_default(&p);
  crisp_shape e1 = shape(4, 2, 0, 128, 128), e2 = shape(0, 2, 4096, 128, 64);
  const crisp_shape* es[2] = {&e1, &e2};
  for (int i = 0; i < 2; ++i) {
    const crisp_shape* s = es[i];
    EXPECT(crisp_estimate(s, &p, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL) == CRISP_OK, "empty estimate %d", i);
    EXPECT(crisp_jsd(s, &p, NULL, NULL, NULL, NULL, NULL, 0, NULL) == CRISP_OK, "empty jsd %d", i);
    EXPECT(crisp_route_select(s, &p, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL, NULL, 0, NULL) ==
               CRISP_OK, "empty select %d", i);
    EXPECT(crisp_sparse_attn(s, 0.f, NULL, NULL, NULL, NULL, NULL, 0, NULL, NULL, 0, NULL) == CRISP_OK,
           "empty sparse %d", i);
    EXPECT(crisp_prefill_attn(s, &p, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL) == CRISP_OK,
           "empty prefill %d", i);
    EXPECT(crisp_dense_attn(s, 0.f, NULL, NULL, NULL, NULL, NULL) == CRISP_OK, "empty dense %d", i);
    EXPECT(crisp_sparse_attn_noalloc(s, 0.f, NULL, NULL, NULL, NULL, NULL, 0, NULL, NULL) == CRISP_OK,
           "empty no-alloc sparse %d", i);
  }
}

static void* other_thread(void* arg) {
  (void)arg;
  crisp_shape s = shape(4, 2, 4096, 64, 128);
  crisp_status st = crisp_dense_attn(&s, 0.f, P256, P256, P256, P256, NULL);
  int ok = st == CRISP_EUNSUPPORTED && strstr(crisp_last_error(), "head_dim") != NULL;
  return ok ? P256 : NULL;
}

static void check_messages(void) {
  EXPECT(strcmp(crisp_status_string(CRISP_OK), "CRISP_OK") == 0, "OK string");
  EXPECT(strcmp(crisp_status_string(CRISP_EINVAL), "CRISP_EINVAL") == 0, "EINVAL string");
  EXPECT(strcmp(crisp_status_string(CRISP_EUNSUPPORTED), "CRISP_EUNSUPPORTED") == 0, "EUNSUPPORTED string");
  EXPECT(strcmp(crisp_status_string(CRISP_EHIP), "CRISP_EHIP") == 0, "EHIP string");
  EXPECT(strcmp(crisp_status_string((crisp_status)7), "CRISP_UNKNOWN") == 0, "unknown status string");
  /* the calling thread's message is its own */
  crisp_shape s = shape(3, 2, 4096, 128, 128);
  crisp_dense_attn(&s, 0.f, P256, P256, P256, P256, NULL);
  char mine[512];
  snprintf(mine, sizeof(mine), "%s", crisp_last_error());
  EXPECT(strstr(mine, "multiple") != NULL, "GQA message: %s", mine);
  pthread_t t;
  void* res = NULL;
  pthread_create(&t, NULL, other_thread, NULL);
  pthread_join(t, &res);
  EXPECT(res != NULL, "other thread saw its own error");
  EXPECT(strcmp(mine, crisp_last_error()) == 0, "message unchanged by another thread's failure");
}

/* With no GPU, a call that passes validation reaches its first launch, which fails:
 * the status must be CRISP_EHIP with a message naming the call. */
static void check_launch_failure(void) {
  crisp_shape s = shape(2, 1, 1024, 128, 128);
  crisp_params p;
  crisp_params_default(&p);
  crisp_status st = crisp_dense_attn(&s, 0.f, P256, P256, P256, P256, NULL);
  EXPECT(st == CRISP_EHIP && strstr(crisp_last_error(), "crisp_dense_attn") != NULL, "dense launch failure: %s",
         crisp_status_string(st));
  st = crisp_sparse_attn_noalloc(&s, 0.f, P256, P256, P256, P256, P256, crisp_col_capacity(&s), P256, NULL);
  EXPECT(st == CRISP_EHIP && strstr(crisp_last_error(), "crisp_sparse_attn_noalloc") != NULL,
         "no-alloc sparse launch failure: %s", crisp_status_string(st));
  size_t ws = 0;
  crisp_workspace_size(&s, &ws);
  st = crisp_estimate(&s, &p, P256, P256, P256, P256, P256, P256, ws, NULL);
  EXPECT(st == CRISP_EHIP && strstr(crisp_last_error(), "crisp_estimate") != NULL, "estimate launch failure: %s",
         crisp_status_string(st));
}

int main(void) {
  check_defaults();
  check_sizes();
  check_shapes();
  check_params();
  check_pointers();
  check_empty();
  check_messages();
  check_launch_failure();
  printf("%d checks, %d failures\n", checks, failures);
  return failures ? 1 : 0;
}
