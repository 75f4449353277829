/*
 * Host-side exercise of the library under AddressSanitizer and
 * UndefinedBehaviorSanitizer (built by tests/test_sanitizers.py with the
 * device code left out).  It calls every entry point that runs without a
 * GPU -- plan enumeration and ranking, explicit tilings, the Eq. (1),
 * closed-form and two-level byte models, the variant table, status strings
 * -- over the benchmark shapes, edge shapes, shapes whose element counts
 * overflow the kernels' indexing, and a few thousand pseudo-random small
 * shapes, plus the argument and plan checks that reject a call before any
 * HIP call.  It prints one line and exits 0 when every call returned a
 * status code of the documented set; the sanitizers abort on the first
 * memory or undefined-behaviour error.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "cnn.h"

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;

/* splitmix64 (Steele, Lea and Flood, 2014) */
static uint64_t next_u64(void) {
  uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

static int64_t pick(int64_t lo, int64_t hi) { return lo + (int64_t)(next_u64() % (uint64_t)(hi - lo + 1)); }

static long calls = 0;
static int bad = 0;

static void check_status(const char* what, int st) {
  ++calls;
  if (st > 0 || st < CNN_E_PLAN) {
    fprintf(stderr, "%s: status %d outside the documented set\n", what, st);
    bad = 1;
  }
  if (st != CNN_OK && (!cnn_last_error() || !cnn_strerror(st))) {
    fprintf(stderr, "%s: missing error text\n", what);
    bad = 1;
  }
}

static const cnn_budget budgets[] = {
    {256, 160 * 1024, 128, 2},
    {1, 16 * 1024, 32, 1},
    {80, 64 * 1024, 64, 4},
};

/* Device addresses that are never dereferenced: every call below is
 * rejected by the library's checks, which only compare address ranges. */
static void* const kFakeIn = (void*)((uintptr_t)1 << 44);
static void* const kFakeKer = (void*)((uintptr_t)2 << 44);
static void* const kFakeOut = (void*)((uintptr_t)3 << 44);

static const int64_t tile_choices[] = {0, 1, 7, 16, 32, 64, 96, 128, 256, 448, 1000, (int64_t)1 << 40};

static void exercise(const cnn_problem* p) {
  for (int dtype = -1; dtype <= 3; ++dtype) {
    for (size_t bi = 0; bi < sizeof(budgets) / sizeof(budgets[0]); ++bi) {
      const cnn_budget* bud = &budgets[bi];
      int n = 0;
      int st = cnn_plan_candidates(p, dtype, bud, NULL, 0, &n);
      check_status("cnn_plan_candidates(count)", st);
      if (st == CNN_OK && n > 0) {
        cnn_plan_t* c = (cnn_plan_t*)calloc((size_t)n, sizeof(cnn_plan_t));
        int n2 = 0;
        check_status("cnn_plan_candidates", cnn_plan_candidates(p, dtype, bud, c, n, &n2));
        for (int i = 0; i < n && i < n2; ++i) {
          double t[3];
          check_status("cnn_hbm_bytes", cnn_hbm_bytes(&c[i], 8, 4 << 20, t));
          check_status("cnn_hbm_bytes(1 xcd)", cnn_hbm_bytes(&c[i], 1, 1, t));
          cnn_plan_t q;
          check_status("cnn_plan_tiles(candidate)",
                       cnn_plan_tiles(p, dtype, c[i].kernel, c[i].tk, c[i].tp, c[i].tc, bud, &q));
          /* edited plans must be rejected before any HIP call */
          cnn_plan_t e = c[i];
          e.tp += 1;
          e.grid += 3;
          st = cnn_fwd_plan_ws(kFakeIn, kFakeKer, kFakeOut, p, dtype, &e, NULL, 0, NULL);
          check_status("cnn_fwd_plan_ws(edited)", st);
          if (st == CNN_OK) {
            fprintf(stderr, "edited plan (kernel %d variant %d) accepted\n", e.kernel, e.variant);
            bad = 1;
          }
          e = c[i];
          e.ws_bytes = CNN_STATIC_SCRATCH_BYTES + 16;
          st = cnn_fwd_plan_static(kFakeIn, kFakeKer, kFakeOut, p, dtype, &e, NULL);
          check_status("cnn_fwd_plan_static(too big)", st);
          if (st != CNN_E_UNSUPPORTED) bad = 1;
        }
        free(c);
      }
      cnn_plan_t pl;
      check_status("cnn_plan", cnn_plan(p, dtype, bud, &pl));
      for (int k = 0; k <= 15; ++k) {
        for (int j = 0; j < 4; ++j) {
          const int64_t tk = tile_choices[pick(0, 11)];
          const int64_t tp = tile_choices[pick(0, 11)];
          const int64_t tc = tile_choices[pick(0, 11)];
          check_status("cnn_plan_tiles", cnn_plan_tiles(p, dtype, k, tk, tp, tc, bud, &pl));
          if (j == 0)
            check_status("cnn_plan_tiles(0)", cnn_plan_tiles(p, dtype, k, 0, 0, 0, bud, &pl));
        }
      }
    }
  }
  double terms[3], fp = 0.0;
  for (int j = 0; j < 8; ++j) {
    cnn_tiles t = {pick(1, 8), pick(1, 300), pick(1, 300), pick(1, 64), pick(1, 64)};
    check_status("cnn_eq1_cost(0)", cnn_eq1_cost(p, &t, 0, terms, &fp));
    check_status("cnn_eq1_cost(1)", cnn_eq1_cost(p, &t, 1, terms, NULL));
    check_status("cnn_slab_cost", cnn_slab_cost(p, pick(1, 512), pick(1, 4096), terms));
    cnn_closed_form_t cf;
    check_status("cnn_closed_form(0)", cnn_closed_form(p, (double)pick(1, 512), 80000.0, 0, &cf));
    check_status("cnn_closed_form(1)", cnn_closed_form(p, (double)pick(1, 512), 700.0, 1, &cf));
  }
}

int main(void) {
  /* benchmark shapes */
  const cnn_problem fixed[] = {
      {1, 16, 16, 16, 16, 3, 3, 1, 1},   {32, 64, 64, 56, 56, 3, 3, 1, 1},
      {64, 128, 256, 28, 28, 3, 3, 2, 2}, {256, 1024, 256, 14, 14, 1, 1, 1, 1},
      {64, 3, 64, 112, 112, 7, 7, 2, 2},  {64, 256, 512, 28, 28, 1, 1, 2, 2},
      {1, 512, 512, 7, 7, 3, 3, 1, 1},
      /* edges: one of everything, stride beyond the stencil, ragged sizes */
      {1, 1, 1, 1, 1, 1, 1, 1, 1},       {1, 1, 1, 1, 1, 7, 7, 3, 3},
      {3, 17, 33, 5, 31, 3, 3, 2, 2},     {2, 8, 8, 64, 1, 1, 1, 2, 1},
      /* indexing limits: element counts at and past 2^31 and 2^63 */
      {1 << 16, 1 << 8, 1 << 8, 1, 1 << 7, 1, 1, 1, 1},
      {(int64_t)1 << 40, 1 << 20, 1 << 20, 1 << 20, 1 << 20, 3, 3, 1, 1},
      {INT64_MAX / 2, 2, 2, 2, 2, 1, 1, 1, 1},
      {1, 1, 1, INT64_MAX / 4, 1, 1, 1, 4, 1},
      /* invalid sizes */
      {0, 1, 1, 1, 1, 1, 1, 1, 1},       {1, 1, 1, 1, 1, 1, 1, 0, 1},
      {-5, 1, 1, 1, 1, 1, 1, 1, 1},
  };
  for (size_t i = 0; i < sizeof(fixed) / sizeof(fixed[0]); ++i) exercise(&fixed[i]);
  for (int i = 0; i < 400; ++i) {
    cnn_problem p = {pick(1, 4), pick(1, 80), pick(1, 80), pick(1, 40), pick(1, 40),
                     pick(1, 7), pick(1, 7), pick(1, 3), pick(1, 3)};
    if (i % 5 == 0) { p.Nc = 16 * pick(1, 8); p.Nh = pick(1, 32); p.Nr = p.Ns = 3; p.sw = p.sh = 2; }
    if (i % 7 == 0) { p.Nc = 8 * pick(1, 16); p.Nr = p.Ns = 1; }
    exercise(&p);
  }
  /* NULL arguments */
  cnn_plan_t pl;
  int n = 0;
  const cnn_problem p0 = fixed[2];
  check_status("cnn_plan(NULL prob)", cnn_plan(NULL, CNN_BF16, &budgets[0], &pl));
  check_status("cnn_plan(NULL plan)", cnn_plan(&p0, CNN_BF16, &budgets[0], NULL));
  check_status("cnn_plan_candidates(NULL count)",
               cnn_plan_candidates(&p0, CNN_BF16, &budgets[0], NULL, 0, NULL));
  check_status("cnn_plan_candidates(NULL out)",
               cnn_plan_candidates(&p0, CNN_BF16, &budgets[0], NULL, 4, &n));
  check_status("cnn_fwd_plan(NULL)", cnn_fwd_plan(NULL, NULL, NULL, &p0, CNN_BF16, &pl, NULL));
  check_status("cnn_fwd_plan_static(NULL)",
               cnn_fwd_plan_static(NULL, NULL, NULL, &p0, CNN_BF16, NULL, NULL));
  check_status("cnn_hbm_bytes(NULL)", cnn_hbm_bytes(NULL, 8, 1, NULL));
  check_status("cnn_eq1_cost(NULL)", cnn_eq1_cost(NULL, NULL, 0, NULL, NULL));
  check_status("cnn_closed_form(NULL)", cnn_closed_form(&p0, 1.0, 1.0, 0, NULL));
  /* the variant table */
  check_status("cnn_variants(count)", cnn_variants(NULL, 0, &n));
  cnn_variant_t* v = (cnn_variant_t*)calloc((size_t)n + 1, sizeof(cnn_variant_t));
  int n2 = 0;
  check_status("cnn_variants", cnn_variants(v, n, &n2));
  check_status("cnn_variants(short)", cnn_variants(v, n / 2, &n2));
  check_status("cnn_variants(NULL)", cnn_variants(NULL, 3, &n2));
  free(v);
  for (int s = -10; s <= 2; ++s)
    if (!cnn_strerror(s)) bad = 1;
  if (cnn_abi_version() != CNN_ABI_VERSION) bad = 1;
  printf("lib host driver: %ld calls, %s\n", calls, bad ? "FAILED" : "ok");
  return bad;
}
