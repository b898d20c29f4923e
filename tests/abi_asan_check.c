/* Drives the host-side paths of libarctopk that need no device: status
 * strings, the host projection, configuration checks (every rejection),
 * the create-time planning of valid layouts (single view, buckets, per-tensor
 * views of many widths, the comparison compressors, and 300 seeded random
 * layouts) and the NULL-context paths.  Built against a copy of the library whose host code carries
 * AddressSanitizer; prints "ok" when every check holds.
 *
 * Without a device, arc_create of a valid configuration plans the layout,
 * then fails at the first HIP call with ARC_ERR_DEVICE and releases what it
 * built; with one, it succeeds and the context is destroyed at once. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "libarctopk.h"

static int failures = 0;

#define CHECK(cond)                                                      \
  do {                                                                   \
    if (!(cond)) {                                                       \
      fprintf(stderr, "check failed at line %d: %s (%s)\n", __LINE__,   \
              #cond, arc_last_error());                                  \
      ++failures;                                                        \
    }                                                                    \
  } while (0)

static arc_config base(void) {
  arc_config c;
  memset(&c, 0, sizeof c);
  c.d = 4096;
  c.n = 64;
  c.K = 3;
  c.seed = 1;
  c.N = 2;
  c.r = 4;
  c.eta = 0.1f;
  return c;
}

static void expect_invalid(const arc_config* c, int line) {
  arc_ctx* out = (arc_ctx*)(void*)0x1;
  const arc_status st = arc_create(c, NULL, &out);
  if (st != ARC_ERR_INVALID || out != NULL || arc_last_error()[0] == '\0') {
    fprintf(stderr, "config of line %d: status %d, out %p\n", line, (int)st, (void*)out);
    ++failures;
  }
}

static void expect_planned(const arc_config* c, int line) {
  arc_ctx* out = NULL;
  const arc_status st = arc_create(c, NULL, &out);
  if (st == ARC_OK) {
    CHECK(out != NULL);
    char buf[512];
    CHECK(arc_describe(out, buf, (int64_t)sizeof buf) == ARC_OK);
    CHECK(strlen(buf) < sizeof buf);
    CHECK(arc_describe(out, buf, 7) == ARC_OK && strlen(buf) == 6);
    CHECK(arc_num_rows(out) > 0 && arc_selected_rows(out) >= 0 && arc_payload_elems(out) >= 0);
    CHECK(arc_destroy(out) == ARC_OK);
  } else if (st != ARC_ERR_DEVICE || out != NULL) {
    fprintf(stderr, "config of line %d: status %d (%s)\n", line, (int)st, arc_last_error());
    ++failures;
  }
}

int main(void) {
  /* status strings */
  for (int s = 0; s <= 5; ++s) CHECK(arc_status_str((arc_status)s) != NULL);
  CHECK(strcmp(arc_status_str((arc_status)99), "ARC_ERR_UNKNOWN") == 0);

  /* host projection, several widths, and its rejections */
  {
    const int64_t widths[] = {1, 3, 147, 768, 2048, 4609};
    const int32_t rs[] = {1, 4, 7, 32};
    for (size_t w = 0; w < sizeof widths / sizeof widths[0]; ++w)
      for (size_t k = 0; k < sizeof rs / sizeof rs[0]; ++k) {
        float* V = (float*)malloc(sizeof(float) * (size_t)(widths[w] * rs[k]));
        CHECK(V != NULL);
        CHECK(arc_projection(2003u + w, (int64_t)k * 7, widths[w], rs[k], V) == ARC_OK);
        free(V);
      }
    float V[16];
    CHECK(arc_projection(1, -1, 4, 4, V) == ARC_ERR_INVALID);
    CHECK(arc_projection(1, 0, 0, 4, V) == ARC_ERR_INVALID);
    CHECK(arc_projection(1, 0, 4, 0, V) == ARC_ERR_INVALID);
    CHECK(arc_projection(1, 0, 4, ARC_MAX_R + 1, V) == ARC_ERR_INVALID);
    CHECK(arc_projection(1, 0, 4, 4, NULL) == ARC_ERR_INVALID);
  }

  /* configuration rejections */
  {
    arc_config c;
    c = base(); c.d = 0; expect_invalid(&c, __LINE__);
    c = base(); c.d = -5; expect_invalid(&c, __LINE__);
    c = base(); c.n = 0; expect_invalid(&c, __LINE__);
    c = base(); c.N = 0; expect_invalid(&c, __LINE__);
    c = base(); c.N = 70000; expect_invalid(&c, __LINE__);
    c = base(); c.r = 0; expect_invalid(&c, __LINE__);
    c = base(); c.r = ARC_MAX_R + 1; expect_invalid(&c, __LINE__);
    c = base(); c.K = -1; expect_invalid(&c, __LINE__);
    c = base(); c.eta = -0.01f; expect_invalid(&c, __LINE__);
    c = base(); c.eta = 1.5f; expect_invalid(&c, __LINE__);
    c = base(); c.grad_dtype = 7; expect_invalid(&c, __LINE__);
    c = base(); c.reserved = 1; expect_invalid(&c, __LINE__);
    c = base(); c.compressor = 3; expect_invalid(&c, __LINE__);
    c = base(); c.d = (int64_t)3 << 31; c.n = 1; expect_invalid(&c, __LINE__);
    c = base(); c.num_buckets = 2; expect_invalid(&c, __LINE__); /* NULL arrays */
    {
      const int64_t begin_bad_end[] = {0, 10, 63}, begin_bad_start[] = {1, 10, 64},
                    begin_empty[] = {0, 10, 10, 64}, ks[] = {1, 1, 1}, kneg[] = {1, -2};
      const int64_t begin_ok[] = {0, 10, 64};
      c = base(); c.num_buckets = 2; c.bucket_row_begin = begin_bad_end; c.bucket_K = ks;
      expect_invalid(&c, __LINE__);
      c.bucket_row_begin = begin_bad_start; expect_invalid(&c, __LINE__);
      c.num_buckets = 3; c.bucket_row_begin = begin_empty; expect_invalid(&c, __LINE__);
      c.num_buckets = 2; c.bucket_row_begin = begin_ok; c.bucket_K = kneg;
      expect_invalid(&c, __LINE__);
    }
    {
      const arc_tensor short_by_one[] = {{64, 96, 5}, {1, 299, 1}};
      const arc_tensor empty[] = {{0, 96, 5}, {1, 6444, 1}};
      const arc_tensor zero_width[] = {{64, 0, 5}, {1, 6444, 1}};
      const arc_tensor overflow[] = {{(int64_t)1 << 40, (int64_t)1 << 40, 1}};
      c = base(); c.n = 0; c.K = 0; c.d = 64 * 96 + 300; c.num_tensors = 2;
      c.tensors = short_by_one; expect_invalid(&c, __LINE__);
      c.tensors = empty; expect_invalid(&c, __LINE__);
      c.tensors = zero_width; expect_invalid(&c, __LINE__);
      c.tensors = NULL; expect_invalid(&c, __LINE__);
      c.tensors = overflow; c.num_tensors = 1; c.d = (int64_t)1 << 40;
      expect_invalid(&c, __LINE__);
    }
    CHECK(arc_create(NULL, NULL, NULL) == ARC_ERR_INVALID);
    c = base();
    CHECK(arc_create(&c, NULL, NULL) == ARC_ERR_INVALID);
  }

  /* valid layouts: planned on the host */
  {
    arc_config c = base();
    expect_planned(&c, __LINE__);
    c.d = 11689512; c.n = 512; c.K = 229; c.N = 8; expect_planned(&c, __LINE__);
    c.d = 1000; c.n = 7; c.K = 1000; expect_planned(&c, __LINE__); /* K >= m, width 7 */
    c.d = 4096; c.n = 1; c.r = 1; c.K = 10; expect_planned(&c, __LINE__);
    c = base(); c.d = 262144; c.n = 4096; c.r = 3; c.K = 5; expect_planned(&c, __LINE__);
    c = base(); c.compressor = ARC_COMP_RANDK; expect_planned(&c, __LINE__);
    c = base(); c.compressor = ARC_COMP_TOPK; c.N = 4; expect_planned(&c, __LINE__);
    {
      const int64_t begin[] = {0, 10, 30, 64}, ks[] = {2, 0, 100};
      c = base(); c.num_buckets = 3; c.bucket_row_begin = begin; c.bucket_K = ks;
      expect_planned(&c, __LINE__);
    }
    {
      /* a ResNet-like mix: conv views out x (in*kh*kw), 1-D tensors, a
       * classifier, widths multiple of 4 and not, long and short tensors */
      const arc_tensor t[] = {{64, 147, 7}, {1, 64, 1}, {1, 64, 1},   {64, 576, 1},
                              {128, 576, 2}, {128, 1152, 2}, {128, 64, 2}, {1, 128, 1},
                              {512, 4608, 6}, {1000, 512, 10}, {1, 1000, 1}, {3, 5, 9}};
      int64_t d = 0;
      for (size_t k = 0; k < sizeof t / sizeof t[0]; ++k) d += t[k].rows * t[k].cols;
      c = base(); c.n = 0; c.K = 0; c.d = d; c.N = 3; c.tensors = t;
      c.num_tensors = (int32_t)(sizeof t / sizeof t[0]);
      expect_planned(&c, __LINE__);
      c.grad_dtype = ARC_DTYPE_BF16; c.r = 8; expect_planned(&c, __LINE__);
      c.compressor = ARC_COMP_TOPK; expect_planned(&c, __LINE__);
      c.compressor = ARC_COMP_RANDK; expect_planned(&c, __LINE__);
    }
  }

  /* seeded random layouts through the planner (single views with buckets,
   * per-tensor mixes, every compressor) */
  {
    uint64_t x = 0x9E3779B97F4A7C15ull;
#define NEXT() (x = x * 6364136223846793005ull + 1442695040888963407ull, (x >> 33))
    for (int it = 0; it < 300; ++it) {
      arc_config c = base();
      c.N = 1 + (int32_t)(NEXT() % 9);
      c.r = 1 + (int32_t)(NEXT() % 8);
      c.compressor = (int32_t)(NEXT() % 3);
      c.grad_dtype = (int32_t)(NEXT() % 2);
      arc_tensor t[12];
      int64_t begin[6], ks[5];
      if (it % 2 == 0) {
        const int64_t widths[] = {1, 3, 4, 7, 64, 100, 147, 256, 512, 768, 2048, 4608};
        const int nt = 1 + (int)(NEXT() % 12);
        int64_t d = 0;
        for (int k = 0; k < nt; ++k) {
          t[k].cols = widths[NEXT() % 12];
          t[k].rows = 1 + (int64_t)(NEXT() % 700);
          t[k].K = (int64_t)(NEXT() % (uint64_t)(t[k].rows + 3));
          d += t[k].rows * t[k].cols;
        }
        c.n = 0;
        c.K = 0;
        c.d = d;
        c.tensors = t;
        c.num_tensors = nt;
      } else {
        c.n = 1 + (int64_t)(NEXT() % 5000);
        c.d = 1 + (int64_t)(NEXT() % 3000000);
        const int64_t m = (c.d + c.n - 1) / c.n;
        c.K = (int64_t)(NEXT() % (uint64_t)(m + 2));
        if (m >= 5 && NEXT() % 2) {
          const int nb = 1 + (int)(NEXT() % 4);
          begin[0] = 0;
          for (int b = 1; b < nb; ++b) begin[b] = begin[b - 1] + 1 + (int64_t)(NEXT() % (uint64_t)(m / nb));
          begin[nb] = m;
          for (int b = 0; b < nb; ++b) ks[b] = (int64_t)(NEXT() % 50);
          c.num_buckets = nb;
          c.bucket_row_begin = begin;
          c.bucket_K = ks;
          c.K = 0;
        }
      }
      expect_planned(&c, __LINE__);
    }
#undef NEXT
  }

  /* NULL-context paths */
  {
    arc_model_config mc;
    memset(&mc, 0, sizeof mc);
    mc.lr = 0.1f;
    float buf[4];
    int64_t steps = 0;
    double ms[ARC_NUM_STAGES];
    char text[16];
    CHECK(arc_destroy(NULL) == ARC_OK);
    CHECK(arc_num_rows(NULL) == -1 && arc_selected_rows(NULL) == -1 &&
          arc_payload_elems(NULL) == -1);
    CHECK(arc_step(NULL, 0, buf, buf, buf, NULL, buf) == ARC_ERR_INVALID);
    CHECK(arc_model_step(NULL, &mc, 0, buf, buf, buf, buf, buf, NULL, NULL, NULL, buf) ==
          ARC_ERR_INVALID);
    CHECK(arc_model_step(NULL, NULL, 0, buf, buf, buf, buf, buf, NULL, NULL, NULL, buf) ==
          ARC_ERR_INVALID);
    CHECK(arc_describe(NULL, text, (int64_t)sizeof text) == ARC_ERR_INVALID);
    CHECK(arc_debug_sigma(NULL, buf) == ARC_ERR_INVALID);
    CHECK(arc_debug_sketch(NULL, buf) == ARC_ERR_INVALID);
    CHECK(arc_debug_projection(NULL, 0, buf) == ARC_ERR_INVALID);
    CHECK(arc_set_projection(NULL, buf) == ARC_ERR_INVALID);
    CHECK(arc_timing_enable(NULL, 1) == ARC_ERR_INVALID);
    CHECK(arc_timing_read(NULL, ms, &steps) == ARC_ERR_INVALID);
  }

  if (failures) {
    printf("%d failures\n", failures);
    return 1;
  }
  printf("ok\n");
  return 0;
}
