// Host-side checks of the C ABI, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code (tests/test_host_sanitizers.py
// builds and runs it): the segment validator on valid, invalid and random
// arrays, and every entry point's argument checks, which must all fail
// before the library touches a device. Exit status 0 when every expected
// status matched; the sanitizers abort the process on any memory error or
// undefined behaviour.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <random>
#include <vector>

#include "ism_attn.h"

static int g_fail = 0;

#define EXPECT(expr, want)                                                        \
  do {                                                                            \
    const int got_ = (int)(expr);                                                 \
    if (got_ != (want)) {                                                         \
      fprintf(stderr, "%s:%d: %s -> %d, expected %d (%s)\n", __FILE__, __LINE__,  \
              #expr, got_, (int)(want), ism_last_error());                        \
      ++g_fail;                                                                   \
    }                                                                             \
  } while (0)

static void *const FAKE = (void *)0x1000;  // never dereferenced

static ism_status check(const std::vector<int32_t> &cu, const std::vector<int32_t> &cs,
                        const std::vector<uint8_t> &fl, int32_t total, int32_t maxlen) {
  // exact-size heap copies, so that any read past an array is an ASan error
  int32_t *a = (int32_t *)malloc(cu.size() * 4 + 1);
  int32_t *b = (int32_t *)malloc(cs.size() * 4 + 1);
  uint8_t *c = (uint8_t *)malloc(fl.size() + 1);
  memcpy(a, cu.data(), cu.size() * 4);
  memcpy(b, cs.data(), cs.size() * 4);
  if (!fl.empty()) memcpy(c, fl.data(), fl.size());
  const ism_status s = ism_check_segments_host(a, b, c, (int32_t)cu.size() - 1,
                                               (int32_t)fl.size(), total, maxlen);
  free(a);
  free(b);
  free(c);
  return s;
}

static void validator_cases() {
  // [Q 3, A 2, Q 2] + [A 2, Q 1]
  EXPECT(check({0, 7, 10}, {0, 3, 5, 7, 9, 10}, {1, 0, 1, 0, 1}, 10, 7), ISM_OK);
  EXPECT(check({0, 1}, {0, 1}, {1}, 1, 1), ISM_OK);
  EXPECT(check({0, 5}, {0, 2, 2, 5}, {1, 0, 1}, 5, 100), ISM_ERR_SEGMENTS);  // empty segment
  EXPECT(check({0, 5}, {0, 3, 2, 5}, {1, 0, 1}, 5, 100), ISM_ERR_SEGMENTS);  // reversed
  EXPECT(check({0, 3, 6}, {0, 2, 6}, {1, 0}, 6, 100), ISM_ERR_SEGMENTS);     // straddles
  EXPECT(check({0, 6}, {0, 2, 5}, {1, 0}, 6, 100), ISM_ERR_SEGMENTS);        // last != total
  EXPECT(check({1, 6}, {1, 2, 6}, {1, 0}, 6, 100), ISM_ERR_SEGMENTS);        // not from 0
  EXPECT(check({0, 0, 4}, {0, 4}, {1}, 4, 100), ISM_ERR_SHAPE);              // empty dialogue
  EXPECT(check({0, 10}, {0, 4, 10}, {1, 0}, 10, 9), ISM_ERR_SHAPE);          // max_seqlen
  EXPECT(ism_check_segments_host(nullptr, (int32_t *)FAKE, (uint8_t *)FAKE, 1, 1, 1, 1),
         ISM_ERR_NULL);
  EXPECT(check({0, 4}, {0, 4}, {1}, 4, 4) == ISM_OK && ism_last_error()[0] == 0, 1);
}

// Random arrays, valid and invalid, with the declared lengths: the
// validator must answer without reading outside them.
static void validator_fuzz() {
  std::mt19937 rng(2408);
  for (int it = 0; it < 20000; ++it) {
    const int batch = 1 + (int)(rng() % 6);
    const int nseg = batch + (int)(rng() % 12);
    std::vector<int32_t> cu(batch + 1), cs(nseg + 1);
    std::vector<uint8_t> fl(nseg);
    const bool sane = rng() % 2;
    int32_t t = 0;
    for (int g = 0; g <= nseg; ++g) {
      cs[g] = sane ? t : (int32_t)(rng() % 64) - 8;
      t += 1 + (int32_t)(rng() % 9);
    }
    const int32_t total = sane ? cs[nseg] : (int32_t)(rng() % 80);
    for (int b = 0; b <= batch; ++b)
      cu[b] = sane ? cs[(int64_t)b * nseg / batch] : (int32_t)(rng() % 64) - 8;
    for (auto &f : fl) f = (uint8_t)(rng() % 3);
    const int32_t maxlen = (int32_t)(rng() % 100);
    const ism_status s = check(cu, cs, fl, total, maxlen);
    if (s != ISM_OK && s != ISM_ERR_SEGMENTS && s != ISM_ERR_SHAPE) {
      fprintf(stderr, "fuzz %d: unexpected status %d\n", it, (int)s);
      ++g_fail;
    }
  }
}

static ism_segments segs(int32_t batch, int32_t nseg, int32_t total, int32_t maxlen) {
  ism_segments s;
  s.cu_seqlens = (const int32_t *)FAKE;
  s.cu_segs = (const int32_t *)FAKE;
  s.seg_is_query = (const uint8_t *)FAKE;
  s.batch = batch;
  s.num_segs = nseg;
  s.total_tokens = total;
  s.max_seqlen = maxlen;
  return s;
}

static void argument_cases() {
  void *ws = (void *)(0x1000 * 256);
  const size_t big = 1 << 20;
  ism_segments sg = segs(1, 1, 10, 10);
  EXPECT(ism_attn_fwd(&sg, nullptr, FAKE, FAKE, FAKE, nullptr, 1, 1, 64, 0.125f, ws, big,
                      nullptr), ISM_ERR_NULL);
  EXPECT(ism_attn_fwd(nullptr, FAKE, FAKE, FAKE, FAKE, nullptr, 1, 1, 64, 0.125f, ws, big,
                      nullptr), ISM_ERR_NULL);
  EXPECT(ism_attn_fwd(&sg, FAKE, FAKE, FAKE, FAKE, nullptr, 3, 2, 64, 0.125f, ws, big,
                      nullptr), ISM_ERR_SHAPE);
  EXPECT(ism_attn_fwd(&sg, FAKE, FAKE, FAKE, FAKE, nullptr, 1, 1, 96, 0.125f, ws, big,
                      nullptr), ISM_ERR_UNSUPPORTED);
  EXPECT(ism_attn_fwd(&sg, FAKE, FAKE, FAKE, FAKE, nullptr, 1, 1, 64, -1.f, ws, big,
                      nullptr), ISM_ERR_SHAPE);
  EXPECT(ism_attn_fwd(&sg, FAKE, FAKE, FAKE, FAKE, nullptr, 1, 1, 64, 0.125f, ws, 4,
                      nullptr), ISM_ERR_WORKSPACE);
  EXPECT(ism_attn_fwd(&sg, FAKE, FAKE, FAKE, FAKE, nullptr, 1, 1, 64, 0.125f, nullptr, 0,
                      nullptr), ISM_ERR_WORKSPACE);
  EXPECT(ism_attn_fwd(&sg, FAKE, FAKE, FAKE, FAKE, nullptr, 1, 1, 64, 0.125f,
                      (char *)ws + 4, big, nullptr), ISM_ERR_WORKSPACE);
  ism_segments sg2 = segs(1, 1, 10, 11);
  EXPECT(ism_attn_fwd(&sg2, FAKE, FAKE, FAKE, FAKE, nullptr, 1, 1, 64, 0.125f, ws, big,
                      nullptr), ISM_ERR_SHAPE);
  EXPECT(ism_attn_bwd(&sg, FAKE, FAKE, FAKE, FAKE, (float *)FAKE, FAKE, nullptr,
                      (float *)FAKE, (float *)FAKE, 1, 1, 64, 0.125f, 0, ws, big, nullptr),
         ISM_ERR_NULL);
  EXPECT(ism_attn_bwd(&sg, FAKE, FAKE, FAKE, FAKE, (float *)FAKE, FAKE, (float *)FAKE,
                      (float *)FAKE, (float *)FAKE, 8, 3, 64, 0.125f, 1, ws, big, nullptr),
         ISM_ERR_SHAPE);
  EXPECT(ism_visibility(&sg, nullptr, (int32_t *)FAKE, nullptr), ISM_ERR_NULL);
  EXPECT(ism_attn_decode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, (const int32_t *)FAKE, 1, 0, FAKE,
                         nullptr, 3, 2, 64, 0.125f, 0, ws, big, nullptr), ISM_ERR_SHAPE);
  EXPECT(ism_attn_decode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, (const int32_t *)FAKE, 1, 65, FAKE,
                         nullptr, 1, 1, 64, 0.125f, 0, ws, big, nullptr), ISM_ERR_CAPACITY);
  EXPECT(ism_attn_decode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, (const int32_t *)FAKE, 1, 0, FAKE,
                         nullptr, 1, 1, 64, 0.125f, 0, ws, 8, nullptr), ISM_ERR_WORKSPACE);
  EXPECT(ism_attn_decode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, (const int32_t *)FAKE, 1, 0, FAKE,
                         nullptr, 1, 1, 64, 0.125f, 5000, ws, big, nullptr), ISM_ERR_SHAPE);
  EXPECT(ism_attn_decode_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, 64, (const int32_t *)FAKE, 64, 0,
                                 FAKE, nullptr, 64, 64, 128, 0.125f, 64, nullptr),
         ISM_ERR_WORKSPACE);
  EXPECT(ism_attn_prefill_cached((const int32_t *)FAKE, 1, 10, 10, FAKE, FAKE, FAKE, FAKE,
                                 FAKE, 8, (const int32_t *)FAKE, FAKE, nullptr, 1, 1, 64,
                                 0.125f, nullptr, 0, nullptr), ISM_ERR_CAPACITY);
  EXPECT(ism_attn_prefill_cached((const int32_t *)FAKE, 1, 10, 10, FAKE, FAKE, FAKE, nullptr,
                                 FAKE, 64, (const int32_t *)FAKE, FAKE, nullptr, 1, 1, 64,
                                 0.125f, nullptr, 0, nullptr), ISM_ERR_NULL);
  EXPECT(ism_attn_prefill_cached((const int32_t *)FAKE, 1, 10, 11, FAKE, FAKE, FAKE, FAKE,
                                 FAKE, 64, (const int32_t *)FAKE, FAKE, nullptr, 1, 1, 64,
                                 0.125f, nullptr, 0, nullptr), ISM_ERR_SHAPE);
  for (int ps : {96, 0, -64})
    EXPECT(ism_attn_prefill_paged((const int32_t *)FAKE, 1, 10, 10, 1, FAKE, FAKE, FAKE, FAKE,
                                  FAKE, 4, ps, (const int32_t *)FAKE, 2, (const int32_t *)FAKE,
                                  FAKE, nullptr, 1, 1, 64, 0.125f, nullptr, 0, nullptr),
           ISM_ERR_UNSUPPORTED);
  EXPECT(ism_attn_decode_paged(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 64, nullptr, 2,
                               (const int32_t *)FAKE, 1, 0, FAKE, nullptr, 1, 1, 64, 0.125f, 0,
                               ws, big, nullptr), ISM_ERR_NULL);
  EXPECT(ism_attn_decode_paged(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 64, (const int32_t *)FAKE,
                               1 << 30, (const int32_t *)FAKE, 1, 0, FAKE, nullptr, 1, 1, 64,
                               0.125f, 0, ws, big, nullptr), ISM_ERR_SHAPE);
  EXPECT(ism_rope2d(nullptr, 0, 4, 1, 64, (const int32_t *)FAKE, (const int32_t *)FAKE,
                    10000.f, 0, nullptr), ISM_ERR_NULL);
  EXPECT(ism_rope2d(FAKE, 2, 4, 1, 64, (const int32_t *)FAKE, (const int32_t *)FAKE, 10000.f,
                    0, nullptr), ISM_ERR_UNSUPPORTED);
  EXPECT(ism_rope2d(FAKE, 0, 4, 1, 64, (const int32_t *)FAKE, (const int32_t *)FAKE, 1.f, 0,
                    nullptr), ISM_ERR_SHAPE);
  ism_segments sg3 = segs(2, 1, 10, 10);
  EXPECT(ism_positions_2d(&sg3, (int32_t *)FAKE, (int32_t *)FAKE, nullptr), ISM_ERR_SHAPE);
  // workspace sizes, including extreme arguments
  EXPECT(ism_attn_workspace_size(ISM_OP_FWD, 1, 1000, 1000, 4, 4, 64, 0) % 256, 0);
  EXPECT(ism_attn_workspace_size(ISM_OP_DECODE, 1, 0, 100, 3, 0, 64, 0), 0);
  EXPECT(ism_attn_workspace_size(ISM_OP_DECODE, 2, 0, 1 << 30, 64, 1, 128, 0) > 0, 1);
  EXPECT(ism_attn_workspace_size(99, 1, 1, 1, 1, 1, 64, 0), 0);
  for (int s = 0; s < 12; ++s) EXPECT(ism_status_string((ism_status)s) != nullptr, 1);
}

int main() {
  validator_cases();
  validator_fuzz();
  argument_cases();
  if (g_fail) {
    fprintf(stderr, "%d check(s) failed\n", g_fail);
    return 1;
  }
  printf("host ABI checks passed\n");
  return 0;
}
