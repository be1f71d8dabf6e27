// Host-side validation of segment metadata and the thread-local error
// string. Pure C++ (no HIP), so it can be built and tested without a GPU.
#include <stdio.h>
#include <string.h>
#include <stdarg.h>

#include "../../include/ism_attn.h"
#include "ism_host.h"

namespace ism {

static thread_local char g_last_error[512] = "";

ism_status fail(ism_status s, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

void clear_error() { g_last_error[0] = '\0'; }

const char *last_error() { return g_last_error; }

}  // namespace ism

extern "C" const char *ism_last_error(void) { return ism::last_error(); }

extern "C" const char *ism_version(void) { return "0.1.0"; }

extern "C" const char *ism_status_string(ism_status s) {
  switch (s) {
    case ISM_OK: return "ok";
    case ISM_ERR_NULL: return "null pointer";
    case ISM_ERR_SHAPE: return "bad shape";
    case ISM_ERR_UNSUPPORTED: return "unsupported configuration";
    case ISM_ERR_SEGMENTS: return "invalid segment metadata";
    case ISM_ERR_WORKSPACE: return "workspace too small or misaligned";
    case ISM_ERR_CAPACITY: return "kv cache capacity exceeded";
    case ISM_ERR_NO_DEVICE: return "no usable gfx950 device";
    case ISM_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

// Invariants of the dialogue structure (Sec. 2.1 sample definition): both
// boundary arrays start at 0, end at total_tokens and strictly increase (no
// empty segment or dialogue); each dialogue boundary is a segment boundary,
// so no segment straddles two dialogues; max_seqlen bounds every dialogue.
extern "C" ism_status ism_check_segments_host(const int32_t *cu_seqlens,
                                              const int32_t *cu_segs,
                                              const uint8_t *seg_is_query,
                                              int32_t batch, int32_t num_segs,
                                              int32_t total_tokens,
                                              int32_t max_seqlen) {
  using ism::fail;
  ism::clear_error();
  if (!cu_seqlens || !cu_segs || !seg_is_query)
    return fail(ISM_ERR_NULL, "segment array is NULL");
  if (batch < 1 || num_segs < batch || total_tokens < num_segs)
    return fail(ISM_ERR_SHAPE,
                "need batch >= 1, num_segs >= batch, total >= num_segs "
                "(batch=%d num_segs=%d total=%d)", batch, num_segs, total_tokens);
  if (cu_seqlens[0] != 0 || cu_segs[0] != 0)
    return fail(ISM_ERR_SEGMENTS, "boundary arrays must start at 0");
  if (cu_seqlens[batch] != total_tokens)
    return fail(ISM_ERR_SEGMENTS, "cu_seqlens[%d]=%d != total_tokens=%d",
                batch, cu_seqlens[batch], total_tokens);
  if (cu_segs[num_segs] != total_tokens)
    return fail(ISM_ERR_SEGMENTS, "cu_segs[%d]=%d != total_tokens=%d",
                num_segs, cu_segs[num_segs], total_tokens);
  for (int32_t g = 0; g < num_segs; ++g)
    if (cu_segs[g + 1] <= cu_segs[g])
      return fail(ISM_ERR_SEGMENTS, "segment %d is empty or reversed (%d..%d)",
                  g, cu_segs[g], cu_segs[g + 1]);
  int32_t g = 0;
  for (int32_t b = 0; b < batch; ++b) {
    const int32_t len = cu_seqlens[b + 1] - cu_seqlens[b];
    if (len <= 0)
      return fail(ISM_ERR_SEGMENTS, "dialogue %d is empty or reversed", b);
    if (len > max_seqlen)
      return fail(ISM_ERR_SHAPE, "dialogue %d has %d tokens > max_seqlen %d",
                  b, len, max_seqlen);
    while (g < num_segs && cu_segs[g] < cu_seqlens[b + 1]) ++g;
    if (cu_segs[g] != cu_seqlens[b + 1])
      return fail(ISM_ERR_SEGMENTS,
                  "dialogue boundary %d is not a segment boundary",
                  cu_seqlens[b + 1]);
  }
  return ISM_OK;
}
