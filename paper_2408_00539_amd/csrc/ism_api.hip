// C ABI of the ISM attention library: argument checks, workspace layout and
// the launch sequence of each entry point. Every check happens on the host
// before any launch; nothing here synchronises the device, except the
// optional segment validation below (ISM_VALIDATE=1).
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "../../include/ism_attn.h"
#include "ism_host.h"
#include "ism_kernels.h"

namespace {

using ism::fail;

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Device check, cached per device ordinal: a gfx950 device must be current.
ism_status check_device() {
  static int ok_cache[64];  // 0 unknown, 1 ok, 2 bad
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count <= 0) {
    (void)hipGetLastError();
    return fail(ISM_ERR_NO_DEVICE, "no HIP device visible");
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(ISM_ERR_NO_DEVICE, "hipGetDevice failed");
  }
  if (dev >= 0 && dev < 64 && ok_cache[dev] == 1) return ISM_OK;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(ISM_ERR_NO_DEVICE, "hipGetDeviceProperties failed");
  }
  const bool ok = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev >= 0 && dev < 64) ok_cache[dev] = ok ? 1 : 2;
  if (!ok)
    return fail(ISM_ERR_NO_DEVICE, "device %d is %s, library is built for gfx950",
                dev, prop.gcnArchName);
  return ISM_OK;
}

ism_status check_heads(int32_t hq, int32_t hkv, int32_t d, float scale) {
  if (hq < 1 || hkv < 1 || hq % hkv != 0)
    return fail(ISM_ERR_SHAPE, "need hq >= 1, hkv >= 1, hq %% hkv == 0 (hq=%d hkv=%d)",
                hq, hkv);
  if (d != 64 && d != 128)
    return fail(ISM_ERR_UNSUPPORTED, "head dim %d not supported (64 or 128)", d);
  // tile transfers address 64 rows of a token-major tensor with 32-bit byte
  // offsets: 64 * hq * d * 2 bytes must stay below 2^31
  if (hq > 8192)
    return fail(ISM_ERR_UNSUPPORTED, "hq %d above the supported 8192 heads", hq);
  if (!(scale > 0.f) || !isfinite(scale))
    return fail(ISM_ERR_SHAPE, "scale must be finite and > 0 (got %g)", (double)scale);
  return ISM_OK;
}

ism_status check_ws(const void *ws, size_t ws_bytes, size_t need) {
  if (need == 0) return ISM_OK;
  if (!ws) return fail(ISM_ERR_WORKSPACE, "workspace of %zu bytes required", need);
  if ((uintptr_t)ws % kAlign)
    return fail(ISM_ERR_WORKSPACE, "workspace must be %zu-byte aligned", kAlign);
  if (ws_bytes < need)
    return fail(ISM_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need);
  return ISM_OK;
}

ism_status check_segments(const ism_segments *sg) {
  if (!sg) return fail(ISM_ERR_NULL, "segments struct is NULL");
  if (!sg->cu_seqlens || !sg->cu_segs || !sg->seg_is_query)
    return fail(ISM_ERR_NULL, "segment array is NULL");
  if (sg->batch < 1 || sg->num_segs < sg->batch || sg->total_tokens < sg->num_segs)
    return fail(ISM_ERR_SHAPE,
                "need batch >= 1, num_segs >= batch, total >= num_segs "
                "(batch=%d num_segs=%d total=%d)",
                sg->batch, sg->num_segs, sg->total_tokens);
  if (sg->max_seqlen < 1 || sg->max_seqlen > sg->total_tokens)
    return fail(ISM_ERR_SHAPE, "max_seqlen %d outside [1, total_tokens=%d]",
                sg->max_seqlen, sg->total_tokens);
  return ISM_OK;
}

ism_status hip_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return ISM_OK;
  return fail(ISM_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Optional validation of the device segment arrays, for debugging: with the
// environment variable ISM_VALIDATE set to 1 (read on every call), an entry
// point that takes an ism_segments waits for its stream, copies the three
// arrays to the host and runs ism_check_segments_host before any launch,
// so malformed metadata fails with its status instead of reaching the
// kernels. A device round trip per call; off by default.
ism_status validate_segments(const ism_segments *sg, hipStream_t stream) {
  const char *v = getenv("ISM_VALIDATE");
  if (!v || strcmp(v, "1") != 0) return ISM_OK;
  std::vector<int32_t> cu, cs;
  std::vector<uint8_t> fl;
  try {  // nothing may throw across the C ABI
    cu.resize(sg->batch + 1);
    cs.resize(sg->num_segs + 1);
    fl.resize(sg->num_segs);
  } catch (...) {
    return fail(ISM_ERR_SHAPE, "ISM_VALIDATE: no host memory for the segment arrays");
  }
  hipError_t e = hipStreamSynchronize(stream);
  if (e == hipSuccess)
    e = hipMemcpy(cu.data(), sg->cu_seqlens, cu.size() * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess)
    e = hipMemcpy(cs.data(), sg->cu_segs, cs.size() * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(fl.data(), sg->seg_is_query, fl.size(), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_status(e, "ISM_VALIDATE: copying the segment arrays");
  return ism_check_segments_host(cu.data(), cs.data(), fl.data(), sg->batch, sg->num_segs,
                                 sg->total_tokens, sg->max_seqlen);
}

// The same for the new-token boundaries of a cached prefill: cu_seqlens_new
// starts at 0, ends at total_new and never decreases, and no dialogue has
// more than max_new new tokens.
ism_status validate_new_lengths(const int32_t *cu_new, int32_t batch, int32_t total_new,
                                int32_t max_new, hipStream_t stream) {
  const char *v = getenv("ISM_VALIDATE");
  if (!v || strcmp(v, "1") != 0) return ISM_OK;
  std::vector<int32_t> cu;
  try {
    cu.resize(batch + 1);
  } catch (...) {
    return fail(ISM_ERR_SHAPE, "ISM_VALIDATE: no host memory for cu_seqlens_new");
  }
  hipError_t e = hipStreamSynchronize(stream);
  if (e == hipSuccess) e = hipMemcpy(cu.data(), cu_new, cu.size() * 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_status(e, "ISM_VALIDATE: copying cu_seqlens_new");
  if (cu[0] != 0 || cu[batch] != total_new)
    return fail(ISM_ERR_SEGMENTS, "cu_seqlens_new must run from 0 to total_new=%d (got %d..%d)",
                total_new, cu[0], cu[batch]);
  for (int32_t b = 0; b < batch; ++b)
    if (cu[b + 1] < cu[b] || cu[b + 1] - cu[b] > max_new)
      return fail(ISM_ERR_SEGMENTS, "dialogue %d has %d new tokens (need 0..max_new=%d)", b,
                  cu[b + 1] - cu[b], max_new);
  return ISM_OK;
}

// Split count of a decode step; `sets` = head sets per dialogue
// (hq / decode_heads_per_set), `target` = workgroups to aim at: about 2048
// four-wave workgroups (two rounds of four per CU) for the vector kernel;
// for the matrix-core kernel, whose long chunks stream faster, about 512
// one-wave workgroups on a dense cache and 768 on a paged one (on 256 slabs
// of 8192 keys: 6.5 and 6.4 TB/s, against 6.2 and 6.4 with 768 for both,
// 6.5 and 6.0 with 512, and 5.5 and 5.5 with 4096). At least 256 keys per
// chunk, at most 64 chunks.
constexpr int kSplitsVector = 2048, kSplitsMmaDense = 512, kSplitsMmaPaged = 768;
int decode_splits(int32_t batch, int32_t sets, int32_t max_len, int32_t req, int target) {
  if (req > 0) return req;
  const int slabs = batch * sets;
  int s = (target + slabs - 1) / slabs;
  const int by_len = (max_len + 255) / 256;
  if (s > by_len) s = by_len;
  if (s > 64) s = 64;
  return s < 1 ? 1 : s;
}

}  // namespace

extern "C" size_t ism_attn_workspace_size(int32_t op, int32_t batch,
                                          int32_t total_tokens, int32_t max_seqlen,
                                          int32_t hq, int32_t hkv, int32_t d,
                                          int32_t num_splits) {
  if (batch < 0 || total_tokens < 0 || hq < 0 || hkv < 0 || d < 0) return 0;
  switch (op) {
    case ISM_OP_FWD:
      return align_up((size_t)total_tokens * 4);
    case ISM_OP_BWD:
      return 2 * align_up((size_t)total_tokens * 4) +
             2 * align_up((size_t)total_tokens * hq * 8);
    case ISM_OP_PREFILL_CACHED:
      return 0;
    case ISM_OP_DECODE: {
      if (hkv < 1 || hq < hkv || hq % hkv) return 0;
      // the larger of the dense and paged split counts
      const int sets = hq / ism::decode_heads_per_set(batch, hq, hkv);
      const size_t s = (size_t)decode_splits(
          batch, sets, max_seqlen, num_splits,
          ism::decode_mma_heads(batch, hq, hkv) > 0 ? kSplitsMmaPaged : kSplitsVector);
      return align_up((size_t)batch * hq * s * d * 4) +
             align_up((size_t)batch * hq * s * 2 * 4);
    }
  }
  return 0;
}

extern "C" ism_status ism_attn_fwd(const ism_segments *sg, const void *q,
                                   const void *k, const void *v, void *o,
                                   float *lse, int32_t hq, int32_t hkv, int32_t d,
                                   float scale, void *ws, size_t ws_bytes,
                                   void *stream) {
  ism::clear_error();
  ism_status st = check_segments(sg);
  if (st) return st;
  if (!q || !k || !v || !o) return fail(ISM_ERR_NULL, "q, k, v and o are required");
  if ((st = check_heads(hq, hkv, d, scale))) return st;
  const size_t need = ism_attn_workspace_size(ISM_OP_FWD, sg->batch, sg->total_tokens,
                                              sg->max_seqlen, hq, hkv, d, 0);
  if ((st = check_ws(ws, ws_bytes, need))) return st;
  if ((st = check_device())) return st;
  if ((st = validate_segments(sg, (hipStream_t)stream))) return st;

  hipStream_t s = (hipStream_t)stream;
  int32_t *lim = (int32_t *)ws;
  if ((st = hip_status(ism::launch_prep_lim(sg->cu_segs, sg->seg_is_query, sg->num_segs,
                                            sg->total_tokens, lim, s),
                       "prep launch")))
    return st;
  ism::FwdArgs a{};
  a.q = q; a.k = k; a.v = v; a.o = o; a.lse = lse;
  a.cu_q = sg->cu_seqlens;
  a.lim = lim;
  a.cache_len = nullptr;
  a.batch = sg->batch; a.hq = hq; a.hkv = hkv;
  a.total_q = sg->total_tokens;
  a.max_rows = sg->max_seqlen;
  a.kv_seq_stride = 0;
  a.kv_head_stride = d;
  a.kv_row_stride = (int64_t)hkv * d;
  a.scale = scale;
  return hip_status(ism::launch_fwd(a, d, false, s), "forward launch");
}

extern "C" ism_status ism_visibility(const ism_segments *sg, int32_t *lim, int32_t *seer,
                                     void *stream) {
  ism::clear_error();
  ism_status st = check_segments(sg);
  if (st) return st;
  if (!lim || !seer) return fail(ISM_ERR_NULL, "lim and seer are required");
  if ((st = check_device())) return st;
  if ((st = validate_segments(sg, (hipStream_t)stream))) return st;
  return hip_status(ism::launch_bwd_prep(sg->cu_segs, sg->seg_is_query, sg->num_segs,
                                         sg->total_tokens, lim, seer, (hipStream_t)stream),
                    "visibility launch");
}

extern "C" ism_status ism_attn_bwd(const ism_segments *sg, const void *q,
                                   const void *k, const void *v, const void *o,
                                   const float *lse, const void *dout, float *dq,
                                   float *dk, float *dv, int32_t hq, int32_t hkv,
                                   int32_t d, float scale, int32_t deterministic,
                                   void *ws, size_t ws_bytes, void *stream) {
  ism::clear_error();
  ism_status st = check_segments(sg);
  if (st) return st;
  if (!q || !k || !v || !o || !lse || !dout || !dq || !dk || !dv)
    return fail(ISM_ERR_NULL, "q, k, v, o, lse, dout, dq, dk, dv are required");
  if ((st = check_heads(hq, hkv, d, scale))) return st;
  const size_t need = ism_attn_workspace_size(ISM_OP_BWD, sg->batch, sg->total_tokens,
                                              sg->max_seqlen, hq, hkv, d, 0);
  if ((st = check_ws(ws, ws_bytes, need))) return st;
  if ((st = check_device())) return st;
  if ((st = validate_segments(sg, (hipStream_t)stream))) return st;

  hipStream_t s = (hipStream_t)stream;
  const size_t tb = align_up((size_t)sg->total_tokens * 4);
  int32_t *lim = (int32_t *)ws;
  int32_t *seer = (int32_t *)((char *)ws + tb);
  uint32_t *lsex = (uint32_t *)((char *)ws + 2 * tb);
  uint32_t *deltax = (uint32_t *)((char *)lsex + align_up((size_t)sg->total_tokens * hq * 8));
  if ((st = hip_status(ism::launch_bwd_prep(sg->cu_segs, sg->seg_is_query, sg->num_segs,
                                            sg->total_tokens, lim, seer, s),
                       "prep launch")))
    return st;
  ism::BwdArgs a{};
  a.q = q; a.k = k; a.v = v; a.o = o; a.dout = dout; a.lse = lse;
  a.dq = dq; a.dk = dk; a.dv = dv; a.lsex = lsex; a.deltax = deltax;
  a.cu_seqlens = sg->cu_seqlens; a.cu_segs = sg->cu_segs;
  a.seg_is_query = sg->seg_is_query; a.lim = lim; a.seer = seer;
  a.batch = sg->batch; a.num_segs = sg->num_segs; a.hq = hq; a.hkv = hkv;
  a.total = sg->total_tokens; a.max_seqlen = sg->max_seqlen;
  a.scale = scale; a.inv_scale = 1.f / scale; a.deterministic = deterministic;
  const hipError_t e = ism::launch_bwd(a, d, s);
  if (e == hipErrorNotSupported)
    return fail(ISM_ERR_UNSUPPORTED, "backward configuration not supported");
  return hip_status(e, "backward launch");
}

extern "C" ism_status ism_attn_prefill_cached(
    const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new, int32_t max_new,
    const void *q_new, const void *k_new, const void *v_new, void *k_cache,
    void *v_cache, int32_t cache_cap, const int32_t *cache_seqlens, void *o,
    float *lse, int32_t hq, int32_t hkv, int32_t d, float scale, void *ws,
    size_t ws_bytes, void *stream) {
  return ism_attn_prefill_cached_segment(cu_seqlens_new, batch, total_new, max_new, 1,
                                         q_new, k_new, v_new, k_cache, v_cache, cache_cap,
                                         cache_seqlens, o, lse, hq, hkv, d, scale, ws,
                                         ws_bytes, stream);
}

namespace {

// A paged KV cache (see the paged entry points); null for a dense cache.
struct Paging {
  const int32_t *block_table;
  int32_t max_pages, num_pages, page_size;
};

ism_status check_paging(const Paging &pg) {
  if (!pg.block_table) return fail(ISM_ERR_NULL, "block_table is NULL");
  if (pg.num_pages < 1 || pg.max_pages < 1)
    return fail(ISM_ERR_SHAPE, "need num_pages >= 1 and max_pages >= 1 (got %d, %d)",
                pg.num_pages, pg.max_pages);
  if (pg.page_size < 64 || pg.page_size % 64 != 0)
    return fail(ISM_ERR_UNSUPPORTED, "page_size %d is not a positive multiple of 64",
                pg.page_size);
  if ((int64_t)pg.max_pages * pg.page_size > INT32_MAX)
    return fail(ISM_ERR_SHAPE, "max_pages * page_size exceeds the int32 position range");
  return ISM_OK;
}

// 2-D rotary positions of the new tokens (see the rope entry points); null
// for none.
struct Rope {
  const int32_t *pos1, *pos2;
  float base;
};

ism_status check_rope_base(float base) {
  if (!(base > 1.f) || !isfinite(base))
    return fail(ISM_ERR_SHAPE, "rope base %g must be finite and > 1", (double)base);
  return ISM_OK;
}

ism_status prefill_impl(const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new,
                        int32_t max_new, int32_t seg_is_query, const void *q_new,
                        const void *k_new, const void *v_new, void *k_cache, void *v_cache,
                        int32_t cache_cap, const int32_t *cache_seqlens, void *o, float *lse,
                        int32_t hq, int32_t hkv, int32_t d, float scale, void *ws,
                        size_t ws_bytes, void *stream, const Paging *pg,
                        const Rope *rp = nullptr) {
  ism::clear_error();
  if (!cu_seqlens_new || !q_new || !k_new || !v_new || !k_cache || !v_cache ||
      !cache_seqlens || !o)
    return fail(ISM_ERR_NULL, "a required pointer is NULL");
  if (pg) {
    const ism_status ps = check_paging(*pg);
    if (ps) return ps;
    cache_cap = pg->max_pages * pg->page_size;
  }
  if (batch < 1 || total_new < 1 || max_new < 1 || max_new > total_new)
    return fail(ISM_ERR_SHAPE,
                "need batch >= 1, 1 <= max_new <= total_new (batch=%d total_new=%d "
                "max_new=%d)", batch, total_new, max_new);
  ism_status st = check_heads(hq, hkv, d, scale);
  if (st) return st;
  if (cache_cap < max_new)
    return fail(ISM_ERR_CAPACITY, "cache_cap %d < max_new %d", cache_cap, max_new);
  if (rp) {
    if (!rp->pos1 || !rp->pos2) return fail(ISM_ERR_NULL, "pos1_new and pos2_new are required");
    if ((st = check_rope_base(rp->base))) return st;
  }
  (void)ws; (void)ws_bytes;
  if ((st = check_device())) return st;
  if ((st = validate_new_lengths(cu_seqlens_new, batch, total_new, max_new,
                                 (hipStream_t)stream)))
    return st;

  hipStream_t s = (hipStream_t)stream;
  const float l2b = rp ? log2f(rp->base) : 0.f;
  const hipError_t ae =
      rp ? ism::launch_cache_append_rope(k_new, v_new, k_cache, v_cache, cu_seqlens_new,
                                         cache_seqlens, rp->pos1, rp->pos2, l2b, batch, max_new,
                                         hkv, d, cache_cap, s)
      : pg ? ism::launch_cache_append_paged(k_new, v_new, k_cache, v_cache, cu_seqlens_new,
                                          cache_seqlens, pg->block_table, pg->max_pages,
                                          pg->num_pages, pg->page_size, batch, max_new, hkv, d,
                                          s)
         : ism::launch_cache_append(k_new, v_new, k_cache, v_cache, cu_seqlens_new,
                                    cache_seqlens, batch, max_new, hkv, d, cache_cap, s);
  if ((st = hip_status(ae, "cache append launch"))) return st;
  ism::FwdArgs a{};
  a.q = q_new; a.k = k_cache; a.v = v_cache; a.o = o; a.lse = lse;
  a.cu_q = cu_seqlens_new;
  a.lim = nullptr;
  a.cache_len = cache_seqlens;
  a.batch = batch; a.hq = hq; a.hkv = hkv;
  a.total_q = total_new;
  a.max_rows = max_new;
  a.kv_seq_stride = (int64_t)hkv * cache_cap * d;
  a.kv_head_stride = (int64_t)cache_cap * d;
  a.kv_row_stride = d;
  a.scale = scale;
  a.cache_causal = seg_is_query ? 0 : 1;
  if (pg) {
    a.block_table = pg->block_table;
    a.max_pages = pg->max_pages;
    a.num_pages = pg->num_pages;
    a.page_size = pg->page_size;
  }
  if (rp) {
    a.rope_pos1 = rp->pos1;
    a.rope_pos2 = rp->pos2;
    a.rope_log2_base = l2b;
  }
  return hip_status(ism::launch_fwd(a, d, true, s), "cached prefill launch");
}

}  // namespace

extern "C" ism_status ism_attn_prefill_cached_segment(
    const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new, int32_t max_new,
    int32_t seg_is_query, const void *q_new, const void *k_new, const void *v_new,
    void *k_cache, void *v_cache, int32_t cache_cap, const int32_t *cache_seqlens, void *o,
    float *lse, int32_t hq, int32_t hkv, int32_t d, float scale, void *ws,
    size_t ws_bytes, void *stream) {
  return prefill_impl(cu_seqlens_new, batch, total_new, max_new, seg_is_query, q_new, k_new,
                      v_new, k_cache, v_cache, cache_cap, cache_seqlens, o, lse, hq, hkv, d,
                      scale, ws, ws_bytes, stream, nullptr);
}

extern "C" ism_status ism_attn_prefill_cached_rope2d(
    const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new, int32_t max_new,
    int32_t seg_is_query, const void *q_new, const void *k_new, const void *v_new,
    void *k_cache, void *v_cache, int32_t cache_cap, const int32_t *cache_seqlens,
    const int32_t *pos1_new, const int32_t *pos2_new, float rope_base, void *o, float *lse,
    int32_t hq, int32_t hkv, int32_t d, float scale, void *ws, size_t ws_bytes, void *stream) {
  const Rope rp{pos1_new, pos2_new, rope_base};
  return prefill_impl(cu_seqlens_new, batch, total_new, max_new, seg_is_query, q_new, k_new,
                      v_new, k_cache, v_cache, cache_cap, cache_seqlens, o, lse, hq, hkv, d,
                      scale, ws, ws_bytes, stream, nullptr, &rp);
}

extern "C" ism_status ism_positions_2d(const ism_segments *sg, int32_t *pos1, int32_t *pos2,
                                       void *stream) {
  ism::clear_error();
  ism_status st = check_segments(sg);
  if (st) return st;
  if (!pos1 || !pos2) return fail(ISM_ERR_NULL, "pos1 and pos2 are required");
  if ((st = check_device())) return st;
  if ((st = validate_segments(sg, (hipStream_t)stream))) return st;
  return hip_status(ism::launch_positions_2d(sg->cu_seqlens, sg->batch, sg->cu_segs,
                                             sg->num_segs, sg->total_tokens, pos1, pos2,
                                             (hipStream_t)stream),
                    "positions launch");
}

extern "C" ism_status ism_rope2d(void *x, int32_t dtype, int32_t total, int32_t heads,
                                 int32_t d, const int32_t *pos1, const int32_t *pos2,
                                 float base, int32_t inverse, void *stream) {
  ism::clear_error();
  if (!x || !pos1 || !pos2) return fail(ISM_ERR_NULL, "x, pos1 and pos2 are required");
  if (dtype != ISM_DTYPE_BF16 && dtype != ISM_DTYPE_F32)
    return fail(ISM_ERR_UNSUPPORTED, "dtype %d is neither ISM_DTYPE_BF16 nor ISM_DTYPE_F32",
                dtype);
  if (total < 0 || heads < 0)
    return fail(ISM_ERR_SHAPE, "total %d and heads %d must be >= 0", total, heads);
  if (d != 64 && d != 128) return fail(ISM_ERR_UNSUPPORTED, "d must be 64 or 128 (got %d)", d);
  ism_status st = check_rope_base(base);
  if (st) return st;
  if ((st = check_device())) return st;
  return hip_status(ism::launch_rope2d(x, dtype == ISM_DTYPE_F32, total, heads, d, pos1, pos2,
                                       log2f(base), inverse != 0, (hipStream_t)stream),
                    "rope launch");
}

extern "C" ism_status ism_attn_prefill_paged(
    const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new, int32_t max_new,
    int32_t seg_is_query, const void *q_new, const void *k_new, const void *v_new,
    void *k_pages, void *v_pages, int32_t num_pages, int32_t page_size,
    const int32_t *block_table, int32_t max_pages, const int32_t *cache_seqlens, void *o,
    float *lse, int32_t hq, int32_t hkv, int32_t d, float scale, void *ws, size_t ws_bytes,
    void *stream) {
  const Paging pg{block_table, max_pages, num_pages, page_size};
  return prefill_impl(cu_seqlens_new, batch, total_new, max_new, seg_is_query, q_new, k_new,
                      v_new, k_pages, v_pages, 0, cache_seqlens, o, lse, hq, hkv, d, scale, ws,
                      ws_bytes, stream, &pg);
}

namespace {

ism_status decode_impl(const void *q, const void *k_new, const void *v_new, void *k_cache,
                       void *v_cache, int32_t cache_cap, const int32_t *cache_seqlens,
                       int32_t batch, int32_t max_seqlen, void *o, float *lse, int32_t hq,
                       int32_t hkv, int32_t d, float scale, int32_t num_splits, void *ws,
                       size_t ws_bytes, void *stream, const Paging *pg) {
  ism::clear_error();
  if (!q || !k_new || !v_new || !k_cache || !v_cache || !cache_seqlens || !o)
    return fail(ISM_ERR_NULL, "a required pointer is NULL");
  if (pg) {
    const ism_status ps = check_paging(*pg);
    if (ps) return ps;
    cache_cap = pg->max_pages * pg->page_size;
  }
  if (batch < 1 || cache_cap < 1)
    return fail(ISM_ERR_SHAPE, "need batch >= 1 and cache_cap >= 1");
  ism_status st = check_heads(hq, hkv, d, scale);
  if (st) return st;
  if (max_seqlen == 0) max_seqlen = cache_cap;
  if (max_seqlen < 1 || max_seqlen > cache_cap)
    return fail(ISM_ERR_CAPACITY, "max_seqlen %d outside [1, cache_cap=%d]", max_seqlen,
                cache_cap);
  if (num_splits < 0 || num_splits > 1024)
    return fail(ISM_ERR_SHAPE, "num_splits %d outside [0, 1024]", num_splits);
  const int set_heads = ism::decode_heads_per_set(batch, hq, hkv);
  const bool mma = ism::decode_mma_heads(batch, hq, hkv) > 0;
  const int splits = decode_splits(batch, hq / set_heads, max_seqlen, num_splits,
                                   !mma ? kSplitsVector : pg ? kSplitsMmaPaged : kSplitsMmaDense);
  const size_t need = ism_attn_workspace_size(ISM_OP_DECODE, batch, 0, max_seqlen, hq,
                                              hkv, d, num_splits);
  if ((st = check_ws(ws, ws_bytes, need))) return st;
  if ((st = check_device())) return st;

  ism::DecodeArgs a{};
  a.q = q; a.k_new = k_new; a.v_new = v_new;
  a.k_cache = k_cache; a.v_cache = v_cache; a.pos = cache_seqlens;
  a.o = o; a.lse = lse;
  a.part_o = (float *)ws;
  a.part_ml = (float *)((char *)ws + align_up((size_t)batch * hq * splits * d * 4));
  a.batch = batch; a.hq = hq; a.hkv = hkv; a.cap = cache_cap;
  a.splits = splits;
  a.scale = scale;
  a.set_heads = set_heads;
  a.mma = mma ? 1 : 0;
  if (pg) {
    a.block_table = pg->block_table;
    a.max_pages = pg->max_pages;
    a.num_pages = pg->num_pages;
    a.page_size = pg->page_size;
  }
  return hip_status(ism::launch_decode(a, d, (hipStream_t)stream), "decode launch");
}

}  // namespace

extern "C" ism_status ism_attn_decode(const void *q, const void *k_new, const void *v_new,
                                      void *k_cache, void *v_cache, int32_t cache_cap,
                                      const int32_t *cache_seqlens, int32_t batch,
                                      int32_t max_seqlen, void *o, float *lse, int32_t hq,
                                      int32_t hkv, int32_t d, float scale, int32_t num_splits,
                                      void *ws, size_t ws_bytes, void *stream) {
  return decode_impl(q, k_new, v_new, k_cache, v_cache, cache_cap, cache_seqlens, batch,
                     max_seqlen, o, lse, hq, hkv, d, scale, num_splits, ws, ws_bytes, stream,
                     nullptr);
}

extern "C" ism_status ism_attn_decode_paged(const void *q, const void *k_new,
                                            const void *v_new, void *k_pages, void *v_pages,
                                            int32_t num_pages, int32_t page_size,
                                            const int32_t *block_table, int32_t max_pages,
                                            const int32_t *cache_seqlens, int32_t batch,
                                            int32_t max_seqlen, void *o, float *lse, int32_t hq,
                                            int32_t hkv, int32_t d, float scale,
                                            int32_t num_splits, void *ws, size_t ws_bytes,
                                            void *stream) {
  const Paging pg{block_table, max_pages, num_pages, page_size};
  return decode_impl(q, k_new, v_new, k_pages, v_pages, 0, cache_seqlens, batch, max_seqlen, o,
                     lse, hq, hkv, d, scale, num_splits, ws, ws_bytes, stream, &pg);
}

// ---------------------------------------------------------------- no-allocation decode

namespace {

// Split partials of ism_attn_decode_noalloc: one array per device, held
// until the process ends. Host code never passes this name to a kernel (on
// the host it is only a stand-in for the device symbol): it uses the device
// address that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[ISM_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
void *g_scratch_ptr[64];  // per device ordinal, set on the first call there

ism_status scratch_address(void **out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(ISM_ERR_NO_DEVICE, "hipGetDevice failed");
  }
  if (dev < 0 || dev >= 64) return fail(ISM_ERR_NO_DEVICE, "device ordinal %d above 63", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(ISM_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                  hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ISM_OK;
}

}  // namespace

extern "C" ism_status ism_attn_decode_noalloc(const void *q, const void *k_new,
                                              const void *v_new, void *k_cache,
                                              void *v_cache, int32_t cache_cap,
                                              const int32_t *cache_seqlens, int32_t batch,
                                              int32_t max_seqlen, void *o, float *lse,
                                              int32_t hq, int32_t hkv, int32_t d, float scale,
                                              int32_t num_splits, void *stream) {
  ism::clear_error();
  ism_status st = check_heads(hq, hkv, d, scale);
  if (st) return st;
  if (batch < 1 || cache_cap < 1) return fail(ISM_ERR_SHAPE, "need batch >= 1 and cache_cap >= 1");
  const int32_t ms = max_seqlen == 0 ? cache_cap : max_seqlen;
  if (ms < 1 || ms > cache_cap)
    return fail(ISM_ERR_CAPACITY, "max_seqlen %d outside [1, cache_cap=%d]", ms, cache_cap);
  if (num_splits < 0 || num_splits > 1024)
    return fail(ISM_ERR_SHAPE, "num_splits %d outside [0, 1024]", num_splits);
  const size_t need = ism_attn_workspace_size(ISM_OP_DECODE, batch, 0, ms, hq, hkv, d,
                                              num_splits);
  if (need > ISM_NOALLOC_SCRATCH_BYTES)
    return fail(ISM_ERR_WORKSPACE,
                "split partials need %zu bytes, above the %zu-byte scratch of the "
                "allocation-free decode (use ism_attn_decode with a workspace)",
                need, (size_t)ISM_NOALLOC_SCRATCH_BYTES);
  if ((st = check_device())) return st;
  void *ws = nullptr;
  if ((st = scratch_address(&ws))) return st;
  return decode_impl(q, k_new, v_new, k_cache, v_cache, cache_cap, cache_seqlens, batch, ms, o,
                     lse, hq, hkv, d, scale, num_splits, ws, ISM_NOALLOC_SCRATCH_BYTES, stream,
                     nullptr);
}
