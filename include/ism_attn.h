/*
 * ism_attn.h - C ABI of the MI355X (gfx950) ISM attention library.
 *
 * Intermittent Semi-working Mask (ISM) attention, arXiv 2408.00539.
 * A packed batch holds several dialogues [P, Q_1, A_1, ..., Q_n, (A_n)]
 * (Sec. 2.1, the sample definition before Eq. 4). By Eq. 5, a token of a query
 * segment sees every earlier token of its dialogue and every token of its own
 * query segment; a token of an answer segment sees the tokens up to and
 * including itself. The attention itself is softmax(scale * Q K^T + M) V
 * with that mask (Sec. 2.3: ISM changes only the causal mask of a standard
 * decoder).
 *
 * Conventions shared by every entry point:
 *  - Tensor pointers are DEVICE pointers owned by the caller. The library
 *    allocates no memory and keeps no state between calls other than a
 *    thread-local error string (and the fixed scratch array of
 *    ism_attn_decode_noalloc, below).
 *  - bf16 tensors are passed as void* and are dense row-major:
 *      q, o: [T, hq, d];  k, v: [T, hkv, d]   (T = tokens of the packed batch)
 *      lse:  [hq, T] float32, natural-log log-sum-exp of the scaled scores.
 *  - Grouped KV heads: query head h reads key/value head h / (hq / hkv);
 *    hq must be a multiple of hkv, hq <= 8192. Supported head dims: d = 64
 *    and d = 128.
 *  - `scale` multiplies Q K^T before the softmax (normally 1/sqrt(d)).
 *  - All work is enqueued on `stream` (a hipStream_t passed as void*, NULL =
 *    the default stream). No call synchronises the device (except under
 *    ISM_VALIDATE=1, below).
 *  - `ws` is a caller-owned device workspace of at least
 *    ism_attn_workspace_size(...) bytes, 256-byte aligned.
 *  - On any error no kernel is launched, outputs are untouched, and a status
 *    other than ISM_OK is returned; ism_last_error() gives the detail.
 *    Faults of kernels already launched surface at the caller's next
 *    synchronisation of the stream, as for any HIP kernel.
 *  - Device-resident segment arrays are not inspected by the entry points
 *    (that would need a synchronising copy); ism_check_segments_host()
 *    validates a host copy of them. For debugging, the environment variable
 *    ISM_VALIDATE=1 (read on every call) makes each entry point that takes
 *    an ism_segments, and each cached prefill (cu_seqlens_new: from 0 to
 *    total_new, non-decreasing, no length above max_new), wait for its
 *    stream, copy those arrays to the host and validate them before any
 *    launch, failing with the validator's status (ISM_ERR_SEGMENTS for
 *    malformed boundaries).
 *  - No entry point aborts, throws or exits the process.
 */
#ifndef ISM_ATTN_H
#define ISM_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ISM_OK = 0,
  ISM_ERR_NULL = 1,        /* a required pointer is NULL                    */
  ISM_ERR_SHAPE = 2,       /* a size is out of range or inconsistent        */
  ISM_ERR_UNSUPPORTED = 3, /* e.g. head dim other than 64 / 128             */
  ISM_ERR_SEGMENTS = 4,    /* segment metadata violates its invariants      */
  ISM_ERR_WORKSPACE = 5,   /* workspace missing, too small or misaligned    */
  ISM_ERR_CAPACITY = 6,    /* KV cache capacity too small                   */
  ISM_ERR_NO_DEVICE = 7,   /* no usable gfx950 device                       */
  ISM_ERR_HIP = 8          /* a HIP runtime call or launch failed           */
} ism_status;

/* Dialogue structure of a packed batch (Sec. 2.1: the sample
 * [P, Q_1, A_1, ..., Q_n] with boundaries m_p, m_{q_k}, m_{a_k}).
 * Dialogue b covers tokens [cu_seqlens[b], cu_seqlens[b+1]); segment g covers
 * [cu_segs[g], cu_segs[g+1]) and is a query segment (bidirectional block,
 * Eq. 5 first two cases) iff seg_is_query[g] != 0, else an answer segment
 * (causal, Eq. 5 third case). The prompt P is passed merged with Q_1 as one
 * query segment (Eq. 5's first case covers both). Invariants: both arrays
 * start at 0 and end at total_tokens, are strictly increasing (no empty
 * segment or dialogue), and every cu_seqlens entry is also a cu_segs entry.
 * max_seqlen must be >= the longest dialogue. Arrays live in device memory. */
typedef struct {
  const int32_t *cu_seqlens;   /* [batch + 1]    */
  const int32_t *cu_segs;      /* [num_segs + 1] */
  const uint8_t *seg_is_query; /* [num_segs]     */
  int32_t batch;
  int32_t num_segs;
  int32_t total_tokens;
  int32_t max_seqlen;
} ism_segments;

/* Workspace query. `op` is one of the ISM_OP_* values; unused arguments may
 * be 0. Returns bytes (a multiple of 256), or 0 if none is needed. */
enum { ISM_OP_FWD = 0, ISM_OP_BWD = 1, ISM_OP_PREFILL_CACHED = 2,
       ISM_OP_DECODE = 3 };
size_t ism_attn_workspace_size(int32_t op, int32_t batch, int32_t total_tokens,
                               int32_t max_seqlen, int32_t hq, int32_t hkv,
                               int32_t d, int32_t num_splits);

/* Training / prefill forward over packed dialogues (Eq. 4 with the bound of
 * Eq. 5, softmax form). Writes o [T, hq, d] bf16 and lse [hq, T] fp32
 * (lse may be NULL). Workspace: ISM_OP_FWD. */
ism_status ism_attn_fwd(const ism_segments *sg, const void *q, const void *k,
                        const void *v, void *o, float *lse, int32_t hq,
                        int32_t hkv, int32_t d, float scale, void *ws,
                        size_t ws_bytes, void *stream);

/* Visibility metadata of a packed batch (Eq. 5, 0-indexed): lim[j] is the
 * last key token j may see (the last token of j's segment if that is a query
 * segment, j itself in an answer segment); seer[i] is the first token of
 * i's dialogue that sees key i (the first token of i's segment if that is a
 * query segment, i itself otherwise). Within a dialogue starting at s_b,
 * token j sees key i iff s_b <= i <= lim[j], equivalently iff seer[i] <= j.
 * These are the bounds from which the attention kernels classify their
 * tiles (skipped, unmasked, masked). lim and seer [total_tokens] int32
 * device, written. */
ism_status ism_visibility(const ism_segments *sg, int32_t *lim, int32_t *seer,
                          void *stream);

/* Backward of ism_attn_fwd (training on whole dialogues in one pass,
 * Sec. 1 and Sec. 3.3). Inputs q, k, v, o, dout bf16 and lse fp32 as written
 * by ism_attn_fwd on the same inputs. Outputs dq [T, hq, d], dk and dv
 * [T, hkv, d] in fp32, overwritten. Every reduction is bitwise repeatable
 * from run to run: each output element is written by one workgroup, with no
 * atomics. `deterministic` is reserved for a non-repeatable mode; today
 * both values run the repeatable path (a one-pass mode that adds dQ with
 * global atomics measured 2.2x slower on MI355X), so the result never
 * depends on it. Workspace: ISM_OP_BWD. */
ism_status ism_attn_bwd(const ism_segments *sg, const void *q, const void *k,
                        const void *v, const void *o, const float *lse,
                        const void *dout, float *dq, float *dk, float *dv,
                        int32_t hq, int32_t hkv, int32_t d, float scale,
                        int32_t deterministic, void *ws, size_t ws_bytes,
                        void *stream);

/* KV-cache reuse, new query segment (Sec. 2.3: reuse the history cache C_h,
 * compute C_q, concatenate [C_h; C_q]). For dialogue b with C_b =
 * cache_seqlens[b] cached tokens and L_b = cu_seqlens_new[b+1] -
 * cu_seqlens_new[b] new tokens, the new keys/values are first written into
 * the cache at positions [C_b, C_b + L_b); then every new row attends to all
 * keys [0, C_b + L_b) (Eq. 5: f = m_{q_n} for the whole current query).
 * q_new [Tn, hq, d], k_new / v_new [Tn, hkv, d] bf16 (Tn = total_new);
 * k_cache / v_cache [batch, hkv, cache_cap, d] bf16, updated in place only in
 * the append range; cache_seqlens [batch] device int32, read only (the
 * caller advances it by L_b afterwards). o [Tn, hq, d] bf16, lse [hq, Tn]
 * fp32 or NULL. The caller guarantees 0 <= C_b and C_b + L_b <= cache_cap
 * (the lengths live on the device, so the call cannot check them): a
 * dialogue outside that range gets NaN in all its rows of o and lse, and
 * only its positions inside the cache are appended. max_new must be >= every
 * L_b. Workspace: ISM_OP_PREFILL_CACHED (none). */
ism_status ism_attn_prefill_cached(
    const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new,
    int32_t max_new, const void *q_new, const void *k_new, const void *v_new,
    void *k_cache, void *v_cache, int32_t cache_cap,
    const int32_t *cache_seqlens, void *o, float *lse, int32_t hq, int32_t hkv,
    int32_t d, float scale, void *ws, size_t ws_bytes, void *stream);

/* The same with the kind of the new segment given: seg_is_query != 0 is the
 * query segment of ism_attn_prefill_cached; seg_is_query == 0 appends an
 * answer segment, whose row r (0-based inside the segment) sees keys
 * [0, C_b + r] (Eq. 5 third case, f(j) = j): an answer prefilled in chunks
 * through the cache, or the causal mask of Eq. 2 for the new rows (the
 * baseline the paper's latency comparison measures ISM against, Sec. 3.6).
 * All other arguments, the append and the errors are as for
 * ism_attn_prefill_cached. */
ism_status ism_attn_prefill_cached_segment(
    const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new,
    int32_t max_new, int32_t seg_is_query, const void *q_new,
    const void *k_new, const void *v_new, void *k_cache, void *v_cache,
    int32_t cache_cap, const int32_t *cache_seqlens, void *o, float *lse,
    int32_t hq, int32_t hkv, int32_t d, float scale, void *ws,
    size_t ws_bytes, void *stream);

/* One answer-token decode step with the reused cache (Sec. 2.3, generation
 * of A_n; Eq. 5 third case f(j) = j: the new token sees every cached token
 * and itself). For dialogue b the new token sits at position
 * p_b = cache_seqlens[b]: its key/value (k_new / v_new [batch, hkv, d]) are
 * written into the cache at p_b, then q [batch, hq, d] attends to keys
 * [0, p_b]. Each dialogue's key range is split into `num_splits` chunks of
 * equal length (0 = choose automatically), processed in parallel and merged
 * exactly. o [batch, hq, d]
 * bf16; lse [hq, batch] fp32 or NULL. The caller guarantees
 * 0 <= p_b < cache_cap and advances cache_seqlens by 1 afterwards; a
 * dialogue with p_b outside that range gets NaN in o and lse and nothing is
 * appended. max_seqlen bounds p_b + 1 for the split choice (0 = cache_cap):
 * the split count, and with it the workspace size, has to be known on the
 * host, where the positions (device memory) are not. Workspace:
 * ism_attn_workspace_size(ISM_OP_DECODE, batch, 0, max_seqlen (with 0
 * replaced by cache_cap), hq, hkv, d, num_splits). Any hq / hkv is
 * supported: with 4 or more query heads per KV head a workgroup serves a
 * set of 4-32 of them on the matrix cores, otherwise 1-3 on the vector
 * ALU, except that a step with fewer than 512 (dialogue, KV head) pairs
 * runs every head set on the matrix cores. */
ism_status ism_attn_decode(const void *q, const void *k_new, const void *v_new,
                           void *k_cache, void *v_cache, int32_t cache_cap,
                           const int32_t *cache_seqlens, int32_t batch,
                           int32_t max_seqlen, void *o, float *lse, int32_t hq,
                           int32_t hkv, int32_t d, float scale,
                           int32_t num_splits, void *ws, size_t ws_bytes,
                           void *stream);

/* The decode step of ism_attn_decode for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same arguments without the
 * workspace. The split partials live in a fixed per-device scratch array of
 * ISM_NOALLOC_SCRATCH_BYTES that the library holds until the process ends
 * (its device address is looked up on the first call on each device); the
 * call allocates nothing. Calls whose partials need more (batch * hq *
 * splits * (d + 2) * 4 bytes, rounded up) fail with ISM_ERR_WORKSPACE
 * before any launch. Every call on a device shares that device's scratch:
 * calls that may overlap on one device (different streams, no ordering
 * between them) race and must be serialised by the caller. Results equal
 * those of ism_attn_decode bit for bit. */
#define ISM_NOALLOC_SCRATCH_BYTES (8u << 20)
ism_status ism_attn_decode_noalloc(const void *q, const void *k_new,
                                   const void *v_new, void *k_cache,
                                   void *v_cache, int32_t cache_cap,
                                   const int32_t *cache_seqlens, int32_t batch,
                                   int32_t max_seqlen, void *o, float *lse,
                                   int32_t hq, int32_t hkv, int32_t d,
                                   float scale, int32_t num_splits,
                                   void *stream);

/* Paged KV cache: the same two operations with the cache held in fixed-size
 * pages instead of one slab per dialogue, so that dialogues of very
 * different lengths share one pool (the multi-turn serving case of Sec. 2.3,
 * where every turn appends to the reused cache). k_pages / v_pages
 * [num_pages, hkv, page_size, d] bf16; block_table [batch, max_pages] int32
 * device: position t of dialogue b is slot t % page_size of page
 * block_table[b * max_pages + t / page_size]. page_size must be a positive
 * multiple of 64; a dialogue holds at most max_pages * page_size positions
 * (this is cache_cap). The caller owns the pages and the table and
 * allocates the pages a turn appends to before the call; table entries are
 * read on the device and clamped into [0, num_pages). Results equal those
 * of the dense entry points on the same logical cache. Workspaces as for
 * ISM_OP_PREFILL_CACHED and ISM_OP_DECODE with cache_cap = max_pages *
 * page_size. */
ism_status ism_attn_prefill_paged(
    const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new,
    int32_t max_new, int32_t seg_is_query, const void *q_new,
    const void *k_new, const void *v_new, void *k_pages, void *v_pages,
    int32_t num_pages, int32_t page_size, const int32_t *block_table,
    int32_t max_pages, const int32_t *cache_seqlens, void *o, float *lse,
    int32_t hq, int32_t hkv, int32_t d, float scale, void *ws,
    size_t ws_bytes, void *stream);

ism_status ism_attn_decode_paged(const void *q, const void *k_new,
                                 const void *v_new, void *k_pages,
                                 void *v_pages, int32_t num_pages,
                                 int32_t page_size, const int32_t *block_table,
                                 int32_t max_pages,
                                 const int32_t *cache_seqlens, int32_t batch,
                                 int32_t max_seqlen, void *o, float *lse,
                                 int32_t hq, int32_t hkv, int32_t d,
                                 float scale, int32_t num_splits, void *ws,
                                 size_t ws_bytes, void *stream);

/* ChatGLM-style 2-D rotary positions, kept when ISM is adapted to a
 * prefix-style backbone (Sec. 2.3: one position encodes the span a token
 * belongs to, the other its offset inside the span; bidirectional attention
 * within query spans, causal within answer spans). Dims [0, d/2) of every
 * head rotate by pos1, dims [d/2, d) by pos2; inside a half of width
 * r = d/2, dims k and k + r/2 (k < r/2) form a pair rotated by the angle
 * pos * base^(-2k/r): x_k' = x_k cos a - x_{k+r/2} sin a,
 * x_{k+r/2}' = x_k sin a + x_{k+r/2} cos a. Angles are formed in fp32
 * revolutions (relative error about 2^-23: ~1e-3 rad at pos * base^(-2k/r)
 * = 10^4) and their fraction goes to the hardware sine / cosine; values are
 * rotated in fp32 and rounded to bf16 (round to nearest even) for bf16
 * tensors. */
enum { ISM_DTYPE_BF16 = 0, ISM_DTYPE_F32 = 1 };

/* Positions of a packed batch from its segments: pos1[j] = index of j's
 * segment counted from its dialogue's first segment, pos2[j] = j minus the
 * first token of its segment. pos1, pos2 [total_tokens] int32 device,
 * written. */
ism_status ism_positions_2d(const ism_segments *sg, int32_t *pos1,
                            int32_t *pos2, void *stream);

/* In-place rotation of x [total, heads, d] (device; dtype ISM_DTYPE_BF16 or
 * ISM_DTYPE_F32) by the positions pos1, pos2 [total] int32 (device) of its
 * tokens; d is 64 or 128; base finite and > 1 (10000 in ChatGLM).
 * `inverse` != 0 rotates by minus the angle: applied to fp32 gradients with
 * respect to rotated queries / keys (ism_attn_bwd on rotated inputs) it
 * gives the gradients with respect to the unrotated ones. Training with the
 * positions: rotate q and k, ism_attn_fwd, ism_attn_bwd, then rotate dq and
 * dk back. */
ism_status ism_rope2d(void *x, int32_t dtype, int32_t total, int32_t heads,
                      int32_t d, const int32_t *pos1, const int32_t *pos2,
                      float base, int32_t inverse, void *stream);

/* ism_attn_prefill_cached_segment with the new tokens' 2-D positions
 * pos1_new, pos2_new [total_new] int32 (device): the new keys are rotated on
 * their way into the cache (which therefore holds rotated keys, as a
 * rotary-position cache does) and each new query row is rotated as the
 * attention loads it; values are not rotated. Equal, bit for bit, to
 * ism_rope2d on q_new and k_new followed by
 * ism_attn_prefill_cached_segment. Dense cache only; a decode step with
 * positions rotates its q and k_new with ism_rope2d first. */
ism_status ism_attn_prefill_cached_rope2d(
    const int32_t *cu_seqlens_new, int32_t batch, int32_t total_new,
    int32_t max_new, int32_t seg_is_query, const void *q_new,
    const void *k_new, const void *v_new, void *k_cache, void *v_cache,
    int32_t cache_cap, const int32_t *cache_seqlens, const int32_t *pos1_new,
    const int32_t *pos2_new, float rope_base, void *o, float *lse, int32_t hq,
    int32_t hkv, int32_t d, float scale, void *ws, size_t ws_bytes,
    void *stream);

/* Host-side validation of segment metadata (HOST pointers). Pure CPU, needs
 * no device. Returns ISM_OK or ISM_ERR_SEGMENTS / ISM_ERR_NULL /
 * ISM_ERR_SHAPE with the first violation in ism_last_error(). */
ism_status ism_check_segments_host(const int32_t *cu_seqlens,
                                   const int32_t *cu_segs,
                                   const uint8_t *seg_is_query, int32_t batch,
                                   int32_t num_segs, int32_t total_tokens,
                                   int32_t max_seqlen);

/* Static description of a status code. */
const char *ism_status_string(ism_status s);

/* Detail of the last failure on the calling thread ("" if none). */
const char *ism_last_error(void);

/* Library version, "major.minor.patch". */
const char *ism_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ISM_ATTN_H */
