// Internal launch interface between the C ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ism {

// Forward attention over row tiles. Two modes share one kernel:
//  * packed (training / prefill): rows and keys live on the packed token axis,
//    key i of dialogue b is row i of k/v (stride hkv*d), and row j sees keys
//    [cu_q[b], lim[j]];
//  * cache (KV reuse): rows are the new tokens of dialogue b, keys are rows
//    of that dialogue's cache slab: all of 0..C_b+L_b-1 for a new query
//    segment, 0..C_b+r for row r of a new answer segment (cache_causal).
struct FwdArgs {
  const void *q;
  const void *k;
  const void *v;
  void *o;
  float *lse;               // may be null
  const int32_t *cu_q;      // [batch+1] row ranges of q / o
  const int32_t *lim;       // packed mode: [T] inclusive key bound per row
  const int32_t *cache_len; // cache mode: [batch] cached tokens C_b
  int32_t batch;
  int32_t hq;
  int32_t hkv;
  int32_t total_q;          // rows of q (T or Tn)
  int32_t max_rows;         // longest row range of a dialogue
  int64_t kv_seq_stride;    // elements between dialogues' K/V (cache mode)
  int64_t kv_head_stride;   // elements between KV heads
  int64_t kv_row_stride;    // elements between consecutive keys
  float scale;
  int32_t cache_causal;     // cache mode: the new segment is an answer
                            // segment (row r sees keys [0, C_b + r])
  // paged cache mode: k / v are page pools [num_pages, hkv, page_size, d];
  // key t of dialogue b is slot t % page_size of page
  // block_table[b * max_pages + t / page_size] (page_size % 64 == 0)
  const int32_t *block_table;
  int32_t page_size, max_pages, num_pages;
  // cache mode: 2-D rotary positions of the new rows (null = none); each
  // query row is rotated as it is loaded (the keys were rotated on append)
  const int32_t *rope_pos1, *rope_pos2;
  float rope_log2_base;
};

hipError_t launch_prep_lim(const int32_t *cu_segs, const uint8_t *seg_is_query,
                           int32_t num_segs, int32_t total, int32_t *lim,
                           hipStream_t stream);

hipError_t launch_fwd(const FwdArgs &a, int d, bool cache_mode,
                      hipStream_t stream);

// Paged cache: where token position t of dialogue b lives. The page index is
// clamped into the pool so that a bad table entry never addresses memory
// outside it. Returns the element offset of (page, head h, slot, 0).
__device__ __forceinline__ int64_t paged_offset(const int32_t *block_table, int32_t max_pages,
                                                int32_t num_pages, int32_t page_size,
                                                int32_t hkv, int32_t d, int b, int h, int t) {
  int page = block_table[(int64_t)b * max_pages + t / page_size];
  page = min(max(page, 0), num_pages - 1);
  return (((int64_t)page * hkv + h) * page_size + t % page_size) * d;
}

// The same for a position that is the same in every lane of the wave (a
// scalar load of the table entry, the offset in scalar registers).
__device__ __forceinline__ int64_t paged_offset_uniform(const int32_t *block_table,
                                                        int32_t max_pages, int32_t num_pages,
                                                        int32_t page_size, int32_t hkv,
                                                        int32_t d, int b, int h, int t) {
  const int idx = __builtin_amdgcn_readfirstlane(b * max_pages + t / page_size);
  int page = __builtin_amdgcn_readfirstlane(block_table[idx]);
  page = min(max(page, 0), num_pages - 1);
  return (((int64_t)page * hkv + h) * page_size + __builtin_amdgcn_readfirstlane(t % page_size)) *
         d;
}

// Cache append: rows [cu_new[b], cu_new[b+1]) of src go to positions
// cache_len[b] + (r - cu_new[b]) of slab b. src is [Tn, hkv, d];
// cache is [batch, hkv, cap, d].
hipError_t launch_cache_append(const void *k_src, const void *v_src,
                               void *k_cache, void *v_cache,
                               const int32_t *cu_new, const int32_t *cache_len,
                               int32_t batch, int32_t max_new, int32_t hkv,
                               int32_t d, int32_t cap, hipStream_t stream);

// The same into a paged cache (layout as in FwdArgs); cap = max_pages *
// page_size positions per dialogue.
hipError_t launch_cache_append_paged(const void *k_src, const void *v_src, void *k_pages,
                                     void *v_pages, const int32_t *cu_new,
                                     const int32_t *cache_len, const int32_t *block_table,
                                     int32_t max_pages, int32_t num_pages, int32_t page_size,
                                     int32_t batch, int32_t max_new, int32_t hkv, int32_t d,
                                     hipStream_t stream);

struct DecodeArgs {
  const void *q;            // [batch, hq, d]
  const void *k_new;        // [batch, hkv, d]
  const void *v_new;
  void *k_cache;            // [batch, hkv, cap, d]
  void *v_cache;
  const int32_t *pos;       // [batch] position of the new token
  void *o;                  // [batch, hq, d]
  float *lse;               // [hq, batch] or null
  float *part_o;            // [batch, hq, splits, d]
  float *part_ml;           // [batch, hq, splits, 2]
  int32_t batch, hq, hkv, cap, splits;
  float scale;
  // paged cache (see FwdArgs)
  const int32_t *block_table;
  int32_t page_size, max_pages, num_pages;
  int32_t set_heads;  // query heads per workgroup (decode_heads_per_set)
  int32_t mma;        // the matrix-core kernel (decode_mma_heads > 0)
};

hipError_t launch_decode(const DecodeArgs &a, int d, hipStream_t stream);

// Decode head sets, with G = hq / hkv query heads per KV head: the
// matrix-core kernel takes sets of the largest divisor of G up to 32 (the
// columns of one product) when that is 4 or more, or, when the step has
// fewer than kDecodeVectorSlabs (dialogue, KV head) slabs, of any size;
// 0 otherwise. Below that slab count its long one-wave chunks stream faster
// than the vector kernel even for one query head (256 slabs of 8192
// positions: 6.5 TB/s against 6.2, 6.0 and 5.9 for 1, 2 and 3 heads; 64
// slabs: 5.6 against 5.2, 4.8 and 4.2); from 1024 slabs on the vector
// kernel's wider grid is faster for 1-3 heads (6.9, 6.7, 6.7 against 6.4).
constexpr int kDecodeVectorSlabs = 512;
inline int decode_mma_heads(int batch, int hq, int hkv) {
  const int g = hq / hkv;
  const int lo = (int64_t)batch * hkv < kDecodeVectorSlabs ? 1 : 4;
  for (int s = g < 32 ? g : 32; s >= lo; --s)
    if (g % s == 0) return s;
  return 0;
}
// Query heads per decode workgroup: the matrix-core set, else (vector kernel,
// G without a divisor between 4 and 32) the largest divisor of G up to 3.
inline int decode_heads_per_set(int batch, int hq, int hkv) {
  const int m = decode_mma_heads(batch, hq, hkv);
  if (m) return m;
  const int g = hq / hkv;
  return g % 3 == 0 ? 3 : g % 2 == 0 ? 2 : 1;
}

struct BwdArgs {
  const void *q, *k, *v, *o, *dout;
  const float *lse;
  float *dq, *dk, *dv;
  // [hq, 2, T] workspace, written by the dQ kernel for the dK/dV kernel:
  // -lse / scale and -delta (delta = rowsum(dO * O)), each as the exact sum
  // of three bf16 values (plane 0: the first two, plane 1: the third and 0)
  uint32_t *lsex, *deltax;
  const int32_t *cu_seqlens;
  const int32_t *cu_segs;
  const uint8_t *seg_is_query;
  const int32_t *lim;       // [T] inclusive key bound per row
  const int32_t *seer;      // [T] first row that sees each key
  int32_t batch, num_segs, hq, hkv, total, max_seqlen;
  float scale, inv_scale;
  int32_t deterministic;
};

hipError_t launch_bwd_prep(const int32_t *cu_segs, const uint8_t *seg_is_query,
                           int32_t num_segs, int32_t total, int32_t *lim, int32_t *seer,
                           hipStream_t stream);

hipError_t launch_bwd(const BwdArgs &a, int d, hipStream_t stream);

// 2-D rotary positions (ism_rope.hip): positions from the segment layout,
// in-place rotation of [total, heads, d] (bf16 or fp32; inverse rotates by
// minus the angle), and the dense cache append with the keys rotated.
hipError_t launch_positions_2d(const int32_t *cu_seqlens, int32_t batch, const int32_t *cu_segs,
                               int32_t num_segs, int32_t total, int32_t *pos1, int32_t *pos2,
                               hipStream_t stream);
hipError_t launch_rope2d(void *x, bool fp32, int32_t total, int32_t heads, int32_t d,
                         const int32_t *pos1, const int32_t *pos2, float log2_base,
                         bool inverse, hipStream_t stream);
hipError_t launch_cache_append_rope(const void *k_src, const void *v_src, void *k_cache,
                                    void *v_cache, const int32_t *cu_new,
                                    const int32_t *cache_len, const int32_t *pos1,
                                    const int32_t *pos2, float log2_base, int32_t batch,
                                    int32_t max_new, int32_t hkv, int32_t d, int32_t cap,
                                    hipStream_t stream);

}  // namespace ism
