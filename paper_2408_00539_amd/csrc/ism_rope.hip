// ChatGLM-style 2-D rotary positions under ISM (the prefix-backbone
// adaptation of Sec. 2.3: the span a token belongs to and its offset inside
// the span are kept as two positions):
//  * positions from the segment layout: pos1 = index of the token's segment
//    counted from its dialogue's first segment, pos2 = offset inside the
//    segment;
//  * in-place rotation of a [T, heads, d] tensor: bf16 queries or keys, or
//    fp32 gradients with the inverse rotation (which maps gradients with
//    respect to rotated queries/keys back to the unrotated ones);
//  * the cache append of a new segment with its keys rotated on the way
//    (the forward rotates the new queries when it loads them), so that a
//    cached prefill needs no separate rotation pass.
// Rotation is HBM-bound elementwise work: a thread owns one (token, head)
// row's 8-dim chunk in the first quarter of a half and its partner chunk d/4
// further, and forms its 8 angles (a few instructions each); each head row
// is read and written whole by d/16 neighbouring threads with 16-byte
// accesses. (Threads that walked all heads with angles formed once had too
// few waves in flight to cover the memory latency: 2x slower.)
#include "ism_common.h"
#include "ism_kernels.h"

namespace ism {

namespace {

__global__ void __launch_bounds__(256)
positions_2d_kernel(const int32_t *__restrict__ cu_seqlens, int32_t batch,
                    const int32_t *__restrict__ cu_segs, int32_t num_segs, int32_t total,
                    int32_t *__restrict__ pos1, int32_t *__restrict__ pos2) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= total) return;
  int lo = 0, hi = num_segs - 1;  // largest g with cu_segs[g] <= j
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_segs[mid] <= j) lo = mid; else hi = mid - 1;
  }
  const int g = lo;
  int blo = 0, bhi = batch - 1;  // largest b with cu_seqlens[b] <= j
  while (blo < bhi) {
    const int mid = (blo + bhi + 1) >> 1;
    if (cu_seqlens[mid] <= j) blo = mid; else bhi = mid - 1;
  }
  const int start = cu_seqlens[blo];
  int g0 = 0, ghi = g;  // the segment that starts at the dialogue's start
  while (g0 < ghi) {
    const int mid = (g0 + ghi) >> 1;
    if (cu_segs[mid] < start) g0 = mid + 1; else ghi = mid;
  }
  pos1[j] = g - g0;
  pos2[j] = j - cu_segs[g];
}

// Angles of this thread's 8 pairs: chunk ci of the first quarter of half hf.
__device__ __forceinline__ void chunk_angles(int pos, int ci, int d, float log2_base,
                                             bool inverse, float (&c)[8], float (&s)[8]) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    rope_cs(pos, ci * 8 + e, d / 2, log2_base, c[e], s[e]);
    if (inverse) s[e] = -s[e];
  }
}

template <typename T>
__global__ void __launch_bounds__(256)
rope2d_kernel(T *__restrict__ x, int32_t total, int32_t heads, int32_t d,
              const int32_t *__restrict__ pos1, const int32_t *__restrict__ pos2,
              float log2_base, int32_t inverse) {
  const int per_row = d / 16;  // pair chunks per head row (d/32 per half)
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)total * heads * per_row) return;
  const int64_t row = i / per_row;  // (token, head)
  const int c = (int)(i % per_row);
  const int t = (int)(row / heads);
  const int half = c / (per_row / 2), ci = c % (per_row / 2);
  const int pos = half ? pos2[t] : pos1[t];
  float cs[8], sn[8];
  chunk_angles(pos, ci, d, log2_base, inverse != 0, cs, sn);
  const int dim = half * (d / 2) + ci * 8;
  T *p = x + row * d + dim;
  if constexpr (sizeof(T) == 2) {
    u32x4 a = *(const u32x4 *)p, b = *(const u32x4 *)(p + d / 4);
    rope_rotate8(a, b, cs, sn);
    *(u32x4 *)p = a;
    *(u32x4 *)(p + d / 4) = b;
  } else {
    f32x4 a0 = *(const f32x4 *)p, a1 = *(const f32x4 *)(p + 4);
    f32x4 b0 = *(const f32x4 *)(p + d / 4), b1 = *(const f32x4 *)(p + d / 4 + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x0 = a0[e], y0 = b0[e], x1 = a1[e], y1 = b1[e];
      a0[e] = fmaf(x0, cs[e], -(y0 * sn[e]));
      b0[e] = fmaf(x0, sn[e], y0 * cs[e]);
      a1[e] = fmaf(x1, cs[e + 4], -(y1 * sn[e + 4]));
      b1[e] = fmaf(x1, sn[e + 4], y1 * cs[e + 4]);
    }
    *(f32x4 *)p = a0;
    *(f32x4 *)(p + 4) = a1;
    *(f32x4 *)(p + d / 4) = b0;
    *(f32x4 *)(p + d / 4 + 4) = b1;
  }
}

// Cache append of a new segment (layout as cache_append_kernel) with the
// keys rotated by the new rows' positions; values are copied.
__global__ void __launch_bounds__(256)
cache_append_rope_kernel(const bf16_t *__restrict__ k_src, const bf16_t *__restrict__ v_src,
                         bf16_t *__restrict__ k_cache, bf16_t *__restrict__ v_cache,
                         const int32_t *__restrict__ cu_new, const int32_t *__restrict__ cache_len,
                         const int32_t *__restrict__ pos1, const int32_t *__restrict__ pos2,
                         float log2_base, int32_t hkv, int32_t d, int32_t cap) {
  const int b = blockIdx.y;
  const int r0 = cu_new[b], n = cu_new[b + 1] - r0;
  const int per_row = d / 16;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n * hkv * per_row) return;
  const int c = (int)(idx % per_row);
  const int h = (int)((idx / per_row) % hkv);
  const int r = (int)(idx / ((int64_t)per_row * hkv));
  const int pos = cache_len[b] + r;
  if (pos < 0 || pos >= cap) return;  // out of contract: never write outside the slab
  const int half = c / (per_row / 2), ci = c % (per_row / 2);
  float cs[8], sn[8];
  chunk_angles(half ? pos2[r0 + r] : pos1[r0 + r], ci, d, log2_base, false, cs, sn);
  const int dim = half * (d / 2) + ci * 8;
  const int64_t src = ((int64_t)(r0 + r) * hkv + h) * d + dim;
  const int64_t dst = (((int64_t)b * hkv + h) * cap + pos) * d + dim;
  u32x4 a = *(const u32x4 *)(k_src + src), bb = *(const u32x4 *)(k_src + src + d / 4);
  rope_rotate8(a, bb, cs, sn);
  *(u32x4 *)(k_cache + dst) = a;
  *(u32x4 *)(k_cache + dst + d / 4) = bb;
  *(u32x4 *)(v_cache + dst) = *(const u32x4 *)(v_src + src);
  *(u32x4 *)(v_cache + dst + d / 4) = *(const u32x4 *)(v_src + src + d / 4);
}

}  // namespace

hipError_t launch_positions_2d(const int32_t *cu_seqlens, int32_t batch, const int32_t *cu_segs,
                               int32_t num_segs, int32_t total, int32_t *pos1, int32_t *pos2,
                               hipStream_t stream) {
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(positions_2d_kernel, dim3((total + 255) / 256), dim3(256), 0, stream,
                     cu_seqlens, batch, cu_segs, num_segs, total, pos1, pos2);
  return hipGetLastError();
}

hipError_t launch_rope2d(void *x, bool fp32, int32_t total, int32_t heads, int32_t d,
                         const int32_t *pos1, const int32_t *pos2, float log2_base,
                         bool inverse, hipStream_t stream) {
  const int64_t threads = (int64_t)total * heads * (d / 16);
  if (threads == 0) return hipSuccess;
  const dim3 grid((unsigned)((threads + 255) / 256));
  if (fp32)
    hipLaunchKernelGGL(rope2d_kernel<float>, grid, dim3(256), 0, stream, (float *)x, total,
                       heads, d, pos1, pos2, log2_base, (int32_t)inverse);
  else
    hipLaunchKernelGGL(rope2d_kernel<bf16_t>, grid, dim3(256), 0, stream, (bf16_t *)x, total,
                       heads, d, pos1, pos2, log2_base, (int32_t)inverse);
  return hipGetLastError();
}

hipError_t launch_cache_append_rope(const void *k_src, const void *v_src, void *k_cache,
                                    void *v_cache, const int32_t *cu_new,
                                    const int32_t *cache_len, const int32_t *pos1,
                                    const int32_t *pos2, float log2_base, int32_t batch,
                                    int32_t max_new, int32_t hkv, int32_t d, int32_t cap,
                                    hipStream_t stream) {
  const int64_t threads = (int64_t)max_new * hkv * (d / 16);
  if (threads == 0 || batch == 0) return hipSuccess;
  hipLaunchKernelGGL(cache_append_rope_kernel, dim3((unsigned)((threads + 255) / 256), batch),
                     dim3(256), 0, stream, (const bf16_t *)k_src, (const bf16_t *)v_src,
                     (bf16_t *)k_cache, (bf16_t *)v_cache, cu_new, cache_len, pos1, pos2,
                     log2_base, hkv, d, cap);
  return hipGetLastError();
}

}  // namespace ism
