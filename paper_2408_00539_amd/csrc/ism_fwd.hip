// Forward ISM attention on gfx950: per-token visibility bounds (Eq. 5) and a
// flash-style online-softmax kernel on bf16 MFMA 32x32x16 with fp32
// accumulation. The same kernel serves the cached prefill of a new query
// segment (Sec. 2.3), where every key of the concatenated cache is visible.
//
// Work decomposition. A workgroup (NWV = 4 or 8 waves) owns a row tile of one
// dialogue and a set of query heads that share one KV head: with G = hq / hkv
// query heads per KV head, hpw = gcd(G, NWV) heads run side by side (one per
// wave column) so that the K/V tile staged in LDS serves all of them, and the
// remaining NWV / hpw waves take consecutive 32-row blocks. Each wave
// computes S^T = K Q^T for a 64-key tile (lane <-> query row, so the softmax
// statistics of a row live in one lane pair), then O^T += V^T P^T.
//
// Mask handling. lim(j) is non-decreasing inside a dialogue, so a wave's
// bounds are lim(first row) and lim(last row): key tiles past lim(last row)
// are never visited, tiles ending at or before lim(first row) run with no
// mask instructions, and only the remaining tiles compare key <= lim(row)
// in registers. No N x N mask exists anywhere.
#include "ism_common.h"
#include "ism_kernels.h"

namespace ism {

// lim[j] = inclusive last visible key of token j (Eq. 5, 0-indexed):
// end-1 of its segment for a query segment, j itself for an answer segment.
__global__ void __launch_bounds__(256)
prep_lim_kernel(const int32_t *__restrict__ cu_segs,
                const uint8_t *__restrict__ seg_is_query, int32_t num_segs,
                int32_t total, int32_t *__restrict__ lim) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= total) return;
  int lo = 0, hi = num_segs - 1;  // largest g with cu_segs[g] <= j
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_segs[mid] <= j) lo = mid; else hi = mid - 1;
  }
  lim[j] = seg_is_query[lo] ? cu_segs[lo + 1] - 1 : j;
}

hipError_t launch_prep_lim(const int32_t *cu_segs, const uint8_t *seg_is_query,
                           int32_t num_segs, int32_t total, int32_t *lim,
                           hipStream_t stream) {
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(prep_lim_kernel, dim3((total + 255) / 256), dim3(256), 0,
                     stream, cu_segs, seg_is_query, num_segs, total, lim);
  return hipGetLastError();
}

// Occupancy target in waves per SIMD (1 or 2), which bounds registers.
#ifndef ISM_FWD_WPE
#define ISM_FWD_WPE 2
#endif

namespace {

constexpr int kBN = 64;  // keys per tile
constexpr int kQW = 32;  // query rows per wave

// K and V tiles of 64 keys, row-major, unpadded rows of D bf16 with the
// swz<D>() chunk swizzle, double-buffered; filled by direct global->LDS
// transfers. K is read as MFMA rows (ds_read_b128), V through transposing
// reads (ds_read_b64_tr_b16) as the V^T operand.
template <int D>
struct FwdSmem {
  bf16_t k[2][kBN * D];
  bf16_t v[2][kBN * D];
};

// 2-D rotary positions of one query row held as MFMA operands: qf[ks] holds
// dims 16 ks + 8 hf .. + 7, so each pair (k, k + D/4) of a half lies in
// qf[ks] and qf[ks + D/64] of the same lane.
template <int D>
__device__ __forceinline__ void rope_queries(bf16x8 (&qf)[D / 16], int hf, int p1, int p2,
                                             float log2_base) {
  constexpr int NKS = D / 16, QK = NKS / 4;  // k steps per quarter of the head
#pragma unroll
  for (int half = 0; half < 2; ++half) {
#pragma unroll
    for (int j = 0; j < QK; ++j) {
      const int ks = half * (NKS / 2) + j;
      const int ci = 2 * j + hf;  // 8-dim chunk inside the half's first quarter
      float c[8], s[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) rope_cs(half ? p2 : p1, ci * 8 + e, D / 2, log2_base, c[e], s[e]);
      u32x4 x = __builtin_bit_cast(u32x4, qf[ks]), y = __builtin_bit_cast(u32x4, qf[ks + QK]);
      rope_rotate8(x, y, c, s);
      qf[ks] = __builtin_bit_cast(bf16x8, x);
      qf[ks + QK] = __builtin_bit_cast(bf16x8, y);
    }
  }
}

// S^T[key][row] = K Q^T for one 64-key tile: two 32-key blocks, D/16 steps.
template <int D>
__device__ __forceinline__ void tile_scores(const char *kl, const SwzOffsets<D> &so,
                                            const bf16x8 (&qf)[D / 16], f32x16 (&s)[2]) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      const bf16x8 kf = *(const bf16x8 *)(kl + kb * 32 * D * 2 + so.rowk[ks]);
      s[kb] = mfma32x32x16(kf, qf[ks], ks == 0 ? f32x16{} : s[kb]);
    }
}

// Keys past the row's bound lim get score -inf.
__device__ __forceinline__ void tile_mask(f32x16 (&s)[2], int c0, int hf, int lim) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = c0 + kb * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
      if (key > lim) s[kb][r] = -INFINITY;
    }
}

// Row max of a tile, combined over the lane pair that holds the row.
__device__ __forceinline__ float tile_max(const f32x16 (&s)[2]) {
  float x[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; r += 2) x[r & 3] = vmax(x[r & 3], vmax(s[kb][r], s[kb][r + 1]));
  return pair_max(vmax(vmax(x[0], x[2]), vmax(x[1], x[3])));
}

// Lazy online-softmax update: the reference max is only raised when a row's
// tile max exceeds it by more than tau (2^8 in probability units); exact
// either way since numerator and denominator share the reference max.
template <int NDB>
__device__ __forceinline__ void raise_max(float mt, float sl2, float tau, float &m_run,
                                          float &l_run, f32x16 (&oacc)[NDB]) {
  if (__builtin_amdgcn_ballot_w64(mt > m_run + tau) != 0) {
    const float mnew = vmax(m_run, mt);
    const float alpha = fast_exp2((m_run - mnew) * sl2);
    m_run = mnew;
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
  }
}

// Probabilities 2^(s sl2 - moff) of one tile as bf16 B operands of the P V
// product, and their fp32 row sum.
__device__ __forceinline__ float tile_probs(const f32x16 (&s)[2], float sl2, float moff,
                                            bf16x8 (&pf)[2][2]) {
  float sum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int bt = 0; bt < 2; ++bt) {
      u32x4 w;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        f32x2 p;
        p[0] = fast_exp2(fmaf(s[kb][8 * bt + 2 * u], sl2, -moff));
        p[1] = fast_exp2(fmaf(s[kb][8 * bt + 2 * u + 1], sl2, -moff));
        sum[u] += p[0] + p[1];
        w[u] = cvt_bf16x2(p);
      }
      pf[kb][bt] = __builtin_bit_cast(bf16x8, w);
    }
  return (sum[0] + sum[1]) + (sum[2] + sum[3]);
}

// O^T[d][row] += V^T[d][key] P^T[key][row] for one 64-key tile.
template <int D>
__device__ __forceinline__ void tile_pv(const char *vl, const SwzOffsets<D> &so,
                                        const bf16x8 (&pf)[2][2], f32x16 (&oacc)[D / 32]) {
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int bt = 0; bt < 2; ++bt) {
        const uint32_t o = (kb * 32 + 16 * bt) * D * 2;
        const bf16x8 vf = tr_operand_at(vl, o + so.trk[db][0], o + so.trk[db][1]);
        oacc[db] = mfma32x32x16(vf, pf[kb][bt], oacc[db]);
      }
  }
}

// One pipelined step in a fixed instruction order: the D/8 products of
// S(t+1) = K(t+1) Q^T (its two 32-key blocks alternating), then the D/8
// products of O^T += V(t)^T P(t)^T (64-key chunks outermost), so that
// consecutive products always use different accumulators. Each product is
// followed by the LDS read of the operand LA = 2 products ahead (K rows, then
// transposed V; a third operand in flight measured ~1 % slower, one only
// ~7 % slower) and by its share of the vector work: during
// the S products the exponentials, row sums and bf16 packing of tile t,
// during the P V products the row max of S(t+1). The order is pinned with
// scheduling barriers so that the matrix core and the vector ALU of a wave
// are busy at the same time. Returns the fp32 row sum of P(t); mt receives
// the (unmasked) row max of S(t+1). With LAST (a wave's last tile) there is
// no S(t+1): the exponentials run alone, then the P V products.
// With PRIO the wave raises its issue priority for the first half (the S
// products and the exponentials, the vector-heavy half) and drops it for the
// P V products, so that of the two waves on a SIMD the one in its
// exponentials issues first and the other one's products fill the matrix
// core around it (about 2 % faster on the packed forward; the paged cache,
// whose transfers all start at the step start, measured ~1 % slower with it).
template <int D, bool LAST, bool PRIO, class Hook>
__device__ __forceinline__ float step_block(const char *kl, const char *vl,
                                            const SwzOffsets<D> &so, const bf16x8 (&qf)[D / 16],
                                            const f32x16 (&cur)[2], f32x16 (&nxt)[2],
                                            f32x16 (&oacc)[D / 32], float sl2, float moff,
                                            float &mt, Hook &&hook) {
  constexpr int NKS = D / 16, NDB = D / 32;
  constexpr int NS = 2 * NKS, NP = 4 * NDB, N = NS + NP, LA = 2;
  constexpr int PPS = 16 / NS;  // probability pairs per S product
  constexpr int MPP = 32 / NP;  // max elements per P V product
  auto read = [&](int n) -> bf16x8 {
    if (n < NS) {
      const int kb = n & 1, ks = n >> 1;
      return *(const bf16x8 *)(kl + kb * 32 * D * 2 + so.rowk[ks]);
    }
    const int j = n - NS, kc = j / NDB, db = j % NDB;
    const uint32_t o = ((kc >> 1) * 32 + 16 * (kc & 1)) * D * 2;
    return tr_operand_at(vl, o + so.trk[db][0], o + so.trk[db][1]);
  };
  constexpr int F = LAST ? NS : 0;  // first product that runs
  bf16x8 op[N];
#pragma unroll
  for (int n = F; n < F + LA; ++n) op[n] = read(n);
  u32x4 w[2][2];
  float sum[2] = {0.f, 0.f}, mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
  for (int n = 0; n < N; ++n) {
    if (PRIO && n == 0) __builtin_amdgcn_s_setprio(1);
    if (PRIO && n == NS) __builtin_amdgcn_s_setprio(0);
    if (n < NS) {
      if (!LAST) {
        const int kb = n & 1, ks = n >> 1;
        nxt[kb] = mfma32x32x16(op[n], qf[ks], ks == 0 ? f32x16{} : nxt[kb]);
      }
    } else {
      const int j = n - NS, kc = j / NDB, db = j % NDB;
      oacc[db] = mfma32x32x16(op[n], __builtin_bit_cast(bf16x8, w[kc >> 1][kc & 1]), oacc[db]);
    }
    hook(n);  // n is a constant once the loop is unrolled
    if (n >= F && n + LA < N) op[n + LA] = read(n + LA);
    if (n < NS) {
#pragma unroll
      for (int c = 0; c < PPS; ++c) {
        const int i = n * PPS + c, kb = i >> 3, bt = (i >> 2) & 1, u = i & 3;
        f32x2 p;
        p[0] = fast_exp2(fmaf(cur[kb][8 * bt + 2 * u], sl2, -moff));
        p[1] = fast_exp2(fmaf(cur[kb][8 * bt + 2 * u + 1], sl2, -moff));
        sum[i & 1] += p[0] + p[1];
        w[kb][bt][u] = cvt_bf16x2(p);
        asm volatile("" : "+v"(sum[i & 1]));  // keep the add in this slot
      }
    } else if (!LAST) {
#pragma unroll
      for (int c = 0; c < MPP; c += 2) {
        const int e = (n - NS) * MPP + c, m = (e >> 1) & 1;
        mx[m] = vmax(mx[m], vmax(nxt[e >> 4][e & 15], nxt[e >> 4][(e & 15) + 1]));
        asm volatile("" : "+v"(mx[m]));
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  mt = LAST ? -INFINITY : pair_max(vmax(mx[0], mx[1]));
  return sum[0] + sum[1];
}

// NT: non-temporal tile transfers, for a cache-mode launch in which every
// (dialogue, head set) group has a single row tile, so that no other
// workgroup reads its K/V (verifying 8 drafted tokens per dialogue through
// the cache ran 11 % faster; with several row tiles per group the same bit
// cost the L2 sharing between them: the workload-3 prefill ran 22 % slower).
template <int D, bool CACHE, int NWV, bool PAGED, bool NT>
__global__ void __launch_bounds__(NWV * 64)
__attribute__((amdgpu_waves_per_eu(ISM_FWD_WPE, ISM_FWD_WPE)))
fwd_kernel(FwdArgs a, int hpw, int tiles, int chunk) {
  constexpr int NDB = D / 32;      // 32-wide d blocks of the output
  constexpr int NKS = D / 16;      // 16-deep k steps of Q K^T
  __shared__ FwdSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int l32 = lane & 31, hf = lane >> 5;

  // Work item: (dialogue, head set) groups in XCD-aware chunks, longest row
  // tile first inside each chunk.
  const int hsets = a.hq / hpw;
  int group, tile;
  if (!xcd_work_item((int)blockIdx.x, a.batch * hsets, tiles, chunk, true, group, tile)) return;
  const int b = group / hsets;
  const int head0 = (group % hsets) * hpw;
  const int wg_rows = (NWV / hpw) * kQW;
  const int s = a.cu_q[b], e = a.cu_q[b + 1];
  const int q0 = s + tile * wg_rows;
  if (q0 >= e) return;

  const int head = head0 + wave % hpw;
  const int kvh = head0 / (a.hq / a.hkv);
  const int wq0 = q0 + (wave / hpw) * kQW;
  const bool active = wq0 < e;
  const int wg_last = min(q0 + wg_rows, e) - 1;

  int key_begin, key_hi, wave_lo, wave_hi, cache_c = 0;
  bool oob = false;  // cache mode: C_b + L_b outside the cache (out of contract)
  const bf16_t *kbase, *vbase;
  if (CACHE) {
    key_begin = 0;
    cache_c = a.cache_len[b];
    // keys [0, C_b + L_b) (query segment) or [0, C_b + r] for row r (answer
    // segment); clamped to the slab for out-of-contract lengths, whose rows
    // get NaN
    const int slab_rows = PAGED ? a.max_pages * a.page_size : (int)(a.kv_head_stride / D);
    oob = cache_c < 0 || cache_c + (e - s) > slab_rows;
    if (a.cache_causal) {
      key_hi = max(min(cache_c + (wg_last - s) + 1, slab_rows) - 1, 0);
      wave_lo = min(cache_c + (min(wq0, e - 1) - s), key_hi);
      wave_hi = active ? min(cache_c + (min(wq0 + kQW, e) - 1 - s), key_hi) : -1;
    } else {
      key_hi = max(min(cache_c + (e - s), slab_rows) - 1, 0);
      wave_lo = key_hi;
      wave_hi = active ? key_hi : -1;
    }
    const int64_t off =
        PAGED ? 0 : (int64_t)b * a.kv_seq_stride + (int64_t)kvh * a.kv_head_stride;
    kbase = (const bf16_t *)a.k + off;
    vbase = (const bf16_t *)a.v + off;
  } else {
    key_begin = s;
    key_hi = a.lim[wg_last];
    wave_lo = a.lim[min(wq0, e - 1)];
    wave_hi = active ? a.lim[min(wq0 + kQW, e) - 1] : s - 1;
    kbase = (const bf16_t *)a.k + (int64_t)kvh * a.kv_head_stride;
    vbase = (const bf16_t *)a.v + (int64_t)kvh * a.kv_head_stride;
  }
  const int64_t rs = a.kv_row_stride;
  const float sl2 = a.scale * kLog2e;
  // first key of tile t of the workgroup's key range (t < its tile count);
  // in the paged cache a 64-key tile lies inside one page
  const int32_t *btab = a.block_table;
  const int pg_max = a.max_pages, pg_num = a.num_pages, pg_size = a.page_size, nkv = a.hkv;
  auto tile_src = [&](const bf16_t *base, int t) __attribute__((always_inline)) {
    if constexpr (PAGED)
      return base + paged_offset_uniform(btab, pg_max, pg_num, pg_size, nkv, D, b, kvh, t * kBN);
    else
      return base + (int64_t)key_begin * rs + (int64_t)t * (kBN * rs);
  };
  // lazy rescale threshold: 2^8 in probability units
  const float tau = 8.f / sl2;

  // Prologue, with its memory latencies overlapped: the transfers of K(0),
  // V(0) and K(1) need only the dialogue's key range in memory (packed mode:
  // keys past the workgroup's bound are real keys of the dialogue, masked
  // like any other invisible key), so they start before the bounds and Q.
  DmaTile<D, kBN, NWV, NT> dma;
  dma.init(tid, rs);
  {
    const int mem_rows = CACHE ? key_hi - key_begin + 1 : e - key_begin;
    const bf16_t *k0 = tile_src(kbase, 0);
    dma.issue(k0, rs, mem_rows, sm.k[0]);
    dma.issue(tile_src(vbase, 0), rs, mem_rows, sm.v[0]);
    if (mem_rows > kBN)
      dma.issue(PAGED ? tile_src(kbase, 1) : k0 + (int64_t)kBN * rs, rs, mem_rows - kBN,
                sm.k[1]);
  }
  // Per-lane query row (clamped into the dialogue; rows past e are computed
  // as copies of the last row and never stored).
  const int rc = min(wq0 + l32, e - 1);
  const int lim_r = !CACHE          ? a.lim[rc]
                    : a.cache_causal ? min(cache_c + (rc - s), key_hi)
                                     : key_hi;
  bf16x8 qf[NKS];
  {
    const bf16_t *qp = (const bf16_t *)a.q + ((int64_t)rc * a.hq + head) * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = *(const bf16x8 *)(qp + ks * 16);
  }
  if constexpr (CACHE) {
    if (a.rope_pos1) rope_queries<D>(qf, hf, a.rope_pos1[rc], a.rope_pos2[rc], a.rope_log2_base);
  }
  wait_loads();  // Q, lim and the transfers above
  __syncthreads();

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  // Software pipeline over key tiles. Tile t's scores S(t) are complete (and
  // masked, the running max raised) when step t starts; step t then issues
  // S(t+1) = K(t+1) Q^T and the P(t) V(t) product in the same basic block as
  // the exponentials of tile t, so matrix and vector work of one wave
  // overlap. LDS holds K(t+1) and V(t) during step t while K(t+2) and V(t+1)
  // are in flight into the other halves of the double buffers.
  const int ntiles = (key_hi - key_begin) / kBN + 1;  // for the workgroup
  const int nw = active ? (wave_hi - key_begin) / kBN + 1 : 0;  // this wave's
  const int64_t tile_elems = (int64_t)kBN * rs;
  const bf16_t *kt = kbase + (int64_t)key_begin * rs;
  const bf16_t *vt = vbase + (int64_t)key_begin * rs;
  // paged cache: sources of K(t+2) and V(t+1) for step t
  const bf16_t *pk2 = PAGED ? tile_src(kbase, min(2, ntiles - 1)) : kt;
  const bf16_t *pv1 = PAGED ? tile_src(vbase, min(1, ntiles - 1)) : vt;
  SwzOffsets<D> so;
  so.init(lane);

  f32x16 sa[2], sb[2];
  if (nw > 0) {
    tile_scores<D>((const char *)sm.k[0], so, qf, sa);
    if (key_begin + kBN - 1 > wave_lo) tile_mask(sa, key_begin, hf, lim_r);
    raise_max(tile_max(sa), sl2, tau, m_run, l_run, oacc);
  }
  lds_barrier();  // every wave is done with K(0) before K(2) overwrites it

  // Step t. MODE 0: K(t+2) and V(t+1) are full tiles, transferred one
  // transfer every third product from the first (a burst of transfers
  // stalls the waves that issue them; one every fourth product, the last
  // near the step end, measured 1.5-3 % slower with the phase priority of
  // step_block); MODE 1: the transfers at once (partial tiles near the end
  // of the key range); MODE 2: the workgroup's last tile, which has no
  // S(t+1) and no transfers, so the waves whose last tile it is run the
  // exponentials and P V only. (A wave whose last tile comes earlier
  // computes an unused S(t+1) there, which keeps one code path per loop.)
  auto step = [&](f32x16 (&cur)[2], f32x16 (&nxt)[2], int t, auto modec) {
    constexpr int MODE = decltype(modec)::value;
    constexpr bool LAST = MODE == 2;
    constexpr int NI = decltype(dma)::NI;
    static_assert(3 * (2 * NI - 1) < 2 * (D / 16) + 4 * (D / 32),
                  "every full-tile transfer falls inside the step's products");
    const int c0 = key_begin + t * kBN;
    const bf16_t *ksrc = PAGED ? pk2 : kt + 2 * tile_elems;
    const bf16_t *vsrc = PAGED ? pv1 : vt + tile_elems;
    if (MODE == 1 || (MODE == 0 && t >= nw)) {
      if (t + 2 < ntiles)
        dma.issue(ksrc, rs, key_hi - (c0 + 2 * kBN) + 1, sm.k[t & 1]);
      dma.issue(vsrc, rs, key_hi - (c0 + kBN) + 1, sm.v[(t + 1) & 1]);
    }
    const char *kl = (const char *)sm.k[(t + 1) & 1];
    const char *vl = (const char *)sm.v[t & 1];
    auto hook = [&](int n) __attribute__((always_inline)) {
      if (MODE == 0 && n % 3 == 0 && n / 3 < 2 * NI) {
        if (n / 3 < NI) dma.issue_one(ksrc, n / 3, sm.k[t & 1]);
        else dma.issue_one(vsrc, n / 3 - NI, sm.v[(t + 1) & 1]);
      }
    };
    if (t < nw) {
      float mt;
      l_run += step_block<D, LAST, !PAGED>(kl, vl, so, qf, cur, nxt, oacc, sl2, m_run * sl2, mt,
                                           hook);
      if (!LAST && t + 1 < nw) {
        if (c0 + 2 * kBN - 1 > wave_lo) {  // S(t+1) crosses some row's bound
          tile_mask(nxt, c0 + kBN, hf, lim_r);
          mt = tile_max(nxt);
        }
        raise_max(mt, sl2, tau, m_run, l_run, oacc);
      }
    }
    if (!LAST) {
      kt += tile_elems;
      vt += tile_elems;
      if constexpr (PAGED) {  // K(t+3) and V(t+2), re-based at page starts
        const int tpp = pg_size / kBN;
        pk2 = (t + 3) % tpp ? pk2 + tile_elems : tile_src(kbase, min(t + 3, ntiles - 1));
        pv1 = (t + 2) % tpp ? pv1 + tile_elems : tile_src(vbase, min(t + 2, ntiles - 1));
      }
    }
    wait_vmem();
    __syncthreads();
  };
  // steps whose K(t+2) and V(t+1) are full tiles, an even count of them
  // (the paged cache looks up each tile's page at the step start and issues
  // its transfers at once)
  int t = 0;
  if constexpr (!PAGED) {
    const int nfull = max((key_hi - key_begin + 1) / kBN - 2, 0) & ~1;
    for (; t < nfull; t += 2) {
      step(sa, sb, t, std::integral_constant<int, 0>{});
      step(sb, sa, t + 1, std::integral_constant<int, 0>{});
    }
  }
  for (; t + 1 < ntiles; t += 2) {
    step(sa, sb, t, std::integral_constant<int, 1>{});
    if (t + 2 < ntiles) step(sb, sa, t + 1, std::integral_constant<int, 1>{});
  }
  if ((ntiles - 1) & 1) step(sb, sa, ntiles - 1, std::integral_constant<int, 2>{});
  else step(sa, sb, ntiles - 1, std::integral_constant<int, 2>{});

  if (!active) return;
  const float lt = pair_sum(l_run);
  const int row = wq0 + l32;
  if (row >= e) return;
  const float inv = oob ? __builtin_nanf("") : 1.f / lt;
  bf16_t *op = (bf16_t *)a.o + ((int64_t)row * a.hq + head) * D + hf * 4;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      u32x2 w;
      w[0] = pack_bf16x2(oacc[db][4 * i + 0] * inv, oacc[db][4 * i + 1] * inv);
      w[1] = pack_bf16x2(oacc[db][4 * i + 2] * inv, oacc[db][4 * i + 3] * inv);
      *(u32x2 *)(op + db * 32 + 8 * i) = w;
    }
  if (a.lse && hf == 0)
    a.lse[(int64_t)head * a.total_q + row] = oob ? __builtin_nanf("") : m_run * a.scale + logf(lt);
}

int gcd_int(int x, int y) {
  while (y) { const int t = x % y; x = y; y = t; }
  return x;
}

template <int D, bool CACHE, int NWV, bool PAGED>
hipError_t launch_fwd_w(const FwdArgs &a, hipStream_t stream) {
  const int hpw = gcd_int(a.hq / a.hkv, NWV);
  const int wg_rows = (NWV / hpw) * kQW;
  const int tiles = (a.max_rows + wg_rows - 1) / wg_rows;
  const int64_t groups = (int64_t)a.batch * (a.hq / hpw);
  if (groups * tiles == 0) return hipSuccess;
  const dim3 grid((unsigned)xcd_grid(groups, tiles));
  if constexpr (CACHE) {
    if (tiles == 1) {
      hipLaunchKernelGGL((fwd_kernel<D, true, NWV, PAGED, true>), grid, dim3(NWV * 64), 0,
                         stream, a, hpw, tiles, ISM_SCHED_CHUNK);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((fwd_kernel<D, CACHE, NWV, PAGED, false>), grid, dim3(NWV * 64), 0,
                     stream, a, hpw, tiles, ISM_SCHED_CHUNK);
  return hipGetLastError();
}

// Grouped KV heads run 8-wave workgroups (one per CU): the heads of a group
// and two 32-row blocks share each staged K/V tile, half the transfers per
// product of 4-wave workgroups. Without grouping, 8 waves would be 256 rows
// of one head, whose waves finish at different key tiles; 4 waves (two
// workgroups per CU) measure as fast there.
template <int D, bool CACHE, bool PAGED>
hipError_t launch_fwd_p(const FwdArgs &a, hipStream_t stream) {
  return a.hq / a.hkv >= 2 ? launch_fwd_w<D, CACHE, 8, PAGED>(a, stream)
                           : launch_fwd_w<D, CACHE, 4, PAGED>(a, stream);
}

template <int D, bool CACHE>
hipError_t launch_fwd_t(const FwdArgs &a, hipStream_t stream) {
  if (CACHE && a.block_table) return launch_fwd_p<D, true, true>(a, stream);
  return launch_fwd_p<D, CACHE, false>(a, stream);
}

}  // namespace

hipError_t launch_fwd(const FwdArgs &a, int d, bool cache_mode,
                      hipStream_t stream) {
  if (d == 128) return cache_mode ? launch_fwd_t<128, true>(a, stream)
                                  : launch_fwd_t<128, false>(a, stream);
  if (d == 64) return cache_mode ? launch_fwd_t<64, true>(a, stream)
                                 : launch_fwd_t<64, false>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace ism
