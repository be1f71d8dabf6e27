// KV-cache reuse path of ISM attention on gfx950 (Sec. 2.3 of the paper):
//  * cache append of a new query segment's keys/values (before the cached
//    prefill, which then runs the forward kernel in cache mode);
//  * one answer-token decode step: the token at position p sees keys
//    [0, p] (Eq. 5 third case). The key range is split into chunks; each
//    workgroup streams one chunk of one (dialogue, KV head) slab with 16-byte
//    coalesced loads and keeps an unnormalised partial (m, l, o); a second
//    kernel merges the partials exactly. The workgroup whose chunk holds p
//    reads the new key/value from the input and also writes it into the
//    cache, so no separate append launch is needed.
//
// Decode is an HBM stream (one query row per head: ~1 FLOP per byte per
// head), so with 1-3 query heads per KV head it can use vector dot
// products; with 4 or more the vector work would bound it, and a
// matrix-core kernel takes those head sets (all heads of a KV head as the
// columns of one product). The matrix-core kernel also takes 1-3 heads when
// the step has few (dialogue, KV head) slabs, where its long one-wave
// chunks stream faster (decode_mma_heads).
#include "ism_common.h"
#include "ism_kernels.h"

namespace ism {

namespace {

__global__ void __launch_bounds__(256)
cache_append_kernel(const bf16_t *__restrict__ k_src,
                    const bf16_t *__restrict__ v_src, bf16_t *__restrict__ k_cache,
                    bf16_t *__restrict__ v_cache, const int32_t *__restrict__ cu_new,
                    const int32_t *__restrict__ cache_len, int32_t hkv, int32_t d,
                    int32_t cap) {
  const int b = blockIdx.y;
  const int r0 = cu_new[b], n = cu_new[b + 1] - r0;
  const int cpr = hkv * (d / 8);  // 16-byte chunks per source row
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n * cpr) return;
  const int r = (int)(idx / cpr), rem = (int)(idx % cpr);
  const int pos = cache_len[b] + r;
  if (pos < 0 || pos >= cap) return;  // out of contract: never write outside the slab
  const int h = rem / (d / 8), c = rem % (d / 8);
  const int64_t src = ((int64_t)(r0 + r) * hkv + h) * d + c * 8;
  const int64_t dst = (((int64_t)b * hkv + h) * cap + pos) * d + c * 8;
  *(u32x4 *)(k_cache + dst) = *(const u32x4 *)(k_src + src);
  *(u32x4 *)(v_cache + dst) = *(const u32x4 *)(v_src + src);
}

__global__ void __launch_bounds__(256)
cache_append_paged_kernel(const bf16_t *__restrict__ k_src, const bf16_t *__restrict__ v_src,
                          bf16_t *__restrict__ k_pages, bf16_t *__restrict__ v_pages,
                          const int32_t *__restrict__ cu_new,
                          const int32_t *__restrict__ cache_len,
                          const int32_t *__restrict__ block_table, int32_t max_pages,
                          int32_t num_pages, int32_t page_size, int32_t hkv, int32_t d) {
  const int b = blockIdx.y;
  const int r0 = cu_new[b], n = cu_new[b + 1] - r0;
  const int cpr = hkv * (d / 8);
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n * cpr) return;
  const int r = (int)(idx / cpr), rem = (int)(idx % cpr);
  const int pos = cache_len[b] + r;
  if (pos < 0 || pos >= max_pages * page_size) return;  // out of contract
  const int h = rem / (d / 8), c = rem % (d / 8);
  const int64_t src = ((int64_t)(r0 + r) * hkv + h) * d + c * 8;
  const int64_t dst =
      paged_offset(block_table, max_pages, num_pages, page_size, hkv, d, b, h, pos) + c * 8;
  *(u32x4 *)(k_pages + dst) = *(const u32x4 *)(k_src + src);
  *(u32x4 *)(v_pages + dst) = *(const u32x4 *)(v_src + src);
}

// Sum of x over each group of N (8 or 16) consecutive lanes, in every lane
// of the group, through DPP lane moves (no LDS round trip, unlike a
// shuffle): quad xor 1, quad xor 2, the mirror inside each 8-lane half row,
// and for N = 16 the mirror inside the 16-lane row. Each step adds two values
// that are uniform over their subgroups, so all lanes end with the same bits.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(N == 8 || N == 16, "groups of 8 or 16 lanes");
  x += dpp_move<0xB1>(x);   // quad_perm [1, 0, 3, 2]
  x += dpp_move<0x4E>(x);   // quad_perm [2, 3, 0, 1]
  x += dpp_move<0x141>(x);  // row_half_mirror
  if constexpr (N == 16) x += dpp_move<0x140>(x);  // row_mirror
  return x;
}

// Split decode step. Each dialogue's key range [0, p] is cut into a.splits
// chunks of equal length rounded up to a whole workgroup iteration (4 KPW
// keys), so every chunk but the last runs whole iterations and the longest
// chunk is as short as the split count allows, whatever the cache capacity;
// trailing chunks of a short dialogue may be empty (partial m = -inf, l = 0).
// PAGED: the cache is a page pool (DecodeArgs); the keys of one wave
// iteration (KPW consecutive, KPW-aligned) lie in one page, whose address
// is looked up once per iteration.
// A workgroup serves GS query heads that share one KV head (GS divides
// G = hq / hkv and is at most 8, so that the per-head registers fit): head
// set hs covers query heads hs GS .. hs GS + GS - 1 of KV head hs GS / G.
// With G > 8 the G / GS sets of a KV head stream its keys separately.
// Sets of 4 or more heads go to decode_mma_kernel below, so GS <= 3 here.
// (Steps with few slabs send every set there.)
template <int D, int GS, bool PAGED>
__global__ void __launch_bounds__(256)
decode_split_kernel(DecodeArgs a) {
  static_assert(GS >= 1 && GS <= 3, "larger head sets run on the matrix cores");
  constexpr int CPK = D / 8;     // lanes per key row (16 bytes each)
  constexpr int KPI = 64 / CPK;  // keys per wave-wide load
  constexpr int U = 8;           // loads in flight per lane per tensor
  constexpr int KPW = U * KPI;   // keys per wave per iteration
  __shared__ float sm_o[4][GS][D];
  __shared__ float sm_m[4][GS], sm_l[4][GS];

  const int split = blockIdx.x, hs = blockIdx.y, b = blockIdx.z;
  const int head0 = hs * GS;
  const int kvh = head0 / (a.hq / a.hkv);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane % CPK, slot = lane / CPK;
  // position of the new token; an out-of-contract position (outside the
  // cache) is clamped so that no access leaves the slab, nothing is
  // appended, and the combine writes NaN for the dialogue
  const int praw = a.pos[b];
  const bool in_cap = praw >= 0 && praw < a.cap;
  const int p = min(max(praw, 0), a.cap - 1);
  // chunk * splits >= p + 1, so the chunks cover [0, p] and p / chunk is a
  // valid split
  constexpr int kGran = 4 * KPW;
  const int chunk = ((p + a.splits) / a.splits + kGran - 1) / kGran * kGran;
  const int k0 = split * chunk;
  const int k1 = min(k0 + chunk, p + 1);
  const int owner = p / chunk;
  const float sl2 = a.scale * kLog2e;

  // element offset of key t's row (dense slab or page pool)
  const int64_t slab = ((int64_t)b * a.hkv + kvh) * a.cap * D;
  auto row_of = [&](int t) -> int64_t {
    if (PAGED)
      return paged_offset_uniform(a.block_table, a.max_pages, a.num_pages, a.page_size, a.hkv,
                                  D, b, kvh, t);
    return slab + (int64_t)t * D;
  };
  const bf16_t *kn = (const bf16_t *)a.k_new + ((int64_t)b * a.hkv + kvh) * D + c * 8;
  const bf16_t *vn = (const bf16_t *)a.v_new + ((int64_t)b * a.hkv + kvh) * D + c * 8;

  if (in_cap && split == owner && head0 % (a.hq / a.hkv) == 0 && tid < CPK) {
    // this chunk (of the KV head's first head set) owns the new token:
    // store it into the cache
    const int64_t prow = row_of(p);
    *(u32x4 *)((bf16_t *)a.k_cache + prow + tid * 8) =
        *(const u32x4 *)((const bf16_t *)a.k_new + ((int64_t)b * a.hkv + kvh) * D + tid * 8);
    *(u32x4 *)((bf16_t *)a.v_cache + prow + tid * 8) =
        *(const u32x4 *)((const bf16_t *)a.v_new + ((int64_t)b * a.hkv + kvh) * D + tid * 8);
  }

  float qv[GS][8];
#pragma unroll
  for (int g = 0; g < GS; ++g) {
    const u32x4 w = *(const u32x4 *)((const bf16_t *)a.q +
                                     ((int64_t)b * a.hq + head0 + g) * D + c * 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      qv[g][2 * i] = bf16_lo(w[i]) * sl2;
      qv[g][2 * i + 1] = bf16_hi(w[i]) * sl2;
    }
  }
  float m[GS], l[GS], o[GS][8];
#pragma unroll
  for (int g = 0; g < GS; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[g][i] = 0.f;
  }

  for (int base = k0 + wave * KPW; base < k1; base += 4 * KPW) {
    u32x4 kr[U], vr[U];
    // keys [base, base + KPW) of this iteration: one page when paged
    const int64_t brow = row_of(base) - (int64_t)base * D;
    const bf16_t *kc = (const bf16_t *)a.k_cache + brow + c * 8;
    const bf16_t *vc = (const bf16_t *)a.v_cache + brow + c * 8;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int key = min(base + u * KPI + slot, p);
      const bool isnew = key == p;
      // non-temporal: the cache is read once per step and must not evict
      // anything (streaming reads reach ~7.1 TB/s this way, ~6.3 TB/s with
      // ordinary loads)
      kr[u] = __builtin_nontemporal_load((const u32x4 *)(isnew ? kn : kc + (int64_t)key * D));
      vr[u] = __builtin_nontemporal_load((const u32x4 *)(isnew ? vn : vc + (int64_t)key * D));
    }
#pragma unroll
    for (int g = 0; g < GS; ++g) {
      float s[U];
      float mt = -INFINITY;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc = fmaf(qv[g][2 * i], bf16_lo(kr[u][i]), acc);
          acc = fmaf(qv[g][2 * i + 1], bf16_hi(kr[u][i]), acc);
        }
        acc = group_sum<CPK>(acc);
        s[u] = (base + u * KPI + slot < k1) ? acc : -INFINITY;
        mt = fmaxf(mt, s[u]);
      }
      const float mnew = fmaxf(m[g], mt);
      const float mref = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = fast_exp2(m[g] - mref);
      m[g] = mnew;
      l[g] *= alpha;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] *= alpha;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float pu = fast_exp2(s[u] - mref);
        l[g] += pu;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          o[g][2 * i] = fmaf(pu, bf16_lo(vr[u][i]), o[g][2 * i]);
          o[g][2 * i + 1] = fmaf(pu, bf16_hi(vr[u][i]), o[g][2 * i + 1]);
        }
      }
    }
  }

  // merge the key slots of the wave (lanes with equal c), then the 4 waves
#pragma unroll
  for (int g = 0; g < GS; ++g) {
#pragma unroll
    for (int x = CPK; x < 64; x <<= 1) {
      const float m2 = __shfl_xor(m[g], x);
      const float l2 = __shfl_xor(l[g], x);
      const float mn = fmaxf(m[g], m2);
      const float mref = mn == -INFINITY ? 0.f : mn;
      const float f1 = fast_exp2(m[g] - mref), f2 = fast_exp2(m2 - mref);
      l[g] = l[g] * f1 + l2 * f2;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float o2 = __shfl_xor(o[g][i], x);
        o[g][i] = o[g][i] * f1 + o2 * f2;
      }
      m[g] = mn;
    }
    if (slot == 0) {
#pragma unroll
      for (int i = 0; i < 8; ++i) sm_o[wave][g][c * 8 + i] = o[g][i];
      if (c == 0) { sm_m[wave][g] = m[g]; sm_l[wave][g] = l[g]; }
    }
  }
  __syncthreads();
  for (int t = tid; t < GS * D; t += 256) {
    const int g = t / D, dd = t % D;
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) mx = fmaxf(mx, sm_m[w][g]);
    const float mref = mx == -INFINITY ? 0.f : mx;
    float lt = 0.f, ot = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = fast_exp2(sm_m[w][g] - mref);
      lt += sm_l[w][g] * f;
      ot += sm_o[w][g][dd] * f;
    }
    const int h = head0 + g;
    const int64_t pi = ((int64_t)b * a.hq + h) * a.splits + split;
    a.part_o[pi * D + dd] = ot;
    if (dd == 0) {
      a.part_ml[pi * 2] = mx;
      a.part_ml[pi * 2 + 1] = lt;
    }
  }
}

// Decode step with matrix cores, for head sets of 4 or more query heads per
// KV head (the vector kernel above is then bound by its FMAs, not by HBM),
// and for sets of any size on steps with few (dialogue, KV head) slabs.
// One wave per workgroup streams one chunk of one (dialogue, KV head) slab
// in 32-key tiles through a 2-stage LDS ring (direct global->LDS transfers,
// the forward kernel's swizzled tile layout) and treats the set's query
// heads as the 32 columns of the forward's products: S^T = K Q^T (lane <->
// head, the columns past the set's heads hold zero queries and are never
// written), an online softmax in exp2 form with the forward's lazy
// rescaling, and O^T += V^T P^T with V^T through transposing reads. The
// chunk holding the new position p patches the new key/value row into its
// LDS tile (the cache row may not hold it yet: the first head set's owner
// chunk writes it to the cache in the same launch). Chunks are whole tiles,
// so a tile of the paged cache lies inside one page (page sizes are
// multiples of 64 positions).
// Partials (m in log2 units, l, o) go to the same split buffers as the
// vector kernel's, merged by decode_combine_kernel.
constexpr int kDecTile = 32;  // keys per tile
template <int D>
struct DecMmaSmem {
  bf16_t k[2][kDecTile * D];
  bf16_t v[2][kDecTile * D];
};

template <int D, bool PAGED>
__global__ void __launch_bounds__(64)
decode_mma_kernel(DecodeArgs a) {
  constexpr int NKS = D / 16, NDB = D / 32, RB = 2 * D;
  using Dma = DmaTile<D, kDecTile, 1, true>;  // the cache is read once per step
  constexpr int NI = Dma::NI;  // transfers per tile and tensor
  __shared__ DecMmaSmem<D> sm;

  const int split = blockIdx.x, hs = blockIdx.y, b = blockIdx.z;
  const int gs = a.set_heads, G = a.hq / a.hkv;
  const int head0 = hs * gs, kvh = head0 / G;
  const int lane = threadIdx.x, l32 = lane & 31, hf = lane >> 5;
  // position of the new token, clamped as in the vector kernel
  const int praw = __builtin_amdgcn_readfirstlane(a.pos[b]);
  const bool in_cap = praw >= 0 && praw < a.cap;
  const int p = min(max(praw, 0), a.cap - 1);
  const int chunk = ((p + a.splits) / a.splits + kDecTile - 1) / kDecTile * kDecTile;
  const int k0 = split * chunk, k1 = min(k0 + chunk, p + 1);
  const int owner = p / chunk;
  const float sl2 = a.scale * kLog2e;
  const int64_t slab = ((int64_t)b * a.hkv + kvh) * a.cap * D;
  auto row_of = [&](int t) -> int64_t {  // element offset of key t's row
    if (PAGED)
      return paged_offset_uniform(a.block_table, a.max_pages, a.num_pages, a.page_size, a.hkv,
                                  D, b, kvh, t);
    return slab + (int64_t)t * D;
  };

  // the new key/value row: 16 bytes per lane in lanes 0 .. D/8 - 1
  constexpr int CPR = D / 8;
  const bool patch = in_cap && split == owner;
  u32x4 knew{}, vnew{};
  if (patch && lane < CPR) {
    const int64_t src = ((int64_t)b * a.hkv + kvh) * D + lane * 8;
    knew = *(const u32x4 *)((const bf16_t *)a.k_new + src);
    vnew = *(const u32x4 *)((const bf16_t *)a.v_new + src);
    if (head0 % G == 0) {  // the KV head's first set stores it into the cache
      const int64_t prow = row_of(p);
      *(u32x4 *)((bf16_t *)a.k_cache + prow + lane * 8) = knew;
      *(u32x4 *)((bf16_t *)a.v_cache + prow + lane * 8) = vnew;
    }
  }
  // B operands of S^T = K Q^T: column l32 is query head head0 + l32
  bf16x8 qf[NKS];
  {
    const bool real = l32 < gs;
    const bf16_t *qp =
        (const bf16_t *)a.q + ((int64_t)b * a.hq + head0 + (real ? l32 : 0)) * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[ks] = real ? *(const bf16x8 *)(qp + ks * 16) : bf16x8{};
  }

  Dma dma;
  dma.init(lane, D);
  SwzOffsets<D> so;
  so.init(lane);
  const int nt = k0 < k1 ? (k1 - k0 + kDecTile - 1) / kDecTile : 0;
  auto issue = [&](int t) __attribute__((always_inline)) {  // tile t into stage t & 1
    const int c = k0 + t * kDecTile;
    const int64_t off = row_of(c);
    const int nv = min(kDecTile, k1 - c);  // rows past it repeat the last valid one
    dma.issue((const bf16_t *)a.k_cache + off, D, nv, sm.k[t & 1]);
    dma.issue((const bf16_t *)a.v_cache + off, D, nv, sm.v[t & 1]);
  };
  wait_loads();  // queries, the new row and its store
  if (nt > 0) issue(0);

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const float tau = 8.f / sl2;  // lazy rescale threshold: 2^8 in probability units
  for (int t = 0; t < nt; ++t) {
    // tile t + 1 goes into the stage tile t - 1 used (its reads are done:
    // their products consumed them); then wait for tile t only
    if (t + 1 < nt) {
      issue(t + 1);
      wait_vmem_but<2 * NI>();
    } else {
      wait_vmem();
    }
    const int c0 = k0 + t * kDecTile;
    bf16_t *kt = sm.k[t & 1];
    bf16_t *vt = sm.v[t & 1];
    if (patch && p - c0 < kDecTile && lane < CPR) {
      const int r = p - c0;
      const int e = r * D + ((lane ^ swz<D>(r)) << 3);
      *(u32x4 *)(kt + e) = knew;
      *(u32x4 *)(vt + e) = vnew;
    }
    const char *kl = (const char *)kt;
    const char *vl = (const char *)vt;
    f32x16 sc;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      sc = mfma32x32x16(*(const bf16x8 *)(kl + so.rowk[ks]), qf[ks], ks == 0 ? f32x16{} : sc);
    if (c0 + kDecTile > k1) {  // the chunk's last tile: keys past k1 - 1 get -inf
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (c0 + (r >> 2) * 8 + hf * 4 + (r & 3) >= k1) sc[r] = -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; r += 2) mt = vmax(mt, vmax(sc[r], sc[r + 1]));
    mt = pair_max(mt);
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
    const float moff = m_run * sl2;
    bf16x8 pf[2];
    float sum = 0.f;
#pragma unroll
    for (int bt = 0; bt < 2; ++bt) {
      u32x4 w;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        f32x2 pr;
        pr[0] = fast_exp2(fmaf(sc[8 * bt + 2 * u], sl2, -moff));
        pr[1] = fast_exp2(fmaf(sc[8 * bt + 2 * u + 1], sl2, -moff));
        sum += pr[0] + pr[1];
        w[u] = cvt_bf16x2(pr);
      }
      pf[bt] = __builtin_bit_cast(bf16x8, w);
    }
    l_run += sum;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int bt = 0; bt < 2; ++bt) {
        const uint32_t o = 16 * bt * RB;
        oacc[db] = mfma32x32x16(tr_operand_at(vl, o + so.trk[db][0], o + so.trk[db][1]),
                                pf[bt], oacc[db]);
      }
  }

  // partials of the set's heads (an empty chunk: m = -inf, l = 0, o = 0)
  const float lt = pair_sum(l_run);
  if (l32 >= gs) return;
  const int64_t pi = ((int64_t)b * a.hq + head0 + l32) * a.splits + split;
  float *po = a.part_o + pi * D + hf * 4;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *(f32x4 *)(po + db * 32 + 8 * i) =
          f32x4{oacc[db][4 * i], oacc[db][4 * i + 1], oacc[db][4 * i + 2], oacc[db][4 * i + 3]};
  if (hf == 0) {
    a.part_ml[pi * 2] = m_run * sl2;
    a.part_ml[pi * 2 + 1] = lt;
  }
}

// Exact merge of the split partials: M = max m_s, L = sum l_s 2^(m_s - M),
// O = sum o_s 2^(m_s - M) / L. Scores were kept in log2 units. A dialogue
// whose position lies outside the cache (out of contract) gets NaN.
template <int D>
__global__ void __launch_bounds__(D)
decode_combine_kernel(DecodeArgs a) {
  const int bh = blockIdx.x;  // b * hq + h
  const int dd = threadIdx.x;
  {
    const int b = bh / a.hq, pb = a.pos[b];
    if (pb < 0 || pb >= a.cap) {
      ((bf16_t *)a.o)[(int64_t)bh * D + dd] = (bf16_t)NAN;
      if (a.lse && dd == 0) a.lse[(int64_t)(bh % a.hq) * a.batch + b] = NAN;
      return;
    }
  }
  const float *ml = a.part_ml + (int64_t)bh * a.splits * 2;
  float mx = -INFINITY;
  for (int s = 0; s < a.splits; ++s) mx = fmaxf(mx, ml[2 * s]);
  const float mref = mx == -INFINITY ? 0.f : mx;
  float lt = 0.f, ot = 0.f;
  const float *po = a.part_o + (int64_t)bh * a.splits * D + dd;
  for (int s = 0; s < a.splits; ++s) {
    const float f = fast_exp2(ml[2 * s] - mref);
    lt += ml[2 * s + 1] * f;
    ot += po[(int64_t)s * D] * f;
  }
  ((bf16_t *)a.o)[(int64_t)bh * D + dd] = (bf16_t)(ot / lt);
  if (a.lse && dd == 0) {
    const int b = bh / a.hq, h = bh % a.hq;
    a.lse[(int64_t)h * a.batch + b] = (mx + log2f(lt)) * kLn2;
  }
}

template <int D, int GS>
hipError_t launch_decode_t(const DecodeArgs &a, hipStream_t stream) {
  const dim3 grid(a.splits, a.hq / GS, a.batch);
  if (a.block_table)
    hipLaunchKernelGGL((decode_split_kernel<D, GS, true>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((decode_split_kernel<D, GS, false>), grid, dim3(256), 0, stream, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((decode_combine_kernel<D>), dim3(a.batch * a.hq), dim3(D),
                     0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_decode_mma(const DecodeArgs &a, hipStream_t stream) {
  const dim3 grid(a.splits, a.hq / a.set_heads, a.batch);
  if (a.block_table)
    hipLaunchKernelGGL((decode_mma_kernel<D, true>), grid, dim3(64), 0, stream, a);
  else
    hipLaunchKernelGGL((decode_mma_kernel<D, false>), grid, dim3(64), 0, stream, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((decode_combine_kernel<D>), dim3(a.batch * a.hq), dim3(D),
                     0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_decode_d(const DecodeArgs &a, hipStream_t stream) {
  if (a.mma) return launch_decode_mma<D>(a, stream);
  switch (a.set_heads) {
    case 1: return launch_decode_t<D, 1>(a, stream);
    case 2: return launch_decode_t<D, 2>(a, stream);
    case 3: return launch_decode_t<D, 3>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_cache_append(const void *k_src, const void *v_src,
                               void *k_cache, void *v_cache,
                               const int32_t *cu_new, const int32_t *cache_len,
                               int32_t batch, int32_t max_new, int32_t hkv,
                               int32_t d, int32_t cap, hipStream_t stream) {
  const int64_t chunks = (int64_t)max_new * hkv * (d / 8);
  if (chunks == 0 || batch == 0) return hipSuccess;
  hipLaunchKernelGGL(cache_append_kernel, dim3((unsigned)((chunks + 255) / 256), batch),
                     dim3(256), 0, stream, (const bf16_t *)k_src,
                     (const bf16_t *)v_src, (bf16_t *)k_cache, (bf16_t *)v_cache,
                     cu_new, cache_len, hkv, d, cap);
  return hipGetLastError();
}

hipError_t launch_cache_append_paged(const void *k_src, const void *v_src, void *k_pages,
                                     void *v_pages, const int32_t *cu_new,
                                     const int32_t *cache_len, const int32_t *block_table,
                                     int32_t max_pages, int32_t num_pages, int32_t page_size,
                                     int32_t batch, int32_t max_new, int32_t hkv, int32_t d,
                                     hipStream_t stream) {
  const int64_t chunks = (int64_t)max_new * hkv * (d / 8);
  if (chunks == 0 || batch == 0) return hipSuccess;
  hipLaunchKernelGGL(cache_append_paged_kernel, dim3((unsigned)((chunks + 255) / 256), batch),
                     dim3(256), 0, stream, (const bf16_t *)k_src, (const bf16_t *)v_src,
                     (bf16_t *)k_pages, (bf16_t *)v_pages, cu_new, cache_len, block_table,
                     max_pages, num_pages, page_size, hkv, d);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs &a, int d, hipStream_t stream) {
  if (d == 128) return launch_decode_d<128>(a, stream);
  if (d == 64) return launch_decode_d<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace ism
