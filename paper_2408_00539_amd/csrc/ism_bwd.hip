// Backward ISM attention on gfx950 (gradients of softmax(scale Q K^T + M) V
// under the Eq. 5 mask), deterministic: no atomics, every output element is
// written by exactly one workgroup.
//
//  1. prep: lim[j] (as in the forward) and seer[i], the first row that sees
//     key i: the start of i's segment if it is a query segment, else i itself
//     (every later row of the dialogue sees i as well, since lim is
//     non-decreasing inside a dialogue and lim(j) >= j).
//  2. dQ kernel, row-tile outer like the forward (lane <-> row): forms its
//     rows' delta[h][j] = sum_d dO[j,h,d] O[j,h,d] (equals sum_i P_ji dP_ji)
//     in its prologue, recomputes S^T and dP^T per 64-key tile and
//     accumulates dQ^T += K^T dS^T. It also stores -lse / scale and -delta
//     of its rows as sums of three bf16 values for the dK/dV kernel, which
//     runs next and adds them to every key of a row with one product per
//     row block.
//  3. dK/dV kernel, key-tile outer: a workgroup owns 128 keys of one KV head
//     (32 per wave pair, lane <-> key), walks the query heads of the group
//     and the 64-row tiles from seer[first key] to the dialogue end, and
//     accumulates dV^T += dO^T P and dK^T += Q^T dS with P = exp(S - LSE),
//     dS = P o (dP - delta), dP = dO V^T. Q and dO tiles are staged in LDS
//     row-major; the products over rows read them through transposing reads.
// All products are bf16 MFMA 32x32x16 with fp32 accumulation; gradients are
// written in fp32.
#include "ism_common.h"
#include "ism_kernels.h"

#ifndef ISM_DKV_WPE
#define ISM_DKV_WPE 2
#endif
#ifndef ISM_DQ_WPE
#define ISM_DQ_WPE 2
#endif

namespace ism {

namespace {

constexpr int kBR = 64;   // rows per tile in the dK/dV kernel
constexpr int kKW = 128;  // keys per dK/dV workgroup (32 per wave)
constexpr int kBK = 64;   // keys per tile in the dQ kernel

__global__ void __launch_bounds__(256)
bwd_prep_kernel(const int32_t *__restrict__ cu_segs,
                const uint8_t *__restrict__ seg_is_query, int32_t num_segs,
                int32_t total, int32_t *__restrict__ lim, int32_t *__restrict__ seer) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= total) return;
  int lo = 0, hi = num_segs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_segs[mid] <= j) lo = mid; else hi = mid - 1;
  }
  const bool q = seg_is_query[lo] != 0;
  lim[j] = q ? cu_segs[lo + 1] - 1 : j;
  seer[j] = q ? cu_segs[lo] : j;
}

// c as the exact sum of three bf16 values: c truncated to bf16, the
// remainder truncated, and the rest (at most 8 significant bits, so exact).
// Word 0 holds the first two (low half first), word 1 the third and zero.
__device__ __forceinline__ void split3_bf16(float c, uint32_t &w0, uint32_t &w1) {
  const uint32_t b0 = __float_as_uint(c) & 0xffff0000u;
  const float r1 = c - __uint_as_float(b0);
  const uint32_t b1 = __float_as_uint(r1) & 0xffff0000u;
  const float r2 = r1 - __uint_as_float(b1);
  w0 = (b0 >> 16) | b1;
  w1 = __float_as_uint(r2) >> 16;
}

// ---------------------------------------------------------------- dK / dV

// Ring of Q / dO tile stages: the tile a dS wave finishes (t - 1), the
// current tile t, and tile t + 1 in flight.
constexpr int kDkvStages = 3;

// Q and dO tiles of 64 rows (unpadded swizzled rows, see swz<D>()) plus the
// per-row -lse / scale and -delta as two planes of bf16 summands, all filled
// by direct global->LDS transfers; and P of the last two tiles for each
// wave pair as fp16 pairs in the element order of the dV product's bf16 B
// operand (lane-private, 4 x 16 bytes per lane, laid out so that
// consecutive lanes touch consecutive bytes). fp16 rather than bf16: P lies
// in [0, 1], where fp16 keeps 3 more mantissa bits, so the dS wave's
// dS = P o (dP - delta) carries one rounding of P 8x smaller than bf16's,
// and its fp16 x fp32 products are single v_fma_mix_f32 instructions.
template <int D>
struct DkvSmem {
  bf16_t q[kDkvStages][kBR * D];
  bf16_t dout[kDkvStages][kBR * D];
  __attribute__((aligned(16))) uint32_t lsex[kDkvStages][2][kBR];
  __attribute__((aligned(16))) uint32_t deltax[kDkvStages][2][kBR];
  __attribute__((aligned(16))) u32x4 p[kDkvStages][4][4 * 64];
};

// 64 consecutive 4-byte values base[min(r0 + l, last)] to lds[l] through one
// global_load_lds_dword.
__device__ __forceinline__ void dma_row_scalars(const void *base, int r0, int last, void *lds,
                                                int lane) {
  const int r = min(r0 + lane, last);
  dma_x1((const char *)base + (int64_t)r * 4, lds_addr(lds));
}

// N products in a fixed order: product n consumes operand n, read from LDS
// LA products ahead; mid() (vector work that later products depend on)
// runs before product K. Scheduling barriers pin the order.
template <int N, int K, int LA, class Rd, class Mm, class Mid>
__device__ __forceinline__ void product_stream(Rd &&rd, Mm &&mm, Mid &&mid) {
  bf16x8 op[N];
#pragma unroll
  for (int n = 0; n < LA && n < N; ++n) op[n] = rd(n);
#pragma unroll
  for (int n = 0; n < N; ++n) {
    if (n == K) {
      mid();
      __builtin_amdgcn_sched_barrier(0);
    }
    mm(n, op[n]);
    if (n + LA < N) op[n + LA] = rd(n + LA);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Eight waves in four pairs; pair p owns the 32 keys c0 + 32 p (lane <->
// key) and its two waves share one SIMD. Per 64-row tile t:
//  * the P wave (p) computes S = Q K^T and P = exp(S - LSE) (masked),
//    accumulates dV^T += dO^T P (P in bf16) and leaves P (fp16) in LDS;
//  * the dS wave (p + 4), one tile behind, forms dS = P o (dP - delta) with
//    its partner's P and accumulates dK^T += Q^T dS, then computes
//    dP = dO V^T of tile t for the next step.
// Each wave does 32 of the 64 products per tile with no product computed
// twice, and the exp / elementwise phase of one wave of a pair falls in the
// other's MFMA phase. Accumulator element r = 4i + j of row block rb holds
// row 32 rb + 8i + 4h + j (h = lane / 32), so bf16 operand kk = 2 rb + bt of
// the products over rows is simply elements 8 bt .. 8 bt + 7 of block rb.
// Visibility needs no per-row bounds: row r sees key i exactly when
// r >= seer[i] (seer is non-decreasing in i).
template <int D>
__global__ void __launch_bounds__(512)
__attribute__((amdgpu_waves_per_eu(ISM_DKV_WPE, ISM_DKV_WPE)))
dkv_kernel(BwdArgs a, int ktiles) {
  constexpr int NKS = D / 16, NDB = D / 32, RB = D * 2, LA = 3;
  constexpr int NRB = kBR / 32, NKK = kBR / 16;  // 32-row blocks, 16-row k steps
  __shared__ DkvSmem<D> sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pair = wave & 3;
  const bool pwave = wave < 4;
  const int hf = lane >> 5;

  // (dialogue, KV head) groups run on one XCD each; early key tiles (the
  // longest row ranges) first.
  int group, kt;
  if (!xcd_work_item((int)blockIdx.x, a.batch * a.hkv, ktiles, ISM_SCHED_CHUNK, false, group,
                     kt))
    return;
  const int b = group / a.hkv, kvh = group % a.hkv;
  const int s = a.cu_seqlens[b], e = a.cu_seqlens[b + 1];
  const int c0 = s + kt * kKW;
  if (c0 >= e) return;
  const int kw0 = c0 + 32 * pair;
  const bool wactive = kw0 < e;
  const int G = a.hq / a.hkv;
  const float sl2 = a.scale * kLog2e;

  // first rows that see the wave's first and last key, and this lane's key
  const int seer_first = wactive ? a.seer[kw0] : e;
  const int seer_last = (wactive && kw0 + 31 < e) ? a.seer[kw0 + 31] : e;
  const int key = kw0 + (lane & 31);
  const int seer_k = key < e ? a.seer[key] : 0x7fffffff;

  const int rstart = a.seer[c0];
  const int nrt = (e - rstart + kBR - 1) / kBR;
  const int iters = G * nrt;
  const int64_t rs = (int64_t)a.hq * D;
  DmaTile<D, kBR, 8> dma;
  dma.init(tid, rs);
  SwzBases<D> so;
  so.init(lane);
  // next tile to transfer: index, head, row tile; it goes to stage st, which
  // callers pass as a constant (nx % kDkvStages)
  int nx = 0, nx_h = kvh * G, nx_rt = 0;
  auto issue_next = [&](int st) __attribute__((always_inline)) {
    const int r0 = rstart + nx_rt * kBR;
    const int64_t base = ((int64_t)r0 * a.hq + nx_h) * D;
    dma.issue((const bf16_t *)a.q + base, rs, e - r0, sm.q[st]);
    dma.issue((const bf16_t *)a.dout + base, rs, e - r0, sm.dout[st]);
    if (wave >= 4) {  // one plane of the split -lse / scale or -delta per dS wave
      const int pl = wave & 1;
      const uint32_t *src = (wave < 6 ? a.lsex : a.deltax) + (int64_t)(2 * nx_h + pl) * a.total;
      dma_row_scalars(src, r0, e - 1, wave < 6 ? sm.lsex[st][pl] : sm.deltax[st][pl], lane);
    }
    ++nx;
    if (++nx_rt == nrt) { nx_rt = 0; ++nx_h; }
  };
  // B operands of this wave's products: K (P wave, for S) or V (dS wave,
  // for dP) of its 32 keys, lane <-> key, 8 head-dim values per k step;
  // the first tile's transfer overlaps their loads (iters >= 1: the first
  // key's own row sees it).
  bf16x8 bop[NKS];
  {
    const int kr = min(key, e - 1);
    const bf16_t *src =
        (const bf16_t *)(pwave ? a.k : a.v) + ((int64_t)kr * a.hkv + kvh) * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) bop[ks] = *(const bf16x8 *)(src + ks * 16);
    issue_next(0);
    wait_loads();  // also drains the first transfer
  }
  // B operand of the products that add a row's -lse / scale (P wave) or
  // -delta (dS wave) to every key of its row: 1 in the k slots 0-2 (lanes
  // 0-31 hold k = 0-7), 0 elsewhere; the matching A operand holds the row's
  // three bf16 summands in those slots (split3_bf16).
  const bf16x8 ones3 = __builtin_bit_cast(
      bf16x8, hf ? u32x4{0u, 0u, 0u, 0u} : u32x4{0x3f803f80u, 0x3f80u, 0u, 0u});
  const int l32 = lane & 31;
  f32x16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};
  f32x16 dp[NRB];         // dS wave: dP of the previous tile
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) dp[rb] = f32x16{};
  bool vis_prev = false;  // dS wave: the previous tile had visible keys

  // A operand of the product that adds row (32 rb + lane % 32)'s summands
  // (plane 0: two bf16, plane 1: the third and zero) to a 32-row block
  auto summands = [&](const uint32_t (*pl)[kBR], int rb) __attribute__((always_inline)) {
    const int r = 32 * rb + l32;
    return __builtin_bit_cast(bf16x8, u32x4{pl[0][r], pl[1][r], 0u, 0u});
  };

  // dS wave, one product stream per step: for the previous tile (stage sp,
  // also its P buffer) dS = P o dP' in 16-row slices, each slice's
  // dK^T[d][key] += Q^T[d][row] dS[row][key] products running beside the
  // elementwise work of the next slice; then (DP) dP'[row][key] = dO V^T -
  // delta of the current tile (stage st): one product per 32-row block
  // starts each accumulator at the row's -delta (it runs after the last dS
  // slice has consumed the previous dP), then the dO V^T products. The
  // empty asm statements keep each slot's vector work in its slot (IR
  // passes would otherwise sink it to its use).
  auto ds_dp = [&](int sp, int st, auto has_ds, auto has_dp) __attribute__((always_inline)) {
    constexpr bool DS = decltype(has_ds)::value, DP = decltype(has_dp)::value;
    constexpr int NK = DS ? NKK * NDB : 0, NX = DP ? NRB : 0;
    constexpr int N = NK + NX + (DP ? NKS * NRB : 0);
    const char *ql = (const char *)sm.q[sp];
    const char *dl = (const char *)sm.dout[st];
    const u32x4 *pp = sm.p[sp][pair];
    u32x4 pw[NKK];
    if constexpr (DS) {
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) pw[kk] = pp[kk * 64 + lane];
    }
    u32x4 fw[NKK];
    // dS elements 2u, 2u + 1 of slice kk (accumulator elements 8 bt + 2u ..)
    auto ds_pair = [&](int kk, int u) __attribute__((always_inline)) {
      const int rb = kk >> 1, e0 = 8 * (kk & 1) + 2 * u;
      f32x2 x;
      x[0] = mul_f16_lo(pw[kk][u], dp[rb][e0]);
      x[1] = mul_f16_hi(pw[kk][u], dp[rb][e0 + 1]);
      uint32_t w = cvt_bf16x2(x);
      asm volatile("" : "+v"(w));
      fw[kk][u] = w;
    };
    auto rd = [&](auto nc) __attribute__((always_inline)) -> bf16x8 {
      constexpr int n = decltype(nc)::value;
      if constexpr (n < NK) {  // n = kk * NDB + db
        constexpr int kk = n / NDB, db = n % NDB;
        return tr_operand_at(ql, 16 * kk * RB + so.tr(db, 0), 16 * kk * RB + so.tr(db, 1));
      } else if constexpr (n < NK + NX) {
        return summands(sm.deltax[st], n - NK);
      } else {  // n - NK - NX = ks * NRB + rb
        constexpr int j = n - NK - NX;
        return *(const bf16x8 *)(dl + (j % NRB) * 32 * RB + so.row(j / NRB));
      }
    };
    auto mm = [&](auto nc, bf16x8 x) __attribute__((always_inline)) {
      constexpr int n = decltype(nc)::value;
      if constexpr (n < NK) {
        constexpr int kk = n / NDB, db = n % NDB;
        acc[db] = mfma32x32x16(x, __builtin_bit_cast(bf16x8, fw[kk]), acc[db]);
      } else if constexpr (n < NK + NX) {
        dp[n - NK] = mfma32x32x16(x, ones3, f32x16{});
      } else {
        constexpr int j = n - NK - NX, ks = j / NRB, rb = j % NRB;
        dp[rb] = mfma32x32x16(x, bop[ks], dp[rb]);
      }
    };
    auto pre = [&](auto nc) __attribute__((always_inline)) {
      constexpr int n = decltype(nc)::value;
      if constexpr (n == 2) {
        if (nx < iters) issue_next((st + 1) % kDkvStages);
      }
      if constexpr (DS && n == 0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) ds_pair(0, u);
      }
    };
    auto work = [&](auto nc) __attribute__((always_inline)) {
      constexpr int n = decltype(nc)::value;
      // slice kk + 1 during the NDB products of slice kk
      if constexpr (DS && n < NK - NDB) {
        constexpr int kk = n / NDB + 1, w = n % NDB, per = 4 / NDB;
#pragma unroll
        for (int c = 0; c < per; ++c) ds_pair(kk, w * per + c);
      }
    };
    product_slots<N, LA>(rd, mm, pre, work);
  };

  // P wave on the current tile (stage st, rows r0.., nvalid valid), one
  // product stream: one product per row block that starts its accumulator
  // at the row's -lse / scale (so that P = exp2(acc * scale * log2 e)), S
  // of row block 0, S of row block 1 beside the exponentials of block 0,
  // dV^T += dO^T P for block 0 beside the exponentials of block 1, then dV
  // for block 1. P goes to LDS as fp16 (and into bf16 operand form) in
  // 16-row slices; rows are masked unless every row sees every key.
  auto p_dv = [&](int st, int r0, int nvalid, bool full) __attribute__((always_inline)) {
    const char *ql = (const char *)sm.q[st];
    const char *dl = (const char *)sm.dout[st];
    u32x4 *pp = sm.p[st][pair];
    f32x16 sacc[NRB];
    u32x4 fw[NKK];
    u32x4 hw;  // the slice being formed, as fp16 pairs for the dS wave
    constexpr int NX = NRB;        // summand products, then
    constexpr int NS = NKS * NRB;  // S products, row-block major
    constexpr int EPS = 16 / NKS;  // exponentials per slot
    auto rd = [&](auto nc) __attribute__((always_inline)) -> bf16x8 {
      constexpr int n = decltype(nc)::value - NX;
      if constexpr (n < 0) {
        return summands(sm.lsex[st], n + NX);
      } else if constexpr (n < NS) {
        return *(const bf16x8 *)(ql + (n / NKS) * 32 * RB + so.row(n % NKS));
      } else {  // n - NS = kk * NDB + db
        constexpr int kk = (n - NS) / NDB, db = (n - NS) % NDB;
        return tr_operand_at(dl, 16 * kk * RB + so.tr(db, 0), 16 * kk * RB + so.tr(db, 1));
      }
    };
    auto mm = [&](auto nc, bf16x8 x) __attribute__((always_inline)) {
      constexpr int n = decltype(nc)::value - NX;
      if constexpr (n < 0) {
        sacc[n + NX] = mfma32x32x16(x, ones3, f32x16{});
      } else if constexpr (n < NS) {
        constexpr int rb = n / NKS, ks = n % NKS;
        sacc[rb] = mfma32x32x16(x, bop[ks], sacc[rb]);
      } else {
        constexpr int kk = (n - NS) / NDB, db = (n - NS) % NDB;
        acc[db] = mfma32x32x16(x, __builtin_bit_cast(bf16x8, fw[kk]), acc[db]);
      }
    };
    auto mask_rb = [&](int rb) __attribute__((always_inline)) {
      // rows at or past nvalid repeat the last row (clamped transfers)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rr = 32 * rb + 8 * (r >> 2) + 4 * hf + (r & 3);
        if (rr >= nvalid || r0 + rr < seer_k) sacc[rb][r] = -INFINITY;
      }
    };
    auto pre = [&](auto nc) __attribute__((always_inline)) {
      constexpr int n = decltype(nc)::value;
      if constexpr (n == 2) {
        if (nx < iters) issue_next((st + 1) % kDkvStages);
      }
      if constexpr (n == NX + NKS || n == NX + 2 * NKS) {
        if (!full) mask_rb((n - NX) / NKS - 1);
      }
    };
    // exponentials of block rb in the NKS slots after its S is complete;
    // each finished 16-row slice goes to LDS and operand form
    auto work = [&](auto nc) __attribute__((always_inline)) {
      constexpr int n = decltype(nc)::value - NX;
      if constexpr (n >= NKS && n < 3 * NKS) {
        constexpr int rb = n / NKS - 1, w = n % NKS;
#pragma unroll
        for (int c = 0; c < EPS; c += 2) {
          const int e0 = w * EPS + c;  // accumulator elements e0, e0 + 1
          f32x2 x;
          x[0] = fast_exp2(sacc[rb][e0] * sl2);
          x[1] = fast_exp2(sacc[rb][e0 + 1] * sl2);
          uint32_t p2 = cvt_bf16x2(x), h2 = cvt_f16x2(x);
          asm volatile("" : "+v"(p2), "+v"(h2));
          fw[2 * rb + (e0 >> 3)][(e0 & 7) >> 1] = p2;
          hw[(e0 & 7) >> 1] = h2;
          if ((e0 & 7) == 6) pp[(2 * rb + (e0 >> 3)) * 64 + lane] = hw;
        }
      }
    };
    product_slots<NX + NS + NKK * NDB, LA>(rd, mm, pre, work);
  };

  using T_ = std::true_type;
  using F_ = std::false_type;
  // The dS waves' first step reads the last stage's Q and P buffer before
  // any tile has filled them (and multiplies them by zeros): clear them. The
  // first tile's transfer goes to stage 0 and is not touched.
  {
    constexpr int L = kDkvStages - 1;
    u32x4 *qz = (u32x4 *)sm.q[L];
    u32x4 *pz = (u32x4 *)sm.p[L];
#pragma unroll
    for (int i = tid; i < kBR * D / 8; i += 512) qz[i] = u32x4{};
#pragma unroll
    for (int i = tid; i < 4 * 4 * 64; i += 512) pz[i] = u32x4{};
  }
  // Start of step it (row tile rt): wait for its tile and synchronize; the
  // transfer of the next tile starts a few products into the step's product
  // stream (off the path to the first product). Returns the tile's first row.
  auto begin_step = [&](int it, int &rt) __attribute__((always_inline)) {
    const int r0 = rstart + rt * kBR;
    if (++rt == nrt) rt = 0;
    wait_vmem();
    // Tile it visible to all waves; every wave is done with tile it - 2 and
    // with the P buffer the P waves write next. A bare s_barrier: the fences
    // of __syncthreads() would also drain the transfers still in flight.
    lds_barrier();
    return r0;
  };
  // The two roles run separate loops (same barrier count) so that each
  // keeps its accumulators in place. Each loop is unrolled by the ring depth
  // so that every tile, P and scalar buffer is a compile-time LDS offset.
  static_assert(kDkvStages == 3, "the role loops below are unrolled by three");
  int rt = 0;
  if (pwave) {
    auto step = [&](int it, auto stc) __attribute__((always_inline)) {
      constexpr int st = decltype(stc)::value;  // it % kDkvStages
      const int r0 = begin_step(it, rt);
      const int nvalid = min(kBR, e - r0);
      if (r0 + nvalid - 1 < seer_first) {  // no row sees these keys: P = 0
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) sm.p[st][pair][kk * 64 + lane] = u32x4{};
        if (nx < iters) issue_next((st + 1) % kDkvStages);
        return;
      }
      p_dv(st, r0, nvalid, nvalid == kBR && r0 >= seer_last);
    };
    for (int it = 0; it < iters; it += kDkvStages) {
      step(it, std::integral_constant<int, 0>{});
      if (it + 1 < iters) step(it + 1, std::integral_constant<int, 1>{});
      if (it + 2 < iters) step(it + 2, std::integral_constant<int, 2>{});
    }
    lds_barrier();
  } else {
    // one stream per step: an invisible previous tile has P = 0 in LDS, so
    // its dK products add nothing; an invisible current tile's dP is never
    // used. The first step's "previous tile" is the zeroed last stage.
    auto step = [&](int it, auto stc) __attribute__((always_inline)) {
      constexpr int st = decltype(stc)::value;  // it % kDkvStages
      const int r0 = begin_step(it, rt);
      const int nvalid = min(kBR, e - r0);
      ds_dp((st + kDkvStages - 1) % kDkvStages, st, T_{}, T_{});
      vis_prev = r0 + nvalid - 1 >= seer_first;
    };
    for (int it = 0; it < iters; it += kDkvStages) {
      step(it, std::integral_constant<int, 0>{});
      if (it + 1 < iters) step(it + 1, std::integral_constant<int, 1>{});
      if (it + 2 < iters) step(it + 2, std::integral_constant<int, 2>{});
    }
    // finish the last tile once its P is in LDS
    lds_barrier();
    if (vis_prev) ds_dp((iters - 1) % kDkvStages, 0, T_{}, F_{});
  }

  if (!wactive || key >= e) return;
  float *out = (pwave ? a.dv : a.dk) + ((int64_t)key * a.hkv + kvh) * D + hf * 4;
  const float mul = pwave ? 1.f : a.scale;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 x;
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = acc[db][4 * i + j] * mul;
      *(f32x4 *)(out + db * 32 + 8 * i) = x;
    }
}

// ---------------------------------------------------------------- dQ

// K and V tiles of 64 keys, unpadded swizzled rows, double-buffered, filled
// by direct global->LDS transfers; K^T is read through transposing reads.
template <int D>
struct DqSmem {
  bf16_t k[2][kBK * D];
  bf16_t v[2][kBK * D];
};

// One wave owns 32 rows of one head (lane <-> row) and walks the 64-key
// tiles its rows see. Per tile, in product order: S^T = K Q^T and dP^T =
// V dO^T for keys 0-31, then for keys 32-63, then dQ^T += K^T dS^T for both
// halves; the exponentials of each S^T half run beside the next dP^T
// products and dS^T = P^T o (dP^T - delta) beside the products after that.
template <int D, int NWV>
__global__ void __launch_bounds__(NWV * 64)
__attribute__((amdgpu_waves_per_eu(ISM_DQ_WPE, ISM_DQ_WPE)))
dq_kernel(BwdArgs a, int hpw, int tiles) {
  constexpr int NKS = D / 16, NDB = D / 32, RB = D * 2, LA = 3;
  __shared__ DqSmem<D> sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hf = lane >> 5;

  const int hsets = a.hq / hpw;
  int group, tile;
  if (!xcd_work_item((int)blockIdx.x, a.batch * hsets, tiles, ISM_SCHED_CHUNK, true, group,
                     tile))
    return;
  const int b = group / hsets;
  const int head0 = (group % hsets) * hpw;
  const int wg_rows = (NWV / hpw) * 32;
  const int s = a.cu_seqlens[b], e = a.cu_seqlens[b + 1];
  const int q0 = s + tile * wg_rows;
  if (q0 >= e) return;
  const int head = head0 + wave % hpw;
  const int kvh = head0 / (a.hq / a.hkv);
  const int wq0 = q0 + (wave / hpw) * 32;
  const bool active = wq0 < e;
  const int key_hi = a.lim[min(q0 + wg_rows, e) - 1];
  const int wave_lo = a.lim[min(wq0, e - 1)];
  const int wave_hi = active ? a.lim[min(wq0 + 32, e) - 1] : s - 1;
  const float sl2 = a.scale * kLog2e;

  // The first K/V tile needs only the dialogue's key range in memory (keys
  // past the workgroup's bound are masked like any other invisible key), so
  // its transfer starts before the bounds, Q and dO arrive.
  const bf16_t *kbase = (const bf16_t *)a.k + (int64_t)kvh * D;
  const bf16_t *vbase = (const bf16_t *)a.v + (int64_t)kvh * D;
  const int64_t rs = (int64_t)a.hkv * D;
  DmaTile<D, kBK, NWV> dma;
  dma.init(tid, rs);
  const bf16_t *kt = kbase + (int64_t)s * rs;
  const bf16_t *vt = vbase + (int64_t)s * rs;
  dma.issue(kt, rs, e - s, sm.k[0]);
  dma.issue(vt, rs, e - s, sm.v[0]);

  const int rc = min(wq0 + l32, e - 1);
  const int lim_r = a.lim[rc];
  const float lse_r = a.lse[(int64_t)head * a.total + rc];
  bf16x8 qf[NKS], df[NKS];
  float ndlt;  // -delta of the lane's row
  {
    const int64_t ro = ((int64_t)rc * a.hq + head) * D + hf * 8;
    const bf16_t *qp = (const bf16_t *)a.q + ro;
    const bf16_t *dp = (const bf16_t *)a.dout + ro;
    const bf16_t *opp = (const bf16_t *)a.o + ro;
    bf16x8 of[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[ks] = *(const bf16x8 *)(qp + ks * 16);
      df[ks] = *(const bf16x8 *)(dp + ks * 16);
      of[ks] = *(const bf16x8 *)(opp + ks * 16);
    }
    wait_loads();  // also drains the transfers above
    // delta = rowsum(dO o O): this lane's half of the head dims, then the pair
    float acc = 0.f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const u32x4 x = __builtin_bit_cast(u32x4, of[ks]), y = __builtin_bit_cast(u32x4, df[ks]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc = fmaf(bf16_lo(x[i]), bf16_lo(y[i]), acc);
        acc = fmaf(bf16_hi(x[i]), bf16_hi(y[i]), acc);
      }
    }
    ndlt = -pair_sum(acc);
  }
  const float lse2 = lse_r * kLog2e;
  // -delta of the row as bf16 summands: for the dK/dV kernel and, as the B
  // operand of one product per key half against a ones A operand (1 in k
  // slots 0-2 of lanes 0-31), to start the dP^T accumulators at -delta
  uint32_t dw0, dw1;
  split3_bf16(ndlt, dw0, dw1);
  const bf16x8 dsum = __builtin_bit_cast(bf16x8, u32x4{dw0, dw1, 0u, 0u});
  const bf16x8 ones3 = __builtin_bit_cast(
      bf16x8, hf ? u32x4{0u, 0u, 0u, 0u} : u32x4{0x3f803f80u, 0x3f80u, 0u, 0u});
  // -lse / scale and -delta of the row as bf16 summands for the dK/dV kernel
  if (active && hf == 0 && wq0 + l32 < e) {
    const int64_t i0 = 2 * (int64_t)head * a.total + wq0 + l32;
    uint32_t w0, w1;
    split3_bf16(-lse_r * a.inv_scale, w0, w1);
    a.lsex[i0] = w0;
    a.lsex[i0 + a.total] = w1;
    a.deltax[i0] = dw0;
    a.deltax[i0 + a.total] = dw1;
  }
  __syncthreads();
  f32x16 dq[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dq[db] = f32x16{};

  const int ntiles = (key_hi - s) / kBK + 1;
  const int nw = active ? (wave_hi - s) / kBK + 1 : 0;  // this wave's tiles
  SwzBases<D> so;
  so.init(lane);
  const int64_t tile_elems = (int64_t)kBK * rs;

  // keys past the row's bound get P = 0 (score -inf)
  auto mask = [&](f32x16 &x, int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (k0 + (r >> 2) * 8 + hf * 4 + (r & 3) > lim_r) x[r] = -INFINITY;
  };

  // one key tile; the loops below run it unrolled by two so that the buffer
  // (t & 1) and with it every LDS address is a compile-time offset. MODE 0:
  // the next tile is full and this wave's transfers of it go out one every
  // second product from the first (~0.5 % faster on the backward than all at
  // the step start); MODE 1: all at the step start (a partial next tile, or
  // none).
  auto step = [&](int t, auto bufc, auto modec) __attribute__((always_inline)) {
    constexpr int buf = decltype(bufc)::value;
    constexpr int MODE = decltype(modec)::value;
    constexpr int NI = decltype(dma)::NI;
    const int c0 = s + t * kBK;
    if (t + 1 < ntiles) {
      kt += tile_elems;
      vt += tile_elems;
      if (MODE == 1 || t >= nw) {
        dma.issue(kt, rs, key_hi - (c0 + kBK) + 1, sm.k[buf ^ 1]);
        dma.issue(vt, rs, key_hi - (c0 + kBK) + 1, sm.v[buf ^ 1]);
      }
    }
    if (t < nw) {
      const bool full = c0 + kBK - 1 <= wave_lo;
      const char *kl = (const char *)sm.k[buf];
      const char *vl = (const char *)sm.v[buf];
      // S^T / P^T and dP^T for the two 32-key halves; dS^T operands
      f32x16 sc[2], pc[2];
      u32x4 ds[2][2];
      constexpr int NH = 2 * NKS;  // products per half (S^T and dP^T)
      constexpr int NX = 2;        // the two -delta products come first
      // products after those (index n - NX): [0, NH) S^T and dP^T half 0
      // (alternating), [NH, 2 NH) half 1, [2 NH, 2 NH + 4 NDB) dQ^T (kb, db, bt)
      auto rd = [&](auto nc) __attribute__((always_inline)) -> bf16x8 {
        constexpr int n = decltype(nc)::value - NX;
        if constexpr (n < 0) {
          return ones3;
        } else if constexpr (n < 2 * NH) {
          constexpr int kb = n / NH, m = n % NH, ks = m >> 1;
          return *(const bf16x8 *)(((m & 1) ? vl : kl) + kb * 32 * RB + so.row(ks));
        } else {
          constexpr int j = n - 2 * NH, kb = j / (2 * NDB), db = (j % (2 * NDB)) >> 1,
                        bt = j & 1;
          constexpr uint32_t o = (kb * 32 + 16 * bt) * RB;
          return tr_operand_at(kl, o + so.tr(db, 0), o + so.tr(db, 1));
        }
      };
      auto mm = [&](auto nc, bf16x8 x) __attribute__((always_inline)) {
        constexpr int n = decltype(nc)::value - NX;
        if constexpr (n < 0) {
          pc[n + NX] = mfma32x32x16(x, dsum, f32x16{});
        } else if constexpr (n < 2 * NH) {
          constexpr int kb = n / NH, m = n % NH, ks = m >> 1;
          if constexpr (m & 1) pc[kb] = mfma32x32x16(x, df[ks], pc[kb]);
          else sc[kb] = mfma32x32x16(x, qf[ks], ks == 0 ? f32x16{} : sc[kb]);
        } else {
          constexpr int j = n - 2 * NH, kb = j / (2 * NDB), db = (j % (2 * NDB)) >> 1,
                        bt = j & 1;
          dq[db] = mfma32x32x16(x, __builtin_bit_cast(bf16x8, ds[kb][bt]), dq[db]);
        }
      };
      // the next tile's transfers (MODE 0); mask a finished S^T half just
      // before its exponentials start
      auto pre = [&](auto nc) __attribute__((always_inline)) {
        constexpr int nr = decltype(nc)::value;
        if constexpr (MODE == 0 && nr % 2 == 0 && nr / 2 < 2 * NI) {
          if constexpr (nr / 2 < NI) dma.issue_one(kt, nr / 2, sm.k[buf ^ 1]);
          else dma.issue_one(vt, nr / 2 - NI, sm.v[buf ^ 1]);
        }
        constexpr int n = nr - NX;
        if constexpr (n == NH) { if (!full) mask(sc[0], c0); }
        if constexpr (n == 2 * NH) { if (!full) mask(sc[1], c0 + 32); }
      };
      // P^T and dS^T of half 0 in the slots of half 1's products (first the
      // exponentials, then dS^T), of half 1 in the slots of half 0's dQ^T
      // products, so that both are complete before the dQ^T products that
      // read them
      // (the empty asm keeps each result in its slot: IR passes would
      // otherwise sink the work past the mask branch to its uses)
      auto exp1 = [&](int kb, int r) __attribute__((always_inline)) {
        float p = fast_exp2(fmaf(sc[kb][r], sl2, -lse2));
        asm volatile("" : "+v"(p));
        sc[kb][r] = p;
      };
      auto ds2 = [&](int kb, int r) __attribute__((always_inline)) {  // elements r, r + 1 (r even)
        f32x2 x;
        x[0] = sc[kb][r] * pc[kb][r];
        x[1] = sc[kb][r + 1] * pc[kb][r + 1];
        uint32_t w = cvt_bf16x2(x);
        asm volatile("" : "+v"(w));
        ds[kb][r >> 3][(r & 7) >> 1] = w;
      };
      auto work = [&](auto nc) __attribute__((always_inline)) {
        constexpr int n = decltype(nc)::value - NX;
        if constexpr (n >= NH && n < 2 * NH) {
          constexpr int E = 32 / NH, w = n - NH;  // element-steps per slot
          if constexpr (w < NH / 2) {
#pragma unroll
            for (int c = 0; c < E; ++c) exp1(0, w * E + c);
          } else {
#pragma unroll
            for (int c = 0; c < E; c += 2) ds2(0, (w - NH / 2) * E + c);
          }
        } else if constexpr (n >= 2 * NH && n < 2 * NH + 2 * NDB) {
          constexpr int E = 16 / NDB, w = n - 2 * NH;
          if constexpr (w < NDB) {
#pragma unroll
            for (int c = 0; c < E; ++c) exp1(1, w * E + c);
          } else {
#pragma unroll
            for (int c = 0; c < E; c += 2) ds2(1, (w - NDB) * E + c);
          }
        }
      };
      static_assert(2 * (2 * NI - 1) < NX + 2 * NH + 4 * NDB,
                    "every transfer of a full next tile falls inside the stream");
      product_slots<NX + 2 * NH + 4 * NDB, LA>(rd, mm, pre, work);
    }
    wait_vmem();
    __syncthreads();
  };
  // steps whose next tile is full, an even count of them; then the rest
  using Z_ = std::integral_constant<int, 0>;
  using O_ = std::integral_constant<int, 1>;
  const int nfull = max((key_hi - s + 1) / kBK - 1, 0) & ~1;
  int t = 0;
  for (; t < nfull; t += 2) {
    step(t, Z_{}, Z_{});
    step(t + 1, O_{}, Z_{});
  }
  for (; t < ntiles; t += 2) {
    step(t, Z_{}, O_{});
    if (t + 1 < ntiles) step(t + 1, O_{}, O_{});
  }

  const int row = wq0 + l32;
  if (!active || row >= e) return;
  float *out = a.dq + ((int64_t)row * a.hq + head) * D + hf * 4;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 x;
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = dq[db][4 * i + j] * a.scale;
      *(f32x4 *)(out + db * 32 + 8 * i) = x;
    }
}

int gcd_i(int x, int y) {
  while (y) { const int t = x % y; x = y; y = t; }
  return x;
}

// dQ workgroups of NWV waves. Eight waves (one workgroup per CU) share each
// staged K/V tile among twice the rows (or the heads of a KV group) of four
// waves: half the transfers per product, measured 1.5-2 % faster on the
// backward than two 4-wave workgroups per CU.
template <int D, int NWV>
hipError_t launch_dq(const BwdArgs &a, hipStream_t stream) {
  const int hpw = gcd_i(a.hq / a.hkv, NWV);
  const int wg_rows = (NWV / hpw) * 32;
  const int tiles = (a.max_seqlen + wg_rows - 1) / wg_rows;
  hipLaunchKernelGGL((dq_kernel<D, NWV>),
                     dim3((unsigned)xcd_grid((int64_t)a.batch * (a.hq / hpw), tiles)),
                     dim3(NWV * 64), 0, stream, a, hpw, tiles);
  return hipGetLastError();
}

// dQ first: it also writes the per-row summands the dK/dV kernel reads.
template <int D>
hipError_t launch_bwd_t(const BwdArgs &a, hipStream_t stream) {
  hipError_t err = launch_dq<D, 8>(a, stream);
  if (err != hipSuccess) return err;
  const int ktiles = (a.max_seqlen + kKW - 1) / kKW;
  hipLaunchKernelGGL((dkv_kernel<D>), dim3((unsigned)xcd_grid((int64_t)a.batch * a.hkv, ktiles)),
                     dim3(512), 0, stream, a, ktiles);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_prep(const int32_t *cu_segs, const uint8_t *seg_is_query,
                           int32_t num_segs, int32_t total, int32_t *lim, int32_t *seer,
                           hipStream_t stream) {
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_prep_kernel, dim3((total + 255) / 256), dim3(256), 0, stream,
                     cu_segs, seg_is_query, num_segs, total, lim, seer);
  return hipGetLastError();
}

hipError_t launch_bwd(const BwdArgs &a, int d, hipStream_t stream) {
  if (d == 128) return launch_bwd_t<128>(a, stream);
  if (d == 64) return launch_bwd_t<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace ism
