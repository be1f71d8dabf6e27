// Backward ISM attention on gfx950 (gradients of softmax(scale Q K^T + M) V
// under the Eq. 5 mask), deterministic: no atomics, every output element is
// written by exactly one workgroup.
//
//  1. prep: lim[j] (as in the forward) and seer[i], the first row that sees
//     key i: the start of i's segment if it is a query segment, else i itself
//     (every later row of the dialogue sees i as well, since lim is
//     non-decreasing inside a dialogue and lim(j) >= j).
//  2. delta[h][j] = sum_d dO[j,h,d] O[j,h,d]  (equals sum_i P_ji dP_ji).
//  3. dK/dV kernel, key-tile outer: a workgroup owns 128 keys of one KV head
//     (32 per wave, lane <-> key), walks the query heads of the group and the
//     32-row tiles from seer[first key] to the dialogue end, and accumulates
//     dV^T += dO^T P and dK^T += Q^T dS with P = exp(S - LSE),
//     dS = P o (dP - delta), dP = dO V^T. Q and dO tiles are staged in LDS
//     both row-major (for S and dP) and transposed (for the two products
//     over rows).
//  4. dQ kernel, row-tile outer like the forward (lane <-> row): recomputes
//     S^T and dP^T per 64-key tile and accumulates dQ^T += K^T dS^T.
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

constexpr int kBR = 32;   // rows per tile in the dK/dV kernel
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

// delta over (row, head) pairs: D/8 lanes per pair, 16-byte loads; also the
// LSE in log2 units (lse * log2 e) that the dK/dV kernel stages per tile.
template <int D>
__global__ void __launch_bounds__(256)
delta_kernel(const bf16_t *__restrict__ o, const bf16_t *__restrict__ dout,
             const float *__restrict__ lse, float *__restrict__ delta,
             float *__restrict__ lse2, int32_t total, int32_t hq) {
  constexpr int LPR = D / 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t pairs = (int64_t)total * hq;
  const int64_t rh = min(gid / LPR, pairs - 1);
  const int c = (int)(gid % LPR);
  const u32x4 x = *(const u32x4 *)(o + rh * D + c * 8);
  const u32x4 y = *(const u32x4 *)(dout + rh * D + c * 8);
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc = fmaf(bf16_lo(x[i]), bf16_lo(y[i]), acc);
    acc = fmaf(bf16_hi(x[i]), bf16_hi(y[i]), acc);
  }
#pragma unroll
  for (int s = 1; s < LPR; s <<= 1) acc += __shfl_xor(acc, s);
  if (c == 0 && gid / LPR < pairs) {
    const int64_t row = rh / hq, h = rh % hq;
    delta[h * total + row] = acc;
    lse2[h * total + row] = lse[h * total + row] * kLog2e;
  }
}

// ---------------------------------------------------------------- dK / dV

constexpr int kDkvStages = 3;  // tiles in flight: compute one, two loading

// Q and dO tiles of 32 rows (unpadded swizzled rows, see swz()) plus the
// per-row LSE (log2 units), delta and lim, all filled by direct global->LDS
// transfers, in a ring of kDkvStages buffers. Transposed operands are read
// with ds_read_b64_tr_b16.
template <int D>
struct DkvSmem {
  bf16_t q[kDkvStages][kBR * D];
  bf16_t dout[kDkvStages][kBR * D];
  __attribute__((aligned(16))) float lse2[kDkvStages][kBR];
  __attribute__((aligned(16))) float delta[kDkvStages][kBR];
  __attribute__((aligned(16))) int lim[kDkvStages][kBR];
};

// 32 consecutive 4-byte values base[min(r0 + l, last)], l < 32, to lds[l]
// through one global_load_lds_dword (lanes 32..63 idle).
__device__ __forceinline__ void dma_row_scalars(const void *base, int r0, int last, void *lds,
                                                int lane) {
  const uint32_t lb = lds_addr(lds);
  if (lane < 32) {
    const int r = min(r0 + lane, last);
    dma_x1((const char *)base + (int64_t)r * 4, lb);
  }
}

// s_waitcnt vmcnt(n) with expcnt / lgkmcnt left unconstrained.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void wait_vmcnt_dyn(int n) {
  switch (n) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<1>(); break;
    case 2: wait_vmcnt<2>(); break;
    default: wait_vmcnt<3>(); break;
  }
}

// 8 waves: waves 0-3 accumulate dV and waves 4-7 dK for the same four
// 32-key blocks, so that each wave holds one accumulator set (64 registers)
// and two waves fit on every SIMD. Both roles recompute S (one extra GEMM in
// five) in exchange for overlapping one role's exp/elementwise work with the
// other's MFMAs.
template <int D>
__global__ void __launch_bounds__(512)
__attribute__((amdgpu_waves_per_eu(ISM_DKV_WPE, ISM_DKV_WPE)))
dkv_kernel(BwdArgs a, int ktiles) {
  constexpr int NKS = D / 16, NDB = D / 32, RB = D * 2;
  __shared__ DkvSmem<D> sm;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kblk = wave & 3, role = wave >> 2;  // role 0: dV, role 1: dK
  const int l32 = lane & 31, hf = lane >> 5;

  // (dialogue, KV head) groups run on one XCD each; early key tiles (the
  // longest row ranges) first.
  const int total = a.batch * a.hkv * ktiles;
  const int per = (total + 7) / 8;
  const int item = (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);
  if (item >= total) return;
  const int group = item / ktiles, kt = item % ktiles;
  const int b = group / a.hkv, kvh = group % a.hkv;
  const int s = a.cu_seqlens[b], e = a.cu_seqlens[b + 1];
  const int c0 = s + kt * kKW;
  if (c0 >= e) return;
  const int kw0 = c0 + 32 * kblk;
  const bool wactive = kw0 < e;
  const int G = a.hq / a.hkv;
  const float sl2 = a.scale * kLog2e;

  // this wave's 32 keys as B operands (lane <-> key, 8 head-dim values)
  bf16x8 kf[NKS], vf[NKS];
  {
    const int key = min(kw0 + l32, e - 1);
    const bf16_t *kp = (const bf16_t *)a.k + ((int64_t)key * a.hkv + kvh) * D + hf * 8;
    const bf16_t *vp = (const bf16_t *)a.v + ((int64_t)key * a.hkv + kvh) * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      kf[ks] = *(const bf16x8 *)(kp + ks * 16);
      vf[ks] = role ? *(const bf16x8 *)(vp + ks * 16) : bf16x8{};
    }
    wait_loads();
  }
  f32x16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};

  const int rstart = a.seer[c0];
  const int nrt = (e - rstart + kBR - 1) / kBR;
  const int iters = G * nrt;
  const int64_t rs = (int64_t)a.hq * D;
  DmaTile<D, kBR, 8> dma;
  dma.init(tid, rs);
  SwzOffsets so;
  so.init(lane, RB);
  // transfers this wave issues per tile: Q and dO blocks, plus one row-scalar
  // array for waves 5, 6, 7
  const int my_ops = 2 * (wave < DmaTile<D, kBR, 8>::T ? 1 : 0) + (wave >= 5 ? 1 : 0);
  // Sources of tile t: Q and dO rows, and the per-row scalars of its head.
  struct TileSrc {
    const bf16_t *q, *d;
    const float *l, *dl;
    int r0;
  };
  auto tile_src = [&](int t) {
    const int h = kvh * G + t / nrt, r0 = rstart + (t % nrt) * kBR;
    const int64_t base = ((int64_t)r0 * a.hq + h) * D;
    return TileSrc{(const bf16_t *)a.q + base, (const bf16_t *)a.dout + base,
                   a.lse2 + (int64_t)h * a.total, a.delta + (int64_t)h * a.total, r0};
  };
  // Transfers of one tile into one stage of the ring. All pointers are
  // __restrict__ so that, once inlined, the transfers carry alias scopes.
  auto issue = [&](const bf16_t *__restrict__ gq, const bf16_t *__restrict__ gd,
                   const float *__restrict__ gl, const float *__restrict__ gdl,
                   const int *__restrict__ glim, int r0, bf16_t *__restrict__ q_n,
                   bf16_t *__restrict__ d_n, float *__restrict__ l_n,
                   float *__restrict__ dl_n, int *__restrict__ lim_n) {
    dma.issue(gq, rs, e - r0, q_n);
    dma.issue(gd, rs, e - r0, d_n);
    if (wave == 5) dma_row_scalars(gl, r0, e - 1, l_n, lane);
    if (wave == 6) dma_row_scalars(gdl, r0, e - 1, dl_n, lane);
    if (wave == 7) dma_row_scalars(glim, r0, e - 1, lim_n, lane);
  };
#pragma unroll
  for (int t = 0; t < kDkvStages - 1; ++t)
    if (t < iters) {
      const TileSrc ts = tile_src(t);
      issue(ts.q, ts.d, ts.l, ts.dl, a.lim, ts.r0, sm.q[t], sm.dout[t], sm.lse2[t],
            sm.delta[t], sm.lim[t]);
    }

  // One step: start the transfers of a later tile into the free stage (the
  // *_n buffers, sources g*) and compute on the current stage (*_c). The
  // __restrict__ qualifiers tell the compiler the stages never overlap, so
  // it does not make the current stage's LDS reads wait for the new
  // transfers.
  auto step = [&](const bf16_t *__restrict__ q_c, const bf16_t *__restrict__ d_c,
                  const float *__restrict__ l_c, const float *__restrict__ dl_c,
                  const int *__restrict__ lim_c, bf16_t *__restrict__ q_n,
                  bf16_t *__restrict__ d_n, float *__restrict__ l_n, float *__restrict__ dl_n,
                  int *__restrict__ lim_n, const bf16_t *__restrict__ gq,
                  const bf16_t *__restrict__ gd, const float *__restrict__ gl,
                  const float *__restrict__ gdl, const int *__restrict__ glim, int rn,
                  bool more, int r0) {
    if (more) issue(gq, gd, gl, gdl, glim, rn, q_n, d_n, l_n, dl_n, lim_n);
    const int nvalid = min(kBR, e - r0);
    const int lim_last = lim_c[nvalid - 1];
    if (!wactive || lim_last < kw0) return;
    // rows at or past nvalid repeat the last row (clamped transfers) and
    // are masked in the partial path
    const bool full = nvalid == kBR && lim_c[0] >= kw0 + 31;
    const char *ql = (const char *)q_c;
    const char *dl = (const char *)d_c;
    const int key = kw0 + l32;
    // S[row][key] (lane <-> key, rows 8i + 4hf + j); role 1 also dP
    f32x16 sacc, pacc;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const uint32_t o = 128 * (ks >> 2) + so.rowk[ks & 3];
      sacc = mfma32x32x16(*(const bf16x8 *)(ql + o), kf[ks], ks == 0 ? f32x16{} : sacc);
    }
    if (role) {
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const uint32_t o = 128 * (ks >> 2) + so.rowk[ks & 3];
        pacc = mfma32x32x16(*(const bf16x8 *)(dl + o), vf[ks], ks == 0 ? f32x16{} : pacc);
      }
    }
    // P = exp(S - LSE) (masked); role 1: dS = P (dP - delta)
    bf16x8 fr[2] = {};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 l2 = *(const f32x4 *)&l_c[8 * i + 4 * hf];
      int lm[4] = {0, 0, 0, 0};
      if (!full) {
        const u32x4 li = *(const u32x4 *)&lim_c[8 * i + 4 * hf];
#pragma unroll
        for (int j = 0; j < 4; ++j) lm[j] = (8 * i + 4 * hf + j < nvalid) ? (int)li[j] : -1;
      }
      f32x2 w[2];
      if (role) {
        const f32x4 dlt = *(const f32x4 *)&dl_c[8 * i + 4 * hf];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float p = fast_exp2(fmaf(sacc[4 * i + j], sl2, -l2[j]));
          if (!full && key > lm[j]) p = 0.f;
          w[j >> 1][j & 1] = p * (pacc[4 * i + j] - dlt[j]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float p = fast_exp2(fmaf(sacc[4 * i + j], sl2, -l2[j]));
          if (!full && key > lm[j]) p = 0.f;
          w[j >> 1][j & 1] = p;
        }
      }
      // rows 8i..8i+3 (+4hf) are slots 4*(i&1).. of operand i>>1
      const int bt = i >> 1, sl = (i & 1) * 2;
      u32x4 x = __builtin_bit_cast(u32x4, fr[bt]);
      x[sl] = cvt_bf16x2(w[0]);
      x[sl + 1] = cvt_bf16x2(w[1]);
      fr[bt] = __builtin_bit_cast(bf16x8, x);
    }
    // role 0: dV^T[d][key] += dO^T P; role 1: dK^T[d][key] += Q^T dS
    const char *src = role ? ql : dl;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const uint32_t cb = ((db & 1) ? so.tro : so.tre) + 64 * db;
#pragma unroll
      for (int bt = 0; bt < 2; ++bt) {
        const uint32_t o = cb + 16 * bt * RB;
        acc[db] = mfma32x32x16(tr_operand_at(src, o, o + 8 * RB), fr[bt], acc[db]);
      }
    }
  };

  for (int it = 0; it < iters; ++it) {
    const int buf = it % kDkvStages, nb = (it + kDkvStages - 1) % kDkvStages;
    const int r0 = rstart + (it % nrt) * kBR;
    // tile it has landed once at most the next tile's transfers are pending
    if (it + 1 < iters) wait_vmcnt_dyn(my_ops); else wait_vmcnt<0>();
    // Tile it visible to all waves, and every wave is done reading tile
    // it - 1 (its reads were consumed by MFMAs). A bare s_barrier: the fences
    // of __syncthreads() would also drain the transfers still in flight.
    lds_barrier();
    const int tn = it + kDkvStages - 1;
    const TileSrc ts = tile_src(tn < iters ? tn : it);
    step(sm.q[buf], sm.dout[buf], sm.lse2[buf], sm.delta[buf], sm.lim[buf], sm.q[nb],
         sm.dout[nb], sm.lse2[nb], sm.delta[nb], sm.lim[nb], ts.q, ts.d, ts.l, ts.dl, a.lim,
         ts.r0, tn < iters, r0);
  }

  const int key = kw0 + l32;
  if (!wactive || key >= e) return;
  float *out = (role ? a.dk : a.dv) + ((int64_t)key * a.hkv + kvh) * D + hf * 4;
  const float mul = role ? a.scale : 1.f;
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

template <int D>
__global__ void __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(ISM_DQ_WPE, ISM_DQ_WPE)))
dq_kernel(BwdArgs a, int hpw, int tiles) {
  constexpr int NKS = D / 16, NDB = D / 32, RB = D * 2;
  __shared__ DqSmem<D> sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;

  const int hsets = a.hq / hpw;
  const int total = a.batch * hsets * tiles;
  const int per = (total + 7) / 8;
  const int item = (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);
  if (item >= total) return;
  const int group = item / tiles;
  const int tile = tiles - 1 - item % tiles;
  const int b = group / hsets;
  const int head0 = (group % hsets) * hpw;
  const int wg_rows = (4 / hpw) * 32;
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

  const int rc = min(wq0 + l32, e - 1);
  const int lim_r = a.lim[rc];
  const float lse2 = a.lse2[(int64_t)head * a.total + rc];
  const float dlt = a.delta[(int64_t)head * a.total + rc];
  bf16x8 qf[NKS], df[NKS];
  {
    const bf16_t *qp = (const bf16_t *)a.q + ((int64_t)rc * a.hq + head) * D + hf * 8;
    const bf16_t *dp = (const bf16_t *)a.dout + ((int64_t)rc * a.hq + head) * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[ks] = *(const bf16x8 *)(qp + ks * 16);
      df[ks] = *(const bf16x8 *)(dp + ks * 16);
    }
    wait_loads();
  }
  f32x16 dq[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dq[db] = f32x16{};

  const bf16_t *kbase = (const bf16_t *)a.k + (int64_t)kvh * D;
  const bf16_t *vbase = (const bf16_t *)a.v + (int64_t)kvh * D;
  const int64_t rs = (int64_t)a.hkv * D;
  const int ntiles = (key_hi - s) / kBK + 1;
  DmaTile<D, kBK> dma;
  dma.init(tid, rs);
  SwzOffsets so;
  so.init(lane, RB);
  const int64_t tile_elems = (int64_t)kBK * rs;
  const bf16_t *kt = kbase + (int64_t)s * rs;
  const bf16_t *vt = vbase + (int64_t)s * rs;
  dma.issue(kt, rs, key_hi - s + 1, sm.k[0]);
  dma.issue(vt, rs, key_hi - s + 1, sm.v[0]);
  wait_vmem();
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int c0 = s + t * kBK;
    if (t + 1 < ntiles) {
      kt += tile_elems;
      vt += tile_elems;
      dma.issue(kt, rs, key_hi - (c0 + kBK) + 1, sm.k[buf ^ 1]);
      dma.issue(vt, rs, key_hi - (c0 + kBK) + 1, sm.v[buf ^ 1]);
    }
    if (active && c0 <= wave_hi) {
      const bool full = c0 + kBK - 1 <= wave_lo;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        // S^T[key][row], dP^T[key][row] for 32 keys, lane <-> row
        f32x16 sacc, pacc;
        const char *kl = (const char *)sm.k[buf];
        const char *vl = (const char *)sm.v[buf];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const uint32_t o = kb * 32 * RB + 128 * (ks >> 2) + so.rowk[ks & 3];
          sacc = mfma32x32x16(*(const bf16x8 *)(kl + o), qf[ks], ks == 0 ? f32x16{} : sacc);
          pacc = mfma32x32x16(*(const bf16x8 *)(vl + o), df[ks], ks == 0 ? f32x16{} : pacc);
        }
        bf16x8 dsf[2];
#pragma unroll
        for (int bt = 0; bt < 2; ++bt) {
          f32x2 w[4];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int r = 8 * bt + u;
            float p = fast_exp2(fmaf(sacc[r], sl2, -lse2));
            if (!full) {
              const int key = c0 + kb * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
              if (key > lim_r) p = 0.f;
            }
            w[u >> 1][u & 1] = p * (pacc[r] - dlt);
          }
          u32x4 x;
#pragma unroll
          for (int u = 0; u < 4; ++u) x[u] = cvt_bf16x2(w[u]);
          dsf[bt] = __builtin_bit_cast(bf16x8, x);
        }
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const uint32_t cb = ((db & 1) ? so.tro : so.tre) + 64 * db;
#pragma unroll
          for (int bt = 0; bt < 2; ++bt) {
            const uint32_t o = cb + (kb * 32 + 16 * bt) * RB;
            dq[db] = mfma32x32x16(tr_operand_at(kl, o, o + 8 * RB), dsf[bt], dq[db]);
          }
        }
      }
    }
    wait_vmem();
    __syncthreads();
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

template <int D>
hipError_t launch_bwd_t(const BwdArgs &a, hipStream_t stream) {
  const int64_t pairs = (int64_t)a.total * a.hq;
  const int64_t thr = pairs * (D / 8);
  hipLaunchKernelGGL((delta_kernel<D>), dim3((unsigned)((thr + 255) / 256)), dim3(256), 0,
                     stream, (const bf16_t *)a.o, (const bf16_t *)a.dout, a.lse, a.delta,
                     a.lse2, a.total, a.hq);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;

  const int ktiles = (a.max_seqlen + kKW - 1) / kKW;
  const int64_t tot_kv = (int64_t)a.batch * a.hkv * ktiles;
  hipLaunchKernelGGL((dkv_kernel<D>), dim3((unsigned)(8 * ((tot_kv + 7) / 8))), dim3(512), 0,
                     stream, a, ktiles);
  if ((err = hipGetLastError()) != hipSuccess) return err;

  const int hpw = gcd_i(a.hq / a.hkv, 4);
  const int wg_rows = (4 / hpw) * 32;
  const int tiles = (a.max_seqlen + wg_rows - 1) / wg_rows;
  const int64_t tot_q = (int64_t)a.batch * (a.hq / hpw) * tiles;
  hipLaunchKernelGGL((dq_kernel<D>), dim3((unsigned)(8 * ((tot_q + 7) / 8))), dim3(256), 0,
                     stream, a, hpw, tiles);
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
