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
#define ISM_DKV_WPE 1
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

// delta over (row, head) pairs: D/8 lanes per pair, 16-byte loads.
template <int D>
__global__ void __launch_bounds__(256)
delta_kernel(const bf16_t *__restrict__ o, const bf16_t *__restrict__ dout,
             float *__restrict__ delta, int32_t total, int32_t hq) {
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
  }
}

// ---------------------------------------------------------------- dK / dV

// Q and dO tiles of 32 rows, unpadded swizzled rows (see swz()), filled by
// direct global->LDS transfers; transposed operands are read with
// ds_read_b64_tr_b16. Per-row LSE (log2), delta and lim ride along.
template <int D>
struct DkvSmem {
  bf16_t q[2][kBR * D];
  bf16_t dout[2][kBR * D];
  __attribute__((aligned(16))) float lse2[2][kBR];
  __attribute__((aligned(16))) float delta[2][kBR];
  __attribute__((aligned(16))) int lim[2][kBR];
};

// Threads 224..255 stage the per-row scalars of a 32-row tile (lim = -1
// marks rows past the end of the dialogue).
struct RowScalars {
  float l2, dl;
  int lm;
  bool has_row;

  __device__ __forceinline__ void init(int tid) { has_row = tid >= 224; }

  __device__ __forceinline__ void load(const BwdArgs &a, int r0, int e, int h) {
    if (!has_row) return;
    const int row = r0 + ((int)threadIdx.x - 224);
    const bool ok = row < e;
    const int rc = ok ? row : e - 1;
    l2 = a.lse[(int64_t)h * a.total + rc] * kLog2e;
    dl = a.delta[(int64_t)h * a.total + rc];
    lm = ok ? a.lim[rc] : -1;
  }

  __device__ __forceinline__ void store(float *lse2, float *delta, int *lim) const {
    if (!has_row) return;
    const int rr = (int)threadIdx.x - 224;
    lse2[rr] = l2;
    delta[rr] = dl;
    lim[rr] = lm;
  }
};

template <int D>
__global__ void __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(ISM_DKV_WPE, ISM_DKV_WPE)))
dkv_kernel(BwdArgs a, int ktiles) {
  constexpr int NKS = D / 16, NDB = D / 32, RB = D * 2;
  __shared__ DkvSmem<D> sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
  const int kw0 = c0 + 32 * wave;
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
      vf[ks] = *(const bf16x8 *)(vp + ks * 16);
    }
  }
  f32x16 dk[NDB], dv[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) { dk[db] = f32x16{}; dv[db] = f32x16{}; }

  const int rstart = a.seer[c0];
  const int nrt = (e - rstart + kBR - 1) / kBR;
  const int iters = G * nrt;
  const int64_t rs = (int64_t)a.hq * D;
  DmaTile<D, kBR> dma;
  dma.init(tid, rs);
  SwzOffsets so;
  so.init(lane, RB);
  RowScalars rsc;
  rsc.init(tid);
  auto issue = [&](int r0, int h, int buf) {
    const int64_t base = ((int64_t)r0 * a.hq + h) * D;
    dma.issue((const bf16_t *)a.q + base, rs, e - r0, sm.q[buf]);
    dma.issue((const bf16_t *)a.dout + base, rs, e - r0, sm.dout[buf]);
    rsc.load(a, r0, e, h);
  };
  issue(rstart, kvh * G, 0);
  rsc.store(sm.lse2[0], sm.delta[0], sm.lim[0]);
  wait_vmem();
  __syncthreads();

  for (int it = 0; it < iters; ++it) {
    const int buf = it & 1;
    const int r0 = rstart + (it % nrt) * kBR;
    if (it + 1 < iters) {
      const int g1 = (it + 1) / nrt, rt1 = (it + 1) % nrt;
      issue(rstart + rt1 * kBR, kvh * G + g1, buf ^ 1);
    }
    const int nvalid = min(kBR, e - r0);
    const int lim_last = sm.lim[buf][nvalid - 1];
    if (wactive && lim_last >= kw0) {
      const bool full = nvalid == kBR && sm.lim[buf][0] >= kw0 + 31;
      // S[row][key] and dP[row][key], lane <-> key, rows 8i + 4hf + j
      f32x16 sacc, pacc;
      const char *ql = (const char *)sm.q[buf];
      const char *dl = (const char *)sm.dout[buf];
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const uint32_t o = 128 * (ks >> 2) + so.rowk[ks & 3];
        sacc = mfma32x32x16(*(const bf16x8 *)(ql + o), kf[ks], ks == 0 ? f32x16{} : sacc);
        pacc = mfma32x32x16(*(const bf16x8 *)(dl + o), vf[ks], ks == 0 ? f32x16{} : pacc);
      }
      const int key = kw0 + l32;
      bf16x8 pfr[2] = {}, dsf[2] = {};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 l2 = *(const f32x4 *)&sm.lse2[buf][8 * i + 4 * hf];
        const f32x4 dl = *(const f32x4 *)&sm.delta[buf][8 * i + 4 * hf];
        int lm[4] = {0, 0, 0, 0};
        if (!full) {
          const u32x4 li = *(const u32x4 *)&sm.lim[buf][8 * i + 4 * hf];
#pragma unroll
          for (int j = 0; j < 4; ++j) lm[j] = (int)li[j];
        }
        f32x2 pp[2], dd[2];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float p = fast_exp2(fmaf(sacc[4 * i + j], sl2, -l2[j]));
          if (!full && key > lm[j]) p = 0.f;
          pp[j >> 1][j & 1] = p;
          dd[j >> 1][j & 1] = p * (pacc[4 * i + j] - dl[j]);
        }
        // rows 8i..8i+3 (+4hf) are slots 4*(i&1).. of operand i>>1
        const int bt = i >> 1, sl = (i & 1) * 2;
        u32x4 wp = __builtin_bit_cast(u32x4, pfr[bt]);
        u32x4 wd = __builtin_bit_cast(u32x4, dsf[bt]);
        wp[sl] = cvt_bf16x2(pp[0]);
        wp[sl + 1] = cvt_bf16x2(pp[1]);
        wd[sl] = cvt_bf16x2(dd[0]);
        wd[sl + 1] = cvt_bf16x2(dd[1]);
        pfr[bt] = __builtin_bit_cast(bf16x8, wp);
        dsf[bt] = __builtin_bit_cast(bf16x8, wd);
      }
      // dV^T[d][key] += dO^T P, dK^T[d][key] += Q^T dS (contraction over rows)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const uint32_t cb = ((db & 1) ? so.tro : so.tre) + 64 * db;
#pragma unroll
        for (int bt = 0; bt < 2; ++bt) {
          const uint32_t o = cb + 16 * bt * RB;
          dv[db] = mfma32x32x16(tr_operand_at(dl, o, o + 8 * RB), pfr[bt], dv[db]);
          dk[db] = mfma32x32x16(tr_operand_at(ql, o, o + 8 * RB), dsf[bt], dk[db]);
        }
      }
    }
    if (it + 1 < iters) rsc.store(sm.lse2[buf ^ 1], sm.delta[buf ^ 1], sm.lim[buf ^ 1]);
    wait_vmem();
    __syncthreads();
  }

  const int key = kw0 + l32;
  if (!wactive || key >= e) return;
  float *dkp = a.dk + ((int64_t)key * a.hkv + kvh) * D + hf * 4;
  float *dvp = a.dv + ((int64_t)key * a.hkv + kvh) * D + hf * 4;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 xk, xv;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        xk[j] = dk[db][4 * i + j] * a.scale;
        xv[j] = dv[db][4 * i + j];
      }
      *(f32x4 *)(dkp + db * 32 + 8 * i) = xk;
      *(f32x4 *)(dvp + db * 32 + 8 * i) = xv;
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
  const float lse2 = a.lse[(int64_t)head * a.total + rc] * kLog2e;
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
                     stream, (const bf16_t *)a.o, (const bf16_t *)a.dout, a.delta, a.total,
                     a.hq);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;

  const int ktiles = (a.max_seqlen + kKW - 1) / kKW;
  const int64_t tot_kv = (int64_t)a.batch * a.hkv * ktiles;
  hipLaunchKernelGGL((dkv_kernel<D>), dim3((unsigned)(8 * ((tot_kv + 7) / 8))), dim3(256), 0,
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
