// Forward ISM attention on gfx950: per-token visibility bounds (Eq. 5) and a
// flash-style online-softmax kernel on bf16 MFMA 32x32x16 with fp32
// accumulation. The same kernel serves the cached prefill of a new query
// segment (Sec. 2.3), where every key of the concatenated cache is visible.
//
// Work decomposition. A workgroup (4 waves) owns a row tile of one dialogue
// and a set of query heads that share one KV head: with G = hq / hkv query
// heads per KV head, hpw = gcd(G, 4) heads run side by side (one per wave
// column) so that the K/V tile staged in LDS serves all of them, and the
// remaining 4 / hpw waves take consecutive 32*NQB-row blocks. Each wave
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

namespace {

constexpr int kBN = 64;  // keys per tile

template <int D>
struct FwdSmem {
  static constexpr int KSTR = D + 8;  // padded K row (bank-conflict-free b128 reads)
  bf16_t k[2][kBN * KSTR];
  bf16_t vt[2][D * kBN];              // V^T, 8-byte units XOR-swizzled by row
};

// Stage one 64-key tile of K (row-major, padded) and V (transposed) through
// registers. Keys past key_hi are clamped to key_hi (always valid memory);
// they are masked out by the caller.
template <int D>
struct TileLoader {
  static constexpr int KCH = kBN * (D / 8) / 256;  // 16-byte K chunks per thread
  u32x4 kr[KCH];
  u32x4 vr[4];

  __device__ __forceinline__ void load(const bf16_t *kbase, const bf16_t *vbase,
                                       int64_t rs, int c0, int key_hi, int tid) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + 256 * i;
      const int row = c / (D / 8), col = c % (D / 8);
      const int key = min(c0 + row, key_hi);
      kr[i] = *(const u32x4 *)(kbase + (int64_t)key * rs + col * 8);
    }
    if (tid < 16 * (D / 8)) {
      const int kg = tid & 15, dc = tid >> 4;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = min(c0 + 4 * kg + r, key_hi);
        vr[r] = *(const u32x4 *)(vbase + (int64_t)key * rs + dc * 8);
      }
    }
  }

  __device__ __forceinline__ void store(FwdSmem<D> &sm, int buf, int tid) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + 256 * i;
      const int row = c / (D / 8), col = c % (D / 8);
      *(u32x4 *)&sm.k[buf][row * FwdSmem<D>::KSTR + col * 8] = kr[i];
    }
    if (tid < 16 * (D / 8)) {
      const int kg = tid & 15, dc = tid >> 4;
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) {
        const int m = dd >> 1;
        uint32_t x0, x1;
        if ((dd & 1) == 0) {
          x0 = (vr[0][m] & 0xffffu) | (vr[1][m] << 16);
          x1 = (vr[2][m] & 0xffffu) | (vr[3][m] << 16);
        } else {
          x0 = (vr[0][m] >> 16) | (vr[1][m] & 0xffff0000u);
          x1 = (vr[2][m] >> 16) | (vr[3][m] & 0xffff0000u);
        }
        const int row = dc * 8 + dd;
        const int pu = kg ^ (row & 15);
        *(u32x2 *)&sm.vt[buf][row * kBN + pu * 4] = u32x2{x0, x1};
      }
    }
  }
};

template <int D, int NQB, bool CACHE>
__global__ void __launch_bounds__(256)
fwd_kernel(FwdArgs a, int hpw, int tiles) {
  constexpr int QW = NQB * 32;     // rows per wave
  constexpr int KSTR = FwdSmem<D>::KSTR;
  constexpr int NDB = D / 32;      // 32-wide d blocks of the output
  constexpr int NKS = D / 16;      // 16-deep k steps of Q K^T
  __shared__ FwdSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;

  // Work item: XCD-aware (consecutive workgroups land on different XCDs, so
  // give each XCD a contiguous run of items), longest row tile first inside
  // each (dialogue, head set) group.
  const int hsets = a.hq / hpw;
  const int total = a.batch * hsets * tiles;
  const int per = (total + 7) / 8;
  const int item = (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);
  if (item >= total) return;
  const int group = item / tiles;
  const int tile = tiles - 1 - item % tiles;
  const int b = group / hsets;
  const int head0 = (group % hsets) * hpw;
  const int wg_rows = (4 / hpw) * QW;
  const int s = a.cu_q[b], e = a.cu_q[b + 1];
  const int q0 = s + tile * wg_rows;
  if (q0 >= e) return;

  const int head = head0 + wave % hpw;
  const int kvh = head0 / (a.hq / a.hkv);
  const int wq0 = q0 + (wave / hpw) * QW;
  const bool active = wq0 < e;
  const int wg_last = min(q0 + wg_rows, e) - 1;

  int key_begin, key_hi, wave_lo, wave_hi;
  const bf16_t *kbase, *vbase;
  if (CACHE) {
    key_begin = 0;
    // keys [0, C_b + L_b); clamped to the slab for out-of-contract lengths
    key_hi = max(min(a.cache_len[b] + (e - s), a.kv_head_stride / D) - 1, 0);
    wave_lo = key_hi;
    wave_hi = active ? key_hi : -1;
    const int64_t off = (int64_t)b * a.kv_seq_stride + (int64_t)kvh * a.kv_head_stride;
    kbase = (const bf16_t *)a.k + off;
    vbase = (const bf16_t *)a.v + off;
  } else {
    key_begin = s;
    key_hi = a.lim[wg_last];
    wave_lo = a.lim[min(wq0, e - 1)];
    wave_hi = active ? a.lim[min(wq0 + QW, e) - 1] : s - 1;
    kbase = (const bf16_t *)a.k + (int64_t)kvh * a.kv_head_stride;
    vbase = (const bf16_t *)a.v + (int64_t)kvh * a.kv_head_stride;
  }
  const int64_t rs = a.kv_row_stride;
  const float sl2 = a.scale * kLog2e;

  // Per-lane query rows (clamped into the dialogue; rows past e are computed
  // as copies of the last row and never stored).
  int lim_r[NQB];
  bf16x8 qf[NQB][NKS];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int rc = min(wq0 + qb * 32 + l32, e - 1);
    lim_r[qb] = CACHE ? key_hi : a.lim[rc];
    const bf16_t *qp = (const bf16_t *)a.q + ((int64_t)rc * a.hq + head) * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[qb][ks] = *(const bf16x8 *)(qp + ks * 16);
  }

  f32x16 oacc[NDB][NQB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][qb][r] = 0.f;
  float m_run[NQB], l_run[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) { m_run[qb] = -INFINITY; l_run[qb] = 0.f; }

  const int ntiles = (key_hi - key_begin) / kBN + 1;
  TileLoader<D> ld;
  ld.load(kbase, vbase, rs, key_begin, key_hi, tid);
  ld.store(sm, 0, tid);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int c0 = key_begin + t * kBN;
    if (t + 1 < ntiles) ld.load(kbase, vbase, rs, c0 + kBN, key_hi, tid);

    if (active && c0 <= wave_hi) {
      const bool full = c0 + kBN - 1 <= wave_lo;
      // S^T[key][row] for two 32-key blocks
      f32x16 sacc[2][NQB];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
          for (int r = 0; r < 16; ++r) sacc[kb][qb][r] = 0.f;
        const bf16_t *kp = &sm.k[buf][(kb * 32 + l32) * KSTR + hf * 8];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const bf16x8 kf = *(const bf16x8 *)(kp + ks * 16);
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb)
            sacc[kb][qb] = mfma32x32x16(kf, qf[qb][ks], sacc[kb][qb]);
        }
      }

      // online softmax, one query row per lane (pair)
      bf16x8 pf[NQB][2][2];
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        float mt = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            float x = sacc[kb][qb][r];
            if (!full) {
              const int key = c0 + kb * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
              if (key > lim_r[qb]) x = -INFINITY;
              sacc[kb][qb][r] = x;
            }
            mt = fmaxf(mt, x);
          }
        mt = fmaxf(mt, swap_halves(mt));
        const float mnew = fmaxf(m_run[qb], mt);
        const float alpha = fast_exp2((m_run[qb] - mnew) * sl2);
        m_run[qb] = mnew;
        const float moff = mnew * sl2;
        float rsum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int bt = 0; bt < 2; ++bt) {
            float p[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              p[u] = fast_exp2(fmaf(sacc[kb][qb][8 * bt + u], sl2, -moff));
              rsum += p[u];
            }
            u32x4 w;
            w[0] = pack_bf16x2(p[0], p[1]);
            w[1] = pack_bf16x2(p[2], p[3]);
            w[2] = pack_bf16x2(p[4], p[5]);
            w[3] = pack_bf16x2(p[6], p[7]);
            pf[qb][kb][bt] = __builtin_bit_cast(bf16x8, w);
          }
        l_run[qb] = fmaf(l_run[qb], alpha, rsum);
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[db][qb][r] *= alpha;
      }

      // O^T[d][row] += V^T[d][key] P^T[key][row]
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int d = db * 32 + l32;
        const bf16_t *vrow = &sm.vt[buf][d * kBN];
        const int sw = l32 & 15;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int bt = 0; bt < 2; ++bt) {
            const int u1 = kb * 8 + 4 * bt + hf;
            const u32x2 lo = *(const u32x2 *)(vrow + ((u1 ^ sw) * 4));
            const u32x2 hi = *(const u32x2 *)(vrow + (((u1 + 2) ^ sw) * 4));
            const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
            const bf16x8 vf = __builtin_bit_cast(bf16x8, w);
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb)
              oacc[db][qb] = mfma32x32x16(vf, pf[qb][kb][bt], oacc[db][qb]);
          }
      }
    }

    if (t + 1 < ntiles) ld.store(sm, buf ^ 1, tid);
    __syncthreads();
  }

  if (!active) return;
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const float lt = l_run[qb] + swap_halves(l_run[qb]);
    const int row = wq0 + qb * 32 + l32;
    if (row >= e) continue;
    const float inv = 1.f / lt;
    bf16_t *op = (bf16_t *)a.o + ((int64_t)row * a.hq + head) * D + hf * 4;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        u32x2 w;
        w[0] = pack_bf16x2(oacc[db][qb][4 * i + 0] * inv, oacc[db][qb][4 * i + 1] * inv);
        w[1] = pack_bf16x2(oacc[db][qb][4 * i + 2] * inv, oacc[db][qb][4 * i + 3] * inv);
        *(u32x2 *)(op + db * 32 + 8 * i) = w;
      }
    if (a.lse && hf == 0)
      a.lse[(int64_t)head * a.total_q + row] = m_run[qb] * a.scale + logf(lt);
  }
}

int gcd_int(int x, int y) {
  while (y) { const int t = x % y; x = y; y = t; }
  return x;
}

template <int D, bool CACHE>
hipError_t launch_fwd_t(const FwdArgs &a, hipStream_t stream) {
  constexpr int NQB = 2;
  const int hpw = gcd_int(a.hq / a.hkv, 4);
  const int wg_rows = (4 / hpw) * NQB * 32;
  const int tiles = (a.max_rows + wg_rows - 1) / wg_rows;
  const int64_t total = (int64_t)a.batch * (a.hq / hpw) * tiles;
  if (total == 0) return hipSuccess;
  const int64_t per = (total + 7) / 8;
  hipLaunchKernelGGL((fwd_kernel<D, NQB, CACHE>), dim3((unsigned)(8 * per)),
                     dim3(256), 0, stream, a, hpw, tiles);
  return hipGetLastError();
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
