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

// Build-time tile configuration: rows per wave = 32 * ISM_FWD_NQB, and the
// occupancy target in waves per SIMD (1 or 2) that bounds registers.
#ifndef ISM_FWD_NQB
#define ISM_FWD_NQB 1
#endif
#ifndef ISM_FWD_WPE
#define ISM_FWD_WPE 2
#endif

namespace {

constexpr int kBN = 64;  // keys per tile

// K and V tiles of 64 keys, row-major, unpadded rows of D bf16 with the
// swz() chunk swizzle, double-buffered; filled by direct global->LDS
// transfers. K is read as MFMA rows (ds_read_b128), V through transposing
// reads (ds_read_b64_tr_b16) as the V^T operand.
template <int D>
struct FwdSmem {
  bf16_t k[2][kBN * D];
  bf16_t v[2][kBN * D];
};

// Online softmax of one 64-key tile held as S^T accumulators (lane <->
// query row; the other 32 keys of the row sit in lane l ^ 32). Writes the
// bf16 probabilities as B operands of the P V product.
template <bool MASK, int NQB, int NDB>
__device__ __forceinline__ void softmax_tile(f32x16 (&sacc)[2][NQB], int c0, int hf,
                                             const int (&lim_r)[NQB], float sl2, float tau,
                                             float (&m_run)[NQB], float (&l_run)[NQB],
                                             f32x16 (&oacc)[NDB][NQB],
                                             bf16x8 (&pf)[NQB][2][2]) {
  float mt[NQB];
  bool grow = false;
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    float x = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (MASK) {
          const int key = c0 + kb * 32 + (r >> 2) * 8 + hf * 4 + (r & 3);
          if (key > lim_r[qb]) sacc[kb][qb][r] = -INFINITY;
        }
        x = fmaxf(x, sacc[kb][qb][r]);
      }
    mt[qb] = pair_max(x);
    grow |= mt[qb] > m_run[qb] + tau;
  }
  if (__builtin_amdgcn_ballot_w64(grow) != 0) {
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const float mnew = fmaxf(m_run[qb], mt[qb]);
      const float alpha = fast_exp2((m_run[qb] - mnew) * sl2);
      m_run[qb] = mnew;
      l_run[qb] *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][qb][r] *= alpha;
    }
  }
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const float moff = m_run[qb] * sl2;
    float rsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int bt = 0; bt < 2; ++bt) {
        f32x2 p[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          p[u][0] = fast_exp2(fmaf(sacc[kb][qb][8 * bt + 2 * u], sl2, -moff));
          p[u][1] = fast_exp2(fmaf(sacc[kb][qb][8 * bt + 2 * u + 1], sl2, -moff));
          rsum += p[u][0] + p[u][1];
        }
        u32x4 w;
#pragma unroll
        for (int u = 0; u < 4; ++u) w[u] = cvt_bf16x2(p[u]);
        pf[qb][kb][bt] = __builtin_bit_cast(bf16x8, w);
      }
    l_run[qb] += rsum;
  }
}

template <int D, int NQB, bool CACHE>
__global__ void __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(ISM_FWD_WPE, ISM_FWD_WPE)))
fwd_kernel(FwdArgs a, int hpw, int tiles) {
  constexpr int QW = NQB * 32;     // rows per wave
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
  wait_loads();

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

  // lazy rescaling: the running max is only raised when a row's tile max
  // exceeds it by more than 2^8 in probability units (exact either way:
  // numerator and denominator share the reference max)
  const float tau = 8.f / sl2;
  bf16x8 pf[NQB][2][2];

  const int ntiles = (key_hi - key_begin) / kBN + 1;
  DmaTile<D, kBN> dma;
  dma.init(tid, rs);
  SwzOffsets so;
  so.init(lane, D * 2);
  const int64_t tile_elems = (int64_t)kBN * rs;
  const bf16_t *kt = kbase + (int64_t)key_begin * rs;
  const bf16_t *vt = vbase + (int64_t)key_begin * rs;
  dma.issue(kt, rs, key_hi - key_begin + 1, sm.k[0]);
  dma.issue(vt, rs, key_hi - key_begin + 1, sm.v[0]);
  wait_vmem();
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int c0 = key_begin + t * kBN;
    if (t + 1 < ntiles) {
      kt += tile_elems;
      vt += tile_elems;
      dma.issue(kt, rs, key_hi - (c0 + kBN) + 1, sm.k[buf ^ 1]);
      dma.issue(vt, rs, key_hi - (c0 + kBN) + 1, sm.v[buf ^ 1]);
    }

    if (active && c0 <= wave_hi) {
      // S^T[key][row] for two 32-key blocks
      f32x16 sacc[2][NQB];
      const char *kl = (const char *)sm.k[buf];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const bf16x8 kf = *(const bf16x8 *)(kl + kb * 32 * D * 2 + 128 * (ks >> 2) +
                                              so.rowk[ks & 3]);
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb)
            sacc[kb][qb] = mfma32x32x16(kf, qf[qb][ks], ks == 0 ? f32x16{} : sacc[kb][qb]);
        }
      }
      // only tiles that cross some row's bound pay for the mask
      if (c0 + kBN - 1 <= wave_lo) {
        softmax_tile<false>(sacc, c0, hf, lim_r, sl2, tau, m_run, l_run, oacc, pf);
      } else {
        softmax_tile<true>(sacc, c0, hf, lim_r, sl2, tau, m_run, l_run, oacc, pf);
      }

      // O^T[d][row] += V^T[d][key] P^T[key][row]
      const char *vl = (const char *)sm.v[buf];
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const uint32_t cb = ((db & 1) ? so.tro : so.tre) + 64 * db;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int bt = 0; bt < 2; ++bt) {
            const uint32_t o = cb + (kb * 32 + 16 * bt) * D * 2;
            const bf16x8 vf = tr_operand_at(vl, o, o + 8 * D * 2);
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb)
              oacc[db][qb] = mfma32x32x16(vf, pf[qb][kb][bt], oacc[db][qb]);
          }
      }
    }

    wait_vmem();
    __syncthreads();
  }

  if (!active) return;
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const float lt = pair_sum(l_run[qb]);
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
  constexpr int NQB = ISM_FWD_NQB;
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
