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

template <int D>
struct FwdSmem {
  static constexpr int KSTR = D + 8;  // padded K row (bank-conflict-free b128 reads)
  bf16_t k[2][kBN * KSTR];
  // V^T: one 128-byte row of 64 keys per head-dim index. Inside a row, key
  // bits 2 and 3 are swapped so that the 8 keys one lane feeds to a P V
  // MFMA are contiguous (one ds_read_b128), and the eight 16-byte chunks are
  // XOR-swizzled with (row & 7) so that the 8 lanes of a read pass hit 8
  // different chunks.
  bf16_t vt[2][D * kBN];
};

// Byte offset of the 16-byte V^T chunk holding keys [32kb + 16bt + 8hf ..)
// in storage order (see FwdSmem) for head-dim row d.
__device__ __forceinline__ uint32_t vt_chunk(int d, int kb, int bt, int hf) {
  return (uint32_t)(d * 128 + (((4 * kb + 2 * bt + hf) ^ (d & 7)) << 4));
}

// Stages one 64-key tile of K (row-major, padded) and V (transposed) through
// registers. Thread-invariant address parts are computed once; a tile's base
// is wave-uniform. Keys past the tile's valid count are clamped to the last
// valid key (always valid memory); the caller masks them.
template <int D>
struct TileLoader {
  static constexpr int KCH = kBN * (D / 8) / 256;  // 16-byte K chunks per thread
  static constexpr int RPI = 256 / (D / 8);         // K rows covered per chunk round
  static constexpr int KSTR = FwdSmem<D>::KSTR;
  u32x4 kr[KCH];
  u32x4 vr[4];
  uint32_t koff;   // byte offset of K chunk 0 of this thread inside a tile
  uint32_t voff;   // byte offset of V row 4kg, chunk dc inside a tile
  uint32_t kls;    // LDS byte offset of K chunk 0
  uint32_t vls;    // LDS byte offset of V^T row dc*8, half (swap2(kg) & 1)
  int krow, vrow, vch, rsb;
  bool vjob;

  __device__ __forceinline__ void init(int64_t rs, int tid) {
    rsb = (int)(rs * 2);
    krow = tid / (D / 8);
    const int col = tid % (D / 8);
    koff = (uint32_t)(krow * rsb + col * 16);
    kls = (uint32_t)((krow * KSTR + col * 8) * 2);
    vjob = tid < 16 * (D / 8);
    const int kg = tid & 15, dc = tid >> 4;
    vrow = 4 * kg;
    voff = (uint32_t)(vrow * rsb + dc * 16);
    const int u = ((kg & 1) << 1) | ((kg >> 1) & 1) | (kg & ~3);  // swap bits 0,1
    vch = u >> 1;
    vls = (uint32_t)(dc * 8 * 128 + (u & 1) * 8);
  }

  // tile = key base of the tile in global memory; nvalid = keys < 64 valid
  __device__ __forceinline__ void load(const char *kt, const char *vt, int nvalid) {
    if (nvalid >= kBN) {
#pragma unroll
      for (int i = 0; i < KCH; ++i)
        kr[i] = *(const u32x4 *)(kt + (int64_t)(RPI * i) * rsb + koff);
      if (vjob) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          vr[r] = *(const u32x4 *)(vt + (int64_t)r * rsb + voff);
      }
    } else {
      const int last = nvalid - 1;
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const int row = min(krow + RPI * i, last);
        kr[i] = *(const u32x4 *)(kt + (int64_t)(row - krow) * rsb + koff);
      }
      if (vjob) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = min(vrow + r, last);
          vr[r] = *(const u32x4 *)(vt + (int64_t)(row - vrow) * rsb + voff);
        }
      }
    }
  }

  __device__ __forceinline__ void store(FwdSmem<D> &sm, int buf) {
    char *kb = (char *)&sm.k[buf][0];
#pragma unroll
    for (int i = 0; i < KCH; ++i)
      *(u32x4 *)(kb + kls + i * RPI * KSTR * 2) = kr[i];
    if (vjob) {
      char *vb = (char *)&sm.vt[buf][0] + vls;
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) {
        const int m = dd >> 1;
        // keys 4kg..4kg+3 of head-dim index 8dc+dd, packed as two bf16 pairs
        const uint32_t sel = (dd & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t x0 = __builtin_amdgcn_perm(vr[1][m], vr[0][m], sel);
        const uint32_t x1 = __builtin_amdgcn_perm(vr[3][m], vr[2][m], sel);
        *(u32x2 *)(vb + dd * 128 + ((vch ^ dd) << 4)) = u32x2{x0, x1};
      }
    }
  }
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

  // lazy rescaling: the running max is only raised when a row's tile max
  // exceeds it by more than 2^8 in probability units (exact either way:
  // numerator and denominator share the reference max)
  const float tau = 8.f / sl2;
  bf16x8 pf[NQB][2][2];

  const int ntiles = (key_hi - key_begin) / kBN + 1;
  TileLoader<D> ld;
  ld.init(rs, tid);
  const int64_t tile_bytes = (int64_t)kBN * rs * 2;
  const char *kt = (const char *)(kbase + (int64_t)key_begin * rs);
  const char *vt = (const char *)(vbase + (int64_t)key_begin * rs);
  ld.load(kt, vt, key_hi - key_begin + 1);
  ld.store(sm, 0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int c0 = key_begin + t * kBN;
    if (t + 1 < ntiles) {
      kt += tile_bytes;
      vt += tile_bytes;
      ld.load(kt, vt, key_hi - (c0 + kBN) + 1);
    }

    if (active && c0 <= wave_hi) {
      // S^T[key][row] for two 32-key blocks
      f32x16 sacc[2][NQB];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16_t *kp = &sm.k[buf][(kb * 32 + l32) * KSTR + hf * 8];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const bf16x8 kf = *(const bf16x8 *)(kp + ks * 16);
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
      const char *vtb = (const char *)&sm.vt[buf][0];
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int bt = 0; bt < 2; ++bt) {
            const bf16x8 vf =
                *(const bf16x8 *)(vtb + vt_chunk(db * 32 + l32, kb, bt, hf));
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb)
              oacc[db][qb] = mfma32x32x16(vf, pf[qb][kb][bt], oacc[db][qb]);
          }
      }
    }

    if (t + 1 < ntiles) ld.store(sm, buf ^ 1);
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
