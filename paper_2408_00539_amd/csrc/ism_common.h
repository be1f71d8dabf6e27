// Internal helpers shared by the HIP kernels of the ISM attention library.
// gfx950 (CDNA4) only: wave64, bf16 MFMA 32x32x16, 160 KiB LDS per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace ism {

typedef __bf16 bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// D(32x32, fp32) += A(32x16, bf16) * B(16x32, bf16).
// Operand layout (lane l, half h = l / 32): A holds row l % 32, k = 8h..8h+7;
// B holds column l % 32, k = 8h..8h+7; the accumulator element r = 4i + j
// of lane l sits at row 8i + 4h + j, column l % 32.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Exchange a value with lane l ^ 32 (the other half of the wave).
__device__ __forceinline__ float swap_halves(float x) {
  return __shfl_xor(x, 32);
}

// IEEE 754-2019 maximum (NaN-propagating): one v_maximum3_f32 for up to three
// operands, with none of the operand quieting that fmaxf needs.
__device__ __forceinline__ float vmax(float a, float b) {
  return __builtin_elementwise_maximum(a, b);
}

// max / sum of x over lanes l and l ^ 32, via v_permlane32_swap: after the
// swap of (x, x) the two results hold, in every lane, the lower-half and the
// upper-half value of that lane pair.
__device__ __forceinline__ float pair_max(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return vmax(__builtin_bit_cast(float, (uint32_t)r[0]),
              __builtin_bit_cast(float, (uint32_t)r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) +
         __builtin_bit_cast(float, (uint32_t)r[1]);
}

__device__ __forceinline__ float fast_exp2(float x) {
  return __builtin_amdgcn_exp2f(x);
}

// Two floats -> packed bf16 pair in one v_cvt_pk_bf16_f32 (round to nearest even).
__device__ __forceinline__ uint32_t cvt_bf16x2(f32x2 v) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return cvt_bf16x2(f32x2{lo, hi});
}

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// Two floats -> packed fp16 pair in one v_cvt_pk_f16_f32 (round to nearest even).
__device__ __forceinline__ uint32_t cvt_f16x2(f32x2 v) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2));
}

// The low / high fp16 half of w times an fp32 value, as one v_fma_mix_f32
// (the conversion is exact, the product rounds once).
__device__ __forceinline__ float mul_f16_lo(uint32_t w, float b) {
  return __builtin_fmaf((float)__builtin_bit_cast(f16x2, w).x, b, 0.f);
}
__device__ __forceinline__ float mul_f16_hi(uint32_t w, float b) {
  return __builtin_fmaf((float)__builtin_bit_cast(f16x2, w).y, b, 0.f);
}

typedef short i16x4 __attribute__((ext_vector_type(4)));

// A operand (32 x 16, bf16) of a 32x32x16 MFMA read from a tile stored with
// the MFMA k index as the row: tile[k * str + m]. Lane l receives row
// m0 + (l % 32) and k = k0 + 4h + {0..3} (slots 0-3), k0 + 8 + 4h + {0..3}
// (slots 4-7), h = l / 32, through two ds_read_b64_tr_b16. That transposing
// read works per 16-lane group: output lane r gets element r % 4 of the
// 8-byte loads of lanes r/4, r/4 + 4, r/4 + 8, r/4 + 12; so lane L of a group
// loads tile row k0 + 4h + L/4, columns m + 4 (L % 4) .. + 3.
__device__ __forceinline__ bf16x8 tr_operand(const bf16_t *tile, int str, int m0, int k0,
                                             int lane) {
  const int g = lane >> 4, L = lane & 15;
  const int m = m0 + 16 * (g & 1) + 4 * (L & 3);
  const int k = k0 + 4 * (g >> 1) + (L >> 2);
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(tile + k * str + m));
  const i16x4 hi =
      __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(tile + (k + 8) * str + m));
  const i16x4 v[2] = {lo, hi};
  return __builtin_bit_cast(bf16x8, v);
}

// Row swizzle of 16-byte chunks in unpadded LDS tiles of D bf16 per row:
// logical chunk c of tile row r is stored at chunk c ^ swz<D>(r). It depends
// on r % 16 only and takes 16 (D = 128) or 8 (D = 64) distinct values there,
// so that both a ds_read_b128 of 16 consecutive rows at one chunk and the
// 4 rows x 32 bytes of each ds_read_b64_tr_b16 lane group hit distinct banks
// (64 banks of 4 bytes, 256 bytes per LDS cycle).
template <int D>
__device__ __forceinline__ int swz(int r) {
  static_assert(D == 64 || D == 128, "head dim 64 or 128");
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return ((r >> 1) & 3) | ((((r >> 1) ^ (r >> 3)) & 1) << 2);
}

// Byte address of a pointer into LDS.
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// global_load_lds_dwordx4 / _dword: each active lane copies 16 / 4 bytes
// from its global address to LDS at lds_base + 16 * lane / 4 * lane
// (lds_base wave-uniform, placed in M0). Written as inline assembly so that
// the compiler does not model the LDS write: the kernels order these
// transfers themselves with counted s_waitcnt vmcnt and barriers, and the
// compiler would otherwise drain every transfer in flight before each LDS
// read of another buffer.
__device__ __forceinline__ void dma_x4(const void *g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(__builtin_amdgcn_readfirstlane(lds_base))
               : "memory", "m0");
}
// The same with a wave-uniform base address in SGPRs and a per-lane 32-bit
// byte offset (the address is base + offset): no 64-bit address arithmetic
// per transfer.
// NT: a non-temporal load (data read once, such as a KV-cache stream).
template <bool NT = false>
__device__ __forceinline__ void dma_x4s(const void *base, uint32_t off, uint32_t lds_base) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt"
                 :
                 : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds_base))
                 : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds_base))
                 : "memory", "m0");
}
__device__ __forceinline__ void dma_x1(const void *g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(g), "s"(__builtin_amdgcn_readfirstlane(lds_base))
               : "memory", "m0");
}

// Workgroup barrier without memory fences, for loops that order their LDS
// traffic with explicit s_waitcnt: outstanding LDS reads are drained first,
// global->LDS transfers are left in flight.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
}

// Compiler-visible wait for all outstanding vector-memory loads of this
// wave (register operands loaded before a pipelined loop), so that the
// compiler's own wait accounting does not carry them into the loop.
__device__ __forceinline__ void wait_loads() {
  __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8));
}

// Wait until this wave's outstanding vector-memory operations, including
// global->LDS transfers, have completed.
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// The same, leaving the wave's N most recent vector-memory operations in
// flight (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vmem_but() {
  static_assert(N >= 0 && N < 64, "vmcnt takes 0..63");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Direct global->LDS staging of a ROWS x D bf16 tile (unpadded, swizzled)
// by the NW waves of a workgroup. Each global_load_lds_dwordx4 writes lane
// l's 16 bytes to LDS bytes [16 l, 16 l + 16) of a 1 KB block, so the swizzle
// is applied by choosing each lane's source chunk. No registers hold the
// data. Block q of the tile is issued by wave q % NW; the workgroup has
// exactly NW waves. NT: non-temporal transfers (see dma_x4s).
template <int D, int ROWS, int NW = 4, bool NT = false>
struct DmaTile {
  static constexpr int CPR = D / 8;                 // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;              // rows per 1 KB transfer
  static constexpr int T = ROWS / RPI;              // transfers per tile
  static constexpr int NI = (T + NW - 1) / NW;      // transfers per wave (max)
  // every wave issues NI transfers (no per-transfer bound check, which the
  // compiler would keep as a branch around each transfer)
  static constexpr bool kEven = T % NW == 0;
  static_assert(ROWS % RPI == 0, "tile rows must fill whole transfers");
  uint32_t loff[NI];  // byte offset of this lane's source chunk (full tile)
  int wave, lane;

  // rs: row stride in elements; ROWS * rs * 2 bytes must fit in 32 bits
  __device__ __forceinline__ void init(int tid, int64_t rs) {
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    lane = tid & 63;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = (i * NW + wave) * RPI + lane / CPR;
      loff[i] = (uint32_t)(r * rs + ((lane % CPR) ^ swz<D>(r)) * 8) * 2u;
    }
  }

  // Transfer i (of NI) of this wave for a tile whose rows are all valid.
  __device__ __forceinline__ void issue_one(const bf16_t *src, int i, bf16_t *lds) const {
    const int q = i * NW + wave;
    if (kEven || q < T) dma_x4s<NT>(src, loff[i], lds_addr(lds) + q * 1024);
  }

  // Rows [0, ROWS) of the tile starting at src (row stride rs elements); rows
  // at or past nvalid repeat row nvalid - 1 (always valid memory).
  __device__ __forceinline__ void issue(const bf16_t *src, int64_t rs, int nvalid,
                                        bf16_t *lds) const {
    const uint32_t lb = lds_addr(lds);
    if (__builtin_amdgcn_readfirstlane(nvalid) >= ROWS) {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int q = i * NW + wave;
        if (kEven || q < T) dma_x4s<NT>(src, loff[i], lb + q * 1024);
      }
    } else {
      // the lane index is re-read here (volatile, so not hoisted): a
      // register kept across the caller's loop for this rare path would cost
      // more than the two instructions
      int ln;
      asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int q = i * NW + wave;
        if (!kEven && q >= T) continue;
        const int r = q * RPI + ln / CPR;
        const int rr = min(r, nvalid - 1);
        dma_x4s<NT>(src, (uint32_t)(rr * rs + ((ln % CPR) ^ swz<D>(r)) * 8) * 2u, lb + q * 1024);
      }
    }
  }
};

// A operand from a swizzled unpadded tile through two transposing reads, at
// precomputed byte offsets (see tr_operand for the lane mapping).
__device__ __forceinline__ bf16x8 tr_operand_at(const char *lds, uint32_t off_lo,
                                                uint32_t off_hi) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(lds + off_lo));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(lds + off_hi));
  const i16x4 v[2] = {lo, hi};
  return __builtin_bit_cast(bf16x8, v);
}

// Per-lane byte offsets for reading MFMA A operands from a swizzled,
// unpadded tile of D bf16 per row.
//  * row operand (ds_read_b128): tile rows r0 + (lane % 32), r0 % 16 == 0,
//    k step ks (head chunk 2 ks + lane / 32): byte row(r0) + rowk[ks];
//  * transposed operand (two ds_read_b64_tr_b16, see tr_operand): tile rows
//    k0 + ..., k0 % 16 == 0, head columns 32 db + ...: bytes row(k0) +
//    trk[db][0] and row(k0) + trk[db][1] (the second read is 8 rows down).
template <int D>
struct SwzOffsets {
  static constexpr int RB = D * 2;  // bytes per tile row
  uint32_t rowk[D / 16];
  uint32_t trk[D / 32][2];

  __device__ __forceinline__ void init(int lane) {
    const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
      rowk[ks] = (uint32_t)(l32 * RB + (((2 * ks + h) ^ swz<D>(l32)) << 4));
    const int g = lane >> 4, L = lane & 15;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int r = 4 * (g >> 1) + (L >> 2) + 8 * s;
        const int m = 32 * db + 16 * (g & 1) + 4 * (L & 3);
        trk[db][s] = (uint32_t)(r * RB + (((m >> 3) ^ swz<D>(r)) << 4) + (m & 7) * 2);
      }
  }
};

// The same offsets in compact form (3 registers instead of D/16 + D/8):
// since the chunk index of k step ks is 2 ks + h and the d block db adds
// 4 db to the chunk index, both enter the swizzled address only by XOR:
// rowk[ks] = rowb ^ (ks << 5) and trk[db][s] = trb[s] ^ (db << 6) (the XOR
// stays inside one tile row, whose byte offset is a multiple of 2 D).
template <int D>
struct SwzBases {
  uint32_t rowb, trb[2];

  __device__ __forceinline__ void init(int lane) {
    SwzOffsets<D> o;
    o.init(lane);
    rowb = o.rowk[0];
    trb[0] = o.trk[0][0];
    trb[1] = o.trk[0][1];
  }
  __device__ __forceinline__ uint32_t row(int ks) const { return rowb ^ (uint32_t)(ks << 5); }
  __device__ __forceinline__ uint32_t tr(int db, int s) const {
    return trb[s] ^ (uint32_t)(db << 6);
  }
};

// A fixed-order sequence of N MFMA products with compile-time slot indices
// (each callback receives std::integral_constant<int, n>): before product n
// pre(n); product n consumes operand n, which rd(n) read from LDS LA
// products earlier; after it, work(n) (the vector work placed beside it).
// Scheduling barriers between slots pin the order.
template <int n, int N, int LA, class Rd, class Mm, class Pre, class Work>
__device__ __forceinline__ void product_slot(bf16x8 *op, Rd &rd, Mm &mm, Pre &pre, Work &work) {
  pre(std::integral_constant<int, n>{});
  mm(std::integral_constant<int, n>{}, op[n]);
  if constexpr (n + LA < N) op[n + LA] = rd(std::integral_constant<int, n + LA>{});
  work(std::integral_constant<int, n>{});
  __builtin_amdgcn_sched_barrier(0);
}
template <int n, int LA, class Rd>
__device__ __forceinline__ void product_prefetch(bf16x8 *op, Rd &rd) {
  if constexpr (n < LA) op[n] = rd(std::integral_constant<int, n>{});
}
template <int N, int LA, class Rd, class Mm, class Pre, class Work, int... Ns>
__device__ __forceinline__ void product_slots_seq(Rd &rd, Mm &mm, Pre &pre, Work &work,
                                                  std::integer_sequence<int, Ns...>) {
  bf16x8 op[N];
  (product_prefetch<Ns, LA>(op, rd), ...);
  (product_slot<Ns, N, LA>(op, rd, mm, pre, work), ...);
}
template <int N, int LA, class Rd, class Mm, class Pre, class Work>
__device__ __forceinline__ void product_slots(Rd &&rd, Mm &&mm, Pre &&pre, Work &&work) {
  product_slots_seq<N, LA>(rd, mm, pre, work, std::make_integer_sequence<int, N>{});
}

// Work order of (group, tile) items over the 8 XCDs. Consecutive workgroup
// ids go to different XCDs (id % 8). With 8 or more groups, XCD x takes the
// groups x, x + 8, x + 16, ... (so every XCD gets the same mix of dialogues)
// and walks them in chunks of `chunk` groups; inside a chunk the tile index
// runs over its groups innermost, in the order tiles-1 .. 0 (`high_first`,
// row tiles of a causal-like mask, longest first) or 0 .. tiles-1 (key
// tiles). The groups of one chunk keep their K/V (or Q/dO) in the XCD's L2
// while their longest tiles start first, which also keeps the chip's last
// workgroups short. With fewer than 8 groups every XCD takes every 8th item
// of the same order over all groups. Returns false for ids past the end.
#ifndef ISM_SCHED_CHUNK
#define ISM_SCHED_CHUNK 4  // groups per scheduling chunk
#endif
__device__ __forceinline__ bool xcd_work_item(int bid, int groups, int tiles, int chunk,
                                              bool high_first, int &group, int &tile) {
  const int x = bid & 7, i = bid >> 3;
  if (groups < 8) {
    const int j = i * 8 + x;
    if (j >= groups * tiles) return false;
    tile = high_first ? tiles - 1 - j / groups : j / groups;
    group = j % groups;
    return true;
  }
  const int ng = (groups - x + 7) >> 3;  // groups of this XCD
  if (i >= ng * tiles) return false;
  const int ck = i / (chunk * tiles);
  const int c0 = ck * chunk;
  const int ce = min(chunk, ng - c0);
  const int j = i - c0 * tiles;
  tile = high_first ? tiles - 1 - j / ce : j / ce;
  group = (c0 + j % ce) * 8 + x;
  return true;
}

// Grid size for xcd_work_item: 8 x the largest per-XCD item count.
inline int64_t xcd_grid(int64_t groups, int64_t tiles) {
  return groups < 8 ? (groups * tiles + 7) / 8 * 8 : 8 * (((groups + 7) >> 3) * tiles);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) {
  return __builtin_bit_cast(float, w << 16);
}
__device__ __forceinline__ float bf16_hi(uint32_t w) {
  return __builtin_bit_cast(float, w & 0xffff0000u);
}

// ChatGLM-style 2-D rotary positions (kept when ISM is adapted to a
// prefix-style backbone, Sec. 2.3): dims [0, d/2) of a head rotate by the
// token's span position pos1, dims [d/2, d) by its offset position pos2;
// inside a half of width r = d/2, dims k and k + r/2 (k < r/2) form a pair
// rotated by the angle pos * base^(-2k/r). Every path that rotates (the
// in-place kernel, the fused cache append, the forward's query load) uses
// these two functions, so they give identical bf16 results.
// The angle is formed in revolutions (pos * base^(-2k/r) / 2 pi, two fp32
// roundings: a relative error of about 2^-23, as forming the angle in fp32
// radians has), and its fraction goes to the hardware sine / cosine, which
// take revolutions: a few instructions instead of a range-reduced sincosf.
__device__ __forceinline__ void rope_cs(int pos, int k, int r, float log2_base, float &c,
                                        float &s) {
  // 2k / r is exact (r is a power of two)
  const float freq_rev = exp2f(-((float)(2 * k) / (float)r) * log2_base) * 0.159154943091895f;
  const float rev = __builtin_amdgcn_fractf((float)pos * freq_rev);
  s = __builtin_amdgcn_sinf(rev);
  c = __builtin_amdgcn_cosf(rev);
}

// Rotate 8 pairs: dims of chunk a with the dims r/2 further in chunk b (8
// bf16 each), angles given by c[i], s[i] (s negated for the inverse).
__device__ __forceinline__ void rope_rotate8(u32x4 &a, u32x4 &b, const float (&c)[8],
                                             const float (&s)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float x0 = bf16_lo(a[i]), x1 = bf16_hi(a[i]);
    float y0 = bf16_lo(b[i]), y1 = bf16_hi(b[i]);
    const float u0 = fmaf(x0, c[2 * i], -(y0 * s[2 * i]));
    const float v0 = fmaf(x0, s[2 * i], y0 * c[2 * i]);
    const float u1 = fmaf(x1, c[2 * i + 1], -(y1 * s[2 * i + 1]));
    const float v1 = fmaf(x1, s[2 * i + 1], y1 * c[2 * i + 1]);
    a[i] = pack_bf16x2(u0, u1);
    b[i] = pack_bf16x2(v0, v1);
  }
}

}  // namespace ism
