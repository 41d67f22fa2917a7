// Internal declarations shared by the HIP sources of libtriroute (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "triroute.h"

namespace tr {

// ------------------------------------------------------------------ dtypes
typedef uint16_t bf16;  // storage of a bfloat16

__device__ __forceinline__ float bf2f(bf16 v) { return __uint_as_float(uint32_t(v) << 16); }

// Round to nearest even (finite inputs).
__device__ __forceinline__ bf16 f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return bf16(u >> 16);
}

// Two floats -> packed bf16 pair (lo in bits 0..15), round to nearest even
// (one v_cvt_pk_bf16_f32; the same bits as f2bf for finite values).
__device__ __forceinline__ uint32_t pk_bf16(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

template <typename T> struct Act;
template <> struct Act<float> {
  static constexpr int bytes = 4;
  __device__ static float ld(const float *p, int64_t i) { return p[i]; }
  __device__ static float cvt(float v) { return v; }
  __device__ static void st(float *p, int64_t i, float v) { p[i] = v; }
};
template <> struct Act<bf16> {
  static constexpr int bytes = 2;
  __device__ static float ld(const bf16 *p, int64_t i) { return bf2f(p[i]); }
  __device__ static float cvt(bf16 v) { return bf2f(v); }
  __device__ static void st(bf16 *p, int64_t i, float v) { p[i] = f2bf(v); }
};

// 8 consecutive elements <-> fp32 (16-byte bf16 / two 16-byte fp32 accesses;
// the address must be aligned to 8 elements).
__device__ __forceinline__ void load8(const bf16 *p, float *v) {
  const uint4 w = *(const uint4 *)p;
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(u[i] << 16);
    v[2 * i + 1] = __uint_as_float(u[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void load8(const float *p, float *v) {
  const float4 a = *(const float4 *)p, b = *(const float4 *)(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void store8(bf16 *p, const float *v) {
  uint4 w;
  w.x = uint32_t(f2bf(v[0])) | (uint32_t(f2bf(v[1])) << 16);
  w.y = uint32_t(f2bf(v[2])) | (uint32_t(f2bf(v[3])) << 16);
  w.z = uint32_t(f2bf(v[4])) | (uint32_t(f2bf(v[5])) << 16);
  w.w = uint32_t(f2bf(v[6])) | (uint32_t(f2bf(v[7])) << 16);
  *(uint4 *)p = w;
}
__device__ __forceinline__ void store8(float *p, const float *v) {
  *(float4 *)p = make_float4(v[0], v[1], v[2], v[3]);
  *(float4 *)(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

// fp64 -> activation dtype as every tensor handed between operators is
// rounded: to fp32 (RNE), then for bf16 to bf16 (RNE).
__device__ __forceinline__ void store8(bf16 *p, const double *v) {
  float f[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = float(v[i]);
  store8(p, f);
}
__device__ __forceinline__ void store8(float *p, const double *v) {
  float f[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = float(v[i]);
  store8(p, f);
}

// --------------------------------------------------------- wave helpers
constexpr int WAVE = 64;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, WAVE);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, WAVE);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, WAVE));
  return v;
}
// Reductions within aligned lane segments of `seg` lanes (seg a power of 2).
// min / max over aligned segments of `seg` lanes (seg a power of two <= 64,
// wave-uniform).  Segments of 16 or more lanes reduce within 16-lane rows by
// row rotations (DPP) and across rows by row-pair and half-wave swaps, with
// no trip through LDS; smaller segments use lane shuffles.
template <bool MAX>
__device__ __forceinline__ float seg_reduce(float v, int seg) {
  auto op = [](float a, float b) { return MAX ? fmaxf(a, b) : fminf(a, b); };
  if (seg >= 16) {
#define TR_ROR(n) __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0x120 + (n), 0xF, 0xF, false))
    v = op(v, TR_ROR(1));
    v = op(v, TR_ROR(2));
    v = op(v, TR_ROR(4));
    v = op(v, TR_ROR(8));
#undef TR_ROR
    if (seg >= 32) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                      false);
      v = op(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    if (seg >= 64) {
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                      false);
      v = op(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    return v;
  }
  for (int m = seg >> 1; m >= 1; m >>= 1) v = op(v, __shfl_xor(v, m, WAVE));
  return v;
}
__device__ __forceinline__ float seg_min(float v, int seg) { return seg_reduce<false>(v, seg); }
// sum over aligned segments of 16, 32 or 64 lanes (same lane pattern)
__device__ __forceinline__ float seg_sum(float v, int seg) {
#define TR_ROR(n) __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0x120 + (n), 0xF, 0xF, false))
  v += TR_ROR(1);
  v += TR_ROR(2);
  v += TR_ROR(4);
  v += TR_ROR(8);
#undef TR_ROR
  if (seg >= 32) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                    false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  if (seg >= 64) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                    false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  return v;
}
__device__ __forceinline__ float seg_max(float v, int seg) { return seg_reduce<true>(v, seg); }
__device__ __forceinline__ uint64_t lanemask_lt() {
  int l = __lane_id();
  return l ? (~0ull >> (64 - l)) : 0ull;
}

// ------------------------------------------------------- direct-to-LDS loads
// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return uint32_t(uintptr_t((const __attribute__((address_space(3))) void *)p));
}

// One wave-wide direct-to-LDS transfer (global_load_lds_dwordx4): each
// active lane moves the 16 bytes at src to LDS address lds + 16 * lane.
// It is issued from inline assembly so that the compiler does not wait for
// every outstanding transfer before each later LDS read; the caller orders
// the data with wait_vm counts of its own (vector-memory ops complete in
// issue order, so a count that ignores other loads is conservative).
__device__ __forceinline__ void dma16(const void *src, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory", "m0");
}

// The same transfer from a wave-uniform base (scalar registers) plus the
// lane's byte offset voff: no per-lane 64-bit address arithmetic.
__device__ __forceinline__ void dma16_s(const void *sbase, uint32_t voff, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1"
      :
      : "v"(voff), "s"(sbase), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory", "m0");
}

// s_waitcnt vmcnt(N) with the other counters left free (gfx9 encoding:
// vmcnt[3:0] at bits 3:0, vmcnt[5:4] at bits 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// ------------------------------------------------------------ KV cache view
// Bits of the physical store of width index bi (bi = 3 keeps the act dtype).
__host__ __device__ inline int pool_bits(int bi, int act_bytes) {
  return bi == 0 ? 2 : bi == 1 ? 4 : bi == 2 ? 8 : 8 * act_bytes;
}

struct CacheView {
  uint8_t *base;
  int32_t *status, *seq_len, *pool_len, *pos;
  int n_seq, capacity, TS, n_tiles;
  int Hkv, dh, G, act_bytes;
  int64_t off_pool[4], tile_bytes[4];
  // paged caches (PT > 0): pool (s, bi) is a list of pages of PT tiles (all
  // kv heads) taken from width bi's page pool; page j of it is
  // page_table[(s * 4 + bi) * max_pages + j]
  int PT, max_pages;
  int32_t *page_table, *alloc, *free_top;
  int32_t *free_list[4], *pos_pool[4];

  __device__ __forceinline__ int page(int s, int bi, int j) const {
    return page_table[(int64_t(s) * 4 + bi) * max_pages + j];
  }
  // positions of the TS slots of tile t of pool (s, bi) (one int32 per slot)
  __device__ __forceinline__ int32_t *pos_tile(int s, int bi, int t) const {
    if (PT) return pos_pool[bi] + (int64_t(page(s, bi, t / PT)) * PT + t % PT) * TS;
    return pos + ((int64_t(s) * 4 + bi) * n_tiles + t) * TS;
  }
  __device__ __forceinline__ int32_t &pos_at(int s, int bi, int slot) const {
    return pos_tile(s, bi, slot / TS)[slot % TS];
  }
  __device__ __forceinline__ uint8_t *tile(int s, int bi, int g, int t) const {
    if (PT)
      return base + off_pool[bi] +
             ((int64_t(page(s, bi, t / PT)) * Hkv + g) * PT + t % PT) * tile_bytes[bi];
    return base + off_pool[bi] + ((int64_t(s) * Hkv + g) * n_tiles + t) * tile_bytes[bi];
  }
  __device__ __forceinline__ int bits(int bi) const { return pool_bits(bi, act_bytes); }
  // byte offsets inside a tile
  __device__ __forceinline__ int v_codes_off(int bi) const { return 512 * bits(bi); }
  __device__ __forceinline__ int k_sz_off(int bi) const { return 1024 * bits(bi); }
  __device__ __forceinline__ int v_sz_off(int bi) const {
    return 1024 * bits(bi) + TS * (dh / G) * 4;
  }
};

// Element placement inside a 64-lane record (see triroute.h).
// K element (slot st in tile, channel c) -> (lane record, element index q).
__device__ __forceinline__ void k_place(int st, int c, int dh, int &lane, int &q) {
  int KS = dh >> 5;
  int blk = st >> 4, n = st & 15;
  int ks = c >> 5, o = (c >> 3) & 3, j = c & 7;
  lane = o * 16 + n;
  q = (blk * KS + ks) * 8 + j;
}
// V element (slot st in tile, channel c) -> (lane record, element index q).
// Within a 32-slot step, element j of lane group o is slot 16*(j/4) + 4*o + j%4:
// the order in which the K-tile MFMA leaves softmax weights in registers.
__device__ __forceinline__ void v_place(int st, int c, int dh, int &lane, int &q) {
  int CB = dh >> 4;
  int kv = st >> 5, r = st & 31;
  int o = (r >> 2) & 3, j = (r >> 4) * 4 + (r & 3);
  int cb = c >> 4, n = c & 15;
  lane = o * 16 + n;
  q = (kv * CB + cb) * 8 + j;
}
// element index q = 8 f + j of a record of bp bits -> (32-bit word, bit offset).
//   2 bits: word q / 16 holds fields 2w (element j at bit 4 j) and 2w + 1
//           (bit 4 j + 2): masking the word with 0x33333333 leaves one code
//           per nibble, an fp4 (e2m1) number worth code / 2;
//   4 bits: word q / 8 holds field f, element j at bit 8 (j % 4) + 4 (j / 4):
//           masking with 0x0F0F0F0F leaves one code per byte, an fp8 (e4m3)
//           number worth code / 512;
//   8 bits: word q / 4, element q at byte q % 4;
//   16 bits: word q / 2, element q at bit 16 (q % 2);
//   32 bits: one element per word.
__device__ __forceinline__ void q_word(int q, int bp, int &word, int &bit) {
  if (bp == 2) {
    word = q >> 4;
    bit = 4 * (q & 7) + 2 * ((q >> 3) & 1);
  } else if (bp == 4) {
    word = q >> 3;
    bit = 8 * (q & 3) + 4 * ((q >> 2) & 1);
  } else if (bp == 8) {
    word = q >> 2;
    bit = 8 * (q & 3);
  } else if (bp == 16) {
    word = q >> 1;
    bit = 16 * (q & 1);
  } else {
    word = q;
    bit = 0;
  }
}

// ------------------------------------------------------------ launch helpers
CacheView make_view(const triroute_cfg &cfg, const triroute_kv_cache &c);

}  // namespace tr
