// Routed attention over the mixed-width cache on bf16 MFMA (gfx950).
//
// Paper Sec. 3.2 (A): a query head at position P reads kv head h / (H/Hkv):
// skip -> 0, local -> keys [P - w + 1, P], full -> [0, P]; softmax over
// q k^T / sqrt(dh) of the dequantized cache (Sec. 3.2 (C)), times v.
//
// One wave processes 32/64-slot tiles of one width pool at a time:
//   S^T = K Q^T   v_mfma_f32_16x16x32_bf16, A = K codes of 16 slots (bf16 of
//                 128 + code, or the code itself for 8-bit, or the stored bf16),
//                 B = up to 16 query columns (GQA heads of one token in decode,
//                 16 tokens of one head in prefill).  The dequantization is
//                 algebraic: per group, s * (acc - off * sum q) + z * sum q.
//   O += P' V     A = P' = fp16(p * s_v) straight from the S^T registers (the
//                 cache stores V in the order that makes this a register
//                 reuse), B = fp16 codes (v_mfma_f32_16x16x32_f16);
//                 the z_v and offset terms are accumulated per query column
//                 and added at the end.  The 16-bit pool multiplies bf16(p)
//                 by the stored bf16 values.
// Online softmax in the exp2 domain.  Decode runs one 8-wave block per
// (sequence, kv head, chunk); each wave streams its share of every pool's
// whole tiles through a private LDS byte FIFO with direct-to-LDS loads issued
// as far ahead as the FIFO allows; the waves merge in LDS and, when a
// sequence is split into chunks, a last kernel merges them with log-sum-exp.
#include <limits.h>

#include <type_traits>

#include "kernels.hpp"

namespace tr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float LOG2E = 1.4426950408889634f;

// Max over the lanes n, n ^ 16, n ^ 32, n ^ 48 (row-pair and half-wave swaps).
__device__ __forceinline__ float max_rows(float x) {
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
  x = fmaxf(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
  return fmaxf(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
}

// Sum over the lanes n, n ^ 16, n ^ 32, n ^ 48 (row-pair and half-wave swaps).
__device__ __forceinline__ float sum_rows(float x) {
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
  x = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
  return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

__device__ __forceinline__ bf16x8 as_op(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ f16x8 as_h(u32x4 v) { return __builtin_bit_cast(f16x8, v); }

// Code fields -> MFMA operands.
//
// 2- and 4-bit fields are laid out so that one mask turns a word into small
// floats of the gfx950 conversion instructions: a 2-bit code sits alone in a
// nibble (fp4 e2m1: code / 2), a 4-bit code alone in a byte (fp8 e4m3:
// code / 512; codes below 16 are the linear subnormal and first normal
// range).  The scaled conversions (power-of-two scale 2 or 512) then give
// the codes themselves as exact fp16 / bf16 pairs, two per instruction.
//
// An 8-bit code c becomes fp16 1024 + c as the 16-bit pattern [c, 0x64]
// (low byte first) by one byte permute (v_perm_b32) per pair; the packed
// fp16 subtraction of 1024 is exact.  Selectors: result bytes 0..3 take
// bytes (0|2, 4, 1|3, 4) of (codes, constant): 0x04010400 pairs bytes 0 and
// 1, 0x04030402 bytes 2 and 3.
constexpr uint32_t SEL01 = 0x04010400u, SEL23 = 0x04030402u;
constexpr uint32_t F16_1024 = 0x64646464u;

// the 32 bits of a packed pair returned by a conversion builtin
template <class V>
__device__ __forceinline__ uint32_t u32_of(V v) {
  static_assert(sizeof(V) == 4, "a packed pair of 16-bit values");
  return __builtin_bit_cast(uint32_t, v);
}

// field f of a 2-bit record: its eight codes, one per nibble
__device__ __forceinline__ uint32_t nibbles2(const uint32_t *w, int f) {
  const uint32_t x = w[f >> 1];
  return ((f & 1) ? x >> 2 : x) & 0x33333333u;
}

// V field of a quantized pool -> fp16 operand holding the codes themselves.
// (A constant left in the operand would be summed over the whole key range
// in the fp32 accumulator.)
template <int BP>
__device__ __forceinline__ f16x8 vfield_h(const uint32_t *w, int f) {
  u32x4 r;
  if constexpr (BP == 2) {
    const uint32_t y = nibbles2(w, f);
    r[0] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(y, 2.f, 0));
    r[1] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(y, 2.f, 1));
    r[2] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(y, 2.f, 2));
    r[3] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(y, 2.f, 3));
    return as_h(r);
  } else if constexpr (BP == 4) {
    const uint32_t lo = w[f] & 0x0F0F0F0Fu, hi = (w[f] >> 4) & 0x0F0F0F0Fu;
    r[0] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(lo, 512.f, false));
    r[1] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(lo, 512.f, true));
    r[2] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(hi, 512.f, false));
    r[3] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_f16_fp8(hi, 512.f, true));
    return as_h(r);
  } else {
#pragma unroll
    for (int p = 0; p < 4; ++p)
      r[p] = __builtin_amdgcn_perm(F16_1024, w[2 * f + (p >> 1)], (p & 1) ? SEL23 : SEL01);
    const f16x8 k1024 = {1024, 1024, 1024, 1024, 1024, 1024, 1024, 1024};
    return as_h(r) - k1024;
  }
}

// K field -> bf16 operand of S^T = K Q^T: the codes themselves (2, 4 and 8
// bits), or the stored values (16 bits).
template <int BP>
__device__ __forceinline__ u32x4 kfield(const uint32_t *w, int f) {
  u32x4 r;
  if constexpr (BP == 2) {
    const uint32_t y = nibbles2(w, f);
    r[0] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(y, 2.f, 0));
    r[1] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(y, 2.f, 1));
    r[2] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(y, 2.f, 2));
    r[3] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(y, 2.f, 3));
  } else if constexpr (BP == 4) {
    const uint32_t lo = w[f] & 0x0F0F0F0Fu, hi = (w[f] >> 4) & 0x0F0F0F0Fu;
    r[0] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 512.f, false));
    r[1] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 512.f, true));
    r[2] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 512.f, false));
    r[3] = u32_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 512.f, true));
  } else if constexpr (BP == 8) {
    // byte -> fp32 (exact), whose upper half is the exact bf16
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t x = w[2 * f + (p >> 1)];
      const float lo = float((x >> (16 * (p & 1))) & 0xFFu);
      const float hi = float((x >> (16 * (p & 1) + 8)) & 0xFFu);
      r[p] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int p = 0; p < 4; ++p) r[p] = w[4 * f + p];
  }
  return r;
}

// 16-bit pool V field: the stored bf16 values.
__device__ __forceinline__ bf16x8 field16(const uint32_t *w, int f) {
  u32x4 r;
#pragma unroll
  for (int p = 0; p < 4; ++p) r[p] = w[4 * f + p];
  return as_op(r);
}

// One K-field product into acc.
template <int BP>
__device__ __forceinline__ f32x4 kmfma(const uint32_t *w, int f, const bf16x8 &q, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_op(kfield<BP>(w, f)), q, acc, 0, 0, 0);
}

template <int BP> struct PoolTraits {
  static constexpr int WORDS = 2 * BP;               // 32-bit words per lane record
  static constexpr bool QUANT = BP < 16;
};

template <int DH> struct Geo {
  static constexpr int TS = 4096 / DH;  // slots per tile
  static constexpr int NB = TS / 16;    // 16-slot blocks per tile
  static constexpr int KS = DH / 32;    // 32-channel k-steps
  static constexpr int CB = DH / 16;    // 16-channel output blocks
  static constexpr int KV = TS / 32;    // 32-slot steps of the P V product
};

// Per-wave running state of the online softmax for 16 query columns.
template <int DH>
struct SoftState {
  float m;               // running max (log2 domain) of column n16
  float l;               // partial denominator of column n16 (this lane's slots)
  float zc[DH / 32];     // partial per-group additive term of column n16
  f32x4 O[DH / 16];      // rows = columns 4*o4 + i, cols = channel n16 + 16 cb
};

// The running max starts at a large finite negative value instead of -inf,
// so that exp2(score - m) of a masked score (-inf) is 0 without a test; a
// column that sees no key keeps l = 0 and yields a zero output.
constexpr float M0 = -1.0e30f;

template <int DH>
__device__ __forceinline__ void state_init(SoftState<DH> &st) {
  st.m = M0;
  st.l = 0.f;
#pragma unroll
  for (int g = 0; g < DH / 32; ++g) st.zc[g] = 0.f;
#pragma unroll
  for (int c = 0; c < DH / 16; ++c) st.O[c] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// Column description: the lane's column n16 takes keys with
// key_lo <= key <= key_hi (slot indices in decode, positions in prefill).
struct ColMask {
  int lo, hi;  // inclusive bounds; lo > hi disables the column
};

// Everything one lane needs of a tile, loaded together so that a tile costs
// one memory round trip (and narrow pools prefetch the next tile): the K and
// V lane records, the fp16 scale/zero words of the lane's slots, and, when
// keys are compared by position, the positions of the lane's slots.
template <int DH, int BP, int G, bool POS>
struct TileRegs {
  using Gm = Geo<DH>;
  static constexpr int NG = DH / G;
  static constexpr int W = PoolTraits<BP>::WORDS;
  static constexpr bool Q = PoolTraits<BP>::QUANT;
  union {
    u32x4 v[W / 4];
    uint32_t w[W];
  } k, v;
  uint32_t ksz[Q ? Gm::NB : 1][4 * NG];        // [block][slot i * NG + g]
  uint32_t vsz[Q ? Gm::KV : 1][2][4 * NG];     // [step][half][slot i * NG + g]
  int key[POS ? Gm::NB : 1][4];                // key positions (INT_MAX past klen)
  int kfirst, klast;  // POS: positions of the tile's first and last slot (klast: INT_MAX if
                      // the tile runs past the pool length)

  // tp: the tile; kpos: positions of the tile's slots (POS only); slot0:
  // pool slot of the tile's first slot; klen: pool length.

  __device__ __forceinline__ void load(const uint8_t *tp, const CacheView &cv, int bi,
                                       int slot0, const int32_t *kpos, int klen) {
    const int lane = threadIdx.x & 63, o4 = lane >> 4;
    const u32x4 *kp = (const u32x4 *)(tp + lane * 8 * BP);
    const u32x4 *vp = (const u32x4 *)(tp + 512 * BP + lane * 8 * BP);
#pragma unroll
    for (int x = 0; x < W / 4; ++x) {
      k.v[x] = kp[x];
      v.v[x] = vp[x];
    }
    if constexpr (Q) {
      const u32x4 *ks = (const u32x4 *)(tp + cv.k_sz_off(bi));
      const u32x4 *vs = (const u32x4 *)(tp + cv.v_sz_off(bi));
#pragma unroll
      for (int blk = 0; blk < Gm::NB; ++blk)
#pragma unroll
        for (int x = 0; x < NG; ++x) {
          const u32x4 t = ks[((blk * 16 + 4 * o4) * NG) / 4 + x];
#pragma unroll
          for (int y = 0; y < 4; ++y) ksz[blk][4 * x + y] = t[y];
        }
#pragma unroll
      for (int kv = 0; kv < Gm::KV; ++kv)
#pragma unroll
        for (int hb = 0; hb < 2; ++hb)
#pragma unroll
          for (int x = 0; x < NG; ++x) {
            const u32x4 t = vs[((32 * kv + 16 * hb + 4 * o4) * NG) / 4 + x];
#pragma unroll
            for (int y = 0; y < 4; ++y) vsz[kv][hb][4 * x + y] = t[y];
          }
    }
    if constexpr (POS) {
      kfirst = kpos[0];
      klast = slot0 + Gm::TS <= klen ? kpos[Gm::TS - 1] : INT_MAX;
#pragma unroll
      for (int blk = 0; blk < Gm::NB; ++blk)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = blk * 16 + 4 * o4 + i;
          // slots past the pool length hold no token
          key[blk][i] = slot0 + r < klen ? kpos[r] : INT_MAX;
        }
    }
  }
};

__device__ __forceinline__ void unpack_sz(uint32_t szw, float &S, float &Z) {
  const uint16_t sb = uint16_t(szw), zb = uint16_t(szw >> 16);
  S = float(*(const _Float16 *)&sb);
  Z = float(*(const _Float16 *)&zb);
}

// Process one tile of width BP, one 32-slot step at a time: S^T for two
// 16-slot blocks, the online-softmax update, then O += P' V for the step.
// `slot0` = pool slot index of the tile's first slot.  Keys are compared
// with the column's bounds by position (POS) or by slot index.
template <int DH, int BP, int G, bool POS>
__device__ __forceinline__ void process_tile(SoftState<DH> &st,
                                             const TileRegs<DH, BP, G, POS> &tr, int slot0,
                                             ColMask cm, const bf16x8 *qop, const float *qsum,
                                             float scale2) {
  using Gm = Geo<DH>;
  using PT = PoolTraits<BP>;
  constexpr int NG = DH / G;    // groups per head vector
  constexpr int gks = G / 32;   // k-steps per group
  const int lane = threadIdx.x & 63, o4 = lane >> 4;
#pragma unroll
  for (int kv = 0; kv < Gm::KV; ++kv) {
    float p[2][4];
    // ---- S^T = K Q^T for blocks 2 kv, 2 kv + 1, dequantized per group
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      const int blk = 2 * kv + hb;
      f32x4 acc[NG];
#pragma unroll
      for (int g = 0; g < NG; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < Gm::KS; ++ks) {
        acc[ks / gks] = kmfma<BP>(tr.k.w, blk * Gm::KS + ks, qop[ks], acc[ks / gks]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float sv = 0.f;
        if constexpr (PT::QUANT) {
#pragma unroll
          for (int g = 0; g < NG; ++g) {
            float S, Z;
            unpack_sz(tr.ksz[blk][i * NG + g], S, Z);
            sv = fmaf(S, acc[g][i], sv);
            sv = fmaf(Z, qsum[g], sv);
          }
        } else {
#pragma unroll
          for (int g = 0; g < NG; ++g) sv += acc[g][i];
        }
        p[hb][i] = sv * scale2;
      }
    }
    // keys outside the column's range: per-key tests only when some lane's
    // range cuts through the tile
    {
      int first, last;
      if constexpr (POS) {
        first = tr.kfirst;
        last = tr.klast;
      } else {
        first = slot0;
        last = slot0 + Gm::TS - 1;
      }
      const bool none = cm.lo > cm.hi || last < cm.lo || first > cm.hi;
      const bool all = first >= cm.lo && last <= cm.hi;
      if (!__builtin_amdgcn_ballot_w64(!none && !all)) {
        if (__builtin_amdgcn_ballot_w64(none)) {
#pragma unroll
          for (int hb = 0; hb < 2; ++hb)
#pragma unroll
            for (int i = 0; i < 4; ++i) p[hb][i] = none ? -INFINITY : p[hb][i];
        }
      } else {
#pragma unroll
        for (int hb = 0; hb < 2; ++hb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            int key;
            if constexpr (POS)
              key = tr.key[2 * kv + hb][i];
            else
              key = slot0 + (2 * kv + hb) * 16 + 4 * o4 + i;
            p[hb][i] = (key >= cm.lo && key <= cm.hi) ? p[hb][i] : -INFINITY;
          }
      }
    }
    // ---- online softmax for this lane's column (lanes n16 + 16 k); the
    // output rows are rescaled only when some column's running max grows
    float mt = fmaxf(fmaxf(fmaxf(p[0][0], p[0][1]), fmaxf(p[0][2], p[0][3])),
                     fmaxf(fmaxf(p[1][0], p[1][1]), fmaxf(p[1][2], p[1][3])));
    mt = max_rows(mt);
    if (__builtin_amdgcn_ballot_w64(mt > st.m)) {
      const float mnew = fmaxf(st.m, mt);
      const float corr = __builtin_amdgcn_exp2f(st.m - mnew);
      st.l *= corr;
#pragma unroll
      for (int g = 0; g < NG; ++g) st.zc[g] *= corr;
      st.m = mnew;
      // column 4 o4 + i lives in lane 4 o4 + i
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float ci = __shfl(corr, 4 * o4 + i, 64);
#pragma unroll
        for (int cb = 0; cb < Gm::CB; ++cb) st.O[cb][i] *= ci;
      }
    }
    float ps = 0.f;
#pragma unroll
    for (int hb = 0; hb < 2; ++hb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[hb][i] = __builtin_amdgcn_exp2f(p[hb][i] - st.m);
        ps += p[hb][i];
      }
    st.l += ps;
    // ---- O += P' V.  Quantized pools: P' = fp16(p * s_v) against fp16
    // codes; the 16-bit pool: P = bf16(p) against the stored bf16.
    u32x4 pk[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
#pragma unroll
      for (int jp = 0; jp < 4; ++jp) {
        uint32_t h2[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int j = 2 * jp + h;
          const float pp = p[j >> 2][j & 3];
          if constexpr (PT::QUANT) {
            float S, Z;
            unpack_sz(tr.vsz[kv][j >> 2][(j & 3) * NG + g], S, Z);
            const _Float16 ph = (_Float16)(pp * S);
            st.zc[g] = fmaf(pp, Z, st.zc[g]);
            h2[h] = uint32_t(*(const uint16_t *)&ph);
          } else {
            h2[h] = uint32_t(f2bf(pp));
          }
        }
        pk[g][jp] = h2[0] | (h2[1] << 16);
      }
    }
#pragma unroll
    for (int cb = 0; cb < Gm::CB; ++cb) {
      const int g = (16 * cb) / G;
      if constexpr (PT::QUANT) {
        const f16x8 bv = vfield_h<BP>(tr.v.w, kv * Gm::CB + cb);
        st.O[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h(pk[g]), bv, st.O[cb], 0, 0, 0);
      } else {
        const bf16x8 bv = field16(tr.v.w, kv * Gm::CB + cb);
        st.O[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_op(pk[g]), bv, st.O[cb], 0, 0, 0);
      }
    }
  }
}

// First index in [0, len) with pos[index] >= p (pos ascending), searched by
// the whole wave: each round probes 64 evenly spaced entries and narrows the
// range 64-fold, so a 32k-entry pool takes two rounds of parallel loads.
// Must be called by all 64 lanes with wave-uniform arguments.
__device__ __forceinline__ int lower_bound_pos(const CacheView &cv, int s, int bi, int len, int p) {
  const int lane = threadIdx.x & 63;
  int lo = 0, hi = len;  // the answer lies in [lo, hi]
  while (hi - lo > 64) {
    const int span = hi - lo;
    const int idx = lo + int(int64_t(span) * (lane + 1) / 64) - 1;
    const uint64_t below = __ballot(cv.pos_at(s, bi, idx) < p);
    const int c = __popcll(below);  // probes 0 .. c-1 lie below p
    const int nlo = c > 0 ? lo + int(int64_t(span) * c / 64) : lo;
    const int nhi = c < 64 ? lo + int(int64_t(span) * (c + 1) / 64) - 1 : hi;
    lo = nlo;
    hi = nhi;
  }
  const int idx = lo + lane;
  const uint64_t below = __ballot(idx < hi && cv.pos_at(s, bi, idx) < p);
  return lo + __popcll(below);
}

// The query operand of column n16 (a row of q, bf16, zero when !valid) and
// its per-group sums, from the raw 16-byte pieces loaded by the caller.
template <int DH, int G>
__device__ __forceinline__ void q_operand(const u32x4 *raw, bool valid, bf16x8 *qop, float *qsum) {
  constexpr int gks = G / 32;
#pragma unroll
  for (int g = 0; g < DH / G; ++g) qsum[g] = 0.f;
#pragma unroll
  for (int ks = 0; ks < DH / 32; ++ks) {
    const u32x4 zero = {0u, 0u, 0u, 0u};
    const u32x4 v = valid ? raw[ks] : zero;
    qop[ks] = as_op(v);
    float sum = 0.f;
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      sum += __uint_as_float(v[y] << 16) + __uint_as_float(v[y] & 0xFFFF0000u);
    }
    qsum[ks / gks] += sum;
  }
#pragma unroll
  for (int g = 0; g < DH / G; ++g) qsum[g] = sum_rows(qsum[g]);
}

// Load the query operand of column n16 (a row of q, bf16) and per-group sums.
template <int DH, int G>
__device__ __forceinline__ void load_q(const bf16 *qrow, bool valid, bf16x8 *qop, float *qsum) {
  const int lane = threadIdx.x & 63, o4 = lane >> 4;
  constexpr int gks = G / 32;
#pragma unroll
  for (int g = 0; g < DH / G; ++g) qsum[g] = 0.f;
#pragma unroll
  for (int ks = 0; ks < DH / 32; ++ks) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (valid) v = *(const u32x4 *)(qrow + 32 * ks + 8 * o4);
    qop[ks] = as_op(v);
    float sum = 0.f;
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      sum += __uint_as_float(v[y] << 16) + __uint_as_float(v[y] & 0xFFFF0000u);
    }
    qsum[ks / gks] += sum;
  }
#pragma unroll
  for (int g = 0; g < DH / G; ++g) {
    qsum[g] += __shfl_xor(qsum[g], 16, 64);
    qsum[g] += __shfl_xor(qsum[g], 32, 64);
  }
}

// Reduce the per-lane partials of every column over the 4 lane groups and
// fold the additive terms into O.  Afterwards lane (0, n) holds in O[cb][i]
// the un-normalised output of column i, channel n + 16 cb; m and l are the
// column's (lane n16 = column).
template <int DH, int G>
__device__ __forceinline__ void state_finish(SoftState<DH> &st) {
  constexpr int NG = DH / G;
  const int lane = threadIdx.x & 63, o4 = lane >> 4;
  st.l += __shfl_xor(st.l, 16, 64);
  st.l += __shfl_xor(st.l, 32, 64);
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    st.zc[g] += __shfl_xor(st.zc[g], 16, 64);
    st.zc[g] += __shfl_xor(st.zc[g], 32, 64);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int col = 4 * o4 + i;
#pragma unroll
    for (int cb = 0; cb < DH / 16; ++cb) {
      const int g = (16 * cb) / G;
      st.O[cb][i] += __shfl(st.zc[g], col, 64);
    }
  }
}

// ------------------------------------------------------------------ decode
struct DecodeArgs {
  CacheView cv;
  const bf16 *q;
  const uint8_t *mode;
  const int32_t *seq_ids;
  float *part;  // [B*H][NS][DH + 2]: m, l, O (NS > 1)
  bf16 *o;      // [B][H][DH] (NS == 1)
  int B, H, R, w, NS;
  float scale2;
};

// Decode streams every pool's tiles through a per-wave LDS ring used as a
// byte FIFO: tiles of different widths are placed back to back (wrapping to
// the ring start when one does not fit before the end), and the wave keeps
// issuing tiles, across pool boundaries, for as long as free ring space
// allows.  The block's 8 rings plus a few words fill the 160 KB of LDS.
constexpr int DEC_WAVES = 8;
// Relative cost of a tile of width index bi in the wave split (bytes moved
// plus dequantisation work, 2 / 4 / 8 / 16 bits).
__device__ constexpr int DEC_COST[4] = {4, 6, 9, 13};
constexpr int DEC_RING = 20 * 1024 - 32;

// Per pool width index bi (2, 4, 8, 16 bits): tile bytes (codes + fp16
// scale/zero), 1 KB wave transfers per tile, ring footprint.
template <int DH, int G>
struct StreamGeo {
  static constexpr int TS = 4096 / DH;
  static constexpr int NG = DH / G;
  __device__ static constexpr int tb(int bi) {
    return 1024 * (2 << bi) + (bi < 3 ? 2 * TS * NG * 4 : 0);
  }
  __device__ static constexpr int ni(int bi) { return (tb(bi) + 1023) / 1024; }
  __device__ static constexpr int foot(int bi) { return (tb(bi) + 255) & ~255; }
  static_assert(((1024 * 16 + 255) & ~255) <= DEC_RING, "a 16-bit tile fits the ring");
};

// s_waitcnt vmcnt(n) for a run-time n, rounded down to a value the tree
// covers (waiting for fewer outstanding transfers is always safe): exact
// below 4, then multiples of 4 up to 24, then multiples of 8 up to 56.
__device__ __forceinline__ void wait_vm_le(int n) {
  if (n >= 12) {
    if (n >= 20) {
      if (n >= 40) {
        if (n >= 56) wait_vm<56>(); else if (n >= 48) wait_vm<48>(); else wait_vm<40>();
      } else if (n >= 24) {
        if (n >= 32) wait_vm<32>(); else wait_vm<24>();
      } else {
        wait_vm<20>();
      }
    } else {
      if (n >= 16) wait_vm<16>(); else wait_vm<12>();
    }
  } else if (n >= 4) {
    if (n >= 8) wait_vm<8>(); else wait_vm<4>();
  } else if (n >= 2) {
    if (n >= 3) wait_vm<3>(); else wait_vm<2>();
  } else {
    if (n >= 1) wait_vm<1>(); else wait_vm<0>();
  }
}

// Copy one whole tile (codes + scale/zero, contiguous in HBM) to LDS address
// dst with direct-to-LDS loads: each lane moves 16 bytes per 1 KB transfer;
// lanes past the tile end sit out the last transfer.
__device__ __forceinline__ void tile_to_lds(const uint8_t *src, uint32_t dst, int tb, int ni) {
  const int lane = threadIdx.x & 63;
  for (int j = 0; j < ni; ++j) {
    const int off = j * 1024 + lane * 16;
    if (off < tb) dma16(src + off, dst + j * 1024);
  }
}

// tile_to_lds for a tile of pool BI (size known at compile time) from a
// wave-uniform address: the transfers are unrolled, only the last one can be
// partial.
template <int DH, int G, int BI>
__device__ __forceinline__ void issue_tile(const uint8_t *src, uint32_t dst) {
  constexpr int TB = StreamGeo<DH, G>::tb(BI), NI = StreamGeo<DH, G>::ni(BI);
  const uint32_t off = (threadIdx.x & 63) * 16;
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    if ((j + 1) * 1024 <= TB || off < uint32_t(TB - j * 1024))
      dma16_s(src + j * 1024, off, dst + j * 1024);
  }
}

// 4 wave-uniform ints picked by a run-time index without a private array.
struct Int4 {
  int v0, v1, v2, v3;
  __device__ __forceinline__ int operator[](int i) const {
    return i == 0 ? v0 : i == 1 ? v1 : i == 2 ? v2 : v3;
  }
  __device__ __forceinline__ void set(int i, int x) {
    if (i == 0) v0 = x; else if (i == 1) v1 = x; else if (i == 2) v2 = x; else v3 = x;
  }
};

// Stream this wave's tiles [w0[bi], w1[bi]) of the four pools, pools in
// order, through its LDS ring (RING bytes at rptr / LDS address rbase) used
// as a byte FIFO: tiles are placed back to back, wrapping to the ring start
// when one does not fit before the end, and the wave keeps issuing tiles,
// across pool boundaries, while free space allows.  With POS each tile is
// followed in the ring by the key positions of its TS slots (int32).  The
// consumer walks the pools in the same order with the pool index known at
// compile time: each resident tile goes to fold(BI, t, lds_pointer), BI an
// std::integral_constant.  On entry no other vector-memory load of the wave
// may be in flight.
template <int DH, int G, int RING = DEC_RING, bool POS = false, class Fold>
__device__ __forceinline__ void stream_tiles(const CacheView &cv, int s, int g, Int4 w0, Int4 w1,
                                             const uint8_t *rptr, uint32_t rbase, Fold &&fold) {
  using SG = StreamGeo<DH, G>;
  constexpr int PB = POS ? 4 * SG::TS : 0;  // position bytes behind a tile
  static_assert(((1024 * 16 + PB + 255) & ~255) <= RING, "a 16-bit tile fits the ring");
  // The producer walks the concatenation of the four ranges with one index
  // kp; pool and tile follow from the range ends without branches.
  const int e1 = w1[0] - w0[0], e2 = e1 + w1[1] - w0[1], e3 = e2 + w1[2] - w0[2];
  const int ktot = e3 + w1[3] - w0[3];
  const int d0 = w0[0], d1 = w0[1] - e1, d2 = w0[2] - e2, d3 = w0[3] - e3;
  int kp = 0;
  int phead = 0, pfree = 0;  // ring end of the newest tile; start of the oldest resident tile
  int nin = 0, issued = 0, consumed = 0;  // tiles resident or in flight; transfers out / used
  int chead = 0;                          // ring end of the last consumed tile
  auto produce = [&]() {
    while (kp < ktot) {
      const int pb = (kp >= e1) + (kp >= e2) + (kp >= e3);
      const int tb = (1024 << (pb + 1)) + (pb < 3 ? SG::tb(0) - 2048 : 0);
      const int sz = (tb + PB + 255) & ~255;
      const int pos = phead + sz <= RING ? phead : 0;
      bool ok = true;
      if (nin > 0) {
        if (pfree < phead)
          ok = pos == phead || sz <= pfree;
        else
          ok = pos == phead && phead + sz <= pfree;
      }
      if (!ok) break;
      const int pt = kp + (pb == 0 ? d0 : pb == 1 ? d1 : pb == 2 ? d2 : d3);
      switch (pb) {
        case 0: issue_tile<DH, G, 0>(cv.tile(s, 0, g, pt), rbase + pos); break;
        case 1: issue_tile<DH, G, 1>(cv.tile(s, 1, g, pt), rbase + pos); break;
        case 2: issue_tile<DH, G, 2>(cv.tile(s, 2, g, pt), rbase + pos); break;
        default: issue_tile<DH, G, 3>(cv.tile(s, 3, g, pt), rbase + pos); break;
      }
      if constexpr (POS) {
        if ((threadIdx.x & 63) < SG::TS / 4)
          dma16(cv.pos_tile(s, pb, pt) + 4 * (threadIdx.x & 63), rbase + pos + tb);
      }
      phead = pos + sz;
      issued += ((tb + 1023) >> 10) + (POS ? 1 : 0);
      ++nin;
      ++kp;
    }
  };
  auto pool = [&](auto BI) {
    constexpr int bi = decltype(BI)::value;
    constexpr int sz = (SG::tb(bi) + PB + 255) & ~255;
    const int t1 = w1[bi];
    for (int t = w0[bi]; t < t1; ++t) {
      produce();
      const int cpos = chead + sz <= RING ? chead : 0;  // the producer's placement rule
      consumed += SG::ni(bi) + (POS ? 1 : 0);
      wait_vm_le(issued - consumed);
      fold(BI, t, rptr + cpos);
      chead = cpos + sz;
      --nin;
      pfree = chead;  // oldest resident tile now starts where this one ended (or the ring wraps)
    }
  };
  pool(std::integral_constant<int, 0>{});
  pool(std::integral_constant<int, 1>{});
  pool(std::integral_constant<int, 2>{});
  pool(std::integral_constant<int, 3>{});
}

// Max over the lanes n16 = h, h + 4, h + 8, h + 12 of each 16-lane row
// (row rotations by 4 and 8), then over the four rows (row-pair and
// half-wave swaps): afterwards every lane holds the maximum over all lanes
// with its lane % 4.
__device__ __forceinline__ float max_lane_mod4(float x) {
  x = fmaxf(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), 0x124, 0xF,
                                                            0xF, false)));
  x = fmaxf(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), 0x128, 0xF,
                                                            0xF, false)));
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
  x = fmaxf(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
  return fmaxf(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
}

// ---- decode with head-packed columns (at most 4 query heads per kv head)
//
// The 16 columns of the S^T = K Q^T product are 4 groups of 4 heads; group
// c multiplies key block c of the tile (its Q operand is zero in the other
// groups' columns), so one accumulator holds every score of the tile with no
// idle column: lane (o4, n16) has head n16 % 4 against slots
// 16 (n16 / 4) + 4 o4 + i.  The softmax state is kept per head (a max over
// the lanes of one head), and P V runs with these 16 "virtual columns" (head,
// key block) as rows: the lane's own probabilities are already in the A
// operand order of the V layout, zero outside its block.  The virtual rows
// of a head are summed once at the end.
//
// The running max starts at M0 (see state_init).

template <int DH>
struct DecState {
  float m;             // running max (log2 domain) of the lane's head
  float l;             // partial denominator (this lane's keys)
  float zc[DH / 32];   // partial additive term per channel group
  f32x4 O[DH / 16];    // rows: virtual columns (key block o4, head i); cols: channel n16 + 16 cb
};

template <int DH>
__device__ __forceinline__ void dec_init(DecState<DH> &st) {
  st.m = M0;
  st.l = 0.f;
#pragma unroll
  for (int g = 0; g < DH / 32; ++g) st.zc[g] = 0.f;
#pragma unroll
  for (int c = 0; c < DH / 16; ++c) st.O[c] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// A tile's K / V lane records and the scale/zero words of the lane's 4 slots.
template <int DH, int BP, int G>
struct DecRegs {
  using Gm = Geo<DH>;
  static constexpr int NG = DH / G;
  static constexpr int W = PoolTraits<BP>::WORDS;
  static constexpr bool Q = PoolTraits<BP>::QUANT;
  union {
    u32x4 v[W / 4];
    uint32_t w[W];
  } k, v;
  uint32_t ksz[Q ? 4 * NG : 1], vsz[Q ? 4 * NG : 1];  // [slot i * NG + g]

  __device__ __forceinline__ void load(const uint8_t *tp, const CacheView &cv, int bi) {
    const int lane = threadIdx.x & 63, o4 = lane >> 4;
    const int blk = min((lane & 15) >> 2, Gm::NB - 1);
    const u32x4 *kp = (const u32x4 *)(tp + lane * 8 * BP);
    const u32x4 *vp = (const u32x4 *)(tp + 512 * BP + lane * 8 * BP);
#pragma unroll
    for (int x = 0; x < W / 4; ++x) {
      k.v[x] = kp[x];
      v.v[x] = vp[x];
    }
    if constexpr (Q) {
      const int st0 = 16 * blk + 4 * o4;
      const u32x4 *ks = (const u32x4 *)(tp + cv.k_sz_off(bi) + st0 * NG * 4);
      const u32x4 *vs = (const u32x4 *)(tp + cv.v_sz_off(bi) + st0 * NG * 4);
#pragma unroll
      for (int x = 0; x < NG; ++x) {
        const u32x4 a = ks[x], b = vs[x];
#pragma unroll
        for (int y = 0; y < 4; ++y) {
          ksz[4 * x + y] = a[y];
          vsz[4 * x + y] = b[y];
        }
      }
    }
  }
};

// Key bounds of the lane's head in one pool, relative to a tile: slot
// 16 c + 4 o4 + i of the tile is a key of the head when lo <= it <= hi.
struct TileMask {
  int lo, hi;
};

// Fold one tile: S^T for its key blocks, the online-softmax update (the
// output rows are rescaled only when some head's running max grows), then
// O += P' V.  `dead`: the lane's key block lies past the tile (d_h 128 has
// two 16-slot blocks per tile, so columns of blocks 2 and 3 are idle).
template <int DH, int BP, int G>
__device__ __forceinline__ void fold_dec(DecState<DH> &st, const DecRegs<DH, BP, G> &tr,
                                         TileMask tm, bool dead, const bf16x8 *qopm,
                                         const float *qsum, float scale2) {
  using Gm = Geo<DH>;
  using PT = PoolTraits<BP>;
  constexpr int NG = DH / G;
  constexpr int gks = G / 32;
  const int lane = threadIdx.x & 63, o4 = lane >> 4, c = (lane & 15) >> 2;
  // ---- scores of the lane's head against slots 16 c + 4 o4 + i
  f32x4 acc[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int blk = 0; blk < Gm::NB; ++blk)
#pragma unroll
    for (int ks = 0; ks < Gm::KS; ++ks)
      acc[ks / gks] = kmfma<BP>(tr.k.w, blk * Gm::KS + ks, qopm[blk * Gm::KS + ks], acc[ks / gks]);
  float p[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float sv = 0.f;
    if constexpr (PT::QUANT) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        float S, Z;
        unpack_sz(tr.ksz[i * NG + g], S, Z);
        sv = fmaf(S, acc[g][i], sv);
        sv = fmaf(Z, qsum[g], sv);
      }
    } else {
#pragma unroll
      for (int g = 0; g < NG; ++g) sv += acc[g][i];
    }
    p[i] = sv * scale2;
  }
  // keys outside the head's range.  Per lane the tile holds all, none or
  // part of the head's keys; the per-key test runs only when some lane has
  // a part (a tile with a window start or the pool's end).
  const int k0 = 16 * c + 4 * o4;
  const bool none = dead || tm.hi < 0 || tm.lo > Gm::TS - 1 || tm.lo > tm.hi;
  const bool all = tm.lo <= 0 && tm.hi >= Gm::TS - 1;
  if (!__builtin_amdgcn_ballot_w64(!none && !all)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = none ? -INFINITY : p[i];
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      p[i] = (!dead && k0 + i >= tm.lo && k0 + i <= tm.hi) ? p[i] : -INFINITY;
  }
  // ---- online softmax per head (lanes of one head: equal lane % 4)
  const float mt = max_lane_mod4(fmaxf(fmaxf(p[0], p[1]), fmaxf(p[2], p[3])));
  if (__builtin_amdgcn_ballot_w64(mt > st.m)) {
    const float mnew = fmaxf(st.m, mt);
    const float corr = __builtin_amdgcn_exp2f(st.m - mnew);
    st.l *= corr;
#pragma unroll
    for (int g = 0; g < NG; ++g) st.zc[g] *= corr;
    st.m = mnew;
    // output rows of head i take head i's factor (lane i holds head i)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float ci = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(corr), i));
#pragma unroll
      for (int cb = 0; cb < Gm::CB; ++cb) st.O[cb][i] *= ci;
    }
  }
  float ps = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    p[i] = __builtin_amdgcn_exp2f(p[i] - st.m);
    ps += p[i];
  }
  st.l += ps;
  // ---- P' (fp16 p * s_v, or bf16 p for the 16-bit pool), two packed pairs per group
  uint32_t ph[NG][2];
#pragma unroll
  for (int g = 0; g < NG; ++g)
#pragma unroll
    for (int jp = 0; jp < 2; ++jp) {
      uint32_t h2[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int i = 2 * jp + hh;
        if constexpr (PT::QUANT) {
          float S, Z;
          unpack_sz(tr.vsz[i * NG + g], S, Z);
          const _Float16 h = (_Float16)(p[i] * S);
          st.zc[g] = fmaf(p[i], Z, st.zc[g]);
          h2[hh] = uint32_t(*(const uint16_t *)&h);
        } else {
          h2[hh] = uint32_t(f2bf(p[i]));
        }
      }
      ph[g][jp] = h2[0] | (h2[1] << 16);
    }
  // ---- O += P' V, one 32-slot step (key blocks 2 kv, 2 kv + 1) at a time
#pragma unroll
  for (int kv = 0; kv < Gm::KV; ++kv) {
    const bool s0 = c == 2 * kv, s1 = c == 2 * kv + 1;
    u32x4 pk[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      pk[g][0] = s0 ? ph[g][0] : 0u;
      pk[g][1] = s0 ? ph[g][1] : 0u;
      pk[g][2] = s1 ? ph[g][0] : 0u;
      pk[g][3] = s1 ? ph[g][1] : 0u;
    }
#pragma unroll
    for (int cb = 0; cb < Gm::CB; ++cb) {
      const int g = (16 * cb) / G;
      if constexpr (PT::QUANT) {
        const f16x8 bv = vfield_h<BP>(tr.v.w, kv * Gm::CB + cb);
        st.O[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h(pk[g]), bv, st.O[cb], 0, 0, 0);
      } else {
        const bf16x8 bv = field16(tr.v.w, kv * Gm::CB + cb);
        st.O[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_op(pk[g]), bv, st.O[cb], 0, 0, 0);
      }
    }
  }
}

// Sum the per-lane partials of each head and its virtual output rows.
// Afterwards lane (o4, n) holds in O[cb][i] the un-normalised output of head
// i, channel n + 16 cb; lanes 0..3 hold m and l of heads 0..3.
template <int DH, int G>
__device__ __forceinline__ void dec_finish(DecState<DH> &st) {
  constexpr int NG = DH / G;
#pragma unroll
  for (int x = 4; x < 64; x <<= 1) {
    st.l += __shfl_xor(st.l, x, 64);
#pragma unroll
    for (int g = 0; g < NG; ++g) st.zc[g] += __shfl_xor(st.zc[g], x, 64);
  }
#pragma unroll
  for (int cb = 0; cb < DH / 16; ++cb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = st.O[cb][i];
      v += __shfl_xor(v, 16, 64);
      v += __shfl_xor(v, 32, 64);
      st.O[cb][i] = v + __shfl(st.zc[(16 * cb) / G], i, 64);
    }
}

// Fold tile t of pool BI, resident in LDS at tp, into a one-head-per-column state.
template <int DH, int G, int BI>
__device__ __forceinline__ void fold_tile(SoftState<DH> &st, const CacheView &cv, int t,
                                          const uint8_t *tp, ColMask cm, const bf16x8 *qop,
                                          const float *qsum, float scale2) {
  constexpr int TS = 4096 / DH, BP = 2 << BI;
  TileRegs<DH, BP, G, false> r;
  r.load(tp, cv, BI, t * TS, nullptr, 0);
  process_tile<DH, BP, G, false>(st, r, t * TS, cm, qop, qsum, scale2);
}

// One block of 8 waves per (sequence, kv head, chunk): the waves split each
// pool's tile range of the chunk into contiguous runs; each wave streams its
// runs of all four pools through its ring.  PACKED (at most 4 query heads per
// kv head): head-packed columns; otherwise one head per column.  With one
// chunk the block writes the normalised output itself; otherwise it leaves
// (m, l, O) partials.
template <int DH, int G, bool PACKED>
__global__ __launch_bounds__(512, 1) void attn_decode_kernel(DecodeArgs a) {
  constexpr int RING = DEC_WAVES * DEC_RING;
  static_assert(RING >= DEC_WAVES * 16 * (DH + 2) * 4, "ring doubles as the merge buffer");
  __shared__ __align__(1024) uint8_t ring[RING];
  __shared__ int bounds[4][2];  // per pool: first slot of the window, length
  const CacheView &cv = a.cv;
  constexpr int TS = 4096 / DH;
  const int Hkv = cv.Hkv;
  const int b = blockIdx.x / Hkv, g = blockIdx.x % Hkv, split = blockIdx.y;
  const int lane = threadIdx.x & 63, n16 = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int R = a.R;
  const int hl = PACKED ? (n16 & 3) : n16;  // the lane's query head within the group
  const int head = g * R + hl;
  // independent loads first: the query row, the sequence id and the modes
  u32x4 qraw[DH / 32];
  {
    const bf16 *qrow = a.q + (int64_t(b) * a.H + g * R + (hl < R ? hl : 0)) * DH + 8 * (lane >> 4);
#pragma unroll
    for (int ks = 0; ks < DH / 32; ++ks) qraw[ks] = *(const u32x4 *)(qrow + 32 * ks);
  }
  const int s = a.seq_ids ? a.seq_ids[b] : b;
  const bool seq_ok = s >= 0 && s < cv.n_seq;
  const int hm = (seq_ok && hl < R) ? int(a.mode[b * a.H + head]) : 0;
  // union of the group's modes (every lane holds one of the R heads)
  const bool any_full = __builtin_amdgcn_ballot_w64(hm == TRIROUTE_FULL) != 0;
  const bool any_local = __builtin_amdgcn_ballot_w64(hm == TRIROUTE_LOCAL) != 0;
  const int U = any_full ? TRIROUTE_FULL : any_local ? TRIROUTE_LOCAL : TRIROUTE_SKIP;
  using State = typename std::conditional<PACKED, DecState<DH>, SoftState<DH>>::type;
  State st;
  if constexpr (PACKED) dec_init(st); else state_init(st);
  if (U > 0 && wave < 4) {  // waves 0..3 find the window start of pools 0..3
    const int bi = wave;
    const int P = cv.seq_len[s] - 1;
    const int len = cv.pool_len[s * 4 + bi];
    // the window start matters only to local heads
    const int lb = any_local ? lower_bound_pos(cv, s, bi, len, P - a.w + 1) : 0;
    if (lane == 0) {
      bounds[bi][0] = lb;
      bounds[bi][1] = len;
    }
  }
  __syncthreads();
  if (U > 0) {
    bf16x8 qop[DH / 32];
    float qsum[DH / G];
    q_operand<DH, G>(qraw, hl < R, qop, qsum);
    wait_vm<0>();  // from here on the only vector-memory traffic is the tile stream
    Int4 w0, w1;
    TileMask tm0[4];  // the lane's key bounds per pool, in pool slots
    int mlo[4], mhi[4];
    // The chunk's tiles of the four pools, taken as one list in pool order,
    // are cut into DEC_WAVES contiguous runs of about equal cost (a tile of
    // width bi costs DEC_COST[bi]: its bytes and its dequantisation work);
    // a tile goes to the run that holds its midpoint.
    int c0[4], nc[4], wsum = 0;
#pragma unroll
    for (int bi = 0; bi < 4; ++bi) {
      const int lb = bounds[bi][0], len = bounds[bi][1];
      const int lo = U == TRIROUTE_FULL ? 0 : lb;
      const int t0 = lo / TS, nt = (len + TS - 1) / TS - t0;
      // nt * NS stays far below 2^31 (capacity / TS tiles, at most 16 chunks)
      c0[bi] = t0 + nt * split / a.NS;
      nc[bi] = t0 + nt * (split + 1) / a.NS - c0[bi];
      wsum += nc[bi] * DEC_COST[bi];
      mlo[bi] = hm == TRIROUTE_FULL ? 0 : hm == TRIROUTE_LOCAL ? lb : 1;
      mhi[bi] = hm == TRIROUTE_SKIP ? 0 : len - 1;
      tm0[bi] = TileMask{mlo[bi], mhi[bi]};
    }
    int pre = 0;  // cost of the earlier pools' tiles
#pragma unroll
    for (int bi = 0; bi < 4; ++bi) {
      // first tile i of run r: DEC_WAVES (2 pre + (2 i + 1) c) >= 2 wsum r
      const int c = DEC_COST[bi];
      auto first = [&](int r) {
        const int num = 2 * wsum * r - DEC_WAVES * (2 * pre + c);
        const int den = 2 * DEC_WAVES * c;
        const int i = num <= 0 ? 0 : (num + den - 1) / den;
        return min(i, nc[bi]);
      };
      w0.set(bi, __builtin_amdgcn_readfirstlane(c0[bi] + first(wave)));
      w1.set(bi, __builtin_amdgcn_readfirstlane(c0[bi] + first(wave + 1)));
      pre += nc[bi] * c;
    }
    const uint8_t *rptr = ring + wave * DEC_RING;
    const uint32_t rbase = lds_addr(ring) + wave * DEC_RING;
    if constexpr (PACKED) {
      // the lane's Q operand, kept only in the columns of key block blk
      constexpr int NB = TS / 16, KS = DH / 32;
      bf16x8 qopm[NB * KS];
      const bf16x8 zero = as_op(u32x4{0u, 0u, 0u, 0u});
#pragma unroll
      for (int blk = 0; blk < NB; ++blk)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qopm[blk * KS + ks] = (n16 >> 2) == blk ? qop[ks] : zero;
      const bool dead = (n16 >> 2) >= NB;
      stream_tiles<DH, G>(cv, s, g, w0, w1, rptr, rbase, [&](auto BI, int t, const uint8_t *tp) {
        constexpr int bi = decltype(BI)::value;
        DecRegs<DH, 2 << bi, G> r;
        r.load(tp, cv, bi);
        const TileMask tm{tm0[bi].lo - t * TS, tm0[bi].hi - t * TS};
        fold_dec<DH, 2 << bi, G>(st, r, tm, dead, qopm, qsum, a.scale2);
      });
      dec_finish<DH, G>(st);
    } else {
      stream_tiles<DH, G>(cv, s, g, w0, w1, rptr, rbase, [&](auto BI, int t, const uint8_t *tp) {
        constexpr int bi = decltype(BI)::value;
        fold_tile<DH, G, bi>(st, cv, t, tp, ColMask{mlo[bi], mhi[bi]}, qop, qsum, a.scale2);
      });
      state_finish<DH, G>(st);
    }
  }
  // merge the waves in LDS (the rings are drained): [wave][col][m, l, O]
  __syncthreads();
  float(*red)[16][DH + 2] = (float(*)[16][DH + 2])ring;
  if (lane < 16) {
    red[wave][lane][0] = st.m;
    red[wave][lane][1] = st.l;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int cb = 0; cb < DH / 16; ++cb)
      red[wave][4 * (lane >> 4) + i][2 + n16 + 16 * cb] = st.O[cb][i];
  __syncthreads();
  for (int idx = threadIdx.x; idx < R * DH; idx += blockDim.x) {
    const int col = idx / DH, c = idx % DH;
    float M = -INFINITY;
#pragma unroll
    for (int wv = 0; wv < DEC_WAVES; ++wv) M = fmaxf(M, red[wv][col][0]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int wv = 0; wv < DEC_WAVES; ++wv) {
        const float mw = red[wv][col][0];
        if (mw == -INFINITY) continue;
        const float f = exp2f(mw - M);
        L += red[wv][col][1] * f;
        O += red[wv][col][2 + c] * f;
      }
    }
    const int hh = g * R + col;
    if (a.NS == 1) {
      a.o[(int64_t(b) * a.H + hh) * DH + c] = f2bf(L > 0.f ? O * (1.f / L) : 0.f);
    } else {
      float *pp = a.part + ((int64_t(b) * a.H + hh) * a.NS + split) * (DH + 2);
      pp[2 + c] = O;
      if (c == 0) {
        pp[0] = M;
        pp[1] = L;
      }
    }
  }
}

template <int DH>
__global__ __launch_bounds__(256) void attn_decode_combine_kernel(const float *__restrict__ part,
                                                                  int BH, int NS,
                                                                  bf16 *__restrict__ o) {
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (item >= BH) return;
  const float *pp = part + int64_t(item) * NS * (DH + 2);
  float M = -INFINITY;
  for (int j = 0; j < NS; ++j) M = fmaxf(M, pp[j * (DH + 2)]);
  float L = 0.f, acc[DH / 64];
#pragma unroll
  for (int r = 0; r < DH / 64; ++r) acc[r] = 0.f;
  if (M != -INFINITY) {
    for (int j = 0; j < NS; ++j) {
      const float mj = pp[j * (DH + 2)];
      if (mj == -INFINITY) continue;
      const float wgt = exp2f(mj - M);
      L += pp[j * (DH + 2) + 1] * wgt;
#pragma unroll
      for (int r = 0; r < DH / 64; ++r) acc[r] += pp[j * (DH + 2) + 2 + lane + 64 * r] * wgt;
    }
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
#pragma unroll
  for (int r = 0; r < DH / 64; ++r) o[int64_t(item) * DH + lane + 64 * r] = f2bf(acc[r] * inv);
}

// ------------------------------------------------------------------ prefill
struct PrefillArgs {
  CacheView cv;
  const bf16 *q;
  const int32_t *seq_ids, *cnt, *idx;
  bf16 *o;
  int B, T, H, Hkv, R, NQ, w, QT;  // NQ = head quartets per kv head, QT = ceil(T / 16)
  float scale2;
};

// Prefill: one block of two waves per (sequence, kv head, head quartet,
// mode, query tile qt); wave w takes the qt-th 16 compacted queries of heads
// 2w and 2w + 1 of the quartet: two 16-column blocks that share every K and
// V operand, so each code field of a tile is converted once per two heads.
// The quartet's queries sit at similar positions; the block streams the
// union of their key ranges from every pool once, through an LDS byte FIFO
// shared by the two waves (each tile followed by its slots' key positions;
// the transfers split over the waves), and every wave masks per head and key
// by position.  A head whose columns all miss a tile skips it.
constexpr int PF_WAVES = 2;
constexpr int PF_HEADS = 2;                    // heads per wave
constexpr int PF_RING = 40 * 1024 - 512;       // four blocks (eight waves) per CU
// Lazy rescale threshold (log2 units): P' = fp16(p * s_v) with p <= 2^PF_TAU
// stays finite for value scales up to 65504 / 2^PF_TAU = 1023.
constexpr float PF_TAU = 6.f;

// v_max3_f32 / v_max_f32 on scores that are never NaN (fmaxf would first
// quiet each operand).
__device__ __forceinline__ float vmax3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
// max_rows without quieting
__device__ __forceinline__ float vmax_rows(float x) {
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
  x = vmax(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
  return vmax(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
}

// fp16(a * s) with s the fp16 in bits 0..15 of sw, rounded once: into bits
// 0..15 of a fresh word (mixlo; bits 16..31 left as they were) or into bits
// 16..31 of w (mixhi; bits 0..15 kept).
__device__ __forceinline__ uint32_t mul_f16_lo(float a, uint32_t sw) {
  uint32_t r;
  asm("v_fma_mixlo_f16 %0, %1, %2, 0 op_sel_hi:[0,1,0]" : "=v"(r) : "v"(a), "v"(sw));
  return r;
}
__device__ __forceinline__ uint32_t mul_f16_hi(uint32_t w, float a, uint32_t sw) {
  asm("v_fma_mixhi_f16 %0, %1, %2, 0 op_sel_hi:[0,1,0]" : "+v"(w) : "v"(a), "v"(sw));
  return w;
}

// Lower bounds, in the sorted key positions of pool k % 4 of sequence s, of
// key[k] for eight (pool, key) pairs at once: each round probes 64 evenly
// spaced entries of every range still longer than 64, the eight loads in
// flight together.  A key <= 0 has bound 0 (positions are >= 0).  Called by
// the whole wave with wave-uniform arguments.
__device__ __forceinline__ void lower_bounds8(const CacheView &cv, int s, const int *len,
                                              const int *key, int *res) {
  const int lane = threadIdx.x & 63;
  int lo[8], hi[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    lo[k] = 0;
    hi[k] = key[k] <= 0 ? 0 : len[k & 3];
  }
  for (;;) {
    bool more = false;
#pragma unroll
    for (int k = 0; k < 8; ++k) more |= hi[k] - lo[k] > 64;
    if (!more) break;
    int v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int span = hi[k] - lo[k];
      v[k] = 0;
      if (span > 64) v[k] = cv.pos_at(s, k & 3, lo[k] + int(int64_t(span) * (lane + 1) / 64) - 1);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int span = hi[k] - lo[k];
      if (span > 64) {
        const int c = __popcll(__ballot(v[k] < key[k]));  // probes 0 .. c-1 lie below the key
        const int nlo = c > 0 ? lo[k] + int(int64_t(span) * c / 64) : lo[k];
        const int nhi = c < 64 ? lo[k] + int(int64_t(span) * (c + 1) / 64) - 1 : hi[k];
        lo[k] = nlo;
        hi[k] = nhi;
      }
    }
  }
  int v[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int idx = lo[k] + lane;
    v[k] = idx < hi[k] ? cv.pos_at(s, k & 3, idx) : INT_MAX;
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) res[k] = lo[k] + __popcll(__ballot(v[k] < key[k]));
}

// What a lane needs of a resident prefill tile of width BP (bf16 layer: the
// 16-bit pool holds bf16), read from LDS in two parts so that the K part is
// dead before the V part is live: the K lane record, the fp16 scale/zero
// words of the lane's slots and their key positions (INT_MAX past the pool
// length); then the V lane record and its scale/zero words.
template <int DH, int BP, int G>
struct PfTile {
  using Gm = Geo<DH>;
  static constexpr int NG = DH / G;
  static constexpr int W = PoolTraits<BP>::WORDS;
  static constexpr bool Q = PoolTraits<BP>::QUANT;
  static constexpr int KSZ = 1024 * BP, VSZ = 1024 * BP + Gm::TS * NG * 4;
  static constexpr int TB = 1024 * BP + (Q ? 2 * Gm::TS * NG * 4 : 0);  // codes + scale/zero
  union Rec {
    u32x4 v[W / 4];
    uint32_t w[W];
  };

  struct K {
    Rec r;
    uint32_t sz[Q ? Gm::NB : 1][4 * NG];  // [block][slot i * NG + g]
    int key[Gm::NB][4];
    int first, last;  // positions of the first and last slot (last INT_MAX past the length)
  };
  struct V {
    Rec r;
    uint32_t sz[Q ? Gm::KV : 1][2][4 * NG];  // [step][half][slot i * NG + g]
  };

  __device__ static __forceinline__ void load_k(K &k, const uint8_t *tp, int slot0, int klen) {
    const int lane = threadIdx.x & 63, o4 = lane >> 4;
    const u32x4 *kp = (const u32x4 *)(tp + lane * 8 * BP);
#pragma unroll
    for (int x = 0; x < W / 4; ++x) k.r.v[x] = kp[x];
    if constexpr (Q) {
      const u32x4 *ks = (const u32x4 *)(tp + KSZ);
#pragma unroll
      for (int blk = 0; blk < Gm::NB; ++blk)
#pragma unroll
        for (int x = 0; x < NG; ++x) {
          const u32x4 t = ks[((blk * 16 + 4 * o4) * NG) / 4 + x];
#pragma unroll
          for (int y = 0; y < 4; ++y) k.sz[blk][4 * x + y] = t[y];
        }
    }
    const int32_t *pp = (const int32_t *)(tp + TB);
#pragma unroll
    for (int blk = 0; blk < Gm::NB; ++blk) {
      const u32x4 t = *(const u32x4 *)(pp + blk * 16 + 4 * o4);
#pragma unroll
      for (int i = 0; i < 4; ++i) k.key[blk][i] = int(t[i]);
    }
    k.first = __builtin_amdgcn_readfirstlane(pp[0]);
    k.last = __builtin_amdgcn_readfirstlane(pp[Gm::TS - 1]);
    if (slot0 + Gm::TS > klen) {  // the pool ends inside this tile
      k.last = INT_MAX;
#pragma unroll
      for (int blk = 0; blk < Gm::NB; ++blk)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          k.key[blk][i] = slot0 + blk * 16 + 4 * o4 + i < klen ? k.key[blk][i] : INT_MAX;
    }
  }

  __device__ static __forceinline__ void load_v(V &v, const uint8_t *tp) {
    const int lane = threadIdx.x & 63, o4 = lane >> 4;
    const u32x4 *vp = (const u32x4 *)(tp + 512 * BP + lane * 8 * BP);
#pragma unroll
    for (int x = 0; x < W / 4; ++x) v.r.v[x] = vp[x];
    if constexpr (Q) {
      const u32x4 *vs = (const u32x4 *)(tp + VSZ);
#pragma unroll
      for (int kv = 0; kv < Gm::KV; ++kv)
#pragma unroll
        for (int hb = 0; hb < 2; ++hb)
#pragma unroll
          for (int x = 0; x < NG; ++x) {
            const u32x4 t = vs[((32 * kv + 16 * hb + 4 * o4) * NG) / 4 + x];
#pragma unroll
            for (int y = 0; y < 4; ++y) v.sz[kv][hb][4 * x + y] = t[y];
          }
    }
  }
};

// How a head's 16 columns meet a tile: every key in every column's range
// (PF_ALL), whole columns out (PF_COLS; `none` per lane), or per key
// (PF_KEYS: key passes iff key - lo <= span, mod 2^32).
enum { PF_ALL = 0, PF_COLS = 1, PF_KEYS = 2 };

struct PfMask {
  uint32_t lo, span;  // lo = 2^32 - 1 and span = 0 for a column without a query
  int mode;
  bool none;
};

// Scores of a whole tile for one head: S^T for the tile's 16-slot blocks
// from the shared K operands, dequantised per group, masked; one
// online-softmax update for the tile; leaves exp2(score - m) in p (block
// blk, slot i at p[4 blk + i]).
template <int DH, int BP, int G>
__device__ __forceinline__ void pf_scores(SoftState<DH> &st, const typename PfTile<DH, BP, G>::K &tk,
                                          const u32x4 (&kop)[Geo<DH>::NB][DH / 32],
                                          const bf16x8 *qop, const float *qsum, float scale2,
                                          const PfMask &mk, float (&p)[4 * Geo<DH>::NB]) {
  constexpr int NB = Geo<DH>::NB, NX = 4 * NB;
  constexpr int NG = DH / G, gks = G / 32, KS = DH / 32, CB = DH / 16;
  constexpr bool QUANT = PoolTraits<BP>::QUANT;
  const int lane = threadIdx.x & 63, o4 = lane >> 4;
  float x[NX];
#pragma unroll
  for (int blk = 0; blk < NB; ++blk) {
    f32x4 acc[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc[ks / gks] =
          __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_op(kop[blk][ks]), qop[ks], acc[ks / gks], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float sv = 0.f;
      if constexpr (QUANT) {
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          float S, Z;
          unpack_sz(tk.sz[blk][i * NG + g], S, Z);
          sv = fmaf(S, acc[g][i], sv);
          sv = fmaf(Z, qsum[g], sv);
        }
      } else {
#pragma unroll
        for (int g = 0; g < NG; ++g) sv += acc[g][i];
      }
      x[4 * blk + i] = sv;
    }
  }
  if (mk.mode == PF_KEYS) {
#pragma unroll
    for (int j = 0; j < NX; ++j)
      x[j] = uint32_t(tk.key[j >> 2][j & 3]) - mk.lo <= mk.span ? x[j] : -INFINITY;
  } else if (mk.mode == PF_COLS) {
#pragma unroll
    for (int j = 0; j < NX; ++j) x[j] = mk.none ? -INFINITY : x[j];
  }
  // scores are x * scale2 (log2 domain); the positive factor commutes with the max
  float mt = vmax3(vmax3(x[0], x[1], x[2]), vmax3(x[3], x[4], x[5]), vmax(x[6], x[7]));
#pragma unroll
  for (int j = 8; j < NX; j += 8)
    mt = vmax3(mt, vmax3(x[j], x[j + 1], x[j + 2]),
               vmax3(vmax3(x[j + 3], x[j + 4], x[j + 5]), x[j + 6], x[j + 7]));
  mt = vmax_rows(mt) * scale2;
  // The running max moves only when some column's tile max exceeds it by
  // more than PF_TAU: below that the stale max still bounds exp2(score - m)
  // by 2^PF_TAU, and O, l and zc keep a common scale, so the quotient is
  // unchanged.
  if (__builtin_amdgcn_ballot_w64(mt > st.m + PF_TAU)) {
    const float mnew = fmaxf(st.m, mt);
    const float corr = __builtin_amdgcn_exp2f(st.m - mnew);
    st.l *= corr;
#pragma unroll
    for (int g = 0; g < NG; ++g) st.zc[g] *= corr;
    st.m = mnew;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float ci = __shfl(corr, 4 * o4 + i, 64);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) st.O[cb][i] *= ci;
    }
  }
  const float nm = -st.m;
  float ps = 0.f;
#pragma unroll
  for (int j = 0; j < NX; ++j) {
    p[j] = __builtin_amdgcn_exp2f(fmaf(x[j], scale2, nm));
    ps += p[j];
  }
  st.l += ps;
}

// P operands of one step for one head: P' = fp16(p * s_v) per group against
// the fp16 codes (quantized pools; the zero term goes to zc), P = bf16(p)
// against the stored bf16 (16-bit pool).
template <int DH, int BP, int G>
__device__ __forceinline__ void pf_pack(SoftState<DH> &st, const typename PfTile<DH, BP, G>::V &tv,
                                        int kv, const float (&p)[4 * Geo<DH>::NB],
                                        u32x4 (&pk)[DH / G]) {
  constexpr int NG = DH / G;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
#pragma unroll
    for (int jp = 0; jp < 4; ++jp) {
      const int j0 = 2 * jp, j1 = 2 * jp + 1;  // step slots: block 2 kv + (j >> 2), slot j & 3
      const float p0 = p[8 * kv + j0], p1 = p[8 * kv + j1];
      if constexpr (PoolTraits<BP>::QUANT) {
        const uint32_t w0 = tv.sz[kv][j0 >> 2][(j0 & 3) * NG + g];
        const uint32_t w1 = tv.sz[kv][j1 >> 2][(j1 & 3) * NG + g];
        pk[g][jp] = mul_f16_hi(mul_f16_lo(p0, w0), p1, w1);
        const uint16_t z0 = uint16_t(w0 >> 16), z1 = uint16_t(w1 >> 16);
        st.zc[g] = fmaf(p0, float(*(const _Float16 *)&z0), st.zc[g]);
        st.zc[g] = fmaf(p1, float(*(const _Float16 *)&z1), st.zc[g]);
      } else {
        pk[g][jp] = pk_bf16(p0, p1);
      }
    }
  }
}

// Fold one resident tile (pool width BP, first slot slot0, pool length klen)
// into the heads' states: the scores of every head from K operands converted
// once, then per 32-slot step O += P' V with each V field converted once.
template <int DH, int BP, int G>
__device__ __forceinline__ void pf_tile(SoftState<DH> (&st)[PF_HEADS], const uint8_t *tp, int slot0,
                                        int klen, const ColMask (&cm)[PF_HEADS],
                                        const uint32_t (&mlo)[PF_HEADS],
                                        const uint32_t (&mspan)[PF_HEADS],
                                        const bool (&act)[PF_HEADS],
                                        const bf16x8 (&qop)[PF_HEADS][DH / 32],
                                        const float (&qsum)[PF_HEADS][DH / G], float scale2) {
  using Gm = Geo<DH>;
  using PT = PfTile<DH, BP, G>;
  constexpr int KS = DH / 32, CB = DH / 16, NG = DH / G;
  typename PT::K tk;
  PT::load_k(tk, tp, slot0, klen);
  PfMask mk[PF_HEADS];
  bool run[PF_HEADS];
#pragma unroll
  for (int hq = 0; hq < PF_HEADS; ++hq) {
    const bool none = cm[hq].lo > cm[hq].hi || tk.last < cm[hq].lo || tk.first > cm[hq].hi;
    const bool all = tk.first >= cm[hq].lo && tk.last <= cm[hq].hi;
    run[hq] = act[hq] && __builtin_amdgcn_ballot_w64(!none) != 0;
    mk[hq].lo = mlo[hq];
    mk[hq].span = mspan[hq];
    mk[hq].none = none;
    mk[hq].mode = __builtin_amdgcn_ballot_w64(!none && !all) ? PF_KEYS
                  : __builtin_amdgcn_ballot_w64(none)        ? PF_COLS
                                                             : PF_ALL;
  }
  float p[PF_HEADS][4 * Gm::NB];
  {
    u32x4 kop[Gm::NB][KS];
#pragma unroll
    for (int blk = 0; blk < Gm::NB; ++blk)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kop[blk][ks] = kfield<BP>(tk.r.w, blk * KS + ks);
#pragma unroll
    for (int hq = 0; hq < PF_HEADS; ++hq)
      if (run[hq]) pf_scores<DH, BP, G>(st[hq], tk, kop, qop[hq], qsum[hq], scale2, mk[hq], p[hq]);
  }
  typename PT::V tv;
  PT::load_v(tv, tp);
#pragma unroll
  for (int kv = 0; kv < Gm::KV; ++kv) {
    u32x4 pk[PF_HEADS][NG];
#pragma unroll
    for (int hq = 0; hq < PF_HEADS; ++hq)
      if (run[hq]) pf_pack<DH, BP, G>(st[hq], tv, kv, p[hq], pk[hq]);
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const int g = (16 * cb) / G;
      if constexpr (PT::Q) {
        const f16x8 bv = vfield_h<BP>(tv.r.w, kv * CB + cb);
#pragma unroll
        for (int hq = 0; hq < PF_HEADS; ++hq)
          if (run[hq])
            st[hq].O[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h(pk[hq][g]), bv, st[hq].O[cb],
                                                                  0, 0, 0);
      } else {
        const bf16x8 bv = field16(tv.r.w, kv * CB + cb);
#pragma unroll
        for (int hq = 0; hq < PF_HEADS; ++hq)
          if (run[hq])
            st[hq].O[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_op(pk[hq][g]), bv,
                                                                   st[hq].O[cb], 0, 0, 0);
      }
    }
  }
}

// This wave's share of the transfers of one tile of pool BI (codes and
// scale/zero from src, then the TS key positions from ps) into LDS address
// dst: transfer x goes to wave x % NW.
template <int DH, int G, int BI, int NW>
__device__ __forceinline__ void issue_tile_split(const uint8_t *src, const int32_t *ps, uint32_t dst,
                                                 int wave) {
  using SG = StreamGeo<DH, G>;
  constexpr int TB = SG::tb(BI), NI = SG::ni(BI);
  const int lane = threadIdx.x & 63;
  const uint32_t off = lane * 16;
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    if (j % NW != wave) continue;
    if ((j + 1) * 1024 <= TB || off < uint32_t(TB - j * 1024))
      dma16_s(src + j * 1024, off, dst + j * 1024);
  }
  if (NI % NW == wave && lane < SG::TS / 4) dma16(ps + 4 * lane, dst + TB);
}

// The block's tiles [w0[bi], w1[bi]) of the four pools, pools in order,
// through one LDS byte FIFO (RING bytes at rptr / LDS address rbase) shared
// by the NW waves: the placement rule of stream_tiles (each tile followed by
// its slots' positions), transfer x of a tile (the positions last) issued by
// wave x % NW.  Before a tile is folded each wave waits for its own
// transfers of it and the block meets at a barrier, which also tells every
// wave that all of them are done with the previous tile, whose space is
// released only then.  A tile that found no room while the previous one was
// resident (two wide tiles and the wrap rule) is issued after an extra
// barrier that releases the previous tile first.  fold(BI, t, lds_pointer)
// as in stream_tiles.  On entry no other vector-memory load of any wave may
// be in flight.
template <int DH, int G, int RING, int NW, class Fold>
__device__ __forceinline__ void stream_tiles_block(const CacheView &cv, int s, int g, Int4 w0,
                                                   Int4 w1, const uint8_t *rptr, uint32_t rbase,
                                                   Fold &&fold) {
  using SG = StreamGeo<DH, G>;
  constexpr int PB = 4 * SG::TS;
  static_assert(((1024 * 16 + PB + 255) & ~255) <= RING, "a 16-bit tile fits the ring");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // transfers of a width-bi tile: ni(bi) code/scale blocks + 1 for the positions
  auto own = [&](int bi) { return max(0, (SG::ni(bi) + 1 - wave + NW - 1) / NW); };
  const int e1 = w1[0] - w0[0], e2 = e1 + w1[1] - w0[1], e3 = e2 + w1[2] - w0[2];
  const int ktot = e3 + w1[3] - w0[3];
  const int d0 = w0[0], d1 = w0[1] - e1, d2 = w0[2] - e2, d3 = w0[3] - e3;
  int kp = 0;
  int phead = 0, pfree = 0;  // ring end of the newest tile; start of the oldest resident tile
  int nin = 0, issued = 0, consumed = 0;  // tiles resident or in flight; own transfers out / used
  int chead = 0;                          // ring end of the last tile handed to fold
  auto produce = [&]() {
    while (kp < ktot) {
      const int pb = (kp >= e1) + (kp >= e2) + (kp >= e3);
      const int tb = (1024 << (pb + 1)) + (pb < 3 ? SG::tb(0) - 2048 : 0);
      const int sz = (tb + PB + 255) & ~255;
      const int pos = phead + sz <= RING ? phead : 0;
      bool ok = true;
      if (nin > 0) {
        if (pfree < phead)
          ok = pos == phead || sz <= pfree;
        else
          ok = pos == phead && phead + sz <= pfree;
      }
      if (!ok) break;
      const int pt = kp + (pb == 0 ? d0 : pb == 1 ? d1 : pb == 2 ? d2 : d3);
      const int32_t *ps = cv.pos_tile(s, pb, pt);
      switch (pb) {  // compile-time pool: no run-time indexing of the cache view's arrays
        case 0: issue_tile_split<DH, G, 0, NW>(cv.tile(s, 0, g, pt), ps, rbase + pos, wave); break;
        case 1: issue_tile_split<DH, G, 1, NW>(cv.tile(s, 1, g, pt), ps, rbase + pos, wave); break;
        case 2: issue_tile_split<DH, G, 2, NW>(cv.tile(s, 2, g, pt), ps, rbase + pos, wave); break;
        default: issue_tile_split<DH, G, 3, NW>(cv.tile(s, 3, g, pt), ps, rbase + pos, wave); break;
      }
      issued += own(pb);
      phead = pos + sz;
      ++nin;
      ++kp;
    }
  };
  produce();
  int gi = 0;         // index of the tile being consumed in the concatenated ranges
  bool held = false;  // the previous tile is still resident
  auto release = [&]() {
    if (held) {
      --nin;
      pfree = chead;
      held = false;
    }
  };
  auto pool = [&](auto BI) {
    constexpr int bi = decltype(BI)::value;
    constexpr int sz = (SG::tb(bi) + PB + 255) & ~255;
    const int t1 = w1[bi];
    for (int t = w0[bi]; t < t1; ++t) {
      if (kp <= gi) {
        // not issued yet: the previous tile left no room for it; once every
        // wave is done with that tile the ring is empty and this one goes in
        __syncthreads();
        release();
        produce();
      }
      const int cpos = chead + sz <= RING ? chead : 0;  // the producer's placement rule
      consumed += own(bi);
      wait_vm_le(issued - consumed);
      __syncthreads();  // this tile is in from every wave; every wave is done with the previous
      release();
      produce();
      fold(BI, t, rptr + cpos);
      chead = cpos + sz;
      held = true;
      ++gi;
    }
  };
  pool(std::integral_constant<int, 0>{});
  pool(std::integral_constant<int, 1>{});
  pool(std::integral_constant<int, 2>{});
  pool(std::integral_constant<int, 3>{});
}

template <int DH, int G>
__global__ __launch_bounds__(64 * PF_WAVES) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_prefill_mfma_kernel(PrefillArgs a) {
  using SG = StreamGeo<DH, G>;
  constexpr int TS = SG::TS, KS = DH / 32, NG = DH / G;
  __shared__ __align__(1024) uint8_t ring[PF_RING];
  const CacheView &cv = a.cv;
  const int lane = threadIdx.x & 63, n16 = lane & 15, o4 = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // heavy blocks first: full mode, and within a mode the query tiles from
  // the latest down, each across all (sequence, kv head, quartet), so that
  // blocks start in decreasing order of their key range
  const int per_qt = a.B * a.Hkv * a.NQ, per_mode = per_qt * a.QT;
  const int m = int(blockIdx.x) < per_mode ? TRIROUTE_FULL : TRIROUTE_LOCAL;
  int r = int(blockIdx.x) % per_mode;
  const int qt = a.QT - 1 - r / per_qt;
  r %= per_qt;
  const int quart = r % a.NQ;
  r /= a.NQ;
  const int g = r % a.Hkv, b = r / a.Hkv;
  const int s = a.seq_ids ? a.seq_ids[b] : b;
  if (s < 0 || s >= cv.n_seq) return;
  const int base = cv.seq_len[s] - a.T;
  // union of the quartet's key ranges (block-uniform: every wave computes it)
  int lo_u = INT_MAX, hi_u = -1;
  for (int k = 0; k < PF_WAVES * PF_HEADS && quart * PF_WAVES * PF_HEADS + k < a.R; ++k) {
    const int sg = (b * a.H + g * a.R + quart * PF_WAVES * PF_HEADS + k) * 2 + (m - 1);
    const int ck = a.cnt[sg];
    if (qt * 16 >= ck) continue;
    const int32_t *lk = a.idx + int64_t(sg) * a.T;
    const int pmin = base + lk[qt * 16], pmax = base + lk[min(qt * 16 + 15, ck - 1)];
    lo_u = min(lo_u, m == TRIROUTE_LOCAL ? pmin - a.w + 1 : 0);
    hi_u = max(hi_u, pmax);
  }
  // this wave's heads: query columns, position bounds, query operands
  int count[PF_HEADS];
  bool act[PF_HEADS];
  ColMask cm[PF_HEADS];
  uint32_t mlo[PF_HEADS], mspan[PF_HEADS];
  bf16x8 qop[PF_HEADS][KS];
  float qsum[PF_HEADS][NG];
#pragma unroll
  for (int hq = 0; hq < PF_HEADS; ++hq) {
    const int hr = (quart * PF_WAVES + wave) * PF_HEADS + hq;
    const int h = g * a.R + min(hr, a.R - 1);
    const int seg = (b * a.H + h) * 2 + (m - 1);
    count[hq] = hr < a.R ? a.cnt[seg] : 0;
    act[hq] = qt * 16 < count[hq];  // wave-uniform
    const int32_t *lst = a.idx + int64_t(seg) * a.T;
    const int j = qt * 16 + n16;
    const bool valid = act[hq] && j < count[hq];
    const int t = valid ? lst[j] : 0;
    const int P = base + t;
    load_q<DH, G>(a.q + (int64_t(b * a.T + t) * a.H + h) * DH, valid, qop[hq], qsum[hq]);
    cm[hq].lo = valid ? (m == TRIROUTE_LOCAL ? P - a.w + 1 : 0) : 1;
    cm[hq].hi = valid ? P : 0;
    mlo[hq] = valid ? uint32_t(cm[hq].lo) : 0xFFFFFFFFu;
    mspan[hq] = valid ? uint32_t(cm[hq].hi - cm[hq].lo) : 0u;
  }
  lo_u = __builtin_amdgcn_readfirstlane(lo_u);
  hi_u = __builtin_amdgcn_readfirstlane(hi_u);
  if (hi_u < 0) return;
  // tile ranges of the union in every pool
  int len[4], key[8], res[8];
#pragma unroll
  for (int bi = 0; bi < 4; ++bi) {
    len[bi] = cv.pool_len[s * 4 + bi];
    key[bi] = lo_u;
    key[4 + bi] = hi_u + 1;
  }
  lower_bounds8(cv, s, len, key, res);
  Int4 w0, w1;
#pragma unroll
  for (int bi = 0; bi < 4; ++bi) {
    const int sa = res[bi], sb = res[4 + bi];
    w0.set(bi, sa < sb ? sa / TS : 0);
    w1.set(bi, sa < sb ? (sb + TS - 1) / TS : 0);
  }
  SoftState<DH> st[PF_HEADS];
#pragma unroll
  for (int hq = 0; hq < PF_HEADS; ++hq) state_init(st[hq]);
  wait_vm<0>();  // from here on the only vector-memory traffic is the tile stream
  stream_tiles_block<DH, G, PF_RING, PF_WAVES>(
      cv, s, g, w0, w1, ring, lds_addr(ring), [&](auto BI, int t, const uint8_t *tp) {
        constexpr int bi = decltype(BI)::value;
        pf_tile<DH, (2 << bi), G>(st, tp, t * TS, len[bi], cm, mlo, mspan, act, qop, qsum,
                                  a.scale2);
      });
  // normalise and write: lane (o4, n) holds column 4 o4 + i, channel n + 16 cb
#pragma unroll
  for (int hq = 0; hq < PF_HEADS; ++hq) {
    if (!act[hq]) continue;
    state_finish<DH, G>(st[hq]);
    const int h = g * a.R + (quart * PF_WAVES + wave) * PF_HEADS + hq;
    const int seg = (b * a.H + h) * 2 + (m - 1);
    const int32_t *lst = a.idx + int64_t(seg) * a.T;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int col = 4 * o4 + i;
      const float lc = __shfl(st[hq].l, col, 64);
      const int jj = qt * 16 + col;
      if (jj >= count[hq]) continue;
      const int tt = lst[jj];
      const float inv = lc > 0.f ? 1.f / lc : 0.f;
      bf16 *orow = a.o + (int64_t(b * a.T + tt) * a.H + h) * DH;
#pragma unroll
      for (int cbk = 0; cbk < DH / 16; ++cbk) orow[n16 + 16 * cbk] = f2bf(st[hq].O[cbk][i] * inv);
    }
  }
}

// ------------------------------------------------------------------ launchers
int decode_splits(int B, int Hkv, int capacity, int TS) {
  (void)capacity;
  (void)TS;
  // one 8-wave block per CU: chunks so that the grid covers the 256 CUs
  const int ns = (256 + B * Hkv - 1) / (B * Hkv);
  return max(1, min(ns, 16));
}

hipError_t launch_attn_mfma_decode(const triroute_cfg &cfg, const CacheView &cv, int B,
                                   const int32_t *seq_ids, const void *q, const uint8_t *mode,
                                   void *o, float *part, hipStream_t st) {
  DecodeArgs a;
  a.cv = cv;
  a.q = (const bf16 *)q;
  a.mode = mode;
  a.seq_ids = seq_ids;
  a.part = part;
  a.o = (bf16 *)o;
  a.B = B;
  a.H = cfg.n_heads;
  a.R = cfg.n_heads / cfg.n_kv_heads;
  a.w = cfg.window;
  a.NS = decode_splits(B, cfg.n_kv_heads, cv.capacity, cv.TS);
  a.scale2 = LOG2E / sqrtf(float(cfg.head_dim));
  dim3 grid(B * cfg.n_kv_heads, a.NS);
  const int BH = B * cfg.n_heads;
  const int G = cfg.kv_group;
  const int threads = 64 * DEC_WAVES;
  const bool packed = a.R <= 4;
#define DEC_LAUNCH(DH_, G_)                                                  \
  (packed ? attn_decode_kernel<DH_, G_, true><<<grid, threads, 0, st>>>(a)   \
          : attn_decode_kernel<DH_, G_, false><<<grid, threads, 0, st>>>(a))
  if (cfg.head_dim == 64) {
    if (G == 64) DEC_LAUNCH(64, 64); else DEC_LAUNCH(64, 32);
    if (a.NS > 1)
      attn_decode_combine_kernel<64><<<(BH + 3) / 4, 256, 0, st>>>(part, BH, a.NS, (bf16 *)o);
  } else {
    if (G == 64) DEC_LAUNCH(128, 64); else DEC_LAUNCH(128, 32);
    if (a.NS > 1)
      attn_decode_combine_kernel<128><<<(BH + 3) / 4, 256, 0, st>>>(part, BH, a.NS, (bf16 *)o);
  }
#undef DEC_LAUNCH
  return hipGetLastError();
}

hipError_t launch_attn_mfma_prefill(const triroute_cfg &cfg, const CacheView &cv, int B, int T,
                                    const int32_t *seq_ids, const void *q,
                                    const triroute_compaction &c, void *o, hipStream_t st) {
  PrefillArgs a;
  a.cv = cv;
  a.q = (const bf16 *)q;
  a.seq_ids = seq_ids;
  a.cnt = c.attn_cnt;
  a.idx = c.attn_idx;
  a.o = (bf16 *)o;
  a.B = B;
  a.T = T;
  a.H = cfg.n_heads;
  a.R = cfg.n_heads / cfg.n_kv_heads;
  a.w = cfg.window;
  a.QT = (T + 15) / 16;
  a.Hkv = cfg.n_kv_heads;
  a.NQ = (a.R + PF_WAVES * PF_HEADS - 1) / (PF_WAVES * PF_HEADS);
  a.scale2 = LOG2E / sqrtf(float(cfg.head_dim));
  const int64_t blocks = int64_t(B) * a.Hkv * a.NQ * 2 * a.QT;
  const dim3 grid{unsigned(blocks)};
  const int G = cfg.kv_group;
  if (cfg.head_dim == 64) {
    if (G == 64)
      attn_prefill_mfma_kernel<64, 64><<<grid, 64 * PF_WAVES, 0, st>>>(a);
    else
      attn_prefill_mfma_kernel<64, 32><<<grid, 64 * PF_WAVES, 0, st>>>(a);
  } else {
    if (G == 64)
      attn_prefill_mfma_kernel<128, 64><<<grid, 64 * PF_WAVES, 0, st>>>(a);
    else
      attn_prefill_mfma_kernel<128, 32><<<grid, 64 * PF_WAVES, 0, st>>>(a);
  }
  return hipGetLastError();
}

}  // namespace tr
