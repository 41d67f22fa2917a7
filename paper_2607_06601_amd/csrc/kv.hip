// Mixed-width KV cache: layout, append (per-token group quantizer of paper
// Sec. 3.2 (C)) and read-back.
//
// Quantizer (bit exact with the CPU oracle): per group of G channels, fp32
// mn/mx, s32 = (mx - mn) / (2^b - 1), s = fp16_rne(s32), z = fp16_rne(mn),
// code = 0 if s == 0 else clamp(rint_even((x - z) / s), 0, 2^b - 1), every
// step in IEEE fp32.  16-bit stores the activation value verbatim.
#include "kernels.hpp"

namespace tr {

__global__ void fill_u32_kernel(uint32_t *__restrict__ p, int64_t n, uint32_t v) {
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * blockDim.x)
    p[i] = v;
}

hipError_t launch_fill_u32(void *p, int64_t n_words, uint32_t v, hipStream_t st) {
  if (n_words <= 0) return hipSuccess;
  int64_t blocks = (n_words + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  fill_u32_kernel<<<dim3(unsigned(blocks)), 256, 0, st>>>((uint32_t *)p, n_words, v);
  return hipGetLastError();
}

// Per batch row: the slot of each new token in its width pool (its rank
// among the row's earlier tokens of that width, after the pool's current
// length), its position in the pool's position array, the new lengths, and
// the pool lengths before the append.  One block of 16 waves per row walks
// the row's tokens 1024 at a time (ballot counts per wave, then per block).
__global__ __launch_bounds__(1024) void kv_slots_kernel(CacheView cv, int T,
                                                        const int32_t *__restrict__ seq_ids,
                                                        const uint8_t *__restrict__ bit,
                                                        int32_t *__restrict__ old_len) {
  constexpr int NW = 16;
  __shared__ int wc[4][NW];
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int s = seq_ids ? seq_ids[b] : b;
  if (s < 0 || s >= cv.n_seq) {
    if (tid == 0) atomicOr(cv.status, int(TRIROUTE_CACHE_BAD_SEQ));
    if (tid < 4) old_len[b * 4 + tid] = -1;
    return;
  }
  const int len0 = cv.seq_len[s];
  if (len0 + T > cv.capacity) {
    if (tid == 0) atomicOr(cv.status, int(TRIROUTE_CACHE_OVERFLOW));
    if (tid < 4) old_len[b * 4 + tid] = -1;
    return;
  }
  int run[4];
#pragma unroll
  for (int bi = 0; bi < 4; ++bi) run[bi] = cv.pool_len[s * 4 + bi];
  if (cv.PT) {
    // paged: count the row's tokens per width, then take the pages the
    // pools grow into from the free stacks (thread bi for width bi)
    __shared__ int cnt_s[4], fail_s;
    if (tid < 4) cnt_s[tid] = 0;
    if (tid == 0) fail_s = 0;
    __syncthreads();
    for (int t0 = 0; t0 < T; t0 += 64 * NW) {
      const int t = t0 + tid;
      const int bi = t < T ? int(bit[int64_t(b) * T + t]) : -1;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint64_t bq = __ballot(bi == q);
        if (lane == 0 && bq) atomicAdd(&cnt_s[q], __popcll(bq));  // a count: order does not matter
      }
    }
    __syncthreads();
    if (tid < 4) {
      const int bi = tid, per = cv.PT * cv.TS;
      const int need = (run[bi] + cnt_s[bi] + per - 1) / per;
      int32_t *held = cv.alloc + s * 4 + bi;
      const int have = *held;
      if (need > have) {
        const int k = need - have;
        const int top = atomicSub(cv.free_top + bi, k);
        if (need > cv.max_pages || top - k < 0) {
          atomicAdd(cv.free_top + bi, k);  // give the claim back
          atomicOr(&fail_s, 1);
        } else {
          for (int q = 0; q < k; ++q)
            cv.page_table[(int64_t(s) * 4 + bi) * cv.max_pages + have + q] = cv.free_list[bi][top - k + q];
          *held = need;
        }
      }
    }
    __syncthreads();
    if (fail_s) {
      if (tid == 0) atomicOr(cv.status, int(TRIROUTE_CACHE_OVERFLOW));
      if (tid < 4) old_len[b * 4 + tid] = -1;
      return;
    }
  }
  if (tid < 4) old_len[b * 4 + tid] = run[tid];
  for (int t0 = 0; t0 < T; t0 += 64 * NW) {
    const int t = t0 + tid;
    const int bi = t < T ? int(bit[int64_t(b) * T + t]) : -1;
    uint64_t bal[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) bal[q] = __ballot(bi == q);
    if (lane < 4) wc[lane][w] = __popcll(bal[lane]);
    __syncthreads();
    if (bi >= 0) {
      int slot = run[bi] + __popcll(bal[bi] & lanemask_lt());
      for (int ww = 0; ww < w; ++ww) slot += wc[bi][ww];
      cv.pos_at(s, bi, slot) = len0 + t;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) run[q] += wc[q][ww];
    __syncthreads();
  }
  if (tid == 0) {
#pragma unroll
    for (int bi = 0; bi < 4; ++bi) cv.pool_len[s * 4 + bi] = run[bi];
    cv.seq_len[s] = len0 + T;
  }
}

// One token per row (decode).  The slot of a row's token (sequence s, width
// bi), in one thread:
// the checks and the page take of kv_slots_kernel for a single token; the
// token's position, the new pool and sequence lengths.  Returns the slot
// (-1: row dropped, status flagged).
__device__ int kv_slot1(const CacheView &cv, int s, int bi) {
  if (s < 0 || s >= cv.n_seq) {
    atomicOr(cv.status, int(TRIROUTE_CACHE_BAD_SEQ));
    return -1;
  }
  const int len0 = cv.seq_len[s];
  if (len0 + 1 > cv.capacity) {
    atomicOr(cv.status, int(TRIROUTE_CACHE_OVERFLOW));
    return -1;
  }
  const int run = cv.pool_len[s * 4 + bi];
  if (cv.PT) {  // paged: the page the pool grows into, from the free stack
    const int per = cv.PT * cv.TS;
    const int need = (run + 1 + per - 1) / per;
    int32_t *held = cv.alloc + s * 4 + bi;
    const int have = *held;
    if (need > have) {
      const int k = need - have;
      const int top = atomicSub(cv.free_top + bi, k);
      if (need > cv.max_pages || top - k < 0) {
        atomicAdd(cv.free_top + bi, k);  // give the claim back
        atomicOr(cv.status, int(TRIROUTE_CACHE_OVERFLOW));
        return -1;
      }
      for (int q = 0; q < k; ++q)
        cv.page_table[(int64_t(s) * 4 + bi) * cv.max_pages + have + q] = cv.free_list[bi][top - k + q];
      *held = need;
    }
  }
  cv.pos_at(s, bi, run) = len0;
  cv.pool_len[s * 4 + bi] = run + 1;
  cv.seq_len[s] = len0 + 1;
  return run;
}

// One token per row (decode), one launch: one block per row; thread 0 takes
// the slot (kv_slot1), then wave w writes kv heads w, w + 4, ...: one
// channel per lane and row of K and V (two on d_h 128): quantize (group
// min/max by lane reductions), write K codes (every 32-bit word of a K
// record belongs to one slot; the token's words are assembled in LDS, each
// lane ORs its element into its word, then one lane per word stores it),
// scales and 8/16-bit V codes (byte and half-word stores).  2- and 4-bit V
// codes share words with slots appended earlier: the token's bits of each
// word are cleared and set in place by word atomics (another row's token of
// the same word, if any, touches other bits).
template <typename T>
__global__ __launch_bounds__(256) void kv_token_kernel(CacheView cv,
                                                       const int32_t *__restrict__ seq_ids,
                                                       const T *__restrict__ kin,
                                                       const T *__restrict__ vin,
                                                       const uint8_t *__restrict__ bit) {
  __shared__ uint32_t kws[4][128];  // per wave: the token's K words (at most 4 dh bits / 32)
  __shared__ int slot_s;
  const int i = blockIdx.x;  // row i = token i
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int bi = __builtin_amdgcn_readfirstlane(int(bit[i]));
  const int s = seq_ids ? __builtin_amdgcn_readfirstlane(seq_ids[i]) : i;
  if (threadIdx.x == 0) slot_s = kv_slot1(cv, s, bi);
  __syncthreads();
  const int slot = __builtin_amdgcn_readfirstlane(slot_s);
  if (slot < 0) return;  // block-uniform: no barrier below
  uint32_t *kwv = kws[w];
  const int Hkv = cv.Hkv, dh = cv.dh, G = cv.G;
  // the wave's kv heads; the scalar bookkeeping (divisions, addresses) runs
  // on the scalar unit and the branches on the width are scalar branches
  for (int g = w; g < Hkv; g += 4) {
    // the wave's own LDS words of the previous head are read: order first
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    __builtin_amdgcn_wave_barrier();
    const int bp = cv.bits(bi);
    const int tile = slot / cv.TS, st = slot % cv.TS;
    uint8_t *tp = cv.tile(s, bi, g, tile);
    const int NR = dh >> 6;  // channels per lane: lane + 64 r
    // both rows first, so that the two loads are in flight together
    T kr[2], vr[2];
    const int64_t row = int64_t(i) * Hkv * dh + g * dh;
#pragma unroll
    for (int r = 0; r < 2; ++r)
      if (r < NR) {
        kr[r] = kin[row + lane + 64 * r];
        vr[r] = vin[row + lane + 64 * r];
      }
    const int KS = dh >> 5;
    const int blk = st >> 4, n = st & 15;
    const int per = bp == 32 ? 1 : 32 / bp;                 // elements per word
    const int q0 = blk * KS * 8, nq = KS * 8;                // this token's elements per record
    const int wpr = (nq + per - 1) / per;                    // its words per record
    const int nw = 4 * wpr;                                  // K words of the token
    for (int x = lane; x < nw; x += 64) kwv[x] = 0u;
    uint8_t *vp = tp + cv.v_codes_off(bi);
#pragma unroll
    for (int kvsel = 0; kvsel < 2; ++kvsel) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        if (r >= NR) break;
        const int c = lane + 64 * r;
        const T raw = kvsel ? vr[r] : kr[r];
        const float x = Act<T>::cvt(raw);
        uint32_t e;
        if (bi == 3) {
          if (sizeof(T) == 2)
            e = uint32_t(*(const uint16_t *)&raw);
          else
            e = __float_as_uint(x);
        } else {
          const int seg = G < 64 ? G : 64;
          const float mn = seg_min(x, seg), mx = seg_max(x, seg);
          const float levels = float((1 << bp) - 1);
          const float s32 = __fdiv_rn(mx - mn, levels);
          const _Float16 s16 = (_Float16)s32;
          const _Float16 z16 = (_Float16)mn;
          const float S = (float)s16, Z = (float)z16;
          float q = 0.f;
          if (S != 0.f) q = fminf(fmaxf(rintf(__fdiv_rn(x - Z, S)), 0.f), levels);
          e = uint32_t(q);
          if ((lane & (seg - 1)) == 0) {
            const int grp = c / G;
            const int off = (kvsel ? cv.v_sz_off(bi) : cv.k_sz_off(bi)) + (st * (dh / G) + grp) * 4;
            const uint32_t pk = uint32_t(*(const uint16_t *)&s16) | (uint32_t(*(const uint16_t *)&z16) << 16);
            *(uint32_t *)(tp + off) = pk;
          }
        }
        if (kvsel == 0) {
          // K element (slot st, channel c): record o, element q = f * 8 + j
          const int ks = c >> 5, o = (c >> 3) & 3, j = c & 7;
          const int q = (blk * KS + ks) * 8 + j;
          int wd, bt;
          q_word(q, bp, wd, bt);
          if (bp == 32)
            kwv[o * wpr + (wd - q0)] = e;
          else
            atomicOr(&kwv[o * wpr + (wd - q0 / per)], e << bt);
        } else {
          int ln, q, wd, bt;
          v_place(st, c, dh, ln, q);
          q_word(q, bp, wd, bt);
          uint8_t *addr = vp + ln * (8 * bp) + wd * 4;
          if (bp <= 4) {
            const uint32_t m = ((1u << bp) - 1u) << bt;
            atomicAnd((uint32_t *)addr, ~m);
            atomicOr((uint32_t *)addr, e << bt);
          } else if (bp == 8)
            addr[bt >> 3] = uint8_t(e);
          else if (bp == 16)
            *(uint16_t *)(addr + (bt >> 3)) = uint16_t(e);
          else
            *(uint32_t *)addr = e;
        }
      }
    }
    // the wave's own LDS words: order its ORs before its reads (no other wave
    // touches them, so no block barrier)
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    __builtin_amdgcn_wave_barrier();
    for (int x = lane; x < nw; x += 64) {
      const int o = x / wpr, wr = x % wpr;
      const int wd = q0 / per + wr;
      *(uint32_t *)(tp + (o * 16 + n) * (8 * bp) + wd * 4) = kwv[x];
    }
  }
}

// Quantizer of one group of N values held by one lane (bit exact with the
// CPU oracle, every step in IEEE fp32): codes, and the fp16 (scale, zero)
// pair packed as scale | zero << 16.
template <int BP, int N>
__device__ __forceinline__ uint32_t quantize_group(const float *x, uint32_t *code) {
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int e = 1; e < N; ++e) {
    mn = fminf(mn, x[e]);
    mx = fmaxf(mx, x[e]);
  }
  const float levels = float((1 << BP) - 1);
  const float s32 = __fdiv_rn(mx - mn, levels);
  const _Float16 s16 = (_Float16)s32;
  const _Float16 z16 = (_Float16)mn;
  const float S = (float)s16, Z = (float)z16;
#pragma unroll
  for (int e = 0; e < N; ++e) {
    float q = 0.f;
    if (S != 0.f) q = fminf(fmaxf(rintf(__fdiv_rn(x[e] - Z, S)), 0.f), levels);
    code[e] = uint32_t(q);
  }
  return uint32_t(*(const uint16_t *)&s16) | (uint32_t(*(const uint16_t *)&z16) << 16);
}

// One 32-slot step of one pool: see kv_step_kernel.  64 channels of one row
// of one token per lane; `code` holds its 64 codes (or raw values).
template <typename T, int DH, int G, int BP>
__device__ __forceinline__ void kv_step(const CacheView &cv, int s, int bi, int g, int step,
                                        int old, int nlen, int len0, int64_t row0,
                                        const T *__restrict__ kin, const T *__restrict__ vin,
                                        uint8_t *stage) {
  constexpr bool Q = BP < 16;
  constexpr int EB = Q ? 1 : BP / 8;  // staged bytes per V element
  constexpr int TS = 4096 / DH, KS = DH / 32, CB = DH / 16, NG = DH / G;
  constexpr int NIT = DH == 128 ? 2 : 1;  // 64-channel row pieces per lane
  const int lane = threadIdx.x & 63, r = lane & 31, hf = lane >> 5;
  const int Hkv = cv.Hkv;
  const int sl = step * 32 + r;
  const bool live = sl >= old && sl < nlen;
  const int tile = (step * 32) / TS, kvs = ((step * 32) % TS) / 32;  // the step within its tile
  uint8_t *tp = cv.tile(s, bi, g, tile);
  const int st = sl % TS;
  if (live) {
    const int t = cv.pos_at(s, bi, sl) - len0;  // the token at the slot's recorded position
    const int64_t rowoff = ((row0 + t) * Hkv + g) * DH;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const bool isv = NIT == 2 ? it == 1 : hf == 1;
      const int c0 = NIT == 2 ? 64 * hf : 0;
      const T *src = (isv ? vin : kin) + rowoff + c0;
      uint32_t code[64];
      if constexpr (Q) {
        float x[64];
#pragma unroll
        for (int e = 0; e < 64; e += 8) load8(src + e, x + e);
        uint8_t *szb = tp + (isv ? cv.v_sz_off(bi) : cv.k_sz_off(bi));
#pragma unroll
        for (int gg = 0; gg < 64 / G; ++gg) {
          const uint32_t sz = quantize_group<BP, G>(x + gg * G, code + gg * G);
          *(uint32_t *)(szb + (st * NG + c0 / G + gg) * 4) = sz;
        }
      } else {
        // the activation value verbatim (bf16 or fp32 bit patterns)
        const uint4 *p4 = (const uint4 *)src;
#pragma unroll
        for (int x4 = 0; x4 < 64 * int(sizeof(T)) / 16; ++x4) {
          const uint4 w = p4[x4];
          const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int y = 0; y < 4; ++y) {
            if constexpr (sizeof(T) == 2) {
              code[8 * x4 + 2 * y] = wv[y] & 0xFFFFu;
              code[8 * x4 + 2 * y + 1] = wv[y] >> 16;
            } else {
              code[4 * x4 + y] = wv[y];
            }
          }
        }
      }
      if (!isv) {
        // K: record o * 16 + st % 16 holds channel 32 ks + 8 o + j of the
        // slot as element q = 8 f + j of field f = (st / 16) KS + ks; this
        // lane's channels are fields f0 and f0 + 1 (ks = c0 / 32 + u),
        // code index 32 u + 8 o + j
        const int f0 = (st >> 4) * KS + (c0 >> 5);
#pragma unroll
        for (int o = 0; o < 4; ++o) {
          uint8_t *rec = tp + (o * 16 + (st & 15)) * 8 * BP;
          const uint32_t *c = code + 8 * o;
          if constexpr (BP == 2) {  // one word holds fields f0 (bits 4 j) and f0 + 1 (4 j + 2)
            uint32_t v = 0;
#pragma unroll
            for (int j = 0; j < 8; ++j) v |= (c[j] << (4 * j)) | (c[32 + j] << (4 * j + 2));
            *(uint32_t *)(rec + 4 * (f0 >> 1)) = v;
          } else if constexpr (BP == 4) {  // one word per field, element j at 8 (j % 4) + 4 (j / 4)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              uint32_t v = 0;
#pragma unroll
              for (int j = 0; j < 8; ++j) v |= c[32 * u + j] << (8 * (j & 3) + 4 * (j >> 2));
              *(uint32_t *)(rec + 4 * (f0 + u)) = v;
            }
          } else if constexpr (BP == 8) {  // byte q
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              uint2 v;
              v.x = c[32 * u] | (c[32 * u + 1] << 8) | (c[32 * u + 2] << 16) | (c[32 * u + 3] << 24);
              v.y = c[32 * u + 4] | (c[32 * u + 5] << 8) | (c[32 * u + 6] << 16) | (c[32 * u + 7] << 24);
              *(uint2 *)(rec + 8 * (f0 + u)) = v;
            }
          } else if constexpr (BP == 16) {  // half-word q
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              uint4 v;
              v.x = c[32 * u] | (c[32 * u + 1] << 16);
              v.y = c[32 * u + 2] | (c[32 * u + 3] << 16);
              v.z = c[32 * u + 4] | (c[32 * u + 5] << 16);
              v.w = c[32 * u + 6] | (c[32 * u + 7] << 16);
              *(uint4 *)(rec + 16 * (f0 + u)) = v;
            }
          } else {  // word q
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              *(uint4 *)(rec + 32 * (f0 + u)) = make_uint4(c[32 * u], c[32 * u + 1], c[32 * u + 2], c[32 * u + 3]);
              *(uint4 *)(rec + 32 * (f0 + u) + 16) = make_uint4(c[32 * u + 4], c[32 * u + 5], c[32 * u + 6], c[32 * u + 7]);
            }
          }
        }
      } else {
        // V codes to the wave's stage: [slot r][channel] in EB bytes
#pragma unroll
        for (int e = 0; e < 64; ++e) {
          uint8_t *d = stage + (r * DH + c0 + e) * EB;
          if constexpr (EB == 1) *d = uint8_t(code[e]);
          else if constexpr (EB == 2) *(uint16_t *)d = uint16_t(code[e]);
          else *(uint32_t *)d = code[e];
        }
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the wave's stage writes are in
  __builtin_amdgcn_wave_barrier();
  // V: record l = lane holds channel 16 cb + l % 16 of slot
  // 16 (j / 4) + 4 (l / 16) + j % 4 of the step as element q = 8 f + j of
  // field f = kvs CB + cb; build every word of the step's fields, keeping
  // the bits of slots appended before this call
  constexpr int EPW = 32 / BP;  // elements per word
  uint32_t *rec = (uint32_t *)(tp + cv.v_codes_off(bi) + lane * 8 * BP);
  const uint32_t mask = BP == 32 ? 0xFFFFFFFFu : ((1u << BP) - 1u);
#pragma unroll 4
  for (int wd = kvs * CB * 8 / EPW; wd < (kvs + 1) * CB * 8 / EPW; ++wd) {
    uint32_t word = 0, keep = 0;
    bool mine = false;  // the word holds a slot of this call (else it is left alone)
#pragma unroll
    for (int e = 0; e < EPW; ++e) {
      const int j = (wd * EPW + e) & 7;
      const int slot = step * 32 + 16 * (j >> 2) + 4 * (lane >> 4) + (j & 3);
      mine |= slot >= old && slot < nlen;
    }
    if (!mine) continue;
#pragma unroll
    for (int e = 0; e < EPW; ++e) {
      const int q = wd * EPW + e, f = q >> 3, j = q & 7;
      const int rs = 16 * (j >> 2) + 4 * (lane >> 4) + (j & 3);
      const int ch = 16 * (f - kvs * CB) + (lane & 15);
      int wq, bt;
      q_word(q, BP, wq, bt);
      const int slot = step * 32 + rs;
      if (slot < old) {
        keep |= mask << bt;
      } else if (slot < nlen) {
        const uint8_t *sp = stage + (rs * DH + ch) * EB;
        const uint32_t cv_ = EB == 1 ? *sp : EB == 2 ? *(const uint16_t *)sp : *(const uint32_t *)sp;
        word |= cv_ << bt;
      }
    }
    rec[wd] = keep ? (rec[wd] & keep) | word : word;
  }
}

// One wave per (batch row b, width pool bi, kv head g, 32-slot step j of the
// slots this append gives pool bi): lanes 0..31 take the step's slots, one
// token each (the token at the slot's recorded position); on d_h 128 lane
// half hf handles channels 64 hf .. 64 hf + 63 of both K and V, on d_h 64
// half 0 does K and half 1 does V.  A lane quantizes its 64 channels of a
// row (one or two groups of G), stores its fp16 scale/zero pairs and its
// slot's K words directly (every K word belongs to one slot), and stages its
// V codes in LDS; then each lane assembles the V words of one record, which
// hold codes of several slots, keeping the bits of slots appended before.
// A step belongs to one wave, so no two waves write a word.
template <typename T, int DH, int G>
__global__ __launch_bounds__(256) void kv_step_kernel(CacheView cv, int B, int T_, int JS,
                                                      const int32_t *__restrict__ seq_ids,
                                                      const T *__restrict__ kin,
                                                      const T *__restrict__ vin,
                                                      const int32_t *__restrict__ old_len) {
  __shared__ __align__(16) uint8_t stage_all[4][32 * DH * sizeof(T)];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int u = __builtin_amdgcn_readfirstlane(int(blockIdx.x) * 4 + wave);
  const int j = u % JS;
  u /= JS;
  const int g = u % cv.Hkv;
  u /= cv.Hkv;
  const int bi = u % 4, b = u / 4;
  if (b >= B) return;
  const int old = __builtin_amdgcn_readfirstlane(old_len[b * 4 + bi]);
  if (old < 0) return;  // row dropped (bad sequence or capacity)
  const int s = seq_ids ? __builtin_amdgcn_readfirstlane(seq_ids[b]) : b;
  const int nlen = __builtin_amdgcn_readfirstlane(cv.pool_len[s * 4 + bi]);
  const int step = old / 32 + j;
  if (step * 32 >= nlen) return;
  const int len0 = __builtin_amdgcn_readfirstlane(cv.seq_len[s]) - T_;
  uint8_t *stage = stage_all[wave];
  const int64_t row0 = int64_t(b) * T_;
  switch (bi) {
    case 0: kv_step<T, DH, G, 2>(cv, s, bi, g, step, old, nlen, len0, row0, kin, vin, stage); break;
    case 1: kv_step<T, DH, G, 4>(cv, s, bi, g, step, old, nlen, len0, row0, kin, vin, stage); break;
    case 2: kv_step<T, DH, G, 8>(cv, s, bi, g, step, old, nlen, len0, row0, kin, vin, stage); break;
    default:
      kv_step<T, DH, G, 8 * int(sizeof(T))>(cv, s, bi, g, step, old, nlen, len0, row0, kin, vin, stage);
      break;
  }
}

// Logical read-back of slots [slot0, slot0 + count) of pool (seq, bi).
template <typename T>
__global__ void kv_export_kernel(CacheView cv, int seq, int bi, int slot0, int count,
                                 uint8_t *__restrict__ kout, uint8_t *__restrict__ vout,
                                 uint16_t *__restrict__ ksz, uint16_t *__restrict__ vsz,
                                 int32_t *__restrict__ pos_out) {
  const int Hkv = cv.Hkv, dh = cv.dh, G = cv.G;
  const int64_t total = int64_t(count) * Hkv * dh;
  const int len = cv.pool_len[seq * 4 + bi];
  const int bp = cv.bits(bi);
  for (int64_t idx = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; idx < total;
       idx += int64_t(gridDim.x) * blockDim.x) {
    const int c = int(idx % dh);
    const int g = int((idx / dh) % Hkv);
    const int r = int(idx / (int64_t(dh) * Hkv));
    const int slot = slot0 + r;
    const bool live = slot < len;
    uint32_t ke = 0, ve = 0;
    uint32_t kszv = 0, vszv = 0;
    if (live) {
      const int tile = slot / cv.TS, st = slot % cv.TS;
      const uint8_t *tp = cv.tile(seq, bi, g, tile);
      int ln, q, wd, bt;
      const uint32_t mask = bp == 32 ? 0xFFFFFFFFu : ((1u << bp) - 1u);
      k_place(st, c, dh, ln, q);
      q_word(q, bp, wd, bt);
      ke = (*(const uint32_t *)(tp + ln * 8 * bp + wd * 4) >> bt) & mask;
      v_place(st, c, dh, ln, q);
      q_word(q, bp, wd, bt);
      ve = (*(const uint32_t *)(tp + cv.v_codes_off(bi) + ln * 8 * bp + wd * 4) >> bt) & mask;
      if (bi < 3 && c % G == 0) {
        kszv = *(const uint32_t *)(tp + cv.k_sz_off(bi) + (st * (dh / G) + c / G) * 4);
        vszv = *(const uint32_t *)(tp + cv.v_sz_off(bi) + (st * (dh / G) + c / G) * 4);
      }
    }
    if (bi < 3) {
      kout[idx] = uint8_t(ke);
      vout[idx] = uint8_t(ve);
      if (c % G == 0) {
        const int64_t so = ((int64_t(r) * Hkv + g) * (dh / G) + c / G) * 2;
        if (ksz) {
          ksz[so] = uint16_t(kszv);
          ksz[so + 1] = uint16_t(kszv >> 16);
        }
        if (vsz) {
          vsz[so] = uint16_t(vszv);
          vsz[so + 1] = uint16_t(vszv >> 16);
        }
      }
    } else if (sizeof(T) == 2) {
      ((uint16_t *)kout)[idx] = uint16_t(ke);
      ((uint16_t *)vout)[idx] = uint16_t(ve);
    } else {
      ((uint32_t *)kout)[idx] = ke;
      ((uint32_t *)vout)[idx] = ve;
    }
    if (pos_out && c == 0 && g == 0)
      pos_out[r] = live ? cv.pos_at(seq, bi, slot) : 0;
  }
}

__global__ __launch_bounds__(256) void kv_paged_init_kernel(CacheView cv, int n0, int n1, int n2,
                                                             int n3) {
  const int np[4] = {n0, n1, n2, n3};
  const int bi = blockIdx.y;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < np[bi]; i += gridDim.x * 256)
    cv.free_list[bi][i] = i;
  if (blockIdx.x == 0 && threadIdx.x == 0) cv.free_top[bi] = np[bi];
}

hipError_t launch_kv_paged_init(const CacheView &cv, const int32_t n_pages[4], hipStream_t st) {
  int mx = 1;
  for (int bi = 0; bi < 4; ++bi) mx = n_pages[bi] > mx ? n_pages[bi] : mx;
  const int bx = (mx + 255) / 256 < 1024 ? (mx + 255) / 256 : 1024;
  kv_paged_init_kernel<<<dim3(bx, 4), 256, 0, st>>>(cv, n_pages[0], n_pages[1], n_pages[2],
                                                    n_pages[3]);
  return hipGetLastError();
}

// Return sequence seq's pages to the free stacks and empty it (one wave per
// width: lane q pushes pages q, q + 64, ...).
__global__ __launch_bounds__(256) void kv_paged_reset_kernel(CacheView cv, int seq) {
  const int bi = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int32_t *held = cv.alloc + seq * 4 + bi;
  const int k = *held;
  int top = 0;
  if (lane == 0 && k > 0) top = atomicAdd(cv.free_top + bi, k);
  top = __shfl(top, 0, 64);
  for (int q = lane; q < k; q += 64)
    cv.free_list[bi][top + q] = cv.page_table[(int64_t(seq) * 4 + bi) * cv.max_pages + q];
  if (lane == 0) {
    *held = 0;
    cv.pool_len[seq * 4 + bi] = 0;
    if (bi == 0) cv.seq_len[seq] = 0;
  }
}

hipError_t launch_kv_paged_reset(const CacheView &cv, int seq, hipStream_t st) {
  kv_paged_reset_kernel<<<dim3(1), 256, 0, st>>>(cv, seq);
  return hipGetLastError();
}

hipError_t launch_kv_append(const triroute_cfg &cfg, const CacheView &cv, int B, int T,
                            const int32_t *seq_ids, const void *k, const void *v,
                            const uint8_t *bit, const KvWs &ws, hipStream_t st) {
  if (T == 1) {  // one token per row: slot and codes in one launch
    if (cfg.act == TRIROUTE_BF16)
      kv_token_kernel<bf16><<<B, 256, 0, st>>>(cv, seq_ids, (const bf16 *)k, (const bf16 *)v, bit);
    else
      kv_token_kernel<float><<<B, 256, 0, st>>>(cv, seq_ids, (const float *)k, (const float *)v,
                                                bit);
    return hipGetLastError();
  }
  kv_slots_kernel<<<B, 1024, 0, st>>>(cv, T, seq_ids, bit, ws.old_len);
  // 32-slot steps an append can touch in one pool: all T tokens, plus the
  // partly filled step it starts in
  const int JS = (T + 31) / 32 + 1;
  const int64_t units = int64_t(B) * 4 * cfg.n_kv_heads * JS;
  const dim3 grid(unsigned((units + 3) / 4));
  const int dh = cfg.head_dim, G = cfg.kv_group;
#define KV_STEP(TT, DH_, G_) \
  kv_step_kernel<TT, DH_, G_><<<grid, 256, 0, st>>>(cv, B, T, JS, seq_ids, (const TT *)k, (const TT *)v, ws.old_len)
#define KV_STEP_T(TT)                                  \
  do {                                                 \
    if (dh == 64) {                                    \
      if (G == 64) KV_STEP(TT, 64, 64); else KV_STEP(TT, 64, 32);    \
    } else {                                           \
      if (G == 64) KV_STEP(TT, 128, 64); else KV_STEP(TT, 128, 32);  \
    }                                                  \
  } while (0)
  if (cfg.act == TRIROUTE_BF16)
    KV_STEP_T(bf16);
  else
    KV_STEP_T(float);
#undef KV_STEP_T
#undef KV_STEP
  return hipGetLastError();
}

hipError_t launch_kv_export(const triroute_cfg &cfg, const CacheView &cv, int seq, int bi,
                            int slot0, int count, void *kout, void *vout, uint16_t *ksz,
                            uint16_t *vsz, int32_t *pos_out, hipStream_t st) {
  int64_t total = int64_t(count) * cv.Hkv * cv.dh;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  if (cfg.act == TRIROUTE_BF16)
    kv_export_kernel<bf16><<<dim3(unsigned(blocks)), 256, 0, st>>>(
        cv, seq, bi, slot0, count, (uint8_t *)kout, (uint8_t *)vout, ksz, vsz, pos_out);
  else
    kv_export_kernel<float><<<dim3(unsigned(blocks)), 256, 0, st>>>(
        cv, seq, bi, slot0, count, (uint8_t *)kout, (uint8_t *)vout, ksz, vsz, pos_out);
  return hipGetLastError();
}

}  // namespace tr
