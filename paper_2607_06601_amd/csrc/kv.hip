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

// Per batch row: slots in each width pool, positions, new lengths.
__global__ __launch_bounds__(256) void kv_slots_kernel(CacheView cv, int T,
                                                       const int32_t *__restrict__ seq_ids,
                                                       const uint8_t *__restrict__ bit,
                                                       int32_t *__restrict__ slots,
                                                       int32_t *__restrict__ old_len) {
  __shared__ int wc[4][4];
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int s = seq_ids ? seq_ids[b] : b;
  if (s < 0 || s >= cv.n_seq) {
    if (tid == 0) atomicOr(cv.status, int(TRIROUTE_CACHE_BAD_SEQ));
    if (tid < 4) old_len[b * 4 + tid] = -1;
    for (int t = tid; t < T; t += 256) slots[int64_t(b) * T + t] = -1;
    return;
  }
  const int len0 = cv.seq_len[s];
  if (len0 + T > cv.capacity) {
    if (tid == 0) atomicOr(cv.status, int(TRIROUTE_CACHE_OVERFLOW));
    if (tid < 4) old_len[b * 4 + tid] = -1;
    for (int t = tid; t < T; t += 256) slots[int64_t(b) * T + t] = -1;
    return;
  }
  int run[4];
#pragma unroll
  for (int bi = 0; bi < 4; ++bi) run[bi] = cv.pool_len[s * 4 + bi];
  if (tid < 4) old_len[b * 4 + tid] = run[tid];
  for (int t0 = 0; t0 < T; t0 += 256) {
    const int t = t0 + tid;
    const int bi = t < T ? int(bit[int64_t(b) * T + t]) : -1;
    uint64_t bal[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) bal[q] = __ballot(bi == q);
    if (lane == 0)
#pragma unroll
      for (int q = 0; q < 4; ++q) wc[q][w] = __popcll(bal[q]);
    __syncthreads();
    if (bi >= 0) {
      int slot = run[bi] + __popcll(bal[bi] & lanemask_lt());
      for (int ww = 0; ww < w; ++ww) slot += wc[bi][ww];
      slots[int64_t(b) * T + t] = slot;
      cv.pos_of(s, bi)[slot] = len0 + t;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) run[q] += wc[q][0] + wc[q][1] + wc[q][2] + wc[q][3];
    __syncthreads();
  }
  if (tid == 0) {
#pragma unroll
    for (int bi = 0; bi < 4; ++bi) cv.pool_len[s * 4 + bi] = run[bi];
    cv.seq_len[s] = len0 + T;
  }
}

// One wave per (token, kv head): quantize K and V, write K codes (every
// 32-bit word of a K record belongs to one slot), scales and 8/16-bit V
// codes (byte and half-word stores); 2- and 4-bit V codes share words with
// neighbouring slots and go to vstage, one byte per element, for
// kv_vpack_kernel (single-token rows: in place, by word atomics).  The K
// words of the token are assembled in LDS: each lane ORs its element into
// its word, then one lane per word stores it.
template <typename T>
__global__ __launch_bounds__(256) void kv_write_kernel(CacheView cv, int T_, int N,
                                                       const int32_t *__restrict__ seq_ids,
                                                       const T *__restrict__ kin,
                                                       const T *__restrict__ vin,
                                                       const uint8_t *__restrict__ bit,
                                                       const int32_t *__restrict__ slots,
                                                       uint8_t *__restrict__ vstage) {
  __shared__ uint32_t kw[4][128];  // per wave: the token's K words (at most 4 dh bits... / 32)
  // the wave index, and all that follows from it, in scalar registers: the
  // per-(token, head) bookkeeping (divisions, addresses) runs on the scalar
  // unit and the branches on the width are scalar branches
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int item = blockIdx.x * 4 + w;
  const int Hkv = cv.Hkv, dh = cv.dh, G = cv.G;
  const int i = item / Hkv, g = item % Hkv;
  const int slot = item < N * Hkv ? __builtin_amdgcn_readfirstlane(slots[i]) : -1;
  if (slot < 0) return;  // wave-uniform: nothing of this wave touches LDS or a barrier
  const int b = i / T_;
  const int s = seq_ids ? __builtin_amdgcn_readfirstlane(seq_ids[b]) : b;
  const int bi = __builtin_amdgcn_readfirstlane(int(bit[i]));
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
  for (int x = lane; x < nw; x += 64) kw[w][x] = 0u;
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
          kw[w][o * wpr + (wd - q0)] = e;
        else
          atomicOr(&kw[w][o * wpr + (wd - q0 / per)], e << bt);
      } else {
        int ln, q, wd, bt;
        v_place(st, c, dh, ln, q);
        q_word(q, bp, wd, bt);
        uint8_t *addr = vp + ln * (8 * bp) + wd * 4;
        if (bp <= 4) {
          if (T_ == 1) {
            // one new token per row: its bits of the shared word are cleared
            // and set in place (another row's token of the same word, if
            // any, touches other bits), and kv_vpack is not needed
            const uint32_t m = ((1u << bp) - 1u) << bt;
            atomicAnd((uint32_t *)addr, ~m);
            atomicOr((uint32_t *)addr, e << bt);
          } else {
            vstage[(int64_t(i) * Hkv + g) * dh + c] = uint8_t(e);
          }
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
    *(uint32_t *)(tp + (o * 16 + n) * (8 * bp) + wd * 4) = kw[w][x];
  }
}

// 2- and 4-bit V words: one wave per (batch row, pool, kv head, 32-slot
// step of the appended range).  A step's words hold only that step's slots,
// so the wave owns them: lane l builds the words of its record l from the
// staged codes of the new slots and keeps the bits of slots appended before.
__global__ __launch_bounds__(256) void kv_vpack_kernel(CacheView cv, int B, int T, int JS,
                                                       const int32_t *__restrict__ seq_ids,
                                                       const int32_t *__restrict__ old_len,
                                                       const uint8_t *__restrict__ vstage) {
  const int lane = threadIdx.x & 63;
  int u = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // scalar bookkeeping
  const int j = u % JS;
  u /= JS;
  const int g = u % cv.Hkv;
  u /= cv.Hkv;
  const int bi = u % 2, b = u / 2;
  if (b >= B) return;
  const int s = seq_ids ? seq_ids[b] : b;
  const int old = old_len[b * 4 + bi];
  if (old < 0) return;  // row dropped (bad sequence or capacity)
  const int nlen = cv.pool_len[s * 4 + bi];
  const int step = old / 32 + j;
  if (step * 32 >= nlen) return;
  const int bp = 2 << bi, dh = cv.dh, TS = cv.TS, CB = dh / 16;
  const int len0 = cv.seq_len[s] - T;
  const int32_t *pos = cv.pos_of(s, bi);
  // token of each slot of the step (lanes 0..31), shuffled to the elements
  const int sl = step * 32 + (lane & 31);
  const int tok = (sl >= old && sl < nlen) ? b * T + (pos[sl] - len0) : -1;
  const int tile = step * 32 / TS, kv = (step * 32 % TS) / 32;
  uint32_t *rec = (uint32_t *)(cv.tile(s, bi, g, tile) + cv.v_codes_off(bi) + lane * 8 * bp);
  const int per = 16 / bp;  // element pairs per word
  const int w0 = kv * CB * 8 / (2 * per), w1 = (kv + 1) * CB * 8 / (2 * per);
  for (int wd = w0; wd < w1; ++wd) {
    uint32_t word = 0, keep = 0;
    for (int h = 0; h < 2 * per; ++h) {
      const int q = 2 * (wd * per + (h >> 1)) + (h & 1);
      const int f = q >> 3, jj = q & 7;
      const int sis = 16 * (jj >> 2) + 4 * (lane >> 4) + (jj & 3);  // slot within the step
      const int ch = 16 * (f % CB) + (lane & 15);
      int wq, bt;
      q_word(q, bp, wq, bt);
      const int slot = step * 32 + sis;
      const int t = __shfl(tok, sis, 64);
      if (slot < old)
        keep |= ((1u << bp) - 1u) << bt;
      else if (t >= 0)
        word |= uint32_t(vstage[(int64_t(t) * cv.Hkv + g) * dh + ch]) << bt;
    }
    rec[wd] = keep ? (rec[wd] & keep) | word : word;
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
      pos_out[r] = live ? cv.pos_of(seq, bi)[slot] : 0;
  }
}

hipError_t launch_kv_append(const triroute_cfg &cfg, const CacheView &cv, int B, int T,
                            const int32_t *seq_ids, const void *k, const void *v,
                            const uint8_t *bit, const KvWs &ws, hipStream_t st) {
  kv_slots_kernel<<<B, 256, 0, st>>>(cv, T, seq_ids, bit, ws.slots, ws.old_len);
  const int N = B * T;
  dim3 grid((N * cfg.n_kv_heads + 3) / 4);
  if (cfg.act == TRIROUTE_BF16)
    kv_write_kernel<bf16><<<grid, 256, 0, st>>>(cv, T, N, seq_ids, (const bf16 *)k,
                                                (const bf16 *)v, bit, ws.slots, ws.vstage);
  else
    kv_write_kernel<float><<<grid, 256, 0, st>>>(cv, T, N, seq_ids, (const float *)k,
                                                 (const float *)v, bit, ws.slots, ws.vstage);
  // 32-slot steps an append can touch in one pool: all T tokens, plus the
  // partly filled step it starts in
  const int JS = (T + 31) / 32 + 1;
  const int64_t units = int64_t(B) * 2 * cfg.n_kv_heads * JS;
  if (T > 1)  // single-token rows wrote their 2- and 4-bit V codes in place
    kv_vpack_kernel<<<dim3(unsigned((units + 3) / 4)), 256, 0, st>>>(cv, B, T, JS, seq_ids,
                                                                      ws.old_len, ws.vstage);
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
