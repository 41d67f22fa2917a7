// Routed attention over the mixed-width cache, vector-ALU form (one wave per
// query head; any act dtype).  Paper Sec. 3.2 (A): query head h of a token at
// position P reads kv head h / (H / Hkv); skip -> 0, local -> keys
// [P - w + 1, P], full -> [0, P]; softmax(q k^T / sqrt(dh)) v over the
// dequantized cache, the token's own key included.
#include "kernels.hpp"

namespace tr {

// First slot of pool (s, bi) whose position is >= p (positions ascend).
__device__ __forceinline__ int pool_lower_bound(const CacheView &cv, int s, int bi, int len,
                                                int p) {
  int lo = 0, hi = len;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (cv.pos_at(s, bi, mid) < p)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

// Dequantized K or V element (slot, channel) of a tile.
__device__ __forceinline__ float cache_elem(const CacheView &cv, const uint8_t *tp, int bi,
                                            int st, int c, bool isv) {
  const int bp = cv.bits(bi);
  int ln, q, wd, bt;
  if (isv)
    v_place(st, c, cv.dh, ln, q);
  else
    k_place(st, c, cv.dh, ln, q);
  q_word(q, bp, wd, bt);
  const uint8_t *rec = tp + (isv ? cv.v_codes_off(bi) : 0) + ln * 8 * bp;
  const uint32_t wv = *(const uint32_t *)(rec + wd * 4);
  if (bi == 3) {
    if (bp == 16) return __uint_as_float(((wv >> bt) & 0xFFFFu) << 16);
    return __uint_as_float(wv);
  }
  const uint32_t code = (wv >> bt) & ((1u << bp) - 1u);
  const int G = cv.G;
  const uint32_t sz =
      *(const uint32_t *)(tp + (isv ? cv.v_sz_off(bi) : cv.k_sz_off(bi)) + (st * (cv.dh / G) + c / G) * 4);
  const uint16_t sb = uint16_t(sz), zb = uint16_t(sz >> 16);
  const float S = float(*(const _Float16 *)&sb), Z = float(*(const _Float16 *)&zb);
  return float(code) * S + Z;
}

struct AttnQuery {
  int row;  // token row in q / o / mode
  int s;    // cache sequence
  int P;    // query position
  int h, m;
};

template <typename T>
__device__ void attend_one(const CacheView &cv, const T *__restrict__ q, T *__restrict__ o,
                           const AttnQuery &aq, int H, int w) {
  const int lane = threadIdx.x & 63;
  const int dh = cv.dh, NR = dh >> 6;
  const int g = aq.h / (H / cv.Hkv);
  const float scale = 1.0f / sqrtf(float(dh));
  float qv[2], acc[2] = {0.f, 0.f};
  for (int r = 0; r < NR; ++r)
    qv[r] = Act<T>::ld(q, (int64_t(aq.row) * H + aq.h) * dh + lane + 64 * r) * scale;
  const int lo = aq.m == TRIROUTE_LOCAL ? max(0, aq.P - w + 1) : 0;
  float mrun = -INFINITY, l = 0.f;
  for (int bi = 0; bi < 4; ++bi) {
    const int len = cv.pool_len[aq.s * 4 + bi];
    const int a = pool_lower_bound(cv, aq.s, bi, len, lo);
    const int e = pool_lower_bound(cv, aq.s, bi, len, aq.P + 1);
    for (int slot = a; slot < e; ++slot) {
      const uint8_t *tp = cv.tile(aq.s, bi, g, slot / cv.TS);
      const int st = slot % cv.TS;
      float part = 0.f;
      for (int r = 0; r < NR; ++r) part = fmaf(qv[r], cache_elem(cv, tp, bi, st, lane + 64 * r, false), part);
      const float sc = wave_sum(part);
      const float mn = fmaxf(mrun, sc);
      const float corr = expf(mrun - mn), pw = expf(sc - mn);
      l = l * corr + pw;
      for (int r = 0; r < NR; ++r)
        acc[r] = acc[r] * corr + pw * cache_elem(cv, tp, bi, st, lane + 64 * r, true);
      mrun = mn;
    }
  }
  const float inv = l > 0.f ? 1.0f / l : 0.f;
  for (int r = 0; r < NR; ++r)
    Act<T>::st(o, (int64_t(aq.row) * H + aq.h) * dh + lane + 64 * r, acc[r] * inv);
}

// Prefill: wave item -> (segment, index in segment).
template <typename T>
__global__ __launch_bounds__(256) void attn_valu_prefill_kernel(
    CacheView cv, int B, int Tq, int H, int w, const int32_t *__restrict__ seq_ids,
    const T *__restrict__ q, const int32_t *__restrict__ cnt, const int32_t *__restrict__ idx,
    T *__restrict__ o) {
  const int64_t item = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nseg = B * H * 2;
  if (item >= int64_t(nseg) * Tq) return;
  const int seg = int(item / Tq), j = int(item % Tq);
  if (j >= cnt[seg]) return;
  AttnQuery aq;
  const int b = seg / (2 * H);
  aq.h = (seg >> 1) % H;
  aq.m = (seg & 1) + 1;
  const int t = idx[int64_t(seg) * Tq + j];
  aq.row = b * Tq + t;
  aq.s = seq_ids ? seq_ids[b] : b;
  if (aq.s < 0 || aq.s >= cv.n_seq) return;
  aq.P = cv.seq_len[aq.s] - Tq + t;
  attend_one<T>(cv, q, o, aq, H, w);
}

// Decode: wave item -> (b, h); skip heads write zeros.
template <typename T>
__global__ __launch_bounds__(256) void attn_valu_decode_kernel(CacheView cv, int B, int H, int w,
                                                               const int32_t *__restrict__ seq_ids,
                                                               const T *__restrict__ q,
                                                               const uint8_t *__restrict__ mode,
                                                               T *__restrict__ o) {
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= B * H) return;
  AttnQuery aq;
  const int b = item / H;
  aq.h = item % H;
  aq.m = mode[item];
  aq.row = b;
  aq.s = seq_ids ? seq_ids[b] : b;
  const bool bad = aq.s < 0 || aq.s >= cv.n_seq;
  aq.P = bad ? 0 : cv.seq_len[aq.s] - 1;
  if (aq.m == TRIROUTE_SKIP || bad) {
    const int lane = threadIdx.x & 63;
    for (int c = lane; c < cv.dh; c += 64) Act<T>::st(o, int64_t(item) * cv.dh + c, 0.f);
    return;
  }
  attend_one<T>(cv, q, o, aq, H, w);
}

hipError_t launch_attn_valu_prefill(const triroute_cfg &cfg, const CacheView &cv, int B, int Tq,
                                    const int32_t *seq_ids, const void *q,
                                    const triroute_compaction &c, void *o, hipStream_t st) {
  const int64_t items = int64_t(B) * cfg.n_heads * 2 * Tq;
  dim3 grid(unsigned((items + 3) / 4));
  if (cfg.act == TRIROUTE_BF16)
    attn_valu_prefill_kernel<bf16><<<grid, 256, 0, st>>>(cv, B, Tq, cfg.n_heads, cfg.window,
                                                         seq_ids, (const bf16 *)q, c.attn_cnt,
                                                         c.attn_idx, (bf16 *)o);
  else
    attn_valu_prefill_kernel<float><<<grid, 256, 0, st>>>(cv, B, Tq, cfg.n_heads, cfg.window,
                                                          seq_ids, (const float *)q, c.attn_cnt,
                                                          c.attn_idx, (float *)o);
  return hipGetLastError();
}

hipError_t launch_attn_valu_decode(const triroute_cfg &cfg, const CacheView &cv, int B,
                                   const int32_t *seq_ids, const void *q, const uint8_t *mode,
                                   void *o, hipStream_t st) {
  dim3 grid(unsigned((B * cfg.n_heads + 3) / 4));
  if (cfg.act == TRIROUTE_BF16)
    attn_valu_decode_kernel<bf16><<<grid, 256, 0, st>>>(cv, B, cfg.n_heads, cfg.window, seq_ids,
                                                        (const bf16 *)q, mode, (bf16 *)o);
  else
    attn_valu_decode_kernel<float><<<grid, 256, 0, st>>>(cv, B, cfg.n_heads, cfg.window,
                                                         seq_ids, (const float *)q, mode,
                                                         (float *)o);
  return hipGetLastError();
}

}  // namespace tr
