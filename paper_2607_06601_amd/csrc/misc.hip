// Second RMSNorm and the expert combine of paper Sec. 3.1 / 3.2 (B):
//   n2 = RMSNorm(xt; g2);  x_out = xt + sum_{slot: e != 0} gate * Y[i*k + slot]
// Slots are summed in slot order (deterministic); a token whose every slot is
// the null expert gets x_out = xt exactly.  The expert GEMMs take n2 and give
// Y in list order (one row per entry of the expert lists, lists back to
// back), so the normalisation writes each token's normalised row to the list
// rows of its assignments and records where each assignment's row went.
#include "kernels.hpp"

namespace tr {

// Few tokens (decode): one wave per list entry pos (8 consecutive elements
// per lane access, d % 64 == 0): token a / k of assignment a = rows[pos],
// normalised, to row pos; slot_of[a] = pos (one launch instead of two; the
// same arithmetic as moe_norm_tok, so the same n2).  Entries past the lists' total do nothing.  The
// norm is evaluated in fp64 (sum of squares, scale, products) and rounded
// once to the activation dtype, so n2 is the correctly rounded value of the
// exact norm: a last-place difference in n2 would otherwise move the expert
// output by far more than its own size.
template <typename T>
__global__ __launch_bounds__(256) void moe_norm_rows_kernel(
    const T *__restrict__ x, const T *__restrict__ g, const int32_t *__restrict__ rows,
    const int32_t *__restrict__ off, int E, int k, int Nk, T *__restrict__ out,
    int32_t *__restrict__ slot_of, int d, float eps) {
  const int pos = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  if (pos >= Nk || pos >= off[E]) return;  // off[E]: end of the last list
  const int a = rows[pos];
  const T *xr = x + int64_t(a / k) * d;
  // rows of up to 1024 elements stay in registers between the two passes
  constexpr int RR = 2;
  float v[RR][8];
  double ss = 0.0;
  if (d <= 512 * RR) {
#pragma unroll
    for (int q = 0; q < RR; ++q) {
      const int c = lane * 8 + 512 * q;
      if (c < d) {
        load8(xr + c, v[q]);
#pragma unroll
        for (int i = 0; i < 8; ++i) ss = fma(double(v[q][i]), double(v[q][i]), ss);
      }
    }
  } else {
    for (int c = lane * 8; c < d; c += 512) {
      float w[8];
      load8(xr + c, w);
#pragma unroll
      for (int i = 0; i < 8; ++i) ss = fma(double(w[i]), double(w[i]), ss);
    }
  }
  ss = wave_sum(ss);
  const double r = 1.0 / sqrt(ss / double(d) + double(eps));
  T *orow = out + int64_t(pos) * d;
  if (d <= 512 * RR) {
#pragma unroll
    for (int q = 0; q < RR; ++q) {
      const int c = lane * 8 + 512 * q;
      if (c < d) {
        float gv[8];
        double o[8];
        load8(g + c, gv);
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = (double(v[q][i]) * r) * double(gv[i]);
        store8(orow + c, o);
      }
    }
  } else {
    for (int c = lane * 8; c < d; c += 512) {
      float w[8], gv[8];
      double o[8];
      load8(xr + c, w);
      load8(g + c, gv);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = (double(w[i]) * r) * double(gv[i]);
      store8(orow + c, o);
    }
  }
  if (lane == 0) slot_of[a] = pos;
}

// List row of every real assignment: slot_of[rows[pos]] = pos for each
// entry pos of the expert lists (one thread per entry).
__global__ __launch_bounds__(256) void moe_slot_of_kernel(const int32_t *__restrict__ rows,
                                                          const int32_t *__restrict__ off, int E,
                                                          int Nk, int32_t *__restrict__ slot_of) {
  const int pos = blockIdx.x * 256 + threadIdx.x;
  if (pos < Nk && pos < off[E]) slot_of[rows[pos]] = pos;  // off[E]: end of the last list
}

// One wave per token i (8 consecutive elements per lane access,
// d % 64 == 0): the row is read once (kept in registers when
// d <= 512 RR, read again for the products otherwise), normalised, and
// written to the list row of each of the token's real assignments.  The
// norm is evaluated in fp64 (sum of squares, scale, products) and rounded
// once to the activation dtype, so n2 is the correctly rounded value of the
// exact norm: a last-place difference in n2 would otherwise move the expert
// output by far more than its own size.
template <typename T, int RR>
__global__ __launch_bounds__(256) void moe_norm_tok_kernel(
    const T *__restrict__ x, const T *__restrict__ g, const int32_t *__restrict__ eidx,
    const int32_t *__restrict__ slot_of, int N, int k, T *__restrict__ out, int d, float eps) {
  const int i = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  if (i >= N) return;
  const T *xr = x + int64_t(i) * d;
  const int32_t *ei = eidx + int64_t(i) * k, *so = slot_of + int64_t(i) * k;
  float v[RR > 0 ? RR : 1][8];
  double ss = 0.0;
  if constexpr (RR > 0) {
#pragma unroll
    for (int q = 0; q < RR; ++q) {
      const int c = lane * 8 + 512 * q;
      if (c < d) {
        load8(xr + c, v[q]);
#pragma unroll
        for (int j = 0; j < 8; ++j) ss = fma(double(v[q][j]), double(v[q][j]), ss);
      }
    }
  } else {
    for (int c = lane * 8; c < d; c += 512) {
      float w[8];
      load8(xr + c, w);
#pragma unroll
      for (int j = 0; j < 8; ++j) ss = fma(double(w[j]), double(w[j]), ss);
    }
  }
  ss = wave_sum(ss);
  const double r = 1.0 / sqrt(ss / double(d) + double(eps));
  // products of the 8 elements at c, rounded, to every real assignment's row
  auto emit = [&](int c, const float *w) {
    float gv[8];
    double o[8];
    load8(g + c, gv);
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = (double(w[j]) * r) * double(gv[j]);
    for (int s = 0; s < k; ++s)
      if (ei[s] != 0) store8(out + int64_t(so[s]) * d + c, o);
  };
  if constexpr (RR > 0) {
#pragma unroll
    for (int q = 0; q < RR; ++q) {
      const int c = lane * 8 + 512 * q;
      if (c < d) emit(c, v[q]);
    }
  } else {
    for (int c = lane * 8; c < d; c += 512) {
      float w[8];
      load8(xr + c, w);
      emit(c, w);
    }
  }
}

// One thread per 8 consecutive features of a token.
template <typename T>
__global__ __launch_bounds__(256) void moe_combine_kernel(const T *__restrict__ xt,
                                                          const float *__restrict__ Y,
                                                          const int32_t *__restrict__ slot_of,
                                                          int ysplit, int64_t yplane,
                                                          const int32_t *__restrict__ eidx,
                                                          const float *__restrict__ egate,
                                                          T *__restrict__ xout, int N, int d,
                                                          int k) {
  const int d8 = d >> 3;
  const int64_t total = int64_t(N) * d8;
  for (int64_t it = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; it < total;
       it += int64_t(gridDim.x) * blockDim.x) {
    const int i = int(it / d8), c = int(it % d8) * 8;
    float acc[8], y[8];
    load8(xt + int64_t(i) * d + c, acc);
#pragma unroll
    for (int u = 0; u < 8; ++u) y[u] = 0.f;
    bool any = false;
    for (int s = 0; s < k; ++s) {
      if (eidx[int64_t(i) * k + s] == 0) continue;
      const float gt = egate[int64_t(i) * k + s];
      float ys[8];
      const float *yr = Y + int64_t(slot_of[int64_t(i) * k + s]) * d + c;
      load8(yr, ys);
      if (ysplit == 2) {  // the second K half's plane, added in order
        float y2[8];
        load8(yr + yplane, y2);
#pragma unroll
        for (int u = 0; u < 8; ++u) ys[u] += y2[u];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) y[u] = fmaf(gt, ys[u], y[u]);
      any = true;
    }
    if (any) {
#pragma unroll
      for (int u = 0; u < 8; ++u) acc[u] += y[u];
    }
    store8(xout + int64_t(i) * d + c, acc);
  }
}

hipError_t launch_moe_norm_rows(const triroute_cfg &cfg, int N, const void *x, const void *g,
                                const triroute_compaction &c, const int32_t *eidx, void *out,
                                int32_t *slot_of, hipStream_t st) {
  const int k = cfg.top_k, Nk = N * k, E = cfg.n_experts, d = cfg.d_model;
  if (Nk <= 2048) {  // few tokens: the launch costs more than normalising a row twice
    if (Nk == 0) return hipSuccess;
    const dim3 g1((Nk + 3) / 4);
    if (cfg.act == TRIROUTE_BF16)
      moe_norm_rows_kernel<bf16><<<g1, 256, 0, st>>>((const bf16 *)x, (const bf16 *)g, c.exp_rows,
                                                     c.exp_off, E, k, Nk, (bf16 *)out, slot_of, d,
                                                     cfg.rms_eps);
    else
      moe_norm_rows_kernel<float><<<g1, 256, 0, st>>>((const float *)x, (const float *)g,
                                                      c.exp_rows, c.exp_off, E, k, Nk,
                                                      (float *)out, slot_of, d, cfg.rms_eps);
    return hipGetLastError();
  }
  moe_slot_of_kernel<<<(Nk + 255) / 256, 256, 0, st>>>(c.exp_rows, c.exp_off, E, Nk, slot_of);
  const dim3 grid((N + 3) / 4);
  auto run = [&](auto tag, auto rr) {
    using T = decltype(tag);
    moe_norm_tok_kernel<T, decltype(rr)::value><<<grid, 256, 0, st>>>(
        (const T *)x, (const T *)g, eidx, slot_of, N, k, (T *)out, d, cfg.rms_eps);
  };
  auto by_width = [&](auto tag) {
    if (d <= 512) run(tag, std::integral_constant<int, 1>{});
    else if (d <= 1024) run(tag, std::integral_constant<int, 2>{});
    else if (d <= 2048) run(tag, std::integral_constant<int, 4>{});
    else run(tag, std::integral_constant<int, 0>{});
  };
  if (cfg.act == TRIROUTE_BF16) by_width(bf16{});
  else by_width(float{});
  return hipGetLastError();
}

hipError_t launch_moe_combine(const triroute_cfg &cfg, int N, const void *xt, const float *Y,
                              const int32_t *slot_of, const int32_t *eidx, const float *egate, void *xout,
                              hipStream_t st) {
  int64_t total = int64_t(N) * (cfg.d_model / 8);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (cfg.act == TRIROUTE_BF16)
    moe_combine_kernel<bf16><<<dim3(unsigned(blocks)), 256, 0, st>>>(
        (const bf16 *)xt, Y, slot_of, moe_ysplit(cfg, N), int64_t(N) * cfg.top_k * cfg.d_model, eidx, egate, (bf16 *)xout, N, cfg.d_model, cfg.top_k);
  else
    moe_combine_kernel<float><<<dim3(unsigned(blocks)), 256, 0, st>>>(
        (const float *)xt, Y, slot_of, moe_ysplit(cfg, N), int64_t(N) * cfg.top_k * cfg.d_model, eidx, egate, (float *)xout, N, cfg.d_model, cfg.top_k);
  return hipGetLastError();
}

// The attention output rows the prefill kernels leave unwritten, zeroed:
// skipped heads (any mode but local or full), and every head of a row whose
// sequence id lies outside the cache (that row is dropped and flagged).  One
// thread per (token, head) row, writing its 16-byte chunks only when the row
// needs zeros; rows of attended heads are not touched.
__global__ __launch_bounds__(256) void attn_zero_rows_kernel(uint4 *__restrict__ o,
                                                             const uint8_t *__restrict__ mode,
                                                             const int32_t *__restrict__ seq_ids,
                                                             int n_seq, uint32_t row_tokens,
                                                             int chunks, uint32_t pairs) {
  const uint32_t pair = blockIdx.x * 256u + threadIdx.x;  // token * H + head (< 2^31, host)
  if (pair >= pairs) return;
  const int b = int(pair / row_tokens);  // row_tokens = H T pairs per batch row
  const int s = seq_ids ? seq_ids[b] : b;
  const int m = mode[pair];  // anything but local or full is in no attention list
  if ((m != TRIROUTE_LOCAL && m != TRIROUTE_FULL) || s < 0 || s >= n_seq) {
    uint4 *row = o + size_t(pair) * chunks;
    for (int c = 0; c < chunks; ++c) row[c] = make_uint4(0u, 0u, 0u, 0u);
  }
}

hipError_t launch_attn_zero_rows(const triroute_cfg &cfg, int B, int T, const uint8_t *mode,
                                 const int32_t *seq_ids, int n_seq, void *o, hipStream_t st) {
  const int chunks = cfg.head_dim * (cfg.act == TRIROUTE_BF16 ? 2 : 4) / 16;
  const int64_t pairs = int64_t(B) * T * cfg.n_heads;
  if (pairs <= 0) return hipSuccess;
  if (pairs >= (int64_t(1) << 31)) return launch_fill_u32(o, pairs * chunks * 4, 0u, st);  // every row
  attn_zero_rows_kernel<<<dim3(unsigned((pairs + 255) / 256)), 256, 0, st>>>(
      (uint4 *)o, mode, seq_ids, n_seq, uint32_t(cfg.n_heads) * uint32_t(T), chunks,
      uint32_t(pairs));
  return hipGetLastError();
}

// Side features of the next layer of a stack (Sec. 3.3: the previous
// layer's decisions among them): the caller's features with the last four
// replaced by this token's decisions in the layer just run, as exact fp32
// quotients: full heads / H, local heads / H, width index / 3, real expert
// slots / k.  One thread per token.
__global__ __launch_bounds__(256) void psi_next_kernel(const float *__restrict__ psi,
                                                       const uint8_t *__restrict__ mode,
                                                       const uint8_t *__restrict__ bit,
                                                       const int32_t *__restrict__ eidx,
                                                       float *__restrict__ out, int N, int dpsi,
                                                       int H, int k) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= N) return;
  for (int j = 0; j < dpsi - 4; ++j) out[int64_t(t) * dpsi + j] = psi[int64_t(t) * dpsi + j];
  int full = 0, local = 0, real = 0;
  for (int h = 0; h < H; ++h) {
    const int m = mode[int64_t(t) * H + h];
    full += m == TRIROUTE_FULL;
    local += m == TRIROUTE_LOCAL;
  }
  for (int j = 0; j < k; ++j) real += eidx[int64_t(t) * k + j] != 0;
  float *o = out + int64_t(t) * dpsi + dpsi - 4;
  o[0] = float(full) / float(H);
  o[1] = float(local) / float(H);
  o[2] = float(bit[t]) / 3.0f;
  o[3] = float(real) / float(k);
}

hipError_t launch_psi_next(const triroute_cfg &cfg, int N, const float *psi, const uint8_t *mode,
                           const uint8_t *bit, const int32_t *eidx, float *out, hipStream_t st) {
  psi_next_kernel<<<dim3((N + 255) / 256), 256, 0, st>>>(psi, mode, bit, eidx, out, N, cfg.d_psi,
                                                         cfg.n_heads, cfg.top_k);
  return hipGetLastError();
}

}  // namespace tr
