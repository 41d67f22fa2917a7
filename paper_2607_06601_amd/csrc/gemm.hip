// Dense and grouped GEMMs of the layer for the fp32 activation dtype (the bf16
// path is gemm_mfma.hip), C = A B^T with both operands K-contiguous, and
// their fused epilogues:
//   QKV   : [n1] x [Wq;Wk;Wv]^T, rotate-half RoPE on q and k
//   O-proj: xt = x + o Wo^T
//   MoE-1 : H = silu(n2 Wgate_e^T) * (n2 Wup_e^T) per expert e (paper Sec.
//           3.2 (B), SwiGLU); n2, H and Y hold one row per entry of the
//           expert lists, in list order (the lists lie back to back)
//   MoE-2 : Y = H Wdown_e^T
// A VALU tiled kernel.  Grouped problems map block -> (expert, row tile) from
// the device-side expert counts, so no host synchronisation is needed.
#include <type_traits>

#include "kernels.hpp"

namespace tr {


struct Tile {
  int m0, n0, mvalid, e, p0;
};

// ------------------------------------------------------------------ problems
template <typename T>
struct QkvProb {
  typedef T elem;
  const T *n1, *Wq, *Wk, *Wv;
  T *q, *k, *v;
  const float2 *rope;  // (cos, sin) of token row, pair j at row * dh / 2 + j
  int N, d, H, Hkv, dh, K, Ncols;
  __device__ bool map(int bx, int by, int BM, Tile &t) const {
    t.m0 = bx * BM;
    t.n0 = by * 128;
    t.mvalid = min(BM, N - t.m0);
    t.e = 0;
    t.p0 = 0;
    return t.mvalid > 0;
  }
  __device__ const T *a_row(const Tile &t, int r) const { return n1 + int64_t(t.m0 + r) * d; }
  __device__ const T *b_row(const Tile &t, int n) const {
    int gc = t.n0 + n;
    const int Hd = H * dh, Kd = Hkv * dh;
    if (gc < Hd) return Wq + int64_t(gc) * d;
    gc -= Hd;
    if (gc < Kd) return Wk + int64_t(gc) * d;
    gc -= Kd;
    if (gc < Kd) return Wv + int64_t(gc) * d;
    return nullptr;
  }
  __device__ void epilogue(const Tile &t, const float *C, int ldc, int r0, int nr,
                           int tid) const {
    const int Hd = H * dh, Kd = Hkv * dh, half = dh >> 1;
    for (int idx = tid; idx < nr * 128; idx += 256) {
      const int r = idx >> 7, c = idx & 127;
      const int row = t.m0 + r0 + r;
      const int gc = t.n0 + c;
      if (r0 + r >= t.mvalid || gc >= Ncols) continue;
      const float x = C[r * ldc + c];
      T *out;
      int ld, col;
      bool rot = true;
      if (gc < Hd) {
        out = q; ld = Hd; col = gc;
      } else if (gc < Hd + Kd) {
        out = k; ld = Kd; col = gc - Hd;
      } else {
        out = v; ld = Kd; col = gc - Hd - Kd; rot = false;
      }
      float y = x;
      if (rot) {
        const int j = col % dh, jj = j % half;
        const float xp = C[r * ldc + (j < half ? c + half : c - half)];
        const float2 a = rope[int64_t(row) * half + jj];
        const float cs = a.x, sn = a.y;
        y = j < half ? x * cs - xp * sn : xp * sn + x * cs;
      }
      Act<T>::st(out, int64_t(row) * ld + col, y);
    }
  }
};

template <typename T>
struct OprojProb {
  typedef T elem;
  const T *o, *Wo, *x;
  T *xt;
  int N, d, K;
  __device__ bool map(int bx, int by, int BM, Tile &t) const {
    t.m0 = bx * BM;
    t.n0 = by * 128;
    t.mvalid = min(BM, N - t.m0);
    t.e = 0;
    t.p0 = 0;
    return t.mvalid > 0;
  }
  __device__ const T *a_row(const Tile &t, int r) const { return o + int64_t(t.m0 + r) * K; }
  __device__ const T *b_row(const Tile &t, int n) const {
    return t.n0 + n < d ? Wo + int64_t(t.n0 + n) * K : nullptr;
  }
  __device__ void epilogue(const Tile &t, const float *C, int ldc, int r0, int nr,
                           int tid) const {
    for (int idx = tid; idx < nr * 128; idx += 256) {
      const int r = idx >> 7, c = idx & 127;
      const int row = t.m0 + r0 + r, col = t.n0 + c;
      if (r0 + r >= t.mvalid || col >= d) continue;
      const int64_t off = int64_t(row) * d + col;
      Act<T>::st(xt, off, Act<T>::ld(x, off) + C[r * ldc + c]);
    }
  }
};

// Map a linear row-tile index to (expert e >= 1, tile within e).
__device__ __forceinline__ bool map_grouped(int bx, int BM, const int32_t *cnt,
                                            const int32_t *off, int E, Tile &t) {
  int rem = bx;
  for (int e = 1; e <= E; ++e) {
    const int c = cnt[e];
    const int nt = (c + BM - 1) / BM;
    if (rem < nt) {
      t.e = e;
      t.p0 = off[e - 1] + rem * BM;
      t.mvalid = min(BM, c - rem * BM);
      t.m0 = 0;
      return true;
    }
    rem -= nt;
  }
  return false;
}

template <typename T>
struct Moe1Prob {
  typedef T elem;
  const T *n2, *Wg, *Wu;
  T *Hm;
  const int32_t *cnt, *off;
  int E, d, dff, K;
  __device__ bool map(int bx, int by, int BM, Tile &t) const {
    if (!map_grouped(bx, BM, cnt, off, E, t)) return false;
    t.n0 = by * 64;
    return true;
  }
  __device__ const T *a_row(const Tile &t, int r) const {
    return n2 + int64_t(t.p0 + r) * d;
  }
  __device__ const T *b_row(const Tile &t, int n) const {
    const int64_t f = int64_t(t.e - 1) * dff + t.n0 + (n & 63);
    return (n < 64 ? Wg : Wu) + f * d;
  }
  __device__ void epilogue(const Tile &t, const float *C, int ldc, int r0, int nr,
                           int tid) const {
    for (int idx = tid; idx < nr * 64; idx += 256) {
      const int r = idx >> 6, c = idx & 63;
      if (r0 + r >= t.mvalid) continue;
      const float g = C[r * ldc + c], u = C[r * ldc + c + 64];
      const float s = g / (1.0f + expf(-g));
      Act<T>::st(Hm, int64_t(t.p0 + r0 + r) * dff + t.n0 + c, s * u);
    }
  }
};

template <typename T>
struct Moe2Prob {
  typedef T elem;
  const T *Hm, *Wd;
  float *Y;
  const int32_t *cnt, *off;
  int E, d, dff, K;
  __device__ bool map(int bx, int by, int BM, Tile &t) const {
    if (!map_grouped(bx, BM, cnt, off, E, t)) return false;
    t.n0 = by * 128;
    return true;
  }
  __device__ const T *a_row(const Tile &t, int r) const { return Hm + int64_t(t.p0 + r) * dff; }
  __device__ const T *b_row(const Tile &t, int n) const {
    return t.n0 + n < d ? Wd + (int64_t(t.e - 1) * d + t.n0 + n) * dff : nullptr;
  }
  __device__ void epilogue(const Tile &t, const float *C, int ldc, int r0, int nr,
                           int tid) const {
    for (int idx = tid; idx < nr * 128; idx += 256) {
      const int r = idx >> 7, c = idx & 127;
      if (r0 + r >= t.mvalid || t.n0 + c >= d) continue;
      Y[int64_t(t.p0 + r0 + r) * d + t.n0 + c] = C[r * ldc + c];
    }
  }
};

// -------------------------------------------------------------- fp32 kernel
// Block tile 64 x 128, K step 16, 4 x 8 outputs per thread.
template <class P>
__global__ __launch_bounds__(256) void gemm_f32_kernel(P p) {
  constexpr int BM = 64, BK = 16, LDC = 132;
  __shared__ __align__(16) float smem[64 * LDC];
  float(*As)[BM + 4] = (float(*)[BM + 4])smem;
  float(*Bs)[128 + 4] = (float(*)[128 + 4])(smem + BK * (BM + 4));
  Tile tc;
  if (!p.map(blockIdx.x, blockIdx.y, BM, tc)) return;
  const int tid = threadIdx.x;
  const int tr = tid >> 4, tcl = tid & 15;
  const int ar = tid >> 2, ak = (tid & 3) * 4;
  const int bn = tid >> 1, bk = (tid & 1) * 8;
  const float *arow = ar < tc.mvalid ? p.a_row(tc, ar) : nullptr;
  const float *brow = p.b_row(tc, bn);
  float acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < p.K; k0 += BK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) As[ak + i][ar] = arow ? arow[k0 + ak + i] : 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) Bs[bk + i][bn] = brow ? brow[k0 + bk + i] : 0.f;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][tr * 4 + i];
#pragma unroll
      for (int j = 0; j < 8; ++j) b[j] = Bs[kk][tcl * 8 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  float *C = smem;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) C[(tr * 4 + i) * LDC + tcl * 8 + j] = acc[i][j];
  __syncthreads();
  p.epilogue(tc, C, LDC, 0, 64, tid);
}

// ------------------------------------------------------------------ launchers
template <class P>
static hipError_t run_gemm(const triroute_cfg &, const P &p, int, int m_tiles64, int n_tiles,
                           hipStream_t st) {
  static_assert(std::is_same<typename P::elem, float>::value, "fp32 problems only");
  if (m_tiles64 > 0) gemm_f32_kernel<P><<<dim3(m_tiles64, n_tiles), 256, 0, st>>>(p);
  return hipGetLastError();
}

// The rotation table (one entry per token and pair serves every q and k
// head of the token), when the first RMSNorm did not already write it.
__global__ __launch_bounds__(256) void rope_table_kernel(int N, const RopeJob r) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= int64_t(N) * r.hd) return;
  r.tab[i] = rope_entry(r, int(i / r.hd), int(i % r.hd));
}

RopeJob make_rope_job(const triroute_cfg &cfg, int Tq, const int32_t *pos_base,
                      const int32_t *pos_idx, int n_base, float *tab) {
  RopeJob r;
  r.pos_base = pos_base;
  r.pos_idx = pos_idx;
  r.n_base = n_base;
  r.Tq = Tq;
  r.hd = cfg.head_dim / 2;
  r.tab = (float2 *)tab;
  for (int j = 0; j < 64; ++j)
    r.inv_freq[j] = j < r.hd ? pow(double(cfg.rope_theta), -2.0 * j / double(cfg.head_dim)) : 0.0;
  return r;
}

size_t qkv_rope_floats(const triroute_cfg &cfg, int N) { return size_t(N) * cfg.head_dim; }

template <typename T>
static hipError_t qkv_t(const triroute_cfg &cfg, int B, int Tq, const void *n1,
                        const triroute_dense_w &w, const float *rope, void *q, void *k, void *v,
                        hipStream_t st) {
  QkvProb<T> p;
  p.n1 = (const T *)n1;
  p.Wq = (const T *)w.Wq;
  p.Wk = (const T *)w.Wk;
  p.Wv = (const T *)w.Wv;
  p.q = (T *)q;
  p.k = (T *)k;
  p.v = (T *)v;
  p.rope = (const float2 *)rope;
  p.N = B * Tq;
  p.d = cfg.d_model;
  p.H = cfg.n_heads;
  p.Hkv = cfg.n_kv_heads;
  p.dh = cfg.head_dim;
  p.K = cfg.d_model;
  p.Ncols = (cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim;
  const int N = p.N;
  return run_gemm(cfg, p, (N + 127) / 128, (N + 63) / 64, (p.Ncols + 127) / 128, st);
}

hipError_t launch_qkv(const triroute_cfg &cfg, int B, int Tq, const void *n1,
                      const triroute_dense_w &w, const int32_t *pos_base, const int32_t *pos_idx,
                      int n_base, void *q, void *k, void *v, float *rope, bool rope_ready,
                      hipStream_t st) {
  const int N = B * Tq;
  if (!rope_ready) {
    const RopeJob r = make_rope_job(cfg, Tq, pos_base, pos_idx, n_base, rope);
    const int64_t n = int64_t(N) * r.hd;
    rope_table_kernel<<<dim3(unsigned((n + 255) / 256)), 256, 0, st>>>(N, r);
  }
  return cfg.act == TRIROUTE_BF16 ? mfma_qkv(cfg, B, Tq, n1, w, rope, q, k, v, st)
                                  : qkv_t<float>(cfg, B, Tq, n1, w, rope, q, k, v, st);
}

template <typename T>
static hipError_t oproj_t(const triroute_cfg &cfg, int N, const void *x, const void *o,
                          const triroute_dense_w &w, void *xt, hipStream_t st) {
  OprojProb<T> p;
  p.o = (const T *)o;
  p.Wo = (const T *)w.Wo;
  p.x = (const T *)x;
  p.xt = (T *)xt;
  p.N = N;
  p.d = cfg.d_model;
  p.K = cfg.n_heads * cfg.head_dim;
  return run_gemm(cfg, p, (N + 127) / 128, (N + 63) / 64, (p.d + 127) / 128, st);
}

hipError_t launch_oproj(const triroute_cfg &cfg, int N, const void *x, const void *o,
                        const triroute_dense_w &w, void *xt, hipStream_t st) {
  return cfg.act == TRIROUTE_BF16 ? mfma_oproj(cfg, N, x, o, w, xt, st)
                                  : oproj_t<float>(cfg, N, x, o, w, xt, st);
}

template <typename T>
static hipError_t moe_gemms_t(const triroute_cfg &cfg, int N, const void *n2,
                              const triroute_moe_w &w, const triroute_compaction &c, void *Hm,
                              float *Y, hipStream_t st) {
  const int E = cfg.n_experts, k = cfg.top_k, d = cfg.d_model, dff = cfg.d_ff;
  const int Nk = N * k;
  Moe1Prob<T> p1;
  p1.n2 = (const T *)n2;
  p1.Wg = (const T *)w.Wgate;
  p1.Wu = (const T *)w.Wup;
  p1.Hm = (T *)Hm;
  p1.cnt = c.exp_cnt;
  p1.off = c.exp_off;
  p1.E = E;
  p1.d = d;
  p1.dff = dff;
  p1.K = d;
  hipError_t err = run_gemm(cfg, p1, Nk / 128 + E, Nk / 64 + E, dff / 64, st);
  if (err != hipSuccess) return err;
  Moe2Prob<T> p2;
  p2.Hm = (const T *)Hm;
  p2.Wd = (const T *)w.Wdown;
  p2.Y = Y;
  p2.cnt = c.exp_cnt;
  p2.off = c.exp_off;
  p2.E = E;
  p2.d = d;
  p2.dff = dff;
  p2.K = dff;
  return run_gemm(cfg, p2, Nk / 128 + E, Nk / 64 + E, (d + 127) / 128, st);
}

hipError_t launch_moe_gemms(const triroute_cfg &cfg, int N, const void *n2,
                            const triroute_moe_w &w, const triroute_compaction &c, void *Hm,
                            float *Y, hipStream_t st) {
  return cfg.act == TRIROUTE_BF16 ? mfma_moe(cfg, N, n2, w, c, Hm, Y, st)
                                  : moe_gemms_t<float>(cfg, N, n2, w, c, Hm, Y, st);
}

}  // namespace tr
