// bf16 GEMMs of the layer on gfx950 MFMA: C = A B^T, both operands
// K-contiguous, fp32 accumulation (v_mfma_f32_16x16x32_bf16).
//
// Block tile BM x BN, K step 64, 8 waves arranged WM x WN, each wave owning a
// (BM/WM) x 64 sub-tile.  A and B tiles are double-buffered in LDS (rows of
// 128 B, 16-byte chunk c of row r stored at c ^ (r & 7)); the next K step is
// fetched into registers while the current one feeds the MFMAs.
//
// Epilogues work on the accumulator registers.  Within a wave's 64 columns
// the B rows are ordered so that column j of 16-column block ni and block
// ni + 2 are partners: gate/up of one expert unit (SwiGLU), or RoPE pair
// (j, j + d_h/2) of one head.  Each lane therefore holds both partners.
//
//   QKV   : [n1] x [Wq;Wk;Wv]^T, rotate-half RoPE on q and k
//   O-proj: xt = x + o Wo^T
//   MoE-1 : H = silu(n2 Wgate_e^T) * (n2 Wup_e^T) per expert (paper Sec. 3.2 (B))
//   MoE-2 : Y[a] = H Wdown_e^T, scattered back to assignment a
#include "kernels.hpp"

namespace tr {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

struct MTile {
  int m0, n0, mvalid, e, p0;
};

// Map a linear row-tile index to (expert e >= 1, tile within e).
__device__ __forceinline__ bool mmap_grouped(int bx, int BM, const int32_t *cnt,
                                             const int32_t *off, int E, MTile &t) {
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

// Physical column n of a BN-wide tile -> (pair index P in the tile, half).
// Wave slice s = n / 64 holds pairs 32 s .. 32 s + 31: first halves in its
// columns 0..31, second halves in 32..63.
__device__ __forceinline__ void col_pair(int n, int &P, int &half) {
  P = (n >> 6) * 32 + (n & 31);
  half = (n >> 5) & 1;
}

// ---------------------------------------------------------------- problems
struct QkvM {
  const bf16 *n1, *Wq, *Wk, *Wv;
  bf16 *q, *k, *v;
  const int32_t *pos_base, *pos_idx;
  int N, Tq, d, H, Hkv, dh, Ncols;
  double inv_freq[64];
  __device__ bool map(int bx, int by, int BM, int BN, MTile &t) const {
    t.m0 = bx * BM;
    t.n0 = by * BN;
    t.mvalid = min(BM, N - t.m0);
    t.e = t.p0 = 0;
    return t.mvalid > 0;
  }
  __device__ int logical_col(const MTile &t, int P, int half) const {
    const int hd = dh >> 1;
    return t.n0 + (P / hd) * dh + (P % hd) + half * hd;
  }
  __device__ const bf16 *a_row(const MTile &t, int r) const { return n1 + int64_t(t.m0 + r) * d; }
  __device__ const bf16 *b_row(const MTile &t, int n) const {
    int P, half;
    col_pair(n, P, half);
    int gc = logical_col(t, P, half);
    if (gc >= Ncols) return nullptr;
    const int Hd = H * dh, Kd = Hkv * dh;
    if (gc < Hd) return Wq + int64_t(gc) * d;
    gc -= Hd;
    if (gc < Kd) return Wk + int64_t(gc) * d;
    return Wv + int64_t(gc - Kd) * d;
  }
  // x1 / x2: first / second half of pair P for tile row r
  __device__ void store_pair(const MTile &t, int r, int P, float x1, float x2) const {
    if (r >= t.mvalid) return;
    const int c1 = logical_col(t, P, 0);
    if (c1 >= Ncols) return;
    const int Hd = H * dh, Kd = Hkv * dh, hd = dh >> 1;
    const int row = t.m0 + r;
    bf16 *out;
    int ld, col;
    bool rot = true;
    if (c1 < Hd) {
      out = q; ld = Hd; col = c1;
    } else if (c1 < Hd + Kd) {
      out = k; ld = Kd; col = c1 - Hd;
    } else {
      out = v; ld = Kd; col = c1 - Hd - Kd; rot = false;
    }
    float y1 = x1, y2 = x2;
    if (rot) {
      const int jj = col % hd;
      const int b = row / Tq, tt = row - b * Tq;
      const int pos = (pos_base ? pos_base[pos_idx ? pos_idx[b] : b] : 0) + tt;
      // angle in fp64, reduced to [-pi, pi], then an accurate fp32 sincos
      const double ang = double(pos) * inv_freq[jj];
      const double kq = rint(ang * 0.15915494309189535);
      double rr = fma(-kq, 6.283185307179586, ang);
      rr = fma(-kq, 2.4492935982947064e-16, rr);
      float sn, cs;
      sincosf(float(rr), &sn, &cs);
      y1 = x1 * cs - x2 * sn;
      y2 = x1 * sn + x2 * cs;
    }
    bf16 *o = out + int64_t(row) * ld + col;
    o[0] = f2bf(y1);
    o[hd] = f2bf(y2);
  }
};

struct OprojM {
  const bf16 *o, *Wo, *x;
  bf16 *xt;
  int N, d, K;
  __device__ bool map(int bx, int by, int BM, int BN, MTile &t) const {
    t.m0 = bx * BM;
    t.n0 = by * BN;
    t.mvalid = min(BM, N - t.m0);
    t.e = t.p0 = 0;
    return t.mvalid > 0;
  }
  __device__ const bf16 *a_row(const MTile &t, int r) const { return o + int64_t(t.m0 + r) * K; }
  __device__ const bf16 *b_row(const MTile &t, int n) const {
    return t.n0 + n < d ? Wo + int64_t(t.n0 + n) * K : nullptr;
  }
  __device__ void store(const MTile &t, int r, int n, float acc) const {
    if (r >= t.mvalid || t.n0 + n >= d) return;
    const int64_t off = int64_t(t.m0 + r) * d + t.n0 + n;
    xt[off] = f2bf(bf2f(x[off]) + acc);
  }
};

struct Moe1M {
  const bf16 *n2, *Wg, *Wu;
  bf16 *Hm;
  const int32_t *cnt, *off, *rows;
  int E, k, d, dff;
  __device__ bool map(int bx, int by, int BM, int BN, MTile &t) const {
    if (!mmap_grouped(bx, BM, cnt, off, E, t)) return false;
    t.n0 = by * (BN / 2);  // BN/2 expert units per tile (gate + up columns)
    return true;
  }
  __device__ const bf16 *a_row(const MTile &t, int r) const {
    return n2 + int64_t(rows[t.p0 + r] / k) * d;
  }
  __device__ const bf16 *b_row(const MTile &t, int n) const {
    int P, half;
    col_pair(n, P, half);
    const int f = t.n0 + P;
    if (f >= dff) return nullptr;
    return (half ? Wu : Wg) + (int64_t(t.e - 1) * dff + f) * d;
  }
  __device__ void store_pair(const MTile &t, int r, int P, float g, float u) const {
    const int f = t.n0 + P;
    if (r >= t.mvalid || f >= dff) return;
    const float s = g / (1.0f + expf(-g));
    Hm[int64_t(t.p0 + r) * dff + f] = f2bf(s * u);
  }
};

struct Moe2M {
  const bf16 *Hm, *Wd;
  float *Y;
  const int32_t *cnt, *off, *rows;
  int E, d, dff;
  __device__ bool map(int bx, int by, int BM, int BN, MTile &t) const {
    if (!mmap_grouped(bx, BM, cnt, off, E, t)) return false;
    t.n0 = by * BN;
    return true;
  }
  __device__ const bf16 *a_row(const MTile &t, int r) const { return Hm + int64_t(t.p0 + r) * dff; }
  __device__ const bf16 *b_row(const MTile &t, int n) const {
    return t.n0 + n < d ? Wd + (int64_t(t.e - 1) * d + t.n0 + n) * dff : nullptr;
  }
  __device__ void store(const MTile &t, int r, int n, float acc) const {
    if (r >= t.mvalid || t.n0 + n >= d) return;
    Y[int64_t(rows[t.p0 + r]) * d + t.n0 + n] = acc;
  }
};

template <class P> struct IsPaired { static constexpr bool value = false; };
template <> struct IsPaired<QkvM> { static constexpr bool value = true; };
template <> struct IsPaired<Moe1M> { static constexpr bool value = true; };

// ------------------------------------------------------------------ kernel
template <class P, int BM, int WM, int WN>
__global__ __launch_bounds__(512, 1) void gemm_mfma_kernel(P p, int K) {
  constexpr int BN = 64 * WN;
  constexpr int TM = BM / WM;      // wave rows
  constexpr int MI = TM / 16;      // 16-row MFMA tiles per wave
  constexpr int LA = BM / 64;      // A chunks per thread per stage
  constexpr int LB = BN / 64;      // B chunks per thread per stage
  constexpr int ABYTES = BM * 128, BBYTES = BN * 128, STAGE = ABYTES + BBYTES;
  __shared__ __align__(16) uint8_t smem[2 * STAGE];
  MTile tc;
  if (!p.map(blockIdx.x, blockIdx.y, BM, BN, tc)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int lr = tid >> 3, lc = tid & 7;
  const bf16 *ap[LA], *bq[LB];
#pragma unroll
  for (int i = 0; i < LA; ++i) {
    const int r = lr + 64 * i;
    ap[i] = r < tc.mvalid ? p.a_row(tc, r) : nullptr;
  }
#pragma unroll
  for (int i = 0; i < LB; ++i) bq[i] = p.b_row(tc, lr + 64 * i);
  uint4 ra[LA], rb[LB];
  const uint4 zero = make_uint4(0, 0, 0, 0);
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < LA; ++i) ra[i] = ap[i] ? *(const uint4 *)(ap[i] + k0 + lc * 8) : zero;
#pragma unroll
    for (int i = 0; i < LB; ++i) rb[i] = bq[i] ? *(const uint4 *)(bq[i] + k0 + lc * 8) : zero;
  };
  auto sstore = [&](int buf) {
    uint8_t *As = smem + buf * STAGE;
    uint8_t *Bs = As + ABYTES;
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      const int r = lr + 64 * i;
      *(uint4 *)(As + r * 128 + ((lc ^ (r & 7)) << 4)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      const int r = lr + 64 * i;
      *(uint4 *)(Bs + r * 128 + ((lc ^ (r & 7)) << 4)) = rb[i];
    }
  };
  f32x4_t acc[MI][4];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int nk = K / 64;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload((kt + 1) * 64);
    const uint8_t *As = smem + (kt & 1) * STAGE;
    const uint8_t *Bs = As + ABYTES;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int ch = ks * 4 + (lane >> 4);
      bf16x8_t b[4];
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int n = wn * 64 + ni * 16 + (lane & 15);
        b[ni] = *(const bf16x8_t *)(Bs + n * 128 + ((ch ^ (n & 7)) << 4));
      }
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) {
        const int r = wm * TM + mi * 16 + (lane & 15);
        const bf16x8_t a = *(const bf16x8_t *)(As + r * 128 + ((ch ^ (r & 7)) << 4));
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[ni], acc[mi][ni], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) sstore((kt + 1) & 1);
    __syncthreads();
  }
  // epilogue from registers: lane holds rows 4 (lane/16) + i of each 16-row
  // tile, column (lane % 16) of each 16-column block
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = wm * TM + mi * 16 + 4 * (lane >> 4) + i;
      if constexpr (IsPaired<P>::value) {
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          const int Pp = wn * 32 + ni * 16 + (lane & 15);
          p.store_pair(tc, r, Pp, acc[mi][ni][i], acc[mi][ni + 2][i]);
        }
      } else {
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          p.store(tc, r, wn * 64 + ni * 16 + (lane & 15), acc[mi][ni][i]);
      }
    }
}

// ------------------------------------------------------------------ launchers
template <class P, int BM, int WM, int WN>
static hipError_t launch(const P &p, int K, int m_tiles, int n_tiles, hipStream_t st) {
  if (m_tiles > 0 && n_tiles > 0)
    gemm_mfma_kernel<P, BM, WM, WN><<<dim3(m_tiles, n_tiles), 512, 0, st>>>(p, K);
  return hipGetLastError();
}

hipError_t mfma_qkv(const triroute_cfg &cfg, int B, int Tq, const void *n1,
                    const triroute_dense_w &w, const int32_t *pos_base, const int32_t *pos_idx,
                    void *q, void *k, void *v, hipStream_t st) {
  QkvM p;
  p.n1 = (const bf16 *)n1;
  p.Wq = (const bf16 *)w.Wq;
  p.Wk = (const bf16 *)w.Wk;
  p.Wv = (const bf16 *)w.Wv;
  p.q = (bf16 *)q;
  p.k = (bf16 *)k;
  p.v = (bf16 *)v;
  p.pos_base = pos_base;
  p.pos_idx = pos_idx;
  p.N = B * Tq;
  p.Tq = Tq;
  p.d = cfg.d_model;
  p.H = cfg.n_heads;
  p.Hkv = cfg.n_kv_heads;
  p.dh = cfg.head_dim;
  p.Ncols = (cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim;
  for (int j = 0; j < 64; ++j)
    p.inv_freq[j] = j < cfg.head_dim / 2
                        ? pow(double(cfg.rope_theta), -2.0 * j / double(cfg.head_dim))
                        : 0.0;
  return launch<QkvM, 256, 4, 2>(p, cfg.d_model, (p.N + 255) / 256, (p.Ncols + 127) / 128, st);
}

hipError_t mfma_oproj(const triroute_cfg &cfg, int N, const void *x, const void *o,
                      const triroute_dense_w &w, void *xt, hipStream_t st) {
  OprojM p;
  p.o = (const bf16 *)o;
  p.Wo = (const bf16 *)w.Wo;
  p.x = (const bf16 *)x;
  p.xt = (bf16 *)xt;
  p.N = N;
  p.d = cfg.d_model;
  p.K = cfg.n_heads * cfg.head_dim;
  return launch<OprojM, 256, 4, 2>(p, p.K, (N + 255) / 256, (p.d + 127) / 128, st);
}

hipError_t mfma_moe(const triroute_cfg &cfg, int N, const void *n2, const triroute_moe_w &w,
                    const triroute_compaction &c, void *Hm, float *Y, hipStream_t st) {
  const int E = cfg.n_experts, k = cfg.top_k, d = cfg.d_model, dff = cfg.d_ff;
  const int Nk = N * k;
  Moe1M p1;
  p1.n2 = (const bf16 *)n2;
  p1.Wg = (const bf16 *)w.Wgate;
  p1.Wu = (const bf16 *)w.Wup;
  p1.Hm = (bf16 *)Hm;
  p1.cnt = c.exp_cnt;
  p1.off = c.exp_off;
  p1.rows = c.exp_rows;
  p1.E = E;
  p1.k = k;
  p1.d = d;
  p1.dff = dff;
  hipError_t err = launch<Moe1M, 256, 2, 4>(p1, d, Nk / 256 + E, (dff + 127) / 128, st);
  if (err != hipSuccess) return err;
  Moe2M p2;
  p2.Hm = (const bf16 *)Hm;
  p2.Wd = (const bf16 *)w.Wdown;
  p2.Y = Y;
  p2.cnt = c.exp_cnt;
  p2.off = c.exp_off;
  p2.rows = c.exp_rows;
  p2.E = E;
  p2.d = d;
  p2.dff = dff;
  return launch<Moe2M, 256, 4, 2>(p2, dff, Nk / 256 + E, (d + 127) / 128, st);
}

}  // namespace tr
