// Backward pass of the relaxed controller (paper Sec. 3.4-3.7, Algorithm 1
// step 7 for the controller): from the language-model gradients of the soft
// samples y~^a, y~^b (the straight-through estimator hands the hard choice's
// gradient to them) and of the selected gates p-bar, plus the regulariser's
// own terms, to the logits, then through the whitened heads, RMSNorm(h; gr),
// the GELU trunk and the first norm to every controller weight and to x and
// psi.  The language-model part of each axis' logit gradient is divided by
// that axis' balance factor rho, which then moves towards the part's norm.
//
// Kernels, in order: the trunk and tail of the forward again (with taps of
// a1, h, h^ and z; deterministic, so the logits equal the forward's), one
// wave per token for the logit gradient and the chain down to da1, fp32
// MFMA grams sum_t A_t^T B_t over fixed token chunks for the weight
// gradients (fp32 within a chunk, chunks added in order in fp64), column
// sums in fp64 for the biases, an fp32 MFMA product da1 W1 for the gradient
// of [n1; psi], the first norm's backward per row, and a final kernel for
// the whitening, the head weights and rho.  Every sum has a fixed order.
#include "kernels.hpp"

namespace tr {

namespace {

constexpr int DR = 128;
// tokens per partial sum of the gram kernels: short chunks for the small
// sums, longer ones for the two trunk weight grams (whose partials are large)
constexpr int GR_CHUNK = 128, GR_CHUNK_W = 512;

__device__ __forceinline__ float gelu_f(float y) {
  return 0.5f * y * (1.0f + erff(y * 0.70710678118654752f));
}
// d GELU / dy = Phi(y) + y phi(y)
__device__ __forceinline__ float gelu_grad_f(float y) {
  return 0.5f * (1.0f + erff(y * 0.70710678118654752f)) +
         y * 0.39894228040143268f * expf(-0.5f * y * y);
}

__device__ __forceinline__ float wsum(float v) { return seg_sum(v, 64); }

struct BwdTokArgs {
  const float *Z, *a1, *hpre, *Wf;  // logits, trunk taps, head weights as applied (folded)
  const float *ya, *yb, *egate;
  const int32_t *eidx, *pos;
  const float *g_ya, *g_yb, *g_gate;
  const float *W2, *gr;
  const double *stats, *usage;  // the forward's batch statistics
  const double *rho;            // [3] or NULL (1)
  const double *lambda;         // [2] or NULL (0)
  float *dz, *dh, *da1, *u, *tgr, *lmsq;
  int N, H, A, E1, k, dh_, w, dkv;
  float inv_ta, inv_tb, zeta, alpha, beta, gamma, eps, kappa_e;
};

// One wave per token.  Lane a < A: attention group a; lane j < E + 1:
// expert j; lanes 0..3: the bit options; every lane: features lane and
// lane + 64 of the 128-wide trunk.
__global__ __launch_bounds__(256) void relax_bwd_tok_kernel(BwdTokArgs p) {
  __shared__ float dzs[4][DR];  // a wave's logit gradients (3 A + E + 5 <= 112), then its dh
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int t = blockIdx.x * 4 + wave;
  if (t >= p.N) return;  // wave-uniform; no block barrier below
  float *dzw = dzs[wave];
  const int NZ = 3 * p.A + p.E1 + 4, HA = p.H / p.A;
  const float *z = p.Z + int64_t(t) * NZ;
  const double *st = p.stats;
  const double rows_a = double(p.N) * p.A, rows = double(p.N);
  const float Df = float(st[TRIROUTE_RS_DENSE]), Dm = float(st[TRIROUTE_RS_DENSE + 1]);
  const float lam_f = p.lambda ? float(p.lambda[0]) : 0.f, lam_m = p.lambda ? float(p.lambda[1]) : 0.f;
  const float rho_a = p.rho ? float(p.rho[0]) : 1.f, rho_e = p.rho ? float(p.rho[1]) : 1.f,
              rho_b = p.rho ? float(p.rho[2]) : 1.f;
  const int P = p.pos[t];
  const float kf = float(P) + 1.f, kl = fminf(kf, float(p.w));
  float sq_a = 0.f, sq_e = 0.f, sq_b = 0.f;  // squares of the language-model parts
  // ---- attention groups
  if (lane < p.A) {
    const int a = lane;
    float y[3], gl[3], gc[3], q[3], zz[3];
    const float kap[3] = {0.f, float(HA) * 2.f * float(p.dh_) * kl, float(HA) * 2.f * float(p.dh_) * kf};
    float zm = -INFINITY;
    for (int m = 0; m < 3; ++m) {
      y[m] = p.ya[(int64_t(t) * p.A + a) * 3 + m];
      gl[m] = p.g_ya[(int64_t(t) * p.A + a) * 3 + m];
      gc[m] = lam_f / Df * kap[m];
      zz[m] = z[3 * a + m];
      zm = fmaxf(zm, zz[m]);
    }
    float qs = 0.f;
    for (int m = 0; m < 3; ++m) { q[m] = expf(zz[m] - zm); qs += q[m]; }
    const float lse = zm + logf(qs);
    float sy_l = 0.f, sy_c = 0.f, sfp = 0.f, slp = 0.f;
    float f[3], Pm[3], lp[3];
    for (int m = 0; m < 3; ++m) {
      q[m] /= qs;
      f[m] = float(st[TRIROUTE_RS_F_ATTN + m]);
      Pm[m] = float(st[TRIROUTE_RS_P_ATTN + m]);
      lp[m] = Pm[m] > 0.f ? logf(Pm[m]) + 1.f : 0.f;
      sy_l += y[m] * gl[m];
      sy_c += y[m] * gc[m];
      sfp += f[m] * q[m];
      slp += lp[m] * q[m];
    }
    const bool ent = p.zeta * logf(3.f) - float(st[TRIROUTE_RS_ENTROPY]) > 0.f;
    for (int m = 0; m < 3; ++m) {
      const float dl = p.inv_ta * y[m] * (gl[m] - sy_l);
      sq_a += dl * dl;
      float d = dl / rho_a + p.inv_ta * y[m] * (gc[m] - sy_c);
      d += p.alpha * 3.f / float(rows_a) * q[m] * (f[m] - sfp);
      d += p.beta * 2.f / float(rows_a) * lse * q[m];
      if (ent) d += p.gamma / float(rows_a) * q[m] * (lp[m] - slp);
      dzw[3 * a + m] = d;
    }
  }
  // ---- experts: the gates over the selected set, then the full softmax
  {
    const float ze = lane < p.E1 ? z[3 * p.A + lane] : -INFINITY;
    const float zmx = seg_max(ze, 64);
    const float ee = lane < p.E1 ? expf(ze - zmx) : 0.f;
    const float es = wsum(ee);
    const float pe = ee / es, lse = zmx + logf(es);
    const float fe = lane < p.E1 ? float(p.usage[lane]) : 0.f;
    const float Pe = lane < p.E1 ? float(p.usage[p.E1 + lane]) : 0.f;
    const float lpe = Pe > 0.f ? logf(Pe) + 1.f : 0.f;
    const float sfp = wsum(fe * pe), slp = wsum(lpe * pe);
    // slot s on lane s: expert, gate, upstream
    const int es_ = lane < p.k ? p.eidx[int64_t(t) * p.k + lane] : -1;
    const float gs = lane < p.k ? p.egate[int64_t(t) * p.k + lane] : 0.f;
    const float gl = lane < p.k ? p.g_gate[int64_t(t) * p.k + lane] : 0.f;
    const float gc = lane < p.k && es_ != 0 ? lam_f / Df * p.kappa_e : 0.f;
    const float sgl = wsum(gs * gl), sgc = wsum(gs * gc);
    const float sl_l = gs * (gl - sgl), sl_c = gs * (gc - sgc);
    float dl = 0.f, dc = 0.f;
    for (int s = 0; s < p.k; ++s) {
      const int e = __shfl(es_, s, 64);
      const float a_l = __shfl(sl_l, s, 64), a_c = __shfl(sl_c, s, 64);
      if (e == lane) { dl += a_l; dc += a_c; }
    }
    const bool ent = p.zeta * logf(float(p.E1)) - float(st[TRIROUTE_RS_ENTROPY + 1]) > 0.f;
    if (lane < p.E1) {
      sq_e += dl * dl;
      float d = dl / rho_e + dc;
      d += p.alpha * float(p.E1) / float(rows) * pe * (fe - sfp);
      d += p.beta * 2.f / float(rows) * lse * pe;
      if (ent) d += p.gamma / float(rows) * pe * (lpe - slp);
      dzw[3 * p.A + lane] = d;
    }
  }
  // ---- bits: y~ over (2, 4, 8, 16)
  {
    const bool on = lane < 4;
    const float zb = on ? z[3 * p.A + p.E1 + lane] : -INFINITY;
    const float y = on ? p.yb[int64_t(t) * 4 + lane] : 0.f;
    const float gl = on ? p.g_yb[int64_t(t) * 4 + lane] : 0.f;
    const float gc = on ? lam_m / Dm * float(p.dkv) * 2.f * float(2 << lane) : 0.f;
    const float zmx = seg_max(zb, 64);
    const float ee = on ? expf(zb - zmx) : 0.f;
    const float es = wsum(ee);
    const float q = ee / es, lse = zmx + logf(es);
    const float f = on ? float(st[TRIROUTE_RS_F_BITS + lane]) : 0.f;
    const float Pb = on ? float(st[TRIROUTE_RS_P_BITS + lane]) : 0.f;
    const float lp = Pb > 0.f ? logf(Pb) + 1.f : 0.f;
    const float sy_l = wsum(y * gl), sy_c = wsum(y * gc), sfp = wsum(f * q), slp = wsum(lp * q);
    const bool ent = p.zeta * logf(4.f) - float(st[TRIROUTE_RS_ENTROPY + 2]) > 0.f;
    if (on) {
      const float dl = p.inv_tb * y * (gl - sy_l);
      sq_b += dl * dl;
      float d = dl / rho_b + p.inv_tb * y * (gc - sy_c);
      d += p.alpha * 4.f / float(rows) * q * (f - sfp);
      d += p.beta * 2.f / float(rows) * lse * q;
      if (ent) d += p.gamma / float(rows) * q * (lp - slp);
      dzw[3 * p.A + p.E1 + lane] = d;
    }
  }
  __builtin_amdgcn_wave_barrier();
  const float sqa = wsum(sq_a), sqe = wsum(sq_e), sqb = wsum(sq_b);
  if (lane < 3) p.lmsq[int64_t(t) * 4 + lane] = lane == 0 ? sqa : lane == 1 ? sqe : sqb;
  for (int r = lane; r < NZ; r += 64) p.dz[int64_t(t) * NZ + r] = dzw[r];
  // ---- dh^ = W'^T dz (lanes own features lane, lane + 64)
  float g0 = 0.f, g1 = 0.f;
  for (int r = 0; r < NZ; ++r) {
    const float d = dzw[r];
    g0 = fmaf(p.Wf[int64_t(r) * DR + lane], d, g0);
    g1 = fmaf(p.Wf[int64_t(r) * DR + lane + 64], d, g1);
  }
  // ---- RMSNorm(h; gr): h^ = h r gr
  const float h0 = p.hpre[int64_t(t) * DR + lane], h1 = p.hpre[int64_t(t) * DR + lane + 64];
  const float rr = 1.0f / sqrtf(wsum(h0 * h0 + h1 * h1) / float(DR) + p.eps);
  p.tgr[int64_t(t) * DR + lane] = g0 * h0 * rr;
  p.tgr[int64_t(t) * DR + lane + 64] = g1 * h1 * rr;
  const float gh0 = g0 * p.gr[lane], gh1 = g1 * p.gr[lane + 64];
  const float dot = wsum(gh0 * h0 + gh1 * h1);
  const float c3 = rr * rr * rr * dot / float(DR);
  const float dh0 = rr * gh0 - c3 * h0, dh1 = rr * gh1 - c3 * h1;
  p.dh[int64_t(t) * DR + lane] = dh0;
  p.dh[int64_t(t) * DR + lane + 64] = dh1;
  // ---- h = W2 u + b2: du_j = sum_i W2[i][j] dh_i
  float* dhs = dzw;  // reuse the wave's row for dh
  __builtin_amdgcn_wave_barrier();
  dhs[lane] = dh0;
  dhs[lane + 64] = dh1;
  __builtin_amdgcn_wave_barrier();
  float u0 = 0.f, u1 = 0.f;
  for (int i = 0; i < DR; ++i) {
    const float d = dhs[i];
    u0 = fmaf(p.W2[int64_t(i) * DR + lane], d, u0);
    u1 = fmaf(p.W2[int64_t(i) * DR + lane + 64], d, u1);
  }
  // ---- u = GELU(a1)
  const float x0 = p.a1[int64_t(t) * DR + lane], x1 = p.a1[int64_t(t) * DR + lane + 64];
  p.u[int64_t(t) * DR + lane] = gelu_f(x0);
  p.u[int64_t(t) * DR + lane + 64] = gelu_f(x1);
  p.da1[int64_t(t) * DR + lane] = u0 * gelu_grad_f(x0);
  p.da1[int64_t(t) * DR + lane + 64] = u1 * gelu_grad_f(x1);
}

// Column sums: part[c][i] = sum over tokens t of chunk c (CS_CHUNK tokens)
// of A[t][i], in fp64: wave w of a block adds tokens c CS_CHUNK + 64 w ..
// + 63 for the block's 64 columns (lane = column), the waves are added in
// order.
constexpr int CS_CHUNK = 256;
__global__ __launch_bounds__(256) void colsum_kernel(const float *__restrict__ A, int lda, int m,
                                                     int N, double *__restrict__ part) {
  __shared__ double ws_[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = blockIdx.x * 64 + lane, c = blockIdx.y;
  const int t0 = c * CS_CHUNK + 64 * wave, t1 = min(N, t0 + 64);
  double s = 0;
  if (i < m) {
    // 16 loads in flight at a time, added in token order
    for (int tb = t0; tb < t1; tb += 16) {
      float v[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) v[q] = A[int64_t(min(tb + q, t1 - 1)) * lda + i];  // clamped
#pragma unroll
      for (int q = 0; q < 16; ++q) s += tb + q < t1 ? double(v[q]) : 0.0;
    }
  }
  ws_[wave][lane] = s;
  __syncthreads();
  if (wave == 0 && i < m)
    part[int64_t(c) * m + i] = ((ws_[0][lane] + ws_[1][lane]) + ws_[2][lane]) + ws_[3][lane];
}
__global__ __launch_bounds__(256) void chunk_sum64_kernel(const double *__restrict__ part, int nc,
                                                          int m, float *__restrict__ out,
                                                          double *__restrict__ out64) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  double s = 0;
  for (int cb = 0; cb < nc; cb += 16) {  // 16 loads in flight, added in chunk order
    double v[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q] = part[int64_t(min(cb + q, nc - 1)) * m + i];  // clamped
#pragma unroll
    for (int q = 0; q < 16; ++q) s += cb + q < nc ? v[q] : 0.0;
  }
  if (out) out[i] = float(s);
  if (out64) out64[i] = s;
}

// out[e] = sum over the nc chunks, in order, of part[c][e] (fp64), as fp32
__global__ __launch_bounds__(256) void chunk_sum_kernel(const float *__restrict__ part, int nc,
                                                        int64_t ne, float *__restrict__ out,
                                                        double *__restrict__ out64) {
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= ne) return;
  double s = 0;
  for (int cb = 0; cb < nc; cb += 16) {  // 16 loads in flight, added in chunk order
    float v[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q] = part[int64_t(min(cb + q, nc - 1)) * ne + e];  // clamped
#pragma unroll
    for (int q = 0; q < 16; ++q) s += cb + q < nc ? double(v[q]) : 0.0;
  }
  if (out) out[e] = float(s);
  if (out64) out64[e] = s;
}

// s = [n1; psi] in fp32 (n1 = x r1 g1, the router's unrounded first norm).
// One wave per token; a lane takes 8 consecutive features at a time (d is a
// multiple of 64, rows of s start 16-byte aligned: d + d_psi is a multiple
// of 4).
template <typename T>
__global__ __launch_bounds__(256) void make_s_kernel(const T *__restrict__ x, const float *__restrict__ g1,
                                                     const float *__restrict__ psi, int N, int d,
                                                     int dpsi, float eps, float *__restrict__ s) {
  const int lane = threadIdx.x & 63, t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= N) return;
  const T *xr = x + int64_t(t) * d;
  float ss = 0.f;
  for (int j = 8 * lane; j < d; j += 512) {
    float v[8];
    load8(xr + j, v);
#pragma unroll
    for (int q = 0; q < 8; ++q) ss += v[q] * v[q];
  }
  const float r = 1.0f / sqrtf(seg_sum(ss, 64) / float(d) + eps);
  float *sr = s + int64_t(t) * (d + dpsi);
  for (int j = 8 * lane; j < d; j += 512) {
    float v[8];
    load8(xr + j, v);
    float o[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) o[q] = (v[q] * r) * g1[j + q];
    *(float4 *)(sr + j) = make_float4(o[0], o[1], o[2], o[3]);
    *(float4 *)(sr + j + 4) = make_float4(o[4], o[5], o[6], o[7]);
  }
  for (int j = lane; j < dpsi; j += 64) sr[d + j] = psi[int64_t(t) * dpsi + j];
}

typedef float f32x4m __attribute__((ext_vector_type(4)));

// C = A^T B over k (A_KMAJOR: A[k][i], the gram of two token-major
// matrices, k = token, one chunk of `kc` tokens per blockIdx.z, written to
// its own plane of C) or C = A B (A[i][k], k within [0, kc), one plane).
// fp32 MFMA 16x16x4: a block of 4 waves takes a 64 x 64 tile of C, wave w its
// rows 16 w .. 16 w + 15 in four 16-column blocks; 16 k-rows of A and B are
// staged in LDS at a time (rows padded to 65 floats: the four k-rows a wave
// reads at once fall in different banks).  Lanes past M, N or the chunk read
// zeros.
template <bool A_KMAJOR>
__global__ __launch_bounds__(256) void mm_f32_kernel(const float *__restrict__ A, int lda,
                                                     const float *__restrict__ B, int ldb, int M,
                                                     int N, int K, int kc, float *__restrict__ C,
                                                     int ldc) {
  __shared__ float As[16][65], Bs[16][65];
  const int i0 = blockIdx.x * 64, j0 = blockIdx.y * 64, z = blockIdx.z;
  const int k_lo = z * kc, k_hi = min(K, k_lo + kc);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  f32x4m acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = f32x4m{0.f, 0.f, 0.f, 0.f};
  for (int k0 = k_lo; k0 < k_hi; k0 += 16) {
    for (int e = threadIdx.x; e < 16 * 64; e += 256) {
      if constexpr (A_KMAJOR) {
        const int kk = e / 64, ii = e % 64;
        As[kk][ii] = (k0 + kk < k_hi && i0 + ii < M) ? A[int64_t(k0 + kk) * lda + i0 + ii] : 0.f;
      } else {
        const int ii = e / 16, kk = e % 16;
        As[kk][ii] = (k0 + kk < k_hi && i0 + ii < M) ? A[int64_t(i0 + ii) * lda + k0 + kk] : 0.f;
      }
      const int kk = e / 64, jj = e % 64;
      Bs[kk][jj] = (k0 + kk < k_hi && j0 + jj < N) ? B[int64_t(k0 + kk) * ldb + j0 + jj] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kq = 0; kq < 16; kq += 4) {
      const float a = As[kq + (lane >> 4)][16 * wave + (lane & 15)];
#pragma unroll
      for (int c = 0; c < 4; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Bs[kq + (lane >> 4)][16 * c + (lane & 15)],
                                                      acc[c], 0, 0, 0);
    }
    __syncthreads();
  }
  float *Cz = C + int64_t(z) * M * ldc;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + 16 * wave + 4 * (lane >> 4) + r, j = j0 + 16 * c + (lane & 15);
      if (i < M && j < N) Cz[int64_t(i) * ldc + j] = acc[c][r];
    }
}

// First norm n1 = x r1 g1: dx = r1 (g1 dn1) - r1^3 x sum(g1 dn1 x) / d; the
// terms dn1 x r1 of dg1 replace dn1 in ds; dpsi is copied out.  One wave
// per token, 8 consecutive features per lane at a time.
template <typename T>
__global__ __launch_bounds__(256) void rms1_bwd_kernel(const T *__restrict__ x, const float *__restrict__ g1,
                                                       float *__restrict__ ds, int N, int d, int dpsi,
                                                       float eps, float *__restrict__ dx,
                                                       float *__restrict__ dpsi_out) {
  const int lane = threadIdx.x & 63, t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= N) return;
  const T *xr = x + int64_t(t) * d;
  float *dr = ds + int64_t(t) * (d + dpsi);
  float ss = 0.f, sg = 0.f;
  for (int j = 8 * lane; j < d; j += 512) {
    float v[8], dn[8];
    load8(xr + j, v);
    load8(dr + j, dn);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      ss += v[q] * v[q];
      sg += g1[j + q] * dn[q] * v[q];
    }
  }
  const float r = 1.0f / sqrtf(seg_sum(ss, 64) / float(d) + eps);
  const float S = seg_sum(sg, 64);
  const float c3 = r * r * r * S / float(d);
  float *dxr = dx + int64_t(t) * d;
  for (int j = 8 * lane; j < d; j += 512) {
    float v[8], dn[8], o[8], tg[8];
    load8(xr + j, v);
    load8(dr + j, dn);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      o[q] = r * (g1[j + q] * dn[q]) - c3 * v[q];
      tg[q] = dn[q] * v[q] * r;
    }
    *(float4 *)(dxr + j) = make_float4(o[0], o[1], o[2], o[3]);
    *(float4 *)(dxr + j + 4) = make_float4(o[4], o[5], o[6], o[7]);
    *(float4 *)(dr + j) = make_float4(tg[0], tg[1], tg[2], tg[3]);
    *(float4 *)(dr + j + 4) = make_float4(tg[4], tg[5], tg[6], tg[7]);
  }
  for (int j = lane; j < dpsi; j += 64) dpsi_out[int64_t(t) * dpsi + j] = dr[d + j];
}

// Head weights from the gram of (dz, h^): with whitening, z = W (h^ - mu) /
// (sd + eps) + c, so dW = (G - dc mu^T) / (sd + eps); biases dc = sum dz.
// Then rho <- (1 - m) rho + m sqrt(sum of the squares of the language-model
// parts).  One thread per head weight.
__global__ __launch_bounds__(256) void heads_final_kernel(const float *__restrict__ G,
                                                          const float *__restrict__ dc, int A, int E1,
                                                          const float *__restrict__ mu,
                                                          const float *__restrict__ sd, float weps,
                                                          float *dWa, float *dca, float *dWe, float *dce,
                                                          float *dWb, float *dcb, const double *lmsq,
                                                          double *rho, float rho_m, double *lm_norm) {
  const int NZ = 3 * A + E1 + 4;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e < NZ * DR) {
    const int r = e / DR, j = e % DR;
    const int ax = r < 3 * A ? 0 : r < 3 * A + E1 ? 1 : 2;
    float v = G[e];
    if (mu) v = (v - dc[r] * mu[ax * DR + j]) / (sd[ax * DR + j] + weps);
    if (ax == 0) dWa[int64_t(r) * DR + j] = v;
    else if (ax == 1) dWe[int64_t(r - 3 * A) * DR + j] = v;
    else dWb[int64_t(r - 3 * A - E1) * DR + j] = v;
    if (j == 0) {
      if (ax == 0) dca[r] = dc[r];
      else if (ax == 1) dce[r - 3 * A] = dc[r];
      else dcb[r - 3 * A - E1] = dc[r];
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < 3) {
    const double nrm = sqrt(lmsq[threadIdx.x]);
    if (lm_norm) lm_norm[threadIdx.x] = nrm;
    if (rho && rho_m > 0.f) rho[threadIdx.x] = (1.0 - rho_m) * rho[threadIdx.x] + rho_m * nrm;
  }
}

hipError_t colsum(const float *A, int lda, int m, int N, float *part, float *out, double *out64,
                  hipStream_t st) {
  const int nc = (N + CS_CHUNK - 1) / CS_CHUNK;
  colsum_kernel<<<dim3((m + 63) / 64, nc), 256, 0, st>>>(A, lda, m, N, (double *)part);
  chunk_sum64_kernel<<<dim3((m + 255) / 256), 256, 0, st>>>((const double *)part, nc, m, out, out64);
  return hipGetLastError();
}

hipError_t gram(const float *A, int lda, int m, const float *B, int ldb, int n, int N, float *part,
                float *out, double *out64, hipStream_t st, int chunk = GR_CHUNK) {
  const int nc = (N + chunk - 1) / chunk;
  mm_f32_kernel<true><<<dim3((m + 63) / 64, (n + 63) / 64, nc), 256, 0, st>>>(A, lda, B, ldb, m, n, N,
                                                                             chunk, part, n);
  const int64_t ne = int64_t(m) * n;
  chunk_sum_kernel<<<dim3(unsigned((ne + 255) / 256)), 256, 0, st>>>(part, nc, ne, out, out64);
  return hipGetLastError();
}

}  // namespace

size_t relax_grad_part_floats(const triroute_cfg &cfg, int N) {
  const size_t nc = (N + GR_CHUNK - 1) / GR_CHUNK, ncw = (N + GR_CHUNK_W - 1) / GR_CHUNK_W;
  const size_t K1 = size_t(cfg.d_model + cfg.d_psi);
  const size_t NZ = size_t(3 * attn_groups(cfg) + cfg.n_experts + 5);
  const size_t ncs = (N + CS_CHUNK - 1) / CS_CHUNK;
  const size_t small = std::max(nc * NZ * DR, 2 * ncs * std::max(K1, std::max(NZ, size_t(DR))));
  const size_t wide = ncw * std::max(size_t(DR) * K1, size_t(DR) * DR);
  return std::max(small, wide);
}

hipError_t launch_relax_backward(const triroute_cfg &cfg, int N, const void *x, const float *psi,
                                 const triroute_router_w &w, const float *Wf,
                                 const float *white_mu, const float *white_sd, float white_eps,
                                 const RelaxBwdJob &j, hipStream_t st) {
  const int A = attn_groups(cfg), E1 = cfg.n_experts + 1, NZ = 3 * A + E1 + 4;
  const int d = cfg.d_model, dpsi = cfg.d_psi, K1 = d + dpsi;
  BwdTokArgs p;
  p.Z = j.z; p.a1 = j.a1; p.hpre = j.hpre; p.Wf = Wf;
  p.ya = j.y_attn; p.yb = j.y_bits; p.egate = j.egate; p.eidx = j.eidx; p.pos = j.pos;
  p.g_ya = j.g_attn; p.g_yb = j.g_bits; p.g_gate = j.g_gate;
  p.W2 = w.W2; p.gr = w.gr; p.stats = j.stats; p.usage = j.usage; p.rho = j.rho_io;
  p.lambda = j.lambda;
  p.dz = j.dz; p.dh = j.dh; p.da1 = j.da1; p.u = j.u; p.tgr = j.tgr; p.lmsq = j.lmsq;
  p.N = N; p.H = cfg.n_heads; p.A = A; p.E1 = E1; p.k = cfg.top_k; p.dh_ = cfg.head_dim;
  p.w = cfg.window; p.dkv = cfg.n_kv_heads * cfg.head_dim;
  p.inv_ta = 1.f / j.tau_a; p.inv_tb = 1.f / j.tau_b; p.zeta = j.zeta; p.alpha = j.alpha;
  p.beta = j.beta; p.gamma = j.gamma; p.eps = cfg.rms_eps;
  p.kappa_e = 3.f * float(cfg.d_model) * float(cfg.d_ff);
  relax_bwd_tok_kernel<<<dim3((N + 3) / 4), 256, 0, st>>>(p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // head weights: gram of (dz, h^) and the bias sums
  const RelaxGradOut &o = j.out;
#define TRY_HIP(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  TRY_HIP(gram(j.dz, NZ, NZ, j.hh, DR, DR, N, j.part, j.G, nullptr, st));
  TRY_HIP(colsum(j.dz, NZ, NZ, N, j.part, j.dc, nullptr, st));
  TRY_HIP(colsum(j.tgr, DR, DR, N, j.part, o.dgr, nullptr, st));
  TRY_HIP(gram(j.dh, DR, DR, j.u, DR, DR, N, j.part, o.dW2, nullptr, st, GR_CHUNK_W));
  TRY_HIP(colsum(j.dh, DR, DR, N, j.part, o.db2, nullptr, st));
  TRY_HIP(colsum(j.da1, DR, DR, N, j.part, o.db1, nullptr, st));
  TRY_HIP(colsum(j.lmsq, 4, 3, N, j.part, nullptr, j.lmsq_sum, st));
  // trunk input [n1; psi]: dW1 = da1^T s, then ds = da1 W1
  if (cfg.act == TRIROUTE_BF16)
    make_s_kernel<bf16><<<dim3((N + 3) / 4), 256, 0, st>>>((const bf16 *)x, w.g1, psi, N, d, dpsi,
                                                           cfg.rms_eps, j.s);
  else
    make_s_kernel<float><<<dim3((N + 3) / 4), 256, 0, st>>>((const float *)x, w.g1, psi, N, d, dpsi,
                                                            cfg.rms_eps, j.s);
  TRY_HIP(gram(j.da1, DR, DR, j.s, K1, K1, N, j.part, o.dW1, nullptr, st, GR_CHUNK_W));
  mm_f32_kernel<false><<<dim3((N + 63) / 64, (K1 + 63) / 64, 1), 256, 0, st>>>(
      j.da1, DR, w.W1, K1, N, K1, DR, DR, j.ds, K1);
  if (cfg.act == TRIROUTE_BF16)
    rms1_bwd_kernel<bf16><<<dim3((N + 3) / 4), 256, 0, st>>>((const bf16 *)x, w.g1, j.ds, N, d, dpsi,
                                                             cfg.rms_eps, o.dx, o.dpsi);
  else
    rms1_bwd_kernel<float><<<dim3((N + 3) / 4), 256, 0, st>>>((const float *)x, w.g1, j.ds, N, d, dpsi,
                                                              cfg.rms_eps, o.dx, o.dpsi);
  TRY_HIP(colsum(j.ds, K1, d, N, j.part, o.dg1, nullptr, st));
  heads_final_kernel<<<dim3((NZ * DR + 255) / 256), 256, 0, st>>>(
      j.G, j.dc, A, E1, white_mu, white_sd, white_eps, o.dWa, o.dca, o.dWe, o.dce, o.dWb, o.dcb,
      j.lmsq_sum, j.rho_io, j.rho_m, o.lm_norm);
#undef TRY_HIP
  return hipGetLastError();
}

}  // namespace tr
