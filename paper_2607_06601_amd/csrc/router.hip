// Controller (paper Sec. 3.3 controller equation) and hard inference
// decisions (Sec. 3.8), fp32 end to end.
//
//   rms_norm1   : r_i = 1/sqrt(mean(x_i^2) + eps); n1 = x r g1 (act out, for QKV)
//   trunk1      : u = GELU(W1 [x r g1 ; psi] + b1)        fp32 tiled GEMM, N x 128
//   tail        : h = W2 u + b2, h^ = RMSNorm(h) gr, z = W_{a,e,b} h^ + c,
//                 argmax / top-k decisions and gates
#include "kernels.hpp"

namespace tr {

// One wave per token row.
template <typename T>
__global__ __launch_bounds__(256) void rms_norm1_kernel(const T *__restrict__ x,
                                                        const float *__restrict__ g,
                                                        float *__restrict__ rinv,
                                                        T *__restrict__ n1, int N, int d,
                                                        float eps) {
  int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (row >= N) return;
  const T *xr = x + int64_t(row) * d;
  float ss = 0.f;
  for (int c = lane; c < d; c += 64) {
    float v = Act<T>::ld(xr, c);
    ss = fmaf(v, v, ss);
  }
  ss = wave_sum(ss);
  float r = 1.0f / sqrtf(ss / float(d) + eps);
  if (lane == 0) rinv[row] = r;
  if (n1) {
    T *nr = n1 + int64_t(row) * d;
    for (int c = lane; c < d; c += 64) Act<T>::st(nr, c, (Act<T>::ld(xr, c) * r) * g[c]);
  }
}

// u[N][128] = GELU([n1 ; psi] W1^T + b1), n1 = x * r * g1 formed on load.
// Block: 64 rows x 128 outputs, 256 threads, 4x8 outputs per thread.
template <typename T>
__global__ __launch_bounds__(256) void trunk1_kernel(const T *__restrict__ x,
                                                     const float *__restrict__ rinv,
                                                     const float *__restrict__ g1,
                                                     const float *__restrict__ psi,
                                                     const float *__restrict__ W1,
                                                     const float *__restrict__ b1,
                                                     float *__restrict__ u, int N, int d,
                                                     int dpsi) {
  constexpr int BM = 64, BN = 128, BK = 16;
  __shared__ __align__(16) float As[BK][BM + 4];
  __shared__ __align__(16) float Bs[BK][BN + 4];
  const int K = d + dpsi;
  const int tid = threadIdx.x;
  const int m0 = blockIdx.x * BM;
  const int tr = tid >> 4, tc = tid & 15;
  float acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  // loaders: A 64x16 (4 per thread), B 128x16 (8 per thread)
  const int ar = tid >> 2, ak = (tid & 3) * 4;
  const int bn = tid >> 1, bk = (tid & 1) * 8;
  const int arow = m0 + ar;
  const float rr = arow < N ? rinv[arow] : 0.f;
  for (int k0 = 0; k0 < K; k0 += BK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int k = k0 + ak + i;
      float v = 0.f;
      if (arow < N && k < K) {
        if (k < d)
          v = (Act<T>::ld(x, int64_t(arow) * d + k) * rr) * g1[k];
        else
          v = psi[int64_t(arow) * dpsi + (k - d)];
      }
      As[ak + i][ar] = v;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int k = k0 + bk + i;
      Bs[bk + i][bn] = k < K ? W1[int64_t(bn) * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][tr * 4 + i];
#pragma unroll
      for (int j = 0; j < 8; ++j) b[j] = Bs[kk][tc * 8 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int row = m0 + tr * 4 + i;
    if (row >= N) continue;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      int col = tc * 8 + j;
      float y = acc[i][j] + b1[col];
      u[int64_t(row) * BN + col] = 0.5f * y * (1.0f + erff(y * 0.70710678118654752f));
    }
  }
}

// Tail: 32 tokens per block, weights staged through LDS in two halves of
// the 128-wide router dimension.  LDS: weights [max(128, NZ)][65],
// activations [32][128], logits [32][NZ] (NZ = 3H + E + 5 <= 112: < 64 KB).
__global__ __launch_bounds__(256) void router_tail_kernel(
    const float *__restrict__ u, const float *__restrict__ W2, const float *__restrict__ b2,
    const float *__restrict__ gr, const float *__restrict__ Wa, const float *__restrict__ ca,
    const float *__restrict__ We, const float *__restrict__ ce, const float *__restrict__ Wb,
    const float *__restrict__ cb, uint8_t *__restrict__ mode, uint8_t *__restrict__ bit,
    int32_t *__restrict__ eidx, float *__restrict__ egate, int N, int H, int E1, int k,
    float eps) {
  constexpr int DR = 128, TB = 32, HALF = 64, LDW = HALF + 1;
  extern __shared__ __align__(16) float lds[];
  const int NZ = 3 * H + E1 + 4;
  const int wrows = NZ > DR ? NZ : DR;
  float *Ws = lds;                   // [wrows][LDW]
  float *Hs = Ws + wrows * LDW;      // [TB][DR]
  float *Zs = Hs + TB * DR;          // [TB][NZ]
  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * TB;
  for (int idx = tid; idx < TB * DR; idx += 256) {
    int t = t0 + idx / DR;
    Hs[idx] = t < N ? u[int64_t(t) * DR + idx % DR] : 0.f;
  }
  // h = W2 u + b2 ; thread: column c, tokens tg, tg + 2, ...
  const int c = tid & (DR - 1), tg = tid >> 7;
  float h[TB / 2];
#pragma unroll
  for (int j = 0; j < TB / 2; ++j) h[j] = b2[c];
  for (int half = 0; half < 2; ++half) {
    __syncthreads();
    for (int idx = tid; idx < DR * HALF; idx += 256)
      Ws[(idx / HALF) * LDW + idx % HALF] = W2[(idx / HALF) * DR + half * HALF + idx % HALF];
    __syncthreads();
    for (int kk = 0; kk < HALF; ++kk) {
      const float wv = Ws[c * LDW + kk];
#pragma unroll
      for (int j = 0; j < TB / 2; ++j)
        h[j] = fmaf(wv, Hs[(tg + 2 * j) * DR + half * HALF + kk], h[j]);
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < TB / 2; ++j) Hs[(tg + 2 * j) * DR + c] = h[j];
  __syncthreads();
  // RMSNorm of h per token (wave w handles tokens w, w + 4, ...)
  {
    const int lane = tid & 63, w = tid >> 6;
    for (int t = w; t < TB; t += 4) {
      const float a = Hs[t * DR + lane], b = Hs[t * DR + lane + 64];
      const float ss = wave_sum(a * a + b * b);
      const float r = 1.0f / sqrtf(ss / float(DR) + eps);
      Hs[t * DR + lane] = (a * r) * gr[lane];
      Hs[t * DR + lane + 64] = (b * r) * gr[lane + 64];
    }
  }
  // logits, the head weights staged in two halves as well
  for (int half = 0; half < 2; ++half) {
    __syncthreads();
    for (int idx = tid; idx < NZ * HALF; idx += 256) {
      const int z = idx / HALF, kk = half * HALF + idx % HALF;
      float wv;
      if (z < 3 * H)
        wv = Wa[z * DR + kk];
      else if (z < 3 * H + E1)
        wv = We[(z - 3 * H) * DR + kk];
      else
        wv = Wb[(z - 3 * H - E1) * DR + kk];
      Ws[z * LDW + idx % HALF] = wv;
    }
    __syncthreads();
    for (int idx = tid; idx < TB * NZ; idx += 256) {
      const int t = idx / NZ, z = idx % NZ;
      float acc = half ? Zs[t * NZ + z] : 0.f;
      for (int kk = 0; kk < HALF; ++kk)
        acc = fmaf(Ws[z * LDW + kk], Hs[t * DR + half * HALF + kk], acc);
      Zs[t * NZ + z] = acc;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < TB * NZ; idx += 256) {
    const int z = idx % NZ;
    const float bias = z < 3 * H ? ca[z] : z < 3 * H + E1 ? ce[z - 3 * H] : cb[z - 3 * H - E1];
    Zs[idx] += bias;
  }
  __syncthreads();
  if (tid < TB && t0 + tid < N) {
    const int t = t0 + tid;
    const float *z = Zs + tid * NZ;
    for (int hh = 0; hh < H; ++hh) {
      const float *za = z + 3 * hh;
      int best = 0;
      if (za[1] > za[best]) best = 1;
      if (za[2] > za[best]) best = 2;
      mode[int64_t(t) * H + hh] = uint8_t(best);
    }
    const float *zb = z + 3 * H + E1;
    int bb = 0;
    for (int j = 1; j < 4; ++j)
      if (zb[j] > zb[bb]) bb = j;
    bit[t] = uint8_t(bb);
    const float *ze = z + 3 * H;
    // top-k by logit (softmax is monotone); ties go to the lower id
    uint64_t taken = 0;
    float zmax = ze[0];
    for (int j = 1; j < E1; ++j) zmax = fmaxf(zmax, ze[j]);
    float tot = 0.f;
    for (int s = 0; s < k; ++s) {
      int best = -1;
      for (int j = 0; j < E1; ++j) {
        if (taken >> j & 1) continue;
        if (best < 0 || ze[j] > ze[best]) best = j;
      }
      taken |= 1ull << best;
      tot += expf(ze[best] - zmax);
    }
    int s = 0;
    for (int j = 0; j < E1; ++j) {
      if (!(taken >> j & 1)) continue;
      eidx[int64_t(t) * k + s] = j;
      egate[int64_t(t) * k + s] = expf(ze[j] - zmax) / tot;
      ++s;
    }
  }
}

size_t router_tail_lds(int H, int E1) {
  const int NZ = 3 * H + E1 + 4;
  const int wrows = NZ > 128 ? NZ : 128;
  return sizeof(float) * (size_t(wrows) * 65 + 32 * 128 + 32 * size_t(NZ));
}

hipError_t launch_router(const triroute_cfg &cfg, int N, const void *x, const float *psi,
                         const triroute_router_w &w, void *n1, uint8_t *mode, uint8_t *bit,
                         int32_t *eidx, float *egate, float *rinv, float *u,
                         hipStream_t st) {
  const int d = cfg.d_model;
  dim3 g1((N + 3) / 4);
  dim3 g2((N + 63) / 64);
  if (cfg.act == TRIROUTE_BF16) {
    rms_norm1_kernel<bf16><<<g1, 256, 0, st>>>((const bf16 *)x, w.g1, rinv, (bf16 *)n1, N, d,
                                               cfg.rms_eps);
    trunk1_kernel<bf16><<<g2, 256, 0, st>>>((const bf16 *)x, rinv, w.g1, psi, w.W1, w.b1, u,
                                            N, d, cfg.d_psi);
  } else {
    rms_norm1_kernel<float><<<g1, 256, 0, st>>>((const float *)x, w.g1, rinv, (float *)n1, N, d,
                                                cfg.rms_eps);
    trunk1_kernel<float><<<g2, 256, 0, st>>>((const float *)x, rinv, w.g1, psi, w.W1, w.b1, u,
                                             N, d, cfg.d_psi);
  }
  size_t lds = router_tail_lds(cfg.n_heads, cfg.n_experts + 1);
  router_tail_kernel<<<dim3((N + 31) / 32), 256, lds, st>>>(u, w.W2, w.b2, w.gr, w.Wa, w.ca, w.We, w.ce, w.Wb,
                                           w.cb, mode, bit, eidx, egate, N, cfg.n_heads,
                                           cfg.n_experts + 1, cfg.top_k, cfg.rms_eps);
  return hipGetLastError();
}

hipError_t router_prepare() { return hipSuccess; }

}  // namespace tr
