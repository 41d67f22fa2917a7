// Controller (paper Sec. 3.3 controller equation) and hard inference
// decisions (Sec. 3.8), fp32 end to end.
//
//   rms_norm1   : r_i = 1/sqrt(mean(x_i^2) + eps); n1 = x r g1 (act out, for QKV; fp64)
//   trunk1      : partial W1 [x r g1 ; psi] over K chunks    fp32 MFMA, N x 128
//   tail        : u = GELU(sum + b1), h = W2 u + b2, h^ = RMSNorm(h) gr,
//                 z = W_{a,e,b} h^ + c, argmax / top-k decisions and gates
#include "kernels.hpp"

namespace tr {

// One wave per token row, 8 consecutive elements per lane access.
template <typename T>
__global__ __launch_bounds__(256) void rms_norm1_kernel(const T *__restrict__ x,
                                                        const float *__restrict__ g,
                                                        float *__restrict__ rinv,
                                                        T *__restrict__ n1, int N, int d,
                                                        float eps, const RopeJob rj) {
  int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (row >= N) return;
  if (rj.tab)  // the token's rotation table entries (one lane per pair)
    for (int j = lane; j < rj.hd; j += 64) rj.tab[int64_t(row) * rj.hd + j] = rope_entry(rj, row, j);
  const T *xr = x + int64_t(row) * d;
  // fp32 scale for the controller (fp32 end to end); fp64 for the n1 the
  // projections read, rounded once to the activation dtype
  float ss = 0.f;
  double sd = 0.0;
  for (int c = lane * 8; c < d; c += 512) {
    float v[8];
    load8(xr + c, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      ss = fmaf(v[i], v[i], ss);
      sd = fma(double(v[i]), double(v[i]), sd);
    }
  }
  ss = wave_sum(ss);
  float r = 1.0f / sqrtf(ss / float(d) + eps);
  if (lane == 0) rinv[row] = r;
  if (n1) {
    sd = wave_sum(sd);
    const double rd = 1.0 / sqrt(sd / double(d) + double(eps));
    T *nr = n1 + int64_t(row) * d;
    for (int c = lane * 8; c < d; c += 512) {
      float v[8], gv[8];
      double o[8];
      load8(xr + c, v);
      load8(g + c, gv);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = (double(v[i]) * rd) * double(gv[i]);
      store8(nr + c, o);
    }
  }
}

typedef float f32x4r __attribute__((ext_vector_type(4)));

// Split of the trunk's K = d + d_psi inputs over blocks, so that a small
// batch (decode) still spreads over the chip: K chunks are multiples of 32.
void router_split(int N, int K, int &ks, int &kchunk) {
  const int mt = (N + 63) / 64;
  int want = (512 + mt - 1) / mt;
  const int kmax = (K + 63) / 64;
  want = want < 1 ? 1 : want > kmax ? kmax : want;
  kchunk = ((K + want - 1) / want + 31) / 32 * 32;
  ks = (K + kchunk - 1) / kchunk;
}

// Partial trunk pre-activations upart[ks][N][128] = [n1 ; psi] W1^T over the
// block's K chunk, with n1 = x r g1 formed on load (fp32 MFMA 16x16x4).
// Block: 64 rows x 128 outputs, 4 waves of 16 rows; the next K step is
// fetched into registers while the current one is multiplied from LDS.
template <typename T>
__global__ __launch_bounds__(256) void trunk1_kernel(const T *__restrict__ x,
                                                     const float *__restrict__ rinv,
                                                     const float *__restrict__ g1,
                                                     const float *__restrict__ psi,
                                                     const float *__restrict__ W1,
                                                     float *__restrict__ upart, int N, int d,
                                                     int dpsi, int kchunk) {
  constexpr int BM = 64, BK = 32, LD = BK + 1;
  __shared__ float As[2][BM][LD];
  __shared__ float Bs[2][128][LD];
  const int K = d + dpsi;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.x * BM;
  const int kb = blockIdx.y * kchunk, ke = min(K, kb + kchunk);
  f32x4r acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = f32x4r{0.f, 0.f, 0.f, 0.f};
  const int ar = tid >> 2, ak = (tid & 3) * 8;
  const int br = tid >> 1, bk = (tid & 1) * 16;
  const int arow = m0 + ar;
  const float rr = arow < N ? rinv[arow] : 0.f;
  float ra[8], rb[16];
  auto fetch = [&](int k0) {
    // A: 8 consecutive inputs of row arow; whole 8-runs inside x use one
    // 16-byte load (d % 64 == 0, so a run never straddles x and psi)
    const int ka = k0 + ak;
    if (arow < N && ka + 8 <= ke && ka + 8 <= d) {
      float xv[8], gv[8];
      load8(x + int64_t(arow) * d + ka, xv);
      load8(g1 + ka, gv);
#pragma unroll
      for (int i = 0; i < 8; ++i) ra[i] = (xv[i] * rr) * gv[i];
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int k = ka + i;
        float v = 0.f;
        if (arow < N && k < ke)
          v = k < d ? (Act<T>::ld(x, int64_t(arow) * d + k) * rr) * g1[k]
                    : psi[int64_t(arow) * dpsi + (k - d)];
        ra[i] = v;
      }
    }
    // B: 16 consecutive inputs of W1 row br (K % 4 == 0: 16-byte aligned)
    const int kb0 = k0 + bk;
    if (kb0 + 16 <= ke) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 w = *(const float4 *)(W1 + int64_t(br) * K + kb0 + 4 * i);
        rb[4 * i] = w.x; rb[4 * i + 1] = w.y; rb[4 * i + 2] = w.z; rb[4 * i + 3] = w.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int k = kb0 + i;
        rb[i] = k < ke ? W1[int64_t(br) * K + k] : 0.f;
      }
    }
  };
  auto put = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 8; ++i) As[buf][ar][ak + i] = ra[i];
#pragma unroll
    for (int i = 0; i < 16; ++i) Bs[buf][br][bk + i] = rb[i];
  };
  fetch(kb);
  put(0);
  __syncthreads();
  int buf = 0;
  for (int k0 = kb; k0 < ke; k0 += BK) {
    const bool more = k0 + BK < ke;
    if (more) fetch(k0 + BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 4) {
      const float av = As[buf][16 * wave + (lane & 15)][kk + (lane >> 4)];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
            av, Bs[buf][16 * j + (lane & 15)][kk + (lane >> 4)], acc[j], 0, 0, 0);
    }
    if (more) put(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  float *out = upart + int64_t(blockIdx.y) * N * 128;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = m0 + 16 * wave + 4 * (lane >> 4) + r;
    if (row >= N) continue;
#pragma unroll
    for (int j = 0; j < 8; ++j) out[int64_t(row) * 128 + 16 * j + (lane & 15)] = acc[j][r];
  }
}

// Tail in 16-token tiles (4 waves per tile, fp32 MFMA 16x16x4), two tiles
// at a time per block (8 waves: two per SIMD, so one tile's latencies hide
// behind the other's work), with W2 and the head weights staged in LDS once
// by coalesced loads:
//   u = GELU(sum of trunk partials + b1); h = W2 u + b2; h^ = RMSNorm(h) gr;
//   z = [Wa; We; Wb] h^ + [ca; ce; cb]; argmax / top-k decisions and gates.
constexpr int RT_TB = 16, RT_DR = 128, RT_LD = RT_DR + 1, RT_NZ = 112;
constexpr size_t RT_LDS = sizeof(float) * (size_t(RT_DR + RT_NZ + 4 * RT_TB) * RT_LD);

__global__ __launch_bounds__(512) void router_tail_kernel(
    const float *__restrict__ upart, int KS, const float *__restrict__ b1,
    const float *__restrict__ W2, const float *__restrict__ b2, const float *__restrict__ gr,
    const float *__restrict__ Wa, const float *__restrict__ ca, const float *__restrict__ We,
    const float *__restrict__ ce, const float *__restrict__ Wb, const float *__restrict__ cb,
    uint8_t *__restrict__ mode, uint8_t *__restrict__ bit, int32_t *__restrict__ eidx,
    float *__restrict__ egate, int N, int H, int A, int E1, int k, float eps, TailTap tap) {
  constexpr int TB = RT_TB, DR = RT_DR, LD = RT_LD;
  extern __shared__ __align__(16) float rt_lds[];
  float(*W2s)[LD] = (float(*)[LD])rt_lds;              // [128][LD]
  float(*Wzs)[LD] = (float(*)[LD])(rt_lds + DR * LD);  // [NZ][LD]
  // group g of 4 waves works on its own tile with its own Us / Zs
  const int g = threadIdx.x >> 8, tid = threadIdx.x & 255, lane = tid & 63, wave = tid >> 6;
  float(*Us)[LD] = (float(*)[LD])(rt_lds + (DR + RT_NZ + 2 * TB * g) * LD);
  float(*Zs)[LD] = (float(*)[LD])(rt_lds + (DR + RT_NZ + 2 * TB * g + TB) * LD);
  const int NZ = 3 * A + E1 + 4;
  for (int i = threadIdx.x; i < DR * DR / 4; i += 512) {
    const int r = i / (DR / 4), c4 = (i % (DR / 4)) * 4;
    const float4 v = *(const float4 *)(W2 + r * DR + c4);
    W2s[r][c4] = v.x; W2s[r][c4 + 1] = v.y; W2s[r][c4 + 2] = v.z; W2s[r][c4 + 3] = v.w;
  }
  for (int i = threadIdx.x; i < NZ * DR / 4; i += 512) {
    const int z = i / (DR / 4), c4 = (i % (DR / 4)) * 4;
    const float *wz = z < 3 * A ? Wa + z * DR
                      : z < 3 * A + E1 ? We + (z - 3 * A) * DR : Wb + (z - 3 * A - E1) * DR;
    const float4 v = *(const float4 *)(wz + c4);
    Wzs[z][c4] = v.x; Wzs[z][c4 + 1] = v.y; Wzs[z][c4 + 2] = v.z; Wzs[z][c4 + 3] = v.w;
  }
  // the weights stay in LDS while the block walks its token tiles; with at
  // most 4 trunk chunks the next tile's partials are loaded while the
  // current tile is computed
  constexpr int EPT = TB * DR / 256;
  float pre[4][EPT];
  auto load_parts = [&](int tt0, int s0, float (*v)[EPT]) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const int idx = tid + 256 * e, t = idx / DR, c = idx % DR;
        v[j][e] = (s0 + j < KS && tt0 + t < N)
                      ? upart[(int64_t(s0 + j) * N + tt0 + t) * DR + c] : 0.f;
      }
  };
  const bool prefetch = KS <= 4;
  // both groups run every round (a group past the last token masks its
  // work), so the block's barriers stay matched
  const int stride = gridDim.x * 2 * TB;
  if (prefetch) load_parts(blockIdx.x * 2 * TB + g * TB, 0, pre);
  for (int base = blockIdx.x * 2 * TB; base < N; base += stride) {
  const int t0 = base + g * TB;
  {
    // u = GELU(sum of the KS trunk partials + b1): thread tid owns elements
    // tid + 256 e of the block's 16 x 128; partials are summed in chunk order
    float sacc[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) sacc[e] = 0.f;
    if (prefetch) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < EPT; ++e) sacc[e] += pre[j][e];
      if (t0 + stride < N) load_parts(t0 + stride, 0, pre);
    } else {
      for (int s0 = 0; s0 < KS; s0 += 4) {
        float v[4][EPT];
        load_parts(t0, s0, v);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < EPT; ++e) sacc[e] += v[j][e];
      }
    }
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int idx = tid + 256 * e, t = idx / DR, c = idx % DR;
      float y = 0.f;
      if (t0 + t < N) {
        y = sacc[e] + b1[c];
        if (tap.a1) tap.a1[int64_t(t0 + t) * DR + c] = y;
        y = 0.5f * y * (1.0f + erff(y * 0.70710678118654752f));
      }
      Us[t][c] = y;
    }
  }
  __syncthreads();
  // h: wave w computes columns 32 w .. 32 w + 31 (two accumulators per
  // column tile, even and odd K steps, so that two MFMA chains interleave)
  f32x4r hacc[2][2];
#pragma unroll
  for (int j = 0; j < 2; ++j) hacc[j][0] = hacc[j][1] = f32x4r{0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int kk = 0; kk < DR; kk += 4) {
    const float av = Us[lane & 15][kk + (lane >> 4)];
#pragma unroll
    for (int j = 0; j < 2; ++j)
      hacc[j][(kk >> 2) & 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(
          av, W2s[32 * wave + 16 * j + (lane & 15)][kk + (lane >> 4)], hacc[j][(kk >> 2) & 1], 0,
          0, 0);
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = 32 * wave + 16 * j + (lane & 15);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float hv = (hacc[j][0][r] + hacc[j][1][r]) + b2[n];
      Us[4 * (lane >> 4) + r][n] = hv;
      const int tr_ = t0 + 4 * (lane >> 4) + r;
      if (tap.hpre && tr_ < N) tap.hpre[int64_t(tr_) * DR + n] = hv;
    }
  }
  __syncthreads();
  {
    // RMSNorm of h: wave w takes tokens w, w + 4, w + 8, w + 12 together
    constexpr int TPW = TB / 4;
    float av[TPW], bv[TPW], ss[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      av[j] = Us[wave + 4 * j][lane];
      bv[j] = Us[wave + 4 * j][lane + 64];
      ss[j] = av[j] * av[j] + bv[j] * bv[j];
    }
#pragma unroll
    for (int j = 0; j < TPW; ++j) ss[j] = seg_sum(ss[j], 64);
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const float r = 1.0f / sqrtf(ss[j] / float(DR) + eps);
      Us[wave + 4 * j][lane] = (av[j] * r) * gr[lane];
      Us[wave + 4 * j][lane + 64] = (bv[j] * r) * gr[lane + 64];
      const int tj = t0 + wave + 4 * j;
      if (tap.h && tj < N) {
        tap.h[int64_t(tj) * DR + lane] = Us[wave + 4 * j][lane];
        tap.h[int64_t(tj) * DR + lane + 64] = Us[wave + 4 * j][lane + 64];
      }
    }
  }
  __syncthreads();
  for (int nt = wave; nt * 16 < NZ; nt += 4) {
    const int z = nt * 16 + (lane & 15);
    const int zr = z < NZ ? z : NZ - 1;
    f32x4r zacc[2] = {f32x4r{0.f, 0.f, 0.f, 0.f}, f32x4r{0.f, 0.f, 0.f, 0.f}};
#pragma unroll 8
    for (int kk = 0; kk < DR; kk += 4)
      zacc[(kk >> 2) & 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(
          Us[lane & 15][kk + (lane >> 4)], Wzs[zr][kk + (lane >> 4)], zacc[(kk >> 2) & 1], 0, 0, 0);
    if (z < NZ) {
      const float bias = z < 3 * A ? ca[z] : z < 3 * A + E1 ? ce[z - 3 * A] : cb[z - 3 * A - E1];
#pragma unroll
      for (int r = 0; r < 4; ++r) Zs[4 * (lane >> 4) + r][z] = (zacc[0][r] + zacc[1][r]) + bias;
    }
  }
  __syncthreads();
  if (tap.z)
    for (int it = tid; it < TB * NZ; it += 256) {
      const int tt = it / NZ, z = it - tt * NZ;
      if (t0 + tt < N) tap.z[int64_t(t0 + tt) * NZ + z] = Zs[tt][z];
    }
  // modes: one thread per (token, head); argmax, first maximum on ties
  const int HA = H / A;  // heads per decision group
  for (int it = tid; it < TB * H; it += 256) {
    const int tt = it / H, hh = it - tt * H;
    if (t0 + tt >= N) continue;
    const float *za = Zs[tt] + 3 * (hh / HA);
    int best = 0;
    if (za[1] > za[best]) best = 1;
    if (za[2] > za[best]) best = 2;
    mode[int64_t(t0 + tt) * H + hh] = uint8_t(best);
  }
  // bit width and experts: wave w takes tokens w, w + 4, ...; lane j holds
  // expert logit j (E + 1 <= 64)
  for (int tt = wave; tt < TB; tt += 4) {
    const int t = t0 + tt;
    if (t >= N) break;  // wave-uniform
    const float *z = Zs[tt];
    if (lane == 0) {
      const float *zb = z + 3 * A + E1;
      int bb = 0;
      for (int j = 1; j < 4; ++j)
        if (zb[j] > zb[bb]) bb = j;
      bit[t] = uint8_t(bb);
    }
    // top-k by logit (softmax is monotone), ties to the lower id; the gate
    // renormalises over the selected set, null included
    const float zj = lane < E1 ? z[3 * A + lane] : -INFINITY;
    const float zmax = seg_max(zj, 64);
    uint64_t taken = 0;
    float tot = 0.f;
    for (int sl = 0; sl < k; ++sl) {
      const float cand = (lane < E1 && !(taken >> lane & 1)) ? zj : -INFINITY;
      const float m = seg_max(cand, 64);
      const uint64_t hit = __ballot(lane < E1 && !(taken >> lane & 1) && cand == m);
      const int best = __ffsll((unsigned long long)hit) - 1;
      taken |= 1ull << best;
      tot += expf(m - zmax);
    }
    if (taken >> lane & 1) {
      const int sl = __popcll(taken & lanemask_lt());
      eidx[int64_t(t) * k + sl] = lane;
      egate[int64_t(t) * k + sl] = expf(zj - zmax) / tot;
    }
  }
  __syncthreads();  // Us / Zs are reused by the next tile
  }
}

// The same tail for few tokens (decode), one 256-thread block per token, so
// that each step's weight reads are all in flight at once instead of a wave
// walking whole rows: thread j < 128 sums the trunk partials of column j (in
// chunk order, then b1); two threads per row of W2 (64 columns each) and
// four per logit row (32 columns each), their partial sums added by lane
// shuffles (every thread of a row ends with the same value).  fp32 either
// way; the products are summed in a different order than the MFMA tail, and
// the decisions do not depend on it above the routing margin.
constexpr int RTB_MAXKS = 48;
__global__ __launch_bounds__(256) void router_tail_blk_kernel(
    const float *__restrict__ upart, int KS, const float *__restrict__ b1,
    const float *__restrict__ W2, const float *__restrict__ b2, const float *__restrict__ gr,
    const float *__restrict__ Wa, const float *__restrict__ ca, const float *__restrict__ We,
    const float *__restrict__ ce, const float *__restrict__ Wb, const float *__restrict__ cb,
    uint8_t *__restrict__ mode, uint8_t *__restrict__ bit, int32_t *__restrict__ eidx,
    float *__restrict__ egate, int N, int H, int A, int E1, int k, float eps, TailTap tap) {
  constexpr int DR = RT_DR;
  __shared__ __align__(16) float us[DR], hs[DR], zs[RT_NZ];
  __shared__ float red[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t = blockIdx.x;  // grid = N
  const int NZ = 3 * A + E1 + 4;
  // u = GELU(sum of the KS trunk partials + b1)
  if (tid < DR) {
    float p[RTB_MAXKS];
#pragma unroll
    for (int s = 0; s < RTB_MAXKS; ++s)
      if (s < KS) p[s] = upart[(int64_t(s) * N + t) * DR + tid];
    float a = 0.f;
#pragma unroll
    for (int s = 0; s < RTB_MAXKS; ++s)
      if (s < KS) a += p[s];
    a += b1[tid];
    if (tap.a1) tap.a1[int64_t(t) * DR + tid] = a;
    us[tid] = 0.5f * a * (1.0f + erff(a * 0.70710678118654752f));
  }
  __syncthreads();
  // h = W2 u + b2, row r = tid / 2; h^ = RMSNorm(h) gr
  {
    const int r = tid >> 1, c0 = (tid & 1) * (DR / 2);
    const float4 *w = (const float4 *)(W2 + r * DR + c0);
    float4 x[DR / 8];
#pragma unroll
    for (int i = 0; i < DR / 8; ++i) x[i] = w[i];
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < DR / 8; ++i) {
      const float4 u = *(const float4 *)(us + c0 + 4 * i);
      acc = fmaf(x[i].x, u.x, acc); acc = fmaf(x[i].y, u.y, acc);
      acc = fmaf(x[i].z, u.z, acc); acc = fmaf(x[i].w, u.w, acc);
    }
    acc += __shfl_xor(acc, 1, 64);
    const float h = acc + b2[r];
    const float ssw = seg_sum((tid & 1) ? 0.f : h * h, 64);  // the wave's 32 rows
    if (lane == 0) red[wave] = ssw;
    __syncthreads();
    const float ss = (red[0] + red[1]) + (red[2] + red[3]);
    const float rr = 1.0f / sqrtf(ss / float(DR) + eps);
    const float hn = (h * rr) * gr[r];
    if ((tid & 1) == 0) {
      hs[r] = hn;
      if (tap.hpre) tap.hpre[int64_t(t) * DR + r] = h;
      if (tap.h) tap.h[int64_t(t) * DR + r] = hn;
    }
  }
  __syncthreads();
  // z = [Wa; We; Wb] h^ + [ca; ce; cb], logit row z0 + tid / 4
  for (int z0 = 0; z0 < NZ; z0 += 64) {
    const int z = z0 + (tid >> 2), c0 = (tid & 3) * (DR / 4);
    float acc = 0.f;
    if (z < NZ) {
      const float *wz = z < 3 * A ? Wa + z * DR : z < 3 * A + E1 ? We + (z - 3 * A) * DR
                                                                  : Wb + (z - 3 * A - E1) * DR;
      float4 x[DR / 16];
#pragma unroll
      for (int i = 0; i < DR / 16; ++i) x[i] = ((const float4 *)(wz + c0))[i];
#pragma unroll
      for (int i = 0; i < DR / 16; ++i) {
        const float4 u = *(const float4 *)(hs + c0 + 4 * i);
        acc = fmaf(x[i].x, u.x, acc); acc = fmaf(x[i].y, u.y, acc);
        acc = fmaf(x[i].z, u.z, acc); acc = fmaf(x[i].w, u.w, acc);
      }
    }
    acc += __shfl_xor(acc, 1, 64);
    acc += __shfl_xor(acc, 2, 64);
    if (z < NZ && (tid & 3) == 0) {
      const float bias = z < 3 * A ? ca[z] : z < 3 * A + E1 ? ce[z - 3 * A] : cb[z - 3 * A - E1];
      zs[z] = acc + bias;
      if (tap.z) tap.z[int64_t(t) * NZ + z] = zs[z];
    }
  }
  __syncthreads();
  if (wave != 0) return;  // decisions by the first wave (no barrier below)
  const int HA = H / A;
  for (int hh = lane; hh < H; hh += 64) {
    const float *za = zs + 3 * (hh / HA);
    int best = 0;
    if (za[1] > za[best]) best = 1;
    if (za[2] > za[best]) best = 2;
    mode[int64_t(t) * H + hh] = uint8_t(best);
  }
  if (lane == 0) {
    const float *zb = zs + 3 * A + E1;
    int bb = 0;
    for (int j = 1; j < 4; ++j)
      if (zb[j] > zb[bb]) bb = j;
    bit[t] = uint8_t(bb);
  }
  const float zj = lane < E1 ? zs[3 * A + lane] : -INFINITY;
  const float zmax = seg_max(zj, 64);
  uint64_t taken = 0;
  float tot = 0.f;
  for (int sl = 0; sl < k; ++sl) {
    const float cand = (lane < E1 && !(taken >> lane & 1)) ? zj : -INFINITY;
    const float m = seg_max(cand, 64);
    const uint64_t hit = __ballot(lane < E1 && !(taken >> lane & 1) && cand == m);
    const int best = __ffsll((unsigned long long)hit) - 1;
    taken |= 1ull << best;
    tot += expf(m - zmax);
  }
  if (taken >> lane & 1) {
    const int sl = __popcll(taken & lanemask_lt());
    eidx[int64_t(t) * k + sl] = lane;
    egate[int64_t(t) * k + sl] = expf(zj - zmax) / tot;
  }
}

hipError_t launch_router(const triroute_cfg &cfg, int N, const void *x, const float *psi,
                         const triroute_router_w &w, void *n1, uint8_t *mode, uint8_t *bit,
                         int32_t *eidx, float *egate, float *rinv, float *u, const RopeJob *rope,
                         hipStream_t st, TailTap tap) {
  RopeJob rj{};
  if (rope) rj = *rope;
  const int d = cfg.d_model;
  int ks, kchunk;
  router_split(N, d + cfg.d_psi, ks, kchunk);
  dim3 g1((N + 3) / 4);
  dim3 g2((N + 63) / 64, ks);
  if (cfg.act == TRIROUTE_BF16) {
    rms_norm1_kernel<bf16><<<g1, 256, 0, st>>>((const bf16 *)x, w.g1, rinv, (bf16 *)n1, N, d,
                                               cfg.rms_eps, rj);
    trunk1_kernel<bf16><<<g2, 256, 0, st>>>((const bf16 *)x, rinv, w.g1, psi, w.W1, u, N, d,
                                            cfg.d_psi, kchunk);
  } else {
    rms_norm1_kernel<float><<<g1, 256, 0, st>>>((const float *)x, w.g1, rinv, (float *)n1, N, d,
                                                cfg.rms_eps, rj);
    trunk1_kernel<float><<<g2, 256, 0, st>>>((const float *)x, rinv, w.g1, psi, w.W1, u, N, d,
                                             cfg.d_psi, kchunk);
  }
  if (N <= 256 && ks <= RTB_MAXKS) {  // few tokens: one block per token
    router_tail_blk_kernel<<<dim3(N), 256, 0, st>>>(
        u, ks, w.b1, w.W2, w.b2, w.gr, w.Wa, w.ca, w.We, w.ce, w.Wb, w.cb, mode, bit, eidx, egate,
        N, cfg.n_heads, attn_groups(cfg), cfg.n_experts + 1, cfg.top_k, cfg.rms_eps, tap);
    return hipGetLastError();
  }
  // one block per CU at most (the weights fill most of its LDS), each
  // loading them once and then taking every 256th token tile
  const int pairs = ((N + RT_TB - 1) / RT_TB + 1) / 2;
  router_tail_kernel<<<dim3(pairs < 256 ? pairs : 256), 512, RT_LDS, st>>>(
      u, ks, w.b1, w.W2, w.b2, w.gr, w.Wa, w.ca, w.We, w.ce, w.Wb, w.cb, mode, bit, eidx, egate, N,
      cfg.n_heads, attn_groups(cfg), cfg.n_experts + 1, cfg.top_k, cfg.rms_eps, tap);
  return hipGetLastError();
}

hipError_t router_prepare() { return hipSuccess; }

}  // namespace tr
