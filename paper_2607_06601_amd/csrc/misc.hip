// Second RMSNorm and the expert combine of paper Sec. 3.1 / 3.2 (B):
//   n2 = RMSNorm(xt; g2);  x_out = xt + sum_{slot: e != 0} gate * Y[i*k + slot]
// Slots are summed in slot order (deterministic); a token whose every slot is
// the null expert gets x_out = xt exactly.
#include "kernels.hpp"

namespace tr {

// One wave per row, 8 consecutive elements per lane access (d % 64 == 0).
template <typename T>
__global__ __launch_bounds__(256) void rms_norm2_kernel(const T *__restrict__ x,
                                                        const T *__restrict__ g,
                                                        T *__restrict__ out, int N, int d,
                                                        float eps) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= N) return;
  const T *xr = x + int64_t(row) * d;
  float ss = 0.f;
  for (int c = lane * 8; c < d; c += 512) {
    float v[8];
    load8(xr + c, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss = fmaf(v[i], v[i], ss);
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / float(d) + eps);
  T *orow = out + int64_t(row) * d;
  for (int c = lane * 8; c < d; c += 512) {
    float v[8], gv[8];
    load8(xr + c, v);
    load8(g + c, gv);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (v[i] * r) * gv[i];
    store8(orow + c, v);
  }
}

// One thread per 8 consecutive features of a token.
template <typename T>
__global__ __launch_bounds__(256) void moe_combine_kernel(const T *__restrict__ xt,
                                                          const float *__restrict__ Y,
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
      load8(Y + (int64_t(i) * k + s) * d + c, ys);
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

hipError_t launch_rms_norm2(const triroute_cfg &cfg, int N, const void *x, const void *g,
                            void *out, hipStream_t st) {
  dim3 grid((N + 3) / 4);
  if (cfg.act == TRIROUTE_BF16)
    rms_norm2_kernel<bf16><<<grid, 256, 0, st>>>((const bf16 *)x, (const bf16 *)g, (bf16 *)out, N,
                                                 cfg.d_model, cfg.rms_eps);
  else
    rms_norm2_kernel<float><<<grid, 256, 0, st>>>((const float *)x, (const float *)g,
                                                  (float *)out, N, cfg.d_model, cfg.rms_eps);
  return hipGetLastError();
}

hipError_t launch_moe_combine(const triroute_cfg &cfg, int N, const void *xt, const float *Y,
                              const int32_t *eidx, const float *egate, void *xout,
                              hipStream_t st) {
  int64_t total = int64_t(N) * (cfg.d_model / 8);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (cfg.act == TRIROUTE_BF16)
    moe_combine_kernel<bf16><<<dim3(unsigned(blocks)), 256, 0, st>>>(
        (const bf16 *)xt, Y, eidx, egate, (bf16 *)xout, N, cfg.d_model, cfg.top_k);
  else
    moe_combine_kernel<float><<<dim3(unsigned(blocks)), 256, 0, st>>>(
        (const float *)xt, Y, eidx, egate, (float *)xout, N, cfg.d_model, cfg.top_k);
  return hipGetLastError();
}

}  // namespace tr
