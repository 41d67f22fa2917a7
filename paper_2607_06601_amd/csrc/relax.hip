// Training-time relaxed controller forward (paper Sec. 3.4-3.7, Algorithm 1
// steps 1-3, 5 and 6): per-axis whitening folded into the head weights, the
// straight-through Gumbel-softmax of the attention and bit heads, the
// top-k softmax of the expert head (the inference tail), the expected costs
// and the per-axis balance, z and entropy-floor losses, the regulariser and
// the dual step.  The controller trunk and tail are the inference kernels
// of router.hip; this file adds the three kernels around them.
//
// Every batch reduction is deterministic: each block folds a fixed token
// range in a fixed order into one column of partial sums (fp64), and one
// wave per field adds that field's column in a fixed order.
#include "kernels.hpp"

namespace tr {

namespace {

constexpr int DR = 128;      // router width
constexpr int RX_BLOCKS = 256, RX_WAVES = 16;
// the fields of one block's partial sums (fp64); expert fields sized for E + 1 <= 64
constexpr int RX_ACNT = 0, RX_AP = 3, RX_ALSE = 6, RX_BCNT = 7, RX_BP = 11, RX_BLSE = 15,
              RX_ELSE = 16, RX_CF = 17, RX_CM = 18, RX_DF = 19, RX_DM = 20, RX_ECNT = 21,
              RX_EP = RX_ECNT + 64, RX_HS = RX_EP + 64, RX_HQ = RX_HS + DR, RX_F = RX_HQ + DR;

__device__ __forceinline__ double wave_sum_d(double v) {
  // fixed butterfly: every lane ends with the same sum, in the same order
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// One block per logit row r of [Wa; We; Wb]: with the axis statistics
// (mu, sd) of that row's head, W'[r][j] = W[r][j] / (sd[j] + eps) and
// c'[r] = c[r] - sum_j W'[r][j] mu[j], so that W' h^ + c' equals
// W ((h^ - mu) / (sd + eps)) + c.
__global__ __launch_bounds__(DR) void white_fold_kernel(
    const float *__restrict__ Wa, const float *__restrict__ ca, const float *__restrict__ We,
    const float *__restrict__ ce, const float *__restrict__ Wb, const float *__restrict__ cb,
    const float *__restrict__ mu, const float *__restrict__ sd, float eps, float *__restrict__ Wf,
    float *__restrict__ cf, int A, int E1) {
  __shared__ float part[2];
  const int r = blockIdx.x, j = threadIdx.x, NA = 3 * A;
  int ax;
  const float *w;
  float c;
  if (r < NA) {
    ax = 0; w = Wa + int64_t(r) * DR; c = ca[r];
  } else if (r < NA + E1) {
    ax = 1; w = We + int64_t(r - NA) * DR; c = ce[r - NA];
  } else {
    ax = 2; w = Wb + int64_t(r - NA - E1) * DR; c = cb[r - NA - E1];
  }
  const float wp = w[j] / (sd[ax * DR + j] + eps);
  Wf[int64_t(r) * DR + j] = wp;
  const float s = seg_sum(wp * mu[ax * DR + j], 64);
  if ((j & 63) == 0) part[j >> 6] = s;
  __syncthreads();
  if (j == 0) cf[r] = c - (part[0] + part[1]);
}

struct RelaxArgs {
  const float *Z;   // [N, NZ] head logits (whitened)
  const float *Hh;  // [N, DR] h^ before whitening
  const float *ga, *gb;
  const int32_t *pos;
  const int32_t *eidx;
  const float *egate;
  uint8_t *mode, *bit;
  float *ya, *yb, *pe, *cfl, *cme;
  double *part;  // [RX_F][RX_BLOCKS]: field f of block b at f * RX_BLOCKS + b
  int N, H, A, E1, k, dh, w;
  float inv_ta, inv_tb;
  float kappa_e;  // 3 d d_ff
  float kv2;      // 2 d_kv
};

// What one lane reads of one token, loaded in one go before any of it is
// used (the next token's while the current one is computed).
struct RxTok {
  int P;
  float za0, za1, za2, ga0, ga1, ga2;  // lane a < A: group a's logits and noise
  float ze;                            // lane j < E + 1: expert logit j
  int es;                              // lane s < k: slot s's expert and gate
  float gs;
  float zb, gbv;                       // lane j < 4: bit logit and noise j
  float h0, h1;                        // h^ features lane, lane + 64
};

__device__ __forceinline__ RxTok rx_load(const RelaxArgs &p, int t, int lane, int NZ) {
  RxTok d;
  const float *z = p.Z + int64_t(t) * NZ;
  d.P = p.pos[t];
  d.za0 = d.za1 = d.za2 = d.ga0 = d.ga1 = d.ga2 = 0.f;
  if (lane < p.A) {
    const float *g = p.ga + (int64_t(t) * p.A + lane) * 3;
    d.za0 = z[3 * lane]; d.za1 = z[3 * lane + 1]; d.za2 = z[3 * lane + 2];
    d.ga0 = g[0]; d.ga1 = g[1]; d.ga2 = g[2];
  }
  d.ze = lane < p.E1 ? z[3 * p.A + lane] : -INFINITY;
  d.es = lane < p.k ? p.eidx[int64_t(t) * p.k + lane] : -1;
  d.gs = lane < p.k ? p.egate[int64_t(t) * p.k + lane] : 0.f;
  d.zb = lane < 4 ? z[3 * p.A + p.E1 + lane] : 0.f;
  d.gbv = lane < 4 ? p.gb[int64_t(t) * 4 + lane] : 0.f;
  d.h0 = p.Hh[int64_t(t) * DR + lane];
  d.h1 = p.Hh[int64_t(t) * DR + lane + 64];
  return d;
}

// The relaxed choices of one token per wave (RX_WAVES waves per block, a
// block taking a contiguous range of tokens).  Lane a < A takes attention
// group a, lane j < E + 1 expert j, lane 0 the bit head and the token's
// scalars; every lane keeps h^ features lane and lane + 64 for the batch
// moments.
__global__ __launch_bounds__(64 * RX_WAVES) void relax_kernel(RelaxArgs p) {
  __shared__ double wpart[RX_WAVES][RX_F];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int NZ = 3 * p.A + p.E1 + 4, HA = p.H / p.A;
  const int chunk = (p.N + gridDim.x - 1) / gridDim.x;
  const int t_lo = blockIdx.x * chunk, t_hi = min(p.N, t_lo + chunk);
  int acnt[3] = {0, 0, 0}, bcnt[4] = {0, 0, 0, 0}, ecnt = 0;
  double aP[3] = {0, 0, 0}, alse = 0, bP[4] = {0, 0, 0, 0}, blse = 0, else_ = 0, eP = 0;
  double csum_f = 0, csum_m = 0, dsum_f = 0, dsum_m = 0;
  double hs0 = 0, hs1 = 0, hq0 = 0, hq1 = 0;
  RxTok nx;
  if (t_lo + wave < t_hi) nx = rx_load(p, t_lo + wave, lane, NZ);
  for (int t = t_lo + wave; t < t_hi; t += RX_WAVES) {
    const RxTok d = nx;
    if (t + RX_WAVES < t_hi) nx = rx_load(p, t + RX_WAVES, lane, NZ);
    const float kf = float(d.P) + 1.f, kl = fminf(kf, float(p.w));
    // attention: ST-Gumbel over (skip, local, full) per decision group
    int yi = 0;
    float cost_a = 0.f;
    if (lane < p.A) {
      const float v0 = d.za0 + d.ga0, v1 = d.za1 + d.ga1, v2 = d.za2 + d.ga2;
      yi = v1 > v0 ? 1 : 0;
      if (v2 > (yi ? v1 : v0)) yi = 2;  // first maximum
      const float vm = fmaxf(v0, fmaxf(v1, v2));
      const float e0 = expf((v0 - vm) * p.inv_ta), e1 = expf((v1 - vm) * p.inv_ta),
                  e2 = expf((v2 - vm) * p.inv_ta);
      const float is = 1.f / (e0 + e1 + e2);
      float *ya = p.ya + (int64_t(t) * p.A + lane) * 3;
      ya[0] = e0 * is; ya[1] = e1 * is; ya[2] = e2 * is;
      cost_a = float(HA) * 2.f * float(p.dh) * (e1 * is * kl + e2 * is * kf);
      const float zm = fmaxf(d.za0, fmaxf(d.za1, d.za2));
      const float q0 = expf(d.za0 - zm), q1 = expf(d.za1 - zm), q2 = expf(d.za2 - zm);
      const float qs = q0 + q1 + q2;
      aP[0] += double(q0 / qs); aP[1] += double(q1 / qs); aP[2] += double(q2 / qs);
      const double lse = double(zm) + double(logf(qs));
      alse += lse * lse;
      acnt[yi] += 1;
    }
    for (int h0 = 0; h0 < p.H; h0 += 64) {
      const int hh = h0 + lane;
      const int src = (hh < p.H ? hh : p.H - 1) / HA;
      const int v = __shfl(yi, src, 64);
      if (hh < p.H) p.mode[int64_t(t) * p.H + hh] = uint8_t(v);
    }
    const float cflops_a = seg_sum(cost_a, 64);
    // experts: softmax(z^e) for the balance statistics; the set and gates
    // are the inference top-k
    const float zmax = seg_max(d.ze, 64);
    const float ej = lane < p.E1 ? expf(d.ze - zmax) : 0.f;
    const float es = seg_sum(ej, 64);
    if (lane < p.E1) {
      const float pj = ej / es;
      eP += double(pj);
      if (p.pe) p.pe[int64_t(t) * p.E1 + lane] = pj;
    }
    float cflops_e = 0.f;
    for (int s = 0; s < p.k; ++s) {
      const int e = __shfl(d.es, s, 64);
      const float g = __shfl(d.gs, s, 64);
      if (e == lane) ++ecnt;
      if (e != 0) cflops_e += g;
    }
    float zb[4], gb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      zb[j] = __shfl(d.zb, j, 64);
      gb[j] = __shfl(d.gbv, j, 64);
    }
    if (lane == 0) {
      const double lse_e = double(zmax) + double(logf(es));
      else_ += lse_e * lse_e;
      // bits: ST-Gumbel over (2, 4, 8, 16)
      float v[4], vm = -INFINITY;
      int bi = 0;
      for (int j = 0; j < 4; ++j) {
        v[j] = zb[j] + gb[j];
        if (v[j] > v[bi]) bi = j;
        vm = fmaxf(vm, v[j]);
      }
      float e[4], esum = 0.f, qm = fmaxf(fmaxf(zb[0], zb[1]), fmaxf(zb[2], zb[3])), q[4], qs = 0.f;
      for (int j = 0; j < 4; ++j) {
        e[j] = expf((v[j] - vm) * p.inv_tb);
        esum += e[j];
        q[j] = expf(zb[j] - qm);
        qs += q[j];
      }
      const float is = 1.f / esum;
      float cmem = 0.f;
      for (int j = 0; j < 4; ++j) {
        p.yb[int64_t(t) * 4 + j] = e[j] * is;
        cmem += e[j] * is * p.kv2 * float(2 << j);
        bP[j] += double(q[j] / qs);
      }
      const double lse_b = double(qm) + double(logf(qs));
      blse += lse_b * lse_b;
      bcnt[bi] += 1;
      p.bit[t] = uint8_t(bi);
      const float cflops = cflops_a + cflops_e * p.kappa_e;
      p.cfl[t] = cflops;
      p.cme[t] = cmem;
      csum_f += double(cflops);
      csum_m += double(cmem);
      dsum_f += double(p.H) * 2.0 * double(p.dh) * double(kf) + double(p.kappa_e);
      dsum_m += double(p.kv2) * 16.0;
    }
    hs0 += double(d.h0); hs1 += double(d.h1);
    hq0 += double(d.h0) * double(d.h0); hq1 += double(d.h1) * double(d.h1);
  }
  // fold the wave's lanes (fixed order) into its row of partial sums
  double *wp = wpart[wave];
  for (int o = 0; o < 3; ++o) {
    const double c = wave_sum_d(double(acnt[o])), s = wave_sum_d(aP[o]);
    if (lane == 0) { wp[RX_ACNT + o] = c; wp[RX_AP + o] = s; }
  }
  const double al = wave_sum_d(alse);
  if (lane == 0) {
    wp[RX_ALSE] = al;
    for (int o = 0; o < 4; ++o) { wp[RX_BCNT + o] = double(bcnt[o]); wp[RX_BP + o] = bP[o]; }
    wp[RX_BLSE] = blse; wp[RX_ELSE] = else_;
    wp[RX_CF] = csum_f; wp[RX_CM] = csum_m; wp[RX_DF] = dsum_f; wp[RX_DM] = dsum_m;
  }
  wp[RX_ECNT + lane] = double(ecnt);
  wp[RX_EP + lane] = eP;
  wp[RX_HS + lane] = hs0; wp[RX_HS + lane + 64] = hs1;
  wp[RX_HQ + lane] = hq0; wp[RX_HQ + lane + 64] = hq1;
  __syncthreads();
  for (int f = threadIdx.x; f < RX_F; f += 64 * RX_WAVES) {
    double s = wpart[0][f];
    for (int w = 1; w < RX_WAVES; ++w) s += wpart[w][f];
    p.part[int64_t(f) * RX_BLOCKS + blockIdx.x] = s;
  }
}

struct FinishArgs {
  const double *tot;  // [RX_F] the batch sums
  int N, A, E1, k;
  double zeta, alpha, beta, gamma, target_f, target_m, lr, ema_m;
  double *dual;   // [4] or NULL
  double *stats;  // [TRIROUTE_RELAX_NSTAT]
  double *usage;  // [2][E1] or NULL
  float *h_mean, *h_var;
};

// Block b, wave w: field f = 16 b + w, summed over the blocks' columns
// (lane l takes blocks l, l + 64, ..., then a fixed butterfly).
__global__ __launch_bounds__(1024) void relax_sum_kernel(const double *__restrict__ part,
                                                         int nblk, double *__restrict__ tot) {
  const int lane = threadIdx.x & 63, f = blockIdx.x * 16 + (threadIdx.x >> 6);
  if (f >= RX_F) return;  // wave-uniform
  const double *col = part + int64_t(f) * RX_BLOCKS;
  double s = 0;
#pragma unroll
  for (int b = 0; b < RX_BLOCKS; b += 64) {
    const double v = col[min(b + lane, nblk - 1)];  // unconditional loads, masked adds
    s += b + lane < nblk ? v : 0.0;
  }
  s = wave_sum_d(s);
  if (lane == 0) tot[f] = s;
}

// One block: one thread per option, then thread x < 3 the losses of axis x
// and thread 0 the costs, the regulariser and the dual step.
__global__ __launch_bounds__(256) void relax_finish_kernel(FinishArgs a) {
  __shared__ double tot[RX_F];
  __shared__ double axreg[3];
  for (int f = threadIdx.x; f < RX_F; f += 256) tot[f] = a.tot[f];
  __syncthreads();
  const double N = a.N, rows_e = double(a.N) * a.k;
  const int x = threadIdx.x;
  if (x < DR) {
    const double m = tot[RX_HS + x] / N;
    if (a.h_mean) a.h_mean[x] = float(m);
    if (a.h_var) a.h_var[x] = float(fmax(0.0, tot[RX_HQ + x] / N - m * m));
  }
  if (a.usage && x < a.E1) {
    a.usage[x] = tot[RX_ECNT + x] / rows_e;
    a.usage[a.E1 + x] = tot[RX_EP + x] / N;
  }
  double *st = a.stats;
  // thread x < 3 + E + 1 + 4 takes one option of one axis (attention
  // options, then experts, then bits): its f_o P_o and P_o log P_o
  __shared__ double fp_o[3 + 64 + 4], plp_o[3 + 64 + 4];
  const int nopt = 3 + a.E1 + 4;
  if (x < nopt) {
    const int ax = x < 3 ? 0 : x < 3 + a.E1 ? 1 : 2;
    const int o = ax == 0 ? x : ax == 1 ? x - 3 : x - 3 - a.E1;
    const int fc = ax == 0 ? RX_ACNT : ax == 1 ? RX_ECNT : RX_BCNT;
    const int fp = ax == 0 ? RX_AP : ax == 1 ? RX_EP : RX_BP;
    const double rows_f = ax == 0 ? N * a.A : ax == 1 ? rows_e : N;
    const double rows_p = ax == 0 ? N * a.A : N;
    const double f = tot[fc + o] / rows_f, P = tot[fp + o] / rows_p;
    fp_o[x] = f * P;
    plp_o[x] = P > 0 ? P * log(P) : 0.0;
    if (ax == 0) { st[TRIROUTE_RS_F_ATTN + o] = f; st[TRIROUTE_RS_P_ATTN + o] = P; }
    if (ax == 2) { st[TRIROUTE_RS_F_BITS + o] = f; st[TRIROUTE_RS_P_BITS + o] = P; }
  }
  __syncthreads();
  if (x < 3) {
    const int nO = x == 0 ? 3 : x == 1 ? a.E1 : 4, o0 = x == 0 ? 0 : x == 1 ? 3 : 3 + a.E1;
    const double rows_p = x == 0 ? N * a.A : N;
    const double lz = tot[x == 0 ? RX_ALSE : x == 1 ? RX_ELSE : RX_BLSE] / rows_p;
    double fP = 0, H = 0;
    for (int o = 0; o < nO; ++o) {
      fP += fp_o[o0 + o];
      H -= plp_o[o0 + o];
    }
    const double lbal = nO * fP, lent = fmax(0.0, a.zeta * log(double(nO)) - H);
    st[TRIROUTE_RS_LBAL + x] = lbal;
    st[TRIROUTE_RS_LZ + x] = lz;
    st[TRIROUTE_RS_LENT + x] = lent;
    st[TRIROUTE_RS_ENTROPY + x] = H;
    axreg[x] = a.alpha * lbal + a.beta * lz + a.gamma * lent;
  }
  __syncthreads();
  if (x != 0) return;
  const double cbar_f = tot[RX_CF] / tot[RX_DF], cbar_m = tot[RX_CM] / tot[RX_DM];
  st[TRIROUTE_RS_CBAR] = cbar_f;
  st[TRIROUTE_RS_CBAR + 1] = cbar_m;
  st[TRIROUTE_RS_COST] = tot[RX_CF];
  st[TRIROUTE_RS_COST + 1] = tot[RX_CM];
  st[TRIROUTE_RS_DENSE] = tot[RX_DF];
  st[TRIROUTE_RS_DENSE + 1] = tot[RX_DM];
  const double lam_f = a.dual ? a.dual[0] : 0.0, lam_m = a.dual ? a.dual[1] : 0.0;
  st[TRIROUTE_RS_REG] = ((axreg[0] + axreg[1]) + axreg[2]) + lam_f * (cbar_f - a.target_f) +
                        lam_m * (cbar_m - a.target_m);
  if (a.dual && a.ema_m > 0) {
    const double ef = (1.0 - a.ema_m) * a.dual[2] + a.ema_m * cbar_f;
    const double em = (1.0 - a.ema_m) * a.dual[3] + a.ema_m * cbar_m;
    a.dual[0] = fmax(0.0, lam_f + a.lr * (ef - a.target_f));
    a.dual[1] = fmax(0.0, lam_m + a.lr * (em - a.target_m));
    a.dual[2] = ef;
    a.dual[3] = em;
  }
}

}  // namespace

size_t relax_part_doubles() { return size_t(RX_BLOCKS) * RX_F + RX_F; }

hipError_t launch_white_fold(const triroute_cfg &cfg, const triroute_router_w &w, const float *mu,
                             const float *sd, float eps, float *Wf, float *cf, hipStream_t st) {
  const int A = attn_groups(cfg), E1 = cfg.n_experts + 1;
  white_fold_kernel<<<dim3(3 * A + E1 + 4), DR, 0, st>>>(w.Wa, w.ca, w.We, w.ce, w.Wb, w.cb, mu,
                                                         sd, eps, Wf, cf, A, E1);
  return hipGetLastError();
}

hipError_t launch_relax(const triroute_cfg &cfg, int N, const RelaxJob &j, hipStream_t st) {
  RelaxArgs p;
  p.Z = j.z; p.Hh = j.h; p.ga = j.g_attn; p.gb = j.g_bits; p.pos = j.pos;
  p.eidx = j.eidx; p.egate = j.egate; p.mode = j.mode; p.bit = j.bit;
  p.ya = j.y_attn; p.yb = j.y_bits; p.pe = j.p_exp; p.cfl = j.c_flops; p.cme = j.c_mem;
  p.part = j.part;
  p.N = N; p.H = cfg.n_heads; p.A = attn_groups(cfg); p.E1 = cfg.n_experts + 1; p.k = cfg.top_k;
  p.dh = cfg.head_dim; p.w = cfg.window;
  p.inv_ta = 1.f / j.tau_a; p.inv_tb = 1.f / j.tau_b;
  p.kappa_e = 3.f * float(cfg.d_model) * float(cfg.d_ff);
  p.kv2 = 2.f * float(cfg.n_kv_heads * cfg.head_dim);
  const int want = (N + 4 * RX_WAVES - 1) / (4 * RX_WAVES);  // at least 4 tokens a wave
  const int nblk = want < RX_BLOCKS ? want : RX_BLOCKS;
  relax_kernel<<<dim3(nblk), 64 * RX_WAVES, 0, st>>>(p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  double *tot = j.part + size_t(RX_BLOCKS) * RX_F;
  relax_sum_kernel<<<dim3((RX_F + 15) / 16), 1024, 0, st>>>(j.part, nblk, tot);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  FinishArgs a;
  a.tot = tot; a.N = N; a.A = p.A; a.E1 = p.E1; a.k = p.k;
  a.zeta = j.zeta; a.alpha = j.alpha; a.beta = j.beta; a.gamma = j.gamma;
  a.target_f = j.target_f; a.target_m = j.target_m; a.lr = j.dual_lr; a.ema_m = j.dual_ema;
  a.dual = j.dual; a.stats = j.stats; a.usage = j.usage_exp; a.h_mean = j.h_mean; a.h_var = j.h_var;
  relax_finish_kernel<<<dim3(1), 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tr
