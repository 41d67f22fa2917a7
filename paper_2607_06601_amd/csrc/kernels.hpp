// Launchers of the device kernels (internal to libtriroute).
#pragma once

#include "common.hpp"

namespace tr {

// Attention decisions per token (cfg.attn_groups, 0 = one per head).
inline int attn_groups(const triroute_cfg &c) { return c.attn_groups > 0 ? c.attn_groups : c.n_heads; }


// router.hip
hipError_t router_prepare();
// trunk K split: ks chunks of kchunk inputs; the trunk partials take
// ks * N * 128 floats of scratch
void router_split(int N, int K, int &ks, int &kchunk);
// Rotation table of rotate-half RoPE (paper Sec. 4 Models): for token row i
// of a [B, Tq] batch and pair j < d_h / 2, (cos, sin) of pos * theta^(-2j/d_h)
// at pos = base + t, base = pos_base[s] with s = pos_idx ? pos_idx[b] : b when
// 0 <= s < n_base, else 0 (a row naming no valid sequence is dropped by the
// append, which flags it; its table entries only need to be finite); the
// angle is taken in fp64 and reduced to [-pi, pi] before an accurate fp32
// sincos.
struct RopeJob {
  const int32_t *pos_base, *pos_idx;
  int n_base;  // entries of pos_base
  int Tq, hd;
  float2 *tab;  // [N][hd]
  double inv_freq[64];
};
RopeJob make_rope_job(const triroute_cfg &cfg, int Tq, const int32_t *pos_base,
                      const int32_t *pos_idx, int n_base, float *tab);
__device__ __forceinline__ float2 rope_entry(const RopeJob &r, int row, int j) {
  const int b = row / r.Tq, tt = row - b * r.Tq;
  const int s = r.pos_idx ? r.pos_idx[b] : b;
  const int pos = (r.pos_base && s >= 0 && s < r.n_base ? r.pos_base[s] : 0) + tt;
  const double ang = double(pos) * r.inv_freq[j];
  const double kq = rint(ang * 0.15915494309189535);
  double rr = fma(-kq, 6.283185307179586, ang);
  rr = fma(-kq, 2.4492935982947064e-16, rr);
  float sn, cs;
  sincosf(float(rr), &sn, &cs);
  return make_float2(cs, sn);
}
// Optional copies of the controller tail's intermediates (any may be NULL):
// h^ [N, 128], the head logits z [N, 3 A + E + 5], the trunk's pre-GELU
// a1 = W1 [n1; psi] + b1 [N, 128] and h = W2 u + b2 before its norm [N, 128].
struct TailTap {
  float *h = nullptr, *z = nullptr, *a1 = nullptr, *hpre = nullptr;
};
// rope (optional): the first RMSNorm also writes that rotation table
hipError_t launch_router(const triroute_cfg &cfg, int N, const void *x, const float *psi,
                         const triroute_router_w &w, void *n1, uint8_t *mode, uint8_t *bit,
                         int32_t *eidx, float *egate, float *rinv, float *u, const RopeJob *rope,
                         hipStream_t st, TailTap tap = TailTap{});
// compact.hip
int compact_hist_ints(int N, int k, int E1);
// attn_lists false: the attention lists are not wanted (decode reads the
// modes themselves) and are left untouched.
hipError_t launch_compact(const triroute_cfg &cfg, int B, int T, const uint8_t *mode,
                          const int32_t *eidx, const triroute_compaction &c, int32_t *hist,
                          hipStream_t st, bool attn_lists = true);
// kv.hip
hipError_t launch_fill_u32(void *p, int64_t n_words, uint32_t v, hipStream_t st);
// append scratch: each row's pool lengths before the append
struct KvWs {
  int32_t *old_len;  // [B][4]
};
// paged caches: fill the free stacks with every page; return a sequence's pages
hipError_t launch_kv_paged_init(const CacheView &cv, const int32_t n_pages[4], hipStream_t st);
hipError_t launch_kv_paged_reset(const CacheView &cv, int seq, hipStream_t st);
hipError_t launch_kv_append(const triroute_cfg &cfg, const CacheView &cv, int B, int T,
                            const int32_t *seq_ids, const void *k, const void *v,
                            const uint8_t *bit, const KvWs &ws, hipStream_t st);
hipError_t launch_kv_export(const triroute_cfg &cfg, const CacheView &cv, int seq, int bi,
                            int slot0, int count, void *kout, void *vout, uint16_t *ksz,
                            uint16_t *vsz, int32_t *pos_out, hipStream_t st);
// gemm.hip
// position of token (b, t) as in RopeJob (pos_base has n_base entries);
// rope: scratch of qkv_rope_floats(cfg, B * Tq) floats (the rotation table)
size_t qkv_rope_floats(const triroute_cfg &cfg, int N);
hipError_t launch_qkv(const triroute_cfg &cfg, int B, int Tq, const void *n1,
                      const triroute_dense_w &w, const int32_t *pos_base, const int32_t *pos_idx,
                      int n_base, void *q, void *k, void *v, float *rope, bool rope_ready,
                      hipStream_t st);
hipError_t launch_oproj(const triroute_cfg &cfg, int N, const void *x, const void *o,
                        const triroute_dense_w &w, void *xt, hipStream_t st);
hipError_t launch_moe_gemms(const triroute_cfg &cfg, int N, const void *n2,
                            const triroute_moe_w &w, const triroute_compaction &c, void *Hm,
                            float *Y, hipStream_t st);
// gemm_mfma.hip (bf16)
hipError_t mfma_qkv(const triroute_cfg &cfg, int B, int Tq, const void *n1,
                    const triroute_dense_w &w, const float *rope, void *q, void *k, void *v,
                    hipStream_t st);
hipError_t mfma_oproj(const triroute_cfg &cfg, int N, const void *x, const void *o,
                      const triroute_dense_w &w, void *xt, hipStream_t st);
hipError_t mfma_moe(const triroute_cfg &cfg, int N, const void *n2, const triroute_moe_w &w,
                    const triroute_compaction &c, void *Hm, float *Y, hipStream_t st);
// attn_valu.hip
hipError_t launch_attn_valu_prefill(const triroute_cfg &cfg, const CacheView &cv, int B, int Tq,
                                    const int32_t *seq_ids, const void *q,
                                    const triroute_compaction &c, void *o, hipStream_t st);
hipError_t launch_attn_valu_decode(const triroute_cfg &cfg, const CacheView &cv, int B,
                                   const int32_t *seq_ids, const void *q, const uint8_t *mode,
                                   void *o, hipStream_t st);
// attn_mfma.hip (bf16)
int decode_splits(int B, int Hkv, int capacity, int TS);
hipError_t launch_attn_mfma_decode(const triroute_cfg &cfg, const CacheView &cv, int B,
                                   const int32_t *seq_ids, const void *q, const uint8_t *mode,
                                   void *o, float *part, hipStream_t st);
hipError_t launch_attn_mfma_prefill(const triroute_cfg &cfg, const CacheView &cv, int B, int T,
                                    const int32_t *seq_ids, const void *q,
                                    const triroute_compaction &c, void *o, hipStream_t st);
// misc.hip
hipError_t launch_moe_norm_rows(const triroute_cfg &cfg, int N, const void *x, const void *g,
                                const triroute_compaction &c, const int32_t *eidx, void *out,
                                int32_t *slot_of, hipStream_t st);
// Few assignments (decode, bf16): the down GEMM splits K in two halves, each
// written to its own plane of Y (N k rows apart); the combine adds the planes
// in order.  Returns the number of planes.
inline int moe_ysplit(const triroute_cfg &c, int N) {
  return c.act == TRIROUTE_BF16 && N * c.top_k <= 2048 && c.d_ff % 128 == 0 ? 2 : 1;
}
// zero the prefill attention rows no attention block writes (skipped heads,
// rows of sequence ids outside [0, n_seq))
hipError_t launch_attn_zero_rows(const triroute_cfg &cfg, int B, int T, const uint8_t *mode,
                                 const int32_t *seq_ids, int n_seq, void *o, hipStream_t st);
hipError_t launch_psi_next(const triroute_cfg &cfg, int N, const float *psi, const uint8_t *mode,
                           const uint8_t *bit, const int32_t *eidx, float *out, hipStream_t st);
hipError_t launch_moe_combine(const triroute_cfg &cfg, int N, const void *xt, const float *Y,
                              const int32_t *slot_of, const int32_t *eidx, const float *egate,
                              void *xout, hipStream_t st);

// relax.hip: the relaxed controller forward around the router kernels
struct RelaxJob {
  const float *z, *h;  // the tail's logits and h^
  const float *g_attn, *g_bits;
  const int32_t *pos, *eidx;
  const float *egate;
  uint8_t *mode, *bit;
  float *y_attn, *y_bits, *p_exp, *c_flops, *c_mem;
  double *part;  // relax_part_doubles() of scratch
  double *dual, *stats, *usage_exp;
  float *h_mean, *h_var;
  float tau_a, tau_b;
  double zeta, alpha, beta, gamma, target_f, target_m, dual_lr, dual_ema;
};
size_t relax_part_doubles();
// whitening folded into the head weights: Wf [3A + E + 5][128], cf [3A + E + 5]
hipError_t launch_white_fold(const triroute_cfg &cfg, const triroute_router_w &w, const float *mu,
                             const float *sd, float eps, float *Wf, float *cf, hipStream_t st);
hipError_t launch_relax(const triroute_cfg &cfg, int N, const RelaxJob &j, hipStream_t st);

// relax_grad.hip: the relaxed controller's backward pass
struct RelaxGradOut {
  float *dW1, *db1, *dW2, *db2, *dgr, *dWa, *dca, *dWe, *dce, *dWb, *dcb, *dg1, *dx, *dpsi;
  double *lm_norm;
};
struct RelaxBwdJob {
  const float *z, *hh, *a1, *hpre;  // taps of the recomputed trunk and tail
  const float *y_attn, *y_bits, *egate;
  const int32_t *eidx, *pos;
  const float *g_attn, *g_bits, *g_gate;
  const double *stats, *usage, *lambda;
  double *rho_io;  // [3] or NULL
  float rho_m;
  float tau_a, tau_b, zeta, alpha, beta, gamma;
  // scratch
  float *dz, *dh, *da1, *u, *tgr, *lmsq, *s, *ds, *part, *G, *dc;
  double *lmsq_sum;
  RelaxGradOut out;
};
size_t relax_grad_part_floats(const triroute_cfg &cfg, int N);
// Wf: the head weights [3A + E + 5][128] as the forward applied them (folded
// with the whitening, or the plain ones); mu / sd NULL: no whitening
hipError_t launch_relax_backward(const triroute_cfg &cfg, int N, const void *x, const float *psi,
                                 const triroute_router_w &w, const float *Wf,
                                 const float *white_mu, const float *white_sd, float white_eps,
                                 const RelaxBwdJob &j, hipStream_t st);
}  // namespace tr
