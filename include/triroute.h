/*
 * triroute.h -- C ABI of an MI355X (gfx950) implementation of the inference
 * forward of one TriRoute-routed transformer layer.
 *
 * The layer (paper Sec. 3.1 block, Sec. 3.2 axes, Sec. 3.3 controller,
 * Sec. 3.8 inference rule):
 *   1. a shared controller decides, per token, an attention mode per query
 *      head (skip / local window / full), a top-k set of SwiGLU experts that
 *      may include the null expert, and the bit width {2,4,8,16} at which the
 *      token's own K/V are written to the cache;
 *   2. tokens are compacted by decision (deterministic prefix sums);
 *   3. K/V are quantized per token and per group of G channels and appended
 *      to a bit-packed mixed-width cache; attention reads that cache and
 *      dequantizes in registers (every read, including a token's own key,
 *      goes through the cache: append, then attend);
 *   4. the experts run as a grouped GEMM in which the null expert is the
 *      identity (never computed).
 *
 * Conventions
 *   - Every pointer is a device pointer unless stated; the caller owns all
 *     memory.  The library never allocates or frees device memory and keeps
 *     no pointer past a call.  Calls are asynchronous on the given stream and
 *     never synchronise it, except triroute_kv_status().
 *   - Tensors are row-major and contiguous.  A batch of B sequences of T
 *     tokens is flattened as token i = b*T + t.  Every activation tensor and
 *     weight (everything but index / decision arrays and psi) must be 16-byte
 *     aligned: the kernels move 16-byte pieces.  A misaligned pointer is
 *     rejected with TRIROUTE_E_INVALID.
 *   - "act" tensors have the activation dtype of cfg->act: IEEE fp32, or
 *     bf16 (16-bit storage, round-to-nearest-even on every write).
 *   - Enumerations: attention mode 0 skip, 1 local, 2 full; bit index 0..3
 *     means 2, 4, 8, 16 bits; expert id 0 is the null expert, 1..E are real.
 *   - Errors: every call validates its arguments on the host first; on error
 *     nothing is launched, outputs are untouched, and the return value is a
 *     negative TRIROUTE_E_* code (message via triroute_last_error(), kept
 *     per thread).  Failures that only the device can see (cache capacity)
 *     set bits of the cache's status word, read with triroute_kv_status().
 *   - No C++ exception crosses this boundary.
 */
#ifndef TRIROUTE_H
#define TRIROUTE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *triroute_stream_t; /* a hipStream_t (NULL = default stream) */

enum triroute_status {
  TRIROUTE_OK = 0,
  TRIROUTE_E_INVALID = -1,     /* null pointer, bad enum, inconsistent sizes */
  TRIROUTE_E_UNSUPPORTED = -2, /* a shape or dtype this build does not run */
  TRIROUTE_E_WORKSPACE = -3,   /* workspace smaller than triroute_workspace_bytes() */
  TRIROUTE_E_CAPACITY = -4,    /* cache too small for the request (host-visible) */
  TRIROUTE_E_HIP = -5          /* a HIP runtime call or kernel launch failed */
};

/* Device-side status bits of a cache (triroute_kv_status). */
enum triroute_cache_flags {
  TRIROUTE_CACHE_OVERFLOW = 1, /* an append would have passed the capacity; that row was dropped */
  TRIROUTE_CACHE_BAD_SEQ = 2   /* a sequence id outside [0, n_seq); that row was dropped */
};

enum triroute_dtype { TRIROUTE_F32 = 0, TRIROUTE_BF16 = 1 };
enum triroute_mode { TRIROUTE_SKIP = 0, TRIROUTE_LOCAL = 1, TRIROUTE_FULL = 2 };

/* Layer shape.  Paper notation: d, H, H_kv, d_h, window w, E experts plus
 * the null, top-k, expert width d_f, quantizer group G, side-feature width
 * d_psi, router width d_r (Sec. 3.1-3.3, Table 2, Table 6).
 * Supported: head_dim in {64, 128}; n_heads a multiple of n_kv_heads with
 * at most 16 query heads per kv head; kv_group in {32, 64} dividing
 * head_dim; d_router == 128; d_psi <= 32 and a multiple of 4 (W1 rows stay
 * 16-byte aligned); 1 <= top_k <= n_experts + 1 <= 64;
 * d_model and d_ff multiples of 64; 3 * A + n_experts + 5 <= 112 (A = attn_groups,
 * n_heads if 0, a divisor of n_heads);
 * rms_eps > 0. */
typedef struct triroute_cfg {
  int32_t d_model;
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t window;    /* local mode reads keys [t - window + 1, t] */
  int32_t n_experts; /* E real experts; the expert head has E + 1 logits */
  int32_t top_k;
  int32_t d_ff;
  int32_t kv_group;  /* G */
  int32_t d_psi;
  int32_t d_router;
  int32_t act;       /* enum triroute_dtype */
  float rms_eps;     /* all three RMSNorms */
  float rope_theta;  /* rotate-half RoPE base */
  /* Attention decisions per token (Sec. 3.2 (A): per head or per head group;
   * the Sec. 5 ablation of a single per-token decision): the attention head
   * has 3 * attn_groups logits and query head h takes the decision of group
   * h / (n_heads / attn_groups).  0 means n_heads (one decision per head);
   * otherwise it must divide n_heads. */
  int32_t attn_groups;
} triroute_cfg;

/* Controller weights, fp32 (Sec. 3.3 controller equation; trunk = two-layer
 * GELU MLP, Table 6).  The frozen per-axis whitening and gradient-balance
 * scales are folded into (W, c) by the caller.
 *   g1 [d]            first RMSNorm gain, shared with the attention sublayer
 *   W1 [d_r, d+d_psi] b1 [d_r]      trunk layer 1 (input [n1 ; psi])
 *   W2 [d_r, d_r]     b2 [d_r]      trunk layer 2
 *   gr [d_r]          RMSNorm gain of h
 *   Wa [3A, d_r]      ca [3A]       attention head, logits [A, 3] for the A =
 *                                   attn_groups (n_heads if 0) decision groups
 *   We [E+1, d_r]     ce [E+1]      expert head (index 0 = null)
 *   Wb [4, d_r]       cb [4]        bit head */
typedef struct triroute_router_w {
  const float *g1, *W1, *b1, *W2, *b2, *gr;
  const float *Wa, *ca, *We, *ce, *Wb, *cb;
} triroute_router_w;

/* Attention projections and the second norm gain, act dtype.
 *   Wq [H*dh, d]  Wk [Hkv*dh, d]  Wv [Hkv*dh, d]  Wo [d, H*dh]  g2 [d] */
typedef struct triroute_dense_w {
  const void *Wq, *Wk, *Wv, *Wo, *g2;
} triroute_dense_w;

/* SwiGLU experts, act dtype: f_e(u) = Wdown_e (silu(Wgate_e u) * Wup_e u).
 *   Wgate [E, d_ff, d]  Wup [E, d_ff, d]  Wdown [E, d, d_ff]
 * (expert id e >= 1 uses slice e - 1). */
typedef struct triroute_moe_w {
  const void *Wgate, *Wup, *Wdown;
} triroute_moe_w;

/* Compaction produced by triroute_router (all device int32 arrays).
 *   attn_cnt [B*H*2]      queries per segment s = (b*H + h)*2 + (m - 1),
 *                         m in {local, full}
 *   attn_idx [B*H*2, T]   segment s lists its token positions t ascending
 *                         in attn_idx[s*T .. s*T + attn_cnt[s])
 *   exp_cnt  [E+1]        assignments per expert id (exp_cnt[0] = nulls)
 *   exp_off  [E+1]        exp_off[0] = 0, exp_off[e] = exp_off[e-1] + exp_cnt[e]
 *   exp_rows [B*T*k]      assignment ids a = i*k + slot of real experts,
 *                         grouped by expert (expert e in
 *                         [exp_off[e-1], exp_off[e])), ascending within */
typedef struct triroute_compaction {
  int32_t *attn_cnt, *attn_idx, *exp_cnt, *exp_off, *exp_rows;
} triroute_compaction;

/* Mixed-width KV cache (paper Sec. 3.2 (C); per-width grouping of tokens).
 * One device allocation of triroute_kv_cache_bytes() holds, for each of
 * n_seq sequences: a length, per width b a pool of `capacity` slots filled
 * in position order, the position of every slot, and the packed codes.
 * Fields are filled by triroute_kv_cache_init; treat them as read-only.
 *
 * Physical layout of one pool (sequence s, width index bi, kv head g): a run
 * of tiles of TS = 4096 / head_dim slots.  A tile holds [K codes | V codes |
 * K scale/zero | V scale/zero] (no scale/zero for 16-bit).  The code block
 * of a tile is 64 lane records of 8*bp bytes (bp = bits, or 16 / 32 for the
 * native bf16 / fp32 store); record l holds 64 elements q = f*8 + j, eight
 * "fields" f of eight elements j:
 *   K: slot 16*(f / (dh/32)) + (l % 16), channel 32*(f % (dh/32)) + 8*(l / 16) + j
 *   V: slot 32*(f / (dh/16)) + 16*(j / 4) + 4*(l / 16) + j % 4,
 *      channel 16*(f % (dh/16)) + (l % 16)
 * Bit position of element q (f = q / 8, j = q % 8) in the record's 32-bit words:
 *   bp = 2:      word q / 16, bit 4*j + 2*(f % 2)
 *   bp = 4:      word q / 8,  bit 8*(j % 4) + 4*(j / 4)
 *   bp = 8:      word q / 4,  bit 8*(q % 4)
 *   bp = 16:     word q / 2,  bit 16*(q % 2)
 *   bp = 32:     word q (one element per word)
 * Scale/zero blocks are [TS slots][dh/G groups][2] fp16 (scale, zero). */
typedef struct triroute_kv_cache {
  void *base;
  int32_t n_seq;
  int32_t capacity;
  int32_t tile_slots;
  int32_t n_tiles;        /* tiles per pool */
  int64_t off_status;     /* int32 status word */
  int64_t off_seq_len;    /* int32 [n_seq] */
  int64_t off_pool_len;   /* int32 [n_seq][4] */
  int64_t off_pos;        /* int32 [n_seq][4][n_tiles * tile_slots] */
  int64_t off_pool[4];    /* first tile of width bi */
  int64_t tile_bytes[4];  /* bytes per tile of width bi */
  int64_t total_bytes;
  /* Paged caches only (page_tiles > 0, see triroute_kv_paged_cache_init):
   * width bi's tiles and slot positions live in a pool of n_pages[bi] pages
   * of page_tiles tiles (every kv head) and page_tiles * tile_slots
   * positions; sequence s's pool of width bi is the list of pages
   * page_table[(s * 4 + bi) * max_pages + j], j < alloc[s * 4 + bi]; the
   * free pages of width bi are free_list[bi][0 .. free_top[bi]). */
  int32_t page_tiles;     /* 0: contiguous pools of `capacity` slots per sequence and width */
  int32_t max_pages;      /* page-table entries per (sequence, width) */
  int32_t n_pages[4];
  int64_t off_alloc;      /* int32 [n_seq][4] */
  int64_t off_page_table; /* int32 [n_seq][4][max_pages] */
  int64_t off_free_top;   /* int32 [4] */
  int64_t off_free_list[4]; /* int32 [n_pages[bi]] */
  int64_t off_pos_pool[4];  /* int32 [n_pages[bi]][page_tiles * tile_slots] */
} triroute_kv_cache;

/* Optional taps of the composite calls: where to also leave intermediates
 * (any field may be NULL).  Shapes as in the per-stage calls. */
typedef struct triroute_layer_taps {
  void *n1;          /* act [N, d] */
  uint8_t *mode;     /* [N, H] */
  uint8_t *bit;      /* [N] */
  int32_t *eidx;     /* [N, k] */
  float *egate;      /* [N, k] */
  void *q, *k, *v;   /* act [N, H*dh], [N, Hkv*dh], [N, Hkv*dh] */
  void *o;           /* act [N, H*dh] */
  void *xt;          /* act [N, d] */
} triroute_layer_taps;

enum triroute_op {
  TRIROUTE_OP_ROUTER = 0,
  TRIROUTE_OP_QKV = 1,
  TRIROUTE_OP_KV_APPEND = 2,
  TRIROUTE_OP_ATTN_PREFILL = 3,
  TRIROUTE_OP_ATTN_DECODE = 4,
  TRIROUTE_OP_MOE = 5,
  TRIROUTE_OP_LAYER_PREFILL = 6,
  TRIROUTE_OP_LAYER_DECODE = 7,
  TRIROUTE_OP_STACK_DECODE = 8,
  TRIROUTE_OP_ROUTER_RELAXED = 9,
  TRIROUTE_OP_ROUTER_RELAXED_BACKWARD = 10
};

/* ---- configuration, errors, sizes ---------------------------------------- */

/* Checks cfg against the supported set; TRIROUTE_OK or E_INVALID/E_UNSUPPORTED. */
int triroute_validate(const triroute_cfg *cfg);
/* Static name of a status code. */
const char *triroute_status_string(int status);
/* Message of the calling thread's last failing call ("" if none). */
const char *triroute_last_error(void);
/* Workspace bytes op needs for B sequences of T tokens (T = 1 for decode). */
int triroute_workspace_bytes(const triroute_cfg *cfg, int op, int B, int T, size_t *bytes);

/* ---- KV cache ------------------------------------------------------------- */

/* Bytes of a cache for n_seq sequences of at most `capacity` tokens. */
int triroute_kv_cache_bytes(const triroute_cfg *cfg, int n_seq, int capacity, size_t *bytes);
/* Lays out `cache` in the caller's allocation `base` (>= cache_bytes, 256-byte
 * aligned) and clears it on `stream` (all sequences empty). */
int triroute_kv_cache_init(const triroute_cfg *cfg, triroute_kv_cache *cache, void *base,
                           size_t bytes, int n_seq, int capacity, triroute_stream_t stream);
/* Empties sequence `seq` (its length and pool lengths) on `stream`; later
 * appends overwrite every bit of the slots they take. */
/* Paged mixed-width cache (the layout above with page_tiles > 0): instead of
 * every sequence reserving `capacity` slots in each of the four width pools,
 * width bi has a pool of n_pages[bi] pages of page_tiles tiles shared by all
 * sequences, and an append takes pages from it as a sequence's pool of that
 * width grows (device-side, no host synchronisation).  capacity still
 * bounds one sequence's length.  An append row whose pages cannot be had
 * (the width's pool is exhausted, or several rows asked at once for the last
 * pages) is dropped and flags TRIROUTE_CACHE_OVERFLOW; pages it already took
 * for other widths stay with its sequence.  triroute_kv_reset_seq returns a
 * sequence's pages.  Every other call takes paged and contiguous caches alike
 * and computes the same results.  page_tiles >= 1; n_pages[bi] >= 0. */
int triroute_kv_paged_cache_bytes(const triroute_cfg *cfg, int n_seq, int capacity,
                                  int page_tiles, const int32_t n_pages[4], size_t *bytes);
int triroute_kv_paged_cache_init(const triroute_cfg *cfg, triroute_kv_cache *cache, void *base,
                                 size_t bytes, int n_seq, int capacity, int page_tiles,
                                 const int32_t n_pages[4], triroute_stream_t stream);
/* Free pages per width of a paged cache (synchronises the stream). */
int triroute_kv_free_pages(const triroute_kv_cache *cache, int32_t free_pages[4],
                           triroute_stream_t stream);
int triroute_kv_reset_seq(const triroute_cfg *cfg, const triroute_kv_cache *cache, int seq,
                          triroute_stream_t stream);
/* Synchronises `stream` and copies the cache status word to *status (host). */
int triroute_kv_status(const triroute_kv_cache *cache, int32_t *status, triroute_stream_t stream);

/* Sec. 3.2 (C) KV bit-width axis: quantize and append T new tokens to each of B cache
 * sequences.  Row b goes to sequence seq_ids[b] (seq_ids NULL: b); its tokens
 * take positions seq_len, seq_len + 1, ... in order, and token (b, t) lands in
 * the pool of width bit[b*T + t] at the next free slot.
 *   k, v  act [B*T, Hkv*dh] (already rotated keys)   bit uint8 [B*T]
 * A row that would pass `capacity` is dropped and sets TRIROUTE_CACHE_OVERFLOW.
 * Quantizer (bit exact): per group of G channels, fp32 mn/mx, s32 = (mx-mn)/(2^b-1),
 * stored s = fp16(s32), z = fp16(mn) (RNE), code = 0 if s == 0 else
 * clamp(rint_even((x - z) / s), 0, 2^b - 1) in fp32; 16-bit keeps x verbatim.
 * Rows must name distinct sequences. */
int triroute_kv_append(const triroute_cfg *cfg, const triroute_kv_cache *cache, int B, int T,
                       const int32_t *seq_ids, const void *k, const void *v, const uint8_t *bit,
                       void *ws, size_t ws_bytes, triroute_stream_t stream);

/* Reads back slots [slot0, slot0 + count) of pool (seq, bi) in logical form:
 *   k_out, v_out  [count, Hkv, dh]: uint8 codes (bi < 3) or act values (bi == 3)
 *   k_sz, v_sz    [count, Hkv, dh/G, 2] fp16 bit patterns (scale, zero); unused for bi == 3
 *   pos_out       int32 [count] token positions
 * Slots beyond the pool's length read as zero.  (Inspection / tests.) */
int triroute_kv_export(const triroute_cfg *cfg, const triroute_kv_cache *cache, int seq, int bi,
                       int slot0, int count, void *k_out, void *v_out, uint16_t *k_sz,
                       uint16_t *v_sz, int32_t *pos_out, triroute_stream_t stream);

/* ---- per-stage calls ------------------------------------------------------ */

/* Sec. 3.3 controller equation, Sec. 3.8 hard decisions:
 *   n1 = RMSNorm(x; g1) (fp32 inside, act out), u = GELU(W1 [n1; psi] + b1),
 *   h = W2 u + b2, h^ = RMSNorm(h; gr), z^a = Wa h^ + ca, z^e = We h^ + ce,
 *   z^b = Wb h^ + cb;  mode[i,h] = argmax_m z^a[h,m] (first maximum),
 *   bit[i] = argmax z^b, S_i = k largest softmax(z^e) (lower id on ties)
 *   stored in ascending id, egate = p_j / sum_{S_i} p (the null's share is
 *   dropped).  Then the compaction `cmp` (see triroute_compaction).
 *   x act [B*T, d], psi f32 [B*T, d_psi]; outputs n1 act [B*T, d],
 *   mode u8 [B*T, H], bit u8 [B*T], eidx i32 [B*T, k], egate f32 [B*T, k]. */
int triroute_router(const triroute_cfg *cfg, int B, int T, const void *x, const float *psi,
                    const triroute_router_w *w, void *n1, uint8_t *mode, uint8_t *bit,
                    int32_t *eidx, float *egate, const triroute_compaction *cmp, void *ws,
                    size_t ws_bytes, triroute_stream_t stream);

/* Sec. 3.1 pre-norm block (the attention projections of Norm(x)) with Sec. 4
 * Models' RoPE: q = Wq n1, k = Wk n1, v = Wv n1 with rotate-half RoPE on q and k
 * at position pos0[b] + t (pos0 NULL: t); pos0 may point into a cache's
 * sequence lengths (see triroute_kv_seq_len_ptr).
 *   n1 act [B*T, d]; q act [B*T, H*dh]; k, v act [B*T, Hkv*dh].
 * ws: device scratch of triroute_workspace_bytes(cfg, TRIROUTE_OP_QKV, B, T)
 * bytes (the per-token rotation table); a shorter one is TRIROUTE_E_WORKSPACE. */
int triroute_qkv(const triroute_cfg *cfg, int B, int T, const void *n1,
                 const triroute_dense_w *w, const int32_t *pos0, void *q, void *k, void *v,
                 void *ws, size_t ws_bytes, triroute_stream_t stream);

/* Device pointer to the int32 [n_seq] sequence lengths of a cache. */
const int32_t *triroute_kv_seq_len_ptr(const triroute_kv_cache *cache);

/* Sec. 3.2 (A) attention-resolution axis: attention of B*T new queries whose K/V were just
 * appended (the T tokens of row b occupy the last T positions of sequence
 * seq_ids[b]).  Query head h of token (b, t) at position P reads kv head
 * h / (H / Hkv): skip -> zeros, local -> keys [P - w + 1, P], full -> [0, P],
 * softmax(q k^T / sqrt(dh)) v over the dequantized cache.  Rows of a
 * sequence id outside [0, n_seq), and heads whose mode byte is neither
 * local nor full, are written as zeros.
 *   q act [B*T, H*dh]; mode u8 [B*T, H]; cmp from triroute_router; o act [B*T, H*dh]. */
int triroute_attn_prefill(const triroute_cfg *cfg, int B, int T, const int32_t *seq_ids,
                          const void *q, const triroute_kv_cache *cache, const uint8_t *mode,
                          const triroute_compaction *cmp, void *o, void *ws, size_t ws_bytes,
                          triroute_stream_t stream);

/* Sec. 3.2 (A) for the Sec. 3.8 left-to-right decode: as triroute_attn_prefill
 * for one new query per sequence (T = 1),
 * split over KV chunks with a log-sum-exp combine.
 *   q act [B, H*dh]; mode u8 [B, H]; o act [B, H*dh]. */
int triroute_attn_decode(const triroute_cfg *cfg, int B, const int32_t *seq_ids, const void *q,
                         const triroute_kv_cache *cache, const uint8_t *mode, void *o, void *ws,
                         size_t ws_bytes, triroute_stream_t stream);

/* Sec. 3.1 pre-norm block, first residual: xt = x + Wo concat_h(o).
 * x, xt act [N, d]. */
int triroute_oproj(const triroute_cfg *cfg, int n_tok, const void *x, const void *o,
                   const triroute_dense_w *w, void *xt, triroute_stream_t stream);

/* Sec. 3.1 second half of the block with the Sec. 3.2 (B) expert axis:
 * n2 = RMSNorm(xt; g2),
 * x_out = xt + sum over slots with eidx != 0 of egate * f_eidx(n2).
 * Null slots are never computed.  eidx/egate/cmp as produced by
 * triroute_router for the same n_tok = B*T tokens. */
int triroute_moe(const triroute_cfg *cfg, int n_tok, const void *xt, const triroute_dense_w *dw,
                 const triroute_moe_w *w, const int32_t *eidx, const float *egate,
                 const triroute_compaction *cmp, void *x_out, void *ws, size_t ws_bytes,
                 triroute_stream_t stream);

/* ---- composites (no host synchronisation inside) ------------------------- */

/* Whole layer for B sequences of T new tokens: router, compaction, QKV at
 * positions continuing each sequence, append, attention, O-proj, experts. */
int triroute_layer_prefill(const triroute_cfg *cfg, int B, int T, const int32_t *seq_ids,
                           const void *x, const float *psi, const triroute_router_w *rw,
                           const triroute_dense_w *dw, const triroute_moe_w *mw,
                           const triroute_kv_cache *cache, void *x_out,
                           const triroute_layer_taps *taps, void *ws, size_t ws_bytes,
                           triroute_stream_t stream);

/* One decode step: one new token per sequence (x [B, d], psi [B, d_psi]). */
int triroute_layer_decode(const triroute_cfg *cfg, int B, const int32_t *seq_ids,
                          const void *x, const float *psi, const triroute_router_w *rw,
                          const triroute_dense_w *dw, const triroute_moe_w *mw,
                          const triroute_kv_cache *cache, void *x_out,
                          const triroute_layer_taps *taps, void *ws, size_t ws_bytes,
                          triroute_stream_t stream);

/* ---- a stack of routed layers ------------------------------------------- */

/* The weights of one routed layer. */
typedef struct triroute_layer_w {
  triroute_router_w router;
  triroute_dense_w dense;
  triroute_moe_w moe;
} triroute_layer_w;

/* One decode step of B sequences through n_layers routed layers (Sec. 3.8:
 * one left-to-right pass, per-token decisions taken layer by layer on the
 * device, no host synchronisation), layer l reading and appending to its own
 * cache caches[l].  Layer 0 takes the caller's side features psi; layer
 * l > 0 takes them with the last four replaced by layer l - 1's decisions
 * of the same token (Sec. 3.3 counts the previous layer's decisions among
 * the side features),
 *   psi'[d_psi - 4] = heads in full mode / H,  psi'[d_psi - 3] = heads in
 *   local mode / H,  psi'[d_psi - 2] = width index / 3,  psi'[d_psi - 1] =
 *   real (non-null) expert slots / k
 * (fp32, exact quotients of small integers).  Layer l's output is layer
 * l + 1's input; the last layer's goes to x_out.  Requires d_psi >= 4.
 *   layers, caches: host arrays of n_layers entries (1 <= n_layers <= 256);
 *   x, x_out act [B, d]; psi f32 [B, d_psi];
 *   ws: triroute_workspace_bytes(cfg, TRIROUTE_OP_STACK_DECODE, B, 1) bytes. */
int triroute_stack_decode(const triroute_cfg *cfg, int n_layers, int B, const int32_t *seq_ids,
                          const void *x, const float *psi, const triroute_layer_w *layers,
                          const triroute_kv_cache *caches, void *x_out, void *ws, size_t ws_bytes,
                          triroute_stream_t stream);

/* ---- training-time relaxed controller forward ----------------------------- */

/* Inputs of the relaxed forward (Sec. 3.4-3.7, Algorithm 1).  Pointers are
 * device memory; N = B * T tokens, A = attention decision groups. */
typedef struct triroute_relax_params {
  const float *g_attn;   /* [N, A, 3] Gumbel(0, 1) noise of the attention choices */
  const float *g_bits;   /* [N, 4] Gumbel(0, 1) noise of the bit choice */
  const int32_t *pos;    /* [N] 0-based position of each token in its sequence */
  const float *white_mu; /* [3, d_r] per-axis running means (attention, experts, bits), or NULL */
  const float *white_sd; /* [3, d_r] per-axis running standard deviations; NULL with white_mu */
  float white_eps;       /* Sec. 3.6 whitening epsilon; sd + eps must be nonzero */
  float tau_a, tau_b;    /* ST-Gumbel temperatures of the attention and bit heads, > 0 */
  float zeta;            /* entropy floor: a fraction of log |O| */
  float alpha, beta, gamma; /* weights of L_bal, L_z and L_ent (Sec. 3.7 total loss) */
  float c_target[2];     /* C*_flops, C*_mem */
  double *dual;          /* [4] lambda_flops, lambda_mem, EMA of C-bar_flops, C-bar_mem, or
                          * NULL (lambda = 0); updated in place when dual_ema > 0 */
  float dual_lr, dual_ema; /* rho_lambda and the EMA momentum m */
} triroute_relax_params;

/* Layout of triroute_relax_out.stats (fp64); the three axes in the order
 * attention, experts, bits. */
enum triroute_relax_stat {
  TRIROUTE_RS_LBAL = 0,     /* [3] Switch balance loss |O| sum_o f_o P_o */
  TRIROUTE_RS_LZ = 3,       /* [3] router z-loss, mean of (log sum_o exp z_o)^2 */
  TRIROUTE_RS_LENT = 6,     /* [3] entropy floor [zeta log |O| - H(P)]_+ */
  TRIROUTE_RS_ENTROPY = 9,  /* [3] H(P) of the mean soft probabilities */
  TRIROUTE_RS_CBAR = 12,    /* [2] C-bar_flops, C-bar_mem: cost / dense cost */
  TRIROUTE_RS_COST = 14,    /* [2] summed expected costs (MACs, bits) */
  TRIROUTE_RS_DENSE = 16,   /* [2] summed dense costs of the same tokens */
  TRIROUTE_RS_REG = 18,     /* the regulariser: sum of alpha L_bal + beta L_z + gamma L_ent
                             * over the axes + sum_r lambda_r (C-bar_r - C*_r) */
  TRIROUTE_RS_F_ATTN = 19,  /* [3] hard-choice fractions of the attention axis */
  TRIROUTE_RS_P_ATTN = 22,  /* [3] mean soft probabilities of the attention axis */
  TRIROUTE_RS_F_BITS = 25,  /* [4] */
  TRIROUTE_RS_P_BITS = 29,  /* [4] */
  TRIROUTE_RELAX_NSTAT = 33
};

/* Outputs of the relaxed forward beyond the hard decisions (device). */
typedef struct triroute_relax_out {
  float *y_attn;     /* [N, A, 3] soft samples of the attention choice */
  float *y_bits;     /* [N, 4] soft samples of the bit choice */
  float *c_flops;    /* [N] expected attention-read plus expert MACs of each token */
  float *c_mem;      /* [N] expected KV bits of each token */
  double *stats;     /* [TRIROUTE_RELAX_NSTAT] */
  float *p_exp;      /* [N, E+1] softmax(z^e), or NULL */
  double *usage_exp; /* [2, E+1] f_o then P_o of the expert axis, or NULL */
  float *h_mean;     /* [d_r] batch mean of h^ (before whitening), or NULL */
  float *h_var;      /* [d_r] batch (population) variance of h^, or NULL */
  float *z;          /* [N, 3A + E + 5] head logits after whitening, or NULL */
} triroute_relax_out;

/* One layer's relaxed controller forward at training time (Algorithm 1
 * steps 1-3, 5, 6; the backward pass is not part of the library):
 *   h^ as in triroute_router; each head reads its own whitening
 *   (h^ - mu) / (sd + eps) (Sec. 3.6; folded into that head's weights on
 *   the device, W' = W / (sd + eps), c' = c - W' mu);
 *   attention and bits (Sec. 3.4): soft sample y~ = softmax((z + g) / tau),
 *   hard choice argmax (z + g) (first maximum), broadcast to the heads of a
 *   decision group in `mode`; experts: the inference top-k and gates;
 *   costs (Sec. 3.5): c_flops = sum_h sum_m y~^a_m 2 d_h keys_m(t) +
 *   3 d d_f sum over the real experts of S_t of their gates (the null costs
 *   nothing), keys_local = min(P + 1, w), keys_full = P + 1; c_mem =
 *   sum_b y~^b_b 2 d_kv b; dense reference H 2 d_h (P + 1) + 3 d d_f and
 *   2 d_kv 16 per token, C-bar = summed cost / summed dense cost;
 *   losses (Sec. 3.6) per axis: f_o hard-choice fractions (attention over
 *   (token, group) rows, experts over the N k assignments), P_o mean of
 *   softmax(z), L_bal = |O| sum f P, L_z = mean (logsumexp z)^2,
 *   L_ent = [zeta log |O| - H(P)]_+; the regulariser of Sec. 3.7 with the
 *   multipliers in `dual` as given; then, when dual_ema > 0, the dual step
 *   ema <- (1 - m) ema + m C-bar, lambda <- max(0, lambda + rho (ema - C*)).
 * Then the compaction of the hard decisions, as triroute_router.  Batch
 * statistics are reduced in a fixed order (deterministic).
 *   x act [B*T, d], psi f32 [B*T, d_psi]; n1, mode, bit, eidx, egate, cmp as
 *   in triroute_router; ws: triroute_workspace_bytes(cfg,
 *   TRIROUTE_OP_ROUTER_RELAXED, B, T) bytes. */
int triroute_router_relaxed(const triroute_cfg *cfg, int B, int T, const void *x,
                            const float *psi, const triroute_router_w *w,
                            const triroute_relax_params *p, void *n1, uint8_t *mode,
                            uint8_t *bit, int32_t *eidx, float *egate,
                            const triroute_compaction *cmp, const triroute_relax_out *out,
                            void *ws, size_t ws_bytes, triroute_stream_t stream);

/* Upstream gradients and balance state of the relaxed backward (device). */
typedef struct triroute_relax_grad_in {
  const float *g_attn;   /* [N, A, 3] dL/dy~^a: the language-model gradient the straight-through
                          * estimator hands from the hard attention choice to its soft sample */
  const float *g_bits;   /* [N, 4] dL/dy~^b */
  const float *g_gate;   /* [N, k] dL/dp-bar of the selected slots (from the expert combine) */
  const double *lambda;  /* [2] the multipliers of the forward's regulariser, or NULL (0) */
  double *rho;           /* [3] gradient-balance factors (attention, experts, bits), in and out,
                          * or NULL (1, no update) */
  float rho_m;           /* EMA momentum of rho; 0 leaves rho as is */
} triroute_relax_grad_in;

/* Gradients of the relaxed backward (device fp32, overwritten): one per
 * router weight, shaped like it (see triroute_router_w), and of the inputs:
 * dx [N, d], dpsi [N, d_psi] (the controller path only: the attention
 * sublayer's share of n1's gradient is the caller's).  lm_norm [3] (fp64,
 * may be NULL): per axis the norm of the language-model part of the logit
 * gradient before balancing. */
typedef struct triroute_relax_grad_out {
  float *dW1, *db1, *dW2, *db2, *dgr;
  float *dWa, *dca, *dWe, *dce, *dWb, *dcb;
  float *dg1, *dx, *dpsi;
  double *lm_norm;
} triroute_relax_grad_out;

/* Backward pass of triroute_router_relaxed (Algorithm 1 step 7 for the
 * controller; Sec. 3.4-3.7).  Differentiates the soft outputs the rest of the
 * layer consumes and the regulariser, with the hard choices, the usage
 * fractions f_o, the whitening statistics and the multipliers held constant:
 *   attention / bits: dz = (1 / tau) y~ (G - <y~, G>) with G = g_attn / rho
 *   (language-model part) plus lambda_r / C_dense^r times the option costs
 *   of Sec. 3.5; experts: dz_j = p-bar_j (G_j - <p-bar, G>) on the selected
 *   slots with G = g_gate / rho plus lambda_flops / C_dense^flops 3 d d_f on
 *   the real experts; each axis adds the gradients of alpha L_bal + beta L_z
 *   + gamma L_ent (the floor only when it is active); then the chain through
 *   the whitened heads, RMSNorm(h; gr), W2, the GELU, W1 and Norm(x; g1).
 *   rho, when given, is used as passed and then set to (1 - rho_m) rho +
 *   rho_m ||language-model part||.
 * x, psi, w, p as given to the forward (the trunk is recomputed; its logits
 * equal the forward's); fwd: the forward's outputs, of which y_attn,
 * y_bits, stats and usage_exp are read (usage_exp must have been
 * requested); eidx, egate: the forward's expert choices.
 * ws: triroute_workspace_bytes(cfg, TRIROUTE_OP_ROUTER_RELAXED_BACKWARD, B, T). */
int triroute_router_relaxed_backward(const triroute_cfg *cfg, int B, int T, const void *x,
                                     const float *psi, const triroute_router_w *w,
                                     const triroute_relax_params *p,
                                     const triroute_relax_out *fwd, const int32_t *eidx,
                                     const float *egate, const triroute_relax_grad_in *gin,
                                     const triroute_relax_grad_out *gout, void *ws,
                                     size_t ws_bytes, triroute_stream_t stream);

/* ---- no-allocation variant ---------------------------------------------- */

/* Bytes of the library's static device scratch (per GPU, held until the
 * process ends). */
#define TRIROUTE_STATIC_SCRATCH_BYTES ((size_t)16 << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): one decode
 * step exactly as triroute_layer_decode (same kernels, same results), with
 * its workspace taken from a static device array of
 * TRIROUTE_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs
 * on, instead of a caller buffer.  The caller still passes every input and
 * output.  A batch whose workspace (triroute_workspace_bytes(cfg,
 * TRIROUTE_OP_LAYER_DECODE, B, 1, .)) exceeds that size is rejected with
 * TRIROUTE_E_WORKSPACE before any launch (16 MiB holds 64 sequences of the
 * 1.3B-class shape, 128 of the 410M-class one).  The call allocates nothing:
 * the array's address on the current device is looked up once per device.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents; nothing in it needs clearing (no step depends on what an
 * earlier call left there), but calls that overlap on one GPU (several
 * streams or threads) race on it and must be serialised by the caller. */
int triroute_layer_decode_noalloc(const triroute_cfg *cfg, int B, const int32_t *seq_ids,
                                  const void *x, const float *psi, const triroute_router_w *rw,
                                  const triroute_dense_w *dw, const triroute_moe_w *mw,
                                  const triroute_kv_cache *cache, void *x_out,
                                  const triroute_layer_taps *taps, triroute_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TRIROUTE_H */
