// Host side of libtriroute: argument validation, cache layout, workspace
// carving and kernel launches on the caller's stream.  No call allocates or
// frees device memory, and only triroute_kv_status synchronises.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <string.h>

#include <mutex>

#include <initializer_list>

#include "kernels.hpp"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

int hip_fail(hipError_t e, const char *what) {
  return fail(TRIROUTE_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define CHECK_HIP(expr, what)                        \
  do {                                               \
    hipError_t e_ = (expr);                          \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

#define REQUIRE(cond, code, ...)                 \
  do {                                           \
    if (!(cond)) return fail(code, __VA_ARGS__); \
  } while (0)

// Static scratch of the no-allocation entry point: one copy per GPU, whose
// device address is looked up once per device (the host-side name of the
// array is not a device address).
__device__ __align__(256) uint8_t scratch[TRIROUTE_STATIC_SCRATCH_BYTES];
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[MAX_DEVICES] = {};

int static_scratch(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= MAX_DEVICES)
    return fail(TRIROUTE_E_UNSUPPORTED, "device %d beyond the %d the library tracks", dev,
                MAX_DEVICES);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return TRIROUTE_OK;
}

int prepare_once() {
  static std::once_flag once;
  static hipError_t err = hipSuccess;
  std::call_once(once, [] { err = tr::router_prepare(); });
  if (err != hipSuccess) return hip_fail(err, "kernel attribute setup");
  return TRIROUTE_OK;
}

int act_bytes(const triroute_cfg &c) { return c.act == TRIROUTE_BF16 ? 2 : 4; }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Bump allocator over a workspace (or a dry run that only counts bytes).
struct Carve {
  uint8_t *base;
  size_t used = 0;
  explicit Carve(void *b) : base((uint8_t *)b) {}
  template <typename T>
  T *take(size_t count) {
    T *p = base ? (T *)(base + used) : nullptr;
    used += align256(count * sizeof(T));
    return p;
  }
};

constexpr int DECODE_MAX_SPLITS = 16;

struct LayerBufs {
  void *n1, *q, *k, *v, *o, *xt;
  uint8_t *mode, *bit;
  int32_t *eidx;
  float *egate;
  triroute_compaction cmp;
};

// --- per-op scratch (the parts a stage needs beyond its outputs)
struct RouterWs {
  float *rinv, *u;
  int32_t *hist;
};
RouterWs carve_router(Carve &cv, const triroute_cfg &c, int N) {
  RouterWs w;
  w.rinv = cv.take<float>(N);
  int ks, kchunk;
  tr::router_split(N, c.d_model + c.d_psi, ks, kchunk);
  w.u = cv.take<float>(size_t(ks) * N * 128);
  w.hist = cv.take<int32_t>(tr::compact_hist_ints(N, c.top_k, c.n_experts + 1));
  return w;
}
struct MoeWs {
  void *n2, *Hm;  // one row per expert-list entry (at most N k)
  float *Y;
  int32_t *slot_of;  // list entry of each assignment
};
MoeWs carve_moe(Carve &cv, const triroute_cfg &c, int N) {
  MoeWs w;
  const size_t ab = act_bytes(c);
  w.n2 = cv.take<uint8_t>(size_t(N) * c.top_k * c.d_model * ab);
  w.Hm = cv.take<uint8_t>(size_t(N) * c.top_k * c.d_ff * ab);
  w.Y = cv.take<float>(size_t(N) * c.top_k * c.d_model * tr::moe_ysplit(c, N));
  w.slot_of = cv.take<int32_t>(size_t(N) * c.top_k);
  return w;
}
tr::KvWs carve_kv(Carve &cv, const triroute_cfg &c, int B, int T) {
  tr::KvWs w;
  w.old_len = cv.take<int32_t>(size_t(B) * 4);
  (void)T;
  return w;
}
float *carve_attn_decode(Carve &cv, const triroute_cfg &c, int B) {
  return cv.take<float>(size_t(B) * c.n_heads * DECODE_MAX_SPLITS * (c.head_dim + 2));
}

LayerBufs carve_layer(Carve &cv, const triroute_cfg &c, int B, int T) {
  const int N = B * T, H = c.n_heads;
  const size_t ab = act_bytes(c);
  LayerBufs L;
  L.n1 = cv.take<uint8_t>(size_t(N) * c.d_model * ab);
  L.mode = cv.take<uint8_t>(size_t(N) * H);
  L.bit = cv.take<uint8_t>(N);
  L.eidx = cv.take<int32_t>(size_t(N) * c.top_k);
  L.egate = cv.take<float>(size_t(N) * c.top_k);
  L.cmp.attn_cnt = cv.take<int32_t>(size_t(B) * H * 2);
  L.cmp.attn_idx = cv.take<int32_t>(size_t(B) * H * 2 * T);
  L.cmp.exp_cnt = cv.take<int32_t>(c.n_experts + 1);
  L.cmp.exp_off = cv.take<int32_t>(c.n_experts + 1);
  L.cmp.exp_rows = cv.take<int32_t>(size_t(N) * c.top_k);
  L.q = cv.take<uint8_t>(size_t(N) * H * c.head_dim * ab);
  L.k = cv.take<uint8_t>(size_t(N) * c.n_kv_heads * c.head_dim * ab);
  L.v = cv.take<uint8_t>(size_t(N) * c.n_kv_heads * c.head_dim * ab);
  L.o = cv.take<uint8_t>(size_t(N) * H * c.head_dim * ab);
  L.xt = cv.take<uint8_t>(size_t(N) * c.d_model * ab);
  return L;
}

float *carve_qkv(Carve &cv, const triroute_cfg &c, int N) {
  return cv.take<float>(tr::qkv_rope_floats(c, N));
}

// A stack's own buffers, ahead of the layer workspace: the activations
// handed between layers (two, used in turn), the next layer's side features
// and the decisions of the layer just run.
struct StackBufs {
  void *xa, *xb;
  float *psi;
  uint8_t *mode, *bit;
  int32_t *eidx;
};

StackBufs carve_stack(Carve &cv, const triroute_cfg &c, int B) {
  const size_t ab = act_bytes(c);
  StackBufs S;
  S.xa = cv.take<uint8_t>(size_t(B) * c.d_model * ab);
  S.xb = cv.take<uint8_t>(size_t(B) * c.d_model * ab);
  S.psi = cv.take<float>(size_t(B) * c.d_psi);
  S.mode = cv.take<uint8_t>(size_t(B) * c.n_heads);
  S.bit = cv.take<uint8_t>(B);
  S.eidx = cv.take<int32_t>(size_t(B) * c.top_k);
  return S;
}

// The relaxed controller forward's scratch beyond the router's: the folded
// head weights, the tail's logits and h^, and the rows of partial sums.
struct RelaxWs {
  float *Wf, *cf, *z, *h;
  double *part;
};
RelaxWs carve_relax(Carve &cv, const triroute_cfg &c, int N) {
  const int NZ = 3 * tr::attn_groups(c) + c.n_experts + 5;
  RelaxWs w;
  w.Wf = cv.take<float>(size_t(NZ) * 128);
  w.cf = cv.take<float>(NZ);
  w.z = cv.take<float>(size_t(N) * NZ);
  w.h = cv.take<float>(size_t(N) * 128);
  w.part = cv.take<double>(tr::relax_part_doubles());
  return w;
}

// The relaxed backward's scratch beyond the forward's: taps of the
// recomputed trunk, the recomputed tail's decisions (discarded), the
// per-token gradients, [n1; psi] and its gradient, and the gram partials.
struct RelaxBwdWs {
  float *a1, *hpre, *dz, *dh, *da1, *u, *tgr, *lmsq, *s, *ds, *part, *G, *dc;
  double *lmsq_sum;
  void *n1;
  uint8_t *mode, *bit;
  int32_t *eidx;
  float *egate;
};
RelaxBwdWs carve_relax_bwd(Carve &cv, const triroute_cfg &c, int N) {
  const int NZ = 3 * tr::attn_groups(c) + c.n_experts + 5, K1 = c.d_model + c.d_psi;
  RelaxBwdWs w;
  w.a1 = cv.take<float>(size_t(N) * 128);
  w.hpre = cv.take<float>(size_t(N) * 128);
  w.dz = cv.take<float>(size_t(N) * NZ);
  w.dh = cv.take<float>(size_t(N) * 128);
  w.da1 = cv.take<float>(size_t(N) * 128);
  w.u = cv.take<float>(size_t(N) * 128);
  w.tgr = cv.take<float>(size_t(N) * 128);
  w.lmsq = cv.take<float>(size_t(N) * 4);
  w.s = cv.take<float>(size_t(N) * K1);
  w.ds = cv.take<float>(size_t(N) * K1);
  w.part = cv.take<float>(tr::relax_grad_part_floats(c, N));
  w.G = cv.take<float>(size_t(NZ) * 128);
  w.dc = cv.take<float>(NZ);
  w.lmsq_sum = cv.take<double>(4);
  w.n1 = cv.take<uint8_t>(size_t(N) * c.d_model * act_bytes(c));
  w.mode = cv.take<uint8_t>(size_t(N) * c.n_heads);
  w.bit = cv.take<uint8_t>(N);
  w.eidx = cv.take<int32_t>(size_t(N) * c.top_k);
  w.egate = cv.take<float>(size_t(N) * c.top_k);
  return w;
}

size_t op_bytes(const triroute_cfg &c, int op, int B, int T) {
  Carve cv(nullptr);
  const int N = B * T;
  switch (op) {
    case TRIROUTE_OP_ROUTER: carve_router(cv, c, N); break;
    case TRIROUTE_OP_QKV: carve_qkv(cv, c, N); break;
    case TRIROUTE_OP_KV_APPEND: carve_kv(cv, c, B, T); break;
    case TRIROUTE_OP_ATTN_PREFILL: break;
    case TRIROUTE_OP_ATTN_DECODE: carve_attn_decode(cv, c, B); break;
    case TRIROUTE_OP_MOE: carve_moe(cv, c, N); break;
    case TRIROUTE_OP_LAYER_PREFILL:
    case TRIROUTE_OP_LAYER_DECODE: {
      carve_layer(cv, c, B, T);
      size_t s = 0;
      // router scratch and rotation table together (the table outlives the router)
      s = std::max(s, op_bytes(c, TRIROUTE_OP_ROUTER, B, T) + op_bytes(c, TRIROUTE_OP_QKV, B, T));
      s = std::max(s, op_bytes(c, TRIROUTE_OP_KV_APPEND, B, T));
      s = std::max(s, op_bytes(c, op == TRIROUTE_OP_LAYER_DECODE ? TRIROUTE_OP_ATTN_DECODE
                                                                 : TRIROUTE_OP_ATTN_PREFILL,
                               B, T));
      s = std::max(s, op_bytes(c, TRIROUTE_OP_MOE, B, T));
      return cv.used + s;
    }
    case TRIROUTE_OP_STACK_DECODE:
      carve_stack(cv, c, B);
      return cv.used + op_bytes(c, TRIROUTE_OP_LAYER_DECODE, B, 1);
    case TRIROUTE_OP_ROUTER_RELAXED:
      carve_router(cv, c, N);
      carve_relax(cv, c, N);
      break;
    case TRIROUTE_OP_ROUTER_RELAXED_BACKWARD:
      carve_router(cv, c, N);
      carve_relax(cv, c, N);
      carve_relax_bwd(cv, c, N);
      break;
    default: return 0;
  }
  return cv.used;
}

int check_cfg(const triroute_cfg *c) {
  REQUIRE(c, TRIROUTE_E_INVALID, "cfg is NULL");
  REQUIRE(c->act == TRIROUTE_F32 || c->act == TRIROUTE_BF16, TRIROUTE_E_INVALID,
          "act must be TRIROUTE_F32 or TRIROUTE_BF16 (got %d)", c->act);
  REQUIRE(c->d_model > 0 && c->n_heads > 0 && c->n_kv_heads > 0 && c->head_dim > 0 &&
              c->window > 0 && c->n_experts > 0 && c->top_k > 0 && c->d_ff > 0 &&
              c->kv_group > 0 && c->d_psi >= 0 && c->d_router > 0,
          TRIROUTE_E_INVALID, "cfg has a non-positive size");
  REQUIRE(c->rms_eps > 0.f && c->rope_theta > 0.f, TRIROUTE_E_INVALID,
          "rms_eps and rope_theta must be positive");
  REQUIRE(c->n_heads % c->n_kv_heads == 0, TRIROUTE_E_INVALID,
          "n_heads (%d) must be a multiple of n_kv_heads (%d)", c->n_heads, c->n_kv_heads);
  REQUIRE(c->top_k <= c->n_experts + 1, TRIROUTE_E_INVALID, "top_k (%d) > n_experts + 1 (%d)",
          c->top_k, c->n_experts + 1);
  REQUIRE(c->head_dim == 64 || c->head_dim == 128, TRIROUTE_E_UNSUPPORTED,
          "head_dim %d not in {64, 128}", c->head_dim);
  REQUIRE(c->kv_group == 32 || c->kv_group == 64, TRIROUTE_E_UNSUPPORTED,
          "kv_group %d not in {32, 64}", c->kv_group);
  REQUIRE(c->head_dim % c->kv_group == 0, TRIROUTE_E_UNSUPPORTED,
          "kv_group %d does not divide head_dim %d", c->kv_group, c->head_dim);
  REQUIRE(c->n_heads / c->n_kv_heads <= 16, TRIROUTE_E_UNSUPPORTED,
          "more than 16 query heads per kv head");
  REQUIRE(c->d_router == 128, TRIROUTE_E_UNSUPPORTED, "d_router %d != 128", c->d_router);
  REQUIRE(c->d_psi <= 32 && c->d_psi % 4 == 0, TRIROUTE_E_UNSUPPORTED,
          "d_psi %d: must be a multiple of 4, at most 32", c->d_psi);
  REQUIRE(c->n_experts + 1 <= 64, TRIROUTE_E_UNSUPPORTED, "n_experts + 1 > 64");
  REQUIRE(c->attn_groups >= 0 && (c->attn_groups == 0 || c->n_heads % c->attn_groups == 0),
          TRIROUTE_E_INVALID, "attn_groups (%d) must be 0 or divide n_heads (%d)", c->attn_groups,
          c->n_heads);
  REQUIRE(3 * tr::attn_groups(*c) + c->n_experts + 5 <= 112, TRIROUTE_E_UNSUPPORTED,
          "router head count 3A + E + 5 > 112");
  REQUIRE(c->d_model % 64 == 0 && c->d_ff % 64 == 0, TRIROUTE_E_UNSUPPORTED,
          "d_model and d_ff must be multiples of 64");
  return TRIROUTE_OK;
}

// Every tensor the kernels read or write in 16-byte pieces must be 16-byte
// aligned (NULL entries are skipped: optional arguments are checked where
// they are required).
int check_aligned(std::initializer_list<const void *> ptrs) {
  for (const void *p : ptrs)
    REQUIRE((uintptr_t(p) & 15) == 0, TRIROUTE_E_INVALID,
            "tensor pointer %p is not 16-byte aligned", p);
  return TRIROUTE_OK;
}

int check_bt(int B, int T) {
  REQUIRE(B >= 1 && T >= 1, TRIROUTE_E_INVALID, "B (%d) and T (%d) must be >= 1", B, T);
  REQUIRE(int64_t(B) * T <= (int64_t(1) << 24), TRIROUTE_E_UNSUPPORTED,
          "B*T = %lld tokens exceeds 2^24", (long long)B * T);
  return TRIROUTE_OK;
}

int check_ws(const triroute_cfg &c, int op, int B, int T, const void *ws, size_t ws_bytes) {
  const size_t need = op_bytes(c, op, B, T);
  REQUIRE(need == 0 || ws, TRIROUTE_E_INVALID, "workspace is NULL (%zu bytes needed)", need);
  REQUIRE(ws_bytes >= need, TRIROUTE_E_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes,
          need);
  REQUIRE((uintptr_t(ws) & 255) == 0, TRIROUTE_E_INVALID, "workspace must be 256-byte aligned");
  return TRIROUTE_OK;
}

int check_cache(const triroute_cfg &c, const triroute_kv_cache *kc, int B, int T) {
  REQUIRE(kc && kc->base, TRIROUTE_E_INVALID, "cache is NULL or not initialised");
  REQUIRE(kc->tile_slots == 4096 / c.head_dim, TRIROUTE_E_INVALID,
          "cache was laid out for another head_dim");
  REQUIRE(B <= kc->n_seq, TRIROUTE_E_INVALID, "B (%d) > cache sequences (%d)", B, kc->n_seq);
  REQUIRE(T <= kc->capacity, TRIROUTE_E_CAPACITY, "T (%d) > cache capacity (%d)", T,
          kc->capacity);
  return TRIROUTE_OK;
}

#define TRY(expr)                 \
  do {                            \
    int r_ = (expr);              \
    if (r_ != TRIROUTE_OK) return r_; \
  } while (0)

void layout_cache(const triroute_cfg &c, int n_seq, int capacity, triroute_kv_cache *kc) {
  memset(kc, 0, sizeof *kc);
  const int dh = c.head_dim, G = c.kv_group, ab = act_bytes(c);
  const int TS = 4096 / dh;
  kc->n_seq = n_seq;
  kc->capacity = capacity;
  kc->tile_slots = TS;
  kc->n_tiles = (capacity + TS - 1) / TS;
  size_t off = 0;
  kc->off_status = off;
  off += 256;
  kc->off_seq_len = off;
  off += align256(size_t(n_seq) * 4);
  kc->off_pool_len = off;
  off += align256(size_t(n_seq) * 16);
  kc->off_pos = off;
  off += align256(size_t(n_seq) * 4 * kc->n_tiles * TS * 4);
  for (int bi = 0; bi < 4; ++bi) {
    const int bp = tr::pool_bits(bi, ab);
    kc->tile_bytes[bi] = align256(size_t(1024) * bp + (bi < 3 ? size_t(2) * TS * (dh / G) * 4 : 0));
    kc->off_pool[bi] = off;
    off += size_t(n_seq) * c.n_kv_heads * kc->n_tiles * kc->tile_bytes[bi];
  }
  kc->total_bytes = off;
}

// Paged layout: the header words, per-sequence lengths, held-page counts and
// page tables, the free stacks, then per width its positions and its tiles
// (page p of width bi: tiles (p Hkv + g) page_tiles + i).
void layout_paged(const triroute_cfg &c, int n_seq, int capacity, int PT, const int32_t np[4],
                  triroute_kv_cache *kc) {
  memset(kc, 0, sizeof *kc);
  const int dh = c.head_dim, G = c.kv_group, ab = act_bytes(c);
  const int TS = 4096 / dh;
  kc->n_seq = n_seq;
  kc->capacity = capacity;
  kc->tile_slots = TS;
  kc->n_tiles = (capacity + TS - 1) / TS;
  kc->page_tiles = PT;
  kc->max_pages = (kc->n_tiles + PT - 1) / PT;
  size_t off = 0;
  kc->off_status = off;
  off += 256;
  kc->off_seq_len = off;
  off += align256(size_t(n_seq) * 4);
  kc->off_pool_len = off;
  off += align256(size_t(n_seq) * 16);
  kc->off_alloc = off;
  off += align256(size_t(n_seq) * 16);
  kc->off_page_table = off;
  off += align256(size_t(n_seq) * 4 * kc->max_pages * 4);
  kc->off_free_top = off;
  off += 256;
  for (int bi = 0; bi < 4; ++bi) {
    kc->n_pages[bi] = np[bi];
    kc->off_free_list[bi] = off;
    off += align256(size_t(np[bi]) * 4);
    kc->off_pos_pool[bi] = off;
    off += align256(size_t(np[bi]) * PT * TS * 4);
  }
  kc->off_pos = kc->off_pos_pool[0];
  for (int bi = 0; bi < 4; ++bi) {
    const int bp = tr::pool_bits(bi, ab);
    kc->tile_bytes[bi] = align256(size_t(1024) * bp + (bi < 3 ? size_t(2) * TS * (dh / G) * 4 : 0));
    kc->off_pool[bi] = off;
    off += size_t(np[bi]) * c.n_kv_heads * PT * kc->tile_bytes[bi];
  }
  kc->total_bytes = off;
}

int check_paged_args(int n_seq, int capacity, int PT, const int32_t *np) {
  REQUIRE(n_seq >= 1 && capacity >= 1, TRIROUTE_E_INVALID, "n_seq and capacity must be >= 1");
  REQUIRE(int64_t(capacity) <= (int64_t(1) << 28), TRIROUTE_E_UNSUPPORTED, "capacity too large");
  REQUIRE(PT >= 1 && PT <= (1 << 16), TRIROUTE_E_INVALID, "page_tiles %d outside [1, 65536]", PT);
  REQUIRE(np, TRIROUTE_E_INVALID, "n_pages is NULL");
  for (int bi = 0; bi < 4; ++bi)
    REQUIRE(np[bi] >= 0 && np[bi] <= (1 << 28), TRIROUTE_E_INVALID,
            "n_pages[%d] = %d outside [0, 2^28]", bi, np[bi]);
  return TRIROUTE_OK;
}

hipError_t run_attn_prefill(const triroute_cfg &c, const triroute_kv_cache &kc, int B, int T,
                            const int32_t *seq_ids, const void *q, const uint8_t *mode,
                            const triroute_compaction &cmp, void *o, hipStream_t st) {
  // the rows no attention block writes: skipped heads, dropped rows
  hipError_t e = tr::launch_attn_zero_rows(c, B, T, mode, seq_ids, kc.n_seq, o, st);
  if (e != hipSuccess) return e;
  const tr::CacheView v = tr::make_view(c, kc);
  return c.act == TRIROUTE_BF16 ? tr::launch_attn_mfma_prefill(c, v, B, T, seq_ids, q, cmp, o, st)
                                : tr::launch_attn_valu_prefill(c, v, B, T, seq_ids, q, cmp, o, st);
}

hipError_t run_attn_decode(const triroute_cfg &c, const triroute_kv_cache &kc, int B,
                           const int32_t *seq_ids, const void *q, const uint8_t *mode, void *o,
                           float *part, hipStream_t st) {
  const tr::CacheView v = tr::make_view(c, kc);
  return c.act == TRIROUTE_BF16 ? tr::launch_attn_mfma_decode(c, v, B, seq_ids, q, mode, o, part, st)
                                : tr::launch_attn_valu_decode(c, v, B, seq_ids, q, mode, o, st);
}

}  // namespace

namespace tr {
CacheView make_view(const triroute_cfg &c, const triroute_kv_cache &k) {
  CacheView v;
  v.base = (uint8_t *)k.base;
  v.status = (int32_t *)(v.base + k.off_status);
  v.seq_len = (int32_t *)(v.base + k.off_seq_len);
  v.pool_len = (int32_t *)(v.base + k.off_pool_len);
  v.pos = (int32_t *)(v.base + k.off_pos);
  v.n_seq = k.n_seq;
  v.capacity = k.capacity;
  v.TS = k.tile_slots;
  v.n_tiles = k.n_tiles;
  v.Hkv = c.n_kv_heads;
  v.dh = c.head_dim;
  v.G = c.kv_group;
  v.act_bytes = act_bytes(c);
  for (int i = 0; i < 4; ++i) {
    v.off_pool[i] = k.off_pool[i];
    v.tile_bytes[i] = k.tile_bytes[i];
  }
  v.PT = k.page_tiles;
  v.max_pages = k.max_pages;
  v.page_table = v.alloc = v.free_top = nullptr;
  for (int i = 0; i < 4; ++i) v.free_list[i] = v.pos_pool[i] = nullptr;
  if (k.page_tiles > 0) {
    v.page_table = (int32_t *)(v.base + k.off_page_table);
    v.alloc = (int32_t *)(v.base + k.off_alloc);
    v.free_top = (int32_t *)(v.base + k.off_free_top);
    for (int i = 0; i < 4; ++i) {
      v.free_list[i] = (int32_t *)(v.base + k.off_free_list[i]);
      v.pos_pool[i] = (int32_t *)(v.base + k.off_pos_pool[i]);
    }
  }
  return v;
}
}  // namespace tr

// ======================================================================= ABI
extern "C" {

const char *triroute_status_string(int s) {
  switch (s) {
    case TRIROUTE_OK: return "ok";
    case TRIROUTE_E_INVALID: return "invalid argument";
    case TRIROUTE_E_UNSUPPORTED: return "unsupported shape or dtype";
    case TRIROUTE_E_WORKSPACE: return "workspace too small";
    case TRIROUTE_E_CAPACITY: return "cache capacity exceeded";
    case TRIROUTE_E_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char *triroute_last_error(void) { return g_err; }

int triroute_validate(const triroute_cfg *cfg) {
  g_err[0] = 0;
  return check_cfg(cfg);
}

int triroute_workspace_bytes(const triroute_cfg *cfg, int op, int B, int T, size_t *bytes) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, T));
  REQUIRE(bytes, TRIROUTE_E_INVALID, "bytes is NULL");
  REQUIRE(op >= TRIROUTE_OP_ROUTER && op <= TRIROUTE_OP_ROUTER_RELAXED_BACKWARD, TRIROUTE_E_INVALID,
          "unknown op %d", op);
  *bytes = op_bytes(*cfg, op, B, T);
  return TRIROUTE_OK;
}

int triroute_kv_cache_bytes(const triroute_cfg *cfg, int n_seq, int capacity, size_t *bytes) {
  TRY(check_cfg(cfg));
  REQUIRE(bytes, TRIROUTE_E_INVALID, "bytes is NULL");
  REQUIRE(n_seq >= 1 && capacity >= 1, TRIROUTE_E_INVALID, "n_seq and capacity must be >= 1");
  REQUIRE(int64_t(capacity) <= (int64_t(1) << 28), TRIROUTE_E_UNSUPPORTED, "capacity too large");
  triroute_kv_cache kc;
  layout_cache(*cfg, n_seq, capacity, &kc);
  *bytes = kc.total_bytes;
  return TRIROUTE_OK;
}

int triroute_kv_cache_init(const triroute_cfg *cfg, triroute_kv_cache *cache, void *base,
                           size_t bytes, int n_seq, int capacity, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  REQUIRE(cache && base, TRIROUTE_E_INVALID, "cache or base is NULL");
  REQUIRE((uintptr_t(base) & 255) == 0, TRIROUTE_E_INVALID, "cache base must be 256-byte aligned");
  REQUIRE(n_seq >= 1 && capacity >= 1, TRIROUTE_E_INVALID, "n_seq and capacity must be >= 1");
  triroute_kv_cache kc;
  layout_cache(*cfg, n_seq, capacity, &kc);
  REQUIRE(bytes >= size_t(kc.total_bytes), TRIROUTE_E_CAPACITY,
          "cache allocation %zu bytes < %lld needed", bytes, (long long)kc.total_bytes);
  kc.base = base;
  CHECK_HIP(tr::launch_fill_u32(base, kc.total_bytes / 4, 0u, (hipStream_t)stream), "cache clear");
  *cache = kc;
  return TRIROUTE_OK;
}

int triroute_kv_paged_cache_bytes(const triroute_cfg *cfg, int n_seq, int capacity,
                                  int page_tiles, const int32_t n_pages[4], size_t *bytes) {
  TRY(check_cfg(cfg));
  REQUIRE(bytes, TRIROUTE_E_INVALID, "bytes is NULL");
  TRY(check_paged_args(n_seq, capacity, page_tiles, n_pages));
  triroute_kv_cache kc;
  layout_paged(*cfg, n_seq, capacity, page_tiles, n_pages, &kc);
  *bytes = kc.total_bytes;
  return TRIROUTE_OK;
}

int triroute_kv_paged_cache_init(const triroute_cfg *cfg, triroute_kv_cache *cache, void *base,
                                 size_t bytes, int n_seq, int capacity, int page_tiles,
                                 const int32_t n_pages[4], triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  REQUIRE(cache && base, TRIROUTE_E_INVALID, "cache or base is NULL");
  REQUIRE((uintptr_t(base) & 255) == 0, TRIROUTE_E_INVALID, "cache base must be 256-byte aligned");
  TRY(check_paged_args(n_seq, capacity, page_tiles, n_pages));
  triroute_kv_cache kc;
  layout_paged(*cfg, n_seq, capacity, page_tiles, n_pages, &kc);
  REQUIRE(bytes >= size_t(kc.total_bytes), TRIROUTE_E_CAPACITY,
          "cache allocation %zu bytes < %lld needed", bytes, (long long)kc.total_bytes);
  kc.base = base;
  hipStream_t st = (hipStream_t)stream;
  // everything is cleared, as for the contiguous layout: the attention
  // kernels read whole tiles, and the slots past a pool's length must hold
  // finite values (their weights are zero); then the free stacks get every
  // page.  A page returned by a reset keeps finite values from its appends.
  CHECK_HIP(tr::launch_fill_u32(base, kc.total_bytes / 4, 0u, st), "cache clear");
  CHECK_HIP(tr::launch_kv_paged_init(tr::make_view(*cfg, kc), kc.n_pages, st), "page stacks");
  *cache = kc;
  return TRIROUTE_OK;
}

int triroute_kv_free_pages(const triroute_kv_cache *cache, int32_t free_pages[4],
                           triroute_stream_t stream) {
  REQUIRE(cache && cache->base && free_pages, TRIROUTE_E_INVALID, "NULL argument");
  REQUIRE(cache->page_tiles > 0, TRIROUTE_E_INVALID, "the cache is not paged");
  CHECK_HIP(hipStreamSynchronize((hipStream_t)stream), "stream sync");
  CHECK_HIP(hipMemcpy(free_pages, (uint8_t *)cache->base + cache->off_free_top, 16,
                      hipMemcpyDeviceToHost),
            "free page read");
  return TRIROUTE_OK;
}

int triroute_kv_reset_seq(const triroute_cfg *cfg, const triroute_kv_cache *cache, int seq,
                          triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  REQUIRE(cache && cache->base, TRIROUTE_E_INVALID, "cache is NULL");
  REQUIRE(seq >= 0 && seq < cache->n_seq, TRIROUTE_E_INVALID, "seq %d out of range", seq);
  hipStream_t st = (hipStream_t)stream;
  if (cache->page_tiles > 0) {  // its pages go back to the free stacks
    CHECK_HIP(tr::launch_kv_paged_reset(tr::make_view(*cfg, *cache), seq, st), "reset");
    return TRIROUTE_OK;
  }
  // Appends overwrite every bit a slot owns, so emptying a sequence only
  // needs its lengths cleared.
  uint8_t *b = (uint8_t *)cache->base;
  CHECK_HIP(tr::launch_fill_u32(b + cache->off_seq_len + 4 * size_t(seq), 1, 0u, st), "reset");
  CHECK_HIP(tr::launch_fill_u32(b + cache->off_pool_len + 16 * size_t(seq), 4, 0u, st), "reset");
  return TRIROUTE_OK;
}

int triroute_kv_status(const triroute_kv_cache *cache, int32_t *status, triroute_stream_t stream) {
  REQUIRE(cache && cache->base && status, TRIROUTE_E_INVALID, "NULL argument");
  CHECK_HIP(hipStreamSynchronize((hipStream_t)stream), "stream sync");
  CHECK_HIP(hipMemcpy(status, (uint8_t *)cache->base + cache->off_status, 4, hipMemcpyDeviceToHost),
            "status read");
  return TRIROUTE_OK;
}

const int32_t *triroute_kv_seq_len_ptr(const triroute_kv_cache *cache) {
  if (!cache || !cache->base) return nullptr;
  return (const int32_t *)((uint8_t *)cache->base + cache->off_seq_len);
}

int triroute_kv_append(const triroute_cfg *cfg, const triroute_kv_cache *cache, int B, int T,
                       const int32_t *seq_ids, const void *k, const void *v, const uint8_t *bit,
                       void *ws, size_t ws_bytes, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, T));
  TRY(check_cache(*cfg, cache, B, T));
  REQUIRE(k && v && bit, TRIROUTE_E_INVALID, "k, v or bit is NULL");
  TRY(check_aligned({k, v}));
  TRY(check_ws(*cfg, TRIROUTE_OP_KV_APPEND, B, T, ws, ws_bytes));
  Carve cv(ws);
  const tr::KvWs kw = carve_kv(cv, *cfg, B, T);
  CHECK_HIP(tr::launch_kv_append(*cfg, tr::make_view(*cfg, *cache), B, T, seq_ids, k, v, bit, kw,
                                 (hipStream_t)stream),
            "kv_append launch");
  return TRIROUTE_OK;
}

int triroute_kv_export(const triroute_cfg *cfg, const triroute_kv_cache *cache, int seq, int bi,
                       int slot0, int count, void *k_out, void *v_out, uint16_t *k_sz,
                       uint16_t *v_sz, int32_t *pos_out, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  REQUIRE(cache && cache->base, TRIROUTE_E_INVALID, "cache is NULL");
  REQUIRE(seq >= 0 && seq < cache->n_seq, TRIROUTE_E_INVALID, "seq out of range");
  REQUIRE(bi >= 0 && bi < 4, TRIROUTE_E_INVALID, "bit index out of range");
  REQUIRE(slot0 >= 0 && count >= 1 && int64_t(slot0) + count <= cache->capacity,
          TRIROUTE_E_INVALID, "slot range outside the capacity");
  REQUIRE(k_out && v_out, TRIROUTE_E_INVALID, "k_out or v_out is NULL");
  CHECK_HIP(tr::launch_kv_export(*cfg, tr::make_view(*cfg, *cache), seq, bi, slot0, count, k_out,
                                 v_out, k_sz, v_sz, pos_out, (hipStream_t)stream),
            "kv_export launch");
  return TRIROUTE_OK;
}

int triroute_router(const triroute_cfg *cfg, int B, int T, const void *x, const float *psi,
                    const triroute_router_w *w, void *n1, uint8_t *mode, uint8_t *bit,
                    int32_t *eidx, float *egate, const triroute_compaction *cmp, void *ws,
                    size_t ws_bytes, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, T));
  REQUIRE(x && (psi || cfg->d_psi == 0) && w && n1 && mode && bit && eidx && egate && cmp,
          TRIROUTE_E_INVALID, "NULL argument");
  REQUIRE(w->g1 && w->W1 && w->b1 && w->W2 && w->b2 && w->gr && w->Wa && w->ca && w->We &&
              w->ce && w->Wb && w->cb,
          TRIROUTE_E_INVALID, "NULL router weight");
  REQUIRE(cmp->attn_cnt && cmp->attn_idx && cmp->exp_cnt && cmp->exp_off && cmp->exp_rows,
          TRIROUTE_E_INVALID, "NULL compaction array");
  TRY(check_aligned({x, n1, w->g1, w->W1, w->W2, w->Wa, w->We, w->Wb}));
  TRY(check_ws(*cfg, TRIROUTE_OP_ROUTER, B, T, ws, ws_bytes));
  TRY(prepare_once());
  Carve cv(ws);
  RouterWs rw = carve_router(cv, *cfg, B * T);
  hipStream_t st = (hipStream_t)stream;
  CHECK_HIP(tr::launch_router(*cfg, B * T, x, psi, *w, n1, mode, bit, eidx, egate, rw.rinv, rw.u,
                              nullptr, st),
            "router launch");
  CHECK_HIP(tr::launch_compact(*cfg, B, T, mode, eidx, *cmp, rw.hist, st), "compaction launch");
  return TRIROUTE_OK;
}

int triroute_router_relaxed(const triroute_cfg *cfg, int B, int T, const void *x,
                            const float *psi, const triroute_router_w *w,
                            const triroute_relax_params *p, void *n1, uint8_t *mode,
                            uint8_t *bit, int32_t *eidx, float *egate,
                            const triroute_compaction *cmp, const triroute_relax_out *out,
                            void *ws, size_t ws_bytes, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, T));
  REQUIRE(x && (psi || cfg->d_psi == 0) && w && p && n1 && mode && bit && eidx && egate && cmp &&
              out,
          TRIROUTE_E_INVALID, "NULL argument");
  REQUIRE(w->g1 && w->W1 && w->b1 && w->W2 && w->b2 && w->gr && w->Wa && w->ca && w->We &&
              w->ce && w->Wb && w->cb,
          TRIROUTE_E_INVALID, "NULL router weight");
  REQUIRE(cmp->attn_cnt && cmp->attn_idx && cmp->exp_cnt && cmp->exp_off && cmp->exp_rows,
          TRIROUTE_E_INVALID, "NULL compaction array");
  REQUIRE(p->g_attn && p->g_bits && p->pos, TRIROUTE_E_INVALID, "NULL noise or position array");
  REQUIRE(!p->white_mu == !p->white_sd, TRIROUTE_E_INVALID,
          "white_mu and white_sd must both be given or both be NULL");
  REQUIRE(isfinite(p->tau_a) && isfinite(p->tau_b) && p->tau_a > 0.f && p->tau_b > 0.f,
          TRIROUTE_E_INVALID, "temperatures must be finite and positive (%g, %g)", p->tau_a,
          p->tau_b);
  REQUIRE(isfinite(p->white_eps) && isfinite(p->zeta) && isfinite(p->alpha) &&
              isfinite(p->beta) && isfinite(p->gamma) && isfinite(p->c_target[0]) &&
              isfinite(p->c_target[1]) && isfinite(p->dual_lr) && isfinite(p->dual_ema),
          TRIROUTE_E_INVALID, "a relaxation parameter is not finite");
  REQUIRE(p->dual_ema >= 0.f && p->dual_ema <= 1.f, TRIROUTE_E_INVALID,
          "dual_ema (%g) outside [0, 1]", p->dual_ema);
  REQUIRE(out->y_attn && out->y_bits && out->c_flops && out->c_mem && out->stats,
          TRIROUTE_E_INVALID, "NULL relaxed output");
  TRY(check_aligned({x, n1, w->g1, w->W1, w->W2, w->Wa, w->We, w->Wb}));
  TRY(check_ws(*cfg, TRIROUTE_OP_ROUTER_RELAXED, B, T, ws, ws_bytes));
  TRY(prepare_once());
  const int N = B * T, A = tr::attn_groups(*cfg), E1 = cfg->n_experts + 1;
  Carve cv(ws);
  RouterWs rw = carve_router(cv, *cfg, N);
  RelaxWs xw = carve_relax(cv, *cfg, N);
  hipStream_t st = (hipStream_t)stream;
  triroute_router_w wf = *w;
  if (p->white_mu) {
    CHECK_HIP(tr::launch_white_fold(*cfg, *w, p->white_mu, p->white_sd, p->white_eps, xw.Wf,
                                    xw.cf, st),
              "whitening fold launch");
    wf.Wa = xw.Wf;
    wf.We = xw.Wf + size_t(3 * A) * 128;
    wf.Wb = xw.Wf + size_t(3 * A + E1) * 128;
    wf.ca = xw.cf;
    wf.ce = xw.cf + 3 * A;
    wf.cb = xw.cf + 3 * A + E1;
  }
  tr::TailTap tap;
  tap.h = xw.h;
  tap.z = out->z ? out->z : xw.z;
  CHECK_HIP(tr::launch_router(*cfg, N, x, psi, wf, n1, mode, bit, eidx, egate, rw.rinv, rw.u,
                              nullptr, st, tap),
            "router launch");
  tr::RelaxJob j;
  j.z = tap.z; j.h = tap.h; j.g_attn = p->g_attn; j.g_bits = p->g_bits; j.pos = p->pos;
  j.eidx = eidx; j.egate = egate; j.mode = mode; j.bit = bit;
  j.y_attn = out->y_attn; j.y_bits = out->y_bits; j.p_exp = out->p_exp;
  j.c_flops = out->c_flops; j.c_mem = out->c_mem; j.part = xw.part; j.dual = p->dual;
  j.stats = out->stats; j.usage_exp = out->usage_exp; j.h_mean = out->h_mean; j.h_var = out->h_var;
  j.tau_a = p->tau_a; j.tau_b = p->tau_b; j.zeta = p->zeta; j.alpha = p->alpha;
  j.beta = p->beta; j.gamma = p->gamma; j.target_f = p->c_target[0]; j.target_m = p->c_target[1];
  j.dual_lr = p->dual_lr; j.dual_ema = p->dual_ema;
  CHECK_HIP(tr::launch_relax(*cfg, N, j, st), "relaxed forward launch");
  CHECK_HIP(tr::launch_compact(*cfg, B, T, mode, eidx, *cmp, rw.hist, st), "compaction launch");
  return TRIROUTE_OK;
}

int triroute_router_relaxed_backward(const triroute_cfg *cfg, int B, int T, const void *x,
                                     const float *psi, const triroute_router_w *w,
                                     const triroute_relax_params *p,
                                     const triroute_relax_out *fwd, const int32_t *eidx,
                                     const float *egate, const triroute_relax_grad_in *gin,
                                     const triroute_relax_grad_out *go, void *ws,
                                     size_t ws_bytes, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, T));
  REQUIRE(x && (psi || cfg->d_psi == 0) && w && p && fwd && eidx && egate && gin && go,
          TRIROUTE_E_INVALID, "NULL argument");
  REQUIRE(w->g1 && w->W1 && w->b1 && w->W2 && w->b2 && w->gr && w->Wa && w->ca && w->We &&
              w->ce && w->Wb && w->cb,
          TRIROUTE_E_INVALID, "NULL router weight");
  REQUIRE(p->pos, TRIROUTE_E_INVALID, "NULL position array");
  REQUIRE(!p->white_mu == !p->white_sd, TRIROUTE_E_INVALID,
          "white_mu and white_sd must both be given or both be NULL");
  REQUIRE(isfinite(p->tau_a) && isfinite(p->tau_b) && p->tau_a > 0.f && p->tau_b > 0.f,
          TRIROUTE_E_INVALID, "temperatures must be finite and positive (%g, %g)", p->tau_a,
          p->tau_b);
  REQUIRE(isfinite(p->white_eps) && isfinite(p->zeta) && isfinite(p->alpha) &&
              isfinite(p->beta) && isfinite(p->gamma),
          TRIROUTE_E_INVALID, "a relaxation parameter is not finite");
  REQUIRE(fwd->y_attn && fwd->y_bits && fwd->stats && fwd->usage_exp, TRIROUTE_E_INVALID,
          "the backward reads the forward's y_attn, y_bits, stats and usage_exp");
  REQUIRE(gin->g_attn && gin->g_bits && gin->g_gate, TRIROUTE_E_INVALID, "NULL upstream gradient");
  REQUIRE(isfinite(gin->rho_m) && gin->rho_m >= 0.f && gin->rho_m <= 1.f, TRIROUTE_E_INVALID,
          "rho_m (%g) outside [0, 1]", gin->rho_m);
  REQUIRE(go->dW1 && go->db1 && go->dW2 && go->db2 && go->dgr && go->dWa && go->dca && go->dWe &&
              go->dce && go->dWb && go->dcb && go->dg1 && go->dx && (go->dpsi || cfg->d_psi == 0),
          TRIROUTE_E_INVALID, "NULL gradient output");
  TRY(check_aligned({x, w->g1, w->W1, w->W2, w->Wa, w->We, w->Wb, go->dx}));
  TRY(check_ws(*cfg, TRIROUTE_OP_ROUTER_RELAXED_BACKWARD, B, T, ws, ws_bytes));
  TRY(prepare_once());
  const int N = B * T, A = tr::attn_groups(*cfg), E1 = cfg->n_experts + 1;
  Carve cv(ws);
  RouterWs rw = carve_router(cv, *cfg, N);
  RelaxWs xw = carve_relax(cv, *cfg, N);
  RelaxBwdWs bw = carve_relax_bwd(cv, *cfg, N);
  hipStream_t st = (hipStream_t)stream;
  // the head weights as the forward applied them, [Wa; We; Wb] in one array
  triroute_router_w wf = *w;
  if (p->white_mu) {
    CHECK_HIP(tr::launch_white_fold(*cfg, *w, p->white_mu, p->white_sd, p->white_eps, xw.Wf,
                                    xw.cf, st),
              "whitening fold launch");
    wf.Wa = xw.Wf;
    wf.We = xw.Wf + size_t(3 * A) * 128;
    wf.Wb = xw.Wf + size_t(3 * A + E1) * 128;
    wf.ca = xw.cf;
    wf.ce = xw.cf + 3 * A;
    wf.cb = xw.cf + 3 * A + E1;
  } else {
    CHECK_HIP(hipMemcpyAsync(xw.Wf, w->Wa, size_t(3 * A) * 128 * 4, hipMemcpyDeviceToDevice, st),
              "head weight copy");
    CHECK_HIP(hipMemcpyAsync(xw.Wf + size_t(3 * A) * 128, w->We, size_t(E1) * 128 * 4,
                             hipMemcpyDeviceToDevice, st),
              "head weight copy");
    CHECK_HIP(hipMemcpyAsync(xw.Wf + size_t(3 * A + E1) * 128, w->Wb, size_t(4) * 128 * 4,
                             hipMemcpyDeviceToDevice, st),
              "head weight copy");
  }
  tr::TailTap tap;
  tap.h = xw.h;
  tap.z = xw.z;
  tap.a1 = bw.a1;
  tap.hpre = bw.hpre;
  CHECK_HIP(tr::launch_router(*cfg, N, x, psi, wf, bw.n1, bw.mode, bw.bit, bw.eidx, bw.egate,
                              rw.rinv, rw.u, nullptr, st, tap),
            "router launch");
  tr::RelaxBwdJob j;
  j.z = xw.z; j.hh = xw.h; j.a1 = bw.a1; j.hpre = bw.hpre;
  j.y_attn = fwd->y_attn; j.y_bits = fwd->y_bits; j.egate = egate; j.eidx = eidx; j.pos = p->pos;
  j.g_attn = gin->g_attn; j.g_bits = gin->g_bits; j.g_gate = gin->g_gate;
  j.stats = fwd->stats; j.usage = fwd->usage_exp; j.lambda = gin->lambda;
  j.rho_io = gin->rho; j.rho_m = gin->rho_m;
  j.tau_a = p->tau_a; j.tau_b = p->tau_b; j.zeta = p->zeta; j.alpha = p->alpha; j.beta = p->beta;
  j.gamma = p->gamma;
  j.dz = bw.dz; j.dh = bw.dh; j.da1 = bw.da1; j.u = bw.u; j.tgr = bw.tgr; j.lmsq = bw.lmsq;
  j.s = bw.s; j.ds = bw.ds; j.part = bw.part; j.G = bw.G; j.dc = bw.dc; j.lmsq_sum = bw.lmsq_sum;
  j.out = tr::RelaxGradOut{go->dW1, go->db1, go->dW2, go->db2, go->dgr, go->dWa, go->dca,
                           go->dWe, go->dce, go->dWb, go->dcb, go->dg1, go->dx, go->dpsi,
                           go->lm_norm};
  CHECK_HIP(tr::launch_relax_backward(*cfg, N, x, psi, *w, xw.Wf, p->white_mu, p->white_sd,
                                      p->white_eps, j, st),
            "relaxed backward launch");
  return TRIROUTE_OK;
}

int triroute_qkv(const triroute_cfg *cfg, int B, int T, const void *n1, const triroute_dense_w *w,
                 const int32_t *pos0, void *q, void *k, void *v, void *ws, size_t ws_bytes,
                 triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, T));
  REQUIRE(n1 && w && w->Wq && w->Wk && w->Wv && q && k && v, TRIROUTE_E_INVALID, "NULL argument");
  TRY(check_aligned({n1, w->Wq, w->Wk, w->Wv, q, k, v}));
  TRY(check_ws(*cfg, TRIROUTE_OP_QKV, B, T, ws, ws_bytes));
  Carve cv(ws);
  float *rope = carve_qkv(cv, *cfg, B * T);
  CHECK_HIP(tr::launch_qkv(*cfg, B, T, n1, *w, pos0, nullptr, B, q, k, v, rope, false,
                           (hipStream_t)stream),
            "qkv launch");
  return TRIROUTE_OK;
}

int triroute_attn_prefill(const triroute_cfg *cfg, int B, int T, const int32_t *seq_ids,
                          const void *q, const triroute_kv_cache *cache, const uint8_t *mode,
                          const triroute_compaction *cmp, void *o, void *ws, size_t ws_bytes,
                          triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, T));
  TRY(check_cache(*cfg, cache, B, T));
  REQUIRE(q && mode && cmp && cmp->attn_cnt && cmp->attn_idx && o, TRIROUTE_E_INVALID,
          "NULL argument");
  TRY(check_aligned({q, o}));
  TRY(check_ws(*cfg, TRIROUTE_OP_ATTN_PREFILL, B, T, ws, ws_bytes));
  CHECK_HIP(run_attn_prefill(*cfg, *cache, B, T, seq_ids, q, mode, *cmp, o, (hipStream_t)stream),
            "attn_prefill launch");
  return TRIROUTE_OK;
}

int triroute_attn_decode(const triroute_cfg *cfg, int B, const int32_t *seq_ids, const void *q,
                         const triroute_kv_cache *cache, const uint8_t *mode, void *o, void *ws,
                         size_t ws_bytes, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, 1));
  TRY(check_cache(*cfg, cache, B, 1));
  REQUIRE(q && mode && o, TRIROUTE_E_INVALID, "NULL argument");
  TRY(check_aligned({q, o}));
  TRY(check_ws(*cfg, TRIROUTE_OP_ATTN_DECODE, B, 1, ws, ws_bytes));
  Carve cv(ws);
  float *part = carve_attn_decode(cv, *cfg, B);
  CHECK_HIP(run_attn_decode(*cfg, *cache, B, seq_ids, q, mode, o, part, (hipStream_t)stream),
            "attn_decode launch");
  return TRIROUTE_OK;
}

int triroute_oproj(const triroute_cfg *cfg, int n_tok, const void *x, const void *o,
                   const triroute_dense_w *w, void *xt, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(n_tok, 1));
  REQUIRE(x && o && w && w->Wo && xt, TRIROUTE_E_INVALID, "NULL argument");
  TRY(check_aligned({x, o, w->Wo, xt}));
  CHECK_HIP(tr::launch_oproj(*cfg, n_tok, x, o, *w, xt, (hipStream_t)stream), "oproj launch");
  return TRIROUTE_OK;
}

static int moe_impl(const triroute_cfg *cfg, int n_tok, const void *xt, const triroute_dense_w *dw,
                    const triroute_moe_w *w, const int32_t *eidx, const float *egate,
                    const triroute_compaction *cmp, void *x_out, Carve &cv, hipStream_t st) {
  MoeWs m = carve_moe(cv, *cfg, n_tok);
  CHECK_HIP(tr::launch_moe_norm_rows(*cfg, n_tok, xt, dw->g2, *cmp, eidx, m.n2, m.slot_of, st),
            "moe_norm_rows launch");
  CHECK_HIP(tr::launch_moe_gemms(*cfg, n_tok, m.n2, *w, *cmp, m.Hm, m.Y, st), "moe gemm launch");
  CHECK_HIP(tr::launch_moe_combine(*cfg, n_tok, xt, m.Y, m.slot_of, eidx, egate, x_out, st),
            "combine launch");
  return TRIROUTE_OK;
}

int triroute_moe(const triroute_cfg *cfg, int n_tok, const void *xt, const triroute_dense_w *dw,
                 const triroute_moe_w *w, const int32_t *eidx, const float *egate,
                 const triroute_compaction *cmp, void *x_out, void *ws, size_t ws_bytes,
                 triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(n_tok, 1));
  REQUIRE(xt && dw && dw->g2 && w && w->Wgate && w->Wup && w->Wdown && eidx && egate && cmp &&
              cmp->exp_cnt && cmp->exp_off && cmp->exp_rows && x_out,
          TRIROUTE_E_INVALID, "NULL argument");
  TRY(check_aligned({xt, dw->g2, w->Wgate, w->Wup, w->Wdown, x_out}));
  TRY(check_ws(*cfg, TRIROUTE_OP_MOE, n_tok, 1, ws, ws_bytes));
  Carve cv(ws);
  return moe_impl(cfg, n_tok, xt, dw, w, eidx, egate, cmp, x_out, cv, (hipStream_t)stream);
}

static int layer_impl(const triroute_cfg *cfg, int B, int T, bool decode, const int32_t *seq_ids,
                      const void *x, const float *psi, const triroute_router_w *rw,
                      const triroute_dense_w *dw, const triroute_moe_w *mw,
                      const triroute_kv_cache *cache, void *x_out, const triroute_layer_taps *taps,
                      void *ws, size_t ws_bytes, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, T));
  TRY(check_cache(*cfg, cache, B, T));
  REQUIRE(x && (psi || cfg->d_psi == 0) && rw && dw && mw && x_out, TRIROUTE_E_INVALID,
          "NULL argument");
  TRY(check_aligned({x, x_out, rw->g1, rw->W1, rw->W2, rw->Wa, rw->We, rw->Wb, dw->Wq, dw->Wk,
                     dw->Wv, dw->Wo, dw->g2, mw->Wgate, mw->Wup, mw->Wdown}));
  if (taps) TRY(check_aligned({taps->n1, taps->q, taps->k, taps->v, taps->o, taps->xt}));
  const int op = decode ? TRIROUTE_OP_LAYER_DECODE : TRIROUTE_OP_LAYER_PREFILL;
  TRY(check_ws(*cfg, op, B, T, ws, ws_bytes));
  TRY(prepare_once());
  hipStream_t st = (hipStream_t)stream;
  Carve cv(ws);
  LayerBufs L = carve_layer(cv, *cfg, B, T);
  if (taps) {
    if (taps->n1) L.n1 = taps->n1;
    if (taps->mode) L.mode = taps->mode;
    if (taps->bit) L.bit = taps->bit;
    if (taps->eidx) L.eidx = taps->eidx;
    if (taps->egate) L.egate = taps->egate;
    if (taps->q) L.q = taps->q;
    if (taps->k) L.k = taps->k;
    if (taps->v) L.v = taps->v;
    if (taps->o) L.o = taps->o;
    if (taps->xt) L.xt = taps->xt;
  }
  const size_t scratch_at = cv.used;
  const int N = B * T;
  // positions continue each sequence: its current length, read on the device
  const int32_t *seq_len = triroute_kv_seq_len_ptr(cache);
  {
    // the router's scratch, then the rotation table: the first RMSNorm
    // writes the table, the QKV epilogue reads it
    Carve sc(ws);
    sc.used = scratch_at;
    RouterWs r = carve_router(sc, *cfg, N);
    float *rope = carve_qkv(sc, *cfg, N);
    const tr::RopeJob job = tr::make_rope_job(*cfg, T, seq_len, seq_ids, cache->n_seq, rope);
    CHECK_HIP(tr::launch_router(*cfg, N, x, psi, *rw, L.n1, L.mode, L.bit, L.eidx, L.egate, r.rinv,
                                r.u, &job, st),
              "router launch");
    // decode attention reads the modes themselves: no attention lists
    CHECK_HIP(tr::launch_compact(*cfg, B, T, L.mode, L.eidx, L.cmp, r.hist, st, !decode),
              "compaction");
    CHECK_HIP(tr::launch_qkv(*cfg, B, T, L.n1, *dw, seq_len, seq_ids, cache->n_seq, L.q, L.k, L.v,
                             rope, true, st),
              "qkv launch");
  }
  {
    Carve sc(ws);
    sc.used = scratch_at;
    const tr::KvWs kw = carve_kv(sc, *cfg, B, T);
    CHECK_HIP(tr::launch_kv_append(*cfg, tr::make_view(*cfg, *cache), B, T, seq_ids, L.k, L.v, L.bit,
                                   kw, st),
              "kv_append launch");
  }
  if (decode) {
    Carve sc(ws);
    sc.used = scratch_at;
    float *part = carve_attn_decode(sc, *cfg, B);
    CHECK_HIP(run_attn_decode(*cfg, *cache, B, seq_ids, L.q, L.mode, L.o, part, st),
              "attn_decode launch");
  } else {
    CHECK_HIP(run_attn_prefill(*cfg, *cache, B, T, seq_ids, L.q, L.mode, L.cmp, L.o, st),
              "attn_prefill launch");
  }
  CHECK_HIP(tr::launch_oproj(*cfg, N, x, L.o, *dw, L.xt, st), "oproj launch");
  {
    Carve sc(ws);
    sc.used = scratch_at;
    TRY(moe_impl(cfg, N, L.xt, dw, mw, L.eidx, L.egate, &L.cmp, x_out, sc, st));
  }
  return TRIROUTE_OK;
}

int triroute_layer_prefill(const triroute_cfg *cfg, int B, int T, const int32_t *seq_ids,
                           const void *x, const float *psi, const triroute_router_w *rw,
                           const triroute_dense_w *dw, const triroute_moe_w *mw,
                           const triroute_kv_cache *cache, void *x_out,
                           const triroute_layer_taps *taps, void *ws, size_t ws_bytes,
                           triroute_stream_t stream) {
  return layer_impl(cfg, B, T, false, seq_ids, x, psi, rw, dw, mw, cache, x_out, taps, ws, ws_bytes,
                    stream);
}

int triroute_layer_decode_noalloc(const triroute_cfg *cfg, int B, const int32_t *seq_ids,
                                  const void *x, const float *psi, const triroute_router_w *rw,
                                  const triroute_dense_w *dw, const triroute_moe_w *mw,
                                  const triroute_kv_cache *cache, void *x_out,
                                  const triroute_layer_taps *taps, triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  TRY(check_bt(B, 1));
  const size_t need = op_bytes(*cfg, TRIROUTE_OP_LAYER_DECODE, B, 1);
  REQUIRE(need <= TRIROUTE_STATIC_SCRATCH_BYTES, TRIROUTE_E_WORKSPACE,
          "decode step of %d sequences needs %zu bytes of scratch > the static %zu", B, need,
          (size_t)TRIROUTE_STATIC_SCRATCH_BYTES);
  void *ws = nullptr;
  TRY(static_scratch(&ws));
  return layer_impl(cfg, B, 1, true, seq_ids, x, psi, rw, dw, mw, cache, x_out, taps, ws,
                    TRIROUTE_STATIC_SCRATCH_BYTES, stream);
}

int triroute_layer_decode(const triroute_cfg *cfg, int B, const int32_t *seq_ids, const void *x,
                          const float *psi, const triroute_router_w *rw, const triroute_dense_w *dw,
                          const triroute_moe_w *mw, const triroute_kv_cache *cache, void *x_out,
                          const triroute_layer_taps *taps, void *ws, size_t ws_bytes,
                          triroute_stream_t stream) {
  return layer_impl(cfg, B, 1, true, seq_ids, x, psi, rw, dw, mw, cache, x_out, taps, ws, ws_bytes,
                    stream);
}

int triroute_stack_decode(const triroute_cfg *cfg, int n_layers, int B, const int32_t *seq_ids,
                          const void *x, const float *psi, const triroute_layer_w *layers,
                          const triroute_kv_cache *caches, void *x_out, void *ws, size_t ws_bytes,
                          triroute_stream_t stream) {
  TRY(check_cfg(cfg));
  REQUIRE(n_layers >= 1 && n_layers <= 256, TRIROUTE_E_INVALID, "n_layers (%d) must be in [1, 256]",
          n_layers);
  REQUIRE(layers && caches && x && psi && x_out, TRIROUTE_E_INVALID, "NULL argument");
  REQUIRE(cfg->d_psi >= 4, TRIROUTE_E_INVALID,
          "a stack needs d_psi >= 4 (the previous layer's decisions)");
  TRY(check_bt(B, 1));
  TRY(check_aligned({x, x_out, psi}));
  TRY(check_ws(*cfg, TRIROUTE_OP_STACK_DECODE, B, 1, ws, ws_bytes));
  Carve cv(ws);
  const StackBufs S = carve_stack(cv, *cfg, B);
  void *lws = (uint8_t *)ws + cv.used;
  const size_t lbytes = ws_bytes - cv.used;
  hipStream_t st = (hipStream_t)stream;
  triroute_layer_taps taps{};
  taps.mode = S.mode;
  taps.bit = S.bit;
  taps.eidx = S.eidx;
  const void *xin = x;
  for (int l = 0; l < n_layers; ++l) {
    void *xo = l == n_layers - 1 ? x_out : (l % 2 == 0 ? S.xa : S.xb);
    TRY(layer_impl(cfg, B, 1, true, seq_ids, xin, l == 0 ? psi : S.psi, &layers[l].router,
                   &layers[l].dense, &layers[l].moe, &caches[l], xo, &taps, lws, lbytes, stream));
    if (l + 1 < n_layers)
      CHECK_HIP(tr::launch_psi_next(*cfg, B, psi, S.mode, S.bit, S.eidx, S.psi, st), "psi launch");
    xin = xo;
  }
  return TRIROUTE_OK;
}

}  // extern "C"
