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
//   MoE-2 : Y = H Wdown_e^T
// n2, H and Y of the experts hold one row per entry of the expert lists, in
// list order (the lists lie back to back), so a tile's rows are contiguous.
#include <algorithm>
#include <initializer_list>
#include <type_traits>

#include "kernels.hpp"

namespace tr {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

struct MTile {
  int m0, n0, mvalid, e, p0;
  int k0 = 0, yp = 0;  // K offset of a split product and its output plane
};

// Row tiles of the grouped problems: lane e - 1 of every wave holds expert
// e's row count and tile count, and an inclusive scan over the lanes gives
// the tiles of experts 1..e, so the mapping costs one parallel load instead
// of a chain of E dependent ones (E <= 63).
struct GroupScan {
  int c = 0, nt = 0, incl = 0, total = 0, start = 0;
};

__device__ __forceinline__ GroupScan group_scan(int BM, const int32_t *cnt, int E) {
  const int lane = threadIdx.x & 63;
  GroupScan g;
  g.c = lane < E ? cnt[lane + 1] : 0;
  g.nt = (g.c + BM - 1) / BM;
  int x = g.nt;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  g.incl = x;
  g.total = __shfl(x, 63, 64);
  // first list position of expert lane + 1: the lists lie back to back in
  // expert order, so it is the sum of the counts before it
  int s = g.c;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(s, d, 64);
    if (lane >= d) s += y;
  }
  g.start = s - g.c;
  return g;
}

// Map a linear row-tile index to (expert e >= 1, tile within e).
__device__ __forceinline__ bool mmap_grouped(int bx, int BM, const GroupScan &gs, MTile &t) {
  const uint64_t m = __ballot(gs.incl > bx);
  if (!m) return false;
  const int l = __ffsll((unsigned long long)m) - 1;
  const int incl = __shfl(gs.incl, l, 64), nt = __shfl(gs.nt, l, 64), c = __shfl(gs.c, l, 64);
  const int rem = bx - (incl - nt);
  t.e = l + 1;
  t.p0 = __shfl(gs.start, l, 64) + rem * BM;
  t.mvalid = min(BM, c - rem * BM);
  t.m0 = 0;
  return true;
}

// Physical column n of a BN-wide tile -> (pair index P in the tile, half).
// Wave slice s = n / 64 holds pairs 32 s .. 32 s + 31: first halves in its
// columns 0..31, second halves in 32..63.
__device__ __forceinline__ void col_pair(int n, int &P, int &half) {
  P = (n >> 6) * 32 + (n & 31);
  half = (n >> 5) & 1;
}

// ---------------------------------------------------------------- problems
// Each problem names its operand rows (a_row, b_row), the LDS column of an
// accumulator after the register pass (EPI_ROPE / EPI_SWIGLU combine the
// partner columns first), and a row-wise epilogue that reads the staged fp32
// tile C (NC columns, row stride LDC) and writes 16-byte chunks.
enum { EPI_PLAIN = 0, EPI_ROPE = 1, EPI_SWIGLU = 2 };

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

__device__ __forceinline__ u32x4_t pack8_bf16(const float *v) {
  u32x4_t w;
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = pk_bf16(v[2 * i], v[2 * i + 1]);
  return w;
}

struct QkvM {
  static constexpr bool DIRECT_W4 = true;
  static constexpr int EPI = EPI_ROPE;
  const bf16 *n1, *Wq, *Wk, *Wv, *Wlo;  // Wlo: the lowest of Wq, Wk, Wv
  bf16 *q, *k, *v;
  const float2 *rope;  // (cos, sin) of token row, pair j at row * dh / 2 + j
  int N, d, H, Hkv, dh, Ncols;
  // four-wave kernel: byte offsets of Wq, Wk, Wv from Wlo less the first
  // column of their range times the row pitch, and the range ends
  uint32_t wq_o, wk_o, wv_o;
  int Hd, HKd;
  static constexpr int out_cols(int BN) { return BN; }
  static constexpr bool GROUPED = false;
  __device__ int tiles(int BM, int ny, const GroupScan &) const { return (N + BM - 1) / BM * ny; }
  __device__ bool map(int bx, int by, int BM, int BN, MTile &t, const GroupScan &) const {
    t.m0 = bx * BM;
    t.n0 = by * BN;
    t.mvalid = min(BM, N - t.m0);
    t.e = t.p0 = 0;
    return t.mvalid > 0;
  }
  // logical column (within the tile) of half `half` of pair P
  __device__ int ccol(int P, int half) const {
    const int hd = dh >> 1;
    return (P / hd) * dh + (P % hd) + half * hd;
  }
  __device__ const bf16 *a_base() const { return n1; }
  __device__ const bf16 *b_base() const { return Wlo; }
  __device__ const bf16 *a_row(const MTile &t, int r) const { return n1 + int64_t(t.m0 + r) * d; }
  __device__ const bf16 *b_row(const MTile &t, int n) const {
    int P, half;
    col_pair(n, P, half);
    int gc = t.n0 + ccol(P, half);
    if (gc >= Ncols) return nullptr;
    const int Hd = H * dh, Kd = Hkv * dh;
    if (gc < Hd) return Wq + int64_t(gc) * d;
    gc -= Hd;
    if (gc < Kd) return Wk + int64_t(gc) * d;
    return Wv + int64_t(gc - Kd) * d;
  }
  // Four-wave kernel (128-column tiles, d_h 64 or 128): wave column wn
  // holds pairs j = jw + 2 c + (ni >> 1) of one head, the first half of the
  // pair in block ni even and the second (j + d_h / 2) in ni odd, where
  // d_h 64: the tile's head wn, jw = 0; d_h 128: the tile's one head, jw = 32 wn.
  // Each lane thus holds both halves of pairs 2 c, 2 c + 1 of its rows.
  __device__ void w4_head(const MTile &t, int wn, int &hcol, int &jw) const {
    hcol = t.n0 + (dh == 64 ? 64 * wn : 0);  // first column of the head
    jw = dh == 64 ? 0 : 32 * wn;
  }
  __device__ uint32_t a_off(const MTile &t, int r) const { return uint32_t(t.m0 + r) * uint32_t(2 * d); }
  // 256-column tiles (d_h 128 only): wave column wn holds the tile's head
  // wn, lane column c pairs j = 4 c + (ni >> 1), first halves in even ni.
  template <int NI>
  __device__ uint32_t b_off_w4(const MTile &t, int wn, int ni, int c) const {
    int hcol, jw;
    if constexpr (NI == 8) {
      hcol = t.n0 + 128 * wn;
      jw = 0;
    } else {
      w4_head(t, wn, hcol, jw);
    }
    const int gc = hcol + jw + (NI / 2) * c + (ni >> 1) + (ni & 1) * (dh >> 1);
    // (arithmetic on the field values: a select of fields by a lane-varying
    // condition becomes a per-lane load from the kernel arguments)
    const uint32_t base = wq_o + uint32_t(gc >= Hd) * (wk_o - wq_o) + uint32_t(gc >= HKd) * (wv_o - wk_o);
    return gc < Ncols ? base + uint32_t(gc) * uint32_t(2 * d) : 0u;
  }
  template <int MI, int NI>
  __device__ void store_w4(const MTile &t, const f32x4_t (&acc)[MI][NI], int wm, int wn, int lane) const {
    if constexpr (NI == 8)
      store_w4_wide(t, acc, wm, wn, lane);
    else
      store_w4_narrow(t, acc, wm, wn, lane);
  }
  // 256-column tiles: each lane holds both halves of pairs j .. j + 3 of
  // head wn; the rotation entries of a row block mi are loaded one block
  // ahead of their use.
  template <int MI, int NI>
  __device__ void store_w4_wide(const MTile &t, const f32x4_t (&acc)[MI][NI], int wm, int wn,
                                int lane) const {
    const int hcol = t.n0 + 128 * wn;
    if (hcol >= Ncols) return;
    const int Hd = H * dh, Kd = Hkv * dh, hd = dh >> 1;
    bf16 *out = q;
    int ld = Hd, col = hcol;
    bool rot = true;
    if (hcol >= Hd + Kd) {
      out = v; ld = Kd; col = hcol - Hd - Kd; rot = false;
    } else if (hcol >= Hd) {
      out = k; ld = Kd; col = hcol - Hd;
    }
    const int j = 4 * (lane & 15);
    auto row_of = [&](int mi, int i) { return wm * MI * 16 + mi * 16 + 4 * (lane >> 4) + i; };
    auto load_cs = [&](int mi, float4 (&cs)[4][2]) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = row_of(mi, i);
        const float4 *tb = (const float4 *)(rope + int64_t(t.m0 + (r < t.mvalid ? r : 0)) * hd + j);
        cs[i][0] = tb[0];
        cs[i][1] = tb[1];
      }
    };
    float4 cur[4][2], nxt[4][2];
    if (rot) load_cs(0, cur);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
      if (rot && mi + 1 < MI) load_cs(mi + 1, nxt);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = row_of(mi, i);
        float y1[4], y2[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float a1 = acc[mi][2 * u][i], a2 = acc[mi][2 * u + 1][i];
          y1[u] = a1;
          y2[u] = a2;
          if (rot) {
            const float4 c4 = cur[i][u >> 1];  // (cos, sin) of pairs j + 2 (u / 2), + 1
            const float cs = (u & 1) ? c4.z : c4.x, sn = (u & 1) ? c4.w : c4.y;
            y1[u] = a1 * cs - a2 * sn;
            y2[u] = a1 * sn + a2 * cs;
          }
        }
        if (r < t.mvalid) {
          bf16 *o = out + int64_t(t.m0 + r) * ld + col + j;
          *(uint2 *)o = make_uint2(pk_bf16(y1[0], y1[1]), pk_bf16(y1[2], y1[3]));
          *(uint2 *)(o + hd) = make_uint2(pk_bf16(y2[0], y2[1]), pk_bf16(y2[2], y2[3]));
        }
      }
      if (rot && mi + 1 < MI) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          cur[i][0] = nxt[i][0];
          cur[i][1] = nxt[i][1];
        }
      }
    }
  }
  template <int MI, int NI>
  __device__ void store_w4_narrow(const MTile &t, const f32x4_t (&acc)[MI][NI], int wm, int wn,
                                  int lane) const {
    static_assert(NI == 4, "two pairs per lane");
    int hcol, jw;
    w4_head(t, wn, hcol, jw);
    if (hcol >= Ncols) return;
    const int Hd = H * dh, Kd = Hkv * dh, hd = dh >> 1;
    bf16 *out = q;
    int ld = Hd, col = hcol;
    bool rot = true;
    if (hcol >= Hd + Kd) {
      out = v; ld = Kd; col = hcol - Hd - Kd; rot = false;
    } else if (hcol >= Hd) {
      out = k; ld = Kd; col = hcol - Hd;
    }
    const int j = jw + 2 * (lane & 15);
    // the rows' rotation entries first, so their loads overlap
    float4 cs[MI][4];
    if (rot) {
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = wm * MI * 16 + mi * 16 + 4 * (lane >> 4) + i;
          cs[mi][i] = *(const float4 *)(rope + int64_t(t.m0 + (r < t.mvalid ? r : 0)) * hd + j);
        }
    }
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * MI * 16 + mi * 16 + 4 * (lane >> 4) + i;
        if (r >= t.mvalid) continue;
        const float a10 = acc[mi][0][i], a20 = acc[mi][1][i], a11 = acc[mi][2][i], a21 = acc[mi][3][i];
        float y10 = a10, y20 = a20, y11 = a11, y21 = a21;
        if (rot) {
          const float4 c4 = cs[mi][i];  // (cos, sin) of pairs j and j + 1
          y10 = a10 * c4.x - a20 * c4.y;
          y20 = a10 * c4.y + a20 * c4.x;
          y11 = a11 * c4.z - a21 * c4.w;
          y21 = a11 * c4.w + a21 * c4.z;
        }
        bf16 *o = out + int64_t(t.m0 + r) * ld + col + j;
        *(uint32_t *)o = pk_bf16(y10, y11);
        *(uint32_t *)(o + hd) = pk_bf16(y20, y21);
      }
  }
  // item = (row, 8 consecutive pairs of one head): rotate-half RoPE on q and
  // k from the token's rotation table; v is copied.
  template <int BM, int NC, int LDC, int NT>
  __device__ void epilogue(const MTile &t, const float *C, int tid) const {
    constexpr int PC = NC / 16;  // 8-pair chunks per row
    const int Hd = H * dh, Kd = Hkv * dh, hd = dh >> 1;
    for (int it = tid; it < BM * PC; it += NT) {
      const int r = it / PC, P0 = (it % PC) * 8;
      const int lc1 = (P0 / hd) * dh + (P0 % hd);
      const int c1 = t.n0 + lc1;
      if (r >= t.mvalid || c1 >= Ncols) continue;
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
      float y1[8], y2[8];
      const float *x1 = C + r * LDC + lc1, *x2 = x1 + hd;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        y1[u] = x1[u];
        y2[u] = x2[u];
      }
      if (rot) {
        const float4 *tb = (const float4 *)(rope + int64_t(row) * hd + col % hd);
#pragma unroll
        for (int u2 = 0; u2 < 4; ++u2) {
          const float4 cs2 = tb[u2];  // pairs 2 u2 and 2 u2 + 1
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int u = 2 * u2 + h;
            const float cs = h ? cs2.z : cs2.x, sn = h ? cs2.w : cs2.y;
            const float a1 = y1[u], a2 = y2[u];
            y1[u] = a1 * cs - a2 * sn;
            y2[u] = a1 * sn + a2 * cs;
          }
        }
      }
      bf16 *o = out + int64_t(row) * ld + col;
      *(u32x4_t *)o = pack8_bf16(y1);
      *(u32x4_t *)(o + hd) = pack8_bf16(y2);
    }
  }
};

struct OprojM {
  static constexpr bool DIRECT_W4 = true;
  static constexpr int EPI = EPI_PLAIN;
  const bf16 *o, *Wo, *x;
  bf16 *xt;
  int N, d, K;
  static constexpr int out_cols(int BN) { return BN; }
  static constexpr bool GROUPED = false;
  __device__ int tiles(int BM, int ny, const GroupScan &) const { return (N + BM - 1) / BM * ny; }
  __device__ bool map(int bx, int by, int BM, int BN, MTile &t, const GroupScan &) const {
    t.m0 = bx * BM;
    t.n0 = by * BN;
    t.mvalid = min(BM, N - t.m0);
    t.e = t.p0 = 0;
    return t.mvalid > 0;
  }
  __device__ const bf16 *a_base() const { return o; }
  __device__ const bf16 *b_base() const { return Wo; }
  __device__ const bf16 *a_row(const MTile &t, int r) const { return o + int64_t(t.m0 + r) * K; }
  __device__ const bf16 *b_row(const MTile &t, int n) const {
    return t.n0 + n < d ? Wo + int64_t(t.n0 + n) * K : nullptr;
  }
  // Four-wave kernel: in wave column wn, MFMA block ni, lane column c holds
  // output column NI (16 wn + c) + ni of the tile, so each lane ends with NI
  // consecutive columns of each of its rows: xt = x + o Wo^T in pieces of
  // NI / 2 words.
  template <int NI>
  __device__ uint32_t b_off_w4(const MTile &t, int wn, int ni, int c) const {
    const int f = t.n0 + NI * (16 * wn + c) + ni;
    return f < d ? uint32_t(f) * uint32_t(2 * K) : 0u;
  }
  __device__ uint32_t a_off(const MTile &t, int r) const { return uint32_t(t.m0 + r) * uint32_t(2 * K); }
  template <int MI, int NI>
  __device__ void store_w4(const MTile &t, const f32x4_t (&acc)[MI][NI], int wm, int wn, int lane) const {
    static_assert(NI % 2 == 0, "whole words");
    const int f = t.n0 + NI * (16 * wn + (lane & 15));
    if (f >= d) return;  // d is a multiple of NI: a lane's columns are all in or all out
    // in halves of the rows (MI / 2 row blocks): each half's residual rows
    // are loaded first, so their loads overlap (all at once would hold 4 MI
    // (NI / 2) registers)
    constexpr int MH = MI / 2;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint32_t xv[MH][4][NI / 2];
#pragma unroll
      for (int m = 0; m < MH; ++m)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = wm * MI * 16 + (h * MH + m) * 16 + 4 * (lane >> 4) + i;
          const uint32_t *xr = (const uint32_t *)(x + int64_t(t.m0 + (r < t.mvalid ? r : 0)) * d + f);
#pragma unroll
          for (int u = 0; u < NI / 2; ++u) xv[m][i][u] = xr[u];
        }
#pragma unroll
      for (int m = 0; m < MH; ++m)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int mi = h * MH + m;
          const int r = wm * MI * 16 + mi * 16 + 4 * (lane >> 4) + i;
          if (r >= t.mvalid) continue;
          uint32_t *yr = (uint32_t *)(xt + int64_t(t.m0 + r) * d + f);
#pragma unroll
          for (int u = 0; u < NI / 2; ++u) {
            const uint32_t w = xv[m][i][u];
            yr[u] = pk_bf16(__uint_as_float(w << 16) + acc[mi][2 * u][i],
                            __uint_as_float(w & 0xFFFF0000u) + acc[mi][2 * u + 1][i]);
          }
        }
    }
  }
  // item = 8 columns of one row: xt = x + o Wo^T
  template <int BM, int NC, int LDC, int NT>
  __device__ void epilogue(const MTile &t, const float *C, int tid) const {
    constexpr int CC = NC / 8;
    for (int it = tid; it < BM * CC; it += NT) {
      const int r = it / CC, c8 = (it % CC) * 8;
      if (r >= t.mvalid || t.n0 + c8 >= d) continue;
      const int64_t off = int64_t(t.m0 + r) * d + t.n0 + c8;
      const u32x4_t xv = *(const u32x4_t *)(x + off);
      float y[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        y[2 * u] = __uint_as_float(xv[u] << 16) + C[r * LDC + c8 + 2 * u];
        y[2 * u + 1] = __uint_as_float(xv[u] & 0xFFFF0000u) + C[r * LDC + c8 + 2 * u + 1];
      }
      *(u32x4_t *)(xt + off) = pack8_bf16(y);
    }
  }
};

struct Moe1M {
  static constexpr int EPI = EPI_SWIGLU;
  const bf16 *n2, *Wg, *Wu, *Wlo;  // n2: normalised rows in list order; Wlo: the lower of Wg, Wu
  bf16 *Hm;
  const int32_t *cnt;
  int E, d, dff;
  static constexpr int out_cols(int BN) { return BN / 2; }
  static constexpr bool GROUPED = true;
  __device__ int tiles(int BM, int ny, const GroupScan &gs) const { return gs.total * ny; }
  __device__ bool map(int bx, int by, int BM, int BN, MTile &t, const GroupScan &gs) const {
    if (!mmap_grouped(bx, BM, gs, t)) return false;
    t.n0 = by * (BN / 2);  // BN/2 expert units per tile (gate + up columns)
    return true;
  }
  __device__ int ccol(int P, int) const { return P; }
  __device__ const bf16 *a_base() const { return n2; }
  __device__ const bf16 *b_base() const { return Wlo; }
  __device__ const bf16 *a_row(const MTile &t, int r) const { return n2 + int64_t(t.p0 + r) * d; }
  __device__ const bf16 *b_row(const MTile &t, int n) const {
    int P, half;
    col_pair(n, P, half);
    const int f = t.n0 + P;
    if (f >= dff) return nullptr;
    return (half ? Wu : Wg) + (int64_t(t.e - 1) * dff + f) * d;
  }
  // Four-wave kernel: in wave column wn, MFMA block ni, lane column c
  // holds expert unit (NI / 2) (16 wn + c) + ni / 2 of the tile, gate for
  // even ni and up for odd, so each lane ends with both halves of NI / 2
  // consecutive units and writes them as one piece per row.
  static constexpr bool DIRECT_W4 = true;
  // Byte offsets from a_base / b_base (32 bits: the host checks the spans).
  // Units past d_ff read unit 0 of the lower matrix instead.
  __device__ uint32_t a_off(const MTile &t, int r) const { return uint32_t(t.p0 + r) * uint32_t(2 * d); }
  template <int NI>
  __device__ uint32_t b_off_w4(const MTile &t, int wn, int ni, int c) const {
    const int f = t.n0 + (NI / 2) * (16 * wn + c) + (ni >> 1);
    if (f >= dff) return 0u;
    const uint32_t m = uint32_t(((ni & 1) ? Wu : Wg) - Wlo) * 2u;
    return m + uint32_t((t.e - 1) * dff + f) * uint32_t(2 * d);
  }
  template <int MI, int NI>
  __device__ void store_w4(const MTile &t, const f32x4_t (&acc)[MI][NI], int wm, int wn, int lane) const {
    static_assert(NI == 8, "4 units per lane, one 8-byte piece per row");
    const int f = t.n0 + (NI / 2) * (16 * wn + (lane & 15));
    if (f >= dff) return;  // d_ff is a multiple of 4: a lane's units are all in or all out
    // SwiGLU of every value first (independent chains for the VALU to
    // overlap), then the stores of the valid rows
    uint32_t w[MI][4][2];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const float g0 = acc[mi][4 * u][i], u0 = acc[mi][4 * u + 1][i];
          const float g1 = acc[mi][4 * u + 2][i], u1 = acc[mi][4 * u + 3][i];
          w[mi][i][u] = pk_bf16(g0 * __builtin_amdgcn_rcpf(1.0f + __expf(-g0)) * u0,
                                g1 * __builtin_amdgcn_rcpf(1.0f + __expf(-g1)) * u1);
        }
    bf16 *out = Hm + int64_t(t.p0) * dff + f;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * MI * 16 + mi * 16 + 4 * (lane >> 4) + i;
        if (r < t.mvalid) *(uint2 *)(out + r * dff) = make_uint2(w[mi][i][0], w[mi][i][1]);
      }
  }
  // item = 8 expert units of one assignment row (C holds silu(g) u)
  template <int BM, int NC, int LDC, int NT>
  __device__ void epilogue(const MTile &t, const float *C, int tid) const {
    constexpr int CC = NC / 8;
    for (int it = tid; it < BM * CC; it += NT) {
      const int r = it / CC, c8 = (it % CC) * 8;
      if (r >= t.mvalid || t.n0 + c8 >= dff) continue;
      *(u32x4_t *)(Hm + int64_t(t.p0 + r) * dff + t.n0 + c8) = pack8_bf16(C + r * LDC + c8);
    }
  }
};

struct Moe2M {
  static constexpr bool DIRECT_W4 = true;
  static constexpr int EPI = EPI_PLAIN;
  const bf16 *Hm, *Wd;
  float *Y;  // rows in list order
  const int32_t *cnt;
  int E, d, dff;
  int ksplit = 1;        // K halves (few-token path), each to its own plane of Y
  int64_t yplane = 0;    // elements between planes
  static constexpr int out_cols(int BN) { return BN; }
  static constexpr bool GROUPED = true;
  __device__ int tiles(int BM, int ny, const GroupScan &gs) const { return gs.total * ny; }
  __device__ bool map(int bx, int by, int BM, int BN, MTile &t, const GroupScan &gs) const {
    if (!mmap_grouped(bx, BM, gs, t)) return false;
    const int ncol = (d + BN - 1) / BN, kh = by / ncol;
    t.n0 = (by - kh * ncol) * BN;
    t.k0 = kh * (dff / ksplit);
    t.yp = kh;
    return true;
  }
  __device__ const bf16 *a_base() const { return Hm; }
  __device__ const bf16 *b_base() const { return Wd; }
  __device__ const bf16 *a_row(const MTile &t, int r) const {
    return Hm + int64_t(t.p0 + r) * dff + t.k0;
  }
  __device__ const bf16 *b_row(const MTile &t, int n) const {
    return t.n0 + n < d ? Wd + (int64_t(t.e - 1) * d + t.n0 + n) * dff + t.k0 : nullptr;
  }
  // Four-wave kernel: in wave column wn, MFMA block ni, lane column c
  // holds output feature NI (16 wn + c) + ni of the tile, so each lane ends
  // with NI consecutive features of each of its rows.
  template <int NI>
  __device__ uint32_t b_off_w4(const MTile &t, int wn, int ni, int c) const {
    const int f = t.n0 + NI * (16 * wn + c) + ni;
    return f < d ? uint32_t((t.e - 1) * d + f) * uint32_t(2 * dff) : 0u;
  }
  __device__ uint32_t a_off(const MTile &t, int r) const { return uint32_t(t.p0 + r) * uint32_t(2 * dff); }
  template <int MI, int NI>
  __device__ void store_w4(const MTile &t, const f32x4_t (&acc)[MI][NI], int wm, int wn, int lane) const {
    static_assert(NI % 2 == 0, "whole 8-byte pieces");
    const int f = t.n0 + NI * (16 * wn + (lane & 15));
    if (f >= d) return;  // d is a multiple of NI: a lane's features are all in or all out
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * MI * 16 + mi * 16 + 4 * (lane >> 4) + i;
        if (r >= t.mvalid) continue;
        float *y = Y + int64_t(t.p0 + r) * d + f;
#pragma unroll
        for (int ni = 0; ni < NI; ni += 2) *(float2 *)(y + ni) = make_float2(acc[mi][ni][i], acc[mi][ni + 1][i]);
      }
  }
  // item = 8 output features of one list row
  template <int BM, int NC, int LDC, int NT>
  __device__ void epilogue(const MTile &t, const float *C, int tid) const {
    constexpr int CC = NC / 8;
    for (int it = tid; it < BM * CC; it += NT) {
      const int r = it / CC, c8 = (it % CC) * 8;
      if (r >= t.mvalid || t.n0 + c8 >= d) continue;
      float *y = Y + t.yp * yplane + int64_t(t.p0 + r) * d + t.n0 + c8;
      const float *c = C + r * LDC + c8;
      *(float4 *)y = make_float4(c[0], c[1], c[2], c[3]);
      *(float4 *)(y + 4) = make_float4(c[4], c[5], c[6], c[7]);
    }
  }
};

// ------------------------------------------------------------------ kernel
// Tiles of the whole problem are handed out XCD by XCD: blocks are issued to
// the 8 XCDs round-robin, so block L runs on XCD L % 8, and it takes tile
// number (its XCD's contiguous share) + L / 8.  Tile t covers row tile t / ny
// and column tile t % ny, so the blocks resident on one XCD share A rows and
// a few weight tiles in that XCD's L2.
__device__ __forceinline__ int xcd_tile(int L, int total) {
  const int per = total >> 3, extra = total & 7, x = L & 7;
  return x * per + min(x, extra) + (L >> 3);
}

// Order of the tiles handed to one XCD.  The 32 CUs of an XCD run 32
// consecutive tiles of its share at a time and stream their K loops in near
// lockstep, so what that XCD's L2 must hold per K step is the union of their
// operand slices.  Walking the tiles in bands of BAND_R row tiles (of one
// expert, for grouped problems), each band in chunks of BAND_R x BAND_C
// tiles with the row fastest, makes that union BAND_R A slices and BAND_C B
// slices instead of one A slice and 32 B slices (the expert weights would
// otherwise stream past the L2 once per row tile).
constexpr int BAND_R = 16, BAND_C = 2;

// Tile t of a rows x ny grid walked in bands -> (row tile i, column tile j).
__device__ __forceinline__ void band_order(int t, int rows, int ny, int &i, int &j) {
  const int band = t / (BAND_R * ny);
  const int rem = t - band * BAND_R * ny;
  const int rb = min(BAND_R, rows - band * BAND_R);  // rows of this band
  const int chunk = rem / (rb * BAND_C);
  const int idx = rem - chunk * rb * BAND_C;
  i = band * BAND_R + idx % rb;
  j = chunk * BAND_C + idx / rb;
}

// The same within each expert of a grouped problem: tile t lies in the
// first expert whose tiles (row tiles x ny, in expert order) reach past it.
__device__ __forceinline__ void grouped_band_order(int t, int ny, const GroupScan &gs, int &bx,
                                                   int &by) {
  const uint64_t m = __ballot(gs.incl * ny > t);
  const int l = __ffsll((unsigned long long)m) - 1;
  const int nt = __shfl(gs.nt, l, 64), first = __shfl(gs.incl, l, 64) - nt;
  int i;
  band_order(t - first * ny, nt, ny, i, by);
  bx = first + i;
}

// LDS chunk (16 bytes) of chunk c of operand row r in a stage whose rows are
// CPR chunks long: a XOR with the row's position in its 256-byte bank span
// makes the 16 rows read by one 16-lane phase (same c) hit 16 distinct
// 16-byte bank groups.
template <int CPR>
__device__ __forceinline__ int swz(int r, int c) {
  if constexpr (CPR == 8)
    return c ^ ((r >> 1) & 7);  // 2 rows per 256-byte span
  else
    return c ^ ((r >> 2) & 3);  // 4 rows per span
}

// vmcnt(n * N) for the run-time n of stages still allowed in flight, n < S - 1
template <int N, int S>
__device__ __forceinline__ void wait_stages(int n) {
  if constexpr (S > 5) if (n >= 4) { wait_vm<4 * N>(); return; }
  if constexpr (S > 4) if (n == 3) { wait_vm<3 * N>(); return; }
  if constexpr (S > 3) if (n == 2) { wait_vm<2 * N>(); return; }
  if constexpr (S > 2) if (n == 1) { wait_vm<N>(); return; }
  wait_vm<0>();
}

// Epilogue register pass: lane holds rows 4 (lane/16) + i of each 16-row tile
// and column (lane % 16) of each 16-column block; in each 64-column slice the
// partner columns (ni, ni + 2) are combined for SwiGLU and kept apart for
// RoPE.  The problem's row-wise pass then reads the staged fp32 tile C.
template <class P, int MI, int NI, int TM, int TN, int LDC>
__device__ __forceinline__ void store_acc(const P &p, float *C, const f32x4_t (&acc)[MI][NI],
                                          int wm, int wn, int lane) {
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = wm * TM + mi * 16 + 4 * (lane >> 4) + i;
      if constexpr (P::EPI == EPI_PLAIN) {
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          C[r * LDC + wn * TN + ni * 16 + (lane & 15)] = acc[mi][ni][i];
      } else {
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
          if ((ni & 3) >= 2) continue;
          int Pp, half;
          col_pair(wn * TN + ni * 16 + (lane & 15), Pp, half);
          const float g = acc[mi][ni][i], u = acc[mi][ni + 2][i];
          if constexpr (P::EPI == EPI_SWIGLU) {
            C[r * LDC + Pp] = g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
          } else {
            C[r * LDC + p.ccol(Pp, 0)] = g;
            C[r * LDC + p.ccol(Pp, 1)] = u;
          }
        }
      }
    }
}

template <class P, int BM, int BN, int WM, int WN, int BK, int S>
__global__ __launch_bounds__(64 * WM * WN, 1) void gemm_mfma_kernel(P p, int K, int ny) {
  constexpr int NW = WM * WN, NT = 64 * NW;  // waves, threads
  constexpr int TM = BM / WM, TN = BN / WN;  // wave tile
  constexpr int MI = TM / 16, NI = TN / 16;  // 16 x 16 MFMA tiles per wave
  constexpr int RB = BK * 2;                 // bytes per operand row per K step
  constexpr int CPR = RB / 16;               // 16-byte chunks per row
  constexpr int RPT = 1024 / RB;             // rows per 1 KB transfer
  constexpr int STAGE = (BM + BN) * RB;
  constexpr int IPW = STAGE / 1024 / NW;     // 1 KB transfers per wave per stage
  static_assert(STAGE % (1024 * NW) == 0 && TN % 64 == 0, "whole transfers, 64-column slices");
  static_assert(S >= 2 && S <= 6 && (BK == 32 || BK == 64), "pipeline shape");
  constexpr int NC = P::out_cols(BN), LDC = NC + 16;  // staged output tile (fp32)
  constexpr int SMEM = S * STAGE > BM * LDC * 4 ? S * STAGE : BM * LDC * 4;
  __shared__ __align__(1024) uint8_t smem[SMEM];
  GroupScan gs;
  if constexpr (P::GROUPED) gs = group_scan(BM, p.cnt, p.E);
  const int total = p.tiles(BM, ny, gs);
  if (int(blockIdx.x) >= total) return;
  const int t = xcd_tile(blockIdx.x, total);
  MTile tc;
  if (!p.map(t / ny, t % ny, BM, BN, tc, gs)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  // Transfer j of this wave fills stage rows RPT g .. RPT g + RPT - 1
  // (g = wave IPW + j; A rows first, then B rows).  Lane l writes LDS chunk
  // l % CPR of row RPT g + l / CPR, which holds the source chunk that swz
  // maps there.  Rows past the valid rows (or past the weight's columns)
  // read a valid row instead: their products land in accumulator rows /
  // columns the epilogue never stores.
  const uint8_t *src[IPW];
  const bf16 *b_fallback = p.b_row(tc, 0);
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int rr = RPT * (wave * IPW + j) + lane / CPR;
    const int c = swz<CPR>(rr, lane % CPR);  // swz is an involution in c
    const bf16 *row;
    if (rr < BM) {
      row = p.a_row(tc, rr < tc.mvalid ? rr : 0);
    } else {
      row = p.b_row(tc, rr - BM);
      if (!row) row = b_fallback;
    }
    src[j] = (const uint8_t *)row + c * 16;
  }
  const uint32_t sbase = lds_addr(smem) + wave * IPW * 1024;
  auto issue = [&](int kt, int stage) {
#pragma unroll
    for (int j = 0; j < IPW; ++j) dma16(src[j] + kt * RB, sbase + stage * STAGE + j * 1024);
  };
  f32x4_t acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int nk = K / BK;
#pragma unroll
  for (int s0 = 0; s0 < S - 1; ++s0)
    if (s0 < nk) issue(s0, s0);
  for (int kt = 0; kt < nk; ++kt) {
    // stage kt has landed once at most the later stages' transfers are out
    wait_stages<IPW, S>(min(S - 2, nk - 1 - kt));
    __syncthreads();  // every wave's part of stage kt is in; stage kt-1 is free
    if (kt + S - 1 < nk) issue(kt + S - 1, (kt + S - 1) % S);
    const uint8_t *As = smem + (kt % S) * STAGE;
    const uint8_t *Bs = As + BM * RB;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      const int ch = ks * 4 + (lane >> 4);
      bf16x8_t b[NI];
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) {
        const int n = wn * TN + ni * 16 + (lane & 15);
        b[ni] = *(const bf16x8_t *)(Bs + n * RB + (swz<CPR>(n, ch) << 4));
      }
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) {
        const int r = wm * TM + mi * 16 + (lane & 15);
        const bf16x8_t a = *(const bf16x8_t *)(As + r * RB + (swz<CPR>(r, ch) << 4));
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[ni], acc[mi][ni], 0, 0, 0);
      }
    }
  }
  __syncthreads();  // every wave is done with the operand stages
  float *C = (float *)smem;
  store_acc<P, MI, NI, TM, TN, LDC>(p, C, acc, wm, wn, lane);
  __syncthreads();
  p.template epilogue<BM, NC, LDC, NT>(tc, C, tid);
}

// ------------------------------------------------------- four-wave kernel
// One wave per SIMD, each wave a (BM/2) x (BN/2) sub-tile: every operand byte
// read from LDS feeds twice the MFMAs of the eight-wave kernel above (per K
// step and CU, 128 KB of fragment reads against 256 MFMAs per SIMD).  With
// no second wave on its SIMD to switch to, a wave hides LDS latency itself:
// the fragments of the next 32-wide K slice are read into a second register
// set while the current slice's MFMAs issue, the reads slotted between the
// MFMAs.  Stages are double-buffered (BK = 64); stage kt + 2 goes into the
// buffer of stage kt as soon as every wave has read it (schedule below).
// acc += a b on the accumulator registers (AGPRs).  With 256 accumulators
// per lane the register allocator, left to itself, parks some of them in
// VGPRs and copies them around every MFMA; pinning them to AGPRs keeps the
// loop free of copies.  As a volatile asm statement it also keeps its place
// relative to the LDS reads and transfers written around it, so the program
// order below is the issue order.
__device__ __forceinline__ void mfma_agpr(f32x4_t &acc, const bf16x8_t &a, const bf16x8_t &b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// acc = a b (the first product of a tile: no zeroing of the accumulators)
__device__ __forceinline__ void mfma_agpr_first(f32x4_t &acc, const bf16x8_t &a, const bf16x8_t &b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=a"(acc) : "v"(a), "v"(b));
}

// The compiler does not see the MFMAs inside the asm statements, so it does
// not keep its own accesses of the accumulators clear of their hazards.
// Each row of accumulators passes through an asm statement that starts with
// `nops` wait states: accesses after it are ordered after the wait, and
// writes before it (zeroing) before the wait.
template <int NI>
__device__ __forceinline__ void acc_fence_row(f32x4_t (&a)[NI]) {
  static_assert(NI == 4 || NI == 6 || NI == 8, "accumulator row widths in use");
  if constexpr (NI == 4)
    asm volatile("s_nop 4" : "+a"(a[0]), "+a"(a[1]), "+a"(a[2]), "+a"(a[3]));
  else if constexpr (NI == 8)
    asm volatile("s_nop 4" : "+a"(a[0]), "+a"(a[1]), "+a"(a[2]), "+a"(a[3]), "+a"(a[4]), "+a"(a[5]),
                 "+a"(a[6]), "+a"(a[7]));
  else
    asm volatile("s_nop 4" : "+a"(a[0]), "+a"(a[1]), "+a"(a[2]), "+a"(a[3]), "+a"(a[4]), "+a"(a[5]));
}

template <class P, int BM, int BN>
__global__ __launch_bounds__(256, 1) void gemm_w4_kernel(P p, int K, int ny) {
  constexpr int NW = 4, NT = 256, WN = 2;
  constexpr int TM = BM / 2, TN = BN / 2;    // wave tile
  constexpr int MI = TM / 16, NI = TN / 16;  // 16 x 16 MFMA tiles per wave
  constexpr int BK = 64, RB = 128, CPR = 8, RPT = 8;
  constexpr int STAGE = (BM + BN) * RB;
  constexpr int IPW = STAGE / 1024 / NW;  // 1 KB transfers per wave per stage
  constexpr int NF = MI + NI;             // fragment reads per K slice
  constexpr int NM = MI * NI;             // MFMAs per K slice
  static_assert(STAGE % (1024 * NW) == 0 && (TN % 64 == 0 || P::DIRECT_W4), "whole transfers, 64-column slices");
  // K step schedule, two barriers: the first, after MFMA B1J of slice 0
  // (every wave's reads of set 1, the last reads of stage kt, are in), frees
  // the buffer of stage kt; the transfers of stage kt + 2 go out one every GAP
  // MFMAs from there until MFMA RS of slice 1, where the second barrier
  // publishes stage kt + 1 (at most this step's IPW transfers still out) for
  // the reads of set 0.  A transfer thus has from slice 0 of step kt to
  // slice 1 of step kt + 1 to land.  (One barrier 16 MFMAs into slice 1, with
  // the transfers after it, left the last ones under 90 MFMAs to land, and a
  // cache-missing transfer stalled the wave at that barrier; spacing the
  // transfers closer than 5 MFMAs slowed the MFMA issue.)
  constexpr int RS = NM - NF < 48 ? NM - NF : 48;
  constexpr int B1J = NF + 4;
  constexpr int NSLOT = (NM - 1 - B1J) + RS;  // slice 0 after B1J, then slice 1 before RS
  constexpr int GAP = NSLOT / IPW < 5 ? NSLOT / IPW : 5;
  static_assert(B1J < NM && RS >= 16 && RS + NF <= NM && GAP >= 1 && GAP * (IPW - 1) < NSLOT,
                "room for the reads and transfers");
  static_assert(P::DIRECT_W4, "results are written from the accumulators");
  __shared__ __align__(1024) uint8_t smem[2 * STAGE];
  // Persistent: block b takes tiles b, b + gridDim.x, ... (one block per CU).
  // The operand stream runs on across tiles: the last two K steps of a tile
  // fetch the first two stages of the block's next tile, so its transfers
  // are in flight while this one's results are written.
  GroupScan gs;
  if constexpr (P::GROUPED) gs = group_scan(BM, p.cnt, p.E);
  const int total = __builtin_amdgcn_readfirstlane(p.tiles(BM, ny, gs));
  int L = blockIdx.x;
  if (L >= total) return;
  auto tile = [&](int l) {  // a tile's fields are wave-uniform: kept in SGPRs
    MTile t;
    const int x = xcd_tile(l, total);
    int bx, by;
    if constexpr (P::GROUPED)
      grouped_band_order(x, ny, gs, bx, by);
    else
      band_order(x, total / ny, ny, bx, by);
    p.map(bx, by, BM, BN, t, gs);  // every index below total maps to a tile
    t.m0 = __builtin_amdgcn_readfirstlane(t.m0);
    t.n0 = __builtin_amdgcn_readfirstlane(t.n0);
    t.mvalid = __builtin_amdgcn_readfirstlane(t.mvalid);
    t.e = __builtin_amdgcn_readfirstlane(t.e);
    t.p0 = __builtin_amdgcn_readfirstlane(t.p0);
    return t;
  };
  MTile tc = tile(L);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, in SGPRs
  const int wm = wave / WN, wn = wave % WN;
  // Transfer j of this wave fills stage rows RPT (wave IPW + j) .. + RPT - 1
  // as in the eight-wave kernel.  A transfer's rows are all A rows or all B
  // rows (RPT divides BM), so each lane keeps one 32-bit byte offset per
  // transfer from that operand's base (the host checks that every operand
  // row lies within 4 GB of it); the base moves on by 128 B per K step.
  // Rows past the valid ones read a valid row instead: their products land
  // in accumulators that are never stored.
  static_assert(BM % RPT == 0, "a transfer stays within one operand");
  auto is_a = [&](int j) { return RPT * (wave * IPW + j) < BM; };  // wave-uniform
  auto gbase = [&](int j) { return (const uint8_t *)(is_a(j) ? p.a_base() : p.b_base()); };
  // (lane-derived terms of the per-tile address arithmetic start from an
  // opaque copy of the lane: hoisted out of the tile loop they would hold
  // registers through the K loop)
  auto pinned_lane = [&]() {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    return ln;
  };
  auto offsets = [&](const MTile &t, uint32_t(&o)[IPW]) {
    const int ln = pinned_lane();
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int rr = RPT * (wave * IPW + j) + ln / CPR;
      const uint32_t c16 = swz<CPR>(rr, ln % CPR) * 16;
      if (is_a(j))
        o[j] = p.a_off(t, rr < t.mvalid ? rr : 0) + c16;
      else
        o[j] = p.template b_off_w4<NI>(t, (rr - BM) / TN, ((rr - BM) % TN) >> 4, (rr - BM) & 15) + c16;
    }
  };
  uint32_t voff[IPW], vnx[IPW];
  offsets(tc, voff);
  const uint32_t sbase = lds_addr(smem) + wave * IPW * 1024;
  // Fragment addresses: row r = (wave row) + 16 i + lane % 16 reads chunk
  // (4 ks + lane / 16) ^ ((r >> 1) & 7); the XOR term depends on the lane only.
  const int l15 = lane & 15, x7 = (lane >> 1) & 7;
  const uint8_t *fa0 = smem + (wm * TM + l15) * RB;
  const uint8_t *fb0 = smem + BM * RB + (wn * TN + l15) * RB;
  int coff[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) coff[ks] = (((ks * 4 + (lane >> 4)) ^ x7) << 4);

  bf16x8_t fa[2][MI], fb[2][NI];
  // piece q of slice ks in buffer buf: q = 0 is A0, 1..NI the B pieces, then A1..
  auto read_piece = [&](int set, int buf, int q) {
    if (q == 0) {
      fa[set][0] = *(const bf16x8_t *)(fa0 + buf * STAGE + coff[set]);
    } else if (q <= NI) {
      fb[set][q - 1] = *(const bf16x8_t *)(fb0 + buf * STAGE + (q - 1) * 16 * RB + coff[set]);
    } else {
      const int mi = q - NI;
      fa[set][mi] = *(const bf16x8_t *)(fa0 + buf * STAGE + mi * 16 * RB + coff[set]);
    }
  };
  f32x4_t acc[MI][NI];
  auto mma = [&](int set, int j) {
    mfma_agpr(acc[j / NI][j % NI], fa[set][j / NI], fb[set][j % NI]);
  };
  auto mma_first = [&](int set, int j) {
    mfma_agpr_first(acc[j / NI][j % NI], fa[set][j / NI], fb[set][j % NI]);
  };

  const int nk = K / BK;  // >= 2 (host)
#pragma unroll
  for (int j = 0; j < IPW; ++j) dma16_s(gbase(j), voff[j], sbase + j * 1024);
#pragma unroll
  for (int j = 0; j < IPW; ++j) dma16_s(gbase(j) + RB, voff[j], sbase + STAGE + j * 1024);
  // the next tile's offsets while stage 0 lands (needed from step nk - 2 on)
  int Ln = L + int(gridDim.x);
  MTile tn = tc;
  if (Ln < total) {
    tn = tile(Ln);
    offsets(tn, vnx);
  }
  wait_vm<IPW>();
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NF; ++q) read_piece(0, 0, q);

  int ph = 0;  // buffer of the tile's stage 0
  for (;;) {
    const bool more = Ln < total;
    // one K step; in the tile's first (FIRST) the slice-0 products start the
    // accumulators
    auto kstep = [&](int kt, auto first) {
      constexpr bool FIRST = decltype(first)::value;
      const int buf = (kt + ph) & 1;
      // stage kt + 2: of this tile, else the next tile's stage kt + 2 - nk,
      // else (the block's last tile) this tile's last stage again, unused
      const bool nxt = kt + 2 >= nk && more;
      const int kn = kt + 2 < nk ? kt + 2 : more ? kt + 2 - nk : nk - 1;
      auto dma_slot = [&](int pos) {  // transfer pos / GAP at slot pos
        if (pos >= 0 && pos % GAP == 0 && pos / GAP < IPW) {
          const int j = pos / GAP;
          dma16_s(gbase(j) + kn * RB, nxt ? vnx[j] : voff[j], sbase + buf * STAGE + j * 1024);
        }
      };
      // slice 0: MFMAs on set 0, the reads of slice 1 into set 1 after the
      // first NF of them, the first barrier after MFMA B1J
#pragma unroll
      for (int j = 0; j < NM; ++j) {
        if constexpr (FIRST)
          mma_first(0, j);
        else
          mma(0, j);
        if (j < NF) read_piece(1, buf, j);
        if (j == B1J) __syncthreads();  // every wave's reads of stage kt are in
        if (j > B1J) dma_slot(j - B1J - 1);
      }
      // slice 1: MFMAs on set 1, the barrier, then the reads of stage
      // kt + 1, slice 0, into set 0 (unused in the last step: the registers
      // are free while the results are written, and read again after)
#pragma unroll
      for (int j = 0; j < NM; ++j) {
        if (j == RS) {
          // stage kt + 1 has landed: loads complete in issue order and only
          // stage kt + 2 may be out (stores in between do not matter)
          wait_vm<IPW>();
          __syncthreads();  // ... in every wave's part
        }
        mma(1, j);
        if (j < RS) dma_slot(NM - 1 - B1J + j);
        if (j >= RS && j - RS < NF) read_piece(0, buf ^ 1, j - RS);
      }
    };
    kstep(0, std::true_type{});
    for (int kt = 1; kt < nk; ++kt) kstep(kt, std::false_type{});
    // the last MFMAs' results are read below: let them drain first
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
    for (int i = 0; i < MI; ++i) acc_fence_row<NI>(acc[i]);
    p.store_w4(tc, acc, wm, wn, pinned_lane());
    if (!more) break;
    ph ^= nk & 1;
    // the next tile's stage 0 is in buffer ph (published by the last step's barrier)
#pragma unroll
    for (int q = 0; q < NF; ++q) read_piece(0, ph, q);
    L = Ln;
    tc = tn;
#pragma unroll
    for (int j = 0; j < IPW; ++j) voff[j] = vnx[j];
    Ln = L + int(gridDim.x);
    if (Ln < total) {
      tn = tile(Ln);
      offsets(tn, vnx);
    }
  }
}

// ------------------------------------------------------------------ launchers
// m_tiles bounds the row tiles (for grouped problems: the most any routing
// can need); the kernel takes the actual count from the problem.
template <class P, int BM, int BN, int WM, int WN, int BK, int S>
static hipError_t launch(const P &p, int K, int m_tiles, int n_tiles, hipStream_t st) {
  if (m_tiles > 0 && n_tiles > 0)
    gemm_mfma_kernel<P, BM, BN, WM, WN, BK, S>
        <<<m_tiles * n_tiles, 64 * WM * WN, 0, st>>>(p, K, n_tiles);
  return hipGetLastError();
}

// CUs of the current device (the tile-shape choice counts rounds of them).
static int cu_count() {
  static int n = 0;
  if (n == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      n = v;
    else
      n = 256;
  }
  return n;
}

// One block per CU at most (a block holds 128 KB of LDS), each walking its
// share of the tiles.
template <class P, int BM, int BN>
static hipError_t launch_w4(const P &p, int K, int m_tiles, int n_tiles, hipStream_t st) {
  const int cu = cu_count();
  if (m_tiles > 0 && n_tiles > 0)
    gemm_w4_kernel<P, BM, BN><<<std::min(m_tiles * n_tiles, cu), 256, 0, st>>>(p, K, n_tiles);
  return hipGetLastError();
}

// The four-wave kernel addresses operand rows by 32-bit byte offsets from the
// lowest of an operand's matrices: *lo gets that pointer, and the result says
// whether every matrix ends within 4 GB of it.
struct Span {
  const void *p;
  size_t bytes;
};
static bool span32(std::initializer_list<Span> ms, const bf16 **lo) {
  uintptr_t a = UINTPTR_MAX, b = 0;
  for (const Span &m : ms) {
    a = std::min(a, uintptr_t(m.p));
    b = std::max(b, uintptr_t(m.p) + m.bytes);
  }
  *lo = (const bf16 *)a;
  return b - a < (uintptr_t(1) << 32);
}

hipError_t mfma_qkv(const triroute_cfg &cfg, int B, int Tq, const void *n1,
                    const triroute_dense_w &w, const float *rope, void *q, void *k, void *v,
                    hipStream_t st) {
  QkvM p;
  p.n1 = (const bf16 *)n1;
  p.Wq = (const bf16 *)w.Wq;
  p.Wk = (const bf16 *)w.Wk;
  p.Wv = (const bf16 *)w.Wv;
  p.Wlo = std::min(p.Wq, std::min(p.Wk, p.Wv));
  p.q = (bf16 *)q;
  p.k = (bf16 *)k;
  p.v = (bf16 *)v;
  p.rope = (const float2 *)rope;
  p.N = B * Tq;
  p.d = cfg.d_model;
  p.H = cfg.n_heads;
  p.Hkv = cfg.n_kv_heads;
  p.dh = cfg.head_dim;
  p.Ncols = (cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim;
  // Few tokens (decode): the product streams the weights; 32-row tiles one
  // head wide put one block on every head and row tile.
  if (p.N <= 2048) {
    if (p.dh == 64)
      return launch<QkvM, 32, 64, 2, 1, 64, 4>(p, cfg.d_model, (p.N + 31) / 32, (p.Ncols + 63) / 64, st);
    if (p.dh == 128)
      return launch<QkvM, 32, 128, 2, 2, 64, 4>(p, cfg.d_model, (p.N + 31) / 32, (p.Ncols + 127) / 128, st);
  }
  const bf16 *lo;
  const bool w4 = (p.dh == 64 || p.dh == 128) && p.Ncols % 128 == 0 && p.d >= 128 &&
                  span32({{p.Wq, size_t(p.H) * p.dh * p.d * sizeof(bf16)},
                          {p.Wk, size_t(p.Hkv) * p.dh * p.d * sizeof(bf16)},
                          {p.Wv, size_t(p.Hkv) * p.dh * p.d * sizeof(bf16)}}, &lo) &&
                  span32({{p.n1, size_t(p.N) * p.d * sizeof(bf16)}}, &lo);
  if (w4) {
    const uint32_t pitch = 2u * uint32_t(p.d);
    p.Hd = p.H * p.dh;
    p.HKd = p.Hd + p.Hkv * p.dh;
    p.wq_o = uint32_t((const uint8_t *)p.Wq - (const uint8_t *)p.Wlo);
    p.wk_o = uint32_t((const uint8_t *)p.Wk - (const uint8_t *)p.Wlo) - uint32_t(p.Hd) * pitch;
    p.wv_o = uint32_t((const uint8_t *)p.Wv - (const uint8_t *)p.Wlo) - uint32_t(p.HKd) * pitch;
    // d_h 128: one head per wave column on 256-column tiles (long K steps,
    // one barrier each), where the columns divide into them
    if (p.dh == 128 && p.Ncols % 256 == 0)
      return launch_w4<QkvM, 256, 256>(p, cfg.d_model, (p.N + 255) / 256, p.Ncols / 256, st);
    return launch_w4<QkvM, 256, 128>(p, cfg.d_model, (p.N + 255) / 256, p.Ncols / 128, st);
  }
  return launch<QkvM, 256, 128, 4, 2, 64, 3>(p, cfg.d_model, (p.N + 255) / 256, (p.Ncols + 127) / 128, st);
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
  const bf16 *lo;
  if (N <= 2048)  // few tokens: weight streaming, narrow tiles as for QKV
    return launch<OprojM, 32, 64, 2, 1, 64, 4>(p, p.K, (N + 31) / 32, (p.d + 63) / 64, st);
  const bool w4 = p.K >= 128 && span32({{p.o, size_t(N) * p.K * sizeof(bf16)}}, &lo) &&
                  span32({{p.Wo, size_t(p.d) * p.K * sizeof(bf16)}}, &lo);
  if (w4) {  // 192- or 256-wide tiles: whichever fills the CUs in fewer rounds of shorter steps
    const int mt = (N + 255) / 256, cu = cu_count();
    const int r192 = p.d % 192 == 0 ? (mt * (p.d / 192) + cu - 1) / cu : 0;
    const int r256 = p.d % 256 == 0 ? (mt * (p.d / 256) + cu - 1) / cu : 0;
    if (r192 > 0 && (r256 == 0 || 3 * r192 <= 4 * r256))
      return launch_w4<OprojM, 256, 192>(p, p.K, mt, p.d / 192, st);
    if (r256 > 0) return launch_w4<OprojM, 256, 256>(p, p.K, mt, p.d / 256, st);
  }
  return launch<OprojM, 256, 128, 4, 2, 64, 3>(p, p.K, (N + 255) / 256, (p.d + 127) / 128, st);
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
  p1.E = E;
  p1.d = d;
  p1.dff = dff;
  const size_t wb = size_t(E) * dff * d * sizeof(bf16);
  const bf16 *alo;
  // Few assignments (decode): each expert's rows fit a 32-row tile and the
  // work is streaming the expert weights, so narrow 32 x 64 tiles (two
  // waves, four stages) put every CU on its own slice of the weights.
  const bool small = Nk <= 2048;
  const bool w4 = span32({{p1.Wg, wb}, {p1.Wu, wb}}, &p1.Wlo) &&
                  span32({{p1.n2, size_t(Nk) * d * sizeof(bf16)}}, &alo);
  hipError_t err =
      small ? launch<Moe1M, 32, 64, 2, 1, 64, 4>(p1, d, Nk / 32 + E, (dff + 31) / 32, st)
      : w4 && d >= 128 ? launch_w4<Moe1M, 256, 256>(p1, d, Nk / 256 + E, (dff + 127) / 128, st)
            : launch<Moe1M, 256, 256, 2, 4, 64, 2>(p1, d, Nk / 256 + E, (dff + 127) / 128, st);
  if (err != hipSuccess) return err;
  Moe2M p2;
  p2.Hm = (const bf16 *)Hm;
  p2.Wd = (const bf16 *)w.Wdown;
  p2.Y = Y;
  p2.cnt = c.exp_cnt;
  p2.E = E;
  p2.d = d;
  p2.dff = dff;
  if (small) {
    p2.ksplit = moe_ysplit(cfg, N);
    p2.yplane = int64_t(Nk) * d;
    return launch<Moe2M, 32, 64, 2, 1, 64, 4>(p2, dff / p2.ksplit, Nk / 32 + E,
                                              (d + 63) / 64 * p2.ksplit, st);
  }
  const bool w4b = dff >= 128 && (d % 192 == 0 || d % 256 == 0) && span32({{p2.Wd, wb}}, &alo) &&
                   span32({{p2.Hm, size_t(Nk) * dff * sizeof(bf16)}}, &alo);
  if (w4b) {  // 192-wide tiles where they divide d (measured faster), else 256
    const int mt = Nk / 256 + E;
    if (d % 192 == 0) return launch_w4<Moe2M, 256, 192>(p2, dff, mt, d / 192, st);
    return launch_w4<Moe2M, 256, 256>(p2, dff, mt, d / 256, st);
  }
  return launch<Moe2M, 256, 128, 4, 2, 64, 3>(p2, dff, Nk / 256 + E, (d + 127) / 128, st);
}

}  // namespace tr
