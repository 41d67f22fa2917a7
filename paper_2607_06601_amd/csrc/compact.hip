// Token compaction by routing decision: deterministic stable partitions by
// prefix sums (no atomics decide any order).
//
//   attention: per (b, h), the ascending t of local and of full queries
//   experts  : per expert 1..E, the ascending assignment ids a = i*k + slot
#include "kernels.hpp"

namespace tr {

constexpr int CHUNK = 1024;  // assignments per expert block

// Blocks [0, B*H): attention lists of one (b, h).  Blocks [B*H, +nbe):
// per-block expert histograms.
__global__ __launch_bounds__(256) void compact_count_kernel(
    const uint8_t *__restrict__ mode, const int32_t *__restrict__ eidx, int B, int T, int H,
    int E1, int Nk, int32_t *__restrict__ attn_cnt, int32_t *__restrict__ attn_idx,
    int32_t *__restrict__ hist) {
  __shared__ int wcnt[2][4];
  __shared__ int lh[64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int bid = blockIdx.x;
  if (bid < B * H) {
    const int b = bid / H, h = bid % H;
    int base[2] = {0, 0};
    for (int t0 = 0; t0 < T; t0 += 256) {
      const int t = t0 + tid;
      const int m = t < T ? mode[(int64_t(b) * T + t) * H + h] : 0;
      uint64_t bal[2];
      bal[0] = __ballot(m == 1);
      bal[1] = __ballot(m == 2);
      if (lane == 0) {
        wcnt[0][w] = __popcll(bal[0]);
        wcnt[1][w] = __popcll(bal[1]);
      }
      __syncthreads();
#pragma unroll
      for (int mm = 0; mm < 2; ++mm) {
        if (m == mm + 1) {
          int off = base[mm] + __popcll(bal[mm] & lanemask_lt());
          for (int ww = 0; ww < w; ++ww) off += wcnt[mm][ww];
          attn_idx[(int64_t(bid) * 2 + mm) * T + off] = t;
        }
      }
#pragma unroll
      for (int mm = 0; mm < 2; ++mm)
        base[mm] += wcnt[mm][0] + wcnt[mm][1] + wcnt[mm][2] + wcnt[mm][3];
      __syncthreads();
    }
    if (tid < 2) attn_cnt[bid * 2 + tid] = base[tid];
    return;
  }
  const int j = bid - B * H;
  for (int e = tid; e < E1; e += 256) lh[e] = 0;
  __syncthreads();
  for (int a = j * CHUNK + tid; a < min(Nk, (j + 1) * CHUNK); a += 256) atomicAdd(&lh[eidx[a]], 1);
  __syncthreads();
  for (int e = tid; e < E1; e += 256) hist[j * E1 + e] = lh[e];
}

// Stable scatter of assignment ids into per-expert lists.  Block j first
// forms each expert's first output position for its chunk from the chunk
// histograms (all chunks' totals give the expert offsets; block 0 also
// writes the counts and offsets).
__global__ __launch_bounds__(256) void compact_scatter_kernel(const int32_t *__restrict__ eidx,
                                                              const int32_t *__restrict__ hist,
                                                              int nbe, int E1, int Nk,
                                                              int32_t *__restrict__ rows,
                                                              int32_t *__restrict__ exp_cnt,
                                                              int32_t *__restrict__ exp_off) {
  __shared__ int wc[4][64];
  __shared__ int run[64], tot[64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int j = blockIdx.x;
  if (tid < E1) {
    int before = 0, all = 0;
    for (int jj = 0; jj < nbe; ++jj) {
      const int v = hist[jj * E1 + tid];
      if (jj < j) before += v;
      all += v;
    }
    run[tid] = before;
    tot[tid] = all;
  }
  __syncthreads();
  if (tid < E1) {
    int start = 0;  // lists of experts 1 .. tid - 1 come first
    for (int ee = 1; ee < tid; ++ee) start += tot[ee];
    if (tid >= 1) run[tid] += start;
    if (j == 0) {
      exp_cnt[tid] = tot[tid];
      exp_off[tid] = tid == 0 ? 0 : start + tot[tid];
    }
  }
  __syncthreads();
  // (sub rounds past the last assignment are skipped: the bound is uniform
  // over the block, so every barrier below is still reached by all threads)
  for (int sub = 0; sub < CHUNK && j * CHUNK + sub < Nk; sub += 256) {
    const int a = j * CHUNK + sub + tid;
    const int e = a < Nk ? eidx[a] : -1;
    int rank = 0;
    for (int ee = 1; ee < E1; ++ee) {
      uint64_t bal = __ballot(e == ee);
      if (e == ee) rank = __popcll(bal & lanemask_lt());
      if (lane == 0) wc[w][ee] = __popcll(bal);
    }
    __syncthreads();
    if (e >= 1) {
      int pos = run[e] + rank;
      for (int ww = 0; ww < w; ++ww) pos += wc[ww][e];
      rows[pos] = a;
    }
    __syncthreads();
    for (int ee = tid; ee < E1; ee += 256)
      if (ee >= 1) run[ee] += wc[0][ee] + wc[1][ee] + wc[2][ee] + wc[3][ee];
    __syncthreads();
  }
}

// Few assignments (one chunk) and no attention lists (decode): the expert
// lists by one block in one launch, histogram, offsets and the same stable
// scatter as the two kernels above (so the same lists).
__global__ __launch_bounds__(256) void compact_experts_one_kernel(const int32_t *__restrict__ eidx,
                                                                  int E1, int Nk,
                                                                  int32_t *__restrict__ rows,
                                                                  int32_t *__restrict__ exp_cnt,
                                                                  int32_t *__restrict__ exp_off) {
  __shared__ int lh[64], run[64];
  __shared__ int wc[4][64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid < E1) lh[tid] = 0;  // E1 <= 64
  __syncthreads();
  for (int a = tid; a < Nk; a += 256) atomicAdd(&lh[eidx[a]], 1);
  __syncthreads();
  if (tid < E1) {
    int start = 0;  // lists of experts 1 .. tid - 1 come first
    for (int ee = 1; ee < tid; ++ee) start += lh[ee];
    run[tid] = start;
    exp_cnt[tid] = lh[tid];
    exp_off[tid] = tid == 0 ? 0 : start + lh[tid];
  }
  __syncthreads();
  for (int sub = 0; sub < Nk; sub += 256) {  // block-uniform bound: every barrier is reached
    const int a = sub + tid;
    const int e = a < Nk ? eidx[a] : -1;
    int rank = 0;
    for (int ee = 1; ee < E1; ++ee) {
      const uint64_t bal = __ballot(e == ee);
      if (e == ee) rank = __popcll(bal & lanemask_lt());
      if (lane == 0) wc[w][ee] = __popcll(bal);
    }
    __syncthreads();
    if (e >= 1) {
      int pos = run[e] + rank;
      for (int ww = 0; ww < w; ++ww) pos += wc[ww][e];
      rows[pos] = a;
    }
    __syncthreads();
    if (tid >= 1 && tid < E1) run[tid] += wc[0][tid] + wc[1][tid] + wc[2][tid] + wc[3][tid];
    __syncthreads();
  }
}
int compact_hist_ints(int N, int k, int E1) { return ((N * k + CHUNK - 1) / CHUNK) * E1; }

hipError_t launch_compact(const triroute_cfg &cfg, int B, int T, const uint8_t *mode,
                          const int32_t *eidx, const triroute_compaction &c, int32_t *hist,
                          hipStream_t st, bool attn_lists) {
  const int H = cfg.n_heads, E1 = cfg.n_experts + 1, Nk = B * T * cfg.top_k;
  const int nbe = (Nk + CHUNK - 1) / CHUNK;
  if (!attn_lists && nbe == 1) {
    compact_experts_one_kernel<<<1, 256, 0, st>>>(eidx, E1, Nk, c.exp_rows, c.exp_cnt, c.exp_off);
    return hipGetLastError();
  }
  compact_count_kernel<<<B * H + nbe, 256, 0, st>>>(mode, eidx, B, T, H, E1, Nk, c.attn_cnt,
                                                    c.attn_idx, hist);
  compact_scatter_kernel<<<nbe, 256, 0, st>>>(eidx, hist, nbe, E1, Nk, c.exp_rows, c.exp_cnt,
                                               c.exp_off);
  return hipGetLastError();
}

}  // namespace tr
