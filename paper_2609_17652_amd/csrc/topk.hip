// fathom_topk: Sec. 2 (top-k decoding) -- per query head, the k largest
// scores over an eligible window, ordered by (score desc, index asc).
//
// Exact radix select on an order-preserving uint32 key (score_key):
//   3 x (histogram pass over the row + pivot) on digits of 11, 11 and 10 bits
//   find the k-th largest key T and how many keys equal to T must be taken;
//   a count pass, a per-row prefix over chunks and a write pass then collect
//   every key > T and the lowest-index keys == T in index order (so ties go to
//   the lower index without sorting the row); a bitonic sort in LDS orders
//   the k winners.  Rows are split into chunks of kChunk elements so that a
//   launch has many workgroups even for a few rows.
#include "common.hpp"

namespace fathom {

constexpr int kTopkThreads = 256;
constexpr int kPerThread = 16;
constexpr int kChunk = kTopkThreads * kPerThread;  // 4096 elements per workgroup
constexpr int kBins = 2048;

struct RowState {
  uint32_t prefix;  // digits fixed so far (the final threshold key T after 3 passes)
  uint32_t mask;    // bits of `prefix` that are fixed
  int32_t need;     // how many still to take among keys matching `prefix`
  int32_t total_gt; // number of eligible keys > T (after the count scan)
};

struct TopkWs {
  uint32_t* hist;  // [R][kBins]
  RowState* state; // [R]
  uint32_t* cnt;   // [R][nchunks][2]
  uint64_t* sel;   // [R][k] composite (key << 32 | ~idx)
};

static inline size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

static inline int64_t topk_chunks(int64_t max_n) { return (max_n + kChunk - 1) / kChunk; }

size_t topk_ws_bytes(int R, int64_t max_n, int k) {
  const int64_t nch = topk_chunks(max_n) > 0 ? topk_chunks(max_n) : 1;
  return align_up((size_t)R * kBins * 4) + align_up((size_t)R * sizeof(RowState)) +
         align_up((size_t)R * nch * 2 * 4) + align_up((size_t)R * k * 8);
}

static TopkWs carve(void* ws, int R, int64_t max_n, int k) {
  const int64_t nch = topk_chunks(max_n) > 0 ? topk_chunks(max_n) : 1;
  char* p = reinterpret_cast<char*>(ws);
  TopkWs w;
  w.hist = reinterpret_cast<uint32_t*>(p); p += align_up((size_t)R * kBins * 4);
  w.state = reinterpret_cast<RowState*>(p); p += align_up((size_t)R * sizeof(RowState));
  w.cnt = reinterpret_cast<uint32_t*>(p); p += align_up((size_t)R * nch * 2 * 4);
  w.sel = reinterpret_cast<uint64_t*>(p);
  return w;
}

struct RowRange {
  int64_t lo, hi;  // eligible window [lo, hi)
};

__device__ __forceinline__ RowRange row_range(const int64_t* n, int u, int64_t cap, int64_t lo,
                                              int64_t tail, uint32_t* st) {
  const int64_t nu = unit_tokens(n, u, cap, st);
  RowRange r;
  r.lo = lo;
  r.hi = nu - tail;
  if (r.hi < r.lo) r.hi = r.lo;
  return r;
}

__global__ void topk_init_kernel(RowState* __restrict__ state, uint32_t* __restrict__ hist, int k) {
  const int r = blockIdx.x;
  for (int b = threadIdx.x; b < kBins; b += blockDim.x) hist[(int64_t)r * kBins + b] = 0u;
  if (threadIdx.x == 0) {
    state[r].prefix = 0u;
    state[r].mask = 0u;
    state[r].need = k;
    state[r].total_gt = 0;
  }
}

// histogram of digit (key >> shift) & (2^bits - 1) over eligible keys matching the prefix
__global__ __launch_bounds__(kTopkThreads) void topk_hist_kernel(const float* __restrict__ scores, int64_t ld_s,
                                                                 const int64_t* __restrict__ n, int G,
                                                                 int64_t lo, int64_t tail, int shift, int bits,
                                                                 const RowState* __restrict__ state,
                                                                 uint32_t* __restrict__ hist,
                                                                 uint32_t* __restrict__ st, int first) {
  __shared__ uint32_t h[kBins];
  const int r = blockIdx.y, u = r / G, tid = threadIdx.x;
  const RowRange rr = row_range(n, u, ld_s, lo, tail, (first && blockIdx.x == 0 && tid == 0) ? st : nullptr);
  const int64_t c0 = rr.lo + (int64_t)blockIdx.x * kChunk;
  if (c0 >= rr.hi) return;
  const uint32_t prefix = state[r].prefix, mask = state[r].mask;
  const uint32_t dmask = (1u << bits) - 1u;
  for (int b = tid; b < kBins; b += kTopkThreads) h[b] = 0u;
  __syncthreads();
  const float* row = scores + (int64_t)r * ld_s;
  bool nonfinite = false;
#pragma unroll 4
  for (int e = 0; e < kPerThread; ++e) {
    const int64_t i = c0 + (int64_t)e * kTopkThreads + tid;
    if (i < rr.hi) {
      const float s = row[i];
      if (first && !(fabsf(s) <= 3.402823466e38f)) nonfinite = true;
      const uint32_t key = score_key(s);
      if ((key & mask) == prefix) atomicAdd(&h[(key >> shift) & dmask], 1u);
    }
  }
  if (first && __ballot(nonfinite) && (tid & 63) == 0) set_status(st, FATHOM_DEV_NONFINITE);
  __syncthreads();
  uint32_t* gh = hist + (int64_t)r * kBins;
  for (int b = tid; b < kBins; b += kTopkThreads)
    if (h[b]) atomicAdd(&gh[b], h[b]);
}

// find the digit holding the need-th largest remaining key; clear the histogram
__global__ __launch_bounds__(kTopkThreads) void topk_pivot_kernel(int shift, int bits, RowState* __restrict__ state,
                                                                  uint32_t* __restrict__ hist) {
  __shared__ uint32_t part[kTopkThreads];
  __shared__ uint32_t hs[kBins];
  const int r = blockIdx.x, tid = threadIdx.x;
  const int nb = 1 << bits;
  uint32_t* gh = hist + (int64_t)r * kBins;
  for (int b = tid; b < kBins; b += kTopkThreads) {
    hs[b] = gh[b];
    gh[b] = 0u;
  }
  __syncthreads();
  // thread t owns digits [nb - (t+1)*per, nb - t*per), i.e. top-down order
  const int per = nb / kTopkThreads;
  const int top = nb - tid * per;
  uint32_t mine = 0;
  for (int d = top - 1; d >= top - per; --d) mine += hs[d];
  part[tid] = mine;
  __syncthreads();
  if (tid == 0) {
    const int need = state[r].need;
    uint32_t above = 0;
    int digit = 0;
    uint32_t above_digit = 0;
    bool found = false;
    for (int t = 0; t < kTopkThreads && !found; ++t) {
      if (above + part[t] >= (uint32_t)need) {
        const int tp = nb - t * per;
        for (int d = tp - 1; d >= tp - per; --d) {
          if (above + hs[d] >= (uint32_t)need) {
            digit = d;
            above_digit = above;
            found = true;
            break;
          }
          above += hs[d];
        }
      } else {
        above += part[t];
      }
    }
    if (!found) {  // fewer candidates than needed: take all of them
      digit = 0;
      above_digit = above - hs[0];
    }
    state[r].prefix |= (uint32_t)digit << shift;
    state[r].mask |= (uint32_t)(nb - 1) << shift;
    state[r].need = need - (int32_t)above_digit;
  }
}

// per chunk: number of eligible keys > T and == T
__global__ __launch_bounds__(kTopkThreads) void topk_count_kernel(const float* __restrict__ scores, int64_t ld_s,
                                                                  const int64_t* __restrict__ n, int G,
                                                                  int64_t lo, int64_t tail, int64_t nch,
                                                                  const RowState* __restrict__ state,
                                                                  uint32_t* __restrict__ cnt) {
  __shared__ uint32_t red[2][kTopkThreads / kWave];
  const int r = blockIdx.y, u = r / G, tid = threadIdx.x;
  const RowRange rr = row_range(n, u, ld_s, lo, tail, nullptr);
  const int64_t c0 = rr.lo + (int64_t)blockIdx.x * kChunk;
  const uint32_t T = state[r].prefix;
  const float* row = scores + (int64_t)r * ld_s;
  int gt = 0, eq = 0;
  for (int e = 0; e < kPerThread; ++e) {
    const int64_t i = c0 + (int64_t)e * kTopkThreads + tid;
    if (i < rr.hi) {
      const uint32_t key = score_key(row[i]);
      gt += key > T;
      eq += key == T;
    }
  }
  gt = wave_sum_int(gt);
  eq = wave_sum_int(eq);
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = gt;
    red[1][tid >> 6] = eq;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t a = 0, b = 0;
    for (int w = 0; w < kTopkThreads / kWave; ++w) {
      a += red[0][w];
      b += red[1][w];
    }
    cnt[((int64_t)r * nch + blockIdx.x) * 2 + 0] = a;
    cnt[((int64_t)r * nch + blockIdx.x) * 2 + 1] = b;
  }
}

// exclusive prefix over chunks (in index order), per row
__global__ void topk_scan_kernel(int64_t nch, RowState* __restrict__ state, uint32_t* __restrict__ cnt) {
  const int r = blockIdx.x;
  if (threadIdx.x != 0) return;
  uint32_t a = 0, b = 0;
  uint32_t* c = cnt + (int64_t)r * nch * 2;
  for (int64_t ch = 0; ch < nch; ++ch) {
    const uint32_t x = c[2 * ch], y = c[2 * ch + 1];
    c[2 * ch] = a;
    c[2 * ch + 1] = b;
    a += x;
    b += y;
  }
  state[r].total_gt = (int32_t)a;
}

// write keys > T, then the first `need` keys == T in index order, to sel[r][*]
__global__ __launch_bounds__(kTopkThreads) void topk_write_kernel(const float* __restrict__ scores, int64_t ld_s,
                                                                  const int64_t* __restrict__ n, int G,
                                                                  int64_t lo, int64_t tail, int64_t nch, int k,
                                                                  const RowState* __restrict__ state,
                                                                  const uint32_t* __restrict__ cnt,
                                                                  uint64_t* __restrict__ sel) {
  __shared__ uint32_t wt[2][kTopkThreads / kWave];
  const int r = blockIdx.y, u = r / G, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const RowRange rr = row_range(n, u, ld_s, lo, tail, nullptr);
  const int64_t c0 = rr.lo + (int64_t)blockIdx.x * kChunk;
  if (c0 >= rr.hi) return;
  const uint32_t T = state[r].prefix;
  const int32_t need = state[r].need, total_gt = state[r].total_gt;
  uint32_t base_gt = cnt[((int64_t)r * nch + blockIdx.x) * 2 + 0];
  uint32_t base_eq = cnt[((int64_t)r * nch + blockIdx.x) * 2 + 1];
  const float* row = scores + (int64_t)r * ld_s;
  uint64_t* out = sel + (int64_t)r * k;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int e = 0; e < kPerThread; ++e) {
    const int64_t i = c0 + (int64_t)e * kTopkThreads + tid;
    uint32_t key = 0;
    bool g = false, q = false;
    if (i < rr.hi) {
      key = score_key(row[i]);
      g = key > T;
      q = key == T;
    }
    const uint64_t bg = __ballot(g), bq = __ballot(q);
    if (lane == 0) {
      wt[0][wave] = (uint32_t)__popcll(bg);
      wt[1][wave] = (uint32_t)__popcll(bq);
    }
    __syncthreads();
    uint32_t og = base_gt, oq = base_eq, tg = 0, tq = 0;
    for (int w = 0; w < kTopkThreads / kWave; ++w) {
      if (w < wave) {
        og += wt[0][w];
        oq += wt[1][w];
      }
      tg += wt[0][w];
      tq += wt[1][w];
    }
    const uint64_t comp = ((uint64_t)key << 32) | (uint64_t)(~(uint32_t)i);
    if (g) out[og + __popcll(bg & lt_mask)] = comp;
    if (q) {
      const uint32_t rank = oq + (uint32_t)__popcll(bq & lt_mask);
      if ((int32_t)rank < need) out[total_gt + rank] = comp;
    }
    base_gt += tg;
    base_eq += tq;
    __syncthreads();
  }
}

// order the winners by (key desc, index asc); empty slots (0) -> (-1, NaN)
__global__ __launch_bounds__(1024) void topk_sort_kernel(const float* __restrict__ scores, int64_t ld_s, int k,
                                                         const uint64_t* __restrict__ sel, int32_t* __restrict__ idx,
                                                         float* __restrict__ val, uint32_t* __restrict__ st) {
  extern __shared__ uint64_t buf[];
  const int r = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
  int P = 1;
  while (P < k) P <<= 1;
  const uint64_t* in = sel + (int64_t)r * k;
  // sel was cleared before the write pass: unwritten slots are 0, the lowest value
  for (int i = tid; i < P; i += nt) buf[i] = i < k ? in[i] : 0ull;
  __syncthreads();
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < P; i += nt) {
        const int j = i ^ stride;
        if (j > i) {
          const bool desc = (i & size) == 0;
          const uint64_t a = buf[i], b = buf[j];
          if (desc ? (a < b) : (a > b)) {
            buf[i] = b;
            buf[j] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  bool shortfall = false;
  const float* row = scores + (int64_t)r * ld_s;
  for (int i = tid; i < k; i += nt) {
    const uint64_t c = buf[i];
    if (c == 0ull) {
      idx[(int64_t)r * k + i] = -1;
      if (val) val[(int64_t)r * k + i] = __uint_as_float(0x7FC00000u);
      shortfall = true;
    } else {
      const int32_t ii = (int32_t)(~(uint32_t)(c & 0xFFFFFFFFull));
      idx[(int64_t)r * k + i] = ii;
      if (val) val[(int64_t)r * k + i] = row[ii];
    }
  }
  if (__syncthreads_or(shortfall) && tid == 0) set_status(st, FATHOM_DEV_TOPK_SHORT);
}

__global__ void topk_clear_sel_kernel(uint64_t* __restrict__ sel, int64_t total) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < total) sel[i] = 0ull;
}

fathom_status launch_topk(const float* scores, int64_t ld_s, const int64_t* n, int U, int G, int k,
                          int64_t lo, int64_t tail, int32_t* idx, float* val, void* ws, uint32_t* st,
                          hipStream_t s) {
  const int R = U * G;
  if (R == 0) return FATHOM_OK;
  const int64_t nch = topk_chunks(ld_s) > 0 ? topk_chunks(ld_s) : 1;
  TopkWs w = carve(ws, R, ld_s, k);
  hipLaunchKernelGGL(topk_init_kernel, dim3(R), dim3(256), 0, s, w.state, w.hist, k);
  const int shifts[3] = {21, 10, 0}, bits[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    hipLaunchKernelGGL(topk_hist_kernel, dim3((unsigned)nch, (unsigned)R), dim3(kTopkThreads), 0, s, scores,
                       ld_s, n, G, lo, tail, shifts[pass], bits[pass], w.state, w.hist, st, pass == 0 ? 1 : 0);
    hipLaunchKernelGGL(topk_pivot_kernel, dim3(R), dim3(kTopkThreads), 0, s, shifts[pass], bits[pass], w.state,
                       w.hist);
  }
  hipLaunchKernelGGL(topk_count_kernel, dim3((unsigned)nch, (unsigned)R), dim3(kTopkThreads), 0, s, scores, ld_s,
                     n, G, lo, tail, nch, w.state, w.cnt);
  hipLaunchKernelGGL(topk_scan_kernel, dim3(R), dim3(64), 0, s, nch, w.state, w.cnt);
  const int64_t total = (int64_t)R * k;
  hipLaunchKernelGGL(topk_clear_sel_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, w.sel, total);
  hipLaunchKernelGGL(topk_write_kernel, dim3((unsigned)nch, (unsigned)R), dim3(kTopkThreads), 0, s, scores, ld_s,
                     n, G, lo, tail, nch, k, w.state, w.cnt, w.sel);
  int P = 1;
  while (P < k) P <<= 1;
  hipLaunchKernelGGL(topk_sort_kernel, dim3(R), dim3(1024), (size_t)P * 8, s, scores, ld_s, k, w.sel, idx, val,
                     st);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

}  // namespace fathom
