// fathom_alloc_depths: Sec. 3.3, Eq. (g) and Eq. (wf) (water-filling), and the
// grouped top-r channel rule of Sec. 2 (uniform-depth mode).
//
// One wave per unit; lane l owns channels l and l + 64.  The water line is
// found exactly: the 4D candidates g_j * 2^-(2m-1) are non-negative doubles,
// so their IEEE bit patterns order like their values, and a 64-step bitwise
// search over the pattern (each step a wave-wide count from ballots) yields the (B+1)-th
// largest candidate with no log, exp or rounding -- a bisection on log(theta)
// carried to the last bit.
#include "common.hpp"

namespace fathom {

__global__ __launch_bounds__(kWave) void alloc_waterfill_kernel(const void* __restrict__ q, fathom_dtype qdt,
                                                                int G, const float* __restrict__ var,
                                                                int B, uint8_t* __restrict__ depths,
                                                                float* __restrict__ theta,
                                                                uint32_t* __restrict__ st) {
  const int u = blockIdx.x, lane = threadIdx.x;
  uint64_t key[2][4];
  uint32_t flags = 0;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int j = lane + 64 * r;
    float s = 0.0f;
    for (int h = 0; h < G; ++h) {
      const float x = load_q(q, qdt, ((int64_t)u * G + h) * kD + j);
      s = __fadd_rn(s, __fmul_rn(x, x));
    }
    const float g = __fmul_rn(s, var[(int64_t)u * kD + j]);
    if (!(g >= 0.0f && g <= 3.402823466e38f)) flags |= FATHOM_DEV_NONFINITE;
#pragma unroll
    for (int m = 1; m <= 4; ++m) {
      const double c = ldexp((double)g, -(2 * m - 1));  // exact
      key[r][m - 1] = c == 0.0 ? 0ull : (uint64_t)__double_as_longlong(c);
    }
  }
  // T = largest pattern with #{keys >= T} >= B + 1, i.e. the (B+1)-th largest key
  uint64_t T = 0;
  if (B < 4 * kD) {
    for (int bit = 63; bit >= 0; --bit) {
      const uint64_t cand = T | (1ull << bit);
      int c = 0;  // wave-wide count from ballots: no cross-lane data movement
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int m = 0; m < 4; ++m) c += __popcll(__ballot(key[r][m] >= cand));
      if (c >= B + 1) T = cand;
    }
  }
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    int t = 0;
#pragma unroll
    for (int m = 0; m < 4; ++m) t += key[r][m] > T;
    depths[(int64_t)u * kD + lane + 64 * r] = (uint8_t)t;
  }
  if (lane == 0 && theta) theta[u] = (float)__longlong_as_double((long long)T);
  uint32_t f = flags;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) f |= __shfl_xor(f, m, kWave);
  if (lane == 0) set_status(st, f);
}

__global__ __launch_bounds__(kWave) void alloc_topr_kernel(const void* __restrict__ q, fathom_dtype qdt,
                                                           int G, int r, uint8_t* __restrict__ depths,
                                                           float* __restrict__ theta,
                                                           uint32_t* __restrict__ st) {
  __shared__ float w[kD];
  const int u = blockIdx.x, lane = threadIdx.x;
  uint32_t flags = 0;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int j = lane + 64 * k;
    float s = 0.0f;
    for (int h = 0; h < G; ++h) s = __fadd_rn(s, fabsf(load_q(q, qdt, ((int64_t)u * G + h) * kD + j)));
    if (!(s <= 3.402823466e38f)) flags |= FATHOM_DEV_NONFINITE;
    w[j] = s;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int j = lane + 64 * k;
    const float wj = w[j];
    int rank = 0;  // position of j in (w desc, j asc) order
    for (int i = 0; i < kD; ++i) {
      const float wi = w[i];
      rank += (wi > wj) || (wi == wj && i < j);
    }
    depths[(int64_t)u * kD + j] = rank < r ? 4 : 0;
    if (theta && rank == r - 1) theta[u] = wj;
  }
  if (theta && r == 0 && lane == 0) theta[u] = 0.0f;
  uint32_t f = flags;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) f |= __shfl_xor(f, m, kWave);
  if (lane == 0) set_status(st, f);
}

fathom_status launch_alloc(const void* q, fathom_dtype qdt, int U, int G, const float* var,
                           fathom_mode mode, int budget_or_r, uint8_t* depths, float* theta,
                           uint32_t* st, hipStream_t s) {
  if (U == 0) return FATHOM_OK;
  if (mode == FATHOM_WATERFILL)
    hipLaunchKernelGGL(alloc_waterfill_kernel, dim3(U), dim3(kWave), 0, s, q, qdt, G, var, budget_or_r,
                       depths, theta, st);
  else
    hipLaunchKernelGGL(alloc_topr_kernel, dim3(U), dim3(kWave), 0, s, q, qdt, G, budget_or_r, depths,
                       theta, st);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

}  // namespace fathom
