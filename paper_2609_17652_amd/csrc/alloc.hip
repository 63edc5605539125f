// fathom_alloc_depths: Sec. 3.3, Eq. (g) and Eq. (wf) (water-filling), and the
// grouped top-r channel rule of Sec. 2 (uniform-depth mode).
//
// One wave per unit; lane l owns channels l and l + 64.  The water line is
// found exactly: the 4D candidates g_j * 2^-(2m-1) are non-negative doubles,
// so their IEEE bit patterns order like their values, and a bitwise search
// over the pattern (each step a wave-wide count from ballots) yields the
// (B+1)-th largest candidate with no log, exp or rounding -- a bisection on
// log(theta) carried to the last bit.  Each candidate is an fp32 value times a
// power of two, held exactly as a normal double: its sign bit and its 29 low
// mantissa bits are zero, and so are those of the answer (one of the
// candidates, or 0), so only bits 62..29 are searched.
#include "common.hpp"

namespace fathom {

template <fathom_dtype QDT>
__device__ __forceinline__ float load_q_as(const void* q, int64_t i) {
  if (QDT == FATHOM_F16)
    return __half2float(__ushort_as_half(((const __attribute__((address_space(1))) uint16_t*)q)[i]));
  return ((const __attribute__((address_space(1))) float*)q)[i];
}

template <fathom_dtype QDT>
__global__ __launch_bounds__(kWave) void alloc_waterfill_kernel(const void* __restrict__ q, int G,
                                                                const float* __restrict__ var,
                                                                int B, uint8_t* __restrict__ depths,
                                                                float* __restrict__ theta,
                                                                uint32_t* __restrict__ st) {
  const int u = blockIdx.x, lane = threadIdx.x;
  __builtin_assume(G >= 1 && G <= kMaxG);
  // every load is issued before the first use: heads past G re-read head G-1
  const float v0 = var[(int64_t)u * kD + lane], v1 = var[(int64_t)u * kD + lane + 64];
  float x[2][kMaxG];
#pragma unroll
  for (int h = 0; h < kMaxG; ++h) {
    const int64_t row = ((int64_t)u * G + min(h, G - 1)) * kD;
    x[0][h] = load_q_as<QDT>(q, row + lane);
    x[1][h] = load_q_as<QDT>(q, row + lane + 64);
  }
  uint64_t key[2][4];
  uint32_t flags = 0;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    float s = 0.0f;  // heads in ascending order
#pragma unroll
    for (int h = 0; h < kMaxG; ++h)
      if (h < G) s = __fadd_rn(s, __fmul_rn(x[r][h], x[r][h]));
    const float g = __fmul_rn(s, r ? v1 : v0);
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
    for (int bit = 62; bit >= 29; --bit) {
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
  {
    if (qdt == FATHOM_F16)
      hipLaunchKernelGGL(alloc_waterfill_kernel<FATHOM_F16>, dim3(U), dim3(kWave), 0, s, q, G, var,
                         budget_or_r, depths, theta, st);
    else
      hipLaunchKernelGGL(alloc_waterfill_kernel<FATHOM_F32>, dim3(U), dim3(kWave), 0, s, q, G, var,
                         budget_or_r, depths, theta, st);
  }
  else
    hipLaunchKernelGGL(alloc_topr_kernel, dim3(U), dim3(kWave), 0, s, q, qdt, G, budget_or_r, depths,
                       theta, st);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

}  // namespace fathom
