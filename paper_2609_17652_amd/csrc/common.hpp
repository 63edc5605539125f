// Internal helpers of libfathom (gfx950, wave64).  Not part of the C ABI.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/fathom.h"

namespace fathom {

constexpr int kWave = 64;
constexpr int kBlockTokens = 64;  // tokens per quantisation block (Sec. 3.2)
constexpr int kPlanes = 4;        // 4-bit codes
constexpr int kD = 128;           // supported head dimension
constexpr int kMaxG = 8;          // query heads per KV head accepted by every entry point

#define FATHOM_LAUNCH_CHECK()                                   \
  do {                                                          \
    hipError_t e_ = hipGetLastError();                          \
    if (e_ != hipSuccess) return FATHOM_ERR_HIP;                \
  } while (0)

__device__ __forceinline__ void set_status(uint32_t* st, uint32_t bits) {
  if (st && bits)
    __hip_atomic_fetch_or((__attribute__((address_space(1))) uint32_t*)st, bits, __ATOMIC_RELAXED,
                          __HIP_MEMORY_SCOPE_AGENT);
}

// n[u] clamped to [0, cap]; raises BAD_N and returns 0 for out-of-range values.
__device__ __forceinline__ int64_t unit_tokens(const int64_t* n, int u, int64_t cap, uint32_t* st) {
  int64_t v = n[u];
  if (v < 0 || v > cap) {
    set_status(st, FATHOM_DEV_BAD_N);
    return 0;
  }
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = __fadd_rn(v, __shfl_xor(v, m, kWave));
  return v;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ __forceinline__ float half_bits_to_float(uint16_t h) {
  return __half2float(__ushort_as_half(h));
}

// Query element i (fp16 converts to fp32 exactly), read through the global
// address space so it never counts against the LDS wait counter.
__device__ __forceinline__ float load_q(const void* q, fathom_dtype qdt, int64_t i) {
  if (qdt == FATHOM_F16)
    return __half2float(__ushort_as_half(((const __attribute__((address_space(1))) uint16_t*)q)[i]));
  return ((const __attribute__((address_space(1))) float*)q)[i];
}

// Order-preserving map fp32 -> uint32: larger score -> larger key; -0 == +0;
// NaN -> 0, below every number (-inf maps to 0x007FFFFF).
__device__ __forceinline__ uint32_t score_key(float s) {
  if (s != s) return 0u;
  if (s == 0.0f) s = 0.0f;
  uint32_t b = __float_as_uint(s);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Block-wide search over a digit histogram hist[0..nb): the largest digit d
// with (number of items in digits >= d) >= need; *above = items in digits > d.
// If the total is below need, d = 0 and *above = total - hist[0].  All threads
// of the block must call it; part[] needs blockDim.x / 64 entries.
__device__ inline void find_crossing(const uint32_t* hist, int nb, uint32_t need, uint32_t* part, int* s_digit,
                                     uint32_t* s_above) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6, nw = nt >> 6;
  const int per = (nb + nt - 1) / nt;
  // thread t owns digits nb-1-t*per down to nb-(t+1)*per (top-down order)
  uint32_t mine = 0;
  for (int x = 0; x < per; ++x) {
    const int d = nb - 1 - tid * per - x;
    if (d >= 0) mine += hist[d];
  }
  uint32_t inc = mine;  // inclusive scan within the wave
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t v = __shfl_up(inc, o, kWave);
    if (lane >= o) inc += v;
  }
  if (lane == 63) part[wave] = inc;
  __syncthreads();
  uint32_t before = 0, total = 0;
  for (int w = 0; w < nw; ++w) {
    if (w < wave) before += part[w];
    total += part[w];
  }
  const uint32_t cum = before + inc, prev = cum - mine;
  if (prev < need && cum >= need) {
    uint32_t above = prev;
    for (int x = 0; x < per; ++x) {
      const int d = nb - 1 - tid * per - x;
      if (d < 0) break;
      if (above + hist[d] >= need) {
        *s_digit = d;
        *s_above = above;
        break;
      }
      above += hist[d];
    }
  }
  if (tid == 0 && total < need) {
    *s_digit = 0;
    *s_above = total - hist[0];
  }
  __syncthreads();
}

}  // namespace fathom
