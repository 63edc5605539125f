// fathom_scan: Sec. 3.2-3.3 -- approximate scores from per-channel plane
// prefixes, all G query heads of a unit at once (the plan is shared by the
// group, so each plane word is read once for all G heads).
//
// One wave per 64-key block, lane i = key 64b + i.  The unit's active
// channels (t_j > 0) are compacted into LDS once per workgroup; per active
// channel the wave reads the block's fp16 scale and the first t plane words
// as wave-uniform (scalar) loads, each lane extracts its t code bits and
// dequantises its key exactly, and every head accumulates one fused
// multiply-add in the documented order:
//   khat = (c^(t) + 1/2 - 2^(t-1)) * a16 * 2^(1-t)   (exact in fp32),
//   acc_h = fmaf(q_hj, khat, acc_h),  channels ascending, acc from +0.
#include "common.hpp"

namespace fathom {

constexpr int kScanThreads = 256;
constexpr int kScanWaves = kScanThreads / kWave;

// Active channel list of one unit: act[a] = j | (t << 8), channels ascending.
__device__ __forceinline__ int build_active(const uint8_t* __restrict__ d, int* act, int* nact) {
  const int tid = threadIdx.x;
  __shared__ int wcount[2];
  int t = 0;
  if (tid < kD) t = d[tid] > kPlanes ? kPlanes : d[tid];  // depths above 4 read as 4
  const bool on = tid < kD && t > 0;
  const uint64_t m = __ballot(on);
  const int lane = tid & 63, wave = tid >> 6;
  if (tid < kD && lane == 0) wcount[wave] = __popcll(m);
  __syncthreads();
  if (on) {
    const int base = wave == 1 ? wcount[0] : 0;
    const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    act[base + __popcll(m & lt)] = tid | (t << 8);
  }
  if (tid == 0) *nact = wcount[0] + wcount[1];
  __syncthreads();
  return *nact;
}

template <int G>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(const uint64_t* __restrict__ planes,
                                                            const uint16_t* __restrict__ scales,
                                                            const int64_t* __restrict__ n, int64_t nb_cap,
                                                            const void* __restrict__ q, fathom_dtype qdt,
                                                            const uint8_t* __restrict__ depths,
                                                            float* __restrict__ scores, int64_t ld_s,
                                                            uint32_t* __restrict__ st) {
  __shared__ int act[kD];
  __shared__ int nact;
  __shared__ float qs[G][kD];
  const int u = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int x = tid; x < G * kD; x += kScanThreads) qs[x / kD][x % kD] = load_q(q, qdt, (int64_t)u * G * kD + x);
  const int A = build_active(depths + (int64_t)u * kD, act, &nact);
  const int64_t nu = unit_tokens(n, u, nb_cap * kBlockTokens, (blockIdx.x == 0 && tid == 0) ? st : nullptr);
  const int64_t b = (int64_t)blockIdx.x * kScanWaves + wave;
  if (b * kBlockTokens >= nu) return;
  const uint64_t* Pu = planes + (int64_t)u * kD * kPlanes * nb_cap;
  const uint16_t* Su = scales + (int64_t)u * kD * nb_cap;
  float acc[G];
#pragma unroll
  for (int h = 0; h < G; ++h) acc[h] = 0.0f;
  for (int a = 0; a < A; ++a) {
    const int e = __builtin_amdgcn_readfirstlane(act[a]);
    const int j = e & 0xFF, t = e >> 8;
    const float af = half_bits_to_float(Su[(int64_t)j * nb_cap + b]);
    const uint64_t* Pj = Pu + (int64_t)j * kPlanes * nb_cap + b;
    uint32_t c = 0;
    for (int p = 0; p < t; ++p) c = 2u * c + (uint32_t)((Pj[(int64_t)p * nb_cap] >> lane) & 1ull);
    const float y = (float)c + (0.5f - (float)(1 << (t - 1)));  // exact half-integer
    const float sc = __uint_as_float((uint32_t)(128 - t) << 23);  // 2^(1-t)
    const float khat = __fmul_rn(y, __fmul_rn(af, sc));            // exact: <= 16 significant bits
#pragma unroll
    for (int h = 0; h < G; ++h) acc[h] = __fmaf_rn(qs[h][j], khat, acc[h]);
  }
  const int64_t i = b * kBlockTokens + lane;
  if (i < nu && i < ld_s) {
#pragma unroll
    for (int h = 0; h < G; ++h) scores[((int64_t)u * G + h) * ld_s + i] = acc[h];
  }
}

template <int G>
static void launch_scan_g(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U, int64_t nb_cap,
                          const void* q, fathom_dtype qdt, const uint8_t* depths, float* scores, int64_t ld_s,
                          uint32_t* st, hipStream_t s) {
  dim3 grid((unsigned)((nb_cap + kScanWaves - 1) / kScanWaves), (unsigned)U);
  hipLaunchKernelGGL(scan_kernel<G>, grid, dim3(kScanThreads), 0, s, planes, scales, n, nb_cap, q, qdt, depths,
                     scores, ld_s, st);
}

fathom_status launch_scan(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U, int64_t nb_cap,
                          const void* q, fathom_dtype qdt, int G, const uint8_t* depths, float* scores,
                          int64_t ld_s, uint32_t* st, hipStream_t s) {
  if (U == 0 || nb_cap == 0) return FATHOM_OK;
  switch (G) {
    case 1: launch_scan_g<1>(planes, scales, n, U, nb_cap, q, qdt, depths, scores, ld_s, st, s); break;
    case 2: launch_scan_g<2>(planes, scales, n, U, nb_cap, q, qdt, depths, scores, ld_s, st, s); break;
    case 3: launch_scan_g<3>(planes, scales, n, U, nb_cap, q, qdt, depths, scores, ld_s, st, s); break;
    case 4: launch_scan_g<4>(planes, scales, n, U, nb_cap, q, qdt, depths, scores, ld_s, st, s); break;
    case 5: launch_scan_g<5>(planes, scales, n, U, nb_cap, q, qdt, depths, scores, ld_s, st, s); break;
    case 6: launch_scan_g<6>(planes, scales, n, U, nb_cap, q, qdt, depths, scores, ld_s, st, s); break;
    case 7: launch_scan_g<7>(planes, scales, n, U, nb_cap, q, qdt, depths, scores, ld_s, st, s); break;
    default: launch_scan_g<8>(planes, scales, n, U, nb_cap, q, qdt, depths, scores, ld_s, st, s); break;
  }
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

}  // namespace fathom
