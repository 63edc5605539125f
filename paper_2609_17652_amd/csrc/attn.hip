// fathom_sparse_attn: Sec. 2 (top-k decoding) -- exact attention of each
// query head over sink + local + its top-k rows, with fp16 K/V rows resident
// in HBM and fp32 arithmetic.
//
// Split over the selected rows (flash-decoding style): the row list of a head
// -- sink rows, local rows, then its top-k entries (entries outside the
// sink/local gap or negative are skipped) -- is cut into chunks of kWaveRows
// positions, one per wave.  A wave loads its rows' K and V together (16 lanes
// per row, 16 bytes each: 4 rows per load instruction, 8 rows per lane), so
// one round of memory latency covers both; it then forms the logits (a
// 16-lane reduction per row), the chunk's max m, sum d of exp(z - m) and
// partial output o = sum exp(z - m) V into the caller's workspace.  A second
// kernel combines the chunks of each head:
//   out = sum_c e^(m_c - M) o_c / sum_c e^(m_c - M) d_c.
#include "common.hpp"

namespace fathom {

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = kAttnThreads / kWave;
constexpr int kWaveRows = 32;                         // row-list positions per wave
constexpr int kRowSteps = kWaveRows / 4;              // 4 rows per load instruction
constexpr int kMaxSinkLocal = 1024;
constexpr int kPart = kD + 2;  // per chunk: m, d, o[D]

static inline int attn_chunks(int k, int n_sink, int n_local) {
  return (n_sink + n_local + k + kWaveRows - 1) / kWaveRows;
}

size_t attn_ws_bytes(int U, int G, int k, int n_sink, int n_local) {
  const int S = attn_chunks(k, n_sink, n_local);
  return (size_t)U * G * (S > 0 ? S : 1) * kPart * sizeof(float);
}

__device__ __forceinline__ float gload_f(const float* p) { return *(const __attribute__((address_space(1))) float*)p; }
__device__ __forceinline__ uint32_t gload_u32(const void* p) {
  return *(const __attribute__((address_space(1))) uint32_t*)p;
}
__device__ __forceinline__ void gstore_f(float* p, float v) { *(__attribute__((address_space(1))) float*)p = v; }

// 8 fp16 values (16 bytes) of a row; VEC: one 16-byte load (16-byte aligned).
typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));
template <bool VEC>
__device__ __forceinline__ uint4 load8h(const uint16_t* p) {
  if constexpr (VEC) {
    const v4u32 v = *(const __attribute__((address_space(1))) v4u32*)p;
    return make_uint4(v.x, v.y, v.z, v.w);
  }
  return make_uint4(gload_u32(p), gload_u32(p + 2), gload_u32(p + 4), gload_u32(p + 6));
}

template <bool VEC>
__global__ __launch_bounds__(kAttnThreads) void attn_chunk_kernel(const void* __restrict__ q, fathom_dtype qdt,
                                                                  const uint16_t* __restrict__ Krows,
                                                                  const uint16_t* __restrict__ Vrows, int64_t ld_tok,
                                                                  int64_t ld_unit, const int64_t* __restrict__ n,
                                                                  int G, const int32_t* __restrict__ idx, int k,
                                                                  int n_sink, int n_local, float sm_scale, int S,
                                                                  float* __restrict__ ws, uint32_t* __restrict__ st) {
  const int r = blockIdx.y, u = r / G, h = r % G;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = blockIdx.x * kAttnWaves + wave;  // this wave's chunk
  if (c >= S) return;
  int64_t nu = *(const __attribute__((address_space(1))) int64_t*)(n + u);
  if (nu < 0) {
    if (lane == 0 && c == 0) set_status(st, FATHOM_DEV_BAD_N);
    nu = 0;
  }
  const int64_t ns = n_sink < nu ? n_sink : nu;
  const int64_t l0 = nu - n_local > ns ? nu - n_local : ns;
  const int64_t nloc = nu - l0;
  float* wp = ws + ((int64_t)r * S + c) * kPart;
  // ---- the row of each of the wave's positions (lane x < 32: position x) ----
  int32_t myrow = -1;
  if (lane < kWaveRows) {
    const int64_t p = (int64_t)c * kWaveRows + lane;
    if (p < ns) {
      myrow = (int32_t)p;
    } else if (p < ns + nloc) {
      myrow = (int32_t)(l0 + (p - ns));
    } else if (p - ns - nloc < k) {
      const int32_t v = *(const __attribute__((address_space(1))) int32_t*)(idx + (int64_t)r * k + (p - ns - nloc));
      if (v >= ns && v < l0) myrow = v;
    }
  }
  // ---- K and V of the rows: lane group g = lane / 16 takes position 4 s + g,
  // lane x = lane mod 16 channels 8x .. 8x + 7 ----
  const int g = lane >> 4, x = lane & 15;
  const uint16_t* Ku = Krows + (int64_t)u * ld_unit + 8 * x;
  const uint16_t* Vu = Vrows + (int64_t)u * ld_unit + 8 * x;
  int32_t row[kRowSteps];
  uint4 kv[kRowSteps], vv[kRowSteps];
#pragma unroll
  for (int s = 0; s < kRowSteps; ++s) {
    row[s] = __shfl(myrow, 4 * s + g, kWave);
    kv[s] = make_uint4(0u, 0u, 0u, 0u);
    vv[s] = make_uint4(0u, 0u, 0u, 0u);
    if (row[s] >= 0) {
      kv[s] = load8h<VEC>(Ku + (int64_t)row[s] * ld_tok);
      vv[s] = load8h<VEC>(Vu + (int64_t)row[s] * ld_tok);
    }
  }
  float qv[8];
  {
    const int64_t qo = ((int64_t)u * G + h) * kD + 8 * x;
#pragma unroll
    for (int e = 0; e < 8; ++e) qv[e] = load_q(q, qdt, qo + e);
  }
  // ---- logits ----
  float z[kRowSteps];
  float zm = -__builtin_huge_valf();
#pragma unroll
  for (int s = 0; s < kRowSteps; ++s) {
    const uint32_t w[4] = {kv[s].x, kv[s].y, kv[s].z, kv[s].w};
    float d = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      d = __fmaf_rn(qv[2 * e], half_bits_to_float((uint16_t)(w[e] & 0xFFFFu)), d);
      d = __fmaf_rn(qv[2 * e + 1], half_bits_to_float((uint16_t)(w[e] >> 16)), d);
    }
#pragma unroll
    for (int m = 1; m < 16; m <<= 1) d = __fadd_rn(d, __shfl_xor(d, m, kWave));
    z[s] = row[s] >= 0 ? __fmul_rn(d, sm_scale) : -__builtin_huge_valf();
    zm = fmaxf(zm, z[s]);
  }
  zm = fmaxf(zm, __shfl_xor(zm, 16, kWave));
  zm = fmaxf(zm, __shfl_xor(zm, 32, kWave));
  if (zm == -__builtin_huge_valf()) {  // no row in this chunk
    if (lane == 0) {
      gstore_f(wp, zm);
      gstore_f(wp + 1, 0.0f);
    }
    return;
  }
  // ---- exp-sum and weighted V rows ----
  float den = 0.0f, o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = 0.0f;
#pragma unroll
  for (int s = 0; s < kRowSteps; ++s) {
    const float pz = row[s] >= 0 ? expf(__fsub_rn(z[s], zm)) : 0.0f;
    den = __fadd_rn(den, pz);
    const uint32_t w[4] = {vv[s].x, vv[s].y, vv[s].z, vv[s].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[2 * e] = __fmaf_rn(pz, half_bits_to_float((uint16_t)(w[e] & 0xFFFFu)), o[2 * e]);
      o[2 * e + 1] = __fmaf_rn(pz, half_bits_to_float((uint16_t)(w[e] >> 16)), o[2 * e + 1]);
    }
  }
  // the four lane groups hold disjoint rows: sum across them
  den = __fadd_rn(den, __shfl_xor(den, 16, kWave));
  den = __fadd_rn(den, __shfl_xor(den, 32, kWave));
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    o[e] = __fadd_rn(o[e], __shfl_xor(o[e], 16, kWave));
    o[e] = __fadd_rn(o[e], __shfl_xor(o[e], 32, kWave));
  }
  if (lane < 16) {
#pragma unroll
    for (int e = 0; e < 8; ++e) gstore_f(wp + 2 + 8 * x + e, o[e]);
  }
  if (lane == 0) {
    gstore_f(wp, zm);
    gstore_f(wp + 1, den);
  }
}

// out = sum_c e^(m_c - M) o_c / sum_c e^(m_c - M) d_c over the chunks of a head.
// One 512-thread workgroup per head: the chunk maxima and sums go to LDS, then
// four groups of 128 threads (one channel each) take every fourth chunk, with
// kCombBatch chunks' loads in flight at a time.
constexpr int kCombThreads = 512;
constexpr int kCombGroups = kCombThreads / kD;
constexpr int kCombBatch = 16;
constexpr int kMaxChunks = (kMaxSinkLocal + FATHOM_MAX_K + kWaveRows - 1) / kWaveRows;
__global__ __launch_bounds__(kCombThreads) void attn_combine_kernel(const float* __restrict__ ws, int S,
                                                                   float* __restrict__ out) {
  __shared__ float em[kMaxChunks];  // m_c, then e^(m_c - M) (0 for a chunk without rows)
  __shared__ float dc[kMaxChunks];
  __shared__ float red[kCombThreads / kWave];
  __shared__ float po[kCombGroups][kD];
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* wp = ws + (int64_t)r * S * kPart;
  float M = -__builtin_huge_valf();
  for (int c = tid; c < S; c += kCombThreads) {
    const float m = gload_f(wp + (int64_t)c * kPart);
    em[c] = m;
    dc[c] = gload_f(wp + (int64_t)c * kPart + 1);
    M = fmaxf(M, m);
  }
  M = wave_max(M);
  if (lane == 0) red[wave] = M;
  __syncthreads();
  M = red[0];
#pragma unroll
  for (int w = 1; w < kCombThreads / kWave; ++w) M = fmaxf(M, red[w]);
  if (M == -__builtin_huge_valf()) {  // no row at all
    if (tid < kD) gstore_f(out + (int64_t)r * kD + tid, 0.0f);
    return;
  }
  for (int c = tid; c < S; c += kCombThreads) {
    const float m = em[c];
    em[c] = m == -__builtin_huge_valf() ? 0.0f : expf(__fsub_rn(m, M));
  }
  __syncthreads();
  const int gi = tid / kD, ch = tid % kD;
  float o = 0.0f;
  for (int c0 = gi; c0 < S; c0 += kCombBatch * kCombGroups) {
    float e[kCombBatch], v[kCombBatch];
#pragma unroll
    for (int j = 0; j < kCombBatch; ++j) {
      const int c = c0 + j * kCombGroups;
      e[j] = c < S ? em[c] : 0.0f;
      v[j] = e[j] != 0.0f ? gload_f(wp + (int64_t)c * kPart + 2 + ch) : 0.0f;  // empty chunks wrote no o
    }
#pragma unroll
    for (int j = 0; j < kCombBatch; ++j) o = __fmaf_rn(e[j], v[j], o);
  }
  po[gi][ch] = o;
  __syncthreads();
  if (tid < kD) {
    float den = 0.0f;
    for (int c = 0; c < S; ++c) den = __fmaf_rn(em[c], dc[c], den);
    float acc = 0.0f;
#pragma unroll
    for (int g = 0; g < kCombGroups; ++g) acc = __fadd_rn(acc, po[g][tid]);
    gstore_f(out + (int64_t)r * kD + tid, acc / den);
  }
}

fathom_status launch_sparse_attn(const void* q, fathom_dtype qdt, const uint16_t* Krows, const uint16_t* Vrows,
                                 int64_t ld_tok, int64_t ld_unit, const int64_t* n, int U, int G,
                                 const int32_t* idx, int k, int n_sink, int n_local, float sm_scale, float* out,
                                 void* ws, uint32_t* st, hipStream_t s) {
  if (U == 0) return FATHOM_OK;
  int S = attn_chunks(k, n_sink, n_local);
  if (S < 1) S = 1;
  float* w = reinterpret_cast<float*>(ws);
  const dim3 grid((unsigned)((S + kAttnWaves - 1) / kAttnWaves), (unsigned)(U * G));
  // 16-byte row loads when every row start is 16-byte aligned
  const bool vec = ((reinterpret_cast<uintptr_t>(Krows) | reinterpret_cast<uintptr_t>(Vrows)) & 15) == 0 &&
                   (ld_tok & 7) == 0 && (ld_unit & 7) == 0;
  if (vec)
    hipLaunchKernelGGL(attn_chunk_kernel<true>, grid, dim3(kAttnThreads), 0, s, q, qdt, Krows, Vrows, ld_tok,
                       ld_unit, n, G, idx, k, n_sink, n_local, sm_scale, S, w, st);
  else
    hipLaunchKernelGGL(attn_chunk_kernel<false>, grid, dim3(kAttnThreads), 0, s, q, qdt, Krows, Vrows, ld_tok,
                       ld_unit, n, G, idx, k, n_sink, n_local, sm_scale, S, w, st);
  hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)(U * G)), dim3(kCombThreads), 0, s, w, S, out);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

int attn_max_sink_local() { return kMaxSinkLocal; }

}  // namespace fathom
