// fathom_sparse_attn: Sec. 2 (top-k decoding) -- exact attention of each
// query head over sink + local + its top-k rows, with fp16 K/V rows resident
// in HBM and fp32 arithmetic.
//
// Split over the selected rows (flash-decoding style): the row list of a head
// -- sink rows, local rows, then its top-k entries (entries outside the
// sink/local gap or negative are skipped) -- is cut into chunks of kChunk
// positions.  Workgroup (chunk, head) computes its rows' logits (4 lanes per
// row, 32 channels each), the chunk's max m, sum d of exp(z - m) and partial
// output o = sum exp(z - m) V (64 lanes x 2 channels, the chunk's rows split
// over 4 waves) into the caller's workspace; a second kernel combines the
// chunks of each head: out = sum_c e^(m_c - M) o_c / sum_c e^(m_c - M) d_c.
#include "common.hpp"

namespace fathom {

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = kAttnThreads / kWave;
constexpr int kChunk = 128;  // row-list positions per workgroup
constexpr int kMaxSinkLocal = 1024;
constexpr int kPart = kD + 2;  // per chunk: m, d, o[D]

static inline int attn_chunks(int k, int n_sink, int n_local) {
  return (n_sink + n_local + k + kChunk - 1) / kChunk;
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

__global__ __launch_bounds__(kAttnThreads) void attn_chunk_kernel(const void* __restrict__ q, fathom_dtype qdt,
                                                                  const uint16_t* __restrict__ Krows,
                                                                  const uint16_t* __restrict__ Vrows, int64_t ld_tok,
                                                                  int64_t ld_unit, const int64_t* __restrict__ n,
                                                                  int G, const int32_t* __restrict__ idx, int k,
                                                                  int n_sink, int n_local, float sm_scale, int S,
                                                                  float* __restrict__ ws, uint32_t* __restrict__ st) {
  __shared__ int32_t rows[kChunk];  // row of each chunk position, -1: none
  __shared__ float pz[kChunk];      // logits, then exp(z - m)
  __shared__ float red[kAttnWaves];
  __shared__ float part[kAttnWaves][kD];
  const int c = blockIdx.x, r = blockIdx.y, u = r / G, h = r % G;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int64_t nu = *(const __attribute__((address_space(1))) int64_t*)(n + u);
  if (nu < 0) {
    if (tid == 0 && c == 0) set_status(st, FATHOM_DEV_BAD_N);
    nu = 0;
  }
  const int64_t ns = n_sink < nu ? n_sink : nu;
  const int64_t l0 = nu - n_local > ns ? nu - n_local : ns;
  const int64_t nloc = nu - l0;
  float* wp = ws + ((int64_t)r * S + c) * kPart;
  // ---- rows of this chunk ----
  if (tid < kChunk) {
    const int64_t p = (int64_t)c * kChunk + tid;
    int32_t row = -1;
    if (p < ns) {
      row = (int32_t)p;
    } else if (p < ns + nloc) {
      row = (int32_t)(l0 + (p - ns));
    } else if (p - ns - nloc < k) {
      const int32_t v = *(const __attribute__((address_space(1))) int32_t*)(idx + (int64_t)r * k + (p - ns - nloc));
      if (v >= ns && v < l0) row = v;
    }
    rows[tid] = row;
  }
  __syncthreads();
  // ---- logits: 4 lanes per row, 32 channels each; 16 rows per wave step ----
  const int cq = lane & 3;
  float qv[32];
  {
    const int64_t qo = ((int64_t)u * G + h) * kD + cq * 32;
#pragma unroll
    for (int x = 0; x < 32; ++x) qv[x] = load_q(q, qdt, qo + x);
  }
  const uint16_t* Ku = Krows + (int64_t)u * ld_unit + cq * 32;
  const uint16_t* Vu = Vrows + (int64_t)u * ld_unit;
#pragma unroll
  for (int step = 0; step < kChunk / (kAttnWaves * 16); ++step) {
    const int slot = (wave * (kChunk / kAttnWaves)) + step * 16 + (lane >> 2);
    const int32_t row = rows[slot];
    float dsum = 0.0f;
    if (row >= 0) {
      uint32_t kk[16];
      const uint16_t* kp = Ku + (int64_t)row * ld_tok;
#pragma unroll
      for (int x = 0; x < 16; ++x) kk[x] = gload_u32(kp + 2 * x);
#pragma unroll
      for (int x = 0; x < 16; ++x) {
        dsum = __fmaf_rn(qv[2 * x], half_bits_to_float((uint16_t)(kk[x] & 0xFFFFu)), dsum);
        dsum = __fmaf_rn(qv[2 * x + 1], half_bits_to_float((uint16_t)(kk[x] >> 16)), dsum);
      }
    }
    dsum = __fadd_rn(dsum, __shfl_xor(dsum, 1, kWave));
    dsum = __fadd_rn(dsum, __shfl_xor(dsum, 2, kWave));
    if (cq == 0) pz[slot] = row >= 0 ? __fmul_rn(dsum, sm_scale) : -__builtin_huge_valf();
  }
  __syncthreads();
  // ---- chunk max and exp-sum ----
  float zm = -__builtin_huge_valf();
  for (int i = tid; i < kChunk; i += kAttnThreads) zm = fmaxf(zm, pz[i]);
  zm = wave_max(zm);
  if (lane == 0) red[wave] = zm;
  __syncthreads();
  zm = red[0];
#pragma unroll
  for (int w = 1; w < kAttnWaves; ++w) zm = fmaxf(zm, red[w]);
  __syncthreads();
  if (zm == -__builtin_huge_valf()) {  // no row in this chunk
    if (tid == 0) {
      gstore_f(wp, zm);
      gstore_f(wp + 1, 0.0f);
    }
    return;
  }
  float den = 0.0f;
  for (int i = tid; i < kChunk; i += kAttnThreads) {
    const float p = rows[i] >= 0 ? expf(__fsub_rn(pz[i], zm)) : 0.0f;
    pz[i] = p;
    den = __fadd_rn(den, p);
  }
  den = wave_sum(den);
  if (lane == 0) red[wave] = den;
  __syncthreads();
  den = 0.0f;
#pragma unroll
  for (int w = 0; w < kAttnWaves; ++w) den = __fadd_rn(den, red[w]);
  // ---- weighted V rows: lane = 2 channels, this wave's share of the chunk ----
  float a0 = 0.0f, a1 = 0.0f;
  constexpr int per = kChunk / kAttnWaves;
  uint32_t vv[per];
#pragma unroll
  for (int x = 0; x < per; ++x) {
    const int32_t row = rows[wave * per + x];
    vv[x] = row >= 0 ? gload_u32(Vu + (int64_t)row * ld_tok + 2 * lane) : 0u;
  }
#pragma unroll
  for (int x = 0; x < per; ++x) {
    const float p = pz[wave * per + x];
    a0 = __fmaf_rn(p, half_bits_to_float((uint16_t)(vv[x] & 0xFFFFu)), a0);
    a1 = __fmaf_rn(p, half_bits_to_float((uint16_t)(vv[x] >> 16)), a1);
  }
  part[wave][2 * lane] = a0;
  part[wave][2 * lane + 1] = a1;
  __syncthreads();
  if (tid < kD) {
    float acc = 0.0f;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) acc = __fadd_rn(acc, part[w][tid]);
    gstore_f(wp + 2 + tid, acc);
  }
  if (tid == 0) {
    gstore_f(wp, zm);
    gstore_f(wp + 1, den);
  }
}

// out = sum_c e^(m_c - M) o_c / sum_c e^(m_c - M) d_c over the chunks of a head.
__global__ __launch_bounds__(kD) void attn_combine_kernel(const float* __restrict__ ws, int S, float* __restrict__ out) {
  const int r = blockIdx.x, tid = threadIdx.x;
  const float* wp = ws + (int64_t)r * S * kPart;
  float M = -__builtin_huge_valf();
  for (int c = 0; c < S; ++c) M = fmaxf(M, gload_f(wp + c * kPart));
  float o = 0.0f;
  if (M > -__builtin_huge_valf()) {
    float den = 0.0f;
    for (int c = 0; c < S; ++c) {
      const float mc = gload_f(wp + c * kPart);
      if (mc == -__builtin_huge_valf()) continue;
      const float e = expf(__fsub_rn(mc, M));
      den = __fmaf_rn(e, gload_f(wp + c * kPart + 1), den);
      o = __fmaf_rn(e, gload_f(wp + c * kPart + 2 + tid), o);
    }
    o = o / den;
  }
  gstore_f(out + (int64_t)r * kD + tid, o);
}

fathom_status launch_sparse_attn(const void* q, fathom_dtype qdt, const uint16_t* Krows, const uint16_t* Vrows,
                                 int64_t ld_tok, int64_t ld_unit, const int64_t* n, int U, int G,
                                 const int32_t* idx, int k, int n_sink, int n_local, float sm_scale, float* out,
                                 void* ws, uint32_t* st, hipStream_t s) {
  if (U == 0) return FATHOM_OK;
  int S = attn_chunks(k, n_sink, n_local);
  if (S < 1) S = 1;
  float* w = reinterpret_cast<float*>(ws);
  hipLaunchKernelGGL(attn_chunk_kernel, dim3((unsigned)S, (unsigned)(U * G)), dim3(kAttnThreads), 0, s, q, qdt,
                     Krows, Vrows, ld_tok, ld_unit, n, G, idx, k, n_sink, n_local, sm_scale, S, w, st);
  hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)(U * G)), dim3(kD), 0, s, w, S, out);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

int attn_max_sink_local() { return kMaxSinkLocal; }

}  // namespace fathom
