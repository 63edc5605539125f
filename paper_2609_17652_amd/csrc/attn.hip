// fathom_sparse_attn: Sec. 2 (top-k decoding) -- exact attention of each
// query head over sink + local + its top-k rows, with fp16 K/V rows resident
// in HBM and fp32 arithmetic.
//
// One workgroup per (unit, head).  The selected row list is built in LDS
// (sink, local, then the top-k entries that fall between them); each wave
// takes every 4th row: 64 lanes x 2 channels read a 256-byte K row with one
// coalesced 4-byte load per lane, a wave sum gives the logit; after the
// block max and exp-sum, each wave accumulates its rows' V contributions for
// its 2 channels per lane and the waves' partials are added in LDS.
#include "common.hpp"

namespace fathom {

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = kAttnThreads / kWave;
constexpr int kMaxSinkLocal = 1024;

__global__ __launch_bounds__(kAttnThreads) void sparse_attn_kernel(const void* __restrict__ q, fathom_dtype qdt,
                                                                   const uint16_t* __restrict__ Krows,
                                                                   const uint16_t* __restrict__ Vrows,
                                                                   int64_t ld_tok, int64_t ld_unit,
                                                                   const int64_t* __restrict__ n, int G,
                                                                   const int32_t* __restrict__ idx, int k,
                                                                   int n_sink, int n_local, float sm_scale,
                                                                   float* __restrict__ out, uint32_t* __restrict__ st) {
  extern __shared__ char smem[];
  const int cap = n_sink + n_local + k;
  int32_t* rows = reinterpret_cast<int32_t*>(smem);
  float* z = reinterpret_cast<float*>(smem + sizeof(int32_t) * cap);
  __shared__ float red[kAttnWaves];
  __shared__ float part[kAttnWaves][kD];
  __shared__ int wcnt[kAttnWaves];

  const int r = blockIdx.x, u = r / G, h = r % G;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int64_t nu = n[u];
  if (nu < 0) {
    if (tid == 0) set_status(st, FATHOM_DEV_BAD_N);
    nu = 0;
  }
  const int64_t ns = n_sink < nu ? n_sink : nu;
  const int64_t l0 = nu - n_local > ns ? nu - n_local : ns;
  // ---- row list: sink, local, then idx entries inside [ns, l0) ----
  const int nfixed = (int)(ns + (nu - l0));
  for (int i = tid; i < nfixed; i += kAttnThreads) rows[i] = i < ns ? i : (int32_t)(l0 + (i - ns));
  int m = nfixed;
  const int32_t* ih = idx ? idx + (int64_t)r * k : nullptr;
  for (int base = 0; base < k; base += kAttnThreads) {
    const int e = base + tid;
    int32_t v = -1;
    if (e < k) v = ih[e];
    const bool keep = e < k && v >= ns && v < l0;
    const uint64_t bm = __ballot(keep);
    if (lane == 0) wcnt[wave] = __popcll(bm);
    __syncthreads();
    int off = m;
    int tot = 0;
    for (int w = 0; w < kAttnWaves; ++w) {
      if (w < wave) off += wcnt[w];
      tot += wcnt[w];
    }
    const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    if (keep) rows[off + __popcll(bm & lt)] = v;
    m += tot;
    __syncthreads();
  }
  float* o = out + (int64_t)r * kD;
  if (m == 0) {
    for (int c = tid; c < kD; c += kAttnThreads) o[c] = 0.0f;
    return;
  }
  // ---- logits ----
  const int64_t qo = ((int64_t)u * G + h) * kD + 2 * lane;
  const float q0 = load_q(q, qdt, qo), q1 = load_q(q, qdt, qo + 1);
  const uint16_t* Ku = Krows + (int64_t)u * ld_unit;
  const uint16_t* Vu = Vrows + (int64_t)u * ld_unit;
  float zmax = -3.402823466e38f;
  for (int i = wave; i < m; i += kAttnWaves) {
    const uint32_t kk = *reinterpret_cast<const uint32_t*>(Ku + (int64_t)rows[i] * ld_tok + 2 * lane);
    const float k0 = half_bits_to_float((uint16_t)(kk & 0xFFFFu)), k1 = half_bits_to_float((uint16_t)(kk >> 16));
    const float d = wave_sum(__fmaf_rn(q1, k1, __fmul_rn(q0, k0)));
    const float zi = __fmul_rn(d, sm_scale);
    if (lane == 0) z[i] = zi;
    zmax = fmaxf(zmax, zi);
  }
  if (lane == 0) red[wave] = zmax;
  __syncthreads();
  zmax = red[0];
  for (int w = 1; w < kAttnWaves; ++w) zmax = fmaxf(zmax, red[w]);
  __syncthreads();
  // ---- softmax weights and denominator ----
  float den = 0.0f;
  for (int i = tid; i < m; i += kAttnThreads) {
    const float p = expf(z[i] - zmax);
    z[i] = p;
    den += p;
  }
  den = wave_sum(den);
  if (lane == 0) red[wave] = den;
  __syncthreads();
  den = 0.0f;
  for (int w = 0; w < kAttnWaves; ++w) den += red[w];
  // ---- weighted V rows ----
  float a0 = 0.0f, a1 = 0.0f;
  for (int i = wave; i < m; i += kAttnWaves) {
    const uint32_t vv = *reinterpret_cast<const uint32_t*>(Vu + (int64_t)rows[i] * ld_tok + 2 * lane);
    const float p = z[i];
    a0 = __fmaf_rn(p, half_bits_to_float((uint16_t)(vv & 0xFFFFu)), a0);
    a1 = __fmaf_rn(p, half_bits_to_float((uint16_t)(vv >> 16)), a1);
  }
  part[wave][2 * lane] = a0;
  part[wave][2 * lane + 1] = a1;
  __syncthreads();
  if (tid < kD) {
    float acc = 0.0f;
    for (int w = 0; w < kAttnWaves; ++w) acc += part[w][tid];
    o[tid] = acc / den;
  }
}

fathom_status launch_sparse_attn(const void* q, fathom_dtype qdt, const uint16_t* Krows, const uint16_t* Vrows,
                                 int64_t ld_tok, int64_t ld_unit, const int64_t* n, int U, int G,
                                 const int32_t* idx, int k, int n_sink, int n_local, float sm_scale, float* out,
                                 uint32_t* st, hipStream_t s) {
  if (U == 0) return FATHOM_OK;
  const size_t lds = (size_t)(n_sink + n_local + k) * 8;
  hipLaunchKernelGGL(sparse_attn_kernel, dim3((unsigned)(U * G)), dim3(kAttnThreads), lds, s, q, qdt, Krows, Vrows,
                     ld_tok, ld_unit, n, G, idx, k, n_sink, n_local, sm_scale, out, st);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

int attn_max_sink_local() { return kMaxSinkLocal; }

}  // namespace fathom
