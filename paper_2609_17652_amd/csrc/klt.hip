// KLT-rotated store: Sec. 3.5 (basis rule).  The rotated variant stores the
// planes of (k - mu) V, mu the mean and V the orthonormal eigenbasis of the
// covariance of a unit's calibration keys, and allocates depths with
// g_j = sum_h ((q_h V)_j)^2 lambda_j -- i.e. the unchanged pack, depth
// allocation and scan run on rotated keys, rotated queries and var = lambda.
//
// fathom_klt_calibrate (one-time, per unit; the unit's own keys calibrate):
//   klt_mean_kernel   kCalChunks token chunks per unit, fp64 channel sums.
//   klt_cov_kernel    the same chunks: fp64 sums of centred outer products,
//                     8 x 8 entries per thread, 32-token tiles in LDS.
//   klt_eig_kernel    one 1024-thread workgroup per unit: fixed-order sums of
//                     the chunk partials, then cyclic Jacobi in fp32 with the
//                     matrix and the basis in LDS -- each sweep is 127 rounds
//                     of 64 disjoint rotations (round-robin pairing), applied
//                     to rows, then columns and the basis -- and finally the
//                     columns ordered by eigenvalue (descending) with each
//                     column's largest-magnitude entry made positive.
// fathom_klt_rotate_keys (prefill) and fathom_klt_rotate_q (per step) compute
// in fp32 in a fixed order: d_j = fl(k_j - mu_j) (no mean for q), then for
// j = 0 .. D-1: acc_c = fl(acc_c + fl(d_j V[j][c])), no fused multiply-add, so
// the rotated operands (and every plane, depth and score built from them) are
// reproducible bit for bit.  The rotation is a dense contraction, but the MFMA
// accumulation order is not this one; it runs once per token at prefill.
#include "common.hpp"

namespace fathom {

constexpr int kCalChunks = 32;        // token chunks per unit in the calibration sums
constexpr int kCalThreads = 256;
constexpr int kCovTile = 32;          // tokens per LDS tile in the covariance pass
constexpr int kEigThreads = 1024;
constexpr int kEigPitch = kD + 1;     // LDS row pitch (column sweeps are conflict free)
constexpr int kJacobiSweeps = 12;     // fp32 cyclic Jacobi on 128 x 128 converges in fewer
constexpr int kRotThreads = 256;
constexpr int kRotTile = 64;          // tokens per rotation tile
constexpr int kRotTilesPerWG = 4;
constexpr int kRotPitch = kRotTile + 4;  // transposed tile row: 16-byte aligned, fewer bank conflicts

size_t klt_ws_bytes(int U) {
  const size_t ms = (size_t)U * kCalChunks * kD * sizeof(double);
  const size_t cs = (size_t)U * kCalChunks * kD * kD * sizeof(double);
  return ((ms + 255) & ~(size_t)255) + cs;
}

template <typename KT>
__device__ __forceinline__ float key_at(const KT* p) {
  if constexpr (sizeof(KT) == 4) return *(const __attribute__((address_space(1))) float*)p;
  return half_bits_to_float(*(const __attribute__((address_space(1))) uint16_t*)p);
}

__device__ __forceinline__ void chunk_range(int64_t nu, int c, int64_t* t0, int64_t* t1) {
  const int64_t cs = (nu + kCalChunks - 1) / kCalChunks;
  *t0 = (int64_t)c * cs < nu ? (int64_t)c * cs : nu;
  *t1 = *t0 + cs < nu ? *t0 + cs : nu;
}

// ---------------------------------------------------------------- calibration
template <typename KT>
__global__ __launch_bounds__(kCalThreads) void klt_mean_kernel(const KT* __restrict__ K, int64_t ld_tok,
                                                              int64_t ld_unit, const int64_t* __restrict__ n,
                                                              int64_t n_cap, double* __restrict__ msum,
                                                              uint32_t* __restrict__ st) {
  __shared__ double half2[kD];
  const int c = blockIdx.x, u = blockIdx.y, tid = threadIdx.x;
  const int ch = tid & (kD - 1), hf = tid >> 7;
  const int64_t nu = unit_tokens(n, u, n_cap, (c == 0 && tid == 0) ? st : nullptr);
  int64_t t0, t1;
  chunk_range(nu, c, &t0, &t1);
  const KT* Ku = K + (int64_t)u * ld_unit + ch;
  double s = 0.0;
  int64_t i = t0 + hf;
  for (; i + 14 < t1; i += 16) {  // 8 loads in flight
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = key_at(Ku + (i + 2 * e) * ld_tok);
#pragma unroll
    for (int e = 0; e < 8; ++e) s += (double)v[e];
  }
  for (; i < t1; i += 2) s += (double)key_at(Ku + i * ld_tok);
  if (hf == 1) half2[ch] = s;
  __syncthreads();
  if (hf == 0) msum[((int64_t)u * kCalChunks + c) * kD + ch] = s + half2[ch];
}

template <typename KT>
__global__ __launch_bounds__(kCalThreads) void klt_cov_kernel(const KT* __restrict__ K, int64_t ld_tok,
                                                             int64_t ld_unit, const int64_t* __restrict__ n,
                                                             int64_t n_cap, const double* __restrict__ msum,
                                                             double* __restrict__ cpart) {
  __shared__ double mu[kD];
  __shared__ double tile[kCovTile][kD];
  const int c = blockIdx.x, u = blockIdx.y, tid = threadIdx.x;
  int64_t nu = n[u];
  if (nu < 0 || nu > n_cap) nu = 0;  // flagged by the mean pass
  if (tid < kD) {
    double s = 0.0;
    for (int x = 0; x < kCalChunks; ++x) s += msum[((int64_t)u * kCalChunks + x) * kD + tid];
    mu[tid] = nu > 0 ? s / (double)nu : 0.0;
  }
  __syncthreads();
  int64_t t0, t1;
  chunk_range(nu, c, &t0, &t1);
  const int jb = 8 * (tid >> 4), lb = 8 * (tid & 15);
  double acc[8][8];
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[a][b] = 0.0;
  const KT* Ku = K + (int64_t)u * ld_unit;
  for (int64_t b0 = t0; b0 < t1; b0 += kCovTile) {
    // centred tile (rows past the chunk are zero and add nothing)
    for (int e = tid; e < kCovTile * kD; e += kCalThreads) {
      const int r = e / kD, x = e % kD;
      tile[r][x] = b0 + r < t1 ? (double)key_at(Ku + (b0 + r) * ld_tok + x) - mu[x] : 0.0;
    }
    __syncthreads();
    for (int r = 0; r < kCovTile; ++r) {
      double dj[8], dl[8];
#pragma unroll
      for (int a = 0; a < 8; ++a) {
        dj[a] = tile[r][jb + a];
        dl[a] = tile[r][lb + a];
      }
#pragma unroll
      for (int a = 0; a < 8; ++a)
#pragma unroll
        for (int b = 0; b < 8; ++b) acc[a][b] = __fma_rn(dj[a], dl[b], acc[a][b]);
    }
    __syncthreads();
  }
  double* out = cpart + ((int64_t)u * kCalChunks + c) * kD * kD;
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b) out[(jb + a) * kD + lb + b] = acc[a][b];
}

__global__ __launch_bounds__(kEigThreads) void klt_eig_kernel(const int64_t* __restrict__ n, int64_t n_cap,
                                                             const double* __restrict__ msum,
                                                             const double* __restrict__ cpart,
                                                             float* __restrict__ mu_out, float* __restrict__ V_out,
                                                             float* __restrict__ lam_out) {
  __shared__ float A[kD * kEigPitch];
  __shared__ float V[kD * kEigPitch];
  __shared__ float rc[kD / 2], rs[kD / 2];
  __shared__ int rp[kD / 2], rq[kD / 2];
  const int u = blockIdx.x, tid = threadIdx.x;
  int64_t nu = n[u];
  if (nu < 0 || nu > n_cap) nu = 0;
  const double inv = nu > 0 ? 1.0 / (double)nu : 0.0;
  // ---- covariance and mean from the chunk partials, summed in chunk order ----
  for (int e = tid; e < kD * kD; e += kEigThreads) {
    double s = 0.0;
    for (int x = 0; x < kCalChunks; ++x) s += cpart[((int64_t)u * kCalChunks + x) * kD * kD + e];
    const int j = e / kD, l = e % kD;
    A[j * kEigPitch + l] = (float)(s * inv);
    V[j * kEigPitch + l] = j == l ? 1.0f : 0.0f;
  }
  if (tid < kD) {
    double s = 0.0;
    for (int x = 0; x < kCalChunks; ++x) s += msum[((int64_t)u * kCalChunks + x) * kD + tid];
    mu_out[(int64_t)u * kD + tid] = (float)(s * inv);
  }
  __syncthreads();
  // ---- cyclic Jacobi: rounds of 64 disjoint pairs (circle method on 128 indices) ----
  for (int sweep = 0; sweep < kJacobiSweeps; ++sweep) {
    for (int r = 0; r < kD - 1; ++r) {
      if (tid < kD / 2) {
        const int i = tid;
        const int p = i == 0 ? kD - 1 : (r + i) % (kD - 1);
        const int q = i == 0 ? r : (r - i + (kD - 1)) % (kD - 1);
        const double apq = A[p * kEigPitch + q];
        double c = 1.0, s = 0.0;
        if (apq != 0.0) {
          // the rotation that zeroes a_pq: tau = (a_qq - a_pp) / (2 a_pq),
          // t the smaller root of t^2 + 2 tau t - 1 = 0
          const double tau = ((double)A[q * kEigPitch + q] - (double)A[p * kEigPitch + p]) / (2.0 * apq);
          const double t = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
          c = 1.0 / sqrt(1.0 + t * t);
          s = t * c;
        }
        rc[i] = (float)c;
        rs[i] = (float)s;
        rp[i] = p;
        rq[i] = q;
      }
      __syncthreads();
      // rows p, q: A <- J^T A
      for (int e = tid; e < (kD / 2) * kD; e += kEigThreads) {
        const int i = e / kD, x = e % kD;
        const float c = rc[i], s = rs[i];
        float* ap = &A[rp[i] * kEigPitch + x];
        float* aq = &A[rq[i] * kEigPitch + x];
        const float a = *ap, b = *aq;
        *ap = c * a - s * b;
        *aq = s * a + c * b;
      }
      __syncthreads();
      // columns p, q: A <- A J, V <- V J
      for (int e = tid; e < (kD / 2) * kD; e += kEigThreads) {
        const int i = e / kD, x = e % kD;
        const float c = rc[i], s = rs[i];
        const int p = rp[i], q = rq[i];
        const float a = A[x * kEigPitch + p], b = A[x * kEigPitch + q];
        A[x * kEigPitch + p] = c * a - s * b;
        A[x * kEigPitch + q] = s * a + c * b;
        const float va = V[x * kEigPitch + p], vb = V[x * kEigPitch + q];
        V[x * kEigPitch + p] = c * va - s * vb;
        V[x * kEigPitch + q] = s * va + c * vb;
      }
      __syncthreads();
    }
  }
  // ---- order by eigenvalue (descending, ties by index), fix signs, write ----
  if (tid < kD) {
    const int c = tid;
    const float lc = A[c * kEigPitch + c];
    int rank = 0;
    for (int x = 0; x < kD; ++x) {
      const float lx = A[x * kEigPitch + x];
      rank += (lx > lc) || (lx == lc && x < c);
    }
    int jm = 0;
    float best = -1.0f;
    for (int j = 0; j < kD; ++j) {
      const float a = fabsf(V[j * kEigPitch + c]);
      if (a > best) {
        best = a;
        jm = j;
      }
    }
    const float sg = V[jm * kEigPitch + c] < 0.0f ? -1.0f : 1.0f;
    float* vo = V_out + (int64_t)u * kD * kD;
    for (int j = 0; j < kD; ++j) vo[j * kD + rank] = sg * V[j * kEigPitch + c];
    lam_out[(int64_t)u * kD + rank] = lc;
  }
}

// ---------------------------------------------------------------- rotations
template <typename KT>
__global__ __launch_bounds__(kRotThreads) void klt_rotate_keys_kernel(const KT* __restrict__ K, int64_t ld_tok,
                                                                     int64_t ld_unit, const int64_t* __restrict__ n,
                                                                     int64_t n_cap, const float* __restrict__ mu,
                                                                     const float* __restrict__ V,
                                                                     float* __restrict__ out, int64_t ld_out,
                                                                     uint32_t* __restrict__ st) {
  __shared__ float Vs[kD * kD];
  __shared__ __attribute__((aligned(16))) float dT[kD * kRotPitch];  // [channel][token]
  const int u = blockIdx.y, tid = threadIdx.x;
  const int64_t nu = unit_tokens(n, u, n_cap, (blockIdx.x == 0 && tid == 0) ? st : nullptr);
  const int64_t base = (int64_t)blockIdx.x * kRotTile * kRotTilesPerWG;
  if (base >= nu) return;
  const float* Vu = V + (int64_t)u * kD * kD;
  for (int e = tid; e < kD * kD; e += kRotThreads) Vs[e] = Vu[e];
  const int ch = tid & (kD - 1), hf = tid >> 7;
  const float muc = mu[(int64_t)u * kD + ch];
  const KT* Ku = K + (int64_t)u * ld_unit;
  float* Ou = out + (int64_t)u * ld_out;
  for (int tt = 0; tt < kRotTilesPerWG; ++tt) {
    const int64_t t0 = base + (int64_t)tt * kRotTile;
    if (t0 >= nu) break;
    __syncthreads();  // Vs written / previous tile's reads done
    // centred tile, transposed: thread (ch, hf) takes tokens hf, hf + 2, ...
    for (int r = hf; r < kRotTile; r += 2) {
      const float k = t0 + r < nu ? key_at(Ku + (t0 + r) * ld_tok + ch) : 0.0f;
      dT[ch * kRotPitch + r] = __fsub_rn(k, muc);
    }
    __syncthreads();
    // thread (c = ch, tokens 32 hf .. 32 hf + 31): acc over j ascending
    float acc[kRotTile / 2];
#pragma unroll
    for (int i = 0; i < kRotTile / 2; ++i) acc[i] = 0.0f;
    for (int j = 0; j < kD; ++j) {
      const float v = Vs[j * kD + ch];
      const float4* dr = reinterpret_cast<const float4*>(&dT[j * kRotPitch + 32 * hf]);
#pragma unroll
      for (int i4 = 0; i4 < kRotTile / 8; ++i4) {
        const float4 d = dr[i4];
        acc[4 * i4] = __fadd_rn(acc[4 * i4], __fmul_rn(d.x, v));
        acc[4 * i4 + 1] = __fadd_rn(acc[4 * i4 + 1], __fmul_rn(d.y, v));
        acc[4 * i4 + 2] = __fadd_rn(acc[4 * i4 + 2], __fmul_rn(d.z, v));
        acc[4 * i4 + 3] = __fadd_rn(acc[4 * i4 + 3], __fmul_rn(d.w, v));
      }
    }
#pragma unroll
    for (int i = 0; i < kRotTile / 2; ++i) {
      const int64_t t = t0 + 32 * hf + i;
      if (t < nu) Ou[t * kD + ch] = acc[i];
    }
  }
}

// One workgroup per unit: V and the unit's queries are staged in LDS with all
// loads in flight, then thread (h, c) forms its dot product from LDS.
__global__ __launch_bounds__(kMaxG * kD) void klt_rotate_q_kernel(const void* __restrict__ q, fathom_dtype qdt,
                                                                 int G, const float* __restrict__ V,
                                                                 float* __restrict__ out) {
  __shared__ float4 Vs4[kD * kD / 4];
  __shared__ float qs[kMaxG * kD];
  const int u = blockIdx.x, tid = threadIdx.x, h = tid / kD, c = tid % kD;
  const float4* Vu = reinterpret_cast<const float4*>(V + (int64_t)u * kD * kD);
  float4 r[kD * kD / 4 / (kMaxG * kD)];
#pragma unroll
  for (int x = 0; x < kD * kD / 4 / (kMaxG * kD); ++x) r[x] = Vu[tid + x * kMaxG * kD];
  const int64_t qo = (int64_t)u * G * kD;
  if (h < G) qs[tid] = load_q(q, qdt, qo + tid);
#pragma unroll
  for (int x = 0; x < kD * kD / 4 / (kMaxG * kD); ++x) Vs4[tid + x * kMaxG * kD] = r[x];
  __syncthreads();
  if (h >= G) return;
  const float* Vs = reinterpret_cast<const float*>(Vs4);
  float acc = 0.0f;
  for (int j = 0; j < kD; ++j) acc = __fadd_rn(acc, __fmul_rn(qs[h * kD + j], Vs[j * kD + c]));
  out[qo + tid] = acc;
}

// ---------------------------------------------------------------- launches
fathom_status launch_klt_calibrate(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                   const int64_t* n, int64_t n_cap, int U, float* mu, float* V, float* lam, void* ws,
                                   uint32_t* st, hipStream_t s) {
  if (U == 0) return FATHOM_OK;
  double* msum = reinterpret_cast<double*>(ws);
  const size_t ms = ((size_t)U * kCalChunks * kD * sizeof(double) + 255) & ~(size_t)255;
  double* cpart = reinterpret_cast<double*>(reinterpret_cast<char*>(ws) + ms);
  const dim3 g((unsigned)kCalChunks, (unsigned)U);
  if (kdt == FATHOM_F32) {
    const float* Kf = reinterpret_cast<const float*>(K);
    hipLaunchKernelGGL(klt_mean_kernel<float>, g, dim3(kCalThreads), 0, s, Kf, ld_tok, ld_unit, n, n_cap, msum, st);
    hipLaunchKernelGGL(klt_cov_kernel<float>, g, dim3(kCalThreads), 0, s, Kf, ld_tok, ld_unit, n, n_cap, msum, cpart);
  } else {
    const __half* Kh = reinterpret_cast<const __half*>(K);
    hipLaunchKernelGGL(klt_mean_kernel<__half>, g, dim3(kCalThreads), 0, s, Kh, ld_tok, ld_unit, n, n_cap, msum, st);
    hipLaunchKernelGGL(klt_cov_kernel<__half>, g, dim3(kCalThreads), 0, s, Kh, ld_tok, ld_unit, n, n_cap, msum,
                       cpart);
  }
  hipLaunchKernelGGL(klt_eig_kernel, dim3((unsigned)U), dim3(kEigThreads), 0, s, n, n_cap, msum, cpart, mu, V, lam);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

fathom_status launch_klt_rotate_keys(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                     const int64_t* n, int64_t n_cap, int U, const float* mu, const float* V,
                                     float* out, int64_t ld_out, uint32_t* st, hipStream_t s) {
  if (U == 0 || n_cap == 0) return FATHOM_OK;
  const int64_t per = (int64_t)kRotTile * kRotTilesPerWG;
  const dim3 g((unsigned)((n_cap + per - 1) / per), (unsigned)U);
  if (kdt == FATHOM_F32)
    hipLaunchKernelGGL(klt_rotate_keys_kernel<float>, g, dim3(kRotThreads), 0, s,
                       reinterpret_cast<const float*>(K), ld_tok, ld_unit, n, n_cap, mu, V, out, ld_out, st);
  else
    hipLaunchKernelGGL(klt_rotate_keys_kernel<__half>, g, dim3(kRotThreads), 0, s,
                       reinterpret_cast<const __half*>(K), ld_tok, ld_unit, n, n_cap, mu, V, out, ld_out, st);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

fathom_status launch_klt_rotate_q(const void* q, fathom_dtype qdt, int U, int G, const float* V, float* out,
                                  hipStream_t s) {
  if (U == 0) return FATHOM_OK;
  hipLaunchKernelGGL(klt_rotate_q_kernel, dim3((unsigned)U), dim3(kMaxG * kD), 0, s, q, qdt, G, V, out);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

}  // namespace fathom
