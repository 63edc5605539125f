// fathom_scan_topk: the decode-step scan + top-k of Sec. 3.2-3.3 and Sec. 2,
// fused so that no score array is written.
//
// The exact result is defined by the documented fp32 scores (exact
// dequantisation, fma(q, khat, acc) over active channels ascending) and the
// (score desc, index asc) order.  To avoid computing those scores for every
// key, each key first gets a cheap proxy with a rigorous error bound:
//   score = sum_j (w_j / 2) z'_j,  w_j = q_hj a16_bj / 8,
//   z'_j  = 2 (c^(t) - 2^(t-1)) 2^(4-t) + 2^(4-t)   (odd multiple, |z'| <= 15),
//   proxy = (delta / 2) sum_j w8_j z'_j  with w8_j = rne(w_j / delta) in int8,
//   delta = a power of two per (block, head), so the proxy is exact in fp32;
//   |score - proxy| <= E = sum_j |w_j - delta w8_j| max|z'_j| / 2 (+ slack for
//   the fp32 rounding of the exact scores).
// Per lane (= key), z' of 4 channels is one dword built from the plane words
// with one EXEC-masked OR per plane bit (the word is the lane mask), and one
// v_dot4_i32_i8 per head folds it in.  Keys whose bound reaches the row's
// threshold tau are re-scored exactly; those with score >= tau are kept.
//
// Passes: (1) proxies of a strided sample of blocks; (2) per row, tau = a rank
// statistic of the sample chosen so that ~1.25 k keys are expected above it; (3) full proxy pass + exact re-scoring of the survivors;
// (4) per row, the k best survivors in order.  If fewer than k keys reach tau
// (or the survivor buffer overflows), pass (4) recomputes the row exactly on
// its own (FATHOM_DEV_TOPK_FALLBACK).  The result never depends on tau.
#include "common.hpp"

namespace fathom {

constexpr int kFT = 256;          // threads per workgroup (4 waves)
constexpr int kFW = kFT / kWave;
constexpr int kSub = 16;          // blocks per weight-setup sub-tile (4 per wave)
constexpr int kRange = 64;        // blocks per workgroup in the full pass
constexpr int kFlush = 256;       // re-score when this many survivors are queued
constexpr int kQueue = kFlush + kSub * kBlockTokens;
constexpr int kMaxDw = kD / 4;    // z' dwords for 128 active channels
constexpr int kSampleBlocks = 512;  // at most this many sampled blocks per row
constexpr int kSelThreads = 1024;
constexpr int kSelCap = 16384;    // LDS composites in the select kernel
constexpr float kNegInf = -__builtin_huge_valf();

struct FusedWs {
  float* tau;       // [R] threshold on exact scores (-inf: every eligible key is kept)
  uint32_t* cnt;    // [R] survivors appended
  uint64_t* cand;   // [R][cap] composites (score_key << 32 | ~index)
  float* sample;    // [R][s_cap] proxies of sampled keys
  int cap;
  int64_t s_stride; // sample every s_stride-th block
  int64_t s_blocks; // sampled blocks per row
};

static inline size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

static inline int fused_cap(int k) {
  const int c = 2 * k + 2048;
  return c < kSelCap ? c : kSelCap;
}

static inline void fused_geometry(int64_t nb_cap, int64_t* stride, int64_t* sblocks) {
  int64_t s = (nb_cap + kSampleBlocks - 1) / kSampleBlocks;
  if (s < 8) s = 8;
  *stride = s;
  *sblocks = (nb_cap + s - 1) / s;
}

size_t fused_ws_bytes(int R, int64_t nb_cap, int k) {
  int64_t s, sb;
  fused_geometry(nb_cap > 0 ? nb_cap : 1, &s, &sb);
  return a256((size_t)R * 4) + a256((size_t)R * 4) + a256((size_t)R * fused_cap(k) * 8) +
         a256((size_t)R * sb * kBlockTokens * 4);
}

static FusedWs fused_carve(void* ws, int R, int64_t nb_cap, int k) {
  FusedWs w;
  fused_geometry(nb_cap > 0 ? nb_cap : 1, &w.s_stride, &w.s_blocks);
  w.cap = fused_cap(k);
  char* p = reinterpret_cast<char*>(ws);
  w.tau = reinterpret_cast<float*>(p); p += a256((size_t)R * 4);
  w.cnt = reinterpret_cast<uint32_t*>(p); p += a256((size_t)R * 4);
  w.cand = reinterpret_cast<uint64_t*>(p); p += a256((size_t)R * w.cap * 8);
  w.sample = reinterpret_cast<float*>(p);
  return w;
}

struct FusedArgs {
  const uint64_t* planes;
  const uint16_t* scales;
  const int64_t* n;
  int64_t nb_cap;
  const void* q;
  fathom_dtype qdt;
  const uint8_t* depths;
  int64_t lo, tail;
  int k;
  FusedWs ws;
  uint32_t* st;
};

template <int G>
struct FusedSmem {
  int act[kD];                      // j | (t << 8), active channels ascending
  float qa[kD][G];                  // fp32 query of active channel a, head h
  uint32_t zinit[kMaxDw];           // constant bits of z' per dword
  uint32_t w8[kSub][kMaxDw][G];     // packed int8 weights
  float hdelta[kSub][G];            // delta / 2
  float ebound[kSub][G];            // error bound (inf: no bound, every key survives)
  float tau[G];
  uint32_t queue[kQueue];
  int nact;
  int qcount;
};

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return lane == 0 ? 0ull : (~0ull >> (64 - lane)); }

// Wave-uniform read of a plane word through the constant address space, so it
// is a scalar (SMEM) load straight into SGPRs.  The store is never written
// while a scan runs.
typedef __attribute__((address_space(4))) const uint64_t cu64;
__device__ __forceinline__ uint64_t sload(const uint64_t* p) { return *(cu64*)(p); }

// z' bits of one channel (byte K of the dword) from its t plane words: one
// EXEC-masked OR per plane, EXEC saved and restored inside the statement.
template <int K>
__device__ __forceinline__ uint32_t gather_channel(uint32_t z, int t, const uint64_t* __restrict__ Pj,
                                                   int64_t pstride) {
  uint64_t sv;
  const uint64_t w0 = sload(Pj);
  if (t == 1) {
    asm volatile(
        "s_mov_b64 %1, exec\n\t"
        "s_andn2_b64 exec, %1, %2\n\t"
        "v_or_b32 %0, %3, %0\n\t"
        "s_mov_b64 exec, %1"
        : "+v"(z), "=&s"(sv)
        : "s"(w0), "i"(0xF0u << (8 * K)));
    return z;
  }
  const uint64_t w1 = sload(Pj + pstride);
  if (t == 2) {
    asm volatile(
        "s_mov_b64 %1, exec\n\t"
        "s_andn2_b64 exec, %1, %2\n\t"
        "v_or_b32 %0, %4, %0\n\t"
        "s_and_b64 exec, %1, %3\n\t"
        "v_or_b32 %0, %5, %0\n\t"
        "s_mov_b64 exec, %1"
        : "+v"(z), "=&s"(sv)
        : "s"(w0), "s"(w1), "i"(0xF0u << (8 * K)), "i"(8u << (8 * K)));
    return z;
  }
  const uint64_t w2 = sload(Pj + 2 * pstride);
  if (t == 3) {
    asm volatile(
        "s_mov_b64 %1, exec\n\t"
        "s_andn2_b64 exec, %1, %2\n\t"
        "v_or_b32 %0, %5, %0\n\t"
        "s_and_b64 exec, %1, %3\n\t"
        "v_or_b32 %0, %6, %0\n\t"
        "s_and_b64 exec, %1, %4\n\t"
        "v_or_b32 %0, %7, %0\n\t"
        "s_mov_b64 exec, %1"
        : "+v"(z), "=&s"(sv)
        : "s"(w0), "s"(w1), "s"(w2), "i"(0xF0u << (8 * K)), "i"(8u << (8 * K)), "i"(4u << (8 * K)));
    return z;
  }
  const uint64_t w3 = sload(Pj + 3 * pstride);
  asm volatile(
      "s_mov_b64 %1, exec\n\t"
      "s_andn2_b64 exec, %1, %2\n\t"
      "v_or_b32 %0, %6, %0\n\t"
      "s_and_b64 exec, %1, %3\n\t"
      "v_or_b32 %0, %7, %0\n\t"
      "s_and_b64 exec, %1, %4\n\t"
      "v_or_b32 %0, %8, %0\n\t"
      "s_and_b64 exec, %1, %5\n\t"
      "v_or_b32 %0, %9, %0\n\t"
      "s_mov_b64 exec, %1"
      : "+v"(z), "=&s"(sv)
      : "s"(w0), "s"(w1), "s"(w2), "s"(w3), "i"(0xF0u << (8 * K)), "i"(8u << (8 * K)), "i"(4u << (8 * K)),
        "i"(2u << (8 * K)));
  return z;
}

// Unit-level setup: active channels, fp32 queries per active channel, z' constants.
template <int G>
__device__ void unit_setup(FusedSmem<G>& sm, const FusedArgs& a, int u) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ int wc[2];
  int t = 0;
  if (tid < kD) {
    t = a.depths[(int64_t)u * kD + tid];
    t = t > kPlanes ? kPlanes : t;
  }
  const bool on = tid < kD && t > 0;
  const uint64_t m = __ballot(on);
  if (tid < kD && lane == 0) wc[wave] = __popcll(m);
  __syncthreads();
  if (on) sm.act[(wave == 1 ? wc[0] : 0) + __popcll(m & lanemask_lt(lane))] = tid | (t << 8);
  if (tid == 0) {
    sm.nact = wc[0] + wc[1];
    sm.qcount = 0;
  }
  __syncthreads();
  const int A = sm.nact;
  for (int x = tid; x < A * G; x += kFT) {
    const int ai = x / G, h = x % G;
    const int j = sm.act[ai] & 0xFF;
    sm.qa[ai][h] = load_q(a.q, a.qdt, ((int64_t)u * G + h) * kD + j);
  }
  for (int d = tid; d < kMaxDw; d += kFT) {
    uint32_t z = 0;
    for (int k = 0; k < 4; ++k) {
      const int ai = 4 * d + k;
      if (ai < A) z |= (8u >> ((sm.act[ai] >> 8) - 1)) << (8 * k);  // 2^(4-t)
    }
    sm.zinit[d] = z;
  }
  __syncthreads();
}

// Weights of up to kSub blocks (block indices from blk_of): 16 threads per
// block, each owning whole dwords of 4 channels.
template <int G, typename BlkOf>
__device__ void weight_setup(FusedSmem<G>& sm, const FusedArgs& a, int u, int64_t nbu, BlkOf blk_of) {
  const int tid = threadIdx.x;
  const int blk = tid >> 4, sl = tid & 15;
  const int A = sm.nact, AD = (A + 3) >> 2;
  const int64_t b = blk_of(blk);
  const bool valid = b >= 0 && b < nbu;
  const uint16_t* Su = a.scales + (int64_t)u * kD * a.nb_cap;
  // pass 1: max |w| per head over the block's active channels
  float mx[G];
#pragma unroll
  for (int h = 0; h < G; ++h) mx[h] = 0.0f;
  bool finite = true;
  if (valid) {
    for (int d = sl; d < AD; d += 16) {
      for (int k = 0; k < 4; ++k) {
        const int ai = 4 * d + k;
        if (ai >= A) break;
        const int j = sm.act[ai] & 0xFF;
        const float af = half_bits_to_float(Su[(int64_t)j * a.nb_cap + b]);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float w = __fmul_rn(__fmul_rn(sm.qa[ai][h], af), 0.125f);
          if (!(fabsf(w) <= 3.402823466e38f)) finite = false;
          mx[h] = fmaxf(mx[h], fabsf(w));
        }
      }
    }
  }
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) mx[h] = fmaxf(mx[h], __shfl_xor(mx[h], o, 16));
  // __any over the 16 lanes of the block
  int fin = finite ? 1 : 0;
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) fin &= __shfl_xor(fin, o, 16);
  float delta[G], inv[G];
  bool ok[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    int e;
    (void)frexpf(mx[h], &e);  // mx in [2^(e-1), 2^e)
    ok[h] = fin && mx[h] >= 0x1p-100f;
    if (mx[h] == 0.0f) ok[h] = fin;
    const int ee = e < -100 ? -100 : e;
    delta[h] = ldexpf(1.0f, ee - 7);  // |w| / delta < 128
    inv[h] = ldexpf(1.0f, 7 - ee);
  }
  // pass 2: quantise, pack, error bound
  float eb[G];
#pragma unroll
  for (int h = 0; h < G; ++h) eb[h] = 0.0f;
  if (valid) {
    for (int d = sl; d < AD; d += 16) {
      uint32_t pk[G];
#pragma unroll
      for (int h = 0; h < G; ++h) pk[h] = 0u;
      for (int k = 0; k < 4; ++k) {
        const int ai = 4 * d + k;
        if (ai >= A) break;
        const int j = sm.act[ai] & 0xFF, t = sm.act[ai] >> 8;
        const float zmax = t == 4 ? 15.0f : t == 3 ? 14.0f : t == 2 ? 12.0f : 8.0f;
        const float af = half_bits_to_float(Su[(int64_t)j * a.nb_cap + b]);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float w = __fmul_rn(__fmul_rn(sm.qa[ai][h], af), 0.125f);
          float r = rintf(__fmul_rn(w, inv[h]));
          r = fminf(fmaxf(r, -127.0f), 127.0f);
          const float err = fabsf(__fsub_rn(w, __fmul_rn(r, delta[h])));
          eb[h] = __fmaf_rn(err, zmax, eb[h]);
          pk[h] |= ((uint32_t)(int)r & 0xFFu) << (8 * k);
        }
      }
#pragma unroll
      for (int h = 0; h < G; ++h) sm.w8[blk][d][h] = pk[h];
    }
  }
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) eb[h] = __fadd_rn(eb[h], __shfl_xor(eb[h], o, 16));
  if (sl == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      sm.hdelta[blk][h] = ok[h] ? 0.5f * delta[h] : 0.0f;
      // half the sum, inflated for the rounding of this sum and of the exact scores
      sm.ebound[blk][h] = ok[h] ? __fmaf_rn(eb[h], 0.5f * (1.0f + 0x1p-10f), __fmul_rn(delta[h], (float)A * 0x1p-6f))
                                : __builtin_huge_valf();
    }
  }
}

// Proxy of the wave's block b for all G heads (lane = key): acc = sum_j w8_j z'_j.
template <int G>
__device__ __forceinline__ void proxy_block(const FusedSmem<G>& sm, const FusedArgs& a, int u, int blk, int64_t b,
                                            int acc[G]) {
  const int A = sm.nact, AD = (A + 3) >> 2;
  const uint64_t* Pu = a.planes + (int64_t)u * kD * kPlanes * a.nb_cap + b;
  const int64_t ps = a.nb_cap;
#pragma unroll
  for (int h = 0; h < G; ++h) acc[h] = 0;
  for (int d = 0; d < AD; ++d) {
    uint32_t z = sm.zinit[d];
    const int a0 = 4 * d;
    {
      const int e = __builtin_amdgcn_readfirstlane(sm.act[a0]);
      z = gather_channel<0>(z, e >> 8, Pu + (int64_t)(e & 0xFF) * kPlanes * ps, ps);
    }
    if (a0 + 1 < A) {
      const int e = __builtin_amdgcn_readfirstlane(sm.act[a0 + 1]);
      z = gather_channel<1>(z, e >> 8, Pu + (int64_t)(e & 0xFF) * kPlanes * ps, ps);
    }
    if (a0 + 2 < A) {
      const int e = __builtin_amdgcn_readfirstlane(sm.act[a0 + 2]);
      z = gather_channel<2>(z, e >> 8, Pu + (int64_t)(e & 0xFF) * kPlanes * ps, ps);
    }
    if (a0 + 3 < A) {
      const int e = __builtin_amdgcn_readfirstlane(sm.act[a0 + 3]);
      z = gather_channel<3>(z, e >> 8, Pu + (int64_t)(e & 0xFF) * kPlanes * ps, ps);
    }
#pragma unroll
    for (int h = 0; h < G; ++h) acc[h] = __builtin_amdgcn_sdot4((int)z, (int)sm.w8[blk][d][h], acc[h], false);
  }
}

// Exact documented scores of key (block b, bit) for all G heads, read from the store.
template <int G>
__device__ __forceinline__ void exact_scores(const int* act, int A, const float (*qa)[G], const FusedArgs& a, int u,
                                             int64_t b, int bit, float acc[G]) {
  const uint64_t* Pu = a.planes + (int64_t)u * kD * kPlanes * a.nb_cap + b;
  const uint16_t* Su = a.scales + (int64_t)u * kD * a.nb_cap + b;
#pragma unroll
  for (int h = 0; h < G; ++h) acc[h] = 0.0f;
  for (int ai = 0; ai < A; ++ai) {
    const int e = act[ai];
    const int j = e & 0xFF, t = e >> 8;
    const float af = half_bits_to_float(Su[(int64_t)j * a.nb_cap]);
    const uint64_t* Pj = Pu + (int64_t)j * kPlanes * a.nb_cap;
    uint32_t c = 0;
    for (int p = 0; p < t; ++p) c = 2u * c + (uint32_t)((Pj[(int64_t)p * a.nb_cap] >> bit) & 1ull);
    const float y = (float)c + (0.5f - (float)(1 << (t - 1)));
    const float khat = __fmul_rn(y, __fmul_rn(af, __uint_as_float((uint32_t)(128 - t) << 23)));
#pragma unroll
    for (int h = 0; h < G; ++h) acc[h] = __fmaf_rn(qa[ai][h], khat, acc[h]);
  }
}

__device__ __forceinline__ void row_window(const FusedArgs& a, int u, int64_t* nu, int64_t* lo, int64_t* hi,
                                           bool flag) {
  int64_t v = a.n[u];
  if (v < 0 || v > a.nb_cap * kBlockTokens) {
    if (flag) set_status(a.st, FATHOM_DEV_BAD_N);
    v = 0;
  }
  *nu = v;
  *lo = a.lo;
  *hi = v - a.tail;
  if (*hi < *lo) *hi = *lo;
}

// ---------------------------------------------------------------- pass 1
template <int G>
__global__ __launch_bounds__(kFT) void fused_sample_kernel(FusedArgs a) {
  __shared__ FusedSmem<G> sm;
  const int u = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  const int64_t nbu = (nu + kBlockTokens - 1) / kBlockTokens;
  const int64_t sb0 = (int64_t)blockIdx.x * kSub;  // first sampled block index of this workgroup
  unit_setup<G>(sm, a, u);
  weight_setup<G>(sm, a, u, nbu, [&](int blk) { return (sb0 + blk) * a.ws.s_stride; });
  __syncthreads();
  for (int r = 0; r < kSub / kFW; ++r) {
    const int blk = wave + kFW * r;
    const int64_t sb = sb0 + blk;
    if (sb >= a.ws.s_blocks) break;
    const int64_t b = sb * a.ws.s_stride;
    const int64_t i = b * kBlockTokens + lane;
    float lb[G];
    if (b < nbu) {
      int acc[G];
      proxy_block<G>(sm, a, u, blk, b, acc);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        // the proxy itself (exact in fp32): tau only steers how many keys are
        // re-scored; the survivor count, not tau, guarantees the result
        lb[h] = __fmul_rn(sm.hdelta[blk][h], (float)acc[h]);
        if (!(i >= lo && i < hi) || !(sm.ebound[blk][h] <= 3.402823466e38f)) lb[h] = kNegInf;
      }
    } else {
#pragma unroll
      for (int h = 0; h < G; ++h) lb[h] = kNegInf;
    }
#pragma unroll
    for (int h = 0; h < G; ++h)
      a.ws.sample[((int64_t)u * G + h) * a.ws.s_blocks * kBlockTokens + sb * kBlockTokens + lane] = lb[h];
  }
}

// ---------------------------------------------------------------- pass 2
// tau = the m-th largest sampled proxy, m ~ 1.25 k * (sampled / eligible) + 16;
// tau = -inf when the row has no more eligible keys than the survivor buffer holds.
__global__ __launch_bounds__(kSelThreads) void fused_tau_kernel(FusedArgs a, int G) {
  __shared__ uint32_t hist[2048];
  __shared__ uint32_t s_prefix, s_mask, s_above;
  __shared__ int s_need, s_digit;
  __shared__ uint32_t s_total;
  __shared__ uint32_t part[kSelThreads / kWave];
  const int r = blockIdx.x, u = r / G, tid = threadIdx.x;
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  const int64_t m_e = hi - lo;
  if (m_e <= a.ws.cap) {
    if (tid == 0) {
      a.ws.tau[r] = kNegInf;
      a.ws.cnt[r] = 0u;
    }
    return;
  }
  const float* smp = a.ws.sample + (int64_t)r * a.ws.s_blocks * kBlockTokens;
  const int64_t ns = a.ws.s_blocks * kBlockTokens;
  // count sampled eligible keys with a usable proxy
  if (tid == 0) s_total = 0u;
  __syncthreads();
  uint32_t c = 0;
  for (int64_t i = tid; i < ns; i += kSelThreads) c += smp[i] > kNegInf;
  atomicAdd(&s_total, c);
  __syncthreads();
  const int64_t m_s = s_total;
  if (m_s == 0) {
    if (tid == 0) {
      a.ws.tau[r] = kNegInf;
      a.ws.cnt[r] = 0u;
    }
    return;
  }
  int64_t m = (5 * (int64_t)a.k * m_s + 4 * m_e - 1) / (4 * m_e) + 16;
  if (m > m_s) m = m_s;
  if (tid == 0) {
    s_prefix = 0u;
    s_mask = 0u;
    s_need = (int)m;
  }
  const int shifts[3] = {21, 10, 0}, bits[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    for (int b = tid; b < 2048; b += kSelThreads) hist[b] = 0u;
    __syncthreads();
    const uint32_t prefix = s_prefix, mask = s_mask, dm = (1u << bits[pass]) - 1u;
    for (int64_t i = tid; i < ns; i += kSelThreads) {
      const float v = smp[i];
      if (v > kNegInf) {
        const uint32_t key = score_key(v);
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shifts[pass]) & dm], 1u);
      }
    }
    __syncthreads();
    find_crossing(hist, (int)dm + 1, (uint32_t)s_need, part, &s_digit, &s_above);
    if (tid == 0) {
      s_prefix = prefix | ((uint32_t)s_digit << shifts[pass]);
      s_mask = mask | (dm << shifts[pass]);
      s_need = s_need - (int)s_above;
    }
    __syncthreads();
  }
  if (tid == 0) {
    const uint32_t key = s_prefix;
    const uint32_t bitsf = (key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key;
    a.ws.tau[r] = __uint_as_float(bitsf);
    a.ws.cnt[r] = 0u;
  }
}

// ---------------------------------------------------------------- pass 3
template <int G>
__device__ void rescore_queue(FusedSmem<G>& sm, const FusedArgs& a, int u, int64_t base_block) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int count = sm.qcount;
  for (int e0 = wave * kWave; e0 < count; e0 += kFT) {
    const int e = e0 + lane;
    uint32_t ent = 0u;
    if (e < count) ent = sm.queue[e];
    const int off = (int)(ent & 0xFFFFu), hm = (int)(ent >> 16);
    const int64_t i = base_block * kBlockTokens + off;
    float s[G];
#pragma unroll
    for (int h = 0; h < G; ++h) s[h] = 0.0f;
    if (hm) exact_scores<G>(sm.act, sm.nact, sm.qa, a, u, i / kBlockTokens, (int)(i % kBlockTokens), s);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float tau = sm.tau[h];
      const bool keep = ((hm >> h) & 1) && (s[h] >= tau || tau == kNegInf);
      const uint64_t bm = __ballot(keep);
      if (bm) {
        const int r = u * G + h;
        uint32_t basep = 0;
        if (lane == __ffsll((unsigned long long)bm) - 1) basep = atomicAdd(&a.ws.cnt[r], (uint32_t)__popcll(bm));
        basep = __shfl(basep, __ffsll((unsigned long long)bm) - 1, kWave);
        if (keep) {
          const uint32_t pos = basep + (uint32_t)__popcll(bm & lanemask_lt(lane));
          if (pos < (uint32_t)a.ws.cap)
            a.ws.cand[(int64_t)r * a.ws.cap + pos] =
                ((uint64_t)score_key(s[h]) << 32) | (uint64_t)(~(uint32_t)i);
        }
      }
    }
  }
}

template <int G>
__global__ __launch_bounds__(kFT) void fused_full_kernel(FusedArgs a) {
  __shared__ FusedSmem<G> sm;
  const int u = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, blockIdx.x == 0 && tid == 0);
  const int64_t nbu = (nu + kBlockTokens - 1) / kBlockTokens;
  const int64_t b0 = (int64_t)blockIdx.x * kRange;
  if (b0 >= nbu || b0 * kBlockTokens >= hi || (b0 + kRange) * kBlockTokens <= lo) return;
  unit_setup<G>(sm, a, u);
  if (tid < G) sm.tau[tid] = a.ws.tau[u * G + tid];
  for (int s0 = 0; s0 < kRange; s0 += kSub) {
    const int64_t sbase = b0 + s0;
    if (sbase >= nbu) break;
    __syncthreads();  // previous sub-tile's weights and queue are consumed
    weight_setup<G>(sm, a, u, nbu, [&](int blk) { return sbase + blk; });
    __syncthreads();
    for (int r = 0; r < kSub / kFW; ++r) {
      const int blk = wave + kFW * r;
      const int64_t b = sbase + blk;
      if (b >= nbu) break;
      int acc[G];
      proxy_block<G>(sm, a, u, blk, b, acc);
      const int64_t i = b * kBlockTokens + lane;
      const bool elig = i >= lo && i < hi;
      int hm = 0;
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float p = __fmul_rn(sm.hdelta[blk][h], (float)acc[h]);
        const float ub = __fadd_rn(p, sm.ebound[blk][h]);
        if (elig && (ub >= sm.tau[h] || sm.tau[h] == kNegInf || ub != ub)) hm |= 1 << h;
      }
      const uint64_t any = __ballot(hm != 0);
      if (any) {
        int basep = 0;
        const int leader = __ffsll((unsigned long long)any) - 1;
        if (lane == leader) basep = atomicAdd(&sm.qcount, __popcll(any));
        basep = __shfl(basep, leader, kWave);
        if (hm) sm.queue[basep + __popcll(any & lanemask_lt(lane))] = (uint32_t)((b - b0) * kBlockTokens + lane) |
                                                                      ((uint32_t)hm << 16);
      }
    }
    __syncthreads();
    const bool last = s0 + kSub >= kRange || sbase + kSub >= nbu;
    if (sm.qcount >= kFlush || last) {
      rescore_queue<G>(sm, a, u, b0);
      __syncthreads();
      if (tid == 0) sm.qcount = 0;
    }
  }
}

// ---------------------------------------------------------------- pass 4
__device__ void bitonic_desc(uint64_t* buf, int P) {
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < P; i += nt) {
        const int j = i ^ stride;
        if (j > i) {
          const bool desc = (i & size) == 0;
          const uint64_t x = buf[i], y = buf[j];
          if (desc ? (x < y) : (x > y)) {
            buf[i] = y;
            buf[j] = x;
          }
        }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ float key_to_score(uint32_t key) {
  if (key == 0u) return __uint_as_float(0x7FC00000u);
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

template <int G>
__global__ __launch_bounds__(kSelThreads) void fused_select_kernel(FusedArgs a, int32_t* __restrict__ idx,
                                                                   float* __restrict__ val) {
  extern __shared__ uint64_t buf[];
  __shared__ int act[kD];         // active channels and queries for the exact fallback
  __shared__ float qa[kD][G];
  __shared__ int nact;
  __shared__ int s_count;
  __shared__ uint64_t s_thr;
  const int r = blockIdx.x, u = r / G, h = r % G, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  const int k = a.k;
  const uint32_t C = a.ws.cnt[r];
  const float tau = a.ws.tau[r];
  const bool fallback = C > (uint32_t)a.ws.cap || (C < (uint32_t)k && tau != kNegInf);
  int count;
  if (!fallback) {
    count = (int)C;
    int P = 1;
    while (P < count) P <<= 1;
    for (int i = tid; i < P; i += kSelThreads) buf[i] = i < count ? a.ws.cand[(int64_t)r * a.ws.cap + i] : 0ull;
    __syncthreads();
    bitonic_desc(buf, P);
  } else {
    // exact recomputation of the row: a streaming top-k over all eligible keys
    if (tid == 0) set_status(a.st, FATHOM_DEV_TOPK_FALLBACK);
    {
      __shared__ int wc[2];
      int t = 0;
      if (tid < kD) {
        t = a.depths[(int64_t)u * kD + tid];
        t = t > kPlanes ? kPlanes : t;
      }
      const bool on = tid < kD && t > 0;
      const uint64_t m = __ballot(on);
      if (tid < kD && lane == 0) wc[wave] = __popcll(m);
      __syncthreads();
      if (on) act[(wave == 1 ? wc[0] : 0) + __popcll(m & lanemask_lt(lane))] = tid | (t << 8);
      if (tid == 0) nact = wc[0] + wc[1];
      __syncthreads();
      for (int x = tid; x < nact * G; x += kSelThreads) {
        const int ai = x / G, hh = x % G;
        qa[ai][hh] = load_q(a.q, a.qdt, ((int64_t)u * G + hh) * kD + (act[ai] & 0xFF));
      }
    }
    if (tid == 0) {
      s_count = 0;
      s_thr = 0ull;
    }
    __syncthreads();
    const int nwaves = kSelThreads / kWave;
    const int64_t bfirst = lo / kBlockTokens, bend = (hi + kBlockTokens - 1) / kBlockTokens;
    for (int64_t bb = bfirst; bb < bend; bb += nwaves) {
      const int64_t b = bb + wave;
      const int64_t i = b * kBlockTokens + lane;
      const bool elig = b < bend && i >= lo && i < hi;
      uint64_t comp = 0ull;
      if (elig) {
        float s[G];
        exact_scores<G>(act, nact, qa, a, u, b, lane, s);
        comp = ((uint64_t)score_key(s[h]) << 32) | (uint64_t)(~(uint32_t)i);
      }
      const uint64_t thr = s_thr;
      const bool add = elig && comp > thr;
      const uint64_t bm = __ballot(add);
      if (bm) {
        int basep = 0;
        const int leader = __ffsll((unsigned long long)bm) - 1;
        if (lane == leader) basep = atomicAdd(&s_count, __popcll(bm));
        basep = __shfl(basep, leader, kWave);
        if (add) buf[basep + __popcll(bm & lanemask_lt(lane))] = comp;
      }
      __syncthreads();
      if (s_count > kSelCap - kSelThreads) {  // room for one more round
        bitonic_desc(buf, kSelCap);
        if (tid == 0) {
          s_count = k;
          s_thr = buf[k - 1];
        }
        for (int x = k + tid; x < kSelCap; x += kSelThreads) buf[x] = 0ull;
        __syncthreads();
      }
    }
    count = s_count;
    for (int x = count + tid; x < kSelCap; x += kSelThreads) buf[x] = 0ull;
    __syncthreads();
    bitonic_desc(buf, kSelCap);
  }
  bool shortfall = false;
  for (int x = tid; x < k; x += kSelThreads) {
    const uint64_t c = x < count ? buf[x] : 0ull;
    if (c == 0ull) {
      idx[(int64_t)r * k + x] = -1;
      if (val) val[(int64_t)r * k + x] = __uint_as_float(0x7FC00000u);
      shortfall = true;
    } else {
      idx[(int64_t)r * k + x] = (int32_t)(~(uint32_t)(c & 0xFFFFFFFFull));
      if (val) val[(int64_t)r * k + x] = key_to_score((uint32_t)(c >> 32));
    }
  }
  if (__syncthreads_or(shortfall) && tid == 0) set_status(a.st, FATHOM_DEV_TOPK_SHORT);
}

// nb_cap == 0: every row is empty (n[u] > 0 is out of range for such a store)
__global__ void fused_empty_kernel(const int64_t* __restrict__ n, int G, int k, int32_t* __restrict__ idx,
                                   float* __restrict__ val, uint32_t* __restrict__ st) {
  const int r = blockIdx.x;
  for (int x = threadIdx.x; x < k; x += blockDim.x) {
    idx[(int64_t)r * k + x] = -1;
    if (val) val[(int64_t)r * k + x] = __uint_as_float(0x7FC00000u);
  }
  if (threadIdx.x == 0) set_status(st, FATHOM_DEV_TOPK_SHORT | (n[r / G] != 0 ? FATHOM_DEV_BAD_N : 0u));
}

template <int G>
static fathom_status launch_fused_g(const FusedArgs& fa, int U, int32_t* idx, float* val, hipStream_t s) {
  const int R = U * G;
  static bool attr = false;
  if (!attr) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(&fused_select_kernel<G>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, kSelCap * 8) != hipSuccess)
      return FATHOM_ERR_HIP;
    attr = true;
  }
  dim3 gs((unsigned)((fa.ws.s_blocks + kSub - 1) / kSub), (unsigned)U);
  hipLaunchKernelGGL(fused_sample_kernel<G>, gs, dim3(kFT), 0, s, fa);
  hipLaunchKernelGGL(fused_tau_kernel, dim3(R), dim3(kSelThreads), 0, s, fa, G);
  dim3 gf((unsigned)((fa.nb_cap + kRange - 1) / kRange), (unsigned)U);
  hipLaunchKernelGGL(fused_full_kernel<G>, gf, dim3(kFT), 0, s, fa);
  hipLaunchKernelGGL(fused_select_kernel<G>, dim3(R), dim3(kSelThreads), (size_t)kSelCap * 8, s, fa, idx, val);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

fathom_status launch_scan_topk_fused(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U,
                                     int64_t nb_cap, const void* q, fathom_dtype qdt, int G, const uint8_t* depths,
                                     int k, int64_t lo, int64_t tail, int32_t* idx, float* val, void* ws,
                                     uint32_t* st, hipStream_t s) {
  if (U == 0) return FATHOM_OK;
  if (nb_cap == 0) {
    hipLaunchKernelGGL(fused_empty_kernel, dim3(U * G), dim3(256), 0, s, n, G, k, idx, val, st);
    FATHOM_LAUNCH_CHECK();
    return FATHOM_OK;
  }
  FusedArgs fa;
  fa.planes = planes;
  fa.scales = scales;
  fa.n = n;
  fa.nb_cap = nb_cap;
  fa.q = q;
  fa.qdt = qdt;
  fa.depths = depths;
  fa.lo = lo;
  fa.tail = tail;
  fa.k = k;
  fa.ws = fused_carve(ws, U * G, nb_cap, k);
  fa.st = st;
  switch (G) {
    case 1: return launch_fused_g<1>(fa, U, idx, val, s);
    case 2: return launch_fused_g<2>(fa, U, idx, val, s);
    case 3: return launch_fused_g<3>(fa, U, idx, val, s);
    case 4: return launch_fused_g<4>(fa, U, idx, val, s);
    case 5: return launch_fused_g<5>(fa, U, idx, val, s);
    case 6: return launch_fused_g<6>(fa, U, idx, val, s);
    case 7: return launch_fused_g<7>(fa, U, idx, val, s);
    default: return launch_fused_g<8>(fa, U, idx, val, s);
  }
}

}  // namespace fathom
