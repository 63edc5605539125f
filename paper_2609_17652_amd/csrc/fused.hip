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
constexpr int kGrp = 8;           // consecutive blocks per wave step: one 64-byte line per plane row
constexpr int kSub = kFW * kGrp;  // 32 blocks per weight-setup sub-tile
constexpr int kRange = 4 * kSub;  // 128 blocks per workgroup in the full pass
constexpr int kFlush = 256;       // re-score when this many survivors are queued
constexpr int kQueue = kFlush + kSub * kBlockTokens;
constexpr int kMaxDw = kD / 4;    // z' dwords for 128 active channels
constexpr int kMaxCells = kD * kPlanes;
constexpr int kSampleGroups = 64; // at most this many sampled groups (512 blocks) per row
constexpr int kSelThreads = 1024;
constexpr int kSelCap = 16384;    // LDS composites in the select kernel
constexpr float kNegInf = -__builtin_huge_valf();

// Per-unit read plan, built once per call: byte offsets (from the unit's plane
// base) of the plane rows the proxy reads, in active-channel order.
struct Plan {
  uint32_t off[kD][4];       // rows of planes 0..3 of active channel a; planes >= t repeat plane t-1
  uint32_t cell[kMaxCells];  // rows of every plane read (p < t), for the L2 prefetch
  uint32_t tpack[kMaxDw];    // depth of channel 4d+k in byte k
  uint32_t zinit[kMaxDw];    // 2^(4-t) in byte k: the constant part of z'
  int32_t A, ncells, pad[62];
};

struct FusedWs {
  float* tau;       // [R] threshold on exact scores (-inf: every eligible key is kept)
  uint32_t* cnt;    // [R] survivors appended
  uint64_t* cand;   // [R][cap] composites (score_key << 32 | ~index)
  float* sample;    // [R][s_groups * 512] proxies of sampled keys
  Plan* plan;       // [U]
  int cap;
  int64_t s_gstride;  // sample every s_gstride-th group of 8 blocks
  int64_t s_groups;   // sampled groups per row
};

static inline size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

static inline int fused_cap(int k) {
  const int c = 2 * k + 2048;
  return c < kSelCap ? c : kSelCap;
}

static inline void fused_geometry(int64_t nb_cap, int64_t* gstride, int64_t* sgroups) {
  const int64_t ng = (nb_cap + kGrp - 1) / kGrp;
  int64_t s = (ng + kSampleGroups - 1) / kSampleGroups;
  if (s < 2) s = 2;
  *gstride = s;
  *sgroups = (ng + s - 1) / s;
}

size_t fused_ws_bytes(int R, int U, int64_t nb_cap, int k) {
  int64_t s, sg;
  fused_geometry(nb_cap > 0 ? nb_cap : 1, &s, &sg);
  return a256((size_t)R * 4) + a256((size_t)R * 4) + a256((size_t)R * fused_cap(k) * 8) +
         a256((size_t)R * sg * kGrp * kBlockTokens * 4) + a256((size_t)U * sizeof(Plan));
}

static FusedWs fused_carve(void* ws, int R, int U, int64_t nb_cap, int k) {
  FusedWs w;
  fused_geometry(nb_cap > 0 ? nb_cap : 1, &w.s_gstride, &w.s_groups);
  w.cap = fused_cap(k);
  char* p = reinterpret_cast<char*>(ws);
  w.tau = reinterpret_cast<float*>(p); p += a256((size_t)R * 4);
  w.cnt = reinterpret_cast<uint32_t*>(p); p += a256((size_t)R * 4);
  w.cand = reinterpret_cast<uint64_t*>(p); p += a256((size_t)R * w.cap * 8);
  w.sample = reinterpret_cast<float*>(p); p += a256((size_t)R * w.s_groups * kGrp * kBlockTokens * 4);
  w.plan = reinterpret_cast<Plan*>(p);
  (void)U;
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
  uint32_t w8[kSub][kMaxDw][G];     // packed int8 weights
  float hdelta[kSub][G];            // delta / 2
  float ebound[kSub][G];            // error bound (inf: no bound, every key survives)
  float tau[G];
  uint32_t queue[kQueue];
  int nact;
  int qcount;
};

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return lane == 0 ? 0ull : (~0ull >> (64 - lane)); }

// Wave-uniform reads through the constant address space are scalar (SMEM)
// loads straight into SGPRs.  Neither the store nor the plan is written while
// a scan runs.
struct Words8 {
  uint64_t w[kGrp];
};
typedef __attribute__((address_space(4))) const uint64_t cu64;
typedef __attribute__((address_space(4))) const uint32_t cu32;
typedef __attribute__((ext_vector_type(4))) unsigned int v4u;
typedef __attribute__((address_space(4))) const v4u cu4;
typedef __attribute__((ext_vector_type(16))) unsigned int v16u;
typedef __attribute__((address_space(4))) const v16u cv16;
__device__ __forceinline__ uint64_t sload64(const void* p) { return *(cu64*)(p); }
__device__ __forceinline__ uint32_t sload32(const void* p) { return *(cu32*)(p); }
__device__ __forceinline__ v4u sload128(const void* p) { return *(cu4*)(p); }
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const char*>(((uint64_t)hi << 32) | lo);
}
// The plane words of the 8 blocks of a group from one row; a group that runs
// past nb_cap (the last one, when nb_cap % 8 != 0) reads only words inside it.
template <bool FULL>
__device__ __forceinline__ Words8 sload_words(const char* row, int64_t nleft) {
  row = uniform_ptr(row);
  Words8 w;
  if constexpr (FULL) {
    const v16u v = *(cv16*)(row);
#pragma unroll
    for (int g = 0; g < kGrp; ++g) w.w[g] = ((uint64_t)v[2 * g + 1] << 32) | v[2 * g];
  } else {
#pragma unroll
    for (int g = 0; g < kGrp; ++g) {
      w.w[g] = 0ull;
      if (g < nleft) w.w[g] = sload64(row + 8 * g);
    }
  }
  return w;
}

// One plane of one channel (byte K of the z' dword) for the 8 blocks of a
// group: lanes whose key has the bit set (the plane word is the lane mask)
// OR in the plane's value; the sign plane ORs 0xF0 where the bit is clear.
// EXEC is saved and restored inside the statement; SCC is clobbered (the
// compiler must not keep a carry or compare result live across it).
template <int K, int P>
__device__ __forceinline__ void or_plane(uint32_t (&z)[kGrp], const Words8& w) {
  uint64_t sv;
  constexpr uint32_t c = P == 0 ? (0xF0u << (8 * K)) : ((8u >> (P > 0 ? P - 1 : 0)) << (8 * K));
  if (P == 0) {
    asm volatile(
        "s_mov_b64 %8, exec\n\t"
        "s_andn2_b64 exec, %8, %9\n\tv_or_b32 %0, %17, %0\n\t"
        "s_andn2_b64 exec, %8, %10\n\tv_or_b32 %1, %17, %1\n\t"
        "s_andn2_b64 exec, %8, %11\n\tv_or_b32 %2, %17, %2\n\t"
        "s_andn2_b64 exec, %8, %12\n\tv_or_b32 %3, %17, %3\n\t"
        "s_andn2_b64 exec, %8, %13\n\tv_or_b32 %4, %17, %4\n\t"
        "s_andn2_b64 exec, %8, %14\n\tv_or_b32 %5, %17, %5\n\t"
        "s_andn2_b64 exec, %8, %15\n\tv_or_b32 %6, %17, %6\n\t"
        "s_andn2_b64 exec, %8, %16\n\tv_or_b32 %7, %17, %7\n\t"
        "s_mov_b64 exec, %8"
        : "+v"(z[0]), "+v"(z[1]), "+v"(z[2]), "+v"(z[3]), "+v"(z[4]), "+v"(z[5]), "+v"(z[6]), "+v"(z[7]),
          "=&s"(sv)
        : "s"(w.w[0]), "s"(w.w[1]), "s"(w.w[2]), "s"(w.w[3]), "s"(w.w[4]), "s"(w.w[5]), "s"(w.w[6]), "s"(w.w[7]),
          "i"(c)
        : "scc");
  } else {
    asm volatile(
        "s_mov_b64 %8, exec\n\t"
        "s_and_b64 exec, %8, %9\n\tv_or_b32 %0, %17, %0\n\t"
        "s_and_b64 exec, %8, %10\n\tv_or_b32 %1, %17, %1\n\t"
        "s_and_b64 exec, %8, %11\n\tv_or_b32 %2, %17, %2\n\t"
        "s_and_b64 exec, %8, %12\n\tv_or_b32 %3, %17, %3\n\t"
        "s_and_b64 exec, %8, %13\n\tv_or_b32 %4, %17, %4\n\t"
        "s_and_b64 exec, %8, %14\n\tv_or_b32 %5, %17, %5\n\t"
        "s_and_b64 exec, %8, %15\n\tv_or_b32 %6, %17, %6\n\t"
        "s_and_b64 exec, %8, %16\n\tv_or_b32 %7, %17, %7\n\t"
        "s_mov_b64 exec, %8"
        : "+v"(z[0]), "+v"(z[1]), "+v"(z[2]), "+v"(z[3]), "+v"(z[4]), "+v"(z[5]), "+v"(z[6]), "+v"(z[7]),
          "=&s"(sv)
        : "s"(w.w[0]), "s"(w.w[1]), "s"(w.w[2]), "s"(w.w[3]), "s"(w.w[4]), "s"(w.w[5]), "s"(w.w[6]), "s"(w.w[7]),
          "i"(c)
        : "scc");
  }
}

// z' byte K of one channel for a group: its t plane rows (the plan repeats row
// t-1 for planes >= t, so the four loads are unconditional and hit one line).
template <int K, bool FULL>
__device__ __forceinline__ void gather_channel(uint32_t (&z)[kGrp], int t, const char* base, const Plan* plan,
                                               int a, int64_t nleft) {
  const v4u o = sload128(&plan->off[a][0]);
  {
    const Words8 w0 = sload_words<FULL>(base + o.x, nleft);
    const Words8 w1 = sload_words<FULL>(base + o.y, nleft);  // row of plane 0 again when t == 1
    or_plane<K, 0>(z, w0);
    if (t > 1) or_plane<K, 1>(z, w1);
  }
  if (t > 2) {
    const Words8 w2 = sload_words<FULL>(base + o.z, nleft);
    const Words8 w3 = sload_words<FULL>(base + o.w, nleft);
    or_plane<K, 2>(z, w2);
    if (t > 3) or_plane<K, 3>(z, w3);
  }
}

// ---------------------------------------------------------------- plan
// One workgroup of 128 threads per unit.
__global__ __launch_bounds__(kD) void fused_plan_kernel(FusedArgs a) {
  __shared__ int act[kD];
  __shared__ int wc[2];
  __shared__ int cstart[kD + 1];
  const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  Plan* pl = a.ws.plan + u;
  int t = a.depths[(int64_t)u * kD + tid];
  t = t > kPlanes ? kPlanes : t;
  const bool on = t > 0;
  const uint64_t m = __ballot(on);
  if (lane == 0) wc[wave] = __popcll(m);
  __syncthreads();
  if (on) act[(wave == 1 ? wc[0] : 0) + __popcll(m & lanemask_lt(lane))] = tid | (t << 8);
  const int A = wc[0] + wc[1];
  __syncthreads();
  const uint32_t rowb = (uint32_t)(a.nb_cap * 8);  // bytes per plane row
  if (tid < A) {
    const int j = act[tid] & 0xFF, tt = act[tid] >> 8;
#pragma unroll
    for (int p = 0; p < 4; ++p) pl->off[tid][p] = (uint32_t)(j * kPlanes + (p < tt ? p : tt - 1)) * rowb;
  } else {
#pragma unroll
    for (int p = 0; p < 4; ++p) pl->off[tid][p] = 0u;  // row 0 of the unit: valid, never ORed
  }
  // prefix of depths for the cell list
  if (tid == 0) {
    int c = 0;
    for (int x = 0; x < A; ++x) {
      cstart[x] = c;
      c += act[x] >> 8;
    }
    cstart[A] = c;
    pl->A = A;
    pl->ncells = c;
  }
  __syncthreads();
  if (tid < A) {
    const int j = act[tid] & 0xFF, tt = act[tid] >> 8;
    for (int p = 0; p < tt; ++p) pl->cell[cstart[tid] + p] = (uint32_t)(j * kPlanes + p) * rowb;
  }
  if (tid < kMaxDw) {
    uint32_t tp = 0u, zi = 0u;
    for (int k2 = 0; k2 < 4; ++k2) {
      const int x = 4 * tid + k2;
      if (x < A) {
        const int tt = act[x] >> 8;
        tp |= (uint32_t)tt << (8 * k2);
        zi |= (8u >> (tt - 1)) << (8 * k2);
      }
    }
    pl->tpack[tid] = tp;
    pl->zinit[tid] = zi;
  }
}

// Unit-level LDS setup: active channels and fp32 queries per active channel.
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
  __syncthreads();
}

// Weights of the kSub blocks of a sub-tile (block indices from blk_of; -1 or
// >= nbu: unused): 8 threads per block, each owning whole dwords of 4 channels.
template <int G, typename BlkOf>
__device__ void weight_setup(FusedSmem<G>& sm, const FusedArgs& a, int u, int64_t nbu, BlkOf blk_of) {
  constexpr int TPB = kFT / kSub;  // threads per block
  const int tid = threadIdx.x;
  const int blk = tid / TPB, sl = tid % TPB;
  const int A = sm.nact, AD = (A + 3) >> 2;
  const int64_t b = blk_of(blk);
  const bool valid = b >= 0 && b < nbu;
  const uint16_t* Su = a.scales + (int64_t)u * kD * a.nb_cap;
  float mx[G];
#pragma unroll
  for (int h = 0; h < G; ++h) mx[h] = 0.0f;
  bool finite = true;
  if (valid) {
    for (int d = sl; d < AD; d += TPB) {
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
    for (int o = TPB / 2; o >= 1; o >>= 1) mx[h] = fmaxf(mx[h], __shfl_xor(mx[h], o, TPB));
  int fin = finite ? 1 : 0;
#pragma unroll
  for (int o = TPB / 2; o >= 1; o >>= 1) fin &= __shfl_xor(fin, o, TPB);
  float delta[G], inv[G];
  bool ok[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    int e;
    (void)frexpf(mx[h], &e);  // mx in [2^(e-1), 2^e)
    ok[h] = fin && (mx[h] >= 0x1p-100f || mx[h] == 0.0f);
    const int ee = e < -100 ? -100 : e;
    delta[h] = ldexpf(1.0f, ee - 7);  // |w| / delta < 128
    inv[h] = ldexpf(1.0f, 7 - ee);
  }
  float eb[G];
#pragma unroll
  for (int h = 0; h < G; ++h) eb[h] = 0.0f;
  if (valid) {
    for (int d = sl; d < AD; d += TPB) {
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
    for (int o = TPB / 2; o >= 1; o >>= 1) eb[h] = __fadd_rn(eb[h], __shfl_xor(eb[h], o, TPB));
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

// Touch the plane lines of a group (one 4-byte load per row, 64 rows per
// instruction) so they are in L2 when the scalar loads ask for them; the
// returned value only keeps the loads alive.
__device__ __forceinline__ uint32_t prefetch_group(const char* base, const Plan* plan, int ncells, bool any) {
  uint32_t acc = 0u;
  if (any) {
    const int lane = threadIdx.x & 63;
    for (int c = lane; c < ncells; c += kWave) acc ^= *reinterpret_cast<const uint32_t*>(base + plan->cell[c]);
  }
  return acc;
}

// Proxy sums of the 8 blocks of a group for all G heads (lane = key):
// acc[g][h] = sum_j w8_j z'_j for block g.
template <int G, bool FULL>
__device__ __forceinline__ void proxy_group_impl(const FusedSmem<G>& sm, const Plan* plan, const char* base,
                                                 int64_t nleft, int blk0, int acc[kGrp][G]) {
  const int A = sm.nact, AD = (A + 3) >> 2;
#pragma unroll
  for (int g = 0; g < kGrp; ++g)
#pragma unroll
    for (int h = 0; h < G; ++h) acc[g][h] = 0;
  for (int d = 0; d < AD; ++d) {
    const uint32_t tp = sload32(&plan->tpack[d]);
    const uint32_t zi = sload32(&plan->zinit[d]);
    uint32_t z[kGrp];
#pragma unroll
    for (int g = 0; g < kGrp; ++g) z[g] = zi;
    gather_channel<0, FULL>(z, (int)(tp & 0xFF), base, plan, 4 * d, nleft);
    if ((tp >> 8) & 0xFF) gather_channel<1, FULL>(z, (int)((tp >> 8) & 0xFF), base, plan, 4 * d + 1, nleft);
    if ((tp >> 16) & 0xFF) gather_channel<2, FULL>(z, (int)((tp >> 16) & 0xFF), base, plan, 4 * d + 2, nleft);
    if (tp >> 24) gather_channel<3, FULL>(z, (int)(tp >> 24), base, plan, 4 * d + 3, nleft);
#pragma unroll
    for (int g = 0; g < kGrp; ++g) {
#pragma unroll
      for (int h = 0; h < G; ++h)
        acc[g][h] = __builtin_amdgcn_sdot4((int)z[g], (int)sm.w8[blk0 + g][d][h], acc[g][h], false);
    }
  }
}

template <int G>
__device__ __forceinline__ void proxy_group(const FusedSmem<G>& sm, const FusedArgs& a, const Plan* plan,
                                            const char* base, int64_t gb, int blk0, int acc[kGrp][G]) {
  if (gb + kGrp <= a.nb_cap)
    proxy_group_impl<G, true>(sm, plan, base, kGrp, blk0, acc);
  else
    proxy_group_impl<G, false>(sm, plan, base, a.nb_cap - gb, blk0, acc);
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
// Each workgroup: 4 sampled groups (one per wave) of the unit.
template <int G>
__global__ __launch_bounds__(kFT) void fused_sample_kernel(FusedArgs a) {
  __shared__ FusedSmem<G> sm;
  const int u = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  const int64_t nbu = (nu + kBlockTokens - 1) / kBlockTokens;
  const Plan* plan = a.ws.plan + u;
  const char* base = reinterpret_cast<const char*>(a.planes + (int64_t)u * kD * kPlanes * a.nb_cap);
  const int64_t sg = (int64_t)blockIdx.x * kFW + wave;  // sampled group index
  const int64_t gb = sg * a.ws.s_gstride * kGrp;        // its first block
  const bool mine = sg < a.ws.s_groups && gb < nbu;
  const uint32_t pf = prefetch_group(base + gb * 8, plan, sload32(&plan->ncells), mine);
  unit_setup<G>(sm, a, u);
  weight_setup<G>(sm, a, u, nbu, [&](int blk) {
    const int64_t s2 = (int64_t)blockIdx.x * kFW + blk / kGrp;
    return s2 < a.ws.s_groups ? s2 * a.ws.s_gstride * kGrp + blk % kGrp : (int64_t)-1;
  });
  __syncthreads();
  if (sg >= a.ws.s_groups) return;
  const int blk0 = wave * kGrp;
  int acc[kGrp][G];
  if (gb < nbu) proxy_group<G>(sm, a, plan, base + gb * 8, gb, blk0, acc);
  asm volatile("" ::"v"(pf));
#pragma unroll
  for (int g = 0; g < kGrp; ++g) {
    const int64_t b = gb + g;
    const int64_t i = b * kBlockTokens + lane;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      // the proxy itself (exact in fp32): tau only steers how many keys are
      // re-scored; the survivor count, not tau, guarantees the result
      float v = kNegInf;
      if (b < nbu && i >= lo && i < hi && sm.ebound[blk0 + g][h] <= 3.402823466e38f)
        v = __fmul_rn(sm.hdelta[blk0 + g][h], (float)acc[g][h]);
      a.ws.sample[((int64_t)u * G + h) * a.ws.s_groups * (kGrp * kBlockTokens) + (sg * kGrp + g) * kBlockTokens +
                  lane] = v;
    }
  }
}

// ---------------------------------------------------------------- pass 2
// tau = the m-th largest sampled proxy, m ~ 1.25 k * (sampled / eligible) + 16;
// tau = -inf when the row has no more eligible keys than the survivor buffer holds.
__global__ __launch_bounds__(kSelThreads) void fused_tau_kernel(FusedArgs a, int G) {
  extern __shared__ uint32_t keys[];  // the row's sample as order-preserving keys (0 = unusable)
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
  const float* smp = a.ws.sample + (int64_t)r * a.ws.s_groups * (kGrp * kBlockTokens);
  const int ns = (int)(a.ws.s_groups * kGrp * kBlockTokens);
  if (tid == 0) s_total = 0u;
  __syncthreads();
  uint32_t c = 0;
  for (int i = tid; i < ns; i += kSelThreads) {
    const float v = smp[i];
    const bool use = v > kNegInf;
    keys[i] = use ? (score_key(v) | 1u) : 0u;  // keep 0 free: NaN proxies do not occur
    c += use;
  }
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
    for (int i = tid; i < ns; i += kSelThreads) {
      const uint32_t key = keys[i];
      if (key && (key & mask) == prefix) atomicAdd(&hist[(key >> shifts[pass]) & dm], 1u);
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
    const uint32_t key = s_prefix & ~1u;  // the low bit was forced on: round the key down
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
  const Plan* plan = a.ws.plan + u;
  const char* base = reinterpret_cast<const char*>(a.planes + (int64_t)u * kD * kPlanes * a.nb_cap);
  const int ncells = (int)sload32(&plan->ncells);
  // L2 prefetch of this wave's first group
  uint32_t pf = prefetch_group(base + (b0 + wave * kGrp) * 8, plan, ncells, b0 + wave * kGrp < nbu);
  unit_setup<G>(sm, a, u);
  if (tid < G) sm.tau[tid] = a.ws.tau[u * G + tid];
  for (int s0 = 0; s0 < kRange; s0 += kSub) {
    const int64_t sbase = b0 + s0;
    if (sbase >= nbu) break;
    __syncthreads();  // previous sub-tile's weights and queue are consumed
    weight_setup<G>(sm, a, u, nbu, [&](int blk) { return sbase + blk; });
    __syncthreads();
    const int64_t gb = sbase + wave * kGrp;
    if (gb < nbu) {
      const int blk0 = wave * kGrp;
      int acc[kGrp][G];
      proxy_group<G>(sm, a, plan, base + gb * 8, gb, blk0, acc);
      asm volatile("" ::"v"(pf));
      const int64_t gnext = gb + kSub;  // prefetch this wave's next group
      pf = prefetch_group(base + gnext * 8, plan, ncells, s0 + kSub < kRange && gnext < nbu);
#pragma unroll
      for (int g = 0; g < kGrp; ++g) {
        const int64_t b = gb + g;
        const int64_t i = b * kBlockTokens + lane;
        const bool elig = b < nbu && i >= lo && i < hi;
        int hm = 0;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float p = __fmul_rn(sm.hdelta[blk0 + g][h], (float)acc[g][h]);
          const float ub = __fadd_rn(p, sm.ebound[blk0 + g][h]);
          if (elig && (ub >= sm.tau[h] || sm.tau[h] == kNegInf || ub != ub)) hm |= 1 << h;
        }
        const uint64_t any = __ballot(hm != 0);
        if (any) {
          int basep = 0;
          const int leader = __ffsll((unsigned long long)any) - 1;
          if (lane == leader) basep = atomicAdd(&sm.qcount, __popcll(any));
          basep = __shfl(basep, leader, kWave);
          if (hm)
            sm.queue[basep + __popcll(any & lanemask_lt(lane))] =
                (uint32_t)((b - b0) * kBlockTokens + lane) | ((uint32_t)hm << 16);
        }
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
  asm volatile("" ::"v"(pf));
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
                            hipFuncAttributeMaxDynamicSharedMemorySize, kSelCap * 8) != hipSuccess ||
        hipFuncSetAttribute(reinterpret_cast<const void*>(&fused_tau_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, kSampleGroups * kGrp * kBlockTokens * 4) !=
            hipSuccess)
      return FATHOM_ERR_HIP;
    attr = true;
  }
  hipLaunchKernelGGL(fused_plan_kernel, dim3(U), dim3(kD), 0, s, fa);
  dim3 gs((unsigned)((fa.ws.s_groups + kFW - 1) / kFW), (unsigned)U);
  hipLaunchKernelGGL(fused_sample_kernel<G>, gs, dim3(kFT), 0, s, fa);
  const size_t tau_lds = (size_t)fa.ws.s_groups * kGrp * kBlockTokens * 4;
  hipLaunchKernelGGL(fused_tau_kernel, dim3(R), dim3(kSelThreads), tau_lds, s, fa, G);
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
  fa.ws = fused_carve(ws, U * G, U, nb_cap, k);
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
