// Shared by the passes of fathom_scan_topk (fused.hip) and its full pass
// (filter.hip): workspace layout, launch geometry, kernel arguments and
// small device helpers.  Not part of the C ABI.
#pragma once

#include "common.hpp"

namespace fathom {

constexpr int kFT = 256;           // threads per workgroup (4 waves)
constexpr int kFW = kFT / kWave;
constexpr int kQB = 4;             // blocks per quad
constexpr int kSQ = 16;            // blocks per superquad at most (8 in the wide full pass)
constexpr int kMaxDw = kD / 4;     // digit dwords (4 channels each)
constexpr int kMaxSl = kD / 16;    // 16-channel slices (one MFMA each)
constexpr int kMaxRg = kD;         // row groups: at most 4 planes x 32 dwords
constexpr int kStP = 65;           // LDS dwords per staged row group (64 lanes + pad)
constexpr int kRing = 3;           // superquads of scales kept for re-scoring
constexpr int kQCap = 64;          // queued candidates per wave at most
constexpr int kSmpW = 8;           // sample proxies kept per (sampled wave, head)
constexpr int kSampleQuads = 64;   // at most this many sampled quads per unit
constexpr int kSmpRow = kSampleQuads * kSmpW;
constexpr int kCntStride = 64;     // survivor counters one 256-byte line apart (device-scope atomics)
constexpr size_t kPlanBytes = 8192;  // workspace slot of a unit's cell plan
constexpr int kPools = 4;          // cell filter: group pools per unit (one per wave of a workgroup)
constexpr int kPoolStride = 32;    // pool counters one 128-byte line apart
constexpr int kSelCap = 16384;     // rows with at most this many eligible keys are computed exactly
constexpr int kThrMax = 1 << 18;   // |S| < 2^17 for A <= 128
constexpr int kNoBound = 1 << 30;  // accumulator start: always (+) or never (-) a candidate
constexpr int kMainWavesTarget = 2048;  // full-pass waves in flight over all units
constexpr int kBackfillUnits = 64;      // from this many units per launch ...
constexpr int kBackfillQpw = 16;        // ... at most this many quads per full-pass wave
constexpr int kNarrow = 3;         // wide-pass classes lie above this
constexpr int64_t kOneNbMax = ((int64_t)1 << 20) - 4096;  // cell filter: byte offsets within a unit's planes (and past them) fit 32 bits
constexpr float kNegInf = -__builtin_huge_valf();

struct FusedWs {
  float* tau;       // [R] threshold on exact scores (-inf: the row is computed exactly)
  uint32_t* cnt;    // [R][kCntStride] word 0: survivors appended to the row's list (counted past its capacity too)
  uint32_t* pool;   // [U][kPools][kPoolStride] word 0: groups taken from the cell filter's pool
  unsigned char* plan;  // [U][kPlanBytes] the cell filter's plan of each unit (built by the sample pass)
  uint64_t* cand;   // [R][lcap] survivors in append order: score_key << 32 | ~index
  uint32_t* uovf;   // [U] from pass 2: (slices of the unit's filter, at least kNarrow + 1 for the wide pass) << 1, 0 = no filter
  float* samp;      // [R][kSmpRow] sampled proxies
  uint32_t* xctl;   // [1 + R] word 1 + r: chunks of row r merged so far (exact rows; word 0 unused)
  uint64_t* part;   // [R][xch][pk] per listed row and chunk: the chunk's top pk composites
  uint32_t* pcnt;   // [R][xch] composites in each partial list
  uint64_t* pmin;   // [R][xch] a lower bound on each full partial list's smallest composite (0: list not full)
  int xch, pk;      // exact pass: chunks per row at most, partial list length
  int cap, lcap;    // rows with at most cap eligible keys are scored directly; survivor list capacity
  int64_t s_stride; // sample every s_stride-th quad
  int s_quads;      // sampled quads per unit
  int qpw;          // full pass: quads per wave (a multiple of 4)
  int64_t nwg;      // full pass: workgroups per unit
};

static inline size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

static inline int fused_cap(int k) {
  const int c = 2 * k + 2048;
  return c < kSelCap ? c : kSelCap;
}
static inline int fused_lcap(int k) { return 2 * fused_cap(k); }

static inline void fused_geometry(int U, int64_t nb_cap, int64_t* stride, int* squads, int* qpw, int64_t* nwg) {
  const int64_t nq = (nb_cap + kQB - 1) / kQB;
  int64_t s = (nq + kSampleQuads - 1) / kSampleQuads;
  if (s < 2) s = 2;
  *stride = s;
  *squads = (int)((nq + s - 1) / s);
  // quads per wave: a multiple of 4 (whole superquads), enough that all units
  // together need about kMainWavesTarget waves
  int64_t per = ((int64_t)U * nq + kMainWavesTarget - 1) / kMainWavesTarget;
  per = (per + 3) & ~(int64_t)3;
  // many units (many resident sessions): their lengths are likely ragged, and
  // short waves let the units' waves backfill each other's slots (16 quads
  // per wave: 0.59 ms against 0.94 ms for 16 ragged sessions); a few long
  // units keep one round of waves (fewer plan set-ups)
  if (U >= kBackfillUnits && per > kBackfillQpw) per = kBackfillQpw;
  if (per < 4) per = 4;
  *qpw = (int)per;
  const int64_t waves = (nq + per - 1) / per;
  *nwg = (waves + kFW - 1) / kFW;
}

// Exact pass geometry: a row's blocks in chunks of kXBlocks (one workgroup
// each, at most kXChunks per row); each chunk keeps its top min(k, chunk keys).
constexpr int kXBlocks = 256;
constexpr int kXKeys = kXBlocks * kBlockTokens;  // 16384 keys per chunk
constexpr int kXChunks = 64;
static inline int exact_chunks(int64_t nb_cap) {
  const int64_t c = (nb_cap + kXBlocks - 1) / kXBlocks;
  return (int)(c < 1 ? 1 : c > kXChunks ? kXChunks : c);
}
static inline int exact_pk(int k) { return k < kXKeys ? k : kXKeys; }
// The head of every chunk's list: its top xs composites.  The merge reads the
// heads, and a chunk's other composites only when its xs-th composite lies
// above the k-th composite of the heads (so a chunk with more than xs of the
// row's top k is read whole).
__host__ __device__ inline int exact_pow2(int k) {  // the merge's sort length
  int p = 2;
  while (p < k) p <<= 1;
  return p;
}
__host__ __device__ inline int exact_split(int k, int nz) {
  int s = (2 * k + nz - 1) / nz;
  if (s < 64) s = 64;
  const int room = (2 * FATHOM_MAX_K - exact_pow2(k)) / nz;  // the heads share LDS with the sorted top k
  if (s > room) s = room;
  return s < k ? s : k;
}

size_t fused_ws_bytes(int R, int U, int64_t nb_cap, int k);

static FusedWs fused_carve(void* ws, int R, int U, int64_t nb_cap, int k) {
  FusedWs w;
  if (nb_cap < 1) nb_cap = 1;
  fused_geometry(U, nb_cap, &w.s_stride, &w.s_quads, &w.qpw, &w.nwg);
  w.cap = fused_cap(k);
  w.lcap = fused_lcap(k);
  char* p = reinterpret_cast<char*>(ws);
  w.tau = reinterpret_cast<float*>(p); p += a256((size_t)R * 4);
  w.cnt = reinterpret_cast<uint32_t*>(p); p += a256((size_t)R * kCntStride * 4);
  w.pool = reinterpret_cast<uint32_t*>(p); p += a256((size_t)U * kPools * kPoolStride * 4);
  w.plan = reinterpret_cast<unsigned char*>(p); p += (size_t)U * kPlanBytes;
  w.cand = reinterpret_cast<uint64_t*>(p); p += a256((size_t)R * w.lcap * 8);
  w.uovf = reinterpret_cast<uint32_t*>(p); p += a256((size_t)U * 4);
  w.samp = reinterpret_cast<float*>(p); p += a256((size_t)R * kSmpRow * 4);
  w.xch = exact_chunks(nb_cap);
  w.pk = exact_pk(k);
  w.xctl = reinterpret_cast<uint32_t*>(p); p += a256((size_t)(1 + R) * 4);
  w.part = reinterpret_cast<uint64_t*>(p); p += a256((size_t)R * w.xch * w.pk * 8);
  w.pcnt = reinterpret_cast<uint32_t*>(p); p += a256((size_t)R * w.xch * 4);
  w.pmin = reinterpret_cast<uint64_t*>(p);
  return w;
}

struct FusedArgs {
  const uint64_t* planes;
  const uint16_t* scales;
  const int64_t* n;
  int64_t nb_cap;
  const void* q;
  fathom_dtype qdt;
  int G;
  const uint8_t* depths;
  int64_t lo, tail;
  int k;
  FusedWs ws;
  uint32_t* st;
  int ccap;  // cells at most of a unit the cell filter takes (64, or 80 when the call's units have 65 to 80 bits)
};

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return lane == 0 ? 0ull : (~0ull >> (64 - lane)); }

// Orders this wave's LDS accesses before its later ones (other lanes).
__device__ __forceinline__ void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Global-memory accesses through the global address space (generic accesses
// would also count against the LDS wait counter).
template <typename T>
__device__ __forceinline__ T gload(const T* p) {
  return *(const __attribute__((address_space(1))) T*)p;
}
template <typename T>
__device__ __forceinline__ void gstore(T* p, T v) {
  *(__attribute__((address_space(1))) T*)p = v;
}
__device__ __forceinline__ uint32_t gatomic_add(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add((__attribute__((address_space(1))) uint32_t*)p, v, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void row_window(const FusedArgs& a, int u, int64_t* nu, int64_t* lo, int64_t* hi,
                                           bool flag) {
  int64_t v = gload(a.n + u);
  if (v < 0 || v > a.nb_cap * kBlockTokens) {
    if (flag) set_status(a.st, FATHOM_DEV_BAD_N);
    v = 0;
  }
  *nu = v;
  *lo = a.lo;
  *hi = v - a.tail;
  if (*hi < *lo) *hi = *lo;
}

// Lane moves within rows of 16 (rotations and quad permutes: every lane has a
// source, so the bound control only lets the move fuse into its user).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}
// Largest of four unsigned values over the wave (non-negative floats may be
// given as their bits, which order as the values), the four reductions
// interleaved step by step; uniform results.
__device__ __forceinline__ void wave_max4_u(uint32_t (&v)[4]) {
#pragma unroll
  for (int h = 0; h < 4; ++h) v[h] = max(v[h], dpp_u<0x128>(v[h]));  // row_ror 8
#pragma unroll
  for (int h = 0; h < 4; ++h) v[h] = max(v[h], dpp_u<0x124>(v[h]));  // row_ror 4
#pragma unroll
  for (int h = 0; h < 4; ++h) v[h] = max(v[h], dpp_u<0x122>(v[h]));  // row_ror 2
#pragma unroll
  for (int h = 0; h < 4; ++h) v[h] = max(v[h], dpp_u<0x121>(v[h]));  // row_ror 1: each lane holds its row's largest
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)v[h], 0);
    const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)v[h], 16);
    const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)v[h], 32);
    const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)v[h], 48);
    const uint32_t m1 = a > b ? a : b, m2 = c > d ? c : d;
    v[h] = m1 > m2 ? m1 : m2;
  }
}

// Inclusive prefix sum over the wave: within rows of 16 lanes by shifted
// adds, then rows 1 and 3 add the last lane of the row before, and rows 2 and
// 3 the last lane of row 1.
__device__ __forceinline__ uint32_t wave_incl_scan_u(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);  // row_shr 1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);  // row_shr 2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);  // row_shr 4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);  // row_shr 8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast 15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast 31
  return v;
}

// The full pass over the units of class 1 (filter.hip); max_cells: the
// caller's bound on a unit's depth bits (0: none), which picks the geometry.
void launch_filter(const FusedArgs& fa, int U, int max_cells, hipStream_t s);

}  // namespace fathom
