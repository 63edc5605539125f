// fathom_scan_topk: the decode-step scan + top-k of Sec. 3.2-3.3 and Sec. 2,
// fused so that no score array is written.
//
// The exact result is defined by the documented fp32 scores (exact
// dequantisation, fma(q, khat, acc) over active channels ascending) and the
// (score desc, index asc) order.  To avoid computing those scores for every
// key, each key first gets a cheap integer proxy with a rigorous error bound.
// With khat = z' a16 / 16, where
//   z' = 2 (c^(t) - 2^(t-1)) 2^(4-t) + 2^(4-t)   (an odd multiple, |z'| <= 15),
// the score is sum_j w_j z'_j / 16 with w_j = q_hj a16_bj.  Per block and
// head, delta is a power of two with max|w| / delta < 1024 and W_j = rne(w_j /
// delta) clamped to [-1020, 1019]; the proxy is (delta / 16) sum_j W_j z'_j,
// exact in fp32, and
//   |score - proxy| <= E = (sum_j |w_j - delta W_j| zmax_j / 16
//                           + (A + 1) 2^-24 sum_j |w_j| + A 2^-120) (1 + 2^-10),
// where the second term covers the rounding of w and the A roundings of the
// documented fma chain (each term |q khat| <= 15/16 |w|), the third any
// subnormal rounding, and the factor the rounding of E's own sums.
//
// W_j has 11 bits, more than an int8 MFMA operand: W = 8 Wh + Wl with Wh in
// [-127, 127] and Wl in [-4, 3].  The digits enter as u_j = U_j / 2 in [0, 15]
// (U_j = sum_{p<t} b_p 2^(4-p), so z'_j = 2 u_j - zmax_j), and the MFMA
// accumulates sum_j (8 u_j) Wh_j + sum_j u_j Wl_j = sum_j u_j W_j into one
// int32: 8 u_j <= 120 still fits the signed byte.  The proxy is then
// (delta / 16) (2 acc + bias) with bias = -sum_j W_j zmax_j per (block, head).
//
// Bits to proxy digits.  A wave holds 64 keys of a block (lane = key).  Four
// channels form a U dword (byte K = u of channel K of 4, plane p at bit
// 8K + 3 - p).  A row group is one plane p of the 4 channels of a U dword;
// staging byte-transposes its 4 plane rows of a block (v_perm_b32) into 8
// words, word m holding keys 8m..8m+7 of the 4 channels (byte K), rotated left
// by 3 - p.  Lane 8m + s then gathers its 4 bits of the row group with one
// v_and_or_b32 against the mask 0x01010101 << ((s + 3 - p) mod 8), building
// the U dword rotated left by s; one v_alignbit_b32 per U dword rotates it
// back.
//
// Passes: (1) proxies of a strided sample of 8-block groups; (2) per row, tau =
// a rank statistic of the sample chosen so that ~1.25 k keys are expected
// above it; (3) the full proxy pass: keys whose proxy + E reaches tau are
// queued per wave and re-scored exactly (their plane lines are still in L2);
// those with score >= tau are appended to the row's survivor list; (4) per
// row, the survivors are sorted and the first k written.  If fewer than k
// reach tau (or the list overflows), pass (4) recomputes the row exactly on
// its own (FATHOM_DEV_TOPK_FALLBACK).  The result never depends on tau.
#include "common.hpp"

namespace fathom {

constexpr int kFT = 256;          // threads per workgroup (4 waves)
constexpr int kFW = kFT / kWave;
constexpr int kGrp = 8;           // blocks per group (one wave step)
constexpr int kChunkRG = 16;      // row groups staged per chunk (a row group: one plane of a U dword's 4 channels)
constexpr int kStageItems = kChunkRG * kGrp / kWave;  // (row group, block) items staged per lane
constexpr int kRgStride = 36;     // LDS dwords per (row group, 4-block half): 8 words x 4 blocks, padded
constexpr int kChunkDw = 8;       // U dwords per chunk
constexpr int kChunkCh = 4 * kChunkDw;  // channels per chunk
constexpr int kScaleK = kD / 8;         // scale loads per lane, first chunk of a group (8 lanes per channel)
constexpr int kMaxDw = kD / 4;
constexpr int kResidentWG = 768;  // full-pass workgroups resident at once on MI355X (256 CUs x 3)
constexpr int kMaxGroupsPerWave = 32;  // keeps a workgroup's key offsets within 16 bits
constexpr int kWGQ = 512;        // full pass: candidate keys a workgroup gathers in LDS before writing
constexpr int kCapPerGroup = 128;  // candidate keys recorded per group of a full-pass workgroup (more: exact fallback)
constexpr int kSlots = 8;        // survivor sub-lists per row (spreads the append counters)
constexpr int kSmp = 64;         // sampled proxies kept per (row, sampled group): 16 lanes x 4
constexpr int kSampleGroups = 64; // at most this many sampled groups (512 blocks) per row
constexpr int kSelThreads = 1024;
constexpr int kSelCap = 16384;    // LDS composites in the select kernel
constexpr float kNegInf = -__builtin_huge_valf();

struct FusedWs {
  float* tau;       // [R] threshold on exact scores (-inf: every eligible key is kept)
  uint32_t* cnt;    // [R][kSlots] survivors appended to sub-list s
  uint64_t* cand;   // [R][kSlots][scap] survivors: score_key << 32 | ~index
  uint32_t* ent;    // [U][nwg][wgcap] key offset from the workgroup's first block | head mask << 16
  uint32_t* uovf;   // [U] a workgroup of the unit overflowed its list: exact fallback for the unit
  int64_t nwg;      // full-pass workgroups per unit
  int gpw;          // full pass: groups per wave, interleaved across the workgroup
  int wgcap;        // candidate keys recorded per full-pass workgroup: kCapPerGroup per group
  float* sample;    // [R][s_groups][128] per sampled group: each lane's two largest proxies
  uint32_t* bnd;    // [R][8] score keys splitting the survivors into kSlots ranges (select pass)
  int cap, scap;  // survivors per row (select kernel), per sub-list
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

static inline int fused_scap(int k) { return fused_cap(k) / 4; }

// Groups per wave: enough that the full pass over all units fits in one round
// of resident workgroups.
static inline int fused_gpw(int U, int64_t nb_cap) {
  const int64_t ng = (nb_cap + kGrp - 1) / kGrp;
  int64_t g = ((int64_t)U * ng + (int64_t)kFW * kResidentWG - 1) / ((int64_t)kFW * kResidentWG);
  return (int)(g < 1 ? 1 : g > kMaxGroupsPerWave ? kMaxGroupsPerWave : g);
}

static inline int64_t fused_nwg(int U, int64_t nb_cap) {
  const int64_t ng = (nb_cap + kGrp - 1) / kGrp, per = (int64_t)kFW * fused_gpw(U, nb_cap);
  return (ng + per - 1) / per;
}

size_t fused_ws_bytes(int R, int U, int64_t nb_cap, int k) {
  int64_t s, sg;
  if (nb_cap < 1) nb_cap = 1;
  fused_geometry(nb_cap, &s, &sg);
  const size_t nw = (size_t)U * fused_nwg(U, nb_cap);
  return a256((size_t)R * 4) + a256((size_t)R * kSlots * 4) + a256((size_t)R * kSlots * fused_scap(k) * 8) +
         a256(nw * (size_t)kCapPerGroup * kFW * fused_gpw(U, nb_cap) * 4) + a256((size_t)U * 4) + a256((size_t)R * kSlots * 4) + a256((size_t)R * sg * kSmp * 4);
}

static FusedWs fused_carve(void* ws, int R, int U, int64_t nb_cap, int k) {
  FusedWs w;
  if (nb_cap < 1) nb_cap = 1;
  fused_geometry(nb_cap, &w.s_gstride, &w.s_groups);
  w.cap = fused_cap(k);
  w.scap = fused_scap(k);
  w.nwg = fused_nwg(U, nb_cap);
  w.gpw = fused_gpw(U, nb_cap);
  w.wgcap = kCapPerGroup * kFW * w.gpw;
  const size_t nw = (size_t)U * w.nwg;
  char* p = reinterpret_cast<char*>(ws);
  w.tau = reinterpret_cast<float*>(p); p += a256((size_t)R * 4);
  w.cnt = reinterpret_cast<uint32_t*>(p); p += a256((size_t)R * kSlots * 4);
  w.cand = reinterpret_cast<uint64_t*>(p); p += a256((size_t)R * kSlots * w.scap * 8);
  w.ent = reinterpret_cast<uint32_t*>(p); p += a256(nw * (size_t)w.wgcap * 4);
  w.uovf = reinterpret_cast<uint32_t*>(p); p += a256((size_t)U * 4);
  w.bnd = reinterpret_cast<uint32_t*>(p); p += a256((size_t)R * kSlots * 4);
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

// Per-unit plan, shared by the waves of a workgroup.  Proxy channel order:
// depth descending, channel ascending (the integer proxy does not depend on
// the order; the exact scores use channel order ascending).  A U dword has as
// many row groups as its first (deepest) channel has planes; a row group lists
// the plane row of each of its 4 channels, kPadRow where the channel is absent
// or shallower.
constexpr uint32_t kPadRow = 0xFFFFFFFFu;
template <int G>
struct alignas(16) UnitLds {
  uint4 rgrow[kD];                // row group g: plane-row index 4j+p of its 4 channels, or kPadRow
  int act[kD];                    // j | t << 8
  int pidx[kD];                   // proxy index of the x-th active channel in channel order
  float qa[kD][G];                // q_hj (fp32) of active channel a
  float zmx[kD];                  // 16 - 2^(4-t): the largest |z'| of channel a
  uint32_t rgp[kD];               // row group g: its plane p
  uint32_t tpk[kMaxDw];           // depths of channels 4d..4d+3, byte K
  uint32_t drg[kMaxDw];           // first row group of dword d, relative to its chunk
  uint32_t dnr[kMaxDw];           // row groups of dword d
  int dch[kMaxDw];                // chunk of dword d
  int chd[kMaxDw + 1];            // chunk c = dwords [chd[c], chd[c+1])
  int chr[kMaxDw + 1];            // first row group of chunk c
  int cnt[2][5];
  int A, nch;
  float tau[G];
};

// Per-wave staging and per-(block, head) state.
template <int G4>
struct alignas(16) WaveLds {
  uint32_t rows[kChunkRG][2][kRgStride];  // [row group][blocks 0-3 | 4-7][4 word m + block], transposed, rotated
  uint16_t scl[kD][kGrp];                 // fp16 scales of the group's active channels (proxy order)
  uint32_t wB[kGrp][G4][kChunkDw];     // int8 Wh: [block][head][U dword], 4 channels a dword
  uint32_t wBl[kGrp][G4][kChunkDw];    // int8 Wl, same layout
  uint32_t zero16[4];                  // a zero MFMA operand for the lanes that carry no weights
  float sdel[kGrp][8];                 // delta (0: no usable bound)
  float sinv[kGrp][8];                 // 1 / delta
  float seb[kGrp][8];                  // sum |w - delta W| zmax
  float ssw[kGrp][8];                  // sum |w|
  int sbias[kGrp][8];                  // bias = -sum W zmax
  int sthr[kGrp][8];                   // full pass: candidate iff acc >= sthr
};

__device__ __forceinline__ uint64_t lanemask_lt(int lane) { return lane == 0 ? 0ull : (~0ull >> (64 - lane)); }

// Orders this wave's LDS writes before its later LDS reads (other lanes).
__device__ __forceinline__ void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Global-memory accesses through the global address space: the pointers live
// in a by-value argument struct, and generic (flat) accesses would also count
// against the LDS wait counter, making every LDS wait wait for HBM loads.
template <typename T>
__device__ __forceinline__ T gload(const T* p) {
  return *(const __attribute__((address_space(1))) T*)p;
}
template <typename T>
__device__ __forceinline__ void gstore(T* p, T v) {
  *(__attribute__((address_space(1))) T*)p = v;
}
__device__ __forceinline__ uint32_t gatomic_add(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add((__attribute__((address_space(1))) uint32_t*)p, v,
                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t rotl32(uint32_t x, int q) {
  return __builtin_amdgcn_alignbit(x, x, (uint32_t)(32 - q) & 31u);
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

// ---------------------------------------------------------------- unit plan
template <int G>
__device__ void unit_setup(UnitLds<G>& P, const FusedArgs& a, int u) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int t = 0;
  if (tid < kD) {
    t = gload(a.depths + (int64_t)u * kD + tid);
    t = t > kPlanes ? kPlanes : t;
  }
  uint64_t bal[5];
#pragma unroll
  for (int v = 1; v <= 4; ++v) bal[v] = __ballot(tid < kD && t == v);
  if (tid < kD && lane == 0) {
#pragma unroll
    for (int v = 1; v <= 4; ++v) P.cnt[wave][v] = __popcll(bal[v]);
  }
  __syncthreads();
  int first[5];
  {
    int pos = 0;
#pragma unroll
    for (int v = 4; v >= 1; --v) {
      first[v] = pos;
      pos += P.cnt[0][v] + P.cnt[1][v];
    }
    if (tid == 0) P.A = pos;
  }
  if (tid < kD && t > 0) {
    const int a_ = first[t] + (wave == 1 ? P.cnt[0][t] : 0) + __popcll(bal[t] & lanemask_lt(lane));
    P.act[a_] = tid | (t << 8);
    const uint64_t on = bal[1] | bal[2] | bal[3] | bal[4];
    const int w0 = P.cnt[0][1] + P.cnt[0][2] + P.cnt[0][3] + P.cnt[0][4];
    P.pidx[(wave == 1 ? w0 : 0) + __popcll(on & lanemask_lt(lane))] = a_;
  }
  __syncthreads();
  const int A = P.A, AD = (A + 3) >> 2;
  for (int x = tid; x < A * G; x += kFT) {
    const int ai = x / G, h = x % G;
    const float qv = load_q(a.q, a.qdt, ((int64_t)u * G + h) * kD + (P.act[ai] & 0xFF));
    P.qa[ai][h] = qv;
  }
  if (tid < A) P.zmx[tid] = (float)(16 - (16 >> (P.act[tid] >> 8)));
  if (tid < AD) {
    uint32_t tp = 0u;
#pragma unroll
    for (int k2 = 0; k2 < 4; ++k2) {
      const int x = 4 * tid + k2;
      if (x < A) tp |= (uint32_t)(P.act[x] >> 8) << (8 * k2);
    }
    P.tpk[tid] = tp;
  }
  __syncthreads();
  if (wave == 0) {  // row groups per dword; greedy chunks of whole dwords, at most kChunkRG row groups
                    // and kChunkDw dwords each
    int nr = 0;
    if (lane < AD) nr = (int)(P.tpk[lane] & 0xFF);  // the first channel of a dword is its deepest
    int c = 0, rows = 0, r0 = 0, ndw = 0, my_row = 0, my_ch = 0;
    for (int d = 0; d < AD; ++d) {
      const int v = __builtin_amdgcn_readlane(nr, d);
      if (rows + v > kChunkRG || ndw == kChunkDw) {
        ++c;
        r0 += rows;
        rows = 0;
        ndw = 0;
        if (lane == 0) {
          P.chd[c] = d;
          P.chr[c] = r0;
        }
      }
      if (lane == d) {
        my_row = rows;
        my_ch = c;
      }
      rows += v;
      ++ndw;
    }
    if (lane < AD) {
      P.drg[lane] = (uint32_t)my_row;
      P.dnr[lane] = (uint32_t)nr;
      P.dch[lane] = my_ch;
    }
    if (lane == 0) {
      const int nch = AD > 0 ? c + 1 : 0;
      P.chd[0] = 0;
      P.chr[0] = 0;
      P.nch = nch;
      P.chd[nch] = AD;
      P.chr[nch] = r0 + rows;
    }
  }
  __syncthreads();
  // row groups of dword d: plane p of its 4 channels
  if (tid < AD) {
    const int d = tid;
    const uint32_t tp = P.tpk[d];
    const int g0 = P.chr[P.dch[d]] + (int)P.drg[d], nr = (int)P.dnr[d];
    for (int p = 0; p < nr; ++p) {
      uint32_t rr[4];
#pragma unroll
      for (int K = 0; K < 4; ++K) {
        const int x = 4 * d + K;
        rr[K] = (x < A && (int)((tp >> (8 * K)) & 0xFF) > p) ? (uint32_t)(4 * (P.act[x] & 0xFF) + p) : kPadRow;
      }
      P.rgrow[g0 + p] = make_uint4(rr[0], rr[1], rr[2], rr[3]);
      P.rgp[g0 + p] = (uint32_t)p;
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------- one wave's pipeline
struct Stage {
  uint64_t rw[kStageItems][4];
  uint32_t sv[kScaleK];
};

// Lane (i, b): row groups i and i + 8 of chunk c for block gb + b and, with
// the first chunk, the scales of active channels i, i + 8, ... (all chunks:
// delta is fixed over every channel of the block).
template <int G>
__device__ __forceinline__ void stage_load(Stage& S, const UnitLds<G>& P, const FusedArgs& a, int u, int64_t gb,
                                           int c) {
  const int lane = threadIdx.x & 63, il = lane >> 3, bl = lane & 7;
  const int rg0 = P.chr[c], nrg = P.chr[c + 1] - rg0;
  const int nsc = c == 0 ? P.A : 0;
  const int64_t b = gb + bl;
  const bool bok = b < a.nb_cap;
  const uint64_t* Pu = a.planes + (int64_t)u * kD * kPlanes * a.nb_cap;
  const uint16_t* Su = a.scales + (int64_t)u * kD * a.nb_cap;
#pragma unroll
  for (int k = 0; k < kStageItems; ++k) {
    const int g = il + 8 * k;
#pragma unroll
    for (int K = 0; K < 4; ++K) S.rw[k][K] = 0ull;
    if (bok && g < nrg) {
      const uint4 rr = P.rgrow[rg0 + g];
      const uint32_t r4[4] = {rr.x, rr.y, rr.z, rr.w};
#pragma unroll
      for (int K = 0; K < 4; ++K)
        if (r4[K] != kPadRow) S.rw[k][K] = gload(Pu + (int64_t)r4[K] * a.nb_cap + b);
    }
  }
#pragma unroll
  for (int k = 0; k < kScaleK; ++k) {
    const int r = il + 8 * k;
    S.sv[k] = 0u;
    if (bok && r < nsc) S.sv[k] = gload(Su + (int64_t)(P.act[r] & 0xFF) * a.nb_cap + b);
  }
}

// Byte transpose of a row group's 4 rows (one block): word m = byte m of rows
// 0..3 in bytes 0..3, i.e. keys 8m..8m+7 of the 4 channels; then rotated left
// by 3 - p.  v_perm_b32 picks bytes 0-3 from its second operand, 4-7 from its first.
template <int G, int G4>
__device__ __forceinline__ void stage_store(const Stage& S, const UnitLds<G>& P, WaveLds<G4>& W, int c) {
  const int lane = threadIdx.x & 63, il = lane >> 3, bl = lane & 7;
  const int rg0 = P.chr[c], nrg = P.chr[c + 1] - rg0;
  const int nsc = c == 0 ? P.A : 0;
#pragma unroll
  for (int k = 0; k < kStageItems; ++k) {
    const int g = il + 8 * k;
    if (g < nrg) {
      const uint32_t rot = (29u + P.rgp[rg0 + g]) & 31u;  // rotate right by 29 + p = left by 3 - p
      uint32_t w[8];
#pragma unroll
      for (int hw = 0; hw < 2; ++hw) {
        const uint32_t r0 = (uint32_t)(S.rw[k][0] >> (32 * hw)), r1 = (uint32_t)(S.rw[k][1] >> (32 * hw));
        const uint32_t r2 = (uint32_t)(S.rw[k][2] >> (32 * hw)), r3 = (uint32_t)(S.rw[k][3] >> (32 * hw));
        const uint32_t t01l = __builtin_amdgcn_perm(r1, r0, 0x05010400u);  // r0.b0 r1.b0 r0.b1 r1.b1
        const uint32_t t01h = __builtin_amdgcn_perm(r1, r0, 0x07030602u);  // r0.b2 r1.b2 r0.b3 r1.b3
        const uint32_t t23l = __builtin_amdgcn_perm(r3, r2, 0x05010400u);
        const uint32_t t23h = __builtin_amdgcn_perm(r3, r2, 0x07030602u);
        w[4 * hw + 0] = __builtin_amdgcn_perm(t23l, t01l, 0x05040100u);
        w[4 * hw + 1] = __builtin_amdgcn_perm(t23l, t01l, 0x07060302u);
        w[4 * hw + 2] = __builtin_amdgcn_perm(t23h, t01h, 0x05040100u);
        w[4 * hw + 3] = __builtin_amdgcn_perm(t23h, t01h, 0x07060302u);
      }
      uint32_t* dst = &W.rows[g][bl >> 2][bl & 3];
#pragma unroll
      for (int m = 0; m < 8; ++m) dst[4 * m] = __builtin_amdgcn_alignbit(w[m], w[m], rot);
    }
  }
#pragma unroll
  for (int k = 0; k < kScaleK; ++k) {
    const int r = il + 8 * k;
    if (r < nsc) W.scl[r][bl] = (uint16_t)S.sv[k];
  }
}

// Weights of chunk c for the 8 blocks of the group.  Lane = (block g, head
// h, channel phase kk): each lane walks the chunk's channels a = kk, kk + KL,
// ... and the per-(block, head) sums are reduced over kk.  first: delta is
// fixed from every active channel; last: the candidate thresholds.  Blocks >= nbu get no bound
// (their keys are never eligible).  A non-finite w leaves delta = 0 (first
// chunk) or a non-finite E: no bound, every key of the block is a candidate.
template <int G, int G4, bool SAMPLE>
__device__ void weights(const UnitLds<G>& P, WaveLds<G4>& W, int c, bool first, bool last, int64_t gb, int64_t nbu) {
  constexpr int Gp = G <= 1 ? 1 : G <= 2 ? 2 : G <= 4 ? 4 : 8;
  constexpr int KL = 8 / Gp;
  const int lane = threadIdx.x & 63, g = lane >> 3, sub = lane & 7, h = sub % Gp, kk = sub / Gp;
  const bool gh = h < G;
  const bool bv = gh && gb + g < nbu;
  const int a0 = 4 * P.chd[c];
  int a1 = 4 * P.chd[c + 1];
  a1 = a1 < P.A ? a1 : P.A;
  const int A = P.A;
  const int hh = gh ? h : 0;
  float delta, inv;
  if (first) {
    float mx = 0.0f;  // fmaxf skips NaN; an infinite w makes mx infinite
    if (bv) {  // over every active channel, not only this chunk's
      for (int ai = kk; ai < A; ai += KL)
        mx = fmaxf(mx, fabsf(__fmul_rn(P.qa[ai][hh], half_bits_to_float(W.scl[ai][g]))));
    }
#pragma unroll
    for (int m = Gp; m < 8; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, kWave));
    int e;
    (void)frexpf(mx, &e);  // mx in [2^(e-1), 2^e)
    const bool ok = mx <= 3.402823466e38f && (mx >= 0x1p-100f || mx == 0.0f);
    const int ee = e < -100 ? -100 : e;
    delta = ok ? ldexpf(1.0f, ee - 10) : 0.0f;  // |w| / delta < 1024
    inv = ok ? ldexpf(1.0f, 10 - ee) : 0.0f;
  } else {
    delta = gh ? W.sdel[g][h] : 0.0f;
    inv = gh ? W.sinv[g][h] : 0.0f;
  }
  float eb = 0.0f, sw = 0.0f, bs = 0.0f;  // bs: sum W zmax, an integer below 2^24
  if (bv) {
    uint8_t* whb = reinterpret_cast<uint8_t*>(&W.wB[g][h][0]);
    uint8_t* wlb = reinterpret_cast<uint8_t*>(&W.wBl[g][h][0]);
    for (int ai = a0 + kk; ai < a1; ai += KL) {
      const int al = ai - a0;
      const float w = __fmul_rn(P.qa[ai][hh], half_bits_to_float(W.scl[ai][g]));
      const float zm = P.zmx[ai];
      const float Wf = fminf(fmaxf(rintf(__fmul_rn(w, inv)), -1020.0f), 1019.0f);
      eb = __fmaf_rn(fabsf(__fmaf_rn(Wf, delta, -w)), zm, eb);
      sw = __fadd_rn(sw, fabsf(w));
      bs = __fmaf_rn(Wf, zm, bs);
      const int Wi = (int)Wf, wh = (Wi + 4) >> 3;
      whb[al] = (uint8_t)(wh & 0xFF);
      wlb[al] = (uint8_t)((Wi - 8 * wh) & 0xFF);
    }
  }
#pragma unroll
  for (int m = Gp; m < 8; m <<= 1) {
    eb = __fadd_rn(eb, __shfl_xor(eb, m, kWave));
    sw = __fadd_rn(sw, __shfl_xor(sw, m, kWave));
    bs = __fadd_rn(bs, __shfl_xor(bs, m, kWave));
  }
  if (gh && kk == 0) {
    const float ebt = first ? eb : __fadd_rn(W.seb[g][h], eb);
    const float swt = first ? sw : __fadd_rn(W.ssw[g][h], sw);
    const int biast = (first ? 0 : W.sbias[g][h]) - (int)bs;
    W.sdel[g][h] = delta;
    W.sinv[g][h] = inv;
    W.seb[g][h] = ebt;
    W.ssw[g][h] = swt;
    W.sbias[g][h] = biast;
    if (last && !SAMPLE) {
      // candidate iff (delta / 16) (2 acc + bias) + E >= tau, made conservative
      // on integers: 2 acc >= floor((tau - E) 16 / delta) - bias - 1
      const float E = __fmul_rn(
          __fmaf_rn(ebt, 0.0625f, __fmaf_rn((float)(A + 1) * 0x1p-24f, swt, (float)A * 0x1p-120f)), 1.0f + 0x1p-10f);
      const float tau = P.tau[h];
      int thr = INT32_MIN;
      if (delta > 0.0f && tau != kNegInf && E <= 3.402823466e38f) {
        const double x = ((double)tau - (double)E) * 16.0 / (double)delta;
        if (x == x) {
          const double X = floor(x) - (double)biast - 1.0;
          const double f = floor((X + 1.0) * 0.5);  // acc >= ceil(X / 2)
          thr = f <= -2147483648.0 ? INT32_MIN : f >= 2147483647.0 ? INT32_MAX : (int)f;
        }
      }
      if (gb + g >= nbu) thr = INT32_MAX;
      W.sthr[g][h] = thr;
    }
  }
}

// Integer proxy sums of chunk c for the 8 blocks, added to acc.  Per 4 U
// dwords (16 channels) two v_mfma_i32_16x16x64_i8 per block: A = the 16
// digits u (then 8 u) of each lane's key; B = Wl (then Wh), block-diagonal, so
// lane group g' of A (keys 16g'..16g'+15) meets only the weights in columns
// 4g'..4g'+3 (heads 0..3): C[i][4g' + h] = sum_j u_{16g'+i, j} W_{j, h}.  Lane l then holds heads
// 4p + l%4 of keys 16((l%16)/4) + 4(l/16) + r, r = 0..3, in acc[g][p][r].
typedef __attribute__((ext_vector_type(4))) int v4i;
template <int G, int G4>
__device__ __forceinline__ void chunk_proxy(const UnitLds<G>& P, const WaveLds<G4>& W, int c,
                                            v4i (&acc)[kGrp][G4 / 4]) {
  constexpr int NP = G4 / 4;
  const int lane = threadIdx.x & 63, sk = lane & 7, m4 = 4 * (lane >> 3);
  const int d0 = uni(P.chd[c]), d1 = uni(P.chd[c + 1]);
  const bool wlane = (lane >> 4) == ((lane & 15) >> 2);
  uint32_t mk[4];  // plane p: this lane's bits of a transposed, rotated word
#pragma unroll
  for (int p = 0; p < 4; ++p) mk[p] = 0x01010101u << ((sk + 3 - p) & 7);
#pragma unroll
  for (int gh = 0; gh < kGrp; gh += 4) {  // blocks gh .. gh+3
    for (int db = d0; db < d1; db += 4) {
      uint32_t zq[4][4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t zr[4] = {0u, 0u, 0u, 0u};
        const int d = db + q;
        if (d < d1) {
          const int nr = uni((int)P.dnr[d]);
          const int rb = uni((int)P.drg[d]);
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            if (p < nr) {
              const uint4 x = *reinterpret_cast<const uint4*>(&W.rows[rb + p][gh >> 2][m4]);
              zr[0] |= x.x & mk[p];
              zr[1] |= x.y & mk[p];
              zr[2] |= x.z & mk[p];
              zr[3] |= x.w & mk[p];
            }
          }
        }
#pragma unroll
        for (int g = 0; g < 4; ++g) zq[q][g] = __builtin_amdgcn_alignbit(zr[g], zr[g], (uint32_t)sk);
      }
      const int mq = (db - d0) >> 2;
#pragma unroll
      for (int pp = 0; pp < NP; ++pp) {
        const int hh = 4 * pp + (lane & 3);
        const bool wl = wlane && hh < G;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int hc = hh < G4 ? hh : 0;
          const v4i bl = *reinterpret_cast<const v4i*>(wl ? &W.wBl[gh + g][hc][4 * mq] : W.zero16);
          const v4i bh = *reinterpret_cast<const v4i*>(wl ? &W.wB[gh + g][hc][4 * mq] : W.zero16);
          const v4i al = {(int)zq[0][g], (int)zq[1][g], (int)zq[2][g], (int)zq[3][g]};
          const v4i ah = {(int)(zq[0][g] << 3), (int)(zq[1][g] << 3), (int)(zq[2][g] << 3), (int)(zq[3][g] << 3)};
          acc[gh + g][pp] = __builtin_amdgcn_mfma_i32_16x16x64_i8(al, bl, acc[gh + g][pp], 0, 0, 0);
          acc[gh + g][pp] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ah, bh, acc[gh + g][pp], 0, 0, 0);
        }
      }
    }
  }
}

// Runs the proxy over `ngroups` groups of unit u (group index gi -> first
// block via group_block), chunk by chunk with the next chunk's loads in flight,
// and hands each finished group to `finish(gb, acc)`.
template <int G, int G4, bool SAMPLE, typename GroupBlock, typename Finish>
__device__ void wave_groups(const UnitLds<G>& P, WaveLds<G4>& W, const FusedArgs& a, int u, int ngroups, int64_t nbu,
                            GroupBlock group_block, Finish finish) {
  const int lane = threadIdx.x & 63;
  const int nch = uni(P.nch);
  if (ngroups <= 0 || nch <= 0) {
    for (int gi = 0; gi < ngroups; ++gi) {  // no active channel: every proxy is 0 with E = 0
      v4i acc[kGrp][G4 / 4];
#pragma unroll
      for (int g = 0; g < kGrp; ++g)
#pragma unroll
        for (int pp = 0; pp < G4 / 4; ++pp) acc[g][pp] = v4i{0, 0, 0, 0};
      const int64_t gb = group_block(gi);
      {
        const int g = lane >> 3, h = lane & 7;
        if (h < G) {
          W.sdel[g][h] = 1.0f;
          W.sinv[g][h] = 1.0f;
          W.seb[g][h] = 0.0f;
          W.ssw[g][h] = 0.0f;
          W.sbias[g][h] = 0;
          int thr = INT32_MIN;
          if (!SAMPLE && P.tau[h] > 0.0f) thr = INT32_MAX;
          if (gb + g >= nbu) thr = INT32_MAX;
          W.sthr[g][h] = thr;
        }
      }
      wave_lds_sync();
      finish(gb, acc);
      wave_lds_sync();
    }
    return;
  }
  const int items = ngroups * nch;
  Stage S;
  stage_load<G>(S, P, a, u, group_block(0), 0);
  if (lane < 4) W.zero16[lane] = 0u;
  v4i acc[kGrp][G4 / 4];
#pragma unroll
  for (int g = 0; g < kGrp; ++g)
#pragma unroll
    for (int pp = 0; pp < G4 / 4; ++pp) acc[g][pp] = v4i{0, 0, 0, 0};
  for (int it = 0; it < items; ++it) {
    const int gi = it / nch, c = it - gi * nch;
    const int64_t gb = group_block(gi);
    stage_store<G, G4>(S, P, W, c);
    if (it + 1 < items) {
      const int gi2 = (it + 1) / nch;
      stage_load<G>(S, P, a, u, group_block(gi2), it + 1 - gi2 * nch);
    }
    wave_lds_sync();
    weights<G, G4, SAMPLE>(P, W, c, c == 0, c == nch - 1, gb, nbu);
    wave_lds_sync();
    chunk_proxy<G, G4>(P, W, c, acc);
    if (c == nch - 1) {
      finish(gb, acc);
#pragma unroll
      for (int g = 0; g < kGrp; ++g)
#pragma unroll
        for (int pp = 0; pp < G4 / 4; ++pp) acc[g][pp] = v4i{0, 0, 0, 0};
    }
    wave_lds_sync();  // this item's LDS reads are done before the next stage_store
  }
}

// ---------------------------------------------------------------- pass 1
// Each workgroup: 4 sampled groups (one per wave) of the unit.
template <int G>
__global__ __launch_bounds__(kFT, 3) void fused_sample_kernel(FusedArgs a) {
  constexpr int G4 = (G + 3) & ~3;
  __shared__ UnitLds<G> P;
  __shared__ WaveLds<G4> WL[kFW];
  const int u = blockIdx.y, lane = threadIdx.x & 63, wave = uni(threadIdx.x >> 6);
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  const int64_t nbu = (nu + kBlockTokens - 1) / kBlockTokens;
  unit_setup<G>(P, a, u);
  const int64_t sg = (int64_t)blockIdx.x * kFW + wave;  // sampled group index
  if (sg >= a.ws.s_groups) return;
  const int64_t gb = sg * a.ws.s_gstride * kGrp;
  WaveLds<G4>& W = WL[wave];
  // lane l holds heads 4p + l%4 of 4 keys per block; it keeps the four largest
  // of its 32 proxies per head: the m-th largest of what the 16 lanes of a
  // head keep is at most the m-th largest sampled proxy
  const int kl = 16 * ((lane & 15) >> 2) + 4 * (lane >> 4);
  auto put = [&](int64_t gbb, v4i (&acc)[kGrp][G4 / 4]) {
#pragma unroll
    for (int pp = 0; pp < G4 / 4; ++pp) {
      const int hh = 4 * pp + (lane & 3);
      const int hc = hh < G ? hh : 0;
      float t[4] = {kNegInf, kNegInf, kNegInf, kNegInf};
#pragma unroll
      for (int g = 0; g < kGrp; ++g) {
        const int64_t b = gbb + g;
        const float del = W.sdel[g][hc];
        const int bias = W.sbias[g][hc];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int64_t i = b * kBlockTokens + kl + q;
          // the proxy itself (exact in fp32): tau only steers how many keys are
          // re-scored; the survivor count, not tau, guarantees the result
          float v = kNegInf;
          if (b < nbu && i >= lo && i < hi && del > 0.0f) v = __fmul_rn(0.0625f * del, (float)(2 * acc[g][pp][q] + bias));
#pragma unroll
          for (int z = 0; z < 4; ++z) {  // insert into the descending t[0..3]
            const float hi2 = fmaxf(t[z], v);
            v = fminf(t[z], v);
            t[z] = hi2;
          }
        }
      }
      if (hh < G) {
        float* dst = a.ws.sample + (((int64_t)u * G + hh) * a.ws.s_groups + sg) * kSmp + (lane >> 2) * 4;
#pragma unroll
        for (int z = 0; z < 4; ++z) gstore(dst + z, t[z]);
      }
    }
  };
  if (gb < nbu) {
    wave_groups<G, G4, true>(P, W, a, u, 1, nbu, [&](int) { return gb; }, put);
  } else {
    for (int pp = 0; pp < G4 / 4; ++pp) {
      const int hh = 4 * pp + (lane & 3);
      if (hh < G) {
        float* dst = a.ws.sample + (((int64_t)u * G + hh) * a.ws.s_groups + sg) * kSmp + (lane >> 2) * 4;
        for (int z = 0; z < 4; ++z) gstore(dst + z, kNegInf);
      }
    }
  }
}

// ---------------------------------------------------------------- pass 2
// tau = the m-th largest kept sample proxy, m ~ 1.25 k * (sampled / eligible)
// + 16; tau = -inf when the row has no more eligible keys than the survivor
// list holds.  The kept proxies stay in registers as order-preserving keys (0
// = unusable); the m-th largest is found bit by bit from the top with
// block-wide counts.  The kept proxies above tau, ranked, also give kSlots - 1
// boundaries that split the expected survivors into ranges of similar size.
constexpr int kTauPer = kSampleGroups * kSmp / kSelThreads;  // kept proxies per thread
__global__ __launch_bounds__(kSelThreads) void fused_tau_kernel(FusedArgs a, int G) {
  __shared__ uint32_t part[2 * (kSelThreads / kWave)];
  __shared__ uint32_t top[kSelThreads];
  __shared__ uint32_t srt[kSelThreads];
  __shared__ int ntop;
  const int r = blockIdx.x, u = r / G, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0 && r % G == 0) a.ws.uovf[u] = 0u;
  if (tid < kSlots) a.ws.cnt[r * kSlots + tid] = 0u;
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  const int64_t m_e = hi - lo;
  if (m_e <= a.ws.cap) {
    if (tid == 0) a.ws.tau[r] = kNegInf;
    return;
  }
  const float* smp = a.ws.sample + (int64_t)r * a.ws.s_groups * kSmp;
  const int ns = (int)(a.ws.s_groups * kSmp);
  uint32_t key[kTauPer];
#pragma unroll
  for (int x = 0; x < kTauPer; ++x) {
    const int i = tid + x * kSelThreads;
    key[x] = 0u;
    if (i < ns) {
      const float v = gload(smp + i);
      if (v > kNegInf) key[x] = score_key(v) | 1u;  // keep 0 free: proxies are never NaN
    }
  }
  // eligible keys of the sampled groups
  uint32_t msg = 0;
  if (tid < a.ws.s_groups) {
    const int64_t k0 = (int64_t)tid * a.ws.s_gstride * kGrp * kBlockTokens, k1 = k0 + kGrp * kBlockTokens;
    const int64_t x0 = k0 > lo ? k0 : lo, x1 = k1 < hi ? k1 : hi;
    msg = x1 > x0 ? (uint32_t)(x1 - x0) : 0u;
  }
  int ph = 0;  // partial sums double-buffered: one barrier per count
  auto block_sum = [&](uint32_t v) {  // v: this wave's total (wave-uniform)
    if (lane == 0) part[ph * (kSelThreads / kWave) + wave] = v;
    __syncthreads();
    uint32_t t = 0;
#pragma unroll
    for (int w = 0; w < kSelThreads / kWave; ++w) t += part[ph * (kSelThreads / kWave) + w];
    ph ^= 1;
    return t;
  };
  uint32_t cw = 0, uw = 0;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) msg += __shfl_xor(msg, o, kWave);
  cw = msg;
#pragma unroll
  for (int x = 0; x < kTauPer; ++x) uw += (uint32_t)__popcll(__ballot(key[x] != 0u));
  const int64_t m_s = block_sum(cw);
  const int64_t usable = block_sum(uw);
  if (m_s == 0 || usable == 0) {
    if (tid == 0) a.ws.tau[r] = kNegInf;
    return;
  }
  int64_t m = (5 * (int64_t)a.k * m_s + 4 * m_e - 1) / (4 * m_e) + 16;
  if (m > usable) m = usable;
  uint32_t prefix = 0u;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    uint32_t cnt = 0;  // wave total from ballots (scalar)
#pragma unroll
    for (int x = 0; x < kTauPer; ++x) cnt += (uint32_t)__popcll(__ballot(key[x] >= cand));
    if ((int64_t)block_sum(cnt) >= m) prefix = cand;
  }
  // rank the kept proxies >= tau (at most kSelThreads of them) for the range boundaries
  if (tid == 0) ntop = 0;
  __syncthreads();
#pragma unroll
  for (int x = 0; x < kTauPer; ++x) {
    if (key[x] >= prefix && key[x] != 0u) {
      const int p2 = atomicAdd(&ntop, 1);
      if (p2 < kSelThreads) top[p2] = key[x];
    }
  }
  __syncthreads();
  const int nt = ntop < kSelThreads ? ntop : kSelThreads;
  if (tid < nt) {
    const uint32_t v = top[tid];
    int rk = 0;
    for (int x = 0; x < nt; ++x) {
      const uint32_t w = top[x];
      rk += (w > v) || (w == v && x < tid);
    }
    srt[rk] = v;
  }
  __syncthreads();
  if (tid == 0) {
    const uint32_t key0 = prefix & ~1u;  // the low bit was forced on: round the key down
    const uint32_t bitsf = (key0 & 0x80000000u) ? (key0 & 0x7FFFFFFFu) : ~key0;
    a.ws.tau[r] = __uint_as_float(bitsf);
  }
  if (tid >= 1 && tid < kSlots) {
    // boundary b: survivors with key > bnd[b] go to ranges < b
    const int at = (int)(((int64_t)tid * nt) / kSlots);
    a.ws.bnd[r * kSlots + tid] = nt > 0 ? (srt[at < nt ? at : nt - 1] & ~1u) : 0u;
  }
  if (tid == 0) a.ws.bnd[r * kSlots] = 0xFFFFFFFFu;
}

// ---------------------------------------------------------------- pass 3
// The documented fp32 scores of key i for all G heads: active channels
// ascending, khat exact, acc = fma(q, khat, acc); the loads of 8 channels are
// issued together.
constexpr int kRsChunk = 8;
template <int G>
__device__ __forceinline__ void exact_scores(const UnitLds<G>& P, const FusedArgs& a, int u, int64_t i,
                                             float (&acc)[G]) {
  const int64_t b = i >> 6;
  const int hw = (int)((i >> 5) & 1), sh = (int)(i & 31), A = P.A;
  const uint64_t* Pu = a.planes + (int64_t)u * kD * kPlanes * a.nb_cap + b;
  const uint16_t* Su = a.scales + (int64_t)u * kD * a.nb_cap + b;
  for (int a0 = 0; a0 < A; a0 += kRsChunk) {
    uint32_t wd[kRsChunk][4];
    uint16_t sc[kRsChunk];
#pragma unroll
    for (int K = 0; K < kRsChunk; ++K) {
      const int x = a0 + K;
      sc[K] = 0;
#pragma unroll
      for (int p = 0; p < 4; ++p) wd[K][p] = 0u;
      if (x < A) {
        const int e2 = P.act[P.pidx[x]], j = e2 & 0xFF, tt = e2 >> 8;
        sc[K] = gload(Su + (int64_t)j * a.nb_cap);
#pragma unroll
        for (int p = 0; p < 4; ++p)
          if (p < tt) wd[K][p] = gload(reinterpret_cast<const uint32_t*>(Pu + (int64_t)(4 * j + p) * a.nb_cap) + hw);
      }
    }
#pragma unroll
    for (int K = 0; K < kRsChunk; ++K) {
      const int x = a0 + K;
      if (x < A) {
        const int pi = P.pidx[x], tt = P.act[pi] >> 8;
        uint32_t c = 0;
#pragma unroll
        for (int p = 0; p < 4; ++p)
          if (p < tt) c = 2u * c + ((wd[K][p] >> sh) & 1u);
        const float y = (float)c + (0.5f - (float)(1 << (tt - 1)));
        const float khat =
            __fmul_rn(y, __fmul_rn(half_bits_to_float(sc[K]), __uint_as_float((uint32_t)(128 - tt) << 23)));
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = __fmaf_rn(P.qa[pi][h], khat, acc[h]);
      }
    }
  }
}

template <int G>
__global__ __launch_bounds__(kFT, 3) void fused_full_kernel(FusedArgs a) {
  constexpr int G4 = (G + 3) & ~3;
  __shared__ UnitLds<G> P;
  __shared__ WaveLds<G4> WL[kFW];
  __shared__ uint32_t wq[kWGQ];  // this workgroup's candidates
  __shared__ int wqn;
  const int u = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, blockIdx.x == 0 && tid == 0);
  const int64_t nbu = (nu + kBlockTokens - 1) / kBlockTokens;
  const int gpw = a.ws.gpw;
  const int64_t g0 = (int64_t)blockIdx.x * kFW * gpw;  // first group of this workgroup
  const int64_t b0 = g0 * kGrp, b1 = (g0 + (int64_t)kFW * gpw) * kGrp;
  const int64_t region = (int64_t)u * a.ws.nwg + blockIdx.x;
  // rows with no more eligible keys than the survivor list holds are
  // computed exactly by pass 4: no candidates from here
  if (b0 >= nbu || b0 * kBlockTokens >= hi || b1 * kBlockTokens <= lo || hi - lo <= a.ws.cap) return;
  if (tid == 0) wqn = 0;
  unit_setup<G>(P, a, u);
  if (tid < G) P.tau[tid] = gload(a.ws.tau + u * G + tid);
  __syncthreads();
  // this wave's groups: g0 + wave + kFW * x, those that hold eligible keys
  // this wave's groups g0 + wave + kFW x that hold eligible keys: a contiguous range of x
  int x_lo = gpw, x_hi = 0;
  for (int x = 0; x < gpw; ++x) {
    const int64_t gbx = (g0 + wave + kFW * x) * kGrp;
    if (gbx < nbu && gbx * kBlockTokens < hi && (gbx + kGrp) * kBlockTokens > lo) {
      x_lo = x < x_lo ? x : x_lo;
      x_hi = x + 1;
    }
  }
  const int ng = x_hi > x_lo ? x_hi - x_lo : 0;
  WaveLds<G4>& W = WL[wave];
  auto gblock = [&](int gi) { return (g0 + wave + kFW * (int64_t)(x_lo + gi)) * kGrp; };
  // lane l holds heads 4p + l%4 of keys 16((l%16)/4) + 4(l/16) + q of each block
  const int kl = 16 * ((lane & 15) >> 2) + 4 * (lane >> 4);
  auto put = [&](int64_t gbb, v4i (&acc)[kGrp][G4 / 4]) {
    // eligibility relative to the group's first key (32-bit)
    const int64_t key0 = gbb * kBlockTokens;
    const int64_t lr = lo - key0, hr = hi - key0, br = nbu - gbb;
    const int lo_r = lr < -1 ? -1 : lr > 1024 ? 1024 : (int)lr;
    const int hi_r = hr < -1 ? -1 : hr > 1024 ? 1024 : (int)hr;
    const int nb_r = br < 0 ? 0 : br > kGrp ? kGrp : (int)br;
#pragma unroll
    for (int pp = 0; pp < G4 / 4; ++pp) {
      const int hh = 4 * pp + (lane & 3);
      int thr[kGrp];
#pragma unroll
      for (int g = 0; g < kGrp; ++g) thr[g] = hh < G ? W.sthr[g][hh] : INT32_MAX;
      uint32_t bits = 0u;  // bit 4g + q: key q of block g reaches its threshold
#pragma unroll
      for (int g = 0; g < kGrp; ++g)
#pragma unroll
        for (int q = 0; q < 4; ++q) bits |= (uint32_t)(acc[g][pp][q] >= thr[g]) << (4 * g + q);
      if (__ballot(bits != 0u)) {
        while (bits) {
          const int bi = __ffs((int)bits) - 1;
          bits &= bits - 1u;
          const int g = bi >> 2, rel = g * kBlockTokens + kl + (bi & 3);
          if (rel >= lo_r && rel < hi_r && g < nb_r) {
            const int pos = atomicAdd(&wqn, 1);
            const uint32_t en = (uint32_t)((gbb - b0) * kBlockTokens + rel) | (1u << (16 + hh));
            if (pos < kWGQ) wq[pos] = en;
            else if (pos < a.ws.wgcap) gstore(&a.ws.ent[region * a.ws.wgcap + pos], en);
          }
        }
      }
    }
  };
  wave_groups<G, G4, false>(P, W, a, u, ng, nbu, gblock, put);
  __syncthreads();
  // exact documented scores of this workgroup's candidates (their plane lines
  // are still in L2); survivors go to the rows' lists through LDS, one append
  // per pass and head
  const int nq = wqn;
  if (nq > a.ws.wgcap) {
    if (tid == 0) set_status(a.ws.uovf + u, 1u);
    return;
  }
  uint64_t(*kept)[kFT] = reinterpret_cast<uint64_t(*)[kFT]>(&WL[0]);  // the staging area is free now
  __shared__ int nk[G];
  __shared__ uint32_t kbase[G];
  for (int e0 = 0; e0 < nq; e0 += kFT) {
    const int slot = (int)((blockIdx.x + e0 / kFT) % kSlots);  // spread the appends over the sub-lists
    if (tid < G) nk[tid] = 0;
    __syncthreads();
    const int e = e0 + tid;
    uint32_t en = 0u;
    if (e < nq) en = e < kWGQ ? wq[e] : gload(a.ws.ent + region * a.ws.wgcap + e);
    const int hm = (int)(en >> 16);
    const int64_t i = b0 * kBlockTokens + (int64_t)(en & 0xFFFFu);
    float acc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) acc[h] = 0.0f;
    if (hm) exact_scores<G>(P, a, u, i, acc);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const bool keep = ((hm >> h) & 1) && acc[h] >= P.tau[h];
      const uint64_t bm = __ballot(keep);
      if (bm) {
        const int leader = __ffsll((unsigned long long)bm) - 1;
        int basep = 0;
        if (lane == leader) basep = atomicAdd(&nk[h], __popcll(bm));
        basep = __shfl(basep, leader, kWave);
        if (keep)
          kept[h][basep + __popcll(bm & lanemask_lt(lane))] =
              ((uint64_t)score_key(acc[h]) << 32) | (uint64_t)(~(uint32_t)i);
      }
    }
    __syncthreads();
    if (tid < G && nk[tid] > 0)
      kbase[tid] = gatomic_add(&a.ws.cnt[(u * G + tid) * kSlots + slot], (uint32_t)nk[tid]);
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) {
      if (tid < nk[h]) {
        const uint32_t pos = kbase[h] + (uint32_t)tid;
        if (pos < (uint32_t)a.ws.scap)
          gstore(&a.ws.cand[((int64_t)(u * G + h) * kSlots + slot) * a.ws.scap + pos], kept[h][tid]);
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- pass 4
// Bitonic sort of buf[0..P) (P a power of two) into descending order; every
// thread owns whole compare-exchange pairs, all loads of a stage issued first.
__device__ void bitonic_desc(uint64_t* buf, int P) {
  const int tid = threadIdx.x, nt = blockDim.x, npairs = P >> 1;
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p0 = 0; p0 < npairs; p0 += 2 * nt) {
        int ii[2];
        uint64_t x[2], y[2];
#pragma unroll
        for (int q2 = 0; q2 < 2; ++q2) {
          const int pid = p0 + tid + q2 * nt;
          ii[q2] = ((pid & ~(stride - 1)) << 1) | (pid & (stride - 1));
          if (pid < npairs) {
            x[q2] = buf[ii[q2]];
            y[q2] = buf[ii[q2] + stride];
          }
        }
#pragma unroll
        for (int q2 = 0; q2 < 2; ++q2) {
          const int pid = p0 + tid + q2 * nt;
          if (pid < npairs) {
            const bool desc = (ii[q2] & size) == 0;
            if (desc ? (x[q2] < y[q2]) : (x[q2] > y[q2])) {
              buf[ii[q2]] = y[q2];
              buf[ii[q2] + stride] = x[q2];
            }
          }
        }
      }
      // pairs of strides <= 64 stay inside one wave's elements from one stage
      // to the next (thread t owns pairs t and t + nt): a wave-level LDS wait
      // suffices unless the next stride is larger
      const int next = stride > 1 ? stride >> 1 : size;  // the next stage's stride
      if (next <= 64 && stride <= 64 && nt % kWave == 0)
        wave_lds_sync();
      else
        __syncthreads();
    }
  }
}

__device__ __forceinline__ float key_to_score(uint32_t key) {
  if (key == 0u) return __uint_as_float(0x7FC00000u);
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// Exact documented score of key (block b, bit) for head h of unit u, for
// the fallback path (channels ascending from the act list).
__device__ __forceinline__ float exact_score1(const int* act, int A, const float* qh, const FusedArgs& a, int u,
                                              int64_t b, int bit) {
  const uint64_t* Pu = a.planes + (int64_t)u * kD * kPlanes * a.nb_cap + b;
  const uint16_t* Su = a.scales + (int64_t)u * kD * a.nb_cap + b;
  float acc = 0.0f;
  for (int ai = 0; ai < A; ++ai) {
    const int e = act[ai], j = e & 0xFF, t = e >> 8;
    const float af = half_bits_to_float(Su[(int64_t)j * a.nb_cap]);
    uint32_t c = 0;
    for (int p = 0; p < t; ++p) c = 2u * c + (uint32_t)((Pu[(int64_t)(4 * j + p) * a.nb_cap] >> bit) & 1ull);
    const float y = (float)c + (0.5f - (float)(1 << (t - 1)));
    const float khat = __fmul_rn(y, __fmul_rn(af, __uint_as_float((uint32_t)(128 - t) << 23)));
    acc = __fmaf_rn(qh[ai], khat, acc);
  }
  return acc;
}

// Pass 4, one workgroup per (score range, row).  Normally the survivors of a
// row are split by the boundaries from pass 2: workgroup b sorts the survivors
// of range b and writes them after the ones of the ranges above.  A row with
// no more eligible keys than the survivor list holds is scored directly, and a
// row whose filter under-collected (or whose lists overflowed) is recomputed
// exactly; both by the range-0 workgroup with a streaming top-k.
template <int G>
__global__ __launch_bounds__(kSelThreads) void fused_select_kernel(FusedArgs a, int32_t* __restrict__ idx,
                                                                   float* __restrict__ val) {
  extern __shared__ uint64_t buf[];
  __shared__ int act[kD];          // active channels ascending (streaming path)
  __shared__ float qa[kD];         // q of this row's head per active channel
  __shared__ int nact;
  __shared__ int s_count, s_above;
  __shared__ uint64_t s_thr;
  __shared__ int wc[2];
  __shared__ uint32_t s_sub[kSlots];
  const int part = blockIdx.x, r = blockIdx.y, u = r / G, h = r % G, tid = threadIdx.x, lane = tid & 63,
            wave = tid >> 6;
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  const int k = a.k;
  if (tid < kSlots) s_sub[tid] = gload(a.ws.cnt + r * kSlots + tid);
  if (tid == 0) {
    s_count = 0;
    s_above = 0;
    s_thr = 0ull;
  }
  __syncthreads();
  uint32_t C = 0;
  bool sub_over = false;
  for (int q2 = 0; q2 < kSlots; ++q2) {
    C += s_sub[q2];
    sub_over |= s_sub[q2] > (uint32_t)a.ws.scap;
  }
  const float tau = gload(a.ws.tau + r);
  const bool direct = hi - lo <= a.ws.cap;
  const bool fallback =
      !direct && (sub_over || C > (uint32_t)kSelCap || C < (uint32_t)k || gload(a.ws.uovf + u) != 0u || tau == kNegInf);
  if (!direct && !fallback) {
    const uint32_t ub = gload(a.ws.bnd + r * kSlots + part);
    const uint32_t lb = part + 1 < kSlots ? gload(a.ws.bnd + r * kSlots + part + 1) : 0u;
    int above = 0;
    for (uint32_t i = tid; i < C; i += kSelThreads) {  // element i of the concatenated sub-lists
      int q2 = 0;
      uint32_t off = i;
      while (off >= s_sub[q2]) off -= s_sub[q2++];
      const uint64_t v = gload(a.ws.cand + ((int64_t)r * kSlots + q2) * a.ws.scap + off);
      const uint32_t key = (uint32_t)(v >> 32);
      if (key > ub) {
        ++above;
      } else if (key > lb) {
        buf[atomicAdd(&s_count, 1)] = v;
      }
    }
    if (above) atomicAdd(&s_above, above);
    __syncthreads();
    const int off0 = s_above, cnt = s_count;
    if (off0 >= k || cnt == 0) return;
    int P2 = 1;
    while (P2 < cnt) P2 <<= 1;
    for (int i = cnt + tid; i < P2; i += kSelThreads) buf[i] = 0ull;
    __syncthreads();
    bitonic_desc(buf, P2);
    for (int x = tid; x < cnt && off0 + x < k; x += kSelThreads) {
      const uint64_t c = buf[x];
      idx[(int64_t)r * k + off0 + x] = (int32_t)(~(uint32_t)(c & 0xFFFFFFFFull));
      if (val) val[(int64_t)r * k + off0 + x] = key_to_score((uint32_t)(c >> 32));
    }
    return;
  }
  if (part != 0) return;
  // streaming top-k over all eligible keys with exact scores
  {
    int t = 0;
    if (tid < kD) {
      t = gload(a.depths + (int64_t)u * kD + tid);
      t = t > kPlanes ? kPlanes : t;
    }
    const bool on = tid < kD && t > 0;
    const uint64_t m = __ballot(on);
    if (tid < kD && lane == 0) wc[wave] = __popcll(m);
    __syncthreads();
    if (on) act[(wave == 1 ? wc[0] : 0) + __popcll(m & lanemask_lt(lane))] = tid | (t << 8);
    if (tid == 0) {
      nact = wc[0] + wc[1];
      if (fallback) set_status(a.st, FATHOM_DEV_TOPK_FALLBACK);
    }
    __syncthreads();
    for (int x = tid; x < nact; x += kSelThreads)
      qa[x] = load_q(a.q, a.qdt, ((int64_t)u * G + h) * kD + (act[x] & 0xFF));
    __syncthreads();
  }
  const int A = nact;
  const int nwaves = kSelThreads / kWave;
  const int64_t bfirst = lo / kBlockTokens, bend = (hi + kBlockTokens - 1) / kBlockTokens;
  for (int64_t bb = bfirst; bb < bend; bb += nwaves) {
    const int64_t b = bb + wave;
    const int64_t i = b * kBlockTokens + lane;
    const bool elig = b < bend && i >= lo && i < hi;
    uint64_t comp = 0ull;
    if (elig) {
      const float s = exact_score1(act, A, qa, a, u, b, lane);
      comp = ((uint64_t)score_key(s) << 32) | (uint64_t)(~(uint32_t)i);
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
      for (int x = s_count + tid; x < kSelCap; x += kSelThreads) buf[x] = 0ull;
      __syncthreads();
      bitonic_desc(buf, kSelCap);
      if (tid == 0) {
        s_count = k;
        s_thr = buf[k - 1];
      }
      for (int x = k + tid; x < kSelCap; x += kSelThreads) buf[x] = 0ull;
      __syncthreads();
    }
  }
  const int count = s_count;
  int P2 = 1;
  while (P2 < count) P2 <<= 1;
  for (int x = count + tid; x < P2; x += kSelThreads) buf[x] = 0ull;
  __syncthreads();
  bitonic_desc(buf, P2 > 1 ? P2 : 2);
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
  dim3 gs((unsigned)((fa.ws.s_groups + kFW - 1) / kFW), (unsigned)U);
  hipLaunchKernelGGL(fused_sample_kernel<G>, gs, dim3(kFT), 0, s, fa);
  hipLaunchKernelGGL(fused_tau_kernel, dim3(R), dim3(kSelThreads), 0, s, fa, G);
  dim3 gf((unsigned)fa.ws.nwg, (unsigned)U);
  hipLaunchKernelGGL(fused_full_kernel<G>, gf, dim3(kFT), 0, s, fa);
  hipLaunchKernelGGL(fused_select_kernel<G>, dim3(kSlots, R), dim3(kSelThreads), (size_t)kSelCap * 8, s, fa, idx, val);
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
