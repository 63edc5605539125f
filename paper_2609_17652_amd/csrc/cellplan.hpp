// The cell plan of a unit for the cell filter (filter.hip): its active
// channels in proxy order (depth descending, channel ascending), the cells
// (channel, plane) packed plane-major, each cell's plane row and scaled query,
// and the tables of the exact re-scoring chain (channels ascending).  The
// sample pass (fused.hip) builds it once per unit and call into the
// workspace; every workgroup of the filter copies it into LDS.  Not part of
// the C ABI.
#pragma once

#include "fused.hpp"

namespace fathom {

constexpr int kCG = 20;          // row groups at most (5 slices of 4)
constexpr int kCC = 4 * kCG;     // cells at most
constexpr int kCA = 80;          // active channels at most

struct alignas(16) CellPlan {
  int A, rg, C, ok;        // active channels, row groups, cells, the unit fits this pass
  int np[4];               // cells of plane p: the channels of depth > p
  int base[5];             // first cell of plane p (base[4] = C)
  double Kc, Kch, Eabs;    // E = unit Kc + delta Kch + Eabs (unit: delta, or delta / 128 for fine weights)
  uint32_t rrow[kCG][2];   // row group g: plane rows 4 j + p of its 4 cells (16-bit halves, kCPad: none)
  alignas(16) float qrg[kCG][4][4];  // row group g, head h, cell k: -q 2^-p of the cell (0 past the cells and for heads >= G)
  alignas(16) int px[kCA];           // ascending position y -> proxy index x (padded to a multiple of 8: x = A)
  alignas(16) float qa[kCA][4];      // q by ascending position and head (re-scoring; 0 on padding)
  alignas(16) float zo[kCA];         // -(1 - 2^-t) by ascending position: khat = (u / 8 + zo) a16, exact (0 on padding)
  float tau[4];
  uint8_t cx[kCC];         // cell -> proxy index of its channel (0 past the cells)
  uint8_t pj[kCA];         // proxy index -> channel
  uint8_t py[kCA];         // proxy index -> ascending position (q of proxy x: qa[py[x]])
};
constexpr uint32_t kCPad = 0xFFFFu;

typedef unsigned int PlanWord __attribute__((ext_vector_type(4)));  // plans move 16 bytes a thread and step
constexpr int kPlanWords = (int)((sizeof(CellPlan) + 15) / 16);
constexpr int kPlanSteps = 2;  // copy steps of 256 threads
static_assert(sizeof(CellPlan) % 16 == 0 && sizeof(CellPlan) <= kPlanBytes, "a unit's plan fits its workspace slot");
static_assert(kPlanWords <= kPlanSteps * kFT, "two 16-byte words per thread copy a plan");

// ---------------------------------------------------------------- plan
// Depth and q of channel tid (< 128), read by the kernel before its other
// preamble work.
struct CellPre {
  int t;
  float q[4];
};
__device__ __forceinline__ CellPre cell_load(const FusedArgs& a, int u) {
  const int tid = threadIdx.x, G = a.G;
  CellPre r;
  r.t = 0;
#pragma unroll
  for (int h = 0; h < 4; ++h) r.q[h] = 0.0f;
  if (tid < kD) {
    r.t = gload(a.depths + (int64_t)u * kD + tid);
#pragma unroll
    for (int h = 0; h < 4; ++h)
      if (h < G) r.q[h] = load_q(a.q, a.qdt, ((int64_t)u * G + h) * kD + tid);
  }
  if (r.t > kPlanes) r.t = kPlanes;
  return r;
}

// Builds the plan of unit u (all threads of the workgroup).  P.ok is false
// when the unit exceeds this pass's limits or has no active channel.
__device__ __forceinline__ void cell_plan(CellPlan& P, const FusedArgs& a, const CellPre& pre) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, G = a.G;
  __shared__ int cnt[2][kPlanes + 1];
  __shared__ int sact[kD];  // proxy index -> channel j | depth << 8
  const int t = pre.t;
  uint64_t bal[kPlanes + 1];
#pragma unroll
  for (int v = 1; v <= kPlanes; ++v) bal[v] = __ballot(tid < kD && t == v);
  if (tid < kD && lane == 0) {
#pragma unroll
    for (int v = 1; v <= kPlanes; ++v) cnt[wave][v] = __popcll(bal[v]);
  }
  __syncthreads();
  int first[kPlanes + 1], A = 0;
#pragma unroll
  for (int v = kPlanes; v >= 1; --v) {
    first[v] = A;
    A += cnt[0][v] + cnt[1][v];
  }
  int np[kPlanes];  // channels with depth > p
#pragma unroll
  for (int p = 0; p < kPlanes; ++p) {
    np[p] = 0;
#pragma unroll
    for (int v = p + 1; v <= kPlanes; ++v) np[p] += cnt[0][v] + cnt[1][v];
  }
  int base[kPlanes + 1];  // cells plane-major without padding: cell base[p] + x = (plane p, proxy channel x)
  base[0] = 0;
#pragma unroll
  for (int p = 0; p < kPlanes; ++p) base[p + 1] = base[p] + np[p];
  const int C = base[kPlanes], rg = (C + 3) >> 2;
  const bool ok = G <= 4 && A > 0 && A <= kCA && C <= kCC;
  if (tid == 0) {
    P.A = A;
    P.rg = rg;
    P.C = C;
    P.ok = ok;
#pragma unroll
    for (int p = 0; p < kPlanes; ++p) {
      P.np[p] = np[p];
      P.base[p] = base[p];
    }
    P.base[kPlanes] = C;
    const double cells = (double)C;
    P.Kc = cells / 4.0 * (1.0 + 0x1p-20);
    P.Kch = (double)A * (double)A * 127.0 * 0x1p-24 * (1.0 + 0x1p-20);
    P.Eabs = (double)A * 0x1p-120;
  }
  if (!ok) {
    __syncthreads();
    return;
  }
  int xp = -1;  // this channel's proxy index
  if (tid < kD && t > 0) {
    xp = first[t] + (wave == 1 ? cnt[0][t] : 0) + __popcll(bal[t] & lanemask_lt(lane));
    sact[xp] = tid | (t << 8);
    P.pj[xp] = (uint8_t)tid;
    // ascending position: active channels below this one
    const uint64_t on = bal[1] | bal[2] | bal[3] | bal[4];
    int y = __popcll(on & lanemask_lt(lane));
    if (wave == 1) y += cnt[0][1] + cnt[0][2] + cnt[0][3] + cnt[0][4];
    P.px[y] = xp;
    P.py[xp] = (uint8_t)y;
    P.zo[y] = -(1.0f - ldexpf(1.0f, -t));
#pragma unroll
    for (int h = 0; h < 4; ++h) P.qa[y][h] = pre.q[h];
  }
  if (tid >= A && tid < ((A + 7) & ~7)) {  // chain padding: q = 0 adds +0 to every head's score
    P.px[tid] = A;
    P.zo[tid] = 0.0f;
#pragma unroll
    for (int h = 0; h < 4; ++h) P.qa[tid][h] = 0.0f;
  }
  __syncthreads();
  // cells: thread c fills cell c = 4 g + k (row group g, byte k).  Its weight
  // uses -q 2^-p, so every cell shares one rounding constant per group and
  // head (the scaling is exact unless q 2^-p is subnormal, and then the cell's
  // weight is 0 either way: |q a16 2^-p| < 2^-110 is far below delta / 2)
  if (tid < kCC) {
    const int c = tid, g = c >> 2, k = c & 3;
    int p = 0;
#pragma unroll
    for (int pp = 1; pp < kPlanes; ++pp) p += c >= base[pp];
    const bool real = c < C;
    const int x = real ? c - base[p] : 0;
    const uint32_t row = real ? (uint32_t)(4 * (sact[x] & 0xFF) + p) : kCPad;
    // cells 0,1 -> rrow[g][0], cells 2,3 -> rrow[g][1] (16-bit halves)
    const uint32_t part = row << (16 * (k & 1));
    const uint32_t other = __shfl_xor(part, 1, kWave);
    if ((k & 1) == 0) P.rrow[g][k >> 1] = part | other;
#pragma unroll
    for (int h = 0; h < 4; ++h) P.qrg[g][h][k] = real && h < G ? -ldexpf(P.qa[P.py[x]][h], -p) : 0.0f;
    P.cx[c] = (uint8_t)x;
  }
  if (tid < 4) P.tau[tid] = kNegInf;
  __syncthreads();
}

}  // namespace fathom
