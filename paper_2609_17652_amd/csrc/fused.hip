// fathom_scan_topk: the decode-step scan + top-k of Sec. 3.2-3.3 and Sec. 2,
// fused so that no score array is written.
//
// The exact result is defined by the documented fp32 scores (exact
// dequantisation, fma(q, khat, acc) over active channels ascending) and the
// (score desc, index asc) order.  To avoid computing those scores for every
// key, each key first gets an integer proxy with a rigorous error bound, and
// only keys the bound cannot exclude are scored exactly.
//
// Proxy.  Per key and active channel a (depth t), the prefix digit
//   u = sum_{p<t} b_p 2^(3-p) in [0, 15]   (= c^(t) << (4 - t))
// gives khat = (2u - zmax) a16 / 16 with zmax = 16 - 2^(4-t).  Per superquad
// (16 consecutive blocks, 8 when A > 64) and head, delta = 2^e is the smallest
// power of two with max |q a16| / delta <= 127 over its blocks and channels, and
// W = rne(q a16 / delta) is an int8 weight per (block, head, channel).  With
//   S = sum_a W_a u_a  and  b = sum_a W_a zmax_a,
// the proxy (delta / 16)(2S - b) differs from the documented score by at most
//   E = delta (sum_a zmax_a / 32 + A^2 127 2^-24) + A 2^-120
// (weight rounding, the A roundings of the fp32 chain, subnormal flushes).
// A key is a candidate for head h iff proxy + E >= tau_h, i.e.
//   S >= thr = floor((floor((tau - E) 16 / delta) - 1 + b) / 2).
//
// That proxy is the wide full pass below (units of more cells than the
// launched cell filter stages); the cell filter (filter.hip) serves the
// others with a per-cell proxy.
//
// Mapping to CDNA4.  A wave handles 4 blocks ("quad", 256 keys) at a time.
// Lane l owns octet m = (l >> 1) & 7, half hb = l & 1 of block l >> 4, i.e.
// keys 8m + 4hb + mu, mu = 0..3.  Row groups (one plane p of the 4 proxy
// channels of a digit dword) are staged in LDS byte-transposed and split into
// nibble copies pre-shifted by 3 - p, so each lane's staged dword holds its 4
// keys' bits at positions mu + 3 - p of byte K; one v_and_or per (row group,
// key) builds the digit dword scaled by 2^mu.  S comes from
// v_mfma_i32_16x16x64_i8 with A = block-diagonal weights (row 4g + h, k-group
// g: block g of the quad, head h) and B = the digit dwords of 16 channels:
// accumulator r of lane l is S for head r of lane l's key mu, scaled by 2^mu.
// The accumulators start at -(thr << mu), so a key is a candidate iff one of
// its four accumulators is >= 0.
//
// Candidates are queued per wave in LDS with their digits; full batches are
// scored exactly (channels ascending, scales kept in an LDS ring) and the keys
// with score >= tau are appended to their row's survivor list.
//
// Passes (launches): (1) sample: exact scores of every s-th quad, the 2
// largest per (block, head), and per unit the rows' call state and the cell
// plan; (2) tau, only for the wide pass or G > 4: per row the m-th largest
// sample, m ~ 1.25 k sampled / eligible + 16 (the cell filter finds the same
// tau itself); (3) the full pass: the cell filter, and the wide pass above
// when launched; (4) select: 8 workgroups per row share out its top k
// positions by a histogram of the survivors' scores and order their share in
// LDS, and rows with at most 2k + 2048 eligible keys, and rows whose
// survivors cannot give the top k (fewer than k reached tau, the list
// overflowed, or too many equal scores for one workgroup's share;
// FATHOM_DEV_TOPK_FALLBACK), are computed from exact scores by a chunked
// selection in the same launch.  The result never depends on tau; it only
// decides how much work is saved.
#include <atomic>
#include <type_traits>
#include <mutex>

#include "cellplan.hpp"

namespace fathom {

size_t fused_ws_bytes(int R, int U, int64_t nb_cap, int k) {
  if (nb_cap < 1) nb_cap = 1;
  const size_t xch = (size_t)exact_chunks(nb_cap), pk = (size_t)exact_pk(k);
  return a256((size_t)R * 4) + a256((size_t)R * kCntStride * 4) + a256((size_t)U * kPools * kPoolStride * 4) +
         (size_t)U * kPlanBytes +
         a256((size_t)R * fused_lcap(k) * 8) +
         a256((size_t)U * 4) +
         a256((size_t)R * kSmpRow * 4) +
         a256((size_t)(1 + R) * 4) + a256((size_t)R * xch * pk * 8) + a256((size_t)R * xch * 4) +
         a256((size_t)R * xch * 8);
}


// ---------------------------------------------------------------- unit plan
// Proxy channel order: depth descending, channel ascending.  Digit dword d
// holds proxy channels 4d..4d+3; its row groups are planes 0 .. t(4d)-1 (its
// first channel is its deepest).  Slice s = dwords 4s..4s+3 = one MFMA.
constexpr uint32_t kPadRow = 0xFFFFu;
struct alignas(16) Plan {
  int A, ndw, nsl, ok;
  double Ku, Eabs;             // E = delta * Ku + Eabs
  int act[kD];                 // proxy order: j | t << 8
  int pord[kD];                // channel-ascending position x -> proxy index
  uint32_t pordb[kD / 4];      // the same, 4 positions per dword (byte x mod 4)
  float qa[kD][4];             // q by channel-ascending position and head (0 for h >= G)
  float za[kD];                // zmax / 16 by channel-ascending position
  float qp[kD][4];             // q (fp32) by proxy index and head (0 for h >= G)
  uint32_t q16[kMaxDw][4][2];  // fp16 q of proxy channels 4d..4d+3, head h: (K0,K1), (K2,K3)
  uint32_t zmx[kMaxDw];        // zmax of proxy channels 4d..4d+3, byte K
  float zm16[kD];              // zmax / 16 by proxy index
  int slrg[kMaxSl + 1];        // slice s: row groups [slrg[s], slrg[s+1])
  uint32_t rgrow[kMaxRg][2];   // row group g: plane rows (4j + p) of bytes K = 0..3 as 16-bit halves
  int rgp[kMaxRg];             // row group g: plane p
  int rgslot[kMaxRg];          // row group g: staging slot 4 * (d mod 4) + p within its slice
  int slmask[kMaxSl];          // slice s: bit 4 dd + p set iff dword 4s + dd has plane p
  float tau[4];
};

// The plan's global reads (thread j < 128: channel j's depth and its q for
// every head), issued by a kernel before its other preamble work.
struct PlanPre {
  int t;
  float q[4];
};
template <bool QF16>
__device__ __forceinline__ PlanPre plan_load(const FusedArgs& a, int u) {
  const int tid = threadIdx.x, G = a.G;
  PlanPre r;
  r.t = 0;
  float x[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (tid < kD) {
    r.t = gload(a.depths + (int64_t)u * kD + tid);
#pragma unroll
    for (int h = 0; h < 4; ++h) {  // heads past G (at most 4 here) re-read head 0
      const int64_t i = ((int64_t)u * G + (h < G ? h : 0)) * kD + tid;
      if (QF16)
        x[h] = __half2float(__ushort_as_half(((const __attribute__((address_space(1))) uint16_t*)a.q)[i]));
      else
        x[h] = ((const __attribute__((address_space(1))) float*)a.q)[i];
    }
  }
#pragma unroll
  for (int h = 0; h < 4; ++h) r.q[h] = h < G ? x[h] : 0.0f;
  return r;
}

__device__ void plan_setup(Plan& P, const FusedArgs& a, int u, const PlanPre& pre) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = a.G;
  __shared__ int cnt[2][5];
  const int t = pre.t > kPlanes ? kPlanes : pre.t;
  float qv4[4];  // this channel's q, loaded with its depth
#pragma unroll
  for (int h = 0; h < 4; ++h) qv4[h] = pre.q[h];
  uint64_t bal[5];
#pragma unroll
  for (int v = 1; v <= 4; ++v) bal[v] = __ballot(tid < kD && t == v);
  if (tid < kD && lane == 0) {
#pragma unroll
    for (int v = 1; v <= 4; ++v) cnt[wave][v] = __popcll(bal[v]);
  }
  __syncthreads();
  int first[5];
  {
    int pos = 0;
#pragma unroll
    for (int v = 4; v >= 1; --v) {
      first[v] = pos;
      pos += cnt[0][v] + cnt[1][v];
    }
    if (tid == 0) {
      P.A = pos;
      P.ndw = (pos + 3) >> 2;
      P.nsl = (pos + 15) >> 4;
      P.ok = G <= 4;
    }
  }
  if (tid < kD && t > 0) {  // this channel's proxy index a_
    const int a_ = first[t] + (wave == 1 ? cnt[0][t] : 0) + __popcll(bal[t] & lanemask_lt(lane));
    P.act[a_] = tid | (t << 8);
    const uint64_t on = bal[1] | bal[2] | bal[3] | bal[4];
    const int w0 = cnt[0][1] + cnt[0][2] + cnt[0][3] + cnt[0][4];
    P.pord[(wave == 1 ? w0 : 0) + __popcll(on & lanemask_lt(lane))] = a_;
#pragma unroll
    for (int h = 0; h < 4; ++h) P.qp[a_][h] = qv4[h];
    P.zm16[a_] = (float)(16 - (16 >> t)) * 0.0625f;
  }
  {
    int nact = 0;
#pragma unroll
    for (int v = 1; v <= 4; ++v) nact += cnt[0][v] + cnt[1][v];
    if (tid >= nact && tid < kD) {  // proxy indices past the active channels
#pragma unroll
      for (int h = 0; h < 4; ++h) P.qp[tid][h] = 0.0f;
      P.zm16[tid] = 0.0f;
    }
  }
  __syncthreads();
  const int A = P.A, ndw = P.ndw;
  if (tid < kMaxDw * 4) {  // q16 pairs and zmax bytes
    const int d = tid >> 2, h = tid & 3;
    uint32_t pr[2] = {0u, 0u};
#pragma unroll
    for (int K = 0; K < 4; ++K) {
      const float qv = P.qp[4 * d + K][h];  // fp16-exact when the queries are fp16
      const uint32_t hb = (uint32_t)__half_as_ushort(__float2half_rn(qv));
      pr[K >> 1] |= hb << (16 * (K & 1));
    }
    P.q16[d][h][0] = pr[0];
    P.q16[d][h][1] = pr[1];
    if (h == 0) {
      uint32_t z = 0u;
#pragma unroll
      for (int K = 0; K < 4; ++K) z |= (uint32_t)(int)(P.zm16[4 * d + K] * 16.0f) << (8 * K);
      P.zmx[d] = z;
    }
  }
  __syncthreads();
  if (tid < kD) {  // channel-ascending copies for the exact re-scoring
    const int ai = tid < A ? P.pord[tid] : 0;
#pragma unroll
    for (int h = 0; h < 4; ++h) P.qa[tid][h] = tid < A ? P.qp[ai][h] : 0.0f;
    P.za[tid] = tid < A ? P.zm16[ai] : 0.0f;
  }
  if (tid < kD / 4) {
    uint32_t w = 0u;
#pragma unroll
    for (int K = 0; K < 4; ++K) w |= (uint32_t)(4 * tid + K < A ? P.pord[4 * tid + K] : 0) << (8 * K);
    P.pordb[tid] = w;
  }
  // row groups, in parallel.  Depths never increase along the proxy order, so
  // within slice s the dwords with plane p are dd < c_p (plane-major order):
  // row group (d = 4 s + dd, p) has index slrg[s] + c_0 + .. + c_(p-1) + dd.
  __shared__ int snr[kMaxDw], scp[kMaxSl][kPlanes], srows[kMaxSl];
  if (tid < kMaxDw) snr[tid] = tid < ndw ? (P.act[4 * tid] >> 8) : 0;  // planes of dword tid
  int zpart = 0;  // sum of zmax over the active channels (wave 0)
  if (wave == 0) {
    zpart = (lane < A ? (int)(P.zm16[lane] * 16.0f) : 0) + (lane + kWave < A ? (int)(P.zm16[lane + kWave] * 16.0f) : 0);
    zpart = wave_sum_int(zpart);
  }
  __syncthreads();
  if (tid < kMaxSl * kPlanes) {  // c_p of slice tid / 4
    const int sl = tid >> 2, p = tid & 3;
    int c = 0;
#pragma unroll
    for (int dd = 0; dd < 4; ++dd) c += snr[4 * sl + dd] > p;
    scp[sl][p] = c;
  }
  __syncthreads();
  if (tid == 0) {
    int g = 0;
    for (int sl = 0; sl < kMaxSl; ++sl) {
      P.slrg[sl] = g;
      srows[sl] = g;
      int msk = 0;
      for (int p = 0; p < kPlanes; ++p) g += scp[sl][p];
      for (int dd = 0; dd < 4; ++dd) msk |= ((1 << snr[4 * sl + dd]) - 1) << (4 * dd);
      P.slmask[sl] = msk;
    }
    P.slrg[kMaxSl] = g;
    const double zs = (double)zpart;
    P.Ku = (zs / 32.0 + (double)A * (double)A * 127.0 * 0x1p-24) * (1.0 + 0x1p-20);
    P.Eabs = (double)A * 0x1p-120;
  }
  __syncthreads();
  if (tid < kMaxDw * kPlanes) {  // row group (dword d, plane p)
    const int d = tid >> 2, p = tid & 3, sl = d >> 2, dd = d & 3;
    if (snr[d] > p) {
      int g = srows[sl] + dd;
      for (int p2 = 0; p2 < p; ++p2) g += scp[sl][p2];
      P.rgslot[g] = 4 * dd + p;
      uint32_t h2[2] = {0u, 0u};
#pragma unroll
      for (int K = 0; K < 4; ++K) {
        const int x = 4 * d + K;
        uint32_t r = kPadRow;
        if (x < A && (P.act[x] >> 8) > p) r = (uint32_t)(4 * (P.act[x] & 0xFF) + p);
        h2[K >> 1] |= r << (16 * (K & 1));
      }
      P.rgrow[g][0] = h2[0];
      P.rgrow[g][1] = h2[1];
      P.rgp[g] = p;
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------- per-wave state
// NSLM slices (16 NSLM proxy channels at most), superquads of SQB blocks, RQ
// superquads of scales kept for re-scoring, QCAP queued candidates.
template <int NSLM, int SQB, int RQ, int QCAP>
struct alignas(16) WaveLdsT {
  uint32_t st[16][kStP];                     // one slice's staged row groups (slot 4 (d mod 4) + p)
  uint32_t W[SQB * 4 * 4 * NSLM];            // int8 weights [block][head][dword < 4 nsl] of the superquad
  int32_t ci[SQB][4][4];                     // [block][mu][head] accumulator start
  uint16_t scl[RQ * SQB * (16 * NSLM + 2)];  // fp16 scales [ring slot][block][proxy channel], rows of 4 ndw + 2
  float amx[16 * NSLM];                      // per proxy channel: largest scale of the superquad
  uint32_t qd[QCAP * 4 * NSLM];              // queued digit dwords, 4 nsl per entry
  uint32_t qi[QCAP];                         // queued key index
  uint32_t qf[QCAP];                         // queued mu | heads << 2 | ring slot << 8 | block << 12
};

typedef __attribute__((ext_vector_type(4))) int v4i;
typedef _Float16 h2t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pkfma16(uint32_t x, uint32_t y, uint32_t z) {
  const h2t r = __builtin_elementwise_fma(__builtin_bit_cast(h2t, x), __builtin_bit_cast(h2t, y),
                                          __builtin_bit_cast(h2t, z));
  return __builtin_bit_cast(uint32_t, r);
}

struct SqInfo {
  int e;          // delta = 2^e (this lane's head: lane >> 4)
  bool valid;     // a bound exists for this superquad and head
};

// Scales of one superquad held in registers between their loads and their
// use: lane x (and x + 64 when NCH = 2) owns proxy channel x, 2 blocks a dword.
template <int NCH, int SQB>
struct SclRegs {
  uint32_t v[NCH][SQB / 2];
};

template <int NCH, int SQB>
__device__ __forceinline__ void scl_issue(SclRegs<NCH, SQB>& r, const Plan& P, const FusedArgs& a, int u,
                                          int64_t sb0) {
  const int lane = threadIdx.x & 63, A = uni(P.A);
  const uint16_t* Su = a.scales + (int64_t)u * kD * a.nb_cap;
  const bool vec = (a.nb_cap & 3) == 0 && sb0 + SQB <= a.nb_cap && (sb0 & 3) == 0 &&
                   (reinterpret_cast<uintptr_t>(a.scales) & 7) == 0;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int x = lane + kWave * c;
#pragma unroll
    for (int i = 0; i < SQB / 2; ++i) r.v[c][i] = 0u;
    if (x < A) {
      const uint16_t* row = Su + (int64_t)(P.act[x] & 0xFF) * a.nb_cap + sb0;
      if (vec) {
#pragma unroll
        for (int i = 0; i < SQB / 4; ++i) {
          const uint64_t v2 = gload(reinterpret_cast<const uint64_t*>(row) + i);
          r.v[c][2 * i] = (uint32_t)v2;
          r.v[c][2 * i + 1] = (uint32_t)(v2 >> 32);
        }
      } else {
#pragma unroll
        for (int b = 0; b < SQB; ++b) {
          const uint32_t h = sb0 + b < a.nb_cap ? (uint32_t)gload(row + b) : 0u;
          r.v[c][b >> 1] |= h << (16 * (b & 1));
        }
      }
    }
  }
}

// Writes the superquad's scales to ring slot `slot` ([block][proxy channel])
// and fixes delta per head: lanes (c, h) reduce max_a |q_ah| amax_a over a = c
// (mod 16).
template <bool QF16, int NCH, int SQB, class WL>
__device__ SqInfo scl_commit(const SclRegs<NCH, SQB>& r, const Plan& P, WL& W, int slot) {
  const int lane = threadIdx.x & 63;
  const int A = uni(P.A), ap = 4 * uni(P.ndw), aps = ap + 2;  // row stride: an odd number of dwords
  uint16_t* sdst = &W.scl[slot * SQB * aps];
  bool nf = false;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int x = lane + kWave * c;
    if (x < ap) {
      uint32_t mx = 0u;
#pragma unroll
      for (int b = 0; b < SQB; ++b) {
        const uint32_t h = (r.v[c][b >> 1] >> (16 * (b & 1))) & 0xFFFFu;
        sdst[b * aps + x] = (uint16_t)h;
        const uint32_t m = h & 0x7FFFu;
        mx = m > mx ? m : mx;
      }
      nf |= mx >= 0x7C00u;
      W.amx[x] = half_bits_to_float((uint16_t)(mx >= 0x7C00u ? 0u : mx));
    }
  }
  nf = __ballot(nf) != 0ull;
  wave_lds_sync();
  const int c = lane & 15, h = lane >> 4;
  float M = 0.0f;
  for (int x = c; x < A; x += 16) M = fmaxf(M, __fmul_rn(fabsf(P.qp[x][h]), W.amx[x]));
#pragma unroll
  for (int m = 1; m < 16; m <<= 1) M = fmaxf(M, __shfl_xor(M, m, kWave));
  SqInfo s;
  s.e = 0;
  s.valid = !nf && M <= 3.402823466e38f;
  if (M > 0.0f && s.valid) {
    int E;
    (void)frexpf(M, &E);  // M in [2^(E-1), 2^E)
    s.e = M <= 127.0f * ldexpf(1.0f, E - 7) ? E - 7 : E - 6;
    if (QF16) s.valid = s.e >= -24 && s.e <= 5;  // 1536 * 2^e is a normal fp16
    else s.valid = s.e >= -100 && s.e <= 100;
  }
  return s;
}

// Weights and accumulator starts of the superquad.  Lane (block beta = lane &
// 15, head h = lane >> 4).
template <bool QF16, int SQB, class WL>
__device__ void superquad_weights(const Plan& P, WL& W, const FusedArgs& a, const SqInfo& si, int slot) {
  const int lane = threadIdx.x & 63, beta = lane & 15, h = lane >> 4;
  const int ndw = uni(P.ndw), aps = 4 * ndw + 2, ws = 4 * uni(P.nsl);
  if (beta < SQB) {
    int bias = 0;
    uint32_t* wdst = &W.W[(beta * 4 + h) * ws];  // dwords ndw .. ws - 1 stay zero
    const uint16_t* srow = &W.scl[(slot * SQB + beta) * aps];
    if (si.valid) {
      if (QF16) {
        const uint32_t cb = (uint32_t)((si.e + 25) << 10 | 0x200);
        const uint32_t c2 = cb | cb << 16;
        for (int d = 0; d < ndw; ++d) {
          const uint2 qq = *reinterpret_cast<const uint2*>(&P.q16[d][h][0]);
          const uint2 aa = make_uint2(*reinterpret_cast<const uint32_t*>(&srow[4 * d]),
                                      *reinterpret_cast<const uint32_t*>(&srow[4 * d + 2]));  // rows: 4-byte aligned
          const uint32_t r0 = pkfma16(qq.x, aa.x, c2), r1 = pkfma16(qq.y, aa.y, c2);
          const uint32_t wd = __builtin_amdgcn_perm(r1, r0, 0x06040200u);
          wdst[d] = wd;
          bias = __builtin_amdgcn_sdot4((int)wd, (int)P.zmx[d], bias, false);
        }
      } else {
        const float c32 = ldexpf(12582912.0f, si.e);  // 1.5 * 2^(23 + e)
        for (int d = 0; d < ndw; ++d) {
          uint32_t r[4];
#pragma unroll
          for (int K = 0; K < 4; ++K)
            r[K] = __float_as_uint(__fmaf_rn(P.qp[4 * d + K][h], half_bits_to_float(srow[4 * d + K]), c32));
          const uint32_t lo = __builtin_amdgcn_perm(r[1], r[0], 0x0c0c0400u);
          const uint32_t hi = __builtin_amdgcn_perm(r[3], r[2], 0x04000c0cu);
          const uint32_t wd = lo | hi;
          wdst[d] = wd;
          bias = __builtin_amdgcn_sdot4((int)wd, (int)P.zmx[d], bias, false);
        }
      }
    } else {
      for (int d = 0; d < ndw; ++d) wdst[d] = 0u;
    }
    for (int d = ndw; d < ws; ++d) wdst[d] = 0u;
    const bool hv = h < a.G && P.tau[h] != kNegInf;
    int c0[4];
    if (!hv) {
#pragma unroll
      for (int mu = 0; mu < 4; ++mu) c0[mu] = -kNoBound;
    } else if (!si.valid) {
#pragma unroll
      for (int mu = 0; mu < 4; ++mu) c0[mu] = kNoBound;
    } else {
      const double del = ldexp(1.0, si.e);
      const double E = del * P.Ku + P.Eabs;
      double X = ((double)P.tau[h] - E) * 16.0 / del;
      X = floor(X) - 1.0;
      X = X < -2.0 * kThrMax ? -2.0 * kThrMax : X > 2.0 * kThrMax ? 2.0 * kThrMax : X;
      int thr = ((int)X + bias) >> 1;
      thr = thr < -kThrMax ? -kThrMax : thr > kThrMax ? kThrMax : thr;
#pragma unroll
      for (int mu = 0; mu < 4; ++mu) c0[mu] = -(thr * (1 << mu));
    }
#pragma unroll
    for (int mu = 0; mu < 4; ++mu) W.ci[beta][mu][h] = c0[mu];
  }
  wave_lds_sync();
}

// Plane words of slice sl for the quad at block qb0: item (row group rl =
// lane >> 2, block beta = lane & 3), 4 rows.
__device__ __forceinline__ void task_issue(uint64_t (&w)[4], const Plan& P, const FusedArgs& a, int u, int64_t qb0,
                                           int sl) {
  const int lane = threadIdx.x & 63, rl = lane >> 2, beta = lane & 3;
  const int g0 = uni(P.slrg[sl]), ng = uni(P.slrg[sl + 1]) - g0;
#pragma unroll
  for (int K = 0; K < 4; ++K) w[K] = 0ull;
  if (rl < ng) {
    const int g = g0 + rl;
    const uint32_t rr0 = P.rgrow[g][0], rr1 = P.rgrow[g][1];
    const uint32_t rows[4] = {rr0 & 0xFFFFu, rr0 >> 16, rr1 & 0xFFFFu, rr1 >> 16};
    const int64_t b = qb0 + beta;
    const uint64_t* Pu = a.planes + (int64_t)u * kD * kPlanes * a.nb_cap + b;
#pragma unroll
    for (int K = 0; K < 4; ++K)
      if (rows[K] != kPadRow && b < a.nb_cap) w[K] = gload(Pu + (int64_t)rows[K] * a.nb_cap);
  }
}

// Stages the loaded row groups of slice sl: byte transpose, then nibble
// copies shifted so that key mu's plane-p bit lands at mu + 3 - p.
template <class WL>
__device__ __forceinline__ void task_stage(const uint64_t (&w)[4], const Plan& P, WL& W, int sl) {
  const int lane = threadIdx.x & 63, rl = lane >> 2, beta = lane & 3;
  const int g0 = uni(P.slrg[sl]), ng = uni(P.slrg[sl + 1]) - g0;
  if (rl < ng) {
    const int p = P.rgp[g0 + rl];
    uint32_t* dst = &W.st[P.rgslot[g0 + rl]][16 * beta];
    const uint32_t sl_ = (uint32_t)(3 - p), sr_ = (uint32_t)(1 + p);
#pragma unroll
    for (int hw = 0; hw < 2; ++hw) {
      const uint32_t a0 = (uint32_t)(w[0] >> (32 * hw)), a1 = (uint32_t)(w[1] >> (32 * hw));
      const uint32_t a2 = (uint32_t)(w[2] >> (32 * hw)), a3 = (uint32_t)(w[3] >> (32 * hw));
      const uint32_t t01l = __builtin_amdgcn_perm(a1, a0, 0x05010400u);
      const uint32_t t01h = __builtin_amdgcn_perm(a1, a0, 0x07030602u);
      const uint32_t t23l = __builtin_amdgcn_perm(a3, a2, 0x05010400u);
      const uint32_t t23h = __builtin_amdgcn_perm(a3, a2, 0x07030602u);
      uint32_t T[4];
      T[0] = __builtin_amdgcn_perm(t23l, t01l, 0x05040100u);
      T[1] = __builtin_amdgcn_perm(t23l, t01l, 0x07060302u);
      T[2] = __builtin_amdgcn_perm(t23h, t01h, 0x05040100u);
      T[3] = __builtin_amdgcn_perm(t23h, t01h, 0x07060302u);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = 4 * hw + j;
        dst[2 * m] = T[j] << sl_;
        dst[2 * m + 1] = T[j] >> sr_;
      }
    }
  }
}

// Exact documented scores of the queued keys (lane e < nq), from their queued
// digits and the scales kept in the ring, and their appends to the survivor
// lists.
template <int SQB, class WL>
__device__ __forceinline__ void rescore_batch(const Plan& P, WL& W, const FusedArgs& a, int u, int nq) {
  const int lane = threadIdx.x & 63, G = a.G;
  wave_lds_sync();
  const bool on = lane < nq;
  const uint32_t i = on ? W.qi[lane] : 0u, f = on ? W.qf[lane] : 0u;
  const int mu = (int)(f & 3u), hm = (int)((f >> 2) & 15u);
  const int rs = (int)((f >> 8) & 15u), bq = (int)((f >> 12) & 15u);
  const int A = uni(P.A), ndw = uni(P.ndw), ap = 4 * ndw, stride = 4 * uni(P.nsl);
  const uint8_t* dg = reinterpret_cast<const uint8_t*>(&W.qd[(on ? lane : 0) * stride]);
  const uint16_t* sv = &W.scl[(rs * SQB + bq) * (ap + 2)];  // scale rows of 4 ndw + 2 halves
  // heads h >= G have q = 0 and are never kept: all four chains run
  float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  constexpr int kC = 8;  // channels whose reads are issued together
  for (int x0 = 0; x0 < A; x0 += kC) {
    const uint32_t p0 = (uint32_t)uni((int)P.pordb[x0 >> 2]), p1 = (uint32_t)uni((int)P.pordb[(x0 >> 2) + 1]);
    uint32_t dv[kC], hv[kC];
    float4 q4[kC];
    float zz[kC];
#pragma unroll
    for (int c = 0; c < kC; ++c) {  // positions past A read valid entries that are not used
      const int ai = (int)(((c < 4 ? p0 : p1) >> (8 * (c & 3))) & 0xFFu);
      dv[c] = dg[ai];
      hv[c] = sv[ai];
      q4[c] = *reinterpret_cast<const float4*>(&P.qa[x0 + c][0]);
      zz[c] = P.za[x0 + c];
    }
#pragma unroll
    for (int c = 0; c < kC; ++c) {
      if (x0 + c < A) {
        const uint32_t u4 = (dv[c] >> mu) & 15u;
        const float af = half_bits_to_float((uint16_t)hv[c]);
        const float khat = __fmaf_rn((float)u4, __fmul_rn(af, 0.125f), -__fmul_rn(af, zz[c]));
        s[0] = __fmaf_rn(q4[c].x, khat, s[0]);
        s[1] = __fmaf_rn(q4[c].y, khat, s[1]);
        s[2] = __fmaf_rn(q4[c].z, khat, s[2]);
        s[3] = __fmaf_rn(q4[c].w, khat, s[3]);
      }
    }
  }
  // lane h reserves head h's slots in its row's list with one atomic
  uint32_t key[4], pre[4] = {0u, 0u, 0u, 0u}, cl = 0u;
  bool keep[4];
  bool any = false;
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    keep[h] = h < G && on && ((hm >> h) & 1) && s[h] >= P.tau[h];
    key[h] = score_key(s[h]);
    const uint64_t bm = __ballot(keep[h]);
    if (bm == 0ull) continue;
    any = true;
    if (lane == h) cl = (uint32_t)__popcll(bm);
    pre[h] = (uint32_t)__popcll(bm & lanemask_lt(lane));
  }
  if (any) {
    uint32_t base = 0u;
    if (cl) base = gatomic_add(&a.ws.cnt[(u * G + lane) * kCntStride], cl);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const uint32_t pos = __shfl(base, h, kWave) + pre[h];
      if (keep[h] && pos < (uint32_t)a.ws.lcap)
        gstore(&a.ws.cand[(int64_t)(u * G + h) * a.ws.lcap + pos], ((uint64_t)key[h] << 32) | (uint64_t)(~i));
    }
  }
  wave_lds_sync();
}


// Runs superquads of SQB blocks over blocks [b0, b1) (b0 a multiple of 4) of
// unit u.  The next quad's plane words (one register set per slice) and the
// next superquad's scales are in flight while the current ones are used.
// Candidates of a quad are queued together; a batch is re-scored at the top
// of the next quad once 48 are queued (or before the ring slot holding their
// scales is reused), with a call only when one quad overflows the queue.
template <bool QF16, int NSLM, int SQB, int RQ, int QCAP>
__device__ void wave_run(const Plan& P, WaveLdsT<NSLM, SQB, RQ, QCAP>& W, const FusedArgs& a, int u, int64_t b0,
                         int64_t b1, int64_t nbu, int64_t lo, int64_t hi) {
  constexpr int NCH = NSLM > 4 ? 2 : 1;
  constexpr int kFlushAt = QCAP * 3 / 4;
  const int lane = threadIdx.x & 63;
  const int nsl = uni(P.nsl), stride = 4 * nsl;
  const int kb = 8 * ((lane >> 1) & 7) + 4 * (lane & 1);  // key of mu = 0 within the block
  const int lb = lane >> 4;                              // block of the quad
  const bool wl = ((lane & 15) >> 2) == lb;              // carries weights in the A operand
  const int wh = lane & 3;
  int pending = 0, oldest = 0;
  SclRegs<NCH, SQB> sr;
  scl_issue(sr, P, a, u, b0);
  // one staging pass per slice
  uint64_t ring[NSLM][4];
#pragma unroll
  for (int sl = 0; sl < NSLM; ++sl)
    if (sl < nsl) task_issue(ring[sl], P, a, u, b0, sl);
  int sqi = 0;
  for (int64_t sb0 = b0; sb0 < b1; sb0 += SQB, ++sqi) {
    const int rslot = sqi % RQ;
    if (pending > 0 && oldest <= sqi - RQ) {  // its scales are about to be overwritten
      rescore_batch<SQB>(P, W, a, u, pending);
      pending = 0;
    }
    const SqInfo si = scl_commit<QF16, NCH, SQB>(sr, P, W, rslot);
    if (sb0 + SQB < b1) scl_issue(sr, P, a, u, sb0 + SQB);
    superquad_weights<QF16, SQB>(P, W, a, si, rslot);
    const int64_t sb1 = sb0 + SQB < b1 ? sb0 + SQB : b1;
    for (int64_t qb0 = sb0; qb0 < sb1; qb0 += kQB) {
      if (pending >= kFlushAt) {
        rescore_batch<SQB>(P, W, a, u, pending);
        pending = 0;
      }
      const int qo = (int)(qb0 - sb0);  // quad offset within the superquad
      const bool more = qb0 + kQB < b1;
      v4i dig[4][NSLM];
      v4i acc[4];
#pragma unroll
      for (int mu = 0; mu < 4; ++mu) acc[mu] = *reinterpret_cast<const v4i*>(&W.ci[qo + lb][mu][0]);
#pragma unroll
      for (int sl = 0; sl < NSLM; ++sl) {
        if (sl < nsl) {
          task_stage(ring[sl], P, W, sl);
          if (more) task_issue(ring[sl], P, a, u, qb0 + kQB, sl);
          wave_lds_sync();
          uint32_t Z[4][4];
#pragma unroll
          for (int dd = 0; dd < 4; ++dd)
#pragma unroll
            for (int mu = 0; mu < 4; ++mu) Z[mu][dd] = 0u;
          const int smask = uni(P.slmask[sl]);
#pragma unroll
          for (int dd = 0; dd < 4; ++dd) {
#pragma unroll
            for (int p = 0; p < 4; ++p) {
              if (smask & (1 << (4 * dd + p))) {
                const uint32_t x = W.st[4 * dd + p][lane];
#pragma unroll
                for (int mu = 0; mu < 4; ++mu) Z[mu][dd] |= x & (0x01010101u << (mu + 3 - p));
              }
            }
          }
#pragma unroll
          for (int mu = 0; mu < 4; ++mu) dig[mu][sl] = v4i{(int)Z[mu][0], (int)Z[mu][1], (int)Z[mu][2], (int)Z[mu][3]};
          v4i wv = v4i{0, 0, 0, 0};
          if (wl) wv = *reinterpret_cast<const v4i*>(&W.W[((qo + lb) * 4 + wh) * stride + 4 * sl]);
#pragma unroll
          for (int mu = 0; mu < 4; ++mu) acc[mu] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wv, dig[mu][sl], acc[mu], 0, 0, 0);
          wave_lds_sync();  // staged reads done before the next slice is staged
        }
      }
      const int64_t kbase = (qb0 + lb) * kBlockTokens + kb;  // key of mu = 0
      const bool inner = qb0 * kBlockTokens >= lo && (qb0 + kQB) * kBlockTokens <= hi && qb0 + kQB <= nbu;
      {
        bool fl[4];
        uint64_t M[4];
        int tot = 0;
#pragma unroll
        for (int mu = 0; mu < 4; ++mu) {
          const int64_t i = kbase + mu;
          const bool el = inner || (i >= lo && i < hi && qb0 + lb < nbu);
          const int mx = max(max(acc[mu][0], acc[mu][1]), max(acc[mu][2], acc[mu][3]));
          fl[mu] = el && mx >= 0;
          M[mu] = __ballot(fl[mu]);
          tot += __popcll(M[mu]);
        }
        if (tot > 0) {
          if (pending + tot > QCAP) {  // make room (rare: the flush at the top of a quad usually does)
            rescore_batch<SQB>(P, W, a, u, pending);
            pending = 0;
          }
          if (pending == 0) oldest = sqi;
          const uint32_t meta = (uint32_t)rslot << 8 | (uint32_t)(qo + lb) << 12;
#pragma unroll
          for (int mu = 0; mu < 4; ++mu) {
            if (M[mu]) {
              if (pending + __popcll(M[mu]) > QCAP) {  // more than QCAP in one quad
                rescore_batch<SQB>(P, W, a, u, pending);
                pending = 0;
                oldest = sqi;
              }
              if (fl[mu]) {
                const int pos = pending + __popcll(M[mu] & lanemask_lt(lane));
                v4i* qdst = reinterpret_cast<v4i*>(&W.qd[pos * stride]);
#pragma unroll
                for (int sl = 0; sl < NSLM; ++sl)
                  if (sl < nsl) qdst[sl] = dig[mu][sl];
                const uint32_t hm = (uint32_t)(acc[mu][0] >= 0) | (uint32_t)(acc[mu][1] >= 0) << 1 |
                                    (uint32_t)(acc[mu][2] >= 0) << 2 | (uint32_t)(acc[mu][3] >= 0) << 3;
                W.qi[pos] = (uint32_t)(kbase + mu);
                W.qf[pos] = (uint32_t)mu | hm << 2 | meta;
              }
              pending += __popcll(M[mu]);
            }
          }
        }
      }
    }
  }
  if (pending > 0) rescore_batch<SQB>(P, W, a, u, pending);
}

// ---------------------------------------------------------------- unit state
// The full-pass class of a unit with sc[v] active channels of depth v
// (v = 1..kPlanes): 0 = no filter (its rows are computed exactly), 1 = the
// cell filter (filter.hip), else the wide pass's slice count (> kNarrow).
__device__ __forceinline__ uint32_t unit_class(const FusedArgs& a, const int (&sc)[kPlanes + 1], int64_t lo,
                                               int64_t hi) {
  const int A = sc[1] + sc[2] + sc[3] + sc[4];
  if (!(a.G <= 4 && A > 0 && hi - lo > a.ws.cap)) return 0u;
  // the launched cell filter takes at most kCA channels and a.ccap cells (one
  // per active channel and plane)
  const int cells = sc[1] + 2 * sc[2] + 3 * sc[3] + 4 * sc[4];
  if (A <= kCA && cells <= a.ccap && a.nb_cap < kOneNbMax) return 1u;
  const uint32_t cls = (uint32_t)((A + 15) >> 4);
  return cls <= (uint32_t)kNarrow ? (uint32_t)(kNarrow + 1) : cls;
}

// The per-call state of unit u's rows, set by the sample pass's workgroup 0
// of the unit (every thread; thread j < 128 holds channel j's depth t): the
// survivor counts and the exact pass's control words cleared, tau = -inf
// until the full pass sets it, and the unit's class.  The tau pass sets the
// same state when it runs.
__device__ __forceinline__ void unit_reset(const FusedArgs& a, int u, int t, int64_t lo, int64_t hi) {
  __shared__ int sc2[2][kPlanes + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, G = a.G;
  if (t > kPlanes) t = kPlanes;
  uint64_t bal[kPlanes + 1];
#pragma unroll
  for (int v = 1; v <= kPlanes; ++v) bal[v] = __ballot(tid < kD && t == v);
  if (tid < kD && lane == 0) {
#pragma unroll
    for (int v = 1; v <= kPlanes; ++v) sc2[wave][v] = __popcll(bal[v]);
  }
  if (tid < G) {
    const int r = u * G + tid;
    gstore(a.ws.cnt + r * kCntStride, 0u);
    gstore(a.ws.xctl + 1 + r, 0u);
    gstore(a.ws.tau + r, kNegInf);
  }
  if (tid < kPools) gstore(a.ws.pool + (u * kPools + tid) * kPoolStride, 0u);
  __syncthreads();
  if (tid == 0) {
    int sc[kPlanes + 1];
    sc[0] = 0;
#pragma unroll
    for (int v = 1; v <= kPlanes; ++v) sc[v] = sc2[0][v] + sc2[1][v];
    gstore(a.ws.uovf + u, unit_class(a, sc, lo, hi) << 1);
  }
}

// ---------------------------------------------------------------- pass 1
// Samples for tau: workgroup x of unit u takes sampled quad x (blocks
// 4 x s_stride .. + 3, one block per wave) and computes the documented exact
// scores of its keys (Sec. 3.2-3.3: prefix dequantisation, fma over the
// active channels ascending from +0, as the re-scoring of the full pass);
// per head, the two largest scores of each block are its samples (-inf where
// the block has fewer eligible keys).  The thread of each active channel
// loads its plane words and scales for the workgroup's 4 blocks as soon as
// it knows its depth and stores them in LDS by the channel's ascending
// position; every lane then reads its block's words back as broadcasts and
// takes its own key's bit.  Workgroup 0 of each unit also sets the rows'
// call state (unit_reset) and builds the unit's cell plan for the filter in
// the workspace while its plane words load.
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
struct alignas(16) SampleLds {
  uint32_t act[kD];                  // ascending position -> channel | depth << 8 (0 on padding)
  float q[kD][4];                    // q by ascending position and head (0 past G and on padding)
  float zo[kD];                      // -(1 - 2^-t): khat = (u / 8 + zo) a16, exact (0 on padding)
  uint32_t w[kFW][2][kD * kPlanes];  // block b's plane words, dword half h of cell 4 y + p
  uint16_t sc[kFW][kD];              // block b's scales by ascending position (0 on padding)
  int cnt[2];                        // active channels of channels 0..63, 64..127
};

__global__ __launch_bounds__(kFT) void fused_sample_kernel(FusedArgs a) {
  __shared__ SampleLds S;
  const int u = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6), G = a.G;
  int t = 0;
  float qv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (tid < kD) {
    t = gload(a.depths + (int64_t)u * kD + tid);
    if (t > kPlanes) t = kPlanes;
#pragma unroll
    for (int h = 0; h < 4; ++h)
      if (h < G) qv[h] = load_q(a.q, a.qdt, ((int64_t)u * G + h) * kD + tid);
  }
  // this channel's words and scales for the workgroup's blocks (0 past the store)
  const int64_t blk0 = (int64_t)blockIdx.x * a.ws.s_stride * kQB;
  uint64_t wd[kQB][kPlanes];
  uint16_t scv[kQB];
#pragma unroll
  for (int b = 0; b < kQB; ++b) {
    const bool inb = tid < kD && t > 0 && blk0 + b < a.nb_cap;
    scv[b] = inb ? gload(a.scales + ((int64_t)u * kD + tid) * a.nb_cap + blk0 + b) : (uint16_t)0;
#pragma unroll
    for (int p = 0; p < kPlanes; ++p)
      wd[b][p] = inb && p < t ? gload(a.planes + (((int64_t)u * kD + tid) * kPlanes + p) * a.nb_cap + blk0 + b) : 0ull;
  }
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  if (blockIdx.x == 0) {  // the unit's call state and its cell plan for the filter, while the words load
    unit_reset(a, u, t, lo, hi);
    __shared__ CellPlan P;
    CellPre pre;
    pre.t = t;
#pragma unroll
    for (int h = 0; h < 4; ++h) pre.q[h] = qv[h];
    cell_plan(P, a, pre);
#pragma unroll
    for (int i = 0; i < kPlanSteps; ++i) {
      const int w = tid + kFT * i;
      if (w < kPlanWords)
        gstore(reinterpret_cast<PlanWord*>(a.ws.plan + (size_t)u * kPlanBytes) + w, reinterpret_cast<const PlanWord*>(&P)[w]);
    }
  }
  if (hi - lo <= a.ws.cap) return;  // computed directly by the exact pass
  // the active channels in ascending order
  const uint64_t on = __ballot(tid < kD && t > 0);
  if (tid < kD && lane == 0) S.cnt[wave] = __popcll(on);
  __syncthreads();
  const int A = S.cnt[0] + S.cnt[1];
  if (tid < kD && t > 0) {
    const int y = __popcll(on & lanemask_lt(lane)) + (wave == 1 ? S.cnt[0] : 0);
    S.act[y] = (uint32_t)tid | (uint32_t)t << 8;
#pragma unroll
    for (int h = 0; h < 4; ++h) S.q[y][h] = qv[h];
    S.zo[y] = -(1.0f - ldexpf(1.0f, -t));
#pragma unroll
    for (int b = 0; b < kQB; ++b) {
      S.sc[b][y] = scv[b];
#pragma unroll
      for (int p = 0; p < kPlanes; ++p) {
        S.w[b][0][4 * y + p] = (uint32_t)wd[b][p];
        S.w[b][1][4 * y + p] = (uint32_t)(wd[b][p] >> 32);
      }
    }
  }
  const int A4 = (A + 3) & ~3;  // the chain in steps of 4 channels; padding adds +0 to every score
  if (tid >= A && tid < A4) {
    S.act[tid] = 0u;
#pragma unroll
    for (int h = 0; h < 4; ++h) S.q[tid][h] = 0.0f;
    S.zo[tid] = 0.0f;
#pragma unroll
    for (int b = 0; b < kQB; ++b) S.sc[b][tid] = 0;
  }
  __syncthreads();
  if (A == 0) return;  // no filter for the unit
  const int64_t nbu = (nu + kBlockTokens - 1) / kBlockTokens;
  const int64_t blk = blk0 + wave;
  const int64_t key = blk * kBlockTokens + lane;
  const bool el = blk < nbu && key >= lo && key < hi;
  float* dst = a.ws.samp + (int64_t)u * G * kSmpRow + (int64_t)blockIdx.x * kSmpW + 2 * wave;
  if (__ballot(el) == 0ull) {  // no eligible key in the block
    if (lane < 2 * G) gstore(dst + (int64_t)(lane >> 1) * kSmpRow + (lane & 1), kNegInf);
    return;
  }
  // this lane's key: the documented chain, 4 channels a step (every read of a
  // step first); a channel's four plane words (of this lane's half) are one
  // 16-byte read, the planes past its depth masked off its digit
  const int half = lane >> 5, bit = lane & 31;
  const uint32_t* wl = &S.w[wave][half][0];
  float sh[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int y0 = 0; y0 < A4; y0 += 4) {
    const v4u ev = *reinterpret_cast<const v4u*>(&S.act[y0]);
    const float4 zv = *reinterpret_cast<const float4*>(&S.zo[y0]);
    const uint2 sv = *reinterpret_cast<const uint2*>(&S.sc[wave][y0]);
    v4u wv[4];
    float4 q4[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      wv[c] = *reinterpret_cast<const v4u*>(&wl[4 * (y0 + c)]);
      q4[c] = *reinterpret_cast<const float4*>(&S.q[y0 + c][0]);
    }
    const uint32_t es[4] = {ev.x, ev.y, ev.z, ev.w};
    const float zs[4] = {zv.x, zv.y, zv.z, zv.w};
    const uint32_t hs[4] = {sv.x & 0xFFFFu, sv.x >> 16, sv.y & 0xFFFFu, sv.y >> 16};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t d = ((wv[c].x >> bit) & 1u) << 3 | ((wv[c].y >> bit) & 1u) << 2 | ((wv[c].z >> bit) & 1u) << 1 |
                         ((wv[c].w >> bit) & 1u);
      const uint32_t dg = d & ((0xF0u >> (es[c] >> 8)) & 0xFu);  // planes p < t
      const float x8 = __fmaf_rn((float)dg, 0.125f, zs[c]);
      const float khat = __fmaf_rn(x8, half_bits_to_float((uint16_t)hs[c]), 0.0f);
      sh[0] = __fmaf_rn(q4[c].x, khat, sh[0]);
      sh[1] = __fmaf_rn(q4[c].y, khat, sh[1]);
      sh[2] = __fmaf_rn(q4[c].z, khat, sh[2]);
      sh[3] = __fmaf_rn(q4[c].w, khat, sh[3]);
    }
  }
  // per head the two largest order-preserving keys (0: none)
  uint32_t k1[4], k2[4];
#pragma unroll
  for (int h = 0; h < 4; ++h) k1[h] = el ? score_key(sh[h]) : 0u;
  uint32_t m1[4] = {k1[0], k1[1], k1[2], k1[3]};
  wave_max4_u(m1);
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const uint64_t at = __ballot(k1[h] == m1[h]);
    k2[h] = lane == (int)__builtin_ctzll(at) ? 0u : k1[h];  // the first lane holding the largest drops out
  }
  wave_max4_u(k2);
  if (lane < 2 * G) {
    const int h = lane >> 1;
    const uint32_t k = (lane & 1) ? (h == 0 ? k2[0] : h == 1 ? k2[1] : h == 2 ? k2[2] : k2[3])
                                  : (h == 0 ? m1[0] : h == 1 ? m1[1] : h == 2 ? m1[2] : m1[3]);
    const float v = k == 0u ? kNegInf : __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
    gstore(dst + (int64_t)h * kSmpRow + (lane & 1), v);
  }
}

// ---------------------------------------------------------------- pass 2
// One workgroup of two waves per row (one thread per channel for the depth
// count), launched for the wide full pass or G > 4 (the cell filter finds tau
// itself).  Sets the row's call state as unit_reset does; tau = the m-th
// largest sample, found by wave 0 with a bitwise search over order-preserving
// keys and ballot counts.  Leaves the unit's class in uovf[u] for pass 3.
constexpr int kTauThreads = kD;
constexpr int kTauPer = kSmpRow / kWave;  // sampled values per lane of wave 0
__global__ __launch_bounds__(kTauThreads) void fused_tau_kernel(FusedArgs a) {
  __shared__ int sc[kPlanes + 1];  // active channels by depth
  const int r = blockIdx.x, G = a.G, u = r / G, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // every load first: the samples (wave 0 keeps the row's 512), the depths, n
  const int ns = wave == 0 ? a.ws.s_quads * kSmpW : 0;
  float sv[kTauPer];
#pragma unroll
  for (int x = 0; x < kTauPer; ++x) {
    const int i = lane + kWave * x;
    sv[x] = i < ns ? gload(a.ws.samp + (int64_t)r * kSmpRow + i) : kNegInf;
  }
  const int t = gload(a.depths + (int64_t)u * kD + tid);
  if (tid == 0) {
    a.ws.cnt[r * kCntStride] = 0u;
    a.ws.xctl[1 + r] = 0u;
  }
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, false);
  if (tid <= kPlanes) sc[tid] = 0;
  __syncthreads();
  if (t > 0) atomicAdd(&sc[t > kPlanes ? kPlanes : t], 1);
  __syncthreads();
  const int A = sc[1] + sc[2] + sc[3] + sc[4];
  const bool ok = G <= 4 && A > 0 && hi - lo > a.ws.cap;
  if (tid == 0 && r % G == 0) {
    const int scv[kPlanes + 1] = {0, sc[1], sc[2], sc[3], sc[4]};
    a.ws.uovf[u] = unit_class(a, scv, lo, hi) << 1;
  }
  if (!ok) {
    if (tid == 0) a.ws.tau[r] = kNegInf;
    return;
  }
  if (wave != 0) return;
  // the row's samples as keys (0 = no sample) and m
  uint32_t key[kTauPer];
  int nv = 0;
#pragma unroll
  for (int x = 0; x < kTauPer; ++x) {
    key[x] = sv[x] > kNegInf ? score_key(sv[x]) | 1u : 0u;  // samples are never NaN; keep 0 free
    nv += __popcll(__ballot(key[x] != 0u));
  }
  int64_t m_s = 0;  // eligible keys in the sampled quads
  for (int x = lane; x < a.ws.s_quads; x += kWave) {
    const int64_t k0 = x * a.ws.s_stride * kQB * kBlockTokens, k1 = k0 + kQB * kBlockTokens;
    const int64_t x0 = k0 > lo ? k0 : lo, x1 = k1 < hi ? k1 : hi;
    m_s += x1 > x0 ? x1 - x0 : 0;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m_s += __shfl_xor(m_s, o, kWave);
  const int64_t m_e = hi - lo;
  int64_t m = m_s > 0 ? (5 * (int64_t)a.k * m_s + 4 * m_e - 1) / (4 * m_e) + 16 : 0;
  if (m > nv) {
    // the samples cannot reach rank m: the smallest sample is used only when
    // the keys expected above it (nv m_e / m_s) are at least 1.1 k, else the
    // row is left unfiltered (exact path) instead of filtered in vain
    m = 10 * (int64_t)nv * m_e >= 11 * (int64_t)a.k * m_s ? nv : 0;
  }
  if (m == 0) {
    if (tid == 0) a.ws.tau[r] = kNegInf;
    return;
  }
  uint32_t prefix = 0u;  // the largest key with at least m samples at or above it
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    int c = 0;
#pragma unroll
    for (int x = 0; x < kTauPer; ++x) c += __popcll(__ballot(key[x] >= cand));
    if (c >= m) prefix = cand;
  }
  const uint32_t k0 = prefix & ~1u;  // the forced low bit rounded down
  if (lane == 0) a.ws.tau[r] = __uint_as_float((k0 & 0x80000000u) ? (k0 & 0x7FFFFFFFu) : ~k0);
}

// ---------------------------------------------------------------- pass 3
// NSLM: the slices this instantiation keeps in registers; a unit is run by
// the narrow (kNarrow) or the wide (8) instantiation according to its slice
// count, which pass 2 leaves in uovf[u] (0: no filter for the unit).
template <bool QF16, int SQB>
__global__ __launch_bounds__(kFT) void fused_main_kernel(FusedArgs a) {
  constexpr int NSLM = kMaxSl;
  __shared__ Plan P;
  __shared__ WaveLdsT<NSLM, SQB, kRing, kQCap> WL[kFW];
  const int u = blockIdx.y, tid = threadIdx.x, wave = uni(tid >> 6);
  // every global read of the preamble first: unit class, n, tau, depths and
  // q (the plan's barriers order the LDS writes)
  const uint32_t uo = gload(a.ws.uovf + u);
  if (tid < 4) P.tau[tid] = tid < a.G ? gload(a.ws.tau + u * a.G + tid) : kNegInf;
  const PlanPre pre = plan_load<QF16>(a, u);
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, blockIdx.x == 0 && tid == 0);
  const int ucls = (int)(uo >> 1);  // slices, or 0
  if (ucls <= kNarrow || ucls > NSLM) return;  // no filter, or the cell filter's
  if (hi - lo <= a.ws.cap) return;
  const int64_t nbu = (nu + kBlockTokens - 1) / kBlockTokens;
  const int64_t gw = (int64_t)blockIdx.x * kFW;       // first wave of this workgroup
  const int64_t qlo = lo / (kQB * kBlockTokens);       // first quad with eligible keys
  const int64_t qhi = (hi + kQB * kBlockTokens - 1) / (kQB * kBlockTokens);
  if (gw * a.ws.qpw >= qhi || (gw + kFW) * a.ws.qpw <= qlo) return;
  plan_setup(P, a, u, pre);
  if (!P.ok || P.A == 0 || P.nsl > NSLM) return;
  bool any = false;
  for (int h = 0; h < a.G; ++h) any |= P.tau[h] != kNegInf;
  if (!any) return;
  int64_t q0 = (gw + wave) * a.ws.qpw, q1 = q0 + a.ws.qpw;
  if (q0 < qlo) q0 = qlo;
  if (q1 > qhi) q1 = qhi;
  if (q0 >= q1) return;
  wave_run<QF16, NSLM, SQB, kRing, kQCap>(P, WL[wave], a, u, q0 * kQB, q1 * kQB < nbu ? q1 * kQB : nbu, nbu, lo,
                                           hi);
}

// ---------------------------------------------------------------- select: ranks
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

// Ranks of filtered rows.  The row's survivor list holds its top k exactly
// when at least k keys survived, the list kept them all (the count goes on
// past the capacity) and the filter ran for the row.  Its top K = min(c, k)
// output positions are shared by kRankParts workgroups: each reads the c
// survivors and builds the same histogram over ns sub-buckets of the score key
// (interpolated between the row's smallest and largest survivor key, not
// decreasing as the key falls), so a survivor's output position is (survivors
// of the sub-buckets before its own) + (survivors of its own sub-bucket with a
// larger composite).  Part z takes the sub-buckets whose first position lies
// in [z K / parts, (z + 1) K / parts) and orders their survivors in LDS; only
// survivors sharing a sub-bucket are compared.  Composites are distinct (they
// carry the index), so the positions are a permutation.  A row whose share
// for some part exceeds kRankCap (many equal scores) is computed exactly by
// its own parts instead; every part reaches the same decision from the same
// histogram.  The parts of a row run on one XCD (workgroups are dealt to the
// 8 XCDs in turn), so the list is read once into that XCD's L2.
constexpr int kRankParts = 8;
constexpr int kRankThreads = 512;   // the rank pass's workgroup (the select pass's is kXThreads)
constexpr int kRankPer = 8;      // survivors per thread read with the count (the rest re-read)
constexpr int kRankCap = 4096;   // survivors one part orders at most
constexpr int kRankSub = 4096;   // sub-buckets at most
constexpr int kRankXcd = 8;
template <int T>
struct RankShared {
  uint32_t s_red[2][T / kWave], s_part[T / kWave];
  uint32_t s_first[kRankParts + 1];  // part z: sub-buckets [s_first[z], s_first[z + 1])
  uint32_t s_c, s_ovf;
  float s_tau;
  int64_t s_n;
};
// Part z of row r (every thread of the workgroup calls it, for a row whose
// list holds its top k); grp and hist are LDS areas of kRankCap composites
// and kRankSub + 1 counts, 16-byte aligned.  Returns true when a part's share
// exceeds kRankCap after all (many equal scores): the row is then computed
// exactly.
template <int T>
__device__ bool rank_part(const FusedArgs& a, int r, int z, int32_t* __restrict__ idx, float* __restrict__ val,
                          uint64_t* grp, uint32_t* hist, RankShared<T>& RS) {
  constexpr int kRankThreads = T;  // threads of the calling workgroup
  auto& s_red = RS.s_red;
  auto& s_part = RS.s_part;
  auto& s_first = RS.s_first;
  auto& s_c = RS.s_c;
  auto& s_ovf = RS.s_ovf;
  auto& s_tau = RS.s_tau;
  auto& s_n = RS.s_n;
  const int G = a.G;
  const int u = r / G, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lcap = a.ws.lcap;
  const uint64_t* src = a.ws.cand + (int64_t)r * lcap;
  uint64_t pv[kRankPer];
#pragma unroll
  for (int x = 0; x < kRankPer; ++x) {  // slots past the count are read but not used
    const int e = tid + kRankThreads * x;
    pv[x] = e < lcap ? gload(src + e) : 0ull;
  }
  if (tid == 0) s_c = gload(a.ws.cnt + r * kCntStride);
  else if (tid == 1) s_tau = gload(a.ws.tau + r);
  else if (tid == 2) s_ovf = gload(a.ws.uovf + u);
  else if (tid == 3) s_n = gload(a.n + u);
  __syncthreads();
  int64_t nu = s_n;
  if (nu < 0 || nu > a.nb_cap * kBlockTokens) nu = 0;
  int64_t lo = a.lo, hi = nu - a.tail;
  if (hi < lo) hi = lo;
  const uint32_t c = s_c, k = (uint32_t)a.k;
  const bool direct = hi - lo <= a.ws.cap;
  const bool complete = c >= k && c <= (uint32_t)lcap && (s_ovf & 1u) == 0u && s_tau != kNegInf;
  if (direct || !complete) return false;  // the caller's row test rules this out
  // visits every survivor: the first kRankPer per thread from registers
  auto each = [&](auto fn) {
#pragma unroll
    for (int x = 0; x < kRankPer; ++x)
      if (tid + kRankThreads * x < (int)c) fn(pv[x]);
    for (uint32_t e = tid + kRankThreads * kRankPer; e < c; e += kRankThreads) fn(gload(src + e));
  };
  int ns = 64;  // sub-buckets: a power of two, at least the survivors
  while (ns < (int)c && ns < kRankSub) ns <<= 1;
  for (int x = tid; x < ns; x += kRankThreads) hist[x] = 0u;
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  each([&](uint64_t v) {
    const uint32_t key = (uint32_t)(v >> 32);
    kmin = key < kmin ? key : kmin;
    kmax = key > kmax ? key : kmax;
  });
  {
    uint32_t mm[4] = {kmax, ~kmin, 0u, 0u};  // the smallest key as the largest complement
    wave_max4_u(mm);
    kmax = mm[0];
    kmin = ~mm[1];
  }
  if (lane == 0) {
    s_red[0][wave] = kmin;
    s_red[1][wave] = kmax;
  }
  __syncthreads();
  kmin = s_red[0][0];
  kmax = s_red[1][0];
#pragma unroll
  for (int x = 1; x < kRankThreads / kWave; ++x) {
    kmin = s_red[0][x] < kmin ? s_red[0][x] : kmin;
    kmax = s_red[1][x] > kmax ? s_red[1][x] : kmax;
  }
  // sub-bucket: floor((kmax - key) * scale), not decreasing as the key falls
  const float scale = kmax > kmin ? (float)(ns - 1) / (float)(kmax - kmin) : 0.0f;
  auto sub_of = [&](uint64_t v) {
    const int sb = (int)__fmul_rn((float)(kmax - (uint32_t)(v >> 32)), scale);
    return sb < ns - 1 ? sb : ns - 1;
  };
  each([&](uint64_t v) { atomicAdd(&hist[sub_of(v)], 1u); });
  __syncthreads();
  // exclusive prefix over the sub-buckets, in place (thread t owns a run of
  // ns / kRankThreads, or one); hist[ns] = c.  Part z's first sub-bucket is
  // the first s with hist[s] >= b_z = z K / parts: for b_z > 0 the one after
  // the sub-bucket whose positions cross b_z.
  const uint32_t K = c < k ? c : k;
  {
    constexpr int kPerMax = kRankSub / kRankThreads;
    static_assert(kPerMax % 4 == 0, "16-byte runs per thread");
    const int per = ns / kRankThreads > 0 ? ns / kRankThreads : 1;
    const int x0 = tid * per;
    uint32_t hv[kPerMax];  // this thread's run of sub-buckets (0 past it)
    if (per == kPerMax) {
#pragma unroll
      for (int v = 0; v < kPerMax / 4; ++v) {
        const uint4 h = *reinterpret_cast<const uint4*>(&hist[x0 + 4 * v]);
        hv[4 * v] = h.x; hv[4 * v + 1] = h.y; hv[4 * v + 2] = h.z; hv[4 * v + 3] = h.w;
      }
    } else {
#pragma unroll
      for (int x = 0; x < kPerMax; ++x) hv[x] = x < per && x0 + x < ns ? hist[x0 + x] : 0u;
    }
    uint32_t run = 0;
#pragma unroll
    for (int x = 0; x < kPerMax; ++x) run += hv[x];
    const uint32_t inc = wave_incl_scan_u(run);
    if (lane == kWave - 1) s_part[wave] = inc;
    __syncthreads();
    uint32_t acc = inc - run;
    for (int x = 0; x < wave; ++x) acc += s_part[x];
    const uint32_t a0 = acc;
    uint32_t ov[kPerMax];  // exclusive prefix of each sub-bucket
#pragma unroll
    for (int x = 0; x < kPerMax; ++x) {
      ov[x] = acc;
      acc += hv[x];
    }
    if (per == kPerMax) {
#pragma unroll
      for (int v = 0; v < kPerMax / 4; ++v)
        *reinterpret_cast<uint4*>(&hist[x0 + 4 * v]) = make_uint4(ov[4 * v], ov[4 * v + 1], ov[4 * v + 2], ov[4 * v + 3]);
    } else {
#pragma unroll
      for (int x = 0; x < kPerMax; ++x)
        if (x < per && x0 + x < ns) hist[x0 + x] = ov[x];
    }
    // part bounds b = zz K / parts inside this thread's positions [a0, acc]
#pragma unroll
    for (int zz = 1; zz <= kRankParts; ++zz) {
      const uint32_t b = (uint32_t)(((uint64_t)zz * K) / kRankParts);
      if (a0 < b && acc >= b) {
#pragma unroll
        for (int x = 0; x < kPerMax; ++x)
          if (ov[x] < b && ov[x] + hv[x] >= b) s_first[zz] = (uint32_t)(x0 + x + 1);
      }
    }
    if (tid == 0) {
      hist[ns] = c;
#pragma unroll
      for (int zz = 0; zz <= kRankParts; ++zz)
        if (((uint64_t)zz * K) / kRankParts == 0) s_first[zz] = 0u;
    }
  }
  __syncthreads();
  bool over = false;
#pragma unroll
  for (int x = 0; x < kRankParts; ++x) over |= hist[s_first[x + 1]] - hist[s_first[x]] > (uint32_t)kRankCap;
  if (over) return true;
  const int s0 = (int)s_first[z], s1 = (int)s_first[z + 1];
  if (s0 == s1) return false;
  const uint32_t start = hist[s0], share = hist[s1] - start;
  __syncthreads();  // every part bound read before hist[s0 .. s1) serve as cursors
  each([&](uint64_t v) {  // group by sub-bucket; hist[s] ends at the group's end
    const int sb = sub_of(v);
    if (sb >= s0 && sb < s1) grp[atomicAdd(&hist[sb], 1u) - start] = v;
  });
  __syncthreads();
  for (uint32_t e = tid; e < share; e += kRankThreads) {
    const uint64_t v = grp[e];
    const int sb = sub_of(v);
    const uint32_t g0 = sb > s0 ? hist[sb - 1] : start, g1 = hist[sb];
    uint32_t rank = g0;
    for (uint32_t x = g0; x < g1; ++x) rank += grp[x - start] > v;
    if (rank < k) {
      idx[(int64_t)r * k + rank] = (int32_t)(~(uint32_t)(v & 0xFFFFFFFFull));
      if (val) val[(int64_t)r * k + rank] = key_to_score((uint32_t)(v >> 32));
    }
  }
  return false;
}

// ---------------------------------------------------------------- exact rows
// Rows whose survivor lists do not determine the top k (direct rows too) are
// computed from exact documented scores, chunk by chunk (the select pass
// below hands out the chunks): the
// exact scores of the chunk's keys go to LDS (kXKeys at a time), and the
// chunk's top min(k, keys) composites (score key << 32 | ~index) to its
// partial list; the workgroup that completes a row's last chunk selects the
// row's top k from its partial lists, orders them and writes the row.  Every
// selection is exact (a radix select on the composites, which are distinct),
// so the result is the documented top k whatever the chunking.
constexpr int kXThreads = 1024;
constexpr int kXWaves = kXThreads / kWave;  // blocks scored per stage, one per wave
constexpr int kXSlots = 4;                  // exact rows in flight (workgroups per chunk index)
constexpr int kXMaxCells = kD * kPlanes;    // (channel, plane) cells of a unit at most
constexpr int kXPre = kXMaxCells * kXWaves / kXThreads;  // plane words staged per thread at most
constexpr int kXPreS = kD * kXWaves / kXThreads;         // scales staged per thread at most
static_assert(kXPre == 8 && kXPreS == 2, "staging registers");
constexpr size_t kXLdsKeys = (size_t)kXKeys * 4;
constexpr size_t kXLdsStw = (size_t)kXMaxCells * kXWaves * 8;  // [block][half][4 slots per channel] u32
constexpr size_t kXLdsSts = (size_t)kD * kXWaves * 8;
constexpr size_t kXLdsTab = (size_t)kD * 4 * 2 + (size_t)kXMaxCells * 4;
constexpr size_t kXLdsHist = 2048 * 4;  // radix histogram; the merge's crossing digit
constexpr size_t kXLdsBytes = kXLdsKeys + kXLdsStw + kXLdsSts + kXLdsTab + kXLdsHist;
static_assert(kXLdsKeys + kXLdsStw >= (size_t)2 * FATHOM_MAX_K * 8, "merge buffer: candidates, then the top k");
static_assert(kXLdsBytes <= 156 * 1024, "exact pass LDS (plus its static part) within one CU's 160 KB");

struct XShared {
  uint32_t part[kXWaves];
  int digit;
  uint32_t above;
  uint32_t cnt;
  uint32_t last;
  uint64_t lb;
  int A, cells;
  int wc[2], wt[2];
  uint32_t pc[kXChunks];
  uint64_t ps[kXChunks];
};

// The largest composite T with #{v >= T} >= need over the elements `each`
// visits (every thread visits its share; need <= their number): an MSB-first
// radix select, 11/11/10 bits per word, that stops once every element with
// the fixed prefix is needed.  Then #{v >= T} == need exactly (composites
// are distinct).  hist holds 2048 words.
template <class Each>
__device__ uint64_t select_threshold(Each each, uint32_t need, uint32_t* hist, XShared& S) {
  uint64_t prefix = 0ull, mask = 0ull;
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int pass = 0; pass < 6; ++pass) {
    const int bits = (pass % 3 == 2) ? 10 : 11;
    const int sh = (pass < 3 ? 32 : 0) + (pass % 3 == 0 ? 21 : pass % 3 == 1 ? 10 : 0);
    const int nb = 1 << bits;
    const uint64_t dm = (uint64_t)(nb - 1);
    for (int x = tid; x < nb; x += nt) hist[x] = 0u;
    __syncthreads();
    each([&](uint64_t v) {
      if ((v & mask) == prefix) atomicAdd(&hist[(v >> sh) & dm], 1u);
    });
    __syncthreads();
    find_crossing(hist, nb, need, S.part, &S.digit, &S.above);
    const int d = S.digit;
    const uint32_t above = S.above, at = hist[d];
    prefix |= (uint64_t)d << sh;
    mask |= dm << sh;
    need -= above;
    __syncthreads();  // hist and the crossing read by all before the next pass
    if (at == need) break;
  }
  return prefix;
}

__device__ __forceinline__ uint64_t key_composite(uint32_t key, int64_t i) {
  return ((uint64_t)key << 32) | (uint64_t)(~(uint32_t)i);
}

// Chunk z of row r computed exactly (every thread of the workgroup calls
// it): the chunk's top composites go to the row's partial list z, and the
// workgroup that completes the row's last chunk merges them and writes the
// row.  xl: the dynamic LDS (kXLdsBytes).
__device__ void exact_chunk(const FusedArgs& a, int r, int z, int32_t* __restrict__ idx, float* __restrict__ val,
                            unsigned char* xl, XShared& S) {
  uint32_t* keys = reinterpret_cast<uint32_t*>(xl);
  uint32_t* stw = reinterpret_cast<uint32_t*>(xl + kXLdsKeys);
  uint64_t* sel = reinterpret_cast<uint64_t*>(xl + kXLdsKeys);  // a pass's selection (stw is free then)
  float2* sts = reinterpret_cast<float2*>(xl + kXLdsKeys + kXLdsStw);  // [channel][block] (a16 / 8, z a16 / 8)
  int* act = reinterpret_cast<int*>(xl + kXLdsKeys + kXLdsStw + kXLdsSts);
  float* qa = reinterpret_cast<float*>(act + kD);
  uint32_t* crow = reinterpret_cast<uint32_t*>(qa + kD);  // cell c: plane row 4 j + p | slot 4 a + p << 9
  uint32_t* hist = reinterpret_cast<uint32_t*>(xl + kXLdsKeys + kXLdsStw + kXLdsSts + kXLdsTab);
  uint64_t* mbuf = reinterpret_cast<uint64_t*>(xl);  // merge: candidates [0, 2 FATHOM_MAX_K - k), then the top k
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = a.G, k = a.k, pk = a.ws.pk;
  {
    const int u = r / G, h = r % G;
    int64_t nu, lo, hi;
    row_window(a, u, &nu, &lo, &hi, false);
    const bool direct = hi - lo <= a.ws.cap;
    const int64_t bfirst = lo / kBlockTokens, bend = hi > lo ? (hi + kBlockTokens - 1) / kBlockTokens : bfirst;
    const int64_t rb = bend - bfirst;  // blocks holding eligible keys
    int nz = (int)((rb + kXBlocks - 1) / kXBlocks);
    if (nz > a.ws.xch) nz = a.ws.xch;
    if (nz < 1) nz = 1;
    if (z >= nz) return;
    const int64_t cbk = (rb + nz - 1) / nz;  // blocks per chunk
    const int64_t cb0 = bfirst + z * cbk, cb1 = cb0 + cbk < bend ? cb0 + cbk : bend;
    // ---- the row's active channels ascending, their q, and their cells: cell
    // (channel a, plane p) is staged in slot 4 a + p, so a channel's words are
    // one aligned 16-byte read
    {
      int t = 0;
      if (tid < kD) {
        t = gload(a.depths + (int64_t)u * kD + tid);
        t = t > kPlanes ? kPlanes : t;
      }
      const int on = tid < kD && t > 0, tc = tid < kD ? t : 0;
      int ion = on, itc = tc;  // inclusive scans within the wave
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int x0 = __shfl_up(ion, o, kWave), x1 = __shfl_up(itc, o, kWave);
        if (lane >= o) {
          ion += x0;
          itc += x1;
        }
      }
      if (wave < 2 && lane == kWave - 1) {
        S.wc[wave] = ion;
        S.wt[wave] = itc;
      }
      __syncthreads();
      if (tid < kD && on) {
        const int ai = ion - 1 + (wave == 1 ? S.wc[0] : 0);
        const int c0 = itc - t + (wave == 1 ? S.wt[0] : 0);
        act[ai] = tid | (t << 8);
        qa[ai] = load_q(a.q, a.qdt, ((int64_t)u * G + h) * kD + tid);
        for (int p = 0; p < t; ++p) crow[c0 + p] = (uint32_t)((kPlanes * tid + p) | ((kPlanes * ai + p) << 9));
      }
      if (tid == 0) {
        S.A = S.wc[0] + S.wc[1];
        S.cells = S.wt[0] + S.wt[1];
      }
      __syncthreads();
    }
    const int A = S.A, nc = S.cells, ns = kPlanes * A;  // slots per (block, half)
    const uint64_t* Pu = a.planes + (int64_t)u * kD * kPlanes * a.nb_cap;
    const uint16_t* Su = a.scales + (int64_t)u * kD * a.nb_cap;
    uint32_t lcnt = 0;      // composites in this chunk's partial list so far
    uint64_t lsplit = 0ull; // its top min(lcnt, xs) composites are those >= lsplit
    uint64_t* plist = a.ws.part + ((int64_t)r * a.ws.xch + z) * pk;
    for (int64_t pb0 = cb0; pb0 < cb1; pb0 += kXBlocks) {  // passes of at most kXKeys keys
      const int64_t pb1 = pb0 + kXBlocks < cb1 ? pb0 + kXBlocks : cb1;
      // ---- exact scores of blocks [pb0, pb1) into keys[]: 16 blocks per stage
      // (one per wave).  Plane words are staged as 32-bit halves, [block][half]
      // [slot]; scales as fp32 times 2^(1-t), [channel][block].  The next
      // stage's words are loaded while this one is scored.
      uint64_t pw[kXPre];
      float2 ps[kXPreS];
      auto issue = [&](int64_t s0) {
#pragma unroll
        for (int i = 0; i < kXPre; ++i) {
          const int x = tid + i * kXThreads;
          pw[i] = 0ull;
          const int64_t b = s0 + (x & (kXWaves - 1));
          if (x < nc * kXWaves && b < pb1)
            pw[i] = gload(Pu + (int64_t)(crow[x / kXWaves] & 0x1FF) * a.nb_cap + b);
        }
#pragma unroll
        for (int i = 0; i < kXPreS; ++i) {
          const int x = tid + i * kXThreads;
          ps[i] = make_float2(0.0f, 0.0f);
          const int64_t b = s0 + (x & (kXWaves - 1));
          if (x < A * kXWaves && b < pb1) {
            // khat = (c^(t) + 1/2 - 2^(t-1)) a16 2^(1-t) = (u + 2^(3-t) - 8) a16 / 8 with
            // u = c^(t) 2^(4-t) the prefix digit: both terms exact in fp32
            const int e = act[x / kXWaves], t = e >> 8;
            const float s8 = __fmul_rn(half_bits_to_float(gload(Su + (int64_t)(e & 0xFF) * a.nb_cap + b)), 0.125f);
            ps[i] = make_float2(s8, __fmul_rn(__fmul_rn((float)(16 >> t), 0.5f) - 8.0f, s8));
          }
        }
      };
      for (int x = tid; x < 2 * kXWaves * ns; x += kXThreads) stw[x] = 0u;  // planes p >= t read as 0
      __syncthreads();
      issue(pb0);
      for (int64_t s0 = pb0; s0 < pb1; s0 += kXWaves) {
#pragma unroll
        for (int i = 0; i < kXPre; ++i) {
          const int x = tid + i * kXThreads;
          if (x < nc * kXWaves) {
            const int bb = x & (kXWaves - 1), slot = crow[x / kXWaves] >> 9;
            stw[(2 * bb) * ns + slot] = (uint32_t)pw[i];
            stw[(2 * bb + 1) * ns + slot] = (uint32_t)(pw[i] >> 32);
          }
        }
#pragma unroll
        for (int i = 0; i < kXPreS; ++i) {
          const int x = tid + i * kXThreads;
          if (x < A * kXWaves) sts[x] = ps[i];
        }
        __syncthreads();
        if (s0 + kXWaves < pb1) issue(s0 + kXWaves);
        const int64_t b = s0 + wave;
        if (b < pb1) {
          // lane's half of every staged word: one aligned 16-byte read per channel
          const uint4* wrow = reinterpret_cast<const uint4*>(stw) + (2 * wave + (lane >> 5)) * A;
          const float2* srow = sts + wave;
          const uint32_t bit = (uint32_t)(lane & 31);
          float acc = 0.0f;
#pragma unroll 4
          for (int ai = 0; ai < A; ++ai) {
            const uint4 w4 = wrow[ai];
            const float2 sb = srow[ai * kXWaves];
            const uint32_t ud = (__builtin_amdgcn_ubfe(w4.x, bit, 1) << 3) | (__builtin_amdgcn_ubfe(w4.y, bit, 1) << 2) |
                                (__builtin_amdgcn_ubfe(w4.z, bit, 1) << 1) | __builtin_amdgcn_ubfe(w4.w, bit, 1);
            acc = __fmaf_rn(qa[ai], __fmaf_rn((float)ud, sb.x, sb.y), acc);
          }
          keys[(b - pb0) * kBlockTokens + lane] = score_key(acc);
        }
        __syncthreads();
      }
      // ---- eligible positions of this pass; the chunk's running top pk
      const int64_t kb = pb0 * kBlockTokens;
      const int p_lo = (int)(lo > kb ? lo - kb : 0);
      const int64_t pe = hi - kb < (pb1 - pb0) * kBlockTokens ? hi - kb : (pb1 - pb0) * kBlockTokens;
      const int p_hi = (int)(pe > p_lo ? pe : p_lo);
      const uint32_t m = (uint32_t)(p_hi - p_lo) + lcnt;  // candidates: this pass and the list so far
      const uint32_t take = m < (uint32_t)pk ? m : (uint32_t)pk;
      auto each = [&](auto f) {
        for (int p = p_lo + tid; p < p_hi; p += kXThreads) f(key_composite(keys[p], kb + p));
        for (uint32_t e = tid; e < lcnt; e += kXThreads) f(plist[e]);
      };
      uint64_t T = 0ull;
      if (m > take) T = select_threshold(each, take, hist, S);
      if (tid == 0) S.cnt = 0u;
      __syncthreads();
      each([&](uint64_t v) {
        if (v >= T) {
          const uint32_t pos = atomicAdd(&S.cnt, 1u);
          if (pos < take) sel[pos] = v;
        }
      });
      __syncthreads();
      lcnt = take;
      if (pb0 + kXBlocks < cb1) {  // another pass follows: the list as it stands
        for (uint32_t e = tid; e < take; e += kXThreads) gstore(plist + e, sel[e]);
        __syncthreads();
        continue;
      }
      // the chunk's final list: its top xs composites (those >= lsplit) first,
      // then the rest (all below lsplit)
      const uint32_t xs = (uint32_t)exact_split(k, nz);
      lsplit = 0ull;
      if (take > xs) {
        auto es = [&](auto f) {
          for (uint32_t e = tid; e < take; e += kXThreads) f(sel[e]);
        };
        lsplit = select_threshold(es, xs, hist, S);
      }
      if (tid == 0) {
        S.cnt = 0u;
        S.above = 0u;
      }
      __syncthreads();
      for (uint32_t e = tid; e < take; e += kXThreads) {
        const uint64_t v = sel[e];
        if (v >= lsplit) gstore(plist + atomicAdd(&S.cnt, 1u), v);
        else gstore(plist + xs + atomicAdd(&S.above, 1u), v);
      }
      __syncthreads();
    }
    if (tid == 0) {
      gstore(a.ws.pcnt + (int64_t)r * a.ws.xch + z, lcnt);
      gstore(a.ws.pmin + (int64_t)r * a.ws.xch + z, lsplit);
    }
    // ---- arrive; the last chunk of the row merges
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      const uint32_t prev = __hip_atomic_fetch_add((__attribute__((address_space(1))) uint32_t*)(a.ws.xctl + 1 + r),
                                                   1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      S.last = prev == (uint32_t)(nz - 1) ? 1u : 0u;
    }
    __syncthreads();
    if (S.last) {
      __threadfence();
      if (tid < nz) {
        const int64_t o = (int64_t)r * a.ws.xch + tid;
        S.pc[tid] = __hip_atomic_load((__attribute__((address_space(1))) uint32_t*)(a.ws.pcnt + o), __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
        S.ps[tid] = __hip_atomic_load((__attribute__((address_space(1))) uint64_t*)(a.ws.pmin + o), __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
      }
      if (tid == 0) {
        S.cnt = 0u;
        S.above = 0u;
      }
      __syncthreads();
      const uint64_t* rl = a.ws.part + (int64_t)r * a.ws.xch * pk;
      const uint32_t xs = (uint32_t)exact_split(k, nz);
      const uint32_t capm = (uint32_t)(2 * FATHOM_MAX_K - exact_pow2(k));  // candidates in LDS at most
      uint64_t* top = mbuf + capm;                              // the row's top k, then ordered
      // (1) the heads (each list's top xs) into LDS
      for (int y = wave; y < nz; y += kXWaves) {
        const uint32_t hy = S.pc[y] < xs ? S.pc[y] : xs;
        uint32_t base = 0u;
        if (lane == 0) base = atomicAdd(&S.cnt, hy);
        base = __shfl(base, 0, kWave);
        for (uint32_t e = lane; e < hy; e += kWave) mbuf[base + e] = gload(rl + (int64_t)y * pk + e);
      }
      __syncthreads();
      const uint32_t H = S.cnt;
      // (2) L = the k-th composite of the heads: at most the row's k-th composite
      uint64_t L = 0ull;
      if (H > (uint32_t)k) {
        auto eh = [&](auto f) {
          for (uint32_t e = tid; e < H; e += kXThreads) f(mbuf[e]);
        };
        L = select_threshold(eh, (uint32_t)k, hist, S);
      }
      // (3) the rest of every list whose xs-th composite lies above L (its
      // other composites may reach L); composites below L are not needed
      if (tid == 0) S.cnt = H;
      __syncthreads();
      for (int y = wave; y < nz; y += kXWaves) {
        if (S.pc[y] <= xs || S.ps[y] <= L) continue;  // the rest is below the split, itself <= L
        const uint64_t* Ly = rl + (int64_t)y * pk;
        for (uint32_t e0 = xs; e0 < S.pc[y]; e0 += kWave) {
          const uint32_t e = e0 + lane;
          const uint64_t v = e < S.pc[y] ? gload(Ly + e) : 0ull;
          const bool keep = e < S.pc[y] && v >= L;
          const uint64_t bm = __ballot(keep);
          if (bm) {
            uint32_t base = 0u;
            if (lane == 0) base = atomicAdd(&S.cnt, (uint32_t)__popcll(bm));
            base = __shfl(base, 0, kWave);
            const uint32_t pos = base + (uint32_t)__popcll(bm & lanemask_lt(lane));
            if (keep && pos < capm) mbuf[pos] = v;
          }
        }
      }
      __syncthreads();
      const uint32_t M = S.cnt;  // heads and kept rests
      uint32_t Mall = 0;
      for (int y = 0; y < nz; ++y) Mall += S.pc[y];
      const uint32_t take = Mall < (uint32_t)k ? Mall : (uint32_t)k;
      uint64_t T = 0ull;
      if (M <= capm) {
        auto each = [&](auto f) {
          for (uint32_t e = tid; e < M; e += kXThreads) {
            const uint64_t v = mbuf[e];
            if (v >= L) f(v);
          }
        };
        if (Mall > take) T = select_threshold(each, take, hist, S);
        if (tid == 0) S.cnt = 0u;
        __syncthreads();
        each([&](uint64_t v) {
          if (v >= T) {
            const uint32_t pos = atomicAdd(&S.cnt, 1u);
            if (pos < take) top[pos] = v;
          }
        });
      } else {  // more candidates than LDS holds (heavy ties): select from the lists themselves
        auto each = [&](auto f) {
          for (int y = 0; y < nz; ++y)
            for (uint32_t e = tid; e < S.pc[y]; e += kXThreads) {
              const uint64_t v = rl[(int64_t)y * pk + e];
              if (v >= L) f(v);
            }
        };
        T = select_threshold(each, take, hist, S);
        if (tid == 0) S.cnt = 0u;
        __syncthreads();
        each([&](uint64_t v) {
          if (v >= T) {
            const uint32_t pos = atomicAdd(&S.cnt, 1u);
            if (pos < take) top[pos] = v;
          }
        });
      }
      __syncthreads();
      int P2 = 2;
      while (P2 < (int)take) P2 <<= 1;
      for (int x = (int)take + tid; x < P2; x += kXThreads) top[x] = 0ull;
      __syncthreads();
      bitonic_desc(top, P2);
      bool shortfall = false;
      for (int x = tid; x < k; x += kXThreads) {
        if (x < (int)take) {
          const uint64_t c = top[x];
          idx[(int64_t)r * k + x] = (int32_t)(~(uint32_t)(c & 0xFFFFFFFFull));
          if (val) val[(int64_t)r * k + x] = key_to_score((uint32_t)(c >> 32));
        } else {
          idx[(int64_t)r * k + x] = -1;
          if (val) val[(int64_t)r * k + x] = __uint_as_float(0x7FC00000u);
          shortfall = true;
        }
      }
      if (__syncthreads_or(shortfall) && tid == 0) set_status(a.st, FATHOM_DEV_TOPK_SHORT);
      if (tid == 0 && !direct) set_status(a.st, FATHOM_DEV_TOPK_FALLBACK);
    }
    __syncthreads();  // LDS reused by the caller's next chunk
  }
}

// Whether row r is computed exactly: a direct row (at most cap eligible keys),
// or a row whose survivor list does not hold its top k (fewer than k
// survivors, more than the list holds, the unit's overflow flag, no tau).
// The rank part decides the same from the same values.
__device__ __forceinline__ bool row_exact(const FusedArgs& a, int r) {
  const int u = r / a.G;
  int64_t nu = gload(a.n + u);
  if (nu < 0 || nu > a.nb_cap * kBlockTokens) nu = 0;
  int64_t lo = a.lo, hi = nu - a.tail;
  if (hi < lo) hi = lo;
  if (hi - lo <= a.ws.cap) return true;
  const uint32_t c = gload(a.ws.cnt + r * kCntStride), ovf = gload(a.ws.uovf + u);
  const float tau = gload(a.ws.tau + r);
  return !(c >= (uint32_t)a.k && c <= (uint32_t)a.ws.lcap && (ovf & 1u) == 0u && tau != kNegInf);
}

// The rank pass, when the rank parts do not fit one round in the select
// pass's workgroups (1024 threads, one a CU): part z of row r as above; a part
// whose share is too large marks the row for the exact rows of the select
// pass that follows (tau = -inf, which every part of the row writes alike,
// before any of them writes a position).
__global__ __launch_bounds__(kRankThreads) void fused_rank_kernel(FusedArgs a, int R, int32_t* __restrict__ idx,
                                                                 float* __restrict__ val) {
  __shared__ uint64_t grp[kRankCap];
  __shared__ __align__(16) uint32_t hist[kRankSub + 4];
  __shared__ RankShared<kRankThreads> RS;
  __shared__ int s_ex;
  const int b = (int)blockIdx.x, j = b / kRankXcd, z = j % kRankParts, r = (j / kRankParts) * kRankXcd + b % kRankXcd;
  if (r >= R) return;
  if (threadIdx.x == 0) s_ex = row_exact(a, r) ? 1 : 0;
  __syncthreads();
  if (s_ex) return;
  if (rank_part<kRankThreads>(a, r, z, idx, val, grp, hist, RS) && threadIdx.x == 0) gstore(a.ws.tau + r, kNegInf);
}

// The select pass: ranks and exact rows in one launch when the rank parts fit
// one round of the chip (ranks set: rank_wg > 0), else the exact rows only
// after the rank pass below.  Workgroup b < rank_wg is part z of row r of the
// ranks above unless the row is computed exactly; a part that finds its
// share too large computes the row's chunks z, z + kRankParts, ... itself.
// Workgroup b < xch kXSlots then takes chunk b mod xch of the rows computed
// exactly with list index s, s + kXSlots, ... (s = b / xch): it marks the
// rows 1024 at a time (the same marks in every workgroup: they follow from
// the filter's counts, tau and flags) and counts them in row order.
static_assert((size_t)kRankCap * 8 + ((size_t)kRankSub + 4) * 4 <= kXLdsBytes, "the rank part's LDS inside the exact part's");
__global__ __launch_bounds__(kXThreads) void fused_select_kernel(FusedArgs a, int R, int rank_wg,
                                                                 int32_t* __restrict__ idx, float* __restrict__ val) {
  extern __shared__ __align__(16) unsigned char xl[];
  __shared__ XShared S;
  __shared__ RankShared<kXThreads> RS;
  __shared__ uint32_t cflg[kXThreads / 32];  // bit i: row r0 + i is computed exactly
  __shared__ int s_ex;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, b = (int)blockIdx.x;
  // marks of rows [r0, r0 + 1024) into cflg (every thread)
  auto mark = [&](int r0) {
    const uint64_t bm = __ballot(r0 + tid < R && row_exact(a, r0 + tid));
    if (lane == 0) {
      cflg[2 * wave] = (uint32_t)bm;
      cflg[2 * wave + 1] = (uint32_t)(bm >> 32);
    }
  };
  mark(0);  // the first rows' marks now: their loads overlap the rank part's
  __syncthreads();
  int cnt0 = 0;  // rows computed exactly among the first 1024
  for (int x = 0; x < kXThreads / 32; ++x) cnt0 += __popc(cflg[x]);
  if (b < rank_wg) {
    const int j = b / kRankXcd, z = j % kRankParts, r = (j / kRankParts) * kRankXcd + b % kRankXcd;
    if (r < R) {
      if (r >= kXThreads && tid == 0) s_ex = row_exact(a, r) ? 1 : 0;
      __syncthreads();
      const bool ex = r < kXThreads ? ((cflg[r >> 5] >> (r & 31)) & 1u) != 0u : s_ex != 0;
      if (!ex) {
        const bool over = rank_part<kXThreads>(a, r, z, idx, val, reinterpret_cast<uint64_t*>(xl),
                                    reinterpret_cast<uint32_t*>(xl + (size_t)kRankCap * 8), RS);
        __syncthreads();
        if (over)
          for (int zz = z; zz < a.ws.xch; zz += kRankParts) exact_chunk(a, r, zz, idx, val, xl, S);
      }
    }
  }
  const int xch = a.ws.xch, zz = b % xch, s = b / xch;
  if (s >= kXSlots) return;
  if (R <= kXThreads && cnt0 <= s) return;  // no exact row for this workgroup (the usual case)
  int before = 0;  // rows computed exactly below r0
  for (int r0 = 0; r0 < R; r0 += kXThreads) {
    if (r0 > 0) {
      __syncthreads();  // the marks of the previous rows are read
      mark(r0);
    }
    __syncthreads();
    int cnt = 0;
    for (int x = 0; x < kXThreads / 32; ++x) cnt += __popc(cflg[x]);
    // list indexes jl = s (mod kXSlots) among this run's rows
    for (int jl = before + (s - before % kXSlots + kXSlots) % kXSlots; jl < before + cnt; jl += kXSlots) {
      int x = 0, left = jl - before;
      while (left >= __popc(cflg[x])) left -= __popc(cflg[x++]);
      uint32_t w = cflg[x];
      for (; left > 0; --left) w &= w - 1u;
      exact_chunk(a, r0 + 32 * x + __builtin_ctz(w), zz, idx, val, xl, S);
    }
    before += cnt;
  }
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

// Compute units of device dev (looked up once per device).
static int device_cus(int dev) {
  static std::atomic<int> cus[64];
  if (dev < 0 || dev >= 64) return 0;
  int c = cus[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      c = -1;  // unknown: no one-launch select pass
    }
    cus[dev].store(c, std::memory_order_relaxed);
  }
  return c > 0 ? c : 0;
}

fathom_status launch_scan_topk_fused(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U,
                                     int64_t nb_cap, const void* q, fathom_dtype qdt, int G, const uint8_t* depths,
                                     int k, int64_t lo, int64_t tail, int max_unit_bits, int32_t* idx, float* val,
                                     void* ws, uint32_t* st, hipStream_t s) {
  if (U == 0) return FATHOM_OK;
  if (nb_cap == 0) {
    hipLaunchKernelGGL(fused_empty_kernel, dim3(U * G), dim3(256), 0, s, n, G, k, idx, val, st);
    FATHOM_LAUNCH_CHECK();
    return FATHOM_OK;
  }
  // the exact pass's dynamic LDS limit, raised once per device (racing
  // callers may both set it; the call is idempotent)
  static std::atomic<uint64_t> attr_set{0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return FATHOM_ERR_HIP;
  }
  const uint64_t bit = dev < 64 ? 1ull << dev : 0ull;
  if (!bit || !(attr_set.load(std::memory_order_acquire) & bit)) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(&fused_select_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)kXLdsBytes) != hipSuccess) {
      (void)hipGetLastError();
      return FATHOM_ERR_HIP;
    }
    attr_set.fetch_or(bit, std::memory_order_release);
  }
  FusedArgs fa;
  fa.planes = planes;
  fa.scales = scales;
  fa.n = n;
  fa.nb_cap = nb_cap;
  fa.q = q;
  fa.qdt = qdt;
  fa.G = G;
  fa.depths = depths;
  fa.lo = lo;
  fa.tail = tail;
  fa.k = k;
  fa.ws = fused_carve(ws, U * G, U, nb_cap, k);
  fa.st = st;
  fa.ccap = max_unit_bits > 64 && max_unit_bits <= 80 ? 80 : 64;
  const int R = U * G;
  const bool f16 = qdt == FATHOM_F16;
  // a unit with at most 80 depth bits has at most 80 cells and channels:
  // with such a bound the cell filter takes every unit, and the wide
  // launches are skipped.  (A unit above the caller's bound is left to the
  // exact rows of the select pass.)
  const bool wide = !(max_unit_bits > 0 && max_unit_bits <= kCC && nb_cap < kOneNbMax);
  if (G <= 4)
    hipLaunchKernelGGL(fused_sample_kernel, dim3((unsigned)fa.ws.s_quads, (unsigned)U), dim3(kFT), 0, s, fa);
  // narrow: the cell filter finds tau itself and the sample pass sets the
  // rows' state, so the tau pass runs only for the wide pass or G > 4
  if (wide || G > 4) hipLaunchKernelGGL(fused_tau_kernel, dim3(R), dim3(kTauThreads), 0, s, fa);
  if (G <= 4) {
    dim3 gm((unsigned)fa.ws.nwg, (unsigned)U);
    launch_filter(fa, U, max_unit_bits, s);
    if (wide) {
      if (f16) hipLaunchKernelGGL((fused_main_kernel<true, 8>), gm, dim3(kFT), 0, s, fa);
      else hipLaunchKernelGGL((fused_main_kernel<false, 8>), gm, dim3(kFT), 0, s, fa);
    }
  }
  const unsigned rank_wg = (unsigned)((R + kRankXcd - 1) / kRankXcd) * kRankXcd * kRankParts;
  const unsigned xg = (unsigned)fa.ws.xch * (unsigned)kXSlots;
  if (rank_wg <= (unsigned)device_cus(dev)) {  // the rank parts fit one round: ranks and exact rows in one launch
    hipLaunchKernelGGL(fused_select_kernel, dim3(rank_wg > xg ? rank_wg : xg), dim3(kXThreads), kXLdsBytes, s, fa, R,
                       (int)rank_wg, idx, val);
  } else {
    hipLaunchKernelGGL(fused_rank_kernel, dim3(rank_wg), dim3(kRankThreads), 0, s, fa, R, idx, val);
    hipLaunchKernelGGL(fused_select_kernel, dim3(xg), dim3(kXThreads), kXLdsBytes, s, fa, R, 0, idx, val);
  }
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

// ---------------------------------------------------------------- no workspace
// fathom_scan_topk_noalloc's workspace: one file-scope array per device,
// loaded with the code object and held until the process ends.  In host code
// the name `scratch` is only a handle; its device address comes from
// hipGetSymbolAddress, called once per device with that device current, and
// only that address is passed to kernels.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kScratchDevices = 64;
static std::atomic<void*> g_scratch_addr[kScratchDevices];
static std::mutex g_scratch_mu;

size_t scratch_capacity() { return kScratchBytes; }

// The current device's address of `scratch` (looked up on its first use).
fathom_status scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return FATHOM_ERR_HIP;
  }
  if (dev < 0 || dev >= kScratchDevices) return FATHOM_ERR_UNSUPPORTED;
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
        (void)hipGetLastError();
        return FATHOM_ERR_HIP;
      }
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return FATHOM_OK;
}

}  // namespace fathom
