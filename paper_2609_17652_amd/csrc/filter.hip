// Full pass of fathom_scan_topk for units of at most 80 cells (one per
// active channel and plane: every unit of at most 80 depth bits, so every
// unit under water-filling at B <= 80 and uniform depth at r <= 16): an int8
// MFMA proxy of every key's four head
// scores over its plane bits, exact re-scoring of the keys the proxy's bound
// cannot exclude, and the appends of keys with exact score >= tau to their
// row's survivor list (Sec. 3.2-3.3 scores, Sec. 2 top-k).
//
// Cells.  With khat = a16 sum_{p<t} 2^-p (b_p - 1/2) (the prefix
// dequantisation of Sec. 3.2 written out; exact), the documented score of a
// key is, as a real number,
//   s = sum over cells (x, p) of w (b - 1/2),   w = q_x a16_x 2^-p,
// one cell per active channel x and plane p < t_x.  Per group (8 blocks)
// and head, delta = 2^e is the smallest power of two with max |q a16| / delta
// <= 127; each cell gets its own int8 weight W = rne(w / delta), so with
// S = sum W b and Wsum = sum W over the cells of a block,
//   |s - delta (S - Wsum / 2)| <= delta cells / 4 + (A^2 127 2^-24) delta
// (weight rounding, then the A roundings of the fp32 chain), plus A 2^-120
// for subnormal results.  A key is a candidate for head h iff
// S >= thr = floor((floor(2 (tau - E) / delta) - 1 + Wsum) / 2).  At three
// and five slices the weights have two levels, W' = 128 W + W_lo in units
// of delta / 128 (the bound's cell term shrinks by 128).
//
// Layout.  Cells are ordered plane-major without padding (plane p's cells are
// its channels, a prefix of the proxy order: depth descending, channel
// ascending); row group g = cells 4 g .. 4 g + 3, which may span two planes.
// The plane words of a quad (4 blocks) are staged in LDS as loaded, cell by
// cell (cells past the unit's read as zero), and ds_read_b64_tr_b8 hands
// lane l the bytes of 8 cells (two row groups) at octet l & 7 of block
// l >> 4: within a 16-lane
// group, output lane 8h + r takes byte r of the words addressed by lanes h,
// h + 2, ..., h + 14.  So lane l owns the 4 keys 8 o + 4 nib + mu (o = l & 7,
// nib = (l >> 3) & 1) of block l >> 4, and with pos = 4 nib + mu,
// X & (0x01010101 << pos) is that key's B operand dword of a row group for
// v_mfma_i32_16x16x64_i8 (byte value b 2^pos, or -128 b at pos 7).  A is
// block diagonal: row 4 g' + h of k-group g' holds block g''s head-h weights,
// negated (-W), so an accumulator holds start - 2^pos S (start + 128 S at
// pos 7).  The starts are thr 2^pos - 1 (-128 thr at pos 7), so a key is a
// candidate for head h iff its accumulator is < 0 (>= 0 at pos 7): the sign
// bits of a lane's 16 accumulators, gathered a byte per head, are its keys'
// candidate heads.
//
// Candidate keys are queued per wave in LDS with their lane's staged
// dwords; a batch is scored exactly in the documented order (channels
// ascending, fmaf from +0) with the scales of the last Slots groups kept in
// an LDS ring, and keys with score >= tau are appended to their row's list.
#include "cellplan.hpp"

namespace fathom {

constexpr int kCSB = 8;          // blocks per group (one delta per head; one loop iteration)
constexpr int kSv = 8;           // survivors per head buffered in LDS before a list append

// Geometry of an instantiation with NS slices of 4 row groups (16 cells):
// NS = 3 serves units of at most 48 cells, NS = 4 of at most 64, NS = 5 of
// at most 80.  The scale ring holds one row of C + 2 halfs per block (an odd
// number of dwords, so the lanes of a re-scoring batch fall in different
// banks) for Slots groups; three workgroups per CU fit the LDS with 6 slots
// at NS = 3 (a wave's 6 groups of the 2^20-token layer: no flush before its
// end), 3 at NS = 4 and 2 at NS = 5 with a queue of 32 candidates (the
// space of the second-level weights; 24 candidates with 3 slots ran as
// fast, 48 with 1 slot 19 % slower).  NS = 3 and 5 have two-level weights
// (at NS = 5 the MFMA loop runs slice by slice so that one slice's two
// weight sets are live at a time); NS = 4 keeps one level.  A lane stages K plane words per quad: 4 cells of its row group up to
// NS = 4, at NS = 5 the cells lane / 4 + 16 k, k < 5.
template <int NS>
struct CGeo {
  static_assert(NS >= 3 && NS <= 5, "three to five slices");
  static constexpr int G = 4 * NS;
  static constexpr int C = 4 * G;
  static constexpr int Slots = NS == 3 ? 6 : NS == 4 ? 3 : 2;
  static constexpr int SclRow = C + 2;
  static constexpr bool Fine = NS != 4;  // two-level weights (slice-outer at five slices, so the registers fit them)
  static constexpr int Q = NS == 5 ? 32 : 64;  // queued candidates per wave; re-scored at a quad boundary once full
  static constexpr int K = NS == 5 ? 5 : 4;    // plane words a lane stages per quad
};
// Fine weights W' = 128 W + W_lo count in units of delta / 128; |W'| <=
// 127 * 128 + 64, so |S'| < 2^21 for up to 80 cells: thresholds are clamped
// to +-2^21 and an accumulator stays below 2^29.
constexpr int kCThrMax = 1 << 21;
constexpr int kCWaves = 4;       // waves per workgroup
constexpr int kCThreads = kCWaves * kWave;
static_assert(kPools == kCWaves, "one pool counter per wave of a workgroup");

template <int NS>
struct alignas(16) FilterLds {
  using Geo = CGeo<NS>;
  uint64_t raw[Geo::C][4];                        // the quad's plane words: cell, block
  uint32_t zero[Geo::G];                          // zero dwords (the A operand of lanes that carry no weights)
  uint32_t W[4][4][Geo::G];                       // int8 weights: block of the quad, head, row group
  uint32_t Wlo[Geo::Fine ? 4 : 1][4][Geo::G];     // fine weights: the residual weights W_lo, likewise
  int32_t ini[4][2][4][4];                        // accumulator starts: block, nibble, mu, head
  uint16_t scl[Geo::Slots][kCSB][Geo::SclRow];    // fp16 scales: ring slot, block, cell (its channel's scale)
  uint32_t qx[Geo::G][Geo::Q];                    // queued keys' staged dwords (digits while re-scored): dword, entry
  uint32_t qi[Geo::Q];                    // queued key index
  uint32_t qf[Geo::Q];                    // pos | slot << 3 (3 bits) | block of the group << 8 | head h at bit 7 + 8 h
  uint64_t sv[4][kSv];                    // survivors per head not yet appended to the row's list
};

typedef __attribute__((ext_vector_type(4))) int v4i;
typedef unsigned int v2u32 __attribute__((ext_vector_type(2)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
constexpr int kRawBufferFlags = 0x00020000;  // raw buffer, 32-bit data format
constexpr uint32_t kPastRange = 0xFFFFFFF0u;  // a buffer offset past every range (loads return zero)

__device__ __forceinline__ int cuni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Orders LDS accesses in the compiler only: a wave's LDS instructions execute
// in program order, so a wave reading what it wrote itself needs no wait.
__device__ __forceinline__ void lds_order() { asm volatile("" ::: "memory"); }
// Keeps the scheduler from moving instructions across this point.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }
__device__ __forceinline__ uint64_t lanes_below(int lane) { return lane == 0 ? 0ull : (~0ull >> (64 - lane)); }

// ---------------------------------------------------------------- scales
// Lane c (< C) holds the 8 scales of cell c's channel (scale row jrow) for the
// group at block sb0, two blocks a dword, and at NS = 5 lane l also those of
// cell 64 + l (row jrow2), read through a buffer descriptor over the unit's
// scale rows (zero past them, and for cells >= C; the lanes of one channel's
// cells read the same bytes).  With 16-byte aligned rows
// (nb_cap a multiple of 8) one 16-byte load per lane; blocks past nb_cap then
// read the next row's scales, which only the (ineligible) keys of those
// blocks and delta see.  Otherwise 8 two-byte loads, each past the range
// beyond nb_cap.  An invalid load (no group of the wave there) reads past the
// range: it is issued, so wait counts stay exact, but fetches nothing.
template <int NS>
struct CScl {
  static constexpr bool Two = CGeo<NS>::C > kWave;  // a second cell per lane
  uint32_t v[kCSB / 2];
  uint32_t v2[Two ? kCSB / 2 : 1];
};
typedef unsigned short u16x1;

template <bool VEC, int NS>
__device__ __forceinline__ void cscl_issue(CScl<NS>& r, const FusedArgs& a, int u, int nc, int jrow, int jrow2, int sb0,
                                           bool valid) {
  const int lane = threadIdx.x & 63;
  const uint64_t base = reinterpret_cast<uint64_t>(a.scales + (int64_t)u * kD * a.nb_cap);
  const uint32_t alo = (uint32_t)cuni((int)(uint32_t)base), ahi = (uint32_t)cuni((int)(uint32_t)(base >> 32));
  const uint32_t bytes = (uint32_t)(kD * 2) * (uint32_t)a.nb_cap;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      reinterpret_cast<void*>(((uint64_t)ahi << 32) | alo), (short)0, (int)bytes, kRawBufferFlags);
  const uint32_t off = lane < nc && valid ? ((uint32_t)jrow * (uint32_t)a.nb_cap + (uint32_t)sb0) * 2u : kPastRange;
  const uint32_t off2 =
      lane + kWave < nc && valid ? ((uint32_t)jrow2 * (uint32_t)a.nb_cap + (uint32_t)sb0) * 2u : kPastRange;
  if constexpr (VEC) {
    const v4u x0 = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off, 0, 0);
    r.v[0] = x0.x; r.v[1] = x0.y; r.v[2] = x0.z; r.v[3] = x0.w;
    if constexpr (CScl<NS>::Two) {
      const v4u x1 = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off2, 0, 0);
      r.v2[0] = x1.x; r.v2[1] = x1.y; r.v2[2] = x1.z; r.v2[3] = x1.w;
    }
  } else {
    const int64_t left = a.nb_cap - (int64_t)sb0;  // blocks of the group inside the row
    uint32_t h[kCSB];
#pragma unroll
    for (int b = 0; b < kCSB; ++b)
      h[b] = __builtin_amdgcn_raw_buffer_load_b16(rs, (int)(b < left && valid ? off + 2u * b : kPastRange), 0, 0);
#pragma unroll
    for (int i = 0; i < kCSB / 2; ++i) r.v[i] = (h[2 * i] & 0xFFFFu) | (h[2 * i + 1] << 16);
    if constexpr (CScl<NS>::Two) {
#pragma unroll
      for (int b = 0; b < kCSB; ++b)
        h[b] = __builtin_amdgcn_raw_buffer_load_b16(rs, (int)(b < left && valid ? off2 + 2u * b : kPastRange), 0, 0);
#pragma unroll
      for (int i = 0; i < kCSB / 2; ++i) r.v2[i] = (h[2 * i] & 0xFFFFu) | (h[2 * i + 1] << 16);
    }
  }
}

// Per group and head: delta = 2^e and whether a bound exists.
struct CDel {
  int e;
  bool valid;
};

// Writes the group's scales to ring slot `slot` (cell order: cell c holds
// its channel's scale, so the plane-0 cell of proxy channel x is cell x) and
// returns delta of head `hq` (every lane: its own head for the weights).  qv:
// q of cell `lane`'s channel for the four heads (0 past the cells), qv2 that
// of cell 64 + lane (NS = 5).
__device__ __forceinline__ uint32_t cscl_absmax(const uint32_t (&v)[kCSB / 2]) {
  uint32_t mx = 0u;
#pragma unroll
  for (int i = 0; i < kCSB / 2; ++i) {
    const uint32_t w = v[i] & 0x7FFF7FFFu;
    const uint32_t m = (w & 0xFFFFu) > (w >> 16) ? (w & 0xFFFFu) : (w >> 16);
    mx = m > mx ? m : mx;
  }
  return mx;
}
template <int NS>
__device__ __forceinline__ CDel cscl_commit(const CScl<NS>& r, FilterLds<NS>& L, int slot, int hq, const float (&qv)[4],
                                            const float (&qv2)[4]) {
  const int lane = threadIdx.x & 63;
  if (lane < CGeo<NS>::C) {
#pragma unroll
    for (int b = 0; b < kCSB; ++b) L.scl[slot][b][lane] = (uint16_t)((r.v[b >> 1] >> (16 * (b & 1))) & 0xFFFFu);
  }
  const uint32_t mx = cscl_absmax(r.v);
  uint32_t mx2 = 0u;
  if constexpr (CScl<NS>::Two) {
    if (lane < CGeo<NS>::C - kWave) {
#pragma unroll
      for (int b = 0; b < kCSB; ++b)
        L.scl[slot][b][kWave + lane] = (uint16_t)((r.v2[b >> 1] >> (16 * (b & 1))) & 0xFFFFu);
    }
    mx2 = cscl_absmax(r.v2);
  }
  const bool nf = __ballot(mx >= 0x7C00u || mx2 >= 0x7C00u) != 0ull;
  const float am = half_bits_to_float((uint16_t)(mx >= 0x7C00u ? 0u : mx));
  uint32_t M[4];
#pragma unroll
  for (int h = 0; h < 4; ++h) M[h] = __float_as_uint(__fmul_rn(fabsf(qv[h]), am));
  if constexpr (CScl<NS>::Two) {
    const float am2 = half_bits_to_float((uint16_t)(mx2 >= 0x7C00u ? 0u : mx2));
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const uint32_t m2 = __float_as_uint(__fmul_rn(fabsf(qv2[h]), am2));
      M[h] = m2 > M[h] ? m2 : M[h];
    }
  }
  wave_max4_u(M);
  const float Mh = __uint_as_float(hq == 0 ? M[0] : hq == 1 ? M[1] : hq == 2 ? M[2] : M[3]);
  CDel d;
  d.e = 0;
  d.valid = !nf && Mh <= 3.402823466e38f;
  if (Mh > 0.0f && d.valid) {
    int E;
    (void)frexpf(Mh, &E);  // Mh in [2^(E-1), 2^E)
    d.e = Mh <= 127.0f * ldexpf(1.0f, E - 7) ? E - 7 : E - 6;
    d.valid = d.e >= -100 && d.e <= 100;
  }
  return d;
}

// ---------------------------------------------------------------- staging
// Lane (block bq = lane & 3 of the quad) loads the plane words of K cells for
// its block through a buffer descriptor over the unit's planes, and stores
// them as raw[cell][bq]: up to NS = 4 the 4 cells of row group g = lane >> 2,
// at NS = 5 the cells lane / 4 + 16 k.  Pad cells (and row groups past the
// unit's) read past the descriptor's range, which returns zero; every other
// load stays inside the unit.
template <int NS>
__device__ __forceinline__ int cstage_cell(int lane, int k) {
  return CGeo<NS>::K == 5 ? (lane >> 2) + 16 * k : 4 * (lane >> 2) + k;
}
template <int NS>
struct CStage {
  __amdgpu_buffer_rsrc_t rs;     // the unit's planes (ub bytes)
  uint32_t boff[CGeo<NS>::K];    // byte offset of word k for block bq of a quad starting at block 0
  uint32_t ub;                   // an offset past the range
};
template <int NS>
struct CRaw {
  uint64_t w[CGeo<NS>::K];  // word k (cell cstage_cell(lane, k)) of block bq
};

// Pad cells get the offset ub: with the quad's offset (at most 8 (nb_cap +
// 40) bytes) added it stays past the range without wrapping (4104 nb_cap +
// 320 < 2^32 for nb_cap < kOneNbMax).
template <int NS>
__device__ __forceinline__ void cstage_setup(CStage<NS>& S, const CellPlan& P, const FusedArgs& a, uint64_t ubase,
                                             uint32_t ub) {
  const int lane = threadIdx.x & 63, g = lane >> 2, bq = lane & 3;
  const uint32_t alo = (uint32_t)cuni((int)(uint32_t)ubase), ahi = (uint32_t)cuni((int)(uint32_t)(ubase >> 32));
  S.rs = __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(((uint64_t)ahi << 32) | alo), (short)0,
                                          (int)(uint32_t)cuni((int)ub), kRawBufferFlags);
  if constexpr (CGeo<NS>::K == 5) {
    // cell c's row: half c & 1 of word (c >> 1) & 1 of row group c >> 2
    // (kCPad for every cell past the unit's)
#pragma unroll
    for (int k = 0; k < 5; ++k) {
      const int c = cstage_cell<NS>(lane, k);
      const uint32_t row = (P.rrow[c >> 2][(c >> 1) & 1] >> (16 * (c & 1))) & 0xFFFFu;
      S.boff[k] = row != kCPad ? (row * (uint32_t)a.nb_cap + (uint32_t)bq) * 8u : ub;
    }
  } else {
    const bool on = g < cuni(P.rg);
    const uint32_t r0 = P.rrow[on ? g : 0][0], r1 = P.rrow[on ? g : 0][1];
    const uint32_t rows[4] = {r0 & 0xFFFFu, r0 >> 16, r1 & 0xFFFFu, r1 >> 16};
#pragma unroll
    for (int k = 0; k < 4; ++k)
      S.boff[k] = on && rows[k] != kCPad ? (rows[k] * (uint32_t)a.nb_cap + (uint32_t)bq) * 8u : ub;
  }
  S.ub = ub;
}

// Loads of the quad whose first block is qb0, issued for every quad the loop
// could reach so that the compiler's wait counts stay exact: an invalid quad
// (no group of the wave there) reads past the range and fetches nothing; a
// valid quad past the unit's blocks reads other rows' words or zeros, which
// no eligible key uses.
template <int NS>
__device__ __forceinline__ void cstage_issue(CRaw<NS>& R, const CStage<NS>& S, int qb0, bool valid) {
  const int so = cuni((int)((uint32_t)qb0 * 8u));
#pragma unroll
  for (int k = 0; k < CGeo<NS>::K; ++k) {
    const v2u32 v = __builtin_amdgcn_raw_buffer_load_b64(S.rs, (int)(valid ? S.boff[k] : S.ub), so, 0);
    R.w[k] = ((uint64_t)v.y << 32) | v.x;
  }
}

template <int NS>
__device__ __forceinline__ void cstage_write(const CRaw<NS>& R, FilterLds<NS>& L) {
  const int lane = threadIdx.x & 63, g = lane >> 2, bq = lane & 3;
  if constexpr (CGeo<NS>::K == 5) {
#pragma unroll
    for (int k = 0; k < 5; ++k) L.raw[cstage_cell<NS>(lane, k)][bq] = R.w[k];
  } else if (g < CGeo<NS>::G) {
#pragma unroll
    for (int k = 0; k < 4; ++k) L.raw[4 * g + k][bq] = R.w[k];
  }
}

// Row groups 2 P and 2 P + 1 of this lane's block and octet (v: its two dwords)
// from the staged words; lane l (as a source) addresses cell 8 P + ((l & 15) >> 1)
// of block l >> 4.
typedef int v2i __attribute__((ext_vector_type(2)));
template <int NS>
__device__ __forceinline__ v2i ctr_read(const FilterLds<NS>& L, uint32_t src_off, int P) {
  const unsigned char* base = reinterpret_cast<const unsigned char*>(&L.raw[0][0]) + src_off + P * 8 * 4 * 8;
  return __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i*)(base));
}

// ---------------------------------------------------------------- weights
// Lanes (block b = lane >> 4 of the quad, head h = (lane >> 2) & 3, part =
// lane & 3): the negated int8 weights -W of row groups g = part (mod 4) of
// block b for head h, their sum, and the accumulator starts of (b, h).  With
// M0 = 1.5 2^(23 + e) the low byte of r = fl(-q 2^-p a16 + M0) is
// W = rne(-q a16 2^-p / delta) as a two's complement byte.  Fine weights add
// W_lo: with K1 = M0 (1 + 2^-7), K1 - r = M0 / 128 - W delta exactly, and the
// low byte of fl(-q 2^-p a16 + (K1 - r)) is the residual rounded in units of
// delta / 128 (|W_lo| <= 64), so W' = 128 W + W_lo is the cell's weight
// rounded to delta / 128 with one rounding.  Pad cells (q = 0) get weight 0;
// a group without thresholds (a head past G, no tau, no valid delta) gets
// fixed starts that no sum of products can cross (|S' 2^pos| < 2^27),
// whatever its weights.
struct CHead {
  float M0;     // rounding constant, 1.5 2^(23 + e)
  float K1;     // M0 (1 + 2^-7): fine weights
  int X;        // floor(2 (tau - E) / delta) - 1, clamped
  bool m0;      // thresholds apply
  int c0, c1;   // the starts of positions 2 part and 2 part + 1 when they do not
};

template <int NS>
__device__ __forceinline__ void cquad_weights(const CellPlan& P, FilterLds<NS>& L, const CHead& H, int slot, int sbq) {
  const int lane = threadIdx.x & 63, b = lane >> 4, h = (lane >> 2) & 3, part = lane & 3;
  const uint16_t* srow = &L.scl[slot][sbq + b][0];
  // every read first: row groups g = part + 4 k, cells 4 g .. 4 g + 3
  float4 qv[NS];
  uint32_t s01[NS], s23[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const int g = part + 4 * k;
    qv[k] = *reinterpret_cast<const float4*>(&P.qrg[g][h][0]);
    s01[k] = *reinterpret_cast<const uint32_t*>(&srow[4 * g]);
    s23[k] = *reinterpret_cast<const uint32_t*>(&srow[4 * g + 2]);
  }
  int wsum = 0, wlo = 0;
  const float Mp = H.M0;
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const int g = part + 4 * k;
    const float a0 = half_bits_to_float((uint16_t)(s01[k] & 0xFFFFu)), a1 = half_bits_to_float((uint16_t)(s01[k] >> 16));
    const float a2 = half_bits_to_float((uint16_t)(s23[k] & 0xFFFFu)), a3 = half_bits_to_float((uint16_t)(s23[k] >> 16));
    const uint32_t r0 = __float_as_uint(__fmaf_rn(qv[k].x, a0, Mp)), r1 = __float_as_uint(__fmaf_rn(qv[k].y, a1, Mp));
    const uint32_t r2 = __float_as_uint(__fmaf_rn(qv[k].z, a2, Mp)), r3 = __float_as_uint(__fmaf_rn(qv[k].w, a3, Mp));
    const uint32_t wd = __builtin_amdgcn_perm(r1, r0, 0x0c0c0400u) | __builtin_amdgcn_perm(r3, r2, 0x04000c0cu);
    L.W[b][h][g] = wd;
    wsum = __builtin_amdgcn_sdot4((int)wd, 0x01010101, wsum, false);
    if constexpr (CGeo<NS>::Fine) {
      const float c0 = H.K1 - __uint_as_float(r0), c1 = H.K1 - __uint_as_float(r1);
      const float c2 = H.K1 - __uint_as_float(r2), c3 = H.K1 - __uint_as_float(r3);
      const uint32_t l0 = __float_as_uint(__fmaf_rn(qv[k].x, a0, c0)), l1 = __float_as_uint(__fmaf_rn(qv[k].y, a1, c1));
      const uint32_t l2 = __float_as_uint(__fmaf_rn(qv[k].z, a2, c2)), l3 = __float_as_uint(__fmaf_rn(qv[k].w, a3, c3));
      const uint32_t wl = __builtin_amdgcn_perm(l1, l0, 0x0c0c0400u) | __builtin_amdgcn_perm(l3, l2, 0x04000c0cu);
      L.Wlo[b][h][g] = wl;
      wlo = __builtin_amdgcn_sdot4((int)wl, 0x01010101, wlo, false);
    }
  }
  if constexpr (CGeo<NS>::Fine) wsum = wsum * 128 + wlo;  // -sum W' of the lane's cells
  wsum += dpp_i<0xB1>(wsum);  // quad_perm [1,0,3,2]
  wsum += dpp_i<0x4E>(wsum);  // quad_perm [2,3,0,1]: -Wsum of (b, h)
  // part writes the starts of positions 2 part, 2 part + 1 (nibble hb = part >> 1);
  // position 7 is part 3's second
  constexpr int tm = CGeo<NS>::Fine ? kCThrMax : kThrMax;
  int thr = (H.X - wsum) >> 1;
  thr = thr < -tm ? -tm : thr > tm ? tm : thr;
  const int hb = part >> 1, mu0 = 2 * (part & 1);
  const int t0 = thr * (1 << (4 * hb + mu0)), t1 = thr * (1 << (4 * hb + mu0 + 1));
  L.ini[b][hb][mu0][h] = H.m0 ? t0 - 1 : H.c0;
  L.ini[b][hb][mu0 + 1][h] = H.m0 ? (part == 3 ? -t1 : t1 - 1) : H.c1;
}

// ---------------------------------------------------------------- survivors
// Appends survivors to the rows' lists: the nb[h] buffered ones of head h and
// this lane's new one of head h when bit h of `keep` is set (composite
// comp[h], rank[h] among the wave's new ones, c[h] of them).  One atomic
// instruction reserves every head's range (lane h for row u G + h), so a
// flush costs one round trip whatever the number of heads.
template <int NS>
__device__ __forceinline__ void cappend(FilterLds<NS>& L, const FusedArgs& a, int u, const int (&nb)[4], const int (&c)[4],
                                        uint32_t keep, const uint64_t (&comp)[4], const int (&rank)[4]) {
  const int lane = threadIdx.x & 63, G = a.G;
  const int tot = lane == 0 ? nb[0] + c[0] : lane == 1 ? nb[1] + c[1] : lane == 2 ? nb[2] + c[2] : nb[3] + c[3];
  uint32_t base = 0u;
  if (lane < G && tot > 0) base = gatomic_add(&a.ws.cnt[(u * G + lane) * kCntStride], (uint32_t)tot);
  const uint32_t lcap = (uint32_t)a.ws.lcap;
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    if (nb[h] + c[h] == 0) continue;  // every head past G
    const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)base, h);
    uint64_t* row = a.ws.cand + (int64_t)(u * G + h) * a.ws.lcap;
    if (lane < nb[h] && b + (uint32_t)lane < lcap) gstore(&row[b + (uint32_t)lane], L.sv[h][lane]);
    const uint32_t pos = b + (uint32_t)nb[h] + (uint32_t)rank[h];
    if (((keep >> h) & 1u) && pos < lcap) gstore(&row[pos], comp[h]);
  }
}

// ---------------------------------------------------------------- re-scoring
// Exact documented scores of the queued keys (lane e < nq) and their appends
// to the survivor lists.  First each entry's staged dwords become digit
// dwords in proxy order (u = sum_p b_p 2^(3-p), byte x of the entry, in
// place: the plane-p dwords of proxy dword i sit at or after dword i), then
// the chain runs over the active channels ascending (padded to a multiple of
// 4 with q = 0, which leaves every score unchanged).
template <int NS>
__device__ __forceinline__ void crescore(const CellPlan& P, FilterLds<NS>& L, const FusedArgs& a, int u, int nq, int (&svn)[4]) {
  const int lane = threadIdx.x & 63, G = a.G;
  const bool on = lane < nq;
  const int e = on ? lane : 0;
  const uint32_t ki = L.qi[e], f = L.qf[e];
  const uint32_t pos = f & 7u, hm = on ? f : 0u;
  const int slot = (int)((f >> 3) & 7u), blk = (int)((f >> 8) & 7u);
  constexpr int Q = CGeo<NS>::Q;
  uint32_t* ent = &L.qx[0][e];  // dword i of the entry at ent[i * Q] (entries side by side: no bank conflicts)
  // digit dword i (proxy channels 4 i .. 4 i + 3): the plane-p bits of its
  // channels are cells base_p + 4 i .., bytes (base_p & 3) .. of row group
  // (base_p + 4 i) >> 2 and the next one (a byte funnel shift), the bytes of
  // channels without plane p masked off; plane 0 is row group i itself, and
  // every other dword read lies past i, so the digits overwrite in place
  int npl[kPlanes], bpl[kPlanes];
#pragma unroll
  for (int p = 0; p < kPlanes; ++p) {
    npl[p] = cuni(P.np[p]);
    bpl[p] = cuni(P.base[p]);
  }
  const int nd0 = (npl[0] + 3) >> 2;
  for (int i = 0; i < nd0; ++i) {
    uint32_t dw = 0u;
#pragma unroll
    for (int p = 0; p < kPlanes; ++p) {
      const int v = npl[p] - 4 * i;  // channels of the dword with plane p
      if (v > 0) {
        const int c0 = bpl[p] + 4 * i, r = c0 >> 2, sh = c0 & 3;
        const int r1 = r + 1 < CGeo<NS>::G ? r + 1 : r;
        const uint32_t lo = ent[r * Q], hi = ent[r1 * Q];
        const uint32_t w = sh ? __builtin_amdgcn_alignbyte(hi, lo, (uint32_t)sh) : lo;
        const uint32_t m = v >= 4 ? 0x01010101u : 0x01010101u >> (8 * (4 - v));
        dw |= ((w >> pos) & m) << (3 - p);
      }
    }
    ent[i * Q] = dw;
  }
  // digit of proxy channel x: byte x & 3 of dword x >> 2
  const uint8_t* dg = reinterpret_cast<const uint8_t*>(ent);
  const uint16_t* sv = &L.scl[slot][blk][0];
  const int A4 = (cuni(P.A) + 3) & ~3;
  float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int y0 = 0; y0 < A4; y0 += 4) {
    const int4 xa = *reinterpret_cast<const int4*>(&P.px[y0]);
    const float4 za = *reinterpret_cast<const float4*>(&P.zo[y0]);
    const int xs[4] = {xa.x, xa.y, xa.z, xa.w};
    const float zs[4] = {za.x, za.y, za.z, za.w};
    uint32_t dv[4], hv[4];
    float4 q4[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      dv[c] = dg[(xs[c] >> 2) * (Q * 4) + (xs[c] & 3)];
      hv[c] = sv[xs[c]];
      q4[c] = *reinterpret_cast<const float4*>(&P.qa[y0 + c][0]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      // (u / 8 + zo) has at most 5 significant bits, its product with a16 at
      // most 16: both steps are exact
      const float x8 = __fmaf_rn((float)dv[c], 0.125f, zs[c]);
      const float khat = __fmaf_rn(x8, half_bits_to_float((uint16_t)hv[c]), 0.0f);
      s[0] = __fmaf_rn(q4[c].x, khat, s[0]);
      s[1] = __fmaf_rn(q4[c].y, khat, s[1]);
      s[2] = __fmaf_rn(q4[c].z, khat, s[2]);
      s[3] = __fmaf_rn(q4[c].w, khat, s[3]);
    }
  }
  // survivors of each head go to the wave's LDS buffer; when one head's
  // would overflow, every head's buffer and new survivors go to the lists
  // together (one atomic instruction), as at the wave's end
  int c[4], rk[4];
  uint64_t comp[4];
  uint32_t keep = 0u;
  bool over = false;
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const bool k = h < G && ((hm >> (7 + 8 * h)) & 1u) && s[h] >= P.tau[h];
    const uint64_t bm = __ballot(k);
    c[h] = __popcll(bm);
    rk[h] = __popcll(bm & lanes_below(lane));
    comp[h] = ((uint64_t)score_key(s[h]) << 32) | (uint64_t)(~ki);
    keep |= (uint32_t)k << h;
    over |= svn[h] + c[h] > kSv;
  }
  if (over) {
    cappend(L, a, u, svn, c, keep, comp, rk);
#pragma unroll
    for (int h = 0; h < 4; ++h) svn[h] = 0;
  } else {
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if ((keep >> h) & 1u) L.sv[h][svn[h] + rk[h]] = comp[h];
      svn[h] += c[h];
    }
  }
  lds_order();
}

// ---------------------------------------------------------------- one wave
// Groups of 8 blocks of unit u: first the wave's ns static groups s0 +
// kCWaves i (the workgroup's waves take its static groups in turn, so two
// waves read the two halves of a 128-byte plane line at about the same time),
// then groups p0 + w + kPools j < pend taken one at a time through counter w
// of the unit's pool (w: the wave's index in its workgroup; kPools counters,
// so each sees a quarter of the atomics), quad by quad (one loop iteration
// per group).  Waves of one SIMD
// progress at unequal rates (older waves issue first), so the pool lets the
// faster ones take more of the unit.  `ready` runs once every first load is
// issued (every wave of the workgroup calls it, so it may hold a barrier); the
// wave stops if it returns false.  The plane words of a quad are loaded one
// group ahead (two register sets), the scales of a group one group ahead, in
// the same order on every path into the loop so that the compiler's load
// counters stay exact (a load with nothing to fetch reads past its range);
// the pool's counter is read a group before the group it names is loaded.  A
// wave's LDS accesses execute in program order, so staged data is read back
// without a wait.  Re-scoring runs at one place: after a quad's candidates,
// when the queue is full, when a quad's candidates do not fit, before
// the ring slot of the oldest queued key is reused, and at the end.
struct CGroups {
  int s0, ns;     // static groups s0 + kCWaves i, i < ns
  int p0, pend;   // the unit's pool of groups
  int ctr;        // the pool counter of this wave: word ctr of the pool counters (-1: no pool)
};
template <bool VEC, int NS, class Ready>
__device__ __forceinline__ void cwave_run(const CellPlan& P, FilterLds<NS>& L, const FusedArgs& a, int u, const CGroups& gs,
                                          int nbu, int lo, int hi, Ready&& ready) {
  using Geo = CGeo<NS>;
  const int lane = threadIdx.x & 63;
  const int bq = lane >> 4, nib = (lane >> 3) & 1, oct = lane & 7;
  const int kb = 8 * oct + 4 * nib;                      // key of mu = 0 within its block
  const bool wl = ((lane & 15) >> 2) == bq;              // carries weights in the A operand
  const int hq = (lane >> 2) & 3;                        // head of this lane's weights
  uint32_t mk[4];
#pragma unroll
  for (int mu = 0; mu < 4; ++mu) mk[mu] = 0x01010101u << (4 * nib + mu);
  const bool top = (lane & 3) == 3;  // as a weight lane: its second start is position 7
  const int C = cuni(P.C);
  const int cxl = P.cx[lane];                  // cell `lane`'s channel (proxy index)
  const int srow = lane < C ? P.pj[cxl] : 0;   // its scale row
  const int yl = P.py[cxl];                    // its ascending position (q: qa[yl])
  // cell 64 + lane's channel (NS = 5; read from the plan where needed, so
  // that no register holds it across the loop)
  auto cell2 = [&]() -> int { return Geo::C > kWave && lane + kWave < C ? P.cx[kWave + lane] : 0; };
  // as a transpose source: cell (l & 15) >> 1 of pair 0, block l >> 4
  const uint32_t src_off = (uint32_t)((((lane & 15) >> 1) * 4 + bq) * 8);
  // the A operand: this lane's weights, or zeros
  const uint32_t* wsrc = wl ? &L.W[bq][lane & 3][0] : &L.zero[0];
  const uint32_t* wlsrc = wl && Geo::Fine ? &L.Wlo[Geo::Fine ? bq : 0][lane & 3][0] : &L.zero[0];
  const uint64_t ubase = reinterpret_cast<uint64_t>(a.planes + (int64_t)u * kD * kPlanes * a.nb_cap);
  const uint32_t ubytes = (uint32_t)(kD * kPlanes * 8) * (uint32_t)a.nb_cap;
  CStage<NS> S;
  cstage_setup<NS>(S, P, a, ubase, ubytes);
  if (lane < Geo::G) L.zero[lane] = 0u;
  int pending = 0, oldest = 0;
  const int b0 = gs.s0 * kCSB;
  const bool any = gs.ns > 0;
  int svn[4] = {0, 0, 0, 0};  // buffered survivors per head
  // the issue order here (scales, quad 0, quad 1) is the loop's steady-state
  // order, so the compiler's load counters agree on every path into the loop
  CScl<NS> sr;
  cscl_issue<VEC, NS>(sr, a, u, C, srow, Geo::C > kWave ? P.pj[cell2()] : 0, b0, any);
  sched_fence();
  CRaw<NS> R0, R1;
  cstage_issue(R0, S, b0, any);
  sched_fence();
  cstage_issue(R1, S, b0 + kQB, any);
  sched_fence();
  if (!ready()) return;
  CHead H;
  int slot = 0;
  // gnxt: the group after the current one (-1: none); grab: the pool's
  // answer for the one after that, requested in the previous iteration
  int gnxt = gs.ns > 1 ? gs.s0 + kCWaves : -1;
  bool dry = gs.ctr < 0, asked = false;
  uint32_t grab = 0u;
  auto quad = [&](CRaw<NS>& R, int qb0, int it, int sbq) {  // sbq: first block of the quad within its group
    cstage_write(R, L);
    sched_fence();
    cstage_issue(R, S, gnxt * kCSB + sbq, gnxt >= 0);  // the same quad of the wave's next group
    sched_fence();
    cquad_weights(P, L, H, slot, sbq);
    lds_order();
    v4i acc[4];
#pragma unroll
    for (int mu = 0; mu < 4; ++mu) acc[mu] = *reinterpret_cast<const v4i*>(&L.ini[bq][nib][mu][0]);
    // every row group of the quad (pads and groups past the unit's are zero)
    uint32_t xr[Geo::G];
#pragma unroll
    for (int pp = 0; pp < Geo::G / 2; ++pp) {
      const v2i v = ctr_read(L, src_off, pp);
      xr[2 * pp] = (uint32_t)v.x;
      xr[2 * pp + 1] = (uint32_t)v.y;
    }
    if constexpr (Geo::Fine && NS == 5) {
      // slices outer: one slice's W and W_lo live at a time, the W chain of
      // each position kept apart and scaled by 128 into the W_lo chain
      v4i ah[4];
#pragma unroll
      for (int mu = 0; mu < 4; ++mu) ah[mu] = v4i{0, 0, 0, 0};
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) {
        const v4i w = *reinterpret_cast<const v4i*>(wsrc + 4 * s2);
        const v4i wlo = *reinterpret_cast<const v4i*>(wlsrc + 4 * s2);
#pragma unroll
        for (int mu = 0; mu < 4; ++mu) {
          const v4i bv = v4i{(int)(xr[4 * s2] & mk[mu]), (int)(xr[4 * s2 + 1] & mk[mu]), (int)(xr[4 * s2 + 2] & mk[mu]),
                             (int)(xr[4 * s2 + 3] & mk[mu])};
          ah[mu] = __builtin_amdgcn_mfma_i32_16x16x64_i8(w, bv, ah[mu], 0, 0, 0);
          acc[mu] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wlo, bv, acc[mu], 0, 0, 0);
        }
      }
#pragma unroll
      for (int mu = 0; mu < 4; ++mu) acc[mu] = acc[mu] + ah[mu] * 128;
    } else {
    v4i wv[NS];
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) wv[s2] = *reinterpret_cast<const v4i*>(wsrc + 4 * s2);
    if constexpr (Geo::Fine) {
      // key position outer, slices inner: the W chain of one position at a
      // time, scaled by 128 into the W_lo chain that started at the thresholds
      v4i wlv[NS];
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) wlv[s2] = *reinterpret_cast<const v4i*>(wlsrc + 4 * s2);
#pragma unroll
      for (int mu = 0; mu < 4; ++mu) {
        v4i ah = v4i{0, 0, 0, 0};
#pragma unroll
        for (int s2 = 0; s2 < NS; ++s2) {
          const v4i bv = v4i{(int)(xr[4 * s2] & mk[mu]), (int)(xr[4 * s2 + 1] & mk[mu]), (int)(xr[4 * s2 + 2] & mk[mu]),
                             (int)(xr[4 * s2 + 3] & mk[mu])};
          ah = __builtin_amdgcn_mfma_i32_16x16x64_i8(wv[s2], bv, ah, 0, 0, 0);
          acc[mu] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wlv[s2], bv, acc[mu], 0, 0, 0);
        }
        acc[mu] = acc[mu] + ah * 128;
      }
    } else {
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) {
        v4i bv[4];
#pragma unroll
        for (int mu = 0; mu < 4; ++mu)
          bv[mu] = v4i{(int)(xr[4 * s2] & mk[mu]), (int)(xr[4 * s2 + 1] & mk[mu]), (int)(xr[4 * s2 + 2] & mk[mu]),
                       (int)(xr[4 * s2 + 3] & mk[mu])};
#pragma unroll
        for (int mu = 0; mu < 4; ++mu) acc[mu] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wv[s2], bv[mu], acc[mu], 0, 0, 0);
      }
    }
    }
    // candidates: this lane's eligible keys (all four inside the window but
    // at the unit's edges), and per key its candidate heads
    const int blk = qb0 + bq;
    const int kbase = blk * kBlockTokens + kb;
    const bool inner = qb0 * kBlockTokens >= lo && (qb0 + 4) * kBlockTokens <= hi && qb0 + 4 <= nbu;
    uint32_t em = 0xFu;
    if (!inner) {
      const int e0 = min(max(lo - kbase, 0), 4), e1 = min(max(hi - kbase, 0), 4);
      em = blk < nbu ? (0xFu << e0) & ~(0xFu << e1) & 0xFu : 0u;
    }
    // byte h of D: bit mu set iff key mu is a candidate for head h (the sign
    // bytes of the four heads' accumulators side by side, flipped at pos 7)
    uint32_t D = 0u;
#pragma unroll
    for (int mu = 0; mu < 4; ++mu) {
      const uint32_t T = __builtin_amdgcn_perm((uint32_t)acc[mu][1], (uint32_t)acc[mu][0], 0x0c0c0703u) |
                         __builtin_amdgcn_perm((uint32_t)acc[mu][3], (uint32_t)acc[mu][2], 0x07030c0cu);
      // mu = 3 sits at pos 7 in nibble 1: its sign bytes flip
      const uint32_t flip = (uint32_t)(-(int)((threadIdx.x >> 3) & 1u));
      D |= ((mu == 3 ? T ^ flip : T) & 0x80808080u) >> (7 - mu);
    }
    D &= em * 0x01010101u;
    uint32_t kmask = (D | D >> 8 | D >> 16 | D >> 24) & 0xFu;
    const bool last = gnxt < 0 && sbq == kCSB - kQB;  // the wave's last quad
    const bool endg = sbq == kCSB - kQB;
    if (__ballot(kmask != 0u) != 0ull && pending == 0) oldest = it;
    const uint32_t meta = (uint32_t)slot << 3 | (uint32_t)(sbq + bq) << 8;
    while (true) {
      // every lane's lowest remaining key, as many as fit; re-score when the
      // queue is full and keys remain, or at the flush points
      const uint64_t want = __ballot(kmask != 0u);
      if (want != 0ull && pending < Geo::Q) {
        const int rank = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(want >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)want, 0u));
        const bool mine = kmask != 0u && rank < Geo::Q - pending;
        if (mine) {
          const int mu = __builtin_ctz(kmask);
          const int qp = pending + rank;
#pragma unroll
          for (int i = 0; i < Geo::G; ++i) L.qx[i][qp] = xr[i];
          L.qi[qp] = (uint32_t)(kbase + mu);
          L.qf[qp] = (uint32_t)(4 * nib + mu) | meta | ((D >> mu) & 0x01010101u) << 7;
          kmask &= kmask - 1u;
        }
        pending += __popcll(__ballot(mine));
        continue;
      }
      // entries of group it + 1 - Slots hold the ring slot rewritten next
      const bool flush = want != 0ull || pending >= Geo::Q ||
                         (pending > 0 && (last || (endg && oldest <= it + 1 - Geo::Slots)));
      if (!flush) break;
      lds_order();
      crescore(P, L, a, u, pending, svn);
      pending = 0;
      oldest = it;
      if (want == 0ull) break;
    }
    lds_order();
  };
  // one loop iteration = one group of 8 blocks (two quads): its scales and
  // delta, then the quads
  int gcur = any ? gs.s0 : -1;
  for (int it = 0; gcur >= 0; ++it) {
    slot = it % Geo::Slots;
    const int gb0 = gcur * kCSB;
    if (it > 0) {  // the group after this one: static, or the pool's answer
      if (asked) {
        const int g = gs.p0 + cuni((int)(threadIdx.x >> 6)) + kPools * cuni((int)grab);
        gnxt = g < gs.pend ? g : -1;
        dry = gnxt < 0;
      } else {
        gnxt = it + 1 < gs.ns ? gs.s0 + kCWaves * (it + 1) : -1;
      }
    }
    // ask the pool for the group after gnxt once the static groups run out
    asked = !dry && gnxt >= 0 && it + 2 >= gs.ns;
    // an increment, not an add: the compiler's atomic optimizer would turn a
    // single-lane add into a wave-aggregated one whose result is read at once
    // (a wait on every load in flight); the result is first read one group later
    if (asked && lane == 0)
      grab = __builtin_amdgcn_atomic_inc32((__attribute__((address_space(1))) uint32_t*)(a.ws.pool + gs.ctr), 0xFFFFFFFFu,
                                           __ATOMIC_RELAXED, "agent");
    sched_fence();
    {
      float qv[4];  // q of cell `lane`'s channel (read here: fewer registers live across the loop)
      {
        const float4 q4 = *reinterpret_cast<const float4*>(&P.qa[yl][0]);
        const bool on = lane < C;
        qv[0] = on ? q4.x : 0.0f; qv[1] = on ? q4.y : 0.0f; qv[2] = on ? q4.z : 0.0f; qv[3] = on ? q4.w : 0.0f;
      }
      float qv2[4] = {0.0f, 0.0f, 0.0f, 0.0f};  // cell 64 + lane's (NS = 5)
      int srow2 = 0;
      if constexpr (Geo::C > kWave) {
        const int x2 = cell2();
        srow2 = P.pj[x2];
        const float4 q4 = *reinterpret_cast<const float4*>(&P.qa[P.py[x2]][0]);
        const bool on = lane + kWave < C;
        qv2[0] = on ? q4.x : 0.0f; qv2[1] = on ? q4.y : 0.0f; qv2[2] = on ? q4.z : 0.0f; qv2[3] = on ? q4.w : 0.0f;
      }
      const CDel dl = cscl_commit(sr, L, slot, hq, qv, qv2);
      sched_fence();
      cscl_issue<VEC, NS>(sr, a, u, C, srow, srow2, gnxt * kCSB, gnxt >= 0);
      sched_fence();
      const float th = P.tau[hq];
      H.M0 = ldexpf(12582912.0f, dl.e);  // 1.5 * 2^(23 + e)
      H.K1 = ldexpf(12582912.0f * (1.0f + 0x1p-7f), dl.e);
      H.X = 0;
      const bool none = hq >= a.G || th == kNegInf;  // no key of this head is a candidate
      H.m0 = !none && dl.valid;
      if (H.m0) {
        const int eu = Geo::Fine ? dl.e - 7 : dl.e;  // the weights' unit: delta, or delta / 128
        const double E = ldexp(P.Kc, eu) + ldexp(P.Kch, dl.e) + P.Eabs;
        double X = ldexp((double)th - E, 1 - eu);  // 2 (tau - E) / unit
        X = floor(X) - 1.0;
        constexpr double xm = 2.0 * (Geo::Fine ? kCThrMax : kThrMax);
        X = X < -xm ? -xm : X > xm ? xm : X;
        H.X = (int)X;
      }
      // no thresholds: every key a candidate (no valid delta) or none
      H.c0 = none ? kNoBound : -kNoBound;
      H.c1 = top ? -H.c0 : H.c0;
    }
    quad(R0, gb0, it, 0);
    quad(R1, gb0 + kQB, it, kQB);
    gcur = gnxt;
  }
  const int none[4] = {0, 0, 0, 0};
  const uint64_t nocomp[4] = {0ull, 0ull, 0ull, 0ull};
  cappend(L, a, u, svn, none, 0u, nocomp, none);
}

// ---------------------------------------------------------------- tau
// Sec. 2 asks for the k largest scores; survivors are the keys whose exact
// score reaches tau, and the result never depends on tau as long as at least
// k keys survive (else the row is computed exactly).  tau of a row is about
// the m-th largest of its samples (the sample pass keeps the two largest
// exact scores of every block of a sampled quad), m = ceil(1.25 k sampled /
// eligible) + 16;
// when fewer samples exist the smallest one is used if about 1.1 k keys are
// expected above it, else tau = -inf (no filter).  Wave w of a workgroup
// finds tau of its unit's row w (w < G) from its lanes' 8 samples each: the
// largest 16-bit prefix of the order-preserving keys with at least m samples
// at or above it, by ballot counts, so tau rounds the m-th sample down to 7
// mantissa bits (a few more survivors, no other effect).
constexpr int kCTauPer = kSmpRow / kWave;

__device__ __forceinline__ float ctau(const FusedArgs& a, const float (&sv)[kCTauPer], int64_t lo, int64_t hi) {
  const int lane = threadIdx.x & 63;
  uint32_t key[kCTauPer];
  int nv = 0;
#pragma unroll
  for (int x = 0; x < kCTauPer; ++x) {
    key[x] = sv[x] > kNegInf ? score_key(sv[x]) | 1u : 0u;  // samples are never NaN; keep 0 free
    nv += __popcll(__ballot(key[x] != 0u));
  }
  // eligible keys in the sampled quads (a unit of this pass has fewer than
  // 2^26 keys and at most kSampleQuads sampled quads: 32-bit products)
  uint32_t m_s = 0u;
  for (int x = lane; x < a.ws.s_quads; x += kWave) {
    const int64_t k0 = x * a.ws.s_stride * kQB * kBlockTokens, k1 = k0 + kQB * kBlockTokens;
    const int64_t x0 = k0 > lo ? k0 : lo, x1 = k1 < hi ? k1 : hi;
    m_s += x1 > x0 ? (uint32_t)(x1 - x0) : 0u;
  }
  m_s = (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan_u(m_s), kWave - 1);
  const uint32_t m_e = (uint32_t)(hi - lo), kk = (uint32_t)a.k;
  uint32_t m = m_s > 0u ? (5u * kk * m_s + 4u * m_e - 1u) / (4u * m_e) + 16u : 0u;
  if (m > (uint32_t)nv) m = 10ull * (uint64_t)nv * m_e >= 11ull * kk * m_s ? (uint32_t)nv : 0u;
  if (m == 0u) return kNegInf;
  // the leading bits shared by the largest and the smallest sample are the
  // answer's too (m <= nv): the search starts below them
  uint32_t ext[4] = {0u, 0u, 0u, 0u};  // largest key, ~smallest (nonzero) key
#pragma unroll
  for (int x = 0; x < kCTauPer; ++x) {
    ext[0] = max(ext[0], key[x]);
    ext[1] = max(ext[1], key[x] != 0u ? ~key[x] : 0u);
  }
  wave_max4_u(ext);
  const uint32_t kmax = ext[0], kmin = ~ext[1];
  const int top = kmax == kmin ? -1 : 31 - __builtin_clz(kmax ^ kmin);  // highest differing bit
  uint32_t prefix = top < 16 ? kmax & 0xFFFF0000u : kmax & ~((2u << top) - 1u);
  for (int bit = top; bit >= 16; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    uint32_t c = 0u;
#pragma unroll
    for (int x = 0; x < kCTauPer; ++x) c += (uint32_t)__popcll(__ballot(key[x] >= cand));
    if (c >= m) prefix = cand;
  }
  // prefix has a nonzero bit (m <= nv samples lie at or above 2^16): the
  // smallest key of its range, as a float
  return __uint_as_float((prefix & 0x80000000u) ? (prefix & 0x7FFFFFFFu) : ~prefix);
}

// ---------------------------------------------------------------- kernel
// Grid (W U): workgroup b takes unit u = b mod U (a unit's workgroups are
// spread over the dispatch order, so over the workgroup slots of the CUs) as
// its x = b / U -th.  The unit's window holds NG groups; each wave takes S of
// them statically, 2/3 of an even share (the workgroup's 4 S groups are
// consecutive, its waves take them in turn), and the rest form the unit's
// pool.  With fewer than 2 static groups per wave every group is static.
// Units of another class (uovf[u] >> 1 != 1: the wide pass, or no filter) and
// rows computed exactly return at once.
// Three workgroups per CU: LDS is handed out in 1280-byte units, so a
// workgroup may hold at most 42 of them (a 53,984-byte build ran two per CU).
constexpr size_t kCLdsMax = 42 * 1280;
template <bool VEC, int NS>
__global__ __launch_bounds__(kCThreads, 3) void fused_filter_kernel(FusedArgs a, int U, int W) {
  static_assert(sizeof(CellPlan) + kCWaves * sizeof(FilterLds<NS>) <= kCLdsMax, "three workgroups per CU");
  __shared__ CellPlan P;
  __shared__ FilterLds<NS> WL[kCWaves];
  const int u = (int)(blockIdx.x % (unsigned)U), x = (int)(blockIdx.x / (unsigned)U);
  const int tid = threadIdx.x, wave = cuni(tid >> 6), lane = tid & 63, G = a.G;
  const uint32_t uo = gload(a.ws.uovf + u);
  // this wave's row's samples first: tau waits on them
  const int nsm = wave < G ? a.ws.s_quads * kSmpW : 0;
  float sv[kCTauPer];
#pragma unroll
  for (int i0 = 0; i0 < kCTauPer; ++i0) {
    const int i = lane + kWave * i0;
    sv[i0] = i < nsm ? gload(a.ws.samp + (int64_t)(u * G + wave) * kSmpRow + i) : kNegInf;
  }
  // the unit's plan (built by the sample pass), up to two 16-byte words per thread
  static_assert(kCThreads == kFT, "the plan's copy steps");
  PlanWord pw[kPlanSteps];
#pragma unroll
  for (int i = 0; i < kPlanSteps; ++i) {
    const int w = tid + kCThreads * i;
    pw[i] = w < kPlanWords ? gload(reinterpret_cast<const PlanWord*>(a.ws.plan + (size_t)u * kPlanBytes) + w)
                           : PlanWord{0u, 0u, 0u, 0u};
  }
  int64_t nu, lo, hi;
  row_window(a, u, &nu, &lo, &hi, x == 0 && tid == 0);
  if ((uo >> 1) != 1u) return;
  if (hi - lo <= a.ws.cap) return;
  const int64_t nbu = (nu + kBlockTokens - 1) / kBlockTokens;
  const int glo = (int)(lo / (kCSB * kBlockTokens));
  const int NG = (int)((hi + kCSB * kBlockTokens - 1) / (kCSB * kBlockTokens)) - glo;
  const int per = kCWaves * W;  // waves of the unit
  int S = (int)((int64_t)NG * 2 / (3 * per)), p0 = NG;
  if (S >= 2) p0 = S * per;
  else S = (NG + per - 1) / per;
  const int sb = x * kCWaves * S;  // the workgroup's first static group
  if (sb >= NG) return;
  // tau of this wave's row first: it needs only the samples and the window,
  // and runs while the plan's loads are in flight
  const float tv = wave < G ? ctau(a, sv, lo, hi) : kNegInf;
#pragma unroll
  for (int i = 0; i < kPlanSteps; ++i)
    if (tid + kCThreads * i < kPlanWords) reinterpret_cast<PlanWord*>(&P)[tid + kCThreads * i] = pw[i];
  __syncthreads();
  if (!P.ok || P.C > CGeo<NS>::C) return;  // more cells than the caller's bound allowed: the exact path
  CGroups gs;  // wave-uniform (read from memory, so held in scalar registers only through readfirstlane)
  const int rem = NG - sb - wave;
  gs.s0 = cuni(glo + sb + wave);
  gs.ns = cuni(rem > 0 ? min(S, (rem + kCWaves - 1) / kCWaves) : 0);
  gs.p0 = cuni(glo + p0);
  gs.pend = cuni(glo + NG);
  gs.ctr = cuni(p0 < NG ? (u * kPools + wave) * kPoolStride : -1);
  // every workgroup finds the same tau; the first of the unit leaves it for
  // the select pass
  auto ready = [&]() -> bool {
    if (wave < G) {
      if (lane == 0) {
        P.tau[wave] = tv;
        if (x == 0) gstore(a.ws.tau + u * G + wave, tv);
      }
    }
    __syncthreads();
    bool any = false;
    for (int h = 0; h < G; ++h) any |= P.tau[h] != kNegInf;
    return any;
  };
  cwave_run<VEC, NS>(P, WL[wave], a, u, gs, (int)nbu, (int)lo, (int)hi, ready);
}

// Workgroups per unit: about kFResident of them over all units (three per
// CU, one round), and no more than one group per wave.
constexpr int64_t kFResident = 3 * 256;
void launch_filter(const FusedArgs& fa, int U, int max_cells, hipStream_t s) {
  const int64_t ngr = (fa.nb_cap + kCSB - 1) / kCSB;
  int64_t W = kFResident / U;
  const int64_t wmax = (ngr + kCWaves - 1) / kCWaves;
  if (W > wmax) W = wmax;
  if (W < 1) W = 1;
  const dim3 grid((unsigned)(W * U));
  // 16-byte aligned scale rows: one 16-byte scale load per lane and group
  const bool vec = (fa.nb_cap & 7) == 0 && (reinterpret_cast<uintptr_t>(fa.scales) & 15) == 0;
  // three slices when no unit can have more than 48 cells, five when units
  // of up to 80 cells take the filter (fa.ccap), else four
  if (max_cells > 0 && max_cells <= CGeo<3>::C) {
    if (vec) hipLaunchKernelGGL((fused_filter_kernel<true, 3>), grid, dim3(kCThreads), 0, s, fa, U, (int)W);
    else hipLaunchKernelGGL((fused_filter_kernel<false, 3>), grid, dim3(kCThreads), 0, s, fa, U, (int)W);
  } else if (fa.ccap > CGeo<4>::C) {
    if (vec) hipLaunchKernelGGL((fused_filter_kernel<true, 5>), grid, dim3(kCThreads), 0, s, fa, U, (int)W);
    else hipLaunchKernelGGL((fused_filter_kernel<false, 5>), grid, dim3(kCThreads), 0, s, fa, U, (int)W);
  } else {
    if (vec) hipLaunchKernelGGL((fused_filter_kernel<true, 4>), grid, dim3(kCThreads), 0, s, fa, U, (int)W);
    else hipLaunchKernelGGL((fused_filter_kernel<false, 4>), grid, dim3(kCThreads), 0, s, fa, U, (int)W);
  }
}

}  // namespace fathom
