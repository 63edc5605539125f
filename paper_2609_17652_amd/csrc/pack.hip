// fathom_pack: Sec. 3.2, Eq. (2) -- per-channel 4-bit quantisation with fp16
// block scales, written channel-major as bit planes.
//
// One workgroup (4 waves) packs kBlocksPerWG consecutive 64-token blocks of one
// unit for all 128 channels.  Per block, the 64 x 128 key tile is read with
// coalesced 16-byte loads into LDS (row pitch 129 floats: column reads are
// bank-conflict free); then lane i of a wave holds token i of one channel at a
// time, the wave max gives the block absmax, four compares against exact
// multiples of the cell width give the code, and four ballots give the plane
// words (ballot bit i = lane i = token 64b + i).  Words and scales collect in
// LDS and leave as contiguous runs of kBlocksPerWG words per (channel, plane).
//
// Append (n_old given): a block's fp16 scale depends on every token in it, so
// a unit growing from n_old to n tokens re-packs blocks floor(n_old/64) ..
// ceil(n/64)-1 from the keys (the last partial block together with the new
// tokens); the grid then covers at most max_blocks blocks per unit, and the
// 128 channels are split over kAppendGroups workgroups (blockIdx.z): an
// append packs few blocks, so its time is one workgroup's channel loop.
#include "common.hpp"

namespace fathom {

constexpr int kPackThreads = 256;
constexpr int kBlocksPerWG = 4;
constexpr int kTilePitch = kD + 1;
constexpr int kAppendGroups = 16;

template <typename KT>
__global__ __launch_bounds__(kPackThreads) void pack_kernel(const KT* __restrict__ K, int64_t ld_tok,
                                                           int64_t ld_unit, const int64_t* __restrict__ n,
                                                           const int64_t* __restrict__ n_old, int64_t max_blocks,
                                                           int64_t nb_cap, uint64_t* __restrict__ planes,
                                                           uint16_t* __restrict__ scales,
                                                           uint32_t* __restrict__ st) {
  __shared__ float tile[kBlockTokens * kTilePitch];
  __shared__ uint64_t outw[kD * kPlanes * kBlocksPerWG];
  __shared__ uint16_t outs[kD * kBlocksPerWG];

  const int u = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // channels [c0, c0 + cpw * 4) of this workgroup, cpw per wave
  const int ngr = (int)gridDim.z, cpw = 32 / ngr, c0 = (int)blockIdx.z * (kD / ngr);
  const int64_t nu = unit_tokens(n, u, nb_cap * kBlockTokens, tid == 0 ? st : nullptr);
  // blocks [bs, be) of this unit are written: all of them, or (append) the
  // ones from the first block holding a new token
  int64_t bs = 0, be = nb_cap;
  if (n_old) {
    const int64_t no = n_old[u];
    if (no < 0 || no > nu || (nu + kBlockTokens - 1) / kBlockTokens - no / kBlockTokens > max_blocks) {
      if (tid == 0) set_status(st, FATHOM_DEV_BAD_N);
      return;  // the unit is left as it was
    }
    bs = no / kBlockTokens;
    be = (nu + kBlockTokens - 1) / kBlockTokens;
  }
  const int64_t b0 = bs + (int64_t)blockIdx.x * kBlocksPerWG;
  if (b0 >= be) return;
  const KT* Ku = K + (int64_t)u * ld_unit;
  uint32_t flags = 0;

  for (int bb = 0; bb < kBlocksPerWG; ++bb) {
    const int64_t b = b0 + bb;
    if (b >= be) break;
    const int64_t tok0 = b * kBlockTokens;
    // ---- stage the 64 x 128 tile (invalid rows as zeros) ----
    if constexpr (sizeof(KT) == 4) {
      const int c4 = tid & 31;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int row = (tid >> 5) + 8 * r;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (tok0 + row < nu) v = *reinterpret_cast<const float4*>(Ku + (tok0 + row) * ld_tok + 4 * c4);
        float* t = &tile[row * kTilePitch + 4 * c4];
        t[0] = v.x; t[1] = v.y; t[2] = v.z; t[3] = v.w;
      }
    } else {
      const int c8 = tid & 15;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = (tid >> 4) + 16 * r;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (tok0 + row < nu) v = *reinterpret_cast<const uint4*>(Ku + (tok0 + row) * ld_tok + 8 * c8);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        float* t = &tile[row * kTilePitch + 8 * c8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          t[2 * e] = half_bits_to_float((uint16_t)(w[e] & 0xFFFFu));
          t[2 * e + 1] = half_bits_to_float((uint16_t)(w[e] >> 16));
        }
      }
    }
    __syncthreads();
    // ---- quantise: wave w owns channels 32w .. 32w+31, lane = token ----
    const bool valid = tok0 + lane < nu;
    for (int jj = 0; jj < cpw; ++jj) {
      const int j = c0 + wave * cpw + jj;
      const float v = tile[lane * kTilePitch + j];
      const bool isn = v != v;
      if (valid && !(fabsf(v) <= 3.402823466e38f)) flags |= FATHOM_DEV_NONFINITE;
      const float av = (valid && !isn) ? fabsf(v) : 0.0f;
      const float a = wave_max(av);
      const __half a16h = __float2half_rn(a);
      const uint16_t a16 = __half_as_ushort(a16h);
      const bool overflow = (a16 & 0x7FFFu) == 0x7C00u;
      const float s = __fmul_rn(__half2float(a16h), 0.125f);  // exact
      int c = 8;
      if (a16 != 0 && !overflow && !isn) {
        // c = clip(floor(v / s), -8, 7) + 8 by binary search on exact
        // thresholds T*s, T integer in [-7, 7] (T*s has <= 14 significant bits)
        c = 0;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int step = 8 >> p;
          const float thr = __fmul_rn((float)(c + step - 8), s);
          if (v >= thr) c += step;
        }
      }
      if (overflow) flags |= FATHOM_DEV_SCALE_OVERFLOW;
      const uint64_t w0 = __ballot(valid && (c & 8));
      const uint64_t w1 = __ballot(valid && (c & 4));
      const uint64_t w2 = __ballot(valid && (c & 2));
      const uint64_t w3 = __ballot(valid && (c & 1));
      if (lane < 4) {
        const uint64_t w = lane == 0 ? w0 : lane == 1 ? w1 : lane == 2 ? w2 : w3;
        outw[(j * kPlanes + lane) * kBlocksPerWG + bb] = w;
      } else if (lane == 4) {
        outs[j * kBlocksPerWG + bb] = a16;
      }
    }
    __syncthreads();
  }
  // ---- contiguous runs of kBlocksPerWG words per (channel, plane) ----
  const int64_t nbw = be - b0 < kBlocksPerWG ? be - b0 : kBlocksPerWG;
  uint64_t* Pu = planes + (int64_t)u * kD * kPlanes * nb_cap;
  const int wc = kD / ngr;  // channels of this workgroup
  for (int w = c0 * kPlanes * kBlocksPerWG + tid; w < (c0 + wc) * kPlanes * kBlocksPerWG; w += kPackThreads) {
    const int row = w / kBlocksPerWG, e = w % kBlocksPerWG;
    if (e < nbw) Pu[(int64_t)row * nb_cap + b0 + e] = outw[w];
  }
  uint16_t* Su = scales + (int64_t)u * kD * nb_cap;
  for (int w = c0 * kBlocksPerWG + tid; w < (c0 + wc) * kBlocksPerWG; w += kPackThreads) {
    const int row = w / kBlocksPerWG, e = w % kBlocksPerWG;
    if (e < nbw) Su[(int64_t)row * nb_cap + b0 + e] = outs[w];
  }
  // one status update per wave
  const uint64_t any = __ballot(flags != 0);
  if (any) {
    uint32_t f = flags;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) f |= __shfl_xor(f, m, kWave);
    if (lane == 0) set_status(st, f);
  }
}

fathom_status launch_pack(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                          const int64_t* n, const int64_t* n_old, int64_t max_new, int U, int64_t nb_cap,
                          uint64_t* planes, uint16_t* scales, uint32_t* st, hipStream_t s) {
  if (U == 0 || nb_cap == 0) return FATHOM_OK;
  // append: new tokens span at most ceil(max_new / 64) + 1 blocks per unit
  int64_t mb = nb_cap;
  if (n_old) {
    mb = (max_new + kBlockTokens - 1) / kBlockTokens + 1;
    if (mb > nb_cap) mb = nb_cap;
  }
  dim3 grid((unsigned)((mb + kBlocksPerWG - 1) / kBlocksPerWG), (unsigned)U, n_old ? kAppendGroups : 1);
  if (kdt == FATHOM_F32)
    hipLaunchKernelGGL(pack_kernel<float>, grid, dim3(kPackThreads), 0, s,
                       reinterpret_cast<const float*>(K), ld_tok, ld_unit, n, n_old, mb, nb_cap, planes, scales, st);
  else
    hipLaunchKernelGGL(pack_kernel<__half>, grid, dim3(kPackThreads), 0, s,
                       reinterpret_cast<const __half*>(K), ld_tok, ld_unit, n, n_old, mb, nb_cap, planes, scales, st);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

}  // namespace fathom
