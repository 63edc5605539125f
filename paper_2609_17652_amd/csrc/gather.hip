// fathom_gather_store: the host-resident store of Sec. 3.6 -- the planes and
// scales stay in pinned host memory and, per decode step, only what the
// allocated depths read crosses the host link into an HBM staging store.
//
// With the layout [U][D][4][nb_cap], the first t planes of channel j are one
// contiguous run of t * nb_cap words, and its scales one run of nb_cap halves:
// one workgroup per (unit, channel) copies the two runs (nothing for t = 0)
// with 16-byte reads of the host memory mapped into the device address space.
#include "common.hpp"

namespace fathom {

constexpr int kGatherThreads = 256;

// bytes [0, nbytes) from src to dst: bytes up to the first 16-byte boundary
// (when both pointers share their offset within 16 bytes, else all bytes),
// then 16-byte words, then the tail bytes
__device__ __forceinline__ void copy_run(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, int64_t nbytes) {
  const uint32_t ms = (uint32_t)reinterpret_cast<uintptr_t>(src) & 15u;
  const uint32_t md = (uint32_t)reinterpret_cast<uintptr_t>(dst) & 15u;
  int64_t head = 0;
  if (ms != md) head = nbytes;
  else if (ms != 0) head = nbytes < (int64_t)(16u - ms) ? nbytes : (int64_t)(16u - ms);
  for (int64_t i = threadIdx.x; i < head; i += kGatherThreads) dst[i] = src[i];
  const int64_t n16 = (nbytes - head) >> 4;
  const uint4* s4 = reinterpret_cast<const uint4*>(src + head);
  uint4* d4 = reinterpret_cast<uint4*>(dst + head);
  for (int64_t i = threadIdx.x; i < n16; i += kGatherThreads) d4[i] = s4[i];
  for (int64_t i = head + (n16 << 4) + threadIdx.x; i < nbytes; i += kGatherThreads) dst[i] = src[i];
}

__global__ __launch_bounds__(kGatherThreads) void gather_kernel(const uint64_t* __restrict__ hplanes,
                                                               const uint16_t* __restrict__ hscales,
                                                               const uint8_t* __restrict__ depths, int64_t nb_cap,
                                                               uint64_t* __restrict__ planes,
                                                               uint16_t* __restrict__ scales) {
  const int j = blockIdx.x, u = blockIdx.y;
  int t = depths[(int64_t)u * kD + j];
  t = t > kPlanes ? kPlanes : t;
  if (t == 0) return;
  const int64_t row = (int64_t)u * kD + j;
  copy_run(reinterpret_cast<const uint8_t*>(hplanes + row * kPlanes * nb_cap),
           reinterpret_cast<uint8_t*>(planes + row * kPlanes * nb_cap), (int64_t)t * nb_cap * 8);
  copy_run(reinterpret_cast<const uint8_t*>(hscales + row * nb_cap), reinterpret_cast<uint8_t*>(scales + row * nb_cap),
           nb_cap * 2);
}

fathom_status launch_gather(const uint64_t* hplanes, const uint16_t* hscales, const uint8_t* depths, int U,
                            int64_t nb_cap, uint64_t* planes, uint16_t* scales, hipStream_t s) {
  if (U == 0 || nb_cap == 0) return FATHOM_OK;
  void* dp = nullptr;
  void* ds = nullptr;
  // pinned host memory only: anything else fails here, before a launch (the
  // runtime's error is cleared so that it is not reported by a later call)
  if (hipHostGetDevicePointer(&dp, const_cast<uint64_t*>(hplanes), 0) != hipSuccess || !dp ||
      hipHostGetDevicePointer(&ds, const_cast<uint16_t*>(hscales), 0) != hipSuccess || !ds) {
    (void)hipGetLastError();
    return FATHOM_ERR_INVALID;
  }
  hipLaunchKernelGGL(gather_kernel, dim3(kD, U), dim3(kGatherThreads), 0, s, static_cast<const uint64_t*>(dp),
                     static_cast<const uint16_t*>(ds), depths, nb_cap, planes, scales);
  FATHOM_LAUNCH_CHECK();
  return FATHOM_OK;
}

}  // namespace fathom
