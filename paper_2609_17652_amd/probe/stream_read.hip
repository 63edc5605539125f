// Streaming-read reference for the bench (not part of libfathom): reads a
// device buffer once with 16-byte loads and reduces it, so that its time is
// the HBM read rate this GPU sustains for a plain coalesced stream.  The
// bench reports the scan's bytes per second against this rate beside the
// published peak.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;
constexpr int kUnroll = 8;  // independent 16-byte loads in flight per thread

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* __restrict__ p, int64_t n16,
                                                               uint32_t* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  uint32_t acc = 0u;
  for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int r = 0; r < kUnroll; ++r) v[r] = __builtin_nontemporal_load(p + i + r * stride);
#pragma unroll
    for (int r = 0; r < kUnroll; ++r) acc ^= v[r].x ^ v[r].y ^ v[r].z ^ v[r].w;
  }
  for (; i < n16; i += stride) {
    const u32x4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  // one word per workgroup keeps the loads live
  __shared__ uint32_t red[kThreads / 64];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc ^= __shfl_xor(acc, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

}  // namespace

extern "C" {

// Workgroups the kernel uses (the size of `out` in words).
int probe_stream_read_groups(void) { return 2048; }

// Reads n16 16-byte words at p (device, 16-byte aligned) on `stream`;
// out (device) receives probe_stream_read_groups() words.  0 on success.
int probe_stream_read(const void* p, int64_t n16, uint32_t* out, void* stream) {
  if (!p || !out || n16 < 0 || (reinterpret_cast<uintptr_t>(p) & 15)) return -1;
  hipLaunchKernelGGL(stream_read_kernel, dim3(2048), dim3(kThreads), 0, reinterpret_cast<hipStream_t>(stream),
                     reinterpret_cast<const u32x4*>(p), n16, out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
