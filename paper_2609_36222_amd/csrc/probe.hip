// Streaming-read probe: the HBM read rate a kernel reaches on this part, as
// the achievable ceiling the FFN's weight stream is compared with.  Not part
// of the method's ABI (include/base.h); bench.py loads it from its own
// library.
//
// Each wavefront reads one contiguous share of the buffer in 4 KiB steps
// (lane l: four 16-byte pieces at 1 KiB apart, the FFN's load shape), four
// steps ahead of their use, and folds the data into one value that is
// written only if it equals a constant no input produces.  Wavefront b
// reads share b % shares: with fewer shares than wavefronts the same bytes
// are read several times, which measures the rate from a working set of
// shares x steps x 4 KiB (L2-, Infinity-Cache- or HBM-resident).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int PD = 4;   // steps in flight

__device__ __forceinline__ u32x4 ld(rsrc_t r, uint32_t v, uint32_t s) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)v, (int)s, 0));
}

__global__ __launch_bounds__(64) void k_stream_read(const uint8_t *buf, uint32_t steps,
                                                    uint32_t shares, uint32_t *sink) {
  const uint32_t bytes = steps * 4096u;
  rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t *>(buf + (size_t)(blockIdx.x % shares) * bytes), 0, (int)bytes,
      0x00020000);
  const uint32_t vo = threadIdx.x * 16u;
  u32x4 b[PD][4], acc = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int p = 0; p < PD; ++p)
#pragma unroll
    for (int t = 0; t < 4; ++t) b[p][t] = ld(r, vo + t * 1024u, (uint32_t)p * 4096u);
  for (uint32_t k = 0; k < steps; k += PD) {
#pragma unroll
    for (int p = 0; p < PD; ++p) {
#pragma unroll
      for (int t = 0; t < 4; ++t) acc ^= b[p][t];
      // past the share's end: out of the resource, zero without a memory access
#pragma unroll
      for (int t = 0; t < 4; ++t) b[p][t] = ld(r, vo + t * 1024u, (k + PD + p) * 4096u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9E3779B9u) sink[0] = 1u;
}

}  // namespace

extern "C" {

// Reads waves * steps * 4 KiB bytes from buf (device, 16-byte aligned), one
// wavefront per share of steps * 4 KiB; wavefront b reads share b % shares
// (shares = 0: waves shares, every byte once), so buf must hold
// min(shares, waves) * steps * 4 KiB bytes.  steps: a multiple of 4; below
// 2^19 (a share under 2 GiB).  sink: one device word.
// start / stop: optional events the dispatch itself records as the kernel
// begins and ends (null: none).  Returns hipErrorInvalidValue for a bad
// argument (nothing launched), else the hipError_t of the launch.
int base_probe_stream_read(const void *buf, uint32_t waves, uint32_t steps, uint32_t shares,
                           void *sink, void *start, void *stop, void *stream) {
  if (!buf || !sink || waves == 0 || steps == 0 || steps % PD || steps >= (1u << 19))
    return (int)hipErrorInvalidValue;
  if (shares == 0 || shares > waves) shares = waves;
  hipExtLaunchKernelGGL(k_stream_read, dim3(waves), dim3(64), 0, (hipStream_t)stream,
                        (hipEvent_t)start, (hipEvent_t)stop, 0, (const uint8_t *)buf, steps,
                        shares, (uint32_t *)sink);
  return (int)hipGetLastError();
}

}  // extern "C"
