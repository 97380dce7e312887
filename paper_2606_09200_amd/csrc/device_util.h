// Device-side helpers shared by the library's kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace occ {

// GPU constant-rate clock (100 MHz on CDNA: 10 ns per tick).
__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

// Kernel timeline: the first workgroup to start lowers stamps[0], the last to
// finish raises stamps[1].  Vector atomics on a caller-provided buffer.
__device__ __forceinline__ void stamp_begin(uint64_t *stamps) {
  if (stamps != nullptr && threadIdx.x == 0)
    atomicMin(reinterpret_cast<unsigned long long *>(stamps), (unsigned long long)now_ticks());
}
__device__ __forceinline__ void stamp_end(uint64_t *stamps) {
  if (stamps != nullptr) {
    __syncthreads();
    if (threadIdx.x == 0)
      atomicMax(reinterpret_cast<unsigned long long *>(stamps + 1), (unsigned long long)now_ticks());
  }
}

// Wave issue priority (s_setprio takes an immediate).
__device__ __forceinline__ void set_wave_priority(int p) {
  switch (p) {
    case 1: __builtin_amdgcn_s_setprio(1); break;
    case 2: __builtin_amdgcn_s_setprio(2); break;
    case 3: __builtin_amdgcn_s_setprio(3); break;
    default: break;
  }
}

}  // namespace occ
