// Device-side helpers shared by the library's kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace occ {

// GPU constant-rate clock (100 MHz on CDNA: 10 ns per tick).
__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

// Optional per-launch tracing.  `stamps` is a [first start, last end] pair
// (atomic min / max over workgroups); `wg` receives one 32-byte record per
// workgroup: {tag, block, HW_ID, XCC_ID} then {t0 lo, t0 hi, t1 lo, t1 hi},
// appended at wg[4 + 8*i] with i taken from the counter wg[0] (records past
// `wg_cap` are dropped).  HW_ID holds the wave's SIMD [5:4], CU [11:8], SH [12]
// and SE [15:13]; XCC_ID [3:0] is the XCD.  All accesses are vector atomics or
// vector stores to the caller's buffer.
struct KTrace {
  uint64_t *stamps;
  uint32_t *wg;
  uint32_t wg_cap;
  uint32_t tag;
};

__device__ __forceinline__ uint64_t trace_begin(const KTrace &t) {
  uint64_t t0 = 0;
  if (threadIdx.x == 0 && (t.stamps != nullptr || t.wg != nullptr)) {
    t0 = now_ticks();
    if (t.stamps != nullptr)
      atomicMin(reinterpret_cast<unsigned long long *>(t.stamps), (unsigned long long)t0);
  }
  return t0;
}

__device__ __forceinline__ void trace_end(const KTrace &t, uint64_t t0) {
  if (t.stamps == nullptr && t.wg == nullptr) return;
  __syncthreads();
  if (threadIdx.x != 0) return;
  uint64_t t1 = now_ticks();
  if (t.stamps != nullptr)
    atomicMax(reinterpret_cast<unsigned long long *>(t.stamps + 1), (unsigned long long)t1);
  if (t.wg != nullptr) {
    uint32_t i = atomicAdd(t.wg, 1u);
    if (i < t.wg_cap) {
      uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);    // HW_REG_HW_ID, 32 bits
      uint32_t xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20);  // HW_REG_XCC_ID, 32 bits
      uint32_t *r = t.wg + 4 + 8 * (size_t)i;
      r[0] = t.tag;
      r[1] = blockIdx.x;
      r[2] = hw;
      r[3] = xcc;
      r[4] = (uint32_t)t0;
      r[5] = (uint32_t)(t0 >> 32);
      r[6] = (uint32_t)t1;
      r[7] = (uint32_t)(t1 >> 32);
    }
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
