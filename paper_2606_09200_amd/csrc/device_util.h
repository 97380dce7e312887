// Device-side helpers shared by the library's kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace occ {

// GPU constant-rate clock (100 MHz on CDNA: 10 ns per tick).
__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

// Shader-clock cycle counter (runs at the engine clock, so cycles / ticks
// over one workgroup's life is the clock it ran at).
__device__ __forceinline__ uint64_t now_cycles() { return __builtin_amdgcn_s_memtime(); }

// Optional per-launch tracing.  `stamps` is a [first start, last end] pair
// (atomic min / max over workgroups); `wg` receives one 48-byte record per
// workgroup: {tag, block, HW_ID, XCC_ID, t0 lo, t0 hi, t1 lo, t1 hi,
// cycles lo, cycles hi, 0, 0}, appended at wg[4 + 12*i] with i taken from the
// counter wg[0] (records past `wg_cap` are dropped).  HW_ID holds the wave's
// SIMD [5:4], CU [11:8], SH [12] and SE [15:13]; XCC_ID [3:0] is the XCD;
// cycles counts engine-clock cycles between t0 and t1.  All accesses are
// vector atomics or vector stores to the caller's buffer.
struct KTrace {
  uint64_t *stamps;
  uint32_t *wg;
  uint32_t wg_cap;
  uint32_t tag;
};

constexpr int kWgRecordWords = 12;

struct TraceStart {
  uint64_t ticks;
  uint64_t cycles;
};

__device__ __forceinline__ TraceStart trace_begin(const KTrace &t) {
  TraceStart s{0, 0};
  if (threadIdx.x == 0 && (t.stamps != nullptr || t.wg != nullptr)) {
    s.ticks = now_ticks();
    s.cycles = now_cycles();
    if (t.stamps != nullptr)
      atomicMin(reinterpret_cast<unsigned long long *>(t.stamps), (unsigned long long)s.ticks);
  }
  return s;
}

__device__ __forceinline__ void trace_end(const KTrace &t, const TraceStart &s) {
  if (t.stamps == nullptr && t.wg == nullptr) return;
  __syncthreads();
  if (threadIdx.x != 0) return;
  const uint64_t c1 = now_cycles();
  const uint64_t t1 = now_ticks();
  if (t.stamps != nullptr)
    atomicMax(reinterpret_cast<unsigned long long *>(t.stamps + 1), (unsigned long long)t1);
  if (t.wg != nullptr) {
    uint32_t i = atomicAdd(t.wg, 1u);
    if (i < t.wg_cap) {
      uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);    // HW_REG_HW_ID, 32 bits
      uint32_t xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20);  // HW_REG_XCC_ID, 32 bits
      const uint64_t cyc = c1 - s.cycles;
      uint32_t *r = t.wg + 4 + (size_t)kWgRecordWords * i;
      r[0] = t.tag;
      r[1] = blockIdx.x;
      r[2] = hw;
      r[3] = xcc;
      r[4] = (uint32_t)s.ticks;
      r[5] = (uint32_t)(s.ticks >> 32);
      r[6] = (uint32_t)t1;
      r[7] = (uint32_t)(t1 >> 32);
      r[8] = (uint32_t)cyc;
      r[9] = (uint32_t)(cyc >> 32);
      r[10] = 0;
      r[11] = 0;
    }
  }
}

// Bandwidth pacing of a streaming loop: with a period of P ticks, trip j of a
// wave starts no earlier than P ticks after trip j-1 started (a wave that
// falls behind does not burst to catch up).  P = 0 disables it.  The wait is
// a scalar loop on the monotonic constant-rate clock, so it always ends.
struct Pacer {
  uint64_t next;
  uint32_t period;
};

__device__ __forceinline__ Pacer pace_start(uint32_t period) {
  return Pacer{period ? now_ticks() + period : 0ull, period};
}

__device__ __forceinline__ void pace_wait(Pacer &p) {
  if (p.period == 0) return;
  uint64_t t = now_ticks();
  while (t < p.next) {
    __builtin_amdgcn_s_sleep(2);
    t = now_ticks();
  }
  p.next = t + p.period;
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
