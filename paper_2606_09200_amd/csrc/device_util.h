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

// Per-launch hooks every kernel runs at its start (hooks_begin) and end
// (hooks_end).  All fields zero / null = off.
//
// Tracing.  `stamps` is a [first start, last end] pair (atomic min / max over
// workgroups); `wg` receives one 48-byte record per workgroup: {tag, block,
// HW_ID, XCC_ID, t0 lo, t0 hi, t1 lo, t1 hi, cycles lo, cycles hi, 0, 0},
// appended at wg[4 + 12*i] with i taken from the counter wg[0] (records past
// `wg_cap` are dropped).  HW_ID holds the wave's SIMD [5:4], CU [11:8],
// SH [12] and SE [15:13]; XCC_ID [3:0] is the XCD; cycles counts
// engine-clock cycles between t0 and t1.  All accesses are vector atomics or
// vector stores to the caller's buffer.
//
// Dependency counter (the per-iteration K_g^i -> K_c^i edge kept on the
// device).  A producer launch sets `signal`: each of its workgroups adds one
// to *signal once all its threads are done (with `release`, after their
// stores are made visible at device scope).  A consumer launch sets `wait`:
// before anything else, thread 0 of each workgroup waits until *wait reaches
// `wait_target` (the producer's workgroup count), at most kDepWaitTicks,
// then (with `acquire`) makes the producer's stores visible to the
// workgroup, and adds one to *ack; the workgroup that brings *ack to
// `ack_target` (the consumer's workgroup count over all its kernels) puts
// *wait and *ack back to zero, which no other workgroup of the consumer reads
// any more.  A wait that runs out sets *err and lets the workgroup go on, so
// every kernel ends.
struct KHooks {
  uint64_t *stamps = nullptr;
  uint32_t *wg = nullptr;
  uint32_t wg_cap = 0;
  uint32_t tag = 0;
  uint32_t *signal = nullptr;
  uint32_t *wait = nullptr;
  uint32_t *ack = nullptr;
  uint32_t *err = nullptr;
  uint32_t wait_target = 0;
  uint32_t ack_target = 0;
  uint32_t release = 0;
  uint32_t acquire = 0;
};

constexpr int kWgRecordWords = 12;
// Longest a consumer workgroup waits for its producer: 2 s of the 100 MHz
// constant-rate clock.
constexpr uint64_t kDepWaitTicks = 200000000ull;

struct HookStart {
  uint64_t ticks;
  uint64_t cycles;
};

__device__ __forceinline__ void dep_wait(const KHooks &t) {
  if (threadIdx.x == 0) {
    const uint64_t t0 = now_ticks();
    bool late = false;
    // poll every ~128 cycles for the first 5 us (launch-bound schedules),
    // then every ~2000 cycles: a long wait (its GEMM takes milliseconds)
    // then puts little load on the memory system the GEMM is using
    while (__hip_atomic_load(t.wait, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < t.wait_target) {
      const uint64_t waited = now_ticks() - t0;
      if (waited > kDepWaitTicks) {
        late = true;
        break;
      }
      if (waited < 500) __builtin_amdgcn_s_sleep(2);
      else __builtin_amdgcn_s_sleep(32);
    }
    if (late) __hip_atomic_store(t.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (t.acquire) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    if (__hip_atomic_fetch_add(t.ack, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u == t.ack_target) {
      __hip_atomic_store(t.ack, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(t.wait, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
}

__device__ __forceinline__ HookStart hooks_begin(const KHooks &t) {
  if (t.wait != nullptr) dep_wait(t);
  HookStart s{0, 0};
  if (threadIdx.x == 0 && (t.stamps != nullptr || t.wg != nullptr)) {
    s.ticks = now_ticks();
    s.cycles = now_cycles();
    if (t.stamps != nullptr)
      atomicMin(reinterpret_cast<unsigned long long *>(t.stamps), (unsigned long long)s.ticks);
  }
  return s;
}

// End of a workgroup: its trace record, then (producer) the dependency
// count, so a consumer never starts before the recorded end.  With
// `release`, every wave's stores are complete and visible at device scope
// before the workgroup counts itself done.
__device__ __forceinline__ void hooks_end(const KHooks &t, const HookStart &s) {
  const bool trace = t.stamps != nullptr || t.wg != nullptr;
  if (t.signal == nullptr && !trace) return;
  if (t.signal != nullptr && t.release) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x != 0) return;
  if (trace) {
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
  if (t.signal != nullptr) __hip_atomic_fetch_add(t.signal, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
