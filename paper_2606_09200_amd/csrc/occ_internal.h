// Internal interfaces of the occ library (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/occ.h"
#include "device_util.h"

namespace occ {

constexpr int kMaxReduceChunks = 64;
constexpr int kMaxPermuteChunks = 512;

// Per-device facts the launch plans depend on (queried once per device).
struct DeviceInfo {
  int ok;
  int num_cus;
  int lds_per_cu;       // bytes
  int max_lds_per_wg;   // bytes
  int clock_khz;
  int gfx950;
};
const DeviceInfo &device_info(int device);
int current_device_info(const DeviceInfo **out);

// ---- GEMM ----------------------------------------------------------------
struct GemmCall {
  const void *A;
  const void *B;
  void *C;
  int M, N, K;
  size_t lds_bytes;
  int grid_cap;         // 0 = one workgroup per tile
  int variant;          // 0 = automatic, else a kernel variant id
  int priority;         // wave priority 0..3 (s_setprio)
  KHooks trace;         // per-launch hooks: tracing, dependency counter (all off by default)
  bool b_kn = false;    // B stored K x N (occ_gemm: C = A B) or N x K (occ_gemm_bt: C = A B^T)
};
int gemm_plan(const GemmCall &c, occ_gemm_plan *plan);
// the plan without the occupancy figure (wg_per_cu = 0): no runtime query
int gemm_launch_plan(const GemmCall &c, occ_gemm_plan *plan);
bool gemm_variant_is_kn(int id);  // a variant that takes B stored K x N
int gemm_launch(const GemmCall &c, hipStream_t s);

// ---- communication-side kernels -----------------------------------------
struct ReduceCall {
  const float *const *bufs;  // host array
  int nchunks;
  size_t len;
  float *out;
  int wgs;                   // 0 = default
  int priority;              // 0..3
  KHooks trace;
  double rate_gbs;           // target bandwidth of the vector path, GB/s; 0 = unpaced
  // when set: the first term of every sum is this bf16 buffer, widened to
  // binary32, and bufs holds the nchunks (>= 0) fp32 terms after it
  const uint16_t *own = nullptr;
};
int reduce_launch(const ReduceCall &c, hipStream_t s);
int reduce_default_wgs(const ReduceCall &c);

struct PermuteCall {
  const void *src;
  void *dst;
  const int32_t *perm;       // host array
  int nchunks;
  size_t chunk_bytes;
  int wgs;
  int priority;
  KHooks trace;
  double rate_gbs;           // as ReduceCall::rate_gbs
};
int permute_launch(const PermuteCall &c, hipStream_t s);
int permute_default_wgs(const PermuteCall &c);

// ---- validation (host only, no HIP calls) --------------------------------
int validate_gemm(const void *A, const void *B, const void *C, int M, int N, int K, bool b_kn = false);
int validate_reduce(const float *const *bufs, int nchunks, size_t len, const float *out);
int validate_reduce_own(const void *own, const float *const *peers, int npeers, size_t len, const float *out);
int validate_permute(const void *src, const void *dst, const int32_t *perm, int nchunks,
                     size_t chunk_bytes);

// Tracing helper: sets npairs [start, end] pairs to [UINT64_MAX, 0] and the
// workgroup-record counter wg[0] to 0 (either pointer may be null).
int trace_reset(uint64_t *stamps, int npairs, uint32_t *wg, hipStream_t s);

}  // namespace occ
