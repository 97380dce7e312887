// Public C entry points: argument validation (host only, before any HIP
// call), device facts, and dispatch to the kernels.
#include "occ_internal.h"

#include <string.h>

namespace occ {

namespace {

bool overlaps(const void *a, size_t abytes, const void *b, size_t bbytes) {
  if (a == nullptr || b == nullptr || abytes == 0 || bbytes == 0) return false;
  uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + bbytes && b0 < a0 + abytes;
}

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

constexpr int kMaxDevices = 64;
DeviceInfo g_info[kMaxDevices];

}  // namespace

int validate_gemm(const void *A, const void *B, const void *C, int M, int N, int K, bool b_kn) {
  if (M < 0 || N < 0 || K < 0 || K % 8 != 0) return OCC_EINVAL;
  if (b_kn && N % 8 != 0) return OCC_EINVAL;  // 16-byte rows of a K x N B
  if (M == 0 || N == 0) return OCC_OK;
  if (C == nullptr || !aligned(C, 16)) return OCC_EINVAL;
  if (K > 0 && (A == nullptr || B == nullptr || !aligned(A, 16) || !aligned(B, 16))) return OCC_EINVAL;
  size_t cb = (size_t)M * N * 2;
  if (K > 0 && (overlaps(C, cb, A, (size_t)M * K * 2) || overlaps(C, cb, B, (size_t)N * K * 2)))
    return OCC_EALIAS;
  return OCC_OK;
}

int validate_reduce(const float *const *bufs, int nchunks, size_t len, const float *out) {
  if (bufs == nullptr || nchunks < 1 || nchunks > kMaxReduceChunks) return OCC_EINVAL;
  if (len == 0) return OCC_OK;
  if (out == nullptr || !aligned(out, 4)) return OCC_EINVAL;
  for (int i = 0; i < nchunks; ++i)
    if (bufs[i] == nullptr || !aligned(bufs[i], 4)) return OCC_EINVAL;
  for (int i = 0; i < nchunks; ++i)
    if (overlaps(out, len * 4, bufs[i], len * 4)) return OCC_EALIAS;
  return OCC_OK;
}

int validate_reduce_own(const void *own, const float *const *peers, int npeers, size_t len,
                        const float *out) {
  if (npeers < 0 || npeers > kMaxReduceChunks - 1 || (npeers > 0 && peers == nullptr)) return OCC_EINVAL;
  if (len == 0) return OCC_OK;
  if (own == nullptr || !aligned(own, 2) || out == nullptr || !aligned(out, 4)) return OCC_EINVAL;
  for (int i = 0; i < npeers; ++i)
    if (peers[i] == nullptr || !aligned(peers[i], 4)) return OCC_EINVAL;
  if (overlaps(out, len * 4, own, len * 2)) return OCC_EALIAS;
  for (int i = 0; i < npeers; ++i)
    if (overlaps(out, len * 4, peers[i], len * 4)) return OCC_EALIAS;
  return OCC_OK;
}

int validate_permute(const void *src, const void *dst, const int32_t *perm, int nchunks,
                     size_t chunk_bytes) {
  if (perm == nullptr || nchunks < 1 || nchunks > kMaxPermuteChunks) return OCC_EINVAL;
  unsigned char seen[kMaxPermuteChunks];
  memset(seen, 0, sizeof seen);
  for (int i = 0; i < nchunks; ++i) {
    int32_t p = perm[i];
    if (p < 0 || p >= nchunks || seen[p]) return OCC_EPERM;
    seen[p] = 1;
  }
  if (chunk_bytes == 0) return OCC_OK;
  if (src == nullptr || dst == nullptr) return OCC_EINVAL;
  size_t total = chunk_bytes * (size_t)nchunks;
  if (overlaps(src, total, dst, total)) return OCC_EALIAS;
  return OCC_OK;
}

const DeviceInfo &device_info(int device) {
  DeviceInfo &d = g_info[device];
  if (!d.ok) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, device) != hipSuccess) return d;
    int v = 0;
    d.num_cus = prop.multiProcessorCount;
    d.lds_per_cu = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, device) == hipSuccess ? v : 0;
    d.max_lds_per_wg = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, device) == hipSuccess ? v : 0;
    d.clock_khz = hipDeviceGetAttribute(&v, hipDeviceAttributeClockRate, device) == hipSuccess ? v : 0;
    d.gfx950 = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    d.ok = d.num_cus > 0 && d.max_lds_per_wg > 0;
  }
  return d;
}

int current_device_info(const DeviceInfo **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return OCC_ENODEV;
  const DeviceInfo &d = device_info(dev);
  if (!d.ok || !d.gfx950) return OCC_ENODEV;
  *out = &d;
  return OCC_OK;
}

int run_overlap_impl(const occ_overlap_cfg *cfg, occ_overlap_result *res);
size_t overlap_workspace_bytes(int n_iter);
int overlap_enqueue_impl(const occ_overlap_cfg *cfg, void *comm_stream, void *workspace, size_t workspace_bytes,
                         uint32_t *err);
int overlap_enqueue_noalloc_impl(const occ_overlap_cfg *cfg, void *comm_stream, uint32_t *err);
int overlap_tune_impl(occ_overlap_cfg *cfg, int tune_reps, occ_overlap_result *res,
                      int *prefer_sequential);

}  // namespace occ

extern "C" {

static int gemm_entry(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
                      int variant, int grid_cap, void *stream, bool b_kn) {
  int st = occ::validate_gemm(A, B, C, M, N, K, b_kn);
  if (st != OCC_OK) return st;
  if (grid_cap < 0 || variant < 0) return OCC_EINVAL;
  occ::GemmCall c{A, B, C, M, N, K, lds_bytes, grid_cap, variant, 0, occ::KHooks{}, b_kn};
  return occ::gemm_launch(c, static_cast<hipStream_t>(stream));
}

static int plan_entry(int M, int N, int K, size_t lds_bytes, int variant, int grid_cap, occ_gemm_plan *plan,
                      bool b_kn) {
  if (plan == nullptr || M < 0 || N < 0 || K < 0 || variant < 0 || grid_cap < 0) return OCC_EINVAL;
  memset(plan, 0, sizeof *plan);
  occ::GemmCall c{nullptr, nullptr, nullptr, M, N, K, lds_bytes, grid_cap, variant, 0, occ::KHooks{}, b_kn};
  return occ::gemm_plan(c, plan);
}

int occ_gemm_ex(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
                int variant, int grid_cap, void *stream) {
  return gemm_entry(A, B, C, M, N, K, lds_bytes, variant, grid_cap, stream, true);
}

int occ_gemm(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
             void *stream) {
  return gemm_entry(A, B, C, M, N, K, lds_bytes, OCC_GEMM_AUTO, 0, stream, true);
}

int occ_gemm_bt_ex(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
                   int variant, int grid_cap, void *stream) {
  return gemm_entry(A, B, C, M, N, K, lds_bytes, variant, grid_cap, stream, false);
}

int occ_gemm_bt(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
                void *stream) {
  return gemm_entry(A, B, C, M, N, K, lds_bytes, OCC_GEMM_AUTO, 0, stream, false);
}

int occ_gemm_plan_query(int M, int N, int K, size_t lds_bytes, int variant, int grid_cap,
                        occ_gemm_plan *plan) {
  return plan_entry(M, N, K, lds_bytes, variant, grid_cap, plan, true);
}

int occ_gemm_bt_plan_query(int M, int N, int K, size_t lds_bytes, int variant, int grid_cap,
                           occ_gemm_plan *plan) {
  return plan_entry(M, N, K, lds_bytes, variant, grid_cap, plan, false);
}

int occ_gemm_info(int *tile_lds_bytes, int *max_lds_per_wg, int *lds_per_cu) {
  if (tile_lds_bytes == nullptr || max_lds_per_wg == nullptr || lds_per_cu == nullptr) return OCC_EINVAL;
  occ_gemm_plan p;
  // the kernel occ_gemm picks for large shapes (any shape with at least one
  // 256x256 tile per CU takes it)
  int st = occ_gemm_plan_query(8192, 8192, 8192, 0, OCC_GEMM_KN_256x256x64_8W_2ST, 0, &p);
  if (st != OCC_OK) return st;
  *tile_lds_bytes = p.tile_lds_bytes;
  *max_lds_per_wg = p.max_lds_per_wg;
  *lds_per_cu = p.lds_per_cu;
  return OCC_OK;
}

int share_reduce_ex(const float *const *bufs, int nchunks, size_t len, float *out, int wgs,
                    int priority, void *stream) {
  int st = occ::validate_reduce(bufs, nchunks, len, out);
  if (st != OCC_OK) return st;
  if (wgs < 0 || priority < 0 || priority > 3) return OCC_EINVAL;
  const occ::DeviceInfo *di = nullptr;
  if (len > 0 && (st = occ::current_device_info(&di)) != OCC_OK) return st;
  occ::ReduceCall c{bufs, nchunks, len, out, wgs, priority, occ::KHooks{}, 0.0};
  return occ::reduce_launch(c, static_cast<hipStream_t>(stream));
}

int share_reduce(const float *const *bufs, int nchunks, size_t len, float *out, void *stream) {
  return share_reduce_ex(bufs, nchunks, len, out, 0, 0, stream);
}

int share_reduce_own(const void *own, const float *const *peers, int npeers, size_t len, float *out,
                     int wgs, int priority, void *stream) {
  int st = occ::validate_reduce_own(own, peers, npeers, len, out);
  if (st != OCC_OK) return st;
  if (wgs < 0 || priority < 0 || priority > 3) return OCC_EINVAL;
  const occ::DeviceInfo *di = nullptr;
  if (len > 0 && (st = occ::current_device_info(&di)) != OCC_OK) return st;
  occ::ReduceCall c{peers, npeers, len, out, wgs, priority, occ::KHooks{}, 0.0,
                    static_cast<const uint16_t *>(own)};
  return occ::reduce_launch(c, static_cast<hipStream_t>(stream));
}

int share_permute_ex(const void *src, void *dst, const int32_t *perm, int nchunks,
                     size_t chunk_bytes, int wgs, int priority, void *stream) {
  int st = occ::validate_permute(src, dst, perm, nchunks, chunk_bytes);
  if (st != OCC_OK) return st;
  if (wgs < 0 || priority < 0 || priority > 3) return OCC_EINVAL;
  const occ::DeviceInfo *di = nullptr;
  if (chunk_bytes > 0 && (st = occ::current_device_info(&di)) != OCC_OK) return st;
  occ::PermuteCall c{src, dst, perm, nchunks, chunk_bytes, wgs, priority, occ::KHooks{}, 0.0};
  return occ::permute_launch(c, static_cast<hipStream_t>(stream));
}

int share_permute(const void *src, void *dst, const int32_t *perm, int nchunks, size_t chunk_bytes,
                  void *stream) {
  return share_permute_ex(src, dst, perm, nchunks, chunk_bytes, 0, 0, stream);
}

int run_overlap(const occ_overlap_cfg *cfg, occ_overlap_result *res) {
  return occ::run_overlap_impl(cfg, res);
}

int occ_overlap_tune(occ_overlap_cfg *cfg, int tune_reps, occ_overlap_result *res,
                     int *prefer_sequential) {
  return occ::overlap_tune_impl(cfg, tune_reps, res, prefer_sequential);
}

size_t occ_overlap_workspace_bytes(int n_iter) { return occ::overlap_workspace_bytes(n_iter); }

int occ_overlap_enqueue(const occ_overlap_cfg *cfg, void *comm_stream, void *workspace, size_t workspace_bytes,
                        uint32_t *err) {
  return occ::overlap_enqueue_impl(cfg, comm_stream, workspace, workspace_bytes, err);
}

int occ_overlap_enqueue_noalloc(const occ_overlap_cfg *cfg, void *comm_stream, uint32_t *err) {
  return occ::overlap_enqueue_noalloc_impl(cfg, comm_stream, err);
}

const char *occ_strerror(int status) {
  switch (status) {
    case OCC_OK: return "OCC_OK: success";
    case OCC_EINVAL: return "OCC_EINVAL: null pointer, bad size or misaligned buffer";
    case OCC_ELDS: return "OCC_ELDS: tile LDS plus pad exceeds the per-workgroup LDS limit";
    case OCC_EPERM: return "OCC_EPERM: perm is not a bijection of [0, nchunks)";
    case OCC_EALIAS: return "OCC_EALIAS: an output overlaps an input";
    case OCC_EHIP: return "OCC_EHIP: HIP runtime error";
    case OCC_ENODEV: return "OCC_ENODEV: no gfx950 device is current";
    case OCC_ETIMEOUT: return "OCC_ETIMEOUT: a collective's bounded wait for its GEMM ran out";
    default: return "unknown occ status";
  }
}

int occ_version(void) { return (OCC_VERSION_MAJOR << 16) | OCC_VERSION_MINOR; }

}  // extern "C"
