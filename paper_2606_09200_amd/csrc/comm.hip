// K_c: one GPU's local share of a collective (Background, item 2).
//
//   share_reduce  -- allreduce share: fixed-order binary32 sum of the chunks.
//   share_permute -- alltoall share: gather of whole chunks by a permutation.
//
// Both are HBM-bound streams: 16-byte non-temporal loads and stores (so the
// stream does not evict the concurrently running GEMM's operands from L2),
// several independent loads in flight per lane, and a grid that is a knob
// (communication kernels are meant to be light, Section 3.1).  The comm
// kernel's wave priority is raised with s_setprio when asked: that is how the
// collective is given precedence over co-resident GEMM waves (Section 3.3).
#include "device_util.h"
#include "occ_internal.h"

#include <string.h>

#include <type_traits>

namespace occ {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// bf16 bit pattern -> binary32 (exact: the bf16 bits are the high half)
__device__ __forceinline__ float widen_bf16(uint32_t bits16) { return __builtin_bit_cast(float, bits16 << 16); }

// Workgroup sizes.  The chunk sum runs two waves per workgroup: at the
// default grid of one workgroup per CU, two of a CU's four SIMDs carry a comm
// wave.  Measured on MI355X against four waves per workgroup: the isolated
// 8-term sum is 8 % faster, and the overlapped schedules are 1.5-8 % shorter
// (8192^3 with 8 x 128 MiB, the same with the own term, and 16 x 28672 x 8192
// with 8 x 64 MiB, at both comm priorities); one wave per workgroup slows the
// isolated sum by 40 % and lengthens the decode-like schedule.  The
// permutation also runs two waves, with twice the loads in flight per lane
// of a four-wave workgroup (kPermuteUnroll): against four waves it is 0.5-1 %
// faster alone and never slower overlapped (8192^3 with 4 x 224 MiB: 0.3-0.9 %
// shorter).
constexpr int kReduceThreads = 128;
constexpr int kPermuteThreads = 128;

struct ChunkPtrs {
  const float *p[kMaxReduceChunks];
};

// Vector path: all chunk pointers and out are 16-byte aligned.  Element j's
// sum is acc = c0[j]; acc = acc + c1[j]; ... exactly in chunk order; the
// loads of all chunks for UNROLL positions are issued before any addition.
// Measured on MI355X: for 8 terms, two positions per trip (16 loads in
// flight per lane, 64 VGPRs) stream as fast as one in the isolated pass and
// make the overlapped 8192^3 schedule 1-2 % shorter (the own-term reduce
// 6 % faster); four positions fall in between.  The default grid is one
// workgroup per CU.
//
// OWN: the first term is a bf16 buffer (this GPU's own contribution, e.g. its
// GEMM output), widened exactly to binary32; the NC (or nchunks) fp32 chunks
// follow it in order.  Its 8 bytes per position are one load.
template <int NC, int UNROLL, bool OFF32, bool OWN>
__global__ __launch_bounds__(kReduceThreads) void reduce_vec_kernel(ChunkPtrs cp, int nchunks, size_t nvec,
                                                                    float *__restrict__ out,
                                                                    const uint16_t *__restrict__ own, int prio,
                                                                    uint32_t pace, KHooks tr) {
  // OFF32: every byte offset the loop forms fits in 32 bits (checked by the
  // host), so each access is a scalar base plus one shared 32-bit lane
  // offset instead of a 64-bit address per chunk: fewer vector instructions
  // per byte, which is issue time a co-running GEMM on the same SIMD gets back.
  using I = typename std::conditional<OFF32, uint32_t, size_t>::type;
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
  Pacer pc = pace_start(pace);
  const int nc = NC > 0 ? NC : nchunks;
  const I n = (I)nvec;
  const I stride = (I)gridDim.x * kReduceThreads;
  I i = (I)blockIdx.x * kReduceThreads + threadIdx.x;
  auto ld = [&](int c, I k) {
    return __builtin_nontemporal_load(
        reinterpret_cast<const f32x4 *>(reinterpret_cast<const char *>(cp.p[c]) + k * (I)sizeof(f32x4)));
  };
  auto st = [&](f32x4 v, I k) {
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(reinterpret_cast<char *>(out) + k * (I)sizeof(f32x4)));
  };
  auto ld_own = [&](I k) {
    const u32x2 w = __builtin_nontemporal_load(
        reinterpret_cast<const u32x2 *>(reinterpret_cast<const char *>(own) + k * (I)sizeof(u32x2)));
    f32x4 r;
    r[0] = widen_bf16(w[0] & 0xFFFFu);
    r[1] = widen_bf16(w[0] >> 16);
    r[2] = widen_bf16(w[1] & 0xFFFFu);
    r[3] = widen_bf16(w[1] >> 16);
    return r;
  };
  constexpr int C0 = OWN ? 0 : 1;  // first fp32 chunk added to the first term

  if constexpr (NC > 0) {
    for (bool first = true; i + (UNROLL - 1) * stride < n; i += UNROLL * stride, first = false) {
      if (!first) pace_wait(pc);
      f32x4 v[NC][UNROLL], o[UNROLL];
      if constexpr (OWN) {
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) o[u] = ld_own(i + u * stride);
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) v[c][u] = ld(c, i + u * stride);
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {
        f32x4 acc = OWN ? o[u] : v[0][u];
#pragma unroll
        for (int c = C0; c < NC; ++c) {
          acc[0] = acc[0] + v[c][u][0];
          acc[1] = acc[1] + v[c][u][1];
          acc[2] = acc[2] + v[c][u][2];
          acc[3] = acc[3] + v[c][u][3];
        }
        st(acc, i + u * stride);
      }
    }
  }
  // Remaining positions (and every position when the chunk count is only
  // known at run time): chunks in batches of 8 loads, folded in order.
  for (bool first = true; i < n; i += stride, first = false) {
    if (NC == 0 && !first) pace_wait(pc);
    f32x4 acc = OWN ? ld_own(i) : ld(0, i);
    for (int c0 = C0; c0 < nc; c0 += 8) {
      f32x4 v[8];
#pragma unroll
      for (int c = 0; c < 8; ++c)
        if (c0 + c < nc) v[c] = ld(c0 + c, i);
#pragma unroll
      for (int c = 0; c < 8; ++c)
        if (c0 + c < nc) {
          acc[0] = acc[0] + v[c][0];
          acc[1] = acc[1] + v[c][1];
          acc[2] = acc[2] + v[c][2];
          acc[3] = acc[3] + v[c][3];
        }
    }
    st(acc, i);
  }
  hooks_end(tr, t0);
}

// Scalar path: elements [first, len) one at a time (the tail after the vector
// path, or everything when a buffer is not 16-byte aligned).
__global__ __launch_bounds__(kReduceThreads) void reduce_scalar_kernel(ChunkPtrs cp, int nchunks,
                                                                       size_t first, size_t len,
                                                                       float *__restrict__ out,
                                                                       const uint16_t *__restrict__ own,
                                                                       int prio, KHooks tr) {
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
  const size_t stride = (size_t)gridDim.x * kReduceThreads;
  for (size_t j = first + (size_t)blockIdx.x * kReduceThreads + threadIdx.x; j < len; j += stride) {
    float acc = own != nullptr ? widen_bf16(own[j]) : cp.p[0][j];
    for (int c = own != nullptr ? 0 : 1; c < nchunks; ++c) acc = acc + cp.p[c][j];
    out[j] = acc;
  }
  hooks_end(tr, t0);
}

struct PermTable {
  int32_t p[kMaxPermuteChunks];
};

// Permutation copy, 16-byte units.  Work item w covers part (w % parts) of
// destination chunk (w / parts); workgroups stride over work items, threads
// over the part's units with UNROLL loads in flight before the stores.
template <int UNROLL, bool OFF32>
__global__ __launch_bounds__(kPermuteThreads) void permute_vec_kernel(const u32x4 *__restrict__ src,
                                                                      u32x4 *__restrict__ dst, PermTable pt,
                                                                      int nchunks, size_t cvec, int parts,
                                                                      int prio, uint32_t pace, KHooks tr) {
  // OFF32: offsets inside a chunk fit in 32 bits (checked by the host): the
  // work item's chunk bases are scalar and the lanes share one 32-bit offset.
  using I = typename std::conditional<OFF32, uint32_t, size_t>::type;
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
  Pacer pc = pace_start(pace);
  bool first = true;
  const int nwork = nchunks * parts;
  for (int w = blockIdx.x; w < nwork; w += gridDim.x) {
    const int chunk = w / parts;
    const int part = w - chunk * parts;
    const I lo = (I)(cvec * part / parts);
    const I hi = (I)(cvec * (part + 1) / parts);
    const char *s = reinterpret_cast<const char *>(src + (size_t)pt.p[chunk] * cvec);
    char *d = reinterpret_cast<char *>(dst + (size_t)chunk * cvec);
    auto at = [](const char *b, I k) { return reinterpret_cast<const u32x4 *>(b + k * (I)sizeof(u32x4)); };
    auto atw = [](char *b, I k) { return reinterpret_cast<u32x4 *>(b + k * (I)sizeof(u32x4)); };
    I i = lo + threadIdx.x;
    for (; i + (UNROLL - 1) * kPermuteThreads < hi; i += UNROLL * kPermuteThreads) {
      if (!first) pace_wait(pc);
      first = false;
      u32x4 v[UNROLL];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) v[u] = __builtin_nontemporal_load(at(s, i + u * kPermuteThreads));
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) __builtin_nontemporal_store(v[u], atw(d, i + u * kPermuteThreads));
    }
    for (; i < hi; i += kPermuteThreads) __builtin_nontemporal_store(__builtin_nontemporal_load(at(s, i)), atw(d, i));
  }
  hooks_end(tr, t0);
}

// Byte path for unaligned buffers or chunk sizes.
__global__ __launch_bounds__(kPermuteThreads) void permute_byte_kernel(const uint8_t *__restrict__ src,
                                                                       uint8_t *__restrict__ dst,
                                                                       PermTable pt, int nchunks,
                                                                       size_t chunk_bytes, int prio,
                                                                       KHooks tr) {
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
  const size_t stride = (size_t)gridDim.x * kPermuteThreads;
  for (int c = 0; c < nchunks; ++c) {
    const uint8_t *s = src + (size_t)pt.p[c] * chunk_bytes;
    uint8_t *d = dst + (size_t)c * chunk_bytes;
    for (size_t b = (size_t)blockIdx.x * kPermuteThreads + threadIdx.x; b < chunk_bytes; b += stride) d[b] = s[b];
  }
  hooks_end(tr, t0);
}

__global__ void stamps_reset_kernel(uint64_t *stamps, int npairs, uint32_t *wg) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (stamps != nullptr && i < npairs) {
    stamps[2 * i] = ~0ull;
    stamps[2 * i + 1] = 0ull;
  }
  if (wg != nullptr && i == 0) wg[0] = 0u;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// At most one workgroup per `threads` work units, at least one.
int clamp_wgs(size_t work_units, int wanted, int threads) {
  size_t cap = (work_units + threads - 1) / threads;
  if (cap < 1) cap = 1;
  return (int)(wanted < (long long)cap ? wanted : cap);
}

// Positions per lane per trip of the vector chunk sum for a number of terms
// (fp32 chunks plus the own term); the launch table and the pacing period
// both take it from here.
constexpr int reduce_unroll(int terms) { return terms == 2 ? 4 : (terms == 4 || terms == 8) ? 2 : 1; }

// Loads in flight per lane of the vector permutation (launch, pacing and the
// 32-bit offset check).  With four-wave workgroups 2 and 8 gave no shorter
// overlapped schedule than 4 (16384x14336x4096 with 64 x 4 MiB, 8192^3 with
// 4 x 224 MiB); the two-wave workgroups take 8, the same bytes per CU.
constexpr int kPermuteUnroll = 8;

// Period (10 ns ticks) between a wave's trips so that the whole grid moves
// trip_bytes per period, i.e. streams at rate_gbs; 0 = unpaced.
uint32_t pace_ticks(double trip_bytes, double rate_gbs) {
  if (!(rate_gbs > 0.0)) return 0;
  double t = trip_bytes / (rate_gbs * 1e9) * 1e8;
  if (t < 1.0) t = 1.0;
  if (t > 4.0e9) t = 4.0e9;
  return (uint32_t)t;
}

}  // namespace

template <bool OFF32, bool OWN>
void launch_reduce(int nchunks, int g, hipStream_t s, const ChunkPtrs &cp, size_t nvec, float *out,
                   const uint16_t *own, int prio, uint32_t pace, const KHooks &tr) {
  // instantiations by the number of terms (own + fp32 chunks)
  switch (nchunks + (OWN ? 1 : 0)) {
    case 2: hipLaunchKernelGGL((reduce_vec_kernel<OWN ? 1 : 2, reduce_unroll(2), OFF32, OWN>), dim3(g), dim3(kReduceThreads), 0, s, cp, nchunks, nvec, out, own, prio, pace, tr); break;
    case 4: hipLaunchKernelGGL((reduce_vec_kernel<OWN ? 3 : 4, reduce_unroll(4), OFF32, OWN>), dim3(g), dim3(kReduceThreads), 0, s, cp, nchunks, nvec, out, own, prio, pace, tr); break;
    case 8: hipLaunchKernelGGL((reduce_vec_kernel<OWN ? 7 : 8, reduce_unroll(8), OFF32, OWN>), dim3(g), dim3(kReduceThreads), 0, s, cp, nchunks, nvec, out, own, prio, pace, tr); break;
    case 16: hipLaunchKernelGGL((reduce_vec_kernel<OWN ? 15 : 16, reduce_unroll(16), OFF32, OWN>), dim3(g), dim3(kReduceThreads), 0, s, cp, nchunks, nvec, out, own, prio, pace, tr); break;
    default: hipLaunchKernelGGL((reduce_vec_kernel<0, 1, OFF32, OWN>), dim3(g), dim3(kReduceThreads), 0, s, cp, nchunks, nvec, out, own, prio, pace, tr); break;
  }
}

int reduce_default_wgs(const ReduceCall &c) {
  const DeviceInfo *di = nullptr;
  int cus = current_device_info(&di) == OCC_OK ? di->num_cus : 256;
  return clamp_wgs(c.len / 4 + 1, cus, kReduceThreads);
}

int reduce_launch(const ReduceCall &c, hipStream_t s) {
  if (c.len == 0) return OCC_OK;
  ChunkPtrs cp;
  memset(&cp, 0, sizeof cp);
  const bool own = c.own != nullptr;
  bool vec = aligned16(c.out) && (!own || (reinterpret_cast<uintptr_t>(c.own) & 7u) == 0);
  for (int i = 0; i < c.nchunks; ++i) {
    cp.p[i] = c.bufs[i];
    vec = vec && aligned16(c.bufs[i]);
  }
  int wgs = c.wgs > 0 ? c.wgs : reduce_default_wgs(c);
  const int prio = c.priority;
  // a dependency wait is acknowledged by every workgroup of every kernel below
  KHooks tr = c.trace;
  if (vec) {
    size_t nvec = c.len / 4;
    const bool tail = nvec * 4 < c.len;
    if (tr.wait != nullptr)
      tr.ack_target = (nvec > 0 ? (uint32_t)clamp_wgs(nvec, wgs, kReduceThreads) : 0u) + (tail ? 1u : 0u);
    if (nvec > 0) {
      int g = clamp_wgs(nvec, wgs, kReduceThreads);
      // positions per lane per trip of each instantiation, and the bytes
      // one position moves
      const int terms = c.nchunks + (own ? 1 : 0);
      const int unroll = reduce_unroll(terms);
      const double pos_bytes = 16.0 * (c.nchunks + 1) + (own ? 8.0 : 0.0);
      const uint32_t pace = pace_ticks((double)g * kReduceThreads * unroll * pos_bytes, c.rate_gbs);
      // 32-bit offsets when the largest byte offset the loop can form, (nvec
      // plus one unrolled grid stride) * 16, stays below 2^32
      const bool off32 = ((double)nvec + 4.0 * g * kReduceThreads) * 16.0 < 4294967296.0;
      if (own) {
        if (off32) launch_reduce<true, true>(c.nchunks, g, s, cp, nvec, c.out, c.own, prio, pace, tr);
        else launch_reduce<false, true>(c.nchunks, g, s, cp, nvec, c.out, c.own, prio, pace, tr);
      } else {
        if (off32) launch_reduce<true, false>(c.nchunks, g, s, cp, nvec, c.out, nullptr, prio, pace, tr);
        else launch_reduce<false, false>(c.nchunks, g, s, cp, nvec, c.out, nullptr, prio, pace, tr);
      }
    }
    if (tail)
      hipLaunchKernelGGL(reduce_scalar_kernel, dim3(1), dim3(kReduceThreads), 0, s, cp, c.nchunks, nvec * 4,
                         c.len, c.out, c.own, prio, tr);
  } else {
    const int g = clamp_wgs(c.len, wgs, kReduceThreads);
    if (tr.wait != nullptr) tr.ack_target = (uint32_t)g;
    hipLaunchKernelGGL(reduce_scalar_kernel, dim3(g), dim3(kReduceThreads), 0, s, cp,
                       c.nchunks, (size_t)0, c.len, c.out, c.own, prio, tr);
  }
  return hipGetLastError() == hipSuccess ? OCC_OK : OCC_EHIP;
}

static int permute_parts(size_t chunk_bytes) {
  // about 256 KiB per work item, at least one
  size_t parts = (chunk_bytes + (256u << 10) - 1) / (256u << 10);
  if (parts < 1) parts = 1;
  if (parts > 4096) parts = 4096;
  return (int)parts;
}

int permute_default_wgs(const PermuteCall &c) {
  const DeviceInfo *di = nullptr;
  int cus = current_device_info(&di) == OCC_OK ? di->num_cus : 256;
  long long items = (long long)c.nchunks * permute_parts(c.chunk_bytes);
  long long want = cus;
  return (int)(items < want ? items : want);
}

int permute_launch(const PermuteCall &c, hipStream_t s) {
  if (c.chunk_bytes == 0) return OCC_OK;
  PermTable pt;
  memset(&pt, 0, sizeof pt);
  for (int i = 0; i < c.nchunks; ++i) pt.p[i] = c.perm[i];
  int wgs = c.wgs > 0 ? c.wgs : permute_default_wgs(c);
  KHooks tr = c.trace;
  if (aligned16(c.src) && aligned16(c.dst) && c.chunk_bytes % 16 == 0) {
    int parts = permute_parts(c.chunk_bytes);
    long long items = (long long)c.nchunks * parts;
    int g = (int)(wgs < items ? wgs : items);
    if (tr.wait != nullptr) tr.ack_target = (uint32_t)g;
    const uint32_t pace = pace_ticks((double)g * kPermuteThreads * kPermuteUnroll * 16.0 * 2.0, c.rate_gbs);
    // 32-bit offsets when a chunk plus one unrolled block stays below 2^32 bytes
    if ((double)c.chunk_bytes + (double)kPermuteUnroll * kPermuteThreads * 16.0 < 4294967296.0)
      hipLaunchKernelGGL((permute_vec_kernel<kPermuteUnroll, true>), dim3(g), dim3(kPermuteThreads), 0, s,
                         static_cast<const u32x4 *>(c.src), static_cast<u32x4 *>(c.dst), pt, c.nchunks,
                         c.chunk_bytes / 16, parts, c.priority, pace, tr);
    else
      hipLaunchKernelGGL((permute_vec_kernel<kPermuteUnroll, false>), dim3(g), dim3(kPermuteThreads), 0, s,
                         static_cast<const u32x4 *>(c.src), static_cast<u32x4 *>(c.dst), pt, c.nchunks,
                         c.chunk_bytes / 16, parts, c.priority, pace, tr);
  } else {
    int g = clamp_wgs(c.chunk_bytes, wgs, kPermuteThreads);
    if (tr.wait != nullptr) tr.ack_target = (uint32_t)g;
    hipLaunchKernelGGL(permute_byte_kernel, dim3(g), dim3(kPermuteThreads), 0, s,
                       static_cast<const uint8_t *>(c.src), static_cast<uint8_t *>(c.dst), pt,
                       c.nchunks, c.chunk_bytes, c.priority, tr);
  }
  return hipGetLastError() == hipSuccess ? OCC_OK : OCC_EHIP;
}

int trace_reset(uint64_t *stamps, int npairs, uint32_t *wg, hipStream_t s) {
  if (stamps == nullptr && wg == nullptr) return OCC_OK;
  int n = npairs > 1 ? npairs : 1;
  hipLaunchKernelGGL(stamps_reset_kernel, dim3((n + 255) / 256), dim3(256), 0, s, stamps, npairs, wg);
  return hipGetLastError() == hipSuccess ? OCC_OK : OCC_EHIP;
}

}  // namespace occ
