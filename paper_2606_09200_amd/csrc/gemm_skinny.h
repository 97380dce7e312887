// Skinny (M <= 16) GEMM kernels (included by gemm.hip only).
#pragma once

#include "gemm_common.h"

namespace occ {
namespace {

// ---------------------------------------------------------------------------
// Skinny kernel for M <= 16 (decode-like GEMMs, HBM-bound on B).  Work unit:
// 16 output columns (16 rows of B) over the whole K.  Persistent workgroups
// (one per CU by default) loop over units; the 4 waves of a workgroup split
// K in quarters and stream their share of the 16 B rows straight from HBM
// into 16x16x32 MFMA operands (non-temporal: every B element is used once),
// UNROLL 32-wide k-blocks of loads in flight per lane.  In a 32-wide k-block
// lane l feeds row l % 16 and k-group l / 16, so one load instruction reads a
// contiguous 64-byte run of each of 16 rows.  A (16 x K, L2-resident) is read
// the same way.  The four partial 16x16 sums are added in wave order
// 0+1+2+3 through LDS, so the result does not depend on timing.
constexpr int kSkinnyKB = 32;

template <int WAVES, int UNROLL>
__global__ __launch_bounds__(64 * WAVES) void gemm_skinny_kernel(const uint16_t *__restrict__ A,
                                                                 const uint16_t *__restrict__ B,
                                                                 uint16_t *__restrict__ C, int M,
                                                                 int N, int K, int prio, KTrace tr) {
  constexpr int kSkinnyUnroll = UNROLL;  // 32-wide k-blocks in flight per lane
  __shared__ f32x4 partial[WAVES - 1][64];
  extern __shared__ __align__(16) unsigned char pad_lds[];  // occupancy pad only
  (void)pad_lds;
  set_wave_priority(prio);
  const TraceStart t0 = trace_begin(tr);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane & 15;   // A row / B row (output column) this lane feeds
  const int g = lane >> 4;   // 8-wide k group inside a 32-wide k-block
  const int nblk = (K + kSkinnyKB - 1) / kSkinnyKB;
  const int b0 = wave * nblk / WAVES, b1 = (wave + 1) * nblk / WAVES;
  const bool arow_ok = r < M;
  const uint16_t *arow = A + (size_t)(arow_ok ? r : 0) * K;
  const int units = (N + 15) / 16;

  for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
    const int n0 = unit * 16;
    const bool brow_ok = n0 + r < N;
    const uint16_t *brow = B + (size_t)(brow_ok ? n0 + r : 0) * K;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    int b = b0;
    for (; b + kSkinnyUnroll <= b1; b += kSkinnyUnroll) {
      u32x4 av[kSkinnyUnroll], bv[kSkinnyUnroll];
#pragma unroll
      for (int u = 0; u < kSkinnyUnroll; ++u) {
        const int k = (b + u) * kSkinnyKB + g * 8;
        u32x4 zb = {0u, 0u, 0u, 0u};
        if (brow_ok && k < K) zb = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(brow + k));
        bv[u] = zb;
      }
#pragma unroll
      for (int u = 0; u < kSkinnyUnroll; ++u) {
        const int k = (b + u) * kSkinnyKB + g * 8;
        u32x4 za = {0u, 0u, 0u, 0u};
        if (arow_ok && k < K) za = *reinterpret_cast<const u32x4 *>(arow + k);
        av[u] = za;
      }
#pragma unroll
      for (int u = 0; u < kSkinnyUnroll; ++u)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av[u]),
                                                      __builtin_bit_cast(bf16x8, bv[u]), acc, 0, 0, 0);
    }
    for (; b < b1; ++b) {
      const int k = b * kSkinnyKB + g * 8;
      u32x4 za = {0u, 0u, 0u, 0u}, zb = {0u, 0u, 0u, 0u};
      if (k < K) {
        if (arow_ok) za = *reinterpret_cast<const u32x4 *>(arow + k);
        if (brow_ok) zb = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(brow + k));
      }
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, za),
                                                    __builtin_bit_cast(bf16x8, zb), acc, 0, 0, 0);
    }

    if (wave > 0) partial[wave - 1][lane] = acc;
    __syncthreads();
    if (wave == 0) {
      f32x4 s = acc;
#pragma unroll
      for (int w = 0; w < WAVES - 1; ++w) {
        f32x4 p = partial[w][lane];
        s[0] = s[0] + p[0];
        s[1] = s[1] + p[1];
        s[2] = s[2] + p[2];
        s[3] = s[3] + p[3];
      }
      // 16x16 MFMA result layout: lane holds column (lane % 16), rows 4*(lane/16) + i.
      const int n = n0 + r;
      if (n < N) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int m = 4 * g + i;
          if (m < M) C[(size_t)m * N + n] = to_bf16(s[i]);
        }
      }
    }
    __syncthreads();  // partial[] is reused by the next unit
  }
  trace_end(tr, t0);
}

// Skinny kernel with A held in registers (M <= 16; K a multiple of
// 64 * WAVES * UNROLL and at most WAVES * KBW * 32).  The same unit, lane
// layout and wave split of K as gemm_skinny_kernel, but each wave loads its
// K-slice of the 16 A rows into registers once (K / (32 * WAVES) 32-wide
// k-blocks, 4 registers each) and keeps it for every unit it processes, so a
// unit streams only its 16 B rows: half the bytes per unit through the memory
// pipeline.  Every k-block is whole, so loads need no bounds checks: a lane
// whose A or B row is past M or N reads row 0 instead and feeds only an output
// row or column that is not stored.  B loads run one chunk (UNROLL k-blocks)
// ahead of the MFMAs that consume them, across unit boundaries too (the even
// chunk count puts the next unit's first chunk in the free buffer).  Partial
// sums are added in wave order through a double-buffered LDS array, one
// barrier per unit.
template <int WAVES, int KBW, int UNROLL>
__global__ __launch_bounds__(64 * WAVES) void gemm_skinny_areg_kernel(const uint16_t *__restrict__ A,
                                                                      const uint16_t *__restrict__ B,
                                                                      uint16_t *__restrict__ C, int M,
                                                                      int N, int K, int prio,
                                                                      KTrace tr) {
  static_assert(KBW % (2 * UNROLL) == 0, "k-blocks per wave must be an even number of chunks");
  constexpr int NCH = KBW / UNROLL;
  __shared__ f32x4 partial[2][WAVES - 1][64];
  extern __shared__ __align__(16) unsigned char pad_lds[];  // occupancy pad only
  (void)pad_lds;
  set_wave_priority(prio);
  const TraceStart t0 = trace_begin(tr);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane & 15;
  const int g = lane >> 4;
  const int bpw = K / (kSkinnyKB * WAVES);  // k-blocks per wave, <= KBW (checked by the host)
  const int nch = bpw / UNROLL;             // chunks, even (checked by the host)
  const int units = (N + 15) / 16;
  // Wave w owns the contiguous K-slice [w * bpw * 32, (w + 1) * bpw * 32):
  // separate sequential streams per wave spread over the HBM channels better
  // (measured) than interleaving the waves' chunks.
  const int kbase = wave * bpw * kSkinnyKB + g * 8;

  u32x4 a[KBW];
  {
    const uint16_t *arow = A + (size_t)(r < M ? r : 0) * K + kbase;
#pragma unroll
    for (int j = 0; j < KBW; ++j) {
      u32x4 z = {0u, 0u, 0u, 0u};
      if (j < bpw) z = *reinterpret_cast<const u32x4 *>(arow + j * kSkinnyKB);
      a[j] = z;
    }
  }
  auto row_of = [&](int unit) { return B + (size_t)(unit * 16 + r < N ? unit * 16 + r : 0) * K + kbase; };
  auto load_chunk = [&](const uint16_t *brow, int ch, u32x4(&bv)[UNROLL]) {
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
      bv[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(brow + (ch * UNROLL + u) * kSkinnyKB));
  };

  u32x4 bv[2][UNROLL];
  if (blockIdx.x < units && nch > 0) load_chunk(row_of(blockIdx.x), 0, bv[0]);
  int par = 0;
  for (int unit = blockIdx.x; unit < units; unit += gridDim.x, par ^= 1) {
    const uint16_t *brow = row_of(unit);
    const int next = unit + (int)gridDim.x;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      if (ch < nch) {
        if (ch + 1 < nch) {
          if (ch + 1 < NCH) load_chunk(brow, ch + 1, bv[(ch + 1) & 1]);
        } else if (next < units) {
          load_chunk(row_of(next), 0, bv[(ch + 1) & 1]);  // (ch + 1) & 1 == 0: nch is even
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[ch * UNROLL + u]),
                                                        __builtin_bit_cast(bf16x8, bv[ch & 1][u]), acc, 0, 0, 0);
      }
    }

    // partial[par] was last read by wave 0 two units ago, before it reached
    // the previous unit's barrier, which every writer has passed since
    if (wave > 0) partial[par][wave - 1][lane] = acc;
    __syncthreads();
    if (wave == 0) {
      f32x4 s = acc;
#pragma unroll
      for (int w = 0; w < WAVES - 1; ++w) {
        f32x4 p = partial[par][w][lane];
        s[0] = s[0] + p[0];
        s[1] = s[1] + p[1];
        s[2] = s[2] + p[2];
        s[3] = s[3] + p[3];
      }
      const int n = unit * 16 + r;
      if (n < N) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int m = 4 * g + i;
          if (m < M) C[(size_t)m * N + n] = to_bf16(s[i]);
        }
      }
    }
  }
  trace_end(tr, t0);
}

}  // namespace
}  // namespace occ
