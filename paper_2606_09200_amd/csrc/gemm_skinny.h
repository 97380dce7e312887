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
                                                                 int N, int K, int prio, KHooks tr) {
  constexpr int kSkinnyUnroll = UNROLL;  // 32-wide k-blocks in flight per lane
  __shared__ f32x4 partial[WAVES - 1][64];
  extern __shared__ __align__(16) unsigned char pad_lds[];  // occupancy pad only
  (void)pad_lds;
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
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
  hooks_end(tr, t0);
}

}  // namespace
}  // namespace occ
