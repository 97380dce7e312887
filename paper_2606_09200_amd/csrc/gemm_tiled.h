// Register-staged tiled GEMM kernel (included by gemm.hip only).
#pragma once

#include "gemm_common.h"

namespace occ {
namespace {

template <class T>
__device__ __forceinline__ void load_tile_regs(const uint16_t *__restrict__ A,
                                               const uint16_t *__restrict__ B, int M, int N,
                                               int K, int m0, int n0, int k0, u32x4 (&ra)[T::A_LOADS],
                                               u32x4 (&rb)[T::B_LOADS]) {
  const int tid = threadIdx.x;
  const int r_in = tid / T::KCH;
  const int c = tid % T::KCH;
  const int k = k0 + c * 8;
  const bool kok = k < K;
#pragma unroll
  for (int p = 0; p < T::A_LOADS; ++p) {
    int m = m0 + p * T::ROWS_PER_PASS + r_in;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (kok && m < M) v = *reinterpret_cast<const u32x4 *>(A + (size_t)m * K + k);
    ra[p] = v;
  }
#pragma unroll
  for (int p = 0; p < T::B_LOADS; ++p) {
    int n = n0 + p * T::ROWS_PER_PASS + r_in;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (kok && n < N) v = *reinterpret_cast<const u32x4 *>(B + (size_t)n * K + k);
    rb[p] = v;
  }
}

template <class T>
__device__ __forceinline__ void store_tile_lds(unsigned char *stage, const u32x4 (&ra)[T::A_LOADS],
                                               const u32x4 (&rb)[T::B_LOADS]) {
  const int tid = threadIdx.x;
  const int r_in = tid / T::KCH;
  const int c = tid % T::KCH;
#pragma unroll
  for (int p = 0; p < T::A_LOADS; ++p) {
    int r = p * T::ROWS_PER_PASS + r_in;
    *reinterpret_cast<u32x4 *>(stage + r * (T::BK * 2) + swz<T::KCH>(r, c) * 16) = ra[p];
  }
  unsigned char *bs = stage + T::A_BYTES;
#pragma unroll
  for (int p = 0; p < T::B_LOADS; ++p) {
    int r = p * T::ROWS_PER_PASS + r_in;
    *reinterpret_cast<u32x4 *>(bs + r * (T::BK * 2) + swz<T::KCH>(r, c) * 16) = rb[p];
  }
}

template <class T>
__global__ __launch_bounds__(T::NT) void gemm_tiled_kernel(const uint16_t *__restrict__ A,
                                                           const uint16_t *__restrict__ B,
                                                           uint16_t *__restrict__ C, int M, int N,
                                                           int K, int tiles_m, int tiles_n,
                                                           int prio, KHooks tr) {
  extern __shared__ __align__(16) unsigned char smem[];  // tile stages, then the unused pad
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / T::WN;
  const int wn = wave % T::WN;
  const int ntiles = tiles_m * tiles_n;
  const int nk = (K + T::BK - 1) / T::BK;

  for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
    int tm, tn;
    tile_coords<8>(xcd_remap(t, ntiles), tiles_m, tiles_n, tm, tn);
    const int m0 = tm * T::BM;
    const int n0 = tn * T::BN;

    f32x16 acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
      for (int j = 0; j < T::FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    u32x4 ra[T::A_LOADS], rb[T::B_LOADS];
    if (nk > 0) {
      load_tile_regs<T>(A, B, M, N, K, m0, n0, 0, ra, rb);
      store_tile_lds<T>(smem, ra, rb);
    }
    __syncthreads();

    // Per-lane LDS offsets of the MFMA operand rows for each 16-wide k-substep.
    const int arow = wm * T::TM + (lane & 31);
    const int brow = wn * T::TN + (lane & 31);
    const int half = lane >> 5;

    for (int kt = 0; kt < nk; ++kt) {
      unsigned char *cur = smem + (kt % T::STAGES) * T::STAGE_BYTES;
      const bool more = kt + 1 < nk;
      if (more) load_tile_regs<T>(A, B, M, N, K, m0, n0, (kt + 1) * T::BK, ra, rb);

#pragma unroll
      for (int ks = 0; ks < T::BK / 16; ++ks) {
        const int c = ks * 2 + half;
        bf16x8 af[T::FM], bfr[T::FN];
#pragma unroll
        for (int i = 0; i < T::FM; ++i) {
          int r = arow + i * 32;
          af[i] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4 *>(cur + r * (T::BK * 2) + swz<T::KCH>(r, c) * 16));
        }
        const unsigned char *bs = cur + T::A_BYTES;
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
          int r = brow + j * 32;
          bfr[j] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4 *>(bs + r * (T::BK * 2) + swz<T::KCH>(r, c) * 16));
        }
#pragma unroll
        for (int i = 0; i < T::FM; ++i)
#pragma unroll
          for (int j = 0; j < T::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      }

      if constexpr (T::STAGES == 1) __syncthreads();
      if (more) store_tile_lds<T>(smem + ((kt + 1) % T::STAGES) * T::STAGE_BYTES, ra, rb);
      __syncthreads();
    }

    // Epilogue.  32x32 MFMA result layout: lane holds column (lane % 32) and
    // rows 8*(r/4) + 4*(lane/32) + r%4 of the block, r = 0..15.
    const int ncol = lane & 31;
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
#pragma unroll
      for (int j = 0; j < T::FN; ++j) {
        const int n = n0 + wn * T::TN + j * 32 + ncol;
        const int mb = m0 + wm * T::TM + i * 32 + 4 * half;
        if (n < N) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = mb + 8 * (r >> 2) + (r & 3);
            if (m < M) C[(size_t)m * N + n] = to_bf16(acc[i][j][r]);
          }
        }
      }
    }
  }
  hooks_end(tr, t0);
}

}  // namespace
}  // namespace occ
