// Skinny (M <= 16) GEMM kernel with B staged through LDS (included by
// gemm.hip only).
#pragma once

#include "gemm_skinny_kn.h"

namespace occ {
namespace {

// ---------------------------------------------------------------------------
// C[M x N] = A[M x K] * B^T, B stored N x K, M <= 16, HBM-bound on B.  The
// unit and wave split of gemm_skinny_areg_kernel (16 output columns, i.e. 16
// rows of B, over the whole K; WAVES waves with contiguous K-slices; each
// wave's slice of A held in registers for every unit), but B reaches the MFMA
// through LDS: each wave streams its slice in blocks of 16 rows x 128 k with
// direct-to-LDS DMA into a private ring of STAGES buffers, so that one DMA
// instruction reads whole 256-byte pieces of 4 rows (the register kernel's
// loads read 64-byte pieces of 16 rows).  B's DMA is non-temporal.  The ring
// keeps running across unit boundaries (the next unit's first blocks are in
// flight while the current one finishes).  Rows past N read as zero through
// the buffer range check.  The WAVES partial 16x16 sums are added in wave
// order through a double-buffered LDS array (one barrier per unit), so the
// result does not depend on timing.  K must be a multiple of 128 * WAVES and
// at most 32 * WAVES * KBW (checked by the host).
constexpr int kSlbKB = 128;                 // k per block
constexpr int kSlbBlockBytes = 16 * kSlbKB * 2;  // 16 rows x 256 B
constexpr int kSlbLoads = kSlbBlockBytes / 1024;  // DMA instructions per block

// Physical 16-byte chunk of logical chunk c in row r of a block: an operand
// read sends 16 rows at one chunk and rows are one 256-byte bank line long,
// so the XOR with r spreads the 16 rows over all 16 chunk slots.
__device__ __forceinline__ int swz_slb(int r, int c) { return c ^ (r & 15); }

template <int WAVES, int STAGES, int KBW>
struct SkinnyLdsB {
  static constexpr int WAVE_BYTES = STAGES * kSlbBlockBytes;
  static constexpr int RING_BYTES = WAVES * WAVE_BYTES;
  static constexpr int PART_BYTES = 2 * (WAVES - 1) * 64 * 16;
  static constexpr int LDS_BYTES = RING_BYTES + PART_BYTES;
  static_assert(KBW % 4 == 0, "A slice in whole blocks");
  static_assert(STAGES >= 2 && (STAGES - 1) * kSlbLoads <= 63, "vmcnt holds at most 63");
};

template <int WAVES, int STAGES, int KBW>
__global__ __launch_bounds__(64 * WAVES) void gemm_skinny_ldsb_kernel(const uint16_t *__restrict__ A,
                                                                      const uint16_t *__restrict__ B,
                                                                      uint16_t *__restrict__ C, int M,
                                                                      int N, int K, int prio, KHooks tr) {
  using G = SkinnyLdsB<WAVES, STAGES, KBW>;
  constexpr int S = STAGES;
  constexpr int NBW = KBW / 4;  // most blocks per wave and unit
  __shared__ __align__(16) unsigned char ring[G::RING_BYTES];
  __shared__ f32x4 partial[2][WAVES - 1][64];
  extern __shared__ __align__(16) unsigned char pad_lds[];  // occupancy pad only
  (void)pad_lds;
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar loop control
  const int r = lane & 15;
  const int g = lane >> 4;
  const int bpw = K / (32 * WAVES);  // 32-wide k-blocks per wave (a multiple of 4, <= KBW)
  const int nbw = bpw / 4;           // LDS blocks per wave and unit
  const int units = (N + 15) / 16;
  const int kslice = wave * bpw * 32;
  unsigned char *mine = ring + wave * G::WAVE_BYTES;
  const uint32_t lds_mine = (uint32_t)(size_t)(__attribute__((address_space(3))) unsigned char *)mine;

  // this wave's slice of the 16 A rows: k-block j (32 k) at register a[j],
  // lane holding row r, k 8g..8g+7 of the block
  u32x4 a[KBW];
  {
    const uint16_t *arow = A + (size_t)(r < M ? r : 0) * K + kslice + g * 8;
#pragma unroll
    for (int j = 0; j < KBW; ++j) {
      u32x4 z = {0u, 0u, 0u, 0u};
      if (j < bpw && r < M) z = *reinterpret_cast<const u32x4 *>(arow + j * 32);
      a[j] = z;
    }
  }

  // DMA instruction q of a block: lane l fills row 4q + l / 16, physical
  // chunk l % 16, i.e. logical chunk (l % 16) ^ row.
  uint32_t voff[kSlbLoads];
#pragma unroll
  for (int q = 0; q < kSlbLoads; ++q) {
    const int row = 4 * q + (lane >> 4);
    voff[q] = (uint32_t)row * (uint32_t)K * 2u + (uint32_t)kslice * 2u + (uint32_t)swz_slb(row, lane & 15) * 16u;
  }
  // operand read of k-substep s (32 k): row r, logical chunk 4s + g
  int b_rd[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) b_rd[s] = r * 256 + swz_slb(r, 4 * s + g) * 16;

  // block stream of this workgroup: sequence number t -> unit blockIdx.x +
  // (t / nbw) * gridDim.x, block t % nbw of this wave's slice
  const int my_units = blockIdx.x < units ? (units - 1 - (int)blockIdx.x) / (int)gridDim.x + 1 : 0;
  const int total = my_units * nbw;
  auto issue = [&](int t) {
    const int unit = blockIdx.x + (t / nbw) * gridDim.x;
    const int i = t % nbw;
    const int rows = min(16, N - unit * 16);
    const i32x4 rsrc = make_rsrc(B + (size_t)unit * 16 * K, (uint32_t)rows * (uint32_t)K * 2u);
    const uint32_t slot = lds_mine + (uint32_t)((t % S) * kSlbBlockBytes);
#pragma unroll
    for (int q = 0; q < kSlbLoads; ++q)
      lds_dma16_nt(rsrc, slot + (uint32_t)(q * 1024), voff[q] + (uint32_t)i * (kSlbKB * 2u));
  };

#pragma unroll
  for (int t = 0; t < S - 1; ++t)
    if (t < total) issue(t);
  int t = 0, par = 0;
  for (int unit = blockIdx.x; unit < units; unit += gridDim.x, par ^= 1) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
      if (i < nbw) {
        // block t has landed once at most min(S-2, total-1-t) later blocks are outstanding
        wait_stages<S - 2, kSlbLoads>(min(S - 2, total - 1 - t));
        // the slot refilled next was read one block ago: those reads are done
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if (t + S - 1 < total) issue(t + S - 1);
        const unsigned char *buf = mine + (t % S) * kSlbBlockBytes;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const bf16x8 bf = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(buf + b_rd[s]));
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[4 * i + s]), bf, acc, 0, 0, 0);
        }
        ++t;
      }
    }

    // partial[par] was last read by wave 0 two units ago, before it reached
    // the previous unit's barrier, which every writer has passed since
    if (wave > 0) partial[par][wave - 1][lane] = acc;
    __syncthreads();
    if (wave == 0) {
      f32x4 sum = acc;
#pragma unroll
      for (int w = 0; w < WAVES - 1; ++w) {
        const f32x4 p = partial[par][w][lane];
        sum[0] = sum[0] + p[0];
        sum[1] = sum[1] + p[1];
        sum[2] = sum[2] + p[2];
        sum[3] = sum[3] + p[3];
      }
      // 16x16 MFMA result layout: lane holds column l % 16, rows 4 * (l / 16) + i
      const int n = unit * 16 + r;
      if (n < N) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = 4 * g + i;
          if (m < M) C[(size_t)m * N + n] = to_bf16(sum[i]);
        }
      }
    }
  }
  hooks_end(tr, t0);
}

}  // namespace
}  // namespace occ
