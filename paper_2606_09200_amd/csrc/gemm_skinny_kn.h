// Skinny (M <= 16) GEMM kernel for B stored K x N (included by gemm.hip only).
#pragma once

#include "gemm_dl.h"

namespace occ {
namespace {

// ---------------------------------------------------------------------------
// C[M x N] = A[M x K] * B[K x N], M <= 16, HBM-bound on B.  Work unit: COLS
// output columns over the whole K, i.e. a 2*COLS-byte piece of every row of B
// (COLS = 128: 256 bytes, two whole cache lines per row).  The WAVES waves of
// a workgroup split K into contiguous slices of 32-row blocks; each wave
// streams its slice through a private ring of STAGES LDS buffers with
// direct-to-LDS DMA (STAGES - 1 blocks in flight, no barriers between waves
// while streaming):
//
//   block buffer = [A: 16 rows x 64 B][B: 32 rows x 2*COLS B]
//
// A (16 x K, L2-resident) comes through the same DMA, so one counter orders
// both; B's DMA is non-temporal (every B byte is used once).  Measured on
// 16 x 28672 x 8192: 256-byte row pieces stream 15-20 % faster than
// 128-byte ones, and the non-temporal policy adds 7-8 %.  MFMA
// v_mfma_f32_16x16x32_bf16, one per 16-column block per k-block: the A
// operand (lane: row l % 16, k-group l / 16) is a 16-byte LDS read; the B
// operand (lane: column l % 16, 8 consecutive k of k-group l / 16) is two LDS
// transpose reads (each 16-lane group of a transpose read hands lane i
// element j of the 8-byte piece that lane 4j + i/4 addressed, so lanes that
// address 4 columns of 4 consecutive rows give each lane 4 consecutive rows
// of one column).  Rows outside K and columns outside N read as zero through
// the buffer range check; rows of A past M likewise.  The WAVES partial
// 16 x COLS sums are added in wave order through LDS, so the result does not
// depend on timing.  Persistent workgroups loop over units.
constexpr int kSknKB = 32;                   // k rows per block
constexpr int kSknABytes = 16 * kSknKB * 2;  // A part of a block buffer: 1 KiB

// Physical 16-byte chunk of logical chunk c in B row r of a block whose rows
// are ROW_BYTES long.  A transpose read touches, per 32 lanes, 8 rows (r..r+3
// and r+8..r+11) at one 32-byte column piece each; the XOR moves those 8
// pieces to 8 different 32-byte slots of the 256-byte bank line (128-byte
// rows: two rows share a line, so each parity class needs 4 slots).
template <int ROW_BYTES>
__device__ __forceinline__ int swz_skn_b(int r, int c) {
  if constexpr (ROW_BYTES == 256) return c ^ (2 * ((r & 3) | (((r >> 3) & 1) << 2)));
  else return c ^ (2 * (((r >> 1) & 1) | (((r >> 3) & 1) << 1)));
}

// Physical chunk of logical chunk g (8 k) in A row m: an operand read sends
// 16 rows at one chunk; rows are 64 bytes, so rows m and m+4 would collide.
__device__ __forceinline__ int swz_skn_a(int m, int g) { return g ^ ((m >> 2) & 3); }

// lds_dma16 with the non-temporal cache policy.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16_nt(i32x4 rsrc, uint32_t lds_addr, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

template <int WAVES, int STAGES, int COLS>
struct SkinnyKn {
  static constexpr int ROW_BYTES = COLS * 2;               // B row piece of a unit
  static constexpr int CPR = ROW_BYTES / 16;               // 16-byte chunks per row piece
  static constexpr int RPI = 64 / CPR;                     // rows per DMA instruction
  static constexpr int B_BYTES = kSknKB * ROW_BYTES;
  static constexpr int B_LOADS = B_BYTES / 1024;
  static constexpr int LOADS = 1 + B_LOADS;                // DMA instructions per block
  static constexpr int BLOCK_BYTES = kSknABytes + B_BYTES;
  static constexpr int NB16 = COLS / 16;                   // 16-column MFMA blocks
  static constexpr int WAVE_BYTES = STAGES * BLOCK_BYTES;
  static constexpr int LDS_BYTES = WAVES * WAVE_BYTES;
  static_assert(COLS == 64 || COLS == 128, "unit of 64 or 128 columns");
  static_assert(WAVE_BYTES >= NB16 * 64 * 16, "a wave's partial sums must fit its ring");
  static_assert(STAGES >= 2 && (STAGES - 1) * LOADS <= 63, "vmcnt holds at most 63");
};

template <int WAVES, int STAGES, int COLS>
__global__ __launch_bounds__(64 * WAVES) void gemm_skinny_kn_kernel(const uint16_t *__restrict__ A,
                                                                    const uint16_t *__restrict__ B,
                                                                    uint16_t *__restrict__ C, int M,
                                                                    int N, int K, int prio, KHooks tr) {
  using G = SkinnyKn<WAVES, STAGES, COLS>;
  constexpr int S = STAGES;
  __shared__ __align__(16) unsigned char ring[G::LDS_BYTES];
  extern __shared__ __align__(16) unsigned char pad_lds[];  // occupancy pad only
  (void)pad_lds;
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar loop control
  const int nblk = (K + kSknKB - 1) / kSknKB;
  const int b0 = wave * nblk / WAVES, b1 = (wave + 1) * nblk / WAVES;
  const int nb = b1 - b0;
  const int units = (N + COLS - 1) / COLS;
  unsigned char *mine = ring + wave * G::WAVE_BYTES;
  const uint32_t lds_mine = (uint32_t)(size_t)(__attribute__((address_space(3))) unsigned char *)mine;

  // DMA slots.  A: lane l fills row l / 4, physical chunk l % 4.  B
  // instruction q: lane l fills row RPI*q + l / CPR, physical chunk l % CPR.
  const int am = lane >> 2;
  const int ag = swz_skn_a(am, lane & 3);
  const i32x4 rsrc_a = make_rsrc(A, (uint32_t)M * (uint32_t)K * 2u);
  const uint32_t a_row_off = (uint32_t)am * (uint32_t)K * 2u;

  // LDS read offsets inside a block buffer.
  const int s16 = lane & 15, grp = lane >> 4;
  const int a_rd = s16 * 64 + swz_skn_a(s16, grp) * 16;
  int b_rd[2][G::NB16];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = 8 * grp + 4 * h + (s16 >> 2);
#pragma unroll
    for (int j = 0; j < G::NB16; ++j)
      b_rd[h][j] = kSknABytes + r * G::ROW_BYTES + swz_skn_b<G::ROW_BYTES>(r, 2 * j + ((s16 & 3) >> 1)) * 16 +
                   8 * (s16 & 1);
  }

  for (int unit = blockIdx.x; unit < units; unit += gridDim.x) {
    const int n0 = unit * COLS;
    // this lane's offset in B instruction q; columns past N get an offset
    // beyond any block's range
    uint32_t vb[G::B_LOADS];
#pragma unroll
    for (int q = 0; q < G::B_LOADS; ++q) {
      const int r = G::RPI * q + lane / G::CPR;
      const int c = swz_skn_b<G::ROW_BYTES>(r, lane % G::CPR);
      vb[q] = (n0 + 8 * c < N) ? (uint32_t)r * (uint32_t)N * 2u + (uint32_t)c * 16u : 0x80000000u;
    }

    auto issue = [&](int i) {  // block b0 + i into ring slot i % S
      const int k0 = (b0 + i) * kSknKB;
      const uint32_t slot = lds_mine + (uint32_t)((i % S) * G::BLOCK_BYTES);
      const uint32_t va = (k0 + 8 * ag < K) ? a_row_off + (uint32_t)(k0 + 8 * ag) * 2u : 0x80000000u;
      lds_dma16(rsrc_a, slot, va);
      // rows k0 .. k0 + have - 1 of columns n0 .. N - 1 lie inside the range
      const int have = min(kSknKB, K - k0);
      const i32x4 rsrc_b = make_rsrc(B + (size_t)k0 * N + n0, (uint32_t)have * (uint32_t)N * 2u - (uint32_t)n0 * 2u);
#pragma unroll
      for (int q = 0; q < G::B_LOADS; ++q) lds_dma16_nt(rsrc_b, slot + (uint32_t)(kSknABytes + q * 1024), vb[q]);
    };

    f32x4 acc[G::NB16];
#pragma unroll
    for (int j = 0; j < G::NB16; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int i = 0; i < S - 1; ++i)
      if (i < nb) issue(i);
    for (int i = 0; i < nb; ++i) {
      // block i has landed once at most min(S-2, nb-1-i) later blocks are outstanding
      wait_stages<S - 2, G::LOADS>(min(S - 2, nb - 1 - i));
      // the slot refilled next was read in iteration i-1: those reads are done
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      if (i + S - 1 < nb) issue(i + S - 1);
      const unsigned char *buf = mine + (i % S) * G::BLOCK_BYTES;
      const bf16x8 af = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(buf + a_rd));
#pragma unroll
      for (int j = 0; j < G::NB16; ++j) {
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4 *)(buf + b_rd[0][j]));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4 *)(buf + b_rd[1][j]));
        const bf16x8 bfr = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bfr, acc[j], 0, 0, 0);
      }
    }

    // Partial sums through the ring (every block of this unit is consumed).
    if (wave > 0) {
#pragma unroll
      for (int j = 0; j < G::NB16; ++j) *reinterpret_cast<f32x4 *>(mine + (j * 64 + lane) * 16) = acc[j];
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int w = 1; w < WAVES; ++w) {
        const unsigned char *p = ring + w * G::WAVE_BYTES;
#pragma unroll
        for (int j = 0; j < G::NB16; ++j) {
          const f32x4 v = *reinterpret_cast<const f32x4 *>(p + (j * 64 + lane) * 16);
          acc[j][0] = acc[j][0] + v[0];
          acc[j][1] = acc[j][1] + v[1];
          acc[j][2] = acc[j][2] + v[2];
          acc[j][3] = acc[j][3] + v[3];
        }
      }
      // 16x16 MFMA result layout: lane holds column l % 16, rows 4 * (l / 16) + i
#pragma unroll
      for (int j = 0; j < G::NB16; ++j) {
        const int n = n0 + 16 * j + s16;
        if (n < N) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = 4 * grp + i;
            if (m < M) C[(size_t)m * N + n] = to_bf16(acc[j][i]);
          }
        }
      }
    }
    __syncthreads();  // the rings are refilled by the next unit
  }
  hooks_end(tr, t0);
}

}  // namespace
}  // namespace occ
