// Types and tile geometry shared by the GEMM kernels (included by gemm.hip only).
#pragma once

#include "device_util.h"
#include "occ_internal.h"

namespace occ {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));  // round to nearest even
}

// ---------------------------------------------------------------------------
// Tiled kernel.  A workgroup owns a BM x BN output tile; WM x WN waves each
// own a (BM/WM) x (BN/WN) sub-tile made of 32x32 MFMA blocks.  Each k-step of
// BK is staged into LDS ([rows][BK] bf16, 16-byte chunks XOR-swizzled by row
// so that the 32 rows of an MFMA operand read hit distinct banks), with the
// next k-step's global loads in flight in registers while the current one is
// multiplied.  STAGES = 2 double-buffers the LDS (one barrier per k-step).
template <int BM_, int BN_, int BK_, int WM_, int WN_, int STAGES_, bool PIPE_ = false, int MINB_ = 1,
          bool BKN_ = false>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_, STAGES = STAGES_;
  static constexpr bool PIPE = PIPE_;  // enforce LDS-read / MFMA interleaving
  static constexpr int MINB = MINB_;   // workgroups per CU the register budget must allow
  // B stored K x N (N-contiguous) instead of N x K: its LDS tile is BK rows of
  // BN columns and MFMA fragments are read with LDS transpose reads
  // (direct-to-LDS kernel only)
  static constexpr bool BKN = BKN_;
  static constexpr int NT = 64 * WM * WN;
  static constexpr int TM = BM / WM, TN = BN / WN;
  static constexpr int FM = TM / 32, FN = TN / 32;
  static constexpr int KCH = BK / 8;              // 16-byte chunks per tile row
  static constexpr int ROWS_PER_PASS = NT / KCH;  // rows the workgroup loads per pass
  static constexpr int BCH = BN / 8;              // 16-byte chunks per K x N B row
  static constexpr int B_RPP = BKN ? NT / BCH : ROWS_PER_PASS;  // B rows per pass
  static constexpr int BROW_BYTES = BN * 2;       // K x N B row in LDS
  static constexpr int A_LOADS = BM / ROWS_PER_PASS;
  static constexpr int B_LOADS = BKN ? BK / B_RPP : BN / ROWS_PER_PASS;
  static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile must be whole 32x32 blocks");
  static_assert(KCH == 4 || KCH == 8, "BK must be 32 or 64");
  static_assert(A_LOADS >= 1 && B_LOADS >= 1, "tile too small for the workgroup");
  static_assert(BM % ROWS_PER_PASS == 0, "uneven load passes");
  static_assert(BKN ? (BK % B_RPP == 0 && B_RPP % 4 == 0 && (BCH >= 16 || BCH == 8))
                    : (BN % ROWS_PER_PASS == 0),
                "uneven load passes");
};

// Physical 16-byte chunk of logical chunk c in tile row r.  The LDS has 64
// banks (256 bytes) and serves a 16-byte-per-lane read 16 lanes at a time;
// an MFMA operand read sends 16 consecutive rows at one logical chunk per
// pass.  Rows are 16*KCH bytes long, so 256/(16*KCH) consecutive rows share a
// bank line at different offsets; XOR-ing the chunk index with the row's
// line number makes all 16 rows of a pass land on distinct banks.  Stores
// (KCH consecutive lanes per row, whole rows per pass) stay conflict-free.
template <int KCH>
__device__ __forceinline__ int swz(int r, int c) {
  if constexpr (KCH == 8) return c ^ ((r >> 1) & 7);
  else return c ^ ((r >> 2) & 3);
}

// Physical 16-byte chunk of logical chunk c in row k of a K x N B tile
// (BCH chunks per row).  A transpose read sends, per 32 lanes, 4 consecutive
// rows at one 64-byte column piece.  Rows of BN*2 >= 256 bytes (BCH >= 16)
// would all hit the same banks: XOR-ing the chunk with 4*(k % 4) moves the 4
// pieces to 4 different 64-byte quarters of the bank line.  Rows of 128 bytes
// (BCH == 8, a 64-column tile) pair up in one bank line, so rows k and k+2
// collide: XOR-ing the chunk with 4 for the second pair of the group swaps
// its two 64-byte halves, and the 4 pieces again fill 4 different quarters.
template <int BCH>
__device__ __forceinline__ int swz_kn(int k, int c) {
  if constexpr (BCH >= 16) return c ^ ((k & 3) << 2);
  else return c ^ ((k & 2) << 1);
}

// XCD-aware order: dispatch hands consecutive workgroups to the 8 XCDs in
// turn, so tile ids are regrouped to give each XCD a contiguous run of the
// grouped order below (and thus shared A/B panels in its own L2).
__device__ __forceinline__ int xcd_remap(int t, int n) {
  int full = n & ~7;
  if (t >= full) return t;
  return (t & 7) * (full >> 3) + (t >> 3);
}

// Grouped tile order: GROUP tile-rows at a time, column-major inside a group.
template <int GROUP>
__device__ __forceinline__ void tile_coords(int id, int tiles_m, int tiles_n, int &tm, int &tn) {
  int per_group = GROUP * tiles_n;
  int g = id / per_group;
  int first = g * GROUP;
  int gs = min(tiles_m - first, GROUP);
  int in = id - g * per_group;
  tm = first + in % gs;
  tn = in / gs;
}

}  // namespace
}  // namespace occ
