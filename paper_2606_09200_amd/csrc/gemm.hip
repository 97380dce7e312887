// K_g: bf16 GEMM on MFMA (gfx950), fp32 accumulation, bf16 output.
//
// Background, item 1: C = A * B, the GEMM of a linear layer, tiled and staged
// through on-chip memory.  Section 3.1: the LDS a workgroup allocates,
// S_blk ~ TILE_M*TILE_K + TILE_K*TILE_N, bounds how many GEMM workgroups
// reside on a CU; an extra dynamic-LDS pad on top of the tile's own LDS lowers
// that residency without changing the kernel's arithmetic.
//
// Layout: A is M x K and C is M x N, row-major.  B is stored K x N (occ_gemm:
// C = A * B, the B tile is staged as stored and read with LDS transpose
// reads) or N x K (occ_gemm_bt: C = A * B^T, a linear layer's weight layout,
// both MFMA operands read from LDS as 16-byte rows).
//
// The kernels live in gemm_dl.h (direct-to-LDS tiles, both layouts),
// gemm_tiled.h (register-staged tiles, the paper's opt1/opt2 with B N x K),
// gemm_skinny.h and gemm_skinny_ldsb.h (M <= 16, B N x K) and
// gemm_skinny_kn.h (M <= 16, B K x N); this file holds the variant table, the
// launch plan and the launcher.
#include "gemm_dl.h"
#include "gemm_skinny.h"
#include "gemm_skinny_kn.h"
#include "gemm_skinny_ldsb.h"
#include "gemm_tiled.h"

#include <algorithm>

namespace occ {
namespace {

// ---------------------------------------------------------------------------
// Variant table.
typedef void (*TiledFn)(const uint16_t *, const uint16_t *, uint16_t *, int, int, int, int, int,
                        int, KHooks);

typedef void (*SkinnyFn)(const uint16_t *, const uint16_t *, uint16_t *, int, int, int, int, KHooks);

struct Variant {
  int id;
  int bm, bn, bk, threads, lds;
  TiledFn fn;        // tiled kernels
  SkinnyFn skinny;   // skinny kernels (M <= 16)
  const char *name;
  int kmax;          // largest K the kernel takes (0 = any)
  int kmult;         // K must be a multiple of this (0 = any)
  bool b_kn;         // takes B stored K x N (and only that)
  int nmax;          // largest N the kernel takes (0 = any)
  int per_cu;        // skinny kernels: persistent workgroups per CU (0 = 1)
};

template <class T>
constexpr Variant make_variant(int id, const char *name) {
  return Variant{id, T::BM, T::BN, T::BK, T::NT, T::LDS_BYTES, gemm_tiled_kernel<T>, nullptr, name, 0, 0, false, 0};
}

// The direct-to-LDS kernel addresses an operand tile with 32-bit byte
// offsets from the tile's first row (row * K * 2 + k * 2) and marks missing
// k with an offset of 2^31: K is capped so that a tile spans at most 2^31
// bytes (no offset wraps and every marked offset is out of range).
template <class T>
constexpr int dl_kmax() {
  return (int)((0x80000000ull / (2ull * (unsigned long long)(T::BM > T::BN ? T::BM : T::BN))) & ~7ull);
}

// A K x N B k-step (BK rows of N) is addressed the same way with N in place of K.
template <class T>
constexpr int dl_nmax() {
  return T::BKN ? (int)((0x80000000ull / (2ull * (unsigned long long)T::BK)) & ~7ull) : 0;
}

template <class T>
constexpr Variant make_dl_variant(int id, const char *name) {
  return Variant{id, T::BM, T::BN, T::BK, T::NT, T::LDS_BYTES, gemm_dl_kernel<T>, nullptr, name,
                 dl_kmax<T>(), 0, T::BKN, dl_nmax<T>()};
}

template <int WAVES, int UNROLL>
constexpr Variant make_skinny_variant(int id, const char *name) {
  return Variant{id, 16, 16, kSkinnyKB * UNROLL, 64 * WAVES, (WAVES - 1) * 64 * 16, nullptr,
                 gemm_skinny_kernel<WAVES, UNROLL>, name, 0, 0, false, 0};
}

// A K x N B block (32 rows of N) is addressed with 32-bit offsets from its
// first row (columns past N marked with 2^31), an A row (M <= 16 rows of K)
// likewise from A.
template <int WAVES, int STAGES, int COLS>
constexpr Variant make_skinny_kn_variant(int id, const char *name) {
  return Variant{id, 16, COLS, kSknKB, 64 * WAVES, SkinnyKn<WAVES, STAGES, COLS>::LDS_BYTES, nullptr,
                 gemm_skinny_kn_kernel<WAVES, STAGES, COLS>, name, (int)((0x80000000ull / 32u) & ~7ull), 0,
                 true, (int)((0x80000000ull / (2u * kSknKB)) & ~7ull), 2};
}

// B staged through LDS in 128-k blocks, A in registers: K a multiple of
// 128 * WAVES, at most 32 * WAVES * KBW.
template <int WAVES, int STAGES, int KBW>
constexpr Variant make_skinny_ldsb_variant(int id, const char *name) {
  return Variant{id, 16, 16, kSlbKB, 64 * WAVES, SkinnyLdsB<WAVES, STAGES, KBW>::LDS_BYTES, nullptr,
                 gemm_skinny_ldsb_kernel<WAVES, STAGES, KBW>, name, 32 * WAVES * KBW, kSlbKB * WAVES, false, 0, 1};
}

// B stored N x K (occ_gemm_bt)
using T64x64_opt1 = Tile<64, 64, 32, 2, 2, 1>;   // Table 1 opt1: 64x64x32
using T64x64_opt2 = Tile<64, 64, 64, 2, 2, 1>;   // Table 1 opt2: 64x64x64
// the opt2 tile with two direct-to-LDS stages: the automatic choice for small
// shapes (one k-step's DMA in flight while the previous one is used)
using D64x64_4w_2s = Tile<64, 64, 64, 2, 2, 2>;
using D128x128_4w_3s = Tile<128, 128, 64, 2, 2, 3>;
using P256x256_8w_2s = Tile<256, 256, 64, 2, 4, 2, true>;
// two workgroups per CU: each has its own barriers, so one computes while the
// other waits (48 KiB of LDS, 4 waves of 128x64 each)
using P128x256k32_4w_2s = Tile<128, 256, 32, 1, 4, 2, true, 2>;

// B stored K x N (occ_gemm): the same tiles with the B tile staged as stored
// and its MFMA operands read with LDS transpose reads
using PKN256x256_8w_2s = Tile<256, 256, 64, 2, 4, 2, true, 1, true>;
using KN128x128_4w_3s = Tile<128, 128, 64, 2, 2, 3, false, 1, true>;
using KN64x64_opt1 = Tile<64, 64, 32, 2, 2, 1, false, 1, true>;   // Table 1 opt1, one stage
using KN64x64_opt2 = Tile<64, 64, 64, 2, 2, 1, false, 1, true>;   // Table 1 opt2, one stage
using KN64x64_4w_2s = Tile<64, 64, 64, 2, 2, 2, false, 1, true>;
using PKN128x256k32_4w_2s = Tile<128, 256, 32, 1, 4, 2, true, 2, true>;

const Variant kVariants[] = {
    // B stored N x K
    make_variant<T64x64_opt1>(6, "64x64x32 opt1, B N x K"),
    make_variant<T64x64_opt2>(7, "64x64x64 opt2, B N x K"),
    make_dl_variant<D64x64_4w_2s>(9, "dl 64x64x64 4w 2st, B N x K"),
    make_dl_variant<D128x128_4w_3s>(14, "dl 128x128x64 4w 3st, B N x K"),
    make_dl_variant<P256x256_8w_2s>(16, "dl+pipe 256x256x64 8w 2st, B N x K"),
    make_skinny_variant<8, 8>(21, "skinny M<=16, 8 waves, unroll 8, B N x K"),
    make_dl_variant<P128x256k32_4w_2s>(25, "dl+pipe 128x256x32 4w 2st 2wg/cu, B N x K"),
    make_skinny_ldsb_variant<8, 2, 32>(34, "skinny M<=16, B via LDS in 256-byte row pieces, A in registers, 8 waves, K<=8192, K%1024==0, B N x K"),
    // B stored K x N
    make_dl_variant<PKN256x256_8w_2s>(32, "dl+pipe 256x256x64 8w 2st, B K x N"),
    make_skinny_kn_variant<4, 2, 128>(33, "skinny M<=16, 128-column units, 4 waves, 2 LDS stages, B K x N"),
    make_dl_variant<KN128x128_4w_3s>(35, "dl 128x128x64 4w 3st, B K x N"),
    make_dl_variant<KN64x64_opt1>(36, "dl 64x64x32 opt1 1st, B K x N"),
    make_dl_variant<KN64x64_opt2>(37, "dl 64x64x64 opt2 1st, B K x N"),
    make_dl_variant<PKN128x256k32_4w_2s>(38, "dl+pipe 128x256x32 4w 2st 2wg/cu, B K x N"),
    make_dl_variant<KN64x64_4w_2s>(39, "dl 64x64x64 4w 2st, B K x N"),
};

constexpr int kMaxVariantId = 63;  // launch-attribute caches are indexed by id
constexpr int kMaxDevices = 64;    // and by device

bool is_skinny(const Variant *v) { return v->skinny != nullptr; }

const Variant *find_variant(int id) {
  for (const Variant &v : kVariants)
    if (v.id == id) return &v;
  return nullptr;
}

int ceil_div(long long a, long long b) { return (int)((a + b - 1) / b); }

// The kernel for a shape: skinny for M <= 16, else the largest tile that
// still gives at least one 256x256 tile per CU (or one 128x128 tile per two
// CUs), else the 64x64x64 tile with two stages.  A K beyond what a
// direct-to-LDS tile addresses with 32-bit offsets takes the 64x64 tile, and
// beyond that (B N x K) the register-staged opt2 tile.
int auto_variant(int M, int N, int K, int num_cus, bool b_kn) {
  if (M <= 16) {
    if (b_kn) return 33;
    // A kept in registers and B staged through LDS when K is whole
    // 1024-wide slices that fit, else 8 k-blocks of A and B in flight per lane
    if (K >= 1024 && K % 1024 == 0 && K <= 8192) return 34;
    return 21;
  }
  const int large = b_kn ? 32 : 16, mid = b_kn ? 35 : 14, small = b_kn ? 39 : 9;
  long long big = (long long)ceil_div(M, 256) * ceil_div(N, 256);
  long long mids = (long long)ceil_div(M, 128) * ceil_div(N, 128);
  int v = big >= num_cus ? large : (mids >= num_cus / 2 ? mid : small);
  const Variant *pv = find_variant(v);
  if (pv->kmax > 0 && K > pv->kmax) {
    v = small;
    pv = find_variant(v);
    if (pv->kmax > 0 && K > pv->kmax && !b_kn) v = 7;
  }
  return v;
}

}  // namespace

bool gemm_variant_is_kn(int id) {
  const Variant *v = find_variant(id);
  return v != nullptr && v->b_kn;
}

static int fill_plan(const GemmCall &c, int variant, const DeviceInfo &di, occ_gemm_plan *p) {
  const Variant *v = find_variant(variant);
  if (v == nullptr) return OCC_EINVAL;
  const bool skinny = is_skinny(v);
  if (skinny && c.M > 16) return OCC_EINVAL;
  if (v->kmax > 0 && c.K > v->kmax) return OCC_EINVAL;
  if (v->kmult > 0 && (c.K == 0 || c.K % v->kmult != 0)) return OCC_EINVAL;
  if (v->b_kn != c.b_kn) return OCC_EINVAL;  // the variant reads B in the other layout
  if (v->nmax > 0 && c.N > v->nmax) return OCC_EINVAL;
  if (v->id < 0 || v->id > kMaxVariantId) return OCC_EINVAL;
  p->tile_m = v->bm;
  p->tile_n = v->bn;
  p->tile_k = v->bk;
  p->threads = v->threads;
  p->tile_lds_bytes = v->lds;
  p->tiles = skinny ? ceil_div(c.N, v->bn) : ceil_div(c.M, v->bm) * ceil_div(c.N, v->bn);
  p->grid = p->tiles;
  const int skinny_grid = di.num_cus * (v->per_cu > 0 ? v->per_cu : 1);
  if (skinny && p->grid > skinny_grid) p->grid = skinny_grid;  // persistent
  if (c.grid_cap > 0 && c.grid_cap < p->grid) p->grid = c.grid_cap;
  p->max_lds_per_wg = di.max_lds_per_wg;
  p->lds_per_cu = di.lds_per_cu;
  p->num_cus = di.num_cus;
  p->kernel_id = variant;
  p->wg_per_cu = 0;
  if (c.lds_bytes > (size_t)di.max_lds_per_wg ||
      (size_t)v->lds + c.lds_bytes > (size_t)di.max_lds_per_wg)
    return OCC_ELDS;
  return OCC_OK;
}

// The launch plan without the occupancy figure: all a launch needs (the
// occupancy query costs host time on every call, which launch-bound
// schedules cannot spare).
int gemm_launch_plan(const GemmCall &c, occ_gemm_plan *plan) {
  const DeviceInfo *di = nullptr;
  int st = current_device_info(&di);
  if (st != OCC_OK) return st;
  int variant = c.variant;
  if (variant == 0) variant = auto_variant(c.M, c.N, c.K, di->num_cus, c.b_kn);
  return fill_plan(c, variant, *di, plan);
}

int gemm_plan(const GemmCall &c, occ_gemm_plan *plan) {
  int st = gemm_launch_plan(c, plan);
  if (st != OCC_OK) return st;
  const Variant *v = find_variant(plan->kernel_id);
  int dyn = (int)(v->fn ? v->lds + c.lds_bytes : c.lds_bytes);
  int nb = 0;
  hipError_t e = v->fn ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, v->fn, v->threads, dyn)
                       : hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, v->skinny, v->threads, dyn);
  if (e != hipSuccess) return OCC_EHIP;
  plan->wg_per_cu = nb;
  return OCC_OK;
}

int gemm_launch(const GemmCall &c, hipStream_t s) {
  occ_gemm_plan p;
  int st = gemm_launch_plan(c, &p);
  if (st != OCC_OK) return st;
  if (c.M == 0 || c.N == 0) return OCC_OK;
  const Variant *v = find_variant(p.kernel_id);
  const uint16_t *A = static_cast<const uint16_t *>(c.A);
  const uint16_t *B = static_cast<const uint16_t *>(c.B);
  uint16_t *C = static_cast<uint16_t *>(c.C);
  // the dynamic-LDS limit is a per-device attribute of each kernel: set it
  // once per device and variant
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return OCC_ENODEV;
  if (v->fn) {
    int dyn = v->lds + (int)c.lds_bytes;
    static bool attr_set[kMaxDevices][kMaxVariantId + 1] = {};
    if (!attr_set[dev][v->id]) {
      if (hipFuncSetAttribute(reinterpret_cast<const void *>(v->fn),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              p.max_lds_per_wg) != hipSuccess)
        return OCC_EHIP;
      attr_set[dev][v->id] = true;
    }
    int tiles_m = ceil_div(c.M, v->bm), tiles_n = ceil_div(c.N, v->bn);
    hipLaunchKernelGGL(v->fn, dim3(p.grid), dim3(v->threads), dyn, s, A, B, C, c.M, c.N, c.K,
                       tiles_m, tiles_n, c.priority, c.trace);
  } else {
    static bool attr_set_skinny[kMaxDevices][kMaxVariantId + 1] = {};
    if (!attr_set_skinny[dev][v->id]) {
      if (hipFuncSetAttribute(reinterpret_cast<const void *>(v->skinny),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              p.max_lds_per_wg - v->lds) != hipSuccess)
        return OCC_EHIP;
      attr_set_skinny[dev][v->id] = true;
    }
    hipLaunchKernelGGL(v->skinny, dim3(p.grid), dim3(v->threads), (int)c.lds_bytes, s, A, B, C,
                       c.M, c.N, c.K, c.priority, c.trace);
  }
  return hipGetLastError() == hipSuccess ? OCC_OK : OCC_EHIP;
}

}  // namespace occ
