// K_g: bf16 GEMM C = A * B^T on MFMA (gfx950), fp32 accumulation, bf16 output.
//
// Background, item 1: the GEMM of a linear layer, tiled and staged through
// on-chip memory.  Section 3.1: the LDS a workgroup allocates,
// S_blk ~ TILE_M*TILE_K + TILE_K*TILE_N, bounds how many GEMM workgroups
// reside on a CU; an extra dynamic-LDS pad on top of the tile's own LDS lowers
// that residency without changing the kernel's arithmetic.
//
// Layout: A is M x K, B is N x K (both K-contiguous, so both MFMA operands are
// read from LDS as 16-byte rows), C is M x N, all row-major.
#include "device_util.h"
#include "occ_internal.h"

#include <algorithm>

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
template <int BM_, int BN_, int BK_, int WM_, int WN_, int STAGES_, bool PIPE_ = false, int MINB_ = 1>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_, STAGES = STAGES_;
  static constexpr bool PIPE = PIPE_;  // enforce LDS-read / MFMA interleaving
  static constexpr int MINB = MINB_;   // workgroups per CU the register budget must allow
  static constexpr int NT = 64 * WM * WN;
  static constexpr int TM = BM / WM, TN = BN / WN;
  static constexpr int FM = TM / 32, FN = TN / 32;
  static constexpr int KCH = BK / 8;              // 16-byte chunks per tile row
  static constexpr int ROWS_PER_PASS = NT / KCH;  // rows the workgroup loads per pass
  static constexpr int A_LOADS = BM / ROWS_PER_PASS;
  static constexpr int B_LOADS = BN / ROWS_PER_PASS;
  static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile must be whole 32x32 blocks");
  static_assert(KCH == 4 || KCH == 8, "BK must be 32 or 64");
  static_assert(A_LOADS >= 1 && B_LOADS >= 1, "tile too small for the workgroup");
  static_assert(BM % ROWS_PER_PASS == 0 && BN % ROWS_PER_PASS == 0, "uneven load passes");
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
                                                           int prio, KTrace tr) {
  extern __shared__ __align__(16) unsigned char smem[];  // tile stages, then the unused pad
  set_wave_priority(prio);
  const TraceStart t0 = trace_begin(tr);
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
  trace_end(tr, t0);
}

// ---------------------------------------------------------------------------
// Direct-to-LDS kernel.  Same tile, LDS layout, MFMA loop and epilogue as
// gemm_tiled_kernel, but each k-step of A and B goes from HBM straight into
// LDS with buffer_load_dwordx4 ... lds: no staging registers, no LDS store
// instructions, STAGES-1 k-steps in flight.  A lane's 16 bytes land at
// M0 + 16*lane, so each lane fetches the logical chunk that the XOR swizzle
// places at its slot.  Buffer range checking supplies the zeros: rows past
// M (N) lie beyond the tile panel's num_records, and chunks past K get an
// offset beyond any panel.
typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ i32x4 make_rsrc(const void *base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = (int)(uint32_t)a;
  r[1] = (int)((a >> 32) & 0xFFFFu);  // stride 0: raw buffer, byte offsets
  r[2] = (int)bytes;                  // num_records: loads at offset >= bytes return 0
  r[3] = 0x00020000;                  // data format for untyped buffer access
  r[0] = __builtin_amdgcn_readfirstlane(r[0]);
  r[1] = __builtin_amdgcn_readfirstlane(r[1]);
  r[2] = __builtin_amdgcn_readfirstlane(r[2]);
  return r;
}

// One 16-byte-per-lane DMA into LDS at M0 + 16*lane.  Issued through asm so
// that the wait for it is explicit (wait_vmcnt) rather than a conservative
// full drain before every later LDS read.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(i32x4 rsrc, uint32_t lds_addr, uint32_t voff) {
  // lds_addr and rsrc are wave-uniform; readfirstlane puts them in SGPRs.
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// Wait until at most `ahead` later stages (of `per_stage` loads each) are
// still in flight.
template <int MAXAHEAD, int PER_STAGE>
__device__ __forceinline__ void wait_stages(int ahead) {
  if constexpr (MAXAHEAD <= 0) {
    wait_vmcnt<0>();
  } else {
    if (ahead >= MAXAHEAD) wait_vmcnt<MAXAHEAD * PER_STAGE>();
    else wait_stages<MAXAHEAD - 1, PER_STAGE>(ahead);
  }
}

template <class T>
__global__ __launch_bounds__(T::NT, T::MINB) void gemm_dl_kernel(const uint16_t *__restrict__ A,
                                                        const uint16_t *__restrict__ B,
                                                        uint16_t *__restrict__ C, int M, int N,
                                                        int K, int tiles_m, int tiles_n, int prio,
                                                        KTrace tr) {
  extern __shared__ __align__(16) unsigned char smem[];  // tile stages, then the unused pad
  set_wave_priority(prio);
  const TraceStart t0 = trace_begin(tr);
  constexpr int S = T::STAGES;
  constexpr int PER_STAGE = T::A_LOADS + T::B_LOADS;
  static_assert(T::ROWS_PER_PASS % 16 == 0, "a lane's swizzle must not change between passes");
  constexpr int ROW_BYTES = T::BK * 2;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / T::WN;
  const int wn = wave % T::WN;
  const int ntiles = tiles_m * tiles_n;
  const int nk = (K + T::BK - 1) / T::BK;
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) unsigned char *)smem;

  // This lane's slot in every load pass: row r_in of the pass, physical
  // chunk q; the swizzle is the same for all passes of a lane, so one offset
  // (plus k0) serves every pass: each pass gets a buffer descriptor of its
  // own, based at the pass's first row, whose num_records covers only the
  // pass's rows that exist.
  const int r_in = threadIdx.x / T::KCH;
  const int q = threadIdx.x % T::KCH;
  const int c = q ^ (swz<T::KCH>(r_in, 0));
  const uint32_t lane_off = (uint32_t)r_in * (uint32_t)K * 2u + (uint32_t)c * 16u;
  const uint32_t wave_lds = (uint32_t)wave * 1024u;

  for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
    int tm, tn;
    tile_coords<8>(xcd_remap(t, ntiles), tiles_m, tiles_n, tm, tn);
    const int m0 = tm * T::BM;
    const int n0 = tn * T::BN;

    auto pass_rsrc = [&](const uint16_t *base, int row0, int rows) {
      const int have = min(T::ROWS_PER_PASS, max(0, rows - row0));
      return make_rsrc(base + (size_t)row0 * K, (uint32_t)have * (uint32_t)K * 2u);
    };
    auto issue = [&](int kt) {
      const int k0 = kt * T::BK;
      const uint32_t sbase = lds0 + (uint32_t)((kt % S) * T::STAGE_BYTES) + wave_lds;
      const uint32_t v = (k0 + c * 8 < K) ? lane_off + (uint32_t)k0 * 2u : 0x80000000u;
#pragma unroll
      for (int p = 0; p < T::A_LOADS; ++p)
        lds_dma16(pass_rsrc(A, m0 + p * T::ROWS_PER_PASS, M), sbase + (uint32_t)(p * T::ROWS_PER_PASS * ROW_BYTES), v);
#pragma unroll
      for (int p = 0; p < T::B_LOADS; ++p)
        lds_dma16(pass_rsrc(B, n0 + p * T::ROWS_PER_PASS, N),
                  sbase + (uint32_t)(T::A_BYTES + p * T::ROWS_PER_PASS * ROW_BYTES), v);
    };

    f32x16 acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
      for (int j = 0; j < T::FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

#pragma unroll
    for (int s = 0; s < S - 1; ++s)
      if (s < nk) issue(s);

    const int arow = wm * T::TM + (lane & 31);
    const int brow = wn * T::TN + (lane & 31);
    const int half = lane >> 5;

    for (int kt = 0; kt < nk; ++kt) {
      // k-step kt has landed once at most min(S-2, nk-1-kt) later steps are
      // outstanding; the barrier then publishes it and retires step kt-1.
      wait_stages<S - 2, PER_STAGE>(min(S - 2, nk - 1 - kt));
      __syncthreads();
      if (kt + S - 1 < nk) issue(kt + S - 1);

      // Fragments of 16-wide k-substep ks+1 are read from LDS while the MFMAs
      // of substep ks run (two register sets); the scheduling groups below
      // interleave one LDS read after each MFMA.
      const unsigned char *cur = smem + (kt % S) * T::STAGE_BYTES;
      constexpr int KS = T::BK / 16;
      bf16x8 af[2][T::FM], bfr[2][T::FN];
      auto load_frags = [&](int ks, bf16x8(&fa)[T::FM], bf16x8(&fb)[T::FN]) {
        const int cc = ks * 2 + half;
#pragma unroll
        for (int i = 0; i < T::FM; ++i) {
          int r = arow + i * 32;
          fa[i] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4 *>(cur + r * ROW_BYTES + swz<T::KCH>(r, cc) * 16));
        }
        const unsigned char *bs = cur + T::A_BYTES;
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
          int r = brow + j * 32;
          fb[j] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4 *>(bs + r * ROW_BYTES + swz<T::KCH>(r, cc) * 16));
        }
      };
      load_frags(0, af[0], bfr[0]);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 1 < KS) load_frags(ks + 1, af[(ks + 1) & 1], bfr[(ks + 1) & 1]);
#pragma unroll
        for (int i = 0; i < T::FM; ++i)
#pragma unroll
          for (int j = 0; j < T::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks & 1][i], bfr[ks & 1][j], acc[i][j], 0, 0, 0);
      }
      if constexpr (T::PIPE) {
        constexpr int NF = T::FM + T::FN;      // LDS reads per substep
        constexpr int NMF = T::FM * T::FN;     // MFMAs per substep
        __builtin_amdgcn_sched_group_barrier(0x100, NF, 0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (ks + 1 < KS) {
#pragma unroll
            for (int x = 0; x < NF; ++x) {
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            if constexpr (NMF > NF) __builtin_amdgcn_sched_group_barrier(0x008, NMF - NF, 0);
          } else {
            __builtin_amdgcn_sched_group_barrier(0x008, NMF, 0);
          }
        }
      }
    }
    __syncthreads();  // every wave is done with the stages before the next tile's prologue

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
        // keep the accumulator reads of one block next to its stores (the
        // scheduler would otherwise hoist all of them and exhaust registers)
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  trace_end(tr, t0);
}

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

// ---------------------------------------------------------------------------
// Variant table.
typedef void (*TiledFn)(const uint16_t *, const uint16_t *, uint16_t *, int, int, int, int, int,
                        int, KTrace);

typedef void (*SkinnyFn)(const uint16_t *, const uint16_t *, uint16_t *, int, int, int, int, KTrace);

struct Variant {
  int id;
  int bm, bn, bk, threads, lds;
  TiledFn fn;        // tiled kernels
  SkinnyFn skinny;   // skinny kernels (M <= 16)
  const char *name;
  int kmax;          // largest K the kernel takes (0 = any)
  int kmult;         // K must be a multiple of this (0 = any)
};

template <class T>
constexpr Variant make_variant(int id, const char *name) {
  return Variant{id, T::BM, T::BN, T::BK, T::NT, T::LDS_BYTES, gemm_tiled_kernel<T>, nullptr, name, 0, 0};
}

template <class T>
constexpr Variant make_dl_variant(int id, const char *name) {
  return Variant{id, T::BM, T::BN, T::BK, T::NT, T::LDS_BYTES, gemm_dl_kernel<T>, nullptr, name, 0, 0};
}

template <int WAVES, int UNROLL>
constexpr Variant make_skinny_variant(int id, const char *name) {
  return Variant{id, 16, 16, kSkinnyKB * UNROLL, 64 * WAVES, (WAVES - 1) * 64 * 16, nullptr,
                 gemm_skinny_kernel<WAVES, UNROLL>, name, 0, 0};
}

template <int WAVES, int KBW, int UNROLL>
constexpr Variant make_skinny_areg_variant(int id, const char *name) {
  return Variant{id, 16, 16, kSkinnyKB * UNROLL, 64 * WAVES, 2 * (WAVES - 1) * 64 * 16, nullptr,
                 gemm_skinny_areg_kernel<WAVES, KBW, UNROLL>, name, WAVES * KBW * kSkinnyKB,
                 2 * WAVES * kSkinnyKB * UNROLL};
}

using T256x256_4w = Tile<256, 256, 64, 2, 2, 2>;
using T256x256_8w = Tile<256, 256, 64, 2, 4, 2>;
using T256x128_4w = Tile<256, 128, 64, 2, 2, 2>;
using T256x128_4w_1s = Tile<256, 128, 64, 2, 2, 1>;
using T128x128_4w = Tile<128, 128, 64, 2, 2, 2>;
using T64x64_opt1 = Tile<64, 64, 32, 2, 2, 1>;   // Table 1 opt1: 64x64x32
using T64x64_opt2 = Tile<64, 64, 64, 2, 2, 1>;   // Table 1 opt2: 64x64x64
using T256x256_k32_1s = Tile<256, 256, 32, 2, 2, 1>;
using D256x256_8w_2s = Tile<256, 256, 64, 2, 4, 2>;
using D256x256k32_8w_4s = Tile<256, 256, 32, 2, 4, 4>;
using D256x256k32_8w_3s = Tile<256, 256, 32, 2, 4, 3>;
using D256x128_4w_3s = Tile<256, 128, 64, 2, 2, 3>;
using D128x128_4w_3s = Tile<128, 128, 64, 2, 2, 3>;
using D256x128_8w_3s = Tile<256, 128, 64, 4, 2, 3>;
using P256x256_8w_2s = Tile<256, 256, 64, 2, 4, 2, true>;
using P256x256k32_8w_4s = Tile<256, 256, 32, 2, 4, 4, true>;
using P256x128_4w_3s = Tile<256, 128, 64, 2, 2, 3, true>;
using P256x256_4w_2s = Tile<256, 256, 64, 2, 2, 2, true>;
// two workgroups per CU: each has its own barriers, so one computes while the
// other waits (48-72 KiB of LDS, 4 waves of 128x64 each)
using P256x128k32_4w_2s = Tile<256, 128, 32, 2, 2, 2, true, 2>;
using P128x256k32_4w_2s = Tile<128, 256, 32, 1, 4, 2, true, 2>;
using P256x128k32_4w_3s = Tile<256, 128, 32, 2, 2, 3, true, 2>;
using P128x256k32_4w_3s = Tile<128, 256, 32, 1, 4, 3, true, 2>;

constexpr int kSkinnyId = 8;

const Variant kVariants[] = {
    make_variant<T256x256_4w>(1, "256x256x64 4w 2st"),
    make_variant<T256x256_8w>(2, "256x256x64 8w 2st"),
    make_variant<T256x128_4w>(3, "256x128x64 4w 2st"),
    make_variant<T256x128_4w_1s>(4, "256x128x64 4w 1st"),
    make_variant<T128x128_4w>(5, "128x128x64 4w 2st"),
    make_variant<T64x64_opt1>(6, "64x64x32 opt1"),
    make_variant<T64x64_opt2>(7, "64x64x64 opt2"),
    make_skinny_variant<4, 16>(kSkinnyId, "skinny M<=16, 4 waves"),
    make_variant<T256x256_k32_1s>(9, "256x256x32 4w 1st"),
    make_dl_variant<D256x256_8w_2s>(10, "dl 256x256x64 8w 2st"),
    make_dl_variant<D256x256k32_8w_4s>(11, "dl 256x256x32 8w 4st"),
    make_dl_variant<D256x256k32_8w_3s>(12, "dl 256x256x32 8w 3st"),
    make_dl_variant<D256x128_4w_3s>(13, "dl 256x128x64 4w 3st"),
    make_dl_variant<D128x128_4w_3s>(14, "dl 128x128x64 4w 3st"),
    make_dl_variant<D256x128_8w_3s>(15, "dl 256x128x64 8w 3st"),
    make_dl_variant<P256x256_8w_2s>(16, "dl+pipe 256x256x64 8w 2st"),
    make_dl_variant<P256x256k32_8w_4s>(17, "dl+pipe 256x256x32 8w 4st"),
    make_dl_variant<P256x128_4w_3s>(18, "dl+pipe 256x128x64 4w 3st"),
    make_dl_variant<P256x256_4w_2s>(19, "dl+pipe 256x256x64 4w 2st"),
    make_skinny_variant<8, 16>(20, "skinny M<=16, 8 waves"),
    make_skinny_variant<8, 8>(21, "skinny M<=16, 8 waves, unroll 8"),
    make_skinny_variant<4, 8>(22, "skinny M<=16, 4 waves, unroll 8"),
    make_skinny_variant<16, 8>(23, "skinny M<=16, 16 waves, unroll 8"),
    make_dl_variant<P256x128k32_4w_2s>(24, "dl+pipe 256x128x32 4w 2st"),
    make_dl_variant<P128x256k32_4w_2s>(25, "dl+pipe 128x256x32 4w 2st"),
    make_dl_variant<P256x128k32_4w_3s>(26, "dl+pipe 256x128x32 4w 3st"),
    make_dl_variant<P128x256k32_4w_3s>(27, "dl+pipe 128x256x32 4w 3st"),
    make_skinny_areg_variant<8, 32, 4>(28, "skinny M<=16, A in registers, 8 waves, K<=8192, K%2048==0"),
    make_skinny_areg_variant<8, 16, 4>(29, "skinny M<=16, A in registers, 8 waves, K<=4096, K%2048==0"),
};

constexpr int kMaxVariantId = 63;  // launch-attribute caches are indexed by id

bool is_skinny(const Variant *v) { return v->skinny != nullptr; }

const Variant *find_variant(int id) {
  for (const Variant &v : kVariants)
    if (v.id == id) return &v;
  return nullptr;
}

int ceil_div(long long a, long long b) { return (int)((a + b - 1) / b); }

int auto_variant(int M, int N, int K, int num_cus) {
  if (M <= 16) {
    // skinny, 8 waves; A kept in registers when K is whole 2048-wide slices
    // that fit, else 8 k-blocks of A and B in flight per lane
    if (K >= 2048 && K % 2048 == 0 && K <= 4096) return 29;
    if (K >= 2048 && K % 2048 == 0 && K <= 8192) return 28;
    return 21;
  }
  long long big = (long long)ceil_div(M, 256) * ceil_div(N, 256);
  if (big >= num_cus) return 16;
  long long mid = (long long)ceil_div(M, 128) * ceil_div(N, 128);
  if (mid >= num_cus / 2) return 5;
  return 7;
}

}  // namespace

static int fill_plan(const GemmCall &c, int variant, const DeviceInfo &di, occ_gemm_plan *p) {
  const Variant *v = find_variant(variant);
  if (v == nullptr) return OCC_EINVAL;
  const bool skinny = is_skinny(v);
  if (skinny && c.M > 16) return OCC_EINVAL;
  if (v->kmax > 0 && c.K > v->kmax) return OCC_EINVAL;
  if (v->kmult > 0 && (c.K == 0 || c.K % v->kmult != 0)) return OCC_EINVAL;
  if (v->id < 0 || v->id > kMaxVariantId) return OCC_EINVAL;
  p->tile_m = v->bm;
  p->tile_n = v->bn;
  p->tile_k = v->bk;
  p->threads = v->threads;
  p->tile_lds_bytes = v->lds;
  p->tiles = skinny ? ceil_div(c.N, 16) : ceil_div(c.M, v->bm) * ceil_div(c.N, v->bn);
  p->grid = p->tiles;
  if (skinny && p->grid > di.num_cus) p->grid = di.num_cus;  // persistent, one per CU
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

int gemm_plan(const GemmCall &c, occ_gemm_plan *plan) {
  const DeviceInfo *di = nullptr;
  int st = current_device_info(&di);
  if (st != OCC_OK) return st;
  int variant = c.variant;
  if (variant == 0) variant = auto_variant(c.M, c.N, c.K, di->num_cus);
  st = fill_plan(c, variant, *di, plan);
  if (st != OCC_OK) return st;
  const Variant *v = find_variant(variant);
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
  int st = gemm_plan(c, &p);
  if (st != OCC_OK) return st;
  if (c.M == 0 || c.N == 0) return OCC_OK;
  const Variant *v = find_variant(p.kernel_id);
  const uint16_t *A = static_cast<const uint16_t *>(c.A);
  const uint16_t *B = static_cast<const uint16_t *>(c.B);
  uint16_t *C = static_cast<uint16_t *>(c.C);
  if (v->fn) {
    int dyn = v->lds + (int)c.lds_bytes;
    static bool attr_set[kMaxVariantId + 1] = {};
    if (!attr_set[v->id]) {
      if (hipFuncSetAttribute(reinterpret_cast<const void *>(v->fn),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              p.max_lds_per_wg) != hipSuccess)
        return OCC_EHIP;
      attr_set[v->id] = true;
    }
    int tiles_m = ceil_div(c.M, v->bm), tiles_n = ceil_div(c.N, v->bn);
    hipLaunchKernelGGL(v->fn, dim3(p.grid), dim3(v->threads), dyn, s, A, B, C, c.M, c.N, c.K,
                       tiles_m, tiles_n, c.priority, c.trace);
  } else {
    static bool attr_set_skinny[kMaxVariantId + 1] = {};
    if (!attr_set_skinny[v->id]) {
      if (hipFuncSetAttribute(reinterpret_cast<const void *>(v->skinny),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              p.max_lds_per_wg - v->lds) != hipSuccess)
        return OCC_EHIP;
      attr_set_skinny[v->id] = true;
    }
    hipLaunchKernelGGL(v->skinny, dim3(p.grid), dim3(v->threads), (int)c.lds_bytes, s, A, B, C,
                       c.M, c.N, c.K, c.priority, c.trace);
  }
  return hipGetLastError() == hipSuccess ? OCC_OK : OCC_EHIP;
}

}  // namespace occ
