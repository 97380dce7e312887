// Direct-to-LDS tiled GEMM kernel (included by gemm.hip only).
#pragma once

#include "gemm_common.h"

namespace occ {
namespace {

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
typedef short i16x4 __attribute__((ext_vector_type(4)));

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
                                                        KHooks tr) {
  extern __shared__ __align__(16) unsigned char smem[];  // tile stages, then the unused pad
  set_wave_priority(prio);
  const HookStart t0 = hooks_begin(tr);
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
  // chunk q; the swizzle is the same for all passes of a lane.  Each operand
  // tile is read through one buffer descriptor based at the tile's first row
  // whose num_records covers only the rows that exist; pass p adds
  // p * ROWS_PER_PASS rows to the lane's offset (a VALU add against a uniform
  // step, so that issuing a pass needs no scalar work that waits on vector
  // results).  Offsets stay below 2^31 (the variant's K limit).
  const int r_in = threadIdx.x / T::KCH;
  const int q = threadIdx.x % T::KCH;
  const int c = q ^ (swz<T::KCH>(r_in, 0));
  const uint32_t lane_off = (uint32_t)r_in * (uint32_t)K * 2u + (uint32_t)c * 16u;
  const uint32_t pass_step = (uint32_t)T::ROWS_PER_PASS * (uint32_t)K * 2u;
  const uint32_t wave_lds = (uint32_t)__builtin_amdgcn_readfirstlane(wave) * 1024u;
  // K x N B: this lane's slot in every B pass, row rB of the pass and
  // physical chunk qB; passes start at multiples of 4 rows, so the logical
  // chunk qB ^ swz is the same in every pass.
  const int rB = threadIdx.x / T::BCH;
  const int cB = swz_kn<T::BCH>(rB, threadIdx.x % T::BCH);
  // K x N B fragment reads (transpose reads, see below): within each group of
  // 16 lanes, lane s reads 4 consecutive columns at row (s / 4) of a 4-row
  // block; the hardware hands lane i of the group element j of lane
  // 4 * j + i / 4, i.e. 4 consecutive k of column i.
  const int tr_k = 8 * ((lane >> 4) >> 1) + ((lane & 15) >> 2);
  const int tr_n = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
    int tm, tn;
    tile_coords<8>(xcd_remap(t, ntiles), tiles_m, tiles_n, tm, tn);
    const int m0 = tm * T::BM;
    const int n0 = tn * T::BN;

    const i32x4 rsrc_a = make_rsrc(A + (size_t)m0 * K, (uint32_t)min(T::BM, M - m0) * (uint32_t)K * 2u);
    const i32x4 rsrc_b = T::BKN ? rsrc_a : make_rsrc(B + (size_t)n0 * K, (uint32_t)min(T::BN, N - n0) * (uint32_t)K * 2u);
    // K x N B: columns past N read as zero through an out-of-range offset,
    // rows past K through the k-step's num_records
    const uint32_t vb = (n0 + cB * 8 < N) ? (uint32_t)rB * (uint32_t)N * 2u + (uint32_t)(n0 + cB * 8) * 2u
                                          : 0x80000000u;
    (void)vb;
    // DMA pass p of k-step kt: A passes first, then B passes.  A k-step past
    // K loads nothing and writes zeros (every offset is out of range).
    auto issue_pass = [&](int kt, int p) {
      const int k0 = kt * T::BK;
      const uint32_t sbase = lds0 + (uint32_t)((kt % S) * T::STAGE_BYTES) + wave_lds;
      const uint32_t v = (k0 + c * 8 < K) ? lane_off + (uint32_t)k0 * 2u : 0x80000000u;
      if (p < T::A_LOADS) {
        lds_dma16(rsrc_a, sbase + (uint32_t)(p * T::ROWS_PER_PASS * ROW_BYTES), v + (uint32_t)p * pass_step);
      } else if constexpr (T::BKN) {
        const int q = p - T::A_LOADS;
        const int have = min(T::BK, max(0, K - k0));
        lds_dma16(make_rsrc(B + (size_t)k0 * N, (uint32_t)have * (uint32_t)N * 2u),
                  sbase + (uint32_t)(T::A_BYTES + q * T::B_RPP * T::BROW_BYTES),
                  vb + (uint32_t)(q * T::B_RPP) * (uint32_t)N * 2u);
      } else {
        const int q = p - T::A_LOADS;
        lds_dma16(rsrc_b, sbase + (uint32_t)(T::A_BYTES + q * T::ROWS_PER_PASS * ROW_BYTES),
                  v + (uint32_t)q * pass_step);
      }
    };
    auto issue = [&](int kt) {
#pragma unroll
      for (int p = 0; p < PER_STAGE; ++p) issue_pass(kt, p);
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

    // MFMA operand fragments of 16-wide k-substep ks of the stage at `cur`
    auto read_a = [&](const unsigned char *cur, int ks, int i) {
      const int r = arow + i * 32;
      return __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4 *>(cur + r * ROW_BYTES + swz<T::KCH>(r, ks * 2 + half) * 16));
    };
    auto read_b = [&](const unsigned char *cur, int ks, int j) {
      const unsigned char *bs = cur + T::A_BYTES;
      if constexpr (T::BKN) {
        const int kr = ks * 16 + tr_k;
        const int n = wn * T::TN + j * 32 + tr_n;
        const int off = swz_kn<T::BCH>(kr, n >> 3) * 16 + (n & 7) * 2;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4 *)(bs + kr * T::BROW_BYTES + off));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4 *)(bs + (kr + 4) * T::BROW_BYTES + off));
        return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      } else {
        const int r = brow + j * 32;
        return __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4 *>(bs + r * ROW_BYTES + swz<T::KCH>(r, ks * 2 + half) * 16));
      }
    };
    constexpr int KS = T::BK / 16;
    constexpr int NF = T::FM + (T::BKN ? 2 : 1) * T::FN;  // LDS reads per substep
    constexpr int NMF = T::FM * T::FN;                     // MFMAs per substep
    bf16x8 af[2][T::FM], bfr[2][T::FN];
    auto load_frags = [&](const unsigned char *cur, int ks, int set) {
#pragma unroll
      for (int i = 0; i < T::FM; ++i) af[set][i] = read_a(cur, ks, i);
#pragma unroll
      for (int j = 0; j < T::FN; ++j) bfr[set][j] = read_b(cur, ks, j);
    };
    auto mfma = [&](int x, int set) {
      const int i = x / T::FN, j = x % T::FN;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[set][i], bfr[set][j], acc[i][j], 0, 0, 0);
    };
    for (int kt = 0; kt < nk; ++kt) {
      // k-step kt has landed once at most min(S-2, nk-1-kt) later steps are
      // outstanding; the barrier then publishes it and retires step kt-1.
      if constexpr (S == 1) {
        // one stage (the paper's tile configurations): every wave is done
        // with the previous k-step before the DMA overwrites it, and the
        // k-step has landed for every wave before any reads it
        __syncthreads();
        issue(kt);
        wait_vmcnt<0>();
        __syncthreads();
      } else {
        wait_stages<S - 2, PER_STAGE>(min(S - 2, nk - 1 - kt));
        __syncthreads();
        if (kt + S - 1 < nk) issue(kt + S - 1);
      }

      // Fragments of 16-wide k-substep ks+1 are read from LDS while the MFMAs
      // of substep ks run (two register sets); the scheduling groups below
      // interleave one LDS read after each MFMA.
      const unsigned char *cur = smem + (kt % S) * T::STAGE_BYTES;
      load_frags(cur, 0, 0);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 1 < KS) load_frags(cur, ks + 1, (ks + 1) & 1);
#pragma unroll
        for (int x = 0; x < NMF; ++x) mfma(x, ks & 1);
      }
      if constexpr (T::PIPE) {
        __builtin_amdgcn_sched_group_barrier(0x100, NF, 0);
#pragma unroll
        for (int ks = 0; ks + 1 < KS; ++ks) {
#pragma unroll
          for (int x = 0; x < NF; ++x) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          if constexpr (NMF > NF) __builtin_amdgcn_sched_group_barrier(0x008, NMF - NF, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NMF, 0);
      }
    }
    __syncthreads();  // every wave is done with the stages before the next tile's prologue

    // C is written once and not read again by this kernel: non-temporal
    // stores keep it from displacing operand lines in the caches (≈ 1 % on
    // 8192^3)
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
            if (m < M) __builtin_nontemporal_store(to_bf16(acc[i][j][r]), &C[(size_t)m * N + n]);
          }
        }
        // keep the accumulator reads of one block next to its stores (the
        // scheduler would otherwise hoist all of them and exhaust registers)
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  hooks_end(tr, t0);
}

}  // namespace
}  // namespace occ
