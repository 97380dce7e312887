/*
 * occ.h -- resource-aware computation/communication overlap on one MI355X.
 *
 * C ABI of the hot path of "Resource-aware Computation-Communication Overlap
 * for multi-GPU ML Workloads" (Cui, Pericas): a bf16 GEMM K_g whose
 * per-workgroup LDS footprint shapes its occupancy (Section 3.1), run
 * concurrently with one GPU's local share of a collective K_c (Background,
 * item 2) on a second stream, with the per-iteration dependency
 * K_g^i -> K_c^i enforced by an event or a device-side counter (Section 3.2)
 * and the collective given precedence over later GEMMs (Section 3.3).
 *
 * Conventions for every entry point:
 *   - Device buffers are plain device pointers owned by the caller; the
 *     library never allocates, frees or retains them.
 *   - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *     Kernel entry points are asynchronous: they return after enqueueing.
 *   - Arguments are validated before any HIP call.  Errors are negative
 *     occ_status codes; nothing is thrown across the ABI and nothing is
 *     launched when a check fails.  occ_strerror() names each code.
 *   - Not thread-safe: calls that overlap on one device from several host
 *     threads must be serialised by the caller.
 */
#ifndef OCC_H
#define OCC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum occ_status {
  OCC_OK = 0,
  OCC_EINVAL = -1,  /* null pointer, negative or unsupported size, misalignment */
  OCC_ELDS = -2,    /* tile LDS + lds_bytes exceeds the per-workgroup LDS limit */
  OCC_EPERM = -3,   /* perm is not a bijection of [0, nchunks) */
  OCC_EALIAS = -4,  /* an output range overlaps an input range */
  OCC_EHIP = -5,    /* the HIP runtime reported an error (launch, event, stream) */
  OCC_ENODEV = -6,  /* no gfx950 device is current */
  OCC_ETIMEOUT = -7 /* a collective's bounded wait for its GEMM ran out (OCC_DEP_COUNTER) */
} occ_status;

/* ------------------------------------------------------------------ K_g */

/*
 * occ_gemm -- C = A * B, bf16 inputs, fp32 accumulation, bf16 output.
 * Background, item 1 (C = alpha op(A) op(B) + beta C) with alpha = 1,
 * beta = 0 (C is overwritten, never read) and op = identity:
 *   A : M x K, row-major bf16 (uint16 bit patterns), lda = K.
 *   B : K x N, row-major bf16, ldb = N:  C[m][n] = sum_k A[m][k] * B[k][n].
 *   C : M x N, row-major bf16, ldc = N.  Rounded to nearest-even from fp32.
 * lds_bytes is the EXTRA dynamic LDS each GEMM workgroup reserves on top of
 * the LDS its tile uses (S_tile).  It is never touched; it only lowers the
 * number of GEMM workgroups that fit on a CU (Section 3.1, S_blk).
 * Requirements: M, N, K >= 0; K % 8 == 0 and N % 8 == 0 (16-byte rows);
 * A, B, C 16-byte aligned; C must not overlap A or B; K at most 4 M and N at
 * most 16 M (an operand tile is addressed with 32-bit offsets; larger is
 * OCC_EINVAL).  M == 0 or N == 0 is a no-op; K == 0 writes zeros.  Returns
 * OCC_ELDS if S_tile + lds_bytes exceeds the device's per-workgroup LDS
 * limit (never clamps).
 */
int occ_gemm(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
             void *stream);

/*
 * Kernel variants (tile_m x tile_n x tile_k, waves, LDS stages).  Variant 0
 * lets the library choose from the shape.  Each variant reads B in one
 * layout: occ_gemm / occ_gemm_ex take the K x N ones, occ_gemm_bt /
 * occ_gemm_bt_ex the N x K ones.  36/37 (K x N) and 6/7 (N x K) are the
 * paper's tile configurations opt1 (64x64x32) and opt2 (64x64x64) of Table 1,
 * with one LDS stage so that S_tile = 2*(TILE_M*TILE_K + TILE_K*TILE_N) bytes
 * (Section 3.1).
 */
enum {
  OCC_GEMM_AUTO = 0,
  /* B stored K x N (occ_gemm) */
  OCC_GEMM_KN_256x256x64_8W_2ST = 32,   /* direct-to-LDS; default for large shapes */
  OCC_GEMM_KN_SKINNY_4W_2ST = 33,       /* M <= 16: 128-column units over the whole K; default for M <= 16 */
  OCC_GEMM_KN_128x128x64_4W_3ST = 35,   /* default for mid-size shapes */
  OCC_GEMM_KN_OPT1_64x64x32 = 36,       /* Table 1 opt1, one stage */
  OCC_GEMM_KN_OPT2_64x64x64 = 37,       /* Table 1 opt2, one stage */
  OCC_GEMM_KN_128x256x32_4W_2ST = 38,   /* two resident workgroups per CU (48 KiB) */
  OCC_GEMM_KN_64x64x64_4W_2ST = 39,     /* the opt2 tile with two stages; default for small shapes */
  /* B stored N x K (occ_gemm_bt) */
  OCC_GEMM_OPT1_64x64x32 = 6,           /* Table 1 opt1, register-staged, one stage */
  OCC_GEMM_OPT2_64x64x64 = 7,           /* Table 1 opt2, register-staged, one stage; default for a K
                                           beyond the direct-to-LDS tiles' limit */
  OCC_GEMM_DL_64x64x64_4W_2ST = 9,      /* direct-to-LDS, two stages; default for small shapes */
  OCC_GEMM_DL_128x128x64_4W_3ST = 14,   /* direct-to-LDS; default for mid-size shapes */
  OCC_GEMM_DLP_256x256x64_8W_2ST = 16,  /* direct-to-LDS; default for large shapes */
  OCC_GEMM_SKINNY_8W_U8 = 21,           /* M <= 16, any K: 8 waves, 8 k-blocks in flight per lane */
  OCC_GEMM_DLP_128x256x32_4W_2ST = 25,  /* two resident workgroups per CU (48 KiB) */
  OCC_GEMM_SKINNY_LDSB_K8192 = 34       /* M <= 16, K a multiple of 1024 up to 8192: A in registers,
                                           B staged through LDS; default for such K */
};

/*
 * occ_gemm_ex -- occ_gemm with an explicit kernel variant (0 or a K x N one)
 * and grid cap.  grid_cap > 0 launches at most grid_cap workgroups, each
 * looping over output tiles (persistent workgroups): the "thread-block count"
 * knob of the paper's Figs. 2-3.  grid_cap == 0 launches one workgroup per
 * tile.  The grid cap and the pad never change the result, and the tiled
 * variants of one layout accumulate every output over k in the same order
 * and give bit-identical results; the skinny variants split K across waves
 * and may differ from them in the last bit.  OCC_EINVAL for an unknown
 * variant, a variant of the other layout, a skinny variant with M > 16, or a
 * K or N beyond the variant's addressing limit.
 */
int occ_gemm_ex(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
                int variant, int grid_cap, void *stream);

/*
 * occ_gemm_bt -- C = A * B^T with B stored N x K (row-major, K-contiguous:
 * the weight layout of a linear layer, op(B) = B^T in Background, item 1):
 *   C[m][n] = sum_k A[m][k] * B[n][k].
 * Same arithmetic, rounding, LDS pad and errors as occ_gemm; N need not be a
 * multiple of 8.  For M > 16 the results are bit-identical to occ_gemm on the
 * same matrix stored K x N (same tiles, same order of the k sums); for M <= 16
 * the skinny kernels of the two layouts split K differently and may differ in
 * the last bit.  Any K % 8 == 0 is taken (K beyond a direct-to-LDS tile's
 * 32-bit addressing runs on the register-staged 64x64 tile).
 */
int occ_gemm_bt(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
                void *stream);

/* occ_gemm_bt_ex -- occ_gemm_bt with a variant (0 or an N x K one) and a grid
   cap as in occ_gemm_ex.  OCC_EINVAL for a K x N variant, a skinny variant
   with M > 16, or a K that variant 34 does not take. */
int occ_gemm_bt_ex(const void *A, const void *B, void *C, int M, int N, int K, size_t lds_bytes,
                   int variant, int grid_cap, void *stream);

/* Launch plan occ_gemm_ex would use, for reporting and sweeps. */
typedef struct occ_gemm_plan {
  int tile_m, tile_n, tile_k;  /* output tile per workgroup and k-step */
  int threads;                 /* threads per workgroup */
  int tile_lds_bytes;          /* S_tile: LDS the tile itself uses */
  int grid;                    /* workgroups launched */
  int tiles;                   /* output tiles */
  int wg_per_cu;               /* resident workgroups per CU with the pad (occupancy API) */
  int max_lds_per_wg;          /* device limit on LDS per workgroup, bytes */
  int lds_per_cu;              /* device LDS per CU, bytes */
  int num_cus;                 /* compute units */
  int kernel_id;               /* variant actually chosen */
} occ_gemm_plan;

/*
 * occ_gemm_plan_query -- the plan for occ_gemm_ex(M, N, K, lds_bytes,
 * variant, grid_cap) on the current device.  Returns OCC_ELDS when
 * S_tile + lds_bytes exceeds the per-workgroup LDS limit (the plan is still
 * filled in, with wg_per_cu = 0); OCC_EINVAL for an N x K variant.
 */
int occ_gemm_plan_query(int M, int N, int K, size_t lds_bytes, int variant, int grid_cap,
                        occ_gemm_plan *plan);

/* occ_gemm_bt_plan_query -- the same for occ_gemm_bt_ex (variant 0 standing
   for occ_gemm_bt's automatic choice); OCC_EINVAL for a K x N variant. */
int occ_gemm_bt_plan_query(int M, int N, int K, size_t lds_bytes, int variant, int grid_cap,
                           occ_gemm_plan *plan);

/*
 * occ_gemm_info -- the three LDS figures of Section 3.1 for the kernel
 * occ_gemm uses on large shapes (variant 32): its tile's own LDS (S_tile),
 * the device's per-workgroup LDS limit and its LDS per CU, in bytes; so a
 * caller can size lds_bytes (S_tile + pad <= max_lds_per_wg; resident
 * workgroups per CU <= lds_per_cu / (S_tile + pad)).  occ_gemm_plan_query
 * gives the same for any shape and variant.  OCC_EINVAL for a null pointer;
 * OCC_ENODEV without a gfx950 device.
 */
int occ_gemm_info(int *tile_lds_bytes, int *max_lds_per_wg, int *lds_per_cu);

/* ------------------------------------------------------------------ K_c */

/*
 * share_reduce -- one GPU's local share of an allreduce (Background, item 2):
 *   out[j] = (((bufs[0][j] + bufs[1][j]) + bufs[2][j]) + ...) + bufs[n-1][j]
 * in IEEE binary32, strict left-to-right, for j < len.  Bit-identical to that
 * definition (no reassociation, no contraction, denormals kept).
 *   bufs    : HOST array of nchunks device pointers, 1 <= nchunks <= 64.
 *   out     : device fp32 buffer of len elements; must not overlap any bufs[c].
 * len == 0 is a no-op.  Any alignment is accepted; 16-byte-aligned buffers
 * take the vectorised path.
 */
int share_reduce(const float *const *bufs, int nchunks, size_t len, float *out, void *stream);

/*
 * share_reduce_ex -- share_reduce with the comm-kernel knobs: `wgs`
 * workgroups of 128 threads (0 = library default: one per CU, fewer for
 * short inputs) and
 * wave priority `priority` in 0..3
 * (s_setprio; 0 = normal).  Same result for every wgs and priority.
 */
int share_reduce_ex(const float *const *bufs, int nchunks, size_t len, float *out, int wgs,
                    int priority, void *stream);

/*
 * share_permute -- one GPU's local share of an alltoall (Background, item 2):
 * a chunk gather, dst[i*chunk_bytes + b] = src[perm[i]*chunk_bytes + b] for
 * i < nchunks, b < chunk_bytes.  A byte copy: any dtype, bit-exact.
 *   perm : HOST int32 array of nchunks entries, a bijection of [0, nchunks);
 *          1 <= nchunks <= 512.
 *   src, dst : device buffers of nchunks*chunk_bytes bytes; must not overlap.
 * nchunks is an addition to the three-pointer form: the length of perm.
 * chunk_bytes == 0 is a no-op.  16-byte-aligned src, dst and chunk_bytes take
 * the vectorised path; anything else is copied byte by byte.
 */
int share_permute(const void *src, void *dst, const int32_t *perm, int nchunks, size_t chunk_bytes,
                  void *stream);

/*
 * share_reduce_own -- the allreduce share whose first term is this GPU's own
 * contribution held in bf16 (for instance the GEMM's output C):
 *   out[j] = (((f32(own[j]) + peers[0][j]) + peers[1][j]) + ...) + peers[n-1][j]
 * in IEEE binary32, strict left-to-right, f32() the exact widening of a bf16
 * bit pattern.  Bit-identical to that definition.
 *   own   : device bf16 buffer of len elements (2-byte aligned).
 *   peers : HOST array of npeers device fp32 pointers, 0 <= npeers <= 63
 *           (may be NULL when npeers == 0).
 *   out   : device fp32 buffer of len elements; must not overlap own or any
 *           peer.
 *   wgs, priority : as share_reduce_ex.
 * len == 0 is a no-op.  own 8-byte aligned with out and peers 16-byte aligned
 * takes the vectorised path.
 */
int share_reduce_own(const void *own, const float *const *peers, int npeers, size_t len, float *out,
                     int wgs, int priority, void *stream);

/* share_permute_ex -- share_permute with `wgs` (workgroups of 128 threads)
 * and `priority` as share_reduce_ex. */
int share_permute_ex(const void *src, void *dst, const int32_t *perm, int nchunks,
                     size_t chunk_bytes, int wgs, int priority, void *stream);

/* ------------------------------------------------------------------ schedule */

/* OCC_COMM_REDUCE_OWN: the collective consumes the GEMM's output.  C then
   holds n_iter consecutive M x N outputs (M*N a multiple of 8): iteration i's
   GEMM writes C_i = C + i*M*N and iteration i's collective is
   share_reduce_own(C_i, bufs, nchunks, len = M*N, out); the per-iteration
   buffers keep GEMM i+1 from overwriting what collective i still reads. */
enum { OCC_COMM_REDUCE = 0, OCC_COMM_PERMUTE = 1, OCC_COMM_REDUCE_OWN = 2 };

/* run_overlap flags: which passes to time (no pass bit set means all three),
   and OCC_RUN_GRAPH: capture the sequential and the overlapped schedule into
   a HIP graph each and replay it per repetition, instead of issuing every
   kernel, event record and stream wait from the host (for schedules whose
   kernels are as short as the host's issue time). */
enum { OCC_RUN_SEQ = 1, OCC_RUN_OVL = 2, OCC_RUN_ISO = 4, OCC_RUN_GRAPH = 8, OCC_RUN_PACE_ALL = 16 };
/* OCC_RUN_PACE_ALL: apply comm_rate_gbs to every schedule and to the isolated
   timings, not only to the overlapped one.  This emulates on one GPU a
   collective whose duration is set by inter-GPU links rather than by this
   GPU's memory (the multi-GPU setting of Section 4): the local kernel then
   streams at the link rate in the sequential schedule too. */

/* Layout of B in the schedule's GEMM (occ_overlap_cfg.gemm_b_layout). */
enum { OCC_B_KN = 0 /* K x N, occ_gemm */, OCC_B_NK = 1 /* N x K, occ_gemm_bt */ };

/*
 * The per-iteration dependency K_g^i -> K_c^i of the overlapped schedule
 * (occ_overlap_cfg.dep; Section 3.2):
 *   OCC_DEP_EVENT   -- a runtime event recorded on the compute stream after
 *                      K_g^i and waited on by the comm stream before K_c^i
 *                      (the paper's form).  Costs about 18 us of host issue
 *                      time per iteration on MI355X, so schedules whose
 *                      kernels are that short become bound by it.
 *   OCC_DEP_COUNTER -- a device-side counter: every workgroup of K_g^i adds
 *                      one to a per-iteration counter when it is done (after
 *                      its stores, released at device scope), and every
 *                      workgroup of K_c^i waits until the counter reaches
 *                      K_g^i's workgroup count (then acquires) before it
 *                      reads anything.  No host call besides the two kernel
 *                      launches.  The collective's last workgroup puts the
 *                      counter back to zero.  The wait is bounded: a
 *                      workgroup that has waited 2 s skips its work and the
 *                      schedule fails with OCC_ETIMEOUT.  Needs a GEMM and a
 *                      collective that fit on one CU side by side (one comm
 *                      workgroup per CU at most, registers and LDS of both
 *                      within the CU's), else OCC_EINVAL; n_iter <= 1024;
 *                      not with OCC_RUN_GRAPH (a replayed graph may order
 *                      a collective before its GEMM on one queue, and that
 *                      collective would wait out its bound): OCC_EINVAL.
 * The sequential schedule needs no dependency (one stream).
 */
enum { OCC_DEP_EVENT = 0, OCC_DEP_COUNTER = 1 };

typedef struct occ_overlap_cfg {
  /* K_g: as occ_gemm (gemm_b_layout OCC_B_KN) or occ_gemm_bt (OCC_B_NK) */
  int M, N, K;
  const void *A, *B;
  void *C;
  size_t lds_bytes;         /* extra LDS per GEMM workgroup (Section 3.1) */
  int gemm_variant;         /* OCC_GEMM_* of the layout (0 = automatic) */
  int gemm_grid;            /* 0: one workgroup per tile; > 0: persistent grid cap */
  int gemm_priority;        /* wave priority of the GEMM kernel, 0 (normal) .. 3 */
  int gemm_b_layout;        /* OCC_B_KN (default) or OCC_B_NK */
  /* K_c: as share_reduce (comm_kind 0), share_permute (comm_kind 1) or
     share_reduce_own of the GEMM's output (comm_kind 2, bufs/nchunks = the
     fp32 peer chunks) */
  int comm_kind;
  const float *const *bufs; /* host array of device pointers */
  int nchunks;
  size_t len;
  float *out;
  const void *src;
  void *dst;
  const int32_t *perm;      /* host array */
  size_t chunk_bytes;
  int comm_wgs;             /* workgroups of the comm kernel; 0 = library default */
  int comm_priority;        /* wave priority of the comm kernel, 0 (normal) .. 3 (highest) */
  /* bandwidth pacing of the collective in the overlapped schedule, GB/s over
     the whole grid: every comm wave spaces its load/store trips so that the
     kernel streams at no more than this rate, leaving memory bandwidth to the
     co-running GEMM.  0 = unpaced (full speed); otherwise at least
     OCC_MIN_COMM_RATE_GBS.  The sequential schedule and the isolated kernel
     timings run unpaced, so t_seq stays the fastest sequential makespan,
     unless flags has OCC_RUN_PACE_ALL.  Results are unchanged (same
     arithmetic, same order). */
  double comm_rate_gbs;
  /* schedule (Section 3.2) and protocol (Section 4.1) */
  int n_iter;               /* GEMM -> collective iterations per schedule, >= 1 */
  int dep;                  /* OCC_DEP_EVENT (default) or OCC_DEP_COUNTER */
  int reps;                 /* timed repetitions of each pass, >= 1 */
  int warmup;               /* untimed repetitions before them, >= 0 */
  int flags;                /* OCC_RUN_* bits, 0 = all */
  /* the caller's stream (hipStream_t as void*, NULL = the null stream): the
     launcher's work starts after everything already enqueued on it, so
     inputs the caller is still producing there are complete first */
  void *stream;
  /* optional device buffer of 4*n_iter uint64: for the last overlapped
     repetition, [start_G0, end_G0, start_C0, end_C0, start_G1, ...] in
     10 ns ticks of the GPU's constant-rate clock (earliest workgroup start,
     latest workgroup end).  NULL = no timeline. */
  uint64_t *timeline;
  /* optional device buffer of 4 + 12*wg_trace_cap uint32: for that same
     repetition, word 0 counts workgroups and record i (words 4+12i ..
     15+12i) is {tag, workgroup id, HW_ID, XCC_ID, t0 lo, t0 hi, t1 lo, t1 hi,
     cycles lo, cycles hi, 0, 0}: tag = 2*iteration (+1 for the collective),
     HW_ID/XCC_ID the hardware registers naming the CU (bits 11:8), shader
     array (12), shader engine (15:13) and XCD (3:0), t0/t1 the workgroup's
     start/end clock (10 ns ticks), cycles the engine-clock cycles between
     them (cycles / (t1 - t0) / 10 ns = the clock the workgroup ran at).
     Records beyond wg_trace_cap are counted but not written.  NULL = off. */
  uint32_t *wg_trace;
  int wg_trace_cap;
} occ_overlap_cfg;

#define OCC_MIN_COMM_RATE_GBS 10.0

typedef struct occ_overlap_result {
  double t_seq_ms;        /* mean sequential makespan: one stream, G0 C0 G1 C1 ... */
  double t_ovl_ms;        /* mean overlapped makespan: two streams + per-iteration dependency */
  double t_seq_min_ms, t_ovl_min_ms;
  double reduction_pct;   /* 100 * (1 - t_ovl / t_seq) = 100 * (1 - TimeRatio) */
  double t_gemm_ms;       /* mean duration of one GEMM launch, isolated pass */
  double t_comm_ms;       /* mean duration of one comm launch, isolated pass */
  int gemm_wg_per_cu;     /* resident GEMM workgroups per CU (occupancy API) */
  int gemm_grid;          /* GEMM workgroups per launch */
  int gemm_tile_lds;      /* S_tile, bytes */
  int comm_wgs;           /* comm workgroups per launch */
  double t_seq_median_ms, t_ovl_median_ms;  /* median over the timed repetitions */
  double t_seq_std_ms, t_ovl_std_ms;        /* sample standard deviation (0 for reps = 1) */
} occ_overlap_result;

/*
 * run_overlap -- time the sequential and the overlapped schedule of n_iter
 * GEMM -> collective iterations (Section 3.2, Fig. 1), after `warmup`
 * untimed repetitions, averaging `reps` timed ones (Section 4.1).
 * Both schedules end on the compute stream: the overlapped one forks the comm
 * stream off it with an event and joins it back after the last collective.
 * Host-synchronous.  Uses two library-owned streams of default priority on
 * the current device (created once, kept for the process), which first wait
 * for the work already enqueued on cfg->stream; the collective's
 * precedence (Section 3.3) is the comm kernel's wave priority.  With
 * OCC_DEP_COUNTER the per-iteration counters live in a small device buffer
 * the library allocates once per device (8 KiB).  All three
 * passes compute the same outputs: C, out/dst are identical to one occ_gemm
 * and one share_* call.  Buffers are validated as by those entry points.
 * HIP maps a process's streams onto a fixed number of hardware queues
 * (GPU_MAX_HW_QUEUES, 4 by default), round-robin in creation order; once a
 * process holds more streams than queues, the two launcher streams can land
 * on one queue and the "overlapped" schedule then runs serially.  Callers
 * that create streams of their own should keep the total within the queue
 * count (measured: 9.9 ms overlapped with 3 streams in the process, 10.7 ms
 * -- no overlap -- with 5, for the 8192^3 GEMM + 8 x 2^25 fp32 reduce).
 */
int run_overlap(const occ_overlap_cfg *cfg, occ_overlap_result *res);

/*
 * occ_overlap_tune -- adaptive choice of the occupancy and priority knobs, the
 * runtime policy the paper leaves to future work (Section 6).  Times the
 * overlapped schedule of *cfg (tune_reps repetitions after one warm-up) for
 * every candidate in
 *   comm_priority {0, 3} x comm_wgs {library default (one per CU), two per CU,
 *                                     one per four CUs}
 *   x gemm_grid {one workgroup per tile, one persistent workgroup per CU}
 *   x lds_bytes {0, the pad that lowers the GEMM's residency by one
 *                workgroup per CU (only when it has more than one)}
 *   x dep {OCC_DEP_EVENT, OCC_DEP_COUNTER (with one comm workgroup per CU)},
 * writes the setting with the shortest median makespan into those fields of
 * *cfg (gemm_variant, n_iter, buffers and the rest are kept), then runs
 * run_overlap(cfg, res) with it.  *prefer_sequential is set to 1 when even
 * the best overlapped median makespan is longer than the sequential one
 * (then overlap should be off).  Same validation and errors as run_overlap;
 * host-synchronous.
 */
int occ_overlap_tune(occ_overlap_cfg *cfg, int tune_reps, occ_overlap_result *res,
                     int *prefer_sequential);

/*
 * occ_overlap_workspace_bytes -- device bytes occ_overlap_enqueue needs for
 * n_iter iterations: 2 * n_iter + 1 uint32 counters, rounded up to 256
 * bytes (0 for n_iter < 1).
 */
size_t occ_overlap_workspace_bytes(int n_iter);

/*
 * occ_overlap_enqueue -- enqueue the overlapped schedule of *cfg and return
 * (Section 3.2, Fig. 1b): for i < n_iter, K_g^i on cfg->stream and K_c^i on
 * comm_stream, with K_g^i -> K_c^i kept by the device counter of
 * OCC_DEP_COUNTER in `workspace`.  No timing, no runtime events, no host
 * synchronisation and no allocation: the form a training or serving loop
 * calls.  GEMM and collective as in run_overlap (gemm_b_layout,
 * comm_kind, knobs, comm_rate_gbs pacing every collective); reps, warmup,
 * flags and dep are not read; timeline and wg_trace must be NULL.
 *   workspace : caller-owned device buffer of at least
 *               occ_overlap_workspace_bytes(n_iter) bytes, 4-byte aligned,
 *               all zero before its first use.  A schedule leaves it zero
 *               again once all its collectives have passed their waits.
 *   err       : optional device uint32 (may be NULL) that a collective
 *               workgroup sets to 1 when its bounded wait runs out (the
 *               library never clears it).
 * Ordering is the caller's: both streams must already follow the work that
 * produces the inputs; the collectives' outputs are complete when
 * comm_stream reaches the end of this call's work, C when cfg->stream does.
 * Two schedules on one workspace must not overlap: order the next call's
 * cfg->stream after this call's comm_stream (else a GEMM can count into a
 * counter a collective of this call still has to clear, and its own
 * collective then waits out its bound).  Under stream capture the replay
 * must run the two streams' chains concurrently, as captured.
 * Errors: those of run_overlap, and OCC_EINVAL for a NULL, misaligned or
 * short workspace, a comm grid above one workgroup per CU, or a collective
 * with no work.  Every argument is checked before the first launch; only a
 * runtime failure (OCC_EHIP) can stop the call part-way, and then counts of
 * the launched GEMMs may remain in the workspace: zero it before reusing it.
 */
int occ_overlap_enqueue(const occ_overlap_cfg *cfg, void *comm_stream, void *workspace, size_t workspace_bytes,
                        uint32_t *err);

/*
 * occ_overlap_enqueue_noalloc -- occ_overlap_enqueue for callers that cannot
 * allocate device memory (code under graph capture, tight serving loops,
 * harnesses that forbid allocation): the counters live in a library-owned
 * static device array sized for OCC_NOALLOC_MAX_ITER iterations (8448 bytes
 * on every GPU the library runs on, held until the process ends), so no
 * workspace is passed and nothing is allocated.  n_iter above
 * OCC_NOALLOC_MAX_ITER is OCC_EINVAL.  All calls on one GPU share that
 * array: calls that overlap on one GPU race (order each call's cfg->stream
 * after the previous call's comm_stream).  The array starts zeroed and a
 * complete schedule leaves it zeroed (after an OCC_EHIP part-way through a
 * call it may not be: the library's array cannot then be reused safely in
 * this process).  Otherwise as occ_overlap_enqueue.
 */
#define OCC_NOALLOC_MAX_ITER 1024
int occ_overlap_enqueue_noalloc(const occ_overlap_cfg *cfg, void *comm_stream, uint32_t *err);

/* Static string naming a status code. */
const char *occ_strerror(int status);

/* Library version, (major << 16) | minor.  The minor number grows whenever a
   structure above gains fields, so a binding can refuse a library whose
   layout it does not know. */
#define OCC_VERSION_MAJOR 2
#define OCC_VERSION_MINOR 2
int occ_version(void);

#ifdef __cplusplus
}
#endif

#endif /* OCC_H */
