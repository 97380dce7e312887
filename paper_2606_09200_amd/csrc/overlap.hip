// Two-stream launcher: sequential vs overlapped schedule of n_iter
// GEMM -> collective iterations (Section 3.2, Fig. 1).
//
//   SEQ: one stream, G0 C0 G1 C1 ... G_{n-1} C_{n-1}.
//   OVL: G_i on the compute stream, C_i on the comm stream after G_i
//        (K_g^i -> K_c^i), so G_{i+1} may run while C_i does.  The edge is an
//        event recorded after G_i and waited on before C_i (OCC_DEP_EVENT),
//        or a device-side counter that G_i's workgroups count up and C_i's
//        workgroups wait on (OCC_DEP_COUNTER).  The collective's precedence
//        over later GEMMs is the comm kernel's wave priority (s_setprio);
//        both streams keep the default queue priority.
//   ISO: SEQ with an event between every two kernels, giving the mean
//        duration of one GEMM and of one collective launch.
//
// Makespans are GPU event intervals.  The protocol follows Section 4.1:
// `warmup` untimed repetitions, then the mean over `reps` timed ones.
#include "occ_internal.h"

#include <string.h>

#include <algorithm>
#include <cmath>
#include <vector>

namespace occ {

namespace {

struct StreamPair {
  hipStream_t comp = nullptr;
  hipStream_t comm = nullptr;
};
StreamPair g_streams[64];

int stream_pair(StreamPair **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return OCC_ENODEV;
  StreamPair &p = g_streams[dev];
  if (p.comp == nullptr) {
    if (hipStreamCreateWithFlags(&p.comp, hipStreamNonBlocking) != hipSuccess) return OCC_EHIP;
    if (hipStreamCreateWithFlags(&p.comm, hipStreamNonBlocking) != hipSuccess) return OCC_EHIP;
  }
  *out = &p;
  return OCC_OK;
}

struct Events {
  std::vector<hipEvent_t> ev;
  ~Events() {
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
  }
  int make(int n, unsigned flags) {
    ev.assign(n, nullptr);
    for (int i = 0; i < n; ++i)
      if (hipEventCreateWithFlags(&ev[i], flags) != hipSuccess) return OCC_EHIP;
    return OCC_OK;
  }
};

// Per-device buffer of the counter dependency: kMaxDepIter counters of
// finished GEMM workgroups (one per iteration), kMaxDepIter counters of
// collective workgroups past their wait, and one error word.  Allocated and
// zeroed once per device; every complete schedule leaves it zeroed again.
constexpr int kMaxDepIter = 1024;
constexpr size_t kDepWords = 2 * kMaxDepIter + 64;
uint32_t *g_dep[64];

int dep_scratch(uint32_t **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return OCC_ENODEV;
  if (g_dep[dev] == nullptr) {
    void *p = nullptr;
    if (hipMalloc(&p, kDepWords * sizeof(uint32_t)) != hipSuccess) return OCC_EHIP;
    if (hipMemset(p, 0, kDepWords * sizeof(uint32_t)) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
      (void)hipFree(p);
      return OCC_EHIP;
    }
    g_dep[dev] = static_cast<uint32_t *>(p);
  }
  *out = g_dep[dev];
  return OCC_OK;
}

#define OCC_TRY(x)                 \
  do {                             \
    int st_ = (x);                 \
    if (st_ != OCC_OK) return st_; \
  } while (0)
#define OCC_HIP(x)                                   \
  do {                                               \
    if ((x) != hipSuccess) return OCC_EHIP;          \
  } while (0)

struct Launcher {
  GemmCall g;
  ReduceCall r;
  PermuteCall p;
  int kind;

  // own: iteration i's GEMM writes its own output C_i (C + i*M*N), which
  // iteration i's collective reduces as its first term
  bool own = false;
  void *c_iter(int i) const { return static_cast<uint16_t *>(g.C) + (own ? (size_t)i * g.M * g.N : 0); }
  int gemm(hipStream_t s, KHooks t, int i) {
    GemmCall c = g;
    c.C = c_iter(i);
    c.trace = t;
    return gemm_launch(c, s);
  }
  // `paced`: the overlapped schedule's launches stream at rate_gbs; the
  // sequential schedule and the isolated timings do too when pace_all.
  double rate_gbs;
  bool pace_all;
  int comm(hipStream_t s, KHooks t, bool paced, int i) {
    paced = paced || pace_all;
    if (kind == OCC_COMM_REDUCE || kind == OCC_COMM_REDUCE_OWN) {
      ReduceCall c = r;
      if (own) c.own = static_cast<const uint16_t *>(c_iter(i));
      c.trace = t;
      c.rate_gbs = paced ? rate_gbs : 0.0;
      return reduce_launch(c, s);
    }
    PermuteCall c = p;
    c.trace = t;
    c.rate_gbs = paced ? rate_gbs : 0.0;
    return permute_launch(c, s);
  }
};

int validate_cfg(const occ_overlap_cfg *c) {
  if (c == nullptr) return OCC_EINVAL;
  if (c->n_iter < 1 || c->reps < 1 || c->warmup < 0) return OCC_EINVAL;
  if (c->comm_priority < 0 || c->comm_priority > 3 || c->comm_wgs < 0) return OCC_EINVAL;
  if (c->gemm_priority < 0 || c->gemm_priority > 3) return OCC_EINVAL;
  if (c->gemm_grid < 0 || c->gemm_variant < 0) return OCC_EINVAL;
  if ((c->flags & ~(OCC_RUN_SEQ | OCC_RUN_OVL | OCC_RUN_ISO | OCC_RUN_GRAPH | OCC_RUN_PACE_ALL)) != 0)
    return OCC_EINVAL;
  if (c->wg_trace != nullptr && c->wg_trace_cap < 0) return OCC_EINVAL;
  if (!(c->comm_rate_gbs == 0.0 || (c->comm_rate_gbs >= OCC_MIN_COMM_RATE_GBS && c->comm_rate_gbs <= 1.0e6)))
    return OCC_EINVAL;
  if (c->gemm_b_layout != OCC_B_KN && c->gemm_b_layout != OCC_B_NK) return OCC_EINVAL;
  if (c->dep != OCC_DEP_EVENT && c->dep != OCC_DEP_COUNTER) return OCC_EINVAL;
  if (c->dep == OCC_DEP_COUNTER && c->n_iter > kMaxDepIter) return OCC_EINVAL;
  // a replayed graph may run its two branches on one queue in any
  // topological order; a collective placed before its GEMM would then wait
  // out its whole bound, so graphs keep the event dependency
  if (c->dep == OCC_DEP_COUNTER && (c->flags & OCC_RUN_GRAPH)) return OCC_EINVAL;
  OCC_TRY(validate_gemm(c->A, c->B, c->C, c->M, c->N, c->K, c->gemm_b_layout == OCC_B_KN));
  size_t cbytes = (size_t)c->M * c->N * 2;
  // K_g writes C while K_c runs: C must not overlap anything K_c touches,
  // and K_c's output must not overlap A or B.
  auto hit = [](const void *a, size_t an, const void *b, size_t bn) {
    if (!a || !b || !an || !bn) return false;
    uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bn && b0 < a0 + an;
  };
  size_t abytes = (size_t)c->M * c->K * 2, bbytes = (size_t)c->N * c->K * 2;
  if (c->comm_kind == OCC_COMM_REDUCE_OWN) {
    // C holds n_iter outputs of M*N each, every one 16-byte aligned; the
    // collective reduces C_i (len = M*N) and the fp32 peer chunks
    const size_t mn = (size_t)c->M * c->N;
    if (mn == 0 || mn % 8 != 0 || c->len != mn) return OCC_EINVAL;
    OCC_TRY(validate_reduce_own(c->C, c->bufs, c->nchunks, c->len, c->out));
    const size_t call = cbytes * (size_t)c->n_iter, lb = c->len * 4;
    for (int i = 0; i < c->nchunks; ++i)
      if (hit(c->C, call, c->bufs[i], lb)) return OCC_EALIAS;
    if (hit(c->C, call, c->out, lb) || hit(c->out, lb, c->A, abytes) || hit(c->out, lb, c->B, bbytes) ||
        hit(c->C, call, c->A, abytes) || hit(c->C, call, c->B, bbytes))
      return OCC_EALIAS;
  } else if (c->comm_kind == OCC_COMM_REDUCE) {
    OCC_TRY(validate_reduce(c->bufs, c->nchunks, c->len, c->out));
    size_t lb = c->len * 4;
    for (int i = 0; i < c->nchunks; ++i)
      if (hit(c->C, cbytes, c->bufs[i], lb)) return OCC_EALIAS;
    if (hit(c->C, cbytes, c->out, lb) || hit(c->out, lb, c->A, abytes) || hit(c->out, lb, c->B, bbytes))
      return OCC_EALIAS;
  } else if (c->comm_kind == OCC_COMM_PERMUTE) {
    OCC_TRY(validate_permute(c->src, c->dst, c->perm, c->nchunks, c->chunk_bytes));
    size_t tb = c->chunk_bytes * (size_t)c->nchunks;
    if (hit(c->C, cbytes, c->src, tb) || hit(c->C, cbytes, c->dst, tb) || hit(c->dst, tb, c->A, abytes) ||
        hit(c->dst, tb, c->B, bbytes))
      return OCC_EALIAS;
  } else {
    return OCC_EINVAL;
  }
  return OCC_OK;
}

}  // namespace

namespace {

// The two schedules, enqueued without timing events (so that they can also be
// captured into a graph).  OVL forks the comm stream off the compute stream
// and joins it back, so the compute stream's next operation follows both.
int enqueue_seq(Launcher &L, hipStream_t s0, int n, const KHooks &off) {
  for (int i = 0; i < n; ++i) {
    OCC_TRY(L.gemm(s0, off, i));
    OCC_TRY(L.comm(s0, off, false, i));
  }
  return OCC_OK;
}

int enqueue_ovl(Launcher &L, hipStream_t s0, hipStream_t s1, hipEvent_t fork, hipEvent_t *deps,
                hipEvent_t join, int n, const KHooks *tg, const KHooks *tc, bool counter) {
  OCC_HIP(hipEventRecord(fork, s0));
  OCC_HIP(hipStreamWaitEvent(s1, fork, 0));
  for (int i = 0; i < n; ++i) {
    OCC_TRY(L.gemm(s0, tg[i], i));
    if (!counter) {
      OCC_HIP(hipEventRecord(deps[i], s0));
      OCC_HIP(hipStreamWaitEvent(s1, deps[i], 0));
    }
    // (with the counter, tg[i] and tc[i] carry the edge to the device)
    OCC_TRY(L.comm(s1, tc[i], true, i));
  }
  // C_{n-1} waits on G_{n-1}, the last GEMM, so the comm stream's end is the
  // end of the schedule; the compute stream waits for it.
  OCC_HIP(hipEventRecord(join, s1));
  OCC_HIP(hipStreamWaitEvent(s0, join, 0));
  return OCC_OK;
}

// Median and sample standard deviation (0 for a single value) of the timed
// repetitions.
void median_and_std(std::vector<double> v, double mean, double *median, double *sd) {
  if (v.empty()) return;
  std::sort(v.begin(), v.end());
  const size_t n = v.size();
  *median = n % 2 ? v[n / 2] : 0.5 * (v[n / 2 - 1] + v[n / 2]);
  double ss = 0;
  for (double x : v) ss += (x - mean) * (x - mean);
  *sd = n > 1 ? std::sqrt(ss / (double)(n - 1)) : 0.0;
}

struct Graph {
  hipGraph_t g = nullptr;
  hipGraphExec_t x = nullptr;
  ~Graph() {
    if (x) (void)hipGraphExecDestroy(x);
    if (g) (void)hipGraphDestroy(g);
  }
  int end_capture(hipStream_t s) {
    if (hipStreamEndCapture(s, &g) != hipSuccess) return OCC_EHIP;
    if (hipGraphInstantiate(&x, g, nullptr, nullptr, 0) != hipSuccess) return OCC_EHIP;
    return OCC_OK;
  }
};

}  // namespace

void make_launcher(const occ_overlap_cfg &c, Launcher *L) {
  const KHooks off{};
  L->kind = c.comm_kind;
  L->g = GemmCall{c.A, c.B, c.C, c.M, c.N, c.K, c.lds_bytes, c.gemm_grid, c.gemm_variant,
                  c.gemm_priority, off, c.gemm_b_layout == OCC_B_KN};
  L->r = ReduceCall{c.bufs, c.nchunks, c.len, c.out, c.comm_wgs, c.comm_priority, off, 0.0};
  L->own = c.comm_kind == OCC_COMM_REDUCE_OWN;
  if (L->own) L->r.own = static_cast<const uint16_t *>(c.C);
  L->p = PermuteCall{c.src, c.dst, c.perm, c.nchunks, c.chunk_bytes, c.comm_wgs, c.comm_priority, off, 0.0};
  L->rate_gbs = c.comm_rate_gbs;
  L->pace_all = (c.flags & OCC_RUN_PACE_ALL) != 0;
}

// Workgroups of one collective launch.
int comm_grid(const occ_overlap_cfg &c, const Launcher &L) {
  return c.comm_wgs > 0 ? c.comm_wgs
                        : (c.comm_kind != OCC_COMM_PERMUTE ? reduce_default_wgs(L.r) : permute_default_wgs(L.p));
}

// Per-iteration hooks of the counter dependency over `n` iterations with
// counters tk[0..n) (GEMM workgroups done) and ack[0..n) (collective
// workgroups past their wait), timeouts reported in *err.
void counter_hook_pair(const Launcher &L, int i, uint32_t gemm_grid, uint32_t *tk, uint32_t *ack, uint32_t *err,
                       KHooks *hg, KHooks *hc) {
  hg->signal = tk + i;
  hg->release = L.own ? 1u : 0u;
  hc->wait = tk + i;
  hc->ack = ack + i;
  hc->err = err;
  hc->wait_target = (L.g.M > 0 && L.g.N > 0) ? gemm_grid : 0u;
  hc->acquire = L.own ? 1u : 0u;
}

void counter_hooks(const Launcher &L, int n, uint32_t gemm_grid, uint32_t *tk, uint32_t *ack, uint32_t *err,
                   std::vector<KHooks> *hg, std::vector<KHooks> *hc) {
  for (int i = 0; i < n; ++i) counter_hook_pair(L, i, gemm_grid, tk, ack, err, &(*hg)[i], &(*hc)[i]);
}

int run_overlap_impl(const occ_overlap_cfg *cfg, occ_overlap_result *res) {
  if (res == nullptr) return OCC_EINVAL;
  OCC_TRY(validate_cfg(cfg));
  memset(res, 0, sizeof *res);
  const occ_overlap_cfg &c = *cfg;
  const int passes = c.flags & (OCC_RUN_SEQ | OCC_RUN_OVL | OCC_RUN_ISO);
  const int flags = (passes ? passes : (OCC_RUN_SEQ | OCC_RUN_OVL | OCC_RUN_ISO)) |
                    (c.flags & (OCC_RUN_GRAPH | OCC_RUN_PACE_ALL));
  const bool graph = (flags & OCC_RUN_GRAPH) != 0;
  const int n = c.n_iter;

  Launcher L;
  make_launcher(c, &L);
  const KHooks off{};

  occ_gemm_plan plan;
  OCC_TRY(gemm_plan(L.g, &plan));
  res->gemm_wg_per_cu = plan.wg_per_cu;
  res->gemm_grid = plan.grid;
  res->gemm_tile_lds = plan.tile_lds_bytes;
  res->comm_wgs = comm_grid(c, L);

  // The counter dependency: every collective workgroup may wait on a CU
  // beside the GEMM, so at most one per CU (then some CU always has room for
  // a GEMM workgroup and the GEMM cannot be starved by waiting workgroups).
  const bool counter = c.dep == OCC_DEP_COUNTER;
  uint32_t *dep = nullptr;
  if (counter) {
    const DeviceInfo *di = nullptr;
    OCC_TRY(current_device_info(&di));
    if (res->comm_wgs > di->num_cus) return OCC_EINVAL;
    // a collective that launches nothing would leave its counter counted up
    if ((c.comm_kind == OCC_COMM_PERMUTE ? c.chunk_bytes : c.len) == 0) return OCC_EINVAL;
    OCC_TRY(dep_scratch(&dep));
  }

  StreamPair *sp = nullptr;
  OCC_TRY(stream_pair(&sp));
  hipStream_t s0 = sp->comp, s1 = sp->comm;

  Events timing, deps, marks;
  OCC_TRY(timing.make(2 * n + 5, hipEventDefault));
  OCC_TRY(deps.make(n, hipEventDisableTiming));
  OCC_TRY(marks.make(3, hipEventDisableTiming));  // fork, join, caller
  hipEvent_t *ev = timing.ev.data();
  hipEvent_t *iso = ev + 4;  // 2n+1 boundaries of the isolated pass

  // Everything runs after the work already queued on the caller's stream
  // (the comm stream forks off s0 in every overlapped schedule).
  OCC_HIP(hipEventRecord(marks.ev[2], static_cast<hipStream_t>(c.stream)));
  OCC_HIP(hipStreamWaitEvent(s0, marks.ev[2], 0));

  // Per-iteration hooks of the overlapped schedule: none with the event
  // dependency; with the counter, G_i counts its finished workgroups in
  // dep[i] and C_i waits for all of them (then acknowledges in
  // dep[kMaxDepIter + i]).  Stores and loads are ordered through the counter
  // only when the collective reads the GEMM's output.
  std::vector<KHooks> hg(n, off), hc(n, off);
  if (counter) {
    counter_hooks(L, n, (uint32_t)plan.grid, dep, dep + kMaxDepIter, dep + 2 * kMaxDepIter, &hg, &hc);
    // every counter at zero (a call that failed half-way may have left some)
    OCC_HIP(hipMemsetAsync(dep, 0, kDepWords * sizeof(uint32_t), s0));
  }

  // Graph mode: capture each schedule once, replay it per repetition.
  Graph gseq, govl;
  if (graph) {
    if (flags & OCC_RUN_SEQ) {
      OCC_HIP(hipStreamBeginCapture(s0, hipStreamCaptureModeRelaxed));
      int st = enqueue_seq(L, s0, n, off);
      int st2 = gseq.end_capture(s0);
      OCC_TRY(st);
      OCC_TRY(st2);
    }
    if (flags & OCC_RUN_OVL) {
      OCC_HIP(hipStreamBeginCapture(s0, hipStreamCaptureModeRelaxed));
      int st = enqueue_ovl(L, s0, s1, marks.ev[0], deps.ev.data(), marks.ev[1], n, hg.data(), hc.data(),
                           counter);
      int st2 = govl.end_capture(s0);
      OCC_TRY(st);
      OCC_TRY(st2);
    }
  }

  double seq_sum = 0, ovl_sum = 0, seq_min = 1e300, ovl_min = 1e300, g_sum = 0, c_sum = 0;
  std::vector<double> seq_t, ovl_t;  // per timed repetition, for median and spread
  int st = OCC_OK;
  for (int rep = 0; rep < c.warmup + c.reps && st == OCC_OK; ++rep) {
    const bool timed = rep >= c.warmup;
    if (flags & OCC_RUN_SEQ) {
      OCC_HIP(hipEventRecord(ev[0], s0));
      if (graph) st = hipGraphLaunch(gseq.x, s0) == hipSuccess ? OCC_OK : OCC_EHIP;
      else st = enqueue_seq(L, s0, n, off);
      OCC_HIP(hipEventRecord(ev[1], s0));
      OCC_HIP(hipEventSynchronize(ev[1]));
      if (st != OCC_OK) break;
      float ms = 0;
      OCC_HIP(hipEventElapsedTime(&ms, ev[0], ev[1]));
      if (timed) {
        seq_sum += ms;
        seq_min = ms < seq_min ? ms : seq_min;
        seq_t.push_back(ms);
      }
    }
    if (flags & OCC_RUN_OVL) {
      OCC_HIP(hipEventRecord(ev[2], s0));
      if (graph) st = hipGraphLaunch(govl.x, s0) == hipSuccess ? OCC_OK : OCC_EHIP;
      else st = enqueue_ovl(L, s0, s1, marks.ev[0], deps.ev.data(), marks.ev[1], n, hg.data(), hc.data(),
                            counter);
      OCC_HIP(hipEventRecord(ev[3], s0));
      OCC_HIP(hipEventSynchronize(ev[3]));
      if (st != OCC_OK) break;
      float ms = 0;
      OCC_HIP(hipEventElapsedTime(&ms, ev[2], ev[3]));
      if (timed) {
        ovl_sum += ms;
        ovl_min = ms < ovl_min ? ms : ovl_min;
        ovl_t.push_back(ms);
      }
    }
    if (flags & OCC_RUN_ISO) {
      OCC_HIP(hipEventRecord(iso[0], s0));
      for (int i = 0; i < n && st == OCC_OK; ++i) {
        st = L.gemm(s0, off, i);
        if (st == OCC_OK && hipEventRecord(iso[2 * i + 1], s0) != hipSuccess) st = OCC_EHIP;
        if (st == OCC_OK) st = L.comm(s0, off, false, i);
        if (st == OCC_OK && hipEventRecord(iso[2 * i + 2], s0) != hipSuccess) st = OCC_EHIP;
      }
      OCC_HIP(hipEventSynchronize(iso[2 * n]));
      if (st != OCC_OK) break;
      if (timed) {
        for (int i = 0; i < n; ++i) {
          float a = 0, b = 0;
          OCC_HIP(hipEventElapsedTime(&a, iso[2 * i], iso[2 * i + 1]));
          OCC_HIP(hipEventElapsedTime(&b, iso[2 * i + 1], iso[2 * i + 2]));
          g_sum += a;
          c_sum += b;
        }
      }
    }
  }
  if (st != OCC_OK) {
    (void)hipStreamSynchronize(s0);
    (void)hipStreamSynchronize(s1);
    return st;
  }

  // Timeline: one more, untimed, overlapped repetition (eager) with every
  // kernel stamping its first-start / last-end clock and, if asked, one record
  // per workgroup (tag = 2*iteration + 0 for the GEMM, + 1 for the collective).
  if (c.timeline != nullptr || c.wg_trace != nullptr) {
    OCC_TRY(trace_reset(c.timeline, 2 * n, c.wg_trace, s0));
    std::vector<KHooks> tg(hg), tc(hc);
    for (int i = 0; i < n; ++i) {
      tg[i].stamps = c.timeline ? c.timeline + 4 * i : nullptr;
      tg[i].wg = c.wg_trace;
      tg[i].wg_cap = (uint32_t)c.wg_trace_cap;
      tg[i].tag = (uint32_t)(2 * i);
      tc[i].stamps = c.timeline ? c.timeline + 4 * i + 2 : nullptr;
      tc[i].wg = c.wg_trace;
      tc[i].wg_cap = (uint32_t)c.wg_trace_cap;
      tc[i].tag = (uint32_t)(2 * i + 1);
    }
    st = enqueue_ovl(L, s0, s1, marks.ev[0], deps.ev.data(), marks.ev[1], n, tg.data(), tc.data(), counter);
    OCC_HIP(hipEventRecord(ev[3], s0));
    OCC_HIP(hipEventSynchronize(ev[3]));
    if (st != OCC_OK) return st;
  }

  // A collective workgroup whose bounded wait ran out: the schedule's
  // ordering was not kept.  Leave the counters zeroed for the next call.
  if (counter) {
    uint32_t err = 0;
    OCC_HIP(hipMemcpy(&err, dep + 2 * kMaxDepIter, sizeof err, hipMemcpyDeviceToHost));
    if (err != 0) {
      OCC_HIP(hipDeviceSynchronize());
      OCC_HIP(hipMemset(dep, 0, kDepWords * sizeof(uint32_t)));
      OCC_HIP(hipDeviceSynchronize());
      return OCC_ETIMEOUT;
    }
  }

  const double R = c.reps;
  if (flags & OCC_RUN_SEQ) {
    res->t_seq_ms = seq_sum / R;
    res->t_seq_min_ms = seq_min;
    median_and_std(seq_t, res->t_seq_ms, &res->t_seq_median_ms, &res->t_seq_std_ms);
  }
  if (flags & OCC_RUN_OVL) {
    res->t_ovl_ms = ovl_sum / R;
    res->t_ovl_min_ms = ovl_min;
    median_and_std(ovl_t, res->t_ovl_ms, &res->t_ovl_median_ms, &res->t_ovl_std_ms);
  }
  if ((flags & OCC_RUN_SEQ) && (flags & OCC_RUN_OVL) && res->t_seq_ms > 0)
    res->reduction_pct = 100.0 * (1.0 - res->t_ovl_ms / res->t_seq_ms);
  if (flags & OCC_RUN_ISO) {
    res->t_gemm_ms = g_sum / (R * n);
    res->t_comm_ms = c_sum / (R * n);
  }
  return OCC_OK;
}

// Adaptive choice of the occupancy and priority knobs (the runtime policy the
// paper names as future work, Section 6): time the overlapped schedule for
// each candidate and keep the one with the shortest median makespan.
// Candidates: comm wave priority {0, 3} x comm workgroups {one per CU (the
// default), two per CU, one per four CUs} x GEMM grid {one workgroup per tile, persistent one
// per CU} x extra LDS pad {0, the pad that lowers the GEMM's residency by one
// workgroup per CU, when one exists} x dependency {event, device counter}
// (the counter only with one comm workgroup per CU).
int overlap_tune_impl(occ_overlap_cfg *cfg, int tune_reps, occ_overlap_result *res,
                      int *prefer_sequential) {
  if (cfg == nullptr || res == nullptr || prefer_sequential == nullptr || tune_reps < 1)
    return OCC_EINVAL;
  OCC_TRY(validate_cfg(cfg));
  const DeviceInfo *di = nullptr;
  OCC_TRY(current_device_info(&di));

  // the pad that takes one resident GEMM workgroup per CU away, if any
  size_t pads[2] = {0, 0};
  int npads = 1;
  {
    GemmCall g{cfg->A, cfg->B, cfg->C, cfg->M, cfg->N, cfg->K, 0, 0, cfg->gemm_variant,
               cfg->gemm_priority, KHooks{}, cfg->gemm_b_layout == OCC_B_KN};
    occ_gemm_plan p0;
    OCC_TRY(gemm_plan(g, &p0));
    if (p0.wg_per_cu > 1) {
      size_t target = (size_t)di->lds_per_cu / (size_t)p0.wg_per_cu + 1;  // fits one fewer
      if (target > (size_t)p0.tile_lds_bytes) {
        g.lds_bytes = target - (size_t)p0.tile_lds_bytes;
        occ_gemm_plan p1;
        if (gemm_plan(g, &p1) == OCC_OK && p1.wg_per_cu == p0.wg_per_cu - 1) pads[npads++] = g.lds_bytes;
      }
    }
  }
  const int prios[2] = {0, 3};
  // comm grids: one workgroup per CU (the default), two per CU, one per four
  // CUs (a lightweight, low-occupancy collective)
  const int wgs[3] = {0, 2 * di->num_cus, di->num_cus / 4 > 0 ? di->num_cus / 4 : 1};
  const int grids[2] = {0, di->num_cus};
  const int deps[2] = {OCC_DEP_EVENT, OCC_DEP_COUNTER};

  occ_overlap_cfg c = *cfg;
  c.reps = tune_reps;
  c.warmup = 1;
  c.flags = OCC_RUN_OVL | (cfg->flags & (OCC_RUN_GRAPH | OCC_RUN_PACE_ALL));
  c.timeline = nullptr;
  c.wg_trace = nullptr;
  double best = 1e300;
  occ_overlap_cfg best_cfg = c;
  for (int a = 0; a < 2; ++a)
    for (int b = 0; b < 3; ++b)
      for (int d = 0; d < 2; ++d)
        for (int e = 0; e < npads; ++e)
          for (int f = 0; f < 2; ++f) {
            if (deps[f] == OCC_DEP_COUNTER &&
                (wgs[b] > di->num_cus || cfg->n_iter > kMaxDepIter || (c.flags & OCC_RUN_GRAPH)))
              continue;
            c.comm_priority = prios[a];
            c.comm_wgs = wgs[b];
            c.gemm_grid = grids[d];
            c.lds_bytes = pads[e];
            c.dep = deps[f];
            occ_overlap_result r;
            int st = run_overlap_impl(&c, &r);
            if (st == OCC_ELDS) continue;
            if (st != OCC_OK) return st;
            if (r.t_ovl_median_ms < best) {
              best = r.t_ovl_median_ms;
              best_cfg = c;
            }
          }
  cfg->comm_priority = best_cfg.comm_priority;
  cfg->comm_wgs = best_cfg.comm_wgs;
  cfg->gemm_grid = best_cfg.gemm_grid;
  cfg->lds_bytes = best_cfg.lds_bytes;
  cfg->dep = best_cfg.dep;
  OCC_TRY(run_overlap_impl(cfg, res));
  *prefer_sequential = (res->t_seq_median_ms > 0 && res->t_ovl_median_ms > res->t_seq_median_ms) ? 1 : 0;
  return OCC_OK;
}

// The overlapped schedule enqueued without timing or runtime events: GEMMs on
// s0, collectives on s1, K_g^i -> K_c^i by the device counters tk/ack (n
// each, zero on entry, zero again once every collective has passed its
// wait).
int enqueue_impl(const occ_overlap_cfg *cfg, hipStream_t s1, uint32_t *tk, uint32_t *ack, int capacity,
                 uint32_t *err, uint32_t *err_sink) {
  if (cfg == nullptr) return OCC_EINVAL;
  occ_overlap_cfg c = *cfg;
  // the fields a timed run uses are not read here
  c.reps = 1;
  c.warmup = 0;
  c.flags = OCC_RUN_OVL;
  c.dep = OCC_DEP_COUNTER;
  if (cfg->timeline != nullptr || cfg->wg_trace != nullptr) return OCC_EINVAL;
  OCC_TRY(validate_cfg(&c));
  if (c.n_iter > capacity) return OCC_EINVAL;
  if ((c.comm_kind == OCC_COMM_PERMUTE ? c.chunk_bytes : c.len) == 0) return OCC_EINVAL;
  const DeviceInfo *di = nullptr;
  OCC_TRY(current_device_info(&di));
  Launcher L;
  make_launcher(c, &L);
  if (comm_grid(c, L) > di->num_cus) return OCC_EINVAL;
  occ_gemm_plan plan;
  OCC_TRY(gemm_launch_plan(L.g, &plan));
  hipStream_t s0 = static_cast<hipStream_t>(c.stream);
  // nothing here allocates: the hooks of each iteration live on the stack
  for (int i = 0; i < c.n_iter; ++i) {
    KHooks hg{}, hc{};
    counter_hook_pair(L, i, (uint32_t)plan.grid, tk, ack, err != nullptr ? err : err_sink, &hg, &hc);
    OCC_TRY(L.gemm(s0, hg, i));
    OCC_TRY(L.comm(s1, hc, true, i));
  }
  return OCC_OK;
}

size_t overlap_workspace_bytes(int n_iter) {
  if (n_iter < 1) return 0;
  const size_t words = 2 * (size_t)n_iter + 1;
  return (words * sizeof(uint32_t) + 255) & ~(size_t)255;
}

// The counters of occ_overlap_enqueue_noalloc: a library-owned device array
// (one copy per GPU, zero from load), for callers that cannot allocate.  In
// host code `scratch` names a host-side stand-in; its device address on the
// current GPU comes from hipGetSymbolAddress, once per device, and only that
// address is passed to kernels.
constexpr int kNoallocMaxIter = OCC_NOALLOC_MAX_ITER;
static __device__ __align__(256) uint32_t scratch[2 * kNoallocMaxIter + 64];
uint32_t *g_scratch[64];  // device address of `scratch`, per device

int noalloc_scratch(uint32_t **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return OCC_ENODEV;
  if (g_scratch[dev] == nullptr) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return OCC_EHIP;
    g_scratch[dev] = static_cast<uint32_t *>(p);
  }
  *out = g_scratch[dev];
  return OCC_OK;
}

int overlap_enqueue_noalloc_impl(const occ_overlap_cfg *cfg, void *comm_stream, uint32_t *err) {
  if (cfg == nullptr || cfg->n_iter < 1 || cfg->n_iter > kNoallocMaxIter) return OCC_EINVAL;
  const DeviceInfo *di = nullptr;
  OCC_TRY(current_device_info(&di));
  uint32_t *w = nullptr;
  OCC_TRY(noalloc_scratch(&w));
  return enqueue_impl(cfg, static_cast<hipStream_t>(comm_stream), w, w + kNoallocMaxIter, kNoallocMaxIter, err,
                      w + 2 * kNoallocMaxIter);
}

int overlap_enqueue_impl(const occ_overlap_cfg *cfg, void *comm_stream, void *workspace, size_t workspace_bytes,
                         uint32_t *err) {
  if (cfg == nullptr || workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 3u) != 0)
    return OCC_EINVAL;
  if (cfg->n_iter < 1 || workspace_bytes < overlap_workspace_bytes(cfg->n_iter)) return OCC_EINVAL;
  uint32_t *w = static_cast<uint32_t *>(workspace);
  const int n = cfg->n_iter;
  return enqueue_impl(cfg, static_cast<hipStream_t>(comm_stream), w, w + n, n, err, w + 2 * n);
}

}  // namespace occ
