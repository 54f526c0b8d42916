// C ABI of the library: state ownership, argument checks, and the launches of
// one step (the kernels themselves are in step.hip, gemm.hip, small.hip and
// online.hip).
//
// The factored step (Appendix A) is four heterogeneous launches on the
// state's stream (see step.hip); a single example with at most 256 target
// pairs takes the two launches of online.hip instead.  Shortcuts of the
// minibatch step, exact in real arithmetic:
//   U_new^{-T} H = -(1/lr) P S^{-1} A^{-1}, so with X = S^{-1} P^T (m x d):
//   U_new^{-T} = U^{-T} - X^T H^T and V_new = V - lr G (U_new^{-T} H)^T
//   = V + sum_i (g_i / a_i) X_i, i.e. c = -val (squared) or b_i / a_i (spherical);
//   Q_new = Q - lr (H grad_H^T + grad_H H^T) + lr^2 H N H^T
//         = Q - lr (H T^T + T H^T) with T = grad_H - (lr/2) H N.
// Every update of the state (U, U^{-T}, Q, V) runs after every check that can
// raise a device error of this step, and skips when the error flag is set.
#include <math.h>
#include <stdlib.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "lst_internal.h"

using namespace lst;

// Workspace of lst_stabilize_noalloc: one array per GPU the library runs on,
// held until the process ends.  12 MiB: the Appendix C workspace (two d x d
// products, split-K partials, vectors, per-round flags) for d <= 512 and up
// to 16 corrections at each end.  Host code takes its device address with
// hipGetSymbolAddress (scratch_device_ptr); the array's name in host code is
// not a device address.
constexpr size_t kScratchFloats = (size_t)3 << 20;
static __device__ __align__(256) float scratch[kScratchFloats];

struct lst_state {
  int kind = 0;  // 0 factored, 1 naive
  int64_t D = 0;
  int d = 0;
  lst_config cfg{};
  int device = 0;
  hipStream_t stream = nullptr;
  float* V = nullptr;      // V (factored) or W (naive), D x d
  float* state = nullptr;  // [Q; U; U^{-T}], 3d x d
  float* Vtmp = nullptr;   // D x d copy for the pristine restore
  int* flags = nullptr;
  // factored workspace
  float *G = nullptr, *Z0 = nullptr, *Yh = nullptr, *NP = nullptr, *aH = nullptr, *bH = nullptr,
        *a = nullptr, *b = nullptr, *cs = nullptr, *T = nullptr, *X = nullptr,
        *ex_val = nullptr, *solve_ws = nullptr, *UHa = nullptr, *c1p = nullptr, *yyd = nullptr,
        *hap = nullptr;
  int *ex_row = nullptr, *ex_cnt = nullptr, *hkey = nullptr, *hmin = nullptr, *hcnt = nullptr,
      *touched = nullptr,
      *own = nullptr, *count = nullptr;
  int last_slots = 0;  // m * K of the last factored step
  int hbits = 0;
  int ld0 = 0;
  float* on_ws = nullptr;  // single-example step workspace
  // solve-from-scratch step: A = U_new^T and its LU factors, pivots, the
  // permutation, Z^T; allocated at its first call.  uit_stale: U^{-T} no
  // longer matches U (lst_step refuses the state until lst_restore).
  float *lu_F = nullptr, *lu_Z = nullptr;
  int *lu_ipiv = nullptr, *lu_perm = nullptr;
  int uit_stale = 0;
  float* Nm = nullptr;  // m_max > 128: m x ldn, N = A C1 A + A C2 B + B C2^T A + B Y^T Y B
  int ldn = 0;
  // shifted spherical loss: sv = [c | s] (W = V U + 1 c^T, s = W^T 1) and the
  // per-example [c^T h_i, s^T h_i] of the current step, then a copy of [c | s]
  float *sv = nullptr, *nt = nullptr;
  int n_c1p = 0;  // partial sums of h^T Q h per example (two per 32-column tile of H^)
  int n_hap_max = 0;  // partial sums of |H^T H| per row for m = m_max
  // naive workspace
  float* O = nullptr;
  float* wsplit = nullptr;
  int naive_ksplit = 1;
  int64_t steps = 0;
  std::vector<void*> allocs;
  // captured steps: one instantiated graph per distinct argument tuple (LRU)
  struct GraphEntry {
    int m, K;
    const void *H, *idx, *val, *loss, *grad;
    uint32_t lr_bits;
    hipGraphExec_t exec;
    uint64_t last_use;
  };
  std::vector<GraphEntry> graphs;
  uint64_t graph_clock = 0;
  int split = 0;       // every task of a step as a launch of its own (profiling aid)
  int use_graphs = 0;  // direct launches: graph replay adds device-side gaps between steps
  hipStream_t cap = nullptr;  // capture stream
  float* scratch = nullptr;   // this device's copy of the static scratch array
  // Appendix C stabilisation: workspace (allocated at first use) and the
  // periodic setting
  float* stab_f = nullptr;
  int* stab_i = nullptr;
  int stab_ksplit = 0, stab_rounds = 0;
  int stab_every = 0;
  lst_stab_config stab_cfg{};
  // profiling: two events per phase per profiled step
  int prof = 0;
  std::vector<hipEvent_t> prof_events;
  std::vector<char> prof_recorded;  // per event slot: recorded in the current profile
  size_t prof_used = 0;
  int64_t prof_steps = 0;
};

namespace {

// Device address of `scratch` on each device, taken once per device with that
// device current (each GPU holds its own copy of the array).
std::mutex g_scratch_mu;
std::vector<float*> g_scratch_ptr;

int scratch_device_ptr(int device, float** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (device < 0) return LST_EINVAL;
  if ((size_t)device >= g_scratch_ptr.size()) g_scratch_ptr.resize(device + 1, nullptr);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return LST_EHIP;
    g_scratch_ptr[device] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[device];
  return LST_OK;
}

// GEMM tile edge of launch 1: 64 when m > 128 and 64 x 64 tiles alone fill
// the 256 compute units (half the bytes per output of 32 x 32 tiles), else 32.
// The edge also fixes the number of h^T Q h and |H^T H| partials.
int launch1_tile(int d, int m) {
  return (m > 128 && (size_t)((m + 63) / 64) * ((3 * d + m + 63) / 64) >= 256) ? 64 : 32;
}
// Stages of launch 1's tiles for m > 128 or more tiles than compute units:
// four (64 KB), so that two tiles share a compute unit and the tiles run in
// one round (c4: 448 tiles of 32 x 32 with eight stages took two rounds, 22
// against 17 us).
constexpr int kLaunch1Stages64 = 4;

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

#define HIPCHK(x)                               \
  do {                                          \
    if ((x) != hipSuccess) return LST_EHIP;     \
  } while (0)

#define OK_OR_RETURN(x)            \
  do {                             \
    int rc_ = (x);                 \
    if (rc_ != LST_OK) return rc_; \
  } while (0)

template <class T>
int dalloc(lst_state* s, T** p, size_t count) {
  if (count == 0) count = 1;
  void* q = nullptr;
  if (hipMalloc(&q, count * sizeof(T)) != hipSuccess) return LST_ENOMEM;
  s->allocs.push_back(q);
  *p = static_cast<T*>(q);
  return LST_OK;
}

// Phases of a step for the profile: the launches, and with split tasks
// (lst_set_split_tasks) each task of launch L as a launch of its own,
// PH_TASK0 + (L - 1) * kTaskKinds + its task kind.
constexpr int kTaskKinds = TK_CLEAR + 1;
enum Phase {
  PH_LAUNCH1 = 0, PH_LAUNCH2, PH_LAUNCH3, PH_LAUNCH4, PH_DRIFT, PH_ONLINE_A, PH_ONLINE_B,
  PH_SCRATCH_FACTOR, PH_SCRATCH_SOLVE, PH_TASK0, PH_COUNT = PH_TASK0 + 4 * kTaskKinds
};
const char* const kTaskNames[kTaskKinds] = {"gemm",  "targets", "yy",   "scalars",
                                            "solve", "scatter", "clear"};
const char* const kLaunchNames[PH_TASK0] = {"launch1",  "launch2",  "launch3",
                                            "launch4",  "drift",    "online_a",
                                            "online_b", "scratch.factor", "scratch.solve"};
// "launch<L>.<task>" for the split-task phases
struct PhaseNames {
  char buf[PH_COUNT][32];
  PhaseNames() {
    for (int p = 0; p < PH_COUNT; ++p) {
      if (p < PH_TASK0) {
        snprintf(buf[p], sizeof buf[p], "%s", kLaunchNames[p]);
      } else {
        const int q = p - PH_TASK0;
        snprintf(buf[p], sizeof buf[p], "launch%d.%s", 1 + q / kTaskKinds,
                 kTaskNames[q % kTaskKinds]);
      }
    }
  }
};
const PhaseNames kPhaseNames;

// Records the begin (end = 0) or end (end = 1) event of a phase on stream st
// when profiling.
int prof_mark(lst_state* s, int phase, int end, hipStream_t st) {
  if (!s->prof) return LST_OK;
  const size_t slot = (size_t)(s->prof_steps - 1) * (2 * PH_COUNT) + 2 * phase + end;
  while (s->prof_events.size() <= slot) {
    hipEvent_t e;
    HIPCHK(hipEventCreate(&e));
    s->prof_events.push_back(e);
    s->prof_recorded.push_back(0);
  }
  HIPCHK(hipEventRecord(s->prof_events[slot], st));
  s->prof_recorded[slot] = 1;
  if (slot + 1 > s->prof_used) s->prof_used = slot + 1;
  return LST_OK;
}

// The start and end events of a launch phase of the current profiled step
// (both null when not profiling): the launch records them around its kernel.
int prof_pair(lst_state* s, int phase, hipEvent_t* e0, hipEvent_t* e1) {
  *e0 = *e1 = nullptr;
  if (!s->prof) return LST_OK;
  const size_t slot = (size_t)(s->prof_steps - 1) * (2 * PH_COUNT) + 2 * phase;
  while (s->prof_events.size() <= slot + 1) {
    hipEvent_t e;
    HIPCHK(hipEventCreate(&e));
    s->prof_events.push_back(e);
    s->prof_recorded.push_back(0);
  }
  *e0 = s->prof_events[slot];
  *e1 = s->prof_events[slot + 1];
  s->prof_recorded[slot] = s->prof_recorded[slot + 1] = 1;
  if (slot + 2 > s->prof_used) s->prof_used = slot + 2;
  return LST_OK;
}

void release(lst_state* s) {
  if (!s) return;
  (void)hipStreamSynchronize(s->stream);
  for (auto& g : s->graphs) (void)hipGraphExecDestroy(g.exec);
  for (void* p : s->allocs) (void)hipFree(p);
  s->allocs.clear();
  if (s->stab_f) (void)hipFree(s->stab_f);
  if (s->stab_i) (void)hipFree(s->stab_i);
  for (hipEvent_t e : s->prof_events) (void)hipEventDestroy(e);
  if (s->cap) (void)hipStreamDestroy(s->cap);
  delete s;
}

float* Qp(lst_state* s) { return s->state; }
float* Up(lst_state* s) { return s->state + (size_t)s->d * s->d; }
float* Uitp(lst_state* s) { return s->state + 2 * (size_t)s->d * s->d; }

int check_config(const lst_config* cfg) {
  if (!cfg) return LST_EINVAL;
  if (cfg->loss != LST_LOSS_SQUARED && cfg->loss != LST_LOSS_SPHERICAL &&
      cfg->loss != LST_LOSS_SPHERICAL_SHIFTED)
    return LST_EINVAL;
  if (cfg->loss != LST_LOSS_SQUARED && !(cfg->sph_eps > 0.f && isfinite(cfg->sph_eps)))
    return LST_EINVAL;
  if (cfg->m_max < 1 || cfg->m_max > 512) return LST_EINVAL;
  if (cfg->K_max < 1 || cfg->K_max > 1024) return LST_EINVAL;
  if ((int64_t)cfg->m_max * cfg->K_max > 16384) return LST_EINVAL;
  if (!(cfg->cond_max >= 0.f) || !isfinite(cfg->cond_max)) return LST_EINVAL;
  return LST_OK;
}

int common_init(lst_state* s, int64_t D, int32_t d, const lst_config* cfg, void* hip_stream) {
  s->D = D;
  s->d = d;
  s->cfg = *cfg;
  HIPCHK(hipGetDevice(&s->device));
  s->stream = static_cast<hipStream_t>(hip_stream);
  HIPCHK(hipStreamCreateWithFlags(&s->cap, hipStreamNonBlocking));
  HIPCHK(configure_kernels());
  OK_OR_RETURN(scratch_device_ptr(s->device, &s->scratch));
  OK_OR_RETURN(dalloc(s, &s->flags, F_COUNT));
  HIPCHK(hipMemsetAsync(s->flags, 0, F_COUNT * sizeof(int), s->stream));
  OK_OR_RETURN(dalloc(s, &s->V, (size_t)D * d));
  return LST_OK;
}

// Split-K C = alpha A^T A with A: K x n (rows K), C n x n symmetric, K large.
int gram_splitk(lst_state* s, const float* A, int64_t Krows, int n, float* C, float alpha) {
  const int tiles = ((n + 127) / 128) * ((n + 127) / 128);
  int64_t ks = (2048 + tiles - 1) / tiles;
  const int64_t max_by_k = (Krows + 255) / 256;
  if (ks > max_by_k) ks = max_by_k;
  if (ks < 1) ks = 1;
  if (ks > 256) ks = 256;
  float* ws = nullptr;
  if (hipMalloc((void**)&ws, (size_t)ks * n * n * sizeof(float)) != hipSuccess) return LST_ENOMEM;
  GemmProblem p = gemm_problem(L_TN, n, n, (int)Krows, vmat(A, n, (int)Krows),
                               vmat(A, n, (int)Krows), ws, n, 1.f, 0.f, EPI_PARTIAL);
  p.ksplit = (int)ks;
  int rc = LST_OK;
  if (gemm_big_launch(p, s->stream) != hipSuccess) rc = LST_EHIP;
  if (rc == LST_OK &&
      gemm_splitk_reduce(ws, (int)ks, n, n, C, n, alpha, 0.f, 1, nullptr, s->stream) != hipSuccess)
    rc = LST_EHIP;
  (void)hipStreamSynchronize(s->stream);
  (void)hipFree(ws);
  return rc;
}

// W = Vsrc U into Wdst (D x d) on stream st, optionally gated on device flags.
int vu_product(lst_state* s, hipStream_t st, const float* Vsrc, float* Wdst, const int* run_if,
               const int* skip_if) {
  GemmProblem p = gemm_problem(L_NN, (int)s->D, s->d, s->d, vmat(Vsrc, s->d, (int)s->D),
                               vmat(Up(s), s->d, s->d), Wdst, s->d, 1.f, 0.f, EPI_STORE);
  HIPCHK(gemm_big_launch(p, st, skip_if, run_if));
  return LST_OK;
}

// Shifted spherical loss: s = W0^T 1 from the D x d W0 (synchronises); other
// losses keep s = 0.
int init_column_sums(lst_state* s, const float* W0) {
  if (s->cfg.loss != LST_LOSS_SPHERICAL_SHIFTED) return LST_OK;
  float* part = nullptr;
  if (hipMalloc((void**)&part, (size_t)column_sum_parts(s->D) * s->d * sizeof(float)) !=
      hipSuccess)
    return LST_ENOMEM;
  const bool ok = column_sums(W0, s->D, s->d, part, s->sv + s->d, s->stream) == hipSuccess;
  const bool synced = hipStreamSynchronize(s->stream) == hipSuccess;
  (void)hipFree(part);
  return ok && synced ? LST_OK : LST_EHIP;
}

int ensure_vtmp(lst_state* s) {
  if (s->Vtmp) return LST_OK;
  return dalloc(s, &s->Vtmp, (size_t)s->D * s->d);
}

int read_flag(lst_state* s, int which, int* out) {
  HIPCHK(hipStreamSynchronize(s->stream));
  HIPCHK(hipMemcpy(out, s->flags + which, sizeof(int), hipMemcpyDeviceToHost));
  return LST_OK;
}

int check_step_args(lst_state* s, int32_t m, int32_t K, const float* H, const int32_t* Y_idx,
                    const float* Y_val, float lr, float* loss, float* grad_H) {
  if (!s) return LST_EINVAL;
  if (m < 1 || m > s->cfg.m_max || K < 1 || K > s->cfg.K_max) return LST_EINVAL;
  if (!H || !Y_idx || !loss || !grad_H) return LST_EINVAL;
  if (s->cfg.loss == LST_LOSS_SQUARED && !Y_val) return LST_EINVAL;
  if (s->cfg.loss != LST_LOSS_SQUARED && K != 1) return LST_EINVAL;
  if (!(lr > 0.f) || !isfinite(lr)) return LST_EINVAL;
  return LST_OK;
}

// Partial sums of |H^T H| per row written by the first GEMM: two per tile
// column (edge t) that holds columns of H^T H (Z0 columns [3d, 3d + m)).
int hap_count(int d, int m, int t) {
  const int first = 3 * d / t, end = (3 * d + m + t - 1) / t;
  return 2 * (end - first);
}

// LDS stages of a launch's GEMM tiles: one per K chunk of the longest problem
// (every chunk issued before the first multiply), at most max_stages.
constexpr int kMaxStages = 9;
int stages_for(const GemmBatch& b, int max_stages = kMaxStages) {
  int nch = 1;
  for (int q = 0; q < b.np; ++q) {
    const int ck = 2048 / (b.p[q].tile == 64 ? 64 : 32);  // k per 16 KB stage
    const int n = (b.p[q].K + ck - 1) / ck;
    if (n > nch) nch = n;
  }
  const int st = nch < max_stages ? nch : max_stages;
  return st < 2 ? 2 : st;
}

// Launches 3 and 4 keep at most 4 stages (64 KB): two blocks share a compute
// unit, so the short tasks run beside the GEMM tiles.
constexpr int kLaunch34Stages = 4;
// Above two tiles per compute unit (c5: 1040 tiles in launch 4) two stages
// (32 KB), so that five tiles share a unit and hide each other's loads:
// launch 4 at c5 89 -> 75 us; with fewer tiles the deeper ring wins (c2 +0.8 us).
constexpr int kManyTiles = 512;
int launch34_stages(GemmBatch& g) {
  int tiles = 0;
  for (int q = 0; q < g.np; ++q) {
    const int t = g.p[q].tile == 64 ? 64 : 32;
    const int tm = (g.p[q].M + t - 1) / t, tn = (g.p[q].N + t - 1) / t;
    tiles += g.p[q].epi == EPI_SYM ? tm * (tm + 1) / 2 : tm * tn;
  }
  return tiles > kManyTiles ? 2 : kLaunch34Stages;
}
constexpr int kLaunch2Stages64 = 4;
// Slots a row needs to be scattered by the launch-4 clear blocks instead of its
// owner in launch 3; at most m K / kHotMinSlots rows qualify, which sizes
// their list.
constexpr int kHotMinSlots = 64;
static_assert(kHotMinSlots <= kSlotCap + 1, "rows scattered in launch 3 must fit their slot list");

// Launch `phase` (PH_LAUNCH1 .. PH_LAUNCH4) of the minibatch step: one grid for
// all of its tasks, or with split tasks one launch per task, in task order
// (the tasks of a launch are independent, so the results are the same).
int run_launch(lst_state* s, const StepCtx& c, StepLaunch& L, int stages, hipStream_t st,
               int phase) {
  hipEvent_t e0, e1;
  if (!s->split) {
    OK_OR_RETURN(prof_pair(s, phase, &e0, &e1));
    HIPCHK(step_launch(c, L, stages, st, e0, e1));
    return LST_OK;
  }
  for (int t = 0; t < L.ntask; ++t) {
    StepLaunch one = L;
    one.ntask = 1;
    one.kind[0] = L.kind[t];
    OK_OR_RETURN(prof_pair(s, PH_TASK0 + (phase - PH_LAUNCH1) * kTaskKinds + L.kind[t], &e0, &e1));
    HIPCHK(step_launch(c, one, stages, st, e0, e1));
  }
  return LST_OK;
}

// Drift control after a step (Appendix C, pristine restore when
// ||U||_F ||U^{-T}||_F > cond_max d).
int enqueue_drift(lst_state* s, hipStream_t st) {
  if (!(s->cfg.cond_max > 0.f)) return LST_OK;
  const int d = s->d;
  int* fl = s->flags;
  OK_OR_RETURN(prof_mark(s, PH_DRIFT, 0, st));
  HIPCHK(drift_check(Up(s), Uitp(s), d, s->cfg.cond_max * (float)d, fl, st));
  HIPCHK(copy_if(s->V, s->Vtmp, (size_t)s->D * d, fl + F_RESTORE, st));
  OK_OR_RETURN(vu_product(s, st, s->Vtmp, s->V, fl + F_RESTORE, fl + F_ERR));
  HIPCHK(set_identity_if(Up(s), d, fl + F_RESTORE, st));
  HIPCHK(set_identity_if(Uitp(s), d, fl + F_RESTORE, st));
  return prof_mark(s, PH_DRIFT, 1, st);
}

// The single-example step (Sherman-Morrison update of U^{-T}).
int enqueue_online(lst_state* s, hipStream_t st, int32_t K, const float* H, const int32_t* Y_idx,
                   const float* Y_val, float lr, float* loss, float* grad_H) {
  OnlineArgs a = online_args(s->d, s->on_ws);
  a.K = K;
  a.loss_kind = s->cfg.loss;
  a.D = s->D;
  a.eps = s->cfg.sph_eps;
  a.lr = lr;
  a.h = H; a.idx = Y_idx; a.val = Y_val;
  a.V = s->V; a.Q = Qp(s); a.U = Up(s); a.Uit = Uitp(s);
  a.own = s->own;
  a.flags = s->flags;
  a.loss = loss; a.grad = grad_H;
  hipEvent_t e0a, e1a, e0b, e1b;
  OK_OR_RETURN(prof_pair(s, PH_ONLINE_A, &e0a, &e1a));
  OK_OR_RETURN(prof_pair(s, PH_ONLINE_B, &e0b, &e1b));
  HIPCHK(online_step(a, st, e0a, e1a, e0b, e1b));
  return enqueue_drift(s, st);
}

// Enqueues the launches of one factored step on stream st.
// scratch: the solve-from-scratch form (section 3.5, last paragraph) instead of
// the Woodbury update: no U^{-T} in launch 1 and no Woodbury solve in launch 2;
// after launch 3, A = U_new^T is formed, factored and solved for Z = U_new^{-T} H
// (lu.hip), then the scatter, the Q and U updates and the clear run as launches
// of their own.  U^{-T} is left as it was.
int enqueue_step(lst_state* s, hipStream_t st, int32_t m, int32_t K, const float* H,
                 const int32_t* Y_idx, const float* Y_val, float lr, float* loss, float* grad_H,
                 bool scratch = false) {
  const bool shifted = s->cfg.loss == LST_LOSS_SPHERICAL_SHIFTED;
  if (!scratch && m == 1 && K <= kOnlineMaxK)
    return enqueue_online(s, st, K, H, Y_idx, Y_val, lr, loss, grad_H);
  const int d = s->d;
  int* fl = s->flags;
  StepCtx c{};
  c.m = m; c.K = K; c.d = d; c.D = s->D;
  c.loss_kind = s->cfg.loss; c.eps = s->cfg.sph_eps; c.lr = lr;
  c.H = H; c.idx = Y_idx; c.val = Y_val;
  c.V = s->V; c.Q = Qp(s); c.U = Up(s); c.Uit = Uitp(s);
  c.Z0 = s->Z0; c.ld0 = s->ld0;
  c.G = s->G; c.Yh = s->Yh; c.NP = s->NP; c.aH = s->aH; c.bH = s->bH;
  c.X = s->X; c.T = s->T; c.UHa = s->UHa;
  const int t1 = launch1_tile(d, m);
  c.c1p = s->c1p; c.ld_c1p = s->n_c1p; c.n_c1p = 2 * ((d + t1 - 1) / t1);
  c.hap = s->hap; c.n_hap = hap_count(d, m, t1);
  c.a = s->a; c.b = s->b; c.cs = s->cs; c.yyd = s->yyd;
  c.loss = loss; c.grad = grad_H;
  c.ex_row = s->ex_row; c.ex_val = s->ex_val; c.ex_cnt = s->ex_cnt;
  c.hkey = s->hkey; c.hmin = s->hmin; c.hcnt = s->hcnt; c.hbits = s->hbits;
  c.own = s->own; c.flags = fl; c.solve_ws = s->solve_ws;
  if (shifted) {
    c.sv = s->sv;
    c.nt = s->nt;
  }
  // rows held by kHotMinSlots or more slots are scattered in launch 4, four
  // waves each, when the step has enough slots for such rows to be worth it
  c.hot_min = (m * K >= 4096) ? kHotMinSlots : 0;
  const bool hot = c.hot_min > 0;
  const float* Hh = s->Z0;          // H^ rows
  const float* UH = s->Z0 + d;      // (U H)^T rows

  {  // launch 1: GEMM 1, gather, target prep
    StepLaunch L{};
    L.ntask = 2;
    L.kind[0] = TK_GEMM; L.kind[1] = TK_TARGETS;
    L.gemm.np = 1;
    GemmProblem& p1 = L.gemm.p[0];
    // [Q; U; U^{-T}; H^T] (scratch: [Q; U; H^T], H^T H lands in the P columns)
    const int nst = scratch ? 2 : 3;
    p1 = gemm_problem(L_NT, m, nst * d + m, d, vmat(H, d, m),
                      vmat2(s->state, d, nst * d, H, d, m), s->Z0, s->ld0, 1.f, 0.f, EPI_STORE);
    GemmExtras& x1 = L.gemm.x;
    x1.dotp = s->c1p; x1.ld_dotp = s->n_c1p; x1.dot_ncols = d;  // h_i^T H^_i partials
    if (!scratch) {
      x1.absp = s->hap; x1.ld_absp = c.n_hap; x1.abs_col0 = 3 * d;  // |H^T H| row partials
    }
    p1.tile = t1;
    const int tiles1 = ((m + t1 - 1) / t1) * ((nst * d + m + t1 - 1) / t1);
    x1.dot_h = H; x1.ld_doth = d;
    L.lk = 1;
    L.timing_slot = 0;
    OK_OR_RETURN(run_launch(s, c, L,
                            stages_for(L.gemm, (m > 128 || tiles1 > 256) ? kLaunch1Stages64 : kMaxStages), st,
                            PH_LAUNCH1));
  }
  {  // launch 2: Y^, C1, C2, C2^T ; solve ; Y^T Y ; per-example scalars
    StepLaunch L{};
    L.ntask = 4;
    L.kind[0] = TK_GEMM; L.kind[1] = TK_SOLVE; L.kind[2] = TK_YY; L.kind[3] = TK_SCALARS;
    if (m > 128) {
      // the solve (H^T H read from memory, many iterations' MFMAs per block)
      // outlasts the GEMM tiles, and the merges of Y^T Y take long for long
      // target lists: their blocks go first
      L.kind[0] = TK_SOLVE; L.kind[1] = TK_YY; L.kind[2] = TK_GEMM;
    }
    if (scratch) {
      L.ntask = 3;
      L.kind[0] = TK_GEMM; L.kind[1] = TK_YY; L.kind[2] = TK_SCALARS;
    }
    GemmBatch& g = L.gemm;
    g.np = 3;
    g.p[0] = gemm_problem(L_NN, m, d, d, vmat(s->G, d, m), vmat(c.U, d, d), s->Yh, d, 1.f, 0.f,
                          EPI_STORE);
    // C1, C2 and C2^T go into NP = [C1 | C2 | C2^T | Y^T Y] (row stride 4m); C2^T is
    // stored by C2's tiles
    g.p[1] = gemm_problem(L_NT, m, m, d, vmat(H, d, m), vmat(Hh, s->ld0, m), s->NP, 4 * m, 1.f,
                          0.f, EPI_STORE);
    g.p[2] = gemm_problem(L_NT, m, m, d, vmat(UH, s->ld0, m), vmat(s->G, d, m), s->NP + m, 4 * m,
                          1.f, 0.f, EPI_STORE_T);
    g.p[2].ct_off = m;
    // m > 128: K (d) is long and 64 x 64 tiles fetch half the bytes per
    // output of 32 x 32 ones; with up to 9 stages all of K is in flight.  N is
    // formed before launch 3 from C2 itself, so C2^T is not computed, and the
    // symmetric C1 = H^T Q H runs on its upper-triangle tiles only.
    if (m > 128) {
      g.p[1].epi = EPI_SYM;
      g.p[2].epi = EPI_STORE;
      for (int q = 0; q < g.np; ++q) g.p[q].tile = 64;
    }
    L.lk = 2;
    L.timing_slot = 1;
    // m > 128: four stages (64 KB) so that a GEMM tile and a solve block (whose
    // B stays in registers) share a compute unit and the tiles need not wait
    // for the solve to end
    OK_OR_RETURN(run_launch(s, c, L, stages_for(g, m > 128 ? kLaunch2Stages64 : kMaxStages), st,
                            PH_LAUNCH2));
  }
  // shifted spherical loss: the all-ones terms of grad_H and N; c and s move
  // (for the solve-from-scratch form after its factorisation, which can fail)
  if (shifted) HIPCHK(shift_terms(c, m <= 128, true, !scratch, st));
  {  // launch 3: grad_H and T ; scatter into V
    StepLaunch L{};
    L.ntask = 2;
    // the scatter's blocks are dispatched first: they are short and must not
    // wait behind the GEMM tiles for a compute unit
    L.kind[0] = TK_SCATTER; L.kind[1] = TK_GEMM;
    GemmBatch& g = L.gemm;
    g.np = 1;
    GemmProblem& pt = g.p[0];
    if (m > 128) {
      // N formed first (m x m, elementwise), then T = grad_H - (lr/2) N H^T
      // at the algorithmic size 2 m^2 d
      HIPCHK(form_n(s->NP, s->a, s->b, m, s->Nm, s->ldn, st));
      pt = gemm_problem(L_NN, m, d, m, vmat(s->Nm, s->ldn, m), vmat(H, d, m), s->T, d,
                        -0.5f * lr, 0.f, EPI_GRADN);
    } else {
      // NP viewed as 2m x 2m (row stride 2m): row 2i = [C1 C2]_i, row 2i+1 = [C2^T Y^T Y]_i;
      // times [a H; b H] it gives both halves of (N H^T)_i, combined in the
      // epilogue: four times the multiply-adds of N H^T, but no pass to form N
      pt = gemm_problem(L_NN, 2 * m, d, 2 * m, vmat(s->NP, 2 * m, 2 * m),
                        vmat2(s->aH, d, m, s->bH, d, m), s->T, d, -0.5f * lr, 0.f, EPI_GRADT);
    }
    GemmExtras& xt = g.x;
    xt.e1 = Hh; xt.lde1 = s->ld0; xt.e2 = s->Yh; xt.lde2 = d;
    xt.s1 = s->a; xt.s2 = s->b; xt.g = grad_H; xt.ldg = d;
    pt.tile = 32;
    L.lk = hot ? 6 : 3;
    L.timing_slot = 2;
    if (scratch) {
      L.ntask = 1;
      L.kind[0] = TK_GEMM;
    }
    OK_OR_RETURN(run_launch(s, c, L, stages_for(g, kLaunch34Stages), st, PH_LAUNCH3));
  }
  if (scratch) {
    // A = U_new^T = U^T - lr H^T (U H A): factor it, Z = A^{-1} H, X_i = -lr a_i z_i
    OK_OR_RETURN(prof_mark(s, PH_SCRATCH_FACTOR, 0, st));
    HIPCHK(transpose_square(c.U, s->lu_F, d, st));
    {
      StepLaunch F{};
      F.lk = 4;
      F.ntask = 1;
      F.kind[0] = TK_GEMM;
      F.gemm.np = 1;
      F.gemm.p[0] = gemm_problem(L_TN, d, d, m, vmat(H, d, m), vmat(s->UHa, d, m), s->lu_F, d,
                                 -lr, 1.f, EPI_STORE);
      F.gemm.p[0].tile = 64;
      HIPCHK(step_launch(c, F, stages_for(F.gemm, kLaunch34Stages), st));
    }
    HIPCHK(lu_factor(s->lu_F, d, s->lu_ipiv, s->lu_perm, fl, st));
    OK_OR_RETURN(prof_mark(s, PH_SCRATCH_FACTOR, 1, st));
    OK_OR_RETURN(prof_mark(s, PH_SCRATCH_SOLVE, 0, st));
    HIPCHK(lu_solve_rows(s->lu_F, s->lu_perm, d, H, m, s->lu_Z, s->X, s->a, lr, st));
    if (shifted) HIPCHK(shift_terms(c, m <= 128, false, true, st));
    OK_OR_RETURN(prof_mark(s, PH_SCRATCH_SOLVE, 1, st));
    StepLaunch L{};
    L.ntask = 1;
    L.kind[0] = TK_SCATTER;
    L.lk = hot ? 6 : 3;
    L.timing_slot = 2;
    hipEvent_t e0, e1;
    OK_OR_RETURN(prof_pair(s, PH_TASK0 + 2 * kTaskKinds + TK_SCATTER, &e0, &e1));
    HIPCHK(step_launch(c, L, kLaunch34Stages, st, e0, e1));
  }
  {  // launch 4: Q -= lr (H T^T + T H^T) ; U and U^{-T} updates ; clear the hash slots
    StepLaunch L{};
    // the clear blocks (which also scatter the hot rows) come last: when the
    // tiles fill more than one pass over the compute units, blocks placed
    // first would hold back the tiles for their own latency-bound work
    L.ntask = 2;
    L.kind[0] = TK_GEMM; L.kind[1] = TK_CLEAR;
    GemmBatch& g = L.gemm;
    g.np = 3;
    g.skip_if = fl + F_ERR;  // every product of this launch updates the state
    g.p[0] = gemm_problem(L_TN, d, d, 2 * m, vmat2(H, d, m, s->T, d, m),
                          vmat2(s->T, d, m, H, d, m), c.Q, d, -lr, 1.f, EPI_SYM);
    g.p[0].tile = 32;
    g.p[1] = gemm_problem(L_TN, d, d, m, vmat(s->UHa, d, m), vmat(H, d, m), c.U, d, -lr, 1.f,
                          EPI_STORE);
    g.p[1].tile = 64;
    g.p[2] = gemm_problem(L_TN, d, d, m, vmat(s->X, d, m), vmat(H, d, m), c.Uit, d, -1.f, 1.f,
                          EPI_STORE);
    g.p[2].tile = 64;
    L.lk = hot ? 7 : 4;
    L.timing_slot = 3;
    if (scratch) {
      g.np = 2;  // no U^{-T}
      L.ntask = 1;
    }
    OK_OR_RETURN(run_launch(s, c, L, stages_for(g, launch34_stages(g)), st, PH_LAUNCH4));
    if (scratch) {
      StepLaunch C{};
      C.ntask = 1;
      C.kind[0] = TK_CLEAR;
      C.lk = L.lk;
      C.timing_slot = 3;
      hipEvent_t e0, e1;
      OK_OR_RETURN(prof_pair(s, PH_TASK0 + 3 * kTaskKinds + TK_CLEAR, &e0, &e1));
      HIPCHK(step_launch(c, C, kLaunch34Stages, st, e0, e1));
      return LST_OK;  // drift control needs U^{-T}
    }
  }
  return enqueue_drift(s, st);
}

int check_stab_config(const lst_stab_config* c) {
  if (!c) return LST_EINVAL;
  if (!(c->sigma_low > 0.f) || !(c->sigma_low <= 1.f) || !(c->sigma_high >= 1.f) ||
      !isfinite(c->sigma_high))
    return LST_EINVAL;
  if (c->squarings < 0 || c->squarings > 16 || c->max_fixes < 1 || c->max_fixes > 16)
    return LST_EINVAL;
  if (c->reinvert < 0 || c->reinvert > 2) return LST_EINVAL;
  return LST_OK;
}

// Enqueues one stabilisation on stream st with the workspace f (floats laid
// out by stab_layout(d, ksplit, cfg.max_fixes)) and the round flags in ints.
int enqueue_stabilize_in(lst_state* s, const lst_stab_config& cfg, hipStream_t st, float* f,
                         int* ints, int ksplit) {
  const StabLayout l = stab_layout(s->d, ksplit, cfg.max_fixes);
  StabArgs a{};
  a.D = s->D;
  a.d = s->d;
  a.V = s->V;
  a.U = Up(s);
  a.Uit = Uitp(s);
  a.flags = s->flags;
  a.sigma_low = cfg.sigma_low;
  a.sigma_high = cfg.sigma_high;
  a.squarings = cfg.squarings;
  a.max_fixes = cfg.max_fixes;
  a.reinvert = cfg.reinvert;
  a.ksplit = ksplit;
  a.G = f + l.G; a.G2 = f + l.G2; a.ws = f + l.ws; a.x = f + l.x; a.u = f + l.u; a.w = f + l.w;
  a.wpart = f + l.wpart; a.scal = f + l.scal; a.sig = f + l.sig; a.trace = f + l.trace;
  a.chain = ints;
  a.stop = ints + 2 * (cfg.max_fixes + 1);
  HIPCHK(stabilize_enqueue(a, st));
  return LST_OK;
}

// Reads the report of the stabilisation just enqueued (synchronises).
int read_stab_report(lst_state* s, const lst_stab_config& cfg, const float* f, const int* ints,
                     int ksplit, lst_stab_report* report) {
  const int R = cfg.max_fixes;
  const StabLayout l = stab_layout(s->d, ksplit, R);
  std::vector<int> chain(2 * (R + 1));
  std::vector<float> sig(2 * R);
  HIPCHK(hipStreamSynchronize(s->stream));
  HIPCHK(hipMemcpy(chain.data(), ints, chain.size() * sizeof(int), hipMemcpyDeviceToHost));
  HIPCHK(hipMemcpy(sig.data(), f + l.sig, sig.size() * sizeof(float), hipMemcpyDeviceToHost));
  int fixes[2] = {0, 0};
  float last[2] = {NAN, NAN};
  for (int e = 0; e < 2; ++e)
    for (int r = 0; r < R; ++r) {
      fixes[e] += chain[e * (R + 1) + r + 1];
      if (chain[e * (R + 1) + r]) last[e] = sig[e * R + r];
    }
  report->fixes_low = fixes[0];
  report->fixes_high = fixes[1];
  report->sigma_min = last[0];
  report->sigma_max = last[1];
  return LST_OK;
}

// Enqueues one stabilisation on stream st (the workspace is sized for the
// largest max_fixes seen so far; a larger one reallocates it).
int enqueue_stabilize(lst_state* s, const lst_stab_config& cfg, hipStream_t st) {
  const int d = s->d;
  if (!s->stab_f || cfg.max_fixes > s->stab_rounds) {
    if (s->stab_f) {
      HIPCHK(hipStreamSynchronize(st));
      (void)hipFree(s->stab_f);
      (void)hipFree(s->stab_i);
      s->stab_f = nullptr;
      s->stab_i = nullptr;
    }
    const int ks = stab_ksplit(d);
    const StabLayout l = stab_layout(d, ks, cfg.max_fixes);
    if (hipMalloc((void**)&s->stab_f, l.floats * sizeof(float)) != hipSuccess) return LST_ENOMEM;
    if (hipMalloc((void**)&s->stab_i, l.ints * sizeof(int)) != hipSuccess) {
      (void)hipFree(s->stab_f);
      s->stab_f = nullptr;
      return LST_ENOMEM;
    }
    s->stab_ksplit = ks;
    s->stab_rounds = cfg.max_fixes;
  }
  return enqueue_stabilize_in(s, cfg, st, s->stab_f, s->stab_i, s->stab_ksplit);
}

}  // namespace

extern "C" {

const char* lst_strerror(int status) {
  switch (status) {
    case LST_OK: return "ok";
    case LST_EINVAL: return "invalid argument";
    case LST_EINDEX: return "target index outside [-1, D) (or missing class for the spherical loss)";
    case LST_ESINGULAR: return "Woodbury matrix H^T H - A^{-1}/lr is singular";
    case LST_ENOMEM: return "device allocation failed";
    case LST_EHIP: return "HIP runtime error";
    case LST_ENONFINITE: return "non-finite loss";
    case LST_ESTATE: return "call not valid for this kind of state";
    case LST_ENOSCRATCH:
      return "problem larger than the static workspace of the no-allocation entry point";
    default: return "unknown status";
  }
}

int lst_init(lst_state** out, int64_t D, int32_t d, const float* V, const float* U,
             const lst_config* cfg, void* hip_stream) {
  if (!out || !V || D < 1 || d < 1 || d > 4096 || D > (int64_t)0x7fffffff) return LST_EINVAL;
  if ((int64_t)D * d > ((int64_t)1 << 40)) return LST_EINVAL;
  int rc = check_config(cfg);
  if (rc != LST_OK) return rc;
  lst_state* s = new lst_state();
  s->kind = 0;
  rc = common_init(s, D, d, cfg, hip_stream);
  const int m = cfg->m_max, K = cfg->K_max;
  auto fail = [&](int code) {
    release(s);
    return code;
  };
  if (rc != LST_OK) return fail(rc);
  s->ld0 = (3 * d + m + 3) / 4 * 4;
  s->ldn = (m + 3) / 4 * 4;
  s->n_c1p = 2 * ((d + 31) / 32);  // the most partials (32-column tiles)
  s->n_hap_max = hap_count(d, m, 32) > hap_count(d, m, 64) ? hap_count(d, m, 32)
                                                           : hap_count(d, m, 64);
  s->hbits = 1;
  while ((1 << s->hbits) < 2 * m * K) ++s->hbits;
  const int hsize = 1 << s->hbits;
  const size_t md = (size_t)m * d;
  // [Q; U; U^{-T}] then [c | s] of the shifted loss (the single-example kernels
  // find c and s right after U^{-T})
  if ((rc = dalloc(s, &s->state, 3 * (size_t)d * d + 2 * (size_t)d)) ||
      (rc = dalloc(s, &s->G, md)) ||
      (rc = dalloc(s, &s->Z0, (size_t)m * s->ld0)) || (rc = dalloc(s, &s->Yh, md)) ||
      (rc = dalloc(s, &s->NP, (size_t)4 * m * m)) ||
      (rc = dalloc(s, &s->Nm, m > 128 ? (size_t)m * s->ldn : 0)) || (rc = dalloc(s, &s->aH, md)) ||
      (rc = dalloc(s, &s->bH, md)) ||
      (rc = dalloc(s, &s->a, m)) || (rc = dalloc(s, &s->b, m)) || (rc = dalloc(s, &s->cs, m)) ||
      (rc = dalloc(s, &s->T, md)) || (rc = dalloc(s, &s->X, md)) ||
      (rc = dalloc(s, &s->solve_ws, solve_workspace_floats(m, d))) ||
      (rc = dalloc(s, &s->ex_row, (size_t)m * K)) || (rc = dalloc(s, &s->ex_val, (size_t)m * K)) ||
      (rc = dalloc(s, &s->ex_cnt, m)) || (rc = dalloc(s, &s->hkey, hsize)) ||
      (rc = dalloc(s, &s->hmin, (size_t)hsize * (1 + kSlotCap) + 1 + hsize / 4)) ||
      (rc = dalloc(s, &s->hcnt, hsize + 1 + (size_t)m * K / kHotMinSlots)) ||
      (rc = dalloc(s, &s->touched, (size_t)m * K)) ||
      (rc = dalloc(s, &s->own, (size_t)m * K)) || (rc = dalloc(s, &s->count, 1)) ||
      (rc = dalloc(s, &s->UHa, md)) || (rc = dalloc(s, &s->yyd, m)) ||
      (rc = dalloc(s, &s->c1p, (size_t)m * s->n_c1p)) ||
      (rc = dalloc(s, &s->hap, (size_t)m * s->n_hap_max)) ||
      (rc = dalloc(s, &s->on_ws, online_workspace_floats(d))) ||
      (rc = dalloc(s, &s->nt, 2 * ((size_t)m + d))))
    return fail(rc);
  s->sv = s->state + 3 * (size_t)d * d;
  if (hipMemsetAsync(s->sv, 0, 2 * (size_t)d * sizeof(float), s->stream) != hipSuccess)
    return fail(LST_EHIP);
  if (fill_ints(s->hkey, -1, hsize, s->stream) != hipSuccess ||
      fill_ints(s->hmin, 0x7fffffff, hsize, s->stream) != hipSuccess ||
      fill_ints(s->hcnt, 0, hsize + 1, s->stream) != hipSuccess)
    return fail(LST_EHIP);
  if (cfg->cond_max > 0.f && (rc = ensure_vtmp(s))) return fail(rc);
  if (hipMemcpyAsync(s->V, V, (size_t)D * d * sizeof(float), hipMemcpyDeviceToDevice, s->stream) !=
      hipSuccess)
    return fail(LST_EHIP);
  if (!U) {
    if (set_identity_if(Up(s), d, nullptr, s->stream) != hipSuccess ||
        set_identity_if(Uitp(s), d, nullptr, s->stream) != hipSuccess)
      return fail(LST_EHIP);
    if ((rc = gram_splitk(s, s->V, D, d, Qp(s), 1.f))) return fail(rc);
    if ((rc = init_column_sums(s, s->V))) return fail(rc);
  } else {
    if (hipMemcpyAsync(Up(s), U, (size_t)d * d * sizeof(float), hipMemcpyDeviceToDevice,
                       s->stream) != hipSuccess)
      return fail(LST_EHIP);
    // U^{-T}: invert U (fp64 Gauss-Jordan), then transpose.  The scratch of
    // the inversion lives only for this call.
    double* work = nullptr;
    float* inv = nullptr;
    if (hipMalloc((void**)&work, (size_t)d * d * sizeof(double)) != hipSuccess)
      return fail(LST_ENOMEM);
    if (hipMalloc((void**)&inv, (size_t)d * d * sizeof(float)) != hipSuccess) {
      (void)hipFree(work);
      return fail(LST_ENOMEM);
    }
    const bool inv_ok = invert_small(Up(s), d, inv, d, d, work, s->flags, 0, s->stream) ==
                            hipSuccess &&
                        transpose_square(inv, Uitp(s), d, s->stream) == hipSuccess;
    const bool synced = hipStreamSynchronize(s->stream) == hipSuccess;
    (void)hipFree(work);
    (void)hipFree(inv);
    if (!inv_ok || !synced) return fail(LST_EHIP);
    // Q = (V U)^T (V U).  With drift control on, the product goes through the
    // restore buffer the state keeps anyway; otherwise through a D x d buffer
    // freed right after.
    float* vu = s->Vtmp;
    if (!vu && hipMalloc((void**)&vu, (size_t)D * d * sizeof(float)) != hipSuccess)
      return fail(LST_ENOMEM);
    rc = vu_product(s, s->stream, s->V, vu, nullptr, nullptr);
    if (rc == LST_OK) rc = gram_splitk(s, vu, D, d, Qp(s), 1.f);  // synchronises
    if (rc == LST_OK) rc = init_column_sums(s, vu);
    if (vu != s->Vtmp) {
      (void)hipStreamSynchronize(s->stream);
      (void)hipFree(vu);
    }
    if (rc) return fail(rc);
  }
  int err = 0;
  if ((rc = read_flag(s, F_ERR, &err))) return fail(rc);
  if (err) return fail(err);
  *out = s;
  return LST_OK;
}

int lst_step(lst_state* s, int32_t m, int32_t K, const float* H, const int32_t* Y_idx,
             const float* Y_val, float lr, float* loss, float* grad_H) {
  int rc = check_step_args(s, m, K, H, Y_idx, Y_val, lr, loss, grad_H);
  if (rc != LST_OK) return rc;
  if (s->kind != 0 || s->uit_stale) return LST_ESTATE;
  DeviceGuard dg(s->device);
  if (s->prof || !s->use_graphs) {
    if (s->prof) s->prof_steps += 1;
    rc = enqueue_step(s, s->stream, m, K, H, Y_idx, Y_val, lr, loss, grad_H);
    if (rc == LST_OK) {
      s->steps += 1;
      s->last_slots = m * K;
      if (s->stab_every > 0 && s->steps % s->stab_every == 0)
        rc = enqueue_stabilize(s, s->stab_cfg, s->stream);
    }
    return rc;
  }
  uint32_t lr_bits;
  memcpy(&lr_bits, &lr, sizeof lr_bits);
  lst_state::GraphEntry* hit = nullptr;
  for (auto& g : s->graphs)
    if (g.m == m && g.K == K && g.H == H && g.idx == Y_idx && g.val == Y_val && g.loss == loss &&
        g.grad == grad_H && g.lr_bits == lr_bits) {
      hit = &g;
      break;
    }
  if (!hit) {
    HIPCHK(hipStreamBeginCapture(s->cap, hipStreamCaptureModeRelaxed));
    rc = enqueue_step(s, s->cap, m, K, H, Y_idx, Y_val, lr, loss, grad_H);
    hipGraph_t graph = nullptr;
    const hipError_t ec = hipStreamEndCapture(s->cap, &graph);
    if (rc != LST_OK || ec != hipSuccess) {
      if (graph) (void)hipGraphDestroy(graph);
      return rc != LST_OK ? rc : LST_EHIP;
    }
    hipGraphExec_t exec = nullptr;
    const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (ei != hipSuccess) return LST_EHIP;
    constexpr size_t kMaxGraphs = 32;
    if (s->graphs.size() >= kMaxGraphs) {
      size_t lru = 0;
      for (size_t i = 1; i < s->graphs.size(); ++i)
        if (s->graphs[i].last_use < s->graphs[lru].last_use) lru = i;
      (void)hipStreamSynchronize(s->stream);
      (void)hipGraphExecDestroy(s->graphs[lru].exec);
      s->graphs.erase(s->graphs.begin() + lru);
    }
    s->graphs.push_back({m, K, H, Y_idx, Y_val, loss, grad_H, lr_bits, exec, 0});
    hit = &s->graphs.back();
  }
  hit->last_use = ++s->graph_clock;
  HIPCHK(hipGraphLaunch(hit->exec, s->stream));
  s->steps += 1;
  s->last_slots = m * K;
  if (s->stab_every > 0 && s->steps % s->stab_every == 0)
    return enqueue_stabilize(s, s->stab_cfg, s->stream);
  return LST_OK;
}

int lst_step_solve(lst_state* s, int32_t m, int32_t K, const float* H, const int32_t* Y_idx,
                   const float* Y_val, float lr, float* loss, float* grad_H) {
  int rc = check_step_args(s, m, K, H, Y_idx, Y_val, lr, loss, grad_H);
  if (rc != LST_OK) return rc;
  if (s->kind != 0) return LST_ESTATE;
  if (s->d > kLuMaxD) return LST_EINVAL;
  DeviceGuard dg(s->device);
  if (!s->lu_F) {
    const int d = s->d;
    if ((rc = dalloc(s, &s->lu_F, (size_t)d * d)) ||
        (rc = dalloc(s, &s->lu_Z, (size_t)s->cfg.m_max * d)) || (rc = dalloc(s, &s->lu_ipiv, d)) ||
        (rc = dalloc(s, &s->lu_perm, d)))
      return rc;
  }
  if (s->prof) s->prof_steps += 1;
  rc = enqueue_step(s, s->stream, m, K, H, Y_idx, Y_val, lr, loss, grad_H, true);
  if (rc == LST_OK) {
    s->steps += 1;
    s->last_slots = m * K;
    s->uit_stale = 1;
  }
  return rc;
}

int lst_stabilize(lst_state* s, const lst_stab_config* cfg, lst_stab_report* report) {
  if (!s) return LST_EINVAL;
  OK_OR_RETURN(check_stab_config(cfg));
  if (s->kind != 0 || s->uit_stale) return LST_ESTATE;
  DeviceGuard dg(s->device);
  OK_OR_RETURN(enqueue_stabilize(s, *cfg, s->stream));
  if (!report) return LST_OK;
  return read_stab_report(s, *cfg, s->stab_f, s->stab_i, s->stab_ksplit, report);
}

int lst_stabilize_noalloc(lst_state* s, const lst_stab_config* cfg, lst_stab_report* report) {
  if (!s) return LST_EINVAL;
  OK_OR_RETURN(check_stab_config(cfg));
  if (s->kind != 0 || s->uit_stale) return LST_ESTATE;
  if (!s->scratch) return LST_EHIP;
  const int ks = stab_ksplit(s->d);
  const StabLayout l = stab_layout(s->d, ks, cfg->max_fixes);
  if (l.floats + l.ints > kScratchFloats) return LST_ENOSCRATCH;
  DeviceGuard dg(s->device);
  float* f = s->scratch;
  int* ints = reinterpret_cast<int*>(s->scratch + l.floats);
  OK_OR_RETURN(enqueue_stabilize_in(s, *cfg, s->stream, f, ints, ks));
  if (!report) return LST_OK;
  return read_stab_report(s, *cfg, f, ints, ks, report);
}

int lst_set_stabilize(lst_state* s, int32_t every, const lst_stab_config* cfg) {
  if (!s || every < 0) return LST_EINVAL;
  if (s->kind != 0) return LST_ESTATE;
  if (every > 0) {
    OK_OR_RETURN(check_stab_config(cfg));
    s->stab_cfg = *cfg;
  }
  s->stab_every = every;
  return LST_OK;
}

int lst_materialize_W(lst_state* s, float* W) {
  if (!s || !W) return LST_EINVAL;
  DeviceGuard dg(s->device);
  if (s->kind == 1) {
    HIPCHK(hipMemcpyAsync(W, s->V, (size_t)s->D * s->d * sizeof(float), hipMemcpyDeviceToDevice,
                          s->stream));
    return LST_OK;
  }
  OK_OR_RETURN(vu_product(s, s->stream, s->V, W, nullptr, nullptr));
  if (s->cfg.loss == LST_LOSS_SPHERICAL_SHIFTED)
    HIPCHK(add_row_vector(W, s->D, s->d, s->sv, s->stream));
  return LST_OK;
}

int lst_get_shift(lst_state* s, float* c, float* s_out) {
  if (!s) return LST_EINVAL;
  if (s->kind != 0 || s->cfg.loss != LST_LOSS_SPHERICAL_SHIFTED) return LST_ESTATE;
  DeviceGuard dg(s->device);
  const size_t bytes = (size_t)s->d * sizeof(float);
  if (c) HIPCHK(hipMemcpyAsync(c, s->sv, bytes, hipMemcpyDeviceToDevice, s->stream));
  if (s_out) HIPCHK(hipMemcpyAsync(s_out, s->sv + s->d, bytes, hipMemcpyDeviceToDevice, s->stream));
  return LST_OK;
}

int lst_get_state(lst_state* s, float* Q, float* U, float* UinvT) {
  if (!s) return LST_EINVAL;
  if (s->kind != 0) return LST_ESTATE;
  DeviceGuard dg(s->device);
  const size_t bytes = (size_t)s->d * s->d * sizeof(float);
  if (Q) HIPCHK(hipMemcpyAsync(Q, Qp(s), bytes, hipMemcpyDeviceToDevice, s->stream));
  if (U) HIPCHK(hipMemcpyAsync(U, Up(s), bytes, hipMemcpyDeviceToDevice, s->stream));
  if (UinvT) HIPCHK(hipMemcpyAsync(UinvT, Uitp(s), bytes, hipMemcpyDeviceToDevice, s->stream));
  return LST_OK;
}

int lst_get_V(lst_state* s, float* V) {
  if (!s || !V) return LST_EINVAL;
  if (s->kind != 0) return LST_ESTATE;
  DeviceGuard dg(s->device);
  HIPCHK(hipMemcpyAsync(V, s->V, (size_t)s->D * s->d * sizeof(float), hipMemcpyDeviceToDevice,
                        s->stream));
  return LST_OK;
}

int lst_touched_rows(lst_state* s, int32_t* rows, int32_t capacity, int32_t* count) {
  if (!s || !count || (capacity > 0 && !rows) || capacity < 0) return LST_EINVAL;
  if (s->kind != 0) return LST_ESTATE;
  DeviceGuard dg(s->device);
  int u = 0;
  if (s->steps > 0 && s->last_slots > 0) {
    HIPCHK(compact_owned(s->own, s->last_slots, s->touched, s->count, s->stream));
    HIPCHK(sort_ints(s->touched, s->count, s->stream));
    HIPCHK(hipStreamSynchronize(s->stream));
    HIPCHK(hipMemcpy(&u, s->count, sizeof(int), hipMemcpyDeviceToHost));
  }
  if (u > capacity) return LST_EINVAL;
  if (u > 0) HIPCHK(hipMemcpy(rows, s->touched, (size_t)u * sizeof(int), hipMemcpyDeviceToHost));
  *count = u;
  return LST_OK;
}

int lst_restore(lst_state* s) {
  if (!s) return LST_EINVAL;
  if (s->kind != 0) return LST_ESTATE;
  DeviceGuard dg(s->device);
  OK_OR_RETURN(ensure_vtmp(s));
  HIPCHK(hipMemcpyAsync(s->Vtmp, s->V, (size_t)s->D * s->d * sizeof(float),
                        hipMemcpyDeviceToDevice, s->stream));
  OK_OR_RETURN(vu_product(s, s->stream, s->Vtmp, s->V, nullptr, nullptr));
  HIPCHK(set_identity_if(Up(s), s->d, nullptr, s->stream));
  HIPCHK(set_identity_if(Uitp(s), s->d, nullptr, s->stream));
  s->uit_stale = 0;
  return LST_OK;
}

int lst_naive_init(lst_state** out, int64_t D, int32_t d, const float* W, const lst_config* cfg,
                   void* hip_stream) {
  if (!out || !W || D < 1 || d < 1 || d > 4096 || D > (int64_t)0x7fffffff) return LST_EINVAL;
  int rc = check_config(cfg);
  if (rc != LST_OK) return rc;
  lst_state* s = new lst_state();
  s->kind = 1;
  rc = common_init(s, D, d, cfg, hip_stream);
  auto fail = [&](int code) {
    release(s);
    return code;
  };
  if (rc != LST_OK) return fail(rc);
  const int m = cfg->m_max;
  const int tiles = ((m + 127) / 128) * ((d + 127) / 128);
  int64_t ks = (512 + tiles - 1) / tiles;
  const int64_t max_by_k = (D + 255) / 256;
  if (ks > max_by_k) ks = max_by_k;
  if (ks > 256) ks = 256;
  if (ks < 1) ks = 1;
  s->naive_ksplit = (int)ks;
  if ((rc = dalloc(s, &s->O, (size_t)m * D)) ||
      (rc = dalloc(s, &s->wsplit, (size_t)ks * m * d)))
    return fail(rc);
  if (hipMemcpyAsync(s->V, W, (size_t)D * d * sizeof(float), hipMemcpyDeviceToDevice, s->stream) !=
      hipSuccess)
    return fail(LST_EHIP);
  if (hipStreamSynchronize(s->stream) != hipSuccess) return fail(LST_EHIP);
  *out = s;
  return LST_OK;
}

int lst_naive_step(lst_state* s, int32_t m, int32_t K, const float* H, const int32_t* Y_idx,
                   const float* Y_val, float lr, float* loss, float* grad_H) {
  int rc = check_step_args(s, m, K, H, Y_idx, Y_val, lr, loss, grad_H);
  if (rc != LST_OK) return rc;
  if (s->kind != 1) return LST_ESTATE;
  DeviceGuard dg(s->device);
  const int d = s->d;
  const int64_t D = s->D;
  hipStream_t st = s->stream;
  const bool sq = s->cfg.loss == LST_LOSS_SQUARED;
  // O (m x D) = H^T W^T: every output of every example, O(D d) each
  HIPCHK(gemm_big_launch(gemm_problem(L_NT, m, (int)D, d, vmat(H, d, m), vmat(s->V, d, (int)D),
                                      s->O, (int)D, 1.f, 0.f, EPI_STORE),
                         st));
  HIPCHK(naive_rowstats(s->O, D, D, m, Y_idx, Y_val, K, s->cfg.loss, s->cfg.sph_eps, loss,
                        s->flags, st));
  {  // grad_H = (dL/dO) W  (K = D, split over K)
    GemmProblem p = gemm_problem(L_NN, m, d, (int)D, vmat(s->O, (int)D, m), vmat(s->V, d, (int)D),
                                 s->wsplit, d, 1.f, 0.f, EPI_PARTIAL);
    p.ksplit = s->naive_ksplit;
    HIPCHK(gemm_big_launch(p, st));
    HIPCHK(gemm_splitk_reduce(s->wsplit, s->naive_ksplit, m, d, grad_H, d, sq ? 2.f : 1.f, 0.f, 0,
                              nullptr, st));
  }
  // W -= lr (dL/dO)^T H^T
  HIPCHK(gemm_big_launch(gemm_problem(L_TN, (int)D, d, m, vmat(s->O, (int)D, m), vmat(H, d, m),
                                      s->V, d, sq ? -2.f * lr : -lr, 1.f, EPI_STORE),
                         st, s->flags + F_ERR));
  s->steps += 1;
  return LST_OK;
}

int lst_sync(lst_state* s) {
  if (!s) return LST_EINVAL;
  DeviceGuard dg(s->device);
  int err = 0;
  OK_OR_RETURN(read_flag(s, F_ERR, &err));
  if (err) {
    const int zero = 0;
    HIPCHK(hipMemcpy(s->flags + F_ERR, &zero, sizeof(int), hipMemcpyHostToDevice));
  }
  return err;
}

int lst_stats(lst_state* s, lst_stats_t* st) {
  if (!s || !st) return LST_EINVAL;
  DeviceGuard dg(s->device);
  int f[F_COUNT];
  HIPCHK(hipStreamSynchronize(s->stream));
  HIPCHK(hipMemcpy(f, s->flags, sizeof(f), hipMemcpyDeviceToHost));
  st->steps = s->steps;
  st->restores = f[F_RESTORES];
  st->last_unique = s->kind == 0 ? f[F_UNIQUE] : 0;
  st->last_nnz = s->kind == 0 ? f[F_NNZ] : 0;
  return LST_OK;
}

int lst_profile_enable(lst_state* s, int32_t enable) {
  if (!s) return LST_EINVAL;
  DeviceGuard dg(s->device);
  HIPCHK(hipStreamSynchronize(s->stream));
  s->prof = enable ? 1 : 0;
  s->prof_used = 0;
  std::fill(s->prof_recorded.begin(), s->prof_recorded.end(), 0);
  s->prof_steps = 0;
  return LST_OK;
}

int lst_profile_read(lst_state* s, double* ms_total, int32_t capacity, int32_t* nphases,
                     int64_t* nsteps) {
  if (!s || !nphases || !nsteps || capacity < 0 || (capacity > 0 && !ms_total))
    return LST_EINVAL;
  DeviceGuard dg(s->device);
  HIPCHK(hipStreamSynchronize(s->stream));
  for (int p = 0; p < capacity && p < PH_COUNT; ++p) ms_total[p] = 0.0;
  for (int64_t st = 0; st < s->prof_steps; ++st) {
    for (int p = 0; p < PH_COUNT && p < capacity; ++p) {
      const size_t b = (size_t)st * (2 * PH_COUNT) + 2 * p;
      if (b + 1 >= s->prof_used || !s->prof_recorded[b] || !s->prof_recorded[b + 1]) continue;
      float ms = 0.f;
      HIPCHK(hipEventElapsedTime(&ms, s->prof_events[b], s->prof_events[b + 1]));
      ms_total[p] += ms;
    }
  }
  *nphases = PH_COUNT;
  *nsteps = s->prof_steps;
  s->prof_used = 0;
  std::fill(s->prof_recorded.begin(), s->prof_recorded.end(), 0);
  s->prof_steps = 0;
  return LST_OK;
}

const char* lst_profile_phase_name(int32_t phase) {
  if (phase < 0 || phase >= PH_COUNT) return nullptr;
  return kPhaseNames.buf[phase];
}

int lst_set_split_tasks(lst_state* s, int32_t enable) {
  if (!s) return LST_EINVAL;
  if (s->kind != 0) return LST_ESTATE;
  DeviceGuard dg(s->device);
  HIPCHK(hipStreamSynchronize(s->stream));
  s->split = enable ? 1 : 0;
  // captured steps hold the other launch sequence
  for (auto& g : s->graphs) (void)hipGraphExecDestroy(g.exec);
  s->graphs.clear();
  return LST_OK;
}

int lst_set_graphs(lst_state* s, int32_t enable) {
  if (!s) return LST_EINVAL;
  DeviceGuard dg(s->device);
  HIPCHK(hipStreamSynchronize(s->stream));
  s->use_graphs = enable ? 1 : 0;
  for (auto& g : s->graphs) (void)hipGraphExecDestroy(g.exec);
  s->graphs.clear();
  return LST_OK;
}

void lst_free(lst_state* s) {
  if (!s) return;
  DeviceGuard dg(s->device);
  release(s);
}

}  // extern "C"
