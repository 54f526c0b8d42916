// Internal declarations shared by the HIP translation units of the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lst.h"

namespace lst {

// ----------------------------------------------------------------- flags
// Device-side int flags of a state.
enum {
  F_ERR = 0,       // sticky status code (0 = ok); update kernels skip when set
  F_RESTORE = 1,   // drift control decided to restore during this step
  F_UNIQUE = 2,    // distinct target rows of the last step
  F_NNZ = 3,       // valid (index, value) pairs of the last step
  F_RESTORES = 4,  // number of restores performed
  F_COUNT = 8
};

// ------------------------------------------------------------------ GEMM
// A "virtual row-major matrix": up to four row blocks stacked on top of each
// other, each with its own base pointer and leading dimension.  Row r of the
// virtual matrix lives in block b with r0[b] <= r < r0[b+1].  An optional
// per-row scale multiplies every element of a row as it is loaded.
struct VMat {
  const float* p[2];
  const float* rscale;  // per-row scale or nullptr
  int ld[2];
  int r1;               // first row of block 1 (nb == 2)
  int nb;
  int vec;              // 1: every block has ld % 4 == 0 and a 16-byte aligned base
};

enum Epi {
  EPI_STORE = 0,    // C = alpha*acc + beta*C
  EPI_SYM = 1,      // upper-triangle tiles only: C[r][c] = C[c][r] = beta_r + alpha*acc (r <= c),
                    // beta_r = C[r][c] when beta != 0, else 0
  EPI_GRADT = 2,    // output rows 2i, 2i+1 pair up into row i (M = 2 x rows of C):
                    //   g = s1[i]*E1[i][c] + s2[i]*E2[i][c]; G[i][c] = g;
                    //   C[i][c] = g + alpha*(s1[i]*acc[2i][c] + s2[i]*acc[2i+1][c])
  EPI_PARTIAL = 3,  // split-K partial: slice z of a M x N workspace, reduced by gemm_splitk_reduce
  EPI_SCALED = 4,   // C = alpha * p * acc + beta * C with p = 2^(-2 ilogb(*s1)) (p = 1 when s1
                    // is null or *s1 is not positive and finite); with g non-null the diagonal
                    // of C is also added into *g (atomically: only its exponent is used)
  EPI_GRADN = 5,    // g = s1[i]*E1[i][c] + s2[i]*E2[i][c]; G[i][c] = g; C[i][c] = g + alpha*acc[i][c]
  EPI_STORE_T = 6   // C[r][c] = alpha*acc and its transpose at C + ct_off: C[ct_off + c*ldc + r]
};
// s1, s2, E1, E2, G (and the row sums of EPI_STORE) are the batch's extras
// (GemmExtras): only batches of one problem use them.

// Layouts of C = op(A) op(B):  M x K times K x N.
enum Layout {
  L_NT = 0,   // A rows are M (K contiguous), B rows are N (K contiguous)
  L_NN = 1,   // A rows are M (K contiguous), B rows are K (N contiguous)
  L_TN = 2    // A rows are K (M contiguous), B rows are K (N contiguous)
};

struct alignas(64) GemmProblem {  // whole kernel-argument cache lines each
  int M, N, K;
  int a_kc, b_kc;   // 1: the operand's rows are the output dimension (K contiguous)
  int ldc;
  float alpha, beta;
  int epi;
  int ksplit;       // EPI_PARTIAL: number of K slices (>= 1)
  int tile;         // step GEMMs: output tile edge, 32 or 64 (0: 32)
  int tiles_m, tiles_n, tile_begin;
  int ct_off;       // EPI_STORE_T: offset of the transpose from C
  VMat A, B;
  float* C;
};

// Epilogue operands that only a batch of one problem uses (its p[0]).
struct GemmExtras {
  // EPI_GRADT / EPI_GRADN (and s1, g of EPI_SCALED)
  const float* e1;
  const float* e2;
  const float* s1;
  const float* s2;
  float* g;
  // EPI_STORE only: per-row partial dot products of the first dot_ncols
  // output columns with dot_h (same row and column), one per (tile column,
  // wave column): dotp[row * ld_dotp + 2 * tile_n + wave_n].
  float* dotp;
  const float* dot_h;
  // EPI_STORE only: per-row partial sums of |C| over the output columns
  // >= abs_col0, one per (tile column, wave column) from the tile column
  // abs_col0 / tile on: absp[row * ld_absp + 2 * (tile_n - abs_col0 / tile) + wave_n].
  float* absp;
  int lde1, lde2, ldg;
  int ld_dotp, dot_ncols, ld_doth;
  int ld_absp, abs_col0;
};

constexpr int kMaxProblems = 3;

struct GemmBatch {
  // Header first: a block finds its problem and its options from these
  // without touching the (large) problem descriptors, whose kernel-argument
  // lines it would otherwise fetch one after another.
  int np;
  int total_tiles;
  int tile_begins[kMaxProblems + 1];  // first tile of each problem; [np] = total_tiles
  int stages;                  // LDS stages of the K pipeline (>= 2)
  int timing_slot;             // record of per-block phase times (builds with LST_TIMING only)
  int first_update;
  const int* skip_if;          // nonzero *skip_if: every block returns at once
  const int* run_if;           // zero *run_if: every block returns at once
  const int* skip_updates_if;  // nonzero: blocks of problems >= first_update return at once
  GemmExtras x;                // with np == 1: the extra operands of p[0]'s epilogue
  GemmProblem p[kMaxProblems];
};

// One-time kernel attribute setup (dynamic LDS limits); call before any launch.
hipError_t configure_kernels();

VMat vmat(const float* p, int ld, int rows, const float* rscale = nullptr);
VMat vmat2(const float* p0, int ld0, int rows0, const float* p1, int ld1, int rows1);
GemmProblem gemm_problem(int layout, int M, int N, int K, const VMat& A, const VMat& B, float* C,
                         int ldc, float alpha, float beta, int epi);
// One large product (EPI_STORE or EPI_PARTIAL) on 128 x 128 double-buffered tiles.
hipError_t gemm_big_launch(GemmProblem p, hipStream_t s, const int* skip_if = nullptr,
                           const int* run_if = nullptr);
// Split-K: C = alpha * sum_z ws[z] + beta * C (sym: r <= c mirrored).
hipError_t gemm_splitk_reduce(const float* ws, int splits, int M, int N, float* C, int ldc,
                              float alpha, float beta, int sym, const int* skip_if,
                              hipStream_t s);

// ------------------------------------------------------------ the step
// Everything the tasks of one factored step read or write (device pointers).
// Slots of a row that its hash entry lists (a row held by more is found by
// searching the examples' target lists instead).
constexpr int kSlotCap = 64;

// Slots per scatter wave: one while a step has at most kScatterOneSlot slots;
// above, about kScatterWaves waves, few enough to be resident together beside
// launch 3's tiles, so that the step's slots are looked up in one pass of
// memory latency instead of one per round of workgroups.
constexpr int kScatterOneSlot = 2048;
constexpr int kScatterWaves = 1024;
__host__ __device__ inline int scatter_slots_per_wave(int slots) {
  if (slots <= kScatterOneSlot) return 1;
  const int s = (slots + kScatterWaves - 1) / kScatterWaves;
  return s > 64 ? 64 : s;
}

// The scalars come first and the pointers after them, so that the struct (a
// kernel argument of every launch of the step) holds no padding.
struct StepCtx {
  int m, K, d;
  // rows held by hot_min or more slots (hot_min 0: none) are not scattered by
  // their owner in launch 3 but listed (hot_list) and scattered by the clear
  // blocks of launch 4, which does not read V
  int hot_min;
  int64_t D;
  int loss_kind;
  float eps, lr;
  int ld0;            // row stride of Z0
  int ld_c1p, n_c1p;  // row stride and number of partials per example of c1p
  int n_hap;          // partials per example of hap
  int hbits;   // hmin's 2^hbits entries are followed by 2^hbits x kSlotCap more: the
               // slots of each row, in no particular order (the first kSlotCap of
               // them; entries past the row's count are stale)
  const float* H;
  const int32_t* idx;
  const float* val;
  float *V, *Q, *U, *Uit;
  float* Z0;   // m x ld0: [H^ | UH | P | H^T H] (rows = examples)
  float *G, *Yh;
  float* NP;   // m x 4m: [C1 | C2 | C2^T | Y^T Y] with C1 = H^T H^, C2 = H^T Y^
  float *X, *T;
  float* UHa;         // m x d: a_i (U h_i)^T, the left factor of the U update
  float *aH, *bH;     // m x d: a_i h_i^T and b_i h_i^T
  float* c1p;         // m x ld_c1p: partial sums of h_i^T Q h_i (from launch 1)
  float* hap;         // m x n_hap: partial sums of |H^T H| along row i (from launch 1)
  float *a, *b, *cs;  // per example
  float* yyd;         // per example: (Y^T Y)_ii
  float *loss, *grad;
  int* ex_row;  // m x K: each example's target rows, ascending (-1 after the valid ones)
  float* ex_val;
  int* ex_cnt;
  int *hkey, *hmin, *hcnt;  // hash table of the step's target rows: smallest slot
                            // and number of slots of each; hcnt's 2^hbits counts
                            // are followed by the hot-row list ([0]: count, then rows)
  int* own;      // m x K: the row of slot i*K + k if that slot owns the row's
                 // scatter in this step (its smallest slot), else -1
  int* flags;
  float* solve_ws;
  // shifted spherical loss only (else null): sv = [c | s] (2 d floats) with
  // W = V U + 1 c^T and s = W^T 1; nt = per example [t_i, n_i] = [c^T h_i, s^T h_i],
  // then a copy of [c | s] as the step found them
  float* sv;
  float* nt;
};
static_assert(sizeof(StepCtx) == 336, "StepCtx is a kernel argument of every launch: keep it small");

enum TaskKind {
  TK_GEMM = 0, TK_TARGETS, TK_YY, TK_SCALARS, TK_SOLVE, TK_SCATTER, TK_CLEAR
};
constexpr int kMaxTasks = 6;

// One heterogeneous launch: block ranges of its tasks (set by step_launch).
// lk selects the kernel built for that launch of the step, which contains only
// the tasks, GEMM layouts and epilogues that launch uses: 1..4 the step's
// launches, 5 the stabilisation's products, 6 and 7 launches 3 and 4 of a step
// that scatters its hot rows in launch 4.
struct StepLaunch {
  int lk;
  int ntask;
  int kind[kMaxTasks];
  int begin[kMaxTasks + 1];
  GemmBatch gemm;  // tiles of the TK_GEMM task (at most one per launch)
  int timing_slot;  // which record of per-block times (builds with LST_TIMING only)
};

// Launches the tasks of L as one grid of 256-thread blocks; each GEMM problem
// has its own tile edge (GemmProblem::tile), all share `stages` LDS stages
// (>= 2).  With ev0 / ev1 the launch records them at the start and the end of
// the kernel's execution.
// N = A C1 A + A C2 B + B C2^T A + B (Y^T Y) B (A = diag(a), B = diag(b)) into
// an m x ldn buffer (columns m .. ldn - 1 zero) from NP = [C1 | C2 | C2^T | Y^T Y].
// The shifted spherical loss (shifted.hip; c.sv = [c | s], W = V U + 1 c^T,
// s = W^T 1): after launch 2, shift_terms adds its all-ones terms to H^, Y^,
// C1 and C2 (and C2^T when with_c2t) when terms is set, and moves c and s when
// update is set (skipped when the step's error flag is set).  c.nt holds
// 2 m + 2 d floats: [t_i, n_i] per example, then the copy of [c | s] the
// targets task of launch 1 makes.
hipError_t shift_terms(const StepCtx& c, bool with_c2t, bool terms, bool update, hipStream_t s);
// out[k] = sum of column k of the rows x cols row-major A, through
// column_sum_parts(rows) x cols floats of partials in part.
int column_sum_parts(int64_t rows);
hipError_t column_sums(const float* A, int64_t rows, int cols, float* part, float* out,
                       hipStream_t s);
// A[r][k] += v[k] for every row r of the rows x cols row-major A.
hipError_t add_row_vector(float* A, int64_t rows, int cols, const float* v, hipStream_t s);

hipError_t form_n(const float* NP, const float* a, const float* b, int m, float* N, int ldn,
                  hipStream_t s);
hipError_t step_launch(const StepCtx& c, StepLaunch& L, int stages, hipStream_t s,
                       hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// 1 when every operand of the batch allows 16-byte LDS-DMA (aligned rows with
// ld % 4 == 0, and K % 4 == 0 where k is the contiguous index).
int gemm_batch_vec16(const GemmBatch& b);
// Floats of global workspace the Woodbury solve needs for its m > 128 fallback.
size_t solve_workspace_floats(int m_max, int d);
// Sorts *n_ptr (<= 16384) ints ascending in place (one block).
hipError_t sort_ints(int* v, const int* n_ptr, hipStream_t s);
// out <- the entries of own[0 .. n) that are >= 0 (unordered); *count <- their number.
hipError_t compact_owned(const int* own, int n, int* out, int* count, hipStream_t s);
hipError_t fill_ints(int* p, int v, int n, hipStream_t s);

// ------------------------------------------------- the single-example step
// Two launches for m = 1 (three for d > 1024; online.hip).  Workspace: one
// float buffer of online_workspace_floats(d), carved by online_args.
constexpr int kOnlineMaxK = 256;
constexpr int kOnlineMaxRows = 16;    // rows per block of launch B (d <= 4096)
constexpr int kOnlineFuseTiles = 16;  // launch B adds the partials itself up to 16 tiles a side
constexpr int kOnlineMaxTiles = 64;   // tiles a side for d = 4096
struct OnlineArgs {
  int d, K, nt, rows_per_block, loss_kind;
  int64_t D;
  float eps, lr;
  const float* h;
  const int32_t* idx;
  const float* val;
  float *V, *Q, *U, *Uit;
  float* part;  // 4 x nt x d: per-tile partial sums of Q h, U h, U^{-T} h, U^T V^T y
  float* vec;   // 4 x d: the same vectors, finished (d > 1024)
  float* sp;    // 3 x nt: per-slab partials of h^T Q h, h^T h, h^T y^ (d > 1024)
  float* scal;  // [0]: y^T y
  float* rsum;  // K: summed value of each owning slot, followed by kOnlineMaxK - K
                // unused entries and 2 d floats: the copy of [c | s] that launch A
                // makes for the shifted loss, whose [c | s] follow U^{-T} (Uit + d^2)
  int* own;     // K: the row of slot k if slot k is the row's first, else -1
  int* flags;
  float *loss, *grad;
};
int online_tiles(int d);
size_t online_workspace_floats(int d);
OnlineArgs online_args(int d, float* ws);
// With e0a/e1a (e0b/e1b) the first (last) launch records them at its start and end.
hipError_t online_step(const OnlineArgs& a, hipStream_t s, hipEvent_t e0a = nullptr,
                       hipEvent_t e1a = nullptr, hipEvent_t e0b = nullptr,
                       hipEvent_t e1b = nullptr);

// ----------------------------------------- the solve-from-scratch step (lu.hip)
constexpr int kLuMaxD = 1024;
// In place P A = L R of the d x d row-major A (partial pivoting); ipiv[k] = the
// row swapped with row k at step k, perm[j] = the row of A that ends at row j.
// LST_ESINGULAR in flags[F_ERR] on a zero or non-finite pivot (the
// factorisation runs on; its output is then meaningless).
hipError_t lu_factor(float* A, int d, int* ipiv, int* perm, int* flags, hipStream_t s);
// With F, perm from lu_factor of A: row i of H (m x d) is h_i^T; writes
// z_i = A^{-1} h_i to row i of X2 and -lr acoef[i] z_i to row i of Xout.
hipError_t lu_solve_rows(const float* F, const int* perm, int d, const float* H, int m, float* X2,
                         float* Xout, const float* acoef, float lr, hipStream_t s);

// ------------------------------------------------------------ small dense
// Sinv = S^{-1} (Gauss-Jordan, partial pivoting); sets F_ERR = LST_ESINGULAR on a zero pivot.
hipError_t invert_small(const float* S, int lds, float* Sinv, int ldi, int m, double* work,
                        int* flags, int check_err, hipStream_t s);
// Drift control: F_RESTORE = (||U||_F ||Uit||_F > thr) and no error.
hipError_t drift_check(const float* U, const float* Uit, int d, float thr, int* flags,
                       hipStream_t s);
hipError_t copy_if(const float* src, float* dst, size_t n, const int* run_if, hipStream_t s);
hipError_t set_identity_if(float* A, int d, const int* run_if, hipStream_t s);
hipError_t set_flag(int* p, int v, hipStream_t s);
hipError_t transpose_square(const float* A, float* At, int d, hipStream_t s);

// ---------------------------------------------------- Appendix C stabilisation
// Everything one stabilisation call reads or writes (device pointers).
struct StabArgs {
  int64_t D;
  int d;
  float *V, *U, *Uit;
  const int* flags;
  float sigma_low, sigma_high;
  int squarings, max_fixes, reinvert, ksplit;
  // workspace (StabLayout offsets into one float buffer, chain in an int buffer)
  float *G, *G2, *ws, *x, *u, *w, *wpart, *scal, *sig;
  float* trace;  // 2 x max_fixes x (kStabMaxSquarings + 1) traces of the round's products
  int* chain;  // 2 x (max_fixes + 1) round flags: [end][0] = no pending error,
               // [end][r + 1] = round r of that end corrected a singular value
  int* stop;   // the same flags negated (the tile products skip while set)
};
constexpr int kStabMaxSquarings = 16;
struct StabLayout {
  size_t G, G2, ws, x, u, w, wpart, scal, sig, trace, floats, ints;
};
StabLayout stab_layout(int d, int ksplit, int max_fixes);
int stab_ksplit(int d);
hipError_t stabilize_enqueue(const StabArgs& a, hipStream_t s);

// ----------------------------------------------------------------- naive
hipError_t naive_rowstats(float* O, int64_t ldo, int64_t D, int m, const int32_t* idx,
                          const float* val, int K, int loss_kind, float eps, float* loss,
                          int* flags, hipStream_t s);

}  // namespace lst
