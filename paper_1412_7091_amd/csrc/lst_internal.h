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
  const float* p[4];
  int ld[4];
  int r0[5];
  int nb;
  int vec;              // 1: every block has ld % 4 == 0 and a 16-byte aligned base
  const float* rscale;  // per-row scale or nullptr
};

enum Epi {
  EPI_STORE = 0,    // C = alpha*acc + beta*C
  EPI_SYM = 1,      // upper-triangle tiles only: C[r][c] = C[c][r] = C[r][c] + alpha*acc (r <= c)
  EPI_GRADT = 2,    // g = s1[r]*E1[r][c] + s2[r]*E2[r][c]; G[r][c] = g; C[r][c] = g + alpha*acc
  EPI_PARTIAL = 3   // split-K partial: slice z of a M x N workspace, reduced by gemm_splitk_reduce
};

// Layouts of C = op(A) op(B):  M x K times K x N.
enum Layout {
  L_NT = 0,   // A rows are M (K contiguous), B rows are N (K contiguous)
  L_NN = 1,   // A rows are M (K contiguous), B rows are K (N contiguous)
  L_TN = 2    // A rows are K (M contiguous), B rows are K (N contiguous)
};

struct GemmProblem {
  int M, N, K;
  int a_kc, b_kc;   // 1: the operand's rows are the output dimension (K contiguous)
  VMat A, B;
  float* C;
  int ldc;
  float alpha, beta;
  int epi;
  int ksplit;       // EPI_PARTIAL: number of K slices (>= 1)
  int tiles_m, tiles_n, tile_begin;
  // EPI_GRADT operands
  const float* e1; int lde1;
  const float* e2; int lde2;
  const float* s1;
  const float* s2;
  float* g; int ldg;
  // A operand generated as N (m x m) from its pieces (a_nmat = 1):
  // N_ij = a_i a_j C1_ij + a_i b_j C2_ij + b_i a_j C2t_ij + b_i b_j yy_ij,
  // C1 = nC12[:, 0:m], C2 = nC12[:, m:2m] (leading dimension nld).
  int a_nmat;
  const float* nC12; int nld;
  const float* nC2t;
  const float* nyy;
  const float* na;
  const float* nb;
  int nm;
};

constexpr int kMaxProblems = 4;

struct GemmBatch {
  GemmProblem p[kMaxProblems];
  int np;
  int total_tiles;
  const int* skip_if;  // nonzero *skip_if: every block returns at once
  const int* run_if;   // zero *run_if: every block returns at once
  const int* skip_updates_if;  // nonzero: blocks of problems >= first_update return at once
  int first_update;
  int kcw_max;                 // K chunk width of the panels (multiple of 16)
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
struct StepCtx {
  int m, K, d;
  int64_t D;
  int loss_kind;
  float eps, lr;
  const float* H;
  const int32_t* idx;
  const float* val;
  float *V, *Q, *U, *Uit;
  float* Z0;   // m x ld0: [H^ | UH | P | H^T H] (rows = examples)
  int ld0;
  float *G, *Yh;
  float* C12;  // m x ldc12: [H^T H^ | H^T Y^]
  int ldc12;
  float* C2t;  // m x m: (H^T Y^)^T
  float *X, *T;
  float *a, *b, *cs;  // per example
  float *loss, *grad;
  int* ex_row;  // m x K: each example's target rows, ascending (-1 after the valid ones)
  float* ex_val;
  int* ex_cnt;
  float* yy;   // m x m: Y^T Y
  int *hkey, *hmin;  // hash table of the step's target rows: smallest slot of each
  int hbits;
  int* touched;  // distinct rows of the step (unordered)
  int* flags;
  float* solve_ws;
};

enum TaskKind {
  TK_GEMM = 0, TK_GATHER, TK_PREP, TK_YY, TK_SCALARS, TK_SOLVE, TK_SCATTER, TK_CLEAR
};
constexpr int kMaxTasks = 6;

// One heterogeneous launch: block ranges of its tasks (set by step_launch).
struct StepLaunch {
  int ntask;
  int kind[kMaxTasks];
  int begin[kMaxTasks + 1];
  GemmBatch gemm;  // tiles of the TK_GEMM task (at most one per launch)
  int timing_slot;  // which record of per-block times (builds with LST_TIMING only)
};

// Launches the tasks of L as one grid of 256-thread blocks; GEMM tiles are
// tile x tile (32 or 64).
hipError_t step_launch(const StepCtx& c, StepLaunch& L, int tile, hipStream_t s);
// Floats of global workspace the Woodbury solve needs for its m > 128 fallback.
size_t solve_workspace_floats(int m_max, int d);
// Sorts *n_ptr (<= 16384) ints ascending in place (one block).
hipError_t sort_ints(int* v, const int* n_ptr, hipStream_t s);
hipError_t fill_ints(int* p, int v, int n, hipStream_t s);

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

// ----------------------------------------------------------------- naive
hipError_t naive_rowstats(float* O, int64_t ldo, int64_t D, int m, const int32_t* idx,
                          const float* val, int K, int loss_kind, float eps, float* loss,
                          int* flags, hipStream_t s);

}  // namespace lst
