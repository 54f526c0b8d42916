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
};

constexpr int kMaxProblems = 3;

struct GemmBatch {
  GemmProblem p[kMaxProblems];
  int np;
  int total_tiles;
  const int* skip_if;  // nonzero *skip_if: every block returns at once
  const int* run_if;   // zero *run_if: every block returns at once
  const int* skip_updates_if;  // nonzero: blocks of problems >= first_update return at once
  int first_update;
};

VMat vmat(const float* p, int ld, int rows, const float* rscale = nullptr);
VMat vmat2(const float* p0, int ld0, int rows0, const float* p1, int ld1, int rows1);
GemmProblem gemm_problem(int layout, int M, int N, int K, const VMat& A, const VMat& B, float* C,
                         int ldc, float alpha, float beta, int epi);
// Launches every problem of the batch in one grid.  tile: 64 or 32 (square
// output tiles), 0 = choose from the number of tiles.
hipError_t gemm_launch(GemmBatch& b, hipStream_t s, int tile = 0);
// Split-K: C = alpha * sum_z ws[z] + beta * C (sym: r <= c mirrored).
hipError_t gemm_splitk_reduce(const float* ws, int splits, int M, int N, float* C, int ldc,
                              float alpha, float beta, int sym, const int* skip_if,
                              hipStream_t s);

// ----------------------------------------------------- sparse target side
struct SparseWs {
  int* ex_row;       // m x K: per-example target rows sorted ascending (then by slot)
  float* ex_val;     // m x K: values in the same order
  int* ex_cnt;       // m: valid pairs per example
  unsigned long long* keys;  // m x K: (row << 32 | slot) or ~0 for unused slots
  int* srt_slot;     // m*K: slots in (row, slot) order
  int* seg_row;      // m*K: distinct rows, ascending
  int* seg_beg;      // m*K + 1: first sorted position of each distinct row
  float* yy;         // m x m: Y^T Y
};

hipError_t prep_examples(const int32_t* idx, const float* val, int m, int K, int64_t D,
                         int one_hot, SparseWs ws, int* flags, hipStream_t s);
hipError_t prep_global_sort(int m, int K, SparseWs ws, int* flags, hipStream_t s);
hipError_t prep_target_gram(int m, int K, SparseWs ws, hipStream_t s);
// G[i, :] = sum_k w_ik V[idx_ik, :]  (w = val, or 1 when one_hot)
hipError_t gather_rows(const float* V, int64_t D, int d, const int32_t* idx, const float* val,
                       int m, int K, int one_hot, float* G, int ldg, hipStream_t s);
// V[r, :] += sum over the pairs (i,k) with idx_ik = r, in slot order, of coef * X[i, :]
// coef = -val[i*K+k] (squared) or cs[i] (per-example coefficient).
hipError_t scatter_rows(float* V, int d, const float* X, int ldx, const float* val,
                        const float* cs, int m, int K, SparseWs ws, const int* flags,
                        hipStream_t s);

// ------------------------------------------------------------ small dense
// Per-example loss terms (loss, a, b, cs = b/a) and the m x m matrix N of the step.
hipError_t minibatch_scalars(int loss_kind, float eps, int64_t D, int m, const float* C12,
                             int ldc12, const float* yy, float* loss, float* a, float* b,
                             float* cs, float* N, int* flags, hipStream_t s);
// X = S^{-1} P^T (m x d) with S = H^T H - diag(1 / (lr a_i)), in 16-column blocks.
hipError_t woodbury_solve(const float* HH, int ldh, const float* P, int ldp, int m, int d,
                          int loss_kind, float eps, int64_t D, float lr, const float* C12,
                          int ldc12, float* X, int ldx, float* gj_ws, int* flags, hipStream_t s);
// Floats of global workspace woodbury_solve needs for its m > 128 fallback.
size_t woodbury_workspace_floats(int m_max, int d);
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
