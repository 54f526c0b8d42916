// The spherical softmax in the shifted form section 3.6 prints,
//   L_i = -log((o_c + eps)^2 / sum_j (o_j + eps)^2),   o = W h_i,
// whose output gradient a_i (o + eps 1) - (2 / u_c) e_c (u = o + eps 1,
// a_i = 2 / S_i) has a part eps a_i 1 along the all-ones vector: every row of
// W moves by the same vector each step.  The factored state absorbs it in a
// row c shared by all rows, W = V U + 1 c^T, and keeps s = W^T 1, so that
// sum_j o_j = s^T h stays O(d).  In the step's notation (H columns h_i,
// t_i = c^T h_i, n_i = s^T h_i, B = diag(b_i)):
//   W^T Y    = U^T (V^T Y) + c 1^T                      (one class per example)
//   grad_H   = (Q H + eps s 1^T) A + (W^T Y) B
//   N        = A C1' A + A C2' B + B C2'^T A + B (Y^T Y) B with
//              C1'_ij = C1_ij + eps (n_i + n_j) + D eps^2,  C2'_ij = C2_ij + t_i + eps
//   c       <- c - lr H (A (t + eps 1))                 (from W (I - lr H A H^T) - lr eps 1 (H a)^T)
//   s       <- s - lr H (A (n + D eps 1) + b)           (s - lr H (dL/dO)^T 1)
// while U, U^{-T}, V (with the scatter weight b_i / a_i) and Q (Appendix B,
// which holds for any dL/dO once grad_H and N are right) move as for the
// other losses.  shift_terms, between launches 2 and 3, adds the eps and c
// terms to H^ = Q H, Y^ and NP, and moves c and s: every check that can fail
// the step has run by then (launches 1 and 2), and no later launch reads them.
// The solve-from-scratch form can still fail later (a zero pivot of U_new),
// so there c and s move in a second, update-only launch after the factorisation.
#include "lst_internal.h"

namespace lst {

namespace {

// Blocks [0, nupd): c and s, 16 columns per block, its 16 groups of 16 threads
// taking every 16th example (eight at a time, loads first), summed in a fixed
// order (skipped when the step's error flag is set, like every state update of
// the step).  The other blocks: one 256-wide column chunk of one example's row:
// H^_i += eps s, Y^_i += c (column < d) and the corrections of C1', C2' (and
// C2'^T when it is stored) (column < m).  These read the copy of [c | s] the
// targets task left after nt, not c.sv, which the first blocks move.
constexpr int kUpdCols = 16;
constexpr int kUpdGroups = 16;

__global__ __launch_bounds__(256) void shift_terms_kernel(StepCtx c, int with_c2t, int nupd,
                                                          int chunks) {
  const int m = c.m, d = c.d;
  const float eps = c.eps;
  if ((int)blockIdx.x < nupd) {
    if (c.flags[F_ERR] != 0) return;  // the whole block
    __shared__ float red[2][kUpdGroups][kUpdCols];
    const int col = threadIdx.x % kUpdCols, g = threadIdx.x / kUpdCols;
    const int k = blockIdx.x * kUpdCols + col;
    const float De = (float)c.D * eps;
    float dc = 0.f, ds = 0.f;
    if (k < d) {
      constexpr int U = 8;
      int i = g;
      for (; i + (U - 1) * kUpdGroups < m; i += U * kUpdGroups) {
        float h[U], a[U], b[U], tt[U], nn[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int e = i + u * kUpdGroups;
          h[u] = c.H[(size_t)e * d + k];
          a[u] = c.a[e];
          b[u] = c.b[e];
          tt[u] = c.nt[2 * e];
          nn[u] = c.nt[2 * e + 1];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          dc += a[u] * (tt[u] + eps) * h[u];
          ds += (a[u] * (nn[u] + De) + b[u]) * h[u];
        }
      }
      for (; i < m; i += kUpdGroups) {
        const float h = c.H[(size_t)i * d + k], a = c.a[i];
        dc += a * (c.nt[2 * i] + eps) * h;
        ds += (a * (c.nt[2 * i + 1] + De) + c.b[i]) * h;
      }
    }
    red[0][g][col] = dc;
    red[1][g][col] = ds;
    __syncthreads();
    if (g == 0 && k < d) {
      float tc = 0.f, ts = 0.f;
#pragma unroll
      for (int q = 0; q < kUpdGroups; ++q) {
        tc += red[0][q][col];
        ts += red[1][q][col];
      }
      c.sv[k] -= c.lr * tc;
      c.sv[d + k] -= c.lr * ts;
    }
    return;
  }
  const int q = blockIdx.x - nupd;
  const int i = q / chunks;
  const int j = (q - i * chunks) * 256 + threadIdx.x;
  const float* snap = c.nt + 2 * m;  // [c | s] as the step found them
  if (j < d) {
    c.Z0[(size_t)i * c.ld0 + j] += eps * snap[d + j];
    c.Yh[(size_t)i * d + j] += snap[j];
  }
  if (j < m) {
    float* r = c.NP + (size_t)i * 4 * m;
    const float ti = c.nt[2 * i], ni = c.nt[2 * i + 1];
    r[j] += eps * (ni + c.nt[2 * j + 1]) + (float)c.D * eps * eps;
    r[m + j] += ti + eps;
    if (with_c2t) r[2 * m + j] += c.nt[2 * j] + eps;
  }
}

// Partial column sums over row blocks of at least kColRows rows (at most
// kColParts blocks), then their sum in block order: the same bits on every run.
constexpr int kColRows = 2048;
constexpr int kColParts = 65535;

int64_t column_rows_per_part(int64_t rows) {
  const int64_t r = (rows + kColParts - 1) / kColParts;
  return r > kColRows ? r : kColRows;
}

__global__ __launch_bounds__(256) void column_partials_kernel(const float* __restrict__ A,
                                                              int64_t rows, int cols,
                                                              int64_t per,
                                                              float* __restrict__ part) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= cols) return;
  const int64_t r0 = (int64_t)blockIdx.y * per;
  const int64_t r1 = r0 + per < rows ? r0 + per : rows;
  float acc = 0.f;
  for (int64_t r = r0; r < r1; ++r) acc += A[r * cols + k];
  part[(size_t)blockIdx.y * cols + k] = acc;
}

__global__ __launch_bounds__(256) void column_finish_kernel(const float* __restrict__ part,
                                                            int nparts, int cols,
                                                            float* __restrict__ out) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= cols) return;
  double acc = 0.0;
  for (int p = 0; p < nparts; ++p) acc += part[(size_t)p * cols + k];
  out[k] = (float)acc;
}

__global__ __launch_bounds__(256) void add_row_kernel(float* __restrict__ A, int64_t rows,
                                                      int cols, const float* __restrict__ v) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= cols) return;
  const float x = v[k];
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) A[r * cols + k] += x;
}

}  // namespace

hipError_t shift_terms(const StepCtx& c, bool with_c2t, bool terms, bool update, hipStream_t s) {
  if (c.m < 1 || c.d < 1 || !c.sv || !c.nt) return hipErrorInvalidValue;
  const int w = c.d > c.m ? c.d : c.m;
  const int chunks = (w + 255) / 256;
  const int nupd = update ? (c.d + kUpdCols - 1) / kUpdCols : 0;
  const int blocks = nupd + (terms ? chunks * c.m : 0);
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(shift_terms_kernel, dim3(blocks), dim3(256), 0, s, c, with_c2t ? 1 : 0,
                     nupd, chunks);
  return hipGetLastError();
}

int column_sum_parts(int64_t rows) {
  const int64_t per = column_rows_per_part(rows);
  return (int)((rows + per - 1) / per);
}

hipError_t column_sums(const float* A, int64_t rows, int cols, float* part, float* out,
                       hipStream_t s) {
  if (rows < 1 || cols < 1) return hipErrorInvalidValue;
  const int64_t per = column_rows_per_part(rows);
  const int np = column_sum_parts(rows);
  if (np > kColParts) return hipErrorInvalidValue;
  hipLaunchKernelGGL(column_partials_kernel, dim3((cols + 255) / 256, np), dim3(256), 0, s, A,
                     rows, cols, per, part);
  hipLaunchKernelGGL(column_finish_kernel, dim3((cols + 255) / 256), dim3(256), 0, s, part, np,
                     cols, out);
  return hipGetLastError();
}

hipError_t add_row_vector(float* A, int64_t rows, int cols, const float* v, hipStream_t s) {
  if (rows < 1 || cols < 1) return hipErrorInvalidValue;
  const int64_t gy = rows < 4096 ? rows : 4096;
  hipLaunchKernelGGL(add_row_kernel, dim3((cols + 255) / 256, (unsigned)gy), dim3(256), 0, s, A,
                     rows, cols, v);
  return hipGetLastError();
}

}  // namespace lst
