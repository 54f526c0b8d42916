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
// other losses.  shift_terms adds the eps and c terms to H^ = Q H, Y^ and NP
// between launches 2 and 3; shift_update moves c and s after launch 4.
#include "lst_internal.h"

namespace lst {

namespace {

// One block row per example i, one thread per column: H^_i += eps s, Y^_i += c
// (j < d) and the corrections of C1', C2' (and C2'^T when it is stored) (j < m).
__global__ __launch_bounds__(256) void shift_terms_kernel(StepCtx c, int with_c2t) {
  const int i = blockIdx.y;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int m = c.m, d = c.d;
  const float eps = c.eps;
  if (j < d) {
    c.Z0[(size_t)i * c.ld0 + j] += eps * c.sv[d + j];
    c.Yh[(size_t)i * d + j] += c.sv[j];
  }
  if (j < m) {
    float* r = c.NP + (size_t)i * 4 * m;
    const float ti = c.nt[2 * i], ni = c.nt[2 * i + 1];
    r[j] += eps * (ni + c.nt[2 * j + 1]) + (float)c.D * eps * eps;
    r[m + j] += ti + eps;
    if (with_c2t) r[2 * m + j] += c.nt[2 * j] + eps;
  }
}

// One thread per column k of c and s; the m examples are summed in order.
// Skips (like every state update of the step) when the error flag is set.
__global__ __launch_bounds__(256) void shift_update_kernel(StepCtx c) {
  if (c.flags[F_ERR] != 0) return;
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  const int d = c.d;
  if (k >= d) return;
  const float eps = c.eps, De = (float)c.D * eps;
  float dc = 0.f, ds = 0.f;
  for (int i = 0; i < c.m; ++i) {
    const float h = c.H[(size_t)i * d + k];
    const float a = c.a[i];
    dc += a * (c.nt[2 * i] + eps) * h;
    ds += (a * (c.nt[2 * i + 1] + De) + c.b[i]) * h;
  }
  float* sv = const_cast<float*>(c.sv);
  sv[k] -= c.lr * dc;
  sv[d + k] -= c.lr * ds;
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

hipError_t shift_terms(const StepCtx& c, bool with_c2t, hipStream_t s) {
  if (c.m < 1 || c.d < 1 || !c.sv || !c.nt) return hipErrorInvalidValue;
  const int w = c.d > c.m ? c.d : c.m;
  hipLaunchKernelGGL(shift_terms_kernel, dim3((w + 255) / 256, c.m), dim3(256), 0, s, c,
                     with_c2t ? 1 : 0);
  return hipGetLastError();
}

hipError_t shift_update(const StepCtx& c, hipStream_t s) {
  if (c.m < 1 || c.d < 1 || !c.sv || !c.nt) return hipErrorInvalidValue;
  hipLaunchKernelGGL(shift_update_kernel, dim3((c.d + 255) / 256), dim3(256), 0, s, c);
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
