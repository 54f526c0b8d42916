// Pivoted LU factorisation and row solves for the solve-from-scratch step
// (section 3.5, last paragraph): instead of carrying U^{-T} from step to step
// through the Woodbury identity, factor A = U_new^T every step and solve
// A z_i = h_i for the m examples of the minibatch, O(d^3) + O(m d^2) work.
//
// Factorisation (right-looking, partial pivoting, P A = L R): panels of 32
// columns.  Per panel three launches:
//   lu_panel_kernel  one workgroup factors the panel (rows j0 .. d) in
//                    registers: per column an arg-max over the rows (ties to
//                    the lower row), the swap, the multipliers and the rank-1
//                    update of the panel's remaining columns;
//   lu_apply_kernel  every other column: the panel's row interchanges (the
//                    rows involved staged in LDS), then right of the panel the
//                    forward substitution with the panel's unit lower triangle;
//   trailing update  A22 -= L21 U12 on the library's 128 x 128 MFMA tiles.
// Row solves, in the examples' row layout (row i of X holds z_i^T): with
// P A = L R, A z = h is z = R^{-1} L^{-1} P h.  Column blocks of 64 go forward
// through L (unit lower, ascending) and back through R (descending); each
// block first takes the product with the entries already solved, then solves
// its 64 x 64 triangle.  The last pass writes X_i = -lr a_i z_i, the form the
// step's scatter consumes.
#include <hip/hip_runtime.h>
#include <math.h>

#include "lst_internal.h"

namespace lst {

namespace {

constexpr int kLuNB = 32;            // panel width
constexpr int kSolveNB = 64;         // column block of the row solves
constexpr int kSolveRows = 16;       // rows of X per workgroup of the row solves

// Panel: columns j0 .. j0 + nc of rows j0 .. d - 1.  Row j0 + t lives in the
// registers of thread t (1024 threads: d <= 1024); per column only the pivot
// row and the arg-max partials go through LDS.  Each column is its own
// template instance, so every register index is a constant.
constexpr int kPanelThreads = kLuMaxD;

struct PanelShared {
  float best[kPanelThreads / 64];
  int bidx[kPanelThreads / 64];
  int p;
  int piv[kLuNB];  // the panel's pivot rows, written to ipiv at the end
  float prow[kLuNB];
  float old[kLuNB];
};

template <int C>
struct PanelColumn {
  __device__ __forceinline__ static void run(float (&a)[kLuNB], PanelShared& sh, int d, int j0,
                                             int nc, int* ipiv, int* flags) {
    if (C < nc) {
      const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
      const int r = j0 + tid, rc = j0 + C;
      // the largest |a| in column C over rows >= rc (ties to the lower row; a
      // NaN counts as infinite)
      float best = -1.f;
      int bidx = 0x7fffffff;
      if (r < d && r >= rc) {
        best = fabsf(a[C]);
        if (best != best) best = INFINITY;
        bidx = r;
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const float ob = __shfl_xor(best, off);
        const int oi = __shfl_xor(bidx, off);
        if (ob > best || (ob == best && oi < bidx)) {
          best = ob;
          bidx = oi;
        }
      }
      if (lane == 0) {
        sh.best[w] = best;
        sh.bidx[w] = bidx;
      }
      __syncthreads();
      if (tid < 64) {
        float b = tid < kPanelThreads / 64 ? sh.best[tid] : -1.f;
        int bi = tid < kPanelThreads / 64 ? sh.bidx[tid] : 0x7fffffff;
#pragma unroll
        for (int off = 8; off > 0; off >>= 1) {
          const float ob = __shfl_xor(b, off);
          const int oi = __shfl_xor(bi, off);
          if (ob > b || (ob == b && oi < bi)) {
            b = ob;
            bi = oi;
          }
        }
        if (tid == 0) {
          sh.p = bi;
          sh.piv[C] = bi;
        }
      }
      __syncthreads();
      const int p = sh.p;
      if (r == p) {
#pragma unroll
        for (int cc = 0; cc < kLuNB; ++cc) sh.prow[cc] = a[cc];
      }
      if (r == rc && p != rc) {
#pragma unroll
        for (int cc = 0; cc < kLuNB; ++cc) sh.old[cc] = a[cc];
      }
      __syncthreads();
      if (p != rc) {
        if (r == rc) {
#pragma unroll
          for (int cc = 0; cc < kLuNB; ++cc) a[cc] = sh.prow[cc];
        } else if (r == p) {
#pragma unroll
          for (int cc = 0; cc < kLuNB; ++cc) a[cc] = sh.old[cc];
        }
      }
      const float piv = sh.prow[C];
      if (tid == 0 && (!(fabsf(piv) > 0.f) || !isfinite(piv)))
        atomicCAS(flags + F_ERR, 0, LST_ESINGULAR);
      if (r < d && r > rc) {
        const float l = a[C] * (1.f / piv);
        a[C] = l;
#pragma unroll
        for (int cc = C + 1; cc < kLuNB; ++cc) a[cc] -= l * sh.prow[cc];
      }
      __syncthreads();  // the pivot row buffers are rewritten for the next column
    }
    PanelColumn<C + 1>::run(a, sh, d, j0, nc, ipiv, flags);
  }
};
template <>
struct PanelColumn<kLuNB> {
  __device__ __forceinline__ static void run(float (&)[kLuNB], PanelShared&, int, int, int, int*,
                                             int*) {}
};

__global__ __launch_bounds__(kPanelThreads) void lu_panel_kernel(float* A, int d, int j0,
                                                                 int* ipiv, int* flags) {
  __shared__ PanelShared sh;
  const int r = j0 + threadIdx.x;
  const int nc = min(kLuNB, d - j0);
  float a[kLuNB];
#pragma unroll
  for (int c = 0; c < kLuNB; ++c) a[c] = (r < d && c < nc) ? A[(size_t)r * d + j0 + c] : 0.f;
  PanelColumn<0>::run(a, sh, d, j0, nc, ipiv, flags);
  if (threadIdx.x < nc) ipiv[j0 + threadIdx.x] = sh.piv[threadIdx.x];
  if (r < d)
#pragma unroll
    for (int c = 0; c < kLuNB; ++c)
      if (c < nc) A[(size_t)r * d + j0 + c] = a[c];
}

// Columns 64 b .. 64 b + 63 outside the panel: the panel's interchanges in
// order (the rows they touch staged in LDS), then, right of the panel, the
// forward substitution with the unit lower triangle L11.  The block after the
// last column slab applies the same interchanges to perm (the row order of the
// right-hand sides).
__global__ __launch_bounds__(64) void lu_apply_kernel(float* A, int d, int j0, const int* ipiv,
                                                      int* perm) {
  __shared__ int s_rows[2 * kLuNB];
  __shared__ int s_slot[kLuNB];
  __shared__ int s_n;
  __shared__ float S[2 * kLuNB][65];
  __shared__ int Sp[2 * kLuNB];
  __shared__ float Ls[kLuNB][kLuNB + 1];
  const int tid = threadIdx.x;
  const int nc = min(kLuNB, d - j0);
  __shared__ int s_piv[kLuNB];
  const bool perm_block = blockIdx.x == gridDim.x - 1;
  const int col = blockIdx.x * 64 + tid;
  if (tid < nc) s_piv[tid] = ipiv[j0 + tid];
  __syncthreads();
  if (tid == 0) {
    int n = nc;
    for (int k = 0; k < nc; ++k) s_rows[k] = j0 + k;
    for (int k = 0; k < nc; ++k) {
      const int p = s_piv[k];
      int slot = -1;
      if (p < j0 + nc) {
        slot = p - j0;
      } else {
        for (int u = nc; u < n; ++u)
          if (s_rows[u] == p) slot = u;
        if (slot < 0) {
          s_rows[n] = p;
          slot = n++;
        }
      }
      s_slot[k] = slot;
    }
    s_n = n;
  }
  if (!perm_block) {
    for (int e0 = 0; e0 < kLuNB * kLuNB; e0 += 8 * 64) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + tid + 64 * u, i = e / kLuNB, k = e - i * kLuNB;
        v[u] = (i < nc && k < nc) ? A[(size_t)(j0 + i) * d + j0 + k] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + tid + 64 * u, i = e / kLuNB, k = e - i * kLuNB;
        Ls[i][k] = v[u];
      }
    }
  }
  __syncthreads();
  const int n = s_n;
  if (perm_block) {
    if (tid < n) Sp[tid] = perm[s_rows[tid]];
    __syncthreads();
    if (tid == 0)
      for (int k = 0; k < nc; ++k) {
        const int sk = s_slot[k];
        const int t = Sp[k];
        Sp[k] = Sp[sk];
        Sp[sk] = t;
      }
    __syncthreads();
    if (tid < n) perm[s_rows[tid]] = Sp[tid];
    return;
  }
  if (col >= d || (col >= j0 && col < j0 + nc)) return;
  {
    float v[2 * kLuNB];
#pragma unroll
    for (int u = 0; u < 2 * kLuNB; ++u) v[u] = u < n ? A[(size_t)s_rows[u] * d + col] : 0.f;
#pragma unroll
    for (int u = 0; u < 2 * kLuNB; ++u) S[u][tid] = v[u];
  }
  for (int k = 0; k < nc; ++k) {
    const int sk = s_slot[k];
    if (sk != k) {
      const float t = S[k][tid];
      S[k][tid] = S[sk][tid];
      S[sk][tid] = t;
    }
  }
  float x[kLuNB];
#pragma unroll
  for (int i = 0; i < kLuNB; ++i) x[i] = S[i][tid];
  if (col >= j0 + nc) {
#pragma unroll
    for (int i = 1; i < kLuNB; ++i) {
      float v = x[i];
#pragma unroll
      for (int k = 0; k < i; ++k) v -= Ls[i][k] * x[k];
      x[i] = v;
    }
  }
#pragma unroll
  for (int u = 0; u < 2 * kLuNB; ++u)
    if (u < n) A[(size_t)s_rows[u] * d + col] = u < kLuNB ? x[u] : S[u][tid];
}

__global__ __launch_bounds__(256) void lu_iota_kernel(int* perm, int d) {
  for (int j = blockIdx.x * 256 + threadIdx.x; j < d; j += gridDim.x * 256) perm[j] = j;
}

// One column block J0 .. J0 + nb of the row solves for rows r0 .. r0 + 15.
// FWD: y = L^{-1} (P h), the right-hand side gathered from H through perm;
// otherwise z = R^{-1} y, written to X2 and, scaled by -lr a_i, to Xout.
template <bool FWD>
__global__ __launch_bounds__(256) void lu_rows_kernel(const float* F, int d, int J0,
                                                      const int* perm, const float* H, int m,
                                                      float* X2, float* Xout, const float* acoef,
                                                      float lr) {
  __shared__ float Xs[kSolveRows][kSolveNB + 1];
  __shared__ float Fs[kSolveNB][kSolveNB + 1];
  __shared__ float Z[kSolveRows][kSolveNB + 1];
  const int tid = threadIdx.x, r0 = blockIdx.x * kSolveRows;
  const int nb = min(kSolveNB, d - J0);
  const int rr = tid >> 4, q = tid & 15, i4 = q * 4;
  const int row = r0 + rr;
  // the right-hand side first (its loads overlap the product's)
  float rhs[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int i = i4 + c;
    rhs[c] = 0.f;
    if (row < m && i < nb)
      rhs[c] = FWD ? H[(size_t)row * d + perm[J0 + i]] : X2[(size_t)row * d + J0 + i];
  }
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  const int kbeg = FWD ? 0 : J0 + nb, kend = FWD ? J0 : d;
  // operands: thread t loads column t & 63 of rows (t >> 6) + 4 u
  const int lc = tid & 63, lr4 = tid >> 6;
  for (int k0 = kbeg; k0 < kend; k0 += kSolveNB) {
    const int kn = min(kSolveNB, kend - k0);
    float xv[kSolveRows / 4], fv[kSolveNB / 4];
#pragma unroll
    for (int u = 0; u < kSolveRows / 4; ++u) {
      const int ro = lr4 + 4 * u;
      xv[u] = (r0 + ro < m && lc < kn) ? X2[(size_t)(r0 + ro) * d + k0 + lc] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kSolveNB / 4; ++u) {
      const int i = lr4 + 4 * u;
      fv[u] = (i < nb && lc < kn) ? F[(size_t)(J0 + i) * d + k0 + lc] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kSolveRows / 4; ++u) Xs[lr4 + 4 * u][lc] = xv[u];
#pragma unroll
    for (int u = 0; u < kSolveNB / 4; ++u) Fs[lr4 + 4 * u][lc] = fv[u];
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < kSolveNB; ++kk) {
      const float x = Xs[rr][kk];
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] += x * Fs[i4 + c][kk];
    }
    __syncthreads();
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) Z[rr][i4 + c] = rhs[c] - acc[c];
  // the diagonal block of F
  {
    float fv[kSolveNB / 4];
#pragma unroll
    for (int u = 0; u < kSolveNB / 4; ++u) {
      const int i = lr4 + 4 * u;
      fv[u] = (i < nb && lc < nb) ? F[(size_t)(J0 + i) * d + J0 + lc] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kSolveNB / 4; ++u) Fs[lr4 + 4 * u][lc] = fv[u];
  }
  __syncthreads();
  // row rr by its 16 lanes (one quarter of a wave): each entry waits for the
  // entries before it (after it, going back), written by lane q == 0 of the
  // same wave; the LDS accesses of a wave complete in order
  if (FWD) {
    for (int i = 0; i < nb; ++i) {
      float s = 0.f;
      for (int k = q; k < i; k += 16) s += Fs[i][k] * Z[rr][k];
      s += __shfl_xor(s, 8);
      s += __shfl_xor(s, 4);
      s += __shfl_xor(s, 2);
      s += __shfl_xor(s, 1);
      if (q == 0) Z[rr][i] -= s;
      asm volatile("" ::: "memory");
    }
  } else {
    for (int i = nb - 1; i >= 0; --i) {
      float s = 0.f;
      for (int k = i + 1 + q; k < nb; k += 16) s += Fs[i][k] * Z[rr][k];
      s += __shfl_xor(s, 8);
      s += __shfl_xor(s, 4);
      s += __shfl_xor(s, 2);
      s += __shfl_xor(s, 1);
      if (q == 0) Z[rr][i] = (Z[rr][i] - s) / Fs[i][i];
      asm volatile("" ::: "memory");
    }
  }
  __syncthreads();
  if (row < m) {
    const float sc = FWD ? 0.f : -lr * acoef[row];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i = i4 + c;
      if (i < nb) {
        const float z = Z[rr][i];
        X2[(size_t)row * d + J0 + i] = z;
        if (!FWD) Xout[(size_t)row * d + J0 + i] = sc * z;
      }
    }
  }
}

}  // namespace

hipError_t lu_factor(float* A, int d, int* ipiv, int* perm, int* flags, hipStream_t s) {
  if (d < 1 || d > kLuMaxD) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lu_iota_kernel, dim3((d + 255) / 256), dim3(256), 0, s, perm, d);
  // the trailing update runs as the GEMM task of a step launch (32 x 32 tiles)
  StepCtx c{};
  c.m = 1;
  c.d = d;
  for (int j0 = 0; j0 < d; j0 += kLuNB) {
    hipLaunchKernelGGL(lu_panel_kernel, dim3(1), dim3(kPanelThreads), 0, s, A, d, j0, ipiv,
                       flags);
    hipLaunchKernelGGL(lu_apply_kernel, dim3((d + 63) / 64 + 1), dim3(64), 0, s, A, d, j0,
                       (const int*)ipiv, perm);
    const int nc = d - j0 < kLuNB ? d - j0 : kLuNB;
    const int rest = d - j0 - nc;
    if (rest > 0) {
      StepLaunch L{};
      L.lk = 2;
      L.ntask = 1;
      L.kind[0] = TK_GEMM;
      L.gemm.np = 1;
      L.gemm.p[0] = gemm_problem(L_NN, rest, rest, nc,
                                 vmat(A + (size_t)(j0 + nc) * d + j0, d, rest),
                                 vmat(A + (size_t)j0 * d + j0 + nc, d, nc),
                                 A + (size_t)(j0 + nc) * d + j0 + nc, d, -1.f, 1.f, EPI_STORE);
      L.gemm.p[0].tile = 32;
      const hipError_t e = step_launch(c, L, 2, s);
      if (e != hipSuccess) return e;
    }
  }
  return hipGetLastError();
}

hipError_t lu_solve_rows(const float* F, const int* perm, int d, const float* H, int m, float* X2,
                         float* Xout, const float* acoef, float lr, hipStream_t s) {
  if (d < 1 || d > kLuMaxD || m < 1) return hipErrorInvalidValue;
  const dim3 grid((m + kSolveRows - 1) / kSolveRows);
  for (int J0 = 0; J0 < d; J0 += kSolveNB)
    hipLaunchKernelGGL(lu_rows_kernel<true>, grid, dim3(256), 0, s, F, d, J0, perm, H, m, X2,
                       Xout, acoef, lr);
  for (int J0 = (d - 1) / kSolveNB * kSolveNB; J0 >= 0; J0 -= kSolveNB)
    hipLaunchKernelGGL(lu_rows_kernel<false>, grid, dim3(256), 0, s, F, d, J0, perm, H, m, X2,
                       Xout, acoef, lr);
  return hipGetLastError();
}

}  // namespace lst
