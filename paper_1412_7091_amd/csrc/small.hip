// Small dense kernels outside the step: the inverse of an initial U, drift
// control (pristine restore), and the naive baseline's row statistics.
#include <math.h>

#include "lst_internal.h"

namespace lst {


// ---------------------------------------------------------------------------
// In-place Gauss-Jordan inverse with partial (row) pivoting, in fp64.  The row
// interchanges make the in-place result the inverse of the row-permuted
// matrix; swapping columns back in reverse order of the interchanges gives
// S^{-1}.  A pivot that is not finite or at most 1e-13 * max|S| marks S as
// singular (LST_ESINGULAR).  One workgroup; LDS storage when m <= 128.
// ---------------------------------------------------------------------------
template <bool IN_LDS, int MAXM>
__global__ __launch_bounds__(1024) void gauss_jordan_kernel(const float* __restrict__ S, int lds,
                                                            float* __restrict__ Sinv, int ldi,
                                                            int m, double* __restrict__ work,
                                                            int* flags, int check_err) {
  if (check_err && flags[F_ERR]) return;
  __shared__ double sh[IN_LDS ? MAXM * MAXM : 1];
  __shared__ double colk[MAXM];
  __shared__ int piv[MAXM];
  __shared__ int s_p, s_bad;
  __shared__ unsigned s_amax;
  double* A = IN_LDS ? sh : work;
  const int tid = threadIdx.x, nt = blockDim.x;
  if (tid == 0) {
    s_bad = 0;
    s_amax = 0u;
  }
  __syncthreads();
  unsigned amax = 0u;
  for (int e = tid; e < m * m; e += nt) {
    const int i = e / m, j = e - i * m;
    const float v = S[(size_t)i * lds + j];
    A[e] = (double)v;
    const float av = fabsf(v);
    const unsigned bits = isfinite(av) ? __float_as_uint(av) : 0x7f800000u;
    amax = max(amax, bits);  // non-negative floats order like their bit patterns
  }
  atomicMax(&s_amax, amax);
  __syncthreads();
  const double tiny = 1e-13 * (double)__uint_as_float(s_amax);
  for (int k = 0; k < m; ++k) {
    if (tid < 64) {
      double best = -1.0;
      int bi = k;
      for (int i = k + tid; i < m; i += 64) {
        const double v = fabs(A[(size_t)i * m + k]);
        if (v > best || (v != v && best == best)) {  // a NaN wins, so it is reported
          best = v;
          bi = i;
        }
      }
      for (int off = 32; off > 0; off >>= 1) {
        const double ob = __shfl_down(best, off);
        const int oi = __shfl_down(bi, off);
        if (ob > best || (ob == best && oi < bi) || (ob != ob && best == best)) {
          best = ob;
          bi = oi;
        }
      }
      if (tid == 0) {
        s_p = bi;
        piv[k] = bi;
        if (!(best > tiny) || !isfinite(best)) s_bad = 1;
      }
    }
    __syncthreads();
    if (s_bad) break;
    const int p = s_p;
    if (p != k) {
      for (int j = tid; j < m; j += nt) {
        const double t = A[(size_t)k * m + j];
        A[(size_t)k * m + j] = A[(size_t)p * m + j];
        A[(size_t)p * m + j] = t;
      }
    }
    __syncthreads();
    const double pinv = 1.0 / A[(size_t)k * m + k];
    for (int i = tid; i < m; i += nt) colk[i] = A[(size_t)i * m + k];
    __syncthreads();
    for (int j = tid; j < m; j += nt) {
      const double v = (j == k) ? 1.0 : A[(size_t)k * m + j];
      A[(size_t)k * m + j] = v * pinv;
    }
    __syncthreads();
    for (int e = tid; e < m * m; e += nt) {
      const int i = e / m, j = e - i * m;
      if (i == k) continue;
      const double v = (j == k) ? 0.0 : A[e];
      A[e] = v - colk[i] * A[(size_t)k * m + j];
    }
    __syncthreads();
  }
  if (s_bad) {
    if (tid == 0) atomicCAS(flags + F_ERR, 0, LST_ESINGULAR);
    return;
  }
  for (int i = tid; i < m; i += nt) {
    for (int k = m - 1; k >= 0; --k) {
      const int p = piv[k];
      if (p != k) {
        const double t = A[(size_t)i * m + k];
        A[(size_t)i * m + k] = A[(size_t)i * m + p];
        A[(size_t)i * m + p] = t;
      }
    }
  }
  __syncthreads();
  for (int e = tid; e < m * m; e += nt) {
    const int i = e / m, j = e - i * m;
    Sinv[(size_t)i * ldi + j] = (float)A[e];
  }
}

hipError_t invert_small(const float* S, int lds, float* Sinv, int ldi, int m, double* work,
                        int* flags, int check_err, hipStream_t s) {
  if (m <= 128) {
    hipLaunchKernelGGL((gauss_jordan_kernel<true, 128>), dim3(1), dim3(1024), 0, s, S, lds, Sinv,
                       ldi, m, work, flags, check_err);
  } else if (m <= 4096) {
    hipLaunchKernelGGL((gauss_jordan_kernel<false, 4096>), dim3(1), dim3(1024), 0, s, S, lds,
                       Sinv, ldi, m, work, flags, check_err);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Drift control (Appendix C): restore when ||U||_F ||U^{-T}||_F > thr.
// The product lies in [cond_2(U), d cond_2(U)] and equals d at U = I.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void drift_check_kernel(const float* __restrict__ U,
                                                           const float* __restrict__ Uit, int d,
                                                           float thr, int* flags) {
  __shared__ double su[1024], si[1024];
  double a = 0.0, b = 0.0;
  const size_t n = (size_t)d * d;
  for (size_t e = threadIdx.x; e < n; e += blockDim.x) {
    a += (double)U[e] * U[e];
    b += (double)Uit[e] * Uit[e];
  }
  su[threadIdx.x] = a;
  si[threadIdx.x] = b;
  __syncthreads();
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if (threadIdx.x < (unsigned)off) {
      su[threadIdx.x] += su[threadIdx.x + off];
      si[threadIdx.x] += si[threadIdx.x + off];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double kappa = sqrt(su[0]) * sqrt(si[0]);
    const int go = (flags[F_ERR] == 0) && !(kappa <= (double)thr);
    flags[F_RESTORE] = go;
    if (go) flags[F_RESTORES] += 1;
  }
}

hipError_t drift_check(const float* U, const float* Uit, int d, float thr, int* flags,
                       hipStream_t s) {
  hipLaunchKernelGGL(drift_check_kernel, dim3(1), dim3(1024), 0, s, U, Uit, d, thr, flags);
  return hipGetLastError();
}

__global__ void copy_if_kernel(const float* __restrict__ src, float* __restrict__ dst, size_t n,
                               const int* run_if) {
  if (run_if && !*run_if) return;
  for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x)
    dst[e] = src[e];
}

hipError_t copy_if(const float* src, float* dst, size_t n, const int* run_if, hipStream_t s) {
  size_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(copy_if_kernel, dim3((unsigned)blocks), dim3(256), 0, s, src, dst, n, run_if);
  return hipGetLastError();
}

__global__ void set_identity_kernel(float* A, int d, const int* run_if) {
  if (run_if && !*run_if) return;
  const size_t n = (size_t)d * d;
  for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x) {
    const size_t i = e / d, j = e - i * d;
    A[e] = (i == j) ? 1.f : 0.f;
  }
}

hipError_t set_identity_if(float* A, int d, const int* run_if, hipStream_t s) {
  size_t blocks = ((size_t)d * d + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(set_identity_kernel, dim3((unsigned)blocks), dim3(256), 0, s, A, d, run_if);
  return hipGetLastError();
}

__global__ void set_flag_kernel(int* p, int v) { *p = v; }

hipError_t set_flag(int* p, int v, hipStream_t s) {
  hipLaunchKernelGGL(set_flag_kernel, dim3(1), dim3(1), 0, s, p, v);
  return hipGetLastError();
}

__global__ void transpose_kernel(const float* __restrict__ A, float* __restrict__ At, int d) {
  const size_t n = (size_t)d * d;
  for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x) {
    const size_t i = e / d, j = e - i * d;
    At[j * d + i] = A[e];
  }
}

hipError_t transpose_square(const float* A, float* At, int d, hipStream_t s) {
  size_t blocks = ((size_t)d * d + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(transpose_kernel, dim3((unsigned)blocks), dim3(256), 0, s, A, At, d);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Naive baseline (sections 2.3 and 3.1): one workgroup per example turns the
// output row o_i = W h_i (stored in O) into dL/do_i / (2 for squared error):
//   squared:   O_i <- o_i - y_i,  loss_i = ||o_i - y_i||^2
//   spherical: O_i <- (2/S) o_i + b e_c,  loss_i = -log(o_c^2+eps) + log S
//   shifted:   O_i <- (2/S) (o_i + eps) - (2/u_c) e_c, u_c = o_c + eps,
//              S = sum_j (o_j + eps)^2,  loss_i = -log(u_c^2) + log S
// Sums run in fp64 in a fixed tree order.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void naive_rowstats_kernel(float* __restrict__ O, int64_t ldo,
                                                              int64_t D,
                                                              const int32_t* __restrict__ idx,
                                                              const float* __restrict__ val, int K,
                                                              int loss_kind, float eps,
                                                              float* __restrict__ loss,
                                                              int* flags) {
  __shared__ double red[1024];
  __shared__ int s_c;
  const int i = blockIdx.x;
  float* o = O + (size_t)i * ldo;
  if (threadIdx.x == 0) {
    s_c = -1;
    for (int k = 0; k < K; ++k) {
      const int r = idx[(size_t)i * K + k];
      const bool bad = (r < -1) || ((int64_t)r >= D) ||
                       (loss_kind != LST_LOSS_SQUARED && r == -1);
      if (bad) {
        atomicCAS(flags + F_ERR, 0, LST_EINDEX);
        continue;
      }
      if (r < 0) continue;
      if (loss_kind == LST_LOSS_SQUARED) {
        o[r] -= val[(size_t)i * K + k];
      } else if (k == 0) {
        s_c = r;
      }
    }
  }
  __syncthreads();
  const bool shifted = loss_kind == LST_LOSS_SPHERICAL_SHIFTED;
  const double sh = shifted ? (double)eps : 0.0;
  double acc = 0.0;
  for (int64_t r = threadIdx.x; r < D; r += blockDim.x) {
    const double u = (double)o[r] + sh;
    acc += u * u;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if (threadIdx.x < (unsigned)off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  const double sumsq = red[0];
  if (loss_kind == LST_LOSS_SQUARED) {
    if (threadIdx.x == 0) {
      const float L = (float)sumsq;
      loss[i] = L;
      if (!isfinite(L)) atomicCAS(flags + F_ERR, 0, LST_ENONFINITE);
    }
    return;
  }
  const int c = s_c;
  const double S = shifted ? sumsq : sumsq + (double)D * eps;
  const double oc = (c >= 0) ? (double)o[c] + sh : 0.0;
  const double num = shifted ? oc * oc : oc * oc + eps;
  const float a = (float)(2.0 / S);
  const float b = shifted ? (float)(-2.0 / oc) : (float)(-2.0 * oc / num);
  __syncthreads();  // every thread has read o[c] before it is rescaled
  for (int64_t r = threadIdx.x; r < D; r += blockDim.x) o[r] = a * (float)((double)o[r] + sh);
  __syncthreads();
  if (threadIdx.x == 0) {
    if (c >= 0) o[c] += b;
    const float L = (float)(-log(num) + log(S));
    loss[i] = L;
    if (!isfinite(L)) atomicCAS(flags + F_ERR, 0, LST_ENONFINITE);
  }
}

hipError_t naive_rowstats(float* O, int64_t ldo, int64_t D, int m, const int32_t* idx,
                          const float* val, int K, int loss_kind, float eps, float* loss,
                          int* flags, hipStream_t s) {
  hipLaunchKernelGGL(naive_rowstats_kernel, dim3(m), dim3(1024), 0, s, O, ldo, D, idx, val, K,
                     loss_kind, eps, loss, flags);
  return hipGetLastError();
}

}  // namespace lst
