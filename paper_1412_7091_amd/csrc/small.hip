// Small dense pieces of the step: per-example loss terms, the m x m matrices
// of the Woodbury update, their inverse, drift control and the naive
// baseline's row statistics.
#include <math.h>

#include "lst_internal.h"

namespace lst {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Per-example scalars and the symmetric m x m matrix N of the step.
//
// With A = diag(a_i) and G the part of dL/dO that is sparse on the targets,
// dL/dO = W H A + G.  Squared error (sections 3.1-3.2): a_i = 2, G = -2 Y.
// Spherical softmax (section 3.6): a_i = 2 / S_i, G = Y diag(b_i),
// S_i = h_i^T Q h_i + D eps, b_i = -2 o_c / (o_c^2 + eps), o_c = h_i^T W^T y_i.
// Inputs C1 = H^T Q H and C2 = H^T (W^T Y) (row i, column j: h_i . (.)_j) and
// Y^T Y.  Outputs:
//   loss_i  = M_ii = C1_ii - 2 C2_ii + (Y^T Y)_ii          (Appendix A, steps 5-6)
//           or -log(o_c^2 + eps) + log S_i                 (spherical)
//   N       = (dL/dO)^T (dL/dO)
//           = A C1 A + A C2 diag(b) + diag(b) C2^T A + diag(b) Y^T Y diag(b)
//             (squared error: N = 4 M, M of Appendix A step 5)
// One thread per entry of N; N_ij and N_ji are evaluated by the same
// expression, so N is exactly symmetric.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void example_terms(int loss_kind, float eps, int64_t D,
                                              const float* C12, int ldc12, const float* yy, int m,
                                              int i, float& a, float& b, float& L) {
  const float c1 = C12[(size_t)i * ldc12 + i];
  const float c2 = C12[(size_t)i * ldc12 + m + i];
  if (loss_kind == LST_LOSS_SQUARED) {
    L = c1 - 2.f * c2 + yy[(size_t)i * m + i];
    a = 2.f;
    b = -2.f;
  } else {
    const float Si = c1 + (float)D * eps;
    const float num = c2 * c2 + eps;
    L = -logf(num) + logf(Si);
    a = 2.f / Si;
    b = -2.f * c2 / num;
  }
}

__global__ __launch_bounds__(256) void minibatch_scalars_kernel(
    int loss_kind, float eps, int64_t D, int m, const float* __restrict__ C12, int ldc12,
    const float* __restrict__ yy, float* __restrict__ loss, float* __restrict__ a_out,
    float* __restrict__ b_out, float* __restrict__ cs_out, float* __restrict__ N, int* flags) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= m * m) return;
  const int i = e / m, j = e - i * m;
  const int p = min(i, j), q = max(i, j);
  float ap, bp, Lp, aq, bq, Lq;
  example_terms(loss_kind, eps, D, C12, ldc12, yy, m, p, ap, bp, Lp);
  example_terms(loss_kind, eps, D, C12, ldc12, yy, m, q, aq, bq, Lq);
  const float* C1 = C12;
  const float* C2 = C12 + m;
  const float c1s = 0.5f * (C1[(size_t)p * ldc12 + q] + C1[(size_t)q * ldc12 + p]);
  const float cross = ap * bq * C2[(size_t)p * ldc12 + q] + bp * aq * C2[(size_t)q * ldc12 + p];
  N[(size_t)i * m + j] = ap * aq * c1s + cross + bp * bq * yy[(size_t)p * m + q];
  if (i == j) {
    loss[i] = Lp;
    if (!isfinite(Lp)) atomicCAS(flags + F_ERR, 0, LST_ENONFINITE);
    a_out[i] = ap;
    b_out[i] = bp;
    cs_out[i] = (loss_kind == LST_LOSS_SQUARED) ? 0.f : bp / ap;
  }
}

hipError_t minibatch_scalars(int loss_kind, float eps, int64_t D, int m, const float* C12,
                             int ldc12, const float* yy, float* loss, float* a, float* b,
                             float* cs, float* N, int* flags, hipStream_t s) {
  const int blocks = (m * m + 255) / 256;
  hipLaunchKernelGGL(minibatch_scalars_kernel, dim3(blocks), dim3(256), 0, s, loss_kind, eps, D,
                     m, C12, ldc12, yy, loss, a, b, cs, N, flags);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// The Woodbury system of step 8 of Appendix A.  With c_i = 1 / (lr a_i)
// (squared error: 1 / (2 lr)), S = H^T H - diag(c) and P = U^{-T} H, the
// updated inverse applied to H is U_new^{-T} H = -(1/lr) P S^{-1} A^{-1}, and
// everything the update needs is X = S^{-1} P^T (m x d).
//
// Each workgroup solves S X_blk = P^T_blk for 16 columns.  Writing
// S = -diag(c) (I - E) with E = diag(1/c) H^T H, X = (I - E)^{-1} B with
// B = -diag(1/c) P^T.  When r = ||E||_inf < 1/2 the Neumann series
// Y_{k+1} = B + E Y_k converges geometrically; it is stopped after the first
// k with r^(k+1) / (1 - r) <= 2^-24, so the truncation error is below fp32
// rounding of the result.  Otherwise (a learning rate so large that
// 2 lr ||H^T H|| is not small) the workgroup runs Gauss-Jordan elimination
// with partial pivoting on the augmented system [S | P^T_blk] (fp64 in LDS
// for m <= 128, fp32 in a global workspace above), flagging LST_ESINGULAR on
// a pivot that is not finite or not above 1e-13 max|S|.  Every workgroup
// evaluates r identically, so they all take the same branch.
// ---------------------------------------------------------------------------
constexpr int kSolveCols = 16;

__device__ __forceinline__ float example_a(int loss_kind, float eps, int64_t D, const float* C12,
                                           int ldc12, int m, int i) {
  if (loss_kind == LST_LOSS_SQUARED) return 2.f;
  const float c1 = C12[(size_t)i * ldc12 + i];
  return 2.f / (c1 + (float)D * eps);
}

template <typename T>
__device__ void gj_augmented(T* A, int lda, int m, int ncol, double* colk, double tiny, int* s_p,
                             int* s_bad) {
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int k = 0; k < m; ++k) {
    if (tid < 64) {
      double best = -1.0;
      int bi = k;
      for (int i = k + tid; i < m; i += 64) {
        const double v = fabs((double)A[(size_t)i * lda + k]);
        if (v > best || (v != v && best == best)) {
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
        *s_p = bi;
        if (!(best > tiny) || !isfinite(best)) *s_bad = 1;
      }
    }
    __syncthreads();
    if (*s_bad) return;
    const int p = *s_p;
    if (p != k) {
      for (int j = tid; j < ncol; j += nt) {
        const T t = A[(size_t)k * lda + j];
        A[(size_t)k * lda + j] = A[(size_t)p * lda + j];
        A[(size_t)p * lda + j] = t;
      }
    }
    __syncthreads();
    const double pinv = 1.0 / (double)A[(size_t)k * lda + k];
    for (int i = tid; i < m; i += nt) colk[i] = (double)A[(size_t)i * lda + k];
    __syncthreads();
    for (int j = tid; j < ncol; j += nt) A[(size_t)k * lda + j] = (T)((double)A[(size_t)k * lda + j] * pinv);
    __syncthreads();
    for (int e = tid; e < m * ncol; e += nt) {
      const int i = e / ncol, j = e - i * ncol;
      if (i == k) continue;
      A[(size_t)i * lda + j] = (T)((double)A[(size_t)i * lda + j] - colk[i] * (double)A[(size_t)k * lda + j]);
    }
    __syncthreads();
  }
}

template <bool SMALL, int MAXM>
__global__ __launch_bounds__(256) void woodbury_solve_kernel(
    const float* __restrict__ HH, int ldh, const float* __restrict__ P, int ldp, int m, int d,
    int loss_kind, float eps, int64_t D, float lr, const float* __restrict__ C12, int ldc12,
    float* __restrict__ X, int ldx, float* __restrict__ gj_ws, int* flags) {
  if (flags[F_ERR]) return;
  extern __shared__ __attribute__((aligned(16))) unsigned char sraw[];
  __shared__ float red[256];
  __shared__ double colk[MAXM];
  __shared__ int s_p, s_bad;
  __shared__ float s_r, s_amax;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int mp = (m + 15) & ~15;
  const int LDE = mp + 4;
  const int c0 = blockIdx.x * kSolveCols;
  float* cinv = reinterpret_cast<float*>(sraw);  // mp
  float* Bt = cinv + mp;                         // kSolveCols x LDE: B^T
  float* Y0 = Bt + kSolveCols * LDE;             // kSolveCols x LDE: Y^T
  float* Y1 = Y0 + kSolveCols * LDE;
  float* Es = Y1 + kSolveCols * LDE;             // mp x LDE (SMALL only)

  for (int i = tid; i < mp; i += 256) {
    if (i < m) {
      const float a = example_a(loss_kind, eps, D, C12, ldc12, m, i);
      cinv[i] = lr * a;  // 1 / c_i
    } else {
      cinv[i] = 0.f;
    }
  }
  if (tid == 0) s_bad = 0;
  __syncthreads();
  // E = diag(1/c) H^T H and r = ||E||_inf ; also max |S| for the pivot threshold
  float rowmax = 0.f, amax = 0.f;
  if (SMALL) {
    for (int e = tid; e < mp * mp; e += 256) {
      const int i = e / mp, j = e - i * mp;
      const float h = (i < m && j < m) ? HH[(size_t)i * ldh + j] : 0.f;
      Es[i * LDE + j] = h * cinv[i];
    }
    __syncthreads();
    for (int i = tid; i < m; i += 256) {
      float sabs = 0.f, hmax = 0.f;
      const float ci = 1.f / cinv[i];
      for (int j = 0; j < m; ++j) {
        const float e = Es[i * LDE + j];
        sabs += fabsf(e);
        const float sv = fabsf(e * ci - (i == j ? ci : 0.f));
        hmax = fmaxf(hmax, sv);
      }
      rowmax = fmaxf(rowmax, sabs);
      amax = fmaxf(amax, hmax);
    }
  } else {
    for (int i = tid; i < m; i += 256) {
      float sabs = 0.f, hmax = 0.f;
      const float ci = 1.f / cinv[i];
      for (int j = 0; j < m; ++j) {
        const float h = HH[(size_t)i * ldh + j];
        sabs += fabsf(h);
        hmax = fmaxf(hmax, fabsf(h - (i == j ? ci : 0.f)));
      }
      rowmax = fmaxf(rowmax, sabs * cinv[i]);
      amax = fmaxf(amax, hmax);
    }
  }
  if (!(rowmax == rowmax)) rowmax = INFINITY;
  red[tid] = rowmax;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) red[tid] = fmaxf(red[tid], red[tid + off]);
    __syncthreads();
  }
  if (tid == 0) s_r = red[0];
  __syncthreads();
  red[tid] = amax;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) red[tid] = fmaxf(red[tid], red[tid + off]);
    __syncthreads();
  }
  if (tid == 0) s_amax = red[0];
  __syncthreads();
  const float r = s_r;

  if (r < 0.5f) {
    // B^T = -(P^T_blk)^T diag(1/c), Y_0 = B
    for (int e = tid; e < kSolveCols * mp; e += 256) {
      const int c = e / mp, i = e - c * mp;
      const float v = (i < m && c0 + c < d) ? -P[(size_t)i * ldp + c0 + c] * cinv[i] : 0.f;
      Bt[c * LDE + i] = v;
      Y0[c * LDE + i] = v;
    }
    int iters = 0;
    if (r > 0.f) {
      const float need = logf(5.9604645e-8f * (1.f - r)) / logf(r);  // r^(k+1) / (1-r) <= 2^-24
      iters = (int)ceilf(need) - 1;
      if (iters < 0) iters = 0;
      if (iters > 64) iters = 64;
    }
    __syncthreads();
    float* Yo = Y0;
    float* Yn = Y1;
    for (int it = 0; it < iters; ++it) {
      for (int rb = wave; rb < mp / 16; rb += 4) {
        floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
        const int arow = rb * 16 + (lane & 15);
        for (int kk = 0; kk < mp; kk += 16) {
          const int k = kk + 4 * (lane >> 4);
          float4 fa;
          if (SMALL) {
            fa = *reinterpret_cast<const float4*>(Es + arow * LDE + k);
          } else {
            fa = make_float4(0.f, 0.f, 0.f, 0.f);
            if (arow < m) {
              const float* hr = HH + (size_t)arow * ldh;
              if (k < m) fa.x = hr[k];
              if (k + 1 < m) fa.y = hr[k + 1];
              if (k + 2 < m) fa.z = hr[k + 2];
              if (k + 3 < m) fa.w = hr[k + 3];
            }
          }
          const float4 fb = *reinterpret_cast<const float4*>(Yo + (lane & 15) * LDE + k);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.x, fb.x, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.y, fb.y, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.z, fb.z, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.w, fb.w, acc, 0, 0, 0);
        }
        const int col = lane & 15;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = rb * 16 + 4 * (lane >> 4) + q;
          const float ey = SMALL ? acc[q] : acc[q] * cinv[row];
          Yn[col * LDE + row] = Bt[col * LDE + row] + ey;
        }
      }
      __syncthreads();
      float* t = Yo;
      Yo = Yn;
      Yn = t;
    }
    for (int e = tid; e < kSolveCols * m; e += 256) {
      const int i = e / kSolveCols, c = e - i * kSolveCols;
      if (c0 + c < d) X[(size_t)i * ldx + c0 + c] = Yo[c * LDE + i];
    }
    return;
  }

  // Fallback: Gauss-Jordan on [S | P^T_blk], S = H^T H - diag(c).
  const int ncol = m + kSolveCols;
  const double tiny = 1e-13 * (double)s_amax;
  if (SMALL) {
    __syncthreads();
    double* A = reinterpret_cast<double*>(sraw);  // aliases the Neumann buffers
    for (int e = tid; e < m * ncol; e += 256) {
      const int i = e / ncol, j = e - i * ncol;
      double v;
      if (j < m) {
        v = (double)HH[(size_t)i * ldh + j];
        if (i == j) v -= 1.0 / (double)(lr * example_a(loss_kind, eps, D, C12, ldc12, m, i));
      } else {
        v = (c0 + j - m < d) ? (double)P[(size_t)i * ldp + c0 + j - m] : 0.0;
      }
      A[(size_t)i * ncol + j] = v;
    }
    __syncthreads();
    gj_augmented<double>(A, ncol, m, ncol, colk, tiny, &s_p, &s_bad);
    if (s_bad) {
      if (tid == 0) atomicCAS(flags + F_ERR, 0, LST_ESINGULAR);
      return;
    }
    for (int e = tid; e < m * kSolveCols; e += 256) {
      const int i = e / kSolveCols, c = e - i * kSolveCols;
      if (c0 + c < d) X[(size_t)i * ldx + c0 + c] = (float)A[(size_t)i * ncol + m + c];
    }
  } else {
    float* A = gj_ws + (size_t)blockIdx.x * m * ncol;
    for (int e = tid; e < m * ncol; e += 256) {
      const int i = e / ncol, j = e - i * ncol;
      float v;
      if (j < m) {
        v = HH[(size_t)i * ldh + j];
        if (i == j) v -= 1.f / (lr * example_a(loss_kind, eps, D, C12, ldc12, m, i));
      } else {
        v = (c0 + j - m < d) ? P[(size_t)i * ldp + c0 + j - m] : 0.f;
      }
      A[(size_t)i * ncol + j] = v;
    }
    __syncthreads();
    gj_augmented<float>(A, ncol, m, ncol, colk, tiny, &s_p, &s_bad);
    if (s_bad) {
      if (tid == 0) atomicCAS(flags + F_ERR, 0, LST_ESINGULAR);
      return;
    }
    for (int e = tid; e < m * kSolveCols; e += 256) {
      const int i = e / kSolveCols, c = e - i * kSolveCols;
      if (c0 + c < d) X[(size_t)i * ldx + c0 + c] = A[(size_t)i * ncol + m + c];
    }
  }
}

size_t woodbury_workspace_floats(int m_max, int d) {
  if (m_max <= 128) return 0;
  const size_t blocks = (size_t)(d + kSolveCols - 1) / kSolveCols;
  return blocks * (size_t)m_max * (m_max + kSolveCols);
}

static bool solve_lds_configured = false;

hipError_t woodbury_solve(const float* HH, int ldh, const float* P, int ldp, int m, int d,
                          int loss_kind, float eps, int64_t D, float lr, const float* C12,
                          int ldc12, float* X, int ldx, float* gj_ws, int* flags, hipStream_t s) {
  constexpr size_t kSmallLds = 128 * (128 + kSolveCols) * sizeof(double);  // fallback matrix
  if (!solve_lds_configured) {
    hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(woodbury_solve_kernel<true, 128>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)kSmallLds);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(woodbury_solve_kernel<false, 512>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, 112 * 1024);
    if (e != hipSuccess) return e;
    solve_lds_configured = true;
  }
  const dim3 grid((d + kSolveCols - 1) / kSolveCols), block(256);
  const int mp = (m + 15) & ~15;
  if (m <= 128) {
    hipLaunchKernelGGL((woodbury_solve_kernel<true, 128>), grid, block, kSmallLds, s, HH, ldh, P,
                       ldp, m, d, loss_kind, eps, D, lr, C12, ldc12, X, ldx, gj_ws, flags);
  } else if (m <= 512) {
    const size_t lds = (size_t)(mp + 3 * kSolveCols * (mp + 4)) * sizeof(float);
    hipLaunchKernelGGL((woodbury_solve_kernel<false, 512>), grid, block, lds, s, HH, ldh, P, ldp,
                       m, d, loss_kind, eps, D, lr, C12, ldc12, X, ldx, gj_ws, flags);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

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
                       (loss_kind == LST_LOSS_SPHERICAL && r == -1);
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
  double acc = 0.0;
  for (int64_t r = threadIdx.x; r < D; r += blockDim.x) acc += (double)o[r] * o[r];
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
  const double S = sumsq + (double)D * eps;
  const double oc = (c >= 0) ? (double)o[c] : 0.0;
  const double num = oc * oc + eps;
  const float a = (float)(2.0 / S);
  const float b = (float)(-2.0 * oc / num);
  __syncthreads();  // every thread has read o[c] before it is rescaled
  for (int64_t r = threadIdx.x; r < D; r += blockDim.x) o[r] *= a;
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
