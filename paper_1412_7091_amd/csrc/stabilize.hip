// Appendix C: correction of the singular values of U that leave the safe
// range [sigma_low, sigma_high], without the O(D d^2) pristine restore.
//
// One call, enqueued on the state's stream with no host synchronisation:
//   1. the smallest singular value of U is estimated by power iteration on
//      U^{-T} (its largest singular value is 1 / sigma_min(U), with the same
//      left singular vector u); while it is below sigma_low, fix-singular-value
//      moves it to 1; at most max_fixes rounds;
//   2. the same for the largest singular value of U against sigma_high.
// A round's power iteration applies A A^T 2^s times to the start vector of
// ones, as s squarings of G = A A^T, which is the same vector in exact
// arithmetic.  Each squaring is scaled by the power of two nearest below
// 1 / trace^2 of the matrix it squares (the trace summed in its epilogue), so
// the top eigenvalue neither overflows nor underflows and the scaling itself
// rounds nothing.  The products run on the step's 32 x 32 MFMA tiles, one
// launch each; only the in-place product of the refinement goes through
// split-K partials.
// fix-singular-value with target 1 and alpha = (1 - sigma) / sigma,
// beta = -alpha / (1 + alpha):
//   U <- U + alpha u (U^T u)^T,  U^{-T} <- U^{-T} + beta u (U^{-1} u)^T,
//   V <- V + beta (V u) u^T  (one pass over V; W = V U and Q do not change).
// U^{-T} is recomputed from U by Newton-Schulz steps Z <- 2 Z - (Z U^T) Z
// (quadratic convergence from any Z with ||I - Z U^T|| < 1): after every
// correction, whose rank-one update of U^{-T} cancels a term of size 1/sigma
// and so loses about log10(1/sigma) digits in fp32, and optionally before
// the search as well (the appendix recomputes it before every check).
// Every kernel is gated by a device flag: a round runs only if the previous
// round of its end corrected something (and no step error is pending), and
// its correction and refinement only if its estimate is out of range.
#include <math.h>

#include "lst_internal.h"

namespace lst {

namespace {

// ------------------------------------------------------------------ kernels
__global__ void stab_begin_kernel(const int* flags, int* chain, int* stop, int rounds, float* sig,
                                  int nsig, float* trace, int ntrace) {
  const int ok = flags[F_ERR] == 0;
  for (int i = threadIdx.x; i < 2 * (rounds + 1); i += blockDim.x) {
    const int v = (i % (rounds + 1) == 0) ? ok : 0;
    chain[i] = v;
    stop[i] = !v;
  }
  for (int i = threadIdx.x; i < nsig; i += blockDim.x) sig[i] = __uint_as_float(0x7fc00000u);
  for (int i = threadIdx.x; i < ntrace; i += blockDim.x) trace[i] = 0.f;
}

// C = alpha * (scale ? *scale : 1) * sum_z ws[z] + beta * C (z ascending).
__global__ void stab_reduce_kernel(const float* __restrict__ ws, int splits, size_t n,
                                   float* __restrict__ C, float alpha, float beta,
                                   const float* __restrict__ scale, const int* run_if) {
  if (run_if && !*run_if) return;
  const float a = scale ? alpha * *scale : alpha;
  for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x) {
    float acc = 0.f;
    for (int z = 0; z < splits; ++z) acc += ws[(size_t)z * n + e];
    C[e] = beta != 0.f ? a * acc + beta * C[e] : a * acc;
  }
}

__global__ __launch_bounds__(256) void stab_rowsum_kernel(const float* __restrict__ G, int d,
                                                          float* __restrict__ x,
                                                          const int* run_if) {
  if (run_if && !*run_if) return;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= d) return;
  float acc = 0.f;
  for (int j = lane; j < d; j += 64) acc += G[(size_t)row * d + j];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) x[row] = acc;
}

__global__ __launch_bounds__(256) void stab_normalize_kernel(const float* __restrict__ x, int d,
                                                             float* __restrict__ u,
                                                             const int* run_if) {
  if (run_if && !*run_if) return;
  __shared__ double red[256];
  double t = 0.0;
  for (int i = threadIdx.x; i < d; i += 256) t += (double)x[i] * x[i];
  red[threadIdx.x] = t;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < (unsigned)off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  const double nrm = sqrt(red[0]);
  const float inv = nrm > 0.0 ? (float)(1.0 / nrm) : 0.f;
  for (int i = threadIdx.x; i < d; i += 256) u[i] = x[i] * inv;
}

// Partial column sums of w1 = U^T u and w2 = (U^{-T})^T u = U^{-1} u over the
// row chunk blockIdx.y (kStabRowChunk rows); thread per column (coalesced).
constexpr int kStabRowChunk = 32;

__global__ __launch_bounds__(256) void stab_matvec_t_kernel(const float* __restrict__ U,
                                                            const float* __restrict__ Uit, int d,
                                                            const float* __restrict__ u,
                                                            float* __restrict__ part,
                                                            const int* run_if) {
  if (run_if && !*run_if) return;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= d) return;
  const int r0 = blockIdx.y * kStabRowChunk, r1 = min(d, r0 + kStabRowChunk);
  float a = 0.f, b = 0.f;
  for (int i = r0; i < r1; ++i) {
    const float ui = u[i];
    a += U[(size_t)i * d + j] * ui;
    b += Uit[(size_t)i * d + j] * ui;
  }
  float* p = part + (size_t)blockIdx.y * 2 * d;
  p[j] = a;
  p[d + j] = b;
}

// Sums the partials into w = [U^T u ; U^{-1} u] (chunks in order), forms the
// estimate of the round (high end: ||U^T u||, low end: 1 / ||U^{-1} u||) and
// the decision; on a correction, alpha and beta of fix-singular-value.
__global__ __launch_bounds__(256) void stab_decide_kernel(const float* __restrict__ part,
                                                          int nchunk, int d,
                                                          float* __restrict__ w, int high,
                                                          float sigma_low, float sigma_high,
                                                          const int* run_if, int* go,
                                                          int* go_stop, float* sig, float* scal) {
  if (!*run_if) {
    if (threadIdx.x == 0) {
      *go = 0;
      *go_stop = 1;
    }
    return;
  }
  __shared__ double red[2][256];
  double s1 = 0.0, s2 = 0.0;
  for (int j = threadIdx.x; j < d; j += 256) {
    float a = 0.f, b = 0.f;
    for (int c = 0; c < nchunk; ++c) {
      a += part[(size_t)c * 2 * d + j];
      b += part[(size_t)c * 2 * d + d + j];
    }
    w[j] = a;
    w[d + j] = b;
    s1 += (double)a * a;
    s2 += (double)b * b;
  }
  red[0][threadIdx.x] = s1;
  red[1][threadIdx.x] = s2;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < (unsigned)off) {
      red[0][threadIdx.x] += red[0][threadIdx.x + off];
      red[1][threadIdx.x] += red[1][threadIdx.x + off];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double sigma = high ? sqrt(red[0][0]) : 1.0 / sqrt(red[1][0]);
    const bool out = high ? (sigma > (double)sigma_high) : (sigma < (double)sigma_low);
    const bool ok = out && sigma > 0.0 && isfinite(sigma);
    *sig = (float)sigma;
    *go = ok ? 1 : 0;
    *go_stop = ok ? 0 : 1;
    if (ok) {
      const double alpha = (1.0 - sigma) / sigma;
      scal[0] = (float)alpha;
      scal[1] = (float)(-alpha / (1.0 + alpha));
    }
  }
}

// U += alpha u (U^T u)^T and U^{-T} += beta u (U^{-1} u)^T.
__global__ void stab_rank1_kernel(float* __restrict__ U, float* __restrict__ Uit, int d,
                                  const float* __restrict__ u, const float* __restrict__ w,
                                  const float* __restrict__ scal, const int* go) {
  if (!*go) return;
  const float alpha = scal[0], beta = scal[1];
  const size_t n = (size_t)d * d;
  for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x) {
    const size_t i = e / d, j = e - i * d;
    const float ui = u[i];
    U[e] += alpha * ui * w[j];
    Uit[e] += beta * ui * w[d + j];
  }
}

// V <- V + beta (V u) u^T: one pass over V, a wave per row at a time (every
// row independent).  VEC: d % 4 == 0 (16-byte rows), d <= 1024.
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <bool VEC>
__global__ __launch_bounds__(256) void stab_fix_v_kernel(float* __restrict__ V, int64_t D, int d,
                                                         const float* __restrict__ u,
                                                         const float* __restrict__ scal,
                                                         const int* go) {
  if (!*go) return;
  const float beta = scal[1];
  const int lane = threadIdx.x & 63;
  const int64_t wave0 = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  if (VEC) {
    // lane owns the 16-byte pieces lane, lane + 64, ... of a row; a wave takes
    // two rows at a time, both rows' loads in flight before either reduction.
    constexpr int NQ = 4, NR = 2;
    const int nq = d / 4;
    f32x4 uq[NQ];
#pragma unroll
    for (int t = 0; t < NQ; ++t) {
      const int q = lane + 64 * t;
      uq[t] = q < nq ? reinterpret_cast<const f32x4*>(u)[q] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int64_t r0 = wave0 * NR; r0 < D; r0 += nwaves * NR) {
      f32x4 v[NR][NQ];
#pragma unroll
      for (int k = 0; k < NR; ++k) {
        const f32x4* row = reinterpret_cast<const f32x4*>(V + (r0 + k) * d);
#pragma unroll
        for (int t = 0; t < NQ; ++t) {
          const int q = lane + 64 * t;
          v[k][t] = (q < nq && r0 + k < D) ? __builtin_nontemporal_load(row + q)
                                           : f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
#pragma unroll
      for (int k = 0; k < NR; ++k) {
        float s = 0.f;
#pragma unroll
        for (int t = 0; t < NQ; ++t)
          s += v[k][t].x * uq[t].x + v[k][t].y * uq[t].y + v[k][t].z * uq[t].z +
               v[k][t].w * uq[t].w;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
        const float c = beta * s;
        f32x4* row = reinterpret_cast<f32x4*>(V + (r0 + k) * d);
#pragma unroll
        for (int t = 0; t < NQ; ++t) {
          const int q = lane + 64 * t;
          if (q < nq && r0 + k < D) __builtin_nontemporal_store(v[k][t] + c * uq[t], row + q);
        }
      }
    }
  } else {
    for (int64_t r = wave0; r < D; r += nwaves) {
      float* row = V + r * d;
      float s = 0.f;
      for (int j = lane; j < d; j += 64) s += row[j] * u[j];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
      const float c = beta * s;
      for (int j = lane; j < d; j += 64) row[j] += c * u[j];
    }
  }
}

// --------------------------------------------------------------- host side
// Newton-Schulz steps on U^{-T}: before the search (from a U^{-T} that only
// drifted) and after a correction (from one that lost up to log10(1/sigma)
// digits; with ||I - Z U^T|| <= 0.1 three steps reach fp32 precision).
constexpr int kRefineBefore = 2;
constexpr int kRefineAfter = 3;

unsigned grid_for(size_t n, unsigned cap) {
  size_t b = (n + 255) / 256;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (unsigned)b;
}

// C (d x d) = alpha * p * A B^T (NT) or A B (NN) + beta * C on the 32 x 32 MFMA tiles of
// the step, one launch: p = 2^(-2 ilogb(*scale_in)) (1 without scale_in), and the
// trace of C added into *trace_out when given.  Skipped while *stop is set.  C must
// not alias A or B.
hipError_t tile_product(const StabArgs& a, int layout, const float* A, const float* B, float* C,
                        float alpha, float beta, const float* scale_in, float* trace_out,
                        const int* stop, hipStream_t s) {
  const int d = a.d;
  StepCtx c{};
  c.m = 1;
  StepLaunch L{};
  L.ntask = 1;
  L.kind[0] = TK_GEMM;
  L.lk = 5;
  L.gemm.np = 1;
  L.gemm.skip_if = stop;
  GemmProblem& p = L.gemm.p[0];
  p = gemm_problem(layout, d, d, d, vmat(A, d, d), vmat(B, d, d), C, d, alpha, beta, EPI_SCALED);
  L.gemm.x.s1 = scale_in;
  L.gemm.x.g = trace_out;
  p.tile = 32;
  int stages = (d + 63) / 64;  // every K chunk resident when it fits
  if (stages > 9) stages = 9;
  if (stages < 2) stages = 2;
  return step_launch(c, L, stages, s);
}

// C (d x d) = alpha * (scale) * op(A) op(B) + beta * C through split-K partials
// (safe when C is also an operand).
hipError_t dd_product(const StabArgs& a, int layout, const float* A, const float* B, float* C,
                      float alpha, float beta, const float* scale, const int* run_if,
                      hipStream_t s) {
  const int d = a.d;
  GemmProblem p = gemm_problem(layout, d, d, d, vmat(A, d, d), vmat(B, d, d), a.ws, d, 1.f, 0.f,
                               EPI_PARTIAL);
  p.ksplit = a.ksplit;
  hipError_t e = gemm_big_launch(p, s, nullptr, run_if);
  if (e != hipSuccess) return e;
  const size_t n = (size_t)d * d;
  hipLaunchKernelGGL(stab_reduce_kernel, dim3(grid_for(n, 2048)), dim3(256), 0, s, a.ws, a.ksplit,
                     n, C, alpha, beta, scale, run_if);
  return hipGetLastError();
}

}  // namespace

StabLayout stab_layout(int d, int ksplit, int max_fixes) {
  StabLayout l;
  const size_t dd = (size_t)d * d;
  const size_t nchunk = (size_t)(d + kStabRowChunk - 1) / kStabRowChunk;
  size_t o = 0;
  l.G = o; o += dd;
  l.G2 = o; o += dd;
  l.ws = o; o += (size_t)ksplit * dd;
  l.x = o; o += d;
  l.u = o; o += d;
  l.w = o; o += 2 * (size_t)d;
  l.wpart = o; o += nchunk * 2 * d;
  l.scal = o; o += 8;
  l.sig = o; o += 2 * (size_t)max_fixes;
  l.trace = o; o += 2 * (size_t)max_fixes * (kStabMaxSquarings + 1);
  l.floats = o;
  l.ints = 4 * ((size_t)max_fixes + 1);  // the round flags, then the same negated
  return l;
}

int stab_ksplit(int d) {
  const int tiles = ((d + 127) / 128) * ((d + 127) / 128);
  int ks = (256 + tiles - 1) / tiles;
  const int max_by_k = (d + 63) / 64;
  if (ks > max_by_k) ks = max_by_k;
  return ks < 1 ? 1 : ks;
}

hipError_t stabilize_enqueue(const StabArgs& a, hipStream_t s) {
  const int d = a.d;
  const size_t dd = (size_t)d * d;
  const int R = a.max_fixes;
  const int nchunk = (d + kStabRowChunk - 1) / kStabRowChunk;
  const int per_round = kStabMaxSquarings + 1;
  hipLaunchKernelGGL(stab_begin_kernel, dim3(1), dim3(256), 0, s, a.flags, a.chain, a.stop, R,
                     a.sig, 2 * R, a.trace, 2 * R * per_round);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int* ok = a.chain;  // chain[0]: no pending step error
  auto stop_of = [&](const int* run) { return a.stop + (run - a.chain); };
  // Z <- 2 Z - (Z U^T) Z on Z = U^{-T}, n times, gated by run; T = Z U^T lives in G2.
  auto refine = [&](int n, const int* run) -> hipError_t {
    hipError_t r = hipSuccess;
    for (int it = 0; it < n && r == hipSuccess; ++it) {
      r = tile_product(a, L_NT, a.Uit, a.U, a.G2, 1.f, 0.f, nullptr, nullptr, stop_of(run), s);
      if (r == hipSuccess) r = dd_product(a, L_NN, a.G2, a.Uit, a.Uit, -1.f, 2.f, nullptr, run, s);
    }
    return r;
  };
  if (a.reinvert >= 2 && (e = refine(kRefineBefore, ok))) return e;
  for (int end = 0; end < 2; ++end) {  // 0: smallest singular value (on U^{-T}), 1: largest (on U)
    const float* A = end ? a.U : a.Uit;
    int* chain = a.chain + end * (R + 1);
    for (int r = 0; r < R; ++r) {
      const int* run = chain + r;
      int* go = chain + r + 1;
      float* tr = a.trace + (size_t)(end * R + r) * per_round;
      // G = A A^T, then squarings G <- p G G (G is symmetric, so G G^T), each
      // scaled by a power of two from the trace of the one before
      if ((e = tile_product(a, L_NT, A, A, a.G, 1.f, 0.f, nullptr, tr, stop_of(run), s)))
        return e;
      float* G = a.G;
      float* G2 = a.G2;
      for (int q = 0; q < a.squarings; ++q) {
        if ((e = tile_product(a, L_NT, G, G, G2, 1.f, 0.f, tr + q, tr + q + 1, stop_of(run), s)))
          return e;
        float* t = G;
        G = G2;
        G2 = t;
      }
      hipLaunchKernelGGL(stab_rowsum_kernel, dim3((d + 3) / 4), dim3(256), 0, s, G, d, a.x, run);
      hipLaunchKernelGGL(stab_normalize_kernel, dim3(1), dim3(256), 0, s, a.x, d, a.u, run);
      hipLaunchKernelGGL(stab_matvec_t_kernel, dim3((d + 255) / 256, nchunk), dim3(256), 0, s,
                         a.U, a.Uit, d, a.u, a.wpart, run);
      hipLaunchKernelGGL(stab_decide_kernel, dim3(1), dim3(256), 0, s, a.wpart, nchunk, d, a.w,
                         end, a.sigma_low, a.sigma_high, run, go, a.stop + (go - a.chain),
                         a.sig + end * R + r, a.scal);
      hipLaunchKernelGGL(stab_rank1_kernel, dim3(grid_for(dd, 1024)), dim3(256), 0, s, a.U, a.Uit,
                         d, a.u, a.w, a.scal, go);
      if (d % 4 == 0 && d <= 1024)
        hipLaunchKernelGGL(stab_fix_v_kernel<true>, dim3(2048), dim3(256), 0, s, a.V, a.D, d, a.u,
                           a.scal, go);
      else
        hipLaunchKernelGGL(stab_fix_v_kernel<false>, dim3(2048), dim3(256), 0, s, a.V, a.D, d,
                           a.u, a.scal, go);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      if (a.reinvert >= 1 && (e = refine(kRefineAfter, go))) return e;
    }
  }
  return hipSuccess;
}

}  // namespace lst
