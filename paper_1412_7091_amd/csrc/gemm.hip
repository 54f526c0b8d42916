// fp32 MFMA GEMM family for the dense contractions of the step.
//
// One kernel template serves every dense product of the minibatch algorithm
// (Appendix A steps 1, 2, 5, 7, 8, 10) and of the naive baseline: a 64 x 64
// output tile per 256-thread workgroup, K staged through LDS 16 at a time,
// each of the four waves owning a 32 x 32 quarter computed with
// v_mfma_f32_16x16x4f32.  Operands are "virtual" row-major matrices (stacked
// row blocks) so that [Q; U; U^{-T}; H] H^T and the rank-2m Q update are
// single products.  Several problems of one layout can share a launch.
#include "lst_internal.h"

namespace lst {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int BM = 64, BN = 64, BK = 16, LDS_STRIDE = BK + 4;

__device__ __forceinline__ void vm_load4(const VMat& v, int row, int col, int nrows, int ncols,
                                         float o[4]) {
  o[0] = o[1] = o[2] = o[3] = 0.f;
  if (row >= nrows) return;
  int b = 0;
  while (b + 1 < v.nb && row >= v.r0[b + 1]) ++b;
  const float* base = v.p[b] + (size_t)(row - v.r0[b]) * (size_t)v.ld[b];
  const float s = v.rscale ? v.rscale[row] : 1.f;
  if (v.vec && col + 3 < ncols) {
    const float4 x = *reinterpret_cast<const float4*>(base + col);
    o[0] = x.x * s; o[1] = x.y * s; o[2] = x.z * s; o[3] = x.w * s;
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (col + j < ncols) o[j] = base[col + j] * s;
  }
}

// Loads the 64 x 16 slice of an operand for output rows/cols [o0, o0+64) and
// k in [k0, k0+16) into registers.  kc: operand rows are the output dimension
// (K contiguous); otherwise operand rows are K.
template <bool KC>
__device__ __forceinline__ void load_tile(const VMat& v, int o0, int k0, int nout, int kend,
                                          float r[4]) {
  const int t = threadIdx.x;
  if (KC) {
    const int row = t >> 2, kq = (t & 3) * 4;
    vm_load4(v, o0 + row, k0 + kq, nout, kend, r);
  } else {
    const int kr = t >> 4, oq = (t & 15) * 4;
    if (k0 + kr < kend) {
      vm_load4(v, k0 + kr, o0 + oq, kend, nout, r);
    } else {
      r[0] = r[1] = r[2] = r[3] = 0.f;
    }
  }
}

template <bool KC>
__device__ __forceinline__ void store_tile(float (*S)[LDS_STRIDE], const float r[4]) {
  const int t = threadIdx.x;
  if (KC) {
    const int row = t >> 2, kq = (t & 3) * 4;
    *reinterpret_cast<float4*>(&S[row][kq]) = make_float4(r[0], r[1], r[2], r[3]);
  } else {
    const int kr = t >> 4, oq = (t & 15) * 4;
#pragma unroll
    for (int j = 0; j < 4; ++j) S[oq + j][kr] = r[j];
  }
}

template <int LAYOUT>
__global__ __launch_bounds__(256) void gemm64_kernel(GemmBatch bt) {
  if (bt.skip_if && *bt.skip_if) return;
  if (bt.run_if && !*bt.run_if) return;
  constexpr bool A_KC = (LAYOUT != L_TN);
  constexpr bool B_KC = (LAYOUT == L_NT);

  int t = blockIdx.x;
  int q = 0;
  while (q + 1 < bt.np && t >= bt.p[q + 1].tile_begin) ++q;
  const GemmProblem& P = bt.p[q];
  int lt = t - P.tile_begin;
  int tm, tn, kb = 0, ke = P.K, z = 0;
  if (P.epi == EPI_SYM) {
    int T = P.tiles_m, r = 0;
    while (lt >= T - r) { lt -= T - r; ++r; }
    tm = r; tn = r + lt;
  } else {
    const int per = P.tiles_m * P.tiles_n;
    z = lt / per;
    lt -= z * per;
    tm = lt / P.tiles_n;
    tn = lt - tm * P.tiles_n;
    if (P.ksplit > 1) {
      const int kc = ((P.K + P.ksplit - 1) / P.ksplit + BK - 1) / BK * BK;
      kb = z * kc;
      ke = min(P.K, kb + kc);
    }
  }
  const int m0 = tm * BM, n0 = tn * BN;

  __shared__ __attribute__((aligned(16))) float As[BM][LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) float Bs[BN][LDS_STRIDE];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  floatx4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  float ra[4], rb[4];
  if (kb < ke) {
    load_tile<A_KC>(P.A, m0, kb, P.M, ke, ra);
    load_tile<B_KC>(P.B, n0, kb, P.N, ke, rb);
  }
  for (int k0 = kb; k0 < ke; k0 += BK) {
    __syncthreads();
    store_tile<A_KC>(As, ra);
    store_tile<B_KC>(Bs, rb);
    __syncthreads();
    if (k0 + BK < ke) {  // prefetch the next slice while this one is multiplied
      load_tile<A_KC>(P.A, m0, k0 + BK, P.M, ke, ra);
      load_tile<B_KC>(P.B, n0, k0 + BK, P.N, ke, rb);
    }
    float4 fa[2], fb[2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
      fa[i] = *reinterpret_cast<const float4*>(&As[wm * 32 + i * 16 + (lane & 15)][4 * (lane >> 4)]);
#pragma unroll
    for (int j = 0; j < 2; ++j)
      fb[j] = *reinterpret_cast<const float4*>(&Bs[wn * 32 + j * 16 + (lane & 15)][4 * (lane >> 4)]);
    // MFMA number q of this slice pairs k = 4*(lane/16) + q of A with the same k of B.
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].x, fb[j].x, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].y, fb[j].y, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].z, fb[j].z, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].w, fb[j].w, acc[i][j], 0, 0, 0);
      }
  }

  // Output element of acc[i][j][r]: row 4*(lane/16) + r, column lane % 16 of the 16 x 16 block.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * 32 + i * 16 + 4 * (lane >> 4) + r;
        const int col = n0 + wn * 32 + j * 16 + (lane & 15);
        if (row >= P.M || col >= P.N) continue;
        const float v = acc[i][j][r];
        if (P.epi == EPI_STORE) {
          float* c = P.C + (size_t)row * P.ldc + col;
          float o = P.alpha * v;
          if (P.beta != 0.f) o += P.beta * *c;
          *c = o;
        } else if (P.epi == EPI_SYM) {
          if (row <= col) {
            const float o = P.C[(size_t)row * P.ldc + col] + P.alpha * v;
            P.C[(size_t)row * P.ldc + col] = o;
            P.C[(size_t)col * P.ldc + row] = o;
          }
        } else if (P.epi == EPI_GRADT) {
          const float g = P.s1[row] * P.e1[(size_t)row * P.lde1 + col] +
                          P.s2[row] * P.e2[(size_t)row * P.lde2 + col];
          P.g[(size_t)row * P.ldg + col] = g;
          P.C[(size_t)row * P.ldc + col] = g + P.alpha * v;
        } else {  // EPI_PARTIAL
          P.C[(size_t)z * P.M * P.N + (size_t)row * P.N + col] = v;
        }
      }
}

__global__ void splitk_reduce_kernel(const float* ws, int splits, int M, int N, float* C, int ldc,
                                     float alpha, float beta, int sym, const int* skip_if) {
  if (skip_if && *skip_if) return;
  const size_t total = (size_t)M * N;
  for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < total;
       e += (size_t)gridDim.x * blockDim.x) {
    const int r = (int)(e / N), c = (int)(e - (size_t)r * N);
    if (sym && r > c) continue;
    float s = 0.f;
    for (int z = 0; z < splits; ++z) s += ws[(size_t)z * total + e];
    float o = alpha * s;
    if (beta != 0.f) o += beta * C[(size_t)r * ldc + c];
    C[(size_t)r * ldc + c] = o;
    if (sym) C[(size_t)c * ldc + r] = o;
  }
}

static int aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

VMat vmat(const float* p, int ld, int rows, const float* rscale) {
  VMat v{};
  v.p[0] = p;
  v.ld[0] = ld;
  v.r0[0] = 0;
  v.r0[1] = rows;
  v.nb = 1;
  v.vec = (ld % 4 == 0) && aligned16(p);
  v.rscale = rscale;
  return v;
}

VMat vmat2(const float* p0, int ld0, int rows0, const float* p1, int ld1, int rows1) {
  VMat v{};
  v.p[0] = p0;
  v.ld[0] = ld0;
  v.p[1] = p1;
  v.ld[1] = ld1;
  v.r0[0] = 0;
  v.r0[1] = rows0;
  v.r0[2] = rows0 + rows1;
  v.nb = 2;
  v.vec = (ld0 % 4 == 0) && (ld1 % 4 == 0) && aligned16(p0) && aligned16(p1);
  v.rscale = nullptr;
  return v;
}

GemmProblem gemm_problem(int M, int N, int K, const VMat& A, const VMat& B, float* C, int ldc,
                         float alpha, float beta, int epi) {
  GemmProblem p{};
  p.M = M; p.N = N; p.K = K;
  p.A = A; p.B = B;
  p.C = C; p.ldc = ldc;
  p.alpha = alpha; p.beta = beta;
  p.epi = epi;
  p.ksplit = 1;
  return p;
}

hipError_t gemm_launch(int layout, GemmBatch& b, hipStream_t s) {
  int total = 0;
  for (int q = 0; q < b.np; ++q) {
    GemmProblem& p = b.p[q];
    p.tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = (p.N + BN - 1) / BN;
    p.tile_begin = total;
    if (p.ksplit < 1) p.ksplit = 1;
    if (p.epi == EPI_SYM) {
      // square C only: upper-triangle tiles
      total += p.tiles_m * (p.tiles_m + 1) / 2;
    } else {
      total += p.tiles_m * p.tiles_n * (p.epi == EPI_PARTIAL ? p.ksplit : 1);
    }
  }
  b.total_tiles = total;
  if (total == 0) return hipSuccess;
  dim3 grid(total), block(256);
  switch (layout) {
    case L_NT: hipLaunchKernelGGL(gemm64_kernel<L_NT>, grid, block, 0, s, b); break;
    case L_NN: hipLaunchKernelGGL(gemm64_kernel<L_NN>, grid, block, 0, s, b); break;
    case L_TN: hipLaunchKernelGGL(gemm64_kernel<L_TN>, grid, block, 0, s, b); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t gemm_splitk_reduce(const float* ws, int splits, int M, int N, float* C, int ldc,
                              float alpha, float beta, int sym, const int* skip_if,
                              hipStream_t s) {
  const size_t total = (size_t)M * N;
  int blocks = (int)((total + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, s, ws, splits, M, N, C,
                     ldc, alpha, beta, sym, skip_if);
  return hipGetLastError();
}

}  // namespace lst
