// fp32 MFMA GEMM for the large products outside the step: the naive
// explicit-W baseline, W = V U, the initial W^T W.  (The step's own small
// products run as panel tiles inside the step kernel; see gemm_tile.h.)
#include "gemm_tile.h"

namespace lst {

// ---------------------------------------------------------------------------
// Large products (the naive explicit-W baseline, V U, the initial W^T W): a
// classic streaming kernel.  128 x 128 output tiles, K in slices of 32 that
// are double-buffered in LDS (the next slice is loaded while the current one
// is multiplied), 2 x 2 waves each owning 64 x 64.  74 KB of LDS lets two
// workgroups share a compute unit.
// ---------------------------------------------------------------------------
constexpr int GB_T = 128, GB_BK = 32, GB_LD = GB_BK + 4;

template <int KC_FLAG>
__device__ __forceinline__ void big_load(const VMat& v, int o0, int nout, int k0, int kend,
                                         float4 r[4]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = t + 256 * q;
    if (KC_FLAG) {
      const int row = idx >> 3, c4 = idx & 7;  // 8 float4 per 32-wide k row
      r[q] = vm_load4(v, o0 + row, k0 + 4 * c4, nout, kend);
    } else {
      const int kr = idx >> 5, c4 = idx & 31;  // 32 float4 per 128-wide output row
      r[q] = vm_load4(v, k0 + kr, o0 + 4 * c4, kend, nout);
    }
  }
}

template <int KC_FLAG>
__device__ __forceinline__ void big_store(float* S, const float4 r[4]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = t + 256 * q;
    if (KC_FLAG) {
      const int row = idx >> 3, c4 = idx & 7;
      *reinterpret_cast<float4*>(S + row * GB_LD + 4 * c4) = r[q];
    } else {
      const int kr = idx >> 5, c4 = idx & 31;
      S[(4 * c4 + 0) * GB_LD + kr] = r[q].x;
      S[(4 * c4 + 1) * GB_LD + kr] = r[q].y;
      S[(4 * c4 + 2) * GB_LD + kr] = r[q].z;
      S[(4 * c4 + 3) * GB_LD + kr] = r[q].w;
    }
  }
}

template <int A_KC, int B_KC>
__global__ __launch_bounds__(256) void gemm_big_kernel(GemmProblem P, const int* skip_if,
                                                       const int* run_if) {
  if (skip_if && *skip_if) return;
  if (run_if && !*run_if) return;
  __shared__ __attribute__((aligned(16))) float As[2][GB_T * GB_LD];
  __shared__ __attribute__((aligned(16))) float Bs[2][GB_T * GB_LD];
  int lt = blockIdx.x;
  const int per = P.tiles_m * P.tiles_n;
  const int z = lt / per;
  lt -= z * per;
  const int tm = lt / P.tiles_n, tn = lt - tm * P.tiles_n;
  int kb = 0, ke = P.K;
  if (P.ksplit > 1) {
    const int kc = ((P.K + P.ksplit - 1) / P.ksplit + GB_BK - 1) / GB_BK * GB_BK;
    kb = z * kc;
    ke = min(P.K, kb + kc);
  }
  const int m0 = tm * GB_T, n0 = tn * GB_T;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  float4 ra[4], rb[4];
  if (kb < ke) {
    big_load<A_KC>(P.A, m0, P.M, kb, ke, ra);
    big_load<B_KC>(P.B, n0, P.N, kb, ke, rb);
    big_store<A_KC>(As[0], ra);
    big_store<B_KC>(Bs[0], rb);
  }
  __syncthreads();
  int buf = 0;
  for (int k0 = kb; k0 < ke; k0 += GB_BK) {
    const bool more = k0 + GB_BK < ke;
    if (more) {
      big_load<A_KC>(P.A, m0, P.M, k0 + GB_BK, ke, ra);
      big_load<B_KC>(P.B, n0, P.N, k0 + GB_BK, ke, rb);
    }
    const float* Aw = As[buf] + (wm * 64 + (lane & 15)) * GB_LD + 4 * (lane >> 4);
    const float* Bw = Bs[buf] + (wn * 64 + (lane & 15)) * GB_LD + 4 * (lane >> 4);
#pragma unroll
    for (int kk = 0; kk < GB_BK; kk += 16) {
      float4 fa[4], fb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) fa[i] = *reinterpret_cast<const float4*>(Aw + i * 16 * GB_LD + kk);
#pragma unroll
      for (int j = 0; j < 4; ++j) fb[j] = *reinterpret_cast<const float4*>(Bw + j * 16 * GB_LD + kk);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].x, fb[j].x, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].y, fb[j].y, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].z, fb[j].z, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].w, fb[j].w, acc[i][j], 0, 0, 0);
        }
    }
    if (more) {
      big_store<A_KC>(As[buf ^ 1], ra);
      big_store<B_KC>(Bs[buf ^ 1], rb);
    }
    __syncthreads();
    buf ^= 1;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * 64 + i * 16 + 4 * (lane >> 4) + r;
        const int col = n0 + wn * 64 + j * 16 + (lane & 15);
        if (row >= P.M || col >= P.N) continue;
        const float v = acc[i][j][r];
        if (P.epi == EPI_PARTIAL) {
          P.C[(size_t)z * P.M * P.N + (size_t)row * P.N + col] = v;
        } else {
          float* c = P.C + (size_t)row * P.ldc + col;
          float o = P.alpha * v;
          if (P.beta != 0.f) o += P.beta * *c;
          *c = o;
        }
      }
}

hipError_t gemm_big_launch(GemmProblem p, hipStream_t s, const int* skip_if, const int* run_if) {
  if (p.epi != EPI_STORE && p.epi != EPI_PARTIAL) return hipErrorInvalidValue;
  if (p.ksplit < 1) p.ksplit = 1;
  p.tiles_m = (p.M + GB_T - 1) / GB_T;
  p.tiles_n = (p.N + GB_T - 1) / GB_T;
  p.tile_begin = 0;
  const int total = p.tiles_m * p.tiles_n * (p.epi == EPI_PARTIAL ? p.ksplit : 1);
  if (total == 0) return hipSuccess;
  const dim3 grid(total), block(256);
  if (p.a_kc && p.b_kc)
    hipLaunchKernelGGL((gemm_big_kernel<1, 1>), grid, block, 0, s, p, skip_if, run_if);
  else if (p.a_kc)
    hipLaunchKernelGGL((gemm_big_kernel<1, 0>), grid, block, 0, s, p, skip_if, run_if);
  else if (p.b_kc)
    hipLaunchKernelGGL((gemm_big_kernel<0, 1>), grid, block, 0, s, p, skip_if, run_if);
  else
    hipLaunchKernelGGL((gemm_big_kernel<0, 0>), grid, block, 0, s, p, skip_if, run_if);
  return hipGetLastError();
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
  v.r1 = rows;
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
  v.r1 = rows0;  // block 1 holds rows [rows0, rows0 + rows1)
  (void)rows1;
  v.nb = 2;
  v.vec = (ld0 % 4 == 0) && (ld1 % 4 == 0) && aligned16(p0) && aligned16(p1);
  v.rscale = nullptr;
  return v;
}

GemmProblem gemm_problem(int layout, int M, int N, int K, const VMat& A, const VMat& B, float* C,
                         int ldc, float alpha, float beta, int epi) {
  GemmProblem p{};
  p.M = M; p.N = N; p.K = K;
  p.a_kc = (layout != L_TN);
  p.b_kc = (layout == L_NT);
  p.A = A; p.B = B;
  p.C = C; p.ldc = ldc;
  p.alpha = alpha; p.beta = beta;
  p.epi = epi;
  p.ksplit = 1;
  return p;
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
