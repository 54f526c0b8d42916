// fp32 MFMA GEMM family for the dense contractions of the step.
//
// The products of the minibatch algorithm (Appendix A steps 1, 2, 5, 7, 8, 10)
// are small (m = 128 .. 512 on one side, d = 500 .. 1024 on the others), so
// their time is dominated by memory latency, not by MFMA throughput.  The
// kernel therefore stages a whole K-chunk of both operands (up to 256 for
// 64 x 64 tiles, 512 for 32 x 32 tiles) into LDS with every global load of
// the chunk in flight at once, then runs the MFMAs out of LDS.  Four waves
// share a tile, each owning a quarter computed with v_mfma_f32_16x16x4f32.
// Operands are "virtual" row-major matrices (stacked row blocks) and each
// problem of a grouped launch carries its own layout and epilogue, so the
// independent products of one phase of the step share a single launch.
#include "lst_internal.h"

namespace lst {

typedef float floatx4 __attribute__((ext_vector_type(4)));

template <int BM, int BN>
struct Panel {
  static constexpr int KC = (32768 / (BM + BN)) / 16 * 16;  // k per LDS chunk
  static constexpr int LD = KC + 4;                          // LDS row stride (floats)
  static constexpr int WM = BM / 2, WN = BN / 2;             // wave tile (2 x 2 waves)
  static constexpr int IM = WM / 16, IN = WN / 16;           // 16 x 16 blocks per wave
  static constexpr int NLA = BM * KC / 4 / 256;              // float4 loads per thread, A
  static constexpr int NLB = BN * KC / 4 / 256;              // float4 loads per thread, B
};

__device__ __forceinline__ float4 vm_load4(const VMat& v, int row, int col, int nrows, int ncols) {
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  if (row >= nrows || col >= ncols) return o;
  int b = 0;
  while (b + 1 < v.nb && row >= v.r0[b + 1]) ++b;
  const float* base = v.p[b] + (size_t)(row - v.r0[b]) * (size_t)v.ld[b];
  if (v.vec && col + 3 < ncols) {
    o = *reinterpret_cast<const float4*>(base + col);
  } else {
    o.x = base[col];
    if (col + 1 < ncols) o.y = base[col + 1];
    if (col + 2 < ncols) o.z = base[col + 2];
    if (col + 3 < ncols) o.w = base[col + 3];
  }
  if (v.rscale) {
    const float s = v.rscale[row];
    o.x *= s; o.y *= s; o.z *= s; o.w *= s;
  }
  return o;
}

// Loads rows [o0, o0+R) of the output dimension and k in [k0, k0+KC) of one
// operand into LDS as S[r * LD + k] (k contiguous).  kc: the operand's rows are
// the output dimension (k contiguous in memory); otherwise its rows are k.
// Elements outside [0, nout) x [k0, kend) are zero.
template <int R, int KC, int LD, int NL>
__device__ __forceinline__ void load_panel(const VMat& v, int kc, int o0, int nout, int k0,
                                           int kend, float* S) {
  float4 r[NL];
  const int t = threadIdx.x;
  if (kc) {
#pragma unroll
    for (int q = 0; q < NL; ++q) {
      const int idx = t + 256 * q;
      const int row = idx / (KC / 4), c4 = idx - row * (KC / 4);
      r[q] = vm_load4(v, o0 + row, k0 + 4 * c4, nout, kend);
    }
#pragma unroll
    for (int q = 0; q < NL; ++q) {
      const int idx = t + 256 * q;
      const int row = idx / (KC / 4), c4 = idx - row * (KC / 4);
      *reinterpret_cast<float4*>(S + row * LD + 4 * c4) = r[q];
    }
  } else {
#pragma unroll
    for (int q = 0; q < NL; ++q) {
      const int idx = t + 256 * q;
      const int kr = idx / (R / 4), c4 = idx - kr * (R / 4);
      r[q] = vm_load4(v, k0 + kr, o0 + 4 * c4, kend, nout);
    }
#pragma unroll
    for (int q = 0; q < NL; ++q) {
      const int idx = t + 256 * q;
      const int kr = idx / (R / 4), c4 = idx - kr * (R / 4);
      S[(4 * c4 + 0) * LD + kr] = r[q].x;
      S[(4 * c4 + 1) * LD + kr] = r[q].y;
      S[(4 * c4 + 2) * LD + kr] = r[q].z;
      S[(4 * c4 + 3) * LD + kr] = r[q].w;
    }
  }
}

template <int BM, int BN>
__global__ __launch_bounds__(256) void gemm_panel_kernel(GemmBatch bt) {
  using C = Panel<BM, BN>;
  if (bt.skip_if && *bt.skip_if) return;
  if (bt.run_if && !*bt.run_if) return;
  extern __shared__ __attribute__((aligned(16))) float smem[];
  float* As = smem;
  float* Bs = smem + BM * C::LD;

  int t = blockIdx.x;
  int q = 0;
  while (q + 1 < bt.np && t >= bt.p[q + 1].tile_begin) ++q;
  if (bt.skip_updates_if && q >= bt.first_update && *bt.skip_updates_if) return;
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
      const int kc = ((P.K + P.ksplit - 1) / P.ksplit + 15) / 16 * 16;
      kb = z * kc;
      ke = min(P.K, kb + kc);
    }
  }
  const int m0 = tm * BM, n0 = tn * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  floatx4 acc[C::IM][C::IN];
#pragma unroll
  for (int i = 0; i < C::IM; ++i)
#pragma unroll
    for (int j = 0; j < C::IN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = kb; k0 < ke; k0 += C::KC) {
    if (k0 != kb) __syncthreads();
    load_panel<BM, C::KC, C::LD, C::NLA>(P.A, P.a_kc, m0, P.M, k0, ke, As);
    load_panel<BN, C::KC, C::LD, C::NLB>(P.B, P.b_kc, n0, P.N, k0, ke, Bs);
    __syncthreads();
    const int kcount = min(C::KC, ke - k0);
    const int kpad = (kcount + 15) & ~15;
    const float* Aw = As + (wm * C::WM + (lane & 15)) * C::LD + 4 * (lane >> 4);
    const float* Bw = Bs + (wn * C::WN + (lane & 15)) * C::LD + 4 * (lane >> 4);
    for (int kk = 0; kk < kpad; kk += 16) {
      float4 fa[C::IM], fb[C::IN];
#pragma unroll
      for (int i = 0; i < C::IM; ++i)
        fa[i] = *reinterpret_cast<const float4*>(Aw + i * 16 * C::LD + kk);
#pragma unroll
      for (int j = 0; j < C::IN; ++j)
        fb[j] = *reinterpret_cast<const float4*>(Bw + j * 16 * C::LD + kk);
      // MFMA number q of a 16-wide k slice pairs k = 4*(lane/16) + q of A with the same k of B.
#pragma unroll
      for (int i = 0; i < C::IM; ++i)
#pragma unroll
        for (int j = 0; j < C::IN; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].x, fb[j].x, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].y, fb[j].y, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].z, fb[j].z, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i].w, fb[j].w, acc[i][j], 0, 0, 0);
        }
    }
  }

  // Element r of acc[i][j]: row 4*(lane/16) + r, column lane % 16 of its 16 x 16 block.
#pragma unroll
  for (int i = 0; i < C::IM; ++i)
#pragma unroll
    for (int j = 0; j < C::IN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * C::WM + i * 16 + 4 * (lane >> 4) + r;
        const int col = n0 + wn * C::WN + j * 16 + (lane & 15);
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

template <int BM, int BN>
static int assign_tiles(GemmBatch& b) {
  int total = 0;
  for (int q = 0; q < b.np; ++q) {
    GemmProblem& p = b.p[q];
    p.tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = (p.N + BN - 1) / BN;
    p.tile_begin = total;
    if (p.ksplit < 1) p.ksplit = 1;
    if (p.epi == EPI_SYM)
      total += p.tiles_m * (p.tiles_m + 1) / 2;  // square C: upper-triangle tiles
    else
      total += p.tiles_m * p.tiles_n * (p.epi == EPI_PARTIAL ? p.ksplit : 1);
  }
  b.total_tiles = total;
  return total;
}

template <int BM, int BN>
static hipError_t launch_tiles(GemmBatch& b, hipStream_t s) {
  using C = Panel<BM, BN>;
  const int total = assign_tiles<BM, BN>(b);
  if (total == 0) return hipSuccess;
  const size_t lds = (size_t)(BM + BN) * C::LD * sizeof(float);
  hipLaunchKernelGGL((gemm_panel_kernel<BM, BN>), dim3(total), dim3(256), lds, s, b);
  return hipGetLastError();
}

static bool lds_configured = false;

static hipError_t configure_lds() {
  if (lds_configured) return hipSuccess;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_panel_kernel<64, 64>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)((64 + 64) * Panel<64, 64>::LD * sizeof(float)));
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_panel_kernel<32, 32>),
                          hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)((32 + 32) * Panel<32, 32>::LD * sizeof(float)));
  if (e != hipSuccess) return e;
  lds_configured = true;
  return hipSuccess;
}

hipError_t gemm_launch(GemmBatch& b, hipStream_t s, int tile) {
  hipError_t e = configure_lds();
  if (e != hipSuccess) return e;
  if (tile == 0) {  // automatic: 64 x 64 unless that leaves most compute units idle
    GemmBatch probe = b;
    tile = assign_tiles<64, 64>(probe) >= 160 ? 64 : 32;
  }
  return tile == 64 ? launch_tiles<64, 64>(b, s) : launch_tiles<32, 32>(b, s);
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
