// One output tile of the fp32 MFMA panel GEMM, as a device function shared by
// the step kernel.
//
// The products of the minibatch algorithm (Appendix A steps 1, 2, 5, 7, 8, 10)
// are small (m = 128 .. 512 on one side, d = 500 .. 1024 on the others), so
// their time goes to memory latency, not to MFMA throughput.  A tile therefore
// stages a whole K-chunk of both operands in LDS with every global load of the
// chunk in flight at once (and the operands of its epilogue prefetched along
// with them), then runs the MFMAs out of LDS.  Four waves share a tile, each
// owning a quarter computed with v_mfma_f32_16x16x4f32.  Operands are
// "virtual" row-major matrices (stacked row blocks); the A operand of the
// product N H^T is instead generated on the fly from the m x m pieces of N.
#pragma once

#include "lst_internal.h"

namespace lst {

typedef float floatx4 __attribute__((ext_vector_type(4)));

template <int BM, int BN>
struct Panel {
  static constexpr int WM = BM / 2, WN = BN / 2;   // wave tile (2 x 2 waves)
  static constexpr int IM = WM / 16, IN = WN / 16; // 16 x 16 blocks per wave
};

// LDS floats a tile with chunk width kcw needs.
__host__ __device__ constexpr int panel_lds_floats(int bm, int bn, int kcw) {
  return (bm + bn) * (kcw + 4);
}

__host__ __device__ __forceinline__ int chunk_width(int kmax, int K) {
  const int k16 = (K + 15) & ~15;
  return k16 < kmax ? k16 : kmax;
}

// Row block of a virtual matrix chosen with constant indices only, so the
// descriptor stays in scalar registers and a lane only selects between them.
__device__ __forceinline__ const float* vm_row(const VMat& v, int row) {
  const float* base = v.p[0];
  int ld = v.ld[0], r0 = 0;
  if (v.nb > 1 && row >= v.r0[1]) { base = v.p[1]; ld = v.ld[1]; r0 = v.r0[1]; }
  if (v.nb > 2 && row >= v.r0[2]) { base = v.p[2]; ld = v.ld[2]; r0 = v.r0[2]; }
  if (v.nb > 3 && row >= v.r0[3]) { base = v.p[3]; ld = v.ld[3]; r0 = v.r0[3]; }
  return base + (size_t)(row - r0) * (size_t)ld;
}

__device__ __forceinline__ float4 vm_load4(const VMat& v, int row, int col, int nrows, int ncols) {
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  if (row >= nrows || col >= ncols) return o;
  const float* base = vm_row(v, row);
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

// N_ij = a_i a_j C1_ij + a_i b_j C2_ij + b_i a_j C2t_ij + b_i b_j (Y^T Y)_ij for
// j = col .. col+3 (zero outside [0, m)).
__device__ __forceinline__ float4 nmat_load4(const GemmProblem& P, int i, int col) {
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  const int m = P.nm;
  if (i >= m || col >= m) return o;
  const float ai = P.na[i], bi = P.nb[i];
  float v[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int j = col + u;
    if (j < m) {
      const float c1 = P.nC12[(size_t)i * P.nld + j];
      const float c2 = P.nC12[(size_t)i * P.nld + m + j];
      const float c2t = P.nC2t[(size_t)i * m + j];
      const float y = P.nyy[(size_t)i * m + j];
      const float aj = P.na[j], bj = P.nb[j];
      v[u] = ai * aj * c1 + ai * bj * c2 + bi * aj * c2t + bi * bj * y;
    }
  }
  o.x = v[0]; o.y = v[1]; o.z = v[2]; o.w = v[3];
  return o;
}

// Loads rows [o0, o0+R) of the output dimension and k in [k0, k0+kcw) of one
// operand into LDS as S[r * ld + k] (k contiguous).  kc: the operand's rows are
// the output dimension (k contiguous in memory); otherwise its rows are k.
// Elements outside [0, nout) x [k0, kend) are zero.  kcw is a multiple of 16.
// NLMAX bounds the float4 loads per thread (R * kcw / 1024).
template <int R, int NLMAX, bool NMAT>
__device__ __forceinline__ void load_panel(const GemmProblem& P, const VMat& v, int kc, int o0,
                                           int nout, int k0, int kend, int kcw, int ld, float* S) {
  float4 r[NLMAX];
  const int t = threadIdx.x;
  const int total = R * kcw / 4;
  if (NMAT || kc) {
    const int per_row = kcw / 4;
#pragma unroll
    for (int q = 0; q < NLMAX; ++q) {
      const int idx = t + 256 * q;
      const int row = idx / per_row, c4 = idx - row * per_row;
      if (idx < total) {
        if (NMAT)
          r[q] = (o0 + row < nout && k0 + 4 * c4 < kend) ? nmat_load4(P, o0 + row, k0 + 4 * c4)
                                                          : make_float4(0.f, 0.f, 0.f, 0.f);
        else
          r[q] = vm_load4(v, o0 + row, k0 + 4 * c4, nout, kend);
      }
    }
#pragma unroll
    for (int q = 0; q < NLMAX; ++q) {
      const int idx = t + 256 * q;
      if (idx < total) {
        const int row = idx / per_row, c4 = idx - row * per_row;
        *reinterpret_cast<float4*>(S + row * ld + 4 * c4) = r[q];
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < NLMAX; ++q) {
      const int idx = t + 256 * q;
      const int kr = idx / (R / 4), c4 = idx - kr * (R / 4);
      if (idx < total) r[q] = vm_load4(v, k0 + kr, o0 + 4 * c4, kend, nout);
    }
#pragma unroll
    for (int q = 0; q < NLMAX; ++q) {
      const int idx = t + 256 * q;
      if (idx < total) {
        const int kr = idx / (R / 4), c4 = idx - kr * (R / 4);
        S[(4 * c4 + 0) * ld + kr] = r[q].x;
        S[(4 * c4 + 1) * ld + kr] = r[q].y;
        S[(4 * c4 + 2) * ld + kr] = r[q].z;
        S[(4 * c4 + 3) * ld + kr] = r[q].w;
      }
    }
  }
}

// Largest chunk width a BM-row panel may use: 16 float4 loads per thread.
__host__ __device__ constexpr int panel_kcw_max(int bm) { return 16384 / bm; }

// Computes tile number t of the batch (problems laid out one after another)
// with chunk width bt.kcw_max (<= panel_kcw_max); smem holds
// panel_lds_floats(BM, BN, bt.kcw_max).
template <int BM, int BN>
__device__ __forceinline__ void panel_tile(const GemmBatch& bt, int t, float* smem) {
  using C = Panel<BM, BN>;
  static_assert(BM == BN, "square tiles");
  constexpr int NLA = 16, NLB = 16;
  int q = 0;
  while (q + 1 < bt.np && t >= bt.p[q + 1].tile_begin) ++q;
  const GemmProblem& P = bt.p[q];
  if (bt.skip_updates_if && q >= bt.first_update && *bt.skip_updates_if) return;
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
  const int kcw = chunk_width(bt.kcw_max, ke - kb);
  const int ld = kcw + 4;
  float* As = smem;
  float* Bs = smem + BM * ld;
  const int m0 = tm * BM, n0 = tn * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Operands of the epilogue, fetched together with the first chunk.
  float pre1[C::IM][C::IN][4], pre2[C::IM][C::IN][4];
#pragma unroll
  for (int i = 0; i < C::IM; ++i)
#pragma unroll
    for (int j = 0; j < C::IN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * C::WM + i * 16 + 4 * (lane >> 4) + r;
        const int col = n0 + wn * C::WN + j * 16 + (lane & 15);
        pre1[i][j][r] = 0.f;
        pre2[i][j][r] = 0.f;
        if (row >= P.M || col >= P.N) continue;
        if ((P.epi == EPI_STORE && P.beta != 0.f) || (P.epi == EPI_SYM && row <= col)) {
          pre1[i][j][r] = P.C[(size_t)row * P.ldc + col];
        } else if (P.epi == EPI_GRADT) {
          pre1[i][j][r] = P.s1[row] * P.e1[(size_t)row * P.lde1 + col];
          pre2[i][j][r] = P.s2[row] * P.e2[(size_t)row * P.lde2 + col];
        }
      }

  floatx4 acc[C::IM][C::IN];
#pragma unroll
  for (int i = 0; i < C::IM; ++i)
#pragma unroll
    for (int j = 0; j < C::IN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = kb; k0 < ke; k0 += kcw) {
    if (k0 != kb) __syncthreads();
    if (P.a_nmat)
      load_panel<BM, NLA, true>(P, P.A, 1, m0, P.M, k0, ke, kcw, ld, As);
    else
      load_panel<BM, NLA, false>(P, P.A, P.a_kc, m0, P.M, k0, ke, kcw, ld, As);
    load_panel<BN, NLB, false>(P, P.B, P.b_kc, n0, P.N, k0, ke, kcw, ld, Bs);
    __syncthreads();
    const int kcount = min(kcw, ke - k0);
    const int kpad = (kcount + 15) & ~15;
    const float* Aw = As + (wm * C::WM + (lane & 15)) * ld + 4 * (lane >> 4);
    const float* Bw = Bs + (wn * C::WN + (lane & 15)) * ld + 4 * (lane >> 4);
    for (int kk = 0; kk < kpad; kk += 16) {
      float4 fa[C::IM], fb[C::IN];
#pragma unroll
      for (int i = 0; i < C::IM; ++i)
        fa[i] = *reinterpret_cast<const float4*>(Aw + i * 16 * ld + kk);
#pragma unroll
      for (int j = 0; j < C::IN; ++j)
        fb[j] = *reinterpret_cast<const float4*>(Bw + j * 16 * ld + kk);
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
          P.C[(size_t)row * P.ldc + col] = P.alpha * v + P.beta * pre1[i][j][r];
        } else if (P.epi == EPI_SYM) {
          if (row <= col) {
            const float o = pre1[i][j][r] + P.alpha * v;
            P.C[(size_t)row * P.ldc + col] = o;
            P.C[(size_t)col * P.ldc + row] = o;
          }
        } else if (P.epi == EPI_GRADT) {
          const float g = pre1[i][j][r] + pre2[i][j][r];
          P.g[(size_t)row * P.ldg + col] = g;
          P.C[(size_t)row * P.ldc + col] = g + P.alpha * v;
        } else {  // EPI_PARTIAL
          P.C[(size_t)z * P.M * P.N + (size_t)row * P.N + col] = v;
        }
      }
}

}  // namespace lst
