// The single-example step (m = 1): Algorithm 1 of the paper, extended to the
// loss family of section 3.6, in two launches.
//
// With one example the products of the minibatch step shrink to matrix-vector
// products and the Woodbury update of U^{-T} to Sherman-Morrison
// (eq. updateU-T), so the step is bound by reading Q, U and U^{-T} twice (for
// the products, then for the rank-one updates) and by the round trip between
// the two passes.  With dL/do = a W h + G (squared error: a = 2, G = -2 y;
// spherical softmax: a = 2 / S, G = b e_c, b = -2 o_c / (o_c^2 + eps)):
//   h^ = Q h, y^ = W^T y = U^T (V^T y), c1 = h^T h^, c2 = h^T y^, y^T y;
//   grad = a h^ + b y^ (squared: b = -2);  N = a^2 c1 + 2 a b c2 + b^2 y^T y;
// the shifted spherical softmax (W = V U + 1 c^T, s = W^T 1, u = o + eps 1)
// adds eps s to h^ and c to y^ (so c2 = u_c - eps), with S = c1 + 2 eps s^T h
// + D eps^2, a = 2 / S, b = -2 / u_c, N = a^2 S + 2 a b u_c + b^2, and moves
// c -= lr a (c^T h + eps) h, s -= lr (a (s^T h + D eps) + b) h;
//   T = grad - (lr / 2) N h;  den = 1 - lr a ||h||^2;
//   Q <- Q - lr (h T^T + T h^T);  U <- U - lr a (U h) h^T;
//   U^{-T} <- U^{-T} + (lr a / den) (U^{-T} h) h^T          (eq. updateU-T);
//   V[r] <- V[r] - (lr / den) G_r (U^{-T} h)^T for every target row r, since
//   U_new^{-T} h = (U^{-T} h) / den                         (eq. updateV).
//
//   launch A  64 x 64 tiles of Q, U, U^{-T}: the tile's partial sums of Q h,
//             U h, U^{-T} h over its columns and of U^T g over its rows, with
//             g = V^T y gathered from the target rows of V.  Block 0 checks
//             the targets and merges repeated rows.
//   launch B  blocks of R rows: every block adds the partials of h^ and y^ in
//             tile order (so all blocks hold the same vectors and scalars),
//             forms T, then updates its rows of Q, U, U^{-T} and the same
//             columns of the target rows of V.
// For d > 1024 (more than 16 tiles a side) a third launch between them adds
// the partials once, and launch B reads the finished vectors.  The partials
// cross blocks only at launch boundaries: a hand-off inside launch A would
// need device-scope fences, each of which writes back the L2 of its XCD.
// Summation orders are fixed, so the step is deterministic.  Q stays bitwise
// symmetric: entries (i, j) and (j, i) get the same correction (sym_pair).
#include <hip/hip_runtime.h>
#include <math.h>

#include "lst_internal.h"

namespace lst {

namespace {

constexpr int kOnTile = 64;

enum { PV_Q = 0, PV_U = 1, PV_P = 2, PV_Y = 3 };

// partial sums of vector v from tile t (launch A)
__device__ __forceinline__ float* on_part(const OnlineArgs& a, int v, int t) {
  return a.part + ((size_t)v * a.nt + t) * a.d;
}

// Sum over the 64 lanes of a wave in a fixed order (xor butterfly).
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// p[0] + p[stride] + ... + p[(n - 1) stride] in that order, n <= MAXN, with
// every load issued before the first add.
template <int MAXN>
__device__ __forceinline__ float sum_parts(const float* p, size_t stride, int n) {
  float v[MAXN];
#pragma unroll
  for (int u = 0; u < MAXN; ++u) v[u] = u < n ? p[(size_t)u * stride] : 0.f;
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < MAXN; ++u)
    if (u < n) s += v[u];
  return s;
}

// The shifted loss's [c | s] (after U^{-T}) and launch A's copy of them (after
// the slot sums), which launch B reads while its blocks move c and s.
__device__ __forceinline__ float* shift_state(const OnlineArgs& a) {
  return a.Uit + (size_t)a.d * a.d;
}
__device__ __forceinline__ float* shift_copy(const OnlineArgs& a) { return a.rsum + kOnlineMaxK; }

// Block 0 of launch A: index checks (LST_EINDEX), and for each slot k whose
// row no earlier slot holds: own[k] = its row, rsum[k] = the values of all the
// row's slots added in slot order; other slots own[k] = -1, rsum[k] = 0.
// Also y^T y, the number of valid pairs and of distinct rows.
__device__ void online_targets(const OnlineArgs& a, int* skey, float* sval, float* red) {
  const int tid = threadIdx.x, K = a.K;
  const bool one_hot = a.loss_kind != LST_LOSS_SQUARED;
  int r = -1;
  bool valid = false;
  if (tid < K) {
    r = a.idx[tid];
    valid = r >= 0 && (int64_t)r < a.D;
    const bool bad = (r < -1) || ((int64_t)r >= a.D) || (one_hot && r == -1);
    if (bad) atomicCAS(a.flags + F_ERR, 0, LST_EINDEX);
    skey[tid] = valid ? r : -1;
    sval[tid] = valid ? (one_hot ? 1.f : a.val[tid]) : 0.f;
  }
  __syncthreads();
  bool owner = valid;
  float sum = 0.f;
  if (valid) {
    for (int k = 0; k < tid && owner; ++k) owner = skey[k] != r;
    if (owner)
      for (int k = tid; k < K; ++k)
        if (skey[k] == r) sum += sval[k];
  }
  if (tid < K) {
    a.own[tid] = owner ? r : -1;
    a.rsum[tid] = owner ? sum : 0.f;
  }
  const float yy = wave_sum(sum * sum);
  const float nnz = wave_sum(valid ? 1.f : 0.f);
  const float nuq = wave_sum(owner ? 1.f : 0.f);
  const int w = tid >> 6;
  if ((tid & 63) == 0) {
    red[w] = yy;
    red[4 + w] = nnz;
    red[8 + w] = nuq;
  }
  __syncthreads();
  if (tid == 0) {
    a.scal[0] = ((red[0] + red[1]) + red[2]) + red[3];
    a.flags[F_NNZ] = (int)(((red[4] + red[5]) + red[6]) + red[7]);
    a.flags[F_UNIQUE] = (int)(((red[8] + red[9]) + red[10]) + red[11]);
  }
}

template <bool VEC>
__global__ __launch_bounds__(256) void online_a_kernel(OnlineArgs a) {
  __shared__ float sU[kOnTile][kOnTile + 1];
  __shared__ float sh[kOnTile], sg[4][kOnTile], scol[4][kOnTile];
  __shared__ int skey[kOnlineMaxK];
  __shared__ float sval[kOnlineMaxK];
  const int tid = threadIdx.x, d = a.d, K = a.K, nt = a.nt;
  if (blockIdx.x == 0) {
    online_targets(a, skey, sval, &scol[0][0]);
    if (a.loss_kind == LST_LOSS_SPHERICAL_SHIFTED) {
      const float* sv = shift_state(a);
      float* cp = shift_copy(a);
      for (int j = tid; j < 2 * d; j += 256) cp[j] = sv[j];
    }
    return;
  }
  const int t = blockIdx.x - 1;
  const int bi = t / nt, bj = t - bi * nt;
  const int r0 = bi * kOnTile, c0 = bj * kOnTile;

  // targets first (their rows of V are the longest chain of loads), then the
  // tile: thread (row i, quarter q) holds 16 consecutive columns of each matrix
  int tr = -1;
  float tv = 0.f;
  if (tid < K) {
    tr = a.idx[tid];
    if (a.loss_kind == LST_LOSS_SQUARED) tv = a.val[tid];
  }
  const int i = tid >> 2, q = tid & 3;
  const int row = r0 + i, col0 = c0 + 16 * q;
  float vq[16], vu[16], vp[16];
  if (VEC && row < d && col0 + 16 <= d) {
    const float4* Qr = reinterpret_cast<const float4*>(a.Q + (size_t)row * d + col0);
    const float4* Ur = reinterpret_cast<const float4*>(a.U + (size_t)row * d + col0);
    const float4* Pr = reinterpret_cast<const float4*>(a.Uit + (size_t)row * d + col0);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float4 x = Qr[c], y = Ur[c], z = Pr[c];
      vq[4 * c] = x.x; vq[4 * c + 1] = x.y; vq[4 * c + 2] = x.z; vq[4 * c + 3] = x.w;
      vu[4 * c] = y.x; vu[4 * c + 1] = y.y; vu[4 * c + 2] = y.z; vu[4 * c + 3] = y.w;
      vp[4 * c] = z.x; vp[4 * c + 1] = z.y; vp[4 * c + 2] = z.z; vp[4 * c + 3] = z.w;
    }
  } else {
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const bool in = row < d && col0 + c < d;
      const size_t o = in ? (size_t)row * d + col0 + c : 0;
      vq[c] = in ? a.Q[o] : 0.f;
      vu[c] = in ? a.U[o] : 0.f;
      vp[c] = in ? a.Uit[o] : 0.f;
    }
  }
  // every tile gathers g over its rows; only block 0 reports bad indices
  if (tid < K) {
    const bool valid = tr >= 0 && (int64_t)tr < a.D;
    skey[tid] = valid ? tr : -1;
    sval[tid] = valid ? (a.loss_kind != LST_LOSS_SQUARED ? 1.f : tv) : 0.f;
  }
  if (tid < kOnTile) sh[tid] = (c0 + tid < d) ? a.h[c0 + tid] : 0.f;
  __syncthreads();
  {  // g over the tile's rows: thread (row j, slot group kq) adds slots kq, kq + 4, ...
    const int j = tid & 63, kq = tid >> 6;
    const int grow = r0 + j;
    float g = 0.f;
    if (grow < d)
      for (int k = kq; k < K; k += 4) {
        const int r = skey[k];
        if (r >= 0) g += sval[k] * a.V[(size_t)r * d + grow];
      }
    sg[kq][j] = g;
  }
  // row partials of Q h, U h, U^{-T} h
  float sq = 0.f, su = 0.f, sp = 0.f;
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const float hv = sh[16 * q + c];
    sq += vq[c] * hv;
    su += vu[c] * hv;
    sp += vp[c] * hv;
    sU[i][16 * q + c] = vu[c];
  }
  sq += __shfl_xor(sq, 1);
  su += __shfl_xor(su, 1);
  sp += __shfl_xor(sp, 1);
  sq += __shfl_xor(sq, 2);
  su += __shfl_xor(su, 2);
  sp += __shfl_xor(sp, 2);
  if (q == 0 && row < d) {
    on_part(a, PV_Q, bj)[row] = sq;
    on_part(a, PV_U, bj)[row] = su;
    on_part(a, PV_P, bj)[row] = sp;
  }
  __syncthreads();
  {  // column partials of U^T g: thread (column j, row quarter qq)
    const int j = tid & 63, qq = tid >> 6;
    float s = 0.f;
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int ir = 16 * qq + rr;
      const float g = ((sg[0][ir] + sg[1][ir]) + sg[2][ir]) + sg[3][ir];
      s += sU[ir][j] * g;
    }
    scol[qq][j] = s;
  }
  __syncthreads();
  if (tid < kOnTile && c0 + tid < d)
    on_part(a, PV_Y, bi)[c0 + tid] = ((scol[0][tid] + scol[1][tid]) + scol[2][tid]) + scol[3][tid];
}

// a b + c d with both products rounded before the sum (no fused multiply-add),
// so that sym_pair(a, b, c, d) and sym_pair(d, c, b, a) are the same bits.
__device__ __forceinline__ float sym_pair(float a, float b, float c, float d) {
#pragma clang fp contract(off)
  return a * b + c * d;
}

// Launch between A and B when d > 1024: block s adds the partials of entries
// 64 s .. 64 s + 63 of the four vectors, and the partial dot products of that
// slab (h^T h^, h^T h, h^T y^).
__global__ __launch_bounds__(256) void online_r_kernel(OnlineArgs a) {
  const int tid = threadIdx.x, d = a.d, nt = a.nt, w = tid >> 6, lane = tid & 63;
  const int r = blockIdx.x * kOnTile + lane;
  const float s = r < d ? sum_parts<kOnlineMaxTiles>(on_part(a, w, 0) + r, d, nt) : 0.f;
  if (r < d) a.vec[(size_t)w * d + r] = s;
  const float hr = r < d ? a.h[r] : 0.f;
  if (w == PV_Q) {
    const float c1 = wave_sum(hr * s);
    const float hh = wave_sum(hr * hr);
    if (lane == 0) {
      a.sp[blockIdx.x] = c1;
      a.sp[nt + blockIdx.x] = hh;
    }
  } else if (w == PV_Y) {
    const float c2 = wave_sum(hr * s);
    if (lane == 0) a.sp[2 * nt + blockIdx.x] = c2;
  }
}

// FUSED: launch B adds the tile partials itself (d <= 1024); otherwise it reads
// the vectors and slab dot products of online_r_kernel.
template <bool VEC, bool FUSED>
__global__ __launch_bounds__(256) void online_b_kernel(OnlineArgs a) {
  extern __shared__ float sm[];
  float* sT = sm;           // h^, then T in place
  float* sY = sm + a.d;     // y^
  float* sH = sm + 2 * a.d;
  __shared__ float red[5][4];
  __shared__ float su[kOnlineMaxRows], spv[kOnlineMaxRows];
  const int tid = threadIdx.x, d = a.d, nt = a.nt, R = a.rows_per_block;
  const int i0 = blockIdx.x * R;
  const int rows = min(R, d - i0);
  float* __restrict__ Q = a.Q;
  float* __restrict__ U = a.U;
  float* __restrict__ P = a.Uit;

  // Loads are issued early so that their latencies overlap: the status flag,
  // the owning slots (whose rows of V are requested as soon as they arrive),
  // the block's first rows of Q, U, U^{-T}, then the prologue's partials.
  const int err0 = a.flags[F_ERR];
  constexpr int kVPre = 2;
  const int nve = a.K * rows;
  int vrow[kVPre];
  float vrs[kVPre], vval[kVPre];
#pragma unroll
  for (int c = 0; c < kVPre; ++c) {
    const int e = tid + 256 * c;
    vrow[c] = -1;
    vrs[c] = 0.f;
    if (e < nve) {
      vrow[c] = a.own[e / rows];
      vrs[c] = a.rsum[e / rows];
    }
  }
  auto load_v = [&]() {
#pragma unroll
    for (int c = 0; c < kVPre; ++c) {
      const int e = tid + 256 * c;
      if (e < nve && vrow[c] >= 0) vval[c] = a.V[(size_t)vrow[c] * d + i0 + e % rows];
    }
  };
  constexpr int kPre = 4;
  const int d4 = d >> 2, ne4 = VEC ? rows * d4 : 0;
  float4 pq[kPre], pu[kPre], pp[kPre];
  if (VEC) {
#pragma unroll
    for (int c = 0; c < kPre; ++c) {
      const int e = tid + 256 * c;
      if (e < ne4) {
        const int ii = e / d4;
        const size_t o = (size_t)(i0 + ii) * d + 4 * (e - ii * d4);
        pq[c] = *reinterpret_cast<const float4*>(Q + o);
        pu[c] = *reinterpret_cast<const float4*>(U + o);
        pp[c] = *reinterpret_cast<const float4*>(P + o);
      }
    }
  }

  // h^, y^ and the dot products: every block the same, in the same order
  // (shifted loss: h^ + eps s and y^ + c, and tt = c^T h, nn = s^T h)
  const bool shifted = a.loss_kind == LST_LOSS_SPHERICAL_SHIFTED;
  const float* cs = shift_copy(a);
  float c1 = 0.f, hh = 0.f, c2 = 0.f, tt = 0.f, nn = 0.f;
  if (FUSED) {
    // thread t: entries 4t .. 4t + 3 (d <= 1024); all of its partials are
    // requested before the first is added
    const int j0 = 4 * tid;
    const bool act = j0 < d;
    float x[4] = {0.f, 0.f, 0.f, 0.f}, y[4] = {0.f, 0.f, 0.f, 0.f};
    if (VEC) {
      float4 px[kOnlineFuseTiles], py[kOnlineFuseTiles];
      if (act) {
#pragma unroll
        for (int u = 0; u < kOnlineFuseTiles; ++u)
          if (u < nt) {
            px[u] = *reinterpret_cast<const float4*>(on_part(a, PV_Q, u) + j0);
            py[u] = *reinterpret_cast<const float4*>(on_part(a, PV_Y, u) + j0);
          }
      }
      load_v();
      if (act) {
#pragma unroll
        for (int u = 0; u < kOnlineFuseTiles; ++u)
          if (u < nt) {
            x[0] += px[u].x; x[1] += px[u].y; x[2] += px[u].z; x[3] += px[u].w;
            y[0] += py[u].x; y[1] += py[u].y; y[2] += py[u].z; y[3] += py[u].w;
          }
      }
    } else {
      float px[kOnlineFuseTiles][4], py[kOnlineFuseTiles][4];
      if (act) {
#pragma unroll
        for (int u = 0; u < kOnlineFuseTiles; ++u)
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const bool in = u < nt && j0 + c < d;
            px[u][c] = in ? on_part(a, PV_Q, u)[j0 + c] : 0.f;
            py[u][c] = in ? on_part(a, PV_Y, u)[j0 + c] : 0.f;
          }
      }
      load_v();
      if (act) {
#pragma unroll
        for (int u = 0; u < kOnlineFuseTiles; ++u)
          if (u < nt)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              x[c] += px[u][c];
              y[c] += py[u][c];
            }
      }
    }
    if (act) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int j = j0 + c;
        if (j < d) {
          const float hv = a.h[j];
          float hx = x[c], yv = y[c];
          if (shifted) {
            const float cj = cs[j], sj = cs[d + j];
            hx += a.eps * sj;
            yv += cj;
            tt += hv * cj;
            nn += hv * sj;
          }
          sT[j] = hx;
          sY[j] = yv;
          sH[j] = hv;
          c1 += hv * x[c];
          c2 += hv * yv;
          hh += hv * hv;
        }
      }
    }
    c1 = wave_sum(c1);
    c2 = wave_sum(c2);
    hh = wave_sum(hh);
    if (shifted) {
      tt = wave_sum(tt);
      nn = wave_sum(nn);
    }
    if ((tid & 63) == 0) {
      red[0][tid >> 6] = c1;
      red[1][tid >> 6] = c2;
      red[2][tid >> 6] = hh;
      red[3][tid >> 6] = tt;
      red[4][tid >> 6] = nn;
    }
    if (tid < rows) {
      su[tid] = sum_parts<kOnlineFuseTiles>(on_part(a, PV_U, 0) + i0 + tid, d, nt);
    } else if (tid >= 64 && tid < 64 + rows) {
      spv[tid - 64] = sum_parts<kOnlineFuseTiles>(on_part(a, PV_P, 0) + i0 + tid - 64, d, nt);
    }
    __syncthreads();
    c1 = ((red[0][0] + red[0][1]) + red[0][2]) + red[0][3];
    c2 = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
    hh = ((red[2][0] + red[2][1]) + red[2][2]) + red[2][3];
    tt = ((red[3][0] + red[3][1]) + red[3][2]) + red[3][3];
    nn = ((red[4][0] + red[4][1]) + red[4][2]) + red[4][3];
  } else {
    load_v();
    for (int u = 0; u < nt; ++u) {
      c1 += a.sp[u];
      hh += a.sp[nt + u];
      c2 += a.sp[2 * nt + u];
    }
#pragma unroll 4
    for (int j = tid; j < d; j += 256) {
      const float hv = a.h[j];
      float hx = a.vec[(size_t)PV_Q * d + j], yv = a.vec[(size_t)PV_Y * d + j];
      if (shifted) {
        const float cj = cs[j], sj = cs[d + j];
        hx += a.eps * sj;
        yv += cj;
        tt += hv * cj;
        nn += hv * sj;
      }
      sT[j] = hx;
      sY[j] = yv;
      sH[j] = hv;
    }
    if (tid < rows) su[tid] = a.vec[(size_t)PV_U * d + i0 + tid];
    else if (tid >= 64 && tid < 64 + rows) spv[tid - 64] = a.vec[(size_t)PV_P * d + i0 + tid - 64];
    if (shifted) {
      tt = wave_sum(tt);
      nn = wave_sum(nn);
      if ((tid & 63) == 0) {
        red[3][tid >> 6] = tt;
        red[4][tid >> 6] = nn;
      }
    }
    __syncthreads();
    if (shifted) {
      tt = ((red[3][0] + red[3][1]) + red[3][2]) + red[3][3];
      nn = ((red[4][0] + red[4][1]) + red[4][2]) + red[4][3];
      c2 += tt;  // h^T (y^ + c)
    }
  }

  const float yy = a.scal[0];
  float L, av, bv, N;
  if (a.loss_kind == LST_LOSS_SQUARED) {
    L = c1 - 2.f * c2 + yy;
    av = 2.f;
    bv = -2.f;
    N = av * av * c1 + 2.f * av * bv * c2 + bv * bv * yy;
  } else if (!shifted) {
    const float S = c1 + (float)a.D * a.eps;
    const float num = c2 * c2 + a.eps;
    L = -logf(num) + logf(S);
    av = 2.f / S;
    bv = -2.f * c2 / num;
    N = av * av * c1 + 2.f * av * bv * c2 + bv * bv * yy;
  } else {
    const float S = c1 + 2.f * a.eps * nn + (float)a.D * a.eps * a.eps;
    const float uc = c2 + a.eps;
    L = logf(S) - 2.f * logf(fabsf(uc));
    av = 2.f / S;
    bv = -2.f / uc;
    N = av * av * S + 2.f * av * bv * uc + bv * bv * yy;
  }
  const float lr = a.lr;
  const float den = 1.f - lr * av * hh;
  int err = 0;
  if (!isfinite(L)) err = LST_ENONFINITE;
  else if (!(den != 0.f) || !isfinite(den)) err = LST_ESINGULAR;
  if (blockIdx.x == 0 && tid == 0) {
    a.loss[0] = L;
    if (err) atomicCAS(a.flags + F_ERR, 0, err);
  }
  const float hn = -0.5f * lr * N;
  for (int j = tid; j < d; j += 256) {
    const float g = av * sT[j] + bv * sY[j];
    sT[j] = g + hn * sH[j];
    if (blockIdx.x == 0) a.grad[j] = g;
  }
  __syncthreads();
  if (err0 != 0 || err != 0) return;
  if (shifted && tid < rows) {  // this block's entries of c and s
    float* sv = shift_state(a);
    const int i = i0 + tid;
    sv[i] -= lr * av * (tt + a.eps) * sH[i];
    sv[d + i] -= lr * (av * (nn + (float)a.D * a.eps) + bv) * sH[i];
  }

  // rows i0 .. i0 + rows of Q, U, U^{-T}
  const float cu = lr * av, cp = lr * av / den;
  if (VEC) {
    // entry e of the block's rows: float4 j4 of row ii
    auto update = [&](int e, float4 qv, float4 uw, float4 pw) {
      const int ii = e / d4, j4 = e - ii * d4;
      const int i = i0 + ii;
      const size_t o = (size_t)i * d + 4 * j4;
      const float hi = sH[i], Ti = sT[i];
      const float wu = cu * su[ii], wp = cp * spv[ii];
      const float4 hj = *reinterpret_cast<const float4*>(sH + 4 * j4);
      const float4 Tj = *reinterpret_cast<const float4*>(sT + 4 * j4);
      qv.x -= lr * sym_pair(hi, Tj.x, Ti, hj.x);
      qv.y -= lr * sym_pair(hi, Tj.y, Ti, hj.y);
      qv.z -= lr * sym_pair(hi, Tj.z, Ti, hj.z);
      qv.w -= lr * sym_pair(hi, Tj.w, Ti, hj.w);
      uw.x -= wu * hj.x; uw.y -= wu * hj.y; uw.z -= wu * hj.z; uw.w -= wu * hj.w;
      pw.x += wp * hj.x; pw.y += wp * hj.y; pw.z += wp * hj.z; pw.w += wp * hj.w;
      *reinterpret_cast<float4*>(Q + o) = qv;
      *reinterpret_cast<float4*>(U + o) = uw;
      *reinterpret_cast<float4*>(P + o) = pw;
    };
#pragma unroll
    for (int c = 0; c < kPre; ++c)
      if (tid + 256 * c < ne4) update(tid + 256 * c, pq[c], pu[c], pp[c]);
    for (int e = tid + 256 * kPre; e < ne4; e += 256) {
      const int ii = e / d4;
      const size_t o = (size_t)(i0 + ii) * d + 4 * (e - ii * d4);
      update(e, *reinterpret_cast<const float4*>(Q + o), *reinterpret_cast<const float4*>(U + o),
             *reinterpret_cast<const float4*>(P + o));
    }
  } else {
    for (int e = tid; e < rows * d; e += 256) {
      const int ii = e / d, j = e - ii * d;
      const int i = i0 + ii;
      const size_t o = (size_t)i * d + j;
      const float hi = sH[i], Ti = sT[i], hj = sH[j], Tj = sT[j];
      Q[o] -= lr * sym_pair(hi, Tj, Ti, hj);
      U[o] -= cu * su[ii] * hj;
      P[o] += cp * spv[ii] * hj;
    }
  }
  // columns i0 .. i0 + rows of the target rows of V
  const float cv = -lr / den;
#pragma unroll
  for (int c = 0; c < kVPre; ++c) {
    const int e = tid + 256 * c;
    if (e < nve && vrow[c] >= 0) {
      const float G = a.loss_kind == LST_LOSS_SQUARED ? -2.f * vrs[c] : bv;
      a.V[(size_t)vrow[c] * d + i0 + e % rows] = vval[c] + (cv * G) * spv[e % rows];
    }
  }
  for (int e = tid + 256 * kVPre; e < nve; e += 256) {
    const int k = e / rows, ii = e - k * rows;
    const int r = a.own[k];
    if (r < 0) continue;
    const float G = a.loss_kind == LST_LOSS_SQUARED ? -2.f * a.rsum[k] : bv;
    a.V[(size_t)r * d + i0 + ii] += (cv * G) * spv[ii];
  }
}

}  // namespace

int online_tiles(int d) { return (d + kOnTile - 1) / kOnTile; }

size_t online_workspace_floats(int d) {
  const size_t nt = (size_t)online_tiles(d);
  return 4 * nt * d + 4 * (size_t)d + 3 * nt + 4 + kOnlineMaxK + 2 * (size_t)d;
}

OnlineArgs online_args(int d, float* ws) {
  OnlineArgs a{};
  const int nt = online_tiles(d);
  a.d = d;
  a.nt = nt;
  a.part = ws;
  a.vec = ws + 4 * (size_t)nt * d;
  a.sp = a.vec + 4 * (size_t)d;
  a.scal = a.sp + 3 * nt;
  a.rsum = a.scal + 4;
  return a;
}

hipError_t online_step(const OnlineArgs& a0, hipStream_t s, hipEvent_t e0a, hipEvent_t e1a,
                       hipEvent_t e0b, hipEvent_t e1b) {
  OnlineArgs a = a0;
  if (a.K < 1 || a.K > kOnlineMaxK || a.d < 1 || a.d > 4096 || a.nt != online_tiles(a.d))
    return hipErrorInvalidValue;
  // launch B: about 256 blocks of R <= 16 rows each
  a.rows_per_block = (a.d + 255) / 256;
  void* args[] = {&a};
  const bool vec = a.d % 4 == 0, fused = a.nt <= kOnlineFuseTiles;
  const dim3 ga(1 + a.nt * a.nt), gb((a.d + a.rows_per_block - 1) / a.rows_per_block);
  const size_t ldsb = (size_t)3 * a.d * sizeof(float);
  const void* ka = vec ? (const void*)online_a_kernel<true> : (const void*)online_a_kernel<false>;
  const void* kb = fused ? (vec ? (const void*)online_b_kernel<true, true>
                                : (const void*)online_b_kernel<false, true>)
                         : (vec ? (const void*)online_b_kernel<true, false>
                                : (const void*)online_b_kernel<false, false>);
  hipError_t e;
  if (e0a && e1a)
    e = hipExtLaunchKernel(ka, ga, dim3(256), args, 0, s, e0a, e1a, 0);
  else
    e = hipLaunchKernel(ka, ga, dim3(256), args, 0, s);
  if (e != hipSuccess) return e;
  if (!fused) {
    e = hipLaunchKernel((const void*)online_r_kernel, dim3(a.nt), dim3(256), args, 0, s);
    if (e != hipSuccess) return e;
  }
  if (e0b && e1b) return hipExtLaunchKernel(kb, gb, dim3(256), args, ldsb, s, e0b, e1b, 0);
  return hipLaunchKernel(kb, gb, dim3(256), args, ldsb, s);
}

}  // namespace lst
