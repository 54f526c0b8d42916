// The factored minibatch step (Appendix A) as four launches on one stream.
//
// Each launch is one grid whose blocks run tiles of several independent tasks
// (a "heterogeneous" launch), so the step pays four launch latencies instead
// of one per task:
//   launch 1  GEMM  Z0 = H^T [Q; U; U^{-T}; H^T]^T -> H^, UH, P, H^T H        (steps 1, 7, 8)
//             gather G = (V^T Y)^T                                         (step 2, sparse part)
//             prep  validate and sort each example's targets; record the
//                   smallest slot of every target row in a hash table
//   launch 2  GEMM  Y^ = G U, C1 = H^T H^, C2 = H^T Y^, C2t = C2^T          (steps 2, 5)
//             solve X = S^{-1} P^T, S = H^T H - diag(1/(lr a_i))           (step 8)
//             yy    Y^T Y                                                  (step 5)
//             scalars per example: loss, a_i, b_i, c_i                     (steps 3-6)
//   launch 3  GEMM  grad_H = H^ A + Y^ diag(b), T = grad_H - (lr/2) N H^T    (step 4)
//                   U -= lr (UH) A H^T, U^{-T} -= X^T H^T                   (steps 7, 8)
//             scatter V[r] += sum over examples j holding r of c_j X_j     (step 9)
//   launch 4  GEMM  Q -= lr (H T^T + T H^T), symmetric                      (step 10)
//             clear the hash slots used by this step
// With A = diag(a_i) and G the part of dL/dO sparse on the targets,
// dL/dO = W H A + G: squared error a_i = 2, G = -2 Y; spherical softmax
// a_i = 2 / S_i, G = Y diag(b_i), S_i = h_i^T Q h_i + D eps,
// b_i = -2 o_c / (o_c^2 + eps), o_c = h_i^T W^T y_i.  N = (dL/dO)^T dL/dO.
// Every update of the state (launches 3 and 4) skips when the step's error
// flag is set; all checks that can set it run in launches 1 and 2.
#include <math.h>

#include "gemm_tile.h"
#include "lst_internal.h"

namespace lst {

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

// sum_j x[j] y[j] by one full wave in a fixed order (lane-strided partial
// sums, then a butterfly), so every wave that evaluates it gets the same bits.
__device__ __forceinline__ float wave_dot(const float* x, const float* y, int n) {
  float s = 0.f;
  for (int j = lane_id(); j < n; j += 64) s += x[j] * y[j];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  return s;
}

__device__ __forceinline__ unsigned row_hash(int r, int bits) {
  return ((unsigned)r * 2654435761u) >> (32 - bits);
}

// a_i of example i (squared error: 2; spherical: 2 / S_i).  Called by a full wave.
__device__ __forceinline__ float example_a(const StepCtx& c, int i) {
  if (c.loss_kind == LST_LOSS_SQUARED) return 2.f;
  const float c1 = wave_dot(c.H + (size_t)i * c.d, c.Z0 + (size_t)i * c.ld0, c.d);
  return 2.f / (c1 + (float)c.D * c.eps);
}

// ------------------------------------------------------------------ gather
// G[i, :] = sum_k w_ik V[idx_ik, :]: one wave per (example, 256-column chunk),
// four consecutive columns per lane, eight rows of V in flight at once.
__device__ __forceinline__ void task_gather(const StepCtx& c, int local) {
  const int nchunk = (c.d + 255) / 256;
  const int item = local * 4 + wave_id();
  if (item >= c.m * nchunk) return;
  const int i = item / nchunk, ch = item - i * nchunk;
  const int col = ch * 256 + lane_id() * 4;
  if (col >= c.d) return;
  const bool vec = (c.d % 4 == 0);
  const bool one_hot = c.loss_kind == LST_LOSS_SPHERICAL;
  const int32_t* ix = c.idx + (size_t)i * c.K;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k0 = 0; k0 < c.K; k0 += 8) {
    float4 rv[8];
    float w[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      rv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      w[u] = 0.f;
      const int k = k0 + u;
      if (k >= c.K) continue;
      const int r = ix[k];
      if (r < 0 || (int64_t)r >= c.D) continue;
      w[u] = one_hot ? 1.f : c.val[(size_t)i * c.K + k];
      const float* row = c.V + (size_t)r * c.d + col;
      if (vec) {
        rv[u] = *reinterpret_cast<const float4*>(row);
      } else {
        rv[u].x = row[0];
        if (col + 1 < c.d) rv[u].y = row[1];
        if (col + 2 < c.d) rv[u].z = row[2];
        if (col + 3 < c.d) rv[u].w = row[3];
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      acc.x += w[u] * rv[u].x;
      acc.y += w[u] * rv[u].y;
      acc.z += w[u] * rv[u].z;
      acc.w += w[u] * rv[u].w;
    }
  }
  float* out = c.G + (size_t)i * c.d + col;
  if (vec) {
    *reinterpret_cast<float4*>(out) = acc;
  } else {
    out[0] = acc.x;
    if (col + 1 < c.d) out[1] = acc.y;
    if (col + 2 < c.d) out[2] = acc.z;
    if (col + 3 < c.d) out[3] = acc.w;
  }
}

// ------------------------------------------------------------------- prep
// Example i: validate its K pairs, sort them by (row, slot) into
// ex_row / ex_val, count them, and record in the hash table the smallest
// slot (i*K + k) holding each row.  K <= 1024.
__device__ __forceinline__ void task_prep(const StepCtx& c, int i, unsigned char* sraw) {
  unsigned long long* keys = reinterpret_cast<unsigned long long*>(sraw);
  int* cnt = reinterpret_cast<int*>(sraw + 1024 * sizeof(unsigned long long));
  const bool one_hot = c.loss_kind == LST_LOSS_SPHERICAL;
  constexpr unsigned long long kNoKey = ~0ull;
  if (threadIdx.x == 0) *cnt = 0;
  __syncthreads();
  const int mask = (1 << c.hbits) - 1;
  for (int k = threadIdx.x; k < c.K; k += blockDim.x) {
    const int r = c.idx[(size_t)i * c.K + k];
    const bool valid = (r >= 0) && ((int64_t)r < c.D);
    const bool bad = (r < -1) || ((int64_t)r >= c.D) || (one_hot && r == -1);
    if (bad) atomicCAS(c.flags + F_ERR, 0, LST_EINDEX);
    keys[k] = valid ? (((unsigned long long)(unsigned)r << 32) | (unsigned)k) : kNoKey;
    if (valid) {
      atomicAdd(cnt, 1);
      const int slot = i * c.K + k;
      unsigned h = row_hash(r, c.hbits);
      for (int probe = 0; probe <= mask; ++probe) {  // the table is at most half full
        const int prev = atomicCAS(c.hkey + h, -1, r);
        if (prev == -1 || prev == r) {
          atomicMin(c.hmin + h, slot);
          break;
        }
        h = (h + 1) & mask;
      }
    }
  }
  __syncthreads();
  for (int k = threadIdx.x; k < c.K; k += blockDim.x) {
    const unsigned long long key = keys[k];
    int rank = 0;
    for (int k2 = 0; k2 < c.K; ++k2) {
      const unsigned long long o = keys[k2];
      rank += (o < key) || (o == key && k2 < k);
    }
    const bool valid = key != kNoKey;
    const int kk = (int)(key & 0xffffffffu);
    c.ex_row[(size_t)i * c.K + rank] = valid ? (int)(key >> 32) : -1;
    c.ex_val[(size_t)i * c.K + rank] =
        valid ? (one_hot ? 1.f : c.val[(size_t)i * c.K + kk]) : 0.f;
  }
  if (threadIdx.x == 0) c.ex_cnt[i] = *cnt;
}

// --------------------------------------------------------------------- Y^T Y
// One thread per (i, j), i <= j, merging the two sorted target lists; a row
// that repeats inside an example contributes the sum of its values.  A block
// owns a 16 x 16 block of pairs on or above the diagonal and stages the 32
// lists it needs in LDS (K <= 64; longer lists are merged from memory).
constexpr int kGramKMax = 64;

__device__ __forceinline__ float merge_dot(const int* ri, const float* vi, int ni, const int* rj,
                                           const float* vj, int nj) {
  float acc = 0.f;
  int a = 0, b = 0;
  while (a < ni && b < nj) {
    const int ra = ri[a], rb = rj[b];
    if (ra < rb) {
      ++a;
    } else if (rb < ra) {
      ++b;
    } else {
      float sa = 0.f, sb = 0.f;
      while (a < ni && ri[a] == ra) sa += vi[a++];
      while (b < nj && rj[b] == rb) sb += vj[b++];
      acc += sa * sb;
    }
  }
  return acc;
}

__device__ __forceinline__ void task_yy(const StepCtx& c, int local, unsigned char* sraw) {
  int(*srow)[kGramKMax] = reinterpret_cast<int(*)[kGramKMax]>(sraw);
  float(*sval)[kGramKMax] = reinterpret_cast<float(*)[kGramKMax]>(sraw + 32 * kGramKMax * 4);
  int* scnt = reinterpret_cast<int*>(sraw + 2 * 32 * kGramKMax * 4);
  const int nb = (c.m + 15) / 16;
  int bi = 0, rem = local;
  while (rem >= nb - bi) { rem -= nb - bi; ++bi; }
  const int bj = bi + rem;
  const int I0 = bi * 16, J0 = bj * 16;
  const bool staged = c.K <= kGramKMax;
  if (staged) {
    for (int e = threadIdx.x; e < 32 * c.K; e += blockDim.x) {
      const int l = e / c.K, k = e - l * c.K;
      const int ex = (l < 16) ? I0 + l : J0 + l - 16;
      if (ex < c.m) {
        srow[l][k] = c.ex_row[(size_t)ex * c.K + k];
        sval[l][k] = c.ex_val[(size_t)ex * c.K + k];
      }
    }
    if (threadIdx.x < 32) {
      const int l = threadIdx.x;
      const int ex = (l < 16) ? I0 + l : J0 + l - 16;
      scnt[l] = ex < c.m ? c.ex_cnt[ex] : 0;
    }
    __syncthreads();
  }
  const int li = threadIdx.x >> 4, lj = threadIdx.x & 15;
  const int i = I0 + li, j = J0 + lj;
  if (i >= c.m || j >= c.m || i > j) return;
  float acc;
  if (staged)
    acc = merge_dot(srow[li], sval[li], scnt[li], srow[16 + lj], sval[16 + lj], scnt[16 + lj]);
  else
    acc = merge_dot(c.ex_row + (size_t)i * c.K, c.ex_val + (size_t)i * c.K, c.ex_cnt[i],
                    c.ex_row + (size_t)j * c.K, c.ex_val + (size_t)j * c.K, c.ex_cnt[j]);
  c.yy[(size_t)i * c.m + j] = acc;
  c.yy[(size_t)j * c.m + i] = acc;
}

// ----------------------------------------------------------------- scalars
// One wave per example: c1 = h^T Q h, c2 = h^T W^T y, (Y^T Y)_ii, then
//   squared:   loss = c1 - 2 c2 + (Y^T Y)_ii (= M_ii, Appendix A step 6), a = 2, b = -2
//   spherical: loss = -log(c2^2 + eps) + log(c1 + D eps), a = 2/(c1 + D eps),
//              b = -2 c2 / (c2^2 + eps), cs = b / a (the scatter weight)
// Block 0 also counts the step's target pairs and resets the distinct-row count.
__device__ __forceinline__ void task_scalars(const StepCtx& c, int local) {
  if (local == 0 && threadIdx.x == 0) {
    int nnz = 0;
    for (int j = 0; j < c.m; ++j) nnz += c.ex_cnt[j];
    c.flags[F_NNZ] = nnz;
    c.flags[F_UNIQUE] = 0;
  }
  const int i = local * 4 + wave_id();
  if (i >= c.m) return;
  const float c1 = wave_dot(c.H + (size_t)i * c.d, c.Z0 + (size_t)i * c.ld0, c.d);
  const float c2 = wave_dot(c.Z0 + (size_t)i * c.ld0 + c.d, c.G + (size_t)i * c.d, c.d);
  if (lane_id() != 0) return;
  float L, a, b, cs;
  if (c.loss_kind == LST_LOSS_SQUARED) {
    const int* ri = c.ex_row + (size_t)i * c.K;
    const float* vi = c.ex_val + (size_t)i * c.K;
    const int n = c.ex_cnt[i];
    const float yy = merge_dot(ri, vi, n, ri, vi, n);
    L = c1 - 2.f * c2 + yy;
    a = 2.f;
    b = -2.f;
    cs = 0.f;
  } else {
    const float Si = c1 + (float)c.D * c.eps;
    const float num = c2 * c2 + c.eps;
    L = -logf(num) + logf(Si);
    a = 2.f / Si;
    b = -2.f * c2 / num;
    cs = b / a;
  }
  c.loss[i] = L;
  c.a[i] = a;
  c.b[i] = b;
  c.cs[i] = cs;
  if (!isfinite(L)) atomicCAS(c.flags + F_ERR, 0, LST_ENONFINITE);
}

// ------------------------------------------------------------------- solve
// The Woodbury system of step 8.  With c_i = 1 / (lr a_i), S = H^T H - diag(c)
// and P = U^{-T} H, U_new^{-T} H = -(1/lr) P S^{-1} A^{-1}: all the update
// needs is X = S^{-1} P^T (m x d).  A block solves S X_blk = P^T_blk for 16
// columns.  Writing S = -diag(c) (I - E), E = diag(1/c) H^T H, gives
// X = (I - E)^{-1} B with B = -diag(1/c) P^T.  When r = ||E||_inf < 1/2 the
// Neumann series Y_{k+1} = B + E Y_k converges geometrically and is stopped
// after the first k with r^(k+1) / (1 - r) <= 2^-24, below fp32 rounding of
// the result.  Otherwise (a learning rate so large that 2 lr ||H^T H|| is not
// small) the block runs Gauss-Jordan elimination with partial pivoting on
// [S | P^T_blk] (fp64 in LDS for m <= 128, fp32 in a global workspace above),
// flagging LST_ESINGULAR on a pivot that is not finite or not above
// 1e-13 max|S|.  Every block evaluates r identically, so all take one branch.
constexpr int kSolveCols = 16;

template <typename TT>
__device__ void gj_augmented(TT* A, int lda, int m, int ncol, double* colk, double tiny, int* s_p,
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
        const TT t = A[(size_t)k * lda + j];
        A[(size_t)k * lda + j] = A[(size_t)p * lda + j];
        A[(size_t)p * lda + j] = t;
      }
    }
    __syncthreads();
    const double pinv = 1.0 / (double)A[(size_t)k * lda + k];
    for (int i = tid; i < m; i += nt) colk[i] = (double)A[(size_t)i * lda + k];
    __syncthreads();
    for (int j = tid; j < ncol; j += nt)
      A[(size_t)k * lda + j] = (TT)((double)A[(size_t)k * lda + j] * pinv);
    __syncthreads();
    for (int e = tid; e < m * ncol; e += nt) {
      const int i = e / ncol, j = e - i * ncol;
      if (i == k) continue;
      A[(size_t)i * lda + j] =
          (TT)((double)A[(size_t)i * lda + j] - colk[i] * (double)A[(size_t)k * lda + j]);
    }
    __syncthreads();
  }
}

// LDS bytes of the solve for m (both branches share the buffer).
__host__ __device__ inline size_t solve_lds_bytes(int m) {
  const int mp = (m + 15) & ~15;
  const size_t neumann =
      (size_t)(mp + 3 * kSolveCols * (mp + 4) + (m <= 128 ? mp * (mp + 4) : 0)) * sizeof(float);
  const size_t gj = m <= 128 ? (size_t)m * (m + kSolveCols) * sizeof(double) : 0;
  const size_t extra = 256 * sizeof(float) + 512 * sizeof(double) + 64;  // red, colk, scalars
  return (neumann > gj ? neumann : gj) + extra;
}

template <bool SMALL>
__device__ __forceinline__ void task_solve(const StepCtx& c, int local, unsigned char* sraw) {
  const int m = c.m, d = c.d;
  const float* HH = c.Z0 + 3 * d;
  const float* P = c.Z0 + 2 * d;
  const int ldh = c.ld0, ldp = c.ld0;
  const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
  const int mp = (m + 15) & ~15;
  const int LDE = mp + 4;
  const int c0 = local * kSolveCols;
  const size_t main_bytes = solve_lds_bytes(m) - (256 * sizeof(float) + 512 * sizeof(double) + 64);
  float* red = reinterpret_cast<float*>(sraw + main_bytes);
  double* colk = reinterpret_cast<double*>(red + 256);
  int* s_int = reinterpret_cast<int*>(colk + 512);  // s_p, s_bad
  float* s_flt = reinterpret_cast<float*>(s_int + 2);  // r, amax
  float* cinv = reinterpret_cast<float*>(sraw);        // mp
  float* Bt = cinv + mp;                               // kSolveCols x LDE: B^T
  float* Y0 = Bt + kSolveCols * LDE;                   // kSolveCols x LDE: Y^T
  float* Y1 = Y0 + kSolveCols * LDE;
  float* Es = Y1 + kSolveCols * LDE;                   // mp x LDE (SMALL only)

  for (int i = wave; i < mp; i += 4) {
    const float a = (i < m) ? example_a(c, i) : 0.f;
    if (lane == 0) cinv[i] = (i < m) ? c.lr * a : 0.f;  // 1 / c_i
  }
  if (tid == 0) s_int[1] = 0;
  __syncthreads();
  float rowmax = 0.f, amax = 0.f;
  if (SMALL) {
    const bool vec4 = (ldh % 4 == 0) && (((uintptr_t)HH & 15) == 0);
    constexpr int NQ = 128 * 128 / 4 / 256;
    float4 r4[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int e4 = tid + 256 * q;
      const int i = e4 / (mp / 4), j = 4 * (e4 - i * (mp / 4));
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (e4 < mp * mp / 4 && i < m) {
        const float* hr = HH + (size_t)i * ldh + j;
        if (vec4 && j + 3 < m) {
          v = *reinterpret_cast<const float4*>(hr);
        } else {
          if (j < m) v.x = hr[0];
          if (j + 1 < m) v.y = hr[1];
          if (j + 2 < m) v.z = hr[2];
          if (j + 3 < m) v.w = hr[3];
        }
      }
      r4[q] = v;
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int e4 = tid + 256 * q;
      if (e4 < mp * mp / 4) {
        const int i = e4 / (mp / 4), j = 4 * (e4 - i * (mp / 4));
        const float ci = cinv[i];
        *reinterpret_cast<float4*>(Es + i * LDE + j) =
            make_float4(r4[q].x * ci, r4[q].y * ci, r4[q].z * ci, r4[q].w * ci);
      }
    }
    __syncthreads();
    for (int i = tid; i < m; i += 256) {
      float sabs = 0.f, hmax = 0.f;
      const float ci = 1.f / cinv[i];
      for (int j = 0; j < m; ++j) {
        const float e = Es[i * LDE + j];
        sabs += fabsf(e);
        hmax = fmaxf(hmax, fabsf(e * ci - (i == j ? ci : 0.f)));
      }
      rowmax = fmaxf(rowmax, sabs);
      amax = fmaxf(amax, hmax);
    }
  } else {
    for (int i = tid; i < m; i += 256) {
      float sabs = 0.f, hmax = 0.f;
      const float ci = 1.f / cinv[i];
      const float* hr = HH + (size_t)i * ldh;
      for (int j0 = 0; j0 < m; j0 += 8) {
        float hv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) hv[u] = (j0 + u < m) ? hr[j0 + u] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          sabs += fabsf(hv[u]);
          hmax = fmaxf(hmax, fabsf(hv[u] - (i == j0 + u ? ci : 0.f)));
        }
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
  if (tid == 0) s_flt[0] = red[0];
  __syncthreads();
  red[tid] = amax;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) red[tid] = fmaxf(red[tid], red[tid + off]);
    __syncthreads();
  }
  if (tid == 0) s_flt[1] = red[0];
  __syncthreads();
  const float r = s_flt[0];

  if (r < 0.5f) {
    for (int e0 = 0; e0 < kSolveCols * mp; e0 += 256 * 8) {
      float pv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + tid + 256 * u;
        const int i = e / kSolveCols, cc = e - i * kSolveCols;
        pv[u] = (e < kSolveCols * mp && i < m && c0 + cc < d) ? P[(size_t)i * ldp + c0 + cc] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + tid + 256 * u;
        if (e < kSolveCols * mp) {
          const int i = e / kSolveCols, cc = e - i * kSolveCols;
          const float v = -pv[u] * cinv[i];
          Bt[cc * LDE + i] = v;
          Y0[cc * LDE + i] = v;
        }
      }
    }
    int iters = 0;
    if (r > 0.f) {
      const float need = logf(5.9604645e-8f * (1.f - r)) / logf(r);  // r^(k+1)/(1-r) <= 2^-24
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
      const int i = e / kSolveCols, cc = e - i * kSolveCols;
      if (c0 + cc < d) c.X[(size_t)i * d + c0 + cc] = Yo[cc * LDE + i];
    }
    return;
  }

  // Fallback: Gauss-Jordan on [S | P^T_blk], S = H^T H - diag(c).  c_i moves
  // to colk first: the fp64 matrix overwrites the buffers that hold 1/c_i.
  const int ncol = m + kSolveCols;
  const double tiny = 1e-13 * (double)s_flt[1];
  for (int i = tid; i < m; i += 256) colk[i] = 1.0 / (double)cinv[i];
  __syncthreads();
  if (SMALL) {
    double* A = reinterpret_cast<double*>(sraw);  // aliases the Neumann buffers
    for (int e = tid; e < m * ncol; e += 256) {
      const int i = e / ncol, j = e - i * ncol;
      double v;
      if (j < m) {
        v = (double)HH[(size_t)i * ldh + j];
        if (i == j) v -= colk[i];
      } else {
        v = (c0 + j - m < d) ? (double)P[(size_t)i * ldp + c0 + j - m] : 0.0;
      }
      A[(size_t)i * ncol + j] = v;
    }
    __syncthreads();
    gj_augmented<double>(A, ncol, m, ncol, colk, tiny, s_int, s_int + 1);
    if (s_int[1]) {
      if (tid == 0) atomicCAS(c.flags + F_ERR, 0, LST_ESINGULAR);
      return;
    }
    for (int e = tid; e < m * kSolveCols; e += 256) {
      const int i = e / kSolveCols, cc = e - i * kSolveCols;
      if (c0 + cc < d) c.X[(size_t)i * d + c0 + cc] = (float)A[(size_t)i * ncol + m + cc];
    }
  } else {
    float* A = c.solve_ws + (size_t)local * m * ncol;
    for (int e = tid; e < m * ncol; e += 256) {
      const int i = e / ncol, j = e - i * ncol;
      float v;
      if (j < m) {
        v = HH[(size_t)i * ldh + j];
        if (i == j) v -= (float)colk[i];
      } else {
        v = (c0 + j - m < d) ? P[(size_t)i * ldp + c0 + j - m] : 0.f;
      }
      A[(size_t)i * ncol + j] = v;
    }
    __syncthreads();
    gj_augmented<float>(A, ncol, m, ncol, colk, tiny, s_int, s_int + 1);
    if (s_int[1]) {
      if (tid == 0) atomicCAS(c.flags + F_ERR, 0, LST_ESINGULAR);
      return;
    }
    for (int e = tid; e < m * kSolveCols; e += 256) {
      const int i = e / kSolveCols, cc = e - i * kSolveCols;
      if (c0 + cc < d) c.X[(size_t)i * d + c0 + cc] = A[(size_t)i * ncol + m + cc];
    }
  }
}

// ----------------------------------------------------------------- scatter
// Step 9: V[r, :] += sum over the examples j whose target holds row r of
// c_j X[j, :], c_j = -(sum of j's values at r) (squared) or cs_j (spherical),
// in increasing j.  One wave per (example, slot) pair; only the pair with the
// smallest slot of its row (read from the hash table) does the work, so every
// row is written once and in a fixed order.  The touched row is appended to
// the step's row list (the hash slots are cleared from it in launch 4).
__device__ __forceinline__ void task_scatter(const StepCtx& c, int local) {
  const int e = local * 4 + wave_id();
  if (e >= c.m * c.K) return;
  const int lane = lane_id();
  const int i = e / c.K, k = e - i * c.K;
  const int r = c.idx[e];
  if (r < 0 || (int64_t)r >= c.D) return;
  const int mask = (1 << c.hbits) - 1;
  unsigned h = row_hash(r, c.hbits);
  int probe = 0;
  while (probe <= mask && c.hkey[h] != r) {
    h = (h + 1) & mask;
    ++probe;
  }
  if (probe > mask || c.hmin[h] != e) return;  // not the owner of row r
  if (lane == 0) {
    const int pos = atomicAdd(c.flags + F_UNIQUE, 1);
    c.touched[pos] = r;
  }
  if (c.flags[F_ERR]) return;
  const bool one_hot = c.loss_kind == LST_LOSS_SPHERICAL;
  const bool vec = (c.d % 4 == 0);
  // columns in groups of 1024 (four 256-column chunks held in registers)
  for (int cg = 0; cg < c.d; cg += 1024) {
    float4 acc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j0 = i; j0 < c.m; j0 += 64) {
      const int j = j0 + lane;
      float cj = 0.f;
      bool found = false;
      if (j < c.m) {
        const int* rows = c.ex_row + (size_t)j * c.K;
        const float* vals = c.ex_val + (size_t)j * c.K;
        const int n = c.ex_cnt[j];
        int lo = 0, hi = n;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (rows[mid] < r) lo = mid + 1; else hi = mid;
        }
        float sum = 0.f;
        while (lo < n && rows[lo] == r) {
          sum += vals[lo];
          ++lo;
          found = true;
        }
        cj = one_hot ? c.cs[j] : -sum;
      }
      unsigned long long bal = __ballot(found);
      while (bal) {
        const int src = __ffsll((long long)bal) - 1;
        bal &= bal - 1;
        const float w = __shfl(cj, src);
        const float* xr = c.X + (size_t)(j0 + src) * c.d;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = cg + q * 256 + lane * 4;
          if (col >= c.d) continue;
          if (vec) {
            const float4 x = *reinterpret_cast<const float4*>(xr + col);
            acc[q].x += w * x.x; acc[q].y += w * x.y; acc[q].z += w * x.z; acc[q].w += w * x.w;
          } else {
            acc[q].x += w * xr[col];
            if (col + 1 < c.d) acc[q].y += w * xr[col + 1];
            if (col + 2 < c.d) acc[q].z += w * xr[col + 2];
            if (col + 3 < c.d) acc[q].w += w * xr[col + 3];
          }
        }
      }
    }
    float* vr = c.V + (size_t)r * c.d;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int col = cg + q * 256 + lane * 4;
      if (col >= c.d) continue;
      if (vec) {
        float4 v = *reinterpret_cast<float4*>(vr + col);
        v.x += acc[q].x; v.y += acc[q].y; v.z += acc[q].z; v.w += acc[q].w;
        *reinterpret_cast<float4*>(vr + col) = v;
      } else {
        vr[col] += acc[q].x;
        if (col + 1 < c.d) vr[col + 1] += acc[q].y;
        if (col + 2 < c.d) vr[col + 2] += acc[q].z;
        if (col + 3 < c.d) vr[col + 3] += acc[q].w;
      }
    }
  }
}

// Launch 4: empty the hash slots of the rows this step touched.
__device__ __forceinline__ void task_clear(const StepCtx& c, int local) {
  const int t = local * 256 + threadIdx.x;
  if (t >= c.flags[F_UNIQUE]) return;
  const int r = c.touched[t];
  const int mask = (1 << c.hbits) - 1;
  unsigned h = row_hash(r, c.hbits);
  for (int probe = 0; probe <= mask; ++probe) {
    if (c.hkey[h] == r) {
      c.hkey[h] = -1;
      c.hmin[h] = 0x7fffffff;
      return;
    }
    h = (h + 1) & mask;
  }
}

// -------------------------------------------------------------- the kernel
#ifdef LST_TIMING
// Per-block (start, end) wall clock of the last launches, for latency studies.
__device__ unsigned long long g_step_times[4][8192][3];
#endif

template <int TILE, bool SMALLM>
__device__ __forceinline__ void run_task(const StepCtx& c, const StepLaunch& L, int t, int local,
                                         unsigned char* sraw) {
  switch (L.kind[t]) {
    case TK_GEMM:
      if (L.gemm.skip_if && *L.gemm.skip_if) return;
      panel_tile<TILE, TILE>(L.gemm, local, reinterpret_cast<float*>(sraw));
      break;
    case TK_GATHER: task_gather(c, local); break;
    case TK_PREP: task_prep(c, local, sraw); break;
    case TK_YY: task_yy(c, local, sraw); break;
    case TK_SCALARS: task_scalars(c, local); break;
    case TK_SOLVE: task_solve<SMALLM>(c, local, sraw); break;
    case TK_SCATTER: task_scatter(c, local); break;
    case TK_CLEAR: task_clear(c, local); break;
    default: break;
  }
}

template <int TILE, bool SMALLM>
__global__ __launch_bounds__(256) void step_kernel(StepCtx c, StepLaunch L) {
  extern __shared__ __attribute__((aligned(16))) unsigned char sraw[];
  const int blk = blockIdx.x;
  int t = 0;
  while (t + 1 < L.ntask && blk >= L.begin[t + 1]) ++t;
  const int local = blk - L.begin[t];
#ifdef LST_TIMING
  const unsigned long long t0 = wall_clock64();
#endif
  run_task<TILE, SMALLM>(c, L, t, local, sraw);
#ifdef LST_TIMING
  __syncthreads();
  if (threadIdx.x == 0 && blk < 8192) {
    g_step_times[L.timing_slot & 3][blk][0] = t0;
    g_step_times[L.timing_slot & 3][blk][1] = wall_clock64();
    g_step_times[L.timing_slot & 3][blk][2] = (unsigned long long)L.kind[t];
  }
#endif
}

// ------------------------------------------------------------------- host
static size_t lds_of(int kind, int tile, int kcw, int m) {
  switch (kind) {
    case TK_GEMM: return (size_t)panel_lds_floats(tile, tile, kcw) * sizeof(float);
    case TK_PREP: return 1024 * sizeof(unsigned long long) + 16;
    case TK_YY: return 2 * 32 * kGramKMax * 4 + 32 * 4;
    case TK_SOLVE: return solve_lds_bytes(m);
    default: return 0;
  }
}

static int tiles_of(GemmBatch& b, int tile) {
  int total = 0;
  for (int q = 0; q < b.np; ++q) {
    GemmProblem& p = b.p[q];
    p.tiles_m = (p.M + tile - 1) / tile;
    p.tiles_n = (p.N + tile - 1) / tile;
    p.tile_begin = total;
    if (p.ksplit < 1) p.ksplit = 1;
    if (p.epi == EPI_SYM)
      total += p.tiles_m * (p.tiles_m + 1) / 2;
    else
      total += p.tiles_m * p.tiles_n * (p.epi == EPI_PARTIAL ? p.ksplit : 1);
  }
  b.total_tiles = total;
  return total;
}

int step_task_blocks(int kind, const StepCtx& c) {
  switch (kind) {
    case TK_GATHER: return (c.m * ((c.d + 255) / 256) + 3) / 4;
    case TK_PREP: return c.m;
    case TK_YY: { const int nb = (c.m + 15) / 16; return nb * (nb + 1) / 2; }
    case TK_SCALARS: return (c.m + 3) / 4;
    case TK_SOLVE: return (c.d + kSolveCols - 1) / kSolveCols;
    case TK_SCATTER: return (c.m * c.K + 3) / 4;
    case TK_CLEAR: return (c.m * c.K + 255) / 256;
    default: return 0;
  }
}

hipError_t step_launch(const StepCtx& c, StepLaunch& L, int tile, hipStream_t s) {
  if (tile != 32 && tile != 64) return hipErrorInvalidValue;
  size_t lds = 0;
  int total = 0;
  for (int t = 0; t < L.ntask; ++t) {
    L.begin[t] = total;
    int n = 0;
    if (L.kind[t] == TK_GEMM) {
      if (L.gemm.kcw_max > panel_kcw_max(tile)) L.gemm.kcw_max = panel_kcw_max(tile);
      n = tiles_of(L.gemm, tile);
    } else {
      n = step_task_blocks(L.kind[t], c);
    }
    const size_t b = lds_of(L.kind[t], tile, L.gemm.kcw_max, c.m);
    if (b > lds) lds = b;
    total += n;
  }
  L.begin[L.ntask] = total;
  if (total == 0) return hipSuccess;
  const bool small = c.m <= 128;
  const dim3 grid(total), block(256);
  if (tile == 32) {
    if (small)
      hipLaunchKernelGGL((step_kernel<32, true>), grid, block, lds, s, c, L);
    else
      hipLaunchKernelGGL((step_kernel<32, false>), grid, block, lds, s, c, L);
  } else {
    if (small)
      hipLaunchKernelGGL((step_kernel<64, true>), grid, block, lds, s, c, L);
    else
      hipLaunchKernelGGL((step_kernel<64, false>), grid, block, lds, s, c, L);
  }
  return hipGetLastError();
}

size_t solve_workspace_floats(int m_max, int d) {
  if (m_max <= 128) return 0;
  const size_t blocks = (size_t)(d + kSolveCols - 1) / kSolveCols;
  return blocks * (size_t)m_max * (m_max + kSolveCols);
}

hipError_t configure_kernels() {
  const int lds_max = 160 * 1024 - 1024;
  const void* ks[] = {reinterpret_cast<const void*>(step_kernel<32, true>),
                      reinterpret_cast<const void*>(step_kernel<32, false>),
                      reinterpret_cast<const void*>(step_kernel<64, true>),
                      reinterpret_cast<const void*>(step_kernel<64, false>)};
  for (const void* k : ks) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Sorts n (<= 16384) ints ascending in place: one block, bitonic in LDS.  Used
// by the debug accessor of the touched rows.
__global__ __launch_bounds__(1024) void sort_ints_kernel(int* v, const int* n_ptr) {
  __shared__ int key[16384];
  const int n = *n_ptr;
  int np2 = 1;
  while (np2 < n) np2 <<= 1;
  for (int e = threadIdx.x; e < np2; e += blockDim.x) key[e] = (e < n) ? v[e] : 0x7fffffff;
  __syncthreads();
  for (int size = 2; size <= np2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int e = threadIdx.x; e < (np2 >> 1); e += blockDim.x) {
        const int lo = 2 * e - (e & (stride - 1));
        const int hi = lo + stride;
        const bool up = ((lo & size) == 0);
        const int a = key[lo], b = key[hi];
        if ((a > b) == up) {
          key[lo] = b;
          key[hi] = a;
        }
      }
      __syncthreads();
    }
  }
  for (int e = threadIdx.x; e < n; e += blockDim.x) v[e] = key[e];
}

#ifdef LST_TIMING
extern "C" int lst_debug_step_times(unsigned long long* out) {
  return hipMemcpyFromSymbol(out, HIP_SYMBOL(g_step_times), sizeof(g_step_times)) == hipSuccess
             ? 0 : -5;
}
#endif

hipError_t sort_ints(int* v, const int* n_ptr, hipStream_t s) {
  hipLaunchKernelGGL(sort_ints_kernel, dim3(1), dim3(1024), 0, s, v, n_ptr);
  return hipGetLastError();
}

__global__ void fill_ints_kernel(int* p, int v, int n) {
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n; e += gridDim.x * blockDim.x) p[e] = v;
}

hipError_t fill_ints(int* p, int v, int n, hipStream_t s) {
  int blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(fill_ints_kernel, dim3(blocks), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

}  // namespace lst
