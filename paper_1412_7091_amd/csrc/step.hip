// The factored minibatch step (Appendix A) as four launches on one stream.
//
// Each launch is one grid whose blocks run tiles of several independent tasks
// (a "heterogeneous" launch), and each launch has its own kernel holding only
// its tasks:
//   launch 1  GEMM    Z0 = H [Q; U; U^{-T}; H^T]^T -> H^, UH, P, H^T H      (steps 1, 7, 8)
//             targets per example: validate and order the targets, (Y^T Y)_ii,
//                     gather G = (V^T Y)^T                                  (step 2, sparse part)
//   launch 2  GEMM    Y^ = G U, C1 = H^T H^, C2 = H^T Y^, C2^T                (steps 2, 5)
//             solve   X = S^{-1} P^T, S = H^T H - diag(1/(lr a_i))         (step 8)
//             yy      Y^T Y                                                (step 5)
//             scalars per example: loss, a_i, b_i, c_i, a h_i, b h_i, and the
//                     hash table of each target row's smallest slot         (steps 3-6)
//   launch 3  GEMM    grad_H = H^ A + Y^ diag(b), T = grad_H - (lr/2) N H^T  (step 4)
//                     with N H^T = A [C1 C2] [AH; BH] + B [C2^T Y^T Y] [AH; BH];
//                     for m > 128 a small kernel forms N between launches 2
//                     and 3 and the GEMM takes N H^T directly
//             scatter V[r] += sum over examples j holding r of c_j X_j     (step 9)
//   launch 4  GEMM    Q -= lr (H T^T + T H^T), symmetric; U -= lr (UH) A H^T;
//                     U^{-T} -= X^T H^T                                     (steps 7, 8, 10)
//             clear   the hash slots used by this step
// With A = diag(a_i) and G the part of dL/dO sparse on the targets,
// dL/dO = W H A + G: squared error a_i = 2, G = -2 Y; spherical softmax
// a_i = 2 / S_i, G = Y diag(b_i), S_i = h_i^T Q h_i + D eps,
// b_i = -2 o_c / (o_c^2 + eps), o_c = h_i^T W^T y_i.  N = (dL/dO)^T dL/dO.
// The shifted spherical softmax (section 3.6 as printed, u = o + eps) adds
// eps 1 a^T to dL/dO, with S_i = h_i^T Q h_i + 2 eps n_i + D eps^2 and
// b_i = -2 / u_c; W = V U + 1 c^T, s = W^T 1, t_i = c^T h_i and n_i = s^T h_i
// (from the targets task of launch 1, which also copies [c | s] after nt).  A
// small kernel between launches 2 and 3 (shifted.hip) adds the extra terms to
// C1, C2, H^ and Y^ from that copy and moves c and s.
// Every update of the state (the scatter, launch 4) skips when the step's
// error flag is set; all checks that can set it run in launches 1 and 2.
#include <hip/hip_ext.h>
#include <math.h>

#include "gemm_tile.h"
#include "lst_internal.h"

namespace lst {

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

__device__ __forceinline__ unsigned row_hash(int r, int bits) {
  return ((unsigned)r * 2654435761u) >> (32 - bits);
}

// The hot-row list, stored after the hash table's slot counts.
__device__ __forceinline__ int* hot_list(const StepCtx& c) { return c.hcnt + (1 << c.hbits); }
__device__ __forceinline__ int* hslot_of(const StepCtx& c) { return c.hmin + (1 << c.hbits); }
// After the slot lists: the number of rows held by two or more slots this step,
// then their hash entries (appended when a row's second slot arrives; at most
// m K / 2 <= 2^hbits / 4 of them).
__device__ __forceinline__ int* multi_rows(const StepCtx& c) {
  return c.hmin + (size_t)(1 << c.hbits) * (1 + kSlotCap);
}

// c1 = h_i^T Q h_i: the partial sums left by the first product of the step,
// added in index order (the same bits wherever it is evaluated).
__device__ __forceinline__ float example_c1(const StepCtx& c, int i) {
  const float* p = c.c1p + (size_t)i * c.ld_c1p;
  const int n = c.n_c1p;
  float s = 0.f;
  int t = 0;
  for (; t + 8 <= n; t += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = p[t + u];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  for (; t < n; ++t) s += p[t];
  return s;
}

// S_i of the spherical losses from c1 = h_i^T Q h_i: sum_j (o_j^2 + eps) =
// c1 + D eps, or for the shifted form sum_j (o_j + eps)^2 = c1 + 2 eps n_i + D eps^2.
__device__ __forceinline__ float example_S(const StepCtx& c, int i, float c1) {
  if (c.loss_kind == LST_LOSS_SPHERICAL_SHIFTED)
    return c1 + 2.f * c.eps * c.nt[2 * i + 1] + (float)c.D * c.eps * c.eps;
  return c1 + (float)c.D * c.eps;
}

// a_i of example i (squared error: 2; spherical: 2 / S_i).
__device__ __forceinline__ float example_a(const StepCtx& c, int i) {
  if (c.loss_kind == LST_LOSS_SQUARED) return 2.f;
  return 2.f / example_S(c, i, example_c1(c, i));
}

// ----------------------------------------------------------------- targets
// Launch 1, one wave per example i (four per block, no block barrier):
//  - load and validate its K (index, value) pairs (LST_EINDEX on a bad index);
//  - order the pairs by (row, slot) into ex_row / ex_val (a sort across the
//    wave's lanes for K <= 64, else a rank sort in its part of LDS) and count
//    them;
//  - (Y^T Y)_ii = sum over distinct rows of (sum of the row's values)^2, each
//    row's values added in slot order;
//  - G_i = sum_k y_ik V[r_ik, :] (Appendix A step 2, the sparse product),
//    slots in order, up to 16 rows of V in flight.
constexpr unsigned long long kNoKey = ~0ull;

// Ascending sort of one 64-bit key per lane across the wave (bitonic network).
__device__ __forceinline__ unsigned long long wave_sort_asc_u64(unsigned long long x) {
  const int lane = lane_id();
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const unsigned long long o = __shfl_xor(x, j);
      const bool up = (lane & k) == 0, low = (lane & j) == 0;
      x = (low == up) ? (o < x ? o : x) : (o > x ? o : x);
    }
  return x;
}

__host__ __device__ inline size_t targets_lds_bytes(int K) {
  return (size_t)4 * K * (sizeof(unsigned long long) + sizeof(float));
}

// Slots per batch of the gather: one batch covers K <= 16.
constexpr int kGatherRows = 16;

// One batch of the gather: rows of slots k0 .. k0 + kGatherRows - 1 (weights
// wv, 0 for slots past K or without a valid target), columns cb + 256 h +
// 4 lane, h < 2.  VEC: d % 4 == 0 (16-byte loads).  Every key is read from
// LDS before the first row is requested, and slots past K request nothing.
template <bool VEC>
__device__ __forceinline__ void gather_load(const StepCtx& c, const unsigned long long* keys,
                                            const float* vals, int k0, int cb,
                                            float4 (&rv)[kGatherRows][2], float (&wv)[kGatherRows]) {
  const int K = c.K, d = c.d, lane = lane_id();
  unsigned long long key[kGatherRows];
#pragma unroll
  for (int u = 0; u < kGatherRows; ++u) key[u] = keys[min(k0 + u, K - 1)];
#pragma unroll
  for (int u = 0; u < kGatherRows; ++u) {
    const bool use = (k0 + u < K) && key[u] != kNoKey;
    wv[u] = use ? vals[min(k0 + u, K - 1)] : 0.f;
    if (k0 + u >= K) continue;  // uniform: K is the same for every lane
    const float* row = c.V + (size_t)(use ? (unsigned)(key[u] >> 32) : 0u) * d;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int col = min(cb + 256 * h + 4 * lane, VEC ? d - 4 : d - 1);
      if (VEC) {
        rv[u][h] = *reinterpret_cast<const float4*>(row + col);
      } else {
        rv[u][h].x = row[col];
        rv[u][h].y = row[min(col + 1, d - 1)];
        rv[u][h].z = row[min(col + 2, d - 1)];
        rv[u][h].w = row[min(col + 3, d - 1)];
      }
    }
  }
}

__device__ __forceinline__ void gather_add(const float4 (&rv)[kGatherRows][2],
                                           const float (&wv)[kGatherRows], float4 (&acc)[2]) {
#pragma unroll
  for (int u = 0; u < kGatherRows; ++u)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // unused slots add nothing (not even a non-finite value of row 0)
      const bool use = wv[u] != 0.f;
      acc[h].x += use ? wv[u] * rv[u][h].x : 0.f;
      acc[h].y += use ? wv[u] * rv[u][h].y : 0.f;
      acc[h].z += use ? wv[u] * rv[u][h].z : 0.f;
      acc[h].w += use ? wv[u] * rv[u][h].w : 0.f;
    }
}

#ifdef LST_TIMING
__device__ unsigned long long g_target_marks[64][6];
#define LST_TMARK(k)                                                            \
  do {                                                                          \
    if (lane == 0 && w == 0 && local < 64) g_target_marks[local][k] = wall_clock64(); \
  } while (0)
#else
#define LST_TMARK(k) \
  do {               \
  } while (0)
#endif

template <bool VEC>
__device__ __forceinline__ void task_targets(const StepCtx& c, int local, unsigned char* sraw) {
  const int w = wave_id(), lane = lane_id();
  const int i = local * 4 + w;
  if (i >= c.m) return;
  if (i == 0 && lane == 0) multi_rows(c)[0] = 0;  // filled in launch 2, read in launch 3
  LST_TMARK(0);
  const int K = c.K, d = c.d;
  if (c.loss_kind == LST_LOSS_SPHERICAL_SHIFTED) {
    // t_i = c^T h_i, n_i = s^T h_i; and a copy of [c | s] after nt (its 2 m
    // entries), striped over the examples' waves, which the terms added between
    // launches 2 and 3 read while the same kernel moves c and s
    const float* hr = c.H + (size_t)i * d;
    float tt = 0.f, nn = 0.f;
    for (int j0 = 0; j0 < d; j0 += 512) {
      float hv[8], cv[8], sv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = min(j0 + lane + 64 * u, d - 1);
        hv[u] = hr[j];
        cv[u] = c.sv[j];
        sv[u] = c.sv[d + j];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (j0 + lane + 64 * u < d) {
          tt += cv[u] * hv[u];
          nn += sv[u] * hv[u];
        }
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      tt += __shfl_xor(tt, off);
      nn += __shfl_xor(nn, off);
    }
    if (lane == 0) {
      c.nt[2 * i] = tt;
      c.nt[2 * i + 1] = nn;
    }
    float* snap = c.nt + 2 * c.m;
    for (int j = 64 * i + lane; j < 2 * d; j += 64 * c.m) snap[j] = c.sv[j];
  }
  unsigned long long* keys = reinterpret_cast<unsigned long long*>(sraw) + (size_t)w * K;
  float* vals = reinterpret_cast<float*>(sraw + (size_t)4 * K * sizeof(unsigned long long)) +
                (size_t)w * K;
  const bool one_hot = c.loss_kind != LST_LOSS_SQUARED;
  const int32_t* ix = c.idx + (size_t)i * K;
  int nvalid = 0;
  for (int k0 = 0; k0 < K; k0 += 64) {
    const int k = k0 + lane;
    const bool in = k < K;
    const int r = in ? ix[k] : -1;
    const float v = (in && !one_hot) ? c.val[(size_t)i * K + k] : 1.f;
    const bool valid = in && r >= 0 && (int64_t)r < c.D;
    const bool bad = in && ((r < -1) || ((int64_t)r >= c.D) || (one_hot && r == -1));
    if (bad) atomicCAS(c.flags + F_ERR, 0, LST_EINDEX);
    if (in) {
      keys[k] = valid ? (((unsigned long long)(unsigned)r << 32) | (unsigned)k) : kNoKey;
      vals[k] = valid ? v : 0.f;
    }
    nvalid += __popcll(__ballot(valid));
  }
  // LDS is read back by other lanes of this wave: the wave's LDS accesses
  // complete in order, so only the compiler must not move them.
  asm volatile("" ::: "memory");

  LST_TMARK(1);
  // The first rows of V are requested now and used after the ordering below,
  // whose latency they overlap.
  float4 rv[kGatherRows][2];
  float wv[kGatherRows];
  gather_load<VEC>(c, keys, vals, 0, 0, rv, wv);

  LST_TMARK(2);
  float yy = 0.f;
  if (K <= 64) {
    // One key per lane, sorted across the wave: lane l then holds the l-th
    // pair in (row, slot) order, and the first lane of each row's run adds
    // the run's values in slot order.
    const unsigned long long key = wave_sort_asc_u64(lane < K ? keys[lane] : kNoKey);
    const bool valid = key != kNoKey;
    const int row = valid ? (int)(unsigned)(key >> 32) : -1;
    const float v = valid ? vals[(unsigned)key] : 0.f;
    const int prev_row = __shfl_up(row, 1);  // every lane takes part in the shuffle
    const bool first = valid && (lane == 0 || prev_row != row);
    float run = v;
    bool more = first;
    for (int t = 1; t < 64 && __ballot(more) != 0ull; ++t) {
      const float vt = __shfl_down(v, t);
      const int rt = __shfl_down(row, t);
      more = more && lane + t < 64 && rt == row;
      if (more) run += vt;
    }
    if (first) yy = run * run;
    if (lane < K) {
      c.ex_row[(size_t)i * K + lane] = row;
      c.ex_val[(size_t)i * K + lane] = v;
    }
  }
  for (int k0 = 0; K > 64 && k0 < K; k0 += 64) {
    const int k = k0 + lane;
    if (k < K) {
      const unsigned long long key = keys[k];
      const unsigned row = (unsigned)(key >> 32);
      int rank = 0;
      bool first = true;
      float run = 0.f;
      for (int k2 = 0; k2 < K; ++k2) {
        const unsigned long long o = keys[k2];
        rank += (o < key) || (o == key && k2 < k);
        if ((unsigned)(o >> 32) == row && o != kNoKey) {
          run += vals[k2];
          first = first && !(k2 < k);
        }
      }
      const bool valid = key != kNoKey;
      if (valid && first) yy += run * run;
      c.ex_row[(size_t)i * K + rank] = valid ? (int)row : -1;
      c.ex_val[(size_t)i * K + rank] = vals[k];
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) yy += __shfl_xor(yy, off);
  if (lane == 0) {
    c.ex_cnt[i] = nvalid;
    c.yyd[i] = yy;
  }

  LST_TMARK(3);
  // G_i = sum_k y_ik V[r_ik, :]: lane l owns columns cb + 256 h + 4 l, slots
  // in order, kGatherRows rows (2 kGatherRows loads) in flight.
  float* gout = c.G + (size_t)i * d;
  for (int cb = 0; cb < d; cb += 512) {
    float4 acc[2] = {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
    for (int k0 = 0; k0 < K; k0 += kGatherRows) {
      if (cb > 0 || k0 > 0) gather_load<VEC>(c, keys, vals, k0, cb, rv, wv);
      gather_add(rv, wv, acc);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int col = cb + 256 * h + 4 * lane;
      if (col >= d) continue;
      if (VEC) {
        *reinterpret_cast<float4*>(gout + col) = acc[h];
      } else {
        gout[col] = acc[h].x;
        if (col + 1 < d) gout[col + 1] = acc[h].y;
        if (col + 2 < d) gout[col + 2] = acc[h].z;
        if (col + 3 < d) gout[col + 3] = acc[h].w;
      }
    }
  }
  LST_TMARK(4);
}

// --------------------------------------------------------------------- Y^T Y
// One thread per (i, j), i <= j, merging the two sorted target lists; a row
// that repeats inside an example contributes the sum of its values.  A block
// owns a 16 x 16 block of pairs on or above the diagonal and stages the 32
// lists it needs in LDS (K <= 64, every load in flight at once; longer lists
// are merged from memory), with a row stride of 65 words so that lanes at the
// same position of different lists fall in different LDS banks.
constexpr int kGramKMax = 64;
constexpr int kGramLd = kGramKMax + 1;

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

// The same sum for lists whose rows are distinct: every step advances the
// side(s) with the smaller row, with no branch inside the loop, so the lanes
// of a wave (each merging its own pair) stay in step.
__device__ __forceinline__ float merge_dot_distinct(const int* ri, const float* vi, int ni,
                                                    const int* rj, const float* vj, int nj) {
  float acc = 0.f;
  int a = 0, b = 0;
  while (a < ni && b < nj) {
    const int ra = ri[a], rb = rj[b];
    const float va = vi[a], vb = vj[b];
    acc += (ra == rb) ? va * vb : 0.f;
    a += (ra <= rb);
    b += (rb <= ra);
  }
  return acc;
}

__device__ __forceinline__ void task_yy(const StepCtx& c, int local, unsigned char* sraw) {
  int(*srow)[kGramLd] = reinterpret_cast<int(*)[kGramLd]>(sraw);
  float(*sval)[kGramLd] = reinterpret_cast<float(*)[kGramLd]>(sraw + 32 * kGramLd * 4);
  int* scnt = reinterpret_cast<int*>(sraw + 2 * 32 * kGramLd * 4);
  const int nb = (c.m + 15) / 16;
  int bi = 0, rem = local;
  while (rem >= nb - bi) { rem -= nb - bi; ++bi; }
  const int bj = bi + rem;
  const int I0 = bi * 16, J0 = bj * 16;
  const bool staged = c.K <= kGramKMax;
  if (staged) {
    constexpr int kPer = 32 * kGramKMax / 256;  // list entries per thread
    int rv[kPer];
    float vv[kPer];
    int cnt = 0;
    if (threadIdx.x < 32) {
      const int l = threadIdx.x;
      const int ex = (l < 16) ? I0 + l : J0 + l - 16;
      cnt = ex < c.m ? c.ex_cnt[ex] : 0;
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int l = e / c.K, k = e - l * c.K;
      const int ex = (l < 16) ? I0 + l : J0 + l - 16;
      const size_t at = (e < 32 * c.K && ex < c.m) ? (size_t)ex * c.K + k : 0;
      rv[u] = c.ex_row[at];
      vv[u] = c.ex_val[at];
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int l = e / c.K, k = e - l * c.K;
      if (e < 32 * c.K) {
        srow[l][k] = rv[u];
        sval[l][k] = vv[u];
      }
    }
    if (threadIdx.x < 32) scnt[threadIdx.x] = cnt;
    __syncthreads();
    // Merge the repeats inside each list (adjacent, the lists being ordered):
    // one list per wave at a time; each run's first entry takes the run's
    // values summed in order and moves to its rank among the runs.  A wave's
    // reads all complete before its writes (its LDS accesses run in order).
    const int lane = lane_id(), w = wave_id();
    for (int l = w; l < 32; l += 4) {
      const int n = scnt[l];
      const int k = lane;
      const int r = k < n ? srow[l][k] : -1;
      const bool head = k < n && (k == 0 || srow[l][k - 1] != r);
      float sum = 0.f;
      if (head)
        for (int k2 = k; k2 < n && srow[l][k2] == r; ++k2) sum += sval[l][k2];
      const unsigned long long heads = __ballot(head);
      const int pos = __popcll(heads & ((1ull << k) - 1ull));
      asm volatile("" ::: "memory");
      if (head) {
        srow[l][pos] = r;
        sval[l][pos] = sum;
      }
      if (lane == 0) scnt[l] = __popcll(heads);
    }
    __syncthreads();
  }
  const int li = threadIdx.x >> 4, lj = threadIdx.x & 15;
  const int i = I0 + li, j = J0 + lj;
  if (i >= c.m || j >= c.m || i > j) return;
  float acc;
  if (staged)
    acc = merge_dot_distinct(srow[li], sval[li], scnt[li], srow[16 + lj], sval[16 + lj],
                             scnt[16 + lj]);
  else
    acc = merge_dot(c.ex_row + (size_t)i * c.K, c.ex_val + (size_t)i * c.K, c.ex_cnt[i],
                    c.ex_row + (size_t)j * c.K, c.ex_val + (size_t)j * c.K, c.ex_cnt[j]);
  float* yy = c.NP + 3 * c.m;  // the Y^T Y block of NP (row stride 4m)
  yy[(size_t)i * 4 * c.m + j] = acc;
  yy[(size_t)j * 4 * c.m + i] = acc;
}

// ----------------------------------------------------------------- scalars
// One wave per example: c1 = h^T Q h (from the partials of launch 1),
// c2 = h^T W^T y = (U h)^T (V^T y), (Y^T Y)_ii (from prep), then
//   squared:   loss = c1 - 2 c2 + (Y^T Y)_ii (= M_ii, Appendix A step 6), a = 2, b = -2
//   spherical: loss = -log(c2^2 + eps) + log(c1 + D eps), a = 2/(c1 + D eps),
//              b = -2 c2 / (c2^2 + eps), cs = b / a (the scatter weight)
//   shifted:   u_c = c2 + t_i + eps, S = c1 + 2 eps n_i + D eps^2,
//              loss = log S - 2 log|u_c|, a = 2/S, b = -2/u_c, cs = b / a
// and the row a (U h)^T of the U update's left factor; also inserts the
// example's target rows into the hash table that decides the scatter's
// owners.  Block 0 also counts the step's target pairs and resets the
// distinct-row count.
__device__ __forceinline__ void task_scalars(const StepCtx& c, int local) {
  if (local == 0 && wave_id() == 0) {
    int nnz = 0;
    for (int j = lane_id(); j < c.m; j += 64) nnz += c.ex_cnt[j];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) nnz += __shfl_xor(nnz, off);
    if (lane_id() == 0) {
      c.flags[F_NNZ] = nnz;
      c.flags[F_UNIQUE] = 0;
      hot_list(c)[0] = 0;  // the list launch 3 fills
    }
  }
  const int i = local * 4 + wave_id();
  if (i >= c.m) return;
  const int lane = lane_id(), d = c.d;
  // Record, for every target row, the smallest slot i*K + k holding it (the
  // owner of the row's scatter in launch 3), the number of slots holding it and
  // (the first kSlotCap of) those slots, and list the rows held by two or more:
  // open addressing, at most half full.
  // The list entry of a lane's first slot is written at the end of the task,
  // so that waiting for its position overlaps the rest of the work.
  int first_at = -1, first_slot = 0;
  {
    const int mask = (1 << c.hbits) - 1;
    for (int k = lane; k < c.K; k += 64) {
      const int r = c.idx[(size_t)i * c.K + k];
      if (r < 0 || (int64_t)r >= c.D) continue;
      const int slot = i * c.K + k;
      unsigned h = row_hash(r, c.hbits);
      for (int probe = 0; probe <= mask; ++probe) {
        const int prev = atomicCAS(c.hkey + h, -1, r);
        if (prev == -1 || prev == r) {
          atomicMin(c.hmin + h, slot);
          const int pos = atomicAdd(c.hcnt + h, 1);
          if (k == lane) {
            first_at = pos < kSlotCap ? (int)h * kSlotCap + pos : -1;
            first_slot = slot;
          } else if (pos < kSlotCap) {
            hslot_of(c)[(size_t)h * kSlotCap + pos] = slot;
          }
          if (pos == 1) {  // the row's second slot: list the row once
            int* mr = multi_rows(c);
            mr[1 + atomicAdd(mr, 1)] = (int)h;
          }
          break;
        }
        h = (h + 1) & mask;
      }
    }
  }
  const float c1 = example_c1(c, i);
  const float Si = (c.loss_kind == LST_LOSS_SQUARED) ? 0.f : example_S(c, i, c1);
  const float a = (c.loss_kind == LST_LOSS_SQUARED) ? 2.f : 2.f / Si;
  const float* uh = c.Z0 + (size_t)i * c.ld0 + d;
  const float* gr = c.G + (size_t)i * d;
  float* uha = c.UHa + (size_t)i * d;
  float s = 0.f;
  for (int j0 = 0; j0 < d; j0 += 512) {
    float xv[8], yv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = min(j0 + lane + 64 * u, d - 1);
      xv[u] = uh[j];
      yv[u] = gr[j];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + lane + 64 * u;
      if (j < d) {
        s += xv[u] * yv[u];
        uha[j] = a * xv[u];
      }
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  const float c2 = s;
  float L, b, cs;
  if (c.loss_kind == LST_LOSS_SQUARED) {
    L = c1 - 2.f * c2 + c.yyd[i];
    b = -2.f;
    cs = 0.f;
  } else if (c.loss_kind == LST_LOSS_SPHERICAL) {
    const float num = c2 * c2 + c.eps;
    L = -logf(num) + logf(Si);
    b = -2.f * c2 / num;
    cs = b / a;
  } else {
    const float uc = c2 + c.nt[2 * i] + c.eps;
    L = logf(Si) - 2.f * logf(fabsf(uc));
    b = -2.f / uc;
    cs = b / a;
  }
  // a h_i and b h_i: the right factor of the product that gives N H^T
  const float* hr = c.H + (size_t)i * d;
  float* ah = c.aH + (size_t)i * d;
  float* bh = c.bH + (size_t)i * d;
  for (int j0 = 0; j0 < d; j0 += 512) {
    float hv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) hv[u] = hr[min(j0 + lane + 64 * u, d - 1)];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + lane + 64 * u;
      if (j < d) {
        ah[j] = a * hv[u];
        bh[j] = b * hv[u];
      }
    }
  }
  if (first_at >= 0) hslot_of(c)[first_at] = first_slot;
  if (lane != 0) return;
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
// Neumann series Y_{k+1} = B + E Y_k converges geometrically; a block stops it
// once, in every one of its columns, a bound on the terms left out falls to
// 2^-20 of that column's largest |B| entry (kNeumannTol, neumann_done), with
// r^(k+1) / (1 - r) <= 2^-20 as the a-priori cap on k.  Otherwise (a learning rate so large that 2 lr ||H^T H|| is not
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
// Row stride (floats) of the solve's column blocks B^T, Y^T (padded).
__host__ __device__ inline int solve_lde(int mp) { return mp + 4; }

__host__ __device__ inline size_t solve_lds_bytes(int m) {
  const int mp = (m + 15) & ~15;
  const int lde = solve_lde(mp);
  // m <= 128: 1/c, B^T, Y^T twice and H^T H; m > 128: 1/c and Y^T twice (each
  // wave keeps its rows of B in registers, so that a GEMM tile fits beside)
  const size_t neumann =
      (size_t)(mp + (m <= 128 ? 3 : 2) * kSolveCols * lde + (m <= 128 ? mp * mp : 0)) *
      sizeof(float);
  const size_t gj = m <= 128 ? (size_t)m * (m + kSolveCols) * sizeof(double) : 0;
  const size_t extra = 256 * sizeof(float) + 512 * sizeof(double) + 64;  // red, colk, scalars
  return (neumann > gj ? neumann : gj) + extra;
}

#ifdef LST_TIMING
// Phase marks of the last solve blocks (latency studies only).
__device__ unsigned long long g_solve_marks[64][8];
#define LST_SMARK(k)                                                        \
  do {                                                                      \
    if (threadIdx.x == 0 && local < 64) g_solve_marks[local][k] = wall_clock64(); \
  } while (0)
#else
#define LST_SMARK(k) \
  do {               \
  } while (0)
#endif

// Relative tolerance of the Neumann series, per column of Y and in the
// infinity norm: the terms left out change no entry of a column by more than
// 2^-20 of the largest entry of that column of B.  B is itself an fp32
// product over d terms (P = U^-T H), whose rounding is of the same order or
// larger, so more terms would not make the solve more accurate.
constexpr float kNeumannTol = 9.5367431640625e-7f;  // 2^-20

// Adaptive end of the series.  Y_k - Y_{k-1} = E^k B and ||E x||_inf <= r ||x||_inf,
// so after iteration k the terms left out add at most
// ||Y_k - Y_{k-1}||_inf r / (1 - r) to any entry of a column.  At an
// iteration's end each lane passes its largest |Y_k - Y_{k-1}| (and, in the
// first iteration, |B|) over its rows of column lane & 15; neumann_post folds
// them over the lanes of the column and stores the wave's column maxima in
// LDS (two sets of slots, by iteration parity, so a wave that runs ahead never
// overwrites maxima another wave still reads); after the workgroup barrier
// neumann_done folds the four waves and returns the same answer in every
// wave.  A NaN counts as infinite, so it never ends the series early.
__device__ __forceinline__ float fold_col16(float v) {
  v = (v == v) ? v : INFINITY;
  v = fmaxf(v, __shfl_xor(v, 16));
  return fmaxf(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ void neumann_post(float* red, int it, float dl, float bl) {
  const int lane = lane_id(), wave = wave_id();
  dl = fold_col16(dl);
  bl = fold_col16(bl);
  if (lane < 16) {
    red[64 + 64 * (it & 1) + 16 * wave + lane] = dl;
    if (it == 0) red[192 + 16 * wave + lane] = bl;
  }
}
__device__ __forceinline__ bool neumann_done(const float* red, int it, float stop_k, float& bcol) {
  const int col = lane_id() & 15;
  const float* s = red + 64 + 64 * (it & 1) + col;
  const float dmax = fmaxf(fmaxf(s[0], s[16]), fmaxf(s[32], s[48]));
  if (it == 0) {
    const float* b = red + 192 + col;
    bcol = fmaxf(fmaxf(b[0], b[16]), fmaxf(b[32], b[48]));
  }
  return __all(dmax * stop_k <= kNeumannTol * bcol);
}

// The Neumann iterations for m > 128 (m % 4 == 0, 16-byte aligned rows of
// H^T H): H^T H (up to 1 MB) does not fit in LDS and is read from memory each
// iteration by every solve block, where it stays L2-resident.  Wave w owns the
// 16-row blocks w, w + 4, ... (RBW of them; a block past the last runs on a
// clamped row, branch-free, and is never stored).  The A fragments are loaded
// NB - 1 k slices ahead of the MFMAs that use them and the stream runs on
// across iteration boundaries (H^T H does not change), so its latency is paid
// once; only the B fragment, read from Y_k in LDS, waits for the barrier that
// ends an iteration.  Columns k >= m of H^T H are read at a clamped position:
// they meet rows of Y_k that are zero.  Returns the buffer holding the result.
//
// r = ||E||_inf is formed from the absolute row sums of H^T H that the first
// iteration accumulates from the fragments it multiplies (every block
// streams all of H^T H in the same order, so all find the same r).  With r
// known the series is capped (r^(k+1) / (1 - r) <= 2^-20) and the adaptive
// stop applies; r >= 1/2 (or not finite) ends it at once, and the caller
// then runs Gauss-Jordan instead.
constexpr int kNeumannMaxIters = 64;

// The iteration cap for r (as many iterations as the a-priori bound needs,
// at least the one already run).
__device__ __forceinline__ int neumann_cap(float r) {
  if (!(r > 0.f)) return 1;
  const float need = logf(kNeumannTol * (1.f - r)) / logf(r);
  return max(1, min(kNeumannMaxIters, (int)ceilf(need) - 1));
}

// The wave's absolute row sums (one per lane & 15 and row block, lanes that
// share a row hold the same sum after the fold) times 1/c, maximised over the
// wave's valid rows and posted to red[8 + wave]; NaN counts as infinite.
__device__ __forceinline__ void neumann_post_r(float* red, float rw) {
  rw = (rw == rw) ? rw : INFINITY;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) rw = fmaxf(rw, __shfl_xor(rw, off));
  if (lane_id() == 0) red[8 + wave_id()] = rw;
}
__device__ __forceinline__ float neumann_read_r(const float* red) {
  return fmaxf(fmaxf(red[8], red[9]), fmaxf(red[10], red[11]));
}
__device__ __forceinline__ float row_abs_fold(float v) {
  v += __shfl_xor(v, 16);
  return v + __shfl_xor(v, 32);
}

template <int RBW>
__device__ __forceinline__ float* neumann_mem(const float* __restrict__ HH, int ldh, int m, int mp,
                                              int LDE, const float* cinv, float* Yo, float* Yn,
                                              float* red, float& r) {
  constexpr int NB = 3;
  const int lane = lane_id(), wave = __builtin_amdgcn_readfirstlane(wave_id());
  const int nsl = mp / 16, nrb = mp / 16;
  const int kl = 4 * (lane >> 4);
  // B's entries of the wave's rows (Y_0 = B), kept in registers
  floatx4 bv[RBW];
#pragma unroll
  for (int t = 0; t < RBW; ++t) {
    const int row = min(wave + 4 * t, nrb - 1) * 16 + kl;
    bv[t] = *reinterpret_cast<const floatx4*>(Yo + (lane & 15) * LDE + row);
  }
  unsigned rofs[RBW];
#pragma unroll
  for (int t = 0; t < RBW; ++t)
    rofs[t] = (unsigned)min((wave + 4 * t) * 16 + (lane & 15), m - 1) * (unsigned)ldh;
  floatx4 fa[NB][RBW];
  auto load = [&](floatx4(&f)[RBW], int sl) {
    const unsigned ko = (unsigned)min(sl * 16 + kl, m - 4);
#pragma unroll
    for (int t = 0; t < RBW; ++t) f[t] = *reinterpret_cast<const floatx4*>(HH + (rofs[t] + ko));
  };
  int lsl = 0;  // slice of the next load
#pragma unroll
  for (int j = 0; j + 1 < NB; ++j) {
    load(fa[j], lsl);
    lsl = (lsl + 1 == nsl) ? 0 : lsl + 1;
  }
  floatx4 acc[RBW];
#pragma unroll
  for (int t = 0; t < RBW; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int yl = (lane & 15) * LDE + kl;
  int total = kNeumannMaxIters * nsl;  // capped once r is known, cut short at convergence
  int sl = 0;               // slice of the next MFMAs
  int it = 0;               // iterations completed
  floatx4 prev[RBW];        // diag(1/c) (H^T H) Y_{k-1} of the wave's rows (Y_0 = B: zero)
  float rs[RBW];            // first iteration: absolute row sums of the wave's rows (partial)
  float bcol = 0.f, stop_k = 0.f;
#pragma unroll
  for (int t = 0; t < RBW; ++t) {
    prev[t] = floatx4{0.f, 0.f, 0.f, 0.f};
    rs[t] = 0.f;
  }
  for (int g0 = 0; g0 < total; g0 += NB) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      // the loads run unconditionally (past the end they re-read H^T H), so
      // the buffers need no copies between unrolled steps
      load(fa[(j + NB - 1) % NB], lsl);
      lsl = (lsl + 1 == nsl) ? 0 : lsl + 1;
      if (g0 + j < total) {
        const floatx4 fb = *reinterpret_cast<const floatx4*>(Yo + yl + sl * 16);
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int t = 0; t < RBW; ++t)
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[j][t][q], fb[q], acc[t], 0, 0, 0);
        if (it == 0 && sl * 16 + kl < m) {
#pragma unroll
          for (int t = 0; t < RBW; ++t)
            rs[t] += (fabsf(fa[j][t][0]) + fabsf(fa[j][t][1])) +
                     (fabsf(fa[j][t][2]) + fabsf(fa[j][t][3]));
        }
        if (++sl == nsl) {
          // Y_{k+1} rows of the wave's blocks
          sl = 0;
          floatx4 cv[RBW];
#pragma unroll
          for (int t = 0; t < RBW; ++t)
            cv[t] = *reinterpret_cast<const floatx4*>(cinv + min(wave + 4 * t, nrb - 1) * 16 + kl);
          if (it == 0) {
            float rw = 0.f;
#pragma unroll
            for (int t = 0; t < RBW; ++t) {
              const float sum = row_abs_fold(rs[t]);
              const int row = (wave + 4 * t) * 16 + (lane & 15);
              if (row < m) rw = fmaxf(rw, (sum == sum) ? sum * cinv[row] : INFINITY);
            }
            neumann_post_r(red, rw);
          }
          float dl = 0.f, bl = 0.f;
#pragma unroll
          for (int t = 0; t < RBW; ++t) {
            const int rb = wave + 4 * t;
            const floatx4 y = acc[t] * cv[t];
            if (rb < nrb) {
              *reinterpret_cast<floatx4*>(Yn + (lane & 15) * LDE + rb * 16 + kl) = bv[t] + y;
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                dl = fmaxf(dl, fabsf(y[q] - prev[t][q]));
                bl = fmaxf(bl, fabsf(bv[t][q]));
              }
            }
            prev[t] = y;
            acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
          }
          neumann_post(red, it, dl, bl);
          lds_barrier();
          float* tt = Yo;
          Yo = Yn;
          Yn = tt;
          if (it == 0) {
            r = neumann_read_r(red);
            stop_k = r / (1.f - r);
            if (!(r < 0.5f)) total = g0 + j + 1;  // the caller falls back
            else total = min(total, neumann_cap(r) * nsl);
          }
          if (neumann_done(red, it, stop_k, bcol)) total = g0 + j + 1;
          ++it;
        }
      }
    }
  }
  return Yo;
}

// neumann_mem for 256 < m <= 512: a wave owns eight 16-row blocks, taken as
// two passes of four per iteration (the same stream of H^T H rows, each row
// read once per iteration), so that the fragments in flight and the
// accumulators are those of four blocks: the kernel then needs at most 256
// VGPRs and two workgroups share a compute unit.
__device__ __forceinline__ float* neumann_mem_two_pass(const float* __restrict__ HH, int ldh, int m,
                                                       int mp, int LDE, const float* cinv,
                                                       float* Yo, float* Yn, float* red, float& r) {
  constexpr int NB = 3, RB = 4;
  const int lane = lane_id(), wave = __builtin_amdgcn_readfirstlane(wave_id());
  const int nsl = mp / 16, nrb = mp / 16;
  const int kl = 4 * (lane >> 4);
  // B's entries of the wave's rows (Y_0 = B), by pass
  floatx4 bv0[RB], bv1[RB];
  unsigned rofs0[RB], rofs1[RB];
#pragma unroll
  for (int t = 0; t < RB; ++t) {
    const int r0 = min(wave + 4 * t, nrb - 1) * 16, r1 = min(wave + 16 + 4 * t, nrb - 1) * 16;
    bv0[t] = *reinterpret_cast<const floatx4*>(Yo + (lane & 15) * LDE + r0 + kl);
    bv1[t] = *reinterpret_cast<const floatx4*>(Yo + (lane & 15) * LDE + r1 + kl);
    rofs0[t] = (unsigned)min(r0 + (lane & 15), m - 1) * (unsigned)ldh;
    rofs1[t] = (unsigned)min(r1 + (lane & 15), m - 1) * (unsigned)ldh;
  }
  floatx4 fa[NB][RB];
  auto load = [&](floatx4(&f)[RB], int sl, int ps) {
    const unsigned ko = (unsigned)min(sl * 16 + kl, m - 4);
#pragma unroll
    for (int t = 0; t < RB; ++t)
      f[t] = *reinterpret_cast<const floatx4*>(HH + ((ps ? rofs1[t] : rofs0[t]) + ko));
  };
  int lsl = 0, lps = 0;  // slice and pass of the next load
  auto advance = [&](int& a, int& b) {
    if (++a == nsl) {
      a = 0;
      b ^= 1;
    }
  };
#pragma unroll
  for (int j = 0; j + 1 < NB; ++j) {
    load(fa[j], lsl, lps);
    advance(lsl, lps);
  }
  floatx4 acc[RB];
#pragma unroll
  for (int t = 0; t < RB; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int yl = (lane & 15) * LDE + kl;
  int total = kNeumannMaxIters * 2 * nsl;  // capped once r is known, cut short at convergence
  int sl = 0, ps = 0;           // slice and pass of the next MFMAs
  int it = 0;                   // iterations completed
  floatx4 prev0[RB], prev1[RB];  // diag(1/c) (H^T H) Y_{k-1} of the wave's rows
  float rs[RB];                  // first iteration: absolute row sums of the pass's rows (partial)
  float bcol = 0.f, dl = 0.f, bl = 0.f, rw = 0.f, stop_k = 0.f;
#pragma unroll
  for (int t = 0; t < RB; ++t) {
    prev0[t] = floatx4{0.f, 0.f, 0.f, 0.f};
    prev1[t] = floatx4{0.f, 0.f, 0.f, 0.f};
    rs[t] = 0.f;
  }
  for (int g0 = 0; g0 < total; g0 += NB) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      // the loads run unconditionally (past the end they re-read H^T H)
      load(fa[(j + NB - 1) % NB], lsl, lps);
      advance(lsl, lps);
      if (g0 + j < total) {
        const floatx4 fb = *reinterpret_cast<const floatx4*>(Yo + yl + sl * 16);
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int t = 0; t < RB; ++t)
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[j][t][q], fb[q], acc[t], 0, 0, 0);
        if (it == 0 && sl * 16 + kl < m) {
#pragma unroll
          for (int t = 0; t < RB; ++t)
            rs[t] += (fabsf(fa[j][t][0]) + fabsf(fa[j][t][1])) +
                     (fabsf(fa[j][t][2]) + fabsf(fa[j][t][3]));
        }
        if (++sl == nsl) {
          // Y_{k+1} rows of the pass's blocks
          sl = 0;
          if (it == 0) {
#pragma unroll
            for (int t = 0; t < RB; ++t) {
              const float sum = row_abs_fold(rs[t]);
              const int row = (wave + 16 * ps + 4 * t) * 16 + (lane & 15);
              if (row < m) rw = fmaxf(rw, (sum == sum) ? sum * cinv[row] : INFINITY);
              rs[t] = 0.f;
            }
            if (ps) neumann_post_r(red, rw);
          }
#pragma unroll
          for (int t = 0; t < RB; ++t) {
            const int rb = wave + 16 * ps + 4 * t;
            const floatx4 cv =
                *reinterpret_cast<const floatx4*>(cinv + min(rb, nrb - 1) * 16 + kl);
            const floatx4 y = acc[t] * cv;
            const floatx4 b = ps ? bv1[t] : bv0[t];
            const floatx4 pv = ps ? prev1[t] : prev0[t];
            if (rb < nrb) {
              *reinterpret_cast<floatx4*>(Yn + (lane & 15) * LDE + rb * 16 + kl) = b + y;
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                dl = fmaxf(dl, fabsf(y[q] - pv[q]));
                bl = fmaxf(bl, fabsf(b[q]));
              }
            }
            if (ps)
              prev1[t] = y;
            else
              prev0[t] = y;
            acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
          }
          if (ps) {  // both passes done: the iteration ends
            neumann_post(red, it, dl, bl);
            lds_barrier();
            float* tt = Yo;
            Yo = Yn;
            Yn = tt;
            if (it == 0) {
              r = neumann_read_r(red);
              stop_k = r / (1.f - r);
              if (!(r < 0.5f)) total = g0 + j + 1;  // the caller falls back
              else total = min(total, neumann_cap(r) * 2 * nsl);
            }
            if (neumann_done(red, it, stop_k, bcol)) total = g0 + j + 1;
            ++it;
            dl = 0.f;
            bl = 0.f;
          }
          ps ^= 1;
        }
      }
    }
  }
  return Yo;
}

template <bool SMALL>
__device__ __forceinline__ void task_solve(const StepCtx& c, int local, unsigned char* sraw) {
  LST_SMARK(0);
  const int m = c.m, d = c.d;
  const float* HH = c.Z0 + 3 * d;
  const float* P = c.Z0 + 2 * d;
  const int ldh = c.ld0, ldp = c.ld0;
  const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
  const int mp = (m + 15) & ~15;
  const int LDE = solve_lde(mp);
  const int c0 = local * kSolveCols;
  const size_t main_bytes = solve_lds_bytes(m) - (256 * sizeof(float) + 512 * sizeof(double) + 64);
  float* red = reinterpret_cast<float*>(sraw + main_bytes);
  double* colk = reinterpret_cast<double*>(red + 256);
  int* s_int = reinterpret_cast<int*>(colk + 512);  // s_p, s_bad
  float* cinv = reinterpret_cast<float*>(sraw);        // mp: 1 / c_i = lr a_i
  float* Bt = cinv + mp;  // kSolveCols x LDE: B^T (m <= 128; above, the waves keep B)
  float* Y0 = SMALL ? Bt + kSolveCols * LDE : cinv + mp;  // kSolveCols x LDE: Y^T
  float* Y1 = Y0 + kSolveCols * LDE;
  float* Hs = Y1 + kSolveCols * LDE;                   // mp x mp: H^T H (SMALL only)

  for (int i = tid; i < mp; i += 256) cinv[i] = (i < m) ? c.lr * example_a(c, i) : 0.f;
  if (tid == 0) s_int[1] = 0;
  LST_SMARK(1);
  // r = ||E||_inf with E = diag(1/c) H^T H; the absolute row sums of H^T H
  // come as partials from the first GEMM.  For m <= 128 this block's columns
  // of P and the partials are fetched first, H^T H (into LDS) after them, and
  // r and the right-hand side are formed while H^T H is still arriving.
  // H^T H in LDS: mp rows of mp floats, the 16-byte slot s of row j stored at
  // slot s ^ (j & hsw) (bank-conflict-free reads down a column and across 16
  // rows); rows and columns beyond m are zero.
  const int hsw = (mp % 32 == 0) ? 7 : 3;  // the XOR must stay inside a row's mp/4 slots
  // m > 128 with m % 4 == 0 and 16-byte aligned rows of H^T H and P: vector
  // loads (the right-hand side and the iterations), and r is found by the
  // first iteration instead of from the partials
  const bool gvec = !SMALL && m % 4 == 0 && d % 4 == 0 && ldh % 4 == 0 &&
                    ((uintptr_t)HH & 15) == 0 && ((uintptr_t)P & 15) == 0;
  float r;
  if (SMALL) {
    // Waves 2 and 3 fetch this block's columns of P and the partial sums
    // first (plain loads, waited for by them alone), then form r and the
    // right-hand side; waves 0 and 1 move H^T H meanwhile.
    const float* zero = g_dma_zero;
    const int q4 = mp / 4;  // slots per row
    const bool vec4 = (ldh % 4 == 0) && (((uintptr_t)HH & 15) == 0) && (m % 4 == 0);
    if (!vec4) {
      for (int e0 = 0; e0 < mp * q4; e0 += 256 * 4) {
        float4 r4[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = e0 + tid + 256 * u;
          const int j = min(e / q4, m - 1), col = 4 * ((e % q4) ^ ((e / q4) & hsw));
          const float* hr = HH + (size_t)j * ldh;
          r4[u].x = hr[min(col, m - 1)];
          r4[u].y = hr[min(col + 1, m - 1)];
          r4[u].z = hr[min(col + 2, m - 1)];
          r4[u].w = hr[min(col + 3, m - 1)];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = e0 + tid + 256 * u;
          if (e < mp * q4) {
            const int j = e / q4, col = 4 * ((e % q4) ^ (j & hsw));
            const bool ok = j < m;
            float4 v;
            v.x = (ok && col < m) ? r4[u].x : 0.f;
            v.y = (ok && col + 1 < m) ? r4[u].y : 0.f;
            v.z = (ok && col + 2 < m) ? r4[u].z : 0.f;
            v.w = (ok && col + 3 < m) ? r4[u].w : 0.f;
            *reinterpret_cast<float4*>(Hs + 4 * e) = v;
          }
        }
      }
    }
    __syncthreads();  // 1 / c_i (and H^T H without DMA) visible to every wave
    if (wave == 3) {
      // Every load below is unconditional at a clamped (valid) address, so
      // all of them are in flight before the first is needed; the values are
      // masked afterwards.
      constexpr int NPV = 128 * kSolveCols / 64;   // P elements per lane for mp = 128
      constexpr int kMaxHap = 2 * (128 / 32 + 1);  // partials per row for m <= 128
      float pv[NPV], hv[2][kMaxHap];
#pragma unroll
      for (int u = 0; u < NPV; ++u) {
        const int e = lane + 64 * u;
        const int i = min(e / kSolveCols, m - 1), cc = min(c0 + e % kSolveCols, d - 1);
        pv[u] = P[(size_t)i * ldp + cc];
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int hrow = min(lane + 64 * h, m - 1);
#pragma unroll
        for (int p = 0; p < kMaxHap; ++p)
          hv[h][p] = c.hap[(size_t)hrow * c.n_hap + min(p, c.n_hap - 1)];
      }
      __builtin_amdgcn_s_barrier();  // the H^T H transfers start after these loads
      float rw = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float sabs = 0.f;
#pragma unroll
        for (int p = 0; p < kMaxHap; ++p) sabs += p < c.n_hap ? hv[h][p] : 0.f;
        const int row = lane + 64 * h;
        if (row < m) {
          const float ri = sabs * cinv[row];
          rw = (ri == ri) ? fmaxf(rw, ri) : INFINITY;
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) rw = fmaxf(rw, __shfl_xor(rw, off));
      if (lane == 0) red[3] = rw;
      // B^T = -(P^T_blk) diag(1/c)^T and Y0 = B^T (used when the series converges)
#pragma unroll
      for (int u = 0; u < NPV; ++u) {
        const int e = lane + 64 * u, i = e / kSolveCols, cc = e % kSolveCols;
        if (i < mp) {
          const float v = (i < m && c0 + cc < d) ? -pv[u] * cinv[i] : 0.f;
          Bt[cc * LDE + i] = v;
          Y0[cc * LDE + i] = v;
        }
      }
    } else {
      __builtin_amdgcn_s_barrier();
      if (vec4) {
        // 16-byte DMA by waves 0-2: instruction q fills slots [64 q, 64 q + 64)
        const unsigned hh = lds_u32(Hs);
        for (int q = wave; q < mp * q4 / 64; q += 3) {
          const int e = 64 * q + lane;
          const int j = e / q4, col = 4 * ((e % q4) ^ (j & hsw));
          dma16((j < m && col < m) ? HH + (size_t)j * ldh + col : zero, hh + 1024u * q);
        }
      }
      if (lane == 0) red[wave] = 0.f;
    }
    LST_SMARK(2);
    wait_vm_le(0);  // H^T H has landed
    lds_barrier();
    r = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  } else if (gvec) {
    // r comes from the first iteration, which streams every row of H^T H
    LST_SMARK(2);
    r = 0.f;
  } else {
    LST_SMARK(2);
    // The partials, m x nh floats stored row after row (m <= 512 and nh <= 34: two
    // per tile column over the m columns of H^T H), are
    // read as one flat array, every load issued before the first is used (each
    // wave's load covers consecutive addresses), then summed row by row through
    // LDS in chunks of 64 rows (Y1 is free until the iterations start).
    constexpr int kChunkRows = 64, kChunks = 4;  // per pass; two passes cover 512 rows
    constexpr int kPerChunk = (kChunkRows * 34 + 255) / 256;
    const int nh = c.n_hap;
    float* stage = Y1;
    float rmax = 0.f;
    for (int pass = 0; pass < 2; ++pass) {
    float hv[kChunks][kPerChunk];
#pragma unroll
    for (int cq = 0; cq < kChunks; ++cq) {
      const int ch = pass * kChunks + cq;
      const int nflat = max(0, min(kChunkRows, m - ch * kChunkRows)) * nh;
      const float* base = c.hap + (size_t)ch * kChunkRows * nh;
#pragma unroll
      for (int u = 0; u < kPerChunk; ++u) {
        const int e = tid + 256 * u;
        hv[cq][u] = e < nflat ? base[e] : 0.f;
      }
    }
#pragma unroll
    for (int cq = 0; cq < kChunks; ++cq) {
      const int ch = pass * kChunks + cq;
      if (ch * kChunkRows < m) {
        const int nflat = min(kChunkRows, m - ch * kChunkRows) * nh;
#pragma unroll
        for (int u = 0; u < kPerChunk; ++u) {
          const int e = tid + 256 * u;
          if (e < nflat) stage[e] = hv[cq][u];
        }
        __syncthreads();
        const int i = ch * kChunkRows + tid;
        if (tid < kChunkRows && i < m) {
          float sabs = 0.f;
          for (int p = 0; p < nh; ++p) sabs += stage[tid * nh + p];
          const float ri = sabs * cinv[i];
          rmax = (ri == ri) ? fmaxf(rmax, ri) : INFINITY;
        }
        __syncthreads();
      }
    }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) rmax = fmaxf(rmax, __shfl_xor(rmax, off));
    if (lane == 0) red[wave] = rmax;
    __syncthreads();
    r = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  }
  LST_SMARK(3);

  if (gvec || r < 0.5f) {
    if (gvec) {
      // Y0 = B = -(P^T_blk) diag(1/c)^T: 16-byte loads, slot e = row
      // e / 4, columns c0 + 4 (e % 4) ... + 3 (all in or all out of range)
      const int nq = 4 * mp;
      for (int e0 = 0; e0 < nq; e0 += 256 * 8) {
        floatx4 pv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = e0 + tid + 256 * u;
          const int i = min(e >> 2, m - 1), col = min(c0 + 4 * (e & 3), d - 4);
          pv[u] = *reinterpret_cast<const floatx4*>(P + (size_t)i * ldp + col);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = e0 + tid + 256 * u;
          if (e < nq) {
            const int i = e >> 2, cq = 4 * (e & 3);
            const bool ok = i < m && c0 + cq < d;
#pragma unroll
            for (int v = 0; v < 4; ++v) Y0[(cq + v) * LDE + i] = ok ? -pv[u][v] * cinv[i] : 0.f;
          }
        }
      }
    } else if (!SMALL) {
      // Y0 = B = -(P^T_blk) diag(1/c)^T.
      for (int e0 = 0; e0 < kSolveCols * mp; e0 += 256 * 8) {
        float pv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = e0 + tid + 256 * u;
          const int i = min(e / kSolveCols, m - 1), cc = min(c0 + e % kSolveCols, d - 1);
          pv[u] = P[(size_t)i * ldp + cc];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = e0 + tid + 256 * u;
          if (e < kSolveCols * mp) {
            const int i = e / kSolveCols, cc = e - i * kSolveCols;
            Y0[cc * LDE + i] = (i < m && c0 + cc < d) ? -pv[u] * cinv[i] : 0.f;
          }
        }
      }
    }
    int iters = gvec ? kNeumannMaxIters : 0;  // gvec: capped once r is known
    const float stop_k = r / (1.f - r);
    if (!gvec && r > 0.f) {
      // at most: r^(k+1) / (1 - r) <= tol (a bound that holds before any
      // iteration); the series usually ends sooner (neumann_done)
      const float need = logf(kNeumannTol * (1.f - r)) / logf(r);
      iters = (int)ceilf(need) - 1;
      if (iters < 0) iters = 0;
      if (iters > kNeumannMaxIters) iters = kNeumannMaxIters;
    }
    if (!SMALL) __syncthreads();
    LST_SMARK(4);
#ifdef LST_TIMING
    if (threadIdx.x == 0 && local < 64) g_solve_marks[local][7] = (unsigned long long)iters;
#endif
    // Y_{k+1} = B + diag(1/c) (H^T H) Y_k.  Wave w owns the 16-row blocks
    // w, w + 4, ...; the B fragment of a k slice is shared by them.
    constexpr int RBW = SMALL ? 2 : 8;
    const int nrb = mp / 16;
    float* Yo = Y0;
    float* Yn = Y1;
    // One 16-wide k slice: B fragment (shared by the wave's row blocks) and
    // the A fragments of its row blocks.
    auto frag = [&](const float* Yk, int kk, float4& fb, float4 (&fa)[RBW]) {
      const int k = kk + 4 * (lane >> 4);
      fb = *reinterpret_cast<const float4*>(Yk + (lane & 15) * LDE + k);
#pragma unroll
      for (int t = 0; t < RBW; ++t) {
        const int arow = min((wave + 4 * t) * 16, mp - 16) + (lane & 15);
        if (SMALL) {
          fa[t] = *reinterpret_cast<const float4*>(Hs + arow * mp + 4 * ((k >> 2) ^ (arow & hsw)));
        } else {
          const float* hr = HH + (size_t)min(arow, m - 1) * ldh;
          const float x0 = hr[min(k, m - 1)], x1 = hr[min(k + 1, m - 1)];
          const float x2 = hr[min(k + 2, m - 1)], x3 = hr[min(k + 3, m - 1)];
          const bool ok = arow < m;
          fa[t].x = (ok && k < m) ? x0 : 0.f;
          fa[t].y = (ok && k + 1 < m) ? x1 : 0.f;
          fa[t].z = (ok && k + 2 < m) ? x2 : 0.f;
          fa[t].w = (ok && k + 3 < m) ? x3 : 0.f;
        }
      }
    };
    if constexpr (SMALL) {
      // m <= 128: at most 8 slices.  The fragment reads go through inline asm
      // one slice ahead of the MFMAs they feed, each slice waiting only for
      // the reads issued a slice earlier (left to the compiler, that wait
      // lands after the next slice's reads and every slice pays the LDS
      // latency); per-lane offsets of every slice are computed once, slices
      // past the last re-read it.
      const int nsl = mp / 16;
      unsigned oa[RBW][8];
#pragma unroll
      for (int t = 0; t < RBW; ++t) {
        const int arow = min((wave + 4 * t) * 16, mp - 16) + (lane & 15);
#pragma unroll
        for (int sl = 0; sl < 8; ++sl) {
          const int k = min(sl, nsl - 1) * 16 + 4 * (lane >> 4);
          oa[t][sl] = lds_u32(Hs + arow * mp + 4 * ((k >> 2) ^ (arow & hsw)));
        }
      }
      const unsigned yl = 4u * (unsigned)((lane & 15) * LDE + 4 * (lane >> 4));
      floatx4 prev[RBW];  // diag(1/c) (H^T H) Y_{k-1} of the wave's rows (Y_0 = B: zero)
      float bcol = 0.f;
#pragma unroll
      for (int t = 0; t < RBW; ++t) prev[t] = floatx4{0.f, 0.f, 0.f, 0.f};
      for (int it = 0; it < iters; ++it) {
        floatx4 acc[RBW];
#pragma unroll
        for (int t = 0; t < RBW; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
        const unsigned yb = lds_u32(Yo) + yl;
        floatx4 fb[2], fa[2][RBW];
        auto rd = [&](int b, int sl) {
          static_assert(RBW == 2, "three reads per slice");
          asm volatile("ds_read_b128 %0, %3\n\tds_read_b128 %1, %4\n\tds_read_b128 %2, %5"
                       : "=&v"(fb[b]), "=&v"(fa[b][0]), "=&v"(fa[b][1])
                       : "v"(yb + 64u * (unsigned)min(sl, nsl - 1)), "v"(oa[0][sl]), "v"(oa[1][sl]));
        };
        auto mm = [&](int b) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int t = 0; t < RBW; ++t)
              acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[b][t][q], fb[b][q], acc[t], 0, 0, 0);
        };
        rd(0, 0);
#pragma unroll
        for (int sl = 0; sl < 8; ++sl) {
          if (sl < nsl) {
            const int b = sl & 1;
            if (sl + 1 < 8) {
              rd(b ^ 1, sl + 1);
              asm volatile("s_waitcnt lgkmcnt(3)" : "+v"(fb[b]), "+v"(fa[b][0]), "+v"(fa[b][1]));
            } else {
              asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fb[b]), "+v"(fa[b][0]), "+v"(fa[b][1]));
            }
            mm(b);
          }
        }
        // the reads of slice nsl (a re-read of the last one) may be outstanding
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        const int col = lane & 15;
        float dl = 0.f, bl = 0.f;
#pragma unroll
        for (int t = 0; t < RBW; ++t) {
          const int rb = wave + 4 * t;
          if (rb >= nrb) break;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = rb * 16 + 4 * (lane >> 4) + q;
            const float bv = Bt[col * LDE + row], y = acc[t][q] * cinv[row];
            Yn[col * LDE + row] = bv + y;
            dl = fmaxf(dl, fabsf(y - prev[t][q]));
            bl = fmaxf(bl, fabsf(bv));
            prev[t][q] = y;
          }
        }
        neumann_post(red, it, dl, bl);
        __syncthreads();
        float* tt = Yo;
        Yo = Yn;
        Yn = tt;
        if (neumann_done(red, it, stop_k, bcol)) break;
      }
    } else if (gvec) {
      Yo = (nrb <= 16) ? neumann_mem<4>(HH, ldh, m, mp, LDE, cinv, Yo, Yn, red, r)
                       : neumann_mem_two_pass(HH, ldh, m, mp, LDE, cinv, Yo, Yn, red, r);
    } else {
    floatx4 prev[RBW];  // diag(1/c) (H^T H) Y_{k-1} of the wave's rows (Y_0 = B: zero)
    floatx4 bvr[RBW];   // B's entries of the wave's rows, read from Y_0 = B
    float bcol = 0.f;
#pragma unroll
    for (int t = 0; t < RBW; ++t) {
      prev[t] = floatx4{0.f, 0.f, 0.f, 0.f};
      const int rb = min(wave + 4 * t, nrb - 1);
#pragma unroll
      for (int q = 0; q < 4; ++q) bvr[t][q] = Yo[(lane & 15) * LDE + rb * 16 + 4 * (lane >> 4) + q];
    }
    for (int it = 0; it < iters; ++it) {
      const int col = lane & 15;
      const int nsl = mp / 16;
      float dl = 0.f, bl = 0.f;
      // the wave's row blocks in passes of four (fragments and accumulators of
      // four blocks at a time keep the kernel within 256 VGPRs)
#pragma unroll
      for (int ps = 0; ps < RBW / 4; ++ps) {
        floatx4 acc[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
        constexpr int NB = 3;
        float4 fb[NB], fa[NB][4];
        auto frag4 = [&](int kk, float4& fbv, float4 (&fav)[4]) {
          const int k = kk + 4 * (lane >> 4);
          fbv = *reinterpret_cast<const float4*>(Yo + (lane & 15) * LDE + k);
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int arow = min((wave + 4 * (4 * ps + t)) * 16, mp - 16) + (lane & 15);
            const float* hr = HH + (size_t)min(arow, m - 1) * ldh;
            const float x0 = hr[min(k, m - 1)], x1 = hr[min(k + 1, m - 1)];
            const float x2 = hr[min(k + 2, m - 1)], x3 = hr[min(k + 3, m - 1)];
            const bool ok = arow < m;
            fav[t].x = (ok && k < m) ? x0 : 0.f;
            fav[t].y = (ok && k + 1 < m) ? x1 : 0.f;
            fav[t].z = (ok && k + 2 < m) ? x2 : 0.f;
            fav[t].w = (ok && k + 3 < m) ? x3 : 0.f;
          }
        };
        // Every wave multiplies all four row blocks of the pass (a block past
        // the last reads a clamped one and is never stored): the waves run side
        // by side, so the extra MFMAs cost no time and the loop has no branches.
        auto mma = [&](const float4& b, const float4 (&av)[4]) {
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[t].x, b.x, acc[t], 0, 0, 0);
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[t].y, b.y, acc[t], 0, 0, 0);
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[t].z, b.z, acc[t], 0, 0, 0);
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[t].w, b.w, acc[t], 0, 0, 0);
          }
        };
        // Three fragment buffers rotate: slice s + 1 is read while slice s is
        // multiplied, into the buffer of slice s - 2 (whose MFMAs are done).
        frag4(0, fb[0], fa[0]);
        for (int sl = 0; sl < nsl; sl += NB) {
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            if (sl + j >= nsl) break;
            frag4(min(sl + j + 1, nsl - 1) * 16, fb[(j + 1) % NB], fa[(j + 1) % NB]);
            mma(fb[j], fa[j]);
          }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int T = 4 * ps + t;
          const int rb = wave + 4 * T;
          if (rb >= nrb) break;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = rb * 16 + 4 * (lane >> 4) + q;
            const float bv = bvr[T][q], y = acc[t][q] * cinv[row];
            Yn[col * LDE + row] = bv + y;
            dl = fmaxf(dl, fabsf(y - prev[T][q]));
            bl = fmaxf(bl, fabsf(bv));
            prev[T][q] = y;
          }
        }
      }
      neumann_post(red, it, dl, bl);
      __syncthreads();
      float* tt = Yo;
      Yo = Yn;
      Yn = tt;
      if (neumann_done(red, it, stop_k, bcol)) break;
    }
    }
    LST_SMARK(5);
    if (!gvec || r < 0.5f) {  // gvec: r from the first iteration decides only now
      for (int e = tid; e < kSolveCols * m; e += 256) {
        const int i = e / kSolveCols, cc = e - i * kSolveCols;
        if (c0 + cc < d) c.X[(size_t)i * d + c0 + cc] = Yo[cc * LDE + i];
      }
      LST_SMARK(6);
      return;
    }
  }

  // Fallback: Gauss-Jordan on [S | P^T_blk], S = H^T H - diag(c).  c_i moves
  // to colk first: the fp64 matrix overwrites the buffers that hold 1/c_i
  // (and the LDS copy of H^T H, whose transfer must have landed first).  The
  // pivot threshold scales with max |S_ij|.
  const int ncol = m + kSolveCols;
  if (SMALL) wait_vm_le(0);
  float amax = 0.f;
  for (int e = tid; e < m * m; e += 256) {
    const int i = e / m, j = e - i * m;
    const float ci = 1.f / cinv[i];
    amax = fmaxf(amax, fabsf(HH[(size_t)i * ldh + j] - (i == j ? ci : 0.f)));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  __syncthreads();  // every wave has read red[0..3] (r) above
  if (lane == 0) red[4 + wave] = amax;
  for (int i = tid; i < m; i += 256) colk[i] = 1.0 / (double)cinv[i];
  __syncthreads();
  const float smax = fmaxf(fmaxf(red[4], red[5]), fmaxf(red[6], red[7]));
  const double tiny = 1e-13 * (double)smax;
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
// in increasing j.  Only the slot (example i, pair k; index i K + k) with the
// smallest index of its row, read from the hash table, does the row's work, so
// every row is written once and in a fixed order.  Each slot records in own[]
// the row it owns (or -1); launch 4 clears the hash slots from that record.
//
// A row held by one slot is written kScatterRows at a time, with all their
// rows of X and V in flight before the first is added.  A row held by several
// slots reads their list from its hash entry, sorts it into slot order and
// adds the examples' rows of X in that order, 16 in flight; a row held by
// more than kSlotCap slots searches the examples' sorted target lists instead
// (kScatterBatch rows in flight).
constexpr int kScatterBatch = 4;
constexpr int kScatterRows = 8;

// The value of x in lane src (the same src in every lane): a scalar read of
// the lane, not a cross-lane shuffle through LDS.
__device__ __forceinline__ int from_lane(int x, int src) {
  return __builtin_amdgcn_readlane(x, src);
}
__device__ __forceinline__ float from_lane(float x, int src) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), src));
}

// Ascending sort of one int per lane across the wave (bitonic network).
__device__ __forceinline__ int wave_sort_asc(int x) {
  const int lane = lane_id();
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int o = __shfl_xor(x, j);
      const bool up = (lane & k) == 0, low = (lane & j) == 0;
      x = (low == up) ? min(x, o) : max(x, o);
    }
  return x;
}

// acc (columns cg + 256 q + 4 lane, q < NQ) += w_l X[j_l, :] over the lanes l
// set in bal, in lane order; with d % 4 == 0, B rows of X in flight at a time
// (a row of a common target, in nearly every example, would otherwise pay the
// memory latency once per example).
template <int NQ, int B>
__device__ __forceinline__ void add_x_rows(const StepCtx& c, int cg, unsigned long long bal,
                                           float w_l, int j_l, float4 (&acc)[4]) {
  const int lane = lane_id();
  if (c.d % 4 == 0) {
    while (bal) {
      float w[B];
      float4 x[B][NQ];
      bool on[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        on[u] = bal != 0;
        const int src = on[u] ? __ffsll((long long)bal) - 1 : 0;
        bal &= bal - 1;
        w[u] = from_lane(w_l, src);
        const int j = from_lane(j_l, src);
        const float* xr = c.X + (size_t)j * c.d;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const int col = cg + q * 256 + lane * 4;
          if (on[u] && col < c.d) x[u][q] = *reinterpret_cast<const float4*>(xr + col);
        }
      }
#pragma unroll
      for (int u = 0; u < B; ++u) {
        if (!on[u]) break;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const int col = cg + q * 256 + lane * 4;
          if (col >= c.d) continue;
          acc[q].x += w[u] * x[u][q].x; acc[q].y += w[u] * x[u][q].y;
          acc[q].z += w[u] * x[u][q].z; acc[q].w += w[u] * x[u][q].w;
        }
      }
    }
    return;
  }
  while (bal) {
    const int src = __ffsll((long long)bal) - 1;
    bal &= bal - 1;
    const float w = from_lane(w_l, src);
    const float* xr = c.X + (size_t)from_lane(j_l, src) * c.d;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int col = cg + q * 256 + lane * 4;
      if (col >= c.d) continue;
      acc[q].x += w * xr[col];
      if (col + 1 < c.d) acc[q].y += w * xr[col + 1];
      if (col + 2 < c.d) acc[q].z += w * xr[col + 2];
      if (col + 3 < c.d) acc[q].w += w * xr[col + 3];
    }
  }
}

// The row r held by cnt slots, owned by slot e (hash entry h): the whole wave.
__device__ __forceinline__ void scatter_row(const StepCtx& c, int r, int h, int cnt, int e) {
  const int lane = lane_id();
  const bool one_hot = c.loss_kind != LST_LOSS_SQUARED;
  const bool listed = cnt <= kSlotCap;
  // listed: lane l < cnt holds the l-th slot of the row in slot order; the
  // first lane of each example's run carries that example and its c_j
  float cj = 0.f;
  int jl = 0;
  unsigned long long lead = 0;
  if (listed) {
    const bool in = lane < cnt;
    const int sl = wave_sort_asc(in ? hslot_of(c)[(size_t)h * kSlotCap + lane] : 0x7fffffff);
    jl = in ? sl / c.K : -1;
    const float v = (in && !one_hot) ? c.val[sl] : 0.f;
    const int jp = __shfl_up(jl, 1);
    const bool leader = in && (lane == 0 || jp != jl);
    // the values of a run, added in slot order by its first lane
    float sum = v;
    bool more = leader;
    for (int t = 1; t < 64 && __ballot(more) != 0; ++t) {
      const float vt = __shfl_down(v, t);
      const int jt = __shfl_down(jl, t);
      more = more && lane + t < cnt && jt == jl;
      if (more) sum += vt;
    }
    if (leader) cj = one_hot ? c.cs[jl] : -sum;
    lead = __ballot(leader);
  }
  const int i = e / c.K;
  // columns in groups of 512 (listed: 16 rows of X in flight) or 1024 (the
  // search, done once per group)
  const int gcols = listed ? 512 : 1024;
  for (int cg = 0; cg < c.d; cg += gcols) {
    float4 acc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (listed) {
      add_x_rows<2, 16>(c, cg, lead, cj, jl, acc);
    } else {
      // examples i, i + 1, ... (i holds the row's smallest slot), 64 at a
      // time, until all cnt slots have been met
      int met = 0;
      for (int j0 = i; j0 < c.m && met < cnt; j0 += 64) {
        const int j = j0 + lane;
        float cw = 0.f;
        bool found = false;
        int nrun = 0;
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
            ++nrun;
            found = true;
          }
          cw = one_hot ? c.cs[j] : -sum;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) nrun += __shfl_xor(nrun, off);
        met += nrun;
        add_x_rows<4, kScatterBatch>(c, cg, __ballot(found), cw, j, acc);
      }
    }
    float* vr = c.V + (size_t)r * c.d;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int col = cg + q * 256 + lane * 4;
      if (col >= c.d || col >= cg + gcols) continue;
      if (c.d % 4 == 0) {
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

// Rows held by one slot each (d % 4 == 0): V[r_l] += w_l X[i_l] for the lanes
// l set in bal, kScatterRows rows at a time, 512 columns at a time.  The sum
// has one term, written as the several-slot rows write theirs (0 + w x, then
// added to V), so a row gives the same bits either way.
__device__ __forceinline__ void scatter_single(const StepCtx& c, unsigned long long bal, int r_l,
                                               int i_l, float w_l) {
  const int lane = lane_id();
  for (int cg = 0; cg < c.d; cg += 512) {
    unsigned long long b = bal;
    while (b) {
      float* vr[kScatterRows];
      float4 x[kScatterRows][2], v[kScatterRows][2];
      int src[kScatterRows];
      bool on[kScatterRows];
#pragma unroll
      for (int u = 0; u < kScatterRows; ++u) {
        on[u] = b != 0;
        src[u] = on[u] ? __ffsll((long long)b) - 1 : 0;
        b &= b - 1;
        const int ru = from_lane(r_l, src[u]), iu = from_lane(i_l, src[u]);
        const float* xr = c.X + (size_t)iu * c.d;
        vr[u] = c.V + (size_t)ru * c.d;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int col = cg + q * 256 + lane * 4;
          if (on[u] && col < c.d) {
            x[u][q] = *reinterpret_cast<const float4*>(xr + col);
            v[u][q] = *reinterpret_cast<const float4*>(vr[u] + col);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kScatterRows; ++u) {
        if (!on[u]) break;
        // the weight's load (issued before the rows') has landed by now
        const float w = from_lane(w_l, src[u]);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int col = cg + q * 256 + lane * 4;
          if (col >= c.d) continue;
          float4 o = v[u][q];
          o.x += 0.f + w * x[u][q].x; o.y += 0.f + w * x[u][q].y;
          o.z += 0.f + w * x[u][q].z; o.w += 0.f + w * x[u][q].w;
          *reinterpret_cast<float4*>(vr[u] + col) = o;
        }
      }
    }
  }
}

__host__ __device__ inline int scatter_lookup_blocks(const StepCtx& c) {
  const int spw = scatter_slots_per_wave(c.m * c.K);
  return (c.m * c.K + 4 * spw - 1) / (4 * spw);
}
// Waves that write the rows held by several slots (taken from the list in
// turn: wave g the rows g, g + kEntryWaves, ...).
constexpr int kEntryWaves = 2048;
__host__ __device__ inline int scatter_entry_blocks(const StepCtx& c) {
  return scatter_slots_per_wave(c.m * c.K) == 1 ? 0 : kEntryWaves / 4;
}

// Blocks [0, scatter_lookup_blocks) take scatter_slots_per_wave(m K)
// consecutive slots per wave and look them up together; a slot that owns its
// row records it in own[], and the rows held by one slot are written here.
// The kEntryWaves waves after them write the rows held by several slots,
// spread evenly over the waves by the list launch 2 made of them (their owner
// slots cluster in the first examples when targets repeat, so the lookup
// waves would get them unevenly).  With one slot per wave (small steps) there
// are no entry waves and the wave writes the row its slot owns, whatever the
// row's count.  With HOT the rows held by c.hot_min or more slots are listed
// for launch 4 instead.
template <bool HOT>
__device__ __forceinline__ void task_scatter(const StepCtx& c, int local) {
  const int lane = lane_id();
  const int spw = scatter_slots_per_wave(c.m * c.K);
  const int nlook = scatter_lookup_blocks(c);
  const bool vec = c.d % 4 == 0;
  // launches 1 and 2 set the error flag: read it while the slots are looked up
  const int err = c.flags[F_ERR];
  int r = -1, cnt = 0, e = 0, h = 0;
  bool mine = false;  // this lane's row is written by scatter_row below
  if (local >= nlook) {
    if (err) return;
    const int* mr = multi_rows(c);
    const int q = ((local - nlook) * 4 + wave_id()) + lane * kEntryWaves;
    if (q < mr[0]) {
      h = mr[1 + q];
      r = c.hkey[h];
      cnt = c.hcnt[h];
      e = c.hmin[h];
      mine = true;
    }
  } else {
    e = (local * 4 + wave_id()) * spw + lane;
    bool owner = false;
    if (lane < spw && e < c.m * c.K) {
      r = c.idx[e];
      if (r >= 0 && (int64_t)r < c.D) {
        const int mask = (1 << c.hbits) - 1;
        unsigned hh = row_hash(r, c.hbits);
        int probe = 0;
        while (probe <= mask && c.hkey[hh] != r) {
          hh = (hh + 1) & mask;
          ++probe;
        }
        owner = probe <= mask && c.hmin[hh] == e;
        if (owner) cnt = c.hcnt[hh];
        h = (int)hh;
      }
      c.own[e] = owner ? r : -1;
    }
    if (err) return;
    const bool single = owner && cnt == 1 && vec;
    const unsigned long long one = __ballot(single);
    if (one) {
      const int i = e / c.K;
      const float w = single ? (c.loss_kind != LST_LOSS_SQUARED ? c.cs[i] : -c.val[e]) : 0.f;
      scatter_single(c, one, r, i, w);
    }
    // with one slot per wave every owned row is written here; otherwise the
    // rows held by one slot of an unaligned V (the entry waves take the rest)
    mine = owner && !single && (spw == 1 || cnt == 1);
  }
  if constexpr (HOT) {
    if (mine && cnt >= c.hot_min) {
      int* hot = hot_list(c);
      hot[1 + atomicAdd(hot, 1)] = r;
      mine = false;
    }
  }
  unsigned long long several = __ballot(mine);
  while (several) {
    const int src = __ffsll((long long)several) - 1;
    several &= several - 1;
    scatter_row(c, from_lane(r, src), from_lane(h, src), from_lane(cnt, src), from_lane(e, src));
  }
}

// Launch 4: the scatter of the rows launch 3 listed as hot (held by so many
// slots that one wave would add them one example at a time), by the nb clear
// blocks.  Work item q = (listed row q / nch, 256-column chunk q % nch);
// block b takes the items b, b + nb, ...  Its four waves split the examples
// into fixed quarters, each adds c_j X_j over its quarter in example order,
// and the four partial sums are added in wave order before the row is
// written once.
constexpr size_t kHotLdsBytes = 3 * 64 * sizeof(float4);

__device__ __forceinline__ void scatter_hot(const StepCtx& c, int local, int nb,
                                            unsigned char* sraw) {
  float4(*part)[64] = reinterpret_cast<float4(*)[64]>(sraw);  // 3 x 64 partial sums
  if (c.flags[F_ERR]) return;
  const int* hot = hot_list(c);
  const int nch = (c.d + 255) / 256;
  const int items = hot[0] * nch;
  const int wave = wave_id(), lane = lane_id();
  const bool one_hot = c.loss_kind != LST_LOSS_SQUARED;
  const bool vec = (c.d % 4 == 0);
  const int span = (c.m + 3) / 4, jb = wave * span, je = min(c.m, jb + span);
  for (int q = local; q < items; q += nb) {
    const int r = hot[1 + q / nch];
    const int col = (q % nch) * 256 + 4 * lane;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j0 = jb; j0 < je; j0 += 64) {
      const int j = j0 + lane;
      float cj = 0.f;
      bool found = false;
      if (j < je) {
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
      // four examples at a time: their rows of X are in flight together
      while (bal) {
        float w[4];
        float4 x[4];
        bool on[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          on[u] = bal != 0;
          const int src = on[u] ? __ffsll((long long)bal) - 1 : 0;
          bal &= bal - 1;
          w[u] = from_lane(cj, src);
          const float* xr = c.X + (size_t)(j0 + src) * c.d;
          x[u] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (on[u] && col < c.d) {
            if (vec) {
              x[u] = *reinterpret_cast<const float4*>(xr + col);
            } else {
              x[u].x = xr[col];
              if (col + 1 < c.d) x[u].y = xr[col + 1];
              if (col + 2 < c.d) x[u].z = xr[col + 2];
              if (col + 3 < c.d) x[u].w = xr[col + 3];
            }
          }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (!on[u]) break;
          acc.x += w[u] * x[u].x; acc.y += w[u] * x[u].y;
          acc.z += w[u] * x[u].z; acc.w += w[u] * x[u].w;
        }
      }
    }
    if (wave > 0) part[wave - 1][lane] = acc;
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        const float4 o = part[p][lane];
        acc.x += o.x; acc.y += o.y; acc.z += o.z; acc.w += o.w;
      }
      float* vr = c.V + (size_t)r * c.d;
      if (col < c.d) vr[col] += acc.x;
      if (col + 1 < c.d) vr[col + 1] += acc.y;
      if (col + 2 < c.d) vr[col + 2] += acc.z;
      if (col + 3 < c.d) vr[col + 3] += acc.w;
    }
    __syncthreads();  // part[] is free for the next item
  }
}

// Launch 4: empty the hash slots of the rows this step touched (found from
// own[]) and count the distinct rows (one atomic per block); with HOT the
// blocks first scatter the hot rows (the longer work, independent of the hash).
template <bool HOT>
__device__ __forceinline__ void task_clear(const StepCtx& c, int local, unsigned char* sraw) {
  if constexpr (HOT) scatter_hot(c, local, (c.m * c.K + 255) / 256, sraw);
  __shared__ int s_cnt[4];
  const int t = local * 256 + threadIdx.x;
  const int r = (t < c.m * c.K) ? c.own[t] : -1;
  if (r >= 0) {
    const int mask = (1 << c.hbits) - 1;
    unsigned h = row_hash(r, c.hbits);
    for (int probe = 0; probe <= mask; ++probe) {
      if (c.hkey[h] == r) {
        c.hkey[h] = -1;
        c.hmin[h] = 0x7fffffff;
        c.hcnt[h] = 0;
        break;
      }
      h = (h + 1) & mask;
    }
  }
  const unsigned long long bal = __ballot(r >= 0);
  if (lane_id() == 0) s_cnt[wave_id()] = __popcll(bal);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int n = s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
    if (n > 0) atomicAdd(c.flags + F_UNIQUE, n);
  }
}

// -------------------------------------------------------------- the kernel
// Dynamic LDS a step launch may use (of the 160 KB of a compute unit).
constexpr size_t kStepLdsMax = 160 * 1024 - 1024;

#ifdef LST_TIMING
// Per-block (start, end) wall clock of the last launches, for latency studies.
__device__ unsigned long long g_step_times[4][8192][3];
#endif

// What each launch kind of the step runs: task kinds, GEMM operand layouts
// (V_*) and GEMM epilogues.  The kernel of a launch kind compiles only these,
// which keeps its code small enough for the instruction cache.
struct LaunchMasks {
  unsigned tasks, vars, epis, tiles;
  bool hot;  // launch 3 lists the hot rows, launch 4's clear blocks scatter them
};
constexpr LaunchMasks kLaunchMasks[8] = {
    {0u, 0u, 0u, 0u},
    {(1u << TK_GEMM) | (1u << TK_TARGETS), V_NT, (1u << EPI_STORE) | (1u << EPX_ROWSUMS), TILE32},
    {(1u << TK_GEMM) | (1u << TK_SOLVE) | (1u << TK_YY) | (1u << TK_SCALARS), V_NN | V_NT,
     (1u << EPI_STORE) | (1u << EPI_STORE_T), TILE32},
    {(1u << TK_GEMM) | (1u << TK_SCATTER), V_NN, 1u << EPI_GRADT, TILE32},
    {(1u << TK_GEMM) | (1u << TK_CLEAR), V_TN,
     (1u << EPI_SYM) | (1u << EPI_STORE) | (1u << EPX_LATE_SKIP), TILE32 | TILE64},
    // the d x d products of the Appendix C stabilisation
    {1u << TK_GEMM, V_NT | V_NN, 1u << EPI_SCALED, TILE32},
    // launches 3 and 4 of a step whose hot rows are scattered in launch 4
    {(1u << TK_GEMM) | (1u << TK_SCATTER), V_NN, 1u << EPI_GRADT, TILE32, true},
    {(1u << TK_GEMM) | (1u << TK_CLEAR), V_TN,
     (1u << EPI_SYM) | (1u << EPI_STORE) | (1u << EPX_LATE_SKIP), TILE32 | TILE64, true},
};

// The kernels of launches 1 and 2 built for m > 128 also compile 64 x 64
// tiles: their products are long in K there (d up to 1024), and 64 x 64 tiles
// fetch half the bytes per output of 32 x 32 ones (launch 1 uses them when
// they alone fill the chip, launch 2 always).  Launch 2's also compiles the
// symmetric epilogue: there C1 = H^T Q H is computed on its upper-triangle
// tiles and mirrored, and C2^T is not computed at all (N is formed from C2).  The launch-3 kernels built for
// m > 128 compile the EPI_GRADN epilogue: there T takes N H^T from the formed
// m x m matrix N instead of the interleaved 2m x 2m view of NP, a quarter of
// the multiply-adds.
constexpr LaunchMasks launch_masks(int lk, bool small) {
  LaunchMasks M = kLaunchMasks[lk];
  if (!small && (lk == 1 || lk == 2)) M.tiles |= TILE64;
  if (!small && lk == 2) M.epis |= 1u << EPI_SYM;  // C1 = H^T H^ on its upper triangle
  if (!small && (lk == 3 || lk == 6)) M.epis |= 1u << EPI_GRADN;
  return M;
}

template <bool SMALLM, int W, int LK>
__device__ __forceinline__ void run_task(const StepCtx& c, const StepLaunch& L, int t, int local,
                                         unsigned char* sraw) {
  constexpr LaunchMasks M = launch_masks(LK, SMALLM);
  const int kind = L.kind[t];
  if constexpr ((M.tasks >> TK_GEMM) & 1u) {
    if (kind == TK_GEMM) {
      if constexpr (!((M.epis >> EPX_LATE_SKIP) & 1u)) {
        if (L.gemm.skip_if && *L.gemm.skip_if) return;
      }
      panel_tile<M.tiles, W, M.vars, M.epis>(L.gemm, local, reinterpret_cast<float*>(sraw));
      return;
    }
  }
  if constexpr ((M.tasks >> TK_TARGETS) & 1u) {
    if (kind == TK_TARGETS) {
      if (c.d % 4 == 0)
        task_targets<true>(c, local, sraw);
      else
        task_targets<false>(c, local, sraw);
      return;
    }
  }
  if constexpr ((M.tasks >> TK_YY) & 1u) {
    if (kind == TK_YY) { task_yy(c, local, sraw); return; }
  }
  if constexpr ((M.tasks >> TK_SCALARS) & 1u) {
    if (kind == TK_SCALARS) { task_scalars(c, local); return; }
  }
  if constexpr ((M.tasks >> TK_SOLVE) & 1u) {
    if (kind == TK_SOLVE) { task_solve<SMALLM>(c, local, sraw); return; }
  }
  if constexpr ((M.tasks >> TK_SCATTER) & 1u) {
    if (kind == TK_SCATTER) { task_scatter<M.hot>(c, local); return; }
  }
  if constexpr ((M.tasks >> TK_CLEAR) & 1u) {
    if (kind == TK_CLEAR) { task_clear<M.hot>(c, local, sraw); return; }
  }
}

template <bool SMALLM, int W, int LK>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(SMALLM || LK != 2 ? 1 : 2)))
void step_kernel(StepCtx c, StepLaunch L) {
  extern __shared__ __attribute__((aligned(16))) unsigned char sraw[];
  // A GEMM block's decoding reads the task table, then the GEMM header, then
  // its problem's descriptor: each a kernel-argument line that the one before
  // selects.  One word of every line it may read is requested up front, so the
  // lines arrive in one round trip rather than one after another (c2 -0.5 us
  // per step; the longer tiles of the m > 128 kernels gain nothing from it).
  if constexpr (SMALLM && ((launch_masks(LK, SMALLM).tasks >> TK_GEMM) & 1u)) {
    asm volatile("" ::"s"(L.ntask), "s"(L.gemm.np), "s"(L.gemm.x.e1), "s"(L.gemm.x.lde1),
                 "s"(L.gemm.p[0].M), "s"(L.gemm.p[0].A.ld[0]), "s"(L.gemm.p[0].C),
                 "s"(L.gemm.p[1].M), "s"(L.gemm.p[1].A.ld[0]), "s"(L.gemm.p[1].C),
                 "s"(L.gemm.p[2].M), "s"(L.gemm.p[2].A.ld[0]), "s"(L.gemm.p[2].C));
  }
  const int blk = blockIdx.x;
  int t = 0;
  while (t + 1 < L.ntask && blk >= L.begin[t + 1]) ++t;
  const int local = blk - L.begin[t];
#ifdef LST_TIMING
  const unsigned long long t0 = wall_clock64();
#endif
  run_task<SMALLM, W, LK>(c, L, t, local, sraw);
#ifdef LST_TIMING
  __syncthreads();
  if (threadIdx.x == 0 && blk < 8192) {
    // kind | GEMM problem + 1 << 4 | HW_ID << 8 | XCC_ID << 40
    unsigned long long tag = (unsigned long long)L.kind[t];
    if (L.kind[t] == TK_GEMM) {
      const int tt = xcd_tile(local, L.gemm.total_tiles);
      int q = 0;
      while (q + 1 < L.gemm.np && tt >= L.gemm.tile_begins[q + 1]) ++q;
      tag |= (unsigned long long)(q + 1) << 4;
    }
    tag |= (unsigned long long)(unsigned)__builtin_amdgcn_s_getreg((31 << 11) | 4) << 8;
    tag |= (unsigned long long)((unsigned)__builtin_amdgcn_s_getreg((3 << 11) | 20) & 15u) << 40;
    g_step_times[L.timing_slot & 3][blk][0] = t0;
    g_step_times[L.timing_slot & 3][blk][1] = wall_clock64();
    g_step_times[L.timing_slot & 3][blk][2] = tag;
  }
#endif
}

// ------------------------------------------------------------------- host
static size_t lds_of(int kind, int stages, int m, int K) {
  switch (kind) {
    case TK_GEMM: return (size_t)stages * kPanelStageBytes;
    case TK_TARGETS: return targets_lds_bytes(K);
    case TK_YY: return 2 * 32 * kGramLd * 4 + 32 * 4;
    case TK_SOLVE: return solve_lds_bytes(m);
    default: return 0;
  }
}

static int tiles_of(GemmBatch& b) {
  int total = 0;
  for (int q = 0; q < b.np; ++q) {
    GemmProblem& p = b.p[q];
    if (p.tile == 0) p.tile = 32;
    p.tiles_m = (p.M + p.tile - 1) / p.tile;
    p.tiles_n = (p.N + p.tile - 1) / p.tile;
    p.tile_begin = total;
    b.tile_begins[q] = total;
    if (p.ksplit < 1) p.ksplit = 1;
    if (p.epi == EPI_SYM)
      total += p.tiles_m * (p.tiles_m + 1) / 2;
    else
      total += p.tiles_m * p.tiles_n * (p.epi == EPI_PARTIAL ? p.ksplit : 1);
  }
  b.total_tiles = total;
  b.tile_begins[b.np] = total;
  return total;
}

int step_task_blocks(int kind, const StepCtx& c) {
  switch (kind) {
    case TK_TARGETS: return (c.m + 3) / 4;
    case TK_YY: { const int nb = (c.m + 15) / 16; return nb * (nb + 1) / 2; }
    case TK_SCALARS: return (c.m + 3) / 4;
    case TK_SOLVE: return (c.d + kSolveCols - 1) / kSolveCols;
    case TK_SCATTER: return scatter_lookup_blocks(c) + scatter_entry_blocks(c);
    case TK_CLEAR: return (c.m * c.K + 255) / 256;
    default: return 0;
  }
}

static int vmat_vec16(const VMat& v) {
  if (!v.vec) return 0;
  for (int b = 0; b < v.nb; ++b)
    if (v.ld[b] % 4 != 0 || ((uintptr_t)v.p[b] & 15) != 0) return 0;
  return 1;
}

int gemm_batch_vec16(const GemmBatch& b) {
  for (int q = 0; q < b.np; ++q) {
    const GemmProblem& p = b.p[q];
    if (!vmat_vec16(p.A) || !vmat_vec16(p.B)) return 0;
    const bool kc = p.a_kc || p.b_kc;
    if (kc && p.K % 4 != 0) return 0;
  }
  return 1;
}

template <bool SMALLM, int W, int LK>
static const void* kfn() {
  return reinterpret_cast<const void*>(step_kernel<SMALLM, W, LK>);
}

// The kernel built for (launch kind, m <= 128, 16-byte DMA); nullptr for a
// combination that is not built.
// Launch kinds with a kernel of their own for m > 128 (64 x 64 tiles, the
// solve's memory-streamed iterations, the T product from N); the others run
// the m <= 128 kernel at every m.
constexpr bool has_large_kernel(int lk) { return lk == 1 || lk == 2 || lk == 3 || lk == 6; }

static const void* step_kernel_for(int lk, bool small, int w16) {
  switch (lk) {
    case 1:
      if (small) return w16 ? kfn<true, 4, 1>() : kfn<true, 1, 1>();
      return w16 ? kfn<false, 4, 1>() : kfn<false, 1, 1>();
    case 2:
      if (small) return w16 ? kfn<true, 4, 2>() : kfn<true, 1, 2>();
      return w16 ? kfn<false, 4, 2>() : kfn<false, 1, 2>();
    case 3:
      if (small) return w16 ? kfn<true, 4, 3>() : kfn<true, 1, 3>();
      return w16 ? kfn<false, 4, 3>() : kfn<false, 1, 3>();
    case 4: return w16 ? kfn<true, 4, 4>() : kfn<true, 1, 4>();
    case 5: return w16 ? kfn<true, 4, 5>() : kfn<true, 1, 5>();
    case 6:
      if (small) return w16 ? kfn<true, 4, 6>() : kfn<true, 1, 6>();
      return w16 ? kfn<false, 4, 6>() : kfn<false, 1, 6>();
    case 7: return w16 ? kfn<true, 4, 7>() : kfn<true, 1, 7>();
    default: return nullptr;
  }
}

// One thread per element of N; row i of NP holds [C1 | C2 | C2^T | Y^T Y]_i.
// N_ij = a_i a_j C1_ij + a_i b_j C2_ij + b_i a_j C2_ji + b_i b_j (Y^T Y)_ij from
// NP = [C1 | C2 | . | Y^T Y] (C2^T is read as C2 transposed): 32 x 32 tiles of N,
// the C2_ji tile through LDS so that every read is along a row.
__global__ __launch_bounds__(256) void form_n_kernel(const float* __restrict__ NP,
                                                     const float* __restrict__ a,
                                                     const float* __restrict__ b, int m,
                                                     float* __restrict__ N, int ldn) {
  __shared__ float T[32][33];
  const int I0 = blockIdx.y * 32, J0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 8 rows of 32 per pass
  const size_t ldp = (size_t)4 * m;
  float c2t[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {  // C2[J0 + r][I0 + tx] for r = ty + 8 u
    const int r = J0 + ty + 8 * u, col = I0 + tx;
    c2t[u] = (r < m && col < m) ? NP[(size_t)r * ldp + m + col] : 0.f;
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) T[ty + 8 * u][tx] = c2t[u];
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = I0 + ty + 8 * u, j = J0 + tx;
    if (i >= m || j >= ldn) continue;
    float v = 0.f;
    if (j < m) {
      const float* r = NP + (size_t)i * ldp;
      const float aj = a[j], bj = b[j];
      v = a[i] * (r[j] * aj + r[m + j] * bj) + b[i] * (T[tx][ty + 8 * u] * aj + r[3 * m + j] * bj);
    }
    N[(size_t)i * ldn + j] = v;
  }
}

hipError_t form_n(const float* NP, const float* a, const float* b, int m, float* N, int ldn,
                  hipStream_t s) {
  if (m <= 0 || ldn < m) return hipErrorInvalidValue;
  hipLaunchKernelGGL(form_n_kernel, dim3((ldn + 31) / 32, (m + 31) / 32), dim3(256), 0, s, NP, a,
                     b, m, N, ldn);
  return hipGetLastError();
}

hipError_t step_launch(const StepCtx& c, StepLaunch& L, int stages, hipStream_t s,
                       hipEvent_t ev0, hipEvent_t ev1) {
  if (L.lk < 1 || L.lk > 7) return hipErrorInvalidValue;
  if (stages < 2 || (size_t)stages * kPanelStageBytes > kStepLdsMax) return hipErrorInvalidValue;
  // the kernel that runs and the masks checked below must be the same build
  const bool small = c.m <= 128 || !has_large_kernel(L.lk);
  const LaunchMasks M = launch_masks(L.lk, small);
  L.gemm.stages = stages;
  L.gemm.timing_slot = L.timing_slot;
  size_t lds = 0;
  int total = 0;
  int w16 = 1;
  for (int t = 0; t < L.ntask; ++t) {
    if (!((M.tasks >> L.kind[t]) & 1u)) return hipErrorInvalidValue;
    L.begin[t] = total;
    int n = 0;
    if (L.kind[t] == TK_GEMM) {
      // the extras belong to a batch of one problem
      const GemmExtras& x = L.gemm.x;
      const bool rowsums = (x.dotp != nullptr || x.absp != nullptr);
      const bool extras = rowsums || x.e1 || x.e2 || x.s1 || x.s2 || x.g;
      if (extras && L.gemm.np != 1) return hipErrorInvalidValue;
      for (int q = 0; q < L.gemm.np; ++q) {
        const GemmProblem& p = L.gemm.p[q];
        const unsigned tbit = (p.tile == 64) ? TILE64 : (p.tile == 32 || p.tile == 0) ? TILE32 : 0u;
        if (!(M.vars & problem_variant(p)) || !((M.epis >> p.epi) & 1u) || !(M.tiles & tbit) ||
            (rowsums && (p.epi != EPI_STORE || !((M.epis >> EPX_ROWSUMS) & 1u))))
          return hipErrorInvalidValue;
      }
      n = tiles_of(L.gemm);
      w16 = gemm_batch_vec16(L.gemm);
    } else {
      n = step_task_blocks(L.kind[t], c);
    }
    size_t b = lds_of(L.kind[t], stages, c.m, c.K);
    if (M.hot && L.kind[t] == TK_CLEAR && b < kHotLdsBytes) b = kHotLdsBytes;
    if (b > lds) lds = b;
    total += n;
  }
  L.begin[L.ntask] = total;
  if (total == 0) {
    // nothing to run: the events still mark this (empty) launch on the stream
    if (ev0 && ev1 && (hipEventRecord(ev0, s) != hipSuccess || hipEventRecord(ev1, s) != hipSuccess))
      return hipErrorUnknown;
    return hipSuccess;
  }
  if (lds > kStepLdsMax) return hipErrorInvalidValue;

  const void* fn = step_kernel_for(L.lk, small, w16);
  if (!fn) return hipErrorInvalidValue;
  StepCtx ca = c;
  StepLaunch la = L;
  void* args[] = {&ca, &la};
  if (ev0 && ev1) return hipExtLaunchKernel(fn, dim3(total), dim3(256), args, lds, s, ev0, ev1, 0);
  return hipLaunchKernel(fn, dim3(total), dim3(256), args, lds, s);
}

size_t solve_workspace_floats(int m_max, int d) {
  if (m_max <= 128) return 0;
  const size_t blocks = (size_t)(d + kSolveCols - 1) / kSolveCols;
  return blocks * (size_t)m_max * (m_max + kSolveCols);
}

hipError_t configure_kernels() {
  for (int lk = 1; lk <= 7; ++lk)
    for (int small = 0; small < 2; ++small)
      for (int w16 = 0; w16 < 2; ++w16) {
        const void* k = step_kernel_for(lk, small != 0, w16);
        if (!k) continue;
        const hipError_t e =
            hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kStepLdsMax);
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
extern "C" int lst_debug_target_marks(unsigned long long* out) {
  return hipMemcpyFromSymbol(out, HIP_SYMBOL(g_target_marks), sizeof(g_target_marks)) == hipSuccess
             ? 0 : -5;
}
extern "C" int lst_debug_solve_marks(unsigned long long* out) {
  return hipMemcpyFromSymbol(out, HIP_SYMBOL(g_solve_marks), sizeof(g_solve_marks)) == hipSuccess
             ? 0 : -5;
}
extern "C" int lst_debug_gemm_marks(unsigned long long* out) {
  return hipMemcpyFromSymbol(out, HIP_SYMBOL(g_gemm_marks), sizeof(g_gemm_marks)) == hipSuccess
             ? 0 : -5;
}
#endif

__global__ __launch_bounds__(1024) void compact_owned_kernel(const int* own, int n, int* out,
                                                             int* count) {
  __shared__ int s_n;
  if (threadIdx.x == 0) s_n = 0;
  __syncthreads();
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int r = own[e];
    if (r >= 0) out[atomicAdd(&s_n, 1)] = r;
  }
  __syncthreads();
  if (threadIdx.x == 0) *count = s_n;
}

hipError_t compact_owned(const int* own, int n, int* out, int* count, hipStream_t s) {
  hipLaunchKernelGGL(compact_owned_kernel, dim3(1), dim3(1024), 0, s, own, n, out, count);
  return hipGetLastError();
}

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
