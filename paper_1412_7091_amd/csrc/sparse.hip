// The K-sparse side of the step: target validation and ordering, the target
// Gram matrix Y^T Y, the gather V^T Y and the scatter into the touched rows of V.
//
// Section 2.1 represents a target as K (index, value) pairs; sections 3.2 and
// Appendix A (steps 2 and 9) touch only the rows of V that appear in the
// minibatch's targets: V^T Y reads K rows per example and the V update writes
// each distinct row once.  Every reduction here runs in a fixed order, so the
// step is bitwise reproducible without float atomics.
#include "lst_internal.h"

namespace lst {

static constexpr unsigned long long kNoKey = ~0ull;

// One workgroup per example: validate the K pairs, sort them by (row, slot) and
// emit the global sort keys.  K <= 1024.
__global__ __launch_bounds__(256) void prep_examples_kernel(const int32_t* __restrict__ idx,
                                                            const float* __restrict__ val, int K,
                                                            int64_t D, int one_hot, SparseWs ws,
                                                            int* flags) {
  __shared__ unsigned long long keys[1024];
  __shared__ int cnt;
  const int i = blockIdx.x;
  if (threadIdx.x == 0) cnt = 0;
  __syncthreads();
  for (int k = threadIdx.x; k < K; k += blockDim.x) {
    const int r = idx[(size_t)i * K + k];
    const bool valid = (r >= 0) && ((int64_t)r < D);
    const bool bad = (r < -1) || ((int64_t)r >= D) || (one_hot && r == -1);
    if (bad) atomicCAS(flags + F_ERR, 0, LST_EINDEX);
    const unsigned slot = (unsigned)(i * K + k);
    const unsigned long long key =
        valid ? (((unsigned long long)(unsigned)r << 32) | slot) : kNoKey;
    keys[k] = key;
    ws.keys[(size_t)i * K + k] = key;
    if (valid) atomicAdd(&cnt, 1);
  }
  __syncthreads();
  // rank sort: keys of valid pairs are distinct (the slot is part of the key)
  for (int k = threadIdx.x; k < K; k += blockDim.x) {
    const unsigned long long key = keys[k];
    int rank = 0;
    for (int k2 = 0; k2 < K; ++k2) {
      const unsigned long long o = keys[k2];
      rank += (o < key) || (o == key && k2 < k);
    }
    const bool valid = key != kNoKey;
    ws.ex_row[(size_t)i * K + rank] = valid ? (int)(key >> 32) : -1;
    const int slot = (int)(key & 0xffffffffu);
    ws.ex_val[(size_t)i * K + rank] = valid ? (one_hot ? 1.f : val[slot]) : 0.f;
  }
  if (threadIdx.x == 0) ws.ex_cnt[i] = cnt;
}

hipError_t prep_examples(const int32_t* idx, const float* val, int m, int K, int64_t D,
                         int one_hot, SparseWs ws, int* flags, hipStream_t s) {
  hipLaunchKernelGGL(prep_examples_kernel, dim3(m), dim3(256), 0, s, idx, val, K, D, one_hot, ws,
                     flags);
  return hipGetLastError();
}

// One workgroup: bitonic sort of all m*K keys in LDS (n <= 16384), then the
// distinct rows and the first sorted position of each.
constexpr int kSortMax = 16384;

__global__ __launch_bounds__(1024) void prep_global_sort_kernel(int n, SparseWs ws, int* flags) {
  __shared__ unsigned long long key[kSortMax];
  __shared__ int scan[1024];
  int np2 = 1;
  while (np2 < n) np2 <<= 1;
  for (int e = threadIdx.x; e < np2; e += blockDim.x) key[e] = (e < n) ? ws.keys[e] : kNoKey;
  __syncthreads();
  for (int size = 2; size <= np2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int e = threadIdx.x; e < (np2 >> 1); e += blockDim.x) {
        const int lo = 2 * e - (e & (stride - 1));
        const int hi = lo + stride;
        const bool up = ((lo & size) == 0);
        const unsigned long long a = key[lo], b = key[hi];
        if ((a > b) == up) {
          key[lo] = b;
          key[hi] = a;
        }
      }
      __syncthreads();
    }
  }
  // number of valid keys and segment starts; each thread owns a contiguous chunk
  __shared__ int s_nnz;
  if (threadIdx.x == 0) s_nnz = np2;
  __syncthreads();
  const int per = (np2 + blockDim.x - 1) / blockDim.x;
  const int e0 = threadIdx.x * per, e1 = min(np2, e0 + per);
  int local = 0;
  for (int e = e0; e < e1; ++e) {
    const unsigned long long k = key[e];
    if (k == kNoKey) {
      if (e == 0 || key[e - 1] != kNoKey) s_nnz = e;  // first unused key (valid keys sort first)
      break;
    }
    const bool start = (e == 0) || ((key[e - 1] >> 32) != (k >> 32));
    local += start;
  }
  scan[threadIdx.x] = local;
  __syncthreads();
  // inclusive scan over the per-thread counts (Hillis-Steele)
  for (int off = 1; off < (int)blockDim.x; off <<= 1) {
    const int v = (threadIdx.x >= (unsigned)off) ? scan[threadIdx.x - off] : 0;
    __syncthreads();
    scan[threadIdx.x] += v;
    __syncthreads();
  }
  int seg = scan[threadIdx.x] - local;  // exclusive prefix
  for (int e = e0; e < e1; ++e) {
    const unsigned long long k = key[e];
    if (k == kNoKey) break;
    const bool start = (e == 0) || ((key[e - 1] >> 32) != (k >> 32));
    if (start) {
      ws.seg_row[seg] = (int)(k >> 32);
      ws.seg_beg[seg] = e;
      ++seg;
    }
    ws.srt_slot[e] = (int)(k & 0xffffffffu);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int u = scan[blockDim.x - 1];
    ws.seg_beg[u] = s_nnz;
    flags[F_NNZ] = s_nnz;
    flags[F_UNIQUE] = u;
  }
}

hipError_t prep_global_sort(int m, int K, SparseWs ws, int* flags, hipStream_t s) {
  const int n = m * K;
  if (n > kSortMax) return hipErrorInvalidValue;
  hipLaunchKernelGGL(prep_global_sort_kernel, dim3(1), dim3(1024), 0, s, n, ws, flags);
  return hipGetLastError();
}

// Y^T Y: one thread per (i, j), i <= j, merging the two sorted target lists;
// a row that repeats inside an example contributes the sum of its values.
__global__ __launch_bounds__(256) void target_gram_kernel(int m, int K, SparseWs ws) {
  const int i = blockIdx.y * 16 + (threadIdx.x >> 4);
  const int j = blockIdx.x * 16 + (threadIdx.x & 15);
  if (i >= m || j >= m || i > j) return;
  const int* ri = ws.ex_row + (size_t)i * K;
  const int* rj = ws.ex_row + (size_t)j * K;
  const float* vi = ws.ex_val + (size_t)i * K;
  const float* vj = ws.ex_val + (size_t)j * K;
  const int ni = ws.ex_cnt[i], nj = ws.ex_cnt[j];
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
  ws.yy[(size_t)i * m + j] = acc;
  ws.yy[(size_t)j * m + i] = acc;
}

hipError_t prep_target_gram(int m, int K, SparseWs ws, hipStream_t s) {
  const int t = (m + 15) / 16;
  hipLaunchKernelGGL(target_gram_kernel, dim3(t, t), dim3(256), 0, s, m, K, ws);
  return hipGetLastError();
}

// G[i, c] = sum_k w_ik V[idx_ik, c]: one wave per (example, 256-column chunk),
// four consecutive columns per lane; K rows of V in flight at once.
template <bool VEC>
__global__ __launch_bounds__(64) void gather_kernel(const float* __restrict__ V, int64_t D, int d,
                                                    const int32_t* __restrict__ idx,
                                                    const float* __restrict__ val, int K,
                                                    int one_hot, float* __restrict__ G, int ldg) {
  const int i = blockIdx.x;
  const int c = blockIdx.y * 256 + threadIdx.x * 4;
  if (c >= d) return;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  const int32_t* ix = idx + (size_t)i * K;
  const float* vx = val + (size_t)i * K;
  for (int k = 0; k < K; ++k) {
    const int r = ix[k];
    if (r < 0 || (int64_t)r >= D) continue;
    const float w = one_hot ? 1.f : vx[k];
    const float* row = V + (size_t)r * d + c;
    if (VEC) {
      const float4 x = *reinterpret_cast<const float4*>(row);
      acc.x += w * x.x; acc.y += w * x.y; acc.z += w * x.z; acc.w += w * x.w;
    } else {
      acc.x += w * row[0];
      if (c + 1 < d) acc.y += w * row[1];
      if (c + 2 < d) acc.z += w * row[2];
      if (c + 3 < d) acc.w += w * row[3];
    }
  }
  float* out = G + (size_t)i * ldg + c;
  if (VEC) {
    *reinterpret_cast<float4*>(out) = acc;
  } else {
    out[0] = acc.x;
    if (c + 1 < d) out[1] = acc.y;
    if (c + 2 < d) out[2] = acc.z;
    if (c + 3 < d) out[3] = acc.w;
  }
}

hipError_t gather_rows(const float* V, int64_t D, int d, const int32_t* idx, const float* val,
                       int m, int K, int one_hot, float* G, int ldg, hipStream_t s) {
  dim3 grid(m, (d + 255) / 256), block(64);
  const bool vec = (d % 4 == 0) && (ldg % 4 == 0) && (((uintptr_t)V & 15) == 0) &&
                   (((uintptr_t)G & 15) == 0);
  if (vec)
    hipLaunchKernelGGL(gather_kernel<true>, grid, block, 0, s, V, D, d, idx, val, K, one_hot, G,
                       ldg);
  else
    hipLaunchKernelGGL(gather_kernel<false>, grid, block, 0, s, V, D, d, idx, val, K, one_hot, G,
                       ldg);
  return hipGetLastError();
}

// V[r, c] += sum over the sorted pairs of row r of coef * X[i, c]: one wave per
// (distinct row, 256-column chunk).  Blocks beyond the number of distinct rows
// of this step return at once.
template <bool VEC>
__global__ __launch_bounds__(64) void scatter_kernel(float* __restrict__ V, int d,
                                                     const float* __restrict__ X, int ldx,
                                                     const float* __restrict__ val,
                                                     const float* __restrict__ cs, int K,
                                                     SparseWs ws, const int* flags) {
  if (flags[F_ERR]) return;
  const int sg = blockIdx.x;
  if (sg >= flags[F_UNIQUE]) return;
  const int c = blockIdx.y * 256 + threadIdx.x * 4;
  if (c >= d) return;
  const int r = ws.seg_row[sg];
  const int p0 = ws.seg_beg[sg], p1 = ws.seg_beg[sg + 1];
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int p = p0; p < p1; ++p) {
    const int slot = ws.srt_slot[p];
    const int i = slot / K;
    const float w = cs ? cs[i] : -val[slot];
    const float* x = X + (size_t)i * ldx + c;
    if (VEC) {
      const float4 v = *reinterpret_cast<const float4*>(x);
      acc.x += w * v.x; acc.y += w * v.y; acc.z += w * v.z; acc.w += w * v.w;
    } else {
      acc.x += w * x[0];
      if (c + 1 < d) acc.y += w * x[1];
      if (c + 2 < d) acc.z += w * x[2];
      if (c + 3 < d) acc.w += w * x[3];
    }
  }
  float* row = V + (size_t)r * d + c;
  if (VEC) {
    float4 v = *reinterpret_cast<float4*>(row);
    v.x += acc.x; v.y += acc.y; v.z += acc.z; v.w += acc.w;
    *reinterpret_cast<float4*>(row) = v;
  } else {
    row[0] += acc.x;
    if (c + 1 < d) row[1] += acc.y;
    if (c + 2 < d) row[2] += acc.z;
    if (c + 3 < d) row[3] += acc.w;
  }
}

hipError_t scatter_rows(float* V, int d, const float* X, int ldx, const float* val,
                        const float* cs, int m, int K, SparseWs ws, const int* flags,
                        hipStream_t s) {
  dim3 grid(m * K, (d + 255) / 256), block(64);
  const bool vec = (d % 4 == 0) && (ldx % 4 == 0) && (((uintptr_t)V & 15) == 0) &&
                   (((uintptr_t)X & 15) == 0);
  if (vec)
    hipLaunchKernelGGL(scatter_kernel<true>, grid, block, 0, s, V, d, X, ldx, val, cs, K, ws,
                       flags);
  else
    hipLaunchKernelGGL(scatter_kernel<false>, grid, block, 0, s, V, d, X, ldx, val, cs, K, ws,
                       flags);
  return hipGetLastError();
}

}  // namespace lst
