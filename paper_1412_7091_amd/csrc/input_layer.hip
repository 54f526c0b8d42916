// The sparse input layer of section 2.2 ("the easy part"): a K-sparse input
// x (K (index, value) pairs per example; index -1 unused) enters the first
// hidden layer through a D_in x d matrix W_in, so that
//   forward: A[i, :] = sum_k v_ik W_in[u_ik, :]           (O(K d) per example)
//   update:  W_in[r, :] -= lr * sum_{(i,k): u_ik = r} v_ik dA[i, :]
// touch only the rows the minibatch refers to.  The update writes each row
// once, from the wave of the row's first slot (in (example, pair) order),
// which adds the contributions of all its slots in that order: deterministic,
// with no atomics on W_in.  A hash table (row -> first slot, number of slots)
// built by a pass over the slots finds the owner of a row in O(1); a row held
// by one slot is updated at once, a repeated row's owner scans the later slots
// until it has met them all, and a row held by kInputHotSlots slots or more is
// summed by a block of sixteen waves (fixed sixteenths of the slots, their sums
// added in order).
#include <math.h>
#include <stdlib.h>

#include <new>

#include "lst_internal.h"

struct lst_input {
  int64_t D = 0;
  int d = 0;
  int device = 0;
  hipStream_t stream = nullptr;
  float* W = nullptr;
  int* flags = nullptr;  // [0]: sticky status
  // open-addressing table of the rows of one update (empty between calls):
  // key (-1 empty), smallest slot, number of slots; and, per slot, the table
  // entry it owns (-1 if none), from which the table is emptied
  int* hkey = nullptr;
  int* hmin = nullptr;
  int* hcnt = nullptr;
  int* own = nullptr;
  // rows held by at least kInputHotSlots slots, summed by input_hot_kernel
  // ([0]: count, then the rows)
  int* hot = nullptr;
};

namespace lst {
namespace {

// Every index in [-1, D); otherwise the sticky status becomes LST_EINDEX.
__global__ void input_validate_kernel(const int32_t* __restrict__ idx, int n, int64_t D,
                                      int* flags) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n) return;
  const int r = idx[e];
  if (r < -1 || (int64_t)r >= D) atomicCAS(flags, 0, LST_EINDEX);
}

// Slots (and table entries) of the row table: twice the largest number of
// slots, so that the table is at most half full.
constexpr int kInputMaxSlots = 65536;
constexpr int kInputHashBits = 17;
constexpr int kInputHashSize = 1 << kInputHashBits;
static_assert(kInputHashSize >= 2 * kInputMaxSlots, "the row table must stay half empty");
// A row held by this many slots or more is summed by a block of 16 waves, each
// over a fixed sixteenth of the slots (the partial sums then added in order).
constexpr int kInputHotSlots = 64;
constexpr int kInputMaxHot = kInputMaxSlots / kInputHotSlots;

__device__ __forceinline__ unsigned input_hash(int r) {
  return ((unsigned)r * 2654435761u) >> (32 - kInputHashBits);
}

// Validates slot e's index and enters its row into the table: the entry keeps
// the smallest slot holding the row and the number of slots holding it.
__global__ void input_insert_kernel(const int32_t* __restrict__ idx, int n, int64_t D,
                                    int* hkey, int* hmin, int* hcnt, int* flags) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n) return;
  const int r = idx[e];
  if (r < -1 || (int64_t)r >= D) {
    atomicCAS(flags, 0, LST_EINDEX);
    return;
  }
  if (r < 0) return;
  unsigned h = input_hash(r);
  for (int probe = 0; probe < kInputHashSize; ++probe) {
    const int prev = atomicCAS(hkey + h, -1, r);
    if (prev == -1 || prev == r) {
      atomicMin(hmin + h, e);
      atomicAdd(hcnt + h, 1);
      return;
    }
    h = (h + 1) & (kInputHashSize - 1);
  }
}

// Empties the entries recorded in own[] (one per distinct row) and the list
// of hot rows.
__global__ void input_clear_kernel(int* own, int n, int* hkey, int* hmin, int* hcnt, int* hot) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e == 0) hot[0] = 0;
  if (e >= n) return;
  const int h = own[e];
  if (h < 0) return;
  hkey[h] = -1;
  hmin[h] = 0x7fffffff;
  hcnt[h] = 0;
  own[e] = -1;
}

// The empty table (init): every key -1, every smallest slot INT_MAX, counts 0.
__global__ void input_table_init_kernel(int* hkey, int* hmin, int* hcnt, int* own, int* hot) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e == 0) hot[0] = 0;
  if (e < kInputHashSize) {
    hkey[e] = -1;
    hmin[e] = 0x7fffffff;
    hcnt[e] = 0;
  }
  if (e < kInputMaxSlots) own[e] = -1;
}

// Pairs (or slots) handled per round: their loads are all issued before the
// first result is used, so a long list pays the memory latency once per round.
constexpr int kInputBatch = 8;
// Slots whose rows of dA an owner wave has in flight at once.
constexpr int kInputRows = 4;

// A[i, :] = sum_k v_ik W[u_ik, :], one wave per example, pairs in order.
// Columns in chunks of 256 (four per lane; 16-byte loads when VEC).
template <bool VEC>
__global__ __launch_bounds__(256) void input_forward_kernel(const float* __restrict__ W,
                                                            int64_t D, int d,
                                                            const int32_t* __restrict__ idx,
                                                            const float* __restrict__ val, int m,
                                                            int K, float* __restrict__ A) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= m) return;
  const int32_t* ip = idx + (size_t)i * K;
  const float* vp = val + (size_t)i * K;
  for (int c0 = 0; c0 < d; c0 += 256) {
    const int col = c0 + 4 * lane;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    for (int k0 = 0; k0 < K; k0 += kInputBatch) {
      float4 w[kInputBatch];
      float v[kInputBatch];
#pragma unroll
      for (int u = 0; u < kInputBatch; ++u) {
        const int k = k0 + u;
        const int r = k < K ? ip[k] : -1;
        // padding, a bad index (flagged elsewhere) and pairs past K add nothing
        const bool on = r >= 0 && (int64_t)r < D;
        v[u] = on ? vp[k] : 0.f;
        const float* row = W + (size_t)(on ? r : 0) * d;
        w[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (on && col < d) {
          if (VEC) {
            w[u] = *reinterpret_cast<const float4*>(row + col);
          } else {
            w[u].x = row[col];
            if (col + 1 < d) w[u].y = row[col + 1];
            if (col + 2 < d) w[u].z = row[col + 2];
            if (col + 3 < d) w[u].w = row[col + 3];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kInputBatch; ++u) {
        if (k0 + u >= K) break;
        a0 += v[u] * w[u].x; a1 += v[u] * w[u].y; a2 += v[u] * w[u].z; a3 += v[u] * w[u].w;
      }
    }
    float* out = A + (size_t)i * d;
    if (VEC) {
      if (col < d) *reinterpret_cast<float4*>(out + col) = make_float4(a0, a1, a2, a3);
    } else {
      if (col < d) out[col] = a0;
      if (col + 1 < d) out[col + 1] = a1;
      if (col + 2 < d) out[col + 2] = a2;
      if (col + 3 < d) out[col + 3] = a3;
    }
  }
}

// Long inputs (K > kInputSplitK): one block per (example, 256-column chunk);
// wave w sums the pairs of the w-th quarter of the example's list in order,
// and the four partial sums are added in wave order, so the result does not
// depend on timing.
constexpr int kInputSplitK = 16;

template <bool VEC>
__global__ __launch_bounds__(256) void input_forward_split_kernel(
    const float* __restrict__ W, int64_t D, int d, const int32_t* __restrict__ idx,
    const float* __restrict__ val, int m, int K, float* __restrict__ A) {
  __shared__ float4 part[3][64];
  const int nch = (d + 255) / 256;
  const int i = blockIdx.x / nch, c0 = (blockIdx.x % nch) * 256;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = c0 + 4 * lane;
  const int q = (K + 3) / 4, kb = wave * q, ke = min(K, kb + q);
  const int32_t* ip = idx + (size_t)i * K;
  const float* vp = val + (size_t)i * K;
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  for (int k0 = kb; k0 < ke; k0 += kInputBatch) {
    float4 w[kInputBatch];
    float v[kInputBatch];
#pragma unroll
    for (int u = 0; u < kInputBatch; ++u) {
      const int k = k0 + u;
      const int r = k < ke ? ip[k] : -1;
      const bool on = r >= 0 && (int64_t)r < D;
      v[u] = on ? vp[k] : 0.f;
      const float* row = W + (size_t)(on ? r : 0) * d;
      w[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (on && col < d) {
        if (VEC) {
          w[u] = *reinterpret_cast<const float4*>(row + col);
        } else {
          w[u].x = row[col];
          if (col + 1 < d) w[u].y = row[col + 1];
          if (col + 2 < d) w[u].z = row[col + 2];
          if (col + 3 < d) w[u].w = row[col + 3];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kInputBatch; ++u) {
      if (k0 + u >= ke) break;
      a0 += v[u] * w[u].x; a1 += v[u] * w[u].y; a2 += v[u] * w[u].z; a3 += v[u] * w[u].w;
    }
  }
  if (wave > 0) part[wave - 1][lane] = make_float4(a0, a1, a2, a3);
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int p = 0; p < 3; ++p) {
    const float4 o = part[p][lane];
    a0 += o.x; a1 += o.y; a2 += o.z; a3 += o.w;
  }
  float* out = A + (size_t)i * d;
  if (VEC) {
    if (col < d) *reinterpret_cast<float4*>(out + col) = make_float4(a0, a1, a2, a3);
  } else {
    if (col < d) out[col] = a0;
    if (col + 1 < d) out[col + 1] = a1;
    if (col + 2 < d) out[col + 2] = a2;
    if (col + 3 < d) out[col + 3] = a3;
  }
}

// One wave per slot e = i*K + k.  The wave of the first slot holding row r
// (from the table) records the entry it owns, then sums v dA over every slot
// holding r, in slot order, and updates the row: at once when the row has one
// slot, else scanning the later slots (kInputBatch chunks of 64 per round)
// until it has met all of them.  With the sticky status set, ownership is still
// recorded (the table must be emptied) but W is left alone.
__global__ __launch_bounds__(256) void input_update_kernel(float* __restrict__ W, int64_t D,
                                                           int d,
                                                           const int32_t* __restrict__ idx,
                                                           const float* __restrict__ val,
                                                           const float* __restrict__ gA, int n,
                                                           int K, float lr, const int* hkey,
                                                           const int* hmin, const int* hcnt,
                                                           int* own, int* hot, const int* flags) {
  const int e = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (e >= n) return;
  const int r = idx[e];
  if (r < 0 || (int64_t)r >= D) return;  // padding, or an index the insert pass flagged
  unsigned h = input_hash(r);
  int probe = 0;
  while (probe < kInputHashSize && hkey[h] != r) {
    h = (h + 1) & (kInputHashSize - 1);
    ++probe;
  }
  if (probe == kInputHashSize || hmin[h] != e) return;
  if (lane == 0) own[e] = (int)h;
  if (*flags) return;
  const int cnt = hcnt[h];
  if (cnt >= kInputHotSlots) {
    if (lane == 0) hot[1 + atomicAdd(hot, 1)] = r;
    return;
  }
  const bool vec = (d % 4 == 0);
  // columns in groups of 1024 (four 256-column chunks per lane); one scan per group
  for (int cg = 0; cg < d; cg += 1024) {
    float4 acc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
    const int nc = min(4, (d - cg + 255) / 256);  // chunks of this group
    int met = 0;
    for (int s0 = e; s0 < n && met < cnt; s0 += 64 * kInputBatch) {
      unsigned long long hits[kInputBatch];
      if (cnt == 1) {
#pragma unroll
        for (int u = 0; u < kInputBatch; ++u) hits[u] = u == 0 ? 1ull : 0ull;
      } else {
        int x[kInputBatch];
#pragma unroll
        for (int u = 0; u < kInputBatch; ++u) {
          const int s = s0 + 64 * u + lane;
          x[u] = s < n ? idx[s] : -1;
        }
#pragma unroll
        for (int u = 0; u < kInputBatch; ++u) hits[u] = __ballot(x[u] == r);
      }
#pragma unroll
      for (int u = 0; u < kInputBatch; ++u) {
        unsigned long long hb = hits[u];
        met += __popcll(hb);
        // kInputRows slots at a time: their rows of dA are in flight together
        while (hb) {
          int t[kInputRows];
          bool on[kInputRows];
#pragma unroll
          for (int q = 0; q < kInputRows; ++q) {
            on[q] = hb != 0;
            t[q] = s0 + 64 * u + (on[q] ? __ffsll((long long)hb) - 1 : 0);
            hb &= hb - 1;
          }
          float v[kInputRows];
          float4 g[kInputRows][4];
#pragma unroll
          for (int q = 0; q < kInputRows; ++q) {
            v[q] = val[on[q] ? t[q] : e];
            const float* gr = gA + (size_t)((on[q] ? t[q] : e) / K) * d;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              const int col = cg + 256 * c + 4 * lane;
              g[q][c] = make_float4(0.f, 0.f, 0.f, 0.f);
              if (c < nc && col < d) {
                if (vec) {
                  g[q][c] = *reinterpret_cast<const float4*>(gr + col);
                } else {
                  g[q][c].x = gr[col];
                  if (col + 1 < d) g[q][c].y = gr[col + 1];
                  if (col + 2 < d) g[q][c].z = gr[col + 2];
                  if (col + 3 < d) g[q][c].w = gr[col + 3];
                }
              }
            }
          }
#pragma unroll
          for (int q = 0; q < kInputRows; ++q) {
            if (!on[q]) break;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              acc[c].x += v[q] * g[q][c].x; acc[c].y += v[q] * g[q][c].y;
              acc[c].z += v[q] * g[q][c].z; acc[c].w += v[q] * g[q][c].w;
            }
          }
        }
      }
    }
    float* row = W + (size_t)r * d;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int col = cg + 256 * c + 4 * lane;
      if (c >= nc || col >= d) continue;
      row[col] -= lr * acc[c].x;
      if (col + 1 < d) row[col + 1] -= lr * acc[c].y;
      if (col + 2 < d) row[col + 2] -= lr * acc[c].z;
      if (col + 3 < d) row[col + 3] -= lr * acc[c].w;
    }
  }
}

// Block b (1024 threads) sums the hot row hot[1 + b / nch] over columns
// [256 (b % nch), +256): wave w adds v dA over the slots of the w-th sixteenth
// of [0, n) that hold the row, in slot order; the sixteen partial sums are then
// added in wave order and the row is updated once.  Blocks past the number of
// hot rows exit.
__global__ __launch_bounds__(1024) void input_hot_kernel(float* __restrict__ W, int d,
                                                         const int32_t* __restrict__ idx,
                                                         const float* __restrict__ val,
                                                         const float* __restrict__ gA, int n,
                                                         int K, float lr, const int* hot,
                                                         const int* flags) {
  __shared__ float4 part[16][64];
  const int nch = (d + 255) / 256;
  const int hid = blockIdx.x / nch;
  if (hid >= hot[0] || *flags) return;
  const int r = hot[1 + hid];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = (blockIdx.x % nch) * 256 + 4 * lane;
  const bool vec = (d % 4 == 0);
  const int span = (n + 15) / 16, sb = wave * span, se = min(n, sb + span);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = sb; s0 < se; s0 += 64 * kInputBatch) {
    unsigned long long hits[kInputBatch];
    {
      int x[kInputBatch];
#pragma unroll
      for (int u = 0; u < kInputBatch; ++u) {
        const int s = s0 + 64 * u + lane;
        x[u] = s < se ? idx[s] : -1;
      }
#pragma unroll
      for (int u = 0; u < kInputBatch; ++u) hits[u] = __ballot(x[u] == r);
    }
#pragma unroll
    for (int u = 0; u < kInputBatch; ++u) {
      unsigned long long hb = hits[u];
      while (hb) {
        int t[kInputRows];
        bool on[kInputRows];
#pragma unroll
        for (int q = 0; q < kInputRows; ++q) {
          on[q] = hb != 0;
          t[q] = s0 + 64 * u + (on[q] ? __ffsll((long long)hb) - 1 : 0);
          hb &= hb - 1;
        }
        float v[kInputRows];
        float4 g[kInputRows];
#pragma unroll
        for (int q = 0; q < kInputRows; ++q) {
          const int tq = on[q] ? t[q] : sb;
          v[q] = val[tq];
          const float* gr = gA + (size_t)(tq / K) * d;
          g[q] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (on[q] && col < d) {
            if (vec) {
              g[q] = *reinterpret_cast<const float4*>(gr + col);
            } else {
              g[q].x = gr[col];
              if (col + 1 < d) g[q].y = gr[col + 1];
              if (col + 2 < d) g[q].z = gr[col + 2];
              if (col + 3 < d) g[q].w = gr[col + 3];
            }
          }
        }
#pragma unroll
        for (int q = 0; q < kInputRows; ++q) {
          if (!on[q]) break;
          acc.x += v[q] * g[q].x; acc.y += v[q] * g[q].y;
          acc.z += v[q] * g[q].z; acc.w += v[q] * g[q].w;
        }
      }
    }
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  float4 sum = part[0][lane];
  for (int w = 1; w < 16; ++w) {
    const float4 o = part[w][lane];
    sum.x += o.x; sum.y += o.y; sum.z += o.z; sum.w += o.w;
  }
  float* row = W + (size_t)r * d;
  if (col < d) row[col] -= lr * sum.x;
  if (col + 1 < d) row[col + 1] -= lr * sum.y;
  if (col + 2 < d) row[col + 2] -= lr * sum.z;
  if (col + 3 < d) row[col + 3] -= lr * sum.w;
}

int check_batch(lst_input* s, int32_t m, int32_t K, const int32_t* idx, const float* val) {
  if (!s || m < 1 || K < 1 || !idx || !val) return LST_EINVAL;
  if ((int64_t)m * K > kInputMaxSlots) return LST_EINVAL;
  return LST_OK;
}

struct DeviceScope {
  int prev = -1;
  explicit DeviceScope(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceScope() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

}  // namespace
}  // namespace lst

using namespace lst;

extern "C" {

int lst_input_init(lst_input** out, int64_t D_in, int32_t d, const float* W_in,
                   void* hip_stream) {
  if (!out || !W_in || D_in < 1 || d < 1 || d > 4096 || D_in > (int64_t)0x7fffffff)
    return LST_EINVAL;
  lst_input* s = new (std::nothrow) lst_input();
  if (!s) return LST_ENOMEM;
  s->D = D_in;
  s->d = d;
  s->stream = static_cast<hipStream_t>(hip_stream);
  auto fail = [&](int code) {
    (void)hipStreamSynchronize(s->stream);
    for (void* p : {(void*)s->W, (void*)s->flags, (void*)s->hkey, (void*)s->hmin, (void*)s->hcnt,
                    (void*)s->own, (void*)s->hot})
      if (p) (void)hipFree(p);
    delete s;
    return code;
  };
  if (hipGetDevice(&s->device) != hipSuccess) return fail(LST_EHIP);
  if (hipMalloc((void**)&s->W, (size_t)D_in * d * sizeof(float)) != hipSuccess ||
      hipMalloc((void**)&s->flags, sizeof(int)) != hipSuccess ||
      hipMalloc((void**)&s->hkey, kInputHashSize * sizeof(int)) != hipSuccess ||
      hipMalloc((void**)&s->hmin, kInputHashSize * sizeof(int)) != hipSuccess ||
      hipMalloc((void**)&s->hcnt, kInputHashSize * sizeof(int)) != hipSuccess ||
      hipMalloc((void**)&s->own, kInputMaxSlots * sizeof(int)) != hipSuccess ||
      hipMalloc((void**)&s->hot, (1 + kInputMaxHot) * sizeof(int)) != hipSuccess)
    return fail(LST_ENOMEM);
  hipLaunchKernelGGL(input_table_init_kernel, dim3(kInputHashSize / 256), dim3(256), 0, s->stream,
                     s->hkey, s->hmin, s->hcnt, s->own, s->hot);
  if (hipMemsetAsync(s->flags, 0, sizeof(int), s->stream) != hipSuccess ||
      hipMemcpyAsync(s->W, W_in, (size_t)D_in * d * sizeof(float), hipMemcpyDeviceToDevice,
                     s->stream) != hipSuccess ||
      hipStreamSynchronize(s->stream) != hipSuccess)
    return fail(LST_EHIP);
  *out = s;
  return LST_OK;
}

int lst_input_forward(lst_input* s, int32_t m, int32_t K, const int32_t* idx, const float* val,
                      float* A) {
  int rc = check_batch(s, m, K, idx, val);
  if (rc != LST_OK) return rc;
  if (!A) return LST_EINVAL;
  DeviceScope g(s->device);
  const int n = m * K;
  hipLaunchKernelGGL(input_validate_kernel, dim3((n + 255) / 256), dim3(256), 0, s->stream, idx,
                     n, s->D, s->flags);
  const bool vec = (s->d % 4 == 0) && (((uintptr_t)A & 15) == 0);
  if (K > kInputSplitK) {
    const dim3 grid((unsigned)(m * ((s->d + 255) / 256)));
    if (vec)
      hipLaunchKernelGGL(input_forward_split_kernel<true>, grid, dim3(256), 0, s->stream, s->W,
                         s->D, s->d, idx, val, m, K, A);
    else
      hipLaunchKernelGGL(input_forward_split_kernel<false>, grid, dim3(256), 0, s->stream, s->W,
                         s->D, s->d, idx, val, m, K, A);
  } else if (vec) {
    hipLaunchKernelGGL(input_forward_kernel<true>, dim3((m + 3) / 4), dim3(256), 0, s->stream,
                       s->W, s->D, s->d, idx, val, m, K, A);
  } else {
    hipLaunchKernelGGL(input_forward_kernel<false>, dim3((m + 3) / 4), dim3(256), 0, s->stream,
                       s->W, s->D, s->d, idx, val, m, K, A);
  }
  return hipGetLastError() == hipSuccess ? LST_OK : LST_EHIP;
}

int lst_input_update(lst_input* s, int32_t m, int32_t K, const int32_t* idx, const float* val,
                     const float* grad_A, float lr) {
  int rc = check_batch(s, m, K, idx, val);
  if (rc != LST_OK) return rc;
  if (!grad_A || !(lr > 0.f) || !isfinite(lr)) return LST_EINVAL;
  DeviceScope g(s->device);
  const int n = m * K;
  hipLaunchKernelGGL(input_insert_kernel, dim3((n + 255) / 256), dim3(256), 0, s->stream, idx, n,
                     s->D, s->hkey, s->hmin, s->hcnt, s->flags);
  hipLaunchKernelGGL(input_update_kernel, dim3((n + 3) / 4), dim3(256), 0, s->stream, s->W, s->D,
                     s->d,
                     idx, val, grad_A, n, K, lr, s->hkey, s->hmin, s->hcnt, s->own, s->hot,
                     s->flags);
  if (n >= kInputHotSlots) {
    const int nch = (s->d + 255) / 256;
    hipLaunchKernelGGL(input_hot_kernel, dim3((unsigned)((n / kInputHotSlots) * nch)), dim3(1024),
                       0, s->stream, s->W, s->d, idx, val, grad_A, n, K, lr, s->hot, s->flags);
  }
  hipLaunchKernelGGL(input_clear_kernel, dim3((n + 255) / 256), dim3(256), 0, s->stream, s->own, n,
                     s->hkey, s->hmin, s->hcnt, s->hot);
  return hipGetLastError() == hipSuccess ? LST_OK : LST_EHIP;
}

int lst_input_get_W(lst_input* s, float* W) {
  if (!s || !W) return LST_EINVAL;
  DeviceScope g(s->device);
  return hipMemcpyAsync(W, s->W, (size_t)s->D * s->d * sizeof(float), hipMemcpyDeviceToDevice,
                        s->stream) == hipSuccess
             ? LST_OK
             : LST_EHIP;
}

int lst_input_sync(lst_input* s) {
  if (!s) return LST_EINVAL;
  DeviceScope g(s->device);
  int err = 0;
  if (hipStreamSynchronize(s->stream) != hipSuccess ||
      hipMemcpy(&err, s->flags, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess)
    return LST_EHIP;
  if (err) {
    const int zero = 0;
    if (hipMemcpy(s->flags, &zero, sizeof(int), hipMemcpyHostToDevice) != hipSuccess)
      return LST_EHIP;
  }
  return err;
}

void lst_input_free(lst_input* s) {
  if (!s) return;
  DeviceScope g(s->device);
  (void)hipStreamSynchronize(s->stream);
  for (void* p : {(void*)s->W, (void*)s->flags, (void*)s->hkey, (void*)s->hmin, (void*)s->hcnt,
                  (void*)s->own, (void*)s->hot})
    (void)hipFree(p);
  delete s;
}

}  // extern "C"
