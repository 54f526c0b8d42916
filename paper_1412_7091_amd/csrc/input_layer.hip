// The sparse input layer of section 2.2 ("the easy part"): a K-sparse input
// x (K (index, value) pairs per example; index -1 unused) enters the first
// hidden layer through a D_in x d matrix W_in, so that
//   forward: A[i, :] = sum_k v_ik W_in[u_ik, :]           (O(K d) per example)
//   update:  W_in[r, :] -= lr * sum_{(i,k): u_ik = r} v_ik dA[i, :]
// touch only the rows the minibatch refers to.  The update writes each row
// once, from the wave of the row's first slot (in (example, pair) order),
// which adds the contributions of all its slots in that order: deterministic,
// with no atomics on W_in.
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
  for (int c0 = 0; c0 < d; c0 += 256) {
    const int col = c0 + 4 * lane;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    for (int k = 0; k < K; ++k) {
      const int r = idx[(size_t)i * K + k];
      if (r < 0 || (int64_t)r >= D) continue;  // padding (a bad index is flagged elsewhere)
      const float v = val[(size_t)i * K + k];
      const float* row = W + (size_t)r * d;
      if (VEC) {
        if (col < d) {
          const float4 w = *reinterpret_cast<const float4*>(row + col);
          a0 += v * w.x; a1 += v * w.y; a2 += v * w.z; a3 += v * w.w;
        }
      } else {
        if (col < d) a0 += v * row[col];
        if (col + 1 < d) a1 += v * row[col + 1];
        if (col + 2 < d) a2 += v * row[col + 2];
        if (col + 3 < d) a3 += v * row[col + 3];
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

// One wave per slot e = i*K + k.  The wave of the first slot holding row r
// sums v dA over every slot holding r, in slot order, and updates the row.
__global__ __launch_bounds__(256) void input_update_kernel(float* __restrict__ W, int d,
                                                           const int32_t* __restrict__ idx,
                                                           const float* __restrict__ val,
                                                           const float* __restrict__ gA, int n,
                                                           int K, float lr, const int* flags) {
  if (*flags) return;
  const int e = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (e >= n) return;
  const int r = idx[e];
  if (r < 0) return;
  // owner: no earlier slot holds r
  for (int c0 = 0; c0 < e; c0 += 64) {
    const int s = c0 + lane;
    const bool hit = s < e && idx[s] == r;
    if (__ballot(hit)) return;
  }
  for (int c0 = 0; c0 < d; c0 += 256) {
    const int col = c0 + 4 * lane;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    for (int s0 = e; s0 < n; s0 += 64) {
      const int s = s0 + lane;
      unsigned long long hits = __ballot(s < n && idx[s] == r);
      while (hits) {
        const int b = __ffsll((long long)hits) - 1;
        hits &= hits - 1;
        const int t = s0 + b;
        const float v = val[t];
        const float* g = gA + (size_t)(t / K) * d;
        if (col < d) a0 += v * g[col];
        if (col + 1 < d) a1 += v * g[col + 1];
        if (col + 2 < d) a2 += v * g[col + 2];
        if (col + 3 < d) a3 += v * g[col + 3];
      }
    }
    float* row = W + (size_t)r * d;
    if (col < d) row[col] -= lr * a0;
    if (col + 1 < d) row[col + 1] -= lr * a1;
    if (col + 2 < d) row[col + 2] -= lr * a2;
    if (col + 3 < d) row[col + 3] -= lr * a3;
  }
}

constexpr int kInputMaxSlots = 65536;

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
    if (s->W) (void)hipFree(s->W);
    if (s->flags) (void)hipFree(s->flags);
    delete s;
    return code;
  };
  if (hipGetDevice(&s->device) != hipSuccess) return fail(LST_EHIP);
  if (hipMalloc((void**)&s->W, (size_t)D_in * d * sizeof(float)) != hipSuccess ||
      hipMalloc((void**)&s->flags, sizeof(int)) != hipSuccess)
    return fail(LST_ENOMEM);
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
  if (vec)
    hipLaunchKernelGGL(input_forward_kernel<true>, dim3((m + 3) / 4), dim3(256), 0, s->stream,
                       s->W, s->D, s->d, idx, val, m, K, A);
  else
    hipLaunchKernelGGL(input_forward_kernel<false>, dim3((m + 3) / 4), dim3(256), 0, s->stream,
                       s->W, s->D, s->d, idx, val, m, K, A);
  return hipGetLastError() == hipSuccess ? LST_OK : LST_EHIP;
}

int lst_input_update(lst_input* s, int32_t m, int32_t K, const int32_t* idx, const float* val,
                     const float* grad_A, float lr) {
  int rc = check_batch(s, m, K, idx, val);
  if (rc != LST_OK) return rc;
  if (!grad_A || !(lr > 0.f) || !isfinite(lr)) return LST_EINVAL;
  DeviceScope g(s->device);
  const int n = m * K;
  hipLaunchKernelGGL(input_validate_kernel, dim3((n + 255) / 256), dim3(256), 0, s->stream, idx,
                     n, s->D, s->flags);
  hipLaunchKernelGGL(input_update_kernel, dim3((n + 3) / 4), dim3(256), 0, s->stream, s->W, s->d,
                     idx, val, grad_A, n, K, lr, s->flags);
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
  (void)hipFree(s->W);
  (void)hipFree(s->flags);
  delete s;
}

}  // extern "C"
