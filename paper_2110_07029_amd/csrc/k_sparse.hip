// Sparse first-layer gradient and update: dW1[f] = sum over the batch entries
// (i, f, x) of x * dA1[i], applied only to the features present in the batch
// (the update pass of Sec. 2.1 restricted to the rows the sparse input
// touches).  Entries are grouped by the radix sort, so each distinct feature
// is one contiguous segment summed by one wavefront in ascending
// (row, position) order: deterministic, no atomics.
#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

constexpr int W1_UNROLL = 16;  // dA1 rows in flight per wavefront
static_assert(64 % W1_UNROLL == 0, "readlane indices stay below 64");

__global__ __launch_bounds__(256) void k_w1_update(float* __restrict__ W1, int F,
                                                   const int32_t* __restrict__ skeys,
                                                   const int32_t* __restrict__ svals, int n_keys,
                                                   const int32_t* __restrict__ row_of, CsrDev x,
                                                   const float* __restrict__ dA1, float lr) {
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= n_keys) return;
  const int f = skeys[j];
  if (f >= F) return;                      // label keys and invalid ids
  if (j > 0 && skeys[j - 1] == f) return;  // not the head of its segment
  const int xbase = x.indptr[0];
  float2* wp = reinterpret_cast<float2*>(W1 + (size_t)f * HID + 2 * lane);
  float2 w = *wp;  // in flight while the segment is summed
  float2 acc = make_float2(0.0f, 0.0f);
  for (int q0 = j;; q0 += 64) {
    const int q = q0 + lane;
    const bool in = q < n_keys && skeys[q] == f;
    int row = 0;
    float xv = 0.0f;
    if (in) {
      const int p = svals[q];
      row = row_of[p];
      xv = x.values[xbase + p];
    }
    const int cnt = __popcll(__ballot(in));  // a segment is contiguous: lanes 0..cnt-1
    // Lanes past the segment read dA1 row 0 and are discarded, so a partial
    // group of 16 costs one round trip like a full one (most segments are short).
    for (int u = 0; u < cnt; u += W1_UNROLL) {
      int ru[W1_UNROLL];
      float xu[W1_UNROLL];
      float2 d[W1_UNROLL];
#pragma unroll
      for (int k = 0; k < W1_UNROLL; ++k) {
        ru[k] = __builtin_amdgcn_readlane(row, u + k);
        xu[k] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, xv), u + k));
      }
#pragma unroll
      for (int k = 0; k < W1_UNROLL; ++k)
        d[k] = *reinterpret_cast<const float2*>(dA1 + (size_t)ru[k] * HID + 2 * lane);
#pragma unroll
      for (int k = 0; k < W1_UNROLL; ++k) {
        if (u + k < cnt) {
          acc.x = fmaf(xu[k], d[k].x, acc.x);
          acc.y = fmaf(xu[k], d[k].y, acc.y);
        }
      }
    }
    if (cnt < 64) break;
  }
  w.x = fmaf(-lr, acc.x, w.x);
  w.y = fmaf(-lr, acc.y, w.y);
  *wp = w;
}

hipError_t launch_w1_update(float* W1, int F, const int32_t* skeys, const int32_t* svals,
                            int n_feat_keys, const int32_t* row_of, const CsrDev& x,
                            const float* dA1, float lr, hipStream_t st) {
  if (n_feat_keys <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_w1_update, dim3((n_feat_keys + 3) / 4), dim3(256), 0, st, W1, F, skeys, svals,
                     n_feat_keys, row_of, x, dA1, lr);
  return hipGetLastError();
}

// Heads of the feature segments, compacted in order by one workgroup.
__global__ __launch_bounds__(1024) void k_touched(const int32_t* __restrict__ skeys, int n, int F,
                                                  int32_t* __restrict__ ids,
                                                  int32_t* __restrict__ count) {
  __shared__ int wsum[16];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int carry = 0;
  for (int base = 0; base < n; base += 1024) {
    const int j = base + threadIdx.x;
    int key = 0, head = 0;
    if (j < n) {
      key = skeys[j];
      head = key < F && (j == 0 || skeys[j - 1] != key);
    }
    int x = head;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    if (w == 0) {
      int s = lane < 16 ? wsum[lane] : 0;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        const int y = __shfl_up(s, o);
        if (lane >= o) s += y;
      }
      if (lane < 16) wsum[lane] = s;
    }
    __syncthreads();
    const int pos = carry + (w > 0 ? wsum[w - 1] : 0) + x - head;
    if (head) ids[pos] = key;
    carry += wsum[15];
    __syncthreads();
  }
  if (threadIdx.x == 0) *count = carry;
}

hipError_t launch_touched(const int32_t* skeys, int n_keys, int F, int32_t* ids, int32_t* count_dev,
                          hipStream_t st) {
  hipLaunchKernelGGL(k_touched, dim3(1), dim3(1024), 0, st, skeys, n_keys, F, ids, count_dev);
  return hipGetLastError();
}

}  // namespace asgd
