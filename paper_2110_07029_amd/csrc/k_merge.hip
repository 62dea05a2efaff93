// Normalized model merge (Alg. 2, final step): w' = sum_i alpha_i w_i +
// gamma (w - w_prev), one streaming pass over all parameters in float4
// vectors, float64 accumulation, one rounding per element.  The replicas
// share the GPU's HBM, so the paper's multi-stream all-reduce becomes a
// single read of every replica.  Also the float64 sum of squares used by the
// L2-per-parameter regularization gate of Alg. 2.
#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

// Replica pointers and weights travel as kernel arguments; the loops over
// them are fully unrolled with a guard so every access is a constant offset.
struct MergeArgs {
  const float4* rep[MERGE_MAX];
  double a[MERGE_MAX];
  float4* bc[MERGE_MAX];
};

// out may alias gp: each element of gp is read before the same element of out is written.
__global__ __launch_bounds__(256) void k_merge(float4* out, const float4* __restrict__ g,
                                               const float4* gp, MergeArgs args, int n, int nb,
                                               double gamma, int64_t count4) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count4; e += stride) {
    double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
#pragma unroll
    for (int i = 0; i < MERGE_MAX; ++i) {
      if (i < n) {
        const float4 v = args.rep[i][e];
        const double ai = args.a[i];
        a0 = fma(ai, (double)v.x, a0);
        a1 = fma(ai, (double)v.y, a1);
        a2 = fma(ai, (double)v.z, a2);
        a3 = fma(ai, (double)v.w, a3);
      }
    }
    if (gp) {
      const float4 x = g[e], y = gp[e];
      a0 = fma(gamma, (double)x.x - (double)y.x, a0);
      a1 = fma(gamma, (double)x.y - (double)y.y, a1);
      a2 = fma(gamma, (double)x.z - (double)y.z, a2);
      a3 = fma(gamma, (double)x.w - (double)y.w, a3);
    }
    const float4 o = make_float4((float)a0, (float)a1, (float)a2, (float)a3);
    out[e] = o;
#pragma unroll
    for (int i = 0; i < MERGE_MAX; ++i)
      if (i < nb) args.bc[i][e] = o;
  }
}

hipError_t launch_merge(float* out, const float* g, const float* gp, const float* const* reps,
                        const double* alpha, int n, double gamma, float* const* bcast, int nb,
                        int64_t count, hipStream_t st) {
  // count is a multiple of 4 (parameter sections are padded); n, nb <= MERGE_MAX.
  const int64_t count4 = count / 4;
  MergeArgs args{};
  for (int i = 0; i < n && i < MERGE_MAX; ++i) {
    args.rep[i] = reinterpret_cast<const float4*>(reps[i]);
    args.a[i] = alpha[i];
  }
  for (int i = 0; i < nb && i < MERGE_MAX; ++i) args.bc[i] = reinterpret_cast<float4*>(bcast[i]);
  int64_t blocks = (count4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_merge, dim3((unsigned)blocks), dim3(256), 0, st, reinterpret_cast<float4*>(out),
                     reinterpret_cast<const float4*>(g),
                     reinterpret_cast<const float4*>(gp), args, n, nb, gamma, count4);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_sqnorm_part(const float* __restrict__ w, int64_t count,
                                                     double* __restrict__ partial) {
  __shared__ double red[4];
  double s = 0.0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count; e += stride) {
    const double v = (double)w[e];
    s = fma(v, v, s);
  }
  s = wave_sum_d(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) partial[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

__global__ __launch_bounds__(256) void k_sqnorm_final(const double* __restrict__ partial, int np,
                                                      double* __restrict__ out) {
  __shared__ double red[4];
  double s = 0.0;
  for (int e = threadIdx.x; e < np; e += 256) s += partial[e];
  s = wave_sum_d(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) *out = ((red[0] + red[1]) + red[2]) + red[3];
}

// The sums of squares of n parameter vectors in one launch: blockIdx.y picks
// the vector, SQNORM_BLOCKS workgroups stream it in float4 loads, and each
// writes its partial; a second launch reduces every vector's partials in a
// fixed order.  partial: n x SQNORM_BLOCKS doubles; out: n doubles, the sums,
// or sqrt(sum) / l2_div when l2_div > 0 (the L2 norm per parameter).
struct SqArgs {
  const float4* w[MERGE_MAX];
};

__global__ __launch_bounds__(256) void k_sqnorm_multi_part(SqArgs a, int64_t count4,
                                                           double* __restrict__ partial) {
  __shared__ double red[4];
  const float4* __restrict__ w = a.w[blockIdx.y];
  double s = 0.0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count4; e += stride) {
    const float4 v = w[e];
    s = fma((double)v.x, (double)v.x, s);
    s = fma((double)v.y, (double)v.y, s);
    s = fma((double)v.z, (double)v.z, s);
    s = fma((double)v.w, (double)v.w, s);
  }
  s = wave_sum_d(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) partial[(size_t)blockIdx.y * SQNORM_BLOCKS + blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

__global__ __launch_bounds__(256) void k_sqnorm_multi_final(const double* __restrict__ partial,
                                                            double* __restrict__ out, double l2_div) {
  __shared__ double red[4];
  const double* p = partial + (size_t)blockIdx.x * SQNORM_BLOCKS;
  double s = 0.0;
  for (int e = threadIdx.x; e < SQNORM_BLOCKS; e += 256) s += p[e];
  s = wave_sum_d(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double t = ((red[0] + red[1]) + red[2]) + red[3];
    out[blockIdx.x] = l2_div > 0.0 ? sqrt(t) / l2_div : t;
  }
}

hipError_t launch_sqnorm_multi(const float* const* w, int n, int64_t count, double* partial, double* out,
                               double l2_div, hipStream_t st) {
  // count is a multiple of 4 (parameter sections are padded); 1 <= n <= MERGE_MAX
  if (n < 1 || n > MERGE_MAX || count % 4) return hipErrorInvalidValue;
  SqArgs a{};
  for (int i = 0; i < n; ++i) a.w[i] = reinterpret_cast<const float4*>(w[i]);
  hipLaunchKernelGGL(k_sqnorm_multi_part, dim3(SQNORM_BLOCKS, n), dim3(256), 0, st, a, count / 4, partial);
  hipLaunchKernelGGL(k_sqnorm_multi_final, dim3(n), dim3(256), 0, st, partial, out, l2_div);
  return hipGetLastError();
}

hipError_t launch_sqnorm(const float* w, int64_t count, double* partial, double* out,
                         hipStream_t st) {
  hipLaunchKernelGGL(k_sqnorm_part, dim3(SQNORM_BLOCKS), dim3(256), 0, st, w, count, partial);
  hipLaunchKernelGGL(k_sqnorm_final, dim3(1), dim3(256), 0, st, partial, SQNORM_BLOCKS, out);
  return hipGetLastError();
}

}  // namespace asgd
