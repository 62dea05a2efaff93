// The optional second dense hidden layer of the sparse MLP (the other reading
// of the paper's "3-layer MLP", Sec. 5.1): A2 = H1 Wh^T + bh, H2 = ReLU(A2),
// with Wh [H x H] row-major (output unit o, input unit k) and H1 = ReLU(A1).
// Its products are B x 128 x 128, a few MFLOP per step, so plain fp32 FMA
// chains over LDS-resident weights serve (a launch costs more than the
// arithmetic); the output layer then reads H2 where it would read H1.
//
//   forward   : A2 = ReLU(A1) Wh^T + bh; H2 = ReLU(A2) in the output layer's
//               operand type (and transposed, for fp32 operands)
//   backward  : dA1 = (dA2 Wh) * [A1 > 0]        (the pre-update Wh)
//               dWh = dA2^T ReLU(A1), dbh = 1^T dA2, Wh -= lr dWh, bh -= lr dbh
#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

constexpr int DN_THREADS = 256;
constexpr int DN_ROWS = 4;   // rows per workgroup of the row-parallel kernels
constexpr int WS = HID + 1;  // LDS row stride of Wh: reads along either index are conflict-free

// Row-parallel product with a resident 128 x 128 weight: thread t computes
// unit j = t % 128 of rows r0 + t / 128 + 2i (i < DN_ROWS / 2).  FWD: out[r][o]
// = bh[o] + sum_k relu(in[r][k]) Wh[o][k]; otherwise out[r][k] = sum_o in[r][o]
// Wh[o][k], masked by [A1 > 0].  Wh sits in LDS as [o][k] with row stride 129,
// so lanes that differ in o (FWD) or in k (backward) hit distinct banks.
template <bool FWD, bool BF16>
__global__ __launch_bounds__(DN_THREADS) void k_dense_rows(const float* __restrict__ in,
                                                          const float* __restrict__ Wh,
                                                          const float* __restrict__ bh, int B,
                                                          int rows_pad, float* __restrict__ out,
                                                          typename Mma<BF16>::elem* __restrict__ Hop,
                                                          typename Mma<BF16>::elem* __restrict__ HopT,
                                                          int ld_t, const float* __restrict__ A1) {
  using E = typename Mma<BF16>::elem;
  __shared__ float w[HID * WS];         // 66 KB
  __shared__ float xs[DN_ROWS][HID];    // the workgroup's input rows
  const int tid = threadIdx.x;
  const int r0 = blockIdx.x * DN_ROWS;
  for (int e = tid; e < HID * HID / 4; e += DN_THREADS) {
    const float4 v = reinterpret_cast<const float4*>(Wh)[e];
    const int o = (4 * e) / HID, k = (4 * e) % HID;
    float* d = w + o * WS + k;
    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
  }
  for (int e = tid; e < DN_ROWS * HID; e += DN_THREADS) {
    const int r = e / HID, k = e % HID;
    const float v = r0 + r < B ? in[(size_t)(r0 + r) * HID + k] : 0.0f;
    xs[r][k] = FWD ? fmaxf(v, 0.0f) : v;
  }
  __syncthreads();
  constexpr int RPT = DN_ROWS / 2;
  const int j = tid % HID, rr = tid / HID;
  float acc[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) acc[i] = FWD ? bh[j] : 0.0f;
#pragma unroll 8
  for (int k = 0; k < HID; ++k) {
    const float wk = FWD ? w[j * WS + k] : w[k * WS + j];
#pragma unroll
    for (int i = 0; i < RPT; ++i) acc[i] = fmaf(xs[rr + 2 * i][k], wk, acc[i]);
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = r0 + rr + 2 * i;
    if (r >= rows_pad) continue;
    const bool live = r < B;
    if constexpr (FWD) {
      // rows past B stay zero in every output, as after the gather
      const float a = live ? acc[i] : 0.0f;
      out[(size_t)r * HID + j] = a;
      const float h = fmaxf(a, 0.0f);
      Hop[(size_t)r * HID + j] = (E)h;
      if constexpr (!BF16) HopT[(size_t)j * ld_t + r] = h;
    } else {
      const float a1 = live ? A1[(size_t)r * HID + j] : 0.0f;
      out[(size_t)r * HID + j] = live && a1 > 0.0f ? acc[i] : 0.0f;
    }
  }
}

// dWh[o][k] = sum_r dA2[r][o] relu(A1[r][k]) and dbh[o] = sum_r dA2[r][o], in
// row order; then the update in place.  Workgroup = 2 output units x 128
// input units; the rows come through LDS in chunks of 64 (all of a chunk's
// loads in flight together), the chunk's dA2 values of the two units beside.
constexpr int WG_CHUNK = 64;
__global__ __launch_bounds__(DN_THREADS) void k_dense_wgrad(const float* __restrict__ dA2,
                                                           const float* __restrict__ A1, int B,
                                                           float lr, float* __restrict__ Wh,
                                                           float* __restrict__ bh) {
  __shared__ float hs[WG_CHUNK][HID];
  __shared__ float ds[WG_CHUNK][2];
  const int tid = threadIdx.x;
  const int k = tid % HID, half = tid / HID;
  const int o = blockIdx.x * 2 + half;
  float acc = 0.0f, db = 0.0f;
  for (int c0 = 0; c0 < B; c0 += WG_CHUNK) {
    const int nr = min(WG_CHUNK, B - c0);
    __syncthreads();  // the previous chunk is consumed
    for (int e = tid; e < nr * HID / 4; e += DN_THREADS) {
      const float4 v = reinterpret_cast<const float4*>(A1 + (size_t)c0 * HID)[e];
      float* d = &hs[0][0] + 4 * e;
      d[0] = fmaxf(v.x, 0.0f); d[1] = fmaxf(v.y, 0.0f); d[2] = fmaxf(v.z, 0.0f); d[3] = fmaxf(v.w, 0.0f);
    }
    for (int e = tid; e < nr * 2; e += DN_THREADS)
      ds[e / 2][e % 2] = dA2[(size_t)(c0 + e / 2) * HID + blockIdx.x * 2 + e % 2];
    __syncthreads();
    for (int r = 0; r < nr; ++r) {
      const float d = ds[r][half];
      acc = fmaf(d, hs[r][k], acc);
      db += d;
    }
  }
  Wh[o * HID + k] = fmaf(-lr, acc, Wh[o * HID + k]);
  if (k == 0) bh[o] = fmaf(-lr, db, bh[o]);
}

hipError_t launch_dense_fwd(bool use_bf16, const float* A1, const float* Wh, const float* bh, int B,
                            int rows_pad, float* A2, void* Hop, void* HopT, int ld_t, hipStream_t st) {
  const dim3 grid((rows_pad + DN_ROWS - 1) / DN_ROWS), block(DN_THREADS);
  if (use_bf16)
    hipLaunchKernelGGL((k_dense_rows<true, true>), grid, block, 0, st, A1, Wh, bh, B, rows_pad, A2,
                       (bf16*)Hop, (bf16*)nullptr, ld_t, nullptr);
  else
    hipLaunchKernelGGL((k_dense_rows<true, false>), grid, block, 0, st, A1, Wh, bh, B, rows_pad, A2,
                       (float*)Hop, (float*)HopT, ld_t, nullptr);
  return hipGetLastError();
}

hipError_t launch_dense_bwd(const float* dA2, const float* A1, float* Wh, float* bh, int B, int rows_pad,
                            float lr, float* dA1, hipStream_t st) {
  // dA1 first: it reads Wh before the update below writes it (same stream)
  hipLaunchKernelGGL((k_dense_rows<false, false>), dim3((rows_pad + DN_ROWS - 1) / DN_ROWS),
                     dim3(DN_THREADS), 0, st, dA2, Wh, nullptr, B, rows_pad, dA1, (float*)nullptr,
                     (float*)nullptr, 0, A1);
  hipLaunchKernelGGL(k_dense_wgrad, dim3(HID / 2), dim3(DN_THREADS), 0, st, dA2, A1, B, lr, Wh, bh);
  return hipGetLastError();
}

}  // namespace asgd
