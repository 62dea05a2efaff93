// Device body of the label grouping of a training step, written for one
// workgroup so that it can ride along inside a larger launch (the output-layer
// forward gives it one workgroup of its own) instead of needing a launch, and
// a cross-stream event, of its own.
#pragma once

#include "asgd_dev.h"

namespace asgd {

// Exclusive scan of one int per thread over the workgroup (NT threads), plus
// the total; wsum: NT/64 ints of LDS.  Ends with a barrier, so wsum can be
// reused right after.
template <int NT>
__device__ __forceinline__ int wg_exclusive_scan(int x, int* wsum, int* total) {
  constexpr int W = NT / 64;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o);
    if (lane >= o) inc += y;
  }
  if (lane == 63) wsum[w] = inc;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int k = 0; k < W; ++k) {
    const int v = wsum[k];
    before += k < w ? v : 0;
    all += v;
  }
  __syncthreads();
  *total = all;
  return before + inc - x;
}

// (row, label) pairs grouped by 32-label block by one workgroup of NT
// threads: a counter per block (cnt: LDS when LDS, else global memory of
// ceil(L/32) ints), an exclusive scan into lbeg, then every valid pair is
// placed in its block's range.  lbeg[b] .. lbeg[b+1] (b < ceil(L/32)) is
// block b's range of lpair, each entry (row << 5) | (label % 32); invalid
// labels (key L) are dropped.  The order of the pairs inside a block is not
// fixed: the backward only ORs them into a bit mask, whose value does not
// depend on it.  wsum: NT/64 ints of LDS.
template <bool LDS>
__device__ __forceinline__ int lb_load(const int32_t* p) {
  if constexpr (LDS)
    return *p;
  else  // counters updated by atomics at L2: read past the L1
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <bool LDS>
__device__ __forceinline__ void lb_sync() {
  if constexpr (!LDS) __threadfence();
  __syncthreads();
}

template <int NT, bool LDS>
__device__ void wg_label_blocks(const int32_t* __restrict__ lkeys, int m, int L,
                                const int32_t* __restrict__ lrow, int32_t* __restrict__ lbeg,
                                int32_t* __restrict__ lpair, int32_t* cnt, int32_t* wsum) {
  const int nb = (L + 31) >> 5;
  const int t = threadIdx.x;
  for (int b = t; b < nb; b += NT) cnt[b] = 0;
  lb_sync<LDS>();
  for (int q = t; q < m; q += NT) {
    const int lab = lkeys[q];
    if (lab >= 0 && lab < L) atomicAdd(&cnt[lab >> 5], 1);
  }
  lb_sync<LDS>();
  // thread t owns the contiguous blocks [t*per, t*per + per)
  const int per = (nb + NT - 1) / NT;
  const int b0 = min(nb, t * per), b1 = min(nb, b0 + per);
  int local = 0;
  for (int b = b0; b < b1; ++b) local += lb_load<LDS>(cnt + b);
  int total;
  int run = wg_exclusive_scan<NT>(local, wsum, &total);
  for (int b = b0; b < b1; ++b) {
    const int c = lb_load<LDS>(cnt + b);
    lbeg[b] = run;
    cnt[b] = run;  // becomes the block's fill cursor
    run += c;
  }
  if (t == 0) lbeg[nb] = total;
  lb_sync<LDS>();
  for (int q = t; q < m; q += NT) {
    const int lab = lkeys[q];
    if (lab >= 0 && lab < L) {
      const int pos = atomicAdd(&cnt[lab >> 5], 1);
      lpair[pos] = (lrow[q] << 5) | (lab & 31);
    }
  }
}

}  // namespace asgd
