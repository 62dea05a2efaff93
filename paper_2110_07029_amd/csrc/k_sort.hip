// Stable LSD radix sort of int32 keys with their original positions as the
// payload.  It orders the batch's feature entries so that the sparse W1
// gradient becomes a segmented reduction over equal feature ids (no contended
// atomics, fixed summation order).
//
// One pass over a digit of up to 11 bits = three launches:
//   hist    : per-workgroup digit counts of a 1024-key chunk (LDS counters),
//             stored block-major: hist[block][digit]
//   scan    : exclusive scan over (digit, workgroup) -> global scatter offsets,
//             every read and write coalesced across the digits
//   scatter : stable ranks inside the chunk from 64-lane ballots (lanes with the
//             same digit in one wave), per-wave running counts, then a prefix
//             over the four waves; keys land at offset + rank.
// hist and scatter size their LDS counters by the pass's digit width (dynamic
// LDS, 4 << bits and 16 << bits bytes), not by the widest digit: a narrow pass
// then fits on a CU beside the output-layer kernels of the other stream.
#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

constexpr int SORT_THREADS = 256;
constexpr int SORT_WAVES = SORT_THREADS / 64;
constexpr int SORT_PER_WAVE = SORT_CHUNK / SORT_WAVES;  // 256
constexpr int SORT_ITERS = SORT_PER_WAVE / 64;         // 4

int sort_blocks(int n) { return (n + SORT_CHUNK - 1) / SORT_CHUNK; }

__global__ __launch_bounds__(SORT_THREADS) void k_sort_hist(const int32_t* __restrict__ keys, int n,
                                                            int shift, int nbits, int nblk,
                                                            int32_t* __restrict__ hist) {
  extern __shared__ int cnt[];  // 1 << nbits counters
  const int nd = 1 << nbits;
  for (int d = threadIdx.x; d < nd; d += SORT_THREADS) cnt[d] = 0;
  __syncthreads();
  const int b0 = blockIdx.x * SORT_CHUNK;
  for (int t = threadIdx.x; t < SORT_CHUNK; t += SORT_THREADS) {
    const int p = b0 + t;
    if (p < n) atomicAdd(&cnt[(keys[p] >> shift) & (nd - 1)], 1);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < nd; d += SORT_THREADS) hist[blockIdx.x * nd + d] = cnt[d];
}

// Scatter offsets offs[b * ndig + d] = (keys with a smaller digit) + (keys with
// digit d in earlier chunks), by one workgroup: thread t owns digits t and
// t + SCAN_THREADS; per chunk b, the threads read consecutive digits (one
// coalesced row of hist), and one block-wide exclusive scan of the per-digit
// totals gives every digit's base.
constexpr int SCAN_THREADS = 1024;
constexpr int SCAN_DPT = (1 << SORT_MAX_BITS) / SCAN_THREADS;  // digits per thread
constexpr int SCAN_BATCH = 16;  // chunk counts loaded together

__global__ __launch_bounds__(SCAN_THREADS) void k_sort_scan(const int32_t* __restrict__ hist,
                                                            int nblk, int ndig,
                                                            int32_t* __restrict__ offs) {
  __shared__ int wsum[SCAN_THREADS / 64];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  // (the chunks' counts are read SCAN_BATCH at a time, all loads in flight
  // before the first sum)
  int tot[SCAN_DPT];
#pragma unroll
  for (int k = 0; k < SCAN_DPT; ++k) tot[k] = 0;
#pragma unroll
  for (int k = 0; k < SCAN_DPT; ++k) {
    const int d = t + k * SCAN_THREADS;
    if (d >= ndig) continue;
    for (int b0 = 0; b0 < nblk; b0 += SCAN_BATCH) {
      int c[SCAN_BATCH];
#pragma unroll
      for (int j = 0; j < SCAN_BATCH; ++j) c[j] = b0 + j < nblk ? hist[(size_t)(b0 + j) * ndig + d] : 0;
#pragma unroll
      for (int j = 0; j < SCAN_BATCH; ++j) tot[k] += c[j];
    }
  }
  // digits in order d = t + k * SCAN_THREADS: scan the block once per k
  int carry = 0;
#pragma unroll
  for (int k = 0; k < SCAN_DPT; ++k) {
    int x = tot[k];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    if (w == 0) {
      int v = lane < SCAN_THREADS / 64 ? wsum[lane] : 0;
#pragma unroll
      for (int o = 1; o < SCAN_THREADS / 64; o <<= 1) {
        const int y = __shfl_up(v, o);
        if (lane >= o) v += y;
      }
      if (lane < SCAN_THREADS / 64) wsum[lane] = v;
    }
    __syncthreads();
    const int base = carry + (w > 0 ? wsum[w - 1] : 0) + x - tot[k];
    carry += wsum[SCAN_THREADS / 64 - 1];
    __syncthreads();
    tot[k] = base;  // becomes the running offset of digit t + k * SCAN_THREADS
  }
#pragma unroll
  for (int k = 0; k < SCAN_DPT; ++k) {
    const int d = t + k * SCAN_THREADS;
    if (d >= ndig) continue;
    for (int b0 = 0; b0 < nblk; b0 += SCAN_BATCH) {
      int c[SCAN_BATCH];
#pragma unroll
      for (int j = 0; j < SCAN_BATCH; ++j) c[j] = b0 + j < nblk ? hist[(size_t)(b0 + j) * ndig + d] : 0;
#pragma unroll
      for (int j = 0; j < SCAN_BATCH; ++j)
        if (b0 + j < nblk) {
          offs[(size_t)(b0 + j) * ndig + d] = tot[k];
          tot[k] += c[j];
        }
    }
  }
}

__global__ __launch_bounds__(SORT_THREADS) void k_sort_scatter(
    const int32_t* __restrict__ keys_in, const int32_t* __restrict__ vals_in, int n, int shift,
    int nbits, int nblk, const int32_t* __restrict__ offs, int32_t* __restrict__ keys_out,
    int32_t* __restrict__ vals_out) {
  extern __shared__ int wcnt_lds[];  // SORT_WAVES x (1 << nbits) counters
  const int nd = 1 << nbits;
  auto wcnt = [&](int ww, int d) -> int& { return wcnt_lds[ww * nd + d]; };
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int d = lane; d < nd; d += 64) wcnt(w, d) = 0;
  __syncthreads();
  const int p0 = blockIdx.x * SORT_CHUNK + w * SORT_PER_WAVE;
  const uint64_t below = (1ull << lane) - 1ull;
  int key[SORT_ITERS], val[SORT_ITERS], rank[SORT_ITERS];
#pragma unroll
  for (int it = 0; it < SORT_ITERS; ++it) {
    const int p = p0 + it * 64 + lane;
    const bool valid = p < n;
    const int k = valid ? keys_in[p] : 0;
    key[it] = k;
    val[it] = valid ? (vals_in ? vals_in[p] : p) : 0;
    const int d = (k >> shift) & (nd - 1);
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (d >> b) & 1;
      const uint64_t bal = __ballot(bit);
      peers &= bit ? bal : ~bal;
    }
    const int before = __popcll(peers & below);
    const int c = wcnt(w, d);  // every peer reads the count before the leader updates it
    rank[it] = c + before;
    if (valid && before == 0) wcnt(w, d) = c + __popcll(peers);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < nd; d += SORT_THREADS) {
    int run = 0;
#pragma unroll
    for (int ww = 0; ww < SORT_WAVES; ++ww) {
      const int c = wcnt(ww, d);
      wcnt(ww, d) = run;
      run += c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < SORT_ITERS; ++it) {
    const int p = p0 + it * 64 + lane;
    if (p < n) {
      const int d = (key[it] >> shift) & (nd - 1);
      const int pos = offs[blockIdx.x * nd + d] + wcnt(w, d) + rank[it];
      keys_out[pos] = key[it];
      vals_out[pos] = val[it];
    }
  }
}

hipError_t launch_sort(const int32_t* keys_in, int n, int key_bits, int32_t* keys_a,
                       int32_t* vals_a, int32_t* keys_b, int32_t* vals_b, int32_t* hist,
                       const int32_t** keys_out, const int32_t** vals_out, hipStream_t st) {
  *keys_out = keys_a;
  *vals_out = vals_a;
  if (n <= 0) return hipSuccess;
  if (key_bits < 1) key_bits = 1;
  const int npass = (key_bits + SORT_MAX_BITS - 1) / SORT_MAX_BITS;
  const int bits = (key_bits + npass - 1) / npass;
  const int nblk = sort_blocks(n);
  int32_t* offs = hist + ((size_t)nblk << SORT_MAX_BITS);
  const int32_t* kin = keys_in;
  const int32_t* vin = nullptr;
  int32_t* kout = keys_a;
  int32_t* vout = vals_a;
  for (int pass = 0; pass < npass; ++pass) {
    const int shift = pass * bits;
    const int nb = key_bits - shift < bits ? key_bits - shift : bits;
    hipLaunchKernelGGL(k_sort_hist, dim3(nblk), dim3(SORT_THREADS), (size_t)4 << nb, st, kin, n,
                       shift, nb, nblk, hist);
    hipLaunchKernelGGL(k_sort_scan, dim3(1), dim3(SCAN_THREADS), 0, st, hist, nblk, 1 << nb, offs);
    hipLaunchKernelGGL(k_sort_scatter, dim3(nblk), dim3(SORT_THREADS),
                       (size_t)SORT_WAVES * 4 << nb, st, kin, vin, n, shift, nb, nblk, offs, kout,
                       vout);
    *keys_out = kout;
    *vals_out = vout;
    kin = kout;
    vin = vout;
    kout = (kout == keys_a) ? keys_b : keys_a;
    vout = (vout == vals_a) ? vals_b : vals_a;
  }
  return hipGetLastError();
}

}  // namespace asgd
