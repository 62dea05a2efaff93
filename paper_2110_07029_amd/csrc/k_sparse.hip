// Sparse first-layer gradient and update: dW1[f] = sum over the batch entries
// (i, f, x) of x * dA1[i], applied only to the features present in the batch
// (the update pass of Sec. 2.1 restricted to the rows the sparse input
// touches), plus the hidden-layer bias update and the batch's mean loss.
// Entries are grouped by the radix sort, so each distinct feature is one
// contiguous segment, summed in ascending (row, position) order: deterministic,
// no atomics.
#include <limits.h>

#include <hip/hip_ext.h>

#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

constexpr int SPU_THREADS = 256;
constexpr int SPU_WAVES = SPU_THREADS / 64;

// db1 = sum_i dA1[i]; b1 -= lr db1; loss = mean_i loss_rows[i]: one workgroup,
// 8 groups of 32 threads x 4 hidden units, rows summed in a fixed order.
__device__ void hidden_bias_wg(int B, const float* __restrict__ dA1, float* __restrict__ b1, float lr,
                               const float* __restrict__ loss_rows, float* __restrict__ loss) {
  constexpr int GROUPS = SPU_THREADS / 32;
  __shared__ float red[GROUPS][HID];
  __shared__ float red_l[SPU_WAVES];
  const int t = threadIdx.x, grp = t >> 5, h4 = (t & 31) * 4;
  float4 s = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll 8
  for (int i = grp; i < B; i += GROUPS) {
    const float4 v = *reinterpret_cast<const float4*>(dA1 + (size_t)i * HID + h4);
    s.x += v.x;
    s.y += v.y;
    s.z += v.z;
    s.w += v.w;
  }
  *reinterpret_cast<float4*>(&red[grp][h4]) = s;
  float ls = 0.0f;
  for (int i = t; i < B; i += SPU_THREADS) ls += loss_rows[i];
  ls = wave_sum(ls);
  if ((t & 63) == 0) red_l[t >> 6] = ls;
  __syncthreads();
  if (t < HID) {
    float tot = red[0][t];
#pragma unroll
    for (int k = 1; k < GROUPS; ++k) tot += red[k][t];
    b1[t] = fmaf(-lr, tot, b1[t]);
  }
  if (t == 0) {
    float l = red_l[0];
    for (int k = 1; k < SPU_WAVES; ++k) l += red_l[k];
    *loss = l / (float)B;
  }
}

// Two launches, one wavefront per window of SPU_WIN consecutive sorted
// entries.  Pieces: the wave sums each run of equal keys inside its window in
// entry order (lanes hold hidden units 2*lane, 2*lane+1; the dA1 and W1 rows
// of all the window's entries are loaded together, an entry's W1 row being its
// feature's).  A segment that lies inside the window is applied to W1 at once;
// the piece that continues a segment from the previous window goes to
// part[2w] and the piece that starts a segment running past the window's end
// to part[2w + 1].  Join: the wave whose window holds the head of such a
// segment finds how many windows it spans (one lane per window), adds their
// continuing pieces to its own in window order and applies the sum.  The
// summation order is fixed (entry order inside a piece, window order across
// pieces), so results do not depend on scheduling, and a long segment (a
// feature in most rows) costs every wave at most one window of entries.  The
// last workgroup of the first launch updates b1 and the loss.
constexpr int SPU_WIN = 32;
constexpr int SPU_BATCH = 16;  // entries whose dA1 and W1 rows are loaded together
int sparse_windows(int n_keys) { return (n_keys + SPU_WIN - 1) / SPU_WIN; }

__global__ __launch_bounds__(SPU_THREADS) void k_sparse_pieces(
    float* __restrict__ W1, int F, const int32_t* __restrict__ skeys, const int32_t* __restrict__ svals,
    int n_keys, const int32_t* __restrict__ row_of, CsrDev x, const float* __restrict__ dA1, float lr, int B,
    float* __restrict__ b1, const float* __restrict__ loss_rows, float* __restrict__ loss,
    float* __restrict__ part, int n_win_blocks) {
  if ((int)blockIdx.x == n_win_blocks) {
    hidden_bias_wg(B, dA1, b1, lr, loss_rows, loss);
    return;
  }
  const int lane = threadIdx.x & 63;
  const int win = blockIdx.x * SPU_WAVES + (threadIdx.x >> 6);
  const int w0 = win * SPU_WIN;
  if (w0 >= n_keys) return;
  // lanes 0..SPU_WIN-1: the window's entries; lane SPU_WIN: the next window's first
  const int q = w0 + lane;
  const int key = lane <= SPU_WIN && q < n_keys ? skeys[q] : INT_MAX;  // invalid ids (>= F) sort last
  if (__builtin_amdgcn_readfirstlane(key) >= F) return;
  const int before = w0 > 0 ? skeys[w0 - 1] : -1;
  const int kn = __shfl_down(key, 1);
  const bool valid = lane < SPU_WIN && key < F;
  // last entry of a run inside the window (at the window's end a run may go on)
  const bool last = valid && (kn != key || lane == SPU_WIN - 1);
  const bool runs_on = __shfl(key, SPU_WIN) == __shfl(key, SPU_WIN - 1);  // for the window's last run
  const bool first_cont = __shfl(key, 0) == before;  // the window starts inside a segment
  int row = 0;
  float xv = 0.0f;
  if (valid) {
    const int p = svals[q];
    row = row_of[p];
    xv = x.values[x.indptr[0] + p];
  }
  const int cnt = __popcll(__ballot(valid));  // valid entries are a prefix of the window
  // dA1 and W1 rows through buffer resources: the row offset is a scalar, the
  // lane's 8 bytes a fixed vector offset, so a load needs no address registers
  const __amdgpu_buffer_rsrc_t rd =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(dA1), (short)0, B * HID * 4, BUF_RSRC_WORD3);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(W1, (short)0, F * HID * 4, BUF_RSRC_WORD3);
  const int voff = lane * 8;
  float2* Wl = reinterpret_cast<float2*>(W1) + lane;
  float2* P = reinterpret_cast<float2*>(part) + lane;
  float2 acc = make_float2(0.0f, 0.0f);
  bool in_first = first_cont;  // the current run continues a segment from the previous window
  // two batches of SPU_BATCH entries: few enough registers for the kernel to
  // share a SIMD with the output-layer backward it overlaps
#pragma unroll 1
  for (int u = 0; u < cnt; u += SPU_BATCH) {
    int rk[SPU_BATCH], fk[SPU_BATCH], lk[SPU_BATCH];
    float xk[SPU_BATCH];
    float2 d[SPU_BATCH], w[SPU_BATCH];
#pragma unroll
    for (int k = 0; k < SPU_BATCH; ++k) {
      rk[k] = __builtin_amdgcn_readlane(row, u + k);
      fk[k] = __builtin_amdgcn_readlane(valid ? key : 0, u + k);
      lk[k] = __builtin_amdgcn_readlane((int)last, u + k);
      xk[k] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, xv), u + k));
    }
    // entries past cnt read dA1 row 0 and W1 row 0 and are discarded
#pragma unroll
    for (int k = 0; k < SPU_BATCH; ++k) {
      d[k] = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(rd, voff, rk[k] * (HID * 4), 0));
      w[k] = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(rw, voff, fk[k] * (HID * 4), 0));
    }
#pragma unroll
    for (int k = 0; k < SPU_BATCH; ++k) {
      const int e = u + k;
      if (e < cnt) {
        acc.x = fmaf(xk[k], d[k].x, acc.x);
        acc.y = fmaf(xk[k], d[k].y, acc.y);
        if (lk[k]) {
          if (in_first)
            P[(size_t)(2 * win) * (HID / 2)] = acc;
          else if (e == SPU_WIN - 1 && runs_on)
            P[(size_t)(2 * win + 1) * (HID / 2)] = acc;
          else
            Wl[(size_t)fk[k] * (HID / 2)] = make_float2(fmaf(-lr, acc.x, w[k].x), fmaf(-lr, acc.y, w[k].y));
          acc = make_float2(0.0f, 0.0f);
          in_first = false;
        }
      }
    }
  }
}

constexpr int JOIN_BATCH = 16;  // continuing pieces loaded together

__global__ __launch_bounds__(SPU_THREADS) void k_sparse_join(float* __restrict__ W1, int F,
                                                              const int32_t* __restrict__ skeys, int n_keys,
                                                              float lr, const float* __restrict__ part) {
  const int lane = threadIdx.x & 63;
  const int win = blockIdx.x * SPU_WAVES + (threadIdx.x >> 6);
  const int w0 = win * SPU_WIN;
  // this window's last entry starts or continues a segment that runs past it ...
  if (w0 + SPU_WIN >= n_keys) return;
  const int f = skeys[w0 + SPU_WIN - 1];
  if (f >= F || skeys[w0 + SPU_WIN] != f) return;
  // ... and the segment's head lies in this window (else an earlier wave joins it)
  if (skeys[w0] == f && w0 > 0 && skeys[w0 - 1] == f) return;
  // windows win+1 .. win+m hold the rest: window v is followed by another piece
  // when it is all f and the next window starts with f (one lane per window)
  int m = 0;
  for (;;) {
    const int v1 = (win + 2 + m + lane) * SPU_WIN;  // first entry after window win+1+m+lane
    const bool more = v1 < n_keys && skeys[v1] == f && skeys[v1 - 1] == f;
    const uint64_t stop = __ballot(!more);
    if (stop) {
      m += __builtin_ctzll(stop) + 1;
      break;
    }
    m += 64;
  }
  const float2* P = reinterpret_cast<const float2*>(part) + lane;
  float2 acc = P[(size_t)(2 * win + 1) * (HID / 2)];
  for (int v0 = 0; v0 < m; v0 += JOIN_BATCH) {
    float2 c[JOIN_BATCH];
#pragma unroll
    for (int k = 0; k < JOIN_BATCH; ++k)
      c[k] = P[(size_t)(2 * (win + 1 + min(v0 + k, m - 1))) * (HID / 2)];
#pragma unroll
    for (int k = 0; k < JOIN_BATCH; ++k)
      if (v0 + k < m) {
        acc.x += c[k].x;
        acc.y += c[k].y;
      }
  }
  float2* wp = reinterpret_cast<float2*>(W1 + (size_t)f * HID) + lane;
  const float2 w = *wp;
  *wp = make_float2(fmaf(-lr, acc.x, w.x), fmaf(-lr, acc.y, w.y));
}

hipError_t launch_sparse_update(float* W1, int F, const int32_t* skeys, const int32_t* svals, int n_keys,
                                const int32_t* row_of, const CsrDev& x, const float* dA1, float lr, int B,
                                float* b1, const float* loss_rows, float* loss, float* part, hipStream_t st,
                                hipEvent_t done) {
  const int nwin = n_keys > 0 ? sparse_windows(n_keys) : 0;
  const int nwb = (nwin + SPU_WAVES - 1) / SPU_WAVES;
  // the last launch completes `done`
  const bool join = nwin > 1;
  const dim3 gp(nwb + 1), gj(nwb), blk(SPU_THREADS);
  if (done && !join)
    hipExtLaunchKernelGGL(k_sparse_pieces, gp, blk, 0, st, nullptr, done, 0, W1, F, skeys, svals, n_keys, row_of, x,
                          dA1, lr, B, b1, loss_rows, loss, part, nwb);
  else
    hipLaunchKernelGGL(k_sparse_pieces, gp, blk, 0, st, W1, F, skeys, svals, n_keys, row_of, x, dA1, lr, B, b1,
                       loss_rows, loss, part, nwb);
  if (join) {
    if (done)
      hipExtLaunchKernelGGL(k_sparse_join, gj, blk, 0, st, nullptr, done, 0, W1, F, skeys, n_keys, lr,
                            (const float*)part);
    else
      hipLaunchKernelGGL(k_sparse_join, gj, blk, 0, st, W1, F, skeys, n_keys, lr, (const float*)part);
  }
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
