// First layer: CSR batch times W1 as coalesced row gathers (sparse input layer
// of the paper's MLP, Sec. 5.1), plus the per-entry sort keys used by the
// backward pass and the model initialisation.
#include <hip/hip_ext.h>

#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

// ---------------------------------------------------------------------------
// Xavier-uniform init from the counter-based splitmix64 stream.
// ---------------------------------------------------------------------------
__global__ void k_init_uniform(float* __restrict__ w, int64_t count, uint64_t key, float bound) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count; e += stride) {
    uint64_t z = (uint64_t)e ^ key;
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    const float u = (float)(uint32_t)(z >> 40) * 0x1p-24f;  // exact: 24-bit grid
    const float t = 2.0f * u - 1.0f;                          // exact in float32
    w[e] = t * bound;                                         // the only rounding
  }
}

hipError_t launch_init_uniform(float* w, int64_t count, uint64_t key, float bound, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_init_uniform, dim3((unsigned)blocks), dim3(256), 0, st, w, count, key, bound);
  return hipGetLastError();
}

__global__ void k_fill_int(int32_t* p, int32_t v, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) p[e] = v;
}

hipError_t launch_fill_int(int32_t* p, int32_t v, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill_int, dim3((unsigned)blocks), dim3(256), 0, st, p, v, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// A1[i] = b1 + sum_{(f, v) in row i} v * W1[f];  H1 = max(A1, 0).
// One workgroup per sample row; for batches whose rows average
// GATHER_LONG_ROW entries or more, GATHER_SPLIT workgroups per row, each
// writing its partial sum, and a second launch adds them (the step time
// follows the longest row, which then spreads over several CUs).  Lane l owns
// hidden units 2l and 2l+1, so every W1 row is one coalesced 512-byte access.
// The row's entries are split into one contiguous range per wavefront; a wavefront
// loads up to 64 (id, value) pairs at once (one per lane, also writing their
// sort keys), broadcasts them with readlane and issues 16 W1 row loads before
// the first is used.  Lanes past the range carry id -1, so a partial group of
// 16 costs one round trip like a full one (the step time follows the longest
// row of the batch, and nnz per row is heavy-tailed).  The partial sums are
// added in wavefront order (then in workgroup order), then b1.
// ---------------------------------------------------------------------------
// Short rows: four wavefronts (one per SIMD), so that the workgroup can start
// on a CU where the output-layer backward leaves room for only one more
// wavefront per SIMD, which is where the next step's gather runs when the
// step is pipelined.  Long rows (split over workgroups; the gather then runs
// alone on the model's stream): eight.
constexpr int gather_waves(int split) { return split > 1 ? 8 : 4; }
constexpr int GATHER_UNROLL = 16;
static_assert(64 % GATHER_UNROLL == 0, "readlane indices stay below 64");

template <bool BF16, int SPLIT>
__global__ __launch_bounds__(64 * gather_waves(SPLIT)) void k_gather_fwd(
    CsrDev x, CsrDev y, int has_y, const float* __restrict__ W1, const float* __restrict__ b1,
    int F, int L, float* __restrict__ A1, typename Mma<BF16>::elem* __restrict__ H1,
    typename Mma<BF16>::elem* __restrict__ H1T, int rows_pad, int ld_t, int32_t* __restrict__ keys,
    int32_t* __restrict__ row_of, int32_t* __restrict__ lkeys, int32_t* __restrict__ lrow,
    float* __restrict__ rw,
    int32_t* __restrict__ err, int validate, float* __restrict__ gpart) {
  using E = typename Mma<BF16>::elem;
  constexpr int WAVES = gather_waves(SPLIT);
  __shared__ float2 part[WAVES][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = (int)blockIdx.x / SPLIT, piece = (int)blockIdx.x % SPLIT;
  const int h0 = 2 * lane;
  if (i >= x.n_rows) {  // padding rows of the output-layer operands are zero
    if (wave == 0 && piece == 0) {
      H1[(size_t)i * HID + h0] = (E)0.0f;
      H1[(size_t)i * HID + h0 + 1] = (E)0.0f;
      if constexpr (!BF16) {  // the transposed copy is read only by the fp32 backward
        H1T[(size_t)h0 * ld_t + i] = (E)0.0f;
        H1T[(size_t)(h0 + 1) * ld_t + i] = (E)0.0f;
      }
    }
    return;
  }
  int bad = 0;
  const int base = x.indptr[0];
  int s = x.indptr[i], e = x.indptr[i + 1];
  if (s < base || e > base + x.nnz || e < s) {
    bad |= ERR_INDPTR;
    s = max(s, base);
    e = min(e, base + x.nnz);
    if (e < s) e = s;
  }
  // wavefront gw of the row's SPLIT * WAVES takes the gw-th contiguous range
  const int gw = piece * WAVES + wave;
  const int per = (e - s + SPLIT * WAVES - 1) / (SPLIT * WAVES);
  const int ws = min(e, s + gw * per), we = min(e, ws + per);
  float2 acc = make_float2(0.0f, 0.0f);
  for (int p0 = ws; p0 < we; p0 += 64) {
    const int p = p0 + lane;
    int f = -1;
    float v = 0.0f;
    if (p < we) {
      f = x.indices[p];
      v = x.values[p];
      int key = f;
      if (f < 0 || f >= F) {
        bad |= ERR_FEATURE_ID;
        key = F;  // sorts after every feature; the W1 update skips it
        f = -1;
      } else if (validate && p > s && x.indices[p - 1] >= f) {
        bad |= ERR_DUPLICATE;
      }
      keys[p - base] = key;
      row_of[p - base] = i;
    }
    const int cnt = min(64, we - p0);
    for (int j = 0; j < cnt; j += GATHER_UNROLL) {
      int fj[GATHER_UNROLL];
      float vj[GATHER_UNROLL];
      float2 wv[GATHER_UNROLL];
#pragma unroll
      for (int u = 0; u < GATHER_UNROLL; ++u) {
        fj[u] = __builtin_amdgcn_readlane(f, j + u);
        vj[u] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), j + u));
      }
#pragma unroll
      for (int u = 0; u < GATHER_UNROLL; ++u)  // id -1 (padding, invalid) reads row 0, discarded below
        wv[u] = *reinterpret_cast<const float2*>(W1 + (size_t)max(fj[u], 0) * HID + h0);
#pragma unroll
      for (int u = 0; u < GATHER_UNROLL; ++u) {
        if (fj[u] >= 0) {
          acc.x = fmaf(vj[u], wv[u].x, acc.x);
          acc.y = fmaf(vj[u], wv[u].y, acc.y);
        }
      }
    }
  }
  part[wave][lane] = acc;

  if (has_y && piece == 0 && wave == WAVES - 1) {
    const int ybase = y.indptr[0];
    int ys = y.indptr[i], ye = y.indptr[i + 1];
    if (ys < ybase || ye > ybase + y.nnz || ye < ys) {
      bad |= ERR_INDPTR;
      ys = max(ys, ybase);
      ye = min(ye, ybase + y.nnz);
      if (ye < ys) ye = ys;
    }
    if (ye == ys) bad |= ERR_EMPTY_LABELS;
    if (lane == 0) rw[i] = ye > ys ? 1.0f / (float)(ye - ys) : 0.0f;
    for (int q = ys + lane; q < ye; q += 64) {
      const int lab = y.indices[q];
      int key = lab;
      if (lab < 0 || lab >= L) {
        bad |= ERR_LABEL_ID;
        key = L;  // dropped when the pairs are grouped by label block
      } else if (validate && q > ys && y.indices[q - 1] >= lab) {
        bad |= ERR_DUPLICATE;
      }
      lkeys[q - ybase] = key;
      lrow[q - ybase] = i;
    }
  }
  if (bad) atomicOr(err, bad);
  __syncthreads();
  if (wave == 0) {
    float2 a = part[0][lane];
#pragma unroll
    for (int k = 1; k < WAVES; ++k) {
      a.x += part[k][lane].x;
      a.y += part[k][lane].y;
    }
    if constexpr (SPLIT > 1) {
      *reinterpret_cast<float2*>(gpart + ((size_t)piece * ld_t + i) * HID + h0) = a;
      return;
    }
    const float2 bb = *reinterpret_cast<const float2*>(b1 + h0);
    a.x = bb.x + a.x;
    a.y = bb.y + a.y;
    *reinterpret_cast<float2*>(A1 + (size_t)i * HID + h0) = a;
    const float r0 = fmaxf(a.x, 0.0f), r1 = fmaxf(a.y, 0.0f);
    H1[(size_t)i * HID + h0] = (E)r0;
    H1[(size_t)i * HID + h0 + 1] = (E)r1;
    if constexpr (!BF16) {
      H1T[(size_t)h0 * ld_t + i] = (E)r0;
      H1T[(size_t)(h0 + 1) * ld_t + i] = (E)r1;
    }
  }
}

// Rows split over GATHER_SPLIT workgroups: A1 = b1 + the pieces' sums in
// piece order, then H1 (and H1^T for fp32 operands) as above.
template <bool BF16>
__global__ __launch_bounds__(64) void k_gather_finish(int n_rows, const float* __restrict__ gpart, int ld_t,
                                                      const float* __restrict__ b1, float* __restrict__ A1,
                                                      typename Mma<BF16>::elem* __restrict__ H1,
                                                      typename Mma<BF16>::elem* __restrict__ H1T) {
  using E = typename Mma<BF16>::elem;
  const int i = blockIdx.x, h0 = 2 * threadIdx.x;
  if (i >= n_rows) return;
  float2 a = *reinterpret_cast<const float2*>(gpart + (size_t)i * HID + h0);
#pragma unroll
  for (int k = 1; k < GATHER_SPLIT; ++k) {
    const float2 v = *reinterpret_cast<const float2*>(gpart + ((size_t)k * ld_t + i) * HID + h0);
    a.x += v.x;
    a.y += v.y;
  }
  const float2 bb = *reinterpret_cast<const float2*>(b1 + h0);
  a.x = bb.x + a.x;
  a.y = bb.y + a.y;
  *reinterpret_cast<float2*>(A1 + (size_t)i * HID + h0) = a;
  const float r0 = fmaxf(a.x, 0.0f), r1 = fmaxf(a.y, 0.0f);
  H1[(size_t)i * HID + h0] = (E)r0;
  H1[(size_t)i * HID + h0 + 1] = (E)r1;
  if constexpr (!BF16) {
    H1T[(size_t)h0 * ld_t + i] = (E)r0;
    H1T[(size_t)(h0 + 1) * ld_t + i] = (E)r1;
  }
}

hipError_t launch_gather_fwd(bool use_bf16, const CsrDev& x, const CsrDev* y, const float* W1,
                             const float* b1, int F, int L, float* A1, void* H1, void* H1T,
                             int rows_pad, int ld_t, int32_t* keys, int32_t* row_of,
                             int32_t* lkeys, int32_t* lrow, float* rw, int32_t* err, int validate,
                             float* gpart, hipStream_t st, hipEvent_t done) {
  CsrDev yy = y ? *y : CsrDev{0, 0, 0, nullptr, nullptr, nullptr};
  const bool split = gpart && x.n_rows > 0 && (int64_t)x.nnz >= (int64_t)GATHER_LONG_ROW * x.n_rows;
  // the last launch completes `done`
  auto go = [&](auto kern, int pieces, auto* h1, auto* h1t, hipEvent_t ev) {
    const dim3 grid(rows_pad * pieces), block(64 * gather_waves(pieces));
    const int has_y = y != nullptr;
    if (ev)
      hipExtLaunchKernelGGL(kern, grid, block, 0, st, nullptr, ev, 0, x, yy, has_y, W1, b1, F, L, A1, h1, h1t,
                            rows_pad, ld_t, keys, row_of, lkeys, lrow, rw, err, validate, gpart);
    else
      hipLaunchKernelGGL(kern, grid, block, 0, st, x, yy, has_y, W1, b1, F, L, A1, h1, h1t, rows_pad, ld_t, keys,
                         row_of, lkeys, lrow, rw, err, validate, gpart);
  };
  auto finish = [&](auto kern, auto* h1, auto* h1t) {
    if (done)
      hipExtLaunchKernelGGL(kern, dim3(x.n_rows), dim3(64), 0, st, nullptr, done, 0, x.n_rows,
                            (const float*)gpart, ld_t, b1, A1, h1, h1t);
    else
      hipLaunchKernelGGL(kern, dim3(x.n_rows), dim3(64), 0, st, x.n_rows, (const float*)gpart, ld_t, b1, A1, h1,
                         h1t);
  };
  if (use_bf16) {
    if (split) {
      go(k_gather_fwd<true, GATHER_SPLIT>, GATHER_SPLIT, (bf16*)H1, (bf16*)H1T, nullptr);
      finish(k_gather_finish<true>, (bf16*)H1, (bf16*)H1T);
    } else {
      go(k_gather_fwd<true, 1>, 1, (bf16*)H1, (bf16*)H1T, done);
    }
  } else {
    if (split) {
      go(k_gather_fwd<false, GATHER_SPLIT>, GATHER_SPLIT, (float*)H1, (float*)H1T, nullptr);
      finish(k_gather_finish<false>, (float*)H1, (float*)H1T);
    } else {
      go(k_gather_fwd<false, 1>, 1, (float*)H1, (float*)H1T, done);
    }
  }
  return hipGetLastError();
}

}  // namespace asgd
