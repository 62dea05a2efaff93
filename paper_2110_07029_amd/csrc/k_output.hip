// Output layer of the sparse MLP (Sec. 5.1): Z = H1 W2^T + b2 over L labels,
// softmax + multi-label cross-entropy, its gradient and the SGD update of W2
// and b2 (Sec. 2.1), and top-k prediction.  Logits are never stored.
//
// Forward (k_out_fwd_train): workgroup = (label split, block of rows).  For
// every 32-label tile: Z^T = W2_tile H1^T on the matrix cores; a single-pass
// online max / sum of exponentials per row; and, with the same
// probabilities, O^T += W2_tile^T P^T.  O/s is sum_l softmax(Z)_l W2[l], the
// dense part of dH1 = (P - T) W2 / B, so the backward never needs a second
// pass over W2 for dH1.  Rows are the N dimension of both products, so all
// per-row state (running max, rescale factor) is per lane.
// Combine (k_out_combine): merges the splits of a row (log-sum-exp, loss,
// dH1 = (O/s - mean_{y in Y_i} W2[y]) / B, dA1 = dH1 * [A1 > 0]).
// Backward (k_out_bwd): workgroup = 128 labels; recompute Z per 32-row block,
// dZ = (softmax - T)/B, dW2 = dZ^T H1, db2 = colsum dZ, and update the fp32
// master W2 / b2 in place from the registers the lane loaded.
#include <float.h>
#include <math.h>

#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <bool BF16>
struct FwdShape {
  static constexpr int NB = BF16 ? 2 : 1;     // 32-row blocks per wave
  static constexpr int RB = 4 * 32 * NB;      // rows per workgroup
  static constexpr int WR = BF16 ? 136 : 132; // leading dim of the row-major tile (elements)
  static constexpr int WT = 36;               // leading dim of the transposed tile (elements)
};

int out_rows_per_block(bool use_bf16) { return use_bf16 ? FwdShape<true>::RB : FwdShape<false>::RB; }

// Cooperative load of one 32-label tile of W2 (fp32 in HBM) by 256 threads:
// thread t reads hidden chunk 4*(t%32) of labels 2a, 2a+1, 2a+16, 2a+17
// (a = t/32), so every load instruction reads whole 512-byte label rows.
struct TileRegs {
  float4 v[4];
  float bias;
};

__device__ __forceinline__ void tile_load(const float* __restrict__ W2, const float* __restrict__ b2,
                                          int L, int tile, TileRegs& r) {
  const int tid = threadIdx.x, a = tid >> 5, q = tid & 31;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int lab = tile * OUT_TILE + 2 * a + (it & 1) + 16 * (it >> 1);
    r.v[it] = lab < L ? *reinterpret_cast<const float4*>(W2 + (size_t)lab * HID + 4 * q)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const int lb = tile * OUT_TILE + tid;
  r.bias = (tid < OUT_TILE && lb < L) ? b2[lb] : 0.0f;
}

template <bool BF16, bool TRANSPOSED>
__device__ __forceinline__ void tile_store(const TileRegs& r, typename Mma<BF16>::elem* wr,
                                           typename Mma<BF16>::elem* wt, float* bt) {
  using E = typename Mma<BF16>::elem;
  constexpr int WR = FwdShape<BF16>::WR, WT = FwdShape<BF16>::WT;
  const int tid = threadIdx.x, a = tid >> 5, q = tid & 31;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int ll = 2 * a + (it & 1) + 16 * (it >> 1);
    E* d = wr + ll * WR + 4 * q;
    if constexpr (BF16) {
      bf16x4 p;
      p[0] = (bf16)r.v[it].x; p[1] = (bf16)r.v[it].y; p[2] = (bf16)r.v[it].z; p[3] = (bf16)r.v[it].w;
      *reinterpret_cast<bf16x4*>(d) = p;
    } else {
      *reinterpret_cast<float4*>(d) = r.v[it];
    }
  }
  if constexpr (TRANSPOSED) {
#pragma unroll
    for (int pr = 0; pr < 2; ++pr) {
      const int ll = 2 * a + 16 * pr;  // even label of the pair
      const float4 x0 = r.v[2 * pr], x1 = r.v[2 * pr + 1];
      const float a0[4] = {x0.x, x0.y, x0.z, x0.w}, a1[4] = {x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        E* d = wt + (4 * q + k) * WT + ll;
        if constexpr (BF16) {
          bf16x2 p;
          p[0] = (bf16)a0[k];
          p[1] = (bf16)a1[k];
          *reinterpret_cast<bf16x2*>(d) = p;
        } else {
          *reinterpret_cast<float2*>(d) = make_float2(a0[k], a1[k]);
        }
      }
    }
  }
  if (threadIdx.x < OUT_TILE) bt[threadIdx.x] = r.bias;
}

template <bool BF16>
__device__ __forceinline__ typename Mma<BF16>::frag frag_row(const typename Mma<BF16>::elem* p,
                                                             int c, int g) {
  if constexpr (BF16)
    return frag_row_bf16(p, c, g);
  else
    return frag_row_f32(p, c, g);
}

template <bool BF16>
__device__ __forceinline__ typename Mma<BF16>::frag frag_acc(const float* v, int c) {
  if constexpr (BF16)
    return frag_acc_bf16(v, c);
  else
    return v[c];
}

// ---------------------------------------------------------------------------
// Forward, training: per (split, row) partial max, sum of exponentials and O.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ __launch_bounds__(256, 1) void k_out_fwd_train(
    const float* __restrict__ W2, const float* __restrict__ b2, int L,
    const typename Mma<BF16>::elem* __restrict__ H1, int B, int tiles_per_split, int n_tiles,
    float* __restrict__ m_part, float* __restrict__ s_part, float* __restrict__ o_part,
    int ld_part) {
  using M = Mma<BF16>;
  using E = typename M::elem;
  using Fr = typename M::frag;
  constexpr int NB = FwdShape<BF16>::NB, WR = FwdShape<BF16>::WR, WT = FwdShape<BF16>::WT;
  constexpr int RB = FwdShape<BF16>::RB;
  constexpr int NCH = 32 / M::KC;
  __shared__ __attribute__((aligned(16))) E wr[2][OUT_TILE * WR];
  __shared__ __attribute__((aligned(16))) E wt[2][HID * WT];
  __shared__ float bt[2][OUT_TILE];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5, n = lane & 31;
  const int split = blockIdx.x;
  const int t_begin = split * tiles_per_split;
  const int t_end = min(n_tiles, t_begin + tiles_per_split);
  const int row0 = blockIdx.y * RB + wave * 32 * NB;
  const bool active = row0 < B;

  // H1^T as the B operand (K = hidden, N = rows), resident for the whole split.
  Fr hf[NB][4][NCH];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const E* hrow = H1 + (size_t)(row0 + nb * 32 + n) * HID;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) hf[nb][kb][c] = frag_row<BF16>(hrow + 32 * kb, c, g);
  }

  float m_run[NB], s_run[NB];
  f32x16 acc_o[NB][4];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = -INFINITY;
    s_run[nb] = 0.0f;
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc_o[nb][hb][r] = 0.0f;
  }

  TileRegs tr;
  if (t_begin < t_end) {
    tile_load(W2, b2, L, t_begin, tr);
    tile_store<BF16, true>(tr, wr[0], wt[0], bt[0]);
  }
  __syncthreads();

  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    const bool has_next = t + 1 < t_end;
    if (has_next) tile_load(W2, b2, L, t + 1, tr);
    if (active) {
      const E* wrb = wr[buf];
      const E* wtb = wt[buf];
      // Z^T tile: A = W2 rows (M = labels, K = hidden), B = H1^T.
      f32x16 z[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) z[nb][r] = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const Fr a = frag_row<BF16>(wrb + n * WR + 32 * kb, c, g);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) z[nb] = M::mma(a, hf[nb][kb][c], z[nb]);
        }
      // bias, label mask, online softmax; probabilities become the K operand of O^T.
      Fr pf[NB][NCH];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        float zz[16];
        float tmax = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ll = 8 * (r >> 2) + 4 * g + (r & 3);
          zz[r] = (t * OUT_TILE + ll < L) ? z[nb][r] + bt[buf][ll] : -INFINITY;
          tmax = fmaxf(tmax, zz[r]);
        }
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        const float mnew = fmaxf(m_run[nb], tmax);
        const float scale = exp_fast(m_run[nb] - mnew);
        float p[16];
        float ps = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          p[r] = exp_fast(zz[r] - mnew);
          ps += p[r];
        }
        s_run[nb] = s_run[nb] * scale + ps;
        if (__any(mnew > m_run[nb])) {
#pragma unroll
          for (int hb = 0; hb < 4; ++hb)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc_o[nb][hb][r] *= scale;
        }
        m_run[nb] = mnew;
#pragma unroll
        for (int c = 0; c < NCH; ++c) pf[nb][c] = frag_acc<BF16>(p, c);
      }
      // O^T += W2_tile^T P^T : A = W2^T rows (M = hidden, K = labels).
#pragma unroll
      for (int hb = 0; hb < 4; ++hb)
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const Fr a = frag_row<BF16>(wtb + (32 * hb + n) * WT, c, g);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc_o[nb][hb] = M::mma(a, pf[nb][c], acc_o[nb][hb]);
        }
    }
    if (has_next) tile_store<BF16, true>(tr, wr[buf ^ 1], wt[buf ^ 1], bt[buf ^ 1]);
    __syncthreads();
  }

  if (active) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int row = row0 + nb * 32 + n;
      const float stot = s_run[nb] + __shfl_xor(s_run[nb], 32);
      if (row < B) {
        if (g == 0) {
          m_part[(size_t)split * ld_part + row] = m_run[nb];
          s_part[(size_t)split * ld_part + row] = stot;
        }
        float* o = o_part + ((size_t)split * ld_part + row) * HID;
#pragma unroll
        for (int hb = 0; hb < 4; ++hb)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *reinterpret_cast<float4*>(o + 32 * hb + 8 * q + 4 * g) =
                make_float4(acc_o[nb][hb][4 * q], acc_o[nb][hb][4 * q + 1], acc_o[nb][hb][4 * q + 2],
                            acc_o[nb][hb][4 * q + 3]);
      }
    }
  }
}

hipError_t launch_out_fwd_train(bool use_bf16, const float* W2, const float* b2, int L, const void* H1,
                                int B, int splits, float* m_part, float* s_part, float* o_part,
                                int ld_part, hipStream_t st) {
  const int n_tiles = (L + OUT_TILE - 1) / OUT_TILE;
  const int tps = (n_tiles + splits - 1) / splits;
  const int s_eff = (n_tiles + tps - 1) / tps;
  const int RB = out_rows_per_block(use_bf16);
  const dim3 grid(s_eff, (B + RB - 1) / RB), block(256);
  if (use_bf16)
    hipLaunchKernelGGL(k_out_fwd_train<true>, grid, block, 0, st, W2, b2, L, (const bf16*)H1, B,
                       tps, n_tiles, m_part, s_part, o_part, ld_part);
  else
    hipLaunchKernelGGL(k_out_fwd_train<false>, grid, block, 0, st, W2, b2, L, (const float*)H1, B,
                       tps, n_tiles, m_part, s_part, o_part, ld_part);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Sum over the 128 threads of a workgroup in a fixed order.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float block_sum_128(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  const float t = red[0] + red[1];
  __syncthreads();
  return t;
}

// ---------------------------------------------------------------------------
// Per row: merge the splits, log-sum-exp, loss, dA1.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ __launch_bounds__(128) void k_out_combine(
    int B, int splits, const float* __restrict__ m_part, const float* __restrict__ s_part,
    const float* __restrict__ o_part, int ld_part, const float* __restrict__ W2,
    const float* __restrict__ b2, int L, const typename Mma<BF16>::elem* __restrict__ H1,
    const float* __restrict__ A1, CsrDev y, int has_y, float invB, float* __restrict__ lse_out,
    float* __restrict__ loss_rows, float* __restrict__ dA1) {
  __shared__ float red[2];
  const int i = blockIdx.x, h = threadIdx.x;
  float M = -INFINITY;
  for (int s = 0; s < splits; ++s) M = fmaxf(M, m_part[(size_t)s * ld_part + i]);
  float St = 0.0f, O = 0.0f;
  for (int s = 0; s < splits; ++s) {
    const float e = exp_fast(m_part[(size_t)s * ld_part + i] - M);
    St = fmaf(e, s_part[(size_t)s * ld_part + i], St);
    O = fmaf(e, o_part[((size_t)s * ld_part + i) * HID + h], O);
  }
  const float lse = M + logf(St);
  if (h == 0) lse_out[i] = lse;
  if (!has_y) return;
  const int ybase = y.indptr[0];
  int ys = y.indptr[i], ye = y.indptr[i + 1];
  ys = max(ys, ybase);
  ye = min(ye, ybase + y.nnz);
  if (ye < ys) ye = ys;
  const float hv = (float)H1[(size_t)i * HID + h];
  float tw = 0.0f, zsum = 0.0f;
  int cnt = 0;
  for (int q = ys; q < ye; ++q) {
    const int lab = y.indices[q];
    if (lab < 0 || lab >= L) continue;
    ++cnt;
    const float w = W2[(size_t)lab * HID + h];
    tw += w;
    float wop = w;
    if constexpr (BF16) wop = (float)(bf16)w;
    const float z = block_sum_128(hv * wop, red);
    zsum += z + b2[lab];
  }
  const float inv_cnt = cnt > 0 ? 1.0f / (float)cnt : 0.0f;
  const float dh = (O / St - tw * inv_cnt) * invB;
  dA1[(size_t)i * HID + h] = A1[(size_t)i * HID + h] > 0.0f ? dh : 0.0f;
  if (h == 0) loss_rows[i] = lse - zsum * inv_cnt;
}

hipError_t launch_out_combine(bool use_bf16, int B, int splits, const float* m_part,
                              const float* s_part, const float* o_part, int ld_part,
                              const float* W2, const float* b2, int L, const void* H1,
                              const float* A1, const CsrDev* y, float* lse, float* loss_rows,
                              float* dA1, hipStream_t st) {
  CsrDev yy = y ? *y : CsrDev{0, 0, 0, nullptr, nullptr, nullptr};
  const float invB = 1.0f / (float)B;
  if (use_bf16)
    hipLaunchKernelGGL(k_out_combine<true>, dim3(B), dim3(128), 0, st, B, splits, m_part, s_part,
                       o_part, ld_part, W2, b2, L, (const bf16*)H1, A1, yy, y != nullptr, invB,
                       lse, loss_rows, dA1);
  else
    hipLaunchKernelGGL(k_out_combine<false>, dim3(B), dim3(128), 0, st, B, splits, m_part, s_part,
                       o_part, ld_part, W2, b2, L, (const float*)H1, A1, yy, y != nullptr, invB,
                       lse, loss_rows, dA1);
  return hipGetLastError();
}

// db1 = sum_i dA1[i, :] (fixed order); b1 -= lr db1; mean loss.
__global__ __launch_bounds__(128) void k_hidden_bias(int B, const float* __restrict__ dA1,
                                                     float* __restrict__ b1, float lr,
                                                     const float* __restrict__ loss_rows,
                                                     float* __restrict__ loss) {
  __shared__ float red[2];
  const int h = threadIdx.x;
  float s = 0.0f;
  for (int i = 0; i < B; ++i) s += dA1[(size_t)i * HID + h];
  b1[h] = fmaf(-lr, s, b1[h]);
  float ls = 0.0f;
  for (int i = h; i < B; i += 128) ls += loss_rows[i];
  const float tot = block_sum_128(ls, red);
  if (h == 0) *loss = tot / (float)B;
}

hipError_t launch_hidden_bias(int B, const float* dA1, float* b1, float lr, const float* loss_rows,
                              float* loss, hipStream_t st) {
  hipLaunchKernelGGL(k_hidden_bias, dim3(1), dim3(128), 0, st, B, dA1, b1, lr, loss_rows, loss);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Backward + update of W2 and b2.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lower_bound_dev(const int32_t* __restrict__ a, int n, int key) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] < key)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

template <bool BF16>
__global__ __launch_bounds__(256) void k_out_bwd(
    float* __restrict__ W2, float* __restrict__ b2, int L, int F,
    const typename Mma<BF16>::elem* __restrict__ H1, const typename Mma<BF16>::elem* __restrict__ H1T,
    int ld_t, int B, const float* __restrict__ lse, const float* __restrict__ rw,
    const int32_t* __restrict__ skeys, const int32_t* __restrict__ svals, int n_keys,
    int label_base, const int32_t* __restrict__ lrow, float lr, float invB) {
  using M = Mma<BF16>;
  using E = typename M::elem;
  using Fr = typename M::frag;
  constexpr int NCH = 32 / M::KC;
  extern __shared__ float smem[];
  const int nrb = (B + 31) >> 5;
  const int bpad = nrb * 32;
  float* lse_s = smem;
  float* rw_s = smem + bpad;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5, n = lane & 31;
  uint32_t* mask = reinterpret_cast<uint32_t*>(smem + 2 * bpad) + wave * 32 * nrb;

  for (int i = threadIdx.x; i < bpad; i += 256) {
    lse_s[i] = i < B ? lse[i] : 0.0f;
    rw_s[i] = i < B ? rw[i] : 0.0f;
  }
  for (int k = lane; k < 32 * nrb; k += 64) mask[k] = 0u;
  __syncthreads();

  const int l0 = blockIdx.x * 128 + wave * 32;
  // true (row, label) pairs of this wave's 32 labels -> bit mask [label][row]
  if (l0 < L) {
    const int lo = lower_bound_dev(skeys, n_keys, F + l0);
    const int hi = lower_bound_dev(skeys, n_keys, F + min(l0 + 32, L));
    for (int q = lo + lane; q < hi; q += 64) {
      const int e = svals[q] - label_base;
      const int row = lrow[e];
      const int ll = skeys[q] - F - l0;
      atomicOr(&mask[ll * nrb + (row >> 5)], 1u << (row & 31));
    }
  }
  __syncthreads();

  const int label = l0 + n;
  const bool lvalid = label < L;
  // The 64 fp32 weights of this lane: hidden 32*kb + 8*q + 4*g + (0..3).
  float4 wreg[4][4];
  const float* wrow = W2 + (size_t)(lvalid ? label : 0) * HID;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int q = 0; q < 4; ++q)
      wreg[kb][q] = lvalid ? *reinterpret_cast<const float4*>(wrow + 32 * kb + 8 * q + 4 * g)
                           : make_float4(0.f, 0.f, 0.f, 0.f);
  const float bias = lvalid ? b2[label] : 0.0f;
  Fr wf[4][NCH];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      if constexpr (BF16) {
        const float4 lo = wreg[kb][2 * c], hi = wreg[kb][2 * c + 1];
        Fr f;
        f[0] = (bf16)lo.x; f[1] = (bf16)lo.y; f[2] = (bf16)lo.z; f[3] = (bf16)lo.w;
        f[4] = (bf16)hi.x; f[5] = (bf16)hi.y; f[6] = (bf16)hi.z; f[7] = (bf16)hi.w;
        wf[kb][c] = f;
      } else {
        const float4 v = wreg[kb][c >> 2];
        const float vs[4] = {v.x, v.y, v.z, v.w};
        wf[kb][c] = vs[c & 3];
      }
    }

  f32x16 accw[4];
#pragma unroll
  for (int hb = 0; hb < 4; ++hb)
#pragma unroll
    for (int r = 0; r < 16; ++r) accw[hb][r] = 0.0f;
  float db2p = 0.0f;

  for (int rb = 0; rb < nrb; ++rb) {
    // Z block: A = H1 rows (M = rows, K = hidden), B = W2^T.
    f32x16 z;
#pragma unroll
    for (int r = 0; r < 16; ++r) z[r] = 0.0f;
    const E* hrow = H1 + (size_t)(rb * 32 + n) * HID;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) z = M::mma(frag_row<BF16>(hrow + 32 * kb, c, g), wf[kb][c], z);
    const uint32_t mw = mask[n * nrb + rb];
    float dz[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = 8 * (r >> 2) + 4 * g + (r & 3);
      const int row = rb * 32 + rl;
      float d = 0.0f;
      if (row < B && lvalid) {
        const float p = exp_fast(z[r] + bias - lse_s[row]);
        const float t = ((mw >> rl) & 1u) ? rw_s[row] : 0.0f;
        d = (p - t) * invB;
      }
      dz[r] = d;
      db2p += d;
    }
    // dW2^T += H1^T dZ : A = H1^T rows (M = hidden, K = rows), B = dZ from the accumulators.
    Fr df[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) df[c] = frag_acc<BF16>(dz, c);
#pragma unroll
    for (int hb = 0; hb < 4; ++hb) {
      const E* trow = H1T + (size_t)(32 * hb + n) * ld_t + rb * 32;
#pragma unroll
      for (int c = 0; c < NCH; ++c) accw[hb] = M::mma(frag_row<BF16>(trow, c, g), df[c], accw[hb]);
    }
  }
  const float db2 = db2p + __shfl_xor(db2p, 32);
  if (lvalid) {
    float* wout = W2 + (size_t)label * HID;
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 w = wreg[hb][q];
        float4 o;
        o.x = fmaf(-lr, accw[hb][4 * q + 0], w.x);
        o.y = fmaf(-lr, accw[hb][4 * q + 1], w.y);
        o.z = fmaf(-lr, accw[hb][4 * q + 2], w.z);
        o.w = fmaf(-lr, accw[hb][4 * q + 3], w.w);
        *reinterpret_cast<float4*>(wout + 32 * hb + 8 * q + 4 * g) = o;
      }
    if (g == 0) b2[label] = fmaf(-lr, db2, bias);
  }
}

hipError_t launch_out_bwd(bool use_bf16, float* W2, float* b2, int L, int F, const void* H1,
                          const void* H1T, int ld_t, int B, const float* lse, const float* rw,
                          const int32_t* skeys, const int32_t* svals, int n_keys, int label_base,
                          const int32_t* lrow, float lr, hipStream_t st) {
  const int nrb = (B + 31) / 32;
  const size_t shm = (size_t)(2 * nrb * 32) * sizeof(float) + (size_t)4 * 32 * nrb * sizeof(uint32_t);
  const dim3 grid((L + 127) / 128), block(256);
  const float invB = 1.0f / (float)B;
  if (use_bf16)
    hipLaunchKernelGGL(k_out_bwd<true>, grid, block, shm, st, W2, b2, L, F, (const bf16*)H1,
                       (const bf16*)H1T, ld_t, B, lse, rw, skeys, svals, n_keys, label_base, lrow,
                       lr, invB);
  else
    hipLaunchKernelGGL(k_out_bwd<false>, grid, block, shm, st, W2, b2, L, F, (const float*)H1,
                       (const float*)H1T, ld_t, B, lse, rw, skeys, svals, n_keys, label_base, lrow,
                       lr, invB);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Prediction: per (split, row) top-k lists of (score, label), ties -> smaller id.
// ---------------------------------------------------------------------------
constexpr int TOPK_MAX = 32;

__device__ __forceinline__ bool better(float s, int i, float ts, int ti) {
  return s > ts || (s == ts && i < ti);
}

template <bool BF16>
__global__ __launch_bounds__(256, 1) void k_out_fwd_topk(
    const float* __restrict__ W2, const float* __restrict__ b2, int L,
    const typename Mma<BF16>::elem* __restrict__ H1, int B, int tiles_per_split, int n_tiles,
    int k, float* __restrict__ part_s, int32_t* __restrict__ part_i, int ld_part) {
  using M = Mma<BF16>;
  using E = typename M::elem;
  using Fr = typename M::frag;
  constexpr int NB = FwdShape<BF16>::NB, WR = FwdShape<BF16>::WR;
  constexpr int RB = FwdShape<BF16>::RB;
  constexpr int NCH = 32 / M::KC;
  constexpr int WROWS = 32 * NB;
  __shared__ __attribute__((aligned(16))) E wr[2][OUT_TILE * WR];
  __shared__ float bt[2][OUT_TILE];
  __shared__ float ls[4][WROWS][TOPK_MAX];
  __shared__ int li[4][WROWS][TOPK_MAX];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5, n = lane & 31;
  const int split = blockIdx.x;
  const int t_begin = split * tiles_per_split;
  const int t_end = min(n_tiles, t_begin + tiles_per_split);
  const int row0 = blockIdx.y * RB + wave * WROWS;
  const bool active = row0 < B;

  for (int e = lane; e < WROWS * TOPK_MAX; e += 64) {
    ls[wave][e / TOPK_MAX][e % TOPK_MAX] = -INFINITY;
    li[wave][e / TOPK_MAX][e % TOPK_MAX] = 0x7fffffff;
  }
  Fr hf[NB][4][NCH];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const E* hrow = H1 + (size_t)(row0 + nb * 32 + n) * HID;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) hf[nb][kb][c] = frag_row<BF16>(hrow + 32 * kb, c, g);
  }
  TileRegs tr;
  if (t_begin < t_end) {
    tile_load(W2, b2, L, t_begin, tr);
    tile_store<BF16, false>(tr, wr[0], nullptr, bt[0]);
  }
  __syncthreads();
  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    const bool has_next = t + 1 < t_end;
    if (has_next) tile_load(W2, b2, L, t + 1, tr);
    if (active) {
      const E* wrb = wr[buf];
      f32x16 z[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) z[nb][r] = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const Fr a = frag_row<BF16>(wrb + n * WR + 32 * kb, c, g);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) z[nb] = M::mma(a, hf[nb][kb][c], z[nb]);
        }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int rloc = nb * 32 + n;
        const bool rvalid = row0 + rloc < B;
        for (int half = 0; half < 2; ++half) {
          if (g == half && rvalid) {
            float* lsr = ls[wave][rloc];
            int* lir = li[wave][rloc];
            for (int r = 0; r < 16; ++r) {
              const int ll = 8 * (r >> 2) + 4 * g + (r & 3);
              const int id = t * OUT_TILE + ll;
              if (id >= L) continue;
              const float sc = z[nb][r] + bt[buf][ll];
              if (!(sc == sc)) continue;  // NaN scores are never ranked
              if (!better(sc, id, lsr[k - 1], lir[k - 1])) continue;
              int pos = k - 1;
              while (pos > 0 && better(sc, id, lsr[pos - 1], lir[pos - 1])) {
                lsr[pos] = lsr[pos - 1];
                lir[pos] = lir[pos - 1];
                --pos;
              }
              lsr[pos] = sc;
              lir[pos] = id;
            }
          }
        }
      }
    }
    if (has_next) tile_store<BF16, false>(tr, wr[buf ^ 1], nullptr, bt[buf ^ 1]);
    __syncthreads();
  }
  if (active) {
    for (int e = lane; e < WROWS * k; e += 64) {
      const int rl = e / k, j = e % k;
      const int row = row0 + rl;
      if (row < B) {
        part_s[((size_t)split * ld_part + row) * k + j] = ls[wave][rl][j];
        part_i[((size_t)split * ld_part + row) * k + j] = li[wave][rl][j];
      }
    }
  }
}

int topk_splits(int B, int n_tiles) {
  const int RB = FwdShape<true>::RB;
  int s = 256 / ((B + RB - 1) / RB);
  if (s > 64) s = 64;
  if (s < 1) s = 1;
  if (s > n_tiles) s = n_tiles;
  return s;
}

hipError_t launch_out_fwd_topk(bool use_bf16, const float* W2, const float* b2, int L, const void* H1,
                               int B, int splits, int k, float* part_s, int32_t* part_i,
                               int ld_part, hipStream_t st) {
  const int n_tiles = (L + OUT_TILE - 1) / OUT_TILE;
  const int tps = (n_tiles + splits - 1) / splits;
  const int s_eff = (n_tiles + tps - 1) / tps;
  const int RB = out_rows_per_block(use_bf16);
  const dim3 grid(s_eff, (B + RB - 1) / RB), block(256);
  if (use_bf16)
    hipLaunchKernelGGL(k_out_fwd_topk<true>, grid, block, 0, st, W2, b2, L, (const bf16*)H1, B,
                       tps, n_tiles, k, part_s, part_i, ld_part);
  else
    hipLaunchKernelGGL(k_out_fwd_topk<false>, grid, block, 0, st, W2, b2, L, (const float*)H1, B,
                       tps, n_tiles, k, part_s, part_i, ld_part);
  return hipGetLastError();
}

// Final top-k of a row from splits*k candidates: k rounds of a block arg-max.
__global__ __launch_bounds__(256) void k_topk_combine(int splits, int k,
                                                      const float* __restrict__ part_s,
                                                      const int32_t* __restrict__ part_i,
                                                      int ld_part, int32_t* __restrict__ ids,
                                                      float* __restrict__ scores) {
  extern __shared__ float csm[];
  const int i = blockIdx.x;
  const int nc = splits * k;
  float* cs = csm;
  int* ci = reinterpret_cast<int*>(csm + nc);
  __shared__ float rs[4];
  __shared__ int ri[4], rp[4];
  for (int e = threadIdx.x; e < nc; e += 256) {
    const int s = e / k, j = e % k;
    cs[e] = part_s[((size_t)s * ld_part + i) * k + j];
    ci[e] = part_i[((size_t)s * ld_part + i) * k + j];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int out = 0; out < k; ++out) {
    float bs = -INFINITY;
    int bi = 0x7fffffff, bp = -1;
    for (int e = threadIdx.x; e < nc; e += 256) {
      if (ci[e] < 0) continue;  // already taken
      if (bp < 0 || better(cs[e], ci[e], bs, bi)) {
        bs = cs[e];
        bi = ci[e];
        bp = e;
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float os = __shfl_xor(bs, o);
      const int oi = __shfl_xor(bi, o), op = __shfl_xor(bp, o);
      if (op >= 0 && (bp < 0 || better(os, oi, bs, bi))) {
        bs = os;
        bi = oi;
        bp = op;
      }
    }
    if (lane == 0) {
      rs[w] = bs;
      ri[w] = bi;
      rp[w] = bp;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      float s0 = rs[0];
      int i0 = ri[0], p0 = rp[0];
      for (int ww = 1; ww < 4; ++ww)
        if (rp[ww] >= 0 && (p0 < 0 || better(rs[ww], ri[ww], s0, i0))) {
          s0 = rs[ww];
          i0 = ri[ww];
          p0 = rp[ww];
        }
      ids[(size_t)i * k + out] = p0 >= 0 ? i0 : -1;
      if (scores) scores[(size_t)i * k + out] = p0 >= 0 ? s0 : -INFINITY;
      if (p0 >= 0) ci[p0] = -1;
    }
    __syncthreads();
  }
}

hipError_t launch_topk_combine(int B, int splits, int k, const float* part_s,
                               const int32_t* part_i, int ld_part, int32_t* ids, float* scores,
                               hipStream_t st) {
  const size_t shm = (size_t)splits * k * (sizeof(float) + sizeof(int));
  hipLaunchKernelGGL(k_topk_combine, dim3(B), dim3(256), shm, st, splits, k, part_s, part_i,
                     ld_part, ids, scores);
  return hipGetLastError();
}

}  // namespace asgd
