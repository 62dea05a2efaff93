// The output layer with stored logits (ASGD_UNFUSED_OUTPUT): the textbook
// layer-by-layer order of the model of Sec. 5.1, kept beside the fused path
// as its reference point and for callers that want the logits.
//
//   k_out_logits     Z = H W2^T + b2 on the matrix cores, written to memory
//                    fp32 [B x ldz] (labels past L hold -inf)
//   k_softmax_part   one pass over Z: per (row, column chunk) the running
//   k_softmax_final  maximum and the sum of exponentials against it (online,
//                    base 2), merged per row into lse; the row's loss is lse
//                    minus the mean of its target logits, read from Z
//   k_unfused_dh     O = P W2 with P = exp(Z - lse) read from Z, per (label
//                    split, row) on the matrix cores
//   k_dh_combine     dH = (sum_splits O - mean_{y in Y_i} W2[y]) / B and
//                    dA = dH * [A > 0]
// The logits launch carries one more workgroup that groups the (row, label)
// pairs by label block for the backward, as the fused forward's launch does.
// The W2 / b2 update is the fused backward of k_out_bwd.hip, which takes lse
// from k_softmax_final and recomputes the logits it needs from H and W2 (that
// costs no memory traffic; reading Z back would cost B*L*4 bytes).
#include <math.h>

#include "asgd_dev.h"
#include "asgd_kernels.h"
#include "aux_dev.h"
#include "out_tile.h"

namespace asgd {

// ---------------------------------------------------------------------------
// Logits.  Workgroup = (label split, 256 rows), 8 waves x 32 rows, H fragments
// resident in registers; W2 tiles double-buffered in LDS, the next one loaded
// into registers while the current one is used.  Lane (g, n) holds row n and
// labels 8q + 4g + 0..3 of the tile (the accumulator's layout); the wave turns
// its 32 x 32 block around in LDS so that each 16-byte store instruction
// writes eight whole 128-byte row segments of Z.  With `exact` the stores go
// element by element and stop at label L (a caller's [B x L] buffer);
// otherwise ldz covers whole tiles.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ __launch_bounds__(FWD_THREADS) void k_out_logits(const float* __restrict__ W2,
                                                            const float* __restrict__ b2, int L,
                                                            const typename Mma<BF16>::elem* __restrict__ H1,
                                                            int B, int tiles_per_split, int n_tiles,
                                                            int s_eff, float* __restrict__ Z, int ldz,
                                                            int exact, int n_fwd, LabelJob lj) {
  using M = Mma<BF16>;
  using E = typename M::elem;
  using Fr = typename M::frag;
  constexpr int RB = FwdShape<BF16>::RB;
  constexpr int NCH = 32 / M::KC;
  __shared__ __attribute__((aligned(16))) E wr[2][tile_elems<BF16>()];
  __shared__ __attribute__((aligned(16))) float bt[2][OUT_TILE];
  constexpr int ZT = OUT_TILE + 4;  // row stride of a wave's transposition block (floats)
  __shared__ __attribute__((aligned(16))) float zt[FwdShape<BF16>::WAVES][32 * ZT];
  if ((int)blockIdx.x >= n_fwd) {  // the label grouping (dispatched last)
    extern __shared__ int32_t job_lds[];
    if (lj.in_lds)
      wg_label_blocks<FWD_THREADS, true>(lj.lkeys, lj.m, L, lj.lrow, lj.lbeg, lj.lpair, job_lds,
                                         job_lds + ((L + 31) >> 5));
    else
      wg_label_blocks<FWD_THREADS, false>(lj.lkeys, lj.m, L, lj.lrow, lj.lbeg, lj.lpair, lj.lcnt, job_lds);
    return;
  }
  const int lane = threadIdx.x & 63, g = lane >> 5, n = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int split = (int)blockIdx.x % s_eff;
  const int t_begin = split * tiles_per_split;
  const int t_end = min(n_tiles, t_begin + tiles_per_split);
  const int row0 = ((int)blockIdx.x / s_eff) * RB + wave * 32;
  const int row = row0 + n;
  const W2Src src = w2_src(W2, b2, L);
  const int rbase[2] = {tw_row_base(n, g, 0), tw_row_base(n, g, 1)};

  Fr hf[4][NCH];
  const E* hrow = H1 + (size_t)row * HID;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int c = 0; c < NCH; ++c) hf[kb][c] = h1_frag<BF16>(hrow, kb, c, g);

  TileRegs tr;
  if (t_begin < t_end) {
    tile_load(src, t_begin, tr);
    tile_store<BF16, false>(tr, L, t_begin, wr[0], nullptr, bt[0]);
    if (t_begin + 1 < t_end) tile_load(src, t_begin + 1, tr);
  }
  __syncthreads();
  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    f32x16 z;
    {
      const float4* bq = reinterpret_cast<const float4*>(bt[buf]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 b = bq[2 * q + g];
        z[4 * q + 0] = b.x; z[4 * q + 1] = b.y; z[4 * q + 2] = b.z; z[4 * q + 3] = b.w;
      }
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) z = M::mma(tile_frag_w<BF16>(wr[buf], rbase, n, kb, c, g), hf[kb][c], z);
    if (!exact) {
      // the accumulator layout into the wave's block (row n, labels 8q + 4g ..), then
      // out as row segments: lane l stores row 8k + l / 8, labels 4 (l % 8) .. + 3
      float* zb = zt[wave];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(zb + n * ZT + 8 * q + 4 * g) =
            make_float4(z[4 * q], z[4 * q + 1], z[4 * q + 2], z[4 * q + 3]);
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int rl = 8 * k + (lane >> 3), cl = 4 * (lane & 7);
        const float4 v = *reinterpret_cast<const float4*>(zb + rl * ZT + cl);
        if (row0 + rl < B) *reinterpret_cast<float4*>(Z + (size_t)(row0 + rl) * ldz + t * OUT_TILE + cl) = v;
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    } else if (row < B) {
      float* zr = Z + (size_t)row * ldz + t * OUT_TILE + 4 * g;
      {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ll = 8 * (r >> 2) + (r & 3);
          if (t * OUT_TILE + 4 * g + ll < L) zr[ll] = z[r];
        }
      }
    }
    if (t + 1 < t_end) tile_store<BF16, false>(tr, L, t + 1, wr[buf ^ 1], nullptr, bt[buf ^ 1]);
    if (t + 2 < t_end) tile_load(src, t + 2, tr);
    __syncthreads();
  }
}

// The job's counters stay in global memory here: dynamic LDS is sized per launch,
// and counters in LDS would take it from every logits workgroup (two of which
// share a CU).
LabelJobPlan logits_label_plan(bool /*use_bf16*/, int /*L*/) {
  LabelJobPlan p{};
  p.ok = 1;
  p.in_lds = 0;
  p.lds_bytes = 4 * (FWD_THREADS / 64);
  return p;
}

hipError_t launch_out_logits(bool use_bf16, const float* W2, const float* b2, int L, const void* H1, int B,
                             float* Z, int ldz, int exact, int n_cu, const LabelJob* job,
                             const LabelJobPlan* plan, hipStream_t st) {
  const int n_tiles = (L + OUT_TILE - 1) / OUT_TILE;
  if (!exact && ldz < n_tiles * OUT_TILE) return hipErrorInvalidValue;
  if (exact && ldz < L) return hipErrorInvalidValue;
  const int RB = out_rows_per_block(use_bf16);
  const int nrb = (B + RB - 1) / RB;
  // two workgroups per CU: the kernel is bound by its stores of Z
  const int want = (2 * n_cu + nrb - 1) / nrb;
  const int splits = want < n_tiles ? want : n_tiles;
  const int tps = (n_tiles + splits - 1) / splits;
  const int s_eff = (n_tiles + tps - 1) / tps;
  const int n_fwd = s_eff * nrb;
  LabelJob lj{};
  int lds = 0, n_job = 0;
  if (job) {
    if (!plan || !plan->ok) return hipErrorInvalidValue;
    lj = *job;
    lj.in_lds = plan->in_lds;
    lds = plan->lds_bytes;
    n_job = 1;
  }
  const dim3 grid(n_fwd + n_job), block(FWD_THREADS);
  if (use_bf16)
    hipLaunchKernelGGL(k_out_logits<true>, grid, block, lds, st, W2, b2, L, (const bf16*)H1, B, tps, n_tiles,
                       s_eff, Z, ldz, exact, n_fwd, lj);
  else
    hipLaunchKernelGGL(k_out_logits<false>, grid, block, lds, st, W2, b2, L, (const float*)H1, B, tps, n_tiles,
                       s_eff, Z, ldz, exact, n_fwd, lj);
  return hipGetLastError();
}

// Entries [*q0, *q1) of row i, kept inside [indptr[0], indptr[0] + nnz) whatever indptr holds.
__device__ __forceinline__ void row_range(const CsrDev& a, int i, int* q0, int* q1) {
  const int base = a.indptr[0];
  const int s = max(a.indptr[i], base), e = min(a.indptr[i + 1], base + a.nnz);
  *q0 = s;
  *q1 = e < s ? s : e;
}

// ---------------------------------------------------------------------------
// Softmax and cross-entropy over the stored logits, one read of Z.  Workgroup
// = (column chunk, row), 256 threads.  Each thread keeps a running maximum m
// (base 2: m = max z log2 e) and s = sum 2^(z log2 e - m) over its share of
// the chunk, rescaling s only when a group of eight float4 loads raises m; the
// wavefront and then the workgroup merge their (m, s) pairs with cross-lane
// reductions.  Entries of -inf (labels past L) contribute nothing.
// ---------------------------------------------------------------------------
// Z is read once by the softmax pass, in whole 16-byte pieces of contiguous
// 1 KB runs per wave: non-temporal loads keep it from displacing what the
// caches hold (measured on the pass alone: 118 -> 103 us for 256 x 670,112).
__device__ __forceinline__ float4 load_nt(const float4* p) {
  const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

constexpr int SM_THREADS = 256;
constexpr int SM_VEC = 8;                          // float4 loads in flight per thread
constexpr int SM_CHUNK = SM_THREADS * SM_VEC * 4 * 4;  // columns per workgroup: four rounds of loads

__device__ __forceinline__ void ms_merge(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;  // both empty
  s = (m == -INFINITY ? 0.0f : s * __builtin_amdgcn_exp2f(m - mm)) +
      (m2 == -INFINITY ? 0.0f : s2 * __builtin_amdgcn_exp2f(m2 - mm));
  m = mm;
}

__global__ __launch_bounds__(SM_THREADS) void k_softmax_part(const float* __restrict__ Z, int ldz,
                                                            float* __restrict__ m_part,
                                                            float* __restrict__ s_part, int ld_part) {
  __shared__ float rm[SM_THREADS / 64], rs[SM_THREADS / 64];
  const int row = blockIdx.y, split = blockIdx.x;
  const int v0 = split * (SM_CHUNK / 4), v1 = min(ldz / 4, v0 + SM_CHUNK / 4);
  const float4* zr = reinterpret_cast<const float4*>(Z + (size_t)row * ldz);
  float m = -INFINITY, s = 0.0f;
  for (int base = v0; base < v1; base += SM_THREADS * SM_VEC) {
    float4 v[SM_VEC];
#pragma unroll
    for (int j = 0; j < SM_VEC; ++j) {
      const int idx = base + j * SM_THREADS + (int)threadIdx.x;
      v[j] = idx < v1 ? load_nt(zr + idx) : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < SM_VEC; ++j) mx = fmaxf(mx, fmaxf(fmaxf(v[j].x, v[j].y), fmaxf(v[j].z, v[j].w)));
    const float mx2 = mx * LOG2E;
    if (mx2 > m) {
      s = m == -INFINITY ? 0.0f : s * __builtin_amdgcn_exp2f(m - mx2);
      m = mx2;
    }
    if (m != -INFINITY) {
      float acc = 0.0f;
#pragma unroll
      for (int j = 0; j < SM_VEC; ++j) {
        acc += __builtin_amdgcn_exp2f(fmaf(v[j].x, LOG2E, -m));
        acc += __builtin_amdgcn_exp2f(fmaf(v[j].y, LOG2E, -m));
        acc += __builtin_amdgcn_exp2f(fmaf(v[j].z, LOG2E, -m));
        acc += __builtin_amdgcn_exp2f(fmaf(v[j].w, LOG2E, -m));
      }
      s += acc;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ms_merge(m, s, __shfl_xor(m, o), __shfl_xor(s, o));
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    rm[w] = m;
    rs[w] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = rm[0], S = rs[0];
    for (int k = 1; k < SM_THREADS / 64; ++k) ms_merge(M, S, rm[k], rs[k]);
    m_part[(size_t)split * ld_part + row] = M;
    s_part[(size_t)split * ld_part + row] = S;
  }
}

// Per row (one wavefront): lse from the chunks' (m, s), in chunk order per
// lane and then a fixed reduction tree; loss = lse - mean of the row's target
// logits.
__global__ __launch_bounds__(64) void k_softmax_final(const float* __restrict__ Z, int ldz, int splits,
                                                      const float* __restrict__ m_part,
                                                      const float* __restrict__ s_part, int ld_part,
                                                      CsrDev y, int has_y, float* __restrict__ lse,
                                                      float* __restrict__ loss_rows) {
  const int row = blockIdx.x, lane = threadIdx.x;
  float m = -INFINITY, s = 0.0f;
  for (int k = lane; k < splits; k += 64)
    ms_merge(m, s, m_part[(size_t)k * ld_part + row], s_part[(size_t)k * ld_part + row]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ms_merge(m, s, __shfl_xor(m, o), __shfl_xor(s, o));
  const float l = (m + __builtin_amdgcn_logf(s)) * LN2;  // v_log_f32 is base 2
  float t = 0.0f;
  int cnt = 0;
  if (has_y) {
    int q0, q1;
    row_range(y, row, &q0, &q1);
    for (int q = q0 + lane; q < q1; q += 64) {
      const int lab = y.indices[q];
      const bool ok = lab >= 0 && lab < y.n_cols;
      if (ok) t += Z[(size_t)row * ldz + lab];
      cnt += ok ? 1 : 0;
    }
    t = wave_sum(t);
    cnt = (int)wave_sum((float)cnt);
  }
  if (lane == 0) {
    lse[row] = l;
    if (has_y) loss_rows[row] = cnt > 0 ? l - t / (float)cnt : 0.0f;
  }
}

hipError_t launch_softmax_ce(const float* Z, int ldz, int B, float* m_part, float* s_part, int ld_part,
                             const CsrDev* y, float* lse, float* loss_rows, hipStream_t st) {
  const int splits = (ldz + SM_CHUNK - 1) / SM_CHUNK;
  if ((int64_t)splits * ld_part < (int64_t)splits * B) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_softmax_part, dim3(splits, B), dim3(SM_THREADS), 0, st, Z, ldz, m_part, s_part,
                     ld_part);
  CsrDev yy = y ? *y : CsrDev{};
  hipLaunchKernelGGL(k_softmax_final, dim3(B), dim3(64), 0, st, Z, ldz, splits, m_part, s_part, ld_part, yy,
                     y != nullptr, lse, loss_rows);
  return hipGetLastError();
}

int softmax_splits(int ldz) { return (ldz + SM_CHUNK - 1) / SM_CHUNK; }

// ---------------------------------------------------------------------------
// O = P W2 from the stored logits.  The workgroup shape of the logits kernel;
// per tile a wave loads its 32 rows x 32 labels of Z (the next tile's while
// the current one is used), forms p = 2^(z log2 e - lse log2 e) in the
// accumulator layout, and adds W2_tile^T P^T into its O^T accumulators.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ __launch_bounds__(FWD_THREADS) void k_unfused_dh(const float* __restrict__ W2,
                                                            const float* __restrict__ b2, int L,
                                                            const float* __restrict__ Z, int ldz,
                                                            const float* __restrict__ lse, int B,
                                                            int tiles_per_split, int n_tiles, int s_eff,
                                                            float* __restrict__ o_part, int ld_part) {
  using M = Mma<BF16>;
  using E = typename M::elem;
  using Fr = typename M::frag;
  constexpr int RB = FwdShape<BF16>::RB;
  constexpr int NCH = 32 / M::KC;
  __shared__ __attribute__((aligned(16))) E wr[2][tile_elems<BF16>()];
  __shared__ __attribute__((aligned(16))) E wt[2][tileT_elems<BF16>()];
  __shared__ __attribute__((aligned(16))) float bt[2][OUT_TILE];
  const int lane = threadIdx.x & 63, g = lane >> 5, n = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int split = (int)blockIdx.x % s_eff;
  const int t_begin = split * tiles_per_split;
  const int t_end = min(n_tiles, t_begin + tiles_per_split);
  const int row0 = ((int)blockIdx.x / s_eff) * RB + wave * 32;
  const int row = row0 + n;
  const bool live = row < B;
  const W2Src src = w2_src(W2, b2, L);
  const int cbase[2] = {tw_col_base(lane, 0), tw_col_base(lane, 1)};
  const float nl2 = live ? -lse[row] * LOG2E : 0.0f;
  const float* zrow = Z + (size_t)(live ? row : 0) * ldz + 4 * g;

  f32x16 acc_o[4];
#pragma unroll
  for (int hb = 0; hb < 4; ++hb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc_o[hb][r] = 0.0f;

  auto load_z = [&](int t, float4 (&zv)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      // (plain loads: a lane reads 16 of a row's 128 bytes per instruction, and
      // non-temporal loads let the line go before the other three quarters
      // are read: 1.5x the bytes from HBM, measured)
      zv[q] = live ? *reinterpret_cast<const float4*>(zrow + t * OUT_TILE + 8 * q)
                   : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
  };
  TileRegs tr;
  float4 zc[4], zn[4];
  if (t_begin < t_end) {
    tile_load(src, t_begin, tr);
    tile_store<BF16, true>(tr, L, t_begin, wr[0], wt[0], bt[0]);
    if (t_begin + 1 < t_end) tile_load(src, t_begin + 1, tr);
    load_z(t_begin, zc);
  }
  __syncthreads();
  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    if (t + 1 < t_end) load_z(t + 1, zn);
    float p[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      p[4 * q + 0] = __builtin_amdgcn_exp2f(fmaf(zc[q].x, LOG2E, nl2));
      p[4 * q + 1] = __builtin_amdgcn_exp2f(fmaf(zc[q].y, LOG2E, nl2));
      p[4 * q + 2] = __builtin_amdgcn_exp2f(fmaf(zc[q].z, LOG2E, nl2));
      p[4 * q + 3] = __builtin_amdgcn_exp2f(fmaf(zc[q].w, LOG2E, nl2));
    }
    Fr pf[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) pf[c] = frag_acc<BF16>(p, c);
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int c = 0; c < NCH; ++c)
        acc_o[hb] = M::mma(tile_frag_wt<BF16>(wr[buf], wt[buf], cbase, hb, c, lane), pf[c], acc_o[hb]);
    if (t + 1 < t_end) tile_store<BF16, true>(tr, L, t + 1, wr[buf ^ 1], wt[buf ^ 1], bt[buf ^ 1]);
    if (t + 2 < t_end) tile_load(src, t + 2, tr);
#pragma unroll
    for (int q = 0; q < 4; ++q) zc[q] = zn[q];
    __syncthreads();
  }
  if (live) {
    float* o = o_part + ((size_t)split * ld_part + row) * HID;
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(o + 32 * hb + 8 * q + 4 * g) =
            make_float4(acc_o[hb][4 * q], acc_o[hb][4 * q + 1], acc_o[hb][4 * q + 2], acc_o[hb][4 * q + 3]);
  }
}

// Per row, 4 groups of 128 threads (one per hidden unit): group c sums the
// splits k = c (mod 4) in order, then the groups are added in order (a fixed
// summation order); dH = (sum_k O_k - rw sum_{y in Y_i} W2[y]) / B and
// dA = dH where A > 0.
constexpr int DHC_GROUPS = 4;
__global__ __launch_bounds__(HID * DHC_GROUPS) void k_dh_combine(const float* __restrict__ o_part, int ld_part,
                                                                 int splits, const float* __restrict__ W2, int L,
                                                                 CsrDev y, const float* __restrict__ rw,
                                                                 const float* __restrict__ A, float invB,
                                                                 float* __restrict__ dA) {
  __shared__ float part[DHC_GROUPS][HID];
  const int row = blockIdx.x, j = threadIdx.x % HID, grp = threadIdx.x / HID;
  float og = 0.0f;
  for (int k = grp; k < splits; k += DHC_GROUPS) og += o_part[((size_t)k * ld_part + row) * HID + j];
  part[grp][j] = og;
  __syncthreads();
  if (grp) return;
  float o = part[0][j];
#pragma unroll
  for (int c = 1; c < DHC_GROUPS; ++c) o += part[c][j];
  int q0, q1;
  row_range(y, row, &q0, &q1);
  float t = 0.0f;
  for (int q = q0; q < q1; ++q) {
    const int lab = y.indices[q];
    if (lab >= 0 && lab < L) t += W2[(size_t)lab * HID + j];
  }
  const float dh = (o - rw[row] * t) * invB;
  dA[(size_t)row * HID + j] = A[(size_t)row * HID + j] > 0.0f ? dh : 0.0f;
}

int unfused_dh_splits(int n_cu, int aux_cus, int B, bool use_bf16, int n_tiles) {
  const int RB = out_rows_per_block(use_bf16);
  const int nrb = (B + RB - 1) / RB;
  const int wgs = n_cu - aux_cus > 1 ? n_cu - aux_cus : 1;
  int s = (wgs + nrb - 1) / nrb;
  if (s > n_tiles) s = n_tiles;
  return s < 1 ? 1 : s;
}

hipError_t launch_unfused_dh(bool use_bf16, const float* W2, const float* b2, int L, const float* Z, int ldz,
                             const float* lse, int B, int splits, float* o_part, int ld_part, const CsrDev& y,
                             const float* rw, const float* A, float* dA, hipStream_t st) {
  const int n_tiles = (L + OUT_TILE - 1) / OUT_TILE;
  if (ldz < n_tiles * OUT_TILE) return hipErrorInvalidValue;
  const int tps = (n_tiles + splits - 1) / splits;
  const int s_eff = (n_tiles + tps - 1) / tps;
  const int RB = out_rows_per_block(use_bf16);
  const dim3 grid(s_eff * ((B + RB - 1) / RB)), block(FWD_THREADS);
  if (use_bf16)
    hipLaunchKernelGGL(k_unfused_dh<true>, grid, block, 0, st, W2, b2, L, Z, ldz, lse, B, tps, n_tiles, s_eff,
                       o_part, ld_part);
  else
    hipLaunchKernelGGL(k_unfused_dh<false>, grid, block, 0, st, W2, b2, L, Z, ldz, lse, B, tps, n_tiles, s_eff,
                       o_part, ld_part);
  hipLaunchKernelGGL(k_dh_combine, dim3(B), dim3(HID * DHC_GROUPS), 0, st, o_part, ld_part, s_eff, W2, L, y, rw,
                     A, 1.0f / (float)B, dA);
  return hipGetLastError();
}

}  // namespace asgd
