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
// Per row, after the forward: k_out_lse_targets merges the splits' (max, sum)
// pairs (log-sum-exp) and forms the target terms and the loss; k_out_dA1
// merges the splits' O (dH1 = (O/s - mean_{y in Y_i} W2[y]) / B,
// dA1 = dH1 * [A1 > 0]); one launch does both when they share a stream.
// The backward with the W2 / b2 update is in k_out_bwd.hip.
#include <float.h>
#include <math.h>

#include <hip/hip_ext.h>

#include "asgd_dev.h"
#include "asgd_kernels.h"
#include "aux_dev.h"
#include "out_tile.h"

namespace asgd {

int out_rows_per_block(bool use_bf16) { return use_bf16 ? FwdShape<true>::RB : FwdShape<false>::RB; }

// ---------------------------------------------------------------------------
// Forward, training: per (split, row) partial max, sum of exponentials and O.
// ---------------------------------------------------------------------------
// LDS ring of W2 tiles: one workgroup barrier per FwdRing::P tiles.  Between
// two barriers the waves read tiles t .. t+P and store t+P+1 .. t+2P, so a ring
// of 2P+1 tiles keeps what is read and what is written apart.  The bf16 tile
// (10 KB) allows P = 2; the fp32 operands (two 17-18 KB layouts per tile) keep
// P = 1.
template <bool BF16>
struct FwdRing {
  static constexpr int P = BF16 ? 2 : 1;
  static constexpr int N = 2 * P + 1;
};

// With a label job, workgroup n_fwd of the launch (dispatched last, on a CU
// the forward leaves free) groups the batch's labels for the backward: it
// depends only on the gather and finishes long before the forward, so the
// backward needs no event from another stream.  Its counters live in the
// launch's dynamic LDS (or in global memory when they do not fit).
template <bool BF16>
__global__ __launch_bounds__(FWD_THREADS) void k_out_fwd_train(
    const float* __restrict__ W2, const float* __restrict__ b2, int L,
    const typename Mma<BF16>::elem* __restrict__ H1, int B, int tiles_per_split, int n_tiles,
    float* __restrict__ m_part, float* __restrict__ s_part, float* __restrict__ o_part,
    int ld_part, int s_eff, int n_fwd, LabelJob lj) {
  using M = Mma<BF16>;
  using E = typename M::elem;
  using Fr = typename M::frag;
  constexpr int RB = FwdShape<BF16>::RB;
  constexpr int NCH = 32 / M::KC;
  static_assert(FwdShape<BF16>::NB == 1, "one 32-row block per wave");
  constexpr int P = FwdRing<BF16>::P, NRING = FwdRing<BF16>::N;
  __shared__ __attribute__((aligned(16))) E wr[NRING][tile_elems<BF16>()];
  __shared__ __attribute__((aligned(16))) E wt[NRING][tileT_elems<BF16>()];
  __shared__ __attribute__((aligned(16))) float bt[NRING][OUT_TILE];

  if ((int)blockIdx.x >= n_fwd) {
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
  // Workgroup -> (split, row block).  Workgroups are dealt to the 8 XCDs in
  // turn (workgroup b to XCD b mod 8), each with its own L2, so the row blocks
  // of one split (which read the same W2 tiles) get consecutive numbers in
  // XCD-major order v: they share an XCD, and its L2 serves the tiles once.
  const int nrb = n_fwd / s_eff;
  const int b = (int)blockIdx.x;
  const int v = n_fwd % 8 == 0 ? (b % 8) * (n_fwd / 8) + b / 8 : b;
  const int split = v / nrb;
  const int t_begin = split * tiles_per_split;
  const int t_end = min(n_tiles, t_begin + tiles_per_split);
  const int t_last = t_end - 1;
  // Rows past B (up to the 256-row padding, zero in H1) are computed like the
  // others and never written out, so the loop has no row-dependent branch.
  const int row0 = (v % nrb) * RB + wave * 32;
  const W2Src src = w2_src(W2, b2, L);
  const int rbase[2] = {tw_row_base(n, g, 0), tw_row_base(n, g, 1)};
  const int cbase[2] = {tw_col_base(lane, 0), tw_col_base(lane, 1)};

  // H1^T as the B operand (K = hidden, N = rows), resident for the whole split.
  Fr hf[4][NCH];
  const E* hrow = H1 + (size_t)(row0 + n) * HID;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int c = 0; c < NCH; ++c) hf[kb][c] = h1_frag<BF16>(hrow, kb, c, g);
  // Redefine the fragments once they have arrived (empty asm), so the loop below
  // never waits on these loads again and its wait counters track only the W2
  // prefetch.
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int c = 0; c < NCH; ++c) asm volatile("" : "+v"(hf[kb][c]));

  // Z^T tile from LDS buffer `buf`: A = W2 rows (M = labels, K = hidden),
  // B = H1^T; the accumulator starts at the labels' biases (-inf past L).
  auto z_tile = [&](int buf) {
    const float4* bq = reinterpret_cast<const float4*>(bt[buf]);
    f32x16 z;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 b = bq[2 * q + g];
      z[4 * q + 0] = b.x; z[4 * q + 1] = b.y; z[4 * q + 2] = b.z; z[4 * q + 3] = b.w;
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) z = M::mma(tile_frag_w<BF16>(wr[buf], rbase, n, kb, c, g), hf[kb][c], z);
    return z;
  };

  float m_run = -INFINITY, s_run = 0.0f;
  f32x16 acc_o[4];
#pragma unroll
  for (int hb = 0; hb < 4; ++hb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc_o[hb][r] = 0.0f;

  // Software pipeline over a ring of LDS tiles and two register tiles.  In the
  // iteration of tile t: the logits of tile t+1 go to the matrix cores while
  // the softmax numerators of tile t are formed; then O^T += W2_t^T P_t^T
  // while tile t+P+1 (loaded into registers two iterations earlier) is
  // converted into the ring and tile t+P+3 is loaded in its place; a barrier
  // closes every P-th iteration.  Tile u lives in ring slot (u - t_begin) mod
  // NRING.  Tile indices are clamped to the split's last tile, so every load,
  // store and product is unconditional (a clamped copy is never consumed).
  // Every split has at least one tile.
  TileRegs tr0, tr1;
  auto slot = [&](int u) { return (u - t_begin) % NRING; };
#pragma unroll
  for (int u = 0; u <= P; ++u) {
    const int tu = min(t_begin + u, t_last);
    tile_load(src, tu, tr0);
    tile_store<BF16, true>(tr0, L, tu, wr[u], wt[u], bt[u]);
  }
  tile_load(src, min(t_begin + P + 1, t_last), tr0);
  tile_load(src, min(t_begin + P + 2, t_last), tr1);
  __syncthreads();
  f32x16 z = z_tile(0);

  // Online softmax in base 2 with lazy rescaling: p = 2^(z log2e - m2) where m2
  // is a per-row reference that is raised only when a tile's maximum exceeds it
  // by more than LAZY (so p <= 2^LAZY); the final normalisation uses the same
  // reference, so the result is exact up to rounding.
  constexpr float LAZY = 8.0f, LAZY_SUM = 256.0f;  // LAZY_SUM = 2^LAZY
  auto iteration = [&](int t, TileRegs& tr) {
    const int b0 = slot(t), b1 = slot(t + 1), bst = slot(t + P + 1);
    // Operands of this iteration's two products, read from LDS first so that
    // their latency is covered by the max / rescale work below: A of the next
    // tile's logits (W2 rows, with the biases as the accumulator's start) and
    // A of this tile's O (W2^T rows).
    // (fp32 operands take 16 chunks per 32-wide block: those are read at use,
    // as holding them all would not fit the register file.)
    constexpr int PRE = BF16 ? NCH : 1;
    Fr za[4][PRE], oa[4][PRE];
    if constexpr (BF16) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int c = 0; c < NCH; ++c) za[kb][c] = tile_frag_w<BF16>(wr[b1], rbase, n, kb, c, g);
    }
    f32x16 zn;
    {
      const float4* bq = reinterpret_cast<const float4*>(bt[b1]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 b = bq[2 * q + g];
        zn[4 * q + 0] = b.x; zn[4 * q + 1] = b.y; zn[4 * q + 2] = b.z; zn[4 * q + 3] = b.w;
      }
    }
    if constexpr (BF16) {
#pragma unroll
      for (int hb = 0; hb < 4; ++hb)
#pragma unroll
        for (int c = 0; c < NCH; ++c) oa[hb][c] = tile_frag_wt<BF16>(wr[b0], wt[b0], cbase, hb, c, lane);
    }

    // The next tile's logits go to the matrix cores first; this tile's
    // numerators are formed on the vector units while they run, against the
    // current reference, and formed again in the rare iteration that raises
    // it, so every p that is used is computed against the reference the row
    // ends with at that point.
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c)
        zn = M::mma(BF16 ? za[kb][c % PRE] : tile_frag_w<BF16>(wr[b1], rbase, n, kb, c, g), hf[kb][c], zn);
    // The tile's maximum is only formed when some lane's numerators sum past
    // 2^LAZY (or are not finite, as on a row's first tile, whose reference is
    // -inf): no numerator exceeds its lane's sum, so every other tile keeps
    // p <= 2^LAZY against the current reference.
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) p[r] = __builtin_amdgcn_exp2f(fmaf(z[r], LOG2E, -m_run));
    float ps = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) ps += p[r];
    if (__any(!(ps <= LAZY_SUM))) {
      // running maximum of this tile (rows are lanes: one max per lane pair)
      float tmax = z[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) tmax = fmaxf(tmax, z[r]);
      tmax = half_swap_max(tmax);
      const float m2c = tmax * LOG2E;
      const float m2n = m2c > m_run + LAZY ? m2c : m_run;
      const float scale = __builtin_amdgcn_exp2f(m_run - m2n);
      s_run *= scale;
#pragma unroll
      for (int hb = 0; hb < 4; ++hb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc_o[hb][r] *= scale;
      m_run = m2n;
      ps = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[r] = __builtin_amdgcn_exp2f(fmaf(z[r], LOG2E, -m_run));
        ps += p[r];
      }
    }
    s_run += ps;
    Fr pf[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) pf[c] = frag_acc<BF16>(p, c);
    // O^T += W2_t^T P^T : A = W2^T rows (M = hidden, K = labels).
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int c = 0; c < NCH; ++c)
        acc_o[hb] = M::mma(BF16 ? oa[hb][c % PRE] : tile_frag_wt<BF16>(wr[b0], wt[b0], cbase, hb, c, lane),
                           pf[c], acc_o[hb]);
    tile_store<BF16, true>(tr, L, min(t + P + 1, t_last), wr[bst], wt[bst], bt[bst]);
    tile_load(src, min(t + P + 3, t_last), tr);
    if ((t - t_begin) % P == P - 1) __syncthreads();
    z = zn;
  };
  for (int t = t_begin; t < t_end; t += 2) {
    iteration(t, tr0);
    if (t + 1 >= t_end) break;
    iteration(t + 1, tr1);
  }

  const int row = row0 + n;
  const float stot = s_run + __shfl_xor(s_run, 32);
  if (row < B) {
    if (g == 0) {
      m_part[(size_t)split * ld_part + row] = m_run * LN2;
      s_part[(size_t)split * ld_part + row] = stot;
    }
    float* o = o_part + ((size_t)split * ld_part + row) * HID;
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(o + 32 * hb + 8 * q + 4 * g) =
            make_float4(acc_o[hb][4 * q], acc_o[hb][4 * q + 1], acc_o[hb][4 * q + 2],
                        acc_o[hb][4 * q + 3]);
  }
}

LabelJobPlan label_job_plan_for(const void* fn, int nthreads, int L) {
  LabelJobPlan p{};
  hipFuncAttributes fa{};
  int dev = 0, lds_max = 0;
  if (hipFuncGetAttributes(&fa, fn) != hipSuccess || hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return p;
  // what the kernel's own arrays leave of a workgroup's LDS (160 KB on gfx950)
  const int budget = lds_max - (int)fa.sharedSizeBytes;
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, budget) != hipSuccess) return p;
  const int ints = (L + 31) / 32 + nthreads / 64;
  p.in_lds = ints * 4 <= budget;
  p.lds_bytes = 4 * (p.in_lds ? ints : nthreads / 64);
  p.ok = p.lds_bytes <= budget;
  return p;
}

LabelJobPlan label_job_plan(bool use_bf16, int L) {
  return label_job_plan_for(use_bf16 ? (const void*)k_out_fwd_train<true> : (const void*)k_out_fwd_train<false>,
                            FWD_THREADS, L);
}

hipError_t launch_out_fwd_train(bool use_bf16, const float* W2, const float* b2, int L, const void* H1,
                                int B, int splits, float* m_part, float* s_part, float* o_part,
                                int ld_part, const LabelJob* job, const LabelJobPlan* plan, hipStream_t st,
                                hipEvent_t t0, hipEvent_t t1) {
  const int n_tiles = (L + OUT_TILE - 1) / OUT_TILE;
  const int tps = (n_tiles + splits - 1) / splits;
  const int s_eff = (n_tiles + tps - 1) / tps;
  const int RB = out_rows_per_block(use_bf16);
  const int n_fwd = s_eff * ((B + RB - 1) / RB);
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
    hipExtLaunchKernelGGL(k_out_fwd_train<true>, grid, block, lds, st, t0, t1, 0, W2, b2, L, (const bf16*)H1, B,
                          tps, n_tiles, m_part, s_part, o_part, ld_part, s_eff, n_fwd, lj);
  else
    hipExtLaunchKernelGGL(k_out_fwd_train<false>, grid, block, lds, st, t0, t1, 0, W2, b2, L, (const float*)H1,
                          B, tps, n_tiles, m_part, s_part, o_part, ld_part, s_eff, n_fwd, lj);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Per row, in two kernels so that only the small one sits between the forward
// and the backward:
//   k_out_lse_targets  lse from the splits' (max, sum) pairs, and the row's
//                      target terms: the mean of W2[y] over y in Y_i (the
//                      pre-update W2, before the backward writes it), the
//                      target logits and the loss;
//   k_out_dA1          the splits' O merged against the same maxima,
//                      dH1 = (O/s - mean_{y in Y_i} W2[y]) / B, dA1 = dH1 [A1 > 0]
//                      (runs beside the backward: it reads no W2).
// A step that forms dA1 on the model's stream anyway runs both in one launch
// (k_out_lse_targets<., true>).
// k_out_lse_targets: 512 threads, one (max, sum) pair per thread merged by
// wavefront reductions, 8 wavefronts x the row's labels for the target terms.
// k_out_dA1: G split groups x 32 threads x 4 hidden units; each group merges
// its splits online against its own running maximum, then the groups are
// rescaled to the row's maximum.  G = 8 (256 threads, 4 KB of LDS, so that it
// fits on a CU beside the backward) or, when nothing runs beside it, 16.
// Every partial is combined in a fixed order, so the results do not depend on
// scheduling.
// ---------------------------------------------------------------------------
constexpr int CMB_THREADS = 512;
constexpr int CMB_WAVES = CMB_THREADS / 64;   // 8
constexpr int DA_GROUPS = 8;        // beside the backward: 256 threads, 4 KB of LDS
constexpr int DA_GROUPS_WIDE = 16;  // on the model's stream, where nothing runs beside it

// (m, s) <- the merge of two (maximum, sum of 2^(x - maximum)) pairs, base 2 or
// natural alike through exp_fast (natural logarithms here)
__device__ __forceinline__ void ms_merge_ln(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;
  s = (m == -INFINITY ? 0.0f : s * exp_fast(m - mm)) + (m2 == -INFINITY ? 0.0f : s2 * exp_fast(m2 - mm));
  m = mm;
}

// Group grp's online merge of splits grp, grp + 16, ...: running maximum mg,
// sum St and (WITH_O) the weighted O of hidden units h4 .. h4 + 3.
template <bool WITH_O, int GROUPS>
__device__ __forceinline__ void merge_splits(int i, int splits, const float* __restrict__ m_part,
                                             const float* __restrict__ s_part, const float* __restrict__ o_part,
                                             int ld_part, int grp, int h4, float& mg, float& St, float4& O) {
  mg = -INFINITY;
  St = 0.0f;
  O = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll 8
  for (int s = grp; s < splits; s += GROUPS) {
    const size_t r = (size_t)s * ld_part + i;
    const float ms = m_part[r];
    const float ss = s_part[r];
    float4 o = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if constexpr (WITH_O) o = *reinterpret_cast<const float4*>(o_part + r * HID + h4);
    // (no split has -inf: each holds at least one label of finite bias)
    const float mn = fmaxf(mg, ms);
    const float a = exp_fast(mg - mn), e = exp_fast(ms - mn);
    St = fmaf(e, ss, St * a);
    if constexpr (WITH_O) {
      O.x = fmaf(e, o.x, O.x * a);
      O.y = fmaf(e, o.y, O.y * a);
      O.z = fmaf(e, o.z, O.z * a);
      O.w = fmaf(e, o.w, O.w * a);
    }
    mg = mn;
  }
}

// Row of workgroup b in a launch of one workgroup per row over n rows.
// Workgroups are dealt to the 8 XCDs in turn; giving each XCD a contiguous
// range of rows lets one L2 serve the cache lines that neighbouring rows share
// in the per-split (max, sum) arrays, instead of every XCD fetching them all.
__device__ __forceinline__ int xcd_row(int b, int n) { return n % 8 == 0 ? (b % 8) * (n / 8) + b / 8 : b; }

// dA1 of row i from the forward's partials, by a workgroup of GROUPS x 32
// threads (every thread calls it): each group merges its splits' O online
// against its own running maximum, then the groups are rescaled to the row's
// maximum; thread t < HID writes hidden unit t, with tw_t the row's mean target
// weight of that unit.  red_o [GROUPS][HID], red_s and red_m [GROUPS]: LDS.
template <int GROUPS>
__device__ __forceinline__ void da1_row(int i, int splits, const float* __restrict__ m_part,
                                        const float* __restrict__ s_part, const float* __restrict__ o_part,
                                        int ld_part, float tw_t, const float* __restrict__ A1, float invB,
                                        float* __restrict__ dA1, float (*red_o)[HID], float* red_s, float* red_m) {
  const int t = threadIdx.x;
  const int grp = t >> 5, h4 = (t & 31) * 4;
  float mg, St;
  float4 O;
  merge_splits<true, GROUPS>(i, splits, m_part, s_part, o_part, ld_part, grp, h4, mg, St, O);
  *reinterpret_cast<float4*>(&red_o[grp][h4]) = O;
  if ((t & 31) == 0) {
    red_s[grp] = St;
    red_m[grp] = mg;
  }
  __syncthreads();
  if (t < HID) {
    float M = red_m[0];
#pragma unroll
    for (int k = 1; k < GROUPS; ++k) M = fmaxf(M, red_m[k]);
    float Ot = 0.0f, Stot = 0.0f;
#pragma unroll
    for (int k = 0; k < GROUPS; ++k) {
      const float e = red_m[k] == -INFINITY ? 0.0f : exp_fast(red_m[k] - M);
      Ot = fmaf(e, red_o[k][t], Ot);
      Stot = fmaf(e, red_s[k], Stot);
    }
    const float dh = (Ot / Stot - tw_t) * invB;
    dA1[(size_t)i * HID + t] = A1[(size_t)i * HID + t] > 0.0f ? dh : 0.0f;
  }
}

// DA: the row's dA1 as well, in the same workgroup (16 split groups), for a
// step that runs it on the model's stream anyway: one launch instead of two.
template <bool BF16, bool DA>
__global__ __launch_bounds__(CMB_THREADS) void k_out_lse_targets(
    int splits, const float* __restrict__ m_part, const float* __restrict__ s_part, int ld_part,
    const float* __restrict__ W2, const float* __restrict__ b2, int L,
    const typename Mma<BF16>::elem* __restrict__ H1, CsrDev y, int has_y, float* __restrict__ lse_out,
    float* __restrict__ loss_rows, float* __restrict__ tw_out, const float* __restrict__ o_part,
    const float* __restrict__ A1, float invB, float* __restrict__ dA1) {
  static_assert(!DA || CMB_THREADS == 32 * DA_GROUPS_WIDE, "dA1 takes the workgroup as 16 split groups");
  __shared__ float red_s[CMB_WAVES];
  __shared__ float red_m[CMB_WAVES];
  __shared__ float red_t[CMB_WAVES][HID];
  __shared__ float red_z[CMB_WAVES];
  const int i = xcd_row((int)blockIdx.x, (int)gridDim.x), t = threadIdx.x, lane = t & 63, w = t >> 6;
  {
    float mg = -INFINITY, St = 0.0f;
    for (int k = t; k < splits; k += CMB_THREADS)
      ms_merge_ln(mg, St, m_part[(size_t)k * ld_part + i], s_part[(size_t)k * ld_part + i]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ms_merge_ln(mg, St, __shfl_xor(mg, o), __shfl_xor(St, o));
    if (lane == 0) {
      red_s[w] = St;
      red_m[w] = mg;
    }
  }
  // target terms: wave w takes labels q = w, w + 8, ... of row i, in that
  // order; lane owns hidden 2l, 2l+1.  The row's label ids are read
  // lane-parallel (every wave counts the valid ones), and a wave's W2 rows load
  // TGT_BATCH at a time ahead of their reductions.
  constexpr int TGT_BATCH = 4;
  float tw0 = 0.0f, tw1 = 0.0f, zw = 0.0f;
  int cnt = 0;
  if (has_y) {
    const int ybase = y.indptr[0];
    int ys = y.indptr[i], ye = y.indptr[i + 1];
    ys = max(ys, ybase);
    ye = min(ye, ybase + y.nnz);
    if (ye < ys) ye = ys;
    const float h0 = (float)H1[(size_t)i * HID + 2 * lane];
    const float h1v = (float)H1[(size_t)i * HID + 2 * lane + 1];
    for (int q0 = ys; q0 < ye; q0 += 64) {
      const int q = q0 + lane;
      const int lab = q < ye ? y.indices[q] : -1;
      cnt += __popcll(__ballot(lab >= 0 && lab < L));
    }
    // this wave's labels: the k-th is q = ys + w + 8k, k < mine; 64 per pass
    const int mine = (ye - ys - w + CMB_WAVES - 1) / CMB_WAVES;
    for (int k0 = 0; k0 < mine; k0 += 64) {
      const int qk = ys + w + CMB_WAVES * (k0 + lane);
      const int labv = k0 + lane < mine ? y.indices[qk] : -1;
      const int nk = min(64, mine - k0);
      for (int u0 = 0; u0 < nk; u0 += TGT_BATCH) {
        float2 wv[TGT_BATCH];
        float bv[TGT_BATCH];
        bool ok[TGT_BATCH];
#pragma unroll
        for (int u = 0; u < TGT_BATCH; ++u) {
          const int lab = __builtin_amdgcn_readlane(labv, min(u0 + u, nk - 1));
          ok[u] = u0 + u < nk && lab >= 0 && lab < L;
          const int lb = ok[u] ? lab : 0;
          wv[u] = *reinterpret_cast<const float2*>(W2 + (size_t)lb * HID + 2 * lane);
          bv[u] = b2[lb];
        }
#pragma unroll
        for (int u = 0; u < TGT_BATCH; ++u) {
          if (!ok[u]) continue;
          tw0 += wv[u].x;
          tw1 += wv[u].y;
          float o0 = wv[u].x, o1 = wv[u].y;
          if constexpr (BF16) {
            o0 = (float)(bf16)wv[u].x;
            o1 = (float)(bf16)wv[u].y;
          }
          zw += wave_sum(fmaf(h0, o0, h1v * o1)) + bv[u];
        }
      }
    }
    red_t[w][2 * lane] = tw0;
    red_t[w][2 * lane + 1] = tw1;
    if (lane == 0) red_z[w] = zw;
  }
  __syncthreads();
  float my_tw = 0.0f;
  if (t < HID) {
    float M = red_m[0], Stot = red_s[0];
#pragma unroll
    for (int k = 1; k < CMB_WAVES; ++k) ms_merge_ln(M, Stot, red_m[k], red_s[k]);
    const float lse = M + logf(Stot);
    if (t == 0) lse_out[i] = lse;
    if (has_y) {
      float tw = red_t[0][t], zs = red_z[0];
#pragma unroll
      for (int k = 1; k < CMB_WAVES; ++k) {
        tw += red_t[k][t];
        zs += red_z[k];
      }
      const float inv_cnt = cnt > 0 ? 1.0f / (float)cnt : 0.0f;
      tw_out[(size_t)i * HID + t] = tw * inv_cnt;
      my_tw = tw * inv_cnt;
      if (t == 0) loss_rows[i] = lse - zs * inv_cnt;
    }
  }
  if constexpr (DA) {
    __shared__ float red_o[DA_GROUPS_WIDE][HID];
    __shared__ float red_s2[DA_GROUPS_WIDE];
    __shared__ float red_m2[DA_GROUPS_WIDE];
    da1_row<DA_GROUPS_WIDE>(i, splits, m_part, s_part, o_part, ld_part, my_tw, A1, invB, dA1, red_o, red_s2,
                            red_m2);
  }
}

template <int GROUPS>
__global__ __launch_bounds__(32 * GROUPS) void k_out_dA1(int splits, const float* __restrict__ m_part,
                                                        const float* __restrict__ s_part,
                                                        const float* __restrict__ o_part, int ld_part,
                                                        const float* __restrict__ tw, const float* __restrict__ A1,
                                                        float invB, float* __restrict__ dA1) {
  __shared__ float red_o[GROUPS][HID];
  __shared__ float red_s[GROUPS];
  __shared__ float red_m[GROUPS];
  const int i = xcd_row((int)blockIdx.x, (int)gridDim.x), t = threadIdx.x;
  const float tw_t = t < HID ? tw[(size_t)i * HID + t] : 0.0f;
  da1_row<GROUPS>(i, splits, m_part, s_part, o_part, ld_part, tw_t, A1, invB, dA1, red_o, red_s, red_m);
}

hipError_t launch_out_lse_targets(bool use_bf16, int B, int splits, const float* m_part, const float* s_part,
                                  int ld_part, const float* W2, const float* b2, int L, const void* H1,
                                  const CsrDev* y, float* lse, float* loss_rows, float* tw, const float* o_part,
                                  const float* A1, float* dA1, hipStream_t st, hipEvent_t done) {
  CsrDev yy = y ? *y : CsrDev{0, 0, 0, nullptr, nullptr, nullptr};
  const bool da = y && dA1;
  const float invB = 1.0f / (float)B;
  auto go = [&](auto kern, auto* h1) {
    if (done)
      hipExtLaunchKernelGGL(kern, dim3(B), dim3(CMB_THREADS), 0, st, nullptr, done, 0, splits, m_part, s_part, ld_part,
                            W2, b2, L, h1, yy, (int)(y != nullptr), lse, loss_rows, tw, o_part, A1, invB, dA1);
    else
      hipLaunchKernelGGL(kern, dim3(B), dim3(CMB_THREADS), 0, st, splits, m_part, s_part, ld_part, W2, b2, L, h1, yy,
                         y != nullptr, lse, loss_rows, tw, o_part, A1, invB, dA1);
  };
  if (use_bf16) {
    if (da)
      go(k_out_lse_targets<true, true>, (const bf16*)H1);
    else
      go(k_out_lse_targets<true, false>, (const bf16*)H1);
  } else {
    if (da)
      go(k_out_lse_targets<false, true>, (const float*)H1);
    else
      go(k_out_lse_targets<false, false>, (const float*)H1);
  }
  return hipGetLastError();
}

hipError_t launch_out_dA1(int B, int splits, const float* m_part, const float* s_part, const float* o_part,
                          int ld_part, const float* tw, const float* A1, float* dA1, bool wide, hipStream_t st) {
  if (wide)
    hipLaunchKernelGGL(k_out_dA1<DA_GROUPS_WIDE>, dim3(B), dim3(32 * DA_GROUPS_WIDE), 0, st, splits, m_part, s_part,
                       o_part, ld_part, tw, A1, 1.0f / (float)B, dA1);
  else
    hipLaunchKernelGGL(k_out_dA1<DA_GROUPS>, dim3(B), dim3(32 * DA_GROUPS), 0, st, splits, m_part, s_part, o_part,
                       ld_part, tw, A1, 1.0f / (float)B, dA1);
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
__global__ __launch_bounds__(FWD_THREADS) void k_out_fwd_topk(
    const float* __restrict__ W2, const float* __restrict__ b2, int L,
    const typename Mma<BF16>::elem* __restrict__ H1, int B, int tiles_per_split, int n_tiles,
    int k, float* __restrict__ part_s, int32_t* __restrict__ part_i, int ld_part) {
  using M = Mma<BF16>;
  using E = typename M::elem;
  using Fr = typename M::frag;
  constexpr int NB = FwdShape<BF16>::NB;
  constexpr int RB = FwdShape<BF16>::RB;
  constexpr int NCH = 32 / M::KC;
  constexpr int WROWS = 32 * NB;
  __shared__ __attribute__((aligned(16))) E wr[2][tile_elems<BF16>()];
  __shared__ __attribute__((aligned(16))) float bt[2][OUT_TILE];
  __shared__ float ls[FwdShape<BF16>::WAVES][WROWS][TOPK_MAX];
  __shared__ int li[FwdShape<BF16>::WAVES][WROWS][TOPK_MAX];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 5, n = lane & 31;
  const int split = blockIdx.x;
  const int t_begin = split * tiles_per_split;
  const int t_end = min(n_tiles, t_begin + tiles_per_split);
  const int row0 = blockIdx.y * RB + wave * WROWS;
  const bool active = row0 < B;
  const W2Src src = w2_src(W2, b2, L);
  const int rbase[2] = {tw_row_base(n, g, 0), tw_row_base(n, g, 1)};

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
      for (int c = 0; c < NCH; ++c) hf[nb][kb][c] = h1_frag<BF16>(hrow, kb, c, g);
  }
  // W2 tiles are loaded three ahead: at the start of iteration t, tile t is in
  // LDS buffer (t - t_begin) & 1 and tiles t+1, t+2, t+3 are in the register
  // sets tr0, tr1, tr2 in turn (the loop is unrolled by three so that every
  // set is named statically); iteration t moves tile t+1 into the other
  // buffer and reloads its set with tile t+4.
  const int t_last = t_end - 1;
  TileRegs tr0, tr1, tr2;
  if (t_begin < t_end) {
    tile_load(src, t_begin, tr0);
    tile_store<BF16, false>(tr0, L, t_begin, wr[0], nullptr, bt[0]);
    tile_load(src, min(t_begin + 1, t_last), tr0);
    tile_load(src, min(t_begin + 2, t_last), tr1);
    tile_load(src, min(t_begin + 3, t_last), tr2);
  }
  __syncthreads();
  auto iteration = [&](int t, TileRegs& trn) {
    const int buf = (t - t_begin) & 1;
    if (active) {
      // the accumulators start from the biases of the tile's labels (rows of Z^T)
      f32x16 z[NB];
      {
        const float4* bq = reinterpret_cast<const float4*>(bt[buf]);
        f32x16 zb;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 bv = bq[2 * q + g];
          zb[4 * q + 0] = bv.x; zb[4 * q + 1] = bv.y; zb[4 * q + 2] = bv.z; zb[4 * q + 3] = bv.w;
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) z[nb] = zb;
      }
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const Fr a = tile_frag_w<BF16>(wr[buf], rbase, n, kb, c, g);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) z[nb] = M::mma(a, hf[nb][kb][c], z[nb]);
        }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int rloc = nb * 32 + n;
        const bool rvalid = row0 + rloc < B;
        // skip the tile unless some lane's best score reaches its row's k-th
        // entry (NaN never does; ties go to the exact test below)
        float m = z[nb][0];
#pragma unroll
        for (int r = 1; r < 16; ++r) m = fmaxf(m, z[nb][r]);
        if (!__any(rvalid && m >= ls[wave][rloc][k - 1])) continue;
        for (int half = 0; half < 2; ++half) {
          if (g == half && rvalid) {
            float* lsr = ls[wave][rloc];
            int* lir = li[wave][rloc];
            // the row's current k-th entry, re-read only after an insertion:
            // most scores fail this test and touch no LDS
            float ts = lsr[k - 1];
            int ti = lir[k - 1];
            for (int r = 0; r < 16; ++r) {
              const int ll = 8 * (r >> 2) + 4 * g + (r & 3);
              const int id = t * OUT_TILE + ll;
              const float sc = z[nb][r];
              if (id >= L || !(sc == sc)) continue;  // NaN scores are never ranked
              if (!better(sc, id, ts, ti)) continue;
              int pos = k - 1;
              while (pos > 0 && better(sc, id, lsr[pos - 1], lir[pos - 1])) {
                lsr[pos] = lsr[pos - 1];
                lir[pos] = lir[pos - 1];
                --pos;
              }
              lsr[pos] = sc;
              lir[pos] = id;
              ts = lsr[k - 1];
              ti = lir[k - 1];
            }
          }
        }
      }
    }
    if (t + 1 < t_end) tile_store<BF16, false>(trn, L, t + 1, wr[buf ^ 1], nullptr, bt[buf ^ 1]);
    if (t + 4 <= t_last) tile_load(src, t + 4, trn);
    __syncthreads();
  };
  for (int t = t_begin; t < t_end; t += 3) {
    iteration(t, tr0);
    if (t + 1 >= t_end) break;
    iteration(t + 1, tr1);
    if (t + 2 >= t_end) break;
    iteration(t + 2, tr2);
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
  const dim3 grid(s_eff, (B + RB - 1) / RB), block(FWD_THREADS);
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
