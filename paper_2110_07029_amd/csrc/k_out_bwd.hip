// Output-layer backward and SGD update of W2 / b2 (Sec. 2.1: backward pass,
// then the update pass), fused so that W2 crosses HBM once in each direction.
//
// Work unit = 32 labels (one wavefront).  For each 32-row block of the batch:
//   Z   = H1 W2_blk^T + b2          (matrix cores, recomputed; logits are never stored)
//   dZ  = (exp(Z - lse) - T) / B    (T = 1/|Y_i| on true labels, from a bit mask)
//   dW2_blk^T += H1^T dZ            (dZ fed straight from the accumulators)
//   db2 += column sums of dZ
// then W2_blk -= lr dW2_blk and b2 -= lr db2 from the fp32 master values the
// lane itself loaded (the accumulator-compatible K order makes the lane that
// loads a weight the lane that owns its gradient).
//
// With bf16 operands H1 is staged in LDS, in the conflict-free tile layout of
// the forward (row stride 160, 16-byte chunks permuted by the row): the logits
// read H1 rows with 16-byte reads, the dW2 product reads H1^T with transposed
// reads (ds_read_b64_tr_b16) from the same copy.  Three kernels, all with
// persistent workgroups:
//   k_out_bwd_prefetch (B <= 256, bf16): 4 wavefronts, the whole batch staged
//           once per workgroup; each wave walks its own label blocks with no
//           barrier, W2 rows moving whole through an LDS staging tile;
//   k_out_bwd, chunked (B > 256, bf16): 8 wavefronts (2 per SIMD); the
//           workgroup takes 8 label blocks at a time and streams the batch
//           through two LDS buffers in 128-row chunks, the dW2 accumulators
//           staying in registers across chunks: while one chunk is in use the
//           next one is copied from global memory straight into the other
//           buffer (global_load_lds, no registers in between);
//   k_out_bwd, global (fp32 operands): H1 and H1^T read from their
//           L2-resident global copies.
#include <hip/hip_ext.h>
#include <math.h>

#include <type_traits>

#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

constexpr int BWD_WAVES = 8;
constexpr int BWD_THREADS = 64 * BWD_WAVES;
constexpr int BWD_CHUNK = 256;  // batches up to this size are staged whole (k_out_bwd_prefetch)
constexpr int BWD_CROWS = 128;  // rows per H1 chunk of the chunked kernel (two chunk buffers)

enum BwdMode { BWD_GLOBAL = 0, BWD_STAGED = 1, BWD_CHUNKED = 2 };  // STAGED: k_out_bwd_prefetch

// Copy rows [r0, r0 + nrows) of H1 (row-major, ld HID) into the LDS tile (row
// r of the chunk at tw_off(r, .)); nrows is a multiple of 32 and inside the
// padded batch (rows past B are zero).  16 lanes store one row: conflict-free.
__device__ __forceinline__ void stage_h1(bf16* h1s, const bf16* __restrict__ H1, int r0, int nrows) {
  for (int e = threadIdx.x; e < nrows * 16; e += BWD_THREADS) {
    const int r = e >> 4, c = e & 15;
    const uint4 v = *reinterpret_cast<const uint4*>(H1 + (size_t)(r0 + r) * HID + c * 8);
    *reinterpret_cast<uint4*>(h1s + r * TW_LD + 8 * (c ^ ((r >> 2) & 3))) = v;
  }
}

// One 16-byte direct copy per lane from global memory into LDS: lane l's
// bytes land at LDS byte lds + 16 l (lds: wave-uniform LDS byte address).
// Written as inline asm so that the compiler's wait-count pass does not treat
// every later LDS access as dependent on the copy (it cannot tell the target
// apart from other LDS data): the kernel waits for its copies itself.  No
// other code in the kernel uses M0.
__device__ __forceinline__ void lds_copy16(const void* src, unsigned lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds)
               : "memory");
}

// RS > 1 (global mode only): the RS wavefronts of a label block split its row
// blocks (rb = rp, rp + RS, ...) and their dW2 / db2 partials meet in LDS, for
// label spaces too small to give every wavefront a block of its own.
template <bool BF16, int MODE, int RS>
__global__ __launch_bounds__(BWD_THREADS) void k_out_bwd(
    float* __restrict__ W2, float* __restrict__ b2, int L,
    const typename Mma<BF16>::elem* __restrict__ H1, const typename Mma<BF16>::elem* __restrict__ H1T,
    int ld_t, int B, const float* __restrict__ lse, const float* __restrict__ rw,
    const int32_t* __restrict__ lbeg, const int32_t* __restrict__ lpair, float lr, float invB,
    float log2_invB) {
  using M = Mma<BF16>;
  using E = typename M::elem;
  using Fr = typename M::frag;
  constexpr int NCH = 32 / M::KC;
  constexpr bool LDS_H1 = MODE != BWD_GLOBAL;
  static_assert(!LDS_H1 || BF16, "LDS staging is for bf16 operands");
  static_assert(MODE != BWD_STAGED, "B <= 256 with bf16 operands runs k_out_bwd_prefetch");
  static_assert(RS == 1 || (MODE == BWD_GLOBAL && BWD_WAVES % RS == 0), "row split: global mode");
  constexpr int LPW = BWD_WAVES / RS;  // label blocks per workgroup at a time (row split)
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  const int nrb = (B + 31) >> 5;
  const int bpad = nrb * 32;
  // rows whose target bits are held at once
  const int span = MODE == BWD_CHUNKED ? BWD_CROWS : bpad;
  const int mstride = span >> 5;  // mask words per label
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5, n = lane & 31;

  char* sp = smem_raw;
  E* h1b = nullptr;  // two chunk buffers of BWD_CROWS rows
  if constexpr (LDS_H1) {
    h1b = reinterpret_cast<E*>(sp);
    sp += 2 * BWD_CROWS * TW_LD * sizeof(E);
  }
  // per row of the batch: the logits' accumulator starts at
  // crow = (log2(1/B) - lse*log2(e)) / log2(e) (-inf for rows past B), so that
  // dZ = 2^(z*log2(e) + bias*log2(e)) = softmax/B with one fma; tw = (1/|Y_i|)/B
  float* crow_s = reinterpret_cast<float*>(sp);
  sp += bpad * sizeof(float);
  float* tw_s = reinterpret_cast<float*>(sp);
  sp += bpad * sizeof(float);
  uint32_t* mask = reinterpret_cast<uint32_t*>(sp) + wave * 32 * mstride;
  sp += BWD_WAVES * 32 * mstride * sizeof(uint32_t);
  // row split: the partial dW2 (64 values per lane) and db2 of wavefronts rp > 0
  float* red = reinterpret_cast<float*>(sp);

  // Row constants of rows [r0, r0 + nrows) at LDS index (row - r0).
  auto stage_rows = [&](int r0, int nrows) {
    for (int i = tid; i < nrows; i += BWD_THREADS) {
      const int r = r0 + i;
      crow_s[i] = r < B ? (log2_invB - lse[r] * LOG2E) * LN2 : -INFINITY;
      tw_s[i] = r < B ? rw[r] * invB : 0.0f;
    }
  };
  // Target bits of this wave's labels for rows [r0, r0 + nrows): mask[label][row block],
  // from the block's (row << 5 | label % 32) pairs in lpair[lo, hi); pr_first is
  // the lane's pair lo + lane, loaded once per block (-1: none).
  auto build_mask = [&](int lo, int hi, int pr_first, int r0, int nrows) {
    for (int k = lane; k < 32 * mstride; k += 64) mask[k] = 0u;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    auto put = [&](int pr) {
      const int row = (pr >> 5) - r0;
      if (row >= 0 && row < nrows)
        atomicOr(&mask[(pr & 31) * mstride + (row >> 5)], 1u << (row & 31));
    };
    if (pr_first >= 0) put(pr_first);
    for (int q = lo + 64 + lane; q < hi; q += 64) put(lpair[q]);
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  };

  // Rows [c0, c0 + BWD_CROWS) of H1 into chunk buffer dst, in the tile layout
  // of stage_h1, by direct global-to-LDS copies: a wave's 16-byte copy fills
  // 1024 consecutive LDS bytes (lane l at byte 16 l), so each lane picks the
  // global chunk that belongs at its LDS slot; the 4 pad slots of a row (bytes
  // 256..319) take an arbitrary chunk of the row.  The rows read stay below
  // round_up(B, BWD_CROWS), inside the H1 buffer (checked by the host).
  auto issue_chunk = [&](int c0, E* dst) {
    if constexpr (MODE == BWD_CHUNKED) {
      constexpr int ROW_B = TW_LD * (int)sizeof(E);  // 320 bytes
      constexpr int N_COPY = BWD_CROWS * ROW_B / 1024;
      static_assert(N_COPY % BWD_WAVES == 0, "chunk copies split evenly over the waves");
      const int wv = __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
      for (int j = 0; j < N_COPY / BWD_WAVES; ++j) {
        const int blk_b = (j * BWD_WAVES + wv) * 1024;
        const int o = blk_b + lane * 16;
        const int r = o / ROW_B;
        const int slot = (o - r * ROW_B) >> 4;
        const int c = slot < 16 ? (slot ^ ((r >> 2) & 3)) : 0;
        lds_copy16(H1 + (size_t)(c0 + r) * HID + 8 * c,
                   __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)dst + blk_b));
      }
    }
  };

  stage_rows(0, bpad);
  __syncthreads();
  // the lane's bases in the LDS tile: H1 row fragments (rows 32 rb + n) and
  // transposed H1^T fragments (hidden 32 hb + n); every offset below is rb, kb,
  // hb, c or hi times a constant
  const int rbase[2] = {tw_row_base(n, g, 0), tw_row_base(n, g, 1)};
  const int cbase[2] = {tw_col_base(lane, 0), tw_col_base(lane, 1)};

  const int n_blocks = (L + 31) >> 5;
  // global: each wave walks its own blocks; chunked: the workgroup walks
  // groups of 8 blocks together (a uniform trip count for the barriers)
  // (row split: groups of LPW blocks, walked by the workgroup together)
  const int n_iter_units = MODE == BWD_CHUNKED ? (n_blocks + BWD_WAVES - 1) / BWD_WAVES
                           : RS > 1            ? (n_blocks + LPW - 1) / LPW
                                               : n_blocks;
  const int first = MODE == BWD_CHUNKED || RS > 1 ? blockIdx.x : blockIdx.x * BWD_WAVES + wave;
  const int step = MODE == BWD_CHUNKED || RS > 1 ? gridDim.x : gridDim.x * BWD_WAVES;
  const int rp = RS > 1 ? wave % RS : 0;  // this wavefront's share of the row blocks
  // chunked: chunks are consumed in the order (unit, chunk); kc counts them,
  // and chunk kc lives in buffer kc & 1.  The first one is requested here.
  const int nch = (bpad + BWD_CROWS - 1) / BWD_CROWS;
  int kc = 0;
  if (MODE == BWD_CHUNKED && first < n_iter_units) issue_chunk(0, h1b);
  for (int unit = first; unit < n_iter_units; unit += step) {
    const int blk = MODE == BWD_CHUNKED ? unit * BWD_WAVES + wave : RS > 1 ? unit * LPW + wave / RS : unit;
    const bool bactive = blk < n_blocks;
    const int l0 = blk * 32;
    const int label = l0 + n;
    const bool lvalid = label < L;
    // W2 rows of this block (fp32 master): hidden 32*kb + 8*q + 4*g + (0..3) per lane.
    // Loads of labels past L read the last row (valid memory) and are never stored.
    float4 wreg[4][4];
    const float* wrow = W2 + (size_t)min(label, L - 1) * HID;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        wreg[kb][q] = *reinterpret_cast<const float4*>(wrow + 32 * kb + 8 * q + 4 * g);
    const float bias = b2[min(label, L - 1)];
    const float bb = lvalid ? bias * LOG2E : -INFINITY;
    // operand fragments of W2 (K = hidden), converted once per block.  bf16:
    // the logits take 8 consecutive hidden units per lane (32kb + 16c + 8g ..
    // + 7, matching the 16-byte H1 reads); the lane holds units 8q + 4g + 0..3,
    // so the two lane halves trade one float4 per pair with v_permlane32_swap
    // (its two results are exactly the pair's lo and hi halves on both halves).
    Fr wf[4][NCH];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        if constexpr (BF16) {
          const float4 a4 = wreg[kb][2 * c], b4 = wreg[kb][2 * c + 1];
          const float av[4] = {a4.x, a4.y, a4.z, a4.w}, bv[4] = {b4.x, b4.y, b4.z, b4.w};
          Fr f;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const auto sw = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, av[j]),
                                                             __builtin_bit_cast(unsigned, bv[j]), false, false);
            f[j] = (bf16)__builtin_bit_cast(float, sw[0]);
            f[4 + j] = (bf16)__builtin_bit_cast(float, sw[1]);
          }
          wf[kb][c] = f;
        } else {
          const float4 v = wreg[kb][c >> 2];
          const float vs[4] = {v.x, v.y, v.z, v.w};
          wf[kb][c] = vs[c & 3];
        }
      }

    // true (row, label) pairs of these 32 labels
    int lo = 0, hi = 0;
    if (bactive) {
      lo = lbeg[blk];
      hi = lbeg[blk + 1];
    }
    const bool has_targets = hi > lo;
    const int pr0 = lo + lane < hi ? lpair[lo + lane] : -1;

    f32x16 accw[4];
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int r = 0; r < 16; ++r) accw[hb][r] = 0.0f;
    float db2p = 0.0f;

    // one 32-row block of the batch (rows grow0 ..): rb indexes its rows in
    // the H1 chunk buffer hbuf and in the target mask
    auto row_block = [&](const E* hbuf, int rb, int grow0) {
      // the accumulator starts at the row constants of rows 8*q + 4*g + (0..3)
      f32x16 z;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 c4 = *reinterpret_cast<const float4*>(crow_s + grow0 + 8 * q + 4 * g);
        z[4 * q + 0] = c4.x; z[4 * q + 1] = c4.y; z[4 * q + 2] = c4.z; z[4 * q + 3] = c4.w;
      }
      if constexpr (LDS_H1) {
        const E* t = hbuf + rb * 32 * TW_LD;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int c = 0; c < NCH; ++c)
            z = M::mma(*reinterpret_cast<const bf16x8*>(t + rbase[c] + 32 * kb), wf[kb][c], z);
      } else {
        const E* hrow = H1 + (size_t)(grow0 + n) * HID;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int c = 0; c < NCH; ++c) z = M::mma(frag_row<BF16>(hrow + 32 * kb, c, g), wf[kb][c], z);
      }
      float dz[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) dz[r] = __builtin_amdgcn_exp2f(fmaf(z[r], LOG2E, bb));
      if (has_targets) {
        const uint32_t mw = mask[n * mstride + rb];
        if (__any(mw != 0u)) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int rl = 8 * (r >> 2) + 4 * g + (r & 3);
            if ((mw >> rl) & 1u) dz[r] -= tw_s[grow0 + rl];
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) db2p += dz[r];
      // dW2^T += H1^T dZ : A = H1^T rows (M = hidden, K = rows), B = dZ from the accumulators.
      Fr df[NCH];
#pragma unroll
      for (int c = 0; c < NCH; ++c) df[c] = frag_acc<BF16>(dz, c);
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) {
        if constexpr (LDS_H1) {
#pragma unroll
          for (int c = 0; c < NCH; ++c) {
            const E* o = hbuf + (rb * 32 + 16 * c) * TW_LD + 32 * hb;
            const bf16x4 lo4 = lds_read_tr16(o + cbase[0]), hi4 = lds_read_tr16(o + cbase[1]);
            bf16x8 af;
            af[0] = lo4[0]; af[1] = lo4[1]; af[2] = lo4[2]; af[3] = lo4[3];
            af[4] = hi4[0]; af[5] = hi4[1]; af[6] = hi4[2]; af[7] = hi4[3];
            accw[hb] = M::mma(af, df[c], accw[hb]);
          }
        } else {
          const E* trow = H1T + (size_t)(32 * hb + n) * ld_t + grow0;
#pragma unroll
          for (int c = 0; c < NCH; ++c) accw[hb] = M::mma(frag_row<BF16>(trow, c, g), df[c], accw[hb]);
        }
      }
    };

    if constexpr (MODE == BWD_CHUNKED) {
      for (int ci = 0; ci < nch; ++ci, ++kc) {
        const int c0 = ci * BWD_CROWS;
        const int crows = min(BWD_CROWS, bpad - c0);
        const E* cur = h1b + (kc & 1) * (BWD_CROWS * TW_LD);
        // this thread's copies into cur have landed; after the barrier all of
        // cur is there and every wave is done with the other buffer
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (ci + 1 < nch || unit + step < n_iter_units)
          issue_chunk(ci + 1 < nch ? c0 + BWD_CROWS : 0, h1b + ((kc + 1) & 1) * (BWD_CROWS * TW_LD));
        if (has_targets) build_mask(lo, hi, pr0, c0, crows);
        if (bactive)
          for (int rb = 0; rb < (crows >> 5); ++rb) row_block(cur, rb, c0 + rb * 32);
      }
    } else {
      if (has_targets) build_mask(lo, hi, pr0, 0, bpad);
      if (bactive)
        for (int rb = rp; rb < nrb; rb += RS) row_block(nullptr, rb, rb * 32);
    }
    if constexpr (RS > 1) {
      // partials of wavefronts rp > 0 to LDS (value-major, lane-contiguous),
      // added by wavefront rp = 0 in rp order
      float* my = red + (size_t)((wave / RS) * (RS - 1) + rp - 1) * 65 * 64;
      if (rp > 0) {
#pragma unroll
        for (int hb = 0; hb < 4; ++hb)
#pragma unroll
          for (int r = 0; r < 16; ++r) my[(16 * hb + r) * 64 + lane] = accw[hb][r];
        my[64 * 64 + lane] = db2p;
      }
      __syncthreads();
      if (rp == 0) {
        for (int k = 1; k < RS; ++k) {
          const float* o = red + (size_t)((wave / RS) * (RS - 1) + k - 1) * 65 * 64;
#pragma unroll
          for (int hb = 0; hb < 4; ++hb)
#pragma unroll
            for (int r = 0; r < 16; ++r) accw[hb][r] += o[(16 * hb + r) * 64 + lane];
          db2p += o[64 * 64 + lane];
        }
      }
      __syncthreads();  // the slots are free again for the next group
    }

    const float db2 = db2p + __shfl_xor(db2p, 32);
    if (bactive && lvalid && rp == 0) {
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
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  }
}

// ---------------------------------------------------------------------------
// Staged batches (B <= 256, bf16) with the next label block's W2 in flight:
// 4 wavefronts, one per SIMD, each with the full register file.  While a wave
// works on one block of 32 labels, the next block's fp32 rows load into
// registers as whole 512-byte rows (the access pattern of a plain streaming
// update); once this block's updated rows have left through the wave's LDS
// staging tile, they enter it, and the products' operand layout is read from
// there.  Inside a block, each step issues the logits of row block rb+1 and
// the dW2 products of rb-1 to the matrix cores while the exponentials of rb
// are formed.
// ---------------------------------------------------------------------------
constexpr int BWP_WAVES = 4;
constexpr int BWP_SLD = 132;  // staging tile row stride (floats): conflict-free both ways
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int BWP_THREADS = 64 * BWP_WAVES;

__global__ __launch_bounds__(BWP_THREADS) void k_out_bwd_prefetch(
    float* __restrict__ W2, float* __restrict__ b2, int L, const bf16* __restrict__ H1, int B,
    const float* __restrict__ lse, const float* __restrict__ rw, const int32_t* __restrict__ lbeg,
    const int32_t* __restrict__ lpair, float lr, float invB, float log2_invB) {
  using M = Mma<true>;
  using Fr = M::frag;
  extern __shared__ __attribute__((aligned(16))) char smem_raw[];
  const int nrb = (B + 31) >> 5;
  const int bpad = nrb * 32;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, n = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  char* sp = smem_raw;
  bf16* h1s = reinterpret_cast<bf16*>(sp);
  sp += BWD_CHUNK * TW_LD * sizeof(bf16);
  float* crow_s = reinterpret_cast<float*>(sp);
  sp += bpad * sizeof(float);
  float* tw_s = reinterpret_cast<float*>(sp);
  sp += bpad * sizeof(float);
  uint32_t* mask = reinterpret_cast<uint32_t*>(sp) + wave * 32 * nrb;
  sp += BWP_WAVES * 32 * nrb * sizeof(uint32_t);
  // the wave's W2 staging tile: 32 label rows of 128 fp32, row stride BWP_SLD
  float* stage = reinterpret_cast<float*>(sp) + wave * 32 * BWP_SLD;

  for (int e = tid; e < bpad * 16; e += BWP_THREADS) {
    const int r = e >> 4, c = e & 15;
    const uint4 v = *reinterpret_cast<const uint4*>(H1 + (size_t)r * HID + c * 8);
    *reinterpret_cast<uint4*>(h1s + r * TW_LD + 8 * (c ^ ((r >> 2) & 3))) = v;
  }
  // per row: the logits' accumulator starts at crow = (log2(1/B) - lse*log2(e)) / log2(e)
  // (-inf past B), so that dZ = 2^(z*log2(e) + bias*log2(e)) = softmax/B with one fma
  for (int i = tid; i < bpad; i += BWP_THREADS) {
    crow_s[i] = i < B ? (log2_invB - lse[i] * LOG2E) * LN2 : -INFINITY;
    tw_s[i] = i < B ? rw[i] * invB : 0.0f;
  }
  __syncthreads();
  const int rbase[2] = {tw_row_base(n, g, 0), tw_row_base(n, g, 1)};
  const int cbase[2] = {tw_col_base(lane, 0), tw_col_base(lane, 1)};

  const int n_blocks = (L + 31) >> 5;
  const int step = gridDim.x * BWP_WAVES;
  // A block's 32 W2 rows move between HBM and the wave's staging tile whole:
  // load or store k covers rows 2k and 2k+1, 16 bytes per lane, so every
  // instruction reads or writes two full 512-byte rows.  The operand layout of
  // the products (lane (g, n): row n, hidden 32kb + 8q + 4g + 0..3) is read
  // from and written to the tile.  W2 and b2 are raw buffers addressed by the
  // lane's offset alone (the block's offset plus the lane's fixed offset plus
  // a constant per row pair), which the buffer's bounds check covers: rows
  // past L read zeros and their stores are dropped.  Also loaded: the block's bias (lane n: label
  // 32 blk + n) and pair range.
  const int crow_l = lane >> 5, ccol = 4 * (lane & 31);  // this lane's row pair slot and column
  const __amdgpu_buffer_rsrc_t w2r = __builtin_amdgcn_make_buffer_rsrc(W2, (short)0, L * HID * 4, BUF_RSRC_WORD3);
  const __amdgpu_buffer_rsrc_t b2r = __builtin_amdgcn_make_buffer_rsrc(b2, (short)0, L * 4, BUF_RSRC_WORD3);
  const int voff = (crow_l * HID + ccol) * 4;
  float4 nv[16];
  float nbias;
  int npr;       // the block's pair lo + lane (-1: none)
  int nlo, nhi;  // its pair range [nlo, nhi), read one block earlier
  auto load_blk = [&](int b, int plo, int phi) {
    const int vb = voff + b * 32 * HID * 4;
#pragma unroll
    for (int k = 0; k < 16; ++k)
      nv[k] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(w2r, vb + k * 2 * HID * 4, 0, 0));
    nbias = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(b2r, n * 4 + b * 32 * 4, 0, 0));
    npr = plo + lane < phi ? lpair[plo + lane] : -1;
    nlo = plo;
    nhi = phi;
  };
  auto stage_frag = [&](int kb, int q) -> float4& {
    return *reinterpret_cast<float4*>(stage + n * BWP_SLD + 32 * kb + 8 * q + 4 * g);
  };

  // The loaded block enters the staging tile right after the previous block's
  // stores, and the block after it is requested at once: every iteration then
  // issues the same memory instructions in the same order (the next block's
  // 17 loads, this block's 16 row stores and one b2 store), so the wait for a
  // block's loads never includes the stores issued after them.
  // (The bias and the first 64 pairs wait in the tile's pad columns HID and
  // HID + 1 + g of row n: a register copy of a loaded value would make the
  // compiler wait for the load right away.)  The pair range of a block is read
  // one block before its loads are issued, so that the pair load need not wait.
  int lo, hi;
  auto stage_loaded = [&]() {
#pragma unroll
    for (int k = 0; k < 16; ++k) *reinterpret_cast<float4*>(stage + (2 * k + crow_l) * BWP_SLD + ccol) = nv[k];
    if (g == 0) stage[n * BWP_SLD + HID] = nbias;
    stage[n * BWP_SLD + HID + 1 + g] = __builtin_bit_cast(float, npr);
    lo = nlo;
    hi = nhi;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  };
  const int first = blockIdx.x * BWP_WAVES + wave;
  if (first >= n_blocks) return;
  load_blk(first, lbeg[first], lbeg[first + 1]);
  stage_loaded();
  {
    const int b = min(first + step, n_blocks - 1);
    load_blk(b, lbeg[b], lbeg[b + 1]);
  }
  for (int blk = first; blk < n_blocks; blk += step) {
    const int bn2 = min(blk + 2 * step, n_blocks - 1);  // the block loaded at the end of this one
    const int plo = lbeg[bn2], phi = lbeg[bn2 + 1];
    const float bias = stage[n * BWP_SLD + HID];
    const int pr0 = __builtin_bit_cast(int, stage[n * BWP_SLD + HID + 1 + g]);
    const int label = blk * 32 + n;
    const bool lvalid = label < L;
    const float bb = lvalid ? bias * LOG2E : -INFINITY;
    // bf16 fragments of the logits' W2 operand: 8 consecutive hidden units per
    // lane (32kb + 16c + 8g .. + 7), read from the staging tile; kept in
    // accumulation registers (matrix instructions read their operands from
    // either half of the register file), which leaves the vector registers to
    // the next block's loads and to deep LDS read pipelines
    Fr wf[4][2];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const float* src = stage + n * BWP_SLD + 32 * kb + 16 * c + 8 * g;
        const float4 a4 = *reinterpret_cast<const float4*>(src);
        const float4 b4 = *reinterpret_cast<const float4*>(src + 4);
        Fr f;
        f[0] = (bf16)a4.x; f[1] = (bf16)a4.y; f[2] = (bf16)a4.z; f[3] = (bf16)a4.w;
        f[4] = (bf16)b4.x; f[5] = (bf16)b4.y; f[6] = (bf16)b4.z; f[7] = (bf16)b4.w;
        i32x4 fi = __builtin_bit_cast(i32x4, f);
        asm volatile("" : "+a"(fi));
        wf[kb][c] = __builtin_bit_cast(Fr, fi);
      }

    const bool has_targets = hi > lo;
    if (has_targets) {
      for (int k = lane; k < 32 * nrb; k += 64) mask[k] = 0u;
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      auto put = [&](int pr) {
        const int row = pr >> 5;
        atomicOr(&mask[(pr & 31) * nrb + (row >> 5)], 1u << (row & 31));
      };
      if (pr0 >= 0) put(pr0);
      for (int q = lo + 64 + lane; q < hi; q += 64) put(lpair[q]);
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
    f32x16 accw[4];
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int r = 0; r < 16; ++r) accw[hb][r] = 0.0f;
    float db2p = 0.0f;

    // The row-block loop, specialised on whether the block has true labels in
    // this batch (most blocks of a wide label space have none), so that its
    // body is straight-line code.  Step rb has two phases: (A) every LDS read
    // of the step (H1^T fragments of row block rb, H1 rows and row constants of
    // rb+1), then (B) the matrix work of two row blocks, the logits of rb+1 and
    // the dW2 products of rb-1, beside the vector work of rb (exponentials,
    // target terms, db2, the bf16 dZ operands).  A row block's dW2 products thus
    // wait one step for their operands and never stand alone at the end of a
    // step.  The scheduling barriers keep the reads ahead of the arithmetic
    // that hides their latency.
    auto rows = [&](auto targets) {
      constexpr bool TGT = decltype(targets)::value;
      auto read_rows = [&](int rb, bf16x8 (&hr)[4][2], f32x16& c) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 c4 = *reinterpret_cast<const float4*>(crow_s + rb * 32 + 8 * q + 4 * g);
          c[4 * q + 0] = c4.x; c[4 * q + 1] = c4.y; c[4 * q + 2] = c4.z; c[4 * q + 3] = c4.w;
        }
        const bf16* t = h1s + rb * 32 * TW_LD;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2) hr[kb][c2] = *reinterpret_cast<const bf16x8*>(t + rbase[c2] + 32 * kb);
      };
      // per row: the accumulator starts at the row constant, then Z += H1 W2^T
      auto logits = [&](const bf16x8 (&hr)[4][2], f32x16 z) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int c = 0; c < 2; ++c) z = M::mma(hr[kb][c], wf[kb][c], z);
        return z;
      };
      auto dw2 = [&](const bf16x8 (&at)[4][2], const Fr (&df)[2]) {
#pragma unroll
        for (int hb = 0; hb < 4; ++hb)
#pragma unroll
          for (int c = 0; c < 2; ++c) accw[hb] = M::mma(at[hb][c], df[c], accw[hb]);
      };
      // Two sets of per-row-block state alternate (no copies): the logits, the
      // H1^T fragments and the bf16 dZ of a row block.
      f32x16 za, zb;
      bf16x8 ata[4][2], atb[4][2];
      Fr dfa[2], dfb[2];
      {
        bf16x8 hr[4][2];
        read_rows(0, hr, za);
        za = logits(hr, za);
      }
      // row block rb from z (its logits) into (at, df); the logits of rb + 1
      // into zn; the dW2 products of rb - 1 from (atp, dfp) when PREV
      auto step = [&](auto prev, int rb, const f32x16& z, f32x16& zn, bf16x8 (&at)[4][2], Fr (&df)[2],
                      const bf16x8 (&atp)[4][2], const Fr (&dfp)[2]) {
        // (A)
#pragma unroll
        for (int hb = 0; hb < 4; ++hb)
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const bf16* o = h1s + (rb * 32 + 16 * c) * TW_LD + 32 * hb;
            const bf16x4 lo4 = lds_read_tr16(o + cbase[0]), hi4 = lds_read_tr16(o + cbase[1]);
            bf16x8 af;
            af[0] = lo4[0]; af[1] = lo4[1]; af[2] = lo4[2]; af[3] = lo4[3];
            af[4] = hi4[0]; af[5] = hi4[1]; af[6] = hi4[2]; af[7] = hi4[3];
            at[hb][c] = af;
          }
        // next row block (the last step recomputes a block and drops it)
        bf16x8 hr[4][2];
        read_rows(min(rb + 1, nrb - 1), hr, zn);
        uint32_t mw = 0;
        float tv[16];
        if constexpr (TGT) {
          mw = mask[n * nrb + rb];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float4 t4 = *reinterpret_cast<const float4*>(tw_s + rb * 32 + 8 * q + 4 * g);
            tv[4 * q + 0] = t4.x; tv[4 * q + 1] = t4.y; tv[4 * q + 2] = t4.z; tv[4 * q + 3] = t4.w;
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        // (B), in eight groups fenced by scheduling barriers: group i issues
        // logits product i of rb+1 and dW2 product i of rb-1 (independent
        // accumulators, so they alternate on the matrix core without a stall),
        // then numerators 2i and 2i+1 of rb, and every fourth group packs 8 of
        // them into the bf16 operand of rb's own dW2 products.
        float dz[16];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          zn = M::mma(hr[i >> 1][i & 1], wf[i >> 1][i & 1], zn);
          if constexpr (decltype(prev)::value)
            accw[i >> 1] = M::mma(atp[i >> 1][i & 1], dfp[i & 1], accw[i >> 1]);
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int r = 2 * i + j;
            dz[r] = __builtin_amdgcn_exp2f(fmaf(z[r], LOG2E, bb));
            if constexpr (TGT) {
              const int rl = 8 * (r >> 2) + 4 * g + (r & 3);
              dz[r] -= ((mw >> rl) & 1u) ? tv[r] : 0.0f;
            }
            db2p += dz[r];
          }
          if ((i & 3) == 3) df[i >> 2] = frag_acc<true>(dz, i >> 2);
          __builtin_amdgcn_sched_barrier(0);
        }
      };
      // row blocks: 0 alone, then pairs (odd rb in set b, even in set a), then
      // the last one alone when nrb is even; its products follow
      step(std::false_type{}, 0, za, zb, ata, dfa, atb, dfb);
      for (int rb = 1; rb + 1 < nrb; rb += 2) {
        step(std::true_type{}, rb, zb, za, atb, dfb, ata, dfa);
        step(std::true_type{}, rb + 1, za, zb, ata, dfa, atb, dfb);
      }
      if (nrb & 1) {
        dw2(ata, dfa);
      } else {
        step(std::true_type{}, nrb - 1, zb, za, atb, dfb, ata, dfa);
        dw2(atb, dfb);
      }
    };
    if (has_targets)
      rows(std::true_type{});
    else
      rows(std::false_type{});

    const float db2 = db2p + __shfl_xor(db2p, 32);
    // W2 -= lr dW2 in the staging tile (the lane's own operand-layout slots),
    // then out as whole rows
#pragma unroll
    for (int hb = 0; hb < 4; ++hb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float4& w = stage_frag(hb, q);
        float4 o;
        o.x = fmaf(-lr, accw[hb][4 * q + 0], w.x);
        o.y = fmaf(-lr, accw[hb][4 * q + 1], w.y);
        o.z = fmaf(-lr, accw[hb][4 * q + 2], w.z);
        o.w = fmaf(-lr, accw[hb][4 * q + 3], w.w);
        w = o;
      }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float4 o = *reinterpret_cast<const float4*>(stage + (2 * k + crow_l) * BWP_SLD + ccol);
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, o), w2r,
                                             voff + blk * 32 * HID * 4 + k * 2 * HID * 4, 0, 0);
    }
    // b2 from every lane, unconditionally (the lanes of half g = 1 and labels
    // past L fall outside the buffer and are dropped)
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, fmaf(-lr, db2, bias)), b2r,
                                          (g == 0 ? n * 4 : L * 4) + blk * 32 * 4, 0, 0);
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    if (blk + step < n_blocks) {
      stage_loaded();
      load_blk(bn2, plo, phi);
    }
  }
}

template <bool BF16, int MODE, int RS>
static hipError_t launch_bwd(int grid, size_t shm, hipStream_t st, hipEvent_t t0, hipEvent_t t1, float* W2,
                             float* b2, int L, const void* H1, const void* H1T, int ld_t, int B, const float* lse,
                             const float* rw, const int32_t* lbeg, const int32_t* lpair, float lr,
                             float invB) {
  using E = typename Mma<BF16>::elem;
  const float log2_invB = (float)log2((double)invB);
  static bool attr_done = false;
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute((const void*)k_out_bwd<BF16, MODE, RS>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_done = true;
  }
  hipExtLaunchKernelGGL((k_out_bwd<BF16, MODE, RS>), dim3(grid), dim3(BWD_THREADS), shm, st, t0, t1, 0, W2, b2,
                        L, (const E*)H1, (const E*)H1T, ld_t, B, lse, rw, lbeg, lpair, lr, invB, log2_invB);
  return hipGetLastError();
}

hipError_t launch_out_bwd(bool use_bf16, float* W2, float* b2, int L, const void* H1,
                          const void* H1T, int ld_t, int B, const float* lse, const float* rw,
                          const int32_t* lbeg, const int32_t* lpair, float lr, int n_cu,
                          hipStream_t st, hipEvent_t t0, hipEvent_t t1) {
  const int nrb = (B + 31) / 32;
  const int mode = !use_bf16 ? BWD_GLOBAL : (B <= BWD_CHUNK ? BWD_STAGED : BWD_CHUNKED);
  const int bpad = nrb * 32;
  const int mspan = mode == BWD_CHUNKED ? BWD_CROWS : bpad;  // rows of one target mask
  size_t shm = (size_t)2 * bpad * sizeof(float) + (size_t)BWD_WAVES * 32 * (mspan / 32) * sizeof(uint32_t);
  if (mode == BWD_CHUNKED) {
    // the chunk copies read whole chunks of H1 rows (ld_t rows allocated)
    if ((B + BWD_CROWS - 1) / BWD_CROWS * BWD_CROWS > ld_t) return hipErrorInvalidValue;
    shm += (size_t)2 * BWD_CROWS * TW_LD * 2;
  }
  const int n_blocks = (L + 31) / 32;
  int grid = (n_blocks + BWD_WAVES - 1) / BWD_WAVES;
  const int cap = mode == BWD_GLOBAL ? 2 * n_cu : n_cu;
  if (grid > cap) grid = cap;
  const float invB = 1.0f / (float)B;
  if (mode == BWD_STAGED) {
    static bool attr_done = false;
    if (!attr_done) {
      hipError_t e = hipFuncSetAttribute((const void*)k_out_bwd_prefetch,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
      if (e != hipSuccess) return e;
      attr_done = true;
    }
    const size_t shp = (size_t)BWD_CHUNK * TW_LD * 2 + (size_t)2 * nrb * 32 * sizeof(float) +
                       (size_t)BWP_WAVES * 32 * nrb * sizeof(uint32_t) +
                       (size_t)BWP_WAVES * 32 * BWP_SLD * sizeof(float);
    int gp = (n_blocks + BWP_WAVES - 1) / BWP_WAVES;
    if (gp > n_cu) gp = n_cu;
    hipExtLaunchKernelGGL(k_out_bwd_prefetch, dim3(gp), dim3(BWP_THREADS), shp, st, t0, t1, 0, W2, b2, L,
                          (const bf16*)H1, B, lse, rw, lbeg, lpair, lr, invB, (float)log2((double)invB));
    return hipGetLastError();
  }
  if (mode == BWD_CHUNKED)
    return launch_bwd<true, BWD_CHUNKED, 1>(grid, shm, st, t0, t1, W2, b2, L, H1, H1T, ld_t, B, lse, rw, lbeg,
                                            lpair, lr, invB);
  // fp32 operands with few label blocks: 4 wavefronts share a block's rows
  // (every wave would otherwise own a block and most of the GPU would idle)
  constexpr int RS = 4;
  if (n_blocks < n_cu * BWD_WAVES / RS && B <= 512) {
    const int units = (n_blocks + BWD_WAVES / RS - 1) / (BWD_WAVES / RS);
    const size_t shr = shm + (size_t)(BWD_WAVES / RS) * (RS - 1) * 65 * 64 * sizeof(float);
    return launch_bwd<false, BWD_GLOBAL, RS>(units < 2 * n_cu ? units : 2 * n_cu, shr, st, t0, t1, W2, b2, L,
                                             H1, H1T, ld_t, B, lse, rw, lbeg, lpair, lr, invB);
  }
  return launch_bwd<false, BWD_GLOBAL, 1>(grid, shm, st, t0, t1, W2, b2, L, H1, H1T, ld_t, B, lse, rw, lbeg,
                                          lpair, lr, invB);
}

}  // namespace asgd
