// W2 tiles of the output layer: the shapes, loads, LDS layouts and operand
// fragments shared by the output-layer kernels (the fused forward and the
// prediction in k_output.hip, the stored-logits path in k_unfused.hip).
#pragma once

#include "asgd_dev.h"
#include "asgd_kernels.h"

namespace asgd {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <bool BF16>
struct FwdShape {
  static constexpr int NB = 1;                // 32-row blocks per wave
  static constexpr int WAVES = 8;             // wavefronts per workgroup (2 per SIMD)
  static constexpr int RB = WAVES * 32 * NB;  // rows per workgroup
  // leading dims chosen so a row step is 2 (mod 4) dwords with an odd half: the
  // 8-byte fragment reads of 16 consecutive lanes then cover all 32 banks
  static constexpr int WR = 132;              // leading dim of the row-major tile (elements)
  static constexpr int WT = 36;               // leading dim of the transposed tile (elements)
};

// Cooperative load of one 32-label tile of W2 (fp32 in HBM) by 512 threads:
// thread t reads hidden chunk 4*(t%32) of labels 2a and 2a+1 (a = t/32), so
// every load instruction reads whole 512-byte label rows and each thread holds
// a label pair for the transposed LDS copy.
constexpr int FWD_THREADS = 512;

struct TileRegs {
  float4 v[2];
  float bias;
};

// W2 and b2 as raw buffer resources: a load past the end returns zeros (no
// clamping or masking), and the uniform tile offset rides in a scalar register
// while the per-thread offset is fixed for the whole kernel.
struct W2Src {
  __amdgpu_buffer_rsrc_t w, b;
  int voff_w;  // bytes: row 2a, hidden 4q
  int voff_b;  // bytes: label slot t % 32
};


__device__ __forceinline__ W2Src w2_src(const float* W2, const float* b2, int L) {
  W2Src s;
  s.w = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(W2), (short)0, L * HID * 4, BUF_RSRC_WORD3);
  s.b = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(b2), (short)0, L * 4, BUF_RSRC_WORD3);
  const int tid = threadIdx.x, a = tid >> 5, q = tid & 31;
  s.voff_w = (2 * a * HID + 4 * q) * 4;
  s.voff_b = (tid & (OUT_TILE - 1)) * 4;
  return s;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// max(v[l], v[l ^ 32]) on every lane, without a trip through LDS: the swap
// exchanges the upper half of one copy with the lower half of the other, so
// the two results hold, on each lane, the lane's value and its partner's.
__device__ __forceinline__ float half_swap_max(float v) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, sw[0]), __builtin_bit_cast(float, sw[1]));
}

__device__ __forceinline__ void tile_load(const W2Src& src, int tile, TileRegs& r) {
  const int base = (int)((unsigned)tile * (unsigned)(OUT_TILE * HID * 4));
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    // (reinterpret the whole vector: bit casts of single elements of the
    // builtin's result are folded into one narrowed load by this compiler)
    const f32x4 v = __builtin_bit_cast(
        f32x4, __builtin_amdgcn_raw_buffer_load_b128(src.w, src.voff_w + it * HID * 4, base, 0));
    r.v[it] = make_float4(v.x, v.y, v.z, v.w);
  }
  r.bias = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(src.b, src.voff_b,
                                                                          tile * OUT_TILE * 4, 0));
}

// Store a loaded tile into LDS as operands.  bf16: the layout above, which
// also serves the transposed operand.  fp32: row-major [label][hidden] (leading
// dim WR) and, if TRANSPOSED, [hidden][label] (leading dim WT).  Biases of
// labels past L become -inf (their weights loaded as zeros, so those labels
// get probability 0).
template <bool BF16>
constexpr int tile_elems() {
  return BF16 ? OUT_TILE * TW_LD : OUT_TILE * FwdShape<BF16>::WR;
}
template <bool BF16>
constexpr int tileT_elems() {
  return BF16 ? 1 : HID * FwdShape<BF16>::WT;
}

template <bool BF16, bool TRANSPOSED>
__device__ __forceinline__ void tile_store(const TileRegs& r, int L, int tile,
                                           typename Mma<BF16>::elem* wr,
                                           typename Mma<BF16>::elem* wt, float* bt) {
  constexpr int WR = FwdShape<BF16>::WR, WT = FwdShape<BF16>::WT;
  const int tid = threadIdx.x, a = tid >> 5, q = tid & 31;
  const float x[2][4] = {{r.v[0].x, r.v[0].y, r.v[0].z, r.v[0].w}, {r.v[1].x, r.v[1].y, r.v[1].z, r.v[1].w}};
  if constexpr (BF16) {
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      bf16x4 p;
      p[0] = (bf16)x[it][0]; p[1] = (bf16)x[it][1]; p[2] = (bf16)x[it][2]; p[3] = (bf16)x[it][3];
      *reinterpret_cast<bf16x4*>(wr + tw_off(2 * a + it, 4 * q)) = p;
    }
  } else {
#pragma unroll
    for (int it = 0; it < 2; ++it)
      *reinterpret_cast<float4*>(wr + (2 * a + it) * WR + 4 * q) =
          make_float4(x[it][0], x[it][1], x[it][2], x[it][3]);
    if constexpr (TRANSPOSED) {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        *reinterpret_cast<float2*>(wt + (4 * q + k) * WT + 2 * a) = make_float2(x[0][k], x[1][k]);
    }
  }
  // every thread writes its label slot's bias (threads sharing a slot write the
  // same value), so the store needs no branch
  const int sl = threadIdx.x & (OUT_TILE - 1);
  bt[sl] = tile * OUT_TILE + sl < L ? r.bias : -INFINITY;
}

// Operand fragments of the logits Z^T = W2_tile H1^T (K = hidden).  With bf16
// operands a lane's 8 values of chunk c of hidden block kb are the consecutive
// units 32 kb + 16 c + 8 g .. + 7 on both sides (one 16-byte read each); fp32
// uses the accumulator-compatible order of frag_row.
template <bool BF16>
__device__ __forceinline__ typename Mma<BF16>::frag h1_frag(const typename Mma<BF16>::elem* hrow, int kb, int c,
                                                            int g) {
  if constexpr (BF16)
    return *reinterpret_cast<const bf16x8*>(hrow + 32 * kb + 16 * c + 8 * g);
  else
    return frag_row<false>(hrow + 32 * kb, c, g);
}
// A fragments of a stored tile: W2 rows (M = labels, K = hidden block kb) and
// W2^T rows (M = hidden block hb, K = labels in the accumulator-compatible
// order, to meet the probabilities taken from the logits' accumulators).
// rb[c] = tw_row_base(n, g, c), cb[hi] = tw_col_base(lane, hi): the lane's bases.
template <bool BF16>
__device__ __forceinline__ typename Mma<BF16>::frag tile_frag_w(const typename Mma<BF16>::elem* wr,
                                                                const int (&rb)[2], int n, int kb, int c, int g) {
  if constexpr (BF16)
    return *reinterpret_cast<const bf16x8*>(wr + rb[c] + 32 * kb);
  else
    return frag_row<false>(wr + n * FwdShape<false>::WR + 32 * kb, c, g);
}
template <bool BF16>
__device__ __forceinline__ typename Mma<BF16>::frag tile_frag_wt(const typename Mma<BF16>::elem* wr,
                                                                 const typename Mma<BF16>::elem* wt,
                                                                 const int (&cb)[2], int hb, int c, int lane) {
  if constexpr (BF16) {
    const bf16* o = wr + 16 * c * TW_LD + 32 * hb;
    const bf16x4 lo = lds_read_tr16(o + cb[0]), hi = lds_read_tr16(o + cb[1]);
    bf16x8 f;
    f[0] = lo[0]; f[1] = lo[1]; f[2] = lo[2]; f[3] = lo[3];
    f[4] = hi[0]; f[5] = hi[1]; f[6] = hi[2]; f[7] = hi[3];
    return f;
  } else {
    return frag_row<false>(wt + (32 * hb + (lane & 31)) * FwdShape<false>::WT, c, lane >> 5);
  }
}

}  // namespace asgd
