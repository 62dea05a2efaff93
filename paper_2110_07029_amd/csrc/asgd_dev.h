// Device-side building blocks shared by the gfx950 kernels.
//
// Matrix-core conventions (CDNA4, wave64):
//   v_mfma_f32_32x32x16_bf16 : D[32x32] += A[32x16] * B[16x32], 8 bf16 per lane
//   v_mfma_f32_32x32x2_f32   : D[32x32] += A[32x2]  * B[2x32],  1 fp32 per lane
// Lane l = 32*g + i (g = l/32).  A lanes own row m = i, B lanes own column
// n = i; the accumulator register r of lane l holds D[8*(r/4) + 4*g + r%4][i].
// Any permutation of the K index is allowed as long as A and B agree.  All
// kernels here use the "accumulator-compatible" K order: inside every block
// of 32 K values, element j of chunk c of lane group g is
//     k = 8*(r/4) + 4*g + r%4 with r = c*KL + j      (KL = values per lane).
// With that order the fp32 accumulators of one product can be fed directly as
// the K-operand of the next product (no register shuffles), and a lane that
// loads the 32 weights it multiplies also owns exactly the gradient entries
// those weights receive.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "asgd_kernels.h"

namespace asgd {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <bool BF16>
struct Mma;

template <>
struct Mma<true> {
  static constexpr int KC = 16;  // K per instruction
  static constexpr int KL = 8;   // K values per lane
  using frag = bf16x8;
  using elem = bf16;
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mma<false> {
  static constexpr int KC = 2;
  static constexpr int KL = 1;
  using frag = float;
  using elem = float;
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// Offset inside a 32-wide K block of element j of chunk c for lane group g.
template <bool BF16>
__device__ __forceinline__ int kofs(int c, int g, int j) {
  const int r = c * Mma<BF16>::KL + j;
  return 8 * (r >> 2) + 4 * g + (r & 3);
}

// Fragment of chunk c (inside the 32-block starting at `p`) from a row whose
// K values are contiguous in memory (global or LDS).
__device__ __forceinline__ bf16x8 frag_row_bf16(const bf16* p, int c, int g) {
  const bf16x4 lo = *reinterpret_cast<const bf16x4*>(p + 16 * c + 4 * g);
  const bf16x4 hi = *reinterpret_cast<const bf16x4*>(p + 16 * c + 8 + 4 * g);
  bf16x8 f;
  f[0] = lo[0]; f[1] = lo[1]; f[2] = lo[2]; f[3] = lo[3];
  f[4] = hi[0]; f[5] = hi[1]; f[6] = hi[2]; f[7] = hi[3];
  return f;
}

__device__ __forceinline__ float frag_row_f32(const float* p, int c, int g) {
  return p[8 * (c >> 2) + 4 * g + (c & 3)];
}

// Fragment of chunk c built from accumulator registers (K = the accumulator's
// row index, 32 per block): values r = c*KL + j.
__device__ __forceinline__ bf16x8 frag_acc_bf16(const float* v, int c) {
  bf16x8 f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (bf16)v[8 * c + j];
  return f;
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

// Word 3 of a raw (unformatted, 32-bit) buffer resource on the gfx9 family; with
// stride 0 a load at or past num_records bytes returns zeros.
constexpr int BUF_RSRC_WORD3 = 0x00020000;

typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---- W2 tile in LDS, bf16 (output-layer forward and backward) ---------------
// [32 labels x 128 hidden], row stride 160 elements, 16-byte chunks XOR-permuted
// by bits 2-3 of the row:
//   (label, h) -> label * 160 + 8 * ((h / 8) ^ ((label / 4) % 4)) + h % 8.
// gfx950's LDS serves 16-byte reads 16 lanes at a time and transposed 8-byte
// reads 32 lanes at a time over 64 banks; this layout keeps both reads of the
// tile (and its 8-byte stores) free of bank conflicts, and the permutation
// touches only the two low chunk bits, so a fragment's address is one of two
// per-lane bases plus a compile-time offset.
constexpr int TW_LD = 160;

__device__ __forceinline__ int tw_off(int row, int col) {
  return row * TW_LD + 8 * ((col >> 3) ^ ((row >> 2) & 3)) + (col & 7);
}
// Row fragments of label row n for lane group g: hidden units 32kb + 16c + 8g
// .. + 7 are at tw_row_base(n, g, c) + 32kb.
__device__ __forceinline__ int tw_row_base(int n, int g, int c) {
  return n * TW_LD + 8 * ((2 * c + g) ^ ((n >> 2) & 3));
}
// Transposed reads: result lane (n, g) receives hidden unit 32hb + n at labels
// 16c + 8hi + 4g + 0..3 from tw_col_base(lane, hi) + 16c * TW_LD + 32hb.  Source
// lane (G, i, a) = (lane / 16, lane / 4 % 4, lane % 4) addresses label
// 8hi + 4(G / 2) + i, hidden units 16(G % 2) + 4a .. + 3 (relative).
__device__ __forceinline__ int tw_col_base(int lane, int hi) {
  const int G = lane >> 4, i = (lane >> 2) & 3, a = lane & 3;
  return (8 * hi + 4 * (G >> 1) + i) * TW_LD + 8 * ((2 * (G & 1) + (a >> 1)) ^ ((2 * hi + (G >> 1)) & 3)) +
         4 * (a & 1);
}

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// ds_read_b64_tr_b16: a 64-bit LDS read whose 4 x 16-bit results are
// transposed inside each group of 16 lanes.  Element i of result lane
// 16G + 4a + b is element b of the 8 bytes that lane 16G + 4i + a addressed.
__device__ __forceinline__ bf16x4 lds_read_tr16(const bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
}

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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

// e^x through the hardware base-2 exponential.
__device__ __forceinline__ float exp_fast(float x) { return __builtin_amdgcn_exp2f(x * LOG2E); }

// Device error flags (bitwise OR into the model's flag word).
enum : int {
  ERR_FEATURE_ID = 1,   // feature id outside [0, F)
  ERR_LABEL_ID = 2,     // label id outside [0, L)
  ERR_INDPTR = 4,       // row extent decreasing or outside [indptr[0], indptr[0] + nnz)
  ERR_DUPLICATE = 8,    // ids of a row not strictly increasing
  ERR_EMPTY_LABELS = 16 // a label row without labels
};

}  // namespace asgd
