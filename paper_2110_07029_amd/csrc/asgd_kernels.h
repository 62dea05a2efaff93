// Host-side launchers of the gfx950 kernels.  Every launcher enqueues on
// `st` and returns the launch status; no launcher allocates memory.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace asgd {

constexpr int HID = 128;  // hidden width H

// Batch view as the kernels see it (device pointers; base = indptr[0] value
// is read on the device).
struct CsrDev {
  int n_rows, n_cols, nnz;
  const int32_t* indptr;
  const int32_t* indices;
  const float* values;
};

// ---- initialisation -------------------------------------------------------
hipError_t launch_init_uniform(float* w, int64_t count, uint64_t key, float bound, hipStream_t st);
hipError_t launch_fill_int(int32_t* p, int32_t v, int64_t n, hipStream_t st);

// ---- first layer forward + sort keys ---------------------------------------
// A1 = X W1 + b1 (fp32), H1 = ReLU(A1) as the output layer's operand type in
// row-major [rows_pad x 128] and, for fp32 operands only, transposed
// [128 x ld_t]; rows in [B, rows_pad) are zero.  Feature entry p (0 <= p < x.nnz): keys[p] = feature id (F if
// invalid), row_of[p] = its row.  With y != NULL, label entry q: lkeys[q] =
// label id (L if invalid), lrow[q] = its row, and rw[i] = 1/|Y_i|.
// Batches whose rows average GATHER_LONG_ROW entries or more split every row
// over GATHER_SPLIT workgroups; gpart: workspace of GATHER_SPLIT x ld_t x HID
// floats for their partial sums (ld_t >= rows_pad).
constexpr int GATHER_SPLIT = 4;
constexpr int GATHER_LONG_ROW = 160;
hipError_t launch_gather_fwd(bool use_bf16, const CsrDev& x, const CsrDev* y, const float* W1,
                             const float* b1, int F, int L, float* A1, void* H1, void* H1T,
                             int rows_pad, int ld_t, int32_t* keys, int32_t* row_of,
                             int32_t* lkeys, int32_t* lrow, float* rw, int32_t* err, int validate,
                             float* gpart, hipStream_t st, hipEvent_t done = nullptr);
// (done: completed by the launcher's last kernel when it has finished, with no
// marker of its own on the stream)

// ---- stable LSD radix sort of (key, position) -----------------------------
constexpr int SORT_CHUNK = 1024;   // keys per workgroup
constexpr int SORT_MAX_BITS = 11;  // digit width limit per pass
int sort_blocks(int n);
// Sorts keys[0..n) (values < 2^key_bits) stably; the payload is the original
// position.  Result in keys_out / vals_out.  tmp buffers of n entries, hist
// and offs of sort_blocks(n) << SORT_MAX_BITS entries.
hipError_t launch_sort(const int32_t* keys_in, int n, int key_bits, int32_t* keys_a,
                       int32_t* vals_a, int32_t* keys_b, int32_t* vals_b, int32_t* hist,
                       const int32_t** keys_out, const int32_t** vals_out, hipStream_t st);

// ---- (label, row) pairs grouped by 32-label block ---------------------------
// For the m label entries: lbeg[b] .. lbeg[b+1] (b < ceil(L/32)) is the range
// of block b's pairs in lpair, each (row << 5) | (label % 32); invalid labels
// (key L) are dropped.  lcnt: ceil(L/32) ints of scratch, used only when the
// counters do not fit in LDS.  Runs as one workgroup of the output-layer
// forward launch.
struct LabelJob {
  const int32_t* lkeys;
  int m;
  const int32_t* lrow;
  int32_t *lbeg, *lpair, *lcnt;
  int in_lds;  // filled in from the plan by the launcher
};
struct LabelJobPlan {
  int ok, lds_bytes, in_lds;
};
LabelJobPlan label_job_plan(bool use_bf16, int L);
// The same for the label-grouping workgroup of another launch of `nthreads` threads.
LabelJobPlan label_job_plan_for(const void* fn, int nthreads, int L);

// ---- output layer -----------------------------------------------------------
constexpr int OUT_TILE = 32;  // labels per forward tile
int out_rows_per_block(bool use_bf16);
// Forward over label splits: per (split, row) running max, sum of exponentials
// and sum_l exp(Z - m) W2[l] (flash-style); one workgroup per (split, row
// block), plus, with job != NULL, one that groups the labels (plan from
// label_job_plan).
hipError_t launch_out_fwd_train(bool use_bf16, const float* W2, const float* b2, int L, const void* H1,
                                int B, int splits, float* m_part, float* s_part, float* o_part,
                                int ld_part, const LabelJob* job, const LabelJobPlan* plan, hipStream_t st,
                                hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
// (t0, t1: optional events that the launch itself completes at the kernel's
// start and end, for timing the kernel alone)
// Per row, after the forward: lse, and with y the loss and tw = mean_{y in Y_i} W2[y]
// [B x 128] (reads W2 before the backward updates it).
// With y and dA1 (non-null), the same launch also forms dA1 = ((O/s - tw) / B) * [A1 > 0]
// from the partials (o_part, A1 as for launch_out_dA1); dA1 null: lse and targets only.
hipError_t launch_out_lse_targets(bool use_bf16, int B, int splits, const float* m_part, const float* s_part,
                                  int ld_part, const float* W2, const float* b2, int L, const void* H1,
                                  const CsrDev* y, float* lse, float* loss_rows, float* tw, const float* o_part,
                                  const float* A1, float* dA1, hipStream_t st, hipEvent_t done = nullptr);
// (done: an event that the launch itself completes when the kernel has
// finished, with no marker of its own on the stream)
// Per row: dA1 = ((O/s - tw) / B) * [A1 > 0] from the forward's partials (reads no W2);
// wide: twice the threads per row (for a launch that runs alone, not beside the backward).
hipError_t launch_out_dA1(int B, int splits, const float* m_part, const float* s_part, const float* o_part,
                          int ld_part, const float* tw, const float* A1, float* dA1, bool wide, hipStream_t st);
// Recompute Z per label tile, dZ = (softmax - T)/B, dW2 = dZ^T H1, db2; update W2, b2 in place.
hipError_t launch_out_bwd(bool use_bf16, float* W2, float* b2, int L, const void* H1,
                          const void* H1T, int ld_t, int B, const float* lse, const float* rw,
                          const int32_t* lbeg, const int32_t* lpair, float lr, int n_cu,
                          hipStream_t st, hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
// (t0, t1 as for launch_out_fwd_train)
// W1[f] -= lr * sum_{entries of f} x * dA1[row], one segment per distinct f
// (keys sorted by feature, invalid ids >= F last); and, in the same launch,
// db1 = sum_i dA1[i]; b1 -= lr db1; loss = mean_i loss_rows[i].
// part: 2 * sparse_windows(n_keys) * HID floats of scratch.
int sparse_windows(int n_keys);
hipError_t launch_sparse_update(float* W1, int F, const int32_t* skeys, const int32_t* svals, int n_keys,
                                const int32_t* row_of, const CsrDev& x, const float* dA1, float lr, int B,
                                float* b1, const float* loss_rows, float* loss, float* part, hipStream_t st,
                                hipEvent_t done = nullptr);  // done: as for launch_gather_fwd
// Distinct sorted feature ids (compaction of segment heads); count to *count_dev.
hipError_t launch_touched(const int32_t* skeys, int n_keys, int F, int32_t* ids, int32_t* count_dev,
                          hipStream_t st);

// ---- the optional second dense hidden layer (k_dense.hip) -------------------------
// A2 = ReLU(A1) Wh^T + bh (fp32, [rows_pad x 128]) and H2 = ReLU(A2) in the operand
// type into Hop (row-major) and, for fp32 operands, HopT ([128 x ld_t]); rows in
// [B, rows_pad) are zero.  Wh [128 x 128] row-major (output, input).
hipError_t launch_dense_fwd(bool use_bf16, const float* A1, const float* Wh, const float* bh, int B,
                            int rows_pad, float* A2, void* Hop, void* HopT, int ld_t, hipStream_t st);
// dA1 = (dA2 Wh) * [A1 > 0] with the pre-update Wh, then Wh -= lr dA2^T ReLU(A1)
// and bh -= lr 1^T dA2 (two launches in that order).
hipError_t launch_dense_bwd(const float* dA2, const float* A1, float* Wh, float* bh, int B, int rows_pad,
                            float lr, float* dA1, hipStream_t st);

// ---- output layer with stored logits (k_unfused.hip) ----------------------------
// Z = H W2^T + b2 into Z [B x ldz] fp32.  exact = 0: ldz >= ceil(L/32)*32 and the
// columns past L hold -inf; exact = 1: ldz >= L and only labels < L are written.
// With job != NULL, one more workgroup of the launch groups the labels (plan from
// logits_label_plan).
LabelJobPlan logits_label_plan(bool use_bf16, int L);
hipError_t launch_out_logits(bool use_bf16, const float* W2, const float* b2, int L, const void* H1, int B,
                             float* Z, int ldz, int exact, int n_cu, const LabelJob* job,
                             const LabelJobPlan* plan, hipStream_t st);
// lse and, with y, loss rows from the stored Z (one pass over it); m_part / s_part
// hold softmax_splits(ldz) x ld_part floats each.
int softmax_splits(int ldz);
hipError_t launch_softmax_ce(const float* Z, int ldz, int B, float* m_part, float* s_part, int ld_part,
                             const CsrDev* y, float* lse, float* loss_rows, hipStream_t st);
// dA = ((P W2 - rw sum_{y in Y_i} W2[y]) / B) * [A > 0] with P = exp(Z - lse) from the stored Z;
// o_part: splits x ld_part x 128 floats.
int unfused_dh_splits(int n_cu, int aux_cus, int B, bool use_bf16, int n_tiles);
hipError_t launch_unfused_dh(bool use_bf16, const float* W2, const float* b2, int L, const float* Z, int ldz,
                             const float* lse, int B, int splits, float* o_part, int ld_part, const CsrDev& y,
                             const float* rw, const float* A, float* dA, hipStream_t st);

// ---- prediction ---------------------------------------------------------------
int topk_splits(int B, int n_tiles);
hipError_t launch_out_fwd_topk(bool use_bf16, const float* W2, const float* b2, int L, const void* H1,
                               int B, int splits, int k, float* part_s, int32_t* part_i,
                               int ld_part, hipStream_t st);
hipError_t launch_topk_combine(int B, int splits, int k, const float* part_s,
                               const int32_t* part_i, int ld_part, int32_t* ids, float* scores,
                               hipStream_t st);

// ---- merge ---------------------------------------------------------------------
constexpr int MERGE_MAX = 16;
// out[e] = sum_i a[i] rep_i[e] + gamma (g[e] - gp[e]) in float64, rounded once;
// out may alias gp.  bcast[i] (nullable array) receives out as well.
hipError_t launch_merge(float* out, const float* g, const float* gp, const float* const* reps,
                        const double* alpha, int n, double gamma, float* const* bcast, int nb,
                        int64_t count, hipStream_t st);
// Deterministic sum of squares (float64) of w[0..count) into *out (device).
hipError_t launch_sqnorm(const float* w, int64_t count, double* partial, double* out,
                         hipStream_t st);
constexpr int SQNORM_BLOCKS = 1024;
// Sums of squares (float64) of n vectors of `count` floats (a multiple of 4) in one
// launch plus a fixed-order reduction: partial n x SQNORM_BLOCKS doubles, out n doubles
// (device): the sums, or sqrt(sum) / l2_div when l2_div > 0.  1 <= n <= MERGE_MAX.
hipError_t launch_sqnorm_multi(const float* const* w, int n, int64_t count, double* partial, double* out,
                               double l2_div, hipStream_t st);

}  // namespace asgd
