// Model object, memory pool and the C ABI of include/asgd.h.
//
// A model owns one parameter allocation [W1 | b1 | (Wh | bh) | W2 | b2] (each
// section padded to 64 floats so the merge streams it as one float4 vector) and one
// workspace allocation carved into the buffers every call needs, sized once
// for the largest batch (the memory pool of Sec. 4 "Scalable Memory
// Management": nothing is allocated while training).
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/asgd.h"
#include "asgd_kernels.h"

using namespace asgd;

namespace {

thread_local std::string g_last_error;

asgd_status fail(asgd_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

asgd_status fail_hip(hipError_t e, const char* what) {
  return fail(ASGD_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(expr)                                   \
  do {                                                  \
    hipError_t e_ = (expr);                             \
    if (e_ != hipSuccess) return fail_hip(e_, #expr);   \
  } while (0)

constexpr int64_t kAlign = 64;  // floats
constexpr int kMaxBatch = 16384;      // rows of one prediction call
constexpr int kMaxTrainBatch = 2048;  // rows of one training step (and of the inspection calls)
// The output-layer forward runs one persistent workgroup per CU except
// kAuxCus, which stay free for the feature sort on the internal stream and
// the forward launch's own label-grouping workgroup.
constexpr int kAuxCus = 16;
// Events that only order work between streams of this device: a device-scope
// release when recorded (a system-scope one writes the caches back for the
// host, which costs several microseconds on the recording stream).
constexpr unsigned kSyncEventFlags = hipEventDisableTiming | hipEventReleaseToDevice;

int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

int bit_width(uint32_t v) {
  int b = 0;
  while (v) {
    ++b;
    v >>= 1;
  }
  return b;
}

}  // namespace

namespace asgd {
asgd_status set_error(asgd_status s, const char* msg) { return fail(s, msg); }
}  // namespace asgd

// Device memory of asgd_models_l2_per_param_noalloc: the per-workgroup partial
// sums of squares of up to MERGE_MAX models (128 KiB), one copy per device,
// held until the process ends.  Host code must not use this name as an address
// (it is a host-side stand-in): the device address comes from
// hipGetSymbolAddress, taken once per device by scratch_on_device().
static __device__ __align__(256) double scratch[MERGE_MAX * SQNORM_BLOCKS];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch_dev[kMaxDevices] = {};

// The device address of `scratch` on `device`, which must be the current device
// the first time (asgd_model_init runs this for its device).
asgd_status scratch_on_device(int device, double** out) {
  if (device < 0 || device >= kMaxDevices) return fail(ASGD_ERANGE, "device ordinal beyond 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return fail_hip(e, "hipGetSymbolAddress(scratch)");
    g_scratch_dev[device] = static_cast<double*>(p);
  }
  *out = g_scratch_dev[device];
  return ASGD_OK;
}
}  // namespace

struct asgd_model {
  asgd_config cfg;
  int F = 0, L = 0;
  bool bf16 = true;
  bool extra = false;    // second dense hidden layer (Wh, bh)
  bool unfused = false;  // logits stored, softmax / cross-entropy as a pass of its own
  hipStream_t stream = nullptr;
  int device = 0;
  int n_cu = 256;
  // internal stream: the label grouping and the feature sort overlap the output layer
  hipStream_t aux = nullptr;
  hipEvent_t ev_fork = nullptr, ev_dA1 = nullptr, ev_join = nullptr;
  LabelJobPlan label_plan{};  // LDS of the forward launch's label-grouping workgroup
  LabelJobPlan label_plan_unf{};  // the same in the stored-logits path's logits launch
  hipEvent_t ev = nullptr;

  // parameters
  float* params = nullptr;
  int64_t off_b1 = 0, off_Wh = 0, off_bh = 0, off_W2 = 0, off_b2 = 0, n_pad = 0, n_params = 0;
  float* W1() const { return params; }
  float* b1() const { return params + off_b1; }
  float* Wh() const { return params + off_Wh; }
  float* bh() const { return params + off_bh; }
  float* W2() const { return params + off_W2; }
  float* b2() const { return params + off_b2; }

  // workspace
  void* ws = nullptr;
  int rows_pad_max = 0;  // rows of the output-layer operands
  int elem = 2;          // bytes per operand element
  float* A1 = nullptr;
  float* gpart = nullptr;  // partial first-layer sums of rows split over several workgroups
  float* A2 = nullptr;   // second hidden layer: pre-activation and its gradient
  float* dA2 = nullptr;
  void* H1 = nullptr;    // the output layer's input in its operand type (H1, or H2 with the extra layer)
  void* H1T = nullptr;
  // H1, H1T and rw are double-buffered: the gather of a step writes one copy
  // while the previous step's backward may still read the other.  H1, H1T and
  // rw above point at the copy of the current call.
  void* H1b[2] = {};
  void* H1Tb[2] = {};
  float* rwb[2] = {};
  int par = 0;
  // true while the last call on the model was a fused training step: its
  // internal stream may then start the next step's gather without waiting for
  // the model's stream (the previous backward only reads the other copies)
  bool pipe = false;
  // whether the gather runs on the internal stream (see asgd_train_step)
  bool gather_aux = false;
  float* tw = nullptr;   // per row: mean of W2[y] over the row's labels (pre-update)
  float* dA1 = nullptr;
  float* lse = nullptr;
  float* loss_rows = nullptr;
  float* rw = nullptr;
  float* loss = nullptr;
  int32_t* err = nullptr;
  int32_t* count = nullptr;
  double* sq_part = nullptr;
  double* sq_out = nullptr;
  double* sqm_part = nullptr;  // sums of squares of up to MERGE_MAX models (this model hosts them)
  double* sqm_out = nullptr;
  int32_t* keys = nullptr;
  int32_t *ka = nullptr, *va = nullptr, *kb = nullptr, *vb = nullptr;
  int32_t* hist = nullptr;
  int32_t* row_of = nullptr;
  float* w1_part = nullptr;  // partial W1 gradients of segments that cross a window
  int32_t* lrow = nullptr;
  int32_t* lkeys = nullptr;
  int32_t* lpair = nullptr;
  int32_t* lbeg = nullptr;
  int32_t* lcnt = nullptr;
  float* m_part = nullptr;
  float* s_part = nullptr;
  float* o_part = nullptr;
  int64_t part_rows = 0;  // capacity in (split, row) pairs
  float* Z = nullptr;     // stored logits [rows_pad_max x ldz] (unfused output only)
  int ldz = 0;
  float* sm_m = nullptr;  // softmax partials per (column chunk, row)
  float* sm_s = nullptr;
  float* tk_s = nullptr;
  int32_t* tk_i = nullptr;
  int64_t tk_rows = 0;

  // kernel timing: per group, a pool of (start, stop) event pairs
  static constexpr int kTimerPool = 1024;
  bool timing = false;
  std::vector<hipEvent_t> tev[ASGD_K_COUNT];
  int tused[ASGD_K_COUNT] = {};
};

namespace {

template <typename T>
T* carve(char*& p, int64_t count) {
  T* r = reinterpret_cast<T*>(p);
  p += round_up(count * (int64_t)sizeof(T), 256);
  return r;
}

// Every buffer of the workspace, laid out twice: once to size it, once to carve it.
int64_t layout_workspace(asgd_model* m, char* base) {
  const asgd_config& c = m->cfg;
  const int RB = out_rows_per_block(m->bf16);
  const int rp = m->rows_pad_max;
  const int64_t n_keys = c.max_nnz;  // the radix sort orders feature entries only
  const int nblk = sort_blocks((int)std::max<int64_t>(n_keys, 1));
  const int64_t n_lblocks = (m->L + 31) / 32;
  const int nrb = rp / RB;
  const int n_tiles = (m->L + OUT_TILE - 1) / OUT_TILE;
  // (split, row) pairs: splits <= min(n_tiles, ceil(n_cu / nRB)) for every nRB <= nrb
  int64_t part_rows = 0;
  for (int r = 1; r <= nrb; ++r) {
    int s = std::min(n_tiles, (m->n_cu + r - 1) / r);
    part_rows = std::max<int64_t>(part_rows, (int64_t)s * r * RB);
  }
  int64_t tk_rows = 0;
  for (int r = 1; r <= nrb; ++r) {
    const int B = r * RB;
    tk_rows = std::max<int64_t>(tk_rows, (int64_t)topk_splits(B, n_tiles) * r * RB);
  }
  char* p = base;
  m->A1 = carve<float>(p, (int64_t)rp * HID);
  m->A2 = carve<float>(p, m->extra ? (int64_t)rp * HID : 0);
  m->dA2 = carve<float>(p, m->extra ? (int64_t)rp * HID : 0);
  for (int b = 0; b < 2; ++b) {
    m->H1b[b] = carve<char>(p, (int64_t)rp * HID * m->elem);
    m->H1Tb[b] = carve<char>(p, (int64_t)rp * HID * m->elem);
    m->rwb[b] = carve<float>(p, rp);
  }
  m->H1 = m->H1b[0];
  m->H1T = m->H1Tb[0];
  m->rw = m->rwb[0];
  // (only a batch with max_nnz >= GATHER_LONG_ROW entries can average that many per row)
  m->gpart = c.max_nnz >= GATHER_LONG_ROW ? carve<float>(p, (int64_t)GATHER_SPLIT * rp * HID) : nullptr;
  m->tw = carve<float>(p, (int64_t)rp * HID);
  m->dA1 = carve<float>(p, (int64_t)rp * HID);
  m->lse = carve<float>(p, rp);
  m->loss_rows = carve<float>(p, rp);
  m->loss = carve<float>(p, 1);
  m->err = carve<int32_t>(p, 1);
  m->count = carve<int32_t>(p, 1);
  m->sq_part = carve<double>(p, SQNORM_BLOCKS);
  m->sq_out = carve<double>(p, 1);
  m->sqm_part = carve<double>(p, (int64_t)MERGE_MAX * SQNORM_BLOCKS);
  m->sqm_out = carve<double>(p, MERGE_MAX);
  m->keys = carve<int32_t>(p, n_keys + 1);
  m->ka = carve<int32_t>(p, n_keys + 1);
  m->va = carve<int32_t>(p, n_keys + 1);
  m->kb = carve<int32_t>(p, n_keys + 1);
  m->vb = carve<int32_t>(p, n_keys + 1);
  m->hist = carve<int32_t>(p, 2 * ((int64_t)nblk << SORT_MAX_BITS));
  m->row_of = carve<int32_t>(p, (int64_t)c.max_nnz + 1);
  m->w1_part = carve<float>(p, 2 * (int64_t)sparse_windows((int)std::max<int64_t>(n_keys, 1)) * HID);
  m->lrow = carve<int32_t>(p, (int64_t)c.max_label_nnz + 1);
  m->lkeys = carve<int32_t>(p, (int64_t)c.max_label_nnz + 1);
  m->lpair = carve<int32_t>(p, (int64_t)c.max_label_nnz + 1);
  m->lbeg = carve<int32_t>(p, n_lblocks + 1);
  m->lcnt = carve<int32_t>(p, n_lblocks + 1);
  m->m_part = carve<float>(p, part_rows);
  m->s_part = carve<float>(p, part_rows);
  m->o_part = carve<float>(p, part_rows * HID);
  m->part_rows = part_rows;
  m->ldz = n_tiles * OUT_TILE;
  const int64_t sm_rows = m->unfused ? (int64_t)softmax_splits(m->ldz) * rp : 0;
  m->Z = carve<float>(p, m->unfused ? (int64_t)rp * m->ldz : 0);
  m->sm_m = carve<float>(p, sm_rows);
  m->sm_s = carve<float>(p, sm_rows);
  m->tk_s = carve<float>(p, tk_rows * 32);
  m->tk_i = carve<int32_t>(p, tk_rows * 32);
  m->tk_rows = tk_rows;
  return (int64_t)(p - base);
}

asgd_status check_csr(const asgd_csr* a, const char* name, int n_cols, bool values, int max_nnz) {
  if (!a) return fail(ASGD_EINVAL, std::string(name) + " is NULL");
  if (a->n_cols != n_cols)
    return fail(ASGD_EINVAL, std::string(name) + ".n_cols does not match the model");
  if (a->n_rows < 1) return fail(ASGD_EINVAL, std::string(name) + ".n_rows must be >= 1");
  if (a->nnz < 0) return fail(ASGD_EINVAL, std::string(name) + ".nnz must be >= 0");
  if (a->nnz > max_nnz)
    return fail(ASGD_ERANGE, std::string(name) + ".nnz exceeds the model's provisioned maximum");
  if (!a->indptr) return fail(ASGD_EINVAL, std::string(name) + ".indptr is NULL");
  if (a->nnz > 0 && !a->indices) return fail(ASGD_EINVAL, std::string(name) + ".indices is NULL");
  if (values && a->nnz > 0 && !a->values)
    return fail(ASGD_EINVAL, std::string(name) + ".values is NULL");
  return ASGD_OK;
}

CsrDev dev(const asgd_csr* a) {
  return CsrDev{a->n_rows, a->n_cols, a->nnz, a->indptr, a->indices, a->values};
}

asgd_status check_batch(asgd_model* m, const asgd_csr* x, const asgd_csr* y, bool train = true) {
  asgd_status s = check_csr(x, "x", m->F, true, m->cfg.max_nnz);
  if (s) return s;
  if (x->n_rows > m->cfg.max_batch)
    return fail(ASGD_ERANGE, "batch larger than the model's max_batch");
  if (train && x->n_rows > kMaxTrainBatch)
    return fail(ASGD_ERANGE, "batches of more than 2048 rows are for prediction only");
  if (y) {
    s = check_csr(y, "y", m->L, false, m->cfg.max_label_nnz);
    if (s) return s;
    if (y->n_rows != x->n_rows) return fail(ASGD_EINVAL, "x and y have different row counts");
  }
  return ASGD_OK;
}

int fwd_splits(asgd_model* m, int B) {
  const int RB = out_rows_per_block(m->bf16);
  const int nrb = (B + RB - 1) / RB;
  const int n_tiles = (m->L + OUT_TILE - 1) / OUT_TILE;
  const int wgs = std::max(1, m->n_cu - kAuxCus);
  return std::max(1, std::min(n_tiles, (wgs + nrb - 1) / nrb));
}

// Start event of the next timed launch of group k (nullptr when not timing).
hipEvent_t timer_start(asgd_model* m, int k, hipStream_t st, hipEvent_t* stop) {
  *stop = nullptr;
  if (!m->timing || m->tused[k] >= asgd_model::kTimerPool) return nullptr;
  std::vector<hipEvent_t>& v = m->tev[k];
  const int i = m->tused[k]++;
  if ((int)v.size() < 2 * (i + 1)) {
    hipEvent_t a = nullptr, b = nullptr;
    if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) {
      --m->tused[k];
      return nullptr;
    }
    v.push_back(a);
    v.push_back(b);
  }
  if (hipEventRecord(v[2 * i], st) != hipSuccess) {
    --m->tused[k];
    return nullptr;
  }
  *stop = v[2 * i + 1];
  return v[2 * i];
}

#define TIMED_ON(m, k, st, expr)                               \
  do {                                                         \
    hipEvent_t stop_ = nullptr;                                \
    timer_start((m), (k), (st), &stop_);                       \
    HIP_TRY(expr);                                             \
    if (stop_) HIP_TRY(hipEventRecord(stop_, (st)));           \
  } while (0)
#define TIMED(m, k, expr) TIMED_ON(m, k, (m)->stream, expr)

// Start and stop events of the next timed launch of group k for a launcher
// that attaches them to its kernel's launch (completed at the kernel's own
// start and end, with no markers around it); nullptr when not timing.
void timer_pair(asgd_model* m, int k, hipEvent_t* t0, hipEvent_t* t1) {
  *t0 = *t1 = nullptr;
  if (!m->timing || m->tused[k] >= asgd_model::kTimerPool) return;
  std::vector<hipEvent_t>& v = m->tev[k];
  const int i = m->tused[k];
  if ((int)v.size() < 2 * (i + 1)) {
    hipEvent_t a = nullptr, b = nullptr;
    if (hipEventCreate(&a) != hipSuccess) return;
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return;
    }
    v.push_back(a);
    v.push_back(b);
  }
  ++m->tused[k];
  *t0 = v[2 * i];
  *t1 = v[2 * i + 1];
}
// expr names the events t0_ and t1_
#define TIMED_LAUNCH(m, k, expr)               \
  do {                                         \
    hipEvent_t t0_ = nullptr, t1_ = nullptr;   \
    timer_pair((m), (k), &t0_, &t1_);          \
    HIP_TRY(expr);                             \
  } while (0)

// Gather forward (+ keys) on stream st into the next copy of H1 / H1T / rw,
// optional validation check.  Leaves H1 / A1 ready.
// done (optional): an event completed once the gather's work has finished on st
asgd_status run_gather(asgd_model* m, const asgd_csr* x, const asgd_csr* y, hipStream_t st, int* rows_pad_out,
                       hipEvent_t done = nullptr) {
  const int B = x->n_rows;
  const int RB = out_rows_per_block(m->bf16);
  const int rows_pad = (int)round_up(B, RB);
  const bool validate = (m->cfg.flags & ASGD_VALIDATE) != 0;
  m->par ^= 1;
  m->H1 = m->H1b[m->par];
  m->H1T = m->H1Tb[m->par];
  m->rw = m->rwb[m->par];
  if (validate) HIP_TRY(launch_fill_int(m->err, 0, 1, st));
  CsrDev xd = dev(x);
  CsrDev yd = y ? dev(y) : CsrDev{};
  TIMED_ON(m, ASGD_K_GATHER, st, launch_gather_fwd(m->bf16, xd, y ? &yd : nullptr, m->W1(), m->b1(), m->F, m->L,
                                                   m->A1, m->H1, m->H1T, rows_pad, m->rows_pad_max, m->keys,
                                                   m->row_of, m->lkeys, m->lrow, m->rw, m->err, validate ? 1 : 0,
                                                   m->gpart, st, m->extra ? nullptr : done));
  if (m->extra) {
    TIMED_ON(m, ASGD_K_DENSE_FWD, st, launch_dense_fwd(m->bf16, m->A1, m->Wh(), m->bh(), B, rows_pad, m->A2,
                                                       m->H1, m->H1T, m->rows_pad_max, st));
    if (done) HIP_TRY(hipEventRecord(done, st));
  }
  if (validate) {
    int32_t e = 0;
    HIP_TRY(hipMemcpyAsync(&e, m->err, sizeof(e), hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    if (e) {
      char buf[160];
      snprintf(buf, sizeof buf,
               "malformed CSR input (flags 0x%x: 1 feature id, 2 label id, 4 indptr, 8 duplicate "
               "id, 16 empty label row)",
               e);
      return fail(ASGD_EINVAL, buf);
    }
  }
  *rows_pad_out = rows_pad;
  return ASGD_OK;
}

asgd_status run_sort(asgd_model* m, hipStream_t st, int n_keys, const int32_t** sk,
                     const int32_t** sv) {
  const int key_bits = bit_width((uint32_t)m->F);  // invalid ids carry key F
  TIMED_ON(m, ASGD_K_SORT, st,
           launch_sort(m->keys, n_keys, key_bits, m->ka, m->va, m->kb, m->vb, m->hist, sk, sv, st));
  return ASGD_OK;
}

// The fused output-layer forward and the per-row lse / target terms on the
// model's stream; with y, dA1 (dA2 with the second hidden layer) follows on
// da_stream, after an event when that is another stream (the training step
// runs it beside the backward).
asgd_status run_forward(asgd_model* m, const asgd_csr* x, const asgd_csr* y, int rows_pad,
                        const LabelJob* labels, hipStream_t da_stream, hipEvent_t fused_done = nullptr) {
  const int B = x->n_rows;
  const int splits = fwd_splits(m, B);
  const int n_tiles = (m->L + OUT_TILE - 1) / OUT_TILE;
  const int tps = (n_tiles + splits - 1) / splits;
  const int s_eff = (n_tiles + tps - 1) / tps;
  if ((int64_t)s_eff * rows_pad > m->part_rows) return fail(ASGD_ERANGE, "partial buffer too small");
  TIMED_LAUNCH(m, ASGD_K_OUT_FWD,
               launch_out_fwd_train(m->bf16, m->W2(), m->b2(), m->L, m->H1, B, splits, m->m_part, m->s_part,
                                    m->o_part, rows_pad, labels, &m->label_plan, m->stream, t0_, t1_));
  CsrDev yd = y ? dev(y) : CsrDev{};
  float* const A = m->extra ? m->A2 : m->A1;
  float* const dA = m->extra ? m->dA2 : m->dA1;
  // dA1 on the model's stream: in the same launch as lse and the target terms
  const bool fused = y && da_stream == m->stream;
  TIMED(m, ASGD_K_OUT_COMBINE, launch_out_lse_targets(m->bf16, B, s_eff, m->m_part, m->s_part, rows_pad, m->W2(),
                                                      m->b2(), m->L, m->H1, y ? &yd : nullptr, m->lse,
                                                      m->loss_rows, m->tw, m->o_part, A, fused ? dA : nullptr,
                                                      m->stream,
                                                      fused ? fused_done
                                                            : y && da_stream != m->stream ? m->ev_dA1 : nullptr));
  if (!y || fused) return ASGD_OK;
  // the event was completed by the lse/targets launch itself: a separate record
  // would put a marker between lse/targets and the backward on the model's
  // stream, and a gap of several microseconds with it
  if (da_stream != m->stream) HIP_TRY(hipStreamWaitEvent(da_stream, m->ev_dA1, 0));
  TIMED_ON(m, ASGD_K_HIDDEN, da_stream, launch_out_dA1(B, s_eff, m->m_part, m->s_part, m->o_part, rows_pad, m->tw,
                                                       A, dA, da_stream == m->stream, da_stream));
  return ASGD_OK;
}

// The output layer with stored logits: Z written by the logits kernel (whose
// launch also groups the labels for the backward), lse and the loss rows
// from one pass over Z, then dA (dA2 with the second hidden layer) from P W2
// with P read back from Z.
asgd_status run_forward_unfused(asgd_model* m, const asgd_csr* x, const asgd_csr* y, int rows_pad,
                                const LabelJob* labels) {
  const int B = x->n_rows;
  const int splits = fwd_splits(m, B);
  const int n_tiles = (m->L + OUT_TILE - 1) / OUT_TILE;
  const int tps = (n_tiles + splits - 1) / splits;
  const int s_eff = (n_tiles + tps - 1) / tps;
  if ((int64_t)s_eff * rows_pad > m->part_rows) return fail(ASGD_ERANGE, "partial buffer too small");
  TIMED(m, ASGD_K_LOGITS, launch_out_logits(m->bf16, m->W2(), m->b2(), m->L, m->H1, B, m->Z, m->ldz, 0,
                                            m->n_cu, labels, &m->label_plan_unf, m->stream));
  CsrDev yd = y ? dev(y) : CsrDev{};
  TIMED(m, ASGD_K_SOFTMAX, launch_softmax_ce(m->Z, m->ldz, B, m->sm_m, m->sm_s, rows_pad, y ? &yd : nullptr,
                                             m->lse, m->loss_rows, m->stream));
  if (y)
    TIMED(m, ASGD_K_DH, launch_unfused_dh(m->bf16, m->W2(), m->b2(), m->L, m->Z, m->ldz, m->lse, B, splits,
                                          m->o_part, rows_pad, yd, m->rw, m->extra ? m->A2 : m->A1,
                                          m->extra ? m->dA2 : m->dA1, m->stream));
  return ASGD_OK;
}

asgd_status sync_events_into(hipStream_t dst, asgd_model* src) {
  if (src->stream == dst) return ASGD_OK;
  HIP_TRY(hipEventRecord(src->ev, src->stream));
  HIP_TRY(hipStreamWaitEvent(dst, src->ev, 0));
  return ASGD_OK;
}

}  // namespace

extern "C" {

const char* asgd_last_error(void) { return g_last_error.c_str(); }

asgd_status asgd_model_init(asgd_model** out, const asgd_config* cfg, uint64_t seed,
                            void* hip_stream) {
  if (!out || !cfg) return fail(ASGD_EINVAL, "out and cfg must be non-NULL");
  *out = nullptr;
  if (cfg->hidden != HID) return fail(ASGD_EINVAL, "hidden must be 128");
  if (cfg->n_features < 1 || cfg->n_labels < 1)
    return fail(ASGD_EINVAL, "n_features and n_labels must be >= 1");
  if ((int64_t)cfg->n_features + cfg->n_labels >= (1 << 30))
    return fail(ASGD_ERANGE, "n_features + n_labels must be < 2^30");
  if (cfg->n_labels >= (1 << 22))  // W2 is read through 32-bit buffer offsets
    return fail(ASGD_ERANGE, "n_labels must be < 2^22");
  if (cfg->n_features >= (1 << 22))  // so are the rows of W1 in its sparse update
    return fail(ASGD_ERANGE, "n_features must be < 2^22");
  if (cfg->max_batch < 1 || cfg->max_batch > kMaxBatch)
    return fail(ASGD_ERANGE, "max_batch must be in [1, 16384]");
  if (cfg->max_nnz < 0 || cfg->max_label_nnz < 0)
    return fail(ASGD_EINVAL, "max_nnz and max_label_nnz must be >= 0");
  if ((int64_t)cfg->max_nnz + cfg->max_label_nnz >= (1LL << 30))
    return fail(ASGD_ERANGE, "max_nnz + max_label_nnz must be < 2^30");
  if (cfg->gemm_bf16 != 0 && cfg->gemm_bf16 != 1) return fail(ASGD_EINVAL, "gemm_bf16 must be 0 or 1");
  if (cfg->extra_hidden_layers != 0 && cfg->extra_hidden_layers != 1)
    return fail(ASGD_EINVAL, "extra_hidden_layers must be 0 or 1");
  if (cfg->flags & ~(ASGD_VALIDATE | ASGD_UNFUSED_OUTPUT)) return fail(ASGD_EINVAL, "unknown flag bits");

  asgd_model* m = new (std::nothrow) asgd_model();
  if (!m) return fail(ASGD_ENOMEM, "host allocation failed");
  m->cfg = *cfg;
  m->F = cfg->n_features;
  m->L = cfg->n_labels;
  m->bf16 = cfg->gemm_bf16 == 1;
  m->extra = cfg->extra_hidden_layers == 1;
  m->unfused = (cfg->flags & ASGD_UNFUSED_OUTPUT) != 0;
  // The gather moves to the internal stream, beside the previous step's
  // backward, when the output layer dominates the step: with many labels per
  // batch entry the internal stream (gather, sort, sparse update: work in
  // proportion to the batch's entries) then stays shorter than the model's
  // stream (work in proportion to L).  Measured: L / max_nnz of 33 (the
  // wide-label workload) gains 5 us per step; 4.9 (wide-feature) and 0.4
  // (tiny) lose 14 and 17 us, the internal stream becoming the longer one.
  m->gather_aux = !m->unfused && (int64_t)cfg->n_labels >= 8 * std::max<int64_t>(cfg->max_nnz, 1);
  m->elem = m->bf16 ? 2 : 4;
  m->stream = (hipStream_t)hip_stream;
  m->rows_pad_max = (int)round_up(cfg->max_batch, out_rows_per_block(m->bf16));
  const int64_t F = m->F, L = m->L;
  m->off_b1 = round_up(F * HID, kAlign);
  m->off_Wh = m->off_b1 + round_up(HID, kAlign);
  m->off_bh = m->off_Wh + (m->extra ? round_up(HID * HID, kAlign) : 0);
  m->off_W2 = m->off_bh + (m->extra ? round_up(HID, kAlign) : 0);
  m->off_b2 = m->off_W2 + round_up(L * HID, kAlign);
  m->n_pad = m->off_b2 + round_up(L, kAlign);
  m->n_params = F * HID + HID + (m->extra ? HID * HID + HID : 0) + L * HID + L;

  hipError_t e = hipGetDevice(&m->device);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&m->n_cu, hipDeviceAttributeMultiprocessorCount, m->device);
  if (e == hipSuccess) {
    double* sp = nullptr;
    const asgd_status ss = scratch_on_device(m->device, &sp);
    if (ss) {
      delete m;
      return ss;
    }
  }
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ev, kSyncEventFlags);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ev_fork, kSyncEventFlags);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ev_join, kSyncEventFlags);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->ev_dA1, kSyncEventFlags);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&m->aux, hipStreamNonBlocking);
  if (e == hipSuccess) {
    m->label_plan = label_job_plan(m->bf16, L);
    if (!m->label_plan.ok) e = hipErrorInvalidConfiguration;
    if (m->unfused) {
      m->label_plan_unf = logits_label_plan(m->bf16, L);
      if (!m->label_plan_unf.ok) e = hipErrorInvalidConfiguration;
    }
  }
  if (e == hipSuccess) e = hipMalloc((void**)&m->params, m->n_pad * sizeof(float));
  if (e != hipSuccess) {
    asgd_model_free(m);
    return fail(e == hipErrorOutOfMemory ? ASGD_ENOMEM : ASGD_EHIP,
                std::string("allocation failed: ") + hipGetErrorString(e));
  }
  const int64_t ws_bytes = layout_workspace(m, nullptr);
  e = hipMalloc(&m->ws, ws_bytes);
  if (e != hipSuccess) {
    asgd_model_free(m);
    return fail(e == hipErrorOutOfMemory ? ASGD_ENOMEM : ASGD_EHIP,
                std::string("workspace allocation failed: ") + hipGetErrorString(e));
  }
  layout_workspace(m, (char*)m->ws);

  const float a1 = (float)sqrt(6.0 / (double)(F + HID));
  const float a2 = (float)sqrt(6.0 / (double)(HID + L));
  e = hipMemsetAsync(m->params, 0, m->n_pad * sizeof(float), m->stream);
  if (e == hipSuccess) e = launch_init_uniform(m->W1(), F * HID, seed ^ (0ull << 56), a1, m->stream);
  if (e == hipSuccess) e = launch_init_uniform(m->W2(), L * HID, seed ^ (1ull << 56), a2, m->stream);
  if (e == hipSuccess && m->extra)
    e = launch_init_uniform(m->Wh(), HID * HID, seed ^ (2ull << 56), (float)sqrt(6.0 / (2.0 * HID)), m->stream);
  if (e == hipSuccess) e = hipMemsetAsync(m->ws, 0, ws_bytes, m->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
  if (e != hipSuccess) {
    asgd_model_free(m);
    return fail_hip(e, "initialisation");
  }
  *out = m;
  return ASGD_OK;
}

asgd_status asgd_model_free(asgd_model* m) {
  if (!m) return ASGD_OK;
  if (m->params || m->ws) (void)hipStreamSynchronize(m->stream);
  if (m->aux) (void)hipStreamSynchronize(m->aux);
  if (m->params) (void)hipFree(m->params);
  if (m->ws) (void)hipFree(m->ws);
  if (m->ev) (void)hipEventDestroy(m->ev);
  if (m->ev_fork) (void)hipEventDestroy(m->ev_fork);
  if (m->ev_join) (void)hipEventDestroy(m->ev_join);
  if (m->ev_dA1) (void)hipEventDestroy(m->ev_dA1);
  if (m->aux) (void)hipStreamDestroy(m->aux);
  for (auto& v : m->tev)
    for (hipEvent_t e : v) (void)hipEventDestroy(e);
  delete m;
  return ASGD_OK;
}

asgd_status asgd_model_set_stream(asgd_model* m, void* hip_stream) {
  if (!m) return fail(ASGD_EINVAL, "model is NULL");
  hipStream_t ns = (hipStream_t)hip_stream;
  m->pipe = false;
  if (ns != m->stream) {
    HIP_TRY(hipEventRecord(m->ev, m->stream));
    HIP_TRY(hipStreamWaitEvent(ns, m->ev, 0));
    m->stream = ns;
  }
  return ASGD_OK;
}

asgd_status asgd_model_copy(asgd_model* dst, const asgd_model* src) {
  if (!dst || !src) return fail(ASGD_EINVAL, "model is NULL");
  if (dst == src) return ASGD_OK;
  if (dst->F != src->F || dst->L != src->L || dst->n_pad != src->n_pad)
    return fail(ASGD_EINVAL, "models differ in shape");
  dst->pipe = false;
  asgd_status s = sync_events_into(dst->stream, const_cast<asgd_model*>(src));
  if (s) return s;
  HIP_TRY(hipMemcpyAsync(dst->params, src->params, dst->n_pad * sizeof(float),
                         hipMemcpyDeviceToDevice, dst->stream));
  // src must not be modified before the copy has read it
  HIP_TRY(hipEventRecord(dst->ev, dst->stream));
  if (src->stream != dst->stream) HIP_TRY(hipStreamWaitEvent(src->stream, dst->ev, 0));
  return ASGD_OK;
}

asgd_status asgd_model_num_params(const asgd_model* m, int64_t* out) {
  if (!m || !out) return fail(ASGD_EINVAL, "NULL argument");
  *out = m->n_params;
  return ASGD_OK;
}

static asgd_status param_span(const asgd_model* m, int32_t which, float** p, size_t* bytes) {
  const int64_t F = m->F, L = m->L;
  switch (which) {
    case ASGD_PARAM_W1: *p = m->W1(); *bytes = (size_t)(F * HID * 4); return ASGD_OK;
    case ASGD_PARAM_B1: *p = m->b1(); *bytes = (size_t)HID * 4; return ASGD_OK;
    case ASGD_PARAM_W2: *p = m->W2(); *bytes = (size_t)(L * HID * 4); return ASGD_OK;
    case ASGD_PARAM_B2: *p = m->b2(); *bytes = (size_t)(L * 4); return ASGD_OK;
    case ASGD_PARAM_WH:
    case ASGD_PARAM_BH:
      if (!m->extra) return fail(ASGD_EINVAL, "the model has no second hidden layer");
      *p = which == ASGD_PARAM_WH ? m->Wh() : m->bh();
      *bytes = (size_t)(which == ASGD_PARAM_WH ? HID * HID * 4 : HID * 4);
      return ASGD_OK;
    default: return fail(ASGD_EINVAL, "unknown parameter selector");
  }
}

asgd_status asgd_model_get_params(const asgd_model* m, int32_t which, void* host, size_t bytes) {
  if (!m || !host) return fail(ASGD_EINVAL, "NULL argument");
  float* p;
  size_t want;
  asgd_status s = param_span(m, which, &p, &want);
  if (s) return s;
  if (bytes != want) return fail(ASGD_EINVAL, "byte count does not match the tensor size");
  HIP_TRY(hipMemcpyAsync(host, p, bytes, hipMemcpyDeviceToHost, m->stream));
  HIP_TRY(hipStreamSynchronize(m->stream));
  return ASGD_OK;
}

asgd_status asgd_model_set_params(asgd_model* m, int32_t which, const void* host, size_t bytes) {
  if (!m || !host) return fail(ASGD_EINVAL, "NULL argument");
  float* p;
  size_t want;
  asgd_status s = param_span(m, which, &p, &want);
  if (s) return s;
  if (bytes != want) return fail(ASGD_EINVAL, "byte count does not match the tensor size");
  m->pipe = false;
  HIP_TRY(hipMemcpyAsync(p, host, bytes, hipMemcpyHostToDevice, m->stream));
  HIP_TRY(hipStreamSynchronize(m->stream));
  return ASGD_OK;
}

asgd_status asgd_train_step(asgd_model* m, const asgd_csr* x, const asgd_csr* y, float lr,
                            float* loss_out) {
  if (!m) return fail(ASGD_EINVAL, "model is NULL");
  if (!y) return fail(ASGD_EINVAL, "y is NULL");
  asgd_status s = check_batch(m, x, y);
  if (s) return s;
  if (!(lr == lr)) return fail(ASGD_EINVAL, "lr is NaN");
  const int B = x->n_rows;
  int rows_pad = 0;
  const int32_t *sk = nullptr, *sv = nullptr;
  const LabelJob labels{m->lkeys, y->nnz, m->lrow, m->lbeg, m->lpair, m->lcnt, 0};
  CsrDev xd = dev(x);
  m->pipe = m->pipe && m->gather_aux;
  if (m->gather_aux) {
    // Two streams.  Internal: gather (after the previous step's W1 update,
    // so it overlaps that step's output-layer backward), feature sort, then,
    // once the forward's partials and target terms exist, dA1, the second
    // hidden layer's backward, the sparse W1 update, b1 and the mean loss.
    // Model's stream: forward (whose launch also groups the labels), lse and
    // target terms, backward with the W2 update; the step ends when both have
    // finished.  Unless the previous call was a training step, the internal
    // stream first waits for the model's stream.
    if (!m->pipe) {
      HIP_TRY(hipEventRecord(m->ev_fork, m->stream));
      HIP_TRY(hipStreamWaitEvent(m->aux, m->ev_fork, 0));
    }
    m->pipe = false;
    s = run_gather(m, x, y, m->aux, &rows_pad, m->ev_fork);
    if (s) return s;
    HIP_TRY(hipStreamWaitEvent(m->stream, m->ev_fork, 0));
    s = run_sort(m, m->aux, x->nnz, &sk, &sv);
    if (s) return s;
    s = run_forward(m, x, y, rows_pad, &labels, m->aux);
    if (s) return s;
    if (m->extra)  // dA1 from dA2 through the second hidden layer, whose update follows
      TIMED_ON(m, ASGD_K_DENSE_BWD, m->aux, launch_dense_bwd(m->dA2, m->A1, m->Wh(), m->bh(), B, rows_pad, lr,
                                                             m->dA1, m->aux));
  } else {
    // The gather and the output layer's forward, and with it dA1, on the
    // model's stream; the feature sort on the internal stream beside them,
    // and the sparse update beside the backward.
    // (the events are completed by the launches themselves: a separate record
    // would put a marker, and a gap, into the model's stream)
    s = run_gather(m, x, y, m->stream, &rows_pad, m->ev_fork);
    if (s) return s;
    HIP_TRY(hipStreamWaitEvent(m->aux, m->ev_fork, 0));
    s = run_sort(m, m->aux, x->nnz, &sk, &sv);
    if (s) return s;
    // dA1's event: completed by the fused lse/targets + dA1 launch, or recorded
    // after the stored-logits path or the second layer's backward
    const bool dA1_by_launch = !m->unfused && !m->extra;
    s = m->unfused ? run_forward_unfused(m, x, y, rows_pad, &labels)
                   : run_forward(m, x, y, rows_pad, &labels, m->stream, dA1_by_launch ? m->ev_dA1 : nullptr);
    if (s) return s;
    if (m->extra)
      TIMED(m, ASGD_K_DENSE_BWD, launch_dense_bwd(m->dA2, m->A1, m->Wh(), m->bh(), B, rows_pad, lr, m->dA1,
                                                  m->stream));
    if (!dA1_by_launch) HIP_TRY(hipEventRecord(m->ev_dA1, m->stream));
    HIP_TRY(hipStreamWaitEvent(m->aux, m->ev_dA1, 0));
  }
  TIMED_ON(m, ASGD_K_W1_UPDATE, m->aux,
           launch_sparse_update(m->W1(), m->F, sk, sv, x->nnz, m->row_of, xd, m->dA1, lr, B, m->b1(),
                                m->loss_rows, m->loss, m->w1_part, m->aux, m->ev_join));
  TIMED_LAUNCH(m, ASGD_K_OUT_BWD,
               launch_out_bwd(m->bf16, m->W2(), m->b2(), m->L, m->H1, m->H1T, m->rows_pad_max, B, m->lse, m->rw,
                              m->lbeg, m->lpair, lr, m->n_cu, m->stream, t0_, t1_));
  HIP_TRY(hipStreamWaitEvent(m->stream, m->ev_join, 0));
  m->pipe = m->gather_aux;
  if (loss_out) return asgd_model_last_loss(m, loss_out);
  return ASGD_OK;
}

asgd_status asgd_model_last_loss(asgd_model* m, float* loss_out) {
  if (!m || !loss_out) return fail(ASGD_EINVAL, "NULL argument");
  float v = 0.0f;
  HIP_TRY(hipMemcpyAsync(&v, m->loss, sizeof(float), hipMemcpyDeviceToHost, m->stream));
  HIP_TRY(hipStreamSynchronize(m->stream));
  *loss_out = v;
  return ASGD_OK;
}

asgd_status asgd_predict_topk(asgd_model* m, const asgd_csr* x, int32_t k, int32_t* ids_dev,
                              float* scores_dev) {
  if (!m) return fail(ASGD_EINVAL, "model is NULL");
  asgd_status s = check_batch(m, x, nullptr, false);
  if (s) return s;
  if (k < 1 || k > 32 || k > m->L) return fail(ASGD_EINVAL, "k must be in [1, min(32, L)]");
  if (!ids_dev) return fail(ASGD_EINVAL, "ids_dev is NULL");
  const int B = x->n_rows;
  int rows_pad = 0;
  m->pipe = false;
  s = run_gather(m, x, nullptr, m->stream, &rows_pad);
  if (s) return s;
  const int n_tiles = (m->L + OUT_TILE - 1) / OUT_TILE;
  const int splits = topk_splits(B, n_tiles);
  const int tps = (n_tiles + splits - 1) / splits;
  const int s_eff = (n_tiles + tps - 1) / tps;
  if ((int64_t)s_eff * rows_pad > m->tk_rows) return fail(ASGD_ERANGE, "top-k buffer too small");
  HIP_TRY(launch_out_fwd_topk(m->bf16, m->W2(), m->b2(), m->L, m->H1, B, splits, k, m->tk_s,
                              m->tk_i, rows_pad, m->stream));
  HIP_TRY(launch_topk_combine(B, s_eff, k, m->tk_s, m->tk_i, rows_pad, ids_dev, scores_dev,
                              m->stream));
  return ASGD_OK;
}

asgd_status asgd_merge(asgd_model* global, asgd_model* prev_global, asgd_model* const* replicas,
                       const float* weights, int32_t n, float gamma, int32_t broadcast) {
  if (!global || !replicas || !weights) return fail(ASGD_EINVAL, "NULL argument");
  if (n < 1 || n > MERGE_MAX) return fail(ASGD_EINVAL, "n must be in [1, 16]");
  if (prev_global == global) return fail(ASGD_EINVAL, "prev_global must differ from global");
  if (prev_global && (prev_global->F != global->F || prev_global->L != global->L ||
                      prev_global->n_pad != global->n_pad))
    return fail(ASGD_EINVAL, "prev_global differs in shape");
  for (int i = 0; i < n; ++i) {
    asgd_model* r = replicas[i];
    if (!r) return fail(ASGD_EINVAL, "replica is NULL");
    if (r == global || r == prev_global) return fail(ASGD_EINVAL, "a replica aliases the global model");
    if (r->F != global->F || r->L != global->L || r->n_pad != global->n_pad)
      return fail(ASGD_EINVAL, "replica differs in shape");
    if (!(weights[i] == weights[i])) return fail(ASGD_EINVAL, "weight is NaN");
    for (int j = 0; j < i; ++j)
      if (replicas[j] == r && broadcast) return fail(ASGD_EINVAL, "duplicate replica with broadcast");
  }
  hipStream_t st = global->stream;
  // every participant's next training step must wait for the merge on its own stream
  global->pipe = false;
  if (prev_global) prev_global->pipe = false;
  for (int i = 0; i < n; ++i) {
    replicas[i]->pipe = false;
    asgd_status s = sync_events_into(st, replicas[i]);
    if (s) return s;
  }
  if (prev_global) {
    asgd_status s = sync_events_into(st, prev_global);
    if (s) return s;
  }
  const float* reps[MERGE_MAX];
  float* bc[MERGE_MAX];
  double alpha[MERGE_MAX];
  for (int i = 0; i < n; ++i) {
    reps[i] = replicas[i]->params;
    bc[i] = replicas[i]->params;
    alpha[i] = (double)weights[i];
  }
  float* out = prev_global ? prev_global->params : global->params;
  TIMED(global, ASGD_K_MERGE, launch_merge(out, global->params, prev_global ? prev_global->params : nullptr, reps, alpha,
                       n, (double)gamma, bc, broadcast ? n : 0, global->n_pad, st));
  if (prev_global) std::swap(global->params, prev_global->params);
  HIP_TRY(hipEventRecord(global->ev, st));
  for (int i = 0; i < n; ++i)
    if (replicas[i]->stream != st) HIP_TRY(hipStreamWaitEvent(replicas[i]->stream, global->ev, 0));
  if (prev_global && prev_global->stream != st)
    HIP_TRY(hipStreamWaitEvent(prev_global->stream, global->ev, 0));
  return ASGD_OK;
}

asgd_status asgd_model_l2_per_param(asgd_model* m, double* out) {
  if (!m || !out) return fail(ASGD_EINVAL, "NULL argument");
  HIP_TRY(launch_sqnorm(m->params, m->n_pad, m->sq_part, m->sq_out, m->stream));
  double s = 0.0;
  HIP_TRY(hipMemcpyAsync(&s, m->sq_out, sizeof(double), hipMemcpyDeviceToHost, m->stream));
  HIP_TRY(hipStreamSynchronize(m->stream));
  *out = sqrt(s) / (double)m->n_params;
  return ASGD_OK;
}

namespace {
// Models whose sums of squares are taken together: same parameter layout; the
// first one's stream runs the kernels after every model's pending work.
asgd_status check_norm_models(asgd_model* const* models, int32_t n, const double* out) {
  if (!models || !out) return fail(ASGD_EINVAL, "NULL argument");
  if (n < 1 || n > MERGE_MAX) return fail(ASGD_ERANGE, "n must be in [1, 16]");
  for (int i = 0; i < n; ++i) {
    if (!models[i]) return fail(ASGD_EINVAL, "model is NULL");
    if (models[i]->n_pad != models[0]->n_pad) return fail(ASGD_EINVAL, "models differ in shape");
  }
  return ASGD_OK;
}

asgd_status norms_on(asgd_model* const* models, int32_t n, double* partial, double* sums_dev, double* out) {
  asgd_model* m0 = models[0];
  hipStream_t st = m0->stream;
  for (int i = 1; i < n; ++i) {
    asgd_status s = sync_events_into(st, models[i]);
    if (s) return s;
  }
  const float* w[MERGE_MAX];
  for (int i = 0; i < n; ++i) w[i] = models[i]->params;
  HIP_TRY(launch_sqnorm_multi(w, n, m0->n_pad, partial, sums_dev, 0.0, st));
  double sums[MERGE_MAX];
  HIP_TRY(hipMemcpyAsync(sums, sums_dev, (size_t)n * sizeof(double), hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  for (int i = 0; i < n; ++i) out[i] = sqrt(sums[i]) / (double)models[i]->n_params;
  return ASGD_OK;
}
}  // namespace

asgd_status asgd_models_l2_per_param(asgd_model* const* models, int32_t n, double* out) {
  asgd_status s = check_norm_models(models, n, out);
  if (s) return s;
  return norms_on(models, n, models[0]->sqm_part, models[0]->sqm_out, out);
}

asgd_status asgd_models_l2_per_param_noalloc(asgd_model* const* models, int32_t n, double* out_dev) {
  asgd_status s = check_norm_models(models, n, out_dev);
  if (s) return s;
  double* partial = nullptr;
  s = scratch_on_device(models[0]->device, &partial);  // resolved when the model was created
  if (s) return s;
  asgd_model* m0 = models[0];
  hipStream_t st = m0->stream;
  for (int i = 1; i < n; ++i) {
    s = sync_events_into(st, models[i]);
    if (s) return s;
  }
  const float* w[MERGE_MAX];
  for (int i = 0; i < n; ++i) w[i] = models[i]->params;
  // every partial the reduction reads is written first by the same enqueued work
  HIP_TRY(launch_sqnorm_multi(w, n, m0->n_pad, partial, out_dev, (double)m0->n_params, st));
  return ASGD_OK;
}

asgd_status asgd_model_set_timing(asgd_model* m, int32_t enable) {
  if (!m) return fail(ASGD_EINVAL, "model is NULL");
  m->timing = enable != 0;
  return ASGD_OK;
}

asgd_status asgd_model_get_timing(asgd_model* m, int32_t kernel, double* total_ms,
                                  int64_t* launches) {
  if (!m || !total_ms || !launches) return fail(ASGD_EINVAL, "NULL argument");
  if (kernel < 0 || kernel >= ASGD_K_COUNT) return fail(ASGD_EINVAL, "unknown kernel group");
  double tot = 0.0;
  const int n = m->tused[kernel];
  for (int i = 0; i < n; ++i) {
    hipEvent_t a = m->tev[kernel][2 * i], b = m->tev[kernel][2 * i + 1];
    HIP_TRY(hipEventSynchronize(b));
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, a, b));
    tot += ms;
  }
  m->tused[kernel] = 0;
  *total_ms = tot;
  *launches = n;
  return ASGD_OK;
}

asgd_status asgd_debug_forward(asgd_model* m, const asgd_csr* x, const asgd_csr* y, float* a1_dev,
                               float* z_dev, float* lse_dev, float* loss_rows_dev) {
  if (!m) return fail(ASGD_EINVAL, "model is NULL");
  asgd_status s = check_batch(m, x, y);
  if (s) return s;
  if (loss_rows_dev && !y) return fail(ASGD_EINVAL, "loss rows need y");
  const int B = x->n_rows;
  int rows_pad = 0;
  m->pipe = false;
  s = run_gather(m, x, y, m->stream, &rows_pad);
  if (s) return s;
  s = m->unfused ? run_forward_unfused(m, x, y, rows_pad, nullptr)
                 : run_forward(m, x, y, rows_pad, nullptr, m->stream);
  if (s) return s;
  if (z_dev) {
    if (m->unfused)  // the step's own stored logits, without their padding columns
      HIP_TRY(hipMemcpy2DAsync(z_dev, (size_t)m->L * 4, m->Z, (size_t)m->ldz * 4, (size_t)m->L * 4, B,
                               hipMemcpyDeviceToDevice, m->stream));
    else
      HIP_TRY(launch_out_logits(m->bf16, m->W2(), m->b2(), m->L, m->H1, B, z_dev, m->L, 1, m->n_cu, nullptr,
                                nullptr, m->stream));
  }
  if (a1_dev)
    HIP_TRY(hipMemcpyAsync(a1_dev, m->A1, (size_t)B * HID * 4, hipMemcpyDeviceToDevice, m->stream));
  if (lse_dev) HIP_TRY(hipMemcpyAsync(lse_dev, m->lse, (size_t)B * 4, hipMemcpyDeviceToDevice, m->stream));
  if (loss_rows_dev)
    HIP_TRY(hipMemcpyAsync(loss_rows_dev, m->loss_rows, (size_t)B * 4, hipMemcpyDeviceToDevice,
                           m->stream));
  return ASGD_OK;
}

asgd_status asgd_debug_touched_rows(asgd_model* m, const asgd_csr* x, int32_t* ids_dev,
                                    int32_t* count_host) {
  if (!m || !ids_dev || !count_host) return fail(ASGD_EINVAL, "NULL argument");
  asgd_status s = check_batch(m, x, nullptr);
  if (s) return s;
  int rows_pad = 0;
  m->pipe = false;
  s = run_gather(m, x, nullptr, m->stream, &rows_pad);
  if (s) return s;
  const int32_t *sk = nullptr, *sv = nullptr;
  s = run_sort(m, m->stream, x->nnz, &sk, &sv);
  if (s) return s;
  HIP_TRY(launch_touched(sk, x->nnz, m->F, ids_dev, m->count, m->stream));
  int32_t c = 0;
  HIP_TRY(hipMemcpyAsync(&c, m->count, sizeof(c), hipMemcpyDeviceToHost, m->stream));
  HIP_TRY(hipStreamSynchronize(m->stream));
  *count_host = c;
  return ASGD_OK;
}

}  // extern "C"
