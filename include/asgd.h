/*
 * asgd.h - C ABI of the MI355X (gfx950) hot path of Adaptive SGD
 * (Ma, Rusu, Wu, Sim: "Adaptive Elastic Training for Sparse Deep Learning on
 * Heterogeneous Multi-GPU Servers", arXiv 2110.07029).
 *
 * The library trains replicas of the paper's sparse extreme-multi-label MLP
 * (Sec. 5.1 "Datasets and Model": sparse input layer, one ReLU hidden layer,
 * softmax + cross-entropy output layer) with mini-batch SGD (Sec. 2.1), and
 * merges replicas with the normalized, momentum-corrected model merge of
 * Alg. 2 (Sec. 3.3).  Batch-size scaling (Alg. 1, Sec. 3.2) and the merge
 * weights run on the host.
 *
 * Model:  A1 = X W1 + b1 ; H1 = ReLU(A1) ; Z = H1 W2^T + b2
 *         loss = mean_i [ logsumexp_j Z_ij - (1/|Y_i|) sum_{y in Y_i} Z_iy ]
 *         (target distribution 1/|Y_i| on each true label; mean over the batch)
 *         With extra_hidden_layers = 1 (the other reading of the paper's
 *         "3-layer MLP"): A2 = H1 Wh^T + bh ; H2 = ReLU(A2) ; Z = H2 W2^T + b2.
 * Shapes: W1 [F x H] row-major, b1 [H], W2 [L x H] row-major (label-major),
 *         b2 [L], Wh [H x H] row-major (output unit, input unit), bh [H];
 *         H = 128.  Parameters are float32.
 *
 * Conventions shared by every entry point
 *  - Every call returns an asgd_status and never throws or aborts.  On a
 *    non-OK status asgd_last_error() gives a message (thread-local).
 *  - Argument and shape errors (EINVAL / ERANGE) are detected on the host
 *    before anything is enqueued; the model is then unchanged.
 *  - EHIP: a HIP runtime call failed; the model's device state is undefined
 *    and the model should be freed.
 *  - Device pointers (CSR arrays, outputs) are owned by the caller and are
 *    only borrowed for the call; they must stay valid until the model's
 *    stream has executed the enqueued work.
 *  - Work is enqueued on the model's HIP stream (hipStream_t passed as
 *    void*; NULL = the default stream).  Calls return before the GPU work
 *    finishes unless stated otherwise.
 *  - A model must not be used from two host threads at once.
 *  - Every kernel bounds-checks feature and label ids and never reads the
 *    caller's index/value arrays outside [indptr[0], indptr[0] + nnz).
 *    Ids out of range are skipped on the device and raise the model's
 *    device error flag; with ASGD_VALIDATE the call then returns EINVAL.
 */
#ifndef ASGD_H
#define ASGD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct asgd_model asgd_model; /* opaque, created and freed only by the library */

typedef enum asgd_status {
  ASGD_OK = 0,
  ASGD_EINVAL = -1, /* invalid argument or malformed CSR content */
  ASGD_ERANGE = -2, /* size beyond what the model was provisioned for */
  ASGD_ENOMEM = -3, /* device or host allocation failed */
  ASGD_EHIP = -4,   /* HIP runtime error */
  ASGD_ESTATE = -5  /* call not valid in the object's current state */
} asgd_status;

/* asgd_config.flags */
#define ASGD_VALIDATE 0x1u       /* check CSR content on the device and synchronize each step */
#define ASGD_UNFUSED_OUTPUT 0x2u /* materialize the logits Z [B x L] fp32 and run the softmax and
                                    cross-entropy as a standalone pass over them (the textbook
                                    layer-by-layer output layer); default: fused, Z never stored */

typedef struct asgd_config {
  int32_t n_features;    /* F in [1, 2^22) */
  int32_t n_labels;      /* L in [1, 2^22) */
  int32_t hidden;        /* H; must be 128 */
  int32_t extra_hidden_layers; /* 0, or 1 for a second dense ReLU layer H -> H (Wh, bh) */
  int32_t max_batch;     /* largest B any call will use, in [1, 16384] (memory pool sized for it,
                            Sec. 4); training steps take at most 2048 rows, prediction all 16384 */
  int32_t max_nnz;       /* largest sum of nnz over the rows of one batch (>= 0) */
  int32_t max_label_nnz; /* largest sum of |Y_i| over the rows of one batch (>= 0;
                            max_nnz + max_label_nnz < 2^30) */
  int32_t gemm_bf16;     /* 1: output-layer products on bf16 operands with fp32 accumulation
                            (fp32 master weights); 0: fp32 operands */
  uint32_t flags;        /* ASGD_VALIDATE | ASGD_UNFUSED_OUTPUT, or 0 */
} asgd_config;

/* A CSR row block living in device memory.  Row i spans entries
 * [indptr[i], indptr[i+1]) of indices/values (absolute offsets, so a batch
 * can be a zero-copy row slice of a larger device-resident dataset whose
 * indptr[0] is not 0).  nnz is the host's copy of indptr[n_rows] - indptr[0].
 * Feature rows must have distinct ids per row; label rows must be non-empty
 * with distinct ids.  values is NULL for label matrices. */
typedef struct asgd_csr {
  int32_t n_rows;         /* B */
  int32_t n_cols;         /* F for features, L for labels */
  int32_t nnz;            /* entries in the block */
  const int32_t* indptr;  /* device, [n_rows + 1] */
  const int32_t* indices; /* device */
  const float* values;    /* device, or NULL for labels */
} asgd_csr;

/* Parameter selectors for get/set. */
enum {
  ASGD_PARAM_W1 = 0,
  ASGD_PARAM_B1 = 1,
  ASGD_PARAM_W2 = 2,
  ASGD_PARAM_B2 = 3,
  ASGD_PARAM_WH = 4, /* models with extra_hidden_layers = 1 only (EINVAL otherwise) */
  ASGD_PARAM_BH = 5
};

/* Merge-weight modes (Alg. 2). */
enum {
  ASGD_WEIGHTS_ALG2 = 0,    /* by batch size if all u_i are equal, else by update count */
  ASGD_WEIGHTS_SAMPLES = 1, /* by samples processed (the alternative named in Sec. 3.3) */
  ASGD_WEIGHTS_UNIFORM = 2  /* 1/n: the plain average of elastic model averaging and of
                               gradient aggregation (Sec. 2.2), the paper's baselines */
};

/* ------------------------------------------------------------------------ */
/* Model lifetime                                                            */
/* ------------------------------------------------------------------------ */

/* Create a model and its workspace (Sec. 4 "Scalable Memory Management":
 * everything is allocated once, for the largest batch).  W1 and W2 are
 * Xavier-uniform with half-width a = fl32(sqrt(6/(fan_in+fan_out))), fans
 * (F,H), (H,L) and (H,H); element e of tensor t (0 = W1, 1 = W2, 2 = Wh, row-major) is
 * fl32(fl32(2u-1) * a) with u = (splitmix64(seed ^ (t << 56) ^ e) >> 40) * 2^-24,
 * splitmix64 being the published generator's output for that state.  Biases
 * start at 0.  Initialisation runs on `hip_stream`; the call returns once it
 * has completed.  *out receives the model; nothing is allocated on error.
 * Errors: EINVAL for a NULL argument, a count below 1 (0 for the nnz maxima),
 * hidden != 128, gemm_bf16 or extra_hidden_layers not 0 or 1 or unknown flag
 * bits; ERANGE for F or L
 * at or above 2^22 (F + L below 2^30), max_batch outside [1, 16384] or
 * max_nnz + max_label_nnz at or above 2^30; ENOMEM / EHIP when the device
 * allocation or the initialisation fails. */
asgd_status asgd_model_init(asgd_model** out, const asgd_config* cfg, uint64_t seed,
                            void* hip_stream);

/* Free the model (synchronizes its stream first).  NULL is accepted. */
asgd_status asgd_model_free(asgd_model* m);

/* Move the model to another HIP stream (subsequent work is enqueued there;
 * the new stream first waits for work already enqueued on the old one). */
asgd_status asgd_model_set_stream(asgd_model* m, void* hip_stream);

/* Copy all parameters of src into dst (same F, L, H).  Enqueued on dst's
 * stream after src's pending work. */
asgd_status asgd_model_copy(asgd_model* dst, const asgd_model* src);

/* Number of parameters P = F*H + H + L*H + L (+ H*H + H with the second hidden layer). */
asgd_status asgd_model_num_params(const asgd_model* m, int64_t* out);

/* Copy one parameter tensor to / from host memory (synchronous).  `bytes`
 * must equal the tensor's size in bytes (F*H*4, H*4, L*H*4, L*4, H*H*4 or H*4). */
asgd_status asgd_model_get_params(const asgd_model* m, int32_t which, void* host, size_t bytes);
asgd_status asgd_model_set_params(asgd_model* m, int32_t which, const void* host, size_t bytes);

/* ------------------------------------------------------------------------ */
/* The per-replica step (Sec. 2.1: forward, backward, update)                */
/* ------------------------------------------------------------------------ */

/* One SGD step on the batch (x, y), B = x->n_rows = y->n_rows, 1 <= B <= min(max_batch, 2048)
 * (ERANGE above):
 * gradients of the mean loss, then theta <- theta - lr * g for W2, b2, b1 and
 * for the rows of W1 whose feature occurs in the batch; other W1 rows are
 * not written.  If loss_out is non-NULL the call synchronizes the stream and
 * stores the batch's mean loss (computed before the update); with NULL the
 * call is fully asynchronous and the loss stays readable with
 * asgd_model_last_loss(). */
asgd_status asgd_train_step(asgd_model* m, const asgd_csr* x, const asgd_csr* y, float lr,
                            float* loss_out);

/* Mean loss of the most recent train step (synchronizes the stream). */
asgd_status asgd_model_last_loss(asgd_model* m, float* loss_out);

/* Top-k labels per row of x by logit Z (ties: smaller label id first), the
 * prediction used for the paper's top-1 accuracy (Sec. 5.1 "Methodology").
 * ids_dev: device int32 [B x k]; scores_dev: device float [B x k] or NULL.
 * 1 <= k <= 32 and k <= L; B up to max_batch (16384 at most).  Asynchronous. */
asgd_status asgd_predict_topk(asgd_model* m, const asgd_csr* x, int32_t k, int32_t* ids_dev,
                              float* scores_dev);

/* ------------------------------------------------------------------------ */
/* Normalized model merging (Alg. 2) and batch-size scaling (Alg. 1)         */
/* ------------------------------------------------------------------------ */

/* The merge step of Alg. 2:  w' = sum_i alpha_i w_i + gamma (w - w_prev);
 * then w_prev <- w and w <- w'.  `global` holds w, `prev_global` holds
 * w_prev (NULL = no momentum term and no history), `replicas[0..n-1]` the
 * w_i, `weights` (host, [n]) the alpha_i.  Sums are formed in float64 per
 * element and rounded once to float32.  All models must share F, L, H;
 * 1 <= n <= 16; replicas may include neither global nor prev_global.
 * broadcast != 0 also writes w' into every replica (replicas restart from the
 * merged model, Sec. 4).  Enqueued on global's stream after the pending work
 * of every participant; the replicas' and prev_global's streams then wait for
 * the merge.  With prev_global, the two models exchange parameter buffers. */
asgd_status asgd_merge(asgd_model* global, asgd_model* prev_global, asgd_model* const* replicas,
                       const float* weights, int32_t n, float gamma, int32_t broadcast);

/* L2 norm of all parameters of a model divided by the parameter count
 * (Alg. 2's regularization gate "||w_i||_2 / |w|").  Synchronous. */
asgd_status asgd_model_l2_per_param(asgd_model* m, double* out);

/* The same for n models at once (1 <= n <= 16, all of one shape): their
 * sums of squares in one launch on models[0]'s stream, after the pending work
 * of every model's stream, and one host synchronization; out: host [n],
 * out[i] = ||w_i||_2 / |w_i|.  ERANGE for n outside [1, 16], EINVAL for a NULL
 * argument or models of different shapes.  The elastic rounds call it for the
 * perturbation gate (Alg. 2) over all replicas. */
asgd_status asgd_models_l2_per_param(asgd_model* const* models, int32_t n, double* out);

/* asgd_models_l2_per_param for callers that cannot allocate memory or wait
 * on the host (code under HIP graph capture, tight serving loops): the same
 * norms, computed by the same kernels, written to out_dev (device, [n]
 * doubles) on models[0]'s stream, asynchronously; nothing is allocated and
 * the host does not wait.  The partial sums live in a fixed device array of
 * the library (16 x 1024 doubles, 128 KiB per device, held until the process
 * ends) instead of a model's workspace; it is shared by every call on that
 * device, so calls that overlap on one device (other streams, other threads)
 * race and must be ordered by the caller.  ERANGE for n outside [1, 16] (the
 * array's capacity); EINVAL for a NULL argument or models of different shapes. */
asgd_status asgd_models_l2_per_param_noalloc(asgd_model* const* models, int32_t n, double* out_dev);

/* Alg. 2 weight computation (host only).  u: updates per replica since the
 * last merge; b: batch sizes; samples: samples processed (used by
 * ASGD_WEIGHTS_SAMPLES, may be NULL otherwise); ASGD_WEIGHTS_UNIFORM gives
 * every replica 1/n.  l2_per_param: per-replica
 * ||w_i||_2/|w| or NULL to disable the perturbation; when every value is
 * < pert_thr and n > 1, alpha_r *= 1 + delta and alpha_s *= 1 - delta for the
 * replica r with the most updates (then largest batch, then lowest index)
 * and s with the fewest (then smallest batch, then highest index).
 * alpha_out: host [n], float32 rounding of the float64 weights. */
asgd_status asgd_merge_weights(int32_t n, const int32_t* u, const int32_t* b,
                               const int64_t* samples, int32_t mode, const double* l2_per_param,
                               double pert_thr, double delta, float* alpha_out);

/* Alg. 1 batch-size scaling (host only), in place on b and lr.  With
 * mu = sum(u)/n: if u_i > mu and b_i + beta (u_i - mu) <= b_max the batch grows,
 * if u_i < mu and b_i - beta (mu - u_i) >= b_min it shrinks, otherwise it is
 * left alone (no clamping).  The new size is the exact value rounded to the
 * nearest integer (halves away from zero); lr_i <- fl32(lr_i * b_new / b_old). */
asgd_status asgd_scale_batches(int32_t n, const int32_t* u, int32_t* b, float* lr, int32_t b_min,
                               int32_t b_max, double beta);

/* ------------------------------------------------------------------------ */
/* Elastic rounds: n replicas on their own HIP streams of one device          */
/* ------------------------------------------------------------------------ */

/* Adaptive SGD's mega-batch loop (Sec. 3.1-3.3) with replicas standing in for
 * GPUs.  One round: batches of consecutive dataset rows are dispatched one at
 * a time to whichever replica is free (dynamic scheduling, Sec. 3.1) until a
 * fixed sample budget (the mega-batch) is spent; a batch never wraps past the
 * dataset end (it is cut there and the cursor restarts at row 0) and the last
 * batch is cut to the remaining budget.  Then Alg. 2 weights the replicas,
 * the merge of Alg. 2 updates the global model (with momentum) and is
 * broadcast to every replica, and Alg. 1 rescales each replica's batch size
 * and learning rate from its update count. */
typedef struct asgd_elastic asgd_elastic; /* opaque */

/* Who takes the next batch of a round. */
enum {
  ASGD_DISPATCH_DYNAMIC = 0, /* the first free replica (Adaptive SGD, Sec. 3.1) */
  ASGD_DISPATCH_STATIC = 1   /* batch k of the round goes to replica k mod n, whatever its speed:
                                the fixed schedule of elastic model averaging and, with a
                                mega-batch of one batch per replica, of gradient aggregation
                                (Sec. 2.2); a round then waits for its slowest replica */
};

enum {
  ASGD_CLOCK_TIMED = 0,  /* a replica is free when its last step's HIP event completed */
  ASGD_CLOCK_VIRTUAL = 1 /* deterministic: replica i's clock advances by
                            slow[i] * (c0 + c1 * rows + c2 * nnz) per step; the
                            replica with the smallest clock (lowest index on
                            ties) takes the next batch */
};

typedef struct asgd_elastic_config {
  int32_t n_replicas;      /* 1..16 */
  int32_t b_min, b_max;    /* batch-size bounds of Alg. 1; every replica starts at b_max */
  double beta;             /* Alg. 1 scaling parameter */
  float lr;                /* learning rate at b_max (linear scaling below) */
  float gamma;             /* momentum of the merge (Alg. 2) */
  int32_t weight_mode;     /* ASGD_WEIGHTS_ALG2, _SAMPLES or _UNIFORM */
  int32_t perturb;         /* 1: Alg. 2 perturbation with the L2-per-parameter gate */
  double pert_thr, delta;  /* perturbation threshold and factor */
  int64_t megabatch;       /* samples per round */
  int32_t dispatch;        /* ASGD_DISPATCH_DYNAMIC or ASGD_DISPATCH_STATIC */
  int32_t clock;           /* ASGD_CLOCK_TIMED or ASGD_CLOCK_VIRTUAL */
  double c0, c1, c2;       /* virtual clock cost model */
  double slow[16];         /* virtual clock per-replica multipliers (0 -> 1) */
} asgd_elastic_config;

/* Per-round record (host memory, filled by asgd_elastic_round). */
typedef struct asgd_elastic_log {
  int32_t n_dispatch;      /* batches dispatched this round */
  int32_t max_dispatch;    /* capacity of the arrays below (set by the caller) */
  int32_t* replica;        /* [max_dispatch] replica of each batch, in dispatch order */
  int32_t* row0;           /* [max_dispatch] first dataset row */
  int32_t* row1;           /* [max_dispatch] one past the last row */
  int32_t u[16];           /* updates per replica this round */
  int64_t samples[16];     /* samples per replica this round */
  int32_t b_used[16];      /* batch sizes used this round */
  float lr_used[16];       /* learning rates used this round */
  float alpha[16];         /* merge weights */
  double l2_per_param[16]; /* replica L2 norm per parameter (perturb only) */
  int32_t b_next[16];      /* batch sizes after Alg. 1 */
  float lr_next[16];       /* learning rates after Alg. 1 */
  int32_t cursor;          /* dataset row the next round starts at */
} asgd_elastic_log;

/* Create n replicas and a global / previous-global model pair, all from the
 * same seed (identical initial models), sized by `model_cfg` (whose
 * max_batch must be >= b_max).  replica_streams: n HIP streams (the
 * replicas' work queues); global_stream: the merge's stream. */
asgd_status asgd_elastic_create(asgd_elastic** out, const asgd_elastic_config* cfg,
                                const asgd_config* model_cfg, uint64_t seed,
                                void* const* replica_streams, void* global_stream);
asgd_status asgd_elastic_free(asgd_elastic* e);

/* One round over the device-resident dataset (x_all, y_all: all rows, the
 * batches are zero-copy row slices; x_indptr_host / y_indptr_host: host
 * copies of the indptr arrays, used for batch nnz counts).  Fills *log (if
 * non-NULL).  Returns after the merge has been enqueued; the replicas'
 * streams wait for it. */
asgd_status asgd_elastic_round(asgd_elastic* e, const asgd_csr* x_all, const asgd_csr* y_all,
                               const int32_t* x_indptr_host, const int32_t* y_indptr_host,
                               asgd_elastic_log* log);

/* Borrow the global model (owned by e) or replica i. */
asgd_status asgd_elastic_model(asgd_elastic* e, int32_t which /* -1 global, else replica */,
                               asgd_model** out);

/* ------------------------------------------------------------------------ */
/* Inspection of intermediates (parity tests)                                */
/* ------------------------------------------------------------------------ */

/* Forward pass only (no update): a1_dev [B x H] the first layer's
 * pre-activation, z_dev [B x L] the logits Z (row-major; written by the
 * logits kernel of the stored-logits path, in either output mode), lse_dev [B]
 * log-sum-exp of the logits, loss_rows_dev [B] per-row loss (needs y; may be
 * NULL together with y).  Every output may be NULL.  Device outputs,
 * asynchronous. */
asgd_status asgd_debug_forward(asgd_model* m, const asgd_csr* x, const asgd_csr* y, float* a1_dev,
                               float* z_dev, float* lse_dev, float* loss_rows_dev);

/* Sorted distinct feature ids of the batch (the W1 rows a step writes), as
 * computed by the step's sort-by-feature pass.  ids_dev: device [>= nnz];
 * *count_host receives the count.  Synchronous. */
asgd_status asgd_debug_touched_rows(asgd_model* m, const asgd_csr* x, int32_t* ids_dev,
                                    int32_t* count_host);

/* ------------------------------------------------------------------------ */
/* Dataset files (host)                                                      */
/* ------------------------------------------------------------------------ */

/* Sparse multi-label datasets in the text format of the Extreme
 * Classification Repository, where the paper's datasets come from (Sec. 5.1,
 * Table 1, libSVM files): an optional header line "n_rows n_features
 * n_labels", then per row "l1,l2,... f1:v1 f2:v2 ..." (labels may be empty;
 * blank lines and lines starting with '#' are skipped).  Feature ids are
 * 0-based, or 1-based with one_based = 1 (as in plain libSVM files); they are
 * shifted to 0-based.  Without a header, n_features / n_labels are one past
 * the largest id seen. */
typedef struct asgd_libsvm_info {
  int64_t n_rows, nnz, label_nnz;
  int64_t n_features, n_labels;
  int64_t header_rows; /* the header's row count, or -1 without a header */
} asgd_libsvm_info;

/* First pass: sizes.  ASGD_EINVAL names the file and line of a syntax
 * error, or an id beyond the header's counts. */
asgd_status asgd_libsvm_scan(const char* path, int32_t one_based, asgd_libsvm_info* info);

/* Second pass into caller-owned host arrays sized from info: indptr and
 * label_indptr [n_rows + 1] (int64, from 0), indices / values [nnz],
 * label_indices [label_nnz]; every row sorted by id.  A repeated id in a row
 * is ASGD_EINVAL; a file that changed since the scan is ASGD_ESTATE. */
asgd_status asgd_libsvm_read(const char* path, int32_t one_based, const asgd_libsvm_info* info,
                             int64_t* indptr, int32_t* indices, float* values, int64_t* label_indptr,
                             int32_t* label_indices);

/* ------------------------------------------------------------------------ */
/* Kernel timing (HIP events on the model's stream)                          */
/* ------------------------------------------------------------------------ */

/* Kernel groups that can be timed. */
enum {
  ASGD_K_GATHER = 0,      /* first-layer gather + sort keys */
  ASGD_K_SORT = 1,        /* radix sort of the batch's feature ids (internal stream) */
  ASGD_K_OUT_FWD = 2,     /* output-layer forward over all labels */
  ASGD_K_OUT_COMBINE = 3, /* per-row merge of the label splits: lse, loss, target terms (and
                             dA1 too, in the same launch, when the step forms dA1 on the
                             model's stream: the wide-label-dominated pipelined step does not) */
  ASGD_K_HIDDEN = 4,      /* per-row dA1 from the forward's partials, when it runs on the
                             internal stream beside the backward */
  ASGD_K_OUT_BWD = 5,     /* output-layer backward + W2/b2 update */
  ASGD_K_W1_UPDATE = 6,   /* sparse W1 gradient + update, b1 update, mean loss (internal stream) */
  ASGD_K_MERGE = 7,       /* normalized merge (timed on the global model) */
  ASGD_K_LABELS = 8,      /* (label, row) pairs grouped by label block: a workgroup of the
                             OUT_FWD (or LOGITS) launch, so never recorded on its own */
  ASGD_K_DENSE_FWD = 9,   /* second hidden layer forward (extra_hidden_layers = 1) */
  ASGD_K_DENSE_BWD = 10,  /* second hidden layer: dA1, and the Wh / bh update */
  ASGD_K_LOGITS = 11,     /* unfused output: the logits Z written to memory */
  ASGD_K_SOFTMAX = 12,    /* unfused output: the softmax / cross-entropy pass over Z (lse, loss) */
  ASGD_K_DH = 13,         /* unfused output: dH = dZ W2 from the stored Z, and dA */
  ASGD_K_COUNT = 14
};

/* enable != 0: from now on, time each kernel group launched for this model
 * with a pair of HIP events (up to 1024 launches per group are recorded
 * between two reads; later launches of that group run untimed).  The output
 * layer's forward and backward (ASGD_K_OUT_FWD, ASGD_K_OUT_BWD) pass the pair
 * to their launch, which completes them at the kernel's own start and end;
 * the other groups record them on their stream before and after their
 * launches, so their durations also count the dispatch.  enable == 0 stops
 * recording. */
asgd_status asgd_model_set_timing(asgd_model* m, int32_t enable);

/* Sum of the event-measured durations (ms) and the number of timed launches
 * of `kernel` since the last read; resets that group's record.  Waits for the
 * recorded events. */
asgd_status asgd_model_get_timing(asgd_model* m, int32_t kernel, double* total_ms,
                                  int64_t* launches);

/* Message describing the last non-OK status returned on this thread. */
const char* asgd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ASGD_H */
