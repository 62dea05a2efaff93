// Elastic rounds of Adaptive SGD on one device: n replicas on their own HIP
// streams stand in for the paper's GPUs; one host thread plays the dynamic
// scheduler (Sec. 4, "Architecture and Workflow").  Per round: dynamic
// dispatch of a fixed sample budget (Sec. 3.1), normalized merge weights and
// the momentum merge (Alg. 2, Sec. 3.3), batch-size scaling (Alg. 1,
// Sec. 3.2).  The same loop runs the paper's baselines (Sec. 2.2, Sec. 5):
// a static schedule with uniform weights, no momentum and fixed batches is
// elastic model averaging, and with one batch per replica per round it is
// gradient aggregation.  Built only on the public C ABI plus HIP events.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <new>
#include <vector>

#include "../../include/asgd.h"

namespace asgd {
asgd_status set_error(asgd_status s, const char* msg);
}

namespace {
asgd_status efail(asgd_status s, const char* msg) { return asgd::set_error(s, msg); }
}  // namespace

struct asgd_elastic {
  asgd_elastic_config cfg{};
  int n = 0;
  std::vector<asgd_model*> reps;
  asgd_model* global = nullptr;
  asgd_model* prev = nullptr;
  std::vector<hipStream_t> streams;
  std::vector<hipEvent_t> done;  // completion of each replica's latest step
  std::vector<int32_t> b;
  std::vector<float> lr;
  int64_t cursor = 0;
};

extern "C" {

asgd_status asgd_elastic_free(asgd_elastic* e) {
  if (!e) return ASGD_OK;
  for (asgd_model* m : e->reps) asgd_model_free(m);
  asgd_model_free(e->global);
  asgd_model_free(e->prev);
  for (hipEvent_t ev : e->done)
    if (ev) (void)hipEventDestroy(ev);
  delete e;
  return ASGD_OK;
}

asgd_status asgd_elastic_create(asgd_elastic** out, const asgd_elastic_config* cfg,
                                const asgd_config* model_cfg, uint64_t seed,
                                void* const* replica_streams, void* global_stream) {
  if (!out || !cfg || !model_cfg || !replica_streams) return efail(ASGD_EINVAL, "NULL argument");
  *out = nullptr;
  const int n = cfg->n_replicas;
  if (n < 1 || n > 16) return efail(ASGD_EINVAL, "n_replicas must be in [1, 16]");
  if (cfg->b_min < 1 || cfg->b_max < cfg->b_min) return efail(ASGD_EINVAL, "need 1 <= b_min <= b_max");
  if (cfg->b_max > model_cfg->max_batch) return efail(ASGD_ERANGE, "b_max exceeds the models' max_batch");
  if (cfg->b_max > 2048) return efail(ASGD_ERANGE, "b_max exceeds 2048, the largest training batch");
  if (cfg->megabatch < 1) return efail(ASGD_EINVAL, "megabatch must be >= 1");
  if (cfg->clock != ASGD_CLOCK_TIMED && cfg->clock != ASGD_CLOCK_VIRTUAL)
    return efail(ASGD_EINVAL, "unknown clock mode");
  if (cfg->weight_mode != ASGD_WEIGHTS_ALG2 && cfg->weight_mode != ASGD_WEIGHTS_SAMPLES &&
      cfg->weight_mode != ASGD_WEIGHTS_UNIFORM)
    return efail(ASGD_EINVAL, "unknown weight mode");
  if (cfg->dispatch != ASGD_DISPATCH_DYNAMIC && cfg->dispatch != ASGD_DISPATCH_STATIC)
    return efail(ASGD_EINVAL, "unknown dispatch mode");
  if (!(cfg->lr == cfg->lr) || !(cfg->beta == cfg->beta)) return efail(ASGD_EINVAL, "NaN parameter");

  asgd_elastic* e = new (std::nothrow) asgd_elastic();
  if (!e) return efail(ASGD_ENOMEM, "host allocation failed");
  e->cfg = *cfg;
  e->n = n;
  for (int i = 0; i < n; ++i) {
    if (cfg->slow[i] <= 0.0) e->cfg.slow[i] = 1.0;
    asgd_model* m = nullptr;
    asgd_status s = asgd_model_init(&m, model_cfg, seed, replica_streams[i]);
    if (s) {
      asgd_elastic_free(e);
      return s;
    }
    e->reps.push_back(m);
    e->streams.push_back((hipStream_t)replica_streams[i]);
    hipEvent_t ev = nullptr;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
      asgd_elastic_free(e);
      return efail(ASGD_EHIP, "event creation failed");
    }
    e->done.push_back(ev);
    e->b.push_back(cfg->b_max);
    e->lr.push_back(cfg->lr);
  }
  asgd_status s = asgd_model_init(&e->global, model_cfg, seed, global_stream);
  if (!s) s = asgd_model_init(&e->prev, model_cfg, seed, global_stream);
  if (s) {
    asgd_elastic_free(e);
    return s;
  }
  *out = e;
  return ASGD_OK;
}

asgd_status asgd_elastic_model(asgd_elastic* e, int32_t which, asgd_model** out) {
  if (!e || !out) return efail(ASGD_EINVAL, "NULL argument");
  if (which == -1) {
    *out = e->global;
    return ASGD_OK;
  }
  if (which < 0 || which >= e->n) return efail(ASGD_EINVAL, "replica index out of range");
  *out = e->reps[which];
  return ASGD_OK;
}

asgd_status asgd_elastic_round(asgd_elastic* e, const asgd_csr* x_all, const asgd_csr* y_all,
                               const int32_t* xh, const int32_t* yh, asgd_elastic_log* log) {
  if (!e || !x_all || !y_all || !xh || !yh) return efail(ASGD_EINVAL, "NULL argument");
  if (x_all->n_rows != y_all->n_rows || x_all->n_rows < 1)
    return efail(ASGD_EINVAL, "x_all and y_all must have the same, non-zero row count");
  const int n = e->n;
  const int64_t n_rows = x_all->n_rows;
  const asgd_elastic_config& c = e->cfg;
  int32_t u[16] = {};
  int64_t samples[16] = {};
  double clock[16] = {};
  int64_t left = c.megabatch;
  int32_t nd = 0;
  if (log) {
    log->n_dispatch = 0;
    for (int i = 0; i < n; ++i) {
      log->b_used[i] = e->b[i];
      log->lr_used[i] = e->lr[i];
    }
  }
  while (left > 0) {
    int w = 0;
    if (c.dispatch == ASGD_DISPATCH_STATIC) {
      w = nd % n;  // fixed schedule: enqueue on the replica's stream whether or not it is busy
    } else if (c.clock == ASGD_CLOCK_VIRTUAL) {
      for (int i = 1; i < n; ++i)
        if (clock[i] < clock[w]) w = i;
    } else {
      // dynamic scheduling: the first replica whose latest step has finished
      for (;;) {
        int free_w = -1;
        for (int i = 0; i < n && free_w < 0; ++i) {
          const hipError_t q = hipEventQuery(e->done[i]);
          if (q == hipSuccess) free_w = i;
          else if (q != hipErrorNotReady) return efail(ASGD_EHIP, hipGetErrorString(q));
        }
        if (free_w >= 0) {
          w = free_w;
          break;
        }
      }
    }
    const int64_t take = std::min<int64_t>(std::min<int64_t>(e->b[w], left), n_rows - e->cursor);
    const int32_t r0 = (int32_t)e->cursor, r1 = (int32_t)(e->cursor + take);
    asgd_csr xb{r1 - r0, x_all->n_cols, xh[r1] - xh[r0], x_all->indptr + r0, x_all->indices,
                x_all->values};
    asgd_csr yb{r1 - r0, y_all->n_cols, yh[r1] - yh[r0], y_all->indptr + r0, y_all->indices,
                nullptr};
    asgd_status s = asgd_train_step(e->reps[w], &xb, &yb, e->lr[w], nullptr);
    if (s) return s;
    if (hipEventRecord(e->done[w], e->streams[w]) != hipSuccess)
      return efail(ASGD_EHIP, "event record failed");
    clock[w] += c.slow[w] * (c.c0 + c.c1 * (double)take + c.c2 * (double)xb.nnz);
    if (log && nd < log->max_dispatch) {
      log->replica[nd] = w;
      log->row0[nd] = r0;
      log->row1[nd] = r1;
    }
    ++nd;
    ++u[w];
    samples[w] += take;
    left -= take;
    e->cursor = r1 < n_rows ? r1 : 0;
  }

  double l2[16] = {};
  if (c.perturb) {  // every replica's norm in one launch and one host synchronization
    asgd_status s = asgd_models_l2_per_param(e->reps.data(), n, l2);
    if (s) return s;
  }
  float alpha[16];
  asgd_status s = asgd_merge_weights(n, u, e->b.data(), samples, c.weight_mode, c.perturb ? l2 : nullptr,
                                     c.pert_thr, c.delta, alpha);
  if (s) return s;
  s = asgd_merge(e->global, e->prev, e->reps.data(), alpha, n, c.gamma, 1);
  if (s) return s;
  s = asgd_scale_batches(n, u, e->b.data(), e->lr.data(), c.b_min, c.b_max, c.beta);
  if (s) return s;
  if (log) {
    log->n_dispatch = nd;
    for (int i = 0; i < n; ++i) {
      log->u[i] = u[i];
      log->samples[i] = samples[i];
      log->alpha[i] = alpha[i];
      log->l2_per_param[i] = l2[i];
      log->b_next[i] = e->b[i];
      log->lr_next[i] = e->lr[i];
    }
    log->cursor = (int32_t)e->cursor;
  }
  return ASGD_OK;
}

}  // extern "C"
