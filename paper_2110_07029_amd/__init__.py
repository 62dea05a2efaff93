"""MI355X (gfx950) hot path of Adaptive SGD (arXiv 2110.07029).

``libasgd.so`` (HIP kernels behind the C ABI of ``include/asgd.h``) does all
the work; this package holds its ctypes binding (same names as the C entry
points), device-resident datasets and the seeded synthetic input generator.
"""
from ._binding import (  # noqa: F401
    ASGD_OK, ASGD_EINVAL, ASGD_ERANGE, ASGD_ENOMEM, ASGD_EHIP, ASGD_ESTATE, ASGD_VALIDATE, ASGD_UNFUSED_OUTPUT,
    ASGD_PARAM_W1, ASGD_PARAM_B1, ASGD_PARAM_W2, ASGD_PARAM_B2, ASGD_PARAM_WH, ASGD_PARAM_BH, ASGD_WEIGHTS_ALG2,
    ASGD_WEIGHTS_SAMPLES, ASGD_WEIGHTS_UNIFORM, ASGD_DISPATCH_DYNAMIC, ASGD_DISPATCH_STATIC, EXPORTS, HIDDEN, AsgdError, asgd_config, asgd_csr, load, library_path,
    asgd_last_error, asgd_model_init, asgd_model_free, asgd_model_set_stream, asgd_model_copy,
    asgd_model_num_params, asgd_model_get_params, asgd_model_set_params, asgd_train_step,
    asgd_model_last_loss, asgd_predict_topk, asgd_merge, asgd_model_l2_per_param, asgd_models_l2_per_param,
    asgd_models_l2_per_param_noalloc,
    asgd_merge_weights, asgd_scale_batches, asgd_debug_forward, asgd_debug_touched_rows,
    asgd_model_set_timing, asgd_model_get_timing, KERNELS, ASGD_CLOCK_TIMED, ASGD_CLOCK_VIRTUAL,
    asgd_elastic_config, asgd_elastic_log, asgd_elastic_create, asgd_elastic_free, asgd_elastic_round,
    asgd_elastic_model, asgd_libsvm_info, asgd_libsvm_scan, asgd_libsvm_read,
)
from .device_data import DeviceCSR  # noqa: F401
