"""MI355X (gfx950) implementation of the hot path of Accumulated Gradient
Normalization (AGN): n simulated workers, lambda local SGD steps each,
normalized commits in a given order, pulls.  The compute runs in the HIP
kernels of libagn.so; this package holds the ctypes binding and the build.
"""
from .agn import (AGN, AGNError, AGN_BF16, AGN_EHIP, AGN_EINVAL, AGN_ENOMEM, AGN_ESTATE, AGN_FP32, AGN_OK, AGN_OPT_ADAM, AGN_OPT_SGD, EXPORTED, KERNEL_CLASSES, LIB_PATH,  # noqa: F401
                  agn_central, agn_create, agn_debug_batch_indices, agn_debug_delta, agn_destroy, agn_evaluate, agn_evaluate_noalloc, agn_kernel_class_work, agn_kernel_timing,
                  agn_last_error, agn_loss, agn_num_params, agn_round, agn_set_central,
                  agn_set_kernel_timing, agn_set_normalization, agn_set_optimizer, agn_set_staleness_scaling, agn_set_stream, agn_staleness, agn_temporal_efficiency, agn_worker_params, load_library)
