"""MI355X-native EventProp training step for LIF networks with learnable delays.

Thin Python binding over the C ABI of ``libsnn.so`` (see ``include/snn.h``):
argument marshalling only.  Every step of the forward and backward pass runs
in the library's HIP kernels; PyTorch only provides device memory and the
stream.  ``load_library()`` and ``Network()`` fail loudly if the library has
not been built (``python -m paper_2501_07331_amd.build``); there is no CPU
fallback.
"""
from .binding import (SNNError, SNNOverflow, Network, lib_path, load_library, SNN_INPUT, SNN_LIF,
                      SNN_LI, SNN_LOSS_CE_SUM, SNN_LOSS_CE_MAX, SNN_LOSS_DMSE, SNN_FLAG_HBM_RINGS,
                      SNN_FLAG_TIMING, SNN_FLAG_SEPARATE_READOUT, SNN_FLAG_CLUSTER, SNN_OPT_SGD, SNN_OPT_ADAM, SNN_OK, SNN_EINVAL, SNN_ENOMEM,
                      SNN_ESTATE, SNN_EOVERFLOW, SNN_EDEVICE, SNN_NOALLOC_SCRATCH_BYTES)
from . import schedules

__all__ = ["SNNError", "SNNOverflow", "Network", "lib_path", "load_library", "SNN_INPUT", "SNN_LIF",
           "SNN_LI", "SNN_LOSS_CE_SUM", "SNN_LOSS_CE_MAX", "SNN_LOSS_DMSE", "SNN_FLAG_HBM_RINGS",
           "SNN_FLAG_TIMING", "SNN_FLAG_SEPARATE_READOUT", "SNN_FLAG_CLUSTER", "SNN_OPT_SGD", "SNN_OPT_ADAM", "SNN_OK", "SNN_EINVAL", "SNN_ENOMEM",
           "SNN_ESTATE", "SNN_EOVERFLOW", "SNN_EDEVICE", "SNN_NOALLOC_SCRATCH_BYTES",
           "schedules"]
