"""MI355X (gfx950) HIP implementation of Ekya's retraining / micro-profiling /
inference hot path, behind the C ABI in include/ekya.h.

`binding` is the ctypes layer over libekya.so (built in-tree by
`python -m paper_2012_10557_amd.build`).
"""
from . import binding  # noqa: F401
from .binding import (  # noqa: F401
    EkyaError,
    ekya_create,
    ekya_destroy,
    ekya_epoch_order,
    ekya_infer,
    ekya_profile,
    ekya_retrain,
    ekya_training_subset,
    ekya_weights_count,
)
