"""MI355X-native scaled-FP8 matmul with fused dynamic rescale and cast
(Scalify scale propagation, arXiv 2407.17353).

The compute path is the HIP library libscalify.so (C ABI in include/scalify.h);
`binding` marshals torch device tensors into it. Build with
`python paper_2407_17353_amd/build.py`.
"""
from .binding import (E4M3, E5M2, F16, F32, RESCALE_AMAX, RESCALE_NONE, ScaledArray,  # noqa: F401
                      ScalifyError, empty_scaled, load_library, scale_tensor, scalify_cast,
                      scalify_matmul, scalify_matmul_scale_log2, scalify_matmul_workspace_size,
                      scalify_rescale, scalify_rescale_workspace_size, scalify_set_scaling)
