"""MI355X-native batched latency attribution (LLMVisor, Sec. 2.1, Eq. 1).

The computation lives in libllmv.so (HIP kernels for gfx950, C ABI in
include/llmv.h); ``llmv`` is its ctypes binding.
"""
from . import llmv  # noqa: F401
from .llmv import (DeviceTrace, LlmvError, admit, attribute, attribute_ext,  # noqa: F401
                   attribute_sweep, batch_sums, features, fit, fit_metrics, fit_workspace, llmv_admit,
                   llmv_attribute, llmv_attribute_ext, llmv_attribute_sweep, llmv_batch_sums,
                   llmv_attribute_sweep_ext, llmv_sweep_workspace_size_ext,
                   llmv_batch_sums_ext, llmv_fit_ext, llmv_fit_metrics_ext, llmv_admit_ext,
                   llmv_features, llmv_shape_constants_ext,
                   llmv_fit, llmv_fit_metrics, llmv_fit_workspace_size, llmv_last_error,
                   llmv_shape_constants, llmv_sweep_workspace_size, llmv_tenant_sums,
                   llmv_validate, llmv_workspace_size, sweep_workspace, tenant_sums, workspace)
