"""NVFP4 ScaleSweep quantization on AMD Instinct MI355X (gfx950).

Thin Python binding of the C library ``libnvfp4ss.so`` (declared in include/nvfp4ss.h).
Every step of the quantizer runs in the library's HIP kernels; this package only marshals
arguments, using PyTorch for device memory and streams.  There is no CPU fallback: if the
library is not built, importing the binding raises.
"""
from .nvfp4 import (  # noqa: F401
    LIB_PATH,
    METHOD_IDS,
    NOALLOC_MAX_TENSORS,
    NVFP4Error,
    block_loss,
    block_optimum,
    channel_sq_norms,
    dequant,
    gap_report,
    gptq_quantize,
    ldlq,
    lib,
    nvfp4_batched_workspace_bytes,
    nvfp4_block_loss,
    nvfp4_block_optimum,
    nvfp4_channel_sq_norms,
    nvfp4_channel_sq_norms_workspace_bytes,
    nvfp4_dequant,
    nvfp4_ldlq,
    nvfp4_ldlq_workspace_bytes,
    nvfp4_quant_batched,
    nvfp4_quant_batched_noalloc,
    nvfp4_quant_absmax,
    nvfp4_quant_four_over_six,
    nvfp4_quant_online,
    nvfp4_quant_scalesweep_mse,
    nvfp4_quant_scalesweep_wmse,
    nvfp4_quant_scalesweep_window,
    nvfp4_scales_bytes,
    nvfp4_status_string,
    nvfp4_sum_f64,
    nvfp4_sum_workspace_bytes,
    nvfp4_workspace_bytes,
    quantize,
    quantize_batched,
    quantize_online,
    quantize_window,
    sum_f64,
    workspace,
)
