"""MI355X (gfx950) LoRA-linear hot path: HIP kernels behind a C ABI.

The Python names mirror the C entry points of include/lora_mi355x.h.
"""
from .lora import (LORA_BF16, LORA_F32, LORA_OP_BWD, LORA_OP_FROZEN_DX, LORA_OP_FWD,  # noqa: F401
                   LoraError, frozen_linear_bwd_dx, frozen_linear_bwd_dx_q, kernel_names, lib,
                   lora_linear_bwd, lora_linear_bwd_noalloc, lora_linear_bwd_q, lora_linear_fwd, lora_linear_fwd_q,
                   lora_ckpt_backward, lora_ckpt_forward, lora_ckpt_sizes,
                   lora_linear_workspace_bytes, lm_head_build_vocab, lm_head_reduced_ce,
                   lm_head_workspace_bytes, profiler_enable, profiler_read, profiler_reset,
                   topk_table_build, lora_linear_plan, handover_giveups, debug_set_handover)
