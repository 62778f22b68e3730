"""conv_einsum engine for AMD Instinct MI355X (gfx950).

Evaluates tensorial convolution layers written as conv_einsum strings
(arXiv 2401.03384) as a FLOP-minimal sequence of pairwise steps, with the
planner and the HIP kernels in libconvein.so (C ABI: include/convein.h).
"""
from .binding import (CeError, ce_backward, ce_backward_noalloc, ce_expr_destroy, ce_expr_output_shape,
                      ce_expr_parse, ce_expr_set_conv, ce_expr_set_feature, ce_expr_set_stride, ce_forward,
                      ce_last_error,
                      ce_plan_checkpoint, ce_plan_cost, ce_plan_create, ce_plan_create_ex, ce_plan_create_limited, ce_plan_create_with_path, ce_plan_describe,
                      ce_plan_destroy, ce_plan_left_to_right_cost, ce_plan_num_steps,
                      ce_plan_step, ce_plan_workspace_size, ce_timing_begin, ce_timing_begin_kernel,
                      ce_timing_end,
                      ce_timing_record, ce_version, lib, LIB_PATH,
                      CE_F32, CE_BF16, CE_COST_FWD, CE_COST_TRAIN_PAPER, CE_FLAG_GENERIC_ONLY,
                      CE_FLAG_NO_FUSION, CE_FLAG_SAVE_INTERMEDIATES, CE_FLAG_WIDE_OFFSETS, CE_NOALLOC_WORKSPACE_BYTES,
                      CE_PAD_SAME_ZERO, CE_PAD_CIRCULAR)
from .layer import GraphStep, Plan, plan, conv_einsum, contract_path, max_batch, step_bytes

__all__ = [
    "CeError", "ce_backward", "ce_backward_noalloc", "ce_expr_destroy", "ce_expr_output_shape", "ce_expr_parse",
    "ce_expr_set_conv", "ce_expr_set_feature", "ce_expr_set_stride", "ce_forward", "ce_last_error", "ce_plan_cost", "ce_plan_create",
    "ce_plan_create_limited", "ce_plan_create_ex", "ce_plan_checkpoint", "ce_plan_create_with_path", "ce_plan_describe", "ce_plan_destroy",
    "ce_plan_left_to_right_cost", "ce_plan_num_steps", "ce_plan_step", "ce_plan_workspace_size",
    "ce_timing_begin", "ce_timing_begin_kernel", "ce_timing_end", "ce_timing_record",
    "ce_version", "lib", "LIB_PATH", "GraphStep", "Plan", "plan", "conv_einsum", "contract_path", "max_batch", "step_bytes",
    "CE_F32", "CE_BF16", "CE_COST_FWD", "CE_COST_TRAIN_PAPER", "CE_FLAG_GENERIC_ONLY",
    "CE_FLAG_NO_FUSION", "CE_FLAG_SAVE_INTERMEDIATES", "CE_FLAG_WIDE_OFFSETS", "CE_NOALLOC_WORKSPACE_BYTES", "CE_PAD_SAME_ZERO", "CE_PAD_CIRCULAR",
]
