"""Mixed-adapter LoRA layer for AMD Instinct MI355X (gfx950).

Python face of liblora_mi355x.so (include/lora.h): ``Table`` (adapter table),
``Plan`` (row grouping by adapter id), ``shrink``, ``expand``, ``apply``,
``apply_ids`` (small batches without a plan), ``linear``, ``grad``, ``grad_x``,
``backward``, ``adamw_step`` and ``token_loss``.  Torch supplies device memory
and streams; the computation runs in the library's HIP kernels.  Nothing here
falls back to another implementation: if the library is not built, every call
raises.  ``Table(..., debug=True)`` runs a table's plans and ops through the
debug build, liblora_mi355x_debug.so.
"""
from .lora import (AdamWTensor, Policy, LOSS_CE, LOSS_IS, LOSS_PPO, LORA_BF16, LORA_BUILD_DEBUG,
                   LORA_DATA_BAD_ID, LORA_DATA_BAD_SEGMENTS, LORA_DATA_BOUNDS, LORA_DATA_EMPTY_SLOT,
                   LORA_F32, LORA_PLAN_M_PERM, LORA_PLAN_PERM, LORA_PLAN_SMALL_ROW, DEBUG_LIB_PATH,
                   LIB_PATH, LoraError, Plan, Table, apply, apply_ids, apply_ids_workspace,
                   apply_noalloc, apply_workspace, expand, adamw_step, backward, backward_workspace,
                   grad, grad_workspace, grad_x, grad_x_workspace, lib, linear, linear_workspace,
                   shrink, token_loss)

__all__ = ["Table", "Plan", "Policy", "shrink", "expand", "apply", "apply_ids",
           "apply_ids_workspace", "apply_noalloc", "linear", "linear_workspace", "grad", "grad_x",
           "backward", "backward_workspace", "adamw_step", "AdamWTensor", "token_loss", "LOSS_CE",
           "LOSS_IS", "LOSS_PPO", "apply_workspace", "grad_workspace", "grad_x_workspace", "lib",
           "LoraError", "LORA_F32", "LORA_BF16", "LORA_DATA_BAD_ID", "LORA_DATA_EMPTY_SLOT",
           "LORA_DATA_BAD_SEGMENTS", "LORA_DATA_BOUNDS", "LORA_BUILD_DEBUG", "LORA_PLAN_PERM",
           "LORA_PLAN_M_PERM", "LORA_PLAN_SMALL_ROW", "LIB_PATH", "DEBUG_LIB_PATH"]
