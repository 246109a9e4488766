"""Float64 CPU oracle for the mixed-adapter LoRA layer.

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library (no kernels, headers, helpers or constants).

Parity pins (tests/test_oracle_pins.py): hand-derived worked examples in
tests/golden/, scalar brute force on tiny inputs, exact linearity of the
masked loss in A, in B and in X (pins the backward and the input gradient),
the merged-weight identity X (W + s B A)^T for the whole layer,
closed forms for permutation / diagonal / rank-1 adapters, integer-valued
exactness, AdamW against torch.optim.AdamW in float64 and its closed forms, the
token losses against torch's cross-entropy, finite differences and closed forms,
and planted-mistake checks that each pin rejects.  No function here is "parity unpinned".
"""
from .lora_oracle import (effective_ids, canonical_plan, plan_bruteforce,
                          segments_to_ids, shrink, expand, apply, delta_rows,
                          apply_bruteforce, linear, linear_rows, linear_bruteforce, grad, grad_bruteforce, grad_x,
                          grad_x_bruteforce, masked_loss, adamw, token_loss, LOSS_CE,
                          LOSS_IS, LOSS_PPO, rel_fro, max_abs)

__all__ = ["effective_ids", "canonical_plan", "plan_bruteforce", "segments_to_ids",
           "shrink", "expand", "apply", "delta_rows", "apply_bruteforce", "linear",
           "linear_rows", "linear_bruteforce", "grad",
           "grad_bruteforce", "grad_x", "grad_x_bruteforce", "masked_loss", "adamw",
           "token_loss", "LOSS_CE", "LOSS_IS", "LOSS_PPO", "rel_fro", "max_abs"]
