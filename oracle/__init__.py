"""Plain fp64 CPU oracle for TF-chunk-masked softmax attention and its JVP.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this package.
The product path (the HIP library and its Python binding) never routes through
it, and this package imports nothing from the product.

Contents
--------
masks      -- the attention mask materialised from its definition (per-token
              chunk ids), for the full, block-causal and teacher-forcing kinds,
              and from an explicit query-group / key-range list (any number
              of key ranges per group).
attention  -- closed-form masked attention O, LSE and the forward-mode tangent
              dO (paper, App. B, the masked-attention and tangent equations),
              and the same JVP with zero tangents on the clean half of a
              teacher-forcing sequence (paper Sec. 3.1.2, TF-sCM tangent).
backward   -- the closed-form gradient (vector-Jacobian product) of the same
              masked attention: gQ, gK, gV and Delta = rowsum(gO o O).
dual       -- a pure-Python dual-number evaluation of the same map, used on
              tiny inputs to pin the closed form (no closed-form tangent used).

Parity status: every function here is pinned by tests in
``tests/test_oracle_pins.py`` (finite differences, dual numbers, PyTorch's
scaled_dot_product_attention and torch.func.jvp, the two-pass TF identity,
hand-derived golden values and invariants).
"""
from .masks import (MASK_FULL, MASK_BLOCK_CAUSAL, MASK_TEACHER_FORCING, MASK_RANGES, allowed_mask, check_groups,
                    count_allowed_pairs)
from .attention import attention_jvp, attention_fwd, attention_jvp_zero_clean
from .backward import attention_vjp

__all__ = [
    "MASK_FULL", "MASK_BLOCK_CAUSAL", "MASK_TEACHER_FORCING", "MASK_RANGES",
    "allowed_mask", "check_groups", "count_allowed_pairs", "attention_jvp", "attention_fwd", "attention_jvp_zero_clean",
    "attention_vjp",
]
