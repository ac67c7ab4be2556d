"""MI355X (gfx950) masked softmax attention forward and forward-mode JVP.

The compute path is the C-ABI library ``libattnjvp.so`` (hand-written HIP
kernels); :mod:`paper_2606_25473_amd.binding` marshals torch tensors into it.
Importing this package does not load the library; the first call does, and it
raises if the library is missing or was built for another target.
"""
from .binding import (attn_jvp_fwd, attn_jvp_fwd_zero_clean, attn_fwd, attn_bwd, count_unmasked_pairs, count_computed_pairs, query_groups,
                      library_path, load_library, AttnError)

__all__ = ["attn_jvp_fwd", "attn_jvp_fwd_zero_clean", "attn_fwd", "attn_bwd", "count_unmasked_pairs", "count_computed_pairs", "query_groups",
           "library_path", "load_library", "AttnError"]
