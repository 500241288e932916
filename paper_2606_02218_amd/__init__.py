"""MI355X (gfx950) group-rollout hot path: ctypes binding of librollout.so.

Every step of the path runs in the library's HIP kernels, and the group-size
controller (Sagc) in the library's host code; this package only marshals
arguments (PyTorch tensors supply device memory and the stream).  Import fails
loudly when the library has not been built.
"""
from ._lib import (  # noqa: F401
    RolloutError, Policy, group_advantage, philox_blocks, gumbel_bits, lib_path, load_library,
    KERNEL_KINDS, exported_symbols, Sagc, sagc_beta_draw, group_filter, grpo_surrogate, decode_attention_chunks, hbm_probe,
)
