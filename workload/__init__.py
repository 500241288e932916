"""Seeded synthetic workloads for the group-rollout hot path.

This package produces *inputs only*: model shapes, random-init weights, prompt
token ids, per-prompt group sizes, forced completion lengths and rewards.  It
holds none of the method's arithmetic (no forward pass, no sampling, no
advantage), so both the CPU oracle and the HIP path can consume its outputs.
"""
from .configs import CONFIGS, ModelShape, Workload, get_config  # noqa: F401
from .gen import (  # noqa: F401
    make_weights, make_prompts, make_group_sizes, make_forced_lengths,
    make_rewards, make_inputs, bf16_round_f32, f32_to_bf16_bits, step_group_lengths, step_rewards,
    drifted_logprobs,
)
