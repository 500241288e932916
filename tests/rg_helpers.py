"""Shared helpers for the GPU parity tests: build a policy from a seeded
workload, run the oracle on the same inputs, and compare."""
from __future__ import annotations

import numpy as np

from oracle.model import OracleModel

MARGIN_TOL = 1e-2      # token decisions with a smaller top-2 gap may differ
LOGIT_TOL = 1e-2       # max-abs logit error under teacher forcing


def oracle_for(shape, weights):
    """The oracle with the model's storage type for its KV cache."""
    return OracleModel(shape, weights, kv_storage="model")


def make_policy(shape, weights, max_seqs, max_prompts, max_prompt_tokens, max_context, kv_pool_pages=0):
    from paper_2606_02218_amd import Policy
    return Policy(shape, weights, max_seqs=max_seqs, max_prompts=max_prompts, max_prompt_tokens=max_prompt_tokens,
                  max_context=max_context, kv_pool_pages=kv_pool_pages)


def prompts_to_device(prompts):
    import torch
    return [torch.as_tensor(np.asarray(p, np.int32)).cuda() for p in prompts]


def compare_free_running(gpu_tokens, gpu_logprobs, ref, lengths, lp_tol):
    """Tokens must agree position by position until the first position where
    the oracle's top-2 margin is below MARGIN_TOL (from there the two
    trajectories may legitimately split).  Every position up to and including
    that one is compared, so the count of compared positions is fixed by the
    oracle alone and is checked here.  Returns (positions compared, sequences
    that split)."""
    checked, split = 0, 0
    expected = 0
    for s in range(gpu_tokens.shape[0]):
        L = int(ref["lengths"][s]) if ref["lengths"][s] > 0 else int(lengths[s])
        low = np.flatnonzero(ref["margins"][s, :L] < MARGIN_TOL)
        expected += int(low[0]) + 1 if len(low) else L
    for s in range(gpu_tokens.shape[0]):
        for t in range(int(lengths[s])):
            if gpu_tokens[s, t] != ref["tokens"][s, t]:
                assert ref["margins"][s, t] < MARGIN_TOL, (
                    f"seq {s} step {t}: gpu {gpu_tokens[s, t]} oracle {ref['tokens'][s, t]} "
                    f"margin {ref['margins'][s, t]}")
                split += 1
                break
            assert abs(gpu_logprobs[s, t] - ref["logprobs"][s, t]) <= lp_tol, (s, t, gpu_logprobs[s, t], ref["logprobs"][s, t])
            checked += 1
            if ref["margins"][s, t] < MARGIN_TOL:
                split += 1
                break
    # a mismatch stops one position early (that position is not counted)
    assert checked + split >= expected, (checked, split, expected)
    return checked, split


def check_structure(tokens, lengths, logprobs, eos, max_new, forced_len=None):
    N = tokens.shape[0]
    for s in range(N):
        L = int(lengths[s])
        assert 1 <= L <= max_new
        if forced_len is not None:
            assert L == int(forced_len[s])
        row = tokens[s]
        assert row[L - 1] == eos or L == max_new
        assert np.all(row[:L - 1] != eos) and np.all(row[:L] >= 0)
        assert np.all(row[L:] == -1)
        assert np.all(logprobs[s, L:] == 0)
        assert np.all(np.isfinite(logprobs[s, :L])) and np.all(logprobs[s, :L] <= 1e-6)
