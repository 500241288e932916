"""Reference group rollout: G completions per prompt (Sec. 3.1, problem
statement), generated one sequence at a time from an explicit KV cache.

Layout: sequence s = off_p + j is sibling j of prompt p, where off is the
exclusive prefix sum of the group sizes (prompt-major order).  Every sibling
starts from the logits of its prompt's last position; its step-0 token is drawn
with its own noise stream (the stream index is s).  Step t >= 1 feeds the
previous token at position Lp + t - 1.  A sequence retires after emitting EOS or
after emitting its max_new-th token; its length counts generated tokens
including the EOS.  Output padding: token -1, log-probability 0.
"""
from __future__ import annotations

import numpy as np

from .model import OracleModel
from .sampling import sample_token


def group_offsets(G) -> np.ndarray:
    G = np.asarray(G, np.int64)
    return np.concatenate([[0], np.cumsum(G)])


def rollout(model: OracleModel, prompts, G, max_new: int, seed: int, forced_len=None,
            temperature: float = 1.0, max_steps=None, prompt_subset=None, record_steps: int = 0,
            on_step=None):
    """Free-running rollout.  ``max_steps`` truncates generation (sequences not
    yet retired keep length 0); ``prompt_subset`` restricts it to some prompts;
    ``record_steps`` keeps the logits of steps t < record_steps; ``on_step``, if
    given, is called as on_step(p, t, n_active) after each decode step (a
    progress hook for long timings; it sees no values of the computation).

    Returns a dict with tokens [N, max_new] int32, lengths [N] int32, logprobs
    [N, max_new] float64, margins [N, max_new] float64 (nan where not sampled)
    and, if requested, logits {(s, t): float64 [V]}."""
    s_ = model.s
    eos = s_.eos_id
    G = np.asarray(G, np.int64)
    off = group_offsets(G)
    N = int(off[-1])
    tokens = np.full((N, max_new), -1, np.int32)
    lengths = np.zeros(N, np.int32)
    logprobs = np.zeros((N, max_new), np.float64)
    margins = np.full((N, max_new), np.nan)
    logits = {}
    limit = max_new if max_steps is None else min(max_new, int(max_steps))
    for p in (range(len(G)) if prompt_subset is None else prompt_subset):
        prompt = np.asarray(prompts[p], np.int64)
        Lp = len(prompt)
        cache = model.new_cache()
        z_last = model.forward(prompt, np.arange(Lp), cache)[-1]
        sibs = [int(off[p]) + j for j in range(int(G[p]))]
        caches = {s: model.copy_cache(cache) for s in sibs}
        z = {s: z_last for s in sibs}
        active, t = sibs, 0
        while active and t < limit:
            still = []
            for s in active:
                L = None if forced_len is None else int(forced_len[s])
                if t < record_steps:
                    logits[(s, t)] = z[s]
                y, lp, mg = sample_token(z[s], seed, t, s, eos, temperature, L)
                tokens[s, t], logprobs[s, t], margins[s, t] = y, lp, mg
                if y == eos or t + 1 == max_new:
                    lengths[s] = t + 1
                else:
                    still.append(s)
            t += 1
            if still and t < limit:
                zz = model.decode_batch([tokens[s, t - 1] for s in still], [Lp + t - 1] * len(still),
                                        [caches[s] for s in still])
                z = {s: zz[i] for i, s in enumerate(still)}
            active = still
            if on_step is not None:
                on_step(p, t, len(active))
    out = dict(tokens=tokens, lengths=lengths, logprobs=logprobs, margins=margins)
    if record_steps:
        out["logits"] = logits
    return out
