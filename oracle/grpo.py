"""GRPO loss forward: teacher-forced log-probabilities of the rollout under the
current policy, and the clipped surrogate built from them (Sec. 2 names GRPO
and DAPO as the training objectives; Sec. 5 trains with both).  The paper
gives no formula; this follows the published objectives it cites:

* Token log-probability (the quantity the rollout reports, Sec. 3.1 setting):
  logprob[s, t] = z_{y_t}/T - logsumexp(z/T), z the logits after the prompt
  and y_0 .. y_{t-1}.  Here every sequence is re-run as ONE causal forward
  over prompt + y_0 .. y_{L-2} with no cache reuse between siblings or steps,
  a different route from the rollout's incremental decode.
* Importance ratio rho = exp(new - old) per token, in float64.
* PPO clipped surrogate per token: min(rho * A, clip(rho, 1 - eps_lo,
  1 + eps_hi) * A), A the sequence's group-relative advantage.  eps_lo =
  eps_hi is the GRPO/PPO form; eps_hi > eps_lo is DAPO's decoupled clip.
* Aggregation: "token" (DAPO) = sum over every counted token / number of
  counted tokens; "seq" (GRPO) = mean over counted sequences of each
  sequence's token mean.  loss = -(aggregate).  No KL term (DAPO drops it;
  GRPO's needs a reference policy, outside this path).
* A token is "clipped" when the clipped term is strictly smaller than the
  unclipped one, i.e. when the min picks the clip.
* keep (optional, per group, e.g. from the zero-variance filter) removes
  every sequence of a dropped group from the aggregate.

Test infrastructure only: the library never calls this module.
"""
from __future__ import annotations

import math

import numpy as np

from .model import OracleModel
from .sampling import logsumexp


def teacher_forced_logprobs(model: OracleModel, prompts, G, tokens, lengths, temperature: float = 1.0):
    """float64 [N, max_new]: log-probability of tokens[s, t] for t < lengths[s],
    0 elsewhere."""
    G = [int(g) for g in G]
    tokens = np.asarray(tokens)
    N, max_new = tokens.shape
    if sum(G) != N:
        raise ValueError("sum(G) != number of sequences")
    out = np.zeros((N, max_new), np.float64)
    s = 0
    for p, g in enumerate(G):
        prompt = np.asarray(prompts[p], np.int64)
        Lp = len(prompt)
        for _ in range(g):
            L = int(lengths[s])
            if not 1 <= L <= max_new:
                raise ValueError("length out of [1, max_new]")
            y = tokens[s, :L].astype(np.int64)
            seq = np.concatenate([prompt, y[:L - 1]])
            z = model.forward(seq, np.arange(len(seq)), model.new_cache())   # [Lp + L - 1, V]
            for t in range(L):
                zt = z[Lp - 1 + t] / float(temperature)
                out[s, t] = zt[y[t]] - logsumexp(zt)
            s += 1
    return out


def clipped_surrogate(new_lp, old_lp, adv, lengths, G, eps_lo: float = 0.2, eps_hi: float = 0.2,
                      mode: str = "token", keep=None):
    """Returns (loss, clipped fraction, counted tokens, counted sequences).
    new_lp, old_lp: [N, max_new]; adv, lengths: [N]; keep: [P] or None."""
    new_lp = np.asarray(new_lp, np.float64)
    old_lp = np.asarray(old_lp, np.float64)
    adv = np.asarray(adv, np.float64)
    G = [int(g) for g in G]
    if any(g < 1 for g in G) or sum(G) != len(adv):
        raise ValueError("group sizes do not partition the sequences")
    if mode not in ("token", "seq"):
        raise ValueError(mode)
    total = 0.0          # token mode: sum of every counted token's term
    seq_total = 0.0      # seq mode: sum of per-sequence means
    n_tok = n_seq = n_clip = 0
    s = 0
    for p, g in enumerate(G):
        for _ in range(g):
            if keep is None or keep[p]:
                L = int(lengths[s])
                a = float(adv[s])
                seq_sum = 0.0
                for t in range(L):
                    rho = math.exp(new_lp[s, t] - old_lp[s, t])
                    unclipped = rho * a
                    clipped = min(max(rho, 1.0 - eps_lo), 1.0 + eps_hi) * a
                    seq_sum += min(unclipped, clipped)
                    n_clip += clipped < unclipped
                total += seq_sum
                seq_total += seq_sum / L
                n_tok += L
                n_seq += 1
            s += 1
    if n_seq == 0:
        return 0.0, 0.0, 0, 0
    agg = total / n_tok if mode == "token" else seq_total / n_seq
    return -agg, n_clip / n_tok, n_tok, n_seq
