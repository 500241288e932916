"""The 7B decoder's widths on the GPU, against the oracle, at two layers.

Every layer of the 7B-shaped decoder runs the same kernels, so two layers at
full width cover what the full depth would: 28 query heads over 4 kv heads
(7 query heads per kv head: the decode attention fills 7 of its 16 MFMA query
columns, and the recompute's row tiles take 16 positions, since 7 x 32 query
rows would need more than 12 waves), projections with K = 3584 and 18944,
QKV N = 4608, gate/up N = 37888, and a 152064-token vocabulary.

* rollout, teacher-forced on the oracle's tokens: every logit within 1e-2
  (max-abs) of the fp64 oracle's, sampling decisions equal except at top-2
  margins below 1e-2, lengths bit-exact;
* free-running from the same inputs follows the oracle's trajectory;
* the teacher-forced recompute of the oracle's tokens reproduces the oracle's
  log-probabilities within 2e-2, and the rollout's own within 2e-2.
"""
import numpy as np
import pytest

from oracle.grpo import teacher_forced_logprobs
from oracle.rollout import rollout as oracle_rollout
from workload import get_config, make_weights, ModelShape
from rg_helpers import (oracle_for, make_policy, prompts_to_device, compare_free_running, check_structure,
                        MARGIN_TOL, LOGIT_TOL)

pytestmark = pytest.mark.gpu

_S = get_config("7b").shape
SHAPE = ModelShape(2, _S.d_model, _S.n_q_heads, _S.n_kv_heads, _S.head_dim, _S.ffn_dim, _S.vocab, _S.rope_theta,
                   dtype="bf16")


@pytest.mark.timeout(400)
def test_7b_widths_rollout_and_recompute():
    import torch
    assert torch.cuda.is_available()
    assert (SHAPE.n_q_heads, SHAPE.n_kv_heads, SHAPE.d_model, SHAPE.ffn_dim, SHAPE.vocab) == (28, 4, 3584, 18944, 152064)
    w = make_weights(SHAPE, 7)
    rng = np.random.default_rng(707)
    prompts = [rng.integers(0, SHAPE.vocab - 1, size=n).astype(np.int32) for n in (61, 20)]
    G, max_new, seed = [5, 3], 16, 77
    L = rng.integers(1, max_new + 1, size=8).astype(np.int32)
    L[0], L[-1] = 1, max_new
    print(f"7B-width case: 2 layers, prompts {[len(p) for p in prompts]}, G {G}, max_new {max_new}", flush=True)
    model = oracle_for(SHAPE, w)
    ref = oracle_rollout(model, prompts, G, max_new, seed, L, record_steps=max_new)
    pol = make_policy(SHAPE, w, max_seqs=8, max_prompts=2, max_prompt_tokens=81, max_context=61 + max_new)
    ft = torch.from_numpy(ref["tokens"]).cuda()
    dp = prompts_to_device(prompts)
    tok, ln, lp, dump = pol.rollout(dp, G, max_new, seed, forced_len=L, force_tokens=ft, dump_steps=max_new)
    torch.cuda.synchronize()
    tok, ln, lp, dump = tok.cpu().numpy(), ln.cpu().numpy(), lp.cpu().numpy(), dump.cpu().numpy()
    np.testing.assert_array_equal(ln, L)
    worst = 0.0
    for s in range(len(L)):
        for t in range(int(L[s])):
            worst = max(worst, float(np.max(np.abs(dump[t, s].astype(np.float64) - ref["logits"][(s, t)]))))
            if tok[s, t] != ref["tokens"][s, t]:
                assert ref["margins"][s, t] < MARGIN_TOL, (s, t, ref["margins"][s, t])
            assert abs(lp[s, t] - ref["logprobs"][s, t]) <= 2 * LOGIT_TOL
    print(f"worst teacher-forced logit gap {worst:.2e}", flush=True)
    assert worst <= LOGIT_TOL, worst

    tok3, ln3, lp3 = pol.rollout(dp, G, max_new, seed, forced_len=L)
    tok3, ln3, lp3 = tok3.cpu().numpy(), ln3.cpu().numpy(), lp3.cpu().numpy()
    check_structure(tok3, ln3, lp3, SHAPE.eos_id, max_new, L)
    compare_free_running(tok3, lp3, ref, ln3, lp_tol=2 * LOGIT_TOL)

    want = teacher_forced_logprobs(model, prompts, G, ref["tokens"], ref["lengths"])
    got = pol.recompute_logprobs(dp, G, ft, torch.from_numpy(ref["lengths"]).cuda()).cpu().numpy()
    valid = np.arange(max_new)[None, :] < ref["lengths"][:, None]
    assert np.all(got[~valid] == 0)
    gap = float(np.max(np.abs(got[valid] - want[valid])))
    print(f"recompute vs oracle logprob gap {gap:.2e}", flush=True)
    assert gap <= 2 * LOGIT_TOL, gap
    assert float(np.max(np.abs(got[valid] - lp[valid]))) <= 2 * LOGIT_TOL
    pol.close()
