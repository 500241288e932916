"""A context longer than one attention chunk's span (16000 tokens): a
19990-token prompt, so the prefill splits every row's context into two chunks
and merges them, decode steps do the same, and the recompute (contexts above
16384 tokens) takes the row-by-row attention instead of row tiles.  Checked
against the oracle: teacher-forced logits within 1e-2, sampling decisions
equal except at top-2 margins below 1e-2, lengths exact, and the recompute
within 2e-2 of the oracle's log-probabilities."""
import numpy as np
import pytest

from oracle.grpo import teacher_forced_logprobs
from oracle.rollout import rollout as oracle_rollout
from workload import ModelShape, make_weights
from rg_helpers import oracle_for, make_policy, prompts_to_device, MARGIN_TOL, LOGIT_TOL

pytestmark = pytest.mark.gpu

SHAPE = ModelShape(1, 128, 2, 1, 64, 256, 512, 1e4, dtype="bf16")
PLEN, MAX_NEW = 19990, 10


@pytest.mark.timeout(400)
def test_context_beyond_one_chunk():
    import torch
    assert torch.cuda.is_available()
    w = make_weights(SHAPE, 21)
    rng = np.random.default_rng(21)
    prompts = [rng.integers(0, SHAPE.vocab - 1, size=PLEN).astype(np.int32)]
    G, L = [2], np.array([MAX_NEW, 4], np.int32)
    print(f"long-context case: prompt {PLEN} tokens, G {G}, max_new {MAX_NEW}", flush=True)
    model = oracle_for(SHAPE, w)
    ref = oracle_rollout(model, prompts, G, MAX_NEW, 5, L, record_steps=MAX_NEW)
    pol = make_policy(SHAPE, w, max_seqs=2, max_prompts=1, max_prompt_tokens=PLEN, max_context=PLEN + MAX_NEW)
    ft = torch.from_numpy(ref["tokens"]).cuda()
    dp = prompts_to_device(prompts)
    tok, ln, lp, dump = pol.rollout(dp, G, MAX_NEW, 5, forced_len=L, force_tokens=ft, dump_steps=MAX_NEW)
    torch.cuda.synchronize()
    tok, ln, lp, dump = tok.cpu().numpy(), ln.cpu().numpy(), lp.cpu().numpy(), dump.cpu().numpy()
    np.testing.assert_array_equal(ln, L)
    worst = 0.0
    for s in range(2):
        for t in range(int(L[s])):
            worst = max(worst, float(np.max(np.abs(dump[t, s].astype(np.float64) - ref["logits"][(s, t)]))))
            if tok[s, t] != ref["tokens"][s, t]:
                assert ref["margins"][s, t] < MARGIN_TOL, (s, t)
            assert abs(float(lp[s, t]) - float(ref["logprobs"][s, t])) <= 2 * LOGIT_TOL
    print(f"worst teacher-forced logit gap {worst:.2e}", flush=True)
    assert worst <= LOGIT_TOL
    want = teacher_forced_logprobs(model, prompts, G, ref["tokens"], ref["lengths"])
    got = pol.recompute_logprobs(dp, G, ft, torch.from_numpy(ref["lengths"]).cuda()).cpu().numpy()
    valid = np.arange(MAX_NEW)[None, :] < ref["lengths"][:, None]
    assert np.all(got[~valid] == 0)
    gap = float(np.max(np.abs(got[valid] - want[valid])))
    print(f"recompute vs oracle {gap:.2e}", flush=True)
    assert gap <= 2 * LOGIT_TOL
    pol.close()
