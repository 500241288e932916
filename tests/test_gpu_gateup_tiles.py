"""Gate/up projections as wide as the 1.5B one (2 x FFN >= 8192 columns) at
33-64 decode rows run on 32 x 64 tiles instead of 32 x 128.  A bf16 model with
FFN 4096 (gate/up 8192 columns, d_model 256, 4 query / 2 kv heads of 64) and
48 sequences (3 prompts x G = 16) puts its first decode steps in the 64-row
bucket on those tiles; as rows retire the later steps fall to the 32-row
bucket and the 128-column tiles.  Teacher-forced on the oracle's tokens: every
logit within 1e-2, log-probabilities within 2e-2, sampling decisions equal
except at top-2 margins below 1e-2, lengths exact.
"""
import numpy as np
import pytest

from oracle.rollout import rollout as oracle_rollout
from workload import ModelShape, make_weights
from rg_helpers import oracle_for, make_policy, prompts_to_device, MARGIN_TOL, LOGIT_TOL

pytestmark = pytest.mark.gpu

SHAPE = ModelShape(2, 256, 4, 2, 64, 4096, 2048, 1e4, dtype="bf16")
P, G, MAX_NEW = 3, 16, 8


@pytest.mark.timeout(300)
def test_gateup_64_column_tiles_teacher_forced():
    import torch
    assert torch.cuda.is_available()
    N = P * G
    rng = np.random.default_rng(2024)
    plens = rng.integers(30, 60, size=P)
    prompts = [rng.integers(0, SHAPE.vocab - 1, size=int(n)).astype(np.int32) for n in plens]
    lengths = rng.integers(1, MAX_NEW + 1, size=N).astype(np.int32)
    lengths[::3] = MAX_NEW
    assert 32 < N <= 64 and 2 * SHAPE.ffn_dim >= 8192
    print(f"gate/up tile case: {N} rows, FFN {SHAPE.ffn_dim}, prompts {list(plens)}", flush=True)
    w = make_weights(SHAPE, 5)
    ref = oracle_rollout(oracle_for(SHAPE, w), prompts, [G] * P, MAX_NEW, 21, lengths, record_steps=MAX_NEW)
    pol = make_policy(SHAPE, w, max_seqs=N, max_prompts=P, max_prompt_tokens=int(plens.sum()),
                      max_context=int(plens.max()) + MAX_NEW)
    ft = torch.from_numpy(ref["tokens"]).cuda()
    tok, ln, lp, dump = pol.rollout(prompts_to_device(prompts), [G] * P, MAX_NEW, 21, forced_len=lengths,
                                    force_tokens=ft, dump_steps=MAX_NEW)
    torch.cuda.synchronize()
    tok, ln, lp, dump = tok.cpu().numpy(), ln.cpu().numpy(), lp.cpu().numpy(), dump.cpu().numpy()
    np.testing.assert_array_equal(ln, lengths)
    worst = 0.0
    for s in range(N):
        for t in range(int(lengths[s])):
            worst = max(worst, float(np.max(np.abs(dump[t, s].astype(np.float64) - ref["logits"][(s, t)]))))
            assert abs(float(lp[s, t]) - float(ref["logprobs"][s, t])) <= 2 * LOGIT_TOL, (s, t)
            if tok[s, t] != ref["tokens"][s, t]:
                assert ref["margins"][s, t] < MARGIN_TOL, (s, t, ref["margins"][s, t])
    print(f"worst teacher-forced logit gap {worst:.2e}", flush=True)
    assert worst <= LOGIT_TOL
    pol.close()
