"""Decode attention at the 1.5B head geometry (12 query / 2 kv heads,
head_dim 128: six query heads per kv head) with contexts long enough that
every decode row's context is cut into several chunks whose partial softmax
results are merged -- the path most decode steps of the 1.5B workload take
once fewer than about 257 rows remain.  Two prompts of 1,700 and 2,300
tokens with 3 and 2 siblings; against the oracle:

* the rollout teacher-forced on the oracle's tokens: every logit within
  1e-2, log-probabilities within 2e-2, sampling decisions equal except at
  top-2 margins below 1e-2, lengths exact; once with the row pass alone and
  once with the group prefix pass (shared prefix pages scored once per
  group, then merged with the rows' own chunks);
* the recompute of the oracle's tokens against the oracle's teacher-forced
  log-probabilities (within 2e-2).
"""
import numpy as np
import pytest

from oracle.grpo import teacher_forced_logprobs
from oracle.rollout import rollout as oracle_rollout
from workload import ModelShape, make_weights
from rg_helpers import oracle_for, make_policy, prompts_to_device, MARGIN_TOL, LOGIT_TOL

pytestmark = pytest.mark.gpu

SHAPE = ModelShape(2, 1536, 12, 2, 128, 2048, 4096, 1e6, dtype="bf16")
PLENS, G, MAX_NEW = (1700, 2300), [3, 2], 10
LENGTHS = np.array([10, 4, 7, 10, 1], np.int32)


@pytest.fixture(scope="module")
def case():
    w = make_weights(SHAPE, 31)
    rng = np.random.default_rng(31)
    prompts = [rng.integers(0, SHAPE.vocab - 1, size=n).astype(np.int32) for n in PLENS]
    model = oracle_for(SHAPE, w)
    ref = oracle_rollout(model, prompts, G, MAX_NEW, 9, LENGTHS, record_steps=MAX_NEW)
    return w, prompts, model, ref


@pytest.mark.timeout(300)
@pytest.mark.parametrize("group_prefix", [False, True])
def test_gqa_multichunk_teacher_forced(case, group_prefix):
    import torch
    import paper_2606_02218_amd as rg
    assert torch.cuda.is_available()
    w, prompts, model, ref = case
    # every decode step of this rollout runs in the 16-row bucket: each row's
    # context is cut into several chunks and merged
    assert rg.decode_attention_chunks(sum(G), SHAPE.n_kv_heads, max(PLENS) + MAX_NEW) >= 3
    print(f"hd-128 GQA multi-chunk case: prompts {PLENS}, G {G}, group prefix pass {group_prefix}", flush=True)
    pol = make_policy(SHAPE, w, max_seqs=sum(G), max_prompts=len(G), max_prompt_tokens=sum(PLENS),
                      max_context=max(PLENS) + MAX_NEW)
    ft = torch.from_numpy(ref["tokens"]).cuda()
    dp = prompts_to_device(prompts)
    tok, ln, lp, dump = pol.rollout(dp, G, MAX_NEW, 9, forced_len=LENGTHS, force_tokens=ft, dump_steps=MAX_NEW,
                                    group_prefix_pass=group_prefix)
    torch.cuda.synchronize()
    tok, ln, lp, dump = tok.cpu().numpy(), ln.cpu().numpy(), lp.cpu().numpy(), dump.cpu().numpy()
    np.testing.assert_array_equal(ln, LENGTHS)
    worst = 0.0
    for s in range(len(LENGTHS)):
        for t in range(int(LENGTHS[s])):
            worst = max(worst, float(np.max(np.abs(dump[t, s].astype(np.float64) - ref["logits"][(s, t)]))))
            assert abs(float(lp[s, t]) - float(ref["logprobs"][s, t])) <= 2 * LOGIT_TOL, (s, t)
            if tok[s, t] != ref["tokens"][s, t]:
                assert ref["margins"][s, t] < MARGIN_TOL, (s, t, ref["margins"][s, t])
    print(f"worst teacher-forced logit gap {worst:.2e}", flush=True)
    assert worst <= LOGIT_TOL
    pol.close()


@pytest.mark.timeout(300)
def test_gqa_multichunk_recompute(case):
    import torch
    w, prompts, model, ref = case
    pol = make_policy(SHAPE, w, max_seqs=sum(G), max_prompts=len(G), max_prompt_tokens=sum(PLENS),
                      max_context=max(PLENS) + MAX_NEW)
    want = teacher_forced_logprobs(model, prompts, G, ref["tokens"], ref["lengths"])
    got = pol.recompute_logprobs(prompts_to_device(prompts), G, torch.from_numpy(ref["tokens"]).cuda(),
                                 torch.from_numpy(ref["lengths"]).cuda()).cpu().numpy()
    valid = np.arange(MAX_NEW)[None, :] < ref["lengths"][:, None]
    assert np.all(got[~valid] == 0)
    gap = float(np.max(np.abs(got[valid] - want[valid])))
    print(f"recompute vs oracle {gap:.2e}", flush=True)
    assert gap <= 2 * LOGIT_TOL
    pol.close()
