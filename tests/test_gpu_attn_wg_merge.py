"""Decode attention whose context chunks are merged by the attention kernel's
own waves (one workgroup per (row, kv head), no merge launch).  That variant
runs for bf16 models when a step has at least 256 (row, kv head) pairs and
each row's context takes 2..8 chunks, so these cases use 128 and 256 rows at
the 1.5B head geometry (12 query / 2 kv heads, head_dim 128) with prompts long
enough for 2-3 chunks.  As rows retire the steps fall to buckets below 256
pairs, which take the per-chunk grid plus the merge launch, so one rollout
covers both.  The rollout is teacher-forced on the oracle's tokens: every
logit within 1e-2, log-probabilities within 2e-2, sampling decisions equal
except at top-2 margins below 1e-2, lengths exact.
"""
import numpy as np
import pytest

from oracle.rollout import rollout as oracle_rollout
from workload import ModelShape, make_weights
from rg_helpers import oracle_for, make_policy, prompts_to_device, MARGIN_TOL, LOGIT_TOL

pytestmark = pytest.mark.gpu

SHAPE = ModelShape(2, 1536, 12, 2, 128, 2048, 4096, 1e6, dtype="bf16")
MAX_NEW = 4
# (prompts, siblings per prompt, shortest and longest prompt)
CASES = {"rows128": (8, 16, 560, 700), "rows256": (16, 16, 300, 420)}


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", sorted(CASES))
def test_attention_merged_in_kernel(name):
    import torch
    import paper_2606_02218_amd as rg
    assert torch.cuda.is_available()
    P, g, lo, hi = CASES[name]
    G = [g] * P
    N = P * g
    rng = np.random.default_rng(77 + N)
    plens = rng.integers(lo, hi + 1, size=P)
    prompts = [rng.integers(0, SHAPE.vocab - 1, size=int(n)).astype(np.int32) for n in plens]
    lengths = rng.integers(1, MAX_NEW + 1, size=N).astype(np.int32)
    lengths[::5] = MAX_NEW
    ctx = int(plens.max()) + MAX_NEW
    chunks = rg.decode_attention_chunks(N, SHAPE.n_kv_heads, ctx)
    # the first decode steps take the in-kernel merge
    assert N * SHAPE.n_kv_heads >= 256 and 2 <= chunks <= 8, chunks
    print(f"in-kernel merge case {name}: {N} rows, prompts {lo}..{hi}, {chunks} chunks", flush=True)
    w = make_weights(SHAPE, 41)
    ref = oracle_rollout(oracle_for(SHAPE, w), prompts, G, MAX_NEW, 13, lengths, record_steps=MAX_NEW)
    pol = make_policy(SHAPE, w, max_seqs=N, max_prompts=P, max_prompt_tokens=int(plens.sum()), max_context=ctx)
    ft = torch.from_numpy(ref["tokens"]).cuda()
    tok, ln, lp, dump = pol.rollout(prompts_to_device(prompts), G, MAX_NEW, 13, forced_len=lengths,
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
