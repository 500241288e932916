"""Seeded random decoders within the supported shapes, against the oracle.

Each case draws a model (bf16 or fp32; head_dim 32/64/128; 1, 2 or 4 kv
heads with 1..8 query heads each; d_model, FFN and vocabulary sizes; 1..3
layers; RoPE theta 1e4 or 1e6), a batch (1..4 ragged prompts, G per prompt,
forced lengths up to max_new), a temperature (1, 0.7 or 1.3), whether the
siblings share their prompt's pages, whether bf16 decode steps take the group
prefix pass, and whether the recompute attends by row tiles or by rows, then
checks:

* the rollout teacher-forced on the oracle's tokens: every logit within 1e-2
  (bf16) / 1e-4 (fp32) of the oracle's, log-probabilities within twice that,
  sampling decisions equal except at top-2 margins below 1e-2, lengths exact;
* free-running from the same inputs follows the oracle's trajectory (tokens
  equal up to the first position whose oracle margin is below 1e-2);
* the recompute of the oracle's tokens against the oracle's teacher-forced
  log-probabilities (same tolerance), zero past each length.

The default run takes 16 small cases; RG_SWEEP_CASES=N sets the count and
RG_SWEEP_BIG=1 draws larger models and batches (d_model up to 1536, FFN up to
6144, vocabularies up to 32000, prompts up to 600 tokens, up to 16 siblings);
RG_SWEEP_LONG=1 draws small models with prompts of 300..2500 tokens, so decode
rows are cut into many context chunks and merged.
"""
import os

import numpy as np
import pytest

from oracle.grpo import teacher_forced_logprobs
from oracle.rollout import rollout as oracle_rollout
from workload import ModelShape, make_weights
from rg_helpers import oracle_for, make_policy, prompts_to_device, compare_free_running, check_structure, MARGIN_TOL

pytestmark = pytest.mark.gpu

BIG = os.environ.get("RG_SWEEP_BIG") == "1"
LONG = os.environ.get("RG_SWEEP_LONG") == "1"
N_CASES = int(os.environ.get("RG_SWEEP_CASES", "16"))


def draw_case(i):
    r = np.random.default_rng((9000 if LONG else (7000 if BIG else 1000)) + i)
    bf = r.random() < 0.8
    hd = int(r.choice([64, 128])) if bf else int(r.choice([32, 64, 128]))
    nkv = int(r.choice([1, 2, 4]))
    rep = int(r.integers(1, 9))
    nq = nkv * rep
    if (nq * hd) % 64:
        nq = nkv * (rep + 1)
    d = 64 * int(r.integers(2, 25 if BIG else 9))
    ffn = 64 * int(r.integers(2, 97 if BIG else 13))
    V = 16 * int(r.integers(32, 2001 if BIG else 257))
    L = int(r.integers(1, 3 if (BIG or LONG) else 4))
    theta = float(r.choice([1e4, 1e6]))
    shape = ModelShape(L, d, nq, nkv, hd, ffn, V, theta, dtype="bf16" if bf else "f32")
    P = int(r.integers(1, 5))
    plens = [int(r.integers(300, 2501) if LONG else r.integers(1, 601 if BIG else 81)) for _ in range(P)]
    G = [int(r.integers(1, 17 if BIG else (4 if LONG else 7))) for _ in range(P)]
    max_new = int(r.integers(1, 49 if BIG else 25))
    lengths = r.integers(1, max_new + 1, size=sum(G)).astype(np.int32)
    prompts = [r.integers(0, V - 1, size=n).astype(np.int32) for n in plens]
    T = float(r.choice([1.0, 0.7, 1.3]))
    share = bool(r.random() < 0.8)
    modes = dict(group_prefix=bool(r.random() < 0.3), row_tiles=bool(r.random() < 0.7))
    return shape, prompts, G, max_new, lengths, T, share, modes


@pytest.mark.timeout(300)
@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape_against_oracle(i):
    import torch
    assert torch.cuda.is_available()
    shape, prompts, G, max_new, L, T, share, modes = draw_case(i)
    print(f"random case {i}: {shape}, prompts {[len(p) for p in prompts]}, G {G}, max_new {max_new}, T {T}, "
          f"shared pages {share}, {modes}", flush=True)
    w = make_weights(shape, 5000 + i)
    model = oracle_for(shape, w)
    ref = oracle_rollout(model, prompts, G, max_new, 77 + i, L, record_steps=max_new, temperature=T)
    pol = make_policy(shape, w, max_seqs=sum(G), max_prompts=len(G), max_prompt_tokens=sum(len(p) for p in prompts),
                      max_context=max(len(p) for p in prompts) + max_new)
    ft = torch.from_numpy(ref["tokens"]).cuda()
    dp = prompts_to_device(prompts)
    tok, ln, lp, dump = pol.rollout(dp, G, max_new, 77 + i, forced_len=L, force_tokens=ft, dump_steps=max_new,
                                    temperature=T, share_prefix=share, group_prefix_pass=modes["group_prefix"])
    torch.cuda.synchronize()
    tok, ln, lp, dump = tok.cpu().numpy(), ln.cpu().numpy(), lp.cpu().numpy(), dump.cpu().numpy()
    tol = 1e-2 if shape.dtype == "bf16" else 1e-4
    np.testing.assert_array_equal(ln, L)
    for s in range(len(L)):
        for t in range(int(L[s])):
            gap = float(np.max(np.abs(dump[t, s].astype(np.float64) - ref["logits"][(s, t)])))
            assert gap <= tol, (s, t, gap)
            assert abs(float(lp[s, t]) - float(ref["logprobs"][s, t])) <= 2 * tol, (s, t)
            if tok[s, t] != ref["tokens"][s, t]:
                assert ref["margins"][s, t] < MARGIN_TOL, (s, t, ref["margins"][s, t])
    tok2, ln2, lp2 = pol.rollout(dp, G, max_new, 77 + i, forced_len=L, temperature=T, share_prefix=share,
                                 group_prefix_pass=modes["group_prefix"])
    tok2, ln2, lp2 = tok2.cpu().numpy(), ln2.cpu().numpy(), lp2.cpu().numpy()
    check_structure(tok2, ln2, lp2, shape.eos_id, max_new, L)
    compare_free_running(tok2, lp2, ref, ln2, lp_tol=2 * tol)
    want = teacher_forced_logprobs(model, prompts, G, ref["tokens"], ref["lengths"], T)
    got = pol.recompute_logprobs(dp, G, ft, torch.from_numpy(ref["lengths"]).cuda(), temperature=T,
                                 share_prefix=share, row_tiles=modes["row_tiles"]).cpu().numpy()
    valid = np.arange(max_new)[None, :] < ref["lengths"][:, None]
    assert np.all(got[~valid] == 0)
    assert float(np.max(np.abs(got[valid] - want[valid]))) <= 2 * tol
    pol.close()
