"""GPU parity of rollout_group against the oracle.

* tiny (fp32): free-running rollouts agree token for token (up to the first
  position whose oracle top-2 margin is < 1e-2), lengths bit-exact.
* teacher forcing: the library consumes the oracle's tokens; every logit is
  within 1e-2 (max-abs) of the oracle's and every sampling decision equals the
  oracle's except at margins < 1e-2.  Shapes: tiny, a GQA bf16 decoder
  (6 query heads per kv head, head_dim 128), and a gpt2s-shaped bf16 decoder
  with ragged prompt lengths (partial KV pages) and variable G.
* shared prompt pages give bit-identical results to per-sibling copies.
* the group prefix pass (each prompt's full prefix pages attended once per
  group) agrees with the row-by-row pass within rounding and with the oracle,
  also for a group larger than one prefix workgroup's 128 query rows.
* temperatures other than 1 (0.7, 1.6): free-running and teacher-forced.
* prompt lengths at KV page boundaries (1, 15, 16, 17, 32, 33 tokens).
* a decode batch of more than 1024 rows (256 x 256 projection tiles).
* graph replay and direct launches (kernel timing) give bit-identical outputs;
  so does a non-default caller stream.
* edge cases: length-1 completions, max_new = 1, natural EOS, errors; an fp32
  model whose vocabulary is wider than every projection (its lm head runs
  through the GEMM partial buffer at the 16-row decode bucket).
"""
import numpy as np
import pytest

from oracle.rollout import rollout as oracle_rollout
from workload import get_config, make_weights, make_inputs, ModelShape
from rg_helpers import (oracle_for, make_policy, prompts_to_device, compare_free_running, check_structure,
                        MARGIN_TOL, LOGIT_TOL)

pytestmark = pytest.mark.gpu

GQA = ModelShape(2, 256, 12, 2, 128, 512, 2048, 1e6, dtype="bf16")
GPT2S = get_config("gpt2s").shape
NAT = ModelShape(2, 64, 2, 2, 32, 128, 16, 1e4, dtype="f32")   # 16-token vocab: EOS comes naturally
WIDE_V = ModelShape(1, 64, 4, 1, 32, 128, 2000, 1e4, dtype="f32")   # vocabulary wider than every projection


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available()
    return torch


def _np(x):
    return x.cpu().numpy()


def _case(shape, seed, plens, G, max_new, len_range):
    rng = np.random.default_rng(seed + 100)
    prompts = [rng.integers(0, shape.vocab - 1, size=n).astype(np.int32) for n in plens]
    N = int(np.sum(G))
    L = rng.integers(len_range[0], len_range[1] + 1, size=N).astype(np.int32)
    L[0] = len_range[0]
    L[-1] = len_range[1]
    return prompts, L


def _run_tf(torch, shape, w, prompts, G, max_new, L, seed, share=True, group_prefix=False, temperature=1.0):
    model = oracle_for(shape, w)
    ref = oracle_rollout(model, prompts, G, max_new, seed, L, record_steps=max_new, temperature=temperature)
    pol = make_policy(shape, w, max_seqs=int(np.sum(G)), max_prompts=len(G), max_prompt_tokens=int(sum(map(len, prompts))),
                      max_context=max(map(len, prompts)) + max_new)
    ft = torch.from_numpy(ref["tokens"]).cuda()
    tok, ln, lp, dump = pol.rollout(prompts_to_device(prompts), G, max_new, seed, forced_len=L, force_tokens=ft,
                                    dump_steps=max_new, share_prefix=share, group_prefix_pass=group_prefix,
                                    temperature=temperature)
    torch.cuda.synchronize()
    return ref, _np(tok), _np(ln), _np(lp), _np(dump), pol


def _check_tf(ref, tok, ln, lp, dump, L):
    np.testing.assert_array_equal(ln, L)
    worst = 0.0
    n_dec = 0
    for s in range(len(L)):
        for t in range(int(L[s])):
            z = ref["logits"][(s, t)]
            err = float(np.max(np.abs(dump[t, s].astype(np.float64) - z)))
            worst = max(worst, err)
            if tok[s, t] != ref["tokens"][s, t]:
                assert ref["margins"][s, t] < MARGIN_TOL, (s, t, ref["margins"][s, t])
            else:
                n_dec += 1
            assert abs(lp[s, t] - ref["logprobs"][s, t]) <= 2 * LOGIT_TOL
    assert worst <= LOGIT_TOL, worst
    return worst, n_dec


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tiny_free_running(torch, seed):
    wl = get_config("tiny")
    w = make_weights(wl.shape, seed)
    inp = make_inputs(wl, seed)
    ref = oracle_rollout(oracle_for(wl.shape, w), inp.prompts, inp.G, wl.max_new, seed, inp.forced_len)
    pol = make_policy(wl.shape, w, 16, 4, 64, wl.prompt_len + wl.max_new)
    tok, ln, lp = pol.rollout(prompts_to_device(inp.prompts), inp.G, wl.max_new, seed, forced_len=inp.forced_len)
    tok, ln, lp = _np(tok), _np(ln), _np(lp)
    check_structure(tok, ln, lp, wl.shape.eos_id, wl.max_new, inp.forced_len)
    checked, split = compare_free_running(tok, lp, ref, ln, lp_tol=1e-4)
    assert checked > 0


@pytest.mark.parametrize("T", [0.7, 1.6])
def test_temperature_other_than_one(torch, T):
    # at T != 1 the sampler scales the logits by 1/T (at T = 1 it takes them as
    # they are): sampling decisions and log-probabilities against the oracle
    wl = get_config("tiny")
    w = make_weights(wl.shape, 1)
    inp = make_inputs(wl, 1)
    ref = oracle_rollout(oracle_for(wl.shape, w), inp.prompts, inp.G, wl.max_new, 3, inp.forced_len, temperature=T)
    pol = make_policy(wl.shape, w, 16, 4, 64, wl.prompt_len + wl.max_new)
    tok, ln, lp = pol.rollout(prompts_to_device(inp.prompts), inp.G, wl.max_new, 3, forced_len=inp.forced_len,
                              temperature=T)
    tok, ln, lp = _np(tok), _np(ln), _np(lp)
    check_structure(tok, ln, lp, wl.shape.eos_id, wl.max_new, inp.forced_len)
    checked, _ = compare_free_running(tok, lp, ref, ln, lp_tol=1e-4)
    assert checked > 0
    wb = make_weights(GQA, 4)
    prompts, L = _case(GQA, 4, [33, 12], [5, 3], 16, (1, 16))
    ref, tok, ln, lp, dump, _ = _run_tf(torch, GQA, wb, prompts, [5, 3], 16, L, 13, temperature=T)
    _check_tf(ref, tok, ln, lp, dump, L)


def test_prompt_lengths_at_page_boundaries(torch):
    # 16-token KV pages: prompts with no full page (1, 15), exactly one or two
    # (16, 32), and one token past a boundary (17, 33), each with siblings
    # that share the full pages and copy the partial one; lengths 1..12
    from oracle.grpo import teacher_forced_logprobs
    prompts, L = _case(GQA, 8, [1, 15, 16, 17, 32, 33], [3, 2, 4, 1, 2, 3], 12, (1, 12))
    G = [3, 2, 4, 1, 2, 3]
    w = make_weights(GQA, 8)
    ref, tok, ln, lp, dump, pol = _run_tf(torch, GQA, w, prompts, G, 12, L, 31)
    _check_tf(ref, tok, ln, lp, dump, L)
    want = teacher_forced_logprobs(oracle_for(GQA, w), prompts, G, ref["tokens"], ref["lengths"])
    got = _np(pol.recompute_logprobs(prompts_to_device(prompts), G, torch.from_numpy(ref["tokens"]).cuda(),
                                     torch.from_numpy(ref["lengths"]).cuda()))
    valid = np.arange(12)[None, :] < ref["lengths"][:, None]
    assert np.all(got[~valid] == 0)
    assert float(np.max(np.abs(got[valid] - want[valid]))) <= 2 * LOGIT_TOL


def test_decode_batch_above_1024_rows(torch):
    # 100 prompts x 8..16 siblings: decode steps with more than 1024 rows run
    # every projection on 256 x 256 tiles with the decode epilogues (QKV with
    # RoPE and KV append, SwiGLU, residual + norm)
    rng = np.random.default_rng(77)
    P = 100
    G = [int(g) for g in rng.integers(8, 17, size=P)]
    prompts = [rng.integers(0, GQA.vocab - 1, size=int(n)).astype(np.int32) for n in rng.integers(1, 25, size=P)]
    N = sum(G)
    assert N > 1024
    L = rng.integers(1, 6, size=N).astype(np.int32)
    L[:1100] = 5                                     # the first steps run above 1024 rows
    w = make_weights(GQA, 9)
    ref, tok, ln, lp, dump, _ = _run_tf(torch, GQA, w, prompts, G, 5, L, 41)
    _check_tf(ref, tok, ln, lp, dump, L)


def test_graph_replay_matches_direct_launches(torch):
    # decode steps replay captured HIP graphs unless kernels are being timed;
    # timing every class, or only the attention class, launches them directly
    # with events around each launch: the outputs must be bit-identical
    w = make_weights(GQA, 12)
    prompts, L = _case(GQA, 12, [40, 7, 19], [5, 3, 4], 24, (1, 24))
    G = [5, 3, 4]
    pol = make_policy(GQA, w, max_seqs=12, max_prompts=3, max_prompt_tokens=66, max_context=64)
    dp = prompts_to_device(prompts)
    base = [_np(x) for x in pol.rollout(dp, G, 24, 17, forced_len=L)]
    for prof in (True, ["attn"]):
        got = [_np(x) for x in pol.rollout(dp, G, 24, 17, forced_len=L, profile=prof)]
        for g, b in zip(got, base):
            np.testing.assert_array_equal(g, b)
        times = pol.kernel_times(1)
        assert times["attn"][1] > 0 and times["attn"][0] > 0
        if prof is True:
            assert all(n > 0 for k, (ms, n) in times.items() if k in ("gemm_qkv", "gemm_o", "gemm_gu", "gemm_down",
                                                                       "gemm_lm", "sample"))


def test_side_stream_matches_default_stream(torch):
    # every entry point launches on the caller's stream (here torch's current
    # stream inside a side-stream context): same outputs, bit for bit
    import paper_2606_02218_amd as rg
    w = make_weights(GQA, 14)
    prompts, L = _case(GQA, 14, [21, 9], [4, 3], 16, (1, 16))
    G = [4, 3]
    pol = make_policy(GQA, w, max_seqs=7, max_prompts=2, max_prompt_tokens=30, max_context=40)
    dp = prompts_to_device(prompts)
    base = [_np(x) for x in pol.rollout(dp, G, 16, 23, forced_len=L)]
    tok0, ln0 = (torch.from_numpy(base[0]).cuda(), torch.from_numpy(base[1]).cuda())
    rec0 = _np(pol.recompute_logprobs(dp, G, tok0, ln0))
    r = torch.from_numpy(np.random.default_rng(3).random(7).astype(np.float32)).cuda()
    Gd = torch.tensor(G, dtype=torch.int32).cuda()
    adv0 = _np(rg.group_advantage(r, Gd))
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        got = pol.rollout(dp, G, 16, 23, forced_len=L)
        rec = pol.recompute_logprobs(dp, G, tok0, ln0)
        adv = rg.group_advantage(r, Gd)
    side.synchronize()
    for g, b in zip(got, base):
        np.testing.assert_array_equal(_np(g), b)
    np.testing.assert_array_equal(_np(rec), rec0)
    np.testing.assert_array_equal(_np(adv), adv0)


def test_tiny_teacher_forced(torch):
    wl = get_config("tiny")
    w = make_weights(wl.shape, 0)
    prompts, L = _case(wl.shape, 0, [16, 9, 23], [4, 3, 2], 32, (1, 32))
    ref, tok, ln, lp, dump, _ = _run_tf(torch, wl.shape, w, prompts, [4, 3, 2], 32, L, 5)
    worst, _ = _check_tf(ref, tok, ln, lp, dump, L)
    assert worst < 1e-4   # fp32 model: only accumulation-order differences


def test_fp32_vocabulary_wider_than_projections(torch):
    # fp32 models run the lm head through the GEMM partial buffer: one
    # sequence decodes in the 16-row bucket, which needs 16 x V elements
    w = make_weights(WIDE_V, 9)
    prompts, L = _case(WIDE_V, 9, [12], [1], 3, (1, 3))
    ref, tok, ln, lp, dump, _ = _run_tf(torch, WIDE_V, w, prompts, [1], 3, L, 34)
    worst, _ = _check_tf(ref, tok, ln, lp, dump, L)
    assert worst < 1e-4


def test_gqa_bf16_teacher_forced(torch):
    w = make_weights(GQA, 3)
    prompts, L = _case(GQA, 3, [40, 16, 7], [6, 1, 3], 24, (1, 24))
    ref, tok, ln, lp, dump, _ = _run_tf(torch, GQA, w, prompts, [6, 1, 3], 24, L, 11)
    _check_tf(ref, tok, ln, lp, dump, L)


def test_gpt2s_ragged_teacher_forced_and_sharing(torch):
    w = make_weights(GPT2S, 0)
    wl = get_config("gpt2s")
    base = make_inputs(wl, 0).prompts
    prompts = [base[0], base[1][:37], base[2][:100]]
    G = [8, 5, 3]
    L = np.random.default_rng(4).integers(1, 41, size=16).astype(np.int32)
    L[0], L[5] = 1, 40
    ref, tok, ln, lp, dump, pol = _run_tf(torch, GPT2S, w, prompts, G, 40, L, 1234)
    _check_tf(ref, tok, ln, lp, dump, L)
    # the same call with private copies of every prompt page is bit-identical
    ft = torch.from_numpy(ref["tokens"]).cuda()
    tok2, ln2, lp2, dump2 = pol.rollout(prompts_to_device(prompts), G, 40, 1234, forced_len=L, force_tokens=ft,
                                        dump_steps=40, share_prefix=False)
    np.testing.assert_array_equal(_np(tok2), tok)
    np.testing.assert_array_equal(_np(ln2), ln)
    np.testing.assert_array_equal(_np(lp2), lp)
    np.testing.assert_array_equal(_np(dump2), dump)
    # attending to the prefix once per group changes only the summation order
    tok4, ln4, lp4, dump4 = pol.rollout(prompts_to_device(prompts), G, 40, 1234, forced_len=L, force_tokens=ft,
                                        dump_steps=40, group_prefix_pass=True)
    _check_tf(ref, _np(tok4), _np(ln4), _np(lp4), _np(dump4), L)
    live = np.zeros(dump.shape[:2], dtype=bool)
    for s in range(len(L)):
        live[: int(L[s]), s] = True
    assert float(np.max(np.abs(_np(dump4)[live] - dump[live]))) < 2e-3
    # free-running from the same inputs follows the oracle's trajectory
    tok3, ln3, lp3 = pol.rollout(prompts_to_device(prompts), G, 40, 1234, forced_len=L)
    tok3, ln3, lp3 = _np(tok3), _np(ln3), _np(lp3)
    check_structure(tok3, ln3, lp3, GPT2S.eos_id, 40, L)
    compare_free_running(tok3, lp3, ref, ln3, lp_tol=2 * LOGIT_TOL)


def test_gqa_bf16_large_group(torch):
    # 30 siblings x 6 query heads per kv head = 180 query rows: two prefix
    # workgroups per (prompt, kv head, chunk); the second group retires early
    w = make_weights(GQA, 5)
    prompts, L = _case(GQA, 5, [70, 33], [30, 2], 12, (1, 12))
    L[30:] = [2, 3]
    ref, tok, ln, lp, dump, _ = _run_tf(torch, GQA, w, prompts, [30, 2], 12, L, 21, group_prefix=True)
    _check_tf(ref, tok, ln, lp, dump, L)


def test_natural_eos(torch):
    w = make_weights(NAT, 2)
    prompts = [np.array([1, 2, 3], np.int32), np.array([4, 5, 6, 7, 8], np.int32)]
    G = [8, 4]
    ref = oracle_rollout(oracle_for(NAT, w), prompts, G, 40, 3, None)
    pol = make_policy(NAT, w, 12, 2, 8, 48)
    tok, ln, lp = pol.rollout(prompts_to_device(prompts), G, 40, 3)
    tok, ln, lp = _np(tok), _np(ln), _np(lp)
    check_structure(tok, ln, lp, NAT.eos_id, 40)
    checked, split = compare_free_running(tok, lp, ref, ln, lp_tol=1e-4)
    if split == 0:
        np.testing.assert_array_equal(ln, ref["lengths"])
    assert checked > 20


def test_max_new_one_and_length_one(torch):
    wl = get_config("tiny")
    w = make_weights(wl.shape, 0)
    prompts = [np.arange(5, dtype=np.int32)]
    pol = make_policy(wl.shape, w, 8, 2, 32, 64)
    ref = oracle_rollout(oracle_for(wl.shape, w), prompts, [3], 1, 9, None)
    tok, ln, lp = pol.rollout(prompts_to_device(prompts), [3], 1, 9)
    np.testing.assert_array_equal(_np(ln), [1, 1, 1])
    compare_free_running(_np(tok), _np(lp), ref, _np(ln), lp_tol=1e-4)
    L = np.array([1, 1, 1], np.int32)
    tok, ln, lp = pol.rollout(prompts_to_device(prompts), [3], 10, 9, forced_len=L)
    assert np.all(_np(tok)[:, 0] == wl.shape.eos_id) and np.all(_np(tok)[:, 1:] == -1)


def test_errors(torch):
    import paper_2606_02218_amd as rg
    from paper_2606_02218_amd._lib import RG_EINVAL, RG_ENOMEM
    wl = get_config("tiny")
    w = make_weights(wl.shape, 0)
    pol = make_policy(wl.shape, w, 8, 2, 32, 48)
    p = prompts_to_device([np.arange(16, dtype=np.int32)])
    with pytest.raises(rg.RolloutError) as e:
        pol.rollout(p, [0], 8, 0)
    assert e.value.code == RG_EINVAL
    with pytest.raises(rg.RolloutError) as e:
        pol.rollout(p, [4], 8, 0, forced_len=[1, 2, 9, 3])
    assert e.value.code == RG_EINVAL
    with pytest.raises(rg.RolloutError) as e:
        pol.rollout(p, [9], 8, 0)
    assert e.value.code == RG_ENOMEM
    with pytest.raises(rg.RolloutError) as e:
        pol.rollout(p, [4], 40, 0)       # 16 + 40 > max_context
    assert e.value.code == RG_ENOMEM
    bad = prompts_to_device([np.array([1, 2, wl.shape.vocab + 5], np.int32)])
    with pytest.raises(rg.RolloutError) as e:
        pol.rollout(bad, [2], 4, 0)
    assert e.value.code == RG_EINVAL
    three = prompts_to_device([np.arange(4, dtype=np.int32)] * 3)
    with pytest.raises(rg.RolloutError) as e:        # 3 prompts > max_prompts = 2
        pol.rollout(three, [1, 1, 1], 4, 0)
    assert e.value.code == RG_ENOMEM and "max_prompts" in str(e.value)
    long2 = prompts_to_device([np.arange(20, dtype=np.int32), np.arange(20, dtype=np.int32)])
    with pytest.raises(rg.RolloutError) as e:        # 40 prompt tokens > max_prompt_tokens = 32
        pol.rollout(long2, [1, 1], 4, 0)
    assert e.value.code == RG_ENOMEM and "prompt tokens" in str(e.value)
    for T in (0.0, -1.0, float("nan"), float("inf")):
        with pytest.raises(rg.RolloutError) as e:
            pol.rollout(p, [4], 8, 0, temperature=T)
        assert e.value.code == RG_EINVAL and "temperature" in str(e.value), T
    # the policy is still usable after errors
    tok, ln, lp = pol.rollout(p, [4], 8, 0, forced_len=[8, 8, 8, 8])
    np.testing.assert_array_equal(_np(ln), [8, 8, 8, 8])


def test_kv_pool_exhaustion(torch):
    from paper_2606_02218_amd import RolloutError
    from paper_2606_02218_amd._lib import RG_ENOMEM
    wl = get_config("tiny")
    w = make_weights(wl.shape, 0)
    # 1 prompt page + 4 sibling pages fit; the second page of each sibling does not
    pol = make_policy(wl.shape, w, 4, 1, 16, 64, kv_pool_pages=5)
    p = prompts_to_device([np.arange(16, dtype=np.int32)])
    with pytest.raises(RolloutError) as e:
        pol.rollout(p, [4], 40, 0, forced_len=[40, 40, 40, 40])
    assert e.value.code == RG_ENOMEM
    tok, ln, lp = pol.rollout(p, [4], 10, 0, forced_len=[10, 3, 7, 1])
    np.testing.assert_array_equal(_np(ln), [10, 3, 7, 1])
