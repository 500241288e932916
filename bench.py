"""Group-step benchmark of the rollout hot path on one MI355X.

One step = rollout_group (prefill, fork, decode until every sequence retires)
+ group_advantage over one batch of the 1.5B-shaped workload: 32 prompts x
G = 16 siblings, 512-token prompts, max_new 4096, forced lognormal(ln 1200, 0.8)
lengths, bf16 random-init weights.  Inputs are resident in HBM before timing.
Prints one JSON line (see the keys below).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12            # MI355X HBM3E, bytes/s
MFMA_BF16_PEAK = 2.5e15      # dense bf16 MFMA, flop/s
FP32_VALU_PEAK = 157.3e12    # fp32 vector FMA (256 CUs x 4 SIMDs x 16 lanes x 2 flop x 2 packed x 2.4 GHz)


def algorithmic_bytes(shape, hist_active, hist_groups, hist_ctx, plen):
    """Per decode step t >= 1 (rows A_t, groups g_t), the bytes the method must
    move, split by kernel class.  Weights once per step; KV: each active
    group's prompt prefix once plus each row's own t generated tokens;
    activations in/out of every projection (fp32)."""
    L, d, F, V = shape.n_layers, shape.d_model, shape.ffn_dim, shape.vocab
    wb = shape.elem_bytes
    kvb = shape.elem_bytes
    qd, kvd = shape.q_dim, shape.kv_dim
    kv_tok_layer = 2 * kvd * kvb
    out = {"gemm_qkv": 0.0, "gemm_o": 0.0, "gemm_gu": 0.0, "gemm_down": 0.0, "gemm_lm": 0.0, "attn": 0.0}
    launches = {k: 0 for k in out}
    for t in range(1, len(hist_active)):
        M = int(hist_active[t])
        if M == 0:
            break
        g = int(hist_groups[t])
        prefix = float(hist_ctx[t]) / M * g if M else 0.0      # sum over active groups of Lp (uniform Lp here)
        ctx_tokens = prefix + M * t                              # prefix once per group + own tokens
        out["gemm_qkv"] += L * ((qd + 2 * kvd) * d * wb + M * d * 4 + M * (qd + 2 * kvd) * 4)
        out["gemm_o"] += L * (d * qd * wb + M * qd * 4 + M * d * 4)
        out["gemm_gu"] += L * (2 * F * d * wb + M * d * 4 + M * 2 * F * 4)
        out["gemm_down"] += L * (d * F * wb + M * F * 4 + M * d * 4)
        out["gemm_lm"] += V * d * wb + M * d * 4 + M * V * 4
        out["attn"] += L * (ctx_tokens * kv_tok_layer + M * qd * 4 * 2)
        for k in ("gemm_qkv", "gemm_o", "gemm_gu", "gemm_down", "attn"):
            launches[k] += L
        launches["gemm_lm"] += 1
    return out, launches


def decode_bytes_total(shape, hist_active, hist_groups, hist_ctx):
    """Whole-step decode bytes: weights + KV read + per-row write."""
    W = shape.decode_weight_bytes()
    kv_tok = shape.kv_bytes_per_token()
    tot = 0.0
    for t in range(1, len(hist_active)):
        M = int(hist_active[t])
        if M == 0:
            break
        g = int(hist_groups[t])
        prefix = float(hist_ctx[t]) / M * g
        tot += W + kv_tok * (prefix + M * t) + M * (kv_tok + shape.d_model * shape.elem_bytes + 8)
    return tot


def prefill_flops(shape, plens):
    """Algorithmic flops of the prefill (one multiply-add = 2 flops): every
    prompt token through every layer's matrices, causal attention (QK^T and
    PV: query i of a prompt scores i + 1 positions), and the lm head at each
    prompt's last position."""
    L, d, V, hd, nq = shape.n_layers, shape.d_model, shape.vocab, shape.head_dim, shape.n_q_heads
    n = np.asarray(plens, np.float64)
    return (2.0 * L * shape.matrix_params_per_layer() * n.sum() + 2.0 * L * nq * hd * float(np.sum(n * (n + 1)))
            + 2.0 * V * d * len(n))


def _oracle_threads() -> int:
    threads = None
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        threads = max([i.get("num_threads", 0) for i in info] or [0]) or None
    except Exception:
        pass
    if threads is None:
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return int(threads)


def cpu_baseline(wl, weights, inputs, n_steps, prompts=(0,), progress=0):
    """The oracle on the host: prefill of the given prompts plus their
    siblings for n_steps decode steps (n_steps None: to the end; prompts None:
    every prompt of the workload)."""
    from oracle.model import OracleModel
    from oracle.rollout import rollout as oracle_rollout
    threads = _oracle_threads()
    model = OracleModel(wl.shape, weights)
    t0 = time.perf_counter()
    def on_step(p, t, n):
        if progress and t % progress == 0:
            print(f"# oracle prompt {p} step {t}: {n} sequences decoding", file=sys.stderr, flush=True)

    out = oracle_rollout(model, inputs.prompts, inputs.G, wl.max_new, 1234, inputs.forced_len,
                         max_steps=n_steps, prompt_subset=None if prompts is None else list(prompts),
                         on_step=on_step)
    dt = time.perf_counter() - t0
    G = np.asarray(inputs.G, np.int64)
    off = np.concatenate([[0], np.cumsum(G)])
    sel = range(len(G)) if prompts is None else prompts
    gen = int(sum(np.sum(out["tokens"][off[p]:off[p + 1]] >= 0) for p in sel))
    n_seq = int(sum(G[p] for p in sel))
    what = "every prompt" if prompts is None else ("prompt " + ", ".join(str(p) for p in sel))
    steps = "to the end" if n_steps is None else f"x {n_steps} decode steps"
    return {"value": gen / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{what} of the {wl.name} workload: prefill ({wl.prompt_len}-token prompts) + {n_seq} sequences "
                      f"{steps} ({gen} tokens) in {dt:.1f} s, float64 numpy"}


def cpu_report(args):
    """The oracle alone (no GPU): the full workload (--cpu-steps 0) or its
    first --cpu-steps decode steps of prompt 0, optionally on one thread.
    Prints one JSON line."""
    from workload import get_config, make_weights, make_inputs
    wl = get_config(args.workload)
    weights = make_weights(wl.shape, 0)
    inp = make_inputs(wl, 0)
    full = args.cpu_steps == 0
    if args.cpu_threads:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=args.cpu_threads):
            r = cpu_baseline(wl, weights, inp, None if full else args.cpu_steps, None if full else (0,), progress=16)
    else:
        r = cpu_baseline(wl, weights, inp, None if full else args.cpu_steps, None if full else (0,), progress=16)
    r["workload"] = wl.name
    print(json.dumps(r), flush=True)


def eb_sweep(args):
    """Static G in {4, 8, 16} against the group-size controller at a fixed
    effective batch of 64 sequences (B = 64 / G prompts per step), on the
    1.5B-shaped policy.  Every training step is one rollout_group plus
    group_advantage with fresh synthetic prompts, forced hierarchical-lognormal
    lengths whose within-group spread narrows from 0.25 to 0.10 over the T
    steps (the same schedule for every arm), and the per-group length
    statistics computed on the GPU.  Prints one JSON line."""
    import torch
    import paper_2606_02218_amd as rg
    from workload import get_config, make_weights, make_inputs, step_group_lengths, step_rewards

    T, EB, sizes = args.eb_sweep, 64, (4, 8, 16)
    wl = get_config(args.workload)
    shape = wl.shape
    pol = rg.Policy(shape, make_weights(shape, 0), max_seqs=EB, max_prompts=EB // min(sizes),
                    max_prompt_tokens=EB // min(sizes) * wl.prompt_len, max_context=wl.prompt_len + wl.max_new)
    pool = make_inputs(wl, 0).prompts
    dev = torch.device("cuda")
    out_tok = torch.empty((EB, wl.max_new), dtype=torch.int32, device=dev)
    out_len = torch.empty(EB, dtype=torch.int32, device=dev)
    out_lp = torch.empty((EB, wl.max_new), dtype=torch.float32, device=dev)
    adv = torch.empty(EB, dtype=torch.float32, device=dev)

    def train_step(t, G, ctl):
        B = EB // G
        sig = 0.25 + (0.10 - 0.25) * t / max(1, T - 1)
        L = step_group_lengths(B, G, wl.max_new, 0, t, sig)
        prompts = torch.from_numpy(pool[[(t * B + i) % len(pool) for i in range(B)]]).to(dev)
        G_dev = torch.full((B,), G, dtype=torch.int32, device=dev)
        rew = torch.from_numpy(step_rewards(B * G, 0, t)).to(dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pol.rollout(prompts, [G] * B, wl.max_new, 5000 + t, forced_len=L,
                    out=(out_tok[:B * G], out_len[:B * G], out_lp[:B * G]))
        rg.group_advantage(rew, G_dev, 1e-6, 1, out=adv[:B * G])
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        stats = ctl.group_stats(out_len[:B * G], G_dev).cpu().numpy()
        return dt, stats, int(L.sum()), int(L.max())

    warm = rg.Sagc(sizes=sizes)
    train_step(0, 16, warm)                    # untimed: first-use set-up
    arms = {}
    for name in ("static-4", "static-8", "static-16", "sagc"):
        ctl = rg.Sagc(sizes=sizes, seed=11)
        G = int(name.split("-")[1]) if name != "sagc" else ctl.G
        rec = {"G": [], "step_s": [], "straggler_rate": [], "tokens": 0, "max_len": []}
        for t in range(T):
            dt, stats, ntok, lmax = train_step(t, G, ctl)
            rec["G"].append(G)
            rec["step_s"].append(round(dt, 3))
            rec["straggler_rate"].append(float(stats[:, 3].mean()))
            rec["max_len"].append(lmax)
            rec["tokens"] += ntok
            if name == "sagc":
                G = ctl.step(stats)
            print(f"# {name} step {t}: G={rec['G'][-1]} {dt:.2f} s, straggler rate {rec['straggler_rate'][-1]:.2f}",
                  file=sys.stderr, flush=True)
        tot = sum(rec["step_s"])
        rec.update({"mean_step_s": round(tot / T, 3), "tokens_per_s": round(rec["tokens"] / tot, 1),
                    "straggler_pct": round(100 * float(np.mean(rec["straggler_rate"])), 1),
                    "s_per_prompt": round(tot / sum(EB // g for g in rec["G"]), 4)})
        if name == "sagc":
            rec["controller"] = ctl.snapshot()
        arms[name] = rec
    print(json.dumps({"sweep": "static G vs group-size controller at EB = 64", "workload": wl.name,
                      "steps_per_arm": T, "effective_batch": EB, "sizes": list(sizes), "arms": arms}), flush=True)


def rows_sweep(args):
    """Decode-step time at fixed small batches: rollouts of N = 16, 32, 64 and
    128 sequences (groups of 16 on the workload's first prompts), every
    completion forced to L tokens, so every decode step runs at N rows with
    contexts from the prompt length to prompt length + L.  Best of two timed
    rollouts after one untimed one; the decode time is the library's own
    device-timeline phase.  Prints one JSON line."""
    import torch
    import paper_2606_02218_amd as rg
    from workload import get_config, make_weights, make_inputs

    L = args.rows_sweep
    wl = get_config(args.workload)
    shape = wl.shape
    inp = make_inputs(wl, 0)
    G, sizes = 16, (16, 32, 64, 128)
    P_max = max(sizes) // G
    if P_max > wl.n_prompts:
        raise SystemExit(f"--rows-sweep needs {P_max} prompts; {wl.name} has {wl.n_prompts}")
    pol = rg.Policy(shape, make_weights(shape, 0), max_seqs=max(sizes), max_prompts=P_max,
                    max_prompt_tokens=P_max * wl.prompt_len, max_context=wl.prompt_len + L)
    dev = torch.device("cuda")
    res = {}
    for N in sizes:
        P = N // G
        prompts = torch.from_numpy(inp.prompts[:P]).to(dev)
        fl = np.full(N, L, dtype=np.int32)
        out = (torch.empty((N, L), dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.int32, device=dev),
               torch.empty((N, L), dtype=torch.float32, device=dev))
        pol.rollout(prompts, [G] * P, L, 7, forced_len=fl, out=out)
        best = None
        for r in range(2):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            pol.rollout(prompts, [G] * P, L, 8 + r, forced_len=fl, out=out)
            torch.cuda.synchronize()
            wall = time.perf_counter() - t0
            pf, dc = pol.phase_times()
            if best is None or dc < best[2]:
                best = (wall, pf, dc)
        wall, pf, dc = best
        res[str(N)] = {"decode_ms": round(dc, 1), "ms_per_step": round(dc / (L - 1), 4), "prefill_ms": round(pf, 2),
                       "wall_s": round(wall, 3)}
        print(f"# {N} rows: {dc / (L - 1):.3f} ms per decode step", file=sys.stderr, flush=True)
    print(json.dumps({"rows_sweep": wl.name, "forced_len": L, "decode_steps": L - 1, "prompt_len": wl.prompt_len,
                      "rows": res}), flush=True)


def launch_floor(n_kernels):
    """Replay cost per kernel of a captured graph of n_kernels dependent tiny
    elementwise kernels (torch's in-place add on 256 floats): the floor that a
    decode step's own kernels sit above.  Prints one JSON line."""
    import torch
    x = torch.zeros(256, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for _ in range(3):
            x.add_(1.0)
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(n_kernels):
            x.add_(1.0)
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    R = 50
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(R):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / R
    expect = float(3 + (3 + R) * n_kernels)
    print(json.dumps({"launch_floor_kernels": n_kernels, "us_per_replay": round(us, 1),
                      "us_per_kernel": round(us / n_kernels, 3), "check": float(x[0].item()) == expect}), flush=True)


def loss_forward_flops(shape, G, plen, lengths):
    """Algorithmic flops (one bf16 product per multiply-add pair) of the
    teacher-forced completion rows, per kernel class: R = sum(L - 1) rows
    through every projection, the lm head over the R rows, and causal
    attention of each row over its context (QK^T and PV)."""
    L, d, F, V = shape.n_layers, shape.d_model, shape.ffn_dim, shape.vocab
    qd, kvd, hd, nq = shape.q_dim, shape.kv_dim, shape.head_dim, shape.n_q_heads
    Ls = np.asarray(lengths, np.int64)
    R = int(np.sum(Ls - 1))
    # context of the row feeding y_t is plen + t + 1 positions, t = 0 .. L - 2
    ctx = int(np.sum((Ls - 1) * (plen + 1) + (Ls - 1) * (Ls - 2) // 2))
    return R, {"gemm_qkv": 2.0 * L * R * (qd + 2 * kvd) * d, "gemm_o": 2.0 * L * R * d * qd,
               "gemm_gu": 2.0 * L * R * 2 * F * d, "gemm_down": 2.0 * L * R * d * F, "gemm_lm": 2.0 * R * V * d,
               "attn": 4.0 * L * nq * hd * ctx}


def loss_forward(args):
    """GRPO loss forward on the rollout of the same workload: one step =
    recompute_logprobs (teacher-forced log-probabilities of every completion
    token) + grpo_surrogate against a drifted copy of the rollout's
    logprobs.  Also checks, at full size, that the recompute reproduces the
    rollout's own logprobs.  Prints one JSON line."""
    import torch
    import paper_2606_02218_amd as rg
    from workload import get_config, make_weights, make_inputs, drifted_logprobs

    wl = get_config(args.workload)
    shape = wl.shape
    inp = make_inputs(wl, 0)
    N = inp.n_seq
    pol = rg.Policy(shape, make_weights(shape, 0), max_seqs=N, max_prompts=wl.n_prompts,
                    max_prompt_tokens=wl.n_prompts * wl.prompt_len, max_context=wl.prompt_len + wl.max_new)
    dev = torch.device("cuda")
    prompts = torch.from_numpy(inp.prompts).to(dev)
    G_dev = torch.from_numpy(inp.G).to(dev)
    rewards = torch.from_numpy(inp.rewards).to(dev)
    tokens, lengths, lp_roll = pol.rollout(prompts, inp.G, wl.max_new, 1234, forced_len=inp.forced_len)
    adv = torch.empty(N, dtype=torch.float32, device=dev)
    ln_np = lengths.cpu().numpy()
    old = torch.from_numpy(drifted_logprobs(lp_roll.cpu().numpy(), ln_np, 0, 0.1)).to(dev)
    new = torch.empty_like(lp_roll)
    print("# rollout done", file=sys.stderr, flush=True)

    def step(prof):
        # advantage and zero-variance filter of the group rewards, then the loss forward
        rg.group_advantage(rewards, G_dev, 1e-6, 1, out=adv)
        keep, _, _ = rg.group_filter(rewards, G_dev)
        pol.recompute_logprobs(prompts, inp.G, tokens, lengths, profile=prof, out=new)
        return rg.grpo_surrogate(new, old, adv, lengths, G_dev, 0.2, 0.28, "token", keep)

    breakdown = {}
    for i in range(args.warmup):
        step(i == 0)
        if i == 0:
            breakdown = {ph: pol.kernel_times(ph) for ph in (0, 1)}
        print(f"# warmup step {i} done", file=sys.stderr, flush=True)
    valid = np.arange(wl.max_new)[None, :] < ln_np[:, None]
    dev_max = float(np.max(np.abs(new.cpu().numpy()[valid] - lp_roll.cpu().numpy()[valid])))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        out = step(False)
        print(f"# timed step {i} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    loss = out.cpu().numpy()
    scored = int(ln_np.sum())
    ms = dt / args.steps * 1e3
    keep, _, _ = rg.group_filter(rewards, G_dev)

    def per_call_us(fn, reps=200):
        # back-to-back calls on torch's current stream, which the library launches on
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        e1.synchronize()
        return round(e0.elapsed_time(e1) * 1e3 / reps, 2)

    small = {"group_advantage": per_call_us(lambda: rg.group_advantage(rewards, G_dev, 1e-6, 1, out=adv)),
             "group_filter": per_call_us(lambda: rg.group_filter(rewards, G_dev)),
             "grpo_surrogate": per_call_us(lambda: rg.grpo_surrogate(new, old, adv, lengths, G_dev, 0.2, 0.28,
                                                                     "token", keep))}
    res = {"metric": "GRPO loss-forward scored tokens/s (group_advantage + group_filter + recompute_logprobs + "
                     "grpo_surrogate)",
           "value": round(scored / (ms / 1e3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(ms, 2), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": wl.name, "prompts": wl.n_prompts, "sequences": N, "prompt_len": wl.prompt_len,
                      "scored_tokens": scored},
           "surrogate": {"loss": float(loss[0]), "clip_frac": float(loss[1]), "tokens": int(loss[2]),
                         "sequences": int(loss[3])},
           "recompute_vs_rollout_logprob_max_abs": round(dev_max, 5),
           "small_calls_us": small}
    if breakdown:
        res["kernel_ms_breakdown"] = {f"{'prefill' if ph == 0 else 'rows'}.{k}": round(v[0], 1)
                                      for ph in (0, 1) for k, v in sorted(breakdown[ph].items(), key=lambda kv: -kv[1][0])
                                      if v[1]}
        R, flops = loss_forward_flops(shape, inp.G, wl.prompt_len, ln_np)
        rows = breakdown[1]
        dom = max((k for k in flops if rows[k][1]), key=lambda k: rows[k][0])
        ms_tot, n = rows[dom]
        achieved = flops[dom] / (ms_tot / 1e3)
        res["roofline"] = {"kernel": dom, "bound": "mfma", "achieved": round(achieved / 1e12, 1),
                           "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK, 4),
                           "traffic": None, "avg_launch_us": round(ms_tot / n * 1e3, 2),
                           "alg_flops_per_launch": round(flops[dom] / n), "launches": n,
                           "timing": "HIP events around each launch, untimed warmup step"}
        res["rows_tflops_by_class"] = {k: round(flops[k] / (rows[k][0] / 1e3) / 1e12, 1) for k in flops if rows[k][1]}
    print(json.dumps(res), flush=True)


# HBM traffic of the roofline kernel comes from rocprofv3 counter passes that
# cannot run inside this process (they slow every dispatch); their result is
# kept as a text summary and reported only while the sources it was measured
# on are unchanged: the attention kernels with their launch mapping and chunk
# plan, and the shared device and kernel headers.
TRAFFIC_SOURCES = ["paper_2606_02218_amd/csrc/k_attn.hip", "paper_2606_02218_amd/csrc/rg_device.h",
                   "paper_2606_02218_amd/csrc/rg_kernels.h"]
TRAFFIC_SUMMARY = "profiles/attention_decode_1.5b_traffic.txt"


def sources_sha256(paths=TRAFFIC_SOURCES):
    import hashlib
    h = hashlib.sha256()
    for rel in paths:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload, kernel):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated) of the
    kernel class on the workload, or None if the summary is for something else
    or any of its sources changed since the counters were taken."""
    import re
    try:
        text = open(os.path.join(ROOT, TRAFFIC_SUMMARY)).read()
    except OSError:
        return None
    kv = dict(re.findall(r"^\s*(workload|kernel|sources_sha256|traffic_bytes_per_launch):\s*(\S+)\s*$", text, re.M))
    if kv.get("workload") != workload or kv.get("kernel") != kernel or "traffic_bytes_per_launch" not in kv:
        return None
    if kv.get("sources_sha256") != sources_sha256():
        return None
    return int(kv["traffic_bytes_per_launch"])


def ceilings():
    """Measured ceilings beside the spec peaks: HBM streaming (torch's device
    copy and sum, and the library's own streaming probe, over 8 GiB) and bf16
    dense MFMA (the platform
    GEMM, hipBLASLt through torch.matmul, on a large square product and on
    the 1.5B projection shapes at 16384 and 512 rows).  Best of 10 timed
    repeats after 3 warmups, HIP events on torch's stream.  Prints one JSON
    line."""
    import torch

    def best_ms(fn, reps=10):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        out = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            out.append(e0.elapsed_time(e1))
        return min(out)

    import paper_2606_02218_amd as rg
    res = {"hbm_peak_spec_GBps": HBM_PEAK / 1e9, "mfma_bf16_peak_spec_TFLOPs": MFMA_BF16_PEAK / 1e12}
    n = 1 << 31                                       # 8 GiB of fp32
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    ms = best_ms(lambda: b.copy_(a))
    res["torch_copy_8GiB"] = {"ms": round(ms, 3), "GBps": round(2 * 4 * n / ms / 1e6, 1)}
    ms = best_ms(lambda: a.sum())
    res["torch_read_sum_8GiB"] = {"ms": round(ms, 3), "GBps": round(4 * n / ms / 1e6, 1)}
    # the library's own streaming probe (16-byte loads, grid-stride), by grid size
    sink = torch.empty(1 << 22, dtype=torch.int32, device="cuda")
    probe = {}
    for blocks in (1024, 2048, 4096, 8192, 16384):
        r_ms = best_ms(lambda: rg.hbm_probe(a, sink, 0, blocks))
        c_ms = best_ms(lambda: rg.hbm_probe(a, b, 1, blocks))
        probe[str(blocks)] = {"read_GBps": round(4 * n / r_ms / 1e6, 1), "copy_GBps": round(2 * 4 * n / c_ms / 1e6, 1)}
    res["probe_8GiB_by_blocks"] = probe
    res["probe_best"] = {"read_GBps": max(v["read_GBps"] for v in probe.values()),
                         "copy_GBps": max(v["copy_GBps"] for v in probe.values())}
    del a, b, sink
    g = {}
    shapes = {"square_8192": (8192, 8192, 8192)}
    for rows in (16384, 512):
        shapes.update({f"gate_up_{rows}": (rows, 17920, 1536), f"down_{rows}": (rows, 1536, 8960),
                       f"qkv_{rows}": (rows, 2048, 1536)})
    for name, (m, nn, k) in shapes.items():
        x = torch.randn(m, k, device="cuda").to(torch.bfloat16)
        w = torch.randn(nn, k, device="cuda").to(torch.bfloat16)
        wt = w.t()
        ms = best_ms(lambda: torch.matmul(x, wt))
        fl = 2.0 * m * nn * k
        g[name] = {"m_n_k": [m, nn, k], "ms": round(ms, 4), "TFLOPs": round(fl / ms / 1e9, 1),
                   "frac_of_spec": round(fl / (ms / 1e3) / MFMA_BF16_PEAK, 4)}
        del x, w, wt
    res["bf16_gemm_torch_matmul"] = g
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1, help="untimed steps; the first one times every kernel class")
    ap.add_argument("--workload", default="1.5b")
    ap.add_argument("--no-profile", action="store_true", help="skip per-kernel event timing")
    ap.add_argument("--cpu-steps", type=int, default=32, help="decode steps of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-report", action="store_true",
                    help="only time the oracle on the host (the full workload with --cpu-steps 0) and exit")
    ap.add_argument("--cpu-threads", type=int, default=0, help="thread limit of the oracle in --cpu-report")
    ap.add_argument("--eb-sweep", type=int, default=0, metavar="T",
                    help="only run the static-G vs controller sweep at EB = 64 with T steps per arm and exit")
    ap.add_argument("--group-prefix", action="store_true",
                    help="decode steps attend to each prompt's shared prefix once per group (RG_FLAG_GROUP_PREFIX)")
    ap.add_argument("--history-out", default="", metavar="PATH",
                    help="write the last rollout's step history (active rows, groups, prompt tokens per step) "
                         "and the per-token KV bytes to PATH (.npz) for `prof phases`")
    ap.add_argument("--loss-forward", action="store_true",
                    help="only run the GRPO loss forward (logprob recompute + clipped surrogate) and exit")
    ap.add_argument("--copy-calib", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (counter calibration) and exit")
    ap.add_argument("--ceilings", action="store_true",
                    help="only measure the HBM copy / read and bf16 GEMM ceilings and exit")
    ap.add_argument("--rows-sweep", type=int, default=0, metavar="L",
                    help="only time decode steps at 16, 32, 64 and 128 rows (completions forced to L tokens) and exit")
    ap.add_argument("--launch-floor", type=int, default=0, metavar="N",
                    help="only time the replay of a graph of N tiny dependent kernels and exit")
    ap.add_argument("--prefill-probe", type=int, default=0, metavar="K",
                    help="only run K rollouts of the workload's prompts with every completion forced to 2 tokens "
                         "(the prefill and one full-batch decode step; a short command for counter passes) and exit")
    args = ap.parse_args()
    if args.cpu_report:
        cpu_report(args)
        return
    if args.ceilings:
        ceilings()
        return
    if args.copy_calib:
        import torch
        n = args.copy_calib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calib_bytes_per_copy": n * 4, "copies": 5}))
        return
    if args.eb_sweep:
        eb_sweep(args)
        return
    if args.rows_sweep:
        rows_sweep(args)
        return
    if args.launch_floor:
        launch_floor(args.launch_floor)
        return
    if args.loss_forward:
        loss_forward(args)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path (prompt groups would shard "
              "across GPUs, one process per GPU; see the design notes).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_02218_amd as rg
    from workload import get_config, make_weights, make_inputs

    wl = get_config(args.workload)
    shape = wl.shape
    weights = make_weights(shape, 0)
    inp = make_inputs(wl, 0)
    N = inp.n_seq
    print(f"# weights and inputs of {wl.name} ready ({N} sequences)", file=sys.stderr, flush=True)
    pol = rg.Policy(shape, weights, max_seqs=N, max_prompts=wl.n_prompts,
                    max_prompt_tokens=wl.n_prompts * wl.prompt_len, max_context=wl.prompt_len + wl.max_new)
    print(f"# policy ready: {pol.device_bytes() / 2**30:.1f} GiB on the device", file=sys.stderr, flush=True)
    dev = torch.device("cuda")
    prompts = torch.from_numpy(inp.prompts).to(dev)
    if args.prefill_probe:
        two = np.full(N, 2, dtype=np.int32)
        out = (torch.empty((N, 2), dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.int32, device=dev),
               torch.empty((N, 2), dtype=torch.float32, device=dev))
        pf = []
        for i in range(args.prefill_probe):
            pol.rollout(prompts, inp.G, 2, 1234 + i, forced_len=two, out=out)
            pf.append(pol.phase_times()[0])
        torch.cuda.synchronize()
        print(json.dumps({"prefill_probe": wl.name, "rollouts": args.prefill_probe, "prefill_ms": [round(v, 2) for v in pf],
                          "prefill_flops": prefill_flops(shape, [wl.prompt_len] * wl.n_prompts)}), flush=True)
        return
    G_dev = torch.from_numpy(inp.G).to(dev)
    rewards = torch.from_numpy(inp.rewards).to(dev)
    tokens = torch.empty((N, wl.max_new), dtype=torch.int32, device=dev)
    lengths = torch.empty(N, dtype=torch.int32, device=dev)
    logprobs = torch.empty((N, wl.max_new), dtype=torch.float32, device=dev)
    adv = torch.empty(N, dtype=torch.float32, device=dev)
    profile = not args.no_profile

    def step(i, prof):
        pol.rollout(prompts, inp.G, wl.max_new, 1234 + i, forced_len=inp.forced_len, profile=prof,
                    group_prefix_pass=args.group_prefix, out=(tokens, lengths, logprobs))
        rg.group_advantage(rewards, G_dev, 1e-6, 1, out=adv)

    breakdown, dom, prefill_kt, by_bucket = {}, None, {}, {}
    for i in range(args.warmup):
        # the first warmup step times every kernel class (untimed step): the
        # per-class breakdown, and the dominant class timed in the timed steps
        step(i, profile and i == 0)
        if profile and i == 0:
            breakdown = pol.kernel_times(1)
            dom = max(breakdown.items(), key=lambda kv: kv[1][0])[0]
            prefill_kt = pol.kernel_times(0)
            by_bucket = {}
            for b, name in enumerate(("16", "32", "64", "128", "256", "384", "512", "more")):
                kb = {k: round(v[0], 2) for k, v in pol.kernel_times(2 + b).items() if v[1]}
                if kb:
                    steps = pol.kernel_times(2 + b)["compact"][1]
                    by_bucket[name] = {"steps": steps, "ms": kb}
        print(f"# warmup step {i} done", file=sys.stderr, flush=True)
    if profile and dom is None:
        dom = "attn"
    torch.cuda.synchronize()
    kt = {}
    phase = [0.0, 0.0]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, [dom] if profile else False)
        pf, dc = pol.phase_times()
        phase[0] += pf
        phase[1] += dc
        if profile:
            ms, n = pol.kernel_times(1)[dom]
            a = kt.setdefault(dom, [0.0, 0])
            a[0] += ms
            a[1] += n
        print(f"# timed step {i} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    gen = int(lengths.sum().item()) * 1  # tokens of the last step; every step has the same forced lengths
    hist_a, hist_g, hist_c = pol.step_history()
    if args.history_out:
        np.savez(args.history_out, active=np.asarray(hist_a), groups=np.asarray(hist_g), ctx=np.asarray(hist_c),
                 n_layers=shape.n_layers, kv_bytes_per_token_layer=2 * shape.kv_dim * shape.elem_bytes,
                 q_bytes_per_row=shape.q_dim * 8)
    assert np.array_equal(lengths.cpu().numpy(), inp.forced_len), "retired lengths differ from the forced lengths"

    ms_per_step = dt / args.steps * 1e3
    value = gen / (ms_per_step / 1e3)
    res = {"metric": "rollout decode tokens/s (group step = rollout_group + group_advantage)",
           "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms_per_step, 2), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "bf16" if shape.dtype == "bf16" else "f32", "data": "synthetic",
           "config": {"workload": wl.name, "prompts": wl.n_prompts,
                      "group_size": wl.group_size if wl.group_size is not None else sorted(set(int(g) for g in inp.G)),
                      "sequences": N, "prompt_len": wl.prompt_len, "max_new": wl.max_new,
                      "generated_tokens": gen, "decode_steps": int(len(hist_a)),
                      "group_prefix_pass": bool(args.group_prefix)},
           "group_step_s": round(ms_per_step / 1e3, 4)}
    # prefill (set-up, prompt tokens through the decoder, last-position lm
    # head, sibling fork) and decode on the device timeline, timed steps
    pf_s, dc_s = phase[0] / args.steps / 1e3, phase[1] / args.steps / 1e3
    F = prefill_flops(shape, [wl.prompt_len] * wl.n_prompts)
    res["prefill_ms"] = round(pf_s * 1e3, 2)
    res["decode_s"] = round(dc_s, 4)
    if shape.dtype == "bf16":
        res["roofline_prefill"] = {"bound": "mfma", "achieved": round(F / pf_s / 1e12, 1),
                                   "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s",
                                   "frac": round(F / pf_s / MFMA_BF16_PEAK, 4),
                                   "issued_frac": round(2 * F / pf_s / MFMA_BF16_PEAK, 4), "alg_flops": F,
                                   "note": "each fp32 activation enters bf16 MFMA as hi + lo planes: two MFMAs per "
                                           "product, so the algorithmic fraction is at most half the issued one"}
    else:   # fp32 models run plain fp32 FMA on the vector ALUs
        res["roofline_prefill"] = {"bound": "alu", "achieved": round(F / pf_s / 1e12, 3),
                                   "peak": FP32_VALU_PEAK / 1e12, "unit": "TFLOP/s",
                                   "frac": round(F / pf_s / FP32_VALU_PEAK, 6), "alg_flops": F}
    dec_b = decode_bytes_total(shape, hist_a, hist_g, hist_c)
    res["roofline_decode"] = {"bound": "hbm", "achieved": round(dec_b / dc_s / 1e9, 1), "peak": HBM_PEAK / 1e9,
                              "unit": "GB/s", "frac": round(dec_b / dc_s / HBM_PEAK, 4), "alg_bytes": dec_b,
                              "note": "whole decode: weights once per step, each active group's prompt KV once, "
                                      "each row's generated KV and its KV write, over the decode device time"}
    if breakdown:
        res["kernel_ms_breakdown_untimed_step"] = {k: round(v[0], 1) for k, v in
                                                   sorted(breakdown.items(), key=lambda kv: -kv[1][0]) if v[1]}
        dec_ms = sum(v[0] for v in breakdown.values())
        tot_b = decode_bytes_total(shape, hist_a, hist_g, hist_c)
        res["decode_hbm_frac_kernel_time"] = round(tot_b / (dec_ms / 1e3) / HBM_PEAK, 4)
        res["kernel_ms_by_row_bucket_untimed_step"] = by_bucket
        res["prefill_kernel_ms_untimed_step"] = {k: round(v[0], 2) for k, v in
                                                 sorted(prefill_kt.items(), key=lambda kv: -kv[1][0]) if v[1]}
    if profile and kt:
        alg, _ = algorithmic_bytes(shape, hist_a, hist_g, hist_c, wl.prompt_len)
        name, (ms_tot, n_tot) = next(iter(kt.items()))
        ms_avg = ms_tot / max(1, n_tot)
        if name in alg:
            per_launch = alg[name] * args.steps / max(1, n_tot)
            achieved = per_launch / (ms_avg / 1e3)
            traffic = measured_traffic(wl.name, name)
            res["roofline"] = {"kernel": name, "bound": "hbm", "achieved": round(achieved / 1e9, 1),
                               "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": round(achieved / HBM_PEAK, 4),
                               "traffic": traffic, "avg_launch_us": round(ms_avg * 1e3, 2),
                               "alg_bytes_per_launch": round(per_launch), "launches": n_tot}
            if traffic is not None:
                res["roofline"]["traffic_unit"] = "bytes per launch"
                res["roofline"]["traffic_vs_alg"] = round(traffic / per_launch, 3)
    if not args.no_cpu_baseline:
        del pol
        torch.cuda.empty_cache()
        res["cpu_baseline"] = cpu_baseline(wl, weights, inp, args.cpu_steps)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
