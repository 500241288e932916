"""Summaries of rocprofv3 CSV output (kernel stats and counter collection).

    python -m paper_2606_02218_amd.prof stats DIR              # per-kernel time table
    python -m paper_2606_02218_amd.prof trace DIR [TOP]        # per kernel and grid size, from kernel_trace.csv
    python -m paper_2606_02218_amd.prof steps DIR              # decode-step time by active-row bucket
    python -m paper_2606_02218_amd.prof steps-full DIR         # the same, every kernel instantiation listed
    python -m paper_2606_02218_amd.prof phases DIR HIST.npz    # decode attention by phase of one rollout
    python -m paper_2606_02218_amd.prof counters DIR REGEX     # mean counter per dispatch
    python -m paper_2606_02218_amd.prof step-counters DIR      # counters per kernel and decode-row bucket
"""
from __future__ import annotations

import collections
import csv
import glob
import os
import re
import sys


def _find(d: str, suffix: str):
    return sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))


def _short(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "")
    return re.sub(r"^void ", "", name)[:100]


def stats_table(d: str) -> str:
    rows = []
    for f in _find(d, "kernel_stats.csv"):
        rows += list(csv.DictReader(open(f)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = [f"{'kernel':100s} {'calls':>9s} {'total_ms':>10s} {'avg_us':>9s} {'pct':>6s}"]
    for r in rows:
        out.append(f"{_short(r['Name']):100s} {int(r['Calls']):9d} {float(r['TotalDurationNs']) / 1e6:10.1f} "
                   f"{float(r['AverageNs']) / 1e3:9.2f} {float(r['Percentage']):6.2f}")
    return "\n".join(out)


def trace_table(d: str, top: int = 60) -> str:
    """Dispatch time grouped by (kernel, grid size): the grid of the row-sized
    kernels tells the row bucket of a decode step."""
    acc = collections.defaultdict(lambda: [0, 0.0])
    span = [None, None]
    for f in _find(d, "kernel_trace.csv"):
        for r in csv.DictReader(open(f)):
            s0, e0 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
            span[0] = s0 if span[0] is None else min(span[0], s0)
            span[1] = e0 if span[1] is None else max(span[1], e0)
            grid = "x".join(r.get(k, "") for k in ("Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z"))
            wg = "x".join(r.get(k, "") for k in ("Workgroup_Size_X", "Workgroup_Size_Y", "Workgroup_Size_Z"))
            name = _short(r.get("Kernel_Name", "?")).split("(")[0]
            a = acc[(name, grid, wg)]
            a[0] += 1
            a[1] += (e0 - s0) / 1e3
    tot = sum(v[1] for v in acc.values())
    out = [f"span_ms {((span[1] or 0) - (span[0] or 0)) / 1e6:.1f}  busy_ms {tot / 1e3:.1f}",
           f"{'kernel':44s} {'grid':>22s} {'wg':>10s} {'calls':>8s} {'total_ms':>10s} {'avg_us':>9s}"]
    for (k, g, w), (n, us) in sorted(acc.items(), key=lambda kv: -kv[1][1])[:top]:
        out.append(f"{k[:44]:44s} {g:>22s} {w:>10s} {n:8d} {us / 1e3:10.1f} {us / n:9.2f}")
    return "\n".join(out)


def _kname(r) -> str:
    return _short(r.get("Kernel_Name", "?")).split("(")[0].split("<")[0]


def steps_table(d: str, full: bool = False) -> str:
    """Decode steps delimited by k_compact; a step's row bound comes from the
    grid of its k_decode_rows launch (one 256-thread block per row).  Reports,
    per row bucket, the steps, GPU-busy and wall span per step, and the busy
    time per kernel name (full: per template instantiation, with launches
    per step and the mean launch duration)."""
    rows = []
    for f in _find(d, "kernel_trace.csv"):
        rows += list(csv.DictReader(open(f)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    buckets = collections.OrderedDict((b, None) for b in (16, 32, 64, 128, 256, 384, 512, 1 << 30))
    acc = {b: {"steps": 0, "busy": 0.0, "span": 0.0, "k": collections.Counter()} for b in buckets}
    cnt, cur_n = collections.Counter(), collections.Counter()
    cur, m, t0, busy = collections.Counter(), None, None, 0.0
    for r in rows:
        name = _kname(r)
        key = _short(r.get("Kernel_Name", "?")).split("(")[0] if full else name
        s0, e0 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        if t0 is None:
            t0 = s0
        dur = (e0 - s0) / 1e3
        cur[key] += dur
        cur_n[key] += 1
        busy += dur
        if name == "k_decode_rows":
            m = int(r.get("Grid_Size_X", "0") or 0) // 256
        if name == "k_compact":
            if m is not None:
                b = next(b for b in buckets if m <= b)
                a = acc[b]
                a["steps"] += 1
                a["busy"] += busy
                a["span"] += (e0 - t0) / 1e3
                a["k"].update(cur)
                a.setdefault("n", collections.Counter()).update(cur_n)
            cur, cur_n, m, t0, busy = collections.Counter(), collections.Counter(), None, None, 0.0
    out = [f"{'rows<=':>8s} {'steps':>6s} {'busy_ms/step':>13s} {'span_ms/step':>13s} {'total_span_s':>13s}  top kernels (us/step)"]
    for b, a in acc.items():
        if not a["steps"]:
            continue
        n = a["steps"]
        top = ", ".join(f"{k} {v / n:.0f}" for k, v in a["k"].most_common(6))
        out.append(f"{b if b < (1 << 30) else 'more':>8} {n:6d} {a['busy'] / n / 1e3:13.3f} {a['span'] / n / 1e3:13.3f} "
                   f"{a['span'] / 1e6:13.2f}" + ("" if full else f"  {top}"))
        if full:
            for k, v in a["k"].most_common():
                c = a["n"][k]
                out.append(f"{'':>8} {k[:70]:70s} {c / n:7.1f}/step {v / n:9.1f} us/step {v / c:8.2f} us")
    return "\n".join(out)


def phases_table(d: str, hist_path: str) -> str:
    """Decode attention of one rollout (the trace's only rollout) by phase:
    steps grouped by their active-row count.  HIST.npz is the step history
    that `bench.py --history-out` writes.  The first n_layers per-row
    attention launches attend the prompt rows; after them decode step t owns
    launches (t-1)*n_layers .. t*n_layers-1, and a merge launch belongs to the
    attention launch before it.  Algorithmic bytes count each active group's
    prompt once; wave-read bytes count it once per row (what the per-row
    pass's waves read, the repeats served by L2)."""
    import numpy as np
    h = np.load(hist_path)
    A, Gr, C = h["active"], h["groups"], h["ctx"]
    L = int(h["n_layers"])
    kvb, qb = float(h["kv_bytes_per_token_layer"]), float(h["q_bytes_per_row"])
    ev = []
    for f in _find(d, "kernel_trace.csv"):
        for r in csv.DictReader(open(f)):
            n = _kname(r)
            if n in ("k_attention_mfma", "k_attn_merge"):
                s0 = int(r["Start_Timestamp"])
                ev.append((s0, int(r["End_Timestamp"]) - s0, n == "k_attn_merge"))
    ev.sort()
    att = []
    for _, dt, is_merge in ev:
        if is_merge:
            if att:
                att[-1][1] += dt
        else:
            att.append([dt, 0])
    bins = [(257, 1 << 30), (129, 256), (65, 128), (33, 64), (17, 32), (1, 16)]
    acc = {b: [0, 0.0, 0.0, 0.0, 0.0] for b in bins}
    used = 0
    for i, (dt, dm) in enumerate(att[L:]):
        t = 1 + i // L
        if t >= len(A) or int(A[t]) == 0:
            break
        M, g = int(A[t]), int(Gr[t])
        alg = (float(C[t]) / M * g + M * t) * kvb + M * qb
        wave = (float(C[t]) + M * t) * kvb + M * qb
        a = acc[next(b for b in bins if b[0] <= M <= b[1])]
        a[0] += 1; a[1] += dt; a[2] += dm; a[3] += alg; a[4] += wave
        used += 1
    out = [f"decode attention launches {len(att) - L} (after {L} prompt-row launches), {used} matched to steps",
           f"{'rows':>9s} {'launches':>9s} {'attn_ms':>8s} {'merge_ms':>9s} {'us/launch':>10s} {'alg_MB':>8s} "
           f"{'alg_TB/s':>9s} {'wave_TB/s':>10s}"]
    ta = tm = 0.0
    for (lo, hi), (n, dt, dm, alg, wave) in acc.items():
        if n:
            ta += dt; tm += dm
            label = f"{lo}+" if hi == 1 << 30 else f"{lo}-{hi}"
            out.append(f"{label:>9s} {n:9d} {dt / 1e6:8.1f} {dm / 1e6:9.1f} {dt / n / 1e3:10.2f} "
                       f"{alg / n / 1e6:8.1f} {alg / dt / 1e3:9.2f} {wave / dt / 1e3:10.2f}")
    out.append(f"total: attention {ta / 1e6:.1f} ms, merge {tm / 1e6:.1f} ms")
    return "\n".join(out)


def counter_table(d: str, regex: str) -> str:
    pat = re.compile(regex)
    acc = collections.defaultdict(lambda: [0, 0.0])
    for f in _find(d, "counter_collection.csv"):
        for r in csv.DictReader(open(f)):
            name = r.get("Kernel_Name", "")
            if not pat.search(name):
                continue
            key = (_short(name), r.get("Counter_Name", "?"))
            a = acc[key]
            a[0] += 1
            a[1] += float(r.get("Counter_Value", 0) or 0)
    out = [f"{'kernel':100s} {'counter':>12s} {'dispatches':>10s} {'mean_per_dispatch':>18s}"]
    for (k, c), (n, v) in sorted(acc.items()):
        out.append(f"{k:100s} {c:>12s} {n:10d} {v / max(1, n):18.1f}")
    return "\n".join(out)


def step_counters(d: str) -> dict:
    """Counter collection grouped like `steps`: dispatches before the first
    k_decode_rows are the prefill; after it, decode steps are delimited by
    k_compact and bucketed by the row bound of their k_decode_rows launch.
    Returns {bucket: {kernel: {"dispatches": n, counter: sum}}}."""
    disp = {}
    for f in _find(d, "counter_collection.csv"):
        for r in csv.DictReader(open(f)):
            key = (f, int(r["Dispatch_Id"]))
            e = disp.get(key)
            if e is None:
                e = disp[key] = {"t": int(r.get("Start_Timestamp", 0) or 0), "name": r.get("Kernel_Name", "?"),
                                 "grid": int(r.get("Grid_Size", 0) or 0), "c": collections.Counter()}
            e["c"][r["Counter_Name"]] += float(r.get("Counter_Value", 0) or 0)
    order = sorted(disp.values(), key=lambda e: e["t"])
    buckets = (16, 32, 64, 128, 256, 384, 512, 1 << 30)
    out = collections.OrderedDict()
    cur, m, decoding = [], None, False

    def flush(label):
        b = out.setdefault(label, {})
        for e in cur:
            k = b.setdefault(_short(e["name"]).split("(")[0], collections.Counter())
            k["dispatches"] += 1
            k.update(e["c"])

    for e in order:
        name = _short(e["name"]).split("(")[0].split("<")[0]
        if name == "k_decode_rows" and not decoding:
            flush("prefill")
            cur, decoding = [], True
        cur.append(e)
        if name == "k_decode_rows":
            m = e["grid"] // 256
        if decoding and name == "k_compact" and m is not None:
            flush(str(next(b for b in buckets if m <= b)))
            cur, m = [], None
    if cur:
        flush("prefill" if not decoding else "tail")
    return out


def step_counters_table(d: str) -> str:
    res = step_counters(d)
    lines = []
    for b, ks in res.items():
        lines.append(f"[{b}]")
        names = sorted({c for k in ks.values() for c in k if c != "dispatches"})
        lines.append(f"  {'kernel':64s} {'dispatches':>10s} " + " ".join(f"{c:>26s}" for c in names))
        for k, v in sorted(ks.items(), key=lambda kv: -kv[1]["dispatches"]):
            n = v["dispatches"]
            lines.append(f"  {k[:64]:64s} {n:10d} " + " ".join(f"{v[c] / n:26.1f}" for c in names))
    return "\n".join(lines)


if __name__ == "__main__":
    if len(sys.argv) >= 3 and sys.argv[1] == "stats":
        print(stats_table(sys.argv[2]))
    elif len(sys.argv) >= 3 and sys.argv[1] == "trace":
        print(trace_table(sys.argv[2], int(sys.argv[3]) if len(sys.argv) > 3 else 60))
    elif len(sys.argv) >= 3 and sys.argv[1] == "steps":
        print(steps_table(sys.argv[2]))
    elif len(sys.argv) >= 3 and sys.argv[1] == "steps-full":
        print(steps_table(sys.argv[2], full=True))
    elif len(sys.argv) >= 4 and sys.argv[1] == "phases":
        print(phases_table(sys.argv[2], sys.argv[3]))
    elif len(sys.argv) >= 4 and sys.argv[1] == "counters":
        print(counter_table(sys.argv[2], sys.argv[3]))
    elif len(sys.argv) >= 3 and sys.argv[1] == "step-counters":
        print(step_counters_table(sys.argv[2]))
    else:
        print(__doc__)
        sys.exit(2)
