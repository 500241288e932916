"""`prof phases` (decode attention by phase of one rollout) on a synthetic
kernel trace: launches map to decode steps in order after the prompt-row
launches, merges attach to the attention launch before them, and the byte
rates follow from the step history."""
import csv
import os

import numpy as np

from paper_2606_02218_amd.prof import phases_table


def _trace(path, events):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for name, s0, dur in events:
            w.writerow({"Kernel_Name": name, "Start_Timestamp": s0, "End_Timestamp": s0 + dur})


def test_phases_table(tmp_path):
    L = 2
    att = "void (anonymous namespace)::k_attention_mfma<128, 2>(float const*, int)"
    merge = "void (anonymous namespace)::k_attn_merge<1>(float const*)"
    ev, t = [], 1000
    ms = 1000000                          # trace timestamps are in ns
    for _ in range(L):                    # prompt rows
        ev.append((att, t, 5 * ms)); t += 10 * ms
    # step 1: 300 rows, one chunk; step 2: 20 rows, a merge after each launch
    for _ in range(L):
        ev.append((att, t, 10 * ms)); t += 20 * ms
    for _ in range(L):
        ev.append((att, t, 4 * ms)); t += 5 * ms
        ev.append((merge, t, 1 * ms)); t += 2 * ms
    ev.append(("void (anonymous namespace)::k_compact(x)", t, 50))
    os.makedirs(tmp_path / "tr" / "sub")
    _trace(tmp_path / "tr" / "sub" / "run_kernel_trace.csv", ev)
    kvb, qb = 1e7, 1e6
    np.savez(tmp_path / "h.npz", active=np.array([300, 300, 20, 0]), groups=np.array([30, 30, 4, 0]),
             ctx=np.array([300 * 50, 300 * 50, 20 * 50, 0]), n_layers=L, kv_bytes_per_token_layer=kvb,
             q_bytes_per_row=qb)
    out = phases_table(str(tmp_path / "tr"), str(tmp_path / "h.npz")).splitlines()
    assert out[0].startswith(f"decode attention launches {2 * L} (after {L} prompt-row launches), {2 * L} matched")
    big = next(l for l in out if l.lstrip().startswith("257+")).split()
    small = next(l for l in out if l.lstrip().startswith("17-32")).split()
    # step 1: alg = (prefix once per group 30*50 + 300*1) * kvb + 300*qb; wave = (300*50 + 300) * kvb + 300*qb
    alg1 = (30 * 50 + 300 * 1) * kvb + 300 * qb
    wave1 = (300 * 50 + 300) * kvb + 300 * qb
    assert int(big[1]) == L and float(big[2]) == 20.0 and float(big[3]) == 0.0 and float(big[4]) == 10000.0
    assert abs(float(big[5]) - alg1 / 1e6) < 0.05
    assert abs(float(big[6]) - alg1 / (10 * ms) / 1e3) < 0.006          # bytes per ns = GB/s
    assert abs(float(big[7]) - wave1 / (10 * ms) / 1e3) < 0.006
    alg2 = (4 * 50 + 20 * 2) * kvb + 20 * qb
    assert int(small[1]) == L and float(small[2]) == 8.0 and float(small[3]) == 2.0
    assert abs(float(small[6]) - alg2 / (4 * ms) / 1e3) < 0.006
    assert out[-1] == "total: attention 28.0 ms, merge 2.0 ms"


def _counters(path, dispatches):
    cols = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp"]
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=cols)
        w.writeheader()
        for i, (name, grid, cnt) in enumerate(dispatches):
            for c, v in cnt.items():
                w.writerow({"Dispatch_Id": i + 1, "Grid_Size": grid, "Kernel_Name": name, "Counter_Name": c,
                            "Counter_Value": v, "Start_Timestamp": 100 * i})


def test_step_counters(tmp_path):
    """Dispatches before the first decode-row set-up are the prefill; each
    decode step (closed by k_compact) lands in the bucket of its row bound
    (the k_decode_rows grid / 256); counters are summed per kernel."""
    from paper_2606_02218_amd.prof import step_counters
    g = "void k_gemm_tiled<32, 128, 1, 4, 1, 64, 4, true>(x)"
    rows = "void k_decode_rows<unsigned short>(int)"
    comp = "void k_compact(int)"
    disp = [("void k_gemm_tiled<256, 256, 4, 8, 1, 64, 2, false>(x)", 9, {"A": 10.0}),
            ("void k_gemm_tiled<256, 256, 4, 8, 1, 64, 2, false>(x)", 9, {"A": 30.0})]
    for m in (20, 20, 300):                 # two steps at <= 32 rows, one at <= 384
        disp += [(rows, 256 * m, {"A": 1.0}), (g, 7, {"A": float(m)}), (comp, 1024, {"A": 0.0})]
    os.makedirs(tmp_path / "pmc" / "x")
    _counters(tmp_path / "pmc" / "x" / "run_counter_collection.csv", disp)
    res = step_counters(str(tmp_path / "pmc"))
    assert list(res) == ["prefill", "32", "384"]
    pre = res["prefill"]["k_gemm_tiled<256, 256, 4, 8, 1, 64, 2, false>"]
    assert pre["dispatches"] == 2 and pre["A"] == 40.0
    k32 = res["32"]["k_gemm_tiled<32, 128, 1, 4, 1, 64, 4, true>"]
    assert k32["dispatches"] == 2 and k32["A"] == 40.0
    assert res["384"]["k_gemm_tiled<32, 128, 1, 4, 1, 64, 4, true>"]["A"] == 300.0
    assert res["32"]["k_compact"]["dispatches"] == 2
