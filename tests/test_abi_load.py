"""The C-ABI library loads on a machine without a GPU and exports every
function that include/*.h declares (no GPU calls here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]
LIB = os.path.join(ROOT, "paper_2606_02218_amd", "librollout.so")


def declared_functions():
    src = "\n".join(open(h).read() for h in HEADERS)
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([A-Za-z_][A-Za-z0-9_]*)\s*\(", src, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "while")))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ["rollout_group", "group_advantage", "rg_policy_create", "rg_policy_destroy", "rg_last_error",
              "rg_philox_blocks", "rg_gumbel_bits", "rg_step_history", "rg_kernel_times", "rg_policy_device_bytes",
              "sagc_init", "sagc_group_stats", "sagc_step", "sagc_beta_draw"]:
        assert n in names, n


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    for n in declared_functions():
        assert hasattr(lib, n), f"{n} declared in include/ but not exported"
    lib.rg_last_error.restype = ctypes.c_char_p
    assert isinstance(lib.rg_last_error(), bytes)


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_argument_validation_without_gpu():
    """Host-side validation answers before any device work."""
    import paper_2606_02218_amd as rg
    from paper_2606_02218_amd import _lib
    lib = rg.load_library()
    # group_advantage rejects bad scalars before launching
    assert lib.group_advantage(None, None, 1, 1, 1e-6, 1, None, None) == _lib.RG_EINVAL
    assert lib.group_advantage(ctypes.c_void_p(16), ctypes.c_void_p(32), 0, 1, 1e-6, 1, ctypes.c_void_p(64), None) == _lib.RG_EINVAL
    assert lib.group_advantage(ctypes.c_void_p(16), ctypes.c_void_p(32), 1, 1, 1e-6, 2, ctypes.c_void_p(64), None) == _lib.RG_EINVAL
    assert b"ddof" in lib.rg_last_error()
    cfg = _lib.rg_config(0, 128, 4, 4, 32, 512, 512, 511, 1e4, 1e-6, 0)
    w = _lib.rg_weights()
    lim = _lib.rg_limits(4, 1, 16, 48, 0)
    h = ctypes.c_void_p()
    assert lib.rg_policy_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(lim), ctypes.byref(h)) == _lib.RG_EINVAL
    cfg = _lib.rg_config(2, 100, 4, 4, 25, 512, 512, 511, 1e4, 1e-6, 0)
    assert lib.rg_policy_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(lim), ctypes.byref(h)) == _lib.RG_EUNSUPPORTED
    assert lib.rollout_group(None, None, None, 1, None, 1, 0, None, None, None, None, None) == _lib.RG_EINVAL


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_argument_validation_cases_without_gpu():
    """Every host-side rejection documented in include/rollout.h, one case each;
    each returns its code before any device work, with a message naming the
    problem."""
    import paper_2606_02218_amd as rg
    from paper_2606_02218_amd import _lib
    lib = rg.load_library()
    E, U = _lib.RG_EINVAL, _lib.RG_EUNSUPPORTED
    # a valid 1.5B-shaped config, then one field broken at a time
    base = dict(n_layers=28, d_model=1536, n_q_heads=12, n_kv_heads=2, head_dim=128, ffn_dim=8960, vocab=151936,
                eos_id=151935, rope_theta=1e6, rms_eps=1e-6, dtype=_lib.RG_DTYPE_BF16)
    cases = [
        (dict(vocab=1, eos_id=0), E, b"invalid config"),
        (dict(eos_id=151936), E, b"invalid config"),
        (dict(rope_theta=0.0), E, b"invalid config"),
        (dict(rms_eps=-1.0), E, b"invalid config"),
        (dict(dtype=7), U, b"dtype"),
        (dict(head_dim=96), U, b"head_dim"),
        (dict(head_dim=32, d_model=384), U, b"bf16 models need head_dim"),
        (dict(n_kv_heads=5), U, b"n_q/n_kv"),
        (dict(n_q_heads=24, n_kv_heads=2), U, b"n_q/n_kv"),
        (dict(d_model=1540), U, b"multiples of 64"),
        (dict(ffn_dim=8961), U, b"multiples of 64"),
        (dict(vocab=151937, eos_id=0), U, b"vocab multiple of 16"),
    ]
    w = _lib.rg_weights()
    lim = _lib.rg_limits(512, 32, 16384, 4608, 0)
    h = ctypes.c_void_p()
    for change, code, msg in cases:
        cfg = _lib.rg_config(**{**base, **change})
        assert lib.rg_policy_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(lim), ctypes.byref(h)) == code, change
        assert msg in lib.rg_last_error(), (change, lib.rg_last_error())
        assert h.value is None
    cfg = _lib.rg_config(**base)
    for bad in [(0, 32, 16384, 4608, 0), (512, 0, 16384, 4608, 0), (512, 32, 0, 4608, 0), (512, 32, 16384, 1, 0),
                (512, 32, 16384, 4608, -1)]:
        lim = _lib.rg_limits(*bad)
        assert lib.rg_policy_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(lim), ctypes.byref(h)) == E, bad
        assert b"invalid limits" in lib.rg_last_error()
    assert lib.rg_policy_create(None, ctypes.byref(w), ctypes.byref(lim), ctypes.byref(h)) == E

    p = [ctypes.c_void_p(16 * (i + 1)) for i in range(8)]   # stand-in device addresses: never dereferenced
    # group_advantage
    assert lib.group_advantage(p[0], p[1], 1, 4, -1e-6, 1, p[2], None) == E and b"eps" in lib.rg_last_error()
    assert lib.group_advantage(p[0], p[1], 1, 4, 1e-6, 1, p[0], None) == E and b"aliases" in lib.rg_last_error()
    assert lib.group_advantage(p[0], p[1], 1, 0, 1e-6, 1, p[2], None) == E
    # group_filter
    assert lib.group_filter(p[0], p[1], 0, 4, p[2], p[3], p[4], None) == E
    assert lib.group_filter(p[0], None, 1, 4, p[2], p[3], p[4], None) == E
    # grpo_surrogate: eps_lo in [0, 1), eps_hi >= 0 and finite, known mode, sizes >= 1
    sur = lib.grpo_surrogate
    ok = dict(P=1, N=4, max_new=8, eps_lo=0.2, eps_hi=0.28, mode=_lib.LOSS_MODES["token"])
    for change, msg in [(dict(eps_lo=1.0), b"eps"), (dict(eps_lo=-0.1), b"eps"), (dict(eps_hi=-0.1), b"eps"),
                        (dict(eps_hi=float("inf")), b"eps"), (dict(mode=5), b"mode"), (dict(P=0), b">= 1"),
                        (dict(max_new=0), b">= 1")]:
        a = {**ok, **change}
        assert sur(p[0], p[1], p[2], p[3], p[4], a["P"], a["N"], a["max_new"], None, a["eps_lo"], a["eps_hi"],
                   a["mode"], p[5], None) == E, change
        assert msg in lib.rg_last_error(), (change, lib.rg_last_error())
    assert sur(None, p[1], p[2], p[3], p[4], 1, 4, 8, None, 0.2, 0.28, 0, p[5], None) == E
    # generator probes
    assert lib.rg_philox_blocks(1, 2, p[0], -1, p[1], None) == E
    assert lib.rg_gumbel_bits(1, 0, 0, 0, p[0], None) == E
    assert lib.rg_gumbel_bits(1, -1, 0, 16, p[0], None) == E


def test_missing_library_fails_loudly(monkeypatch):
    """Without librollout.so every entry point raises: there is no fallback."""
    from paper_2606_02218_amd import _lib
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "_LIB_PATH", os.path.join(ROOT, "paper_2606_02218_amd", "no_such_librollout.so"))
    with pytest.raises(ImportError, match="no fallback"):
        _lib.load_library()
    with pytest.raises(ImportError):
        _lib.group_advantage(None, None)
    with pytest.raises(ImportError):
        _lib.group_filter(None, None)


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_decode_attention_chunk_plan():
    """The chunk plan a decode step's attention takes (host logic, no GPU):
    the multi-chunk GPU test's rollout and the 1.5B workload at every row
    count cut each row's context into several chunks; from 512 to 2048
    (row, kv head) pairs two, merged inside the kernel; beyond that, or for
    contexts under 512 tokens, one."""
    import paper_2606_02218_amd as rg
    assert rg.decode_attention_chunks(5, 2, 2300 + 10) >= 3
    for rows in (1, 16, 64, 128, 256):
        assert rg.decode_attention_chunks(rows, 2, 512 + 4096) >= 2, rows
    for rows in (384, 512, 1024):
        assert rg.decode_attention_chunks(rows, 2, 512 + 4096) == 2, rows
    assert rg.decode_attention_chunks(2048, 2, 512 + 4096) == 1
    assert rg.decode_attention_chunks(512, 2, 400) == 1
    with pytest.raises(rg.RolloutError):
        rg.decode_attention_chunks(0, 2, 100)
