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
