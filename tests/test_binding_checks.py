"""The Python binding checks shapes, dtypes, devices and contiguity before it
calls into the library, so that a buffer sized differently from what a
kernel indexes is refused on the host (CPU only: every case raises before
any ctypes call or device work)."""
import os

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2606_02218_amd", "librollout.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")


def _policy():
    """A Policy object without a device-side handle: only the host-side
    argument checks run (each case must raise before any library call)."""
    from paper_2606_02218_amd import _lib
    from workload import ModelShape
    pol = object.__new__(_lib.Policy)
    pol.shape = ModelShape(1, 128, 2, 1, 64, 256, 512, 1e4, dtype="bf16")
    pol._h = None
    return pol


def test_tensor_check_order():
    from paper_2606_02218_amd._lib import _dev, _gpu
    t = torch.zeros((2, 3), dtype=torch.int32)
    with pytest.raises(TypeError, match="torch.Tensor"):
        _dev("x", np.zeros((2, 3), np.int32), torch.int32, (2, 3))
    with pytest.raises(TypeError, match="dtype"):
        _dev("x", t.float(), torch.int32, (2, 3))
    with pytest.raises(ValueError, match="shape"):
        _dev("x", t, torch.int32, (3, 2))
    with pytest.raises(ValueError, match="dimension"):
        _dev("x", t, torch.int32, ndim=1)
    with pytest.raises(ValueError, match="contiguous"):
        _dev("x", t.t(), torch.int32, (3, 2))
    assert _dev("x", t, torch.int32, (2, 3)) is t
    with pytest.raises(TypeError, match="GPU memory"):
        _gpu(x=t)


def test_rollout_rejects_bad_inputs():
    pol = _policy()
    cpu_prompts = torch.zeros((2, 8), dtype=torch.int32)
    with pytest.raises(TypeError, match="GPU memory"):
        pol.rollout(cpu_prompts, [2, 2], 4, 0)
    with pytest.raises(TypeError, match="dtype"):
        pol.rollout(cpu_prompts.long(), [2, 2], 4, 0)
    with pytest.raises(ValueError, match="at least one"):
        pol.rollout([], [], 4, 0)
    with pytest.raises(ValueError, match="dimension"):
        pol.rollout([torch.zeros((2, 2), dtype=torch.int32)], [1], 4, 0)


def test_recompute_rejects_bad_inputs():
    pol = _policy()
    prompts = [torch.zeros(8, dtype=torch.int32)]
    with pytest.raises(TypeError, match="GPU memory"):
        pol.recompute_logprobs(prompts, [2], torch.zeros((2, 4), dtype=torch.int32), torch.ones(2, dtype=torch.int32))


def test_free_functions_reject_bad_inputs():
    from paper_2606_02218_amd import _lib
    r32 = torch.zeros(8, dtype=torch.float32)
    g32 = torch.tensor([4, 4], dtype=torch.int32)
    with pytest.raises(TypeError, match="dtype"):
        _lib.group_advantage(r32.double(), g32)
    with pytest.raises(TypeError, match="dtype"):
        _lib.group_advantage(r32, g32.long())
    with pytest.raises(ValueError, match="dimension"):
        _lib.group_filter(r32.view(2, 4), g32)
    with pytest.raises(TypeError, match="GPU memory"):
        _lib.group_filter(r32, g32)
    new = torch.zeros((8, 5), dtype=torch.float32)
    with pytest.raises(ValueError, match="shape"):
        _lib.grpo_surrogate(new, torch.zeros((8, 4)), r32, torch.ones(8, dtype=torch.int32), g32)
    with pytest.raises(ValueError, match="shape"):
        _lib.grpo_surrogate(new, new.clone(), torch.zeros(7), torch.ones(8, dtype=torch.int32), g32)
    with pytest.raises(TypeError, match="dtype"):
        _lib.grpo_surrogate(new, new.clone(), r32, torch.ones(8, dtype=torch.int64), g32)
    with pytest.raises(ValueError, match="shape"):
        _lib.grpo_surrogate(new, new.clone(), r32, torch.ones(8, dtype=torch.int32), g32,
                            keep=torch.ones(3, dtype=torch.int32))
    with pytest.raises(ValueError, match="shape"):
        _lib.philox_blocks(1, 2, torch.zeros((3, 3), dtype=torch.int64))


def test_rollout_checks_every_buffer_before_the_device():
    """Shapes and dtypes of every argument are checked before any of them is
    required to be in GPU memory, so these cases run on the CPU."""
    pol = _policy()
    pr = torch.zeros((2, 8), dtype=torch.int32)
    with pytest.raises(ValueError, match="one entry per prompt"):
        pol.rollout(pr, [2], 4, 0)
    with pytest.raises(ValueError, match="forced_len must have N = 4"):
        pol.rollout(pr, [2, 2], 4, 0, forced_len=[4, 4, 4])
    with pytest.raises(TypeError, match="integers"):
        pol.rollout(pr, [2, 2], 4, 0, forced_len=np.full(4, 2.0))
    with pytest.raises(ValueError, match="force_tokens must have shape"):
        pol.rollout(pr, [2, 2], 4, 0, force_tokens=torch.zeros((4, 3), dtype=torch.int32))
    good = (torch.zeros((4, 4), dtype=torch.int32), torch.zeros(4, dtype=torch.int32), torch.zeros((4, 4)))
    for k, bad in [(0, torch.zeros((4, 5), dtype=torch.int32)), (1, torch.zeros(3, dtype=torch.int32)),
                   (2, torch.zeros((4, 4), dtype=torch.float64))]:
        out = list(good)
        out[k] = bad
        with pytest.raises((ValueError, TypeError)):
            pol.rollout(pr, [2, 2], 4, 0, out=tuple(out))
    with pytest.raises(TypeError, match="GPU memory"):
        pol.rollout(pr, [2, 2], 4, 0, forced_len=[4, 4, 4, 4], out=good)


def test_recompute_checks_every_buffer_before_the_device():
    pol = _policy()
    pr = [torch.zeros(8, dtype=torch.int32), torch.zeros(5, dtype=torch.int32)]
    tok = torch.zeros((3, 4), dtype=torch.int32)
    with pytest.raises(ValueError, match="rows"):
        pol.recompute_logprobs(pr, [2, 2], tok, torch.ones(4, dtype=torch.int32))
    with pytest.raises(ValueError, match="lengths must have shape"):
        pol.recompute_logprobs(pr, [2, 1], tok, torch.ones(4, dtype=torch.int32))
    with pytest.raises(TypeError, match="dtype"):
        pol.recompute_logprobs(pr, [2, 1], tok.long(), torch.ones(3, dtype=torch.int32))
    with pytest.raises(ValueError, match="logprobs"):
        pol.recompute_logprobs(pr, [2, 1], tok, torch.ones(3, dtype=torch.int32), out=torch.zeros((3, 5)))


def test_hbm_probe_rejects_bad_inputs():
    from paper_2606_02218_amd import _lib
    src = torch.zeros(64, dtype=torch.int32)
    with pytest.raises(ValueError, match="contiguous"):
        _lib.hbm_probe(torch.zeros((8, 8), dtype=torch.int32).t(), src, 1)
    with pytest.raises(ValueError, match="at least"):
        _lib.hbm_probe(src, torch.zeros(16, dtype=torch.int32), 1)
    with pytest.raises(ValueError, match="at least"):
        _lib.hbm_probe(src, torch.zeros(64, dtype=torch.int32), 0, blocks=1)
    with pytest.raises(TypeError, match="GPU memory"):
        _lib.hbm_probe(src, torch.zeros(64, dtype=torch.int32), 1)
