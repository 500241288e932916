"""GPU per-group length statistics (sagc_group_stats) against the oracle:
bit-exact (l_max, l_median, R, S) on ragged groups, plus the NaN rows for
groups outside the kernel's bounds, and the statistics of a real rollout
driving one controller step."""
import numpy as np
import pytest

from oracle import sagc as O

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available()
    return torch


def _expected(L, G, tau):
    return np.array([[np.float32(v) for v in s] for s in O.group_stats(L, G, tau)], dtype=np.float32)


def test_group_stats_match_oracle(torch):
    import paper_2606_02218_amd as rg
    rng = np.random.default_rng(0)
    G = [1, 2, 3, 4, 5, 8, 16, 17, 32, 64, 255, 256, 1024, 7]
    L = rng.integers(1, 4097, size=sum(G)).astype(np.int32)
    L[sum(G[:5]):sum(G[:6])] = 9            # a group of equal lengths: R = 1
    c = rg.Sagc(tau=1.25)
    got = c.group_stats(torch.from_numpy(L).cuda(), torch.tensor(G, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), _expected(L, G, 1.25))


def test_group_stats_bounds_give_nan(torch):
    import paper_2606_02218_amd as rg
    L = np.arange(1, 41, dtype=np.int32)
    G = [4, 0, 1025, 4, 40]                   # size 0, size > 1024, and a group running past N
    c = rg.Sagc()
    got = c.group_stats(torch.from_numpy(L).cuda(), torch.tensor(G, dtype=torch.int32, device="cuda")).cpu().numpy()
    assert np.isnan(got[1]).all() and np.isnan(got[2]).all() and np.isnan(got[4]).all()
    # offsets keep counting the declared sizes, so group 3 starts at 4 + 0 + 1025 > N: NaN as well
    assert np.isnan(got[3]).all()
    np.testing.assert_array_equal(got[0], _expected(L[:4], [4], 1.25)[0])


def test_rollout_lengths_drive_a_step(torch):
    import paper_2606_02218_amd as rg
    from workload import get_config, make_weights, make_inputs
    from rg_helpers import make_policy, prompts_to_device
    wl = get_config("tiny")
    w = make_weights(wl.shape, 1)
    inp = make_inputs(wl, 1)
    G = [4, 4, 4]
    prompts = [inp.prompts[0], inp.prompts[0][:9], inp.prompts[0][:13]]
    L = np.array([3, 30, 4, 5, 8, 8, 9, 8, 1, 32, 2, 2], np.int32)
    pol = make_policy(wl.shape, w, 12, 3, 48, wl.prompt_len + wl.max_new)
    tok, ln, lp = pol.rollout(prompts_to_device(prompts), G, wl.max_new, 9, forced_len=L)
    c = rg.Sagc(seed=4)
    st = c.group_stats(ln, torch.tensor(G, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.cpu().numpy(), _expected(L, G, 1.25))
    cfg = O.SagcConfig(seed=4)
    ref = O.sagc_init(cfg)
    assert c.step(st) == O.sagc_step(cfg, ref, [float(s) for s in _expected(L, G, 1.25)[:, 3]])
