"""grpo_surrogate_noalloc, the clipped surrogate for callers that cannot
allocate device memory, called through the C ABI: on two calls in a row (the
second with fewer groups and sequences than the first, so stale records of
the first call sit in the static scratch beyond the second's N) its output
equals grpo_surrogate's bit for bit, and both match the oracle to 1e-10
relative; N above the scratch's 65536 records is refused on the host."""
import ctypes as C

import numpy as np
import pytest

from oracle.grpo import clipped_surrogate

pytestmark = pytest.mark.gpu


def _inputs(seed, G, T):
    rng = np.random.default_rng(seed)
    N = int(np.sum(G))
    L = rng.integers(1, T + 1, size=N).astype(np.int32)
    old = rng.normal(-2.0, 1.0, size=(N, T)).astype(np.float32)
    new = (old + rng.normal(0, 0.25, size=(N, T))).astype(np.float32)
    adv = rng.normal(size=N).astype(np.float32)
    keep = (rng.random(len(G)) < 0.7).astype(np.int32)
    return new, old, adv, L, keep


def _call(lib, fn, d, G_dev, P, N, T, keep, eps, mode, out, stream):
    return fn(d["new"].data_ptr(), d["old"].data_ptr(), d["adv"].data_ptr(), d["L"].data_ptr(), G_dev.data_ptr(),
              P, N, T, 0 if keep is None else keep.data_ptr(), C.c_double(eps[0]), C.c_double(eps[1]), mode,
              out.data_ptr(), stream)


@pytest.mark.timeout(120)
def test_noalloc_surrogate_matches_the_allocating_entry_point():
    import torch
    import paper_2606_02218_amd as rg
    from paper_2606_02218_amd import _lib
    assert torch.cuda.is_available()
    lib = rg.load_library()
    stream = torch.cuda.current_stream().cuda_stream
    rng = np.random.default_rng(77)
    cases = [(list(rng.integers(1, 33, size=400)), 48, (0.2, 0.28), 0),   # ~6,600 sequences, token mean
             (list(rng.integers(1, 9, size=37)), 20, (0.2, 0.2), 1)]       # fewer groups and sequences, seq mean
    for k, (G, T, eps, mode) in enumerate(cases):
        new, old, adv, L, keep = _inputs(900 + k, G, T)
        P, N = len(G), int(np.sum(G))
        print(f"no-alloc surrogate call {k}: P {P}, N {N}, max_new {T}, mode {mode}", flush=True)
        d = {n: torch.from_numpy(np.ascontiguousarray(a)).cuda() for n, a in
             (("new", new), ("old", old), ("adv", adv), ("L", L))}
        G_dev = torch.from_numpy(np.asarray(G, np.int32)).cuda()
        keep_dev = torch.from_numpy(keep).cuda()
        for kp, kd in ((None, None), (keep, keep_dev)):
            out_a = torch.full((4,), -7.0, dtype=torch.float64, device="cuda")
            out_b = torch.full((4,), -7.0, dtype=torch.float64, device="cuda")
            assert _call(lib, lib.grpo_surrogate, d, G_dev, P, N, T, kd, eps, mode, out_a, stream) == _lib.RG_OK
            assert _call(lib, lib.grpo_surrogate_noalloc, d, G_dev, P, N, T, kd, eps, mode, out_b,
                         stream) == _lib.RG_OK
            torch.cuda.synchronize()
            a, b = out_a.cpu().numpy(), out_b.cpu().numpy()
            assert np.array_equal(a, b), (a, b)
            want = clipped_surrogate(new, old, adv, L, G, *eps, mode="token" if mode == 0 else "seq", keep=kp)
            assert b[2] == want[2] and b[3] == want[3], (b, want)
            assert b[0] == pytest.approx(want[0], rel=1e-10, abs=1e-14)
            assert b[1] == pytest.approx(want[1], rel=1e-10, abs=1e-14)


def test_noalloc_surrogate_refuses_n_beyond_its_scratch():
    import paper_2606_02218_amd as rg
    from paper_2606_02218_amd import _lib
    lib = rg.load_library()
    p = [C.c_void_p(256 * (i + 1)) for i in range(6)]
    rc = lib.grpo_surrogate_noalloc(p[0], p[1], p[2], p[3], p[4], 1, 65537, 8, None, C.c_double(0.2),
                                    C.c_double(0.2), 0, p[5], None)
    assert rc == _lib.RG_EINVAL
    assert b"static scratch" in lib.rg_last_error()
