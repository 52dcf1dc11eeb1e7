"""The allocation-free entry point (lsgd_replica_sign_sync_static) against
lsgd_replica_sign_sync with caller-owned scratch, through the C ABI."""
import ctypes

import numpy as np
import pytest
import torch

from gpu_util import device

pytestmark = pytest.mark.gpu


def _inputs(K, P, seed, ef):
    g = torch.Generator().manual_seed(seed)
    ws = torch.randn(P, generator=g)
    W = ws[None] + 1e-3 * torch.randn(K, P, generator=g)
    W[:, ::17] = ws[::17]          # exact zeros in the differences
    E = 1e-4 * torch.randn(K, P, generator=g) if ef else None
    dev = device()
    return (W.to(dev), ws.to(dev), None if E is None else E.to(dev))


@pytest.mark.parametrize("ef", [False, True])
def test_static_scratch_sign_sync_matches_the_allocating_entry_point(ef):
    """Two calls in a row (the second on a smaller problem, which reuses the
    array the first one filled): replicas, the synchronised model and the
    error memories bit-identical to the entry point with its own scratch."""
    from paper_1808_07217_amd import lsgd as L
    for K, P, seed in ((16, 1841164, 1), (5, 30004, 2)):
        print(f"static sign sync ef={ef} K={K} P={P}", flush=True)
        W, ws, E = _inputs(K, P, seed, ef)
        W2, ws2 = W.clone(), ws.clone()
        E2 = None if E is None else E.clone()
        L.replica_sign_sync(W, ws, E)
        L.replica_sign_sync_static(W2, ws2, E2)
        torch.cuda.synchronize()
        assert torch.equal(W, W2) and torch.equal(ws, ws2)
        if ef:
            assert torch.equal(E, E2)
        # the replicas all hold the new synchronised model
        assert torch.equal(W2[0], ws2) and torch.equal(W2[-1], ws2)


def test_static_scratch_refuses_problems_beyond_its_size():
    """A problem whose scratch exceeds the static array is refused with
    LSGD_E_WORKSPACE before any launch; bad sizes with LSGD_E_INVALID."""
    from paper_1808_07217_amd import lsgd as L
    lib = L._lib
    nb = ctypes.c_size_t()
    K, P = 64, 1 << 21
    assert lib.lsgd_sign_sync_scratch_bytes(K, P, ctypes.byref(nb)) == 0
    assert nb.value > (16 << 20)
    fake = ctypes.c_void_p(256)
    assert lib.lsgd_replica_sign_sync_static(fake, K, P, fake, None, None) == 2
    assert lib.lsgd_replica_sign_sync_static(fake, 4, 6, fake, None, None) == 1
    assert lib.lsgd_replica_sign_sync_static(None, 4, 8, fake, None, None) == 1
