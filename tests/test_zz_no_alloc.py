"""The allocation-free weighted CE (dflare_weighted_ce_noalloc) against the entry point
with a caller workspace (dflare_weighted_ce), through the C ABI: two calls in a row, the
second with a smaller input, each bitwise equal to the workspace call on the same input
(the same kernels in the same order), and the first also within the oracle's bar."""
import numpy as np
import pytest
import torch

from oracle import training_oracle as tr
from paper_2606_02091_amd import dflare as dfl
import parity as P

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("needs a GPU", allow_module_level=True)


def _inputs(n_blocks, V, B, seed):
    rng = np.random.default_rng(seed)
    z = (3.0 * rng.standard_normal((n_blocks * B, V))).astype(np.float32)
    y = rng.integers(0, V, size=n_blocks * B).astype(np.int32)
    y[rng.random(n_blocks * B) < 0.1] = -1
    return z, y


@pytest.mark.parametrize("V", [1000, 151936])
def test_noalloc_weighted_ce_matches_workspace_entry(V):
    B, gamma = 16, 4.5
    print(f"[no_alloc] weighted CE V={V}", flush=True)
    for call, n_blocks in enumerate((9, 3)):  # the second call is smaller
        z, y = _inputs(n_blocks, V, B, seed=20 + call)
        zt, yt = torch.from_numpy(z).cuda(), torch.from_numpy(y).cuda()
        rows = n_blocks * B
        loss = torch.full((1,), float("nan"), device="cuda")
        ce = torch.full((rows,), float("nan"), device="cuda")
        dz = torch.full((rows, V), float("nan"), device="cuda")
        dfl.weighted_ce_noalloc(zt, yt, B, gamma, loss, ce, dz)
        rloss, rce, rdz = dfl.weighted_ce(zt, yt, B, gamma)
        torch.cuda.synchronize()
        assert torch.equal(loss, rloss), (call, loss, rloss)
        assert torch.equal(ce, rce), call
        assert torch.equal(dz, rdz), call
        if call == 0:
            oloss, oce, odz = tr.weighted_ce(z.astype(np.float64), y, B, gamma)
            assert abs(float(loss.cpu()[0]) - oloss) <= 1e-5 * max(1.0, abs(oloss))
            assert P.relinf(ce.cpu().numpy(), oce) <= 1e-5
            assert P.relinf(dz.cpu().numpy(), odz) <= 1e-5


def test_noalloc_weighted_ce_rejects_more_rows_than_its_scratch():
    B, V = 16, 64
    rows = dfl.WEIGHTED_CE_NOALLOC_MAX_ROWS + B
    z = torch.zeros((rows, V), device="cuda")
    y = torch.zeros(rows, dtype=torch.int32, device="cuda")
    loss = torch.zeros(1, device="cuda")
    ce = torch.zeros(rows, device="cuda")
    with pytest.raises(dfl.DFlareError) as ei:
        dfl.weighted_ce_noalloc(z, y, B, 4.5, loss, ce, z)
    assert ei.value.status == dfl.ERR_INVALID_ARG
