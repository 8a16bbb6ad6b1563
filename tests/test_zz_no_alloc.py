"""The allocation-free loss entry point (grpo_token_loss_noalloc) against
grpo_token_loss on the same inputs: two calls in a row, the second smaller
(the static scratch keeps the first call's contents), both bit-identical to
the workspace entry point (same kernels) and within 1e-5 relative of the
oracle; sizes above the static maximum rejected before any work."""
import numpy as np
import pytest
import torch

import oracle
from paper_2510_17158_amd import api

from gpu_util import require_gpu, say

pytestmark = pytest.mark.gpu


def _inputs(N, Tr, seed):
    rng = np.random.default_rng(seed)
    lp = (rng.standard_normal((N, Tr)) * 0.5 - 2.0).astype(np.float32)
    lo = (lp + rng.standard_normal((N, Tr)) * 0.2).astype(np.float32)
    lr = (lp + rng.standard_normal((N, Tr)) * 0.1).astype(np.float32)
    mask = (rng.random((N, Tr)) < 0.8).astype(np.uint8)
    mask[0, :] = 0                                  # a sequence with no trained token
    adv = rng.standard_normal(N).astype(np.float32)
    return lp, lo, lr, mask, adv


@pytest.mark.parametrize("agg", [0, 1])
def test_noalloc_matches_workspace_entry_point(agg):
    require_gpu()
    for N, Tr, seed in ((64, 2048, 1), (24, 700, 2)):     # second call smaller
        say("no-alloc loss", N, Tr, "agg", agg)
        h = _inputs(N, Tr, seed)
        d = [torch.from_numpy(a).cuda() for a in h]
        outs = []
        for noalloc in (False, True):
            loss = torch.full((1,), float("nan"), device="cuda")
            tl = torch.full((N, Tr), float("nan"), device="cuda")
            dl = torch.full((N, Tr), float("nan"), device="cuda")
            st = torch.full((4,), float("nan"), device="cuda")
            if noalloc:
                api.token_loss_noalloc(*d, 0.2, 0.04, agg, loss, tl, dl, st)
            else:
                ws = api.alloc_workspace(None, api.OP_LOSS, N, Tr)
                api.token_loss(*d, 0.2, 0.04, agg, loss, tl, dl, st, ws=ws)
            torch.cuda.synchronize()
            outs.append([t.cpu().numpy() for t in (loss, tl, dl, st)])
        for a, b in zip(*outs):
            np.testing.assert_array_equal(a, b)
        ref = oracle.token_loss(*[a.astype(np.float64) if a.dtype == np.float32 else a
                                  for a in h], 0.2, 0.04, agg=agg)
        got = float(outs[1][0][0])
        assert abs(got - ref["loss"]) <= 1e-5 * abs(ref["loss"]) + 1e-7, (got, ref["loss"])


def test_noalloc_rejects_sizes_above_the_static_maximum():
    require_gpu()
    N = 16385
    d = [torch.zeros(N, 1, device="cuda") for _ in range(3)]
    mask = torch.ones(N, 1, dtype=torch.uint8, device="cuda")
    adv = torch.zeros(N, device="cuda")
    loss = torch.zeros(1, device="cuda")
    with pytest.raises(api.GrpoError) as e:
        api.token_loss_noalloc(*d, mask, adv, 0.2, 0.04, 0, loss)
    assert e.value.code == api.INVALID_ARG and "static scratch" in str(e.value)
