"""zo_subspace_refresh_noalloc (static per-GPU scratch, no allocation) against
zo_subspace_refresh (caller workspace) on the same panels: the two run the same
kernels in the same order, so Q, diag(R) and info must agree bit for bit.  Two
calls in a row, the second smaller than the first (the scratch then holds the
first call's partial results, which must not be read)."""
import numpy as np
import pytest
import torch

import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import dev_f32, host

pytestmark = pytest.mark.gpu


def _panels(seed, rows_list, r):
    return [zd.f32(zd.draw(seed, "OMEGA_V", (i, rows, r), (rows, r))) for i, rows in enumerate(rows_list)]


def _both(panels, r):
    om = [dev_f32(p) for p in panels]
    rd_a = [torch.empty(r, dtype=torch.float32, device="cuda") for _ in om]
    rd_b = [torch.empty(r, dtype=torch.float32, device="cuda") for _ in om]
    info_a = torch.full((len(om),), -7, dtype=torch.int32, device="cuda")
    info_b = torch.full((len(om),), -7, dtype=torch.int32, device="cuda")
    qa = zo.subspace_refresh(om, r, r_diag=rd_a, info=info_a)
    qb = [torch.full_like(o, float("nan")) for o in om]
    zo.subspace_refresh_noalloc(om, r, qb, r_diag=rd_b, info=info_b)
    torch.cuda.synchronize()
    for a, b in zip(qa + rd_a, qb + rd_b):
        np.testing.assert_array_equal(host(a).view(np.uint32), host(b).view(np.uint32))
    np.testing.assert_array_equal(info_a.cpu().numpy(), info_b.cpu().numpy())
    assert np.all(info_b.cpu().numpy() == 0)
    Q = host(qb[0])
    assert np.abs(Q.T @ Q - np.eye(r)).max() <= 1e-6


@pytest.mark.parametrize("r,first,second", [
    (64, [20480, 5120, 5120, 20480], [4096, 300]),   # OPT-13B-shaped panels, then smaller ones
    (128, [20480, 5120], [2049]),                    # the wide (64 < r <= 128) kernels
    (4, [27648, 5120, 1024, 8], [256, 8]),           # Qwen LoRA factor panels, then the Tiny ones
])
def test_noalloc_matches_workspace_refresh(r, first, second):
    _both(_panels(1, first, r), r)
    _both(_panels(2, second, r), r)


def test_noalloc_rejects_oversized_call():
    r = 64
    # 4M rows: 2048 row chunks of one 64 x 64 float64 partial each (64 MiB) plus the panel's rest.
    om = torch.empty((1 << 22, r), dtype=torch.float32, device="cuda")
    out = torch.empty_like(om)
    with pytest.raises(zo.ZoError, match="static scratch"):
        zo.subspace_refresh_noalloc([om], r, [out])
