"""Parity of the loss helpers (zo_sq_loss, zo_combine_central, zo_combine_forward) with the
oracle, for every output type the perturbed linear produces (fp32, bf16, fp16).

The device loss reads the exact 16-bit values and reduces in float64, so it matches the
oracle's float64 sum of the same values to rounding order (relative 1e-12); the estimates
divide float64 losses and round once to fp32.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import dev_bf16, dev_f16, dev_f32, host

pytestmark = pytest.mark.gpu


def values(a64, dt):
    if dt == "bf16":
        bits, v = zd.as_bf16_values(a64)
        return dev_bf16(bits), v
    if dt == "f16":
        h, v = zd.as_f16_values(a64)
        return dev_f16(h), v
    v = zd.f32(a64).astype(np.float64)
    return dev_f32(v), v


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("nblk,T,m", [(8, 64, 256), (3, 37, 50), (2, 300, 1024), (1, 1, 8)])
def test_sq_loss_parity(dt, nblk, T, m):
    Yd, Yv = values(zd.draw(5, "X", (nblk, T, m), (nblk * T, m)), dt)
    Sd, Sv = values(zd.draw(5, "WSTAR", (T, m), (T, m)), dt)
    L = host(zo.sq_loss(Yd, Sd, nblk, T))
    torch.cuda.synchronize()
    ref = np.array([oracle.sq_loss(Yv[b * T:(b + 1) * T], Sv) for b in range(nblk)])
    np.testing.assert_allclose(L, ref, rtol=1e-12, atol=0)


@pytest.mark.parametrize("q", [1, 4, 100])
def test_estimates_parity(q):
    Lc = 6.0 + zd.draw(6, "G", (q, 1), (2 * q,), 1e-4)
    eps = float(np.float32(1e-3))
    g = host(zo.combine_central(torch.from_numpy(Lc).cuda(), eps))
    ref = oracle.central_estimate(Lc[0::2], Lc[1::2], eps)
    np.testing.assert_array_equal(g, ref.astype(np.float32).astype(np.float64))
    Lf = 6.0 + zd.draw(6, "G", (q, 2), (q + 1,), 1e-4)
    g = host(zo.combine_forward(torch.from_numpy(Lf).cuda(), eps))
    ref = oracle.forward_estimate(Lf[1:], Lf[0], eps)
    np.testing.assert_array_equal(g, ref.astype(np.float32).astype(np.float64))
