"""Parity of zo_subspace_refresh (HIP TSQR) with the oracle's Haar QR (Eq. 11, Alg. 1).

The sign-corrected thin Q is unique, so every column must agree in sign with the
oracle's (a bitwise decision), the values to e(., ., 1) <= 1e-5, and the output
must be orthonormal to 1e-6 with a positive R diagonal.
"""
import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import dev_f32, ferr, host

pytestmark = pytest.mark.gpu


def run(panels_np, r, inplace=False):
    om = [dev_f32(p) for p in panels_np]
    out = om if inplace else None
    rd = [torch.empty(r, dtype=torch.float32, device="cuda") for _ in om]
    info = torch.full((len(om),), -7, dtype=torch.int32, device="cuda")
    qs = zo.subspace_refresh(om, r, out=out, r_diag=rd, info=info)
    torch.cuda.synchronize()
    return [host(q) for q in qs], [host(d) for d in rd], info.cpu().numpy()


def check(Q, rd, Om):
    U, R, bad = oracle.haar_qr(Om.astype(np.float64))
    assert bad == -1
    r = Q.shape[1]
    dots = np.einsum("ij,ij->j", Q, U)
    assert np.all(dots > 0), "column sign decision differs from the oracle"
    assert ferr(Q, U, 1.0) <= 1e-5
    assert np.abs(Q.T @ Q - np.eye(r)).max() <= 1e-6
    assert np.all(rd > 0)
    np.testing.assert_allclose(rd, np.diag(R), rtol=1e-5)


@pytest.mark.parametrize("rows,r", [
    (256, 4), (512, 4),                  # Tiny
    (2048, 16), (8192, 16),              # OPT-1.3B
    (4096, 32), (11008, 32),             # LLaMA-7B
    (5120, 64), (20480, 64),             # OPT-13B
    (8, 4), (27648, 4),                  # Qwen LoRA factors
    (64, 64), (65, 64), (257, 64), (300, 37), (1, 1), (1025, 3),
    (5120, 128), (20480, 128),           # the paper's full-tuning rank at OPT-13B sizes
    (128, 128), (65, 65), (300, 100), (1025, 96), (2049, 72), (4096, 24),
])
def test_refresh_parity(rows, r):
    Om = zd.f32(zd.draw(0, "OMEGA_U", (rows, r), (rows, r)))
    Q, rd, info = run([Om], r)
    assert info[0] == 0
    check(Q[0], rd[0], Om)


def test_refresh_batched_mixed_rows_inplace():
    r = 16
    rows = [16, 100, 2048, 4097, 333] * 8  # 40 panels: more than one launch holds
    Oms = [zd.f32(zd.draw(1, "OMEGA_V", (i,), (rw, r))) for i, rw in enumerate(rows)]
    Q, rd, info = run(Oms, r, inplace=True)
    assert np.all(info == 0)
    for q, d, om in zip(Q, rd, Oms):
        check(q, d, om)


def test_refresh_batched_wide_rank():
    """r = 128 over 50 panels of mixed rows (two launches of the wide kernels)."""
    r = 128
    rows = [128, 300, 2048, 1100, 129] * 10
    Oms = [zd.f32(zd.draw(4, "OMEGA_V", (i,), (rw, r))) for i, rw in enumerate(rows)]
    Q, rd, info = run(Oms, r, inplace=True)
    assert np.all(info == 0)
    for q, d, om in zip(Q, rd, Oms):
        check(q, d, om)


@pytest.mark.parametrize("r,zero_col", [(6, 3), (128, 70), (100, 0)])
def test_refresh_rank_deficient_flag(r, zero_col):
    Om = zd.f32(zd.draw(2, "OMEGA_U", (0,), (500, r)))
    Om[:, zero_col] = 0.0
    Q, rd, info = run([Om], r)
    assert info[0] == zero_col + 1  # first zero diagonal at that column
    assert rd[0][zero_col] == 0.0
    assert np.all(Q[0][:, zero_col] == 0.0)
    # The other columns are the Haar factor of the panel without that column.
    keep = [c for c in range(r) if c != zero_col]
    U, R, bad = oracle.haar_qr(np.delete(Om, zero_col, axis=1).astype(np.float64))
    assert bad == -1
    assert ferr(Q[0][:, keep], U, 1.0) <= 1e-5
    np.testing.assert_allclose(rd[0][keep], np.diag(R), rtol=1e-5)


@pytest.mark.parametrize("rows,r", [(5120, 64), (5120, 128)])
def test_refresh_deterministic(rows, r):
    Om = zd.f32(zd.draw(3, "OMEGA_U", (0,), (rows, r)))
    a = run([Om], r)[0][0]
    b = run([Om], r)[0][0]
    assert np.array_equal(a, b)


@pytest.mark.parametrize("seed", [0, 42])
def test_haar_ks_on_gpu(seed):
    """Appendix Haar validation setup (m = 50, r = 10, 2000 trials) through the GPU path:
    the first coordinate of the first column follows the exact Haar marginal."""
    m, r, n = 50, 10, 2000
    Oms = [zd.f32(zd.draw(seed, "OMEGA_U", (99999, i), (m, r))) for i in range(n)]
    Q, _, info = run(Oms, r)
    assert np.all(info == 0)
    x = np.array([q[0, 0] for q in Q])
    cdf = lambda v: 0.5 + 0.5 * np.sign(v) * scipy.special.betainc(0.5, (m - 1) / 2.0, v * v)
    ks = scipy.stats.kstest(x, cdf)
    assert ks.pvalue > 0.05, ks
