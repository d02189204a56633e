"""Parity of zo_lora_perturbed_linear (HIP) with the float64 oracle (LoRA scheme: both
adapter factors perturbed in their own subspaces, Eq. 4 / Alg. 2 per trainable matrix).

The oracle materialises A', B' and W + scale B' A'; the GPU never does.  Bars as
for the full-tuning layer: fp32 paths e(., ., 1) <= 1e-5; bf16 outputs
e(., ., 1e-3) <= 1e-2 and normwise <= 1e-2.  At the paper's initialisation
(B = 0) and eps = 1e-3 the adapter branch is far below bf16 resolution of Y,
so the branch is also checked through fp32 outputs with X shared by the +/-
blocks, and at eps = 1 with a non-zero B.
"""
import hashlib

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import dev_bf16, dev_f16, dev_f32, ferr, host, normwise, orth

pytestmark = pytest.mark.gpu

SCALE = zd.QWEN_LORA_ALPHA / zd.QWEN_LORA_RANK


def make_case(T, m, n, rl, r, q, nblk, shared_x, bf16, zero_b=False, seed=0, same_x_pairs=False, f16=False):
    """The frozen base W and X are bf16 (bf16=True), fp16 (f16=True) or fp32."""
    W64 = zd.draw(seed, "W0", (m, n), (m, n), 0.02)
    X0 = zd.draw(seed, "X", (T, n, 0), (T, n))
    if f16:
        Wh, Wv = zd.as_f16_values(W64)
        X0h, X0v = zd.as_f16_values(X0)
        Wd, X0d = dev_f16(Wh), dev_f16(X0h)
    elif bf16:
        Wb, Wv = zd.as_bf16_values(W64)
        X0b, X0v = zd.as_bf16_values(X0)
        Wd, X0d = dev_bf16(Wb), dev_bf16(X0b)
    else:
        Wv = zd.f32(W64).astype(np.float64)
        X0v = zd.f32(X0).astype(np.float64)
        Wd, X0d = dev_f32(Wv), dev_f32(X0v)
    step = T // nblk
    if shared_x:
        shift = [0] * nblk
        Xd, xs = X0d, 0
    else:
        shift = [(b // 2 if same_x_pairs else b) * step for b in range(nblk)]
        Xd, xs = torch.cat([torch.roll(X0d, sh, 0) for sh in shift]).contiguous(), T * n
    A = zd.f32(zd.draw(seed, "LORA_A", (m, n), (rl, n), 0.02))
    B = np.zeros((m, rl), np.float32) if zero_b else zd.f32(zd.draw(seed, "LORA_B", (m, n), (m, rl), 0.02))
    UA, VA = orth(seed, (11, rl, n), rl, r), orth(seed, (12, rl, n), n, r)
    UB, VB = orth(seed, (13, m, rl), m, r), orth(seed, (14, m, rl), rl, r)
    ZA = np.stack([zd.f32(zd.draw(seed, "Z", (0, j, 1), (r, r))) for j in range(q)])
    ZB = np.stack([zd.f32(zd.draw(seed, "Z", (0, j, 2), (r, r))) for j in range(q)])
    bq = [b // 2 % q for b in range(nblk)]
    bs = [1 if b % 2 == 0 else -1 for b in range(nblk)]
    host_f = dict(A=A, UA=UA, VA=VA, ZA=ZA, B=B, UB=UB, VB=VB, ZB=ZB)
    dev = {k: dev_f32(v) for k, v in host_f.items()}
    return dict(T=T, m=m, n=n, rl=rl, r=r, q=q, nblk=nblk, Wv=Wv, X0v=X0v, shift=shift, bq=bq, bs=bs,
                Wd=Wd, Xd=Xd, xs=xs, h={k: v.astype(np.float64) for k, v in host_f.items()}, d=dev)


def xblock(c, b, rows=None):
    T = c["T"]
    idx = np.arange(T) if rows is None else np.asarray(rows)
    return c["X0v"][(idx - c["shift"][b]) % T]


def layer(c, eps, out_dtype=None):
    d = c["d"]
    return zo.LoraPerturbedLinear(c["Xd"], c["Wd"], d["A"], d["UA"], d["VA"], d["ZA"], d["B"], d["UB"], d["VB"],
                                  d["ZB"], c["bq"], c["bs"], eps, SCALE, c["T"], x_block_stride=c["xs"],
                                  out_dtype=out_dtype)


def run_gpu(c, eps, out_dtype=None):
    Y = layer(c, eps, out_dtype)()
    torch.cuda.synchronize()
    return host(Y).reshape(c["nblk"], c["T"], c["m"])


def run_oracle(c, eps, blocks=None, rows=None):
    h = c["h"]
    blocks = range(c["nblk"]) if blocks is None else blocks
    out = []
    for b in blocks:
        out += oracle.lora_perturbed_linear_blocks([xblock(c, b, rows)], c["Wv"], h["A"], h["UA"], h["VA"], h["ZA"],
                                                   h["B"], h["UB"], h["VB"], h["ZB"], [c["bq"][b]], [c["bs"][b]],
                                                   eps, SCALE)
    return out


@pytest.mark.parametrize("T,m,n,rl,r,q,nblk,shared,zero_b", [
    (64, 256, 512, 8, 4, 4, 8, True, False),     # Tiny-sized layer, shared X
    (37, 50, 70, 3, 2, 3, 6, False, False),      # ragged everything
    (1, 3, 1, 1, 1, 1, 1, False, False),         # degenerate sizes
    (130, 72, 300, 8, 4, 2, 4, False, True),     # B = 0 (paper initialisation)
])
def test_fp32_parity(T, m, n, rl, r, q, nblk, shared, zero_b):
    c = make_case(T, m, n, rl, r, q, nblk, shared, bf16=False, zero_b=zero_b)
    Y = run_gpu(c, 1e-3)
    ref = run_oracle(c, 1e-3)
    for b in range(nblk):
        assert ferr(Y[b], ref[b], 1.0) <= 1e-5, b


@pytest.mark.parametrize("T,m,n,rl,r,q,nblk,shared,zero_b", [
    (300, 264, 200, 8, 4, 2, 4, False, False),   # ragged token, column and K tails
    (256, 1024, 512, 8, 4, 4, 8, False, True),   # v-projection-like m, B = 0
    (96, 520, 136, 16, 8, 3, 6, True, False),    # wider adapter, shared X
    (8, 8, 8, 1, 1, 1, 2, False, False),         # smallest legal bf16 shape
])
@pytest.mark.parametrize("out", ["bf16", "f32"])
def test_bf16_parity(T, m, n, rl, r, q, nblk, shared, zero_b, out):
    c = make_case(T, m, n, rl, r, q, nblk, shared, bf16=True, zero_b=zero_b)
    Y = run_gpu(c, 1e-3, out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = run_oracle(c, 1e-3)
    for b in range(nblk):
        assert ferr(Y[b], ref[b], 1e-3) <= 1e-2, b
        assert normwise(Y[b], ref[b]) <= 1e-2, b
        if out == "f32":
            assert ferr(Y[b], ref[b], 1.0) <= 1e-4, b


@pytest.mark.parametrize("T,m,n,rl,r,q,nblk,shared,zero_b", [
    (300, 264, 200, 8, 4, 2, 4, False, False),   # ragged tails (generic tile kernel)
    (256, 1024, 512, 8, 4, 4, 8, False, True),   # v-projection-like m, B = 0 (main kernel)
    (96, 520, 136, 16, 8, 3, 6, True, False),    # wider adapter, shared X
])
@pytest.mark.parametrize("out", ["f16", "f32"])
def test_f16_parity(T, m, n, rl, r, q, nblk, shared, zero_b, out):
    """fp16 frozen base (the paper's precision for its LoRA runs)."""
    c = make_case(T, m, n, rl, r, q, nblk, shared, bf16=False, zero_b=zero_b, f16=True)
    Y = run_gpu(c, 1e-3, out_dtype=torch.float16 if out == "f16" else torch.float32)
    ref = run_oracle(c, 1e-3)
    for b in range(nblk):
        assert ferr(Y[b], ref[b], 1e-3) <= 1e-2, b
        assert normwise(Y[b], ref[b]) <= 2e-3, b
        if out == "f32":
            assert ferr(Y[b], ref[b], 1.0) <= 1e-4, b


def test_bf16_eps_one_adapter_visible():
    """At eps = 1 with a non-zero B the adapter branch and both perturbations are large enough
    to be checked through bf16 outputs."""
    c = make_case(200, 128, 256, 8, 4, 2, 4, False, bf16=True)
    Y = run_gpu(c, 1.0)
    ref = run_oracle(c, 1.0)
    h = c["h"]
    for b in range(4):
        base = xblock(c, b) @ (c["Wv"] + SCALE * h["B"] @ h["A"]).T
        assert normwise(Y[b], ref[b]) <= 1e-2
        assert normwise(base, ref[b]) > 5e-2


@pytest.mark.parametrize("zero_b", [True, False])
@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_adapter_channel_fp32_out(zero_b, dt):
    """X_{2j} = X_{2j+1}: (Y+ - Y-)/(2 eps) is the odd part of the branch,
    scale X [(U_A Z_A V_A^T)^T B^T + A^T (U_B Z_B V_B^T)^T], which a kernel that dropped or
    mis-signed either perturbation would fail (it is below 16-bit resolution of Y)."""
    T, m, n, rl, r, q = 256, 256, 512, 8, 4, 3
    c = make_case(T, m, n, rl, r, q, 2 * q, False, bf16=dt == "bf16", zero_b=zero_b, same_x_pairs=True,
                  f16=dt == "f16")
    eps = 1e-3
    Y = run_gpu(c, eps, out_dtype=torch.float32)
    h = c["h"]
    for j in range(q):
        X = xblock(c, 2 * j)
        PA = h["UA"] @ h["ZA"][j] @ h["VA"].T
        PB = h["UB"] @ h["ZB"][j] @ h["VB"].T
        odd = SCALE * X @ (h["B"] @ PA + PB @ h["A"]).T
        d = (Y[2 * j] - Y[2 * j + 1]) / (2 * eps)
        assert normwise(d, odd) <= 1e-2, j
        assert ferr(d, odd, 1e-1) <= 5e-2, j


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_frozen_tensors_bitwise_unchanged(dt):
    c = make_case(128, 256, 256, 8, 4, 4, 8, False, bf16=dt == "bf16", f16=dt == "f16")
    hs = lambda t: hashlib.sha256(t.contiguous().view(torch.int16 if t.element_size() == 2 else torch.int32)
                                  .cpu().numpy().tobytes()).hexdigest()
    before = [hs(c["Wd"]), hs(c["d"]["A"]), hs(c["d"]["B"])]
    for _ in range(3):
        run_gpu(c, 1e-3)
    assert before == [hs(c["Wd"]), hs(c["d"]["A"]), hs(c["d"]["B"])]


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
def test_prepare_apply_equals_one_call(dt):
    c = make_case(300, 264, 200, 8, 4, 2, 4, False, bf16=dt == "bf16", f16=dt == "f16")
    one = run_gpu(c, 1e-3)
    pl = layer(c, 1e-3)
    pl.prepare()
    Y = pl.apply()
    torch.cuda.synchronize()
    assert np.array_equal(host(Y).reshape(one.shape), one)


@pytest.mark.parametrize("name", ["q", "v"])
@pytest.mark.parametrize("zero_b", [True, False])
def test_qwen32b_lora_full_size_sampled(name, zero_b):
    """The adapted projections of the Qwen-32B-shaped stack at full size (T = 4096, q = 4,
    8 blocks, r_L = 8, r = 4); sampled token rows checked against the oracle row by row."""
    cfg = zd.CONFIGS["qwen-32b-lora"]
    m, n = {"q": (5120, 5120), "v": (1024, 5120)}[name]
    T, q = cfg["T"], cfg["q"]
    nblk = 2 * q
    c = make_case(T, m, n, zd.QWEN_LORA_RANK, cfg["r"], q, nblk, False, bf16=True, zero_b=zero_b)
    Y = layer(c, 1e-3)()
    torch.cuda.synchronize()
    rows = np.array([0, 1, 255, 256, T // 2 + 1, T - 1])
    Yh = Y.view(nblk, T, m)
    for b in [0, 1, nblk - 1]:
        got = host(Yh[b][torch.from_numpy(rows).cuda()])
        ref = run_oracle(c, 1e-3, blocks=[b], rows=rows)[0]
        assert ferr(got, ref, 1e-3) <= 1e-2, b
        assert normwise(got, ref) <= 1e-2, b


def test_adapter_factor_update():
    """The LoRA factors are fp32 trainable matrices: one subspace Adam step on A (r_L x n) and
    B (m x r_L) with their own subspaces, sharing the q global estimates (Eqs. 6-10)."""
    m, n, rl, r, q = 1024, 5120, 8, 4, 4
    c = make_case(8, m, n, rl, r, q, 2, False, bf16=False)
    h, d = c["h"], c["d"]
    g = zd.f32(zd.draw(3, "G", (1,), (q,), 1e-2))
    items, refs = [], []
    for W, U, V, Z in ((h["A"], h["UA"], h["VA"], h["ZA"]), (h["B"], h["UB"], h["VB"], h["ZB"])):
        M1 = zd.f32(zd.draw(3, "MOM", W.shape + (1,), (r, r), 0.1))
        M2 = zd.f32(np.abs(zd.draw(3, "MOM", W.shape + (2,), (r, r), 0.01)))
        items.append(dict(W=dev_f32(W), U=dev_f32(U), V=dev_f32(V), Z=dev_f32(Z), M1=dev_f32(M1), M2=dev_f32(M2)))
        refs.append(oracle.subspace_adam_update(W, U, V, Z, g.astype(np.float64), M1, M2, 2,
                                                float(np.float32(1e-2)), float(np.float32(0.9)),
                                                float(np.float32(0.95)), float(np.float32(1e-8))))
    zo.subspace_adam_update(items, dev_f32(g), 2, 1e-2, 0.9, 0.95, 1e-8)
    torch.cuda.synchronize()
    for it, ref in zip(items, refs):
        assert ferr(host(it["W"]), ref["W"], 1.0) <= 1e-5
        np.testing.assert_allclose(host(it["M1"]), ref["M1"], rtol=1e-6, atol=1e-12)
        np.testing.assert_allclose(host(it["M2"]), ref["M2"], rtol=1e-6, atol=1e-14)
