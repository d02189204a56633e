"""Parity of zo_perturbed_linear (HIP) with the float64 oracle (Eq. 4 in the forward of Eq. 5).

The oracle materialises W + s eps U Z V^T; the GPU never does.  Tolerances
(floored relative error e(a, b, tau) = max |a-b| / max(|b|, tau rms(b))):
fp32 paths e(., ., 1) <= 1e-5; bf16 outputs e(., ., 1e-3) <= 1e-2 and
normwise <= 1e-2 (bf16 rounding of the output alone reaches 2^-9 relative);
fp16 outputs the same floored bar and normwise <= 2e-3 (fp16 rounding is
2^-11); 16-bit inputs with fp32 outputs e(., ., 1) <= 1e-4.
"""
import hashlib

import numpy as np
import pytest
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import cast, dev_bf16, dev_f16, dev_f32, ferr, host, normwise, orth

pytestmark = pytest.mark.gpu


def make_case(T, m, n, r, q, nblk, shared_x, bf16, seed=0, wsig=0.02, f16=False):
    """Inputs on host (exact float64 values the GPU receives) and on device; W and X are
    bf16 (bf16=True), fp16 (f16=True) or fp32.

    Block b's activations are the base block X0 with its rows rolled by
    b * floor(T / nblk) (zd.block_roll_rows); the stacked device tensor is built
    with the same roll on the device so the host keeps only X0.
    """
    W64 = zd.draw(seed, "W0", (m, n), (m, n), wsig)
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
        Xd, xs = X0d, 0
    else:
        Xd, xs = torch.cat([torch.roll(X0d, b * step, 0) for b in range(nblk)]).contiguous(), T * n
    U = orth(seed, (1, m, r), m, r)
    V = orth(seed, (2, n, r), n, r)
    Z = zd.z_draws(seed, 0, 0, q, r)
    bq = [b // 2 % q for b in range(nblk)]
    bs = [1 if b % 2 == 0 else -1 for b in range(nblk)]
    shift = [0 if shared_x else b * step for b in range(nblk)]
    return dict(T=T, m=m, n=n, r=r, q=q, nblk=nblk, Wv=Wv, X0v=X0v, shift=shift, U=U, V=V, Z=Z,
                bq=bq, bs=bs, Wd=Wd, Xd=Xd, Ud=dev_f32(U), Vd=dev_f32(V), Zd=dev_f32(Z), xs=xs)


def xblock(c, b, rows=None):
    """float64 activations of block b (optionally only the given rows)."""
    T = c["T"]
    idx = np.arange(T) if rows is None else np.asarray(rows)
    return c["X0v"][(idx - c["shift"][b]) % T]


def run_gpu(c, eps, out_dtype=None):
    Y = zo.perturbed_linear(c["Xd"], c["Wd"], c["Ud"], c["Vd"], c["Zd"], c["bq"], c["bs"], eps, c["T"],
                            x_block_stride=c["xs"], out_dtype=out_dtype)
    torch.cuda.synchronize()
    return host(Y).reshape(c["nblk"], c["T"], c["m"])


def run_oracle(c, eps, blocks=None, rows=None):
    blocks = range(c["nblk"]) if blocks is None else blocks
    out = []
    for b in blocks:
        out += oracle.perturbed_linear_blocks([xblock(c, b, rows)], c["Wv"], c["U"].astype(np.float64),
                                              c["V"].astype(np.float64), c["Z"].astype(np.float64),
                                              [c["bq"][b]], [c["bs"][b]], eps)
    return out


@pytest.mark.parametrize("T,m,n,r,q,nblk,shared", [
    (64, 256, 512, 4, 4, 8, True),      # the Tiny configuration's layer
    (37, 50, 70, 5, 3, 6, False),       # ragged everything
    (1, 3, 1, 1, 1, 1, False),          # degenerate sizes
    (130, 72, 300, 20, 2, 4, True),
    (64, 200, 300, 128, 2, 4, False),   # r = 128, the paper's full-tuning rank
    (50, 100, 200, 80, 2, 4, False),    # 64 < r <= 96 (rp = 80 of a 96-column product)
])
def test_fp32_parity(T, m, n, r, q, nblk, shared):
    c = make_case(T, m, n, r, q, nblk, shared, bf16=False)
    Y = run_gpu(c, 1e-3)
    ref = run_oracle(c, 1e-3)
    for b in range(nblk):
        assert ferr(Y[b], ref[b], 1.0) <= 1e-5, b


@pytest.mark.parametrize("T,m,n,r,q,nblk,shared", [
    (300, 264, 200, 16, 2, 4, False),   # ragged token, column and K tails; several tiles
    (256, 512, 512, 64, 4, 8, False),   # exact tiles, r = 64
    (96, 520, 136, 24, 3, 6, True),     # r not a multiple of 16, shared X
    (513, 256, 1024, 4, 1, 2, False),   # one row past a tile
    (8, 8, 8, 1, 1, 1, True),           # smallest legal bf16 shape
    (192, 256, 384, 128, 2, 4, False),  # r = 128, the paper's full-tuning rank
    (100, 136, 264, 100, 3, 6, True),   # r = 100 padded to 128
    (200, 264, 256, 80, 2, 4, False),   # r = 80 padded to 96
])
@pytest.mark.parametrize("out", ["bf16", "f32"])
def test_bf16_parity(T, m, n, r, q, nblk, shared, out):
    c = make_case(T, m, n, r, q, nblk, shared, bf16=True)
    Y = run_gpu(c, 1e-3, out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = run_oracle(c, 1e-3)
    for b in range(nblk):
        assert ferr(Y[b], ref[b], 1e-3) <= 1e-2, b
        assert normwise(Y[b], ref[b]) <= 1e-2, b
        if out == "f32":
            # fp32 accumulation of exact bf16 products: far inside the bf16 bound.
            assert ferr(Y[b], ref[b], 1.0) <= 1e-4, b


@pytest.mark.parametrize("T,m,n,r,q,nblk,shared", [
    (300, 264, 200, 16, 2, 4, False),   # ragged tails; n % 32 != 0 takes the generic tile kernel
    (256, 512, 512, 64, 4, 8, False),   # exact tiles, r = 64 (the main kernel)
    (96, 520, 136, 24, 3, 6, True),     # r not a multiple of 16, shared X
    (513, 256, 1024, 4, 1, 2, False),   # one row past a tile
    (8, 8, 8, 1, 1, 1, True),           # smallest legal 16-bit shape
    (192, 256, 384, 128, 2, 4, False),  # r = 128
])
@pytest.mark.parametrize("out", ["f16", "f32"])
def test_f16_parity(T, m, n, r, q, nblk, shared, out):
    """fp16 W and X (the paper's precision): X W^T on the fp16 MFMA, the rank-r segment on bf16
    hi/lo operands, X V from the fp16 split of 256 V."""
    c = make_case(T, m, n, r, q, nblk, shared, bf16=False, f16=True)
    Y = run_gpu(c, 1e-3, out_dtype=torch.float16 if out == "f16" else torch.float32)
    ref = run_oracle(c, 1e-3)
    for b in range(nblk):
        assert ferr(Y[b], ref[b], 1e-3) <= 1e-2, b
        assert normwise(Y[b], ref[b]) <= 2e-3, b
        if out == "f32":
            assert ferr(Y[b], ref[b], 1.0) <= 1e-4, b


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_eps_one_correction_visible(dt):
    """At eps = 1 the rank-r term is large enough to be checked through 16-bit outputs."""
    c = make_case(200, 128, 256, 8, 2, 4, False, bf16=dt == "bf16", f16=dt == "f16")
    Y = run_gpu(c, 1.0)
    ref = run_oracle(c, 1.0)
    base = [xblock(c, b) @ c["Wv"].T for b in range(4)]
    for b in range(4):
        assert normwise(Y[b], ref[b]) <= 1e-2
        assert normwise(base[b], ref[b]) > 5e-2  # the correction matters at this eps


@pytest.mark.parametrize("r", [16, 128])
@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_correction_channel_fp32_out(r, dt):
    """X_{2j} = X_{2j+1}: (Y+ - Y-)/(2 eps) isolates (X V)(U Z_j)^T, which a kernel that dropped
    or mis-signed the rank-r term would fail (it is below 16-bit resolution of Y)."""
    T, m, n, q = 256, 256, 512, 3
    c = make_case(T, m, n, r, q, 2 * q, False, bf16=dt == "bf16", f16=dt == "f16")
    X0 = c["X0v"]
    c["Xd"] = torch.cat([c["Xd"][:T]] * (2 * q)).contiguous()  # block 0 (unrolled) for every block
    c["bq"] = [b // 2 for b in range(2 * q)]
    eps = 1e-3
    Y = run_gpu(c, eps, out_dtype=torch.float32)
    U, V = c["U"].astype(np.float64), c["V"].astype(np.float64)
    for j in range(q):
        d = (Y[2 * j] - Y[2 * j + 1]) / (2 * eps)
        exact = (X0 @ V) @ (U @ c["Z"][j].astype(np.float64)).T
        assert normwise(d, exact) <= 1e-2, j
        assert ferr(d, exact, 1e-1) <= 5e-2, j


def test_w_bitwise_unchanged():
    """W is read only: its bytes are identical after the 2q queries (no in-place perturb/unperturb)."""
    c = make_case(128, 256, 256, 16, 4, 8, False, bf16=True)
    h0 = hashlib.sha256(c["Wd"].view(torch.int16).cpu().numpy().tobytes()).hexdigest()
    for _ in range(3):
        run_gpu(c, 1e-3)
    h1 = hashlib.sha256(c["Wd"].view(torch.int16).cpu().numpy().tobytes()).hexdigest()
    assert h0 == h1


def test_zero_eps_is_plain_gemm():
    c = make_case(128, 256, 192, 8, 2, 4, False, bf16=True)
    Y = run_gpu(c, 0.0, out_dtype=torch.float32)
    for b in range(4):
        plain = np.matmul(xblock(c, b), c["Wv"].T)
        assert ferr(Y[b], plain, 1.0) <= 1e-4


def test_deterministic_repeat():
    c = make_case(300, 264, 200, 16, 2, 4, False, bf16=True)
    a = run_gpu(c, 1e-3)
    b = run_gpu(c, 1e-3)
    assert np.array_equal(a, b)


def _distinct_shapes(cfg):
    seen = []
    for _, m, n in cfg["mats"]:
        if (m, n) not in seen:
            seen.append((m, n))
    return seen


FULL_SIZE = [(name, m, n) for name in ("opt-1.3b", "llama-7b", "opt-13b")
             for m, n in _distinct_shapes(zd.CONFIGS[name])]


FULL_SIZE_R128 = [("opt-13b", m, n, 128, "bf16") for m, n in _distinct_shapes(zd.CONFIGS["opt-13b"])]
FULL_SIZE_R24 = [("opt-13b", m, n, 24, "bf16") for m, n in _distinct_shapes(zd.CONFIGS["opt-13b"])]
FULL_SIZE_F16 = [("opt-13b", m, n, None, "f16") for m, n in _distinct_shapes(zd.CONFIGS["opt-13b"])]


@pytest.mark.parametrize("name,m,n,rank,dt", [(*x, None, "bf16") for x in FULL_SIZE] + FULL_SIZE_R128
                         + FULL_SIZE_R24 + FULL_SIZE_F16)
def test_full_size_sampled(name, m, n, rank, dt):
    """Every distinct matrix shape of the OPT-1.3B, LLaMA-7B and OPT-13B stacks at full size
    (T tokens per block, 2q blocks, the config's r; the OPT-13B shapes also at the paper's
    full-tuning rank r = 128, at its r = 24 and in fp16, the paper's precision) in the launch
    configuration the benchmark times; sampled token rows of several blocks checked against
    the oracle row by row."""
    cfg = zd.CONFIGS[name]
    T, q = cfg["T"], cfg["q"]
    r = rank or cfg["r"]
    nblk = 2 * q
    c = make_case(T, m, n, r, q, nblk, False, bf16=dt == "bf16", f16=dt == "f16")
    Y = zo.perturbed_linear(c["Xd"], c["Wd"], c["Ud"], c["Vd"], c["Zd"], c["bq"], c["bs"], 1e-3, T,
                            x_block_stride=c["xs"])
    torch.cuda.synchronize()
    rows = np.array([0, 1, 255, 256, T // 2 + 1, T - 1])
    blocks = sorted({0, 1, nblk // 2 - 1, nblk - 1})
    Yh = Y.view(nblk, T, m)
    for b in blocks:
        got = host(Yh[b][torch.from_numpy(rows).cuda()])
        ref = run_oracle(c, 1e-3, blocks=[b], rows=rows)[0]
        assert ferr(got, ref, 1e-3) <= 1e-2, b
        assert normwise(got, ref) <= (2e-3 if dt == "f16" else 1e-2), b


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
def test_prepare_apply_equals_one_call(dt):
    """zo_perturbed_linear_prepare + zo_perturbed_linear_apply is the one-call result, bit for bit."""
    c = make_case(300, 264, 200, 16, 2, 4, False, bf16=dt == "bf16", f16=dt == "f16")
    one = run_gpu(c, 1e-3)
    pl = zo.PerturbedLinear(c["Xd"], c["Wd"], c["Ud"], c["Vd"], c["Zd"], c["bq"], c["bs"], 1e-3, c["T"],
                            x_block_stride=c["xs"])
    pl.prepare()
    Y = pl.apply()
    torch.cuda.synchronize()
    assert np.array_equal(host(Y).reshape(one.shape), one)


def test_max_blocks_and_queries():
    """ZO_MAX_BLOCKS blocks over ZO_MAX_QUERIES queries (every block's query and sign decoded
    from the per-call table), small T; every block against the oracle."""
    T, m, n, r = 16, 64, 128, 4
    nblk = zo.ZO_MAX_BLOCKS
    q = 256
    c = make_case(T, m, n, r, q, nblk, False, bf16=True)
    c["bq"] = [(7 * b) % q for b in range(nblk)]
    c["bs"] = [(1, -1, 0)[b % 3] for b in range(nblk)]
    Y = run_gpu(c, 1e-1, out_dtype=torch.float32)
    ref = run_oracle(c, 1e-1)
    for b in range(nblk):
        assert ferr(Y[b], ref[b], 1.0) <= 1e-4, b


def test_forward_difference_paper_k_full_size_sampled():
    """The paper's K = 99 queries and a baseline block at the OPT-13B shape and token count
    (nblk = 100, T = 8192: M = 819200 rows, 5120 x 5120 W, r = 64, distinct activations per
    block) in the launch configuration the benchmark's forward-difference run times; sampled
    rows of the baseline, the first, a middle and the last query block against the oracle,
    and the baseline block against the plain product."""
    cfg = zd.CONFIGS["opt-13b"]
    T, m, n, r, q = cfg["T"], 5120, 5120, cfg["r"], 99
    nblk = q + 1
    c = make_case(T, m, n, r, q, nblk, False, bf16=True)
    c["bq"] = [0] + list(range(q))
    c["bs"] = [0] + [1] * q
    Y = zo.perturbed_linear(c["Xd"], c["Wd"], c["Ud"], c["Vd"], c["Zd"], c["bq"], c["bs"], 1e-3, T,
                            x_block_stride=c["xs"])
    torch.cuda.synchronize()
    del c["Xd"]
    rows = np.array([0, 1, 255, 256, T // 2 + 1, T - 1])
    Yh = Y.view(nblk, T, m)
    for b in (0, 1, 50, 99):
        got = host(Yh[b][torch.from_numpy(rows).cuda()])
        ref = run_oracle(c, 1e-3, blocks=[b], rows=rows)[0]
        assert ferr(got, ref, 1e-3) <= 1e-2, b
        assert normwise(got, ref) <= 1e-2, b
        if b == 0:
            plain = xblock(c, 0, rows) @ c["Wv"].T
            assert ferr(got, plain, 1e-3) <= 1e-2


def test_prepare_group_rejects_shared_workspace():
    """Linears that would share one workspace (the default per-stream buffer) cannot be prepared
    as a group: each must keep its own prepared operands until its apply."""
    T, n, r, q, nblk = 64, 256, 8, 2, 4
    Xd, _ = cast(zd.draw(32, "X", (T, n), (nblk * T, n)), "bf16")
    plins = []
    for i in range(2):
        Wd, _ = cast(zd.draw(32, "W0", (i, n), (128, n), 0.05), "bf16")
        U, V, Z = orth(32, (i, 1), 128, r), orth(32, (i, 2), n, r), zd.z_draws(32, 0, i, q, r)
        plins.append(zo.PerturbedLinear(Xd, Wd, dev_f32(U), dev_f32(V), dev_f32(Z), [0, 0, 1, 1], [1, -1, 1, -1],
                                        1e-2, T, x_block_stride=T * n))
    assert plins[0].ws.data_ptr() == plins[1].ws.data_ptr()
    with pytest.raises(zo.ZoError, match="overlap"):
        zo.prepare_group(plins)


def test_forward_difference_layout_at_paper_k():
    """The paper's K = 99 queries with a baseline block (nblk = 100: block 0 unperturbed, block
    1 + k query k with sign +), as the forward estimator of Eq. 6 lays them out."""
    T, m, n, r, q = 32, 128, 256, 8, 99
    nblk = q + 1
    c = make_case(T, m, n, r, q, nblk, True, bf16=True)
    c["bq"] = [0] + list(range(q))
    c["bs"] = [0] + [1] * q
    Y = run_gpu(c, 1e-3, out_dtype=torch.float32)
    ref = run_oracle(c, 1e-3)
    for b in range(nblk):
        assert ferr(Y[b], ref[b], 1.0) <= 1e-4, b
    # the baseline block is the plain product X W^T
    np.testing.assert_allclose(Y[0], c["X0v"] @ c["Wv"].T, rtol=0, atol=1e-4 * np.abs(Y[0]).max())


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("shared", [False, True])
@pytest.mark.parametrize("T,n,r,ms", [
    (200, 264, 20, [256, 128, 72]),   # K not a multiple of 32: fp32 projection, then the combine
    (300, 512, 64, [256, 128, 72]),   # 3 x 128 stacked rows: the main GEMM, combine in its epilogue
    (260, 320, 24, [64, 200, 136]),   # 3 x 64 rows (rp = 32) on the main GEMM
    (130, 256, 40, [96, 160]),        # 2 x 128 rows: one whole 256-row tile
    (300, 320, 20, [96, 160]),        # 2 x 64 rows (rp = 32): one k_proj tile holds both factors
])
def test_prepare_group_equals_separate(dt, shared, T, n, r, ms):
    """zo_perturbed_linear_prepare_group (one projection pass for matrices that read the same X,
    of different heights) then each apply: bitwise the separate prepares and applies (a single
    16-bit factor of 64 or 128 rows projects in k_proj)."""
    q, nblk = 2, 4
    xs = 0 if shared else T * n
    Xd, _ = cast(zd.draw(31, "X", (T, n), ((1 if shared else nblk) * T, n)), dt)
    bq, bs = [b // 2 for b in range(nblk)], [1, -1] * (nblk // 2)
    plins, refs = [], []
    for i, m in enumerate(ms):
        Wd, _ = cast(zd.draw(31, "W0", (i, m, n), (m, n), 0.05), dt)
        U, V = orth(31, (i, 1, m), m, r), orth(31, (i, 2, n), n, r)
        Z = zd.z_draws(31, 0, i, q, r)
        args = (Xd, Wd, dev_f32(U), dev_f32(V), dev_f32(Z), bq, bs, 1e-2, T)
        ws = torch.empty(zo.lib().zo_perturbed_linear_workspace(T, m, n, r, q, nblk, xs, zo._lib._DT[Xd.dtype]),
                         dtype=torch.uint8, device="cuda")
        plins.append(zo.PerturbedLinear(*args, x_block_stride=xs, workspace=ws))
        ref = zo.PerturbedLinear(*args, x_block_stride=xs)
        ref.prepare()
        refs.append(ref.apply().clone())
    zo.prepare_group(plins)
    for p, ref in zip(plins, refs):
        Y = p.apply()
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.uint8), ref.view(torch.uint8))


def _epi_ref(y, epi, R):
    if epi == zo.ZO_EPI_RELU:
        return np.maximum(y, 0.0)
    if epi == zo.ZO_EPI_RESIDUAL:
        return y + R
    if epi == zo.ZO_EPI_SILU_MUL:
        return y * oracle.silu(R)
    return y


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("epi", ["none", "relu", "residual", "silu_mul"])
def test_shared_x_epilogues(dt, epi):
    """One X shared by every block (x_block_stride = 0): X W^T is computed once and each block
    adds its rank-r term (plain and ReLU epilogues), or the blocks take the per-block path
    (residual and gated epilogues, R per block).  Several tiles with ragged edges in tokens and
    output columns; every block against the oracle with the epilogue applied in float64."""
    T, m, n, r, q, nblk = 600, 520, 136, 24, 3, 6
    c = make_case(T, m, n, r, q, nblk, True, bf16=dt == "bf16", f16=dt == "f16")
    code = {"none": zo.ZO_EPI_NONE, "relu": zo.ZO_EPI_RELU, "residual": zo.ZO_EPI_RESIDUAL,
            "silu_mul": zo.ZO_EPI_SILU_MUL}[epi]
    R64 = Rd = None
    if code in (zo.ZO_EPI_RESIDUAL, zo.ZO_EPI_SILU_MUL):
        Rd, R64 = cast(zd.draw(5, "X", (T, m, 3), (nblk * T, m)), dt)
    pl = zo.PerturbedLinear(c["Xd"], c["Wd"], c["Ud"], c["Vd"], c["Zd"], c["bq"], c["bs"], 1e-3, T, x_block_stride=0)
    pl.prepare()
    Y = host(pl.apply(code, Rd)).reshape(nblk, T, m)
    ref = run_oracle(c, 1e-3)
    for b in range(nblk):
        Rb = None if R64 is None else R64.reshape(nblk, T, m)[b]
        want = _epi_ref(ref[b], code, Rb)
        assert ferr(Y[b], want, 1e-3) <= 1e-2, b
        assert normwise(Y[b], want) <= (2e-3 if dt == "f16" else 1e-2), b


@pytest.mark.parametrize("name", ["opt-13b", "llama-7b"])
def test_shared_x_full_size_sampled(name):
    """The first layer's q/k/v shape at full size with one shared X (T tokens, 2q blocks, the
    config's r), in the launch configuration the benchmark's shared-X report times; sampled token
    rows of several blocks against the oracle, and the difference of the two blocks of a query
    (the correction channel, X W^T cancels exactly) against (X V)(eps U Z_j)^T in fp32 output."""
    cfg = zd.CONFIGS[name]
    T, q, r = cfg["T"], cfg["q"], cfg["r"]
    m = n = cfg["mats"][0][1]
    nblk = 2 * q
    c = make_case(T, m, n, r, q, nblk, True, bf16=True)
    rows = np.array([0, 1, 255, 256, T // 2 + 1, T - 1])
    blocks = sorted({0, 1, nblk // 2 - 1, nblk - 1})
    for out in (None, torch.float32):
        Y = zo.perturbed_linear(c["Xd"], c["Wd"], c["Ud"], c["Vd"], c["Zd"], c["bq"], c["bs"], 1e-3, T,
                                x_block_stride=0, out_dtype=out)
        torch.cuda.synchronize()
        Yh = Y.view(nblk, T, m)
        got = {b: host(Yh[b][torch.from_numpy(rows).cuda()]) for b in blocks}
        refs = {b: run_oracle(c, 1e-3, blocks=[b], rows=rows)[0] for b in blocks}
        for b in blocks:
            if out is None:
                assert ferr(got[b], refs[b], 1e-3) <= 1e-2, b
                assert normwise(got[b], refs[b]) <= 1e-2, b
            else:
                assert ferr(got[b], refs[b], 1.0) <= 1e-4, b
        if out is not None:  # blocks 0 and 1: query 0, + and -
            d = (got[0] - got[1]) / 2e-3
            xv = xblock(c, 0, rows) @ c["V"].astype(np.float64)
            want = xv @ (c["U"].astype(np.float64) @ c["Z"][0].astype(np.float64)).T
            assert ferr(d, want, 1.0) <= 2e-2
