"""Parity of the LLaMA-family layer pieces (RMS norm, rotary positions, the SwiGLU epilogue
and the whole layer, as the network a query evaluates in the forward of Eq. 5) with the
float64 oracle.

Bars as for the pre-LN decoder layer: a 16-bit kernel output on exact 16-bit inputs is held
to the bar of one rounding (floored relative error <= 1e-2 at floor 1e-3 rms, normwise
<= 2e-3), fp32 RMS norm to 1e-5, attention to one ulp plus 2^-14 of the softmax average
of |V|.  The layer is checked stage by stage, each stage fed the
GPU's own previous output; the one-call layer is bitwise that sequence of calls; and the
end-to-end output is held against the oracle layer that rounds every stored activation to
the same type.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import cast, check16, check_attention, dev_f32, ferr, host, normwise, orth, rnd, ulp16

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ RMS norm
@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("rows,d", [(37, 96), (64, 4096), (5, 8), (300, 5120),
                                    # every register bucket, its edges, and the re-reading path
                                    (7, 1032), (6, 5128), (5, 8192), (3, 8200), (2, 11008)])
def test_rmsnorm_parity(dt, rows, d):
    Xd, Xv = cast(zd.draw(21, "X", (rows, d), (rows, d)) * 2.0 + 0.5, dt)
    g = zd.f32(1.0 + 0.1 * zd.draw(21, "W0", (d, 1), (d,)))
    Y = host(zo.rmsnorm(Xd, dev_f32(g), 1e-6))
    ref = oracle.rms_norm(Xv, g.astype(np.float64), 1e-6)
    if dt == "f32":
        assert ferr(Y, ref, 1.0) <= 1e-5
    else:
        check16(Y, ref, dt)


def test_rmsnorm_in_place_and_scale_invariance():
    """Y = RMS(X) may overwrite X; with eps = 0 and a power-of-two scale of X (exact in bf16)
    the output is the same bits."""
    Xd, _ = cast(zd.draw(22, "X", (0,), (64, 512)), "bf16")
    g = torch.ones(512, device="cuda")
    ref = zo.rmsnorm(Xd, g, 0.0)
    Xs = (Xd.float() * 8.0).to(torch.bfloat16)
    torch.testing.assert_close(zo.rmsnorm(Xs, g, 0.0).view(torch.int16), ref.view(torch.int16), rtol=0, atol=0)
    zo.rmsnorm(Xd, g, 0.0, out=Xd)
    torch.cuda.synchronize()
    assert torch.equal(Xd.view(torch.int16), ref.view(torch.int16))


# ------------------------------------------------------------------ rotary positions
@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("rows,seq_len,d,heads", [
    (128, 64, 256, 2),       # dh = 128
    (200, 100, 128, 2),      # dh = 64, sequences not a multiple of 64
    (96, 32, 240, 3),        # dh = 80: 16-multiple head dims other than 64 and 128
    (8192, 4096, 256, 2),    # positions up to 4095
    (512, 256, 4096, 32),    # the LLaMA-7B width
])
def test_rope_parity(dt, rows, seq_len, d, heads):
    Xd, Xv = cast(zd.draw(23, "X", (rows, d, heads), (rows, d)), dt)
    zo.rope(Xd, seq_len, heads)
    Y = host(Xd)
    ref = oracle.rope(Xv, seq_len, heads)
    check16(Y, ref, dt)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_rope_position_zero_is_identity(dt):
    """seq_len = 1 puts every row at position 0: cos 0 = 1, sin 0 = 0, X unchanged bit for bit."""
    Xd, _ = cast(zd.draw(24, "X", (0,), (64, 512)), dt)
    X0 = Xd.clone()
    zo.rope(Xd, 1, 4)
    torch.cuda.synchronize()
    assert torch.equal(Xd.view(torch.int16), X0.view(torch.int16))


def test_rope_other_base_and_relative_positions():
    """A non-default base, and the defining property of the rotation: the dot product of a
    rotated query at position p and a rotated key at position p' depends on p - p' only.
    Each fp16 output carries a relative rounding of at most 2^-11, so each dot product is
    within 2 * 2^-11 |q| |k| of its exact value; 6 * 2^-11 leaves room for the angles'
    fp32 errors."""
    d, heads, L = 128, 1, 64
    base = 500000.0
    q = zd.draw(25, "X", (1,), (d,))
    k = zd.draw(25, "X", (2,), (d,))
    Xq = np.tile(q, (L, 1))
    Xk = np.tile(k, (L, 1))
    Qd, Qv = cast(Xq, "f16")
    Kd, Kv = cast(Xk, "f16")
    zo.rope(Qd, L, heads, base)
    zo.rope(Kd, L, heads, base)
    Qh, Kh = host(Qd), host(Kd)
    check16(Qh, oracle.rope(Qv, L, heads, base), "q")
    check16(Kh, oracle.rope(Kv, L, heads, base), "k")
    # <R_p q, R_p' k> for (p, p') = (5, 2) and (40, 37): the same offset
    a = float(Qh[5] @ Kh[2])
    b = float(Qh[40] @ Kh[37])
    scale = float(np.linalg.norm(Qv[0]) * np.linalg.norm(Kv[0]))
    assert abs(a - b) <= 6 * 2.0 ** -11 * scale


# ------------------------------------------------------------------ SwiGLU epilogue
@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("n", [512, 200])   # the main kernel, and the generic tile kernel
@pytest.mark.parametrize("shared", [False, True])
def test_apply_silu_mul(dt, n, shared):
    T, m, r, q, nblk = 192, 256, 8, 2, 4
    Wd, Wv = cast(zd.draw(26, "W0", (m, n), (m, n), 0.05), dt)
    Xd, Xv = cast(zd.draw(26, "X", (T, n), (nblk * T, n)), dt)
    U, V = orth(26, (1, m), m, r), orth(26, (2, n), n, r)
    Z = zd.z_draws(26, 0, 0, q, r)
    bq, bs = [b // 2 for b in range(nblk)], [1, -1] * (nblk // 2)
    eps = 1e-2
    pl = zo.PerturbedLinear(Xd, Wd, dev_f32(U), dev_f32(V), dev_f32(Z), bq, bs, eps, T, x_block_stride=T * n)
    pl.prepare()
    # gate values over a few units either side of zero, where silu bends
    Gd, Gv = cast(3.0 * zd.draw(26, "WSTAR", (m,), ((1 if shared else nblk) * T, m)), dt)
    Y = host(pl.apply(zo.ZO_EPI_SILU_MUL, Gd))
    for b in range(nblk):
        lin = oracle.perturbed_linear(Xv[b * T:(b + 1) * T], Wv, U.astype(np.float64), V.astype(np.float64),
                                      Z[bq[b]].astype(np.float64), bs[b], eps)
        Gb = Gv if shared else Gv[b * T:(b + 1) * T]
        check16(Y[b * T:(b + 1) * T], oracle.silu(Gb) * lin, b)


# ------------------------------------------------------------------ the layer
def llama_case(seed, dt, d, ffn, r, q):
    shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d),
              "down": (d, ffn)}
    dev, ref = {}, {}
    for i, (nm, (m, n)) in enumerate(shapes.items()):
        Wd, Wv = cast(zd.draw(seed, "W0", (i, m, n), (m, n), 0.03), dt)
        U, V = orth(seed, (i, 1, m), m, r), orth(seed, (i, 2, n), n, r)
        Z = zd.z_draws(seed, 0, i, q, r)
        dev[nm] = dict(W=Wd, U=dev_f32(U), V=dev_f32(V), Z=dev_f32(Z))
        ref[nm] = dict(W=Wv, U=U.astype(np.float64), V=V.astype(np.float64), Z=Z.astype(np.float64))
    g1 = zd.f32(1.0 + 0.1 * zd.draw(seed, "W0", (99, 0), (d,)))
    g2 = zd.f32(1.0 + 0.1 * zd.draw(seed, "W0", (99, 1), (d,)))
    ref.update(rms1_g=g1.astype(np.float64), rms2_g=g2.astype(np.float64))
    return dev, dict(rms1_gamma=dev_f32(g1), rms2_gamma=dev_f32(g2)), ref


# ffn = 688 is not a multiple of the GEMM tiles: ragged rows of gate and up, a ragged
# reduction of down.
LL = dict(T=128, seq_len=64, r=8, q=2, nblk=4, eps=1e-2)
SHAPES = [dict(d=256, heads=2, ffn=688), dict(d=256, heads=4, ffn=512)]


def blocks():
    nblk, q = LL["nblk"], LL["q"]
    return [b // 2 % q for b in range(nblk)], [1 if b % 2 == 0 else -1 for b in range(nblk)]


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("shared", [True, False])
@pytest.mark.parametrize("shape", range(len(SHAPES)))
def test_llama_layer_stagewise_and_one_call(dt, shared, shape):
    T, L, r, q, nblk, eps = (LL[k] for k in ("T", "seq_len", "r", "q", "nblk", "eps"))
    d, heads, ffn = (SHAPES[shape][k] for k in ("d", "heads", "ffn"))
    dev, norms, ref = llama_case(31 + shape, dt, d, ffn, r, q)
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(31, "X", (T, d), ((1 if shared else nblk) * T, d)), dt)
    out = zo.LlamaLayer(dev, norms, bq, bs, eps, T, L, heads)(Hd)
    torch.cuda.synchronize()

    def lin(nm, X, xs):
        mt = dev[nm]
        p = zo.PerturbedLinear(X, mt["W"], mt["U"], mt["V"], mt["Z"], bq, bs, eps, T, x_block_stride=xs)
        p.prepare()
        return p

    def lin_ref(nm, Xv_b, b):
        mt = ref[nm]
        return oracle.perturbed_linear(Xv_b, mt["W"], mt["U"], mt["V"], mt["Z"][bq[b]], bs[b], eps)

    def rows(b):
        return slice(b * T, (b + 1) * T)

    hT = 0 if shared else T * d
    A = zo.rmsnorm(Hd, norms["rms1_gamma"], 1e-6)
    Ah = host(A)
    check16(Ah, oracle.rms_norm(Hv, ref["rms1_g"], 1e-6), "rms1")
    QKV = []
    for nm in ("q", "k", "v"):
        Y = lin(nm, A, hT).apply().clone()
        Yh = host(Y)
        for b in range(nblk):
            check16(Yh[rows(b)], lin_ref(nm, Ah if shared else Ah[rows(b)], b), (nm, b))
        if nm != "v":
            zo.rope(Y, L, heads)
            Rh = host(Y)
            for b in range(nblk):
                check16(Rh[rows(b)], oracle.rope(Yh[rows(b)], L, heads), ("rope", nm, b))
            Yh = Rh
        QKV.append((Y, Yh))
    (Qd, Qh), (Kd, Kh), (Vd, Vh) = QKV
    C = zo.causal_attention(Qd, Kd, Vd, nblk, T, L, heads)
    Ch = host(C)
    for b in range(nblk):
        check_attention(Ch[rows(b)], Qh[rows(b)], Kh[rows(b)], Vh[rows(b)], heads, L, dt, ("attn", b))
    H2 = lin("o", C, T * d).apply(zo.ZO_EPI_RESIDUAL, Hd).clone()
    H2h = host(H2)
    for b in range(nblk):
        check16(H2h[rows(b)], (Hv if shared else Hv[rows(b)]) + lin_ref("o", Ch[rows(b)], b), ("o", b))
    A2 = zo.rmsnorm(H2, norms["rms2_gamma"], 1e-6)
    A2h = host(A2)
    check16(A2h, oracle.rms_norm(H2h, ref["rms2_g"], 1e-6), "rms2")
    G = lin("gate", A2, T * d).apply().clone()
    Gh = host(G)
    for b in range(nblk):
        check16(Gh[rows(b)], lin_ref("gate", A2h[rows(b)], b), ("gate", b))
    F = lin("up", A2, T * d).apply(zo.ZO_EPI_SILU_MUL, G).clone()
    Fh = host(F)
    for b in range(nblk):
        check16(Fh[rows(b)], oracle.silu(Gh[rows(b)]) * lin_ref("up", A2h[rows(b)], b), ("up", b))
    H3 = lin("down", F, T * ffn).apply(zo.ZO_EPI_RESIDUAL, H2)
    H3h = host(H3)
    for b in range(nblk):
        check16(H3h[rows(b)], H2h[rows(b)] + lin_ref("down", Fh[rows(b)], b), ("down", b))
    # The one-call layer is exactly that sequence.
    assert torch.equal(out.view(torch.int16), H3.view(torch.int16))


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("shape", range(len(SHAPES)))
def test_llama_layer_end_to_end(dt, shape):
    """Against the oracle layer that rounds each stored activation to the same type.  As for
    the pre-LN layer, a one-ulp flip of a stored H2_i reaches output i undamped through the
    residual stream, so each output is held to one ulp of H2_i plus one ulp of its own value
    plus 2e-3 rms (the propagated flips of the narrower paths), and the block to the normwise
    bar of a single rounding."""
    T, L, r, q, nblk, eps = (LL[k] for k in ("T", "seq_len", "r", "q", "nblk", "eps"))
    d, heads, ffn = (SHAPES[shape][k] for k in ("d", "heads", "ffn"))
    dev, norms, ref = llama_case(41 + shape, dt, d, ffn, r, q)
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(41, "X", (T, d), (nblk * T, d)), dt)
    out = host(zo.LlamaLayer(dev, norms, bq, bs, eps, T, L, heads)(Hd))
    for b in range(nblk):
        rr = slice(b * T, (b + 1) * T)
        tr = {}
        want = oracle.llama_layer(Hv[rr], ref, bs[b], eps, bq[b], heads, L, store=rnd(dt), trace=tr)
        assert normwise(out[rr], want) <= 2e-3, b
        rms = float(np.sqrt(np.mean(want ** 2)))
        bound = ulp16(tr["H2"], dt) + ulp16(want, dt) + 2e-3 * rms
        err = np.abs(out[rr] - want)
        assert np.all(err <= bound), (b, float(np.max(err / bound)))


def test_llama_loss_central_difference_at_large_eps():
    """L+- of a real two-layer LLaMA-family forward.  The target is the input itself, so the
    loss measures what the layers' branches add to the residual stream; at eps = 1 the
    central difference of that loss stands far above the bf16 forward's rounding noise
    (about 1% of the larger estimate here) and matches the oracle's."""
    T, L, r, q, nblk = (LL[k] for k in ("T", "seq_len", "r", "q", "nblk"))
    d, heads, ffn = (SHAPES[0][k] for k in ("d", "heads", "ffn"))
    eps = 1.0
    layers = [llama_case(51 + i, "bf16", d, ffn, r, q) for i in range(2)]
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(51, "X", (T, d), (T, d)), "bf16")
    H = Hd
    for dev, norms, _ in layers:
        H = zo.LlamaLayer(dev, norms, bq, bs, eps, T, L, heads)(H)
    Lb = zo.sq_loss(H, Hd, nblk, T)
    g = host(zo.combine_central(Lb, eps))
    Lh = host(Lb)
    Lref = []
    for b in range(nblk):
        x = Hv
        for _, _, ref in layers:
            x = oracle.llama_layer(x, ref, bs[b], eps, bq[b], heads, L, store=oracle.round_bf16)
        Lref.append(oracle.sq_loss(x, Hv))
    np.testing.assert_allclose(Lh, Lref, rtol=2e-3)
    gref = oracle.central_estimate(Lref[0::2], Lref[1::2], eps)
    np.testing.assert_allclose(g, gref, rtol=2e-2, atol=2e-2 * np.abs(gref).max())
