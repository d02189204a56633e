"""Parity of the decoder-layer pieces (the network each query evaluates, the forward of
Eq. 5 inside Alg. 3) with the float64 oracle.

Bars: each kernel on exact 16-bit inputs as the perturbed linear: e(., ., 1e-3) <= 1e-2 and
normwise <= 2e-3 for 16-bit outputs (one rounding of 2^-9 / 2^-11), e(., ., 1) <= 1e-5 for
fp32 layer norm; attention elementwise within one ulp plus 2^-14 of the softmax average
of |V| (the accuracy of its P V product), normwise 2e-3.  The decoder layer is checked stage by stage with each stage fed the GPU's
own previous output (so the bars stay those of single kernels), the one-call layer is
bitwise the sequence of single calls, and the end-to-end output is compared with the
oracle layer that rounds every stored activation to the same type.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import cast, check16, check_attention, dev_f32, ferr, host, normwise, orth, rnd, ulp16

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ layer norm
@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("rows,d", [(37, 96), (300, 5120), (5, 8), (64, 2048),
                                    # every register bucket and its edges, and the re-reading path
                                    (7, 1032), (9, 4096), (6, 5128), (5, 8192), (3, 8200)])
def test_layernorm_parity(dt, rows, d):
    Xd, Xv = cast(zd.draw(7, "X", (rows, d), (rows, d)) * 2.0 + 0.5, dt)
    g = zd.f32(1.0 + 0.1 * zd.draw(7, "W0", (d, 1), (d,)))
    b = zd.f32(0.1 * zd.draw(7, "W0", (d, 2), (d,)))
    Y = host(zo.layernorm(Xd, dev_f32(g), dev_f32(b), 1e-5))
    ref = oracle.layer_norm(Xv, g.astype(np.float64), b.astype(np.float64), 1e-5)
    if dt == "f32":
        assert ferr(Y, ref, 1.0) <= 1e-5
    else:
        check16(Y, ref, dt)


def test_layernorm_in_place():
    Xd, Xv = cast(zd.draw(8, "X", (0,), (64, 512)), "bf16")
    g, b = torch.ones(512, device="cuda"), torch.zeros(512, device="cuda")
    ref = host(zo.layernorm(Xd, g, b))
    zo.layernorm(Xd, g, b, out=Xd)
    torch.cuda.synchronize()
    assert np.array_equal(host(Xd), ref)


# ------------------------------------------------------------------ attention
def attn_case(seed, nblk, T, d, dt):
    out = []
    for k, kind in enumerate(("X", "W0", "WSTAR")):
        out.append(cast(zd.draw(seed, kind, (nblk, T, d, k), (nblk * T, d)), dt))
    return out


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("nblk,T,seq_len,d,heads", [
    (2, 256, 128, 256, 2),    # dh = 128, two query tiles per sequence
    (1, 200, 100, 128, 2),    # dh = 64, sequences not a multiple of the 64-query tile
    (3, 64, 64, 512, 4),      # one tile per sequence
    (1, 1024, 512, 256, 2),   # the OPT-13B sequence length
    (1, 1024, 512, 128, 2),   # dh = 64 at a sequence length that takes the 8-wave workgroups
])
def test_attention_parity(dt, nblk, T, seq_len, d, heads):
    (Qd, Qv), (Kd, Kv), (Vd, Vv) = attn_case(9, nblk, T, d, dt)
    O = host(zo.causal_attention(Qd, Kd, Vd, nblk, T, seq_len, heads))
    for b in range(nblk):
        r = slice(b * T, (b + 1) * T)
        check_attention(O[r], Qv[r], Kv[r], Vv[r], heads, seq_len, dt, (dt, b))


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_attention_single_token_sequences_return_v(dt):
    """seq_len = 1: each query sees only its own key, so O = V bit for bit (P = 2^12 exactly)."""
    (Qd, _), (Kd, _), (Vd, _) = attn_case(10, 2, 32, 256, dt)
    O = zo.causal_attention(Qd, Kd, Vd, 2, 32, 1, 2)
    torch.cuda.synchronize()
    assert torch.equal(O.view(torch.int16), Vd.view(torch.int16))


def test_attention_large_logits_stay_finite():
    """Scaled logits of several hundred (sharp attention) must not overflow the softmax."""
    (Qd, Qv), (Kd, Kv), (Vd, Vv) = attn_case(11, 1, 128, 128, "bf16")
    Qd, Qv = cast(Qv * 40.0, "bf16")
    O = host(zo.causal_attention(Qd, Kd, Vd, 1, 128, 128, 1))
    assert np.isfinite(O).all()
    check_attention(O, Qv, Kv, Vv, 1, 128, "bf16", "sharp")


# ------------------------------------------------------------------ fused epilogues
@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("n", [512, 200])   # the main kernel, and the generic tile kernel
@pytest.mark.parametrize("epi", ["relu", "residual", "residual_shared"])
def test_apply_epilogues(dt, n, epi):
    T, m, r, q, nblk = 192, 256, 8, 2, 4
    Wd, Wv = cast(zd.draw(12, "W0", (m, n), (m, n), 0.05), dt)
    Xd, Xv = cast(zd.draw(12, "X", (T, n), (nblk * T, n)), dt)
    U, V = orth(12, (1, m), m, r), orth(12, (2, n), n, r)
    Z = zd.z_draws(12, 0, 0, q, r)
    bq, bs = [b // 2 for b in range(nblk)], [1, -1] * (nblk // 2)
    eps = 1e-2
    pl = zo.PerturbedLinear(Xd, Wd, dev_f32(U), dev_f32(V), dev_f32(Z), bq, bs, eps, T, x_block_stride=T * n)
    pl.prepare()
    shared = epi == "residual_shared"
    Rd, Rv = cast(zd.draw(12, "WSTAR", (m,), ((1 if shared else nblk) * T, m)), dt)
    if epi == "relu":
        Y = host(pl.apply(zo.ZO_EPI_RELU))
    else:
        Y = host(pl.apply(zo.ZO_EPI_RESIDUAL, Rd))
    for b in range(nblk):
        lin = oracle.perturbed_linear(Xv[b * T:(b + 1) * T], Wv, U.astype(np.float64), V.astype(np.float64),
                                      Z[bq[b]].astype(np.float64), bs[b], eps)
        if epi == "relu":
            ref = np.maximum(lin, 0.0)
        else:
            ref = lin + (Rv if shared else Rv[b * T:(b + 1) * T])
        check16(Y[b * T:(b + 1) * T], ref, (epi, b))


def test_apply_residual_in_place():
    """R may be Y itself: Y <- Y + the perturbed product."""
    T, m, n, r, q, nblk = 128, 256, 256, 8, 1, 2
    Wd, Wv = cast(zd.draw(13, "W0", (m, n), (m, n), 0.05), "bf16")
    Xd, Xv = cast(zd.draw(13, "X", (T, n), (nblk * T, n)), "bf16")
    U, V = orth(13, (1, m), m, r), orth(13, (2, n), n, r)
    Z = zd.z_draws(13, 0, 0, q, r)
    Yd, Yv = cast(zd.draw(13, "WSTAR", (m,), (nblk * T, m)), "bf16")
    pl = zo.PerturbedLinear(Xd, Wd, dev_f32(U), dev_f32(V), dev_f32(Z), [0, 0], [1, -1], 1e-2, T,
                            x_block_stride=T * n, Y=Yd)
    pl.prepare()
    Y = host(pl.apply(zo.ZO_EPI_RESIDUAL, Yd))
    for b, s in enumerate([1, -1]):
        lin = oracle.perturbed_linear(Xv[b * T:(b + 1) * T], Wv, U.astype(np.float64), V.astype(np.float64),
                                      Z[0].astype(np.float64), s, 1e-2)
        check16(Y[b * T:(b + 1) * T], lin + Yv[b * T:(b + 1) * T], b)


# ------------------------------------------------------------------ the decoder layer
def decoder_case(seed, dt, d, ffn, r, q):
    shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "fc1": (ffn, d), "fc2": (d, ffn)}
    dev, ref = {}, {}
    for i, (nm, (m, n)) in enumerate(shapes.items()):
        Wd, Wv = cast(zd.draw(seed, "W0", (i, m, n), (m, n), 0.02), dt)
        U, V = orth(seed, (i, 1, m), m, r), orth(seed, (i, 2, n), n, r)
        Z = zd.z_draws(seed, 0, i, q, r)
        dev[nm] = dict(W=Wd, U=dev_f32(U), V=dev_f32(V), Z=dev_f32(Z))
        ref[nm] = dict(W=Wv, U=U.astype(np.float64), V=V.astype(np.float64), Z=Z.astype(np.float64))
    ln = {}
    for k, nm in enumerate(("ln1_gamma", "ln1_beta", "ln2_gamma", "ln2_beta")):
        base = 1.0 if nm.endswith("gamma") else 0.0
        ln[nm] = zd.f32(base + 0.1 * zd.draw(seed, "W0", (99, k), (d,)))
    ref.update(ln1_g=ln["ln1_gamma"].astype(np.float64), ln1_b=ln["ln1_beta"].astype(np.float64),
               ln2_g=ln["ln2_gamma"].astype(np.float64), ln2_b=ln["ln2_beta"].astype(np.float64))
    return dev, {k: dev_f32(v) for k, v in ln.items()}, ref


DEC = dict(T=128, seq_len=64, d=256, heads=2, ffn=512, r=8, q=2, nblk=4, eps=1e-2)


def blocks():
    nblk = DEC["nblk"]
    return [b // 2 % DEC["q"] for b in range(nblk)], [1 if b % 2 == 0 else -1 for b in range(nblk)]


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("shared", [True, False])
def test_decoder_layer_stagewise_and_one_call(dt, shared):
    T, L, d, heads, ffn, r, q, nblk, eps = (DEC[k] for k in ("T", "seq_len", "d", "heads", "ffn", "r", "q",
                                                             "nblk", "eps"))
    dev, lnd, ref = decoder_case(14, dt, d, ffn, r, q)
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(14, "X", (T, d), ((1 if shared else nblk) * T, d)), dt)
    out = zo.DecoderLayer(dev, lnd, bq, bs, eps, T, L, heads)(Hd)
    torch.cuda.synchronize()

    # The same layer as a sequence of single calls, each stage checked against the oracle
    # on the GPU's own input to that stage.
    def lin(nm, X, xs, Y=None):
        mt = dev[nm]
        return zo.PerturbedLinear(X, mt["W"], mt["U"], mt["V"], mt["Z"], bq, bs, eps, T, x_block_stride=xs, Y=Y)

    def lin_ref(nm, Xv_b, b):
        mt = ref[nm]
        return oracle.perturbed_linear(Xv_b, mt["W"], mt["U"], mt["V"], mt["Z"][bq[b]], bs[b], eps)

    hT = 0 if shared else T * d
    A = zo.layernorm(Hd, lnd["ln1_gamma"], lnd["ln1_beta"])
    Ah = host(A)
    check16(Ah, oracle.layer_norm(Hv, ref["ln1_g"], ref["ln1_b"]), "ln1")
    QKV = []
    for nm in ("q", "k", "v"):
        p = lin(nm, A, hT)
        p.prepare()
        Y = p.apply()
        Yh = host(Y)
        for b in range(nblk):
            Ab = Ah if shared else Ah[b * T:(b + 1) * T]
            check16(Yh[b * T:(b + 1) * T], lin_ref(nm, Ab, b), (nm, b))
        QKV.append((Y.clone(), Yh))
    (Qd, Qh), (Kd, Kh), (Vd, Vh) = QKV
    C = zo.causal_attention(Qd, Kd, Vd, nblk, T, L, heads)
    Ch = host(C)
    for b in range(nblk):
        rr = slice(b * T, (b + 1) * T)
        check_attention(Ch[rr], Qh[rr], Kh[rr], Vh[rr], heads, L, dt, ("attn", b))
    p = lin("o", C, T * d)
    p.prepare()
    H2 = p.apply(zo.ZO_EPI_RESIDUAL, Hd).clone()
    H2h = host(H2)
    for b in range(nblk):
        rr = slice(b * T, (b + 1) * T)
        Hb = Hv if shared else Hv[rr]
        check16(H2h[rr], Hb + lin_ref("o", Ch[rr], b), ("o", b))
    A2 = zo.layernorm(H2, lnd["ln2_gamma"], lnd["ln2_beta"])
    A2h = host(A2)
    check16(A2h, oracle.layer_norm(H2h, ref["ln2_g"], ref["ln2_b"]), "ln2")
    p = lin("fc1", A2, T * d)
    p.prepare()
    F = p.apply(zo.ZO_EPI_RELU).clone()
    Fh = host(F)
    for b in range(nblk):
        rr = slice(b * T, (b + 1) * T)
        check16(Fh[rr], np.maximum(lin_ref("fc1", A2h[rr], b), 0.0), ("fc1", b))
    p = lin("fc2", F, T * ffn)
    p.prepare()
    H3 = p.apply(zo.ZO_EPI_RESIDUAL, H2)
    H3h = host(H3)
    for b in range(nblk):
        rr = slice(b * T, (b + 1) * T)
        check16(H3h[rr], H2h[rr] + lin_ref("fc2", Fh[rr], b), ("fc2", b))
    # The one-call layer is exactly that sequence.
    assert torch.equal(out.view(torch.int16), H3.view(torch.int16))


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_decoder_layer_end_to_end(dt):
    """Against the oracle layer that rounds each stored activation to the same type.  Where the
    two roundings of a stored value land on different sides of a rounding boundary (a one-ulp
    flip), the difference propagates; through the residual stream it does so undamped:
    H_out = H2 + F W2'^T carries a flip of H2_i into output i whole, even where the MLP branch
    cancels H2_i and the output is near zero.  So each output is held to one ulp of H2_i plus
    one ulp of its own value plus 2e-3 rms (the propagated flips of the narrower paths), and
    the block to the normwise bar of a single rounding (2e-3)."""
    T, L, d, heads, ffn, r, q, nblk, eps = (DEC[k] for k in ("T", "seq_len", "d", "heads", "ffn", "r", "q",
                                                             "nblk", "eps"))
    dev, lnd, ref = decoder_case(15, dt, d, ffn, r, q)
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(15, "X", (T, d), (nblk * T, d)), dt)
    out = host(zo.DecoderLayer(dev, lnd, bq, bs, eps, T, L, heads)(Hd))
    for b in range(nblk):
        rr = slice(b * T, (b + 1) * T)
        tr = {}
        want = oracle.decoder_layer(Hv[rr], ref, bs[b], eps, bq[b], heads, L, store=rnd(dt), trace=tr)
        assert normwise(out[rr], want) <= 2e-3, b
        rms = float(np.sqrt(np.mean(want ** 2)))
        bound = ulp16(tr["H2"], dt) + ulp16(want, dt) + 2e-3 * rms
        err = np.abs(out[rr] - want)
        assert np.all(err <= bound), (b, float(np.max(err / bound)))


def test_decoder_loss_central_difference_at_large_eps():
    """L+- of a real two-layer forward: at eps = 0.5 the central difference of the squared loss
    is far above the bf16 forward's rounding noise and matches the oracle's."""
    T, L, d, heads, ffn, r, q, nblk = (DEC[k] for k in ("T", "seq_len", "d", "heads", "ffn", "r", "q", "nblk"))
    eps = 0.5
    layers = [decoder_case(16 + i, "bf16", d, ffn, r, q) for i in range(2)]
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(16, "X", (T, d), (T, d)), "bf16")
    Ysd, Ysv = cast(zd.draw(16, "WSTAR", (T, d), (T, d)), "bf16")
    H = Hd
    for dev, lnd, _ in layers:
        H = zo.DecoderLayer(dev, lnd, bq, bs, eps, T, L, heads)(H)
    Lb = zo.sq_loss(H, Ysd, nblk, T)
    g = host(zo.combine_central(Lb, eps))
    Lh = host(Lb)
    Lref = []
    for b in range(nblk):
        x = Hv
        for _, _, ref in layers:
            x = oracle.decoder_layer(x, ref, bs[b], eps, bq[b], heads, L, store=oracle.round_bf16)
        Lref.append(oracle.sq_loss(x, Ysv))
    np.testing.assert_allclose(Lh, Lref, rtol=2e-3)
    gref = oracle.central_estimate(Lref[0::2], Lref[1::2], eps)
    np.testing.assert_allclose(g, gref, rtol=2e-2, atol=2e-2 * np.abs(gref).max())
