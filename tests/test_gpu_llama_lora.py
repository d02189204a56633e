"""Parity of grouped key/value attention and of the LoRA scheme's LLaMA-family layer (the Qwen
models of the experiments: grouped heads, frozen base, adapters on q and v perturbed per block,
Eq. 4 on the adapter factors, inside the forward of Eq. 5) with the float64 oracle.

Bars as for the other layers: attention within one ulp plus 2^-14 of the softmax average of
|V|; the layer stage by stage at the single-kernel bars on the GPU's own inputs (the frozen
products checked through the perturbed linear at eps = 0, which adds exact zeros); the
one-call layer bitwise the sequence of calls; end to end against the oracle layer that rounds
each stored activation, at the residual-stream bound; a two-layer central difference; and the
full size of the Qwen-32B-shaped layer against the exact layer, relative to the oracle's
16-bit pipeline.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import cast, check16, check_attention, dev_f32, host, normwise, orth, rnd, ulp16

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ grouped attention
@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("nblk,T,seq_len,d,heads,kv", [
    (2, 256, 128, 512, 4, 1),    # dh = 128, one key/value head for four query heads
    (1, 200, 100, 256, 4, 2),    # dh = 64, ragged query tiles
    (2, 512, 256, 1280, 10, 2),  # the Qwen-32B ratio (5 query heads per key/value head)
    (1, 1024, 512, 512, 4, 2),   # dh = 128, sequences of 512 (8-wave workgroups)
    (1, 1024, 512, 256, 4, 2),   # dh = 64, sequences of 512 (8-wave workgroups)
])
def test_grouped_attention_parity(dt, nblk, T, seq_len, d, heads, kv):
    dkv = d // heads * kv
    Qd, Qv = cast(zd.draw(71, "X", (nblk, T, d), (nblk * T, d)), dt)
    Kd, Kv = cast(zd.draw(71, "W0", (nblk, T, dkv), (nblk * T, dkv)), dt)
    Vd, Vv = cast(zd.draw(71, "WSTAR", (nblk, T, dkv), (nblk * T, dkv)), dt)
    O = host(zo.causal_attention(Qd, Kd, Vd, nblk, T, seq_len, heads, kv_heads=kv))
    for b in range(nblk):
        r = slice(b * T, (b + 1) * T)
        check_attention(O[r], Qv[r], Kv[r], Vv[r], heads, seq_len, dt, (dt, b), kv)
        ref = oracle.causal_attention(Qv[r], Kv[r], Vv[r], heads, seq_len, kv)
        assert normwise(O[r], ref) <= 2e-3


def test_grouped_attention_equals_repeated_heads():
    """Grouped heads are bitwise the plain kernel on K and V with each head repeated."""
    nblk, T, L, d, heads, kv = 1, 128, 64, 512, 4, 2
    dh, dkv = d // heads, d // heads * kv
    Qd, _ = cast(zd.draw(72, "X", (0,), (nblk * T, d)), "bf16")
    Kd, _ = cast(zd.draw(72, "W0", (0,), (nblk * T, dkv)), "bf16")
    Vd, _ = cast(zd.draw(72, "WSTAR", (0,), (nblk * T, dkv)), "bf16")
    rep = lambda X: X.view(nblk * T, kv, 1, dh).expand(nblk * T, kv, heads // kv, dh).reshape(nblk * T, d)
    a = zo.causal_attention(Qd, Kd, Vd, nblk, T, L, heads, kv_heads=kv)
    b = zo.causal_attention(Qd, rep(Kd).contiguous(), rep(Vd).contiguous(), nblk, T, L, heads)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


# ------------------------------------------------------------------ the layer
def lora_case(seed, dt, d, dkv, ffn, rl, r, q):
    shapes = {"q": (d, d), "k": (dkv, d), "v": (dkv, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d),
              "down": (d, ffn)}
    dev, ref = {}, {}
    for i, (nm, (m, n)) in enumerate(shapes.items()):
        Wd, Wv = cast(zd.draw(seed, "W0", (i, m, n), (m, n), 0.03), dt)
        dev[nm], ref[nm] = dict(W=Wd), dict(W=Wv)
        if nm in ("q", "v"):
            A = zd.f32(zd.draw(seed, "LORA_A", (i,), (rl, n), 0.05))
            B = zd.f32(zd.draw(seed, "LORA_B", (i,), (m, rl), 0.05))
            fac = dict(A=A, B=B, UA=orth(seed, (i, 1), rl, r), VA=orth(seed, (i, 2), n, r),
                       UB=orth(seed, (i, 3), m, r), VB=orth(seed, (i, 4), rl, r),
                       ZA=zd.z_draws(seed, 0, 2 * i, q, r), ZB=zd.z_draws(seed, 0, 2 * i + 1, q, r))
            dev[nm].update({k: dev_f32(v) for k, v in fac.items()})
            ref[nm].update({k: v.astype(np.float64) for k, v in fac.items()})
    g1 = zd.f32(1.0 + 0.1 * zd.draw(seed, "W0", (99, 0), (d,)))
    g2 = zd.f32(1.0 + 0.1 * zd.draw(seed, "W0", (99, 1), (d,)))
    ref.update(rms1_g=g1.astype(np.float64), rms2_g=g2.astype(np.float64))
    return dev, dict(rms1_gamma=dev_f32(g1), rms2_gamma=dev_f32(g2)), ref


LL = dict(T=128, seq_len=64, rl=4, r=4, q=2, nblk=4, eps=1e-2, scale=2.0)
SHAPES = [dict(d=256, heads=2, kv=1, ffn=688), dict(d=256, heads=4, kv=2, ffn=512)]


def blocks():
    nblk, q = LL["nblk"], LL["q"]
    return [b // 2 % q for b in range(nblk)], [1 if b % 2 == 0 else -1 for b in range(nblk)]


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("shared", [True, False])
@pytest.mark.parametrize("shape", range(len(SHAPES)))
def test_lora_layer_stagewise_and_one_call(dt, shared, shape):
    T, L, rl, r, q, nblk, eps, scale = (LL[k] for k in ("T", "seq_len", "rl", "r", "q", "nblk", "eps", "scale"))
    d, heads, kv, ffn = (SHAPES[shape][k] for k in ("d", "heads", "kv", "ffn"))
    dkv = d // heads * kv
    dev, norms, ref = lora_case(81 + shape, dt, d, dkv, ffn, rl, r, q)
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(81, "X", (T, d), ((1 if shared else nblk) * T, d)), dt)
    out = zo.LlamaLoraLayer(dev, norms, bq, bs, eps, scale, T, L, heads, kv, rope_base=1e6)(Hd)
    torch.cuda.synchronize()

    def rows(b):
        return slice(b * T, (b + 1) * T)

    def frozen(nm, X, xs):
        # The perturbed linear at eps = 0: its rank-r segment adds exact zeros, so this is the
        # frozen product.
        m, n = dev[nm]["W"].shape
        z = lambda *sh: torch.zeros(sh, dtype=torch.float32, device="cuda")
        return zo.PerturbedLinear(X, dev[nm]["W"], z(m, r), z(n, r), z(q, r, r), bq, bs, 0.0, T, x_block_stride=xs)

    def adapted(nm, X, xs):
        m = dev[nm]
        return zo.LoraPerturbedLinear(X, m["W"], m["A"], m["UA"], m["VA"], m["ZA"], m["B"], m["UB"], m["VB"], m["ZB"],
                                      bq, bs, eps, scale, T, x_block_stride=xs)()

    def adapted_ref(nm, Xb, b):
        m = ref[nm]
        return oracle.lora_perturbed_linear(Xb, m["W"], m["A"], m["UA"], m["VA"], m["ZA"][bq[b]], m["B"], m["UB"],
                                            m["VB"], m["ZB"][bq[b]], bs[b], eps, scale)

    hT = 0 if shared else T * d
    A = zo.rmsnorm(Hd, norms["rms1_gamma"], 1e-6)
    Ah = host(A)
    check16(Ah, oracle.rms_norm(Hv, ref["rms1_g"], 1e-6), "rms1")
    Ab = lambda b: Ah if shared else Ah[rows(b)]
    Qd = adapted("q", A, hT).clone()
    Qh = host(Qd)
    Kd = frozen("k", A, hT)
    Kd.prepare()
    Kd = Kd.apply().clone()
    Kh = host(Kd)
    Vd = adapted("v", A, hT).clone()
    Vh = host(Vd)
    for b in range(nblk):
        check16(Qh[rows(b)], adapted_ref("q", Ab(b), b), ("q", b))
        check16(Kh[rows(b)], Ab(b) @ ref["k"]["W"].T, ("k", b))
        check16(Vh[rows(b)], adapted_ref("v", Ab(b), b), ("v", b))
    zo.rope(Qd, L, heads, 1e6)
    zo.rope(Kd, L, kv, 1e6)
    Qr, Kr = host(Qd), host(Kd)
    for b in range(nblk):
        check16(Qr[rows(b)], oracle.rope(Qh[rows(b)], L, heads, 1e6), ("rope q", b))
        check16(Kr[rows(b)], oracle.rope(Kh[rows(b)], L, kv, 1e6), ("rope k", b))
    C = zo.causal_attention(Qd, Kd, Vd, nblk, T, L, heads, kv_heads=kv)
    Ch = host(C)
    for b in range(nblk):
        check_attention(Ch[rows(b)], Qr[rows(b)], Kr[rows(b)], Vh[rows(b)], heads, L, dt, ("attn", b), kv)
        assert normwise(Ch[rows(b)], oracle.causal_attention(Qr[rows(b)], Kr[rows(b)], Vh[rows(b)], heads, L,
                                                             kv)) <= 2e-3
    p = frozen("o", C, T * d)
    p.prepare()
    H2 = p.apply(zo.ZO_EPI_RESIDUAL, Hd).clone()
    H2h = host(H2)
    for b in range(nblk):
        check16(H2h[rows(b)], (Hv if shared else Hv[rows(b)]) + Ch[rows(b)] @ ref["o"]["W"].T, ("o", b))
    A2 = zo.rmsnorm(H2, norms["rms2_gamma"], 1e-6)
    A2h = host(A2)
    check16(A2h, oracle.rms_norm(H2h, ref["rms2_g"], 1e-6), "rms2")
    p = frozen("gate", A2, T * d)
    p.prepare()
    G = p.apply().clone()
    Gh = host(G)
    p = frozen("up", A2, T * d)
    p.prepare()
    F = p.apply(zo.ZO_EPI_SILU_MUL, G).clone()
    Fh = host(F)
    for b in range(nblk):
        check16(Gh[rows(b)], A2h[rows(b)] @ ref["gate"]["W"].T, ("gate", b))
        check16(Fh[rows(b)], oracle.silu(Gh[rows(b)]) * (A2h[rows(b)] @ ref["up"]["W"].T), ("up", b))
    p = frozen("down", F, T * ffn)
    p.prepare()
    H3 = p.apply(zo.ZO_EPI_RESIDUAL, H2)
    H3h = host(H3)
    for b in range(nblk):
        check16(H3h[rows(b)], H2h[rows(b)] + Fh[rows(b)] @ ref["down"]["W"].T, ("down", b))
    assert torch.equal(out.view(torch.int16), H3.view(torch.int16))


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("shape", range(len(SHAPES)))
def test_lora_layer_end_to_end(dt, shape):
    """Against the oracle layer that rounds each stored activation to the same type, at the
    residual-stream bound of the other layer tests."""
    T, L, rl, r, q, nblk, eps, scale = (LL[k] for k in ("T", "seq_len", "rl", "r", "q", "nblk", "eps", "scale"))
    d, heads, kv, ffn = (SHAPES[shape][k] for k in ("d", "heads", "kv", "ffn"))
    dev, norms, ref = lora_case(91 + shape, dt, d, d // heads * kv, ffn, rl, r, q)
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(91, "X", (T, d), (nblk * T, d)), dt)
    out = host(zo.LlamaLoraLayer(dev, norms, bq, bs, eps, scale, T, L, heads, kv)(Hd))
    for b in range(nblk):
        rr = slice(b * T, (b + 1) * T)
        tr = {}
        want = oracle.llama_lora_layer(Hv[rr], ref, bs[b], eps, bq[b], heads, kv, L, scale, store=rnd(dt), trace=tr)
        assert normwise(out[rr], want) <= 2e-3, b
        rms = float(np.sqrt(np.mean(want ** 2)))
        bound = ulp16(tr["H2"], dt) + ulp16(want, dt) + 2e-3 * rms
        err = np.abs(out[rr] - want)
        assert np.all(err <= bound), (b, float(np.max(err / bound)))


def test_lora_layer_central_difference_at_large_eps():
    """Two layers, the input as the target: at eps = 1 the central difference of the loss is
    far above the bf16 forward's rounding noise and matches the oracle's."""
    T, L, rl, r, q, nblk, scale = (LL[k] for k in ("T", "seq_len", "rl", "r", "q", "nblk", "scale"))
    d, heads, kv, ffn = (SHAPES[1][k] for k in ("d", "heads", "kv", "ffn"))
    eps = 1.0
    layers = [lora_case(101 + i, "bf16", d, d // heads * kv, ffn, rl, r, q) for i in range(2)]
    bq, bs = blocks()
    Hd, Hv = cast(zd.draw(101, "X", (T, d), (T, d)), "bf16")
    H = Hd
    for dev, norms, _ in layers:
        H = zo.LlamaLoraLayer(dev, norms, bq, bs, eps, scale, T, L, heads, kv)(H)
    Lb = zo.sq_loss(H, Hd, nblk, T)
    g = host(zo.combine_central(Lb, eps))
    Lh = host(Lb)
    Lref = []
    for b in range(nblk):
        x = Hv
        for _, _, ref in layers:
            x = oracle.llama_lora_layer(x, ref, bs[b], eps, bq[b], heads, kv, L, scale, store=oracle.round_bf16)
        Lref.append(oracle.sq_loss(x, Hv))
    np.testing.assert_allclose(Lh, Lref, rtol=2e-3)
    gref = oracle.central_estimate(Lref[0::2], Lref[1::2], eps)
    np.testing.assert_allclose(g, gref, rtol=2e-2, atol=2e-2 * np.abs(gref).max())


def test_lora_layer_full_size_sampled():
    """The Qwen-32B-shaped layer (d = 5120, 40 query heads over 8 key/value heads, ffn = 27648,
    adapters r_L = 8 with r = 4 subspaces, 2q blocks of T tokens) with three sampled
    (block, sequence) pairs against the exact layer: the device's normwise error within 5 % of
    the oracle's bf16 pipeline's and its largest element error within 1.5x the pipeline's."""
    cfg = zd.CONFIGS["qwen-32b-lora"]
    dec = cfg["decoder"]
    T, q, r, eps = cfg["T"], cfg["q"], cfg["r"], cfg["eps"]
    d, heads, kv, ffn, L = dec["d"], dec["heads"], dec["kv_heads"], dec["ffn"], dec["seq_len"]
    rl, scale = zd.QWEN_LORA_RANK, zd.QWEN_LORA_ALPHA / zd.QWEN_LORA_RANK
    nblk = 2 * q
    dev, norms, ref = lora_case(111, "bf16", d, d // heads * kv, ffn, rl, r, q)
    bq, bs = [b // 2 for b in range(nblk)], [1 if b % 2 == 0 else -1 for b in range(nblk)]
    step = T // nblk
    H0d, H0v = cast(zd.draw(111, "X", (T, d), (T, d)), "bf16")
    H = torch.cat([torch.roll(H0d, b * step, 0) for b in range(nblk)])
    out = zo.LlamaLoraLayer(dev, norms, bq, bs, eps, scale, T, L, heads, kv, rope_base=dec["rope_base"])(H)
    torch.cuda.synchronize()
    del H
    nseq = T // L
    for b, s in [(0, 0), (nblk - 1, nseq - 1), (nblk // 2 + 1, nseq // 2)]:
        got = host(out[b * T + s * L:b * T + (s + 1) * L])
        Hb = np.roll(H0v, b * step, axis=0)[s * L:(s + 1) * L]
        kw = dict(rope_base=dec["rope_base"])
        exact = oracle.llama_lora_layer(Hb, ref, bs[b], eps, bq[b], heads, kv, L, scale, **kw)
        pipe = oracle.llama_lora_layer(Hb, ref, bs[b], eps, bq[b], heads, kv, L, scale, store=oracle.round_bf16, **kw)
        nw_dev, nw_pipe = normwise(got, exact), normwise(pipe, exact)
        assert nw_dev <= 1.05 * nw_pipe, (b, s, nw_dev, nw_pipe)
        mx_dev, mx_pipe = float(np.max(np.abs(got - exact))), float(np.max(np.abs(pipe - exact)))
        assert mx_dev <= 1.5 * mx_pipe, (b, s, mx_dev, mx_pipe)
