"""The decoder layers at the full sizes the benchmark's decoder step runs (OPT-13B, OPT-1.3B and
LLaMA-7B shapes: every block of T tokens, 2q blocks, the config's r and eps, bf16; OPT-13B also
in fp16, the paper's precision), in the
same one-call launch sequence, with sampled (block, sequence) pairs checked against the
float64 oracle.

Each block has its own input (the first block's rows rolled by b * T / nblk, as in the
benchmark), so the per-block projections and attention are exercised at scale.

The bar at these sizes is accuracy against the exact layer, relative to the oracle's own
16-bit pipeline (the same layer with every stored activation rounded to the layer's type
where the device stores one).  Stage by stage the device agrees with that pipeline on its own inputs to a
fraction of a percent of one-ulp flips; but a flip of a stored value moves every later sum
that reads it, and over d = 4096-5120, 512 keys and K = 20480 those moves cross rounding
boundaries ever more often (at the OPT-13B shape: 0.2 % of Q, K, V differ, 4 % of the
attention output, 12 % of H2, 45 % of the layer output, by an ulp).  Two correct 16-bit
evaluations therefore differ by about the pipeline's own error, and what can be asked is
that the device be as accurate as the pipeline: its normwise error against the exact layer
within 5 % of the pipeline's, and its largest element error within 1.5 times the
pipeline's largest.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import cast, dev_f32, host, normwise, orth, rnd

pytestmark = pytest.mark.gpu


def full_layer(name, seed, dt="bf16"):
    cfg = zd.CONFIGS[name]
    dec = cfg["decoder"]
    d, ffn, r, q = dec["d"], dec["ffn"], cfg["r"], cfg["q"]
    llama = dec.get("family") == "llama"
    if llama:
        shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d),
                  "down": (d, ffn)}
    else:
        shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "fc1": (ffn, d), "fc2": (d, ffn)}
    dev, ref = {}, {}
    for i, (nm, (m, n)) in enumerate(shapes.items()):
        Wd, Wv = cast(zd.draw(seed, "W0", (i, m, n), (m, n), 0.02), dt)
        U, V = orth(seed, (i, 1, m), m, r), orth(seed, (i, 2, n), n, r)
        Z = zd.z_draws(seed, 0, i, q, r)
        dev[nm] = dict(W=Wd, U=dev_f32(U), V=dev_f32(V), Z=dev_f32(Z))
        ref[nm] = dict(W=Wv, U=U.astype(np.float64), V=V.astype(np.float64), Z=Z.astype(np.float64))
    g = zd.f32(1.0 + 0.05 * zd.draw(seed, "W0", (99,), (4, d)))
    if llama:
        norms = dict(rms1_gamma=dev_f32(g[0]), rms2_gamma=dev_f32(g[2]))
        ref.update(rms1_g=g[0].astype(np.float64), rms2_g=g[2].astype(np.float64))
    else:
        b1, b2 = zd.f32(g[1] - 1.0), zd.f32(g[3] - 1.0)
        norms = dict(ln1_gamma=dev_f32(g[0]), ln1_beta=dev_f32(b1), ln2_gamma=dev_f32(g[2]), ln2_beta=dev_f32(b2))
        ref.update(ln1_g=g[0].astype(np.float64), ln1_b=b1.astype(np.float64), ln2_g=g[2].astype(np.float64),
                   ln2_b=b2.astype(np.float64))
    return cfg, dec, llama, dev, norms, ref


@pytest.mark.parametrize("name,dt", [("opt-13b", "bf16"), ("opt-1.3b", "bf16"), ("llama-7b", "bf16"),
                                     ("opt-13b", "f16")])   # fp16: the paper's precision for OPT-13B
def test_layer_full_size_sampled(name, dt):
    seed = 61
    cfg, dec, llama, dev, norms, ref = full_layer(name, seed, dt)
    T, q, eps = cfg["T"], cfg["q"], cfg["eps"]
    d, heads, L = dec["d"], dec["heads"], dec["seq_len"]
    nblk = 2 * q
    bq, bs = [b // 2 for b in range(nblk)], [1 if b % 2 == 0 else -1 for b in range(nblk)]
    step = T // nblk
    H0d, H0v = cast(zd.draw(seed, "X", (T, d), (T, d)), dt)
    H = torch.cat([torch.roll(H0d, b * step, 0) for b in range(nblk)])
    Layer = zo.LlamaLayer if llama else zo.DecoderLayer
    out = Layer(dev, norms, bq, bs, eps, T, L, heads)(H)
    torch.cuda.synchronize()
    del H
    nseq = T // L
    fn = oracle.llama_layer if llama else oracle.decoder_layer
    for b, s in [(0, 0), (nblk - 1, nseq - 1), (nblk // 2 + 1, nseq // 2)]:
        rows = slice(b * T + s * L, b * T + (s + 1) * L)
        got = host(out[rows])
        Hb = np.roll(H0v, b * step, axis=0)[s * L:(s + 1) * L]
        exact = fn(Hb, ref, bs[b], eps, bq[b], heads, L)
        pipe = fn(Hb, ref, bs[b], eps, bq[b], heads, L, store=rnd(dt))
        nw_dev, nw_pipe = normwise(got, exact), normwise(pipe, exact)
        assert nw_dev <= 1.05 * nw_pipe, (b, s, nw_dev, nw_pipe)
        mx_dev, mx_pipe = float(np.max(np.abs(got - exact))), float(np.max(np.abs(pipe - exact)))
        assert mx_dev <= 1.5 * mx_pipe, (b, s, mx_dev, mx_pipe)
