"""Parity of zo_subspace_adam_update (HIP) with the float64 oracle (Eqs. 6-10).

Bars: fp32 W e(., W_exact, 1) <= 1e-5.  bf16 W: (i) the fp32 pre-rounding
hook e(., W_exact, 1) <= 2e-3 (we also hold it to 5e-5, and every entry to the
error bound of the kernel's arithmetic, see update_bound); (ii) the stored bf16
is exactly RNE of the hook, and within 1 ulp of round_bf16(W_exact) wherever
that bound is below half an ulp; (iii) normwise <= 2e-3.  The fraction of
1-ulp flips is reported (and held below 1% for bf16).  fp16 W: the same bars
with fp16 rounding and ulp; its ulp is 8x finer, so the 1-ulp bar applies to
fewer entries (where the delta cancels W, the split's ~2^-17 of sum |L||V| can
reach a few fp16 ulps).  The 1-ulp bar must cover at least half of the entries
(bf16 at every learning rate tested; fp16 at the full-tuning rate 1e-3, where it
covers 70-100%; at 1e-2 it covers 1-99% and the first two bars carry the check).
The moments are fp32 state: relative 1e-6.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15665_amd as zo
import zo_draws as zd
from _common import dev_bf16, dev_f16, dev_f32, ferr, host, normwise, orth

pytestmark = pytest.mark.gpu

F32 = lambda x: float(np.float32(x))  # hyper-parameters cross the ABI as fp32


def make_item(seed, idx, m, n, r, q, bf16, moments=False, f16=False):
    """W is bf16 (bf16=True), fp16 (f16=True) or fp32."""
    W64 = zd.draw(seed, "W0", idx, (m, n), 0.02)
    if f16:
        Wh, Wv = zd.as_f16_values(W64)
        Wd = dev_f16(Wh)
    elif bf16:
        Wb, Wv = zd.as_bf16_values(W64)
        Wd = dev_bf16(Wb)
    else:
        Wv = zd.f32(W64).astype(np.float64)
        Wd = dev_f32(Wv)
    U = orth(seed, idx + (1,), m, r)
    V = orth(seed, idx + (2,), n, r)
    Z = np.stack([zd.f32(zd.draw(seed, "Z", idx + (j,), (r, r))) for j in range(q)])
    if moments:
        M1 = zd.f32(zd.draw(seed, "MOM", idx + (1,), (r, r), 0.1))
        M2 = zd.f32(np.abs(zd.draw(seed, "MOM", idx + (2,), (r, r), 0.01)))
    else:
        M1 = np.zeros((r, r), np.float32)
        M2 = np.zeros((r, r), np.float32)
    return dict(m=m, n=n, Wv=Wv, U=U, V=V, Z=Z, M1h=M1, M2h=M2, f16=f16,
                dev=dict(W=Wd, U=dev_f32(U), V=dev_f32(V), Z=dev_f32(Z), M1=dev_f32(M1), M2=dev_f32(M2),
                         zbar_out=torch.empty((r, r), dtype=torch.float32, device="cuda"),
                         w_f32_out=torch.empty((m, n), dtype=torch.float32, device="cuda")))


def expected(it, g, t, lr, b1, b2, ea):
    return oracle.subspace_adam_update(it["Wv"], it["U"], it["V"], it["Z"], g, it["M1h"], it["M2h"], t,
                                       F32(lr), F32(b1), F32(b2), F32(ea))


def update_bound(U, V, S, lr, W_exact):
    """Per-entry bound on |hook - W_exact| for the bf16-W path (Eq. 10 in its arithmetic):
    L = lr U S is formed in fp32 over r terms and S is held in fp32; L and V enter the MFMA as
    hi + lo bf16 pairs (each pair keeps x to 2^-18 |x|, and the dropped lo*lo product is
    below 2^-18 |L V|), so every product is off by at most 3 * 2^-18 of |L_ia V_ja|; the
    3 rp products (rp = r rounded up to 32) accumulate in fp32; W - delta rounds once."""
    r = U.shape[1]
    rp = -(-r // 32) * 32
    A = (F32(lr) * (np.abs(U).astype(np.float64) @ np.abs(S))) @ np.abs(V).astype(np.float64).T
    return (3 * 2.0 ** -18 + (3 * rp + r + 4) * 2.0 ** -24) * A + 2.0 ** -23 * np.abs(W_exact)


def check_bf16_storage(got_w, got_hook, W_exact, E, f16=False, min_held=0.5):
    """Stored 16-bit W (bf16, or fp16 with f16=True): the hook within E of W_exact everywhere;
    the stored value exactly RNE of the hook; within 1 ulp of the exactly rounded W_exact
    wherever E is below half an ulp (where E is not, the first two already bound the stored
    value by E + half an ulp), which must hold for at least min_held of the entries (None: no
    floor); returns the fraction of 1-ulp flips."""
    rnd = oracle.round_f16 if f16 else oracle.round_bf16
    assert np.all(np.abs(got_hook - W_exact) <= E)
    assert np.array_equal(got_w, rnd(got_hook))
    rne = rnd(W_exact)
    e = np.frexp(rne)[1]
    ulp = np.ldexp(1.0, np.maximum(e - 11, -24)) if f16 else np.ldexp(1.0, e - 8)
    held = ulp >= 2 * E
    print(f"1-ulp bar covers {np.mean(held):.3f} of the entries")
    if min_held is not None:
        # bf16's ulp leaves E far below half an ulp almost everywhere; fp16's is 8x finer, and
        # where the delta cancels W the split's ~2^-17 of sum|L||V| can reach a few fp16 ulps.
        assert np.mean(held) >= min_held
    assert np.all((np.abs(got_w - rne) <= ulp * (1 + 1e-12))[held])
    return float(np.mean(got_w != rne))


def check_item(it, ref, bf16, lr, min_held=0.5):
    got_hook = host(it["dev"]["w_f32_out"])
    got_w = host(it["dev"]["W"])
    # Our own bound, tighter than the 2e-3 bar: the hi+lo bf16 split keeps ~2^-16 of the delta.
    assert ferr(got_hook, ref["W"], 1.0) <= 5e-5
    if bf16:
        assert ferr(got_hook, ref["W"], 1.0) <= 2e-3
        E = update_bound(it["U"], it["V"], ref["S"], lr, ref["W"])
        flips = check_bf16_storage(got_w, got_hook, ref["W"], E, it["f16"], min_held)
        assert normwise(got_w, ref["W"]) <= 2e-3
        print(f"16-bit storage flips vs exact rounding: {flips:.2e}")
        if not it["f16"]:
            assert flips < 1e-2, flips
    else:
        assert ferr(got_w, ref["W"], 1.0) <= 1e-5
    np.testing.assert_allclose(host(it["dev"]["M1"]), ref["M1"], rtol=1e-6, atol=1e-12)
    np.testing.assert_allclose(host(it["dev"]["M2"]), ref["M2"], rtol=1e-6, atol=1e-14)
    np.testing.assert_allclose(host(it["dev"]["zbar_out"]), ref["Zbar"], rtol=1e-6, atol=1e-9)


@pytest.mark.parametrize("m,n,r,q,t,moments", [
    (300, 264, 16, 4, 1, False),    # ragged against the 128 x 256 workgroup tile
    (256, 512, 64, 8, 3, True),     # r = 64 (two 32-deep K steps)
    (130, 1000, 100, 2, 7, True),   # r = 100 padded to 128
    (256, 512, 128, 4, 2, True),    # r = 128, the paper's full-tuning rank
    (17, 8, 4, 4, 1, False),        # tiny, r = 4 padded to 32
    (1024, 2048, 32, 4, 2, True),
])
def test_bf16_update_parity(m, n, r, q, t, moments):
    it = make_item(0, (m, n, r), m, n, r, q, True, moments)
    g = zd.f32(zd.draw(0, "G", (m, n, r), (q,), 1e-2))
    lr, b1, b2, ea = 1e-2, 0.9, 0.95, 1e-8
    ref = expected(it, g.astype(np.float64), t, lr, b1, b2, ea)
    zo.subspace_adam_update([it["dev"]], dev_f32(g), t, lr, b1, b2, ea)
    torch.cuda.synchronize()
    check_item(it, ref, True, lr)


@pytest.mark.parametrize("m,n,r,q,t,moments", [
    (300, 264, 16, 4, 1, False),    # ragged against the 128 x 256 workgroup tile
    (256, 512, 64, 8, 3, True),
    (130, 1000, 100, 2, 7, True),   # r = 100 padded to 128
    (256, 512, 128, 4, 2, True),
    (17, 8, 4, 4, 1, False),
])
@pytest.mark.parametrize("lr", [1e-3, 1e-2])
def test_f16_update_parity(m, n, r, q, t, moments, lr):
    """fp16 W (the paper's precision): the same kernel with fp16 conversions of W; stored values
    RNE to fp16 of the fp32 hook, held to the fp16 ulp.  At the full-tuning learning rate 1e-3
    the 1-ulp bar covers at least half of the entries; at 1e-2 the update's rounding bound
    exceeds half an fp16 ulp on most entries (down to 1% covered at r = 128), so there the
    hook bound and the exact rounding of the hook carry the check."""
    it = make_item(21, (m, n, r), m, n, r, q, False, moments, f16=True)
    g = zd.f32(zd.draw(21, "G", (m, n, r), (q,), 1e-2))
    b1, b2, ea = 0.9, 0.95, 1e-8
    ref = expected(it, g.astype(np.float64), t, lr, b1, b2, ea)
    zo.subspace_adam_update([it["dev"]], dev_f32(g), t, lr, b1, b2, ea)
    torch.cuda.synchronize()
    check_item(it, ref, True, lr, min_held=0.5 if lr <= 1e-3 else None)


@pytest.mark.parametrize("m,n,r,q", [(256, 512, 4, 4), (33, 71, 5, 3), (1, 1, 1, 1), (200, 264, 128, 2)])
def test_fp32_update_parity(m, n, r, q):
    it = make_item(1, (m, n, r), m, n, r, q, False, True)
    g = zd.f32(zd.draw(1, "G", (m, n, r), (q,), 1e-1))
    ref = expected(it, g.astype(np.float64), 2, 1e-2, 0.9, 0.999, 1e-8)
    zo.subspace_adam_update([it["dev"]], dev_f32(g), 2, 1e-2, 0.9, 0.999, 1e-8)
    torch.cuda.synchronize()
    check_item(it, ref, False, 1e-2)


def test_update_subspace_invariant():
    """U^T (W_new - W_old) V = -lr S (through the fp32 hook)."""
    m, n, r, q = 512, 768, 16, 4
    it = make_item(2, (9,), m, n, r, q, True, True)
    g = zd.f32(zd.draw(2, "G", (9,), (q,), 1e-2))
    ref = expected(it, g.astype(np.float64), 4, 1e-2, 0.9, 0.95, 1e-8)
    zo.subspace_adam_update([it["dev"]], dev_f32(g), 4, 1e-2, 0.9, 0.95, 1e-8)
    torch.cuda.synchronize()
    D = host(it["dev"]["w_f32_out"]) - it["Wv"]
    proj = it["U"].astype(np.float64).T @ D @ it["V"].astype(np.float64)
    assert normwise(proj, -F32(1e-2) * ref["S"]) <= 1e-4


def test_nonfinite_estimate_leaves_state_untouched():
    m, n, r, q = 64, 128, 8, 4
    it = make_item(3, (1,), m, n, r, q, True, True)
    g = np.array([1.0, np.nan, 0.5, 0.1], np.float32)
    w0 = it["dev"]["W"].clone()
    m10, m20 = it["dev"]["M1"].clone(), it["dev"]["M2"].clone()
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    it["dev"]["w_f32_out"] = None
    zo.subspace_adam_update([it["dev"]], dev_f32(g), 1, 1e-2, 0.9, 0.95, 1e-8, nonfinite_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 1
    assert torch.equal(it["dev"]["W"].view(torch.int16), w0.view(torch.int16))
    assert torch.equal(it["dev"]["M1"], m10) and torch.equal(it["dev"]["M2"], m20)


def test_batched_heterogeneous_items():
    """Mixed shapes in one call (more than one group of the descriptor fill), one global g."""
    r, q = 16, 4
    shapes = [(64 + 8 * i, 256 + 64 * (i % 3)) for i in range(21)]
    items = [make_item(4, (i,), m, n, r, q, True, i % 2 == 1) for i, (m, n) in enumerate(shapes)]
    g = zd.f32(zd.draw(4, "G", (0,), (q,), 1e-2))
    refs = [expected(it, g.astype(np.float64), 5, 5e-3, 0.9, 0.95, 1e-8) for it in items]
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    zo.subspace_adam_update([it["dev"] for it in items], dev_f32(g), 5, 5e-3, 0.9, 0.95, 1e-8, nonfinite_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0
    for it, ref in zip(items, refs):
        check_item(it, ref, True, 5e-3)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_many_items_mixed_hooks(dt):
    """150 items in one call: the descriptor table takes ten fill launches and the workgroup ->
    item search two rounds; every third item has no check hook and no zbar_out, so the
    hook-writing kernel variant also runs items without a hook buffer."""
    bf16 = dt == "bf16"
    r, q, lr, t = 8, 2, 5e-3, 2
    shapes = [(16 + 8 * (i % 7), 64 + 64 * (i % 3)) for i in range(150)]
    items = [make_item(6, (i,), m, n, r, q, bf16, i % 2 == 1) for i, (m, n) in enumerate(shapes)]
    for i, it in enumerate(items):
        if i % 3 == 2:
            it["dev"]["w_f32_out"] = None
            it["dev"]["zbar_out"] = None
    g = zd.f32(zd.draw(6, "G", (0,), (q,), 1e-2))
    refs = [expected(it, g.astype(np.float64), t, lr, 0.9, 0.95, 1e-8) for it in items]
    zo.subspace_adam_update([it["dev"] for it in items], dev_f32(g), t, lr, 0.9, 0.95, 1e-8)
    torch.cuda.synchronize()
    for i, (it, ref) in enumerate(zip(items, refs)):
        if it["dev"]["w_f32_out"] is not None:
            check_item(it, ref, bf16, lr)
            continue
        got_w = host(it["dev"]["W"])
        if bf16:
            # No hook: the stored value is RNE of a value within E of W_exact.
            E = update_bound(it["U"], it["V"], ref["S"], lr, ref["W"])
            half_ulp = np.maximum(np.exp2(np.frexp(got_w)[1] - 9.0), np.exp2(np.frexp(ref["W"])[1] - 9.0))
            assert np.all(np.abs(got_w - ref["W"]) <= E + half_ulp), i
            assert normwise(got_w, ref["W"]) <= 2e-3
        else:
            assert ferr(got_w, ref["W"], 1.0) <= 1e-5, i
        np.testing.assert_allclose(host(it["dev"]["M1"]), ref["M1"], rtol=1e-6, atol=1e-12)
        np.testing.assert_allclose(host(it["dev"]["M2"]), ref["M2"], rtol=1e-6, atol=1e-14)


def test_thousands_of_items():
    """4500 tiny items in one call: 282 fill launches and a three-round workgroup -> item search
    (4500 > 64 * 64), for the bf16 path; every item checked against the oracle."""
    r, q, lr, t = 4, 2, 1e-2, 1
    shapes = [(8 + 8 * (i % 5), 8 + 8 * (i % 2)) for i in range(4500)]
    items = [make_item(7, (i,), m, n, r, q, True, False) for i, (m, n) in enumerate(shapes)]
    g = zd.f32(zd.draw(7, "G", (0,), (q,), 1e-2))
    refs = [expected(it, g.astype(np.float64), t, lr, 0.9, 0.95, 1e-8) for it in items]
    zo.subspace_adam_update([it["dev"] for it in items], dev_f32(g), t, lr, 0.9, 0.95, 1e-8)
    torch.cuda.synchronize()
    got_hook = host(torch.cat([it["dev"]["w_f32_out"].reshape(-1) for it in items]))
    want = np.concatenate([ref["W"].reshape(-1) for ref in refs])
    assert ferr(got_hook, want, 1.0) <= 5e-5
    for i in (0, 1, 63, 64, 4095, 4096, 4499):
        check_item(items[i], refs[i], True, lr)


@pytest.mark.parametrize("name,m,n,rank,f16", [("opt-1.3b", 8192, 2048, None, False),
                                                ("llama-7b", 11008, 4096, None, False),
                                                ("llama-7b", 4096, 11008, None, False),
                                                ("opt-13b", 20480, 5120, None, False),
                                                ("opt-13b", 5120, 20480, None, False),
                                                ("opt-13b", 20480, 5120, 128, False),
                                                ("opt-13b", 5120, 20480, 128, False),
                                                ("opt-13b", 20480, 5120, None, True),
                                                ("opt-13b", 5120, 20480, None, True)])
def test_full_size_sampled(name, m, n, rank, f16):
    """Full-size update of the largest matrices of each stack (the config's r, q, lr, betas; the
    OPT-13B shapes also at the paper's full-tuning rank r = 128 and with fp16 W, the paper's
    precision); sampled rows vs the oracle."""
    cfg = zd.CONFIGS[name]
    q, lr, b1, b2 = cfg["q"], cfg["lr"], cfg["beta1"], cfg["beta2"]
    r = rank or cfg["r"]
    it = make_item(5, (m, n), m, n, r, q, not f16, True, f16=f16)
    g = zd.f32(zd.draw(5, "G", (m, n), (q,), 1e-2))
    zo.subspace_adam_update([it["dev"]], dev_f32(g), 3, lr, b1, b2, 1e-8)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 127, 128, m // 2 + 3, m - 1])
    Zbar = oracle.aggregate(g.astype(np.float64), it["Z"])
    _, _, S = oracle.adam_direction(it["M1h"], it["M2h"], Zbar, 3, F32(b1), F32(b2), F32(1e-8))
    W_rows = it["Wv"][rows] - F32(lr) * (it["U"][rows].astype(np.float64) @ S @ it["V"].astype(np.float64).T)
    got_hook = host(it["dev"]["w_f32_out"][torch.from_numpy(rows).cuda()])
    got_w = host(it["dev"]["W"][torch.from_numpy(rows).cuda()])
    assert ferr(got_hook, W_rows, 1.0) <= 5e-5
    E = update_bound(it["U"][rows], it["V"], S, lr, W_rows)
    assert check_bf16_storage(got_w, got_hook, W_rows, E, f16) < 1e-2
    np.testing.assert_allclose(host(it["dev"]["M1"]), oracle.adam_direction(
        it["M1h"], it["M2h"], Zbar, 3, F32(b1), F32(b2), F32(1e-8))[0], rtol=1e-6, atol=1e-12)


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("m,n,r,q", [(300, 264, 16, 4), (512, 1024, 64, 8), (129, 72, 5, 1)])
def test_sgd_update_parity(dt, m, n, r, q):
    """Subspace SGD (S = Zbar; q = 1 is SubZero's update): the same bars as the Adam update;
    moments given to the call are left untouched."""
    bf16, f16 = dt == "bf16", dt == "f16"
    it = make_item(11, (m, n, 7), m, n, r, q, bf16, moments=True, f16=f16)
    g = zd.f32(zd.draw(11, "G", (m, n, 7), (q,), 1e-2))
    M1_before = host(it["dev"]["M1"]).copy()
    zo.subspace_sgd_update([it["dev"]], dev_f32(g), 1e-3)
    torch.cuda.synchronize()
    ref = oracle.subspace_sgd_update(it["Wv"], it["U"], it["V"], it["Z"], g.astype(np.float64), F32(1e-3))
    got_hook = host(it["dev"]["w_f32_out"])
    got_w = host(it["dev"]["W"])
    if bf16 or f16:
        assert ferr(got_hook, ref["W"], 1.0) <= 5e-5
        E = update_bound(it["U"], it["V"], ref["Zbar"], 1e-3, ref["W"])
        assert check_bf16_storage(got_w, got_hook, ref["W"], E, f16) < 1e-2
        assert normwise(got_w, ref["W"]) <= 2e-3
    else:
        assert ferr(got_w, ref["W"], 1.0) <= 1e-5
    np.testing.assert_allclose(host(it["dev"]["zbar_out"]), ref["Zbar"], rtol=1e-6, atol=1e-9)
    np.testing.assert_array_equal(host(it["dev"]["M1"]), M1_before)


def test_sgd_update_without_moments_and_nonfinite_guard():
    m, n, r, q = 256, 512, 16, 4
    it = make_item(12, (m, n), m, n, r, q, True)
    dev = {k: v for k, v in it["dev"].items() if k not in ("M1", "M2")}
    W0 = host(dev["W"]).copy()
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    g = dev_f32(np.array([1.0, np.nan, 0.5, 0.0], np.float32))
    zo.subspace_sgd_update([dev], g, 1e-2, nonfinite_flag=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 1
    np.testing.assert_array_equal(host(dev["W"]), W0)
    g = zd.f32(zd.draw(12, "G", (m, n), (q,), 1e-2))
    zo.subspace_sgd_update([dev], dev_f32(g), 1e-2)
    torch.cuda.synchronize()
    ref = oracle.subspace_sgd_update(it["Wv"], it["U"], it["V"], it["Z"], g.astype(np.float64), F32(1e-2))
    assert ferr(host(dev["w_f32_out"]), ref["W"], 1.0) <= 5e-5


def test_max_queries_aggregate():
    """q = ZO_MAX_QUERIES coefficient matrices aggregated with their global estimates (Eq. 6)."""
    m, n, r, q = 64, 128, 8, 256
    it = make_item(31, (m, n, r), m, n, r, q, True, True)
    g = zd.f32(zd.draw(31, "G", (m, n, r), (q,), 1e-2))
    lr, b1, b2, ea = 1e-2, 0.9, 0.95, 1e-8
    ref = expected(it, g.astype(np.float64), 2, lr, b1, b2, ea)
    zo.subspace_adam_update([it["dev"]], dev_f32(g), 2, lr, b1, b2, ea)
    torch.cuda.synchronize()
    check_item(it, ref, True, lr)
