"""Shared helpers of the tests: tolerance measures and host<->device conversions."""
import numpy as np

import zo_draws as zd


def ferr(a, b, tau):
    """Floored relative error max_i |a_i - b_i| / max(|b_i|, tau * rms(b))."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    rms = float(np.sqrt(np.mean(b * b))) if b.size else 0.0
    den = np.maximum(np.abs(b), tau * rms)
    den = np.where(den == 0.0, 1.0, den)
    return float(np.max(np.abs(a - b) / den)) if a.size else 0.0


def normwise(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def orth(seed, idx, rows, r):
    """A column-orthonormal float32 test matrix (LAPACK QR of a keyed draw)."""
    Q, _ = np.linalg.qr(zd.draw(seed, "OMEGA_U", (7777,) + tuple(idx), (rows, r)))
    return Q.astype(np.float32)


def dev_f32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def dev_bf16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)).view(torch.bfloat16).cuda()


def dev_f16(h):
    import torch
    return torch.from_numpy(np.ascontiguousarray(h, dtype=np.float16)).cuda()


def host_bf16_values(t):
    """float64 values of a bf16 device tensor."""
    import torch
    bits = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return zd.bf16_to_f32(bits).astype(np.float64)


def host(t):
    import torch
    if t.dtype == torch.bfloat16:
        return host_bf16_values(t)
    return t.detach().cpu().numpy().astype(np.float64)


def cast(a64, dt):
    """(device tensor, exact float64 values) of a float64 array in dtype dt."""
    if dt == "bf16":
        bits, v = zd.as_bf16_values(a64)
        return dev_bf16(bits), v
    if dt == "f16":
        h, v = zd.as_f16_values(a64)
        return dev_f16(h), v
    v = zd.f32(a64).astype(np.float64)
    return dev_f32(v), v


def rnd(dt):
    """The oracle's rounding of a stored activation of type dt."""
    import oracle
    return oracle.round_f16 if dt == "f16" else oracle.round_bf16


def check16(got, ref, what):
    """The bar of one 16-bit rounding of a kernel's output: floored relative error <= 1e-2 at
    floor 1e-3 rms, normwise <= 2e-3."""
    assert ferr(got, ref, 1e-3) <= 1e-2, what
    assert normwise(got, ref) <= 2e-3, what


def ulp16(x, dt):
    """Spacing of 16-bit values (fp16 with its subnormals, or bf16) at |x|."""
    e = np.frexp(x)[1]
    return np.ldexp(1.0, np.maximum(e - 11, -24)) if dt == "f16" else np.ldexp(1.0, e - 8)


def check_attention(got, Q, K, V, heads, seq_len, dt, what, kv_heads=None):
    """Causal attention held to the bar its arithmetic sets.  P enters the P V product as a
    hi + lo pair of 16-bit values (relative error <= 2^-17 for bf16 pairs, less for fp16), and
    the fp32 logits carry an absolute error of a few 2^-24 |q| |k|, which moves P by under
    2^-16 relative at logits of a few hundred.  So before its rounding each output is within
    2^-14 softmax(S) |V| (the same average taken of |V|, with margin) of the exact one, and
    after it within one ulp more; blockwise it keeps the normwise bar of a single rounding."""
    import oracle
    ref = oracle.causal_attention(Q, K, V, heads, seq_len, kv_heads)
    mag = oracle.causal_attention(Q, K, np.abs(V), heads, seq_len, kv_heads)
    assert normwise(got, ref) <= 2e-3, what
    bound = ulp16(ref, dt) + 2.0 ** -14 * mag
    err = np.abs(np.asarray(got, np.float64) - ref)
    assert np.all(err <= bound), (what, float(np.max(err / bound)))


def spacing32(y):
    """Spacing of float32 values at |y| (one ulp)."""
    return np.spacing(np.abs(np.asarray(y, np.float64)).astype(np.float32)).astype(np.float64)


def estimate_noise_bar(Yplus, Yminus, Ystar, eps, r, T, g, k=6.0, rel=1e-5):
    """Per-query bar on |g_gpu - g_exact| / max(|g_exact|, rms(g_exact)) for estimates formed
    from fp32 outputs of the fp32 perturbed linear.

    Yplus[j] is the exact output of query j's + block (the oracle's).  Central estimate,
    g_j = (L(Y+_j) - L(Y-_j)) / (2 eps): Yminus[j] is the exact output of its - block.
    Forward estimate, g_j = (L(Y+_j) - L(Y_0)) / eps: Yminus is None (the baseline block
    adds exact zeros as its rank-r term, so its output carries no rounding that the + block
    does not share).  L = 0.5 sum (Y - Y*)^2 / T is accumulated in fp64, so its own error is
    negligible; what moves g is the rounding of Y.  The two sides of a difference share
    X W^T bit for bit (same X, same W, same summation order); the rank-r term is then added
    by r fused multiply-adds, each rounding at the scale of |Y| with an error uniform in
    +-ulp/2 (variance ulp^2 / 12), independently for the two sides.  The shared error of
    X W^T enters only through Y+ - Y- = O(eps), and W, U, V differ from the oracle's
    float64 ones by fp32 rounding: both are covered by the `rel` term.  So

        var(T * delta(L+_j - L-_j)) = sum_i (Y+_ji - Y*_i)^2 r ulp(Y+_ji)^2 / 12
                                      + the same for Y-_j (central only)

    and the bar is k = 6 standard deviations plus rel |g_j|, over the floored |g_j|."""
    Ystar = np.asarray(Ystar, np.float64)
    g = np.asarray(g, np.float64)
    floor = np.maximum(np.abs(g), np.sqrt(np.mean(g * g)))

    def var(Y):
        Y = np.asarray(Y, np.float64)
        return np.sum((Y - Ystar) ** 2 * r * spacing32(Y) ** 2 / 12.0)

    out = []
    for j, Yp in enumerate(Yplus):
        v = var(Yp) + (var(Yminus[j]) if Yminus is not None else 0.0)
        sigma = np.sqrt(v) / (T * (2.0 * eps if Yminus is not None else eps))
        out.append((k * sigma + rel * abs(g[j])) / floor[j])
    return np.array(out)
