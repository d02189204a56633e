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
