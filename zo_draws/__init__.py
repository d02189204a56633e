"""Seeded synthetic inputs for the SubZero+ hot path.

This module is shared by the CPU oracle (``oracle/``) and by the GPU path's
tests and benchmark.  It draws random numbers and builds input tensors; it
holds none of the method's arithmetic (no QR, no perturbation, no loss, no
optimizer step).

Draw contract
-------------
The paper fixes no generator, fill order or stream split for its Gaussian
draws (Alg. 1 first step, Alg. 2 per-layer draw, Alg. 3 per-query seed).
Every draw here is keyed, so any array can be regenerated on its own:

    draw(seed, kind, idx, shape, sigma)

fills ``shape`` in C order with ``sigma * N(0, 1)`` in float64.  The flat
array is cut into chunks of ``CHUNK`` elements; chunk ``c`` comes from
``numpy.random.Generator(PCG64(SeedSequence(entropy=seed,
spawn_key=(KIND[kind],) + idx + (c,)))).standard_normal``.  Chunks are
independent streams, so large arrays are filled by several threads with a
result that does not depend on the thread count.

Casts: float64 -> float32 by ``astype`` (round to nearest even); float32 ->
bfloat16 by integer round-to-nearest-even on the float32 bit pattern.  The
bf16 value of a float64 draw is therefore rounded twice, deliberately, and
the same bits are handed to both sides.
"""
from __future__ import annotations

import hashlib
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNK = 1 << 22

KIND = {
    "W0": 1,        # initial weight of a matrix
    "X": 2,         # activations (one T x n block per distinct n)
    "WSTAR": 3,     # Tiny target: W* = W + N(0, 0.01^2)
    "OMEGA_U": 4,   # Gaussian input of the left projection QR
    "OMEGA_V": 5,   # Gaussian input of the right projection QR
    "Z": 6,         # per-query r x r perturbation coefficients
    "LORA_A": 7,
    "LORA_B": 8,
    "G": 9,         # synthetic per-query estimates (update-only tests)
    "MOM": 10,      # synthetic Adam moments (update-only tests)
}


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _fill_chunk(out_flat: np.ndarray, seed: int, key: tuple, c: int) -> None:
    lo = c * CHUNK
    hi = min(out_flat.size, lo + CHUNK)
    ss = np.random.SeedSequence(entropy=seed, spawn_key=key + (c,))
    gen = np.random.Generator(np.random.PCG64(ss))
    gen.standard_normal(hi - lo, dtype=np.float64, out=out_flat[lo:hi])


def draw(seed: int, kind: str, idx: tuple, shape, sigma: float = 1.0) -> np.ndarray:
    """sigma * N(0,1) array of ``shape`` (float64, C order), keyed by (seed, kind, idx)."""
    shape = tuple(int(s) for s in (shape if isinstance(shape, (tuple, list)) else (shape,)))
    key = (KIND[kind],) + tuple(int(i) for i in idx)
    out = np.empty(shape, dtype=np.float64)
    flat = out.reshape(-1)
    nchunk = (flat.size + CHUNK - 1) // CHUNK
    if nchunk <= 1:
        if flat.size:
            _fill_chunk(flat, seed, key, 0)
    else:
        with ThreadPoolExecutor(max_workers=_threads()) as ex:
            list(ex.map(lambda c: _fill_chunk(flat, seed, key, c), range(nchunk)))
    if sigma != 1.0:
        out *= sigma
    return out


def f32(a: np.ndarray) -> np.ndarray:
    """float64 -> float32, round to nearest even."""
    return np.asarray(a, dtype=np.float64).astype(np.float32)


def bf16_bits(a32: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), integer round-to-nearest-even."""
    a32 = np.ascontiguousarray(a32, dtype=np.float32)
    u = a32.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(a32)
    if nan.any():
        rounded[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return rounded


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float32 (exact)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def as_bf16_values(a64: np.ndarray):
    """Cast a float64 draw to bf16: returns (bits uint16, exact float64 values of those bits)."""
    bits = bf16_bits(f32(a64))
    return bits, bf16_to_f32(bits).astype(np.float64)


def as_f16_values(a64: np.ndarray):
    """Cast a float64 draw to IEEE binary16 via float32 (both steps round to nearest even):
    returns (float16 array, exact float64 values of it)."""
    h = f32(a64).astype(np.float16)
    return h, h.astype(np.float64)


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def block_roll_rows(x0: np.ndarray, nblk: int) -> np.ndarray:
    """Distinct activations per block: block b is x0 with its rows rolled by b*floor(T/nblk).

    Returns the stacked (nblk*T, n) array.  Stands in for the per-query inputs
    that a real network hands to a layer after the first one.
    """
    T = x0.shape[0]
    step = T // max(nblk, 1)
    return np.concatenate([np.roll(x0, b * step, axis=0) for b in range(nblk)], axis=0)


# --------------------------------------------------------------------------
# Tiny configuration: one fp32 linear layer W 256x512, X 64x512, r=4, q=4.
# --------------------------------------------------------------------------
TINY = dict(m=256, n=512, T=64, r=4, q=4, eps=1e-3, lr=1e-2, beta1=0.9,
            beta2=0.999, eps_adam=1e-8, steps=20, F=5, seed=0)


def tiny_inputs(seed: int = 0) -> dict:
    """W, X, W*, Y* of the Tiny configuration as float32 (Y* = fp32 of X W*^T in fp64)."""
    c = TINY
    W = f32(draw(seed, "W0", (0,), (c["m"], c["n"]), 0.02))
    X = f32(draw(seed, "X", (0,), (c["T"], c["n"]), 1.0))
    Wstar = f32(W.astype(np.float64) + draw(seed, "WSTAR", (0,), (c["m"], c["n"]), 0.01))
    Ystar = f32(X.astype(np.float64) @ Wstar.astype(np.float64).T)
    return dict(W=W, X=X, Wstar=Wstar, Ystar=Ystar)


def omega_pair(seed: int, t_refresh: int, mat: int, m: int, n: int, r: int):
    """Gaussian inputs (Omega_U: m x r, Omega_V: n x r) as float32 for a refresh at step t."""
    ou = f32(draw(seed, "OMEGA_U", (t_refresh, mat), (m, r)))
    ov = f32(draw(seed, "OMEGA_V", (t_refresh, mat), (n, r)))
    return ou, ov


def z_draws(seed: int, t: int, mat: int, q: int, r: int) -> np.ndarray:
    """Per-query coefficients Z[q, r, r] (float32) for matrix ``mat`` at step ``t``."""
    return np.stack([f32(draw(seed, "Z", (t, j, mat), (r, r))) for j in range(q)])


# --------------------------------------------------------------------------
# Model-shaped stacks (shapes only; weights are synthetic).
# --------------------------------------------------------------------------
def _stack(name, layers, mats, T, r, q, eps=1e-3, lr=1e-3, F=100, beta1=0.9, beta2=0.95, decoder=None):
    return dict(name=name, layers=layers, mats=mats, T=T, r=r, q=q, eps=eps, lr=lr,
                F=F, beta1=beta1, beta2=beta2, eps_adam=1e-8, decoder=decoder)


CONFIGS = {
    "opt-1.3b": _stack("opt-1.3b", 24,
                       [("q", 2048, 2048), ("k", 2048, 2048), ("v", 2048, 2048),
                        ("o", 2048, 2048), ("fc1", 8192, 2048), ("fc2", 2048, 8192)],
                       T=4096, r=16, q=4, F=500,
                       decoder=dict(d=2048, heads=32, ffn=8192, seq_len=256)),   # 16 sequences x 256
    "llama-7b": _stack("llama-7b", 32,
                       [("q", 4096, 4096), ("k", 4096, 4096), ("v", 4096, 4096),
                        ("o", 4096, 4096), ("gate", 11008, 4096), ("up", 11008, 4096),
                        ("down", 4096, 11008)],
                       T=4096, r=32, q=4,
                       decoder=dict(d=4096, heads=32, ffn=11008, seq_len=256, family="llama")),  # 16 x 256
    "opt-13b": _stack("opt-13b", 40,
                      [("q", 5120, 5120), ("k", 5120, 5120), ("v", 5120, 5120),
                       ("o", 5120, 5120), ("fc1", 20480, 5120), ("fc2", 5120, 20480)],
                      T=8192, r=64, q=8,
                      decoder=dict(d=5120, heads=40, ffn=20480, seq_len=512)),  # batch 16 x 512
    # LoRA on q and v of a frozen base; each factor has its own r=4 subspace.
    "qwen-32b-lora": _stack("qwen-32b-lora", 64,
                            [("q", 5120, 5120), ("k", 1024, 5120), ("v", 1024, 5120),
                             ("o", 5120, 5120), ("gate", 27648, 5120), ("up", 27648, 5120),
                             ("down", 5120, 27648)],
                            T=4096, r=4, q=4, lr=1e-2,
                            decoder=dict(d=5120, heads=40, kv_heads=8, ffn=27648, seq_len=256,  # 16 x 256
                                         family="llama-lora", rope_base=1e6)),
}
QWEN_LORA_RANK = 8
QWEN_LORA_ALPHA = 16
