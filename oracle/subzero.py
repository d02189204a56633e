"""float64 reference of every step on the SubZero+ hot path (test infrastructure).

Each function cites the passage of the paper it follows.  Readings of points
where the paper is silent or ambiguous are marked READING and listed in the
design notes of the repository.

Pins (independent checks that this file is right) live in
``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "householder_qr", "haar_qr", "raw_qr_first_column",
    "perturbation", "perturbed_weight", "perturbed_linear", "perturbed_linear_blocks",
    "lora_perturbed_factors", "lora_perturbed_linear", "lora_perturbed_linear_blocks",
    "layer_norm", "causal_attention", "DECODER_MATS", "decoder_layer",
    "rms_norm", "rope", "silu", "LLAMA_MATS", "llama_layer", "LORA_LAYER_MATS", "llama_lora_layer",
    "sq_loss", "central_estimate", "forward_estimate", "aggregate",
    "adam_direction", "subspace_adam_update", "subspace_sgd_update", "round_bf16", "round_f16", "tiny_run",
]


# ---------------------------------------------------------------------------
# Subspace construction: Eq. 11 / Alg. 1 (HaarProjMatrix)
# ---------------------------------------------------------------------------
def householder_qr(A):
    """Thin QR of a tall matrix by Householder reflections (textbook algorithm).

    Returns (Q, R) with A = Q R, Q rows x r with orthonormal columns, R r x r
    upper triangular.  The sign of each R_kk is whatever the reflector choice
    gives (alpha = -sign(x_0) ||x||, the choice that avoids cancellation), i.e.
    an implementation-dependent convention -- exactly the situation the paper's
    sign correction addresses (Sec. "QR Subspace Construction with Sign
    Correction").  A column that is already zero below and on the diagonal
    gets no reflector and R_kk = 0.
    """
    A = np.array(A, dtype=np.float64, copy=True)
    rows, r = A.shape
    if rows < r:
        raise ValueError("householder_qr needs rows >= columns")
    vs = []
    for k in range(r):
        x = A[k:, k]
        normx = math.sqrt(float(np.dot(x, x)))
        if normx == 0.0:
            vs.append(None)
            continue
        alpha = -math.copysign(normx, x[0])
        v = x.copy()
        v[0] -= alpha
        v /= math.sqrt(float(np.dot(v, v)))
        # H = I - 2 v v^T applied to the trailing block.
        A[k:, k:] -= 2.0 * np.outer(v, v @ A[k:, k:])
        A[k + 1:, k] = 0.0
        vs.append(v)
    R = np.triu(A[:r, :])
    Q = np.zeros((rows, r), dtype=np.float64)
    Q[:r, :r] = np.eye(r)
    for k in reversed(range(r)):
        v = vs[k]
        if v is None:
            continue
        Q[k:, :] -= 2.0 * np.outer(v, v @ Q[k:, :])
    return Q, R


def haar_qr(Omega):
    """Haar-distributed orthonormal factor: Eq. 11 / Alg. 1.

    QR of the Gaussian matrix, then each column of Q is multiplied by the sign
    of the matching diagonal entry of R, so that the corrected R has a positive
    diagonal.  READING: sgn(0) := +1 (the paper leaves it undefined); a zero
    diagonal entry is reported through ``rank_deficient_col`` (first such
    column, or -1).

    Returns (U, R_corrected, rank_deficient_col).
    """
    Q, R = householder_qr(Omega)
    d = np.diag(R)
    s = np.where(d < 0.0, -1.0, 1.0)
    zero = np.nonzero(d == 0.0)[0]
    return Q * s[None, :], R * s[:, None], (int(zero[0]) if zero.size else -1)


def raw_qr_first_column(Omega):
    """First column of Q from the same QR without the sign correction (negative control)."""
    Q, _ = householder_qr(Omega)
    return Q[:, 0]


# ---------------------------------------------------------------------------
# Perturbation: Eq. 4, Alg. 2 (PerturbParams), linear layer of Eq. 5
# ---------------------------------------------------------------------------
def perturbation(U, Z, V):
    """Full-space perturbation U Z V^T of one matrix for one query (Eq. 4)."""
    U = np.asarray(U, np.float64)
    V = np.asarray(V, np.float64)
    Z = np.asarray(Z, np.float64)
    return U @ Z @ V.T


def perturbed_weight(W, U, V, Z, sign, eps):
    """W + sign * eps * U Z V^T, materialised (Alg. 2 with scale sign*eps)."""
    return np.asarray(W, np.float64) + (sign * eps) * perturbation(U, Z, V)


def perturbed_linear(X, W, U, V, Z, sign, eps):
    """Output of a linear layer (nn.Linear layout, W is out x in) under the
    perturbed weight: X (W + sign eps U Z V^T)^T (Eq. 5's forward, one layer)."""
    Wp = perturbed_weight(W, U, V, Z, sign, eps)
    return np.asarray(X, np.float64) @ Wp.T


def perturbed_linear_blocks(Xb, W, U, V, Zs, blk_query, blk_sign, eps, rows=None):
    """Blocks b = 0..nblk-1: Y_b = X_b (W + s_b eps U Z_{j(b)} V^T)^T.

    ``Xb`` is a list of per-block activations (T x n).  ``rows`` optionally
    restricts each block to a subset of its rows (the layer is row-wise, so
    sampled rows are computed exactly as in the full product).
    """
    out = []
    for b, X in enumerate(Xb):
        Xr = np.asarray(X, np.float64) if rows is None else np.asarray(X, np.float64)[rows]
        out.append(perturbed_linear(Xr, W, U, V, Zs[blk_query[b]], float(blk_sign[b]), eps))
    return out


# ---------------------------------------------------------------------------
# LoRA scheme: the trainable parameters are the two adapter factors
# (Sec. "Algorithm" -- SubZero+ applies to the trainable parameters of each
# scheme; Sec. "Experiments" -- LoRA with r = 8, alpha = 16)
# ---------------------------------------------------------------------------
def lora_perturbed_factors(A, UA, VA, ZA, B, UB, VB, ZB, sign, eps):
    """Both adapter factors under one query, each in its own subspace (Eq. 4
    applied to every trainable matrix, Alg. 2):

        A' = A + sign eps U_A Z_A V_A^T   (r_L x n),
        B' = B + sign eps U_B Z_B V_B^T   (m x r_L).

    READING: the two factors of a layer take part in the same query with the
    same sign, as every trainable matrix does in Alg. 3.
    """
    return (perturbed_weight(A, UA, VA, ZA, sign, eps),
            perturbed_weight(B, UB, VB, ZB, sign, eps))


def lora_perturbed_linear(X, W, A, UA, VA, ZA, B, UB, VB, ZB, sign, eps, scale):
    """Output of a LoRA-adapted linear layer under one query, materialised:
    X (W + scale B' A')^T with the frozen base W (out x in).

    READING: scale = alpha / r_L, the usual LoRA scaling (2 for r_L = 8,
    alpha = 16).
    """
    Ap, Bp = lora_perturbed_factors(A, UA, VA, ZA, B, UB, VB, ZB, sign, eps)
    Weff = np.asarray(W, np.float64) + scale * (Bp @ Ap)
    return np.asarray(X, np.float64) @ Weff.T


def lora_perturbed_linear_blocks(Xb, W, A, UA, VA, ZAs, B, UB, VB, ZBs, blk_query, blk_sign,
                                 eps, scale, rows=None):
    """Blocks b = 0..nblk-1 of the LoRA layer: query j(b), sign s(b); ``rows``
    optionally restricts each block to a subset of its rows."""
    out = []
    for b, X in enumerate(Xb):
        Xr = np.asarray(X, np.float64) if rows is None else np.asarray(X, np.float64)[rows]
        j = blk_query[b]
        out.append(lora_perturbed_linear(Xr, W, A, UA, VA, ZAs[j], B, UB, VB, ZBs[j],
                                         float(blk_sign[b]), eps, scale))
    return out


# ---------------------------------------------------------------------------
# The network whose loss each query evaluates (Eq. 5; Alg. 3 query loop): a
# pre-LN decoder layer of the OPT family with every weight matrix perturbed
# ---------------------------------------------------------------------------
def layer_norm(X, gamma, beta, eps_ln=1e-5):
    """Row-wise layer normalisation (x - mean) / sqrt(var + eps_ln) * gamma + beta, with the
    population variance of each row (the normalisation inside the OPT decoder layers the
    paper fine-tunes).  READING: eps_ln = 1e-5."""
    X = np.asarray(X, np.float64)
    mu = X.mean(axis=1, keepdims=True)
    var = ((X - mu) ** 2).mean(axis=1, keepdims=True)
    return (X - mu) / np.sqrt(var + eps_ln) * np.asarray(gamma, np.float64) + np.asarray(beta, np.float64)


def causal_attention(Q, K, V, heads, seq_len, kv_heads=None):
    """Multi-head causal self-attention of one block of T token rows holding T / seq_len
    sequences one after another: for each sequence and head h (columns h dh .. (h+1) dh - 1,
    dh = d / heads), query t attends to keys t' <= t of its own sequence with weights
    softmax_t'(q_t . k_t' / sqrt(dh)) and returns the weighted sum of the v_t'.
    ``kv_heads`` (grouped key/value heads, a divisor of heads): K and V hold kv_heads heads
    of dh columns, and query head h reads key/value head h // (heads / kv_heads)."""
    Q, K, V = (np.asarray(a, np.float64) for a in (Q, K, V))
    T, d = Q.shape
    dh = d // heads
    group = heads // (kv_heads or heads)
    O = np.zeros_like(Q)
    future = np.triu(np.ones((seq_len, seq_len), dtype=bool), 1)
    for s0 in range(0, T, seq_len):
        rows = slice(s0, s0 + seq_len)
        for h in range(heads):
            c = slice(h * dh, (h + 1) * dh)
            ckv = slice((h // group) * dh, (h // group + 1) * dh)
            S = Q[rows, c] @ K[rows, ckv].T / math.sqrt(dh)
            S[future] = -np.inf
            S = S - S.max(axis=1, keepdims=True)
            P = np.exp(S)
            P = P / P.sum(axis=1, keepdims=True)
            O[rows, c] = P @ V[rows, ckv]
    return O


DECODER_MATS = ("q", "k", "v", "o", "fc1", "fc2")


def decoder_layer(H, layer, sign, eps, j, heads, seq_len, store=None, eps_ln=1e-5, trace=None):
    """One pre-LN decoder layer under query j with sign s: each of its six weight matrices W
    (q, k, v, o, fc1, fc2; each with its own U, V and coefficients Z_j) enters as
    W + s eps U Z_j V^T (Eq. 4), and
        A = LN1(H);   Q, K, V = A Wq'^T, A Wk'^T, A Wv'^T;   C = attention(Q, K, V)
        H2 = H + C Wo'^T;   F = relu(LN2(H2) W1'^T);   H3 = H2 + F W2'^T.
    ``store`` (optional) rounds each tensor the layer writes to memory, at the points where
    a device path stores one (e.g. round_bf16); all arithmetic is float64.  ``trace`` (an
    optional dict) receives the stored intermediates A, Q, K, V, C, H2, A2, F.
    READING: no biases (the perturbed parameters are the weight matrices); ReLU, as in OPT."""
    st = store if store is not None else (lambda x: x)
    lin = lambda X, name: perturbed_linear(X, layer[name]["W"], layer[name]["U"], layer[name]["V"],
                                           layer[name]["Z"][j], sign, eps)
    A = st(layer_norm(H, layer["ln1_g"], layer["ln1_b"], eps_ln))
    Q, K, Vv = st(lin(A, "q")), st(lin(A, "k")), st(lin(A, "v"))
    C = st(causal_attention(Q, K, Vv, heads, seq_len))
    H2 = st(np.asarray(H, np.float64) + lin(C, "o"))
    A2 = st(layer_norm(H2, layer["ln2_g"], layer["ln2_b"], eps_ln))
    F = st(np.maximum(lin(A2, "fc1"), 0.0))
    if trace is not None:
        trace.update(A=A, Q=Q, K=K, V=Vv, C=C, H2=H2, A2=A2, F=F)
    return st(H2 + lin(F, "fc2"))


# ---------------------------------------------------------------------------
# The same for a decoder layer of the LLaMA family (the other full-tuning
# family of the experiments): RMS normalisation, rotary positions, SwiGLU MLP
# ---------------------------------------------------------------------------
def rms_norm(X, gamma, eps_rms=1e-6):
    """Row-wise RMS normalisation x / sqrt(mean(x^2) + eps_rms) * gamma (no centring, no bias).
    READING: eps_rms = 1e-6."""
    X = np.asarray(X, np.float64)
    ms = (X * X).mean(axis=1, keepdims=True)
    return X / np.sqrt(ms + eps_rms) * np.asarray(gamma, np.float64)


def rope(X, seq_len, heads, base=10000.0):
    """Rotary position embedding of query or key rows of one block (T token rows holding
    T / seq_len sequences one after another; a row's position is its index within its
    sequence).  In each head of dh = d / heads columns, dimension i < dh/2 and its partner
    i + dh/2 are rotated together by the angle p * base^(-2i/dh):
        (a, b) -> (a cos - b sin, b cos + a sin).
    READING: the half-split pairing and base 10000 of the LLaMA checkpoints' usual form."""
    X = np.asarray(X, np.float64)
    T, d = X.shape
    dh = d // heads
    half = dh // 2
    pos = (np.arange(T) % seq_len).astype(np.float64)
    theta = base ** (-2.0 * np.arange(half, dtype=np.float64) / dh)
    ang = pos[:, None] * theta[None, :]
    c, s = np.cos(ang), np.sin(ang)
    out = X.copy()
    for h in range(heads):
        a = X[:, h * dh:h * dh + half]
        b = X[:, h * dh + half:(h + 1) * dh]
        out[:, h * dh:h * dh + half] = a * c - b * s
        out[:, h * dh + half:(h + 1) * dh] = b * c + a * s
    return out


def silu(x):
    """x * sigmoid(x), the gate non-linearity of the SwiGLU MLP."""
    x = np.asarray(x, np.float64)
    return x / (1.0 + np.exp(-x))


LLAMA_MATS = ("q", "k", "v", "o", "gate", "up", "down")


def llama_layer(H, layer, sign, eps, j, heads, seq_len, store=None, eps_rms=1e-6, rope_base=10000.0,
                trace=None):
    """One pre-norm decoder layer of the LLaMA family under query j with sign s, each of its
    seven weight matrices (q, k, v, o, gate, up, down; each with its own U, V and Z_j)
    entering as W + s eps U Z_j V^T (Eq. 4):
        A = RMS1(H);   Q = rope(A Wq'^T);  K = rope(A Wk'^T);  V = A Wv'^T
        C = attention(Q, K, V);   H2 = H + C Wo'^T;   A2 = RMS2(H2)
        F = silu(A2 Wg'^T) * (A2 Wu'^T);   H3 = H2 + F Wd'^T.
    ``store`` rounds each tensor at the points where the device path stores one (Q and K
    are stored before and after the rotation; the gate output before it enters F); all
    arithmetic float64.  ``trace`` receives A, Q, K, V, C, H2, A2, G, F."""
    st = store if store is not None else (lambda x: x)
    lin = lambda X, name: perturbed_linear(X, layer[name]["W"], layer[name]["U"], layer[name]["V"],
                                           layer[name]["Z"][j], sign, eps)
    A = st(rms_norm(H, layer["rms1_g"], eps_rms))
    Q = st(rope(st(lin(A, "q")), seq_len, heads, rope_base))
    K = st(rope(st(lin(A, "k")), seq_len, heads, rope_base))
    Vv = st(lin(A, "v"))
    C = st(causal_attention(Q, K, Vv, heads, seq_len))
    H2 = st(np.asarray(H, np.float64) + lin(C, "o"))
    A2 = st(rms_norm(H2, layer["rms2_g"], eps_rms))
    G = st(lin(A2, "gate"))
    F = st(silu(G) * lin(A2, "up"))
    if trace is not None:
        trace.update(A=A, Q=Q, K=K, V=Vv, C=C, H2=H2, A2=A2, G=G, F=F)
    return st(H2 + lin(F, "down"))


LORA_LAYER_MATS = ("q", "k", "v", "o", "gate", "up", "down")


def llama_lora_layer(H, layer, sign, eps, j, heads, kv_heads, seq_len, scale, store=None, eps_rms=1e-6,
                     rope_base=1e6, trace=None):
    """The LLaMA-family layer of the LoRA scheme (the Qwen models of the experiments): grouped
    key/value heads (k and v project to kv_heads * dh columns), frozen base weights, and LoRA
    adapters on q and v whose factors are the perturbed parameters (Eq. 4 on A and B, as in
    lora_perturbed_linear):
        A = RMS1(H);   Q = rope(A (Wq + scale B_q' A_q')^T);   K = rope(A Wk^T)
        V = A (Wv + scale B_v' A_v')^T;   C = attention(Q, K, V; kv_heads)
        H2 = H + C Wo^T;   A2 = RMS2(H2);   F = silu(A2 Wg^T) * (A2 Wu^T);   H3 = H2 + F Wd^T.
    layer["q"], layer["v"]: W, A, UA, VA, ZA (q x r x r), B, UB, VB, ZB; the others: W.
    ``store`` rounds each tensor where a device path stores one (as in llama_layer).
    READING: rope_base 1e6 (the Qwen2.5 models); no biases, as for the other layers."""
    st = store if store is not None else (lambda x: x)
    lin = lambda X, name: np.asarray(X, np.float64) @ np.asarray(layer[name]["W"], np.float64).T

    def lora(X, name):
        m = layer[name]
        return lora_perturbed_linear(X, m["W"], m["A"], m["UA"], m["VA"], m["ZA"][j], m["B"], m["UB"], m["VB"],
                                     m["ZB"][j], sign, eps, scale)

    A = st(rms_norm(H, layer["rms1_g"], eps_rms))
    Q = st(rope(st(lora(A, "q")), seq_len, heads, rope_base))
    K = st(rope(st(lin(A, "k")), seq_len, kv_heads, rope_base))
    Vv = st(lora(A, "v"))
    C = st(causal_attention(Q, K, Vv, heads, seq_len, kv_heads))
    H2 = st(np.asarray(H, np.float64) + lin(C, "o"))
    A2 = st(rms_norm(H2, layer["rms2_g"], eps_rms))
    G = st(lin(A2, "gate"))
    F = st(silu(G) * lin(A2, "up"))
    if trace is not None:
        trace.update(A=A, Q=Q, K=K, V=Vv, C=C, H2=H2, A2=A2, G=G, F=F)
    return st(H2 + lin(F, "down"))


# ---------------------------------------------------------------------------
# Losses and the estimate: Eqs. 3, 5, 6; Alg. 3 query loop
# ---------------------------------------------------------------------------
def sq_loss(Y, Ystar):
    """Squared loss of the Tiny configuration: 0.5 ||Y - Y*||_F^2 / T (T = rows)."""
    D = np.asarray(Y, np.float64) - np.asarray(Ystar, np.float64)
    return 0.5 * float(np.sum(D * D)) / D.shape[0]


def central_estimate(Lp, Lm, eps):
    """Central difference (L+ - L-) / (2 eps) per query (the two-point scheme of
    Eq. 3, applied to every query; READING: the central scheme replaces the
    forward difference of Eq. 6 / Alg. 3 for this hot path)."""
    return (np.asarray(Lp, np.float64) - np.asarray(Lm, np.float64)) / (2.0 * eps)


def forward_estimate(L, L0, eps):
    """Forward difference rho_k = (l_k - l_0) / eps (Eq. 6, Alg. 3)."""
    return (np.asarray(L, np.float64) - float(L0)) / eps


def aggregate(g, Zs):
    """Aggregated low-rank gradient Zbar = (1/K) sum_k rho_k Z^(k) (Sec. 3.1, Alg. 3)."""
    g = np.asarray(g, np.float64)
    Zs = np.asarray(Zs, np.float64)
    acc = np.zeros(Zs.shape[1:], dtype=np.float64)
    for k in range(len(g)):
        acc += g[k] * Zs[k]
    return acc / len(g)


# ---------------------------------------------------------------------------
# Subspace Adam: Eqs. 7-10
# ---------------------------------------------------------------------------
def adam_direction(M1, M2, Zbar, t, beta1, beta2, eps_adam):
    """One step of Adam on the r x r aggregated gradient (Eqs. 7-9).

    READING: t is the 1-based step index (the paper's loop counts from 0,
    which would divide by zero in the bias correction).  Returns
    (M1_new, M2_new, S) with S = Mhat / (sqrt(Vhat) + eps_adam), eps_adam
    outside the square root.
    """
    if t < 1:
        raise ValueError("Adam step index is 1-based")
    Zbar = np.asarray(Zbar, np.float64)
    M1n = beta1 * np.asarray(M1, np.float64) + (1.0 - beta1) * Zbar
    M2n = beta2 * np.asarray(M2, np.float64) + (1.0 - beta2) * (Zbar * Zbar)
    mhat = M1n / (1.0 - beta1 ** t)
    vhat = M2n / (1.0 - beta2 ** t)
    S = mhat / (np.sqrt(vhat) + eps_adam)
    return M1n, M2n, S


def subspace_adam_update(W, U, V, Zs, g, M1, M2, t, lr, beta1, beta2, eps_adam):
    """Full once-per-step update of one matrix (Alg. 3 tail, Eqs. 7-10).

    Zbar = (1/q) sum_j g_j Z_j; Adam in r x r; W_new = W - lr U S V^T (exact,
    float64).  READING: the trailing factor of Eq. 10 is the n x r right
    projection (dimension check), the denominator uses the r x r moment.
    Returns dict(W=W_new, M1, M2, S, Zbar).
    """
    Zbar = aggregate(g, Zs)
    M1n, M2n, S = adam_direction(M1, M2, Zbar, t, beta1, beta2, eps_adam)
    Wn = np.asarray(W, np.float64) - lr * (np.asarray(U, np.float64) @ S @ np.asarray(V, np.float64).T)
    return dict(W=Wn, M1=M1n, M2=M2n, S=S, Zbar=Zbar)


# ---------------------------------------------------------------------------
# bfloat16 storage rounding (format, not method): single rounding from float64
# ---------------------------------------------------------------------------
def subspace_sgd_update(W, U, V, Zs, g, lr):
    """Plain SGD in the subspace (the "SubZero+/SGD" rows of the experiments; with q = 1
    SubZero's update W - eta rho U Z V^T of Sec. "Preliminaries"):
    Zbar = (1/q) sum_j g_j Z_j, W_new = W - lr U Zbar V^T (exact, float64).
    Returns dict(W=W_new, Zbar)."""
    Zbar = aggregate(g, Zs)
    W_new = np.asarray(W, np.float64) - lr * (np.asarray(U, np.float64) @ Zbar @ np.asarray(V, np.float64).T)
    return dict(W=W_new, Zbar=Zbar)


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 (8 significant bits), ties to even.

    Written from the format definition: x = f 2^e with 0.5 <= |f| < 1; the
    bf16 quantum at that binade is 2^(e-8); rint() rounds half to even.
    Overflow/subnormal ranges are not needed for weights and are not handled.
    """
    x = np.asarray(x, dtype=np.float64)
    f, e = np.frexp(x)
    q = np.ldexp(1.0, e - 8)
    return np.rint(x / q) * q


def round_f16(x):
    """Round float64 values to the nearest IEEE binary16 value, ties to even.

    Written from the format definition: 11 significant bits, so the quantum
    in the binade [2^(e-1), 2^e) is 2^(e-11); below the smallest normal
    2^-14 the quantum stays 2^-24 (subnormals); a result beyond the largest
    finite value (2 - 2^-10) 2^15 = 65504 becomes an infinity of x's sign.
    """
    x = np.asarray(x, dtype=np.float64)
    f, e = np.frexp(x)
    q = np.ldexp(1.0, np.maximum(e - 11, -24))
    y = np.rint(x / q) * q
    return np.where(np.abs(y) > 65504.0, np.copysign(np.inf, x), y)


# ---------------------------------------------------------------------------
# Tiny configuration end to end (Alg. 3 with the central estimate)
# ---------------------------------------------------------------------------
def tiny_run(inputs, omega_fn, z_fn, cfg, g_override=None, estimator="central"):
    """Alg. 3 on the one-layer Tiny problem, float64.

    inputs: dict(W, X, Ystar) arrays.  omega_fn(t) -> (Omega_U, Omega_V) for a
    refresh at step t; z_fn(t) -> Z[q, r, r].  g_override(t, g) may replace
    the estimates (teacher forcing).  Per step t = 0..steps-1: refresh if
    t mod F == 0; for each query j the loss of W + eps U Z_j V^T and either
    the loss of W - eps U Z_j V^T, g_j = (L+ - L-)/(2 eps) (estimator
    "central"), or the baseline loss of W, g_j = (L+ - L0)/eps (estimator
    "forward", Eq. 6); Adam update with step index t+1.
    Returns a list of per-step records.
    """
    W = np.asarray(inputs["W"], np.float64)
    X = np.asarray(inputs["X"], np.float64)
    Ystar = np.asarray(inputs["Ystar"], np.float64)
    r, q, eps = cfg["r"], cfg["q"], cfg["eps"]
    M1 = np.zeros((r, r))
    M2 = np.zeros((r, r))
    U = V = None
    recs = []
    for t in range(cfg["steps"]):
        if t % cfg["F"] == 0:
            ou, ov = omega_fn(t)
            U, _, _ = haar_qr(ou)
            V, _, _ = haar_qr(ov)
        Zs = np.asarray(z_fn(t), np.float64)
        Lp = np.array([sq_loss(perturbed_linear(X, W, U, V, Zs[j], +1.0, eps), Ystar) for j in range(q)])
        if estimator == "forward":
            Lm = None
            L0 = sq_loss(X @ W.T, Ystar)
            g = forward_estimate(Lp, L0, eps)
        else:
            Lm = np.array([sq_loss(perturbed_linear(X, W, U, V, Zs[j], -1.0, eps), Ystar) for j in range(q)])
            L0 = None
            g = central_estimate(Lp, Lm, eps)
        if g_override is not None:
            g = np.asarray(g_override(t, g), np.float64)
        upd = subspace_adam_update(W, U, V, Zs, g, M1, M2, t + 1, cfg["lr"],
                                   cfg["beta1"], cfg["beta2"], cfg["eps_adam"])
        W_before = W
        W, M1, M2 = upd["W"], upd["M1"], upd["M2"]
        recs.append(dict(t=t, U=U, V=V, Z=Zs, Lp=Lp, Lm=Lm, L0=L0, g=g, S=upd["S"], Zbar=upd["Zbar"],
                         W_before=W_before, W=W, M1=M1, M2=M2,
                         loss=sq_loss(X @ W.T, Ystar)))
    return recs
