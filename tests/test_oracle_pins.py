"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every test here checks the oracle against something other than itself:
hand-derived values (tests/golden), closed forms, invariants, library special
cases (LAPACK QR, Cholesky, Kronecker products, torch.optim.Adam) and exact
distributions.  No GPU is used.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.special
import scipy.stats

import oracle
import zo_draws as zd

RNG = np.random.default_rng(1234)


def _orth(rows, r, seed):
    Q, _ = np.linalg.qr(np.random.default_rng(seed).standard_normal((rows, r)))
    return Q


# --------------------------------------------------------------------------- QR
def test_qr_hand_cases(golden_dir):
    """Eq. 11 / Alg. 1: the sign-corrected thin QR equals the hand-derived unique factor."""
    cases = json.load(open(os.path.join(golden_dir, "qr_hand.json")))["cases"]
    for c in cases:
        U, R, bad = oracle.haar_qr(np.array(c["omega"]))
        np.testing.assert_allclose(U, np.array(c["Q"]), rtol=0, atol=1e-15, err_msg=c["name"])
        np.testing.assert_allclose(R, np.array(c["R"]), rtol=0, atol=1e-15, err_msg=c["name"])
        assert bad == -1


@pytest.mark.parametrize("rows,r", [(200, 8), (50, 10), (33, 33), (1000, 64)])
def test_qr_first_column_closed_form(rows, r):
    """With diag(R) > 0 the first column is Omega[:,0] / ||Omega[:,0]|| exactly."""
    Om = RNG.standard_normal((rows, r))
    U, R, _ = oracle.haar_qr(Om)
    np.testing.assert_allclose(U[:, 0], Om[:, 0] / np.linalg.norm(Om[:, 0]), rtol=0, atol=1e-14)
    assert R[0, 0] == pytest.approx(np.linalg.norm(Om[:, 0]), rel=1e-14)


@pytest.mark.parametrize("rows,r", [(64, 4), (512, 16), (300, 37), (2048, 64)])
def test_qr_matches_cholesky_form(rows, r):
    """Uniqueness: R = chol(Omega^T Omega)^T (positive diagonal) and Q = Omega R^-1."""
    Om = RNG.standard_normal((rows, r))
    U, R, _ = oracle.haar_qr(Om)
    Rc = np.linalg.cholesky(Om.T @ Om).T
    Qc = scipy.linalg.solve_triangular(Rc, Om.T, trans="T", lower=False).T
    np.testing.assert_allclose(R, Rc, rtol=0, atol=1e-10 * np.abs(Rc).max())
    np.testing.assert_allclose(U, Qc, rtol=0, atol=1e-10)


@pytest.mark.parametrize("rows,r", [(100, 1), (256, 4), (512, 32), (4096, 64)])
def test_qr_matches_lapack_with_sign_fix(rows, r):
    """Library special case: LAPACK's thin QR followed by the column sign fix."""
    Om = RNG.standard_normal((rows, r))
    Ql, Rl = np.linalg.qr(Om, mode="reduced")
    s = np.where(np.diag(Rl) < 0, -1.0, 1.0)
    U, R, _ = oracle.haar_qr(Om)
    np.testing.assert_allclose(U, Ql * s, rtol=0, atol=1e-12)
    np.testing.assert_allclose(R, Rl * s[:, None], rtol=0, atol=1e-12 * np.abs(Rl).max())


@pytest.mark.parametrize("rows,r", [(512, 16), (777, 5), (2000, 64)])
def test_qr_invariants(rows, r):
    Om = RNG.standard_normal((rows, r))
    U, R, bad = oracle.haar_qr(Om)
    assert bad == -1
    assert np.abs(U.T @ U - np.eye(r)).max() < 1e-13
    assert np.abs(U @ R - Om).max() < 1e-12 * np.abs(Om).max()
    assert np.all(np.diag(R) > 0)
    assert np.abs(np.tril(U.T @ Om, -1)).max() < 1e-12


def test_qr_rank_deficient_column_reported():
    """READING of sgn(0): a zero column gives R_kk = 0, reported as rank-deficient."""
    Om = RNG.standard_normal((40, 6))
    Om[:, 3] = 0.0
    U, R, bad = oracle.haar_qr(Om)
    assert bad == 3
    assert R[3, 3] == 0.0
    # The other columns are still orthonormal and the factorisation still holds.
    assert np.abs(U @ R - Om).max() < 1e-12


def _coord_cdf(m):
    """Exact CDF of one coordinate of a uniform unit vector in R^m:
    x^2 ~ Beta(1/2, (m-1)/2) and the distribution is symmetric."""
    def cdf(x):
        x = np.asarray(x)
        return 0.5 + 0.5 * np.sign(x) * scipy.special.betainc(0.5, (m - 1) / 2.0, x * x)
    return cdf


@pytest.mark.parametrize("seed", [0, 42])
def test_haar_ks_appendix_setup(seed, golden_dir):
    """Appendix Haar validation (Table 9 setup: m = 50, r = 10, 2000 trials).

    The corrected first column must follow the exact Haar marginal (KS p > 0.05);
    the uncorrected one (negative control) must be rejected.  Our draws differ
    from the paper's, so the paper's D values are compared only in size.
    """
    g = json.load(open(os.path.join(golden_dir, "paper_haar_ks.json")))
    m, r, n = g["m"], g["r"], g["trials"]
    corr = np.empty(n)
    raw = np.empty(n)
    corr1 = np.empty(n)
    for i in range(n):
        Om = zd.draw(seed, "OMEGA_U", (99999, i), (m, r))
        U, _, _ = oracle.haar_qr(Om)
        corr[i] = U[0, 0]
        corr1[i] = U[1, 0]
        raw[i] = oracle.raw_qr_first_column(Om)[0]
    cdf = _coord_cdf(m)
    kc = scipy.stats.kstest(corr, cdf)
    kc1 = scipy.stats.kstest(corr1, cdf)
    kr = scipy.stats.kstest(raw, cdf)
    assert kc.pvalue > 0.05 and kc1.pvalue > 0.05
    assert kc.statistic < 2.5 * g["corrected"]["seed0"]["D"]
    assert kr.pvalue < 1e-3
    # Coordinate variance of a uniform unit vector is exactly 1/m.
    var = float(np.mean(corr ** 2))
    assert abs(var - 1.0 / m) < 4 * math.sqrt(2.0 / n) / m + 1e-12
    assert g["theory_variance"] == pytest.approx(1.0 / m)


# ------------------------------------------------------------- perturbed linear
def test_perturbed_linear_hand_example():
    """X = [1, 2], W = I, U = e1, V = e2, Z = 3, eps = 0.5: W+ = [[1, 1.5], [0, 1]], Y = [4, 2]."""
    X = np.array([[1.0, 2.0]])
    W = np.eye(2)
    U = np.array([[1.0], [0.0]])
    V = np.array([[0.0], [1.0]])
    Z = np.array([[3.0]])
    np.testing.assert_array_equal(oracle.perturbed_linear(X, W, U, V, Z, +1.0, 0.5), [[4.0, 2.0]])
    np.testing.assert_array_equal(oracle.perturbed_linear(X, W, U, V, Z, -1.0, 0.5), [[-2.0, 2.0]])


def _pl_case(T=37, m=48, n=64, r=5, seed=7):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, n))
    W = 0.02 * rng.standard_normal((m, n))
    U = _orth(m, r, seed + 1)
    V = _orth(n, r, seed + 2)
    Z = rng.standard_normal((r, r))
    return X, W, U, V, Z


def test_perturbed_linear_special_cases():
    X, W, U, V, Z = _pl_case()
    base = np.matmul(X, W.T)
    np.testing.assert_allclose(oracle.perturbed_linear(X, W, U, V, Z, 1.0, 0.0), base, rtol=0, atol=1e-14)
    np.testing.assert_allclose(oracle.perturbed_linear(X, W, U, V, 0 * Z, -1.0, 1e-3), base, rtol=0, atol=1e-14)


@pytest.mark.parametrize("eps", [1e-3, 1.0])
def test_perturbed_linear_factored_identity(eps):
    """X (W + s eps U Z V^T)^T = X W^T + s eps (X V)(U Z)^T (the route that never forms U Z V^T)."""
    X, W, U, V, Z = _pl_case()
    for s in (+1.0, -1.0):
        fact = X @ W.T + s * eps * (X @ V) @ (U @ Z).T
        np.testing.assert_allclose(oracle.perturbed_linear(X, W, U, V, Z, s, eps), fact, rtol=0, atol=1e-12)
    yp = oracle.perturbed_linear(X, W, U, V, Z, 1.0, eps)
    ym = oracle.perturbed_linear(X, W, U, V, Z, -1.0, eps)
    np.testing.assert_allclose(yp + ym, 2 * X @ W.T, rtol=0, atol=1e-12)


def test_lemma1_kronecker_and_norm():
    """Lemma 1 of SubZero (restated in the Preliminaries): vec(U Z V^T) = (V kron U) vec(Z),
    and with column-orthonormal U, V the Frobenius norm is preserved."""
    _, _, U, V, Z = _pl_case(m=20, n=30, r=4)
    P = oracle.perturbation(U, Z, V)
    vec = lambda A: A.reshape(-1, order="F")
    np.testing.assert_allclose(vec(P), np.kron(V, U) @ vec(Z), rtol=0, atol=1e-14)
    assert np.linalg.norm(P) == pytest.approx(np.linalg.norm(Z), rel=1e-13)
    K = np.kron(V, U)
    assert np.abs(K.T @ K - np.eye(16)).max() < 1e-13


def test_perturbed_linear_blocks_rows_subset():
    X, W, U, V, Z = _pl_case(T=20)
    Zs = np.stack([Z, 2 * Z])
    Xb = [X, X[::-1].copy(), X, X]
    full = oracle.perturbed_linear_blocks(Xb, W, U, V, Zs, [0, 0, 1, 1], [1, -1, 1, -1], 1e-2)
    rows = np.array([0, 5, 19])
    part = oracle.perturbed_linear_blocks(Xb, W, U, V, Zs, [0, 0, 1, 1], [1, -1, 1, -1], 1e-2, rows=rows)
    for b in range(4):
        np.testing.assert_array_equal(part[b], full[b][rows])
    np.testing.assert_allclose(full[2], X @ (W + 1e-2 * U @ (2 * Z) @ V.T).T, atol=1e-13)


# ------------------------------------------------------------------ LoRA scheme
def test_lora_hand_example():
    """Worked by hand: n = 2, m = r_L = r = 1, W = 0, X = [1, 2], A = [1, 0], B = [[2]],
    U_A = U_B = V_B = [[1]], V_A = e2, Z_A = 3, Z_B = -1, eps = 0.5, scale = 2.
    s = +1: A' = [1, 1.5], B' = 1.5, W_eff = 2 * 1.5 * A' = [3, 4.5], Y = 3 + 9 = 12.
    s = -1: A' = [1, -1.5], B' = 2.5, W_eff = [5, -7.5], Y = 5 - 15 = -10."""
    X = np.array([[1.0, 2.0]])
    W = np.zeros((1, 2))
    A = np.array([[1.0, 0.0]])
    B = np.array([[2.0]])
    one = np.array([[1.0]])
    VA = np.array([[0.0], [1.0]])
    args = (X, W, A, one, VA, np.array([[3.0]]), B, one, one, np.array([[-1.0]]))
    np.testing.assert_array_equal(oracle.lora_perturbed_linear(*args, +1.0, 0.5, 2.0), [[12.0]])
    np.testing.assert_array_equal(oracle.lora_perturbed_linear(*args, -1.0, 0.5, 2.0), [[-10.0]])


def _lora_case(T=9, m=7, n=11, rl=3, r=2, seed=11, zero_b=False):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, n))
    W = 0.02 * rng.standard_normal((m, n))
    A = 0.02 * rng.standard_normal((rl, n))
    B = np.zeros((m, rl)) if zero_b else 0.02 * rng.standard_normal((m, rl))
    UA, VA = _orth(rl, r, seed + 1), _orth(n, r, seed + 2)
    UB, VB = _orth(m, r, seed + 3), _orth(rl, r, seed + 4)
    ZA, ZB = rng.standard_normal((r, r)), rng.standard_normal((r, r))
    return X, W, A, UA, VA, ZA, B, UB, VB, ZB


def test_lora_brute_force_loops():
    """Element-by-element loops over the definition on a tiny case."""
    X, W, A, UA, VA, ZA, B, UB, VB, ZB = _lora_case(T=3, m=4, n=5, rl=2, r=2)
    s, eps, scale = -1.0, 0.3, 2.0
    T, n = X.shape
    m, rl = B.shape
    r = UA.shape[1]
    Ap = np.zeros((rl, n))
    for c in range(rl):
        for k in range(n):
            acc = A[c, k]
            for e in range(r):
                for f in range(r):
                    acc += s * eps * UA[c, e] * ZA[e, f] * VA[k, f]
            Ap[c, k] = acc
    Bp = np.zeros((m, rl))
    for i in range(m):
        for c in range(rl):
            acc = B[i, c]
            for e in range(r):
                for f in range(r):
                    acc += s * eps * UB[i, e] * ZB[e, f] * VB[c, f]
            Bp[i, c] = acc
    Y = np.zeros((T, m))
    for t in range(T):
        for i in range(m):
            acc = 0.0
            for k in range(n):
                w = W[i, k]
                for c in range(rl):
                    w += scale * Bp[i, c] * Ap[c, k]
                acc += X[t, k] * w
            Y[t, i] = acc
    got = oracle.lora_perturbed_linear(X, W, A, UA, VA, ZA, B, UB, VB, ZB, s, eps, scale)
    np.testing.assert_allclose(got, Y, rtol=0, atol=1e-13)


@pytest.mark.parametrize("eps", [1e-3, 0.5])
def test_lora_output_is_quadratic_in_eps(eps):
    """Both factors are affine in eps, so Y(s eps) = Y0 + s eps Y1 + eps^2 Y2 exactly:
    the even part isolates the product of the two perturbations and the odd part the two
    first-order terms.  A factor left unperturbed, or perturbed with the opposite sign,
    breaks one of the two."""
    X, W, A, UA, VA, ZA, B, UB, VB, ZB = _lora_case()
    scale = 2.0
    f = lambda s, e: oracle.lora_perturbed_linear(X, W, A, UA, VA, ZA, B, UB, VB, ZB, s, e, scale)
    PA = UA @ ZA @ VA.T
    PB = UB @ ZB @ VB.T
    Y0 = X @ (W + scale * B @ A).T
    Y1 = scale * X @ (B @ PA + PB @ A).T
    Y2 = scale * X @ (PB @ PA).T
    np.testing.assert_allclose(f(1.0, 0.0), Y0, rtol=0, atol=1e-14)
    np.testing.assert_allclose((f(1.0, eps) - f(-1.0, eps)) / (2 * eps), Y1, rtol=0, atol=1e-10)
    np.testing.assert_allclose((f(1.0, eps) + f(-1.0, eps)) / 2 - Y0, eps ** 2 * Y2, rtol=0, atol=1e-14)


def test_lora_reduces_to_full_tuning_case():
    """With A = I (r_L = n), Z_A = 0 and B = 0 the adapter is B' itself, so the layer is the
    full-tuning perturbed linear with Z scaled by the LoRA scale."""
    X, W, _, UA, VA, ZA, _, _, _, ZB = _lora_case(n=6, rl=6)
    m, n = W.shape
    UB, VB = _orth(m, 2, 5), _orth(n, 2, 6)
    A = np.eye(n)
    B = np.zeros((m, n))
    for s in (1.0, -1.0):
        got = oracle.lora_perturbed_linear(X, W, A, UA, VA, 0 * ZA, B, UB, VB, ZB, s, 1e-2, 2.0)
        ref = oracle.perturbed_linear(X, W, UB, VB, 2.0 * ZB, s, 1e-2)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-14)


def test_lora_zero_b_first_order_only_through_b():
    """Paper initialisation B = 0 with Z_A = 0: the branch is exactly linear in eps and
    equals scale * s eps X A^T (U_B Z_B V_B^T)^T."""
    X, W, A, UA, VA, ZA, B, UB, VB, ZB = _lora_case(zero_b=True)
    for s in (1.0, -1.0):
        got = oracle.lora_perturbed_linear(X, W, A, UA, VA, 0 * ZA, B, UB, VB, ZB, s, 0.25, 2.0)
        lin = X @ W.T + 2.0 * s * 0.25 * X @ A.T @ (UB @ ZB @ VB.T).T
        np.testing.assert_allclose(got, lin, rtol=0, atol=1e-14)


def test_lora_blocks_use_their_query_and_sign():
    X, W, A, UA, VA, ZA, B, UB, VB, ZB = _lora_case()
    ZAs, ZBs = np.stack([ZA, -2 * ZA]), np.stack([ZB, 3 * ZB])
    Xb = [X, X[::-1].copy(), X]
    out = oracle.lora_perturbed_linear_blocks(Xb, W, A, UA, VA, ZAs, B, UB, VB, ZBs, [1, 0, 1],
                                              [-1, 1, 0], 1e-2, 2.0, rows=np.array([0, 4]))
    ref0 = oracle.lora_perturbed_linear(X, W, A, UA, VA, -2 * ZA, B, UB, VB, 3 * ZB, -1.0, 1e-2, 2.0)
    np.testing.assert_array_equal(out[0], ref0[[0, 4]])
    np.testing.assert_allclose(out[2], (X @ (W + 2.0 * B @ A).T)[[0, 4]], rtol=0, atol=1e-14)


# --------------------------------------------------------------- loss, estimate
def test_sq_loss_hand():
    assert oracle.sq_loss([[1.0, 2.0]], [[0.0, 0.0]]) == 2.5
    assert oracle.sq_loss([[1.0], [3.0]], [[0.0], [1.0]]) == pytest.approx(0.5 * (1 + 4) / 2)


def _quad_problem(T=64, m=32, n=48, r=4, seed=3):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, n))
    W = 0.02 * rng.standard_normal((m, n))
    Ys = X @ (W + 0.01 * rng.standard_normal((m, n))).T
    U = _orth(m, r, seed + 10)
    V = _orth(n, r, seed + 11)
    grad = (X @ W.T - Ys).T @ X / T
    return X, W, Ys, U, V, grad


@pytest.mark.parametrize("eps", [1e-3, 1.0, 7.5])
def test_central_difference_exact_on_quadratic(eps):
    """On L(W) = 0.5||X W^T - Y*||^2 / T the central difference equals <grad L, U Z V^T>
    exactly for every eps (the quadratic terms cancel)."""
    X, W, Ys, U, V, grad = _quad_problem()
    Z = np.random.default_rng(9).standard_normal((4, 4))
    Lp = oracle.sq_loss(oracle.perturbed_linear(X, W, U, V, Z, 1.0, eps), Ys)
    Lm = oracle.sq_loss(oracle.perturbed_linear(X, W, U, V, Z, -1.0, eps), Ys)
    g = oracle.central_estimate([Lp], [Lm], eps)[0]
    exact = float(np.sum(grad * (U @ Z @ V.T)))
    assert g == pytest.approx(exact, rel=2e-9 if eps < 1e-2 else 1e-11, abs=1e-13)


def test_estimator_unbiased_monte_carlo():
    """E_Z[<grad L, U Z V^T> Z] = U^T grad L V (E[z z^T] = I); Monte Carlo with a 4-sigma bound."""
    X, W, Ys, U, V, grad = _quad_problem()
    target = U.T @ grad @ V
    N = 20000
    rng = np.random.default_rng(5)
    Zs = rng.standard_normal((N, 4, 4))
    # Exact central differences on a quadratic equal the directional derivative.
    g = np.array([np.sum(grad * (U @ Z @ V.T)) for Z in Zs])
    est = oracle.aggregate(g, Zs)
    bound = 4 * np.linalg.norm(target) * math.sqrt((16 + 1) / N)
    assert np.linalg.norm(est - target) < bound
    # Through the oracle's own loss route on a subset of draws (same expectation).
    sub = Zs[:200]
    gl = [oracle.central_estimate([oracle.sq_loss(oracle.perturbed_linear(X, W, U, V, Z, 1, 1e-2), Ys)],
                                  [oracle.sq_loss(oracle.perturbed_linear(X, W, U, V, Z, -1, 1e-2), Ys)], 1e-2)[0]
          for Z in sub]
    np.testing.assert_allclose(gl, g[:200], rtol=1e-8, atol=1e-12)


def test_forward_difference_unbiased_on_quadratic():
    """Eq. 6's forward difference: on a quadratic, E[(L(W+eps D)-L(W))/eps Z] is also U^T grad V
    (the eps^2 term is even in Z, its product with Z has zero mean)."""
    X, W, Ys, U, V, grad = _quad_problem(r=2)
    target = U.T @ grad @ V
    N = 20000
    Zs = np.random.default_rng(8).standard_normal((N, 2, 2))
    eps = 1e-3
    L0 = oracle.sq_loss(X @ W.T, Ys)
    XWt = X @ W.T - Ys
    # Closed-form loss of the perturbed weight keeps this fast: L(W+eps D) = 0.5||R + eps X D^T||^2/T.
    XV = X @ V
    Ls = np.array([0.5 * np.sum((XWt + eps * XV @ (U @ Z).T) ** 2) / X.shape[0] for Z in Zs[:2000]])
    Lchk = np.array([oracle.sq_loss(oracle.perturbed_linear(X, W, U, V, Z, 1, eps), Ys) for Z in Zs[:20]])
    np.testing.assert_allclose(Ls[:20], Lchk, rtol=1e-13)
    rho = oracle.forward_estimate(Ls, L0, eps)
    est = oracle.aggregate(rho, Zs[:2000])
    assert np.linalg.norm(est - target) < 4 * np.linalg.norm(target) * math.sqrt(5 / 2000) + 1e-6


@pytest.mark.parametrize("eps", [1e-3, 0.5])
def test_forward_difference_closed_form_on_quadratic(eps):
    """Eq. 6 on the quadratic L(W) = 0.5||X W^T - Y*||^2 / T: with P = U Z V^T,
    (L(W + eps P) - L(W)) / eps = <grad L, P> + (eps / 2) ||X P^T||^2 / T exactly."""
    X, W, Ys, U, V, grad = _quad_problem(r=3)
    Z = np.random.default_rng(31).standard_normal((3, 3))
    P = U @ Z @ V.T
    L0 = oracle.sq_loss(X @ W.T, Ys)
    L1 = oracle.sq_loss(oracle.perturbed_linear(X, W, U, V, Z, 1.0, eps), Ys)
    rho = oracle.forward_estimate(np.array([L1]), L0, eps)[0]
    exact = np.sum(grad * P) + 0.5 * eps * np.sum((X @ P.T) ** 2) / X.shape[0]
    assert rho == pytest.approx(exact, rel=1e-7 if eps < 1e-2 else 1e-11, abs=1e-12)


def test_tiny_forward_run_matches_its_definition():
    """The forward-difference variant of the Tiny loop: each step's g is (L(W + eps U Z_j V^T) - L(W)) / eps
    of that step's W, and a teacher-forced zero estimate leaves W unchanged."""
    inp = zd.tiny_inputs(0)
    cfg = dict(zd.TINY, steps=3)
    om = lambda t: zd.omega_pair(0, t, 0, cfg["m"], cfg["n"], cfg["r"])
    zf = lambda t: zd.z_draws(0, t, 0, cfg["q"], cfg["r"])
    recs = oracle.tiny_run(inp, om, zf, cfg, estimator="forward")
    X, Ys = inp["X"].astype(np.float64), inp["Ystar"]
    for rec in recs:
        L0 = oracle.sq_loss(X @ rec["W_before"].T, Ys)
        assert rec["L0"] == pytest.approx(L0, rel=1e-15)
        np.testing.assert_allclose(rec["g"], (rec["Lp"] - L0) / cfg["eps"], rtol=1e-12)
        assert rec["Lm"] is None
    zero = oracle.tiny_run(inp, om, zf, cfg, estimator="forward", g_override=lambda t, g: np.zeros_like(g))
    np.testing.assert_array_equal(zero[-1]["W"], inp["W"].astype(np.float64))


def test_aggregate_one_hot_and_linearity():
    Zs = RNG.standard_normal((5, 3, 3))
    np.testing.assert_allclose(oracle.aggregate([0, 0, 5.0, 0, 0], Zs), Zs[2], rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.aggregate(np.ones(5), Zs), Zs.mean(0), rtol=0, atol=1e-15)


# ------------------------------------------------------------------------- Adam
def test_adam_first_step_closed_form():
    """Step 1: Mhat = Zbar, Vhat = Zbar^2, so S = Zbar / (|Zbar| + eps_adam) whatever the betas."""
    Zb = RNG.standard_normal((6, 6))
    for b1, b2 in [(0.9, 0.999), (0.9, 0.95), (0.0, 0.0), (0.5, 0.3)]:
        _, _, S = oracle.adam_direction(np.zeros((6, 6)), np.zeros((6, 6)), Zb, 1, b1, b2, 1e-8)
        np.testing.assert_allclose(S, Zb / (np.abs(Zb) + 1e-8), rtol=1e-14, atol=0)


def test_adam_zero_betas_every_step():
    M1 = RNG.standard_normal((4, 4))
    M2 = RNG.random((4, 4))
    Zb = RNG.standard_normal((4, 4))
    for t in (1, 2, 17):
        _, _, S = oracle.adam_direction(M1, M2, Zb, t, 0.0, 0.0, 1e-8)
        np.testing.assert_allclose(S, Zb / (np.abs(Zb) + 1e-8), rtol=1e-14)


def test_adam_step_index_is_one_based():
    with pytest.raises(ValueError):
        oracle.adam_direction(np.zeros((2, 2)), np.zeros((2, 2)), np.ones((2, 2)), 0, 0.9, 0.95, 1e-8)


def test_adam_matches_torch_optim():
    """Library special case: torch.optim.Adam on an r x r parameter with gradient Zbar_t moves the
    parameter by exactly -lr * S_t each step (Eqs. 7-10 are Adam in the r x r space)."""
    torch = pytest.importorskip("torch")
    r, lr, b1, b2, ea = 5, 1e-2, 0.9, 0.95, 1e-8
    p = torch.zeros((r, r), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=lr, betas=(b1, b2), eps=ea)
    M1 = np.zeros((r, r))
    M2 = np.zeros((r, r))
    rng = np.random.default_rng(11)
    for t in range(1, 8):
        Zb = rng.standard_normal((r, r)) * (10.0 ** rng.integers(-3, 2))
        before = p.detach().clone().numpy()
        p.grad = torch.from_numpy(Zb.copy())
        opt.step()
        M1, M2, S = oracle.adam_direction(M1, M2, Zb, t, b1, b2, ea)
        np.testing.assert_allclose(p.detach().numpy() - before, -lr * S, rtol=1e-9, atol=1e-15)


def test_update_invariants():
    """U^T (W_new - W_old) V = -lr S and rank(W_new - W_old) <= r."""
    m, n, r, q = 40, 56, 4, 3
    U, V = _orth(m, r, 1), _orth(n, r, 2)
    W = 0.02 * RNG.standard_normal((m, n))
    Zs = RNG.standard_normal((q, r, r))
    g = RNG.standard_normal(q)
    out = oracle.subspace_adam_update(W, U, V, Zs, g, np.zeros((r, r)), np.zeros((r, r)), 1, 1e-2, 0.9, 0.95, 1e-8)
    D = out["W"] - W
    np.testing.assert_allclose(U.T @ D @ V, -1e-2 * out["S"], rtol=0, atol=1e-15)
    assert np.linalg.matrix_rank(D, tol=1e-12) <= r
    np.testing.assert_allclose(out["Zbar"], np.tensordot(g, Zs, 1) / q, rtol=1e-14)


def test_zero_estimates_leave_w_unchanged():
    m, n, r, q = 16, 24, 3, 4
    U, V = _orth(m, r, 3), _orth(n, r, 4)
    W = RNG.standard_normal((m, n))
    out = oracle.subspace_adam_update(W, U, V, RNG.standard_normal((q, r, r)), np.zeros(q),
                                      np.zeros((r, r)), np.zeros((r, r)), 1, 1e-2, 0.9, 0.95, 1e-8)
    np.testing.assert_array_equal(out["W"], W)


# ------------------------------------------------------------------ bf16 format
def test_sgd_update_single_query_is_subzero_step():
    """q = 1: W - lr g U Z V^T (SubZero's update), and U^T (W_new - W) V = -lr Zbar for any q."""
    rng = np.random.default_rng(21)
    m, n, r = 30, 20, 3
    W = rng.standard_normal((m, n))
    U, V = _orth(m, r, 1), _orth(n, r, 2)
    Z = rng.standard_normal((1, r, r))
    out = oracle.subspace_sgd_update(W, U, V, Z, [0.7], 0.1)
    np.testing.assert_allclose(out["W"], W - 0.1 * 0.7 * U @ Z[0] @ V.T, rtol=0, atol=1e-14)
    Zs = rng.standard_normal((4, r, r))
    g = rng.standard_normal(4)
    out = oracle.subspace_sgd_update(W, U, V, Zs, g, 0.05)
    Zbar = np.einsum("j,jab->ab", g, Zs) / 4
    np.testing.assert_allclose(U.T @ (out["W"] - W) @ V, -0.05 * Zbar, rtol=0, atol=1e-13)
    assert np.linalg.matrix_rank(out["W"] - W, tol=1e-10) <= r
    zero = oracle.subspace_sgd_update(W, U, V, Zs, np.zeros(4), 0.05)
    np.testing.assert_array_equal(zero["W"], W)


def test_round_bf16_hand_cases(golden_dir):
    cases = json.load(open(os.path.join(golden_dir, "bf16_rounding.json")))["cases"]
    for c in cases:
        assert oracle.round_bf16(c["x_value"]) == c["bf16"], c["x"]


def test_round_bf16_matches_torch_on_fp32_inputs():
    """For float32-representable inputs one rounding to bf16 is torch's float32->bfloat16 cast."""
    torch = pytest.importorskip("torch")
    x32 = (RNG.standard_normal(200000) * 10.0 ** RNG.uniform(-6, 3, 200000)).astype(np.float32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float32).numpy().astype(np.float64)
    np.testing.assert_array_equal(oracle.round_bf16(x32.astype(np.float64)), ref)


def test_round_f16_hand_cases(golden_dir):
    cases = json.load(open(os.path.join(golden_dir, "f16_rounding.json")))["cases"]
    for c in cases:
        got = oracle.round_f16(c["x_value"])
        assert got == float(c["f16"]), c["x"]
        assert np.signbit(got) == np.signbit(float(c["f16"])) or float(c["f16"]) == 0.0, c["x"]


def test_round_f16_matches_library_casts():
    """One rounding float64 -> binary16 is numpy's float16 cast, over normal, subnormal and
    overflowing magnitudes; on float32-representable inputs it is also torch's float32 ->
    float16 cast (torch's float64 -> float16 goes through float32, a double rounding)."""
    torch = pytest.importorskip("torch")
    x = RNG.standard_normal(200000) * 10.0 ** RNG.uniform(-9, 5.2, 200000)
    with np.errstate(over="ignore"):
        ref_np = x.astype(np.float16).astype(np.float64)
    got = oracle.round_f16(x)
    np.testing.assert_array_equal(got, ref_np)
    assert np.isinf(got).any() and (np.abs(got[np.isfinite(got)]) < 2.0 ** -14).any()
    x32 = x.astype(np.float32)
    ref_t = torch.from_numpy(x32).to(torch.float16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_f16(x32.astype(np.float64)), ref_t)


def test_fp32_in_place_restore_is_not_exact():
    """Alg. 2 adds then subtracts eps U Z V^T in place; in float32 that does not give W back
    bit for bit (why the GPU path never writes W during the queries)."""
    m, n, r = 256, 512, 4
    W = zd.f32(zd.draw(0, "W0", (0,), (m, n), 0.02))
    U, V = _orth(m, r, 5).astype(np.float32), _orth(n, r, 6).astype(np.float32)
    D = (1e-3 * (U @ RNG.standard_normal((r, r)).astype(np.float32) @ V.T)).astype(np.float32)
    back = (W + D) - D
    assert np.count_nonzero(back != W) > 0


# ------------------------------------------------------------------------ Tiny
def test_tiny_loop_teacher_forced_zero_is_identity():
    c = dict(zd.TINY, steps=3)
    inp = zd.tiny_inputs(0)
    recs = oracle.tiny_run(inp, lambda t: zd.omega_pair(0, t, 0, c["m"], c["n"], c["r"]),
                           lambda t: zd.z_draws(0, t, 0, c["q"], c["r"]), c,
                           g_override=lambda t, g: np.zeros_like(g))
    np.testing.assert_array_equal(recs[-1]["W"], inp["W"].astype(np.float64))


def test_tiny_loop_decreases_loss():
    c = zd.TINY
    inp = zd.tiny_inputs(0)
    recs = oracle.tiny_run(inp, lambda t: zd.omega_pair(0, t, 0, c["m"], c["n"], c["r"]),
                           lambda t: zd.z_draws(0, t, 0, c["q"], c["r"]), c)
    L0 = oracle.sq_loss(inp["X"].astype(np.float64) @ inp["W"].astype(np.float64).T, inp["Ystar"])
    assert recs[-1]["loss"] < L0
    # The g's are exact directional derivatives of a quadratic (checked above), so each g_j equals
    # <grad L(W_t), U Z_j V^T> up to the float64 cancellation of the difference.
    rec = recs[7]
    X = inp["X"].astype(np.float64)
    grad = (X @ rec["W_before"].T - inp["Ystar"]).T @ X / X.shape[0]
    exact = [np.sum(grad * (rec["U"] @ Z @ rec["V"].T)) for Z in rec["Z"]]
    np.testing.assert_allclose(rec["g"], exact, rtol=1e-6, atol=1e-9)


@pytest.mark.parametrize("estimator", ["central", "forward"])
def test_tiny_run_state_carried_across_steps_and_refreshes(estimator):
    """The 20-step loop's state from step to step, pinned against things other than the loop:
    - torch.optim.Adam (betas and eps of the run), stepped once per loop step with the run's own
      Zbar_t as the gradient of an r x r parameter, moves that parameter by exactly the run's
      subspace coordinates of the weight change, U_t^T (W_{t+1} - W_t) V_t = -lr S_t (Eq. 10
      with orthonormal U, V).  Torch keeps its moments across every step and refresh and
      counts steps from 1, so moments that were reset, not carried, or bias-corrected with the
      wrong index fail here;
    - W carries over: step t + 1 starts from step t's W;
    - the subspace is the sign-corrected LAPACK QR of Omega(t) at t mod F = 0 and unchanged in
      between (an off-by-one in the refresh cadence fails);
    - Zbar_t = (1/q) sum_j g_j Z_j;
    - each g_j is the exact directional derivative of the quadratic loss at W_t (central), or
      that plus eps/2 ||X P_j^T||^2 / T (forward, P_j = U Z_j V^T)."""
    torch = pytest.importorskip("torch")
    c = zd.TINY
    inp = zd.tiny_inputs(0)
    om = lambda t: zd.omega_pair(0, t, 0, c["m"], c["n"], c["r"])
    recs = oracle.tiny_run(inp, om, lambda t: zd.z_draws(0, t, 0, c["q"], c["r"]), c, estimator=estimator)
    assert len(recs) == c["steps"]
    r, X, Ys = c["r"], inp["X"].astype(np.float64), inp["Ystar"]
    p = torch.zeros((r, r), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=c["lr"], betas=(c["beta1"], c["beta2"]), eps=c["eps_adam"])
    W_prev = inp["W"].astype(np.float64)
    for t, rec in enumerate(recs):
        np.testing.assert_array_equal(rec["W_before"], W_prev)
        if t % c["F"] == 0:
            for got, omega in zip((rec["U"], rec["V"]), om(t)):
                Q, R = np.linalg.qr(np.asarray(omega, np.float64))
                np.testing.assert_allclose(got, Q * np.sign(np.diag(R))[None, :], rtol=0, atol=1e-12)
        else:
            np.testing.assert_array_equal(rec["U"], recs[t - 1]["U"])
            np.testing.assert_array_equal(rec["V"], recs[t - 1]["V"])
        np.testing.assert_allclose(rec["Zbar"], np.tensordot(rec["g"], rec["Z"], axes=1) / c["q"],
                                   rtol=1e-13, atol=1e-16)
        grad = (X @ rec["W_before"].T - Ys).T @ X / X.shape[0]
        P = [rec["U"] @ Z @ rec["V"].T for Z in rec["Z"]]
        exact = np.array([np.sum(grad * Pj) for Pj in P])
        if estimator == "forward":
            exact += np.array([0.5 * c["eps"] * np.sum((X @ Pj.T) ** 2) / X.shape[0] for Pj in P])
        np.testing.assert_allclose(rec["g"], exact, rtol=1e-6, atol=1e-9)
        before = p.detach().clone().numpy()
        p.grad = torch.from_numpy(np.array(rec["Zbar"], np.float64))
        opt.step()
        moved = rec["U"].T @ (rec["W"] - rec["W_before"]) @ rec["V"]
        np.testing.assert_allclose(moved, p.detach().numpy() - before, rtol=1e-8, atol=1e-13)
        W_prev = rec["W"]


# ---------------------------------------------------------------------------
# The decoder layer the queries run through (Eq. 5 inside Alg. 3)
# ---------------------------------------------------------------------------
def test_layer_norm_hand_case(golden_dir):
    c = json.load(open(os.path.join(golden_dir, "layernorm_hand.json")))
    x = np.array([c["x"]])
    n = oracle.layer_norm(x, np.ones(4), np.zeros(4), c["eps_ln"])[0]
    np.testing.assert_allclose(n, c["normalised"], rtol=0, atol=1e-15)
    y = oracle.layer_norm(x, np.array(c["gamma"]), np.array(c["beta"]), c["eps_ln"])[0]
    np.testing.assert_allclose(y, c["y"], rtol=0, atol=1e-15)


def test_layer_norm_closed_forms_and_torch():
    torch = pytest.importorskip("torch")
    X = RNG.standard_normal((37, 96)) * 3.0 + RNG.standard_normal((37, 1))
    eps_ln = 1e-5
    Y = oracle.layer_norm(X, np.ones(96), np.zeros(96), eps_ln)
    var = X.var(axis=1)
    np.testing.assert_allclose(Y.mean(axis=1), 0.0, atol=1e-13)
    np.testing.assert_allclose((Y ** 2).mean(axis=1), var / (var + eps_ln), rtol=1e-12)
    # eps = 0: invariant to a positive scale and a shift of each row.
    a, c = RNG.uniform(0.5, 4.0, (37, 1)), RNG.standard_normal((37, 1))
    np.testing.assert_allclose(oracle.layer_norm(a * X + c, np.ones(96), np.zeros(96), 0.0),
                               oracle.layer_norm(X, np.ones(96), np.zeros(96), 0.0), atol=1e-12)
    g, b = RNG.standard_normal(96), RNG.standard_normal(96)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(X), (96,), torch.from_numpy(g), torch.from_numpy(b),
                                         eps_ln).numpy()
    np.testing.assert_allclose(oracle.layer_norm(X, g, b, eps_ln), ref, rtol=1e-12, atol=1e-12)


def test_causal_attention_matches_torch_sdpa():
    torch = pytest.importorskip("torch")
    S, L, heads, dh = 3, 20, 4, 16
    Q, K, V = (RNG.standard_normal((S * L, heads * dh)) for _ in range(3))
    got = oracle.causal_attention(Q, K, V, heads, L)
    to4 = lambda A: torch.from_numpy(A).reshape(S, L, heads, dh).permute(0, 2, 1, 3)
    ref = torch.nn.functional.scaled_dot_product_attention(to4(Q), to4(K), to4(V), is_causal=True)
    ref = ref.permute(0, 2, 1, 3).reshape(S * L, heads * dh).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_causal_attention_closed_forms():
    S, L, heads, dh = 2, 12, 2, 16
    Q, K, V = (RNG.standard_normal((S * L, heads * dh)) for _ in range(3))
    O = oracle.causal_attention(Q, K, V, heads, L)
    # The first token of each sequence sees only itself.
    for s0 in range(0, S * L, L):
        np.testing.assert_allclose(O[s0], V[s0], rtol=0, atol=1e-15)
    # Q = 0: uniform weights over the visible keys, i.e. prefix means of V per sequence.
    O0 = oracle.causal_attention(np.zeros_like(Q), K, V, heads, L)
    for s0 in range(0, S * L, L):
        pref = np.cumsum(V[s0:s0 + L], axis=0) / np.arange(1, L + 1)[:, None]
        np.testing.assert_allclose(O0[s0:s0 + L], pref, rtol=1e-13, atol=1e-13)
    # One-hot keys k_t = e_t and q_t = lam e_t: logit a = lam / sqrt(dh) on the diagonal, 0 off it,
    # so o_t = (e^a v_t + sum_{t' < t} v_t') / (e^a + t).
    lam = 3.0
    Kh = np.zeros((L, dh)); Kh[np.arange(L), np.arange(L)] = 1.0
    Vh = RNG.standard_normal((L, dh))
    Oh = oracle.causal_attention(lam * Kh, Kh, Vh, 1, L)
    ea = math.exp(lam / math.sqrt(dh))
    for t in range(L):
        np.testing.assert_allclose(Oh[t], (ea * Vh[t] + Vh[:t].sum(axis=0)) / (ea + t), rtol=1e-13, atol=1e-14)
    # Sequences do not see each other.
    V2 = V.copy(); V2[L:] += 1.0
    np.testing.assert_array_equal(oracle.causal_attention(Q, K, V2, heads, L)[:L], O[:L])


def _decoder_params(seed, d, ffn, r, q, zero=False):
    shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "fc1": (ffn, d), "fc2": (d, ffn)}
    layer = {}
    for i, (nm, (m, n)) in enumerate(shapes.items()):
        W = np.zeros((m, n)) if zero else zd.draw(seed, "W0", (i, m, n), (m, n), 0.05)
        U, _ = np.linalg.qr(zd.draw(seed, "OMEGA_U", (i, m), (m, r)))
        V, _ = np.linalg.qr(zd.draw(seed, "OMEGA_V", (i, n), (n, r)))
        layer[nm] = dict(W=W, U=U, V=V, Z=zd.z_draws(seed, 0, i, q, r).astype(np.float64))
    layer["ln1_g"], layer["ln1_b"] = 1.0 + 0.1 * RNG.standard_normal(d), 0.1 * RNG.standard_normal(d)
    layer["ln2_g"], layer["ln2_b"] = 1.0 + 0.1 * RNG.standard_normal(d), 0.1 * RNG.standard_normal(d)
    return layer


def test_decoder_layer_zero_weights_is_identity():
    d, ffn, r, q = 32, 64, 4, 2
    layer = _decoder_params(1, d, ffn, r, q, zero=True)
    H = RNG.standard_normal((24, d))
    np.testing.assert_array_equal(oracle.decoder_layer(H, layer, 1.0, 0.0, 0, 4, 8), H)


def test_decoder_layer_single_token_sequences():
    """seq_len = 1: attention returns V, so H2 = H + (LN1(H) Wv'^T) Wo'^T, written out with the
    perturbed weights formed directly from Eq. 4."""
    d, ffn, r, q = 32, 64, 4, 2
    layer = _decoder_params(2, d, ffn, r, q)
    H = RNG.standard_normal((10, d))
    s, eps, j = -1.0, 0.3, 1
    Wp = {nm: layer[nm]["W"] + s * eps * layer[nm]["U"] @ layer[nm]["Z"][j] @ layer[nm]["V"].T
          for nm in oracle.DECODER_MATS}
    mu = H.mean(1, keepdims=True); sd = np.sqrt(H.var(1, keepdims=True) + 1e-5)
    A = (H - mu) / sd * layer["ln1_g"] + layer["ln1_b"]
    H2 = H + (A @ Wp["v"].T) @ Wp["o"].T
    mu2 = H2.mean(1, keepdims=True); sd2 = np.sqrt(H2.var(1, keepdims=True) + 1e-5)
    A2 = (H2 - mu2) / sd2 * layer["ln2_g"] + layer["ln2_b"]
    H3 = H2 + np.maximum(A2 @ Wp["fc1"].T, 0.0) @ Wp["fc2"].T
    np.testing.assert_allclose(oracle.decoder_layer(H, layer, s, eps, j, 4, 1), H3, rtol=1e-12, atol=1e-12)


def test_decoder_layer_matches_torch_modules():
    """The layer against torch's own layer_norm, scaled_dot_product_attention and relu in float64,
    with the perturbed weights formed from Eq. 4."""
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    d, ffn, r, q, heads, L, S = 64, 128, 4, 3, 4, 10, 3
    layer = _decoder_params(3, d, ffn, r, q)
    H = RNG.standard_normal((S * L, d))
    s, eps, j = 1.0, 0.05, 2
    Wp = {nm: torch.from_numpy(layer[nm]["W"] + s * eps * layer[nm]["U"] @ layer[nm]["Z"][j] @ layer[nm]["V"].T)
          for nm in oracle.DECODER_MATS}
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    Ht = t(H)
    A = F.layer_norm(Ht, (d,), t(layer["ln1_g"]), t(layer["ln1_b"]), 1e-5)
    heads4 = lambda X: X.reshape(S, L, heads, d // heads).permute(0, 2, 1, 3)
    C = F.scaled_dot_product_attention(heads4(F.linear(A, Wp["q"])), heads4(F.linear(A, Wp["k"])),
                                       heads4(F.linear(A, Wp["v"])), is_causal=True)
    C = C.permute(0, 2, 1, 3).reshape(S * L, d)
    H2 = Ht + F.linear(C, Wp["o"])
    A2 = F.layer_norm(H2, (d,), t(layer["ln2_g"]), t(layer["ln2_b"]), 1e-5)
    H3 = H2 + F.linear(F.relu(F.linear(A2, Wp["fc1"])), Wp["fc2"])
    np.testing.assert_allclose(oracle.decoder_layer(H, layer, s, eps, j, heads, L), H3.numpy(),
                               rtol=1e-11, atol=1e-11)


# ---------------------------------------------------------------------------
# The LLaMA-family layer (RMS normalisation, rotary positions, SwiGLU MLP)
# ---------------------------------------------------------------------------
def test_rms_norm_hand_case_and_torch():
    torch = pytest.importorskip("torch")
    # (3, 4): mean square 12.5, so the row divides by sqrt(12.5).
    np.testing.assert_allclose(oracle.rms_norm(np.array([[3.0, 4.0]]), np.ones(2), 0.0)[0],
                               [0.848528137423857, 1.131370849898476], rtol=0, atol=1e-15)
    X = RNG.standard_normal((29, 80)) * 2.0 + 0.5
    g = 1.0 + 0.1 * RNG.standard_normal(80)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(X), (80,), torch.from_numpy(g), 1e-6).numpy()
    np.testing.assert_allclose(oracle.rms_norm(X, g, 1e-6), ref, rtol=1e-13, atol=1e-13)
    # eps = 0: invariant to a positive scale of each row (but not to a shift).
    a = RNG.uniform(0.5, 4.0, (29, 1))
    np.testing.assert_allclose(oracle.rms_norm(a * X, g, 0.0), oracle.rms_norm(X, g, 0.0), rtol=1e-13, atol=1e-13)
    assert np.abs(oracle.rms_norm(X + 1.0, g, 0.0) - oracle.rms_norm(X, g, 0.0)).max() > 1e-2


def test_rope_hand_cases_and_properties():
    # One head of dh = 4: dimension 0 pairs with 2 (angle p * 1), dimension 1 with 3 (angle p * 0.01).
    X = np.array([[1.0, 0.0, 0.0, 0.0], [1.0, 0.0, 0.0, 0.0], [0.0, 1.0, 0.0, 0.0], [0.0, 0.0, 2.0, 0.0]])
    Y = oracle.rope(X, 4, 1)  # positions 0, 1, 2, 3
    np.testing.assert_allclose(Y[0], [1.0, 0.0, 0.0, 0.0], atol=1e-16)
    np.testing.assert_allclose(Y[1], [math.cos(1.0), 0.0, math.sin(1.0), 0.0], atol=1e-16)
    np.testing.assert_allclose(Y[2], [0.0, math.cos(0.02), 0.0, math.sin(0.02)], atol=1e-16)
    np.testing.assert_allclose(Y[3], [-2.0 * math.sin(3.0), 0.0, 2.0 * math.cos(3.0), 0.0], atol=1e-15)
    L, heads, dh = 16, 3, 32
    Q, K = RNG.standard_normal((L, heads * dh)), RNG.standard_normal((L, heads * dh))
    Rq, Rk = oracle.rope(Q, L, heads), oracle.rope(K, L, heads)
    # Rotations: every (i, i + dh/2) pair keeps its length; position 0 is untouched.
    for h in range(heads):
        a, b = slice(h * dh, h * dh + dh // 2), slice(h * dh + dh // 2, (h + 1) * dh)
        np.testing.assert_allclose(Rq[:, a] ** 2 + Rq[:, b] ** 2, Q[:, a] ** 2 + Q[:, b] ** 2, rtol=1e-13)
    np.testing.assert_array_equal(Rq[0], Q[0])
    # Scores depend on positions only through their difference: q at p, k at s.
    def score(p, s, h=1):
        q = np.zeros((L, heads * dh)); k = np.zeros((L, heads * dh))
        q[p], k[s] = Q[3], K[5]
        qr, kr = oracle.rope(q, L, heads)[p], oracle.rope(k, L, heads)[s]
        c = slice(h * dh, (h + 1) * dh)
        return float(qr[c] @ kr[c])
    np.testing.assert_allclose(score(9, 4), score(12, 7), rtol=1e-12)
    assert abs(score(9, 4) - score(9, 6)) > 1e-3
    # Positions restart with every sequence of the block.
    np.testing.assert_array_equal(oracle.rope(np.vstack([Q, Q]), L, heads)[L:], Rq)


def test_rope_matches_transformers():
    torch = pytest.importorskip("torch")
    ml = pytest.importorskip("transformers.models.llama.modeling_llama")
    L, heads, dh, base = 12, 2, 16, 10000.0
    Q, K = RNG.standard_normal((L, heads * dh)), RNG.standard_normal((L, heads * dh))
    inv = 1.0 / base ** (torch.arange(0, dh, 2, dtype=torch.float64) / dh)
    ang = torch.arange(L, dtype=torch.float64)[:, None] * inv[None, :]
    emb = torch.cat([ang, ang], dim=-1)
    to4 = lambda A: torch.from_numpy(A).reshape(1, L, heads, dh).permute(0, 2, 1, 3)
    qr, kr = ml.apply_rotary_pos_emb(to4(Q), to4(K), emb.cos()[None], emb.sin()[None])
    back = lambda A: A.permute(0, 2, 1, 3).reshape(L, heads * dh).numpy()
    np.testing.assert_allclose(oracle.rope(Q, L, heads), back(qr), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(oracle.rope(K, L, heads), back(kr), rtol=1e-13, atol=1e-13)


def test_silu_closed_forms_and_torch():
    torch = pytest.importorskip("torch")
    x = RNG.standard_normal(200) * 4.0
    np.testing.assert_allclose(oracle.silu(x) - oracle.silu(-x), x, rtol=1e-14, atol=1e-14)
    assert oracle.silu(0.0) == 0.0
    np.testing.assert_allclose(oracle.silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(), rtol=1e-14)


def _llama_params(seed, d, ffn, r, q, zero=False):
    shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d), "down": (d, ffn)}
    layer = {}
    for i, (nm, (m, n)) in enumerate(shapes.items()):
        W = np.zeros((m, n)) if zero else zd.draw(seed, "W0", (i, m, n), (m, n), 0.05)
        U, _ = np.linalg.qr(zd.draw(seed, "OMEGA_U", (i, m), (m, r)))
        V, _ = np.linalg.qr(zd.draw(seed, "OMEGA_V", (i, n), (n, r)))
        layer[nm] = dict(W=W, U=U, V=V, Z=zd.z_draws(seed, 0, i, q, r).astype(np.float64))
    layer["rms1_g"], layer["rms2_g"] = 1.0 + 0.1 * RNG.standard_normal(d), 1.0 + 0.1 * RNG.standard_normal(d)
    return layer


def test_llama_layer_zero_weights_and_causality():
    d, ffn, r, q, heads, L = 32, 64, 4, 2, 4, 8
    zero = _llama_params(4, d, ffn, r, q, zero=True)
    H = RNG.standard_normal((3 * L, d))
    np.testing.assert_array_equal(oracle.llama_layer(H, zero, 1.0, 0.0, 0, heads, L), H)
    layer = _llama_params(5, d, ffn, r, q)
    out = oracle.llama_layer(H, layer, -1.0, 0.2, 1, heads, L)
    # Changing the last tokens of the second sequence leaves every earlier row as it was.
    H2 = H.copy(); H2[L + 5:2 * L] += RNG.standard_normal((3, d))
    out2 = oracle.llama_layer(H2, layer, -1.0, 0.2, 1, heads, L)
    np.testing.assert_array_equal(out2[:L + 5], out[:L + 5])
    np.testing.assert_array_equal(out2[2 * L:], out[2 * L:])
    assert np.abs(out2[L + 5:2 * L] - out[L + 5:2 * L]).max() > 1e-3


def test_llama_layer_matches_transformers():
    """The layer against transformers' LlamaDecoderLayer (its RMS norm and rotary tables are
    float32 inside, hence the 2e-6 bar), with the perturbed weights formed from Eq. 4."""
    torch = pytest.importorskip("torch")
    transformers = pytest.importorskip("transformers")
    ml = pytest.importorskip("transformers.models.llama.modeling_llama")
    d, ffn, r, q, heads, L, S = 64, 128, 4, 3, 4, 10, 3
    layer = _llama_params(6, d, ffn, r, q)
    H = RNG.standard_normal((S * L, d))
    s, eps, j = 1.0, 0.05, 2
    Wp = {nm: layer[nm]["W"] + s * eps * layer[nm]["U"] @ layer[nm]["Z"][j] @ layer[nm]["V"].T
          for nm in oracle.LLAMA_MATS}
    cfg = transformers.LlamaConfig(hidden_size=d, intermediate_size=ffn, num_attention_heads=heads,
                                   num_key_value_heads=heads, rms_norm_eps=1e-6, attention_bias=False,
                                   mlp_bias=False, hidden_act="silu", max_position_embeddings=4 * L)
    cfg._attn_implementation = "sdpa"
    mod = ml.LlamaDecoderLayer(cfg, 0).double()
    rot = ml.LlamaRotaryEmbedding(cfg).double()
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    with torch.no_grad():
        att, mlp = mod.self_attn, mod.mlp
        for lin, nm in ((att.q_proj, "q"), (att.k_proj, "k"), (att.v_proj, "v"), (att.o_proj, "o"),
                        (mlp.gate_proj, "gate"), (mlp.up_proj, "up"), (mlp.down_proj, "down")):
            lin.weight.copy_(t(Wp[nm]))
        mod.input_layernorm.weight.copy_(t(layer["rms1_g"]))
        mod.post_attention_layernorm.weight.copy_(t(layer["rms2_g"]))
        x = t(H).reshape(S, L, d)
        pos = torch.arange(L).unsqueeze(0).expand(S, L)
        out = mod(x, attention_mask=None, position_ids=pos, position_embeddings=rot(x, pos))
        out = out[0] if isinstance(out, tuple) else out
    ref = out.reshape(S * L, d).numpy()
    got = oracle.llama_layer(H, layer, s, eps, j, heads, L)
    np.testing.assert_allclose(got, ref, rtol=2e-6, atol=2e-6 * np.abs(ref).max())


def test_grouped_kv_attention():
    """Grouped key/value heads: kv_heads = heads is the plain multi-head attention bit for bit;
    in general the result equals multi-head attention on K and V with each key/value head
    repeated for its group of query heads, and torch's grouped scaled-dot-product attention."""
    torch = pytest.importorskip("torch")
    T, L, heads, kv, dh = 24, 12, 6, 2, 8
    Q = RNG.standard_normal((T, heads * dh))
    K, V = RNG.standard_normal((T, kv * dh)), RNG.standard_normal((T, kv * dh))
    Kf, Vf = RNG.standard_normal((T, heads * dh)), RNG.standard_normal((T, heads * dh))
    np.testing.assert_array_equal(oracle.causal_attention(Q, Kf, Vf, heads, L, heads),
                                  oracle.causal_attention(Q, Kf, Vf, heads, L))
    rep = lambda X: np.repeat(X.reshape(T, kv, dh), heads // kv, axis=1).reshape(T, heads * dh)
    got = oracle.causal_attention(Q, K, V, heads, L, kv)
    np.testing.assert_array_equal(got, oracle.causal_attention(Q, rep(K), rep(V), heads, L))
    F = torch.nn.functional
    sh = lambda X, h: torch.from_numpy(X).reshape(T // L, L, h, dh).transpose(1, 2)
    ref = F.scaled_dot_product_attention(sh(Q, heads), sh(K, kv), sh(V, kv), is_causal=True, enable_gqa=True)
    ref = ref.transpose(1, 2).reshape(T, heads * dh).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def _lora_layer_params(seed, d, dkv, ffn, rl, r, q):
    shapes = {"q": (d, d), "k": (dkv, d), "v": (dkv, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d),
              "down": (d, ffn)}
    layer = {}
    for i, (nm, (m, n)) in enumerate(shapes.items()):
        layer[nm] = dict(W=zd.draw(seed, "W0", (i, m, n), (m, n), 0.05))
        if nm in ("q", "v"):
            orth = lambda rows, k: np.linalg.qr(zd.draw(seed, "OMEGA_U", (i, rows, k), (rows, r)))[0]
            layer[nm].update(A=zd.draw(seed, "LORA_A", (i,), (rl, n), 0.05), B=zd.draw(seed, "LORA_B", (i,), (m, rl), 0.05),
                             UA=orth(rl, 0), VA=orth(n, 1), UB=orth(m, 2), VB=orth(rl, 3),
                             ZA=zd.z_draws(seed, 0, 2 * i, q, r).astype(np.float64),
                             ZB=zd.z_draws(seed, 0, 2 * i + 1, q, r).astype(np.float64))
    layer["rms1_g"], layer["rms2_g"] = 1.0 + 0.1 * RNG.standard_normal(d), 1.0 + 0.1 * RNG.standard_normal(d)
    return layer


def test_llama_lora_layer_matches_transformers_qwen2():
    """The LoRA-scheme layer against transformers' Qwen2DecoderLayer (grouped key/value heads,
    rotary base 1e6; its q/k/v biases set to zero, the reading of no biases), with q and v
    given the effective weights W + scale B'A' of Eq. 4 on the adapter factors."""
    torch = pytest.importorskip("torch")
    transformers = pytest.importorskip("transformers")
    mq = pytest.importorskip("transformers.models.qwen2.modeling_qwen2")
    d, heads, kv, ffn, rl, r, q, L, S = 64, 8, 2, 96, 4, 2, 3, 10, 2
    dkv = kv * d // heads
    layer = _lora_layer_params(8, d, dkv, ffn, rl, r, q)
    H = RNG.standard_normal((S * L, d))
    s, eps, j, scale = -1.0, 0.1, 1, 2.0
    Weff = {nm: layer[nm]["W"] for nm in oracle.LORA_LAYER_MATS}
    for nm in ("q", "v"):
        m = layer[nm]
        Ap, Bp = oracle.lora_perturbed_factors(m["A"], m["UA"], m["VA"], m["ZA"][j], m["B"], m["UB"], m["VB"],
                                               m["ZB"][j], s, eps)
        Weff[nm] = m["W"] + scale * Bp @ Ap
    cfg = transformers.Qwen2Config(hidden_size=d, intermediate_size=ffn, num_attention_heads=heads,
                                   num_key_value_heads=kv, rms_norm_eps=1e-6, rope_theta=1e6,
                                   hidden_act="silu", max_position_embeddings=4 * L)
    cfg._attn_implementation = "sdpa"
    mod = mq.Qwen2DecoderLayer(cfg, 0).double()
    rot = mq.Qwen2RotaryEmbedding(cfg).double()
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    with torch.no_grad():
        att, mlp = mod.self_attn, mod.mlp
        for lin, nm in ((att.q_proj, "q"), (att.k_proj, "k"), (att.v_proj, "v"), (att.o_proj, "o"),
                        (mlp.gate_proj, "gate"), (mlp.up_proj, "up"), (mlp.down_proj, "down")):
            lin.weight.copy_(t(Weff[nm]))
            if lin.bias is not None:
                lin.bias.zero_()
        mod.input_layernorm.weight.copy_(t(layer["rms1_g"]))
        mod.post_attention_layernorm.weight.copy_(t(layer["rms2_g"]))
        x = t(H).reshape(S, L, d)
        pos = torch.arange(L).unsqueeze(0).expand(S, L)
        out = mod(x, attention_mask=None, position_ids=pos, position_embeddings=rot(x, pos))
        out = out[0] if isinstance(out, tuple) else out
    ref = out.reshape(S * L, d).numpy()
    got = oracle.llama_lora_layer(H, layer, s, eps, j, heads, kv, L, scale)
    np.testing.assert_allclose(got, ref, rtol=2e-6, atol=2e-6 * np.abs(ref).max())
    # The frozen base alone: eps = 0 and B = 0 leave q and v at their base weights.
    zeroB = {nm: dict(layer[nm]) for nm in oracle.LORA_LAYER_MATS}
    zeroB.update(rms1_g=layer["rms1_g"], rms2_g=layer["rms2_g"])
    for nm in ("q", "v"):
        zeroB[nm]["B"] = np.zeros_like(layer[nm]["B"])
    base = oracle.llama_lora_layer(H, zeroB, s, 0.0, j, heads, kv, L, scale)
    assert np.abs(base - got).max() > 1e-4   # the adapters and their perturbation do act
