"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formula: each checks it against an
independent route (a library routine, the explicit mn x mn Kronecker form,
a closed form, a brute-force optimisation, or an invariance of the method),
chosen so that a dropped term, a wrong scale, a transposed operand or a
swapped side fails at least one of them.
"""
import numpy as np
import pytest
import scipy.linalg as sla
import scipy.optimize as sopt
from scipy.stats import multivariate_normal

import oracle
import synth

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# ----------------------------------------------------------------- helpers

def rand_spd(dim, rng, cond=10.0):
    Q = synth.haar_orthogonal(dim, rng)
    lam = np.geomspace(1.0, 1.0 / cond, dim)
    return (Q * lam) @ Q.T


def matrix_normal(N, A, B, rng):
    """Samples with Cov(vec G) = A (x) B (column-major vec)."""
    m, n = B.shape[0], A.shape[0]
    SA = np.linalg.cholesky(A)
    SB = np.linalg.cholesky(B)
    Z = rng.standard_normal((N, m, n))
    return SB[None] @ Z @ SA.T[None]


def vec_cm(G):
    """Column-major vec of each sample: (N, m n)."""
    return np.stack([g.reshape(-1, order="F") for g in G])


def explicit_H(G):
    V = vec_cm(G)
    return V.T @ V / G.shape[0]


def explicit_loglik(G, A, B):
    """Gaussian log-likelihood with the explicit mn x mn covariance A (x) B."""
    K = np.kron(A, B)
    return float(np.sum(multivariate_normal(mean=np.zeros(K.shape[0]), cov=K).logpdf(vec_cm(G))))


def normalised(A, B):
    c = np.trace(A) / A.shape[0]
    return A / c, B * c


# -------------------------------------------------- p1: textbook reduction

def test_first_half_step_is_uncentred_second_moment():
    """With A = I the B update is the second moment of the N n columns
    (Table 1 'Marginal'/'Input' factors; Appendix B start from I)."""
    rng = np.random.default_rng(1)
    N, m, n = 7, 5, 9
    G = rng.standard_normal((N, m, n))
    cols = G.transpose(1, 0, 2).reshape(m, N * n)          # every column g of every sample
    mom = np.cov(cols, bias=True) + np.outer(cols.mean(1), cols.mean(1))
    B1 = oracle.half_step_B(G, np.eye(n))
    np.testing.assert_allclose(B1, mom, rtol=1e-13, atol=1e-14)
    rows = G.reshape(N * m, n)                               # every row of every sample
    momA = np.cov(rows.T, bias=True) + np.outer(rows.mean(0), rows.mean(0))
    A1 = oracle.half_step_A(G, np.eye(m))
    np.testing.assert_allclose(A1, momA, rtol=1e-13, atol=1e-14)


def test_damping_adds_mean_diagonal():
    """Appendix B damping: X + kappa * mean(diag X) * I."""
    rng = np.random.default_rng(2)
    G = rng.standard_normal((6, 4, 5))
    r = oracle.flipflop(G, 1, damping=0.1, keep_half_steps=True)
    _, _, B1 = r.half_steps[0]
    cols = G.transpose(1, 0, 2).reshape(4, -1)
    mom = cols @ cols.T / cols.shape[1]
    np.testing.assert_allclose(B1, mom + 0.1 * np.mean(np.diag(mom)) * np.eye(4), rtol=1e-13)


# ------------------------------------------- p2: orthogonal design, exact

@pytest.mark.parametrize("m,n", [(5, 7), (4, 3), (1, 6), (6, 1)])
def test_orthogonal_design_recovers_truth_in_one_iteration(m, n):
    """N = m n samples sqrt(mn) S_B e_k e_l^T S_A^T make the sample H exactly
    A (x) B, so one iteration must return (A, B) up to the trace scale."""
    rng = np.random.default_rng(3 + m + n)
    A = rand_spd(n, rng, 30.0)
    B = rand_spd(m, rng, 20.0)
    SA = np.linalg.cholesky(A)
    SB = np.linalg.cholesky(B)
    G = []
    for k in range(m):
        for l in range(n):
            Z = np.zeros((m, n))
            Z[k, l] = np.sqrt(m * n)
            G.append(SB @ Z @ SA.T)
    G = np.array(G)
    np.testing.assert_allclose(explicit_H(G), np.kron(A, B), atol=1e-12)
    r = oracle.flipflop(G, 1)
    At, Bt = normalised(A, B)
    assert oracle.kron_rel_error(r.A, r.B, At, Bt) < 1e-13
    np.testing.assert_allclose(r.A, At, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(r.B, Bt, rtol=1e-12, atol=1e-13)


# -------------------------------------------------- p3: trace identity

@pytest.mark.parametrize("order", ["B_FIRST", "A_FIRST"])
def test_trace_identity_after_every_half_step(order):
    """(1/mn) tr(H (A(x)B)^-1) = 1 after each maximum-likelihood half step,
    with H and the Kronecker inverse formed explicitly (Section 5)."""
    rng = np.random.default_rng(4)
    N, m, n = 30, 3, 4
    G = matrix_normal(N, rand_spd(n, rng), rand_spd(m, rng), rng)
    H = explicit_H(G)
    r = oracle.flipflop(G, 4, order=order, keep_half_steps=True)
    assert len(r.half_steps) == 8
    for _, A, B in r.half_steps:
        t = np.trace(H @ np.linalg.inv(np.kron(A, B))) / (m * n)
        assert abs(t - 1.0) < 1e-12
        assert abs(oracle.trace_identity(G, A, B) - 1.0) < 1e-12


# ------------------------------------------- p4: monotone log-likelihood

def test_loglik_matches_explicit_gaussian_and_is_monotone():
    rng = np.random.default_rng(5)
    N, m, n = 25, 3, 4
    G = matrix_normal(N, rand_spd(n, rng, 50), rand_spd(m, rng, 50), rng)
    G += 0.3 * rng.standard_normal(G.shape)                  # not exactly Kronecker
    r = oracle.flipflop(G, 6, keep_half_steps=True)
    prev = explicit_loglik(G, np.eye(n), np.eye(m))
    for _, A, B in r.half_steps:
        ll = explicit_loglik(G, A, B)
        assert abs(ll - oracle.loglik(G, A, B)) < 1e-9 * abs(ll)
        assert ll >= prev - 1e-9 * abs(prev)
        prev = ll
    # the normalisation leaves the likelihood unchanged
    A, B = r.half_steps[-1][1], r.half_steps[-1][2]
    assert abs(explicit_loglik(G, 3.0 * A, B / 3.0) - explicit_loglik(G, A, B)) < 1e-9 * abs(prev)


# ----------------------------------------------------- p5: brute force

def test_fixed_point_matches_brute_force_mle():
    """Maximise the explicit mn x mn Gaussian likelihood over Cholesky
    parameters of A and B with BFGS; the flip-flop fixed point must agree."""
    rng = np.random.default_rng(6)
    N, m, n = 40, 2, 3
    G = matrix_normal(N, rand_spd(n, rng, 8), rand_spd(m, rng, 8), rng)
    G += 0.2 * rng.standard_normal(G.shape)
    V = vec_cm(G)
    S = V.T @ V

    il_n = np.tril_indices(n)
    il_m = np.tril_indices(m)

    def unpack(th):
        LA = np.zeros((n, n))
        LA[il_n] = th[:len(il_n[0])]
        LB = np.zeros((m, m))
        LB[il_m] = th[len(il_n[0]):]
        return LA @ LA.T, LB @ LB.T

    def nll(th):
        A, B = unpack(th)
        K = np.kron(A, B)
        sign, logdet = np.linalg.slogdet(K)
        if sign <= 0:
            return 1e30
        return 0.5 * N * logdet + 0.5 * np.trace(np.linalg.solve(K, S))

    th0 = np.concatenate([np.eye(n)[il_n], np.eye(m)[il_m]])
    best = sopt.minimize(nll, th0, method="BFGS", options={"gtol": 1e-10, "maxiter": 10000})
    Ab, Bb = normalised(*unpack(best.x))
    r = oracle.flipflop(G, 300)
    assert oracle.kron_rel_error(r.A, r.B, Ab, Bb) < 1e-5


# ------------------------------------------------- p6: order independence

def test_fixed_point_independent_of_update_order():
    rng = np.random.default_rng(7)
    N, m, n = 50, 6, 8
    G = matrix_normal(N, rand_spd(n, rng, 20), rand_spd(m, rng, 20), rng)
    G += 0.3 * rng.standard_normal(G.shape)
    rb = oracle.flipflop(G, 400, order="B_FIRST")
    ra = oracle.flipflop(G, 400, order="A_FIRST")
    assert oracle.kron_rel_error(rb.A, rb.B, ra.A, ra.B) < 1e-9
    # ... but a few iterations in, the two orders are different iterates
    rb2 = oracle.flipflop(G, 2, order="B_FIRST")
    ra2 = oracle.flipflop(G, 2, order="A_FIRST")
    assert oracle.kron_rel_error(rb2.A, rb2.B, ra2.A, ra2.B) > 1e-6


# ------------------------------------------------------ p7: consistency

def test_recovers_truth_at_rate_n_to_minus_half():
    """Noise-free matrix-normal samples: the error of A (x) B against the
    true factors falls like N^-1/2 (the iteration is the MLE)."""
    w = synth.Workload("consistency", 6, 5, 0, 30, 1.0, 1.0, "normal", 0, 0.0, "f32", 0)
    Ns = [50, 200, 800, 3200]
    errs = []
    for N in Ns:
        e = []
        for s in range(6):
            d = synth.generate(w.scaled(N=N), seed=1000 + s, threads=1)
            r = oracle.flipflop(d.G, 30)
            e.append(oracle.kron_rel_error(r.A, r.B, *normalised(d.A_true, d.B_true)))
        errs.append(np.mean(e))
    slope = np.polyfit(np.log(Ns), np.log(errs), 1)[0]
    assert -0.65 < slope < -0.35, (slope, errs)
    assert errs[-1] < 0.05


# ------------------------------------------------------ p8: equivariance

def test_equivariance_rotations_scale_permutation():
    rng = np.random.default_rng(8)
    N, m, n = 20, 5, 7
    G = matrix_normal(N, rand_spd(n, rng, 10), rand_spd(m, rng, 10), rng)
    G += 0.2 * rng.standard_normal(G.shape)
    base = oracle.flipflop(G, 5)
    U = synth.haar_orthogonal(m, rng)
    V = synth.haar_orthogonal(n, rng)
    rot = oracle.flipflop(U[None] @ G @ V.T[None], 5)
    np.testing.assert_allclose(rot.A, V @ base.A @ V.T, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(rot.B, U @ base.B @ U.T, rtol=1e-9, atol=1e-10)
    sc = oracle.flipflop(3.0 * G, 5)
    np.testing.assert_allclose(sc.A, base.A, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(sc.B, 9.0 * base.B, rtol=1e-11, atol=1e-12)
    perm = oracle.flipflop(G[rng.permutation(N)], 5)
    np.testing.assert_allclose(perm.A, base.A, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(perm.B, base.B, rtol=1e-11, atol=1e-12)


# ------------------------------------------------- p10: degenerate shapes

def test_single_row_and_single_column_layers():
    """m = 1: B is a scalar b; A b is the second moment S of the rows after
    one iteration and stays there.  n = 1 is the mirror image."""
    rng = np.random.default_rng(9)
    N, n = 40, 6
    G = rng.standard_normal((N, 1, n)) @ np.diag(np.linspace(0.5, 2.0, n))
    rows = G[:, 0, :]
    S = rows.T @ rows / N
    for it in (1, 2, 5):
        r = oracle.flipflop(G, it)
        np.testing.assert_allclose(r.A, n * S / np.trace(S), rtol=1e-12)
        np.testing.assert_allclose(r.B, [[np.trace(S) / n]], rtol=1e-12)
    Gt = np.transpose(G, (0, 2, 1))                            # n = 1, m = 6
    r = oracle.flipflop(Gt, 3)
    np.testing.assert_allclose(r.A * r.B, S, rtol=1e-12)
    assert r.A.shape == (1, 1) and abs(r.A[0, 0] - 1.0) < 1e-15


# ---------------------------------------------- failures (Section 2 convention)

def test_rank_deficient_samples_raise_not_spd():
    rng = np.random.default_rng(10)
    G = rng.standard_normal((2, 3, 9))        # N m = 6 < n = 9: A-update singular
    with pytest.raises(oracle.NotSPDError) as ei:
        oracle.flipflop(G, 3)
    assert ei.value.iteration == 2             # A_1 is singular, B_2 needs A_1^-1
    r = oracle.flipflop(G, 3, damping=0.1)     # damping makes it well posed
    assert np.all(np.linalg.eigvalsh(r.A) > 0)
    Gn = rng.standard_normal((4, 3, 3))
    Gn[1, 0, 0] = np.nan
    with pytest.raises(oracle.NotSPDError):
        oracle.flipflop(Gn, 1)


# ---------------------------------------------------- metric and apply pins

def test_kron_rel_error_matches_explicit_kronecker():
    rng = np.random.default_rng(11)
    A, Ar = rand_spd(4, rng), rand_spd(4, rng)
    B, Br = rand_spd(3, rng), rand_spd(3, rng)
    ref = np.linalg.norm(np.kron(A, B) - np.kron(Ar, Br)) / np.linalg.norm(np.kron(Ar, Br))
    assert abs(oracle.kron_rel_error(A, B, Ar, Br) - ref) < 1e-14
    # tiny perturbations: the stable form keeps digits the expanded form loses
    dA = 1e-9 * rng.standard_normal((4, 4))
    e = oracle.kron_rel_error(Ar + dA, Br, Ar, Br)
    assert abs(e - np.linalg.norm(dA) / np.linalg.norm(Ar)) < 1e-6 * e


def test_scale_free_error_matches_explicit_kronecker():
    """The scale-free error against its definition on the explicit products,
    its blindness to scale, and its small-error limit."""
    rng = np.random.default_rng(12)
    A, Ar = rand_spd(4, rng), rand_spd(4, rng)
    B, Br = rand_spd(3, rng), rand_spd(3, rng)
    K, Kr = np.kron(A, B), np.kron(Ar, Br)
    ref = np.linalg.norm(K / np.linalg.norm(K) - Kr / np.linalg.norm(Kr))
    assert abs(oracle.kron_rel_error_scale_free(A, B, Ar, Br) - ref) < 1e-14
    # a common scale, and a scale moved between the factors, are invisible
    assert abs(oracle.kron_rel_error_scale_free(3.0 * A, 0.5 * B, Ar, 7.0 * Br) - ref) < 1e-14
    assert oracle.kron_rel_error_scale_free(2.0 * Ar, Br / 2.0, Ar, Br) < 1e-15
    # while the plain error sees a scale of the whole product
    assert abs(oracle.kron_rel_error(1.01 * Ar, Br, Ar, Br) - 0.01) < 1e-12
    # small direction errors agree with the plain error to first order
    dA = 1e-7 * rng.standard_normal((4, 4))
    dA -= np.sum(dA * Ar) / np.sum(Ar * Ar) * Ar  # orthogonal to Ar: no change of scale
    e1 = oracle.kron_rel_error_scale_free(Ar + dA, Br, Ar, Br)
    e2 = oracle.kron_rel_error(Ar + dA, Br, Ar, Br)
    assert abs(e1 - e2) < 1e-6 * e2


def test_kron_apply_matches_explicit_kronecker():
    rng = np.random.default_rng(12)
    m, n = 3, 5
    A, B = rand_spd(n, rng), rand_spd(m, rng)
    X = rng.standard_normal((2, m, n))
    Y = oracle.kron_apply(A, B, X)
    K = np.kron(A, B)
    for b in range(2):
        np.testing.assert_allclose(Y[b].reshape(-1, order="F"), K @ X[b].reshape(-1, order="F"),
                                   rtol=1e-12)
    Yi = oracle.kron_apply(A, B, X, inverse=True)
    for b in range(2):
        np.testing.assert_allclose(Yi[b].reshape(-1, order="F"),
                                   np.linalg.solve(K, X[b].reshape(-1, order="F")), rtol=1e-10)


# ------------------------------------------------- p9: mismatch factor

def test_mismatch_factor_identities():
    """Section 4: Phi >= 1 with equality iff H is proportional to A (x) B;
    eq. (6) ties log Phi to the KL divergence minimised over a scale; and
    since each half step minimises Phi over one factor, Phi never rises."""
    rng = np.random.default_rng(13)
    m, n = 2, 3
    N = 60                                      # N >= mn: H nonsingular
    G = matrix_normal(N, rand_spd(n, rng, 5), rand_spd(m, rng, 5), rng)
    G += 0.5 * rng.standard_normal(G.shape)
    H = explicit_H(G)
    A, B = rand_spd(n, rng), rand_spd(m, rng)
    assert abs(oracle.mismatch_factor(7.0 * np.kron(A, B), A, B) - 1.0) < 1e-12
    phi = oracle.mismatch_factor(H, A, B)
    assert phi > 1.0
    K = np.kron(A, B)
    d = m * n

    def kl(s):   # KL(N(0,H) || N(0, sK))
        Ks = s * K
        return 0.5 * (np.trace(np.linalg.solve(Ks, H)) - d
                      + np.linalg.slogdet(Ks)[1] - np.linalg.slogdet(H)[1])

    best = sopt.minimize_scalar(lambda t: kl(np.exp(t)), bracket=(-5, 5), tol=1e-12)
    assert abs(np.log(phi) - 2.0 / d * best.fun) < 1e-9
    r = oracle.flipflop(G, 5, keep_half_steps=True)
    prev = oracle.mismatch_factor(H, np.eye(n), np.eye(m))
    for kind, A, B in r.half_steps:
        phi = oracle.mismatch_factor(H, A, B)
        assert phi <= prev * (1 + 1e-12)
        prev = phi
        if kind == "A":    # trace identity: Phi |H|^(1/mn) = |A|^(1/n) |B|^(1/m)
            lhs = np.log(phi) + np.linalg.slogdet(H)[1] / d
            rhs = np.linalg.slogdet(A)[1] / n + np.linalg.slogdet(B)[1] / m
            assert abs(lhs - rhs) < 1e-10


def test_objective_is_mismatch_factor_up_to_the_data_term():
    """Section 4: psi = log Phi(H, A (x) B) + log|H| / (m n), with Phi taken
    as the AM/GM ratio of the generalised eigenvalues of (H, A (x) B) (an
    independent route through the explicit mn x mn matrices), at factors that
    are not a fixed point; invariant under A -> cA, B -> B/c; never rising
    over flip-flop half steps; and after an A half step it equals
    -2 l / (N m n) - (1 + log 2 pi) with l the log-likelihood."""
    rng = np.random.default_rng(17)
    m, n = 2, 3
    N = 40                                      # N >= mn: H nonsingular
    G = matrix_normal(N, rand_spd(n, rng, 4), rand_spd(m, rng, 6), rng)
    G += 0.3 * rng.standard_normal(G.shape)
    H = explicit_H(G)
    d = m * n
    A, B = rand_spd(n, rng, 3), rand_spd(m, rng, 8)
    psi = oracle.objective(G, A, B)
    ref = np.log(oracle.mismatch_factor(H, A, B)) + np.linalg.slogdet(H)[1] / d
    assert abs(psi - ref) < 1e-11
    assert abs(oracle.objective(G, 3.7 * A, B / 3.7) - psi) < 1e-12
    r = oracle.flipflop(G, 4, keep_half_steps=True)
    prev = oracle.objective(G, np.eye(n), np.eye(m))
    for kind, A, B in r.half_steps:
        cur = oracle.objective(G, A, B)
        assert cur <= prev + 1e-12
        prev = cur
        if kind == "A":
            ll = oracle.loglik(G, A, B)
            assert abs(cur - (-2.0 * ll / (N * d) - 1.0 - np.log(2 * np.pi))) < 1e-10
    # rank-deficient H (N < mn): psi is still finite and scale-invariant
    Gs = G[:3]
    assert np.isfinite(oracle.objective(Gs, A, B))


# ------------------------------------------------- rank-one (per-token) form

def test_token_half_steps_equal_dense_half_steps_on_materialised_samples():
    """Section 5's rank-one half steps (weights x^T A^-1 x and g^T B^-1 g)
    against the dense half steps on G_t = g_t x_t^T, at arbitrary factors;
    a whole run (both orders, damping) against the dense oracle; and the
    token log-likelihood and objective against the dense ones."""
    rng = np.random.default_rng(31)
    T, m, n = 400, 5, 7
    x = rng.standard_normal((T, n)) * np.linspace(0.5, 2.0, n)
    g = rng.standard_normal((T, m)) @ rand_spd(m, rng, 4)
    G = oracle.materialise(x, g)
    A, B = rand_spd(n, rng, 6), rand_spd(m, rng, 9)
    assert np.allclose(oracle.half_step_B_tokens(x, g, A), oracle.half_step_B(G, A), rtol=1e-12, atol=0)
    assert np.allclose(oracle.half_step_A_tokens(x, g, B), oracle.half_step_A(G, B), rtol=1e-12, atol=0)
    for order, kappa in (("B_FIRST", 0.0), ("A_FIRST", 0.1)):
        rt = oracle.flipflop_tokens(x, g, 6, order=order, damping=kappa)
        rd = oracle.flipflop(G, 6, order=order, damping=kappa)
        assert oracle.kron_rel_error(rt.A, rt.B, rd.A, rd.B) < 1e-12
    r = oracle.flipflop_tokens(x, g, 4)
    assert abs(oracle.loglik_tokens(x, g, r.A, r.B) - oracle.loglik(G, r.A, r.B)) < 1e-9 * T * m * n
    assert abs(oracle.objective_tokens(x, g, A, B) - oracle.objective(G, A, B)) < 1e-12


def test_token_fixed_point_recovers_independent_kronecker_factors():
    """Inputs and gradients independent (one component): H = E[xx^T] (x)
    E[gg^T] is a Kronecker product, and the fixed point is that product up
    to scale (error shrinking like T^-1/2)."""
    rng = np.random.default_rng(32)
    m, n = 4, 6
    At, Bt = rand_spd(n, rng, 5), rand_spd(m, rng, 5)
    errs = []
    for T in (4000, 64000):
        x = rng.standard_normal((T, n)) @ np.linalg.cholesky(At).T
        g = rng.standard_normal((T, m)) @ np.linalg.cholesky(Bt).T
        r = oracle.flipflop_tokens(x, g, 30)
        errs.append(oracle.kron_rel_error(r.A, r.B, At, Bt))
    assert errs[1] < 0.5 * errs[0] and errs[1] < 0.03


# ------------------------------------------------------------- WaterKron

def test_rev_cholesky_definition_and_inverse():
    """RevCholesky(M) is lower triangular with L^T L = M; its inverse is the
    Cholesky factor of M^-1 (Section 3 background)."""
    rng = np.random.default_rng(41)
    M = rand_spd(7, rng, 50)
    L = oracle.rev_cholesky(M)
    assert np.allclose(np.triu(L, 1), 0) and np.all(np.diag(L) > 0)
    assert np.allclose(L.T @ L, M, atol=1e-12)
    assert np.allclose(np.linalg.inv(L), np.linalg.cholesky(np.linalg.inv(M)), atol=1e-10)
    # the normalised inverse (Algorithm 2's error-spreading matrix) is unit
    # lower triangular and L times it is diagonal with L's own diagonal
    Lt = oracle.normalised_inverse(M)
    assert np.allclose(np.triu(Lt, 1), 0) and np.allclose(np.diag(Lt), 1.0)
    assert np.allclose(L @ Lt, np.diag(np.diag(L)), atol=1e-10)


def test_waterfilling_scales_of_the_babai_figure():
    """The Babai-rounding figure: L = [[2, 0], [1, 3]] gives the optimal input
    scales (3/sqrt 6, 2/sqrt 6) (volume-preserving, alpha_j proportional to
    1/L_jj)."""
    L = np.array([[2.0, 0.0], [1.0, 3.0]])
    alpha, beta = oracle.waterfilling_scales(L.T @ L, np.eye(1), 1.0)
    assert np.allclose(alpha, [3 / np.sqrt(6), 2 / np.sqrt(6)], atol=1e-14)
    assert np.allclose(beta, [1.0])


def test_two_sided_gptq_reductions():
    """Algorithm 2 with B = I is Algorithm 1; Algorithm 2 is Algorithm 1 on
    vec(W)^T with the Kronecker factor A (x) B and scales alpha (x) beta (the
    proof of the achievability corollary); the error lies in the Babai cell:
    |(L^B (V - W) L^A^T)_ij| <= alpha_j beta_i L^A_jj L^B_ii / 2."""
    rng = np.random.default_rng(42)
    m, n = 5, 6
    A, B = rand_spd(n, rng, 20), rand_spd(m, rng, 30)
    W = rng.standard_normal((m, n))
    alpha, beta = oracle.waterfilling_scales(A, B, 0.3)
    Z1, _ = oracle.gptq(W, A, alpha, np.full(m, beta[0]))
    Z2, _ = oracle.two_sided_gptq(W, A, np.eye(m), alpha, np.full(m, beta[0]))
    assert np.array_equal(Z1, Z2)
    Z, V = oracle.two_sided_gptq(W, A, B, alpha, beta)
    wv = W.reshape(1, -1, order="F")
    Zv, _ = oracle.gptq(wv, np.kron(A, B), np.kron(alpha, beta), np.ones(1))
    assert np.array_equal(Zv.reshape(m, n, order="F"), Z)
    LA, LB = oracle.rev_cholesky(A), oracle.rev_cholesky(B)
    Err = LB @ (V - W) @ LA.T
    cell = np.outer(beta * np.diag(LB), alpha * np.diag(LA)) / 2
    assert np.all(np.abs(Err) <= cell * (1 + 1e-9))


def test_high_rate_distortion():
    """Achievability corollary: D_{A,B} -> (gamma^2 / 12) |A|^(1/n) |B|^(1/m)
    as gamma -> 0 (Gaussian W)."""
    rng = np.random.default_rng(43)
    m, n = 24, 20
    A, B = rand_spd(n, rng, 40), rand_spd(m, rng, 60)
    W = rng.standard_normal((m, n))
    gamma = 1e-3
    alpha, beta = oracle.waterfilling_scales(A, B, gamma)
    _, V = oracle.two_sided_gptq(W, A, B, alpha, beta)
    D = oracle.distortion(V, W, A, B)
    pred = gamma ** 2 / 12 * np.exp(np.linalg.slogdet(A)[1] / n + np.linalg.slogdet(B)[1] / m)
    assert abs(D / pred - 1.0) < 0.1


# ------------------------------------------- Table 1 variants (Section 5 and 6)

def _rearranged(H, m, n):
    """R[(j, j'), (i, i')] = H[j m + i, j' m + i'] (column-major vec), so that
    ||H - A (x) B||_F = ||R - vec(A) vec(B)^T||_F (Van Loan and Pitsianis's
    rearrangement: the best Kronecker approximation is R's top singular pair)."""
    return H.reshape(n, m, n, m).transpose(0, 2, 1, 3).reshape(n * n, m * m)


def _second_moment(G):
    N, m, n = G.shape
    V = G.transpose(0, 2, 1).reshape(N, m * n)      # column-major vec: index j m + i
    return V.T @ V / N


def test_frobenius_converges_to_the_best_kronecker_approximation():
    """Section 5: replacing the inverses by the factors gives a power
    iteration minimising ||H - A (x) B||_F.  Its fixed point must be the top
    singular pair of the rearranged H."""
    rng = np.random.default_rng(11)
    m, n, N = 3, 4, 30
    G = rng.standard_normal((N, m, n))
    G += 0.8 * rng.standard_normal((N, m, 1)) * rng.standard_normal((1, 1, n))
    H = _second_moment(G)
    U, S, Vt = np.linalg.svd(_rearranged(H, m, n))
    assert S[0] > 1.5 * S[1]
    As = U[:, 0].reshape(n, n)
    Bs = Vt[0].reshape(m, m)
    As *= n / np.trace(As)
    Bs /= np.trace(Bs)
    res = oracle.frobenius(G, 200)
    np.testing.assert_allclose(res.A, As, rtol=0, atol=1e-9 * np.abs(As).max())
    np.testing.assert_allclose(res.B / np.trace(res.B), Bs, rtol=0, atol=1e-9 * np.abs(Bs).max())
    # and it is the best Kronecker product in Frobenius norm: the FlipFlop
    # factors, optimally scaled, are no closer to H
    def resid(A, B):
        K = np.kron(A, B)
        s = np.sum(H * K) / np.sum(K * K)
        return np.linalg.norm(H - s * K)
    ff = oracle.flipflop(G, 50)
    assert resid(res.A, res.B) <= resid(ff.A, ff.B) + 1e-12


def test_frobenius_and_flipflop_recover_kronecker_factors_on_an_orthogonal_design():
    """G = S_B Z S_A^T over the complete design Z = sqrt(mn) e_k e_l^T has
    H = A0 (x) B0 exactly; one iteration of either estimator returns A0, B0
    (up to the scale exchanged between them)."""
    rng = np.random.default_rng(12)
    m, n = 3, 5
    SA, SB = rng.standard_normal((n, n)), rng.standard_normal((m, m))
    A0, B0 = SA @ SA.T, SB @ SB.T
    G = np.stack([SB @ (np.sqrt(m * n) * np.outer(np.eye(m)[k], np.eye(n)[l])) @ SA.T
                  for k in range(m) for l in range(n)])
    np.testing.assert_allclose(_second_moment(G), np.kron(A0, B0), atol=1e-10)
    for res in (oracle.frobenius(G, 1), oracle.flipflop(G, 1)):
        np.testing.assert_allclose(res.A, A0 * n / np.trace(A0), rtol=1e-10, atol=1e-10)
        np.testing.assert_allclose(res.B / np.trace(res.B), B0 / np.trace(B0), rtol=1e-10,
                                   atol=1e-10)


def test_marginal_equals_flipflop_and_frobenius_for_independent_tokens():
    """Tokens made of every pair (x, g) of two sets have H = E[x x^T] (x) E[g g^T]
    exactly: Marginal (Table 1) must equal the answer of both iterations."""
    rng = np.random.default_rng(13)
    m, n, p, q = 4, 6, 9, 7
    X = rng.standard_normal((p, n)) * np.linspace(0.5, 2.0, n)
    Gm = rng.standard_normal((q, m))
    x = np.repeat(X, q, axis=0)
    g = np.tile(Gm, (p, 1))
    A, B = oracle.marginal_tokens(x, g)
    np.testing.assert_allclose(np.trace(A), n)
    for res in (oracle.flipflop_tokens(x, g, 1), oracle.flipflop_tokens(x, g, 3),
                oracle.frobenius_tokens(x, g, 2)):
        np.testing.assert_allclose(res.A, A, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(res.B / np.trace(res.B), B / np.trace(B), rtol=1e-10,
                                   atol=1e-12)
    # FlipFlop keeps the scale of H: its product is the marginal product
    ff = oracle.flipflop_tokens(x, g, 1)
    np.testing.assert_allclose(np.kron(ff.A, ff.B), np.kron(X.T @ X / p, Gm.T @ Gm / q),
                               rtol=1e-10, atol=1e-12)
    # Input: the same A, B = c I
    Ai, Bi = oracle.input_tokens(x, m)
    np.testing.assert_allclose(Ai, A, rtol=1e-12)
    np.testing.assert_allclose(Bi, Bi[0, 0] * np.eye(m))


def test_frobenius_tokens_equal_dense_frobenius_on_materialised_samples():
    rng = np.random.default_rng(14)
    x = rng.standard_normal((40, 5))
    g = rng.standard_normal((40, 3))
    a = oracle.frobenius_tokens(x, g, 3, damping=0.1)
    b = oracle.frobenius(oracle.materialise(x, g), 3, damping=0.1)
    np.testing.assert_allclose(a.A, b.A, rtol=1e-11)
    np.testing.assert_allclose(a.B, b.B, rtol=1e-11)
    c = oracle.frobenius_tokens(x, g, 3, order="A_FIRST")
    d = oracle.frobenius(oracle.materialise(x, g), 3, order="A_FIRST")
    np.testing.assert_allclose(c.A, d.A, rtol=1e-11)


# ------------------------------------------- row oracles of the half steps

def _block_half_steps(G, A, B):
    """Both half steps from the explicit second moment H (column-major vec):
    with H4[j, a, k, b] = E[G_aj G_bk], E[G A^-1 G^T]_ab = sum_jk (A^-1)_jk H4[j,a,k,b]
    and E[G^T B^-1 G]_jk = sum_ab (B^-1)_ab H4[j,a,k,b]."""
    N, m, n = G.shape
    H4 = explicit_H(G).reshape(n, m, n, m)
    Bh = np.einsum("jk,jakb->ab", np.linalg.inv(A), H4) / n
    Ah = np.einsum("ab,jakb->jk", np.linalg.inv(B), H4) / m
    return Ah, Bh


@pytest.mark.parametrize("bf16", [False, True])
def test_half_step_row_oracles_every_row_unscaled(bf16):
    """The row oracles used at full size give every row of the half steps,
    unscaled, with a non-identity factor: against the dense half steps and
    against the explicit Kronecker form; the identity branch against the
    sample second moment."""
    rng = np.random.default_rng(31)
    m, n, N = 7, 5, 9
    A, B = rand_spd(n, rng, 30.0), rand_spd(m, rng, 20.0)
    G = matrix_normal(N, A, B, rng)
    if bf16:
        G = synth.f32_to_bf16_bits(G.astype(np.float32))
    G64 = oracle.as_f64_samples(G)
    A0, B0 = rand_spd(n, rng, 50.0), rand_spd(m, rng, 50.0)
    rb = oracle.half_step_B_rows(G, A0, np.arange(m))
    ra = oracle.half_step_A_rows(G, B0, np.arange(n))
    np.testing.assert_allclose(rb, oracle.half_step_B(G64, A0), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(ra, oracle.half_step_A(G64, B0), rtol=1e-12, atol=1e-13)
    Ah, _ = _block_half_steps(G64, np.eye(n), B0)
    _, Bh = _block_half_steps(G64, A0, np.eye(m))
    np.testing.assert_allclose(rb, Bh, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(ra, Ah, rtol=1e-10, atol=1e-12)
    # a subset of rows in any order, and the identity branch
    sel = np.array([4, 0, 2])
    np.testing.assert_allclose(oracle.half_step_B_rows(G, A0, sel), rb[sel], rtol=1e-13)
    np.testing.assert_allclose(oracle.half_step_A_rows(G, B0, sel), ra[sel], rtol=1e-13)
    X = G64.transpose(0, 2, 1).reshape(N * n, m)              # stacked G_i^T
    np.testing.assert_allclose(oracle.half_step_B_rows(G, None, np.arange(m)), X.T @ X / (N * n),
                               rtol=1e-12)
    Y = G64.reshape(N * m, n)
    np.testing.assert_allclose(oracle.half_step_A_rows(G, None, np.arange(n)), Y.T @ Y / (N * m),
                               rtol=1e-12)


def test_token_row_oracle_every_row_unscaled():
    """Rows of the per-token B half step, unscaled, with a non-identity A and
    a chunk size that splits the tokens: against the token half step and
    against the dense row oracle on the materialised samples g_t x_t^T."""
    rng = np.random.default_rng(32)
    T, m, n = 57, 6, 4
    x, g = rng.standard_normal((T, n)), rng.standard_normal((T, m))
    A0 = rand_spd(n, rng, 40.0)
    rows = np.arange(m)
    r = oracle.half_step_B_tokens_rows(x, g, A0, rows, chunk=10)
    np.testing.assert_allclose(r, oracle.half_step_B_tokens(x, g, A0), rtol=1e-12)
    Gt = g[:, :, None] * x[:, None, :]
    np.testing.assert_allclose(r, oracle.half_step_B_rows(Gt, A0, rows), rtol=1e-12)
    np.testing.assert_allclose(oracle.half_step_B_tokens_rows(x, g, None, rows, chunk=7),
                               oracle.half_step_B_rows(Gt, None, rows), rtol=1e-12)
