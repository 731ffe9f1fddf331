"""Pins of the float64 oracle against what the paper and the mathematics fix.

Each test ties one oracle function to something other than itself: a closed
form (SVD functional calculus, Props. 1-2 of App. D), an invariant (unit row
norms, trace of Gamma, Frobenius norms of T), a textbook routine (Higham's
Newton-Schulz polar iteration), a worked example of the paper (App. A), a
special case where the sketch must be exact (Alg. 2), or the published
known-answer vectors of Philox4x32-10.
"""
import math
import os

import numpy as np
import pytest

from oracle import normpre_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(20240917)


def _rand(m, n, scale=1.0):
    return RNG.standard_normal((m, n)) * scale


# ------------------------------------------------------------------ Philox / Omega
def test_philox_known_answer_vectors():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "philox4x32_10_kat.txt"))
            if l.strip() and not l.startswith("#")]
    for r in rows:
        vals = [int(v, 16) for v in r]
        ctr = np.array([vals[0:4]], dtype=np.uint32)
        out = O.philox4x32_10(ctr, (vals[4], vals[5]))[0]
        assert [int(v) for v in out] == vals[6:10]


def test_omega_is_standard_normal():
    om = O.sketch_omega(1337, 7, 3, 4000, 25).ravel()
    # Kolmogorov-Smirnov distance against the N(0,1) CDF.
    xs = np.sort(om)
    cdf = 0.5 * (1.0 + np.vectorize(math.erf)(xs / math.sqrt(2.0)))
    emp = np.arange(1, xs.size + 1) / xs.size
    ks = np.max(np.abs(emp - cdf))
    assert ks < 1.63 / math.sqrt(xs.size)          # 1% critical value
    assert abs(om.mean()) < 5.0 / math.sqrt(om.size)
    assert abs(om.var() - 1.0) < 0.03


def test_omega_counter_layout():
    # Different (t, matrix id) give independent draws; same key reproduces.
    a = O.sketch_omega(1, 2, 3, 50, 8)
    assert np.array_equal(a, O.sketch_omega(1, 2, 3, 50, 8))
    assert not np.allclose(a, O.sketch_omega(1, 3, 3, 50, 8))
    assert not np.allclose(a, O.sketch_omega(1, 2, 4, 50, 8))
    # Element (i, j) uses linear index e = j*b + i: the first column is the
    # leading block of the flat stream.
    big = O.sketch_omega(1, 2, 3, 50, 8)
    flat = O.sketch_omega(1, 2, 3, 400, 1)[:, 0]
    assert np.allclose(big.T.ravel(), flat)


# ------------------------------------------------------------------ momentum
def test_momentum_matches_geometric_sum():
    mu = 0.95
    gs = [_rand(5, 7) for _ in range(6)]
    m = np.zeros((5, 7))
    for g in gs:
        m = O.momentum_update(m, g, mu)
    expect = sum(mu ** (len(gs) - 1 - s) * g for s, g in enumerate(gs))
    assert np.allclose(m, expect, rtol=0, atol=1e-13)


# ------------------------------------------------------------------ relaxed tangent
def test_relaxed_tangent_decomposition():
    # App. D: x = g_tan + (1 - ||w||^2) g_rad with g_rad the projection onto w.
    m, w = _rand(9, 13), _rand(9, 13, 0.4)
    x = O.relaxed_tangent(m, w)
    for i in range(9):
        wi, mi = w[i], m[i]
        g_rad = (mi @ wi) / (wi @ wi) * wi
        g_tan = mi - g_rad
        assert np.allclose(x[i], g_tan + (1.0 - wi @ wi) * g_rad, atol=1e-12)


def test_relaxed_tangent_unit_rows_is_strict_tangent():
    m, w = _rand(6, 10), _rand(6, 10)
    w /= np.linalg.norm(w, axis=1, keepdims=True)
    x = O.relaxed_tangent(m, w)
    assert np.allclose(np.sum(x * w, axis=1), 0.0, atol=1e-12)


def test_relaxed_tangent_zero_weight_is_identity():
    m = _rand(4, 5)
    assert np.array_equal(O.relaxed_tangent(m, np.zeros((4, 5))), m)


# ------------------------------------------------------------------ normalization
def test_normalization_invariants():
    x = _rand(12, 30)
    x[3] = 0.0
    psi = O.diagonal_gram_normalize(x)
    norms = np.linalg.norm(psi, axis=1)
    assert norms[3] == 0.0
    assert np.allclose(np.delete(norms, 3), 1.0, atol=1e-14)
    gamma = psi @ psi.T
    assert np.allclose(np.delete(np.diag(gamma), 3), 1.0)
    assert math.isclose(np.trace(gamma), 11.0, rel_tol=1e-14)
    # Off-diagonal entries are row cosines (Sec. 2.2).
    cos01 = x[0] @ x[1] / (np.linalg.norm(x[0]) * np.linalg.norm(x[1]))
    assert math.isclose(gamma[0, 1], cos01, rel_tol=1e-12)


def test_scale_dominated_rows_example():
    # Sec. 1: one row of norm 1e4, others 1e-3 with fixed directions.  The
    # leading Gram eigenvector follows the big row; Psi does not see scales.
    dirs = _rand(5, 8)
    dirs /= np.linalg.norm(dirs, axis=1, keepdims=True)
    scales = np.array([1e4, 1e-3, 1e-3, 1e-3, 1e-3])
    x = scales[:, None] * dirs
    _, vecs = np.linalg.eigh(x @ x.T)
    assert abs(vecs[0, -1]) > 1.0 - 1e-12
    assert np.allclose(O.diagonal_gram_normalize(x), dirs, atol=1e-14)


def test_orthogonal_rows_worked_example():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "orthogonal_rows_example.txt"))
            if l.strip() and not l.startswith("#")]
    a = np.array([float(r[0]) for r in rows])
    q, _ = np.linalg.qr(_rand(6, 4))
    x = a[:, None] * q.T                  # 4 orthogonal rows in R^6 with norms a
    ghat = O.trace_matched_gram(x)
    assert np.allclose(np.sort(np.linalg.eigvalsh(ghat)), [float(r[1]) for r in rows])
    psi = O.diagonal_gram_normalize(x)
    assert np.allclose(np.linalg.eigvalsh(psi @ psi.T), [float(r[2]) for r in rows])


# ------------------------------------------------------------------ Newton-Schulz
def _odd_poly(coeffs, s):
    a, b, c = coeffs
    return a * s + b * s ** 3 + c * s ** 5


@pytest.mark.parametrize("shape", [(7, 19), (19, 7), (16, 16), (1, 9), (40, 90)])
def test_newton_schulz_is_odd_functional_calculus(shape):
    # X_{k+1} = a X + (b A + c A^2) X with A = X X^T acts on the singular values
    # through f(s) = a s + b s^3 + c s^5 and leaves the singular vectors alone.
    psi = O.diagonal_gram_normalize(_rand(*shape))
    u, s, vt = np.linalg.svd(psi, full_matrices=False)
    s = s / (np.linalg.norm(psi) + 1e-7)
    for _ in range(5):
        s = _odd_poly(O.MUON_NS_COEFFS, s)
    expect = u @ np.diag(s) @ vt
    got = O.newton_schulz(psi, 5, O.MUON_NS_COEFFS)
    assert np.allclose(got, expect, atol=1e-12)


def test_newton_schulz_transpose_rule():
    psi = _rand(11, 29)
    assert np.allclose(O.newton_schulz(psi.T), O.newton_schulz(psi).T, atol=1e-13)


def test_cubic_newton_schulz_converges_to_polar_factor():
    # Higham's iteration X <- 1.5 X - 0.5 X X^T X converges to msign(X) = U V^T.
    psi = O.diagonal_gram_normalize(_rand(10, 24))
    t = O.newton_schulz(psi, 60, O.CUBIC_NS_COEFFS)
    assert np.allclose(t, O.msign_svd(psi), atol=1e-10)
    # ||T^G||_F^2 = m for full row rank (App. D).
    assert math.isclose(np.linalg.norm(t) ** 2, 10.0, rel_tol=1e-10)


def test_newton_schulz_on_orthonormal_rows_is_proportional():
    q, _ = np.linalg.qr(_rand(20, 6))
    psi = q.T                                   # Gamma = I
    t = O.newton_schulz(psi)
    ratio = t / psi
    assert np.allclose(ratio, ratio.flat[0])


# ------------------------------------------------------------------ NormPre-L
def _svd_clip_topr(psi, r):
    """Props. 1-2: T = U diag(s') V^T, s'_i = 1 for the top-min(r, |A|) s_i > 1."""
    u, s, vt = np.linalg.svd(psi, full_matrices=False)
    s2 = s.copy()
    active = np.flatnonzero(s > 1.0)[:r]
    s2[active] = 1.0
    return u @ np.diag(s2) @ vt


def _correlated_psi(m, n, rank=3, noise=0.3):
    x = _rand(m, rank) @ _rand(rank, n) + noise * _rand(m, n)
    return O.diagonal_gram_normalize(x)


@pytest.mark.parametrize("r", [1, 2, 4, 100])
def test_localized_exact_matches_svd_closed_form(r):
    psi = _correlated_psi(14, 33)
    u_sel, lam_sel = O.localized_exact(psi, r)
    t = O.localized_apply(psi, u_sel, lam_sel)
    assert np.allclose(t, _svd_clip_topr(psi, r), atol=1e-12)


def test_regularized_projection_clips_singular_values():
    # Prop. 1 with r >= |A|: singular values min(s, 1), and T is the nearest
    # matrix with ||T||_op <= 1 (checked against random feasible points).
    psi = _correlated_psi(8, 20)
    u_sel, lam_sel = O.localized_exact(psi, 8)
    t = O.localized_apply(psi, u_sel, lam_sel)
    s_psi = np.linalg.svd(psi, compute_uv=False)
    s_t = np.linalg.svd(t, compute_uv=False)
    assert np.allclose(s_t, np.minimum(s_psi, 1.0), atol=1e-12)
    best = np.linalg.norm(t - psi)
    for _ in range(200):
        cand = t + 0.05 * _rand(*t.shape)
        cand /= max(1.0, np.linalg.norm(cand, 2))
        assert np.linalg.norm(cand - psi) >= best - 1e-12


def test_localized_eigen_and_svd_paths_agree_and_contract():
    psi = _correlated_psi(16, 40)
    u_sel, lam_sel = O.localized_exact(psi, 3)
    t = O.localized_apply(psi, u_sel, lam_sel)
    # ||T^L||^2 = |C| + sum_{i not in C} lambda_i <= m  (App. D)
    lam = np.sort(np.linalg.eigvalsh(psi @ psi.T))[::-1]
    expect = len(lam_sel) + lam[len(lam_sel):].sum()
    assert math.isclose(np.linalg.norm(t) ** 2, expect, rel_tol=1e-12)
    assert np.linalg.norm(t) ** 2 <= 16.0 + 1e-9
    # sigma_i(T) <= sigma_i(Psi): eig(P^L) in (0, 1]
    assert np.all(np.linalg.svd(t, compute_uv=False) <= np.linalg.svd(psi, compute_uv=False) + 1e-12)


def test_sketch_exact_when_rank_fits():
    # rank(Psi) <= l: the sketch spans range(Psi) and equals exact-L.
    m, n, k = 60, 80, 5
    psi = O.diagonal_gram_normalize(_rand(m, k) @ _rand(k, n))
    om = O.sketch_omega(11, 0, 0, n, 12)
    sk = O.interaction_sketch(psi, 4, 8, 1, om)
    resid = np.linalg.norm(psi - sk.q @ (sk.q.T @ psi)) / np.linalg.norm(psi)
    assert resid < 1e-13
    t_sk = O.localized_apply(psi, sk.u_sel, sk.lam_sel)
    u_ex, lam_ex = O.localized_exact(psi, 4)
    assert np.allclose(t_sk, O.localized_apply(psi, u_ex, lam_ex), atol=1e-11)


def test_sketch_exact_when_l_equals_rows():
    psi = _correlated_psi(10, 50)
    om = O.sketch_omega(5, 1, 2, 50, 10)
    sk = O.interaction_sketch(psi, 6, 8, 1, om)      # l = min(10, 14) = 10
    assert sk.ell == 10
    u_ex, lam_ex = O.localized_exact(psi, 6)
    assert np.allclose(O.localized_apply(psi, sk.u_sel, sk.lam_sel),
                       O.localized_apply(psi, u_ex, lam_ex), atol=1e-11)


def test_sketch_ritz_values_interlace_and_norm_closed_form():
    psi = _correlated_psi(120, 200, rank=8, noise=0.5)
    om = O.sketch_omega(3, 4, 5, 200, 20)
    sk = O.interaction_sketch(psi, 12, 8, 1, om)
    lam = np.sort(np.linalg.eigvalsh(psi @ psi.T))[::-1]
    assert np.all(sk.ritz_values <= lam[: sk.ritz_values.size] + 1e-10)
    t = O.localized_apply(psi, sk.u_sel, sk.lam_sel)
    closed = np.linalg.norm(psi) ** 2 - np.sum(sk.lam_sel - 1.0)
    assert math.isclose(np.linalg.norm(t) ** 2, closed, rel_tol=1e-12)


def test_sketch_basis_invariance():
    # Rayleigh-Ritz does not depend on which orthonormal basis of span(Y) is used.
    psi = _correlated_psi(50, 70, rank=6)
    om = O.sketch_omega(9, 9, 9, 70, 14)
    sk = O.interaction_sketch(psi, 6, 8, 1, om)
    rot, _ = np.linalg.qr(_rand(14, 14))
    q2 = sk.q @ rot
    b2 = q2.T @ psi
    ev, z = np.linalg.eigh(b2 @ b2.T)
    order = np.argsort(-ev, kind="stable")[:6]
    lam2, u2 = ev[order], q2 @ z[:, order]
    keep = lam2 > 1.0
    t2 = O.localized_apply(psi, u2[:, keep], lam2[keep])
    assert np.allclose(t2, O.localized_apply(psi, sk.u_sel, sk.lam_sel), atol=1e-11)


def _psi_from_factors(a, b, sig, seed):
    """Psi = U diag(sig) V^T with Haar-like orthonormal U (a x k), V (b x k)."""
    rng = np.random.default_rng(seed)
    k = len(sig)
    u, _ = np.linalg.qr(rng.standard_normal((a, k)))
    v, _ = np.linalg.qr(rng.standard_normal((b, k)))
    return u, np.asarray(sig, float), v, (u * np.asarray(sig, float)) @ v.T


def _projector(basis):
    return basis @ basis.T


@pytest.mark.parametrize("p", [0, 1, 2])
def test_candidate_subspace_is_the_power_iterated_range(p):
    # Alg. 2: range(Y) = range((Psi Psi^T)^p Psi Omega).  With Psi = U S V^T
    # that is range(U S^(2p+1) V^T Omega), formed here from the factors alone.
    # Each p gives a different l-dimensional subspace (rank 30 > l = 8), so a
    # dropped, repeated or skipped power iteration fails the projector match.
    sig = np.linspace(2.0, 0.5, 30)
    u, s, v, psi = _psi_from_factors(40, 60, sig, 100 + p)
    omega = O.sketch_omega(21, 3, 1, 60, 8)
    q = O.candidate_subspace(psi, omega, p)
    assert np.allclose(q.T @ q, np.eye(8), atol=1e-12)
    expect = {}
    for pp in range(4):
        y = u @ (s[:, None] ** (2 * pp + 1) * (v.T @ omega))
        expect[pp], _ = np.linalg.qr(y)
    assert np.linalg.norm(_projector(q) - _projector(expect[p]), 2) < 1e-9
    for pp in range(4):
        if pp != p:
            assert np.linalg.norm(_projector(q) - _projector(expect[pp]), 2) > 1e-2
    # and the whole sketch uses exactly hp.power_iters of them
    sk = O.interaction_sketch(psi, 4, 4, p, omega)
    assert np.linalg.norm(_projector(sk.q) - _projector(expect[p]), 2) < 1e-9


def test_power_iteration_converges_to_the_leading_eigenpairs():
    # Spectral gap after r = 4: sigma = (3, 2.8, 2.6, 2.4 | 0.5 ...).  Subspace
    # iteration contracts the error by (sigma_5 / sigma_4)^2 per pass, so with
    # p = 30 the top-r Ritz values are the top-r eigenvalues of Gamma to
    # rounding; with p = 0 a 6-dimensional random subspace of a 50-dimensional
    # range misses them by a wide margin, and each extra pass gets closer.
    sig = np.concatenate([[3.0, 2.8, 2.6, 2.4], np.linspace(0.5, 0.05, 46)])
    u, s, v, psi = _psi_from_factors(50, 80, sig, 7)
    omega = O.sketch_omega(5, 0, 0, 80, 6)
    lam_true = s[:4] ** 2
    err = []
    for p in range(6):
        sk = O.interaction_sketch(psi, 4, 2, p, omega)
        err.append(np.max(np.abs(sk.ritz_values - lam_true) / lam_true))
    sk30 = O.interaction_sketch(psi, 4, 2, 30, omega)
    assert np.allclose(sk30.ritz_values, lam_true, rtol=1e-10, atol=0)
    # the selected eigenvectors are the leading left singular vectors
    assert np.linalg.norm(_projector(sk30.u_sel) - _projector(u[:, :4]), 2) < 1e-9
    assert err[0] > 0.05
    assert all(err[i + 1] < err[i] for i in range(5)), err


def test_topr_then_threshold_equals_threshold_then_topr():
    psi = _correlated_psi(30, 45, rank=10, noise=0.2)
    om = O.sketch_omega(2, 2, 2, 45, 13)
    sk = O.interaction_sketch(psi, 5, 8, 1, om)
    ev = np.linalg.eigvalsh(sk.gamma_q)
    ev = np.sort(ev)[::-1]
    expect = ev[ev > 1.0][:5]
    assert np.allclose(sk.lam_sel, expect)


# ------------------------------------------------------------------ RMS + update
def test_rms_and_update():
    hp = O.HParams(lr=1e-2)
    w, g, mp = _rand(12, 20, 0.02), _rand(12, 20), _rand(12, 20)
    for variant in ("G", "L"):
        out = O.normpre_step(w, g, mp, 0, hp, variant)
        assert math.isclose(np.linalg.norm(out["update"]), 0.2 * math.sqrt(240), rel_tol=1e-12)
        # lr = 0 leaves W unchanged
        hp0 = O.HParams(lr=0.0)
        assert np.array_equal(O.normpre_step(w, g, mp, 0, hp0, variant)["w_new"], w)


def test_zero_signal_gives_pure_decay():
    hp = O.HParams(lr=0.5, weight_decay=0.1)
    w = _rand(6, 9)
    z = np.zeros((6, 9))
    for variant in ("G", "L"):
        out = O.normpre_step(w, z, z, 1, hp, variant)
        assert np.all(out["update"] == 0.0)
        assert np.allclose(out["w_new"], (1.0 - 0.05) * w)


# ------------------------------------------------------------------ whole step
@pytest.mark.parametrize("variant", ["G", "L"])
def test_transpose_equivariance(variant):
    w, g, mp = _rand(9, 21, 0.1), _rand(9, 21), _rand(9, 21)
    hr = O.HParams(orientation="row", rank=3)
    hc = O.HParams(orientation="col", rank=3)
    a = O.normpre_step(w, g, mp, 4, hr, variant)
    b = O.normpre_step(w.T, g.T, mp.T, 4, hc, variant)
    assert np.allclose(a["update"], b["update"].T, atol=1e-12)


@pytest.mark.parametrize("variant", ["G", "L"])
def test_scale_and_row_permutation(variant):
    hp = O.HParams(orientation="row", rank=4)
    w, g, mp = _rand(15, 26, 0.05), _rand(15, 26), _rand(15, 26)
    base = O.normpre_step(w, g, mp, 2, hp, variant)["update"]
    scaled = O.normpre_step(w, 3.7 * g, 3.7 * mp, 2, hp, variant)["update"]
    assert np.allclose(base, scaled, atol=1e-12)
    perm = RNG.permutation(15)
    permuted = O.normpre_step(w[perm], g[perm], mp[perm], 2, hp, variant)["update"]
    assert np.allclose(base[perm], permuted, atol=1e-11)


def test_both_axes_rank_one_closed_form():
    # W = 0 makes the relaxed tangent the identity (X = M).  For M = a b^T the
    # row pass gives sign(a_i) b / ||b||, and the column pass then scales each
    # column to unit norm: Psi_ij = sign(a_i) sign(b_j) / sqrt(m).
    m, n = 7, 11
    a = RNG.standard_normal(m)
    b = RNG.standard_normal(n)
    w = np.zeros((m, n))
    g = np.outer(a, b)
    hp = O.HParams(orientation="both")
    for t in (0, 1):
        out = O.normpre_step(w, g, np.zeros((m, n)), t, hp, "NORM")
        assert out["k"] == t % 2
        expect = np.outer(np.sign(a), np.sign(b)) / math.sqrt(m)
        assert np.allclose(out["psi"], expect, atol=1e-14)


def test_both_axes_unit_columns_and_preconditioner_side():
    w, g, mp = _rand(9, 14), _rand(9, 14), _rand(9, 14)
    hp = O.HParams(orientation="both", rank=3)
    r0 = O.normpre_step(w, g, mp, 0, hp, "L")
    r1 = O.normpre_step(w, g, mp, 1, hp, "L")
    # the same Psi for both parities, every column of unit norm
    assert np.allclose(r0["psi"], r1["psi"], atol=1e-15)
    assert np.allclose(np.linalg.norm(r0["psi"], axis=0), 1.0)
    # the localized preconditioner acts on rows for t even, on columns for t odd
    assert r0["k"] == 0 and r1["k"] == 1
    assert r0["ell"] == min(9, 3 + 8) and r1["ell"] == min(14, 3 + 8)
    # it differs from row-only normalization (the column pass took effect)
    row = O.normpre_step(w, g, mp, 0, O.HParams(orientation="row", rank=3), "L")
    assert O.relative_fro(row["psi"], r0["psi"]) > 1e-3


def test_source_x_orthogonal_rows_closed_form():
    # App. A's worked example: mutually orthogonal rows with norms a_i have a
    # diagonal trace-matched Gram with eigenvalues d a_i^2 / sum_j a_j^2.  With
    # the interaction source X the exact localized step then scales each
    # selected row of Psi (a unit row) by lambda_i^{-1/2} and leaves the rest.
    d, n = 6, 10
    q, _ = np.linalg.qr(RNG.standard_normal((n, d)))
    norms = np.array([5.0, 0.5, 3.0, 1.0, 0.2, 2.5])
    x = (q.T * norms[:, None])                       # orthogonal rows
    w = np.zeros((d, n))
    lam = d * norms ** 2 / np.sum(norms ** 2)
    hp = O.HParams(rank=2, source="x", lr=1.0, weight_decay=0.0, orientation="row")
    out = O.normpre_step(w, x, np.zeros((d, n)), 0, hp, "L", l_mode="exact")
    top = np.sort(lam[lam > 1.0])[::-1][:2]
    assert np.allclose(out["lam_sel"], top, rtol=1e-12)
    psi = x / norms[:, None]
    expect = psi.copy()
    for v in top:
        i = int(np.argmin(np.abs(lam - v)))
        expect[i] *= v ** -0.5
    assert np.allclose(out["t"], expect, atol=1e-12)


@pytest.mark.parametrize("l_mode", ["exact", "sketch"])
def test_source_x_equal_row_norms_reduces_to_psi(l_mode):
    # Equal active-row norms make G_X = Gamma, so both sources coincide.
    w = np.zeros((12, 20))
    g = _rand(12, 20)
    g = g / np.linalg.norm(g, axis=1, keepdims=True) * 3.0
    zero = np.zeros((12, 20))
    for t in (0,):
        a = O.normpre_step(w, g, zero, t, O.HParams(rank=3, source="x", orientation="row"), "L", l_mode=l_mode)
        b = O.normpre_step(w, g, zero, t, O.HParams(rank=3, source="psi", orientation="row"), "L", l_mode=l_mode)
        assert np.allclose(a["update"], b["update"], atol=1e-10)
    # unequal norms: the sources differ
    g2 = g * np.linspace(0.2, 3.0, 12)[:, None]
    a = O.normpre_step(w, g2, zero, 0, O.HParams(rank=3, source="x", orientation="row"), "L", l_mode=l_mode)
    b = O.normpre_step(w, g2, zero, 0, O.HParams(rank=3, source="psi", orientation="row"), "L", l_mode=l_mode)
    assert O.relative_fro(a["update"], b["update"]) > 1e-3


def test_orientation_alternates_with_t():
    hp = O.HParams()
    w, g, mp = _rand(5, 8), _rand(5, 8), _rand(5, 8)
    assert O.normpre_step(w, g, mp, 0, hp, "G")["k"] == 0
    assert O.normpre_step(w, g, mp, 1, hp, "G")["k"] == 1
    # k = 1 normalises the columns of the W layout
    psi = O.normpre_step(w, g, mp, 1, hp, "G")["psi"]
    assert np.allclose(np.linalg.norm(psi, axis=0), 1.0)


# ------------------------------------------------------------------ reference steps and ablations
def test_strict_tangent_removes_the_radial_component():
    # Exact tangent projection (App. A.4): <x_i, w_i> = 0 for any weight scale,
    # equal to the relaxed form on unit rows (Sec. 3.1), identity on zero rows.
    m, w = _rand(9, 14), _rand(9, 14, 3.0)
    w[4] = 0.0
    x = O.strict_tangent(m, w)
    assert np.max(np.abs(np.sum(x * w, axis=1))) < 1e-12 * np.max(np.abs(m)) * np.max(np.abs(w)) * 14
    np.testing.assert_allclose(x[4], m[4], rtol=0, atol=0)
    wu = w / np.maximum(np.linalg.norm(w, axis=1, keepdims=True), 1e-300)
    wu[4] = 0.0
    np.testing.assert_allclose(O.strict_tangent(m, wu), O.relaxed_tangent(m, wu), rtol=1e-13, atol=1e-13)
    # a plausible slip (dividing by ||w|| instead of ||w||^2) breaks orthogonality
    d = np.sum(m * w, axis=1) / np.linalg.norm(w, axis=1).clip(1e-300)
    bad = m - d[:, None] * w
    assert np.max(np.abs(np.sum(bad * w, axis=1))) > 1e-3


def test_tangent_none_normalizes_the_momentum_rows():
    w, g, mp = _rand(6, 11), _rand(6, 11), _rand(6, 11)
    hp = O.HParams(tangent="none", lr=1.0, weight_decay=0.0)
    r = O.normpre_step(w, g, mp, 0, hp, "NORM")
    m = hp.momentum * mp + g
    np.testing.assert_allclose(r["psi"], m / np.linalg.norm(m, axis=1, keepdims=True), rtol=1e-13, atol=1e-14)


def test_normalize_only_rows_and_rms():
    # T = Psi: every active row of U has the same norm 0.2 sqrt(mn / a) and
    # points along x_i (Sec. 2.2 with P = I, Sec. 3.1 RMS).
    w, g, mp = _rand(12, 7), _rand(12, 7), _rand(12, 7)
    hp = O.HParams(lr=1.0, weight_decay=0.0)
    for t in (0, 1):
        r = O.normpre_step(w, g, mp, t, hp, "NORM")
        u_act = O.orient(r["update"], r["k"])
        a = u_act.shape[0]
        np.testing.assert_allclose(np.linalg.norm(u_act, axis=1), 0.2 * math.sqrt(w.size / a), rtol=1e-12)
        x = O.relaxed_tangent(O.orient(hp.momentum * mp + g, r["k"]), O.orient(w, r["k"]))
        cos = np.sum(u_act * x, axis=1) / (np.linalg.norm(u_act, axis=1) * np.linalg.norm(x, axis=1))
        np.testing.assert_allclose(cos, 1.0, rtol=0, atol=1e-12)


def test_normalize_only_equals_g_on_orthogonal_rows():
    # Orthonormal Psi rows: the Newton-Schulz map scales Psi uniformly, so after
    # the RMS match NormPre-G and the P = I step give the same update.
    q, _ = np.linalg.qr(RNG.standard_normal((20, 6)))
    g = (q.T * RNG.uniform(0.5, 3.0, 6)[:, None])   # 6 x 20, orthogonal rows
    z = np.zeros_like(g)
    hp = O.HParams(lr=1.0, weight_decay=0.0, orientation="row")
    rg = O.normpre_step(z, g, z, 0, hp, "G")
    rn = O.normpre_step(z, g, z, 0, hp, "NORM")
    np.testing.assert_allclose(rg["update"], rn["update"], rtol=1e-10, atol=1e-12)


def test_muon_with_cubic_iteration_is_scaled_polar_factor():
    # Muon (Sec. 2.1): msign of the momentum; with Higham's cubic iterated to
    # convergence U = 0.2 sqrt(max(m, n)) U_M V_M^T and ||U||_F = 0.2 sqrt(mn).
    for shape in [(8, 21), (21, 8)]:
        w, g, mp = _rand(*shape), _rand(*shape), _rand(*shape)
        hp = O.HParams(lr=1.0, weight_decay=0.0, ns_iters=60, ns_coeffs=O.CUBIC_NS_COEFFS)
        r = O.normpre_step(w, g, mp, 0, hp, "MUON")
        m = hp.momentum * mp + g
        np.testing.assert_allclose(r["update"], 0.2 * math.sqrt(max(shape)) * O.msign_svd(m), rtol=0, atol=1e-10)
        assert math.isclose(np.linalg.norm(r["update"]), 0.2 * math.sqrt(w.size), rel_tol=1e-10)


def test_muon_invariances():
    w, g, mp = _rand(10, 16), _rand(10, 16), _rand(10, 16)
    hp = O.HParams(lr=1.0, weight_decay=0.0, ns_eps=0.0)
    r = O.normpre_step(w, g, mp, 0, hp, "MUON")
    # scale of (G, M_prev) drops out (Frobenius pre-scaling, exact with no
    # epsilon); t has no effect
    r2 = O.normpre_step(w, 7.0 * g, 7.0 * mp, 1, hp, "MUON")
    np.testing.assert_allclose(r2["update"], r["update"], rtol=1e-9, atol=1e-12)
    # transposed inputs give the transposed update (odd polynomial in X X^T)
    rt = O.normpre_step(w.T, g.T, mp.T, 0, hp, "MUON")
    np.testing.assert_allclose(rt["update"], r["update"].T, rtol=1e-9, atol=1e-12)
    # and, unlike NormPre, Muon does not equalize row scales: scaling one row
    # of G and M_prev changes the update
    g3, m3 = g.copy(), mp.copy()
    g3[2] *= 10.0
    m3[2] *= 10.0
    r3 = O.normpre_step(w, g3, m3, 0, hp, "MUON")
    assert O.relative_fro(r3["update"], r["update"]) > 1e-2


# ------------------------------------------------- spectral diagnostics (App. A)
def test_interaction_spectrum_worked_example():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "orthogonal_rows_example.txt"))
            if l.strip() and not l.startswith("#")]
    a = np.array([float(r[0]) for r in rows])
    q, _ = np.linalg.qr(_rand(6, 4))
    x = a[:, None] * q.T
    before = O.interaction_spectrum(x, normalized=False)
    after = O.interaction_spectrum(x, normalized=True)
    assert np.allclose(before, sorted((float(r[1]) for r in rows), reverse=True))
    assert np.allclose(after, [float(r[2]) for r in rows])
    assert abs(before.sum() - 4.0) < 1e-12 and abs(after.sum() - 4.0) < 1e-12   # both have trace d
    split = O.energy_split(after, 4, 32)
    assert split["global"] < 1e-24                        # Gamma = I: nothing to transform


@pytest.mark.parametrize("shape,r", [((30, 70), 4), ((50, 20), 3), ((40, 40), 100)])
def test_energy_split_closed_forms(shape, r):
    # Low-rank-plus-noise rows: several singular values of Psi above one,
    # the rest below.
    x = _rand(shape[0], 5) @ _rand(5, shape[1]) + 0.3 * _rand(*shape)
    psi = O.diagonal_gram_normalize(x)
    lam = O.interaction_spectrum(x, normalized=True)
    count = min(shape)
    split = O.energy_split(lam, count, r)
    # Global preconditioning sends every singular value to one: the total is
    # the squared distance of Psi to its polar factor.
    assert math.isclose(split["global"], np.linalg.norm(psi - O.msign_svd(psi)) ** 2, rel_tol=1e-9)
    # Localized preconditioning changes exactly the modes of C: E_top is the
    # squared distance of Psi to the exact NormPre-L output.
    u_sel, lam_sel = O.localized_exact(psi, r)
    t_loc = O.localized_apply(psi, u_sel, lam_sel)
    assert math.isclose(split["top"], np.linalg.norm(psi - t_loc) ** 2, rel_tol=1e-9, abs_tol=1e-18)
    # Brute force over the singular values.
    sv = np.linalg.svd(psi, compute_uv=False)
    assert math.isclose(split["sub"], float(np.sum((sv[(sv > 1e-9) & (sv < 1)] - 1) ** 2)), rel_tol=1e-9)
    assert math.isclose(split["top"] + split["remain"], float(np.sum((sv[sv > 1] - 1) ** 2)), rel_tol=1e-9)


# ------------------------------------------------- descent alignment (App. A)
def test_descent_alignment_closed_forms():
    g = _rand(20, 30)
    q = _rand(20, 30)
    q -= np.sum(q * g) / np.sum(g * g) * g          # orthogonal to g
    cos, mean = O.descent_alignment([g, g, g, g], [3.0 * g, -0.5 * g, q, np.zeros_like(g)])
    assert np.allclose(cos, [1.0, -1.0, 0.0, 0.0], atol=1e-14)
    assert math.isclose(mean, 0.0, abs_tol=1e-14)


def test_descent_alignment_of_normalize_only_step():
    # W = 0 and M_prev = 0: x_i = g_i, Psi = D(G)^-1 G and U = c Psi (c > 0),
    # so <G, U> / (||G|| ||U||) = sum_i ||g_i|| / (sqrt(m) ||G||_F): the
    # Cauchy-Schwarz ratio of the row norms (1 exactly when they are equal).
    rng = np.random.default_rng(3)
    g = rng.standard_normal((12, 40)) * rng.uniform(0.1, 5.0, (12, 1))
    z = np.zeros_like(g)
    out = O.normpre_step(z, g, z, 0, O.HParams(lr=1.0, weight_decay=0.0), "NORM")
    cos, _ = O.descent_alignment([g], [out["update"]])
    rn = np.linalg.norm(g, axis=1)
    assert math.isclose(cos[0], rn.sum() / (math.sqrt(12) * np.linalg.norm(g)), rel_tol=1e-13)
    g_eq = g / rn[:, None]
    out = O.normpre_step(z, g_eq, z, 0, O.HParams(lr=1.0, weight_decay=0.0), "NORM")
    assert math.isclose(O.descent_alignment([g_eq], [out["update"]])[0][0], 1.0, rel_tol=1e-13)
