"""The Gram-space schedule of the Newton-Schulz iteration is exact algebra.

For matrices with L >= 2 s the library runs the five Newton-Schulz iterations
of NormPre-G (Sec. 3.2, the quintic of Muon) on s x s matrices: with
X_k = Q_k X_0, A_k = X_k X_k^T and P_k = a I + b A_k + c A_k^2,

    Q_{k+1} = P_k Q_k,        A_{k+1} = P_k A_k P_k,

and X is formed only at X_3 = Q_3 X_0 (where a fresh Gram A_3 is taken) and
T = X_5 = Q_5 X_3.  These tests carry out that schedule in float64 and check
that it reproduces the oracle's plain iteration to rounding, for wide and tall
matrices and for other polynomial coefficients.  They pin the reformulation,
not the GPU code (whose fp16 results the GPU parity tests compare with the
oracle).
"""
import numpy as np
import pytest

from oracle import normpre_oracle as O

RNG = np.random.default_rng(31)


def gram_space_ns(x, coeffs=O.MUON_NS_COEFFS, restart=3, steps=5):
    """Gram-space schedule on the short side: rows of x are the s short-side
    vectors (x is s x L); returns X_steps (s x L)."""
    a, b, c = coeffs
    base = x / (np.linalg.norm(x) + 1e-7)
    s = base.shape[0]
    eye = np.eye(s)
    A = base @ base.T
    Q = eye
    for k in range(steps):
        if k == restart:
            A = base @ base.T
            Q = eye
        P = a * eye + b * A + c * A @ A
        Q = P @ Q
        if k == restart - 1 or k == steps - 1:
            base = Q @ base
        else:
            A = P @ A @ P
    return base


@pytest.mark.parametrize("shape", [(24, 64), (40, 100), (64, 256), (32, 96)])
def test_gram_space_schedule_matches_plain_iteration_wide(shape):
    psi = RNG.standard_normal(shape)
    psi /= np.linalg.norm(psi, axis=1, keepdims=True)
    ref = O.newton_schulz(psi, 5, O.MUON_NS_COEFFS)
    got = gram_space_ns(psi)
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < 1e-11


@pytest.mark.parametrize("shape", [(100, 40), (256, 64)])
def test_gram_space_schedule_matches_plain_iteration_tall(shape):
    # Tall matrices iterate on the transpose (s = number of columns).
    psi = RNG.standard_normal(shape)
    psi /= np.linalg.norm(psi, axis=1, keepdims=True)
    ref = O.newton_schulz(psi, 5, O.MUON_NS_COEFFS)
    got = gram_space_ns(psi.T).T
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < 1e-11


def test_gram_space_schedule_other_coefficients_and_low_rank():
    # Rank-deficient input (zero singular values stay zero) and the cubic
    # Newton-Schulz coefficients: the identity holds for any odd polynomial.
    u = RNG.standard_normal((30, 5))
    v = RNG.standard_normal((5, 90))
    psi = u @ v
    for coeffs in (O.MUON_NS_COEFFS, O.CUBIC_NS_COEFFS, (2.0, -1.5, 0.5)):
        ref = O.newton_schulz(psi, 5, coeffs)
        got = gram_space_ns(psi, coeffs)
        assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < 1e-11


def test_gram_space_schedule_detects_a_wrong_update():
    # A plausible slip (A_{k+1} = P_k A_k instead of P_k A_k P_k) is caught.
    psi = RNG.standard_normal((24, 64))
    ref = O.newton_schulz(psi, 5, O.MUON_NS_COEFFS)
    a, b, c = O.MUON_NS_COEFFS
    x = psi / (np.linalg.norm(psi) + 1e-7)
    A = x @ x.T
    Q = np.eye(24)
    for _ in range(5):
        P = a * np.eye(24) + b * A + c * A @ A
        Q = P @ Q
        A = P @ A
    got = Q @ x
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) > 1e-3
