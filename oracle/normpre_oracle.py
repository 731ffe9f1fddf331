"""Plain float64 CPU oracle for one NormPre optimizer step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, constants
table or helper with the HIP library; the only thing both sides consume is
the seeded input data handed to them by the callers.

Everything here is written out from the paper "Normalize-Then-Precondition"
(arXiv 2609.36692): the step of Algorithm 1 (the NormPre optimizer, Sec. 3.1)
in its order, and the randomized interaction sketch of Algorithm 2 (App. B)
from what it computes: an orthonormal basis of the power-iterated sketch of
range(Psi), the Rayleigh-Ritz pairs of Gamma = Psi Psi^T on it, and the
selection of the over-amplified modes.  Library routines used as single
steps: ``@`` (matmul), ``np.linalg.qr`` (an orthonormal basis),
``np.linalg.svd`` (the eigenpairs of Gamma_Q = B B^T from the singular pairs
of B) and ``np.linalg.eigh`` (the exact variant of App. B).

Conventions the paper leaves open:
  * Newton-Schulz polynomial: the quintic used by Muon, coefficients
    (3.4445, -4.7750, 2.0315), Frobenius pre-scaling with +1e-7 (Sec. 3.2
    names Muon's iteration without giving its coefficients).
  * Orientation: k = t mod 2 with k = 0 acting on rows of W (Alg. 1).
  * Zero rows: psi_i = x_i / max(||x_i||, eps), eps = 1e-12 (Eq. 2 needs
    non-zero rows; this keeps a zero row at zero).
  * Gaussian test matrix Omega of Alg. 2: Philox4x32-10 counter-based
    generator (Salmon et al., SC'11) + Box-Muller, keyed by (seed, t, matrix
    id); see ``sketch_omega``.  Parity of this convention with the authors'
    code is unpinned: the paper does not name an RNG.
  * Selection: strict lambda > 1 among the top-min(r, l) Ritz values, ties
    broken by lower index (Alg. 2 and App. B).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

MUON_NS_COEFFS = (3.4445, -4.7750, 2.0315)
CUBIC_NS_COEFFS = (1.5, -0.5, 0.0)   # Higham's Newton-Schulz polar iteration
TARGET_RMS = 0.2                     # Sec. 3.1, "Consistent Update RMS"


@dataclass
class HParams:
    """Hyperparameters of Alg. 1 / Alg. 2 (defaults: optimizer table, App. A)."""
    lr: float = 6e-4
    momentum: float = 0.95
    weight_decay: float = 0.1
    target_rms: float = TARGET_RMS
    ns_iters: int = 5
    ns_coeffs: tuple = MUON_NS_COEFFS
    rank: int = 32
    oversample: int = 8
    power_iters: int = 1
    seed: int = 1337
    norm_eps: float = 1e-12
    ns_eps: float = 1e-7
    orientation: str = "alternating"   # "alternating" | "row" | "col" | "both" (App. A.4)
    tangent: str = "relaxed"           # "relaxed" (Sec. 3.1) | "none" | "strict" (App. A.4)
    source: str = "psi"                # NormPre-L interaction source: "psi" | "x" (App. A.4)


# --------------------------------------------------------------------------
# Alg. 1, line "M_t <- mu M_{t-1} + G_t"  (Sec. 3.1)
# --------------------------------------------------------------------------
def momentum_update(m_prev: np.ndarray, g: np.ndarray, mu: float) -> np.ndarray:
    """Heavy-ball momentum M_t = mu * M_{t-1} + G_t (no dampening, no Nesterov)."""
    return mu * np.asarray(m_prev, np.float64) + np.asarray(g, np.float64)


# --------------------------------------------------------------------------
# Alg. 1 orientation: k_t = t mod 2, O_0(A) = A, O_1(A) = A^T  (Sec. 3.1)
# --------------------------------------------------------------------------
def orientation_of(t: int, mode: str = "alternating") -> int:
    """Active side k of step t.  "both" normalizes rows and then columns every
    step (the Row+Column/Step ablation of App. A.4); its preconditioner keeps
    the alternating active side."""
    if mode in ("alternating", "both"):
        return int(t) % 2
    if mode == "row":
        return 0
    if mode == "col":
        return 1
    raise ValueError(f"unknown orientation mode {mode!r}")


def orient(a: np.ndarray, k: int) -> np.ndarray:
    """O_k(A): identity for k = 0, transpose for k = 1."""
    return a if k == 0 else a.T


def orient_inv(a: np.ndarray, k: int) -> np.ndarray:
    """O_k^{-1}: maps an active-orientation matrix back to the W layout."""
    return a if k == 0 else a.T


# --------------------------------------------------------------------------
# Relaxed tangent momentum (Sec. 3.1):  x_i = m_i - <m_i, w_i> w_i
# (w_i is NOT normalised; App. D shows x_i = g_tan + (1 - ||w_i||^2) g_rad)
# --------------------------------------------------------------------------
def relaxed_tangent(m_bar: np.ndarray, w_bar: np.ndarray) -> np.ndarray:
    d = np.sum(m_bar * w_bar, axis=1)
    return m_bar - d[:, None] * w_bar


# --------------------------------------------------------------------------
# Momentum-processing ablations (App. A.4, "Ablations on Marginally
# Normalized Update"): "none" leaves the momentum unchanged; "strict" removes
# the whole radial component, the orthogonal projection onto w_i^perp (the
# relaxed form coincides with it when ||w_i|| = 1, Sec. 3.1).  A zero w_i has
# no radial direction and leaves m_i unchanged.
# --------------------------------------------------------------------------
def strict_tangent(m_bar: np.ndarray, w_bar: np.ndarray) -> np.ndarray:
    d = np.sum(m_bar * w_bar, axis=1)
    ww = np.sum(w_bar * w_bar, axis=1)
    coef = np.divide(d, ww, out=np.zeros_like(d), where=ww > 0)
    return m_bar - coef[:, None] * w_bar


def momentum_processing(m_bar: np.ndarray, w_bar: np.ndarray, mode: str = "relaxed") -> np.ndarray:
    if mode == "relaxed":
        return relaxed_tangent(m_bar, w_bar)
    if mode == "strict":
        return strict_tangent(m_bar, w_bar)
    if mode == "none":
        return m_bar.copy()
    raise ValueError(f"unknown tangent mode {mode!r}")


# --------------------------------------------------------------------------
# Diagonal-Gram normalisation, Eq. (2):  Psi = D(X)^{-1} X,
# D(X) = Diag(||x_1||, ..., ||x_m||)  (Sec. 2.2)
# --------------------------------------------------------------------------
def diagonal_gram_normalize(x: np.ndarray, eps: float = 1e-12) -> np.ndarray:
    norms = np.sqrt(np.sum(x * x, axis=1))
    return x / np.maximum(norms, eps)[:, None]


def interaction_source_x(x: np.ndarray) -> np.ndarray:
    """X_s = sqrt(d / tr(X X^T)) X, so that X_s X_s^T is the trace-matched Gram
    G_X of App. A (d = active rows); zero X gives zero."""
    tot = float(np.sum(x * x))
    return x * math.sqrt(x.shape[0] / tot) if tot > 0 else np.zeros_like(x)


def both_axes_normalize(w: np.ndarray, m: np.ndarray, tangent: str = "relaxed",
                        eps: float = 1e-12) -> np.ndarray:
    """Row+Column/Step ablation (App. A.4, orientation table): the row-active
    momentum processing and Eq. (2) on the rows of W, then Eq. (2) applied to
    the columns of the result.  Reading: the second axis is a plain marginal
    normalization (no second tangent step).  Returns Psi in the W layout."""
    psi_rows = diagonal_gram_normalize(momentum_processing(m, w, tangent), eps)
    return diagonal_gram_normalize(psi_rows.T, eps).T


# --------------------------------------------------------------------------
# NormPre-G: T = msign(Psi) approximated with Newton-Schulz (Sec. 3.2);
# the input is transposed when needed so the Gram matrix is s x s,
# s = min(m, n) (App. C).
# --------------------------------------------------------------------------
def newton_schulz(psi: np.ndarray, steps: int = 5, coeffs=MUON_NS_COEFFS,
                  eps: float = 1e-7) -> np.ndarray:
    a, b, c = coeffs
    tall = psi.shape[0] > psi.shape[1]
    x = psi.T if tall else psi
    x = x / (np.linalg.norm(x) + eps)
    for _ in range(steps):
        gram = x @ x.T
        poly = b * gram + c * (gram @ gram)
        x = a * x + poly @ x
    return x.T if tall else x


def msign_svd(x: np.ndarray) -> np.ndarray:
    """msign(X) = U V^T from the thin SVD (Sec. 2.1).  Used only in pins."""
    u, _, vt = np.linalg.svd(x, full_matrices=False)
    return u @ vt


# --------------------------------------------------------------------------
# Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
# easy as 1, 2, 3", SC'11) -- the counter-based generator that feeds the
# Gaussian sketch Omega of Alg. 2.  Exact uint32 arithmetic in uint64.
# --------------------------------------------------------------------------
_PHILOX_M0 = 0xD2511F53
_PHILOX_M1 = 0xCD9E8D57
_PHILOX_W0 = 0x9E3779B9
_PHILOX_W1 = 0xBB67AE85
_MASK32 = 0xFFFFFFFF


def philox4x32_10(counters: np.ndarray, key) -> np.ndarray:
    """counters: (N, 4) uint32, key: (k0, k1) -> (N, 4) uint32 outputs."""
    c = np.asarray(counters, dtype=np.uint64).copy()
    k0 = np.uint64(int(key[0]) & _MASK32)
    k1 = np.uint64(int(key[1]) & _MASK32)
    m0 = np.uint64(_PHILOX_M0)
    m1 = np.uint64(_PHILOX_M1)
    mask = np.uint64(_MASK32)
    sh = np.uint64(32)
    for rnd in range(10):
        if rnd > 0:
            k0 = np.uint64((int(k0) + _PHILOX_W0) & _MASK32)
            k1 = np.uint64((int(k1) + _PHILOX_W1) & _MASK32)
        p0 = m0 * c[:, 0]
        p1 = m1 * c[:, 2]
        hi0, lo0 = p0 >> sh, p0 & mask
        hi1, lo1 = p1 >> sh, p1 & mask
        c = np.stack([hi1 ^ c[:, 1] ^ k0, lo1, hi0 ^ c[:, 3] ^ k1, lo0], axis=1)
    return c.astype(np.uint32)


def sketch_omega(seed: int, t: int, matrix_id: int, b: int, ell: int) -> np.ndarray:
    """Omega in R^{b x l}, Omega_ij ~ N(0, 1) (Alg. 2, Gaussian sketch line).

    Element (i, j) has linear index e = j*b + i.  Philox block e >> 2 with
    counter (e >> 2, matrix_id, t mod 2^32, t >> 32) and key (seed mod 2^32,
    seed >> 32) gives four words x0..x3; Box-Muller turns (x0, x1) into
    (z0, z1) and (x2, x3) into (z2, z3) with u1 = ((x >> 8) + 1) 2^-24 in
    (0, 1] and u2 = (x >> 8) 2^-24 in [0, 1):
        z_even = sqrt(-2 ln u1) cos(2 pi u2),  z_odd = sqrt(-2 ln u1) sin(2 pi u2).
    Element e takes z_{e mod 4} of its block.
    """
    n = b * ell
    if n == 0:
        return np.zeros((b, ell))
    nblk = (n + 3) // 4
    blk = np.arange(nblk, dtype=np.uint64)
    ctr = np.zeros((nblk, 4), dtype=np.uint64)
    ctr[:, 0] = blk & np.uint64(_MASK32)
    ctr[:, 1] = np.uint64(matrix_id & _MASK32)
    ctr[:, 2] = np.uint64(t & _MASK32)
    ctr[:, 3] = np.uint64((t >> 32) & _MASK32)
    x = philox4x32_10(ctr, (seed & _MASK32, (seed >> 32) & _MASK32)).astype(np.float64)
    two24 = 2.0 ** -24
    z = np.empty((nblk, 4))
    for pair in (0, 2):
        u1 = (np.floor(x[:, pair] / 256.0) + 1.0) * two24
        u2 = np.floor(x[:, pair + 1] / 256.0) * two24
        rad = np.sqrt(-2.0 * np.log(u1))
        z[:, pair] = rad * np.cos(2.0 * math.pi * u2)
        z[:, pair + 1] = rad * np.sin(2.0 * math.pi * u2)
    flat = z.reshape(-1)[:n]
    return flat.reshape(ell, b).T.copy()


# --------------------------------------------------------------------------
# NormPre-L, Alg. 2 (randomized interaction sketch) + Rayleigh-Ritz
# --------------------------------------------------------------------------
@dataclass
class SketchResult:
    ell: int
    q: np.ndarray            # a x l orthonormal basis of the candidate subspace
    b_mat: np.ndarray        # l x b,  Q^T Psi
    gamma_q: np.ndarray      # l x l,  Rayleigh-Ritz matrix
    ritz_values: np.ndarray  # top-min(r, l) Ritz values, descending
    ritz_vectors: np.ndarray  # l x min(r, l), matching Z
    selected: np.ndarray     # boolean mask over the top-min(r, l) values (lambda > 1)
    u_sel: np.ndarray = field(default=None)      # a x |C|
    lam_sel: np.ndarray = field(default=None)    # |C|


def _desc_order(vals: np.ndarray) -> np.ndarray:
    """Descending order, ties resolved towards the lower index."""
    return np.argsort(-vals, kind="stable")


def candidate_subspace(psi: np.ndarray, omega: np.ndarray, power_iters: int) -> np.ndarray:
    """Orthonormal basis Q (a x l) of the candidate subspace of Alg. 2:
    range((Psi Psi^T)^p Psi Omega), the Gaussian sketch of the column space of
    Psi sharpened by p power iterations (each one multiplies by Psi^T, then by
    Psi, so the leading directions of Gamma = Psi Psi^T gain weight lambda per
    pass).  ``np.linalg.qr`` supplies the orthonormal basis."""
    y = psi @ omega
    for _ in range(power_iters):
        y = psi @ (psi.T @ y)
    basis, _ = np.linalg.qr(y, mode="reduced")
    return basis


def rayleigh_ritz(psi: np.ndarray, basis: np.ndarray):
    """Ritz pairs of Gamma = Psi Psi^T on range(Q) (Alg. 2, Ritz pairs; App. B):
    with B = Q^T Psi the projected matrix is Gamma_Q = B B^T, whose eigenpairs
    are the squared singular values of B and its left singular vectors.
    Returns (B, Gamma_Q, values descending, l x l eigenvector matrix)."""
    b_mat = basis.T @ psi
    ell = basis.shape[1]
    z, sv, _ = np.linalg.svd(b_mat, full_matrices=True)
    vals = np.zeros(ell)
    vals[: sv.size] = sv ** 2
    return b_mat, b_mat @ b_mat.T, vals, z


def select_modes(vals_desc: np.ndarray, rank: int, force_count: int | None = None) -> np.ndarray:
    """Spectral budget and threshold of Alg. 2 / Eq. (P^L): of the leading
    min(r, l) Ritz values keep those strictly above one (the modes that the
    normalized geometry over-amplifies).  Returns a mask over the leading
    min(r, l) values."""
    top = min(rank, vals_desc.size)
    if force_count is None:
        return vals_desc[:top] > 1.0
    sel = np.zeros(top, bool)
    sel[:force_count] = True
    return sel


def interaction_sketch(psi: np.ndarray, rank: int, oversample: int,
                       power_iters: int, omega: np.ndarray,
                       force_count: int | None = None) -> SketchResult:
    """Randomized interaction sketch (Alg. 2, App. B): sketch width
    l = min(a, r + o) for a active rows, the candidate subspace, its Ritz
    pairs, the leading min(r, l) of them, and the selected set C.

    ``force_count`` (tests only) selects exactly that many leading Ritz pairs
    instead of applying the threshold, to compare against a run whose
    r-th boundary fell inside a near-tie.
    """
    ell = min(psi.shape[0], rank + oversample)
    basis = candidate_subspace(psi, omega[:, :ell], power_iters)
    b_mat, gamma_q, vals, z = rayleigh_ritz(psi, basis)
    top = min(rank, ell)
    sel = select_modes(vals, rank, force_count)
    lam, z_top = vals[:top], z[:, :top]
    u_hat = basis @ z_top
    return SketchResult(ell=ell, q=basis, b_mat=b_mat, gamma_q=gamma_q,
                        ritz_values=lam, ritz_vectors=z_top, selected=sel,
                        u_sel=u_hat[:, sel], lam_sel=lam[sel])


def localized_apply(psi: np.ndarray, u_sel: np.ndarray, lam_sel: np.ndarray) -> np.ndarray:
    """T = (I + U_C (Lambda_C^{-1/2} - I) U_C^T) Psi  (Alg. 1, NormPre-L line)."""
    if u_sel.shape[1] == 0:
        return psi.copy()
    coef = lam_sel ** -0.5 - 1.0
    return psi + u_sel @ (coef[:, None] * (u_sel.T @ psi))


def localized_exact(psi: np.ndarray, rank: int):
    """Exact eigenspace extraction (App. B): eig of Gamma = Psi Psi^T,
    A = {lambda > 1}, C = the min(r, |A|) largest of A."""
    gamma = psi @ psi.T
    evals, evecs = np.linalg.eigh(gamma)
    order = _desc_order(evals)
    evals, evecs = evals[order], evecs[:, order]
    active = np.flatnonzero(evals > 1.0)
    chosen = active[:rank]
    return evecs[:, chosen], evals[chosen]


# --------------------------------------------------------------------------
# Consistent update RMS (Sec. 3.1):  R_k(T) = 0.2 O_k^{-1}(T) / RMS(T),
# RMS(T) = ||T||_F / sqrt(mn);  W <- W - eta (R_k(T) + lambda_wd W)  (Alg. 1)
# --------------------------------------------------------------------------
def rms_scale(t_active: np.ndarray, k: int, target: float = TARGET_RMS) -> np.ndarray:
    t_w = orient_inv(t_active, k)
    fro = np.linalg.norm(t_w)
    if fro == 0.0:
        return np.zeros_like(t_w)
    rms = fro / math.sqrt(t_w.size)
    return target * t_w / rms


def parameter_update(w: np.ndarray, u: np.ndarray, lr: float, wd: float) -> np.ndarray:
    return w - lr * (u + wd * w)


# --------------------------------------------------------------------------
# One full step of Alg. 1 for one matrix.
# --------------------------------------------------------------------------
def normpre_step(w, g, m_prev, t: int, hp: HParams, variant: str = "G",
                 matrix_id: int = 0, omega: np.ndarray | None = None,
                 force_count: int | None = None, l_mode: str = "sketch") -> dict:
    """Returns a dict with the new momentum, Psi (W layout), T (W layout),
    the RMS-matched update U, the new W and, for NormPre-L, sketch diagnostics.

    variant: "G" (Newton-Schulz msign) or "L" (localized; l_mode "sketch" per
    Alg. 2 or "exact" per App. B); the reference steps "MUON" (``muon_step``)
    and "NORM" (normalize-only: the step with P = I, T = Psi, Sec. 2.2).
    """
    if variant == "MUON":
        return muon_step(w, g, m_prev, hp)
    w = np.asarray(w, np.float64)
    g = np.asarray(g, np.float64)
    m_prev = np.asarray(m_prev, np.float64)
    m = momentum_update(m_prev, g, hp.momentum)
    k = orientation_of(t, hp.orientation)
    x = None
    if hp.orientation == "both":
        psi = orient(both_axes_normalize(w, m, hp.tangent, hp.norm_eps), k)
    else:
        w_bar, m_bar = orient(w, k), orient(m, k)
        x = momentum_processing(m_bar, w_bar, hp.tangent)
        psi = diagonal_gram_normalize(x, hp.norm_eps)
    out = {"k": k, "momentum": m, "psi": orient_inv(psi, k)}
    if variant == "NORM":
        t_act = psi
    elif variant == "G":
        t_act = newton_schulz(psi, hp.ns_iters, hp.ns_coeffs, hp.ns_eps)
    elif variant == "L":
        a, b = psi.shape
        ell = min(a, hp.rank + hp.oversample)
        # Interaction source (App. A.4): the eigenpairs come from Psi, or from
        # the update before normalization through its trace-matched Gram
        # G_X = a X X^T / tr(X X^T) (App. A); either way they act on Psi.
        if hp.source == "psi":
            src = psi
        elif hp.source == "x" and x is not None:
            src = interaction_source_x(x)
        else:
            raise ValueError(f"interaction source {hp.source!r} with orientation {hp.orientation!r}")
        if l_mode == "exact":
            u_sel, lam_sel = localized_exact(src, hp.rank)
            out["lam_sel"] = lam_sel
        else:
            if omega is None:
                omega = sketch_omega(hp.seed, t, matrix_id, b, ell)
            sk = interaction_sketch(src, hp.rank, hp.oversample, hp.power_iters,
                                    omega, force_count)
            u_sel, lam_sel = sk.u_sel, sk.lam_sel
            out.update(ell=sk.ell, ritz_values=sk.ritz_values,
                       n_selected=int(sk.selected.sum()), omega=omega)
        t_act = localized_apply(psi, u_sel, lam_sel)
    else:
        raise ValueError(f"unknown variant {variant!r}")
    u = rms_scale(t_act, k, hp.target_rms)
    out["t"] = orient_inv(t_act, k)
    out["update"] = u
    out["w_new"] = parameter_update(w, u, hp.lr, hp.weight_decay)
    return out


# --------------------------------------------------------------------------
# Muon reference step (Sec. 2.1; configuration of App. A.1): heavy-ball
# momentum, then the same q-step Newton-Schulz iteration applied to the
# momentum itself (no tangent processing, no normalization, no orientation),
# and the RMS-matching convention the paper uses for Muon on LLaMA / Qwen3:
# U = 0.2 sqrt(max(m, n)) T.  Weight decay as in Alg. 1.
# --------------------------------------------------------------------------
def muon_step(w, g, m_prev, hp: HParams) -> dict:
    w = np.asarray(w, np.float64)
    g = np.asarray(g, np.float64)
    m_prev = np.asarray(m_prev, np.float64)
    m = momentum_update(m_prev, g, hp.momentum)
    t_mat = newton_schulz(m, hp.ns_iters, hp.ns_coeffs, hp.ns_eps)
    u = hp.target_rms * math.sqrt(max(m.shape)) * t_mat
    return {"k": 0, "momentum": m, "psi": m / (np.linalg.norm(m) + hp.ns_eps), "t": t_mat,
            "update": u, "w_new": parameter_update(w, u, hp.lr, hp.weight_decay)}


# --------------------------------------------------------------------------
# Spectral diagnostics of App. A (used by pins on the worked examples)
# --------------------------------------------------------------------------
def trace_matched_gram(x: np.ndarray) -> np.ndarray:
    """G_X = d X X^T / tr(X X^T), d = number of active rows (App. A)."""
    gram = x @ x.T
    return x.shape[0] * gram / np.trace(gram)


def interaction_spectrum(x_bar: np.ndarray, normalized: bool = True, eps: float = 1e-12) -> np.ndarray:
    """Eigenvalues, descending, of Gamma = Psi Psi^T with Psi = D(X)^-1 X
    (normalized) or of the trace-matched G_X (before normalization), for the
    update X in its active orientation (App. A, spectral dynamics: both have
    trace d, so their spectra are compared directly)."""
    g = (lambda p: p @ p.T)(diagonal_gram_normalize(x_bar, eps)) if normalized else trace_matched_gram(x_bar)
    return np.sort(np.linalg.eigvalsh(g))[::-1]


def energy_split(eigs, count: int, rank: int) -> dict:
    """Spectral transformation energy (App. A): e_i = (sqrt(lambda_i) - 1)^2
    over the nonzero eigenvalues (the first `count`, descending, positive);
    C = the largest at most `rank` eigenvalues above one.  E_top sums e_i
    over C, E_remain over the other eigenvalues above one, E_sub over those
    in (0, 1); E_global is the total."""
    lam = [float(v) for v in list(eigs)[:count] if v > 0.0]
    above = [v for v in lam if v > 1.0]
    chosen = above[:rank]
    e = lambda v: (math.sqrt(v) - 1.0) ** 2
    top = sum(e(v) for v in chosen)
    remain = sum(e(v) for v in above[len(chosen):])
    sub = sum(e(v) for v in lam if v < 1.0)
    return {"top": top, "remain": remain, "sub": sub, "global": top + remain + sub}


def descent_alignment(grads, updates):
    """Descent alignment (App. A, training dynamics): for each matrix the
    cosine of its gradient G and its update direction Phi before
    learning-rate scaling, decoupled weight decay excluded (for NormPre the
    RMS-matched update U of Alg. 1); Align_t is their plain mean.  A zero G or
    Phi gives cosine 0.  Returns (cosines, mean)."""
    cos = []
    for g, phi in zip(grads, updates):
        g = np.asarray(g, np.float64)
        phi = np.asarray(phi, np.float64)
        den = np.linalg.norm(g) * np.linalg.norm(phi)
        cos.append(float(np.sum(g * phi) / den) if den > 0 else 0.0)
    return cos, (sum(cos) / len(cos) if cos else 0.0)


def relative_fro(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (den if den > 0 else 1.0))
