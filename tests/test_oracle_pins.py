"""Pins of the float64 oracle against facts that do not come from the oracle
itself: brute-force least squares, closed forms derived from the paper's
appendix, hand-worked examples, counting and invariance properties.

Each test names the passage of the DuoGPT paper it follows.  A plausible slip
in the oracle (a dropped a/b/c term, a wrong sign of the residual, a transposed
G, the wrong column feeding the lazy residual update, a wrong tie order)
fails at least one of them.
"""

import itertools
import json
import os

import numpy as np
import pytest

from oracle import duo_ref as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


def _layer(seed, n, k, m, scale_sigma=0.5, outliers=0):
    rng = np.random.default_rng(seed)
    s = np.exp(scale_sigma * rng.standard_normal(k))
    if outliers:
        s[rng.choice(k, outliers, replace=False)] *= 20.0
    X = rng.standard_normal((m, k)) * s
    W = 0.02 * rng.standard_normal((n, k))
    return W, X


def _ridge(A, y, lam):
    """argmin_v |A v - y|^2 + lam |v|^2 and its value, by lstsq on the stacked
    system (no normal equations)."""
    q = A.shape[1]
    if q == 0:
        return np.zeros(0), float(y @ y)
    M = np.vstack([A, np.sqrt(lam) * np.eye(q)])
    t = np.concatenate([y, np.zeros(q)])
    v, *_ = np.linalg.lstsq(M, t, rcond=None)
    return v, float(np.sum((A @ v - y) ** 2) + lam * v @ v)


# ---------------------------------------------------------------------------
# Activation rule (Preliminaries, "Activation Sparsity")
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("k,p_x", [(7, 0.5), (16, 0.6), (10, 0.0), (9, 0.99), (12, 0.25)])
def test_sparsify_bruteforce_keys(k, p_x):
    rng = np.random.default_rng(k)
    # coarse values: many exact magnitude ties, signed zeros
    X = rng.integers(-3, 4, size=(40, k)).astype(np.float64)
    X[X == 0] = np.where(rng.random((X == 0).sum()) < 0.5, 0.0, -0.0)
    Xh, keep = R.sparsify_tokens(X, p_x)
    z = int(np.floor(p_x * k + 0.5))
    for t in range(X.shape[0]):
        assert (~keep[t]).sum() == z
        dropped = [(abs(X[t, c]), c) for c in range(k) if not keep[t, c]]
        kept = [(abs(X[t, c]), c) for c in range(k) if keep[t, c]]
        if dropped and kept:
            assert max(dropped) < min(kept)      # lexicographic (|x|, channel)
    assert np.array_equal(Xh, np.where(keep, X, 0.0))


def test_zero_count_rounding():
    assert R.act_zero_count(11008, 0.6) == 6605          # 6604.8
    assert R.act_zero_count(4096, 0.5) == 2048
    assert R.act_zero_count(2, 0.5) == 1                 # 1.5 rounds half up
    assert R.act_zero_count(3, 0.5) == 2


# ---------------------------------------------------------------------------
# Eq. 3 against direct constrained ridge least squares (App. A.1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_eq3_closed_form_equals_bruteforce(seed):
    rng = np.random.default_rng(seed)
    k, m = 8, 30
    X = rng.standard_normal((m, k)) * np.exp(rng.standard_normal(k))
    Xh, _ = R.sparsify_tokens(X, 0.5)
    w = rng.standard_normal(k)
    lam = 0.3
    for p in range(k):
        Lp, dw = R.obs_closed_form(w, Xh, X, lam, p)
        Lb, dwb = R.obs_bruteforce(w, Xh, X, lam, p)
        assert abs(Lp - Lb) <= 1e-9 * max(1.0, abs(Lb))
        np.testing.assert_allclose(dw, dwb, rtol=1e-8, atol=1e-10)
        assert abs(dw[p] + w[p]) < 1e-10                 # constraint dw e_p^T + w_p = 0


@pytest.mark.parametrize("k", [4, 6, 10])
def test_bruteforce_over_masks_single_weight(k):
    """Tiny layer: trying every one-weight mask by least squares finds the
    same optimum as minimising the Eq. 3 loss over p."""
    rng = np.random.default_rng(100 + k)
    X = rng.standard_normal((3 * k, k)) * np.exp(0.7 * rng.standard_normal(k))
    Xh, _ = R.sparsify_tokens(X, 0.5)
    w = rng.standard_normal(k)
    lam = 0.1
    closed = [R.obs_closed_form(w, Xh, X, lam, p)[0] for p in range(k)]
    brute = [R.obs_bruteforce(w, Xh, X, lam, p)[0] for p in range(k)]
    assert int(np.argmin(closed)) == int(np.argmin(brute))
    assert abs(min(closed) - min(brute)) <= 1e-9 * max(1.0, min(brute))


def test_theorem1_single_step_gain():
    """Theorem 1 (proof in App. A.5): for one step the DuoGPT loss is below the
    SparseGPT loss by r Xh^T H^-1_{-p} Xh r^T >= 0."""
    rng = np.random.default_rng(7)
    k, m, lam = 6, 25, 0.2
    X = rng.standard_normal((m, k))
    Xh, _ = R.sparsify_tokens(X, 0.5)
    w = rng.standard_normal(k)
    Hl = Xh.T @ Xh + lam * np.eye(k)
    Hinv = np.linalg.inv(Hl)
    r = (X - Xh) @ w
    for p in range(k):
        h = Hinv[p, p]
        dw_s = -(w[p] / h) * Hinv[p, :]
        loss_s = np.sum((Xh @ dw_s - r) ** 2) + lam * dw_s @ dw_s
        loss_d, _ = R.obs_closed_form(w, Xh, X, lam, p)
        Hm = Hinv - np.outer(Hinv[:, p], Hinv[p, :]) / h
        gain = (Xh.T @ r) @ Hm @ (Xh.T @ r)
        assert gain >= 0
        assert abs((loss_s - loss_d) - gain) <= 1e-9 * max(1.0, loss_s)


# ---------------------------------------------------------------------------
# Score factor, D and the Cholesky identities (Eq. 7, App. A.2-A.4)
# ---------------------------------------------------------------------------

def _terms(seed, k=9, m=40, p_x=0.5, damp=0.05):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((m, k)) * np.exp(0.8 * rng.standard_normal(k))
    H, G, a = R.hessian_terms(X, p_x)
    L, lam = R.inverse_cholesky(H, damp)
    fac, D, (aa, b, c) = R.score_terms(G, L, a)
    Xh, _ = R.sparsify_tokens(X, p_x)
    return X, Xh, H, G, a, L, lam, fac, D


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_score_factor_is_constrained_ridge(seed):
    """With columns < p frozen, removing w_p costs w_p^2 * fac_p where
    fac_p = lam + min_v |Xh_{>p} v - X_dense_p|^2 + lam |v|^2 (the residual of
    regressing the dense column p on the later sparse columns), and the optimal
    correction of the later weights is w_p * v*.  In the sweep that correction
    is w_p * (D[p, j] - L[j, p] / L[p, p])."""
    X, Xh, H, G, a, L, lam, fac, D = _terms(seed)
    k = X.shape[1]
    for p in range(k):
        v, val = _ridge(Xh[:, p + 1:], X[:, p], lam)
        assert abs(fac[p] - (lam + val)) <= 1e-8 * max(1.0, abs(fac[p]))
        step = D[p, p + 1:] - L[p + 1:, p] / L[p, p]
        np.testing.assert_allclose(step, v, rtol=1e-7, atol=1e-9)
        assert fac[p] >= lam * (1 - 1e-12)


@pytest.mark.parametrize("seed", [0, 1])
def test_D_is_residual_regression(seed):
    """A kept weight w_p still moves the later weights by w_p * D[p, >p], the
    ridge regression of dX_p on the later sparse columns (Eq. 3 update term,
    App. A.4)."""
    X, Xh, H, G, a, L, lam, fac, D = _terms(seed)
    k = X.shape[1]
    dX = X - Xh
    for p in range(k):
        u, _ = _ridge(Xh[:, p + 1:], dX[:, p], lam)
        np.testing.assert_allclose(D[p, p + 1:], u, rtol=1e-7, atol=1e-9)
        assert np.all(D[p, :p + 1] == 0.0)


def test_last_column_closed_form():
    X, Xh, H, G, a, L, lam, fac, D = _terms(5)
    k = X.shape[1]
    assert abs(fac[k - 1] - (X[:, k - 1] @ X[:, k - 1] + lam)) <= 1e-10 * fac[k - 1]
    # k = 1: the score of the only weight is w^2 (|x|^2 + lam)
    x = np.array([[3.0], [-2.0], [0.5]])
    H, G, a = R.hessian_terms(x, 0.0)
    L, lam = R.inverse_cholesky(H, 0.1)
    fac1, _, _ = R.score_terms(G, L, a)
    assert abs(fac1[0] - (x[:, 0] @ x[:, 0] + lam)) < 1e-12


@pytest.mark.parametrize("seed", [0, 1])
def test_cholesky_identities(seed):
    """App. A.2: L_{p+1:,p+1:} L_{p+1:,p+1:}^T is the inverse of the trailing
    block of H.  App. A.3: after Gaussian elimination of columns < p (the
    update of Sec. 3), column p of H^-1 divided by its diagonal equals
    L[:, p] / L[p, p]."""
    X, Xh, H, G, a, L, lam, fac, D = _terms(seed)
    k = X.shape[1]
    Hl = H + lam * np.eye(k)
    for p in range(k - 1):
        np.testing.assert_allclose(L[p + 1:, p + 1:] @ L[p + 1:, p + 1:].T,
                                   np.linalg.inv(Hl[p + 1:, p + 1:]), rtol=1e-8, atol=1e-14)
    Hinv = np.linalg.inv(Hl)
    for p in range(k):
        np.testing.assert_allclose(Hinv[:, p] / Hinv[p, p], L[:, p] / L[p, p], rtol=1e-8, atol=1e-12)
        Hinv = Hinv - np.outer(Hinv[:, p], Hinv[p, :]) / Hinv[p, p]


def test_bc_terms_explicit():
    """b and c as first defined in Sec. 4.3 (before the Cholesky rewrite)."""
    X, Xh, H, G, a, L, lam, fac, D = _terms(11)
    k = X.shape[1]
    dX = X - Xh
    Hl = H + lam * np.eye(k)
    _, _, (aa, b, c) = R.score_terms(G, L, a)
    Hinv = np.linalg.inv(Hl)
    for p in range(k):
        z = dX[:, p] @ Xh                          # dX_p Xh^T
        Hm = np.zeros((k, k))
        Hm[p + 1:, p + 1:] = np.linalg.inv(Hl[p + 1:, p + 1:])
        assert abs(b[p] - z @ Hm @ z) <= 1e-8 * max(1.0, abs(b[p]))
        # c_p = dX_p Xh^T H^-1_{:,p} / [H^-1]_pp with the inverse after eliminating < p
        Hp = np.zeros((k, k))
        Hp[p:, p:] = np.linalg.inv(Hl[p:, p:])
        assert abs(c[p] - z @ Hp[:, p] / Hp[p, p]) <= 1e-8 * max(1.0, abs(c[p]))
    np.testing.assert_allclose(aa, np.sum(dX * dX, axis=0))


# ---------------------------------------------------------------------------
# Hand-worked examples
# ---------------------------------------------------------------------------

def _golden():
    with open(GOLDEN) as f:
        return json.load(f)["examples"]


@pytest.mark.parametrize("ex", _golden(), ids=lambda e: e["name"])
def test_hand_examples(ex):
    X = np.array(ex["X"])
    W = np.array(ex["W"])
    e = ex["expect"]
    _, keep_x = R.sparsify_tokens(X, ex["p_x"])
    assert keep_x.tolist() == e["keep_x"]
    out = R.prune_layer(W, X, ex["p_x"], ex["p_w"], damp=ex["damp"], B=ex["B"])
    tol = dict(rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out["H"], e["H"], **tol)
    np.testing.assert_allclose(out["G"], e["G"], **tol)
    np.testing.assert_allclose(out["a"], e["a"], **tol)
    assert abs(out["lam"] - e["lam"]) < 1e-12
    np.testing.assert_allclose(out["L"], e["L"], **tol)
    np.testing.assert_allclose(out["b"], e["b"], **tol)
    np.testing.assert_allclose(out["c"], e["c"], **tol)
    np.testing.assert_allclose(out["D"], e["D"], **tol)
    np.testing.assert_allclose(out["fac"], e["fac"], **tol)
    assert out["keep"].tolist() == e["keep_w"]
    np.testing.assert_allclose(out["W_hat"], e["W_hat"], **tol)
    J = R.objective(W, out["W_hat"], X, ex["p_x"])
    assert abs(J - e["objective"]) < 1e-9


# ---------------------------------------------------------------------------
# Sweep: counts, special cases, lazy == eager, objective, invariances
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n,k,p_w,B", [(7, 50, 0.5, 16), (5, 33, 0.6, 8), (3, 10, 0.37, 4), (4, 12, 0.0, 5)])
def test_mask_counts_exact(n, k, p_w, B):
    W, X = _layer(n * k, n, k, 4 * k)
    out = R.prune_layer(W, X, 0.5, p_w, damp=0.01, B=B)
    keep = out["keep"]
    counts = R.block_prune_counts(n, k, p_w, B)
    for bi, j0 in enumerate(range(0, k, B)):
        assert (~keep[:, j0:j0 + B]).sum() == counts[bi]
        assert abs(counts[bi] - p_w * n * min(B, k - j0)) <= 1.0
    assert (~keep).sum() == int(np.floor(p_w * n * k + 0.5))
    assert np.all(out["W_hat"][~keep] == 0.0)


def test_selected_scores_are_lowest():
    W, X = _layer(3, 12, 40, 160)
    scores = []
    out = R.prune_layer(W, X, 0.5, 0.5, B=16, scores_out=scores)
    for bi, j0 in enumerate(range(0, 40, 16)):
        S = scores[bi]
        keep = out["keep"][:, j0:j0 + 16]
        assert S[~keep].max() <= S[keep].min()


def test_zero_sparsity_returns_weights_bit_unchanged():
    W, X = _layer(9, 6, 24, 80)
    out = R.prune_layer(W, X, 0.0, 0.0, B=8)
    assert np.array_equal(out["W_hat"], W)
    assert np.all(out["D"] == 0.0) and np.all(out["a"] == 0.0)


def test_weight_sparsity_zero_still_corrects():
    W, X = _layer(10, 6, 24, 80)
    out = R.prune_layer(W, X, 0.5, 0.0, B=8)
    assert out["keep"].all()
    assert np.max(np.abs(out["W_hat"] - W)) > 1e-6
    J_duo = R.objective(W, out["W_hat"], X, 0.5)
    J_id = R.objective(W, W, X, 0.5)
    assert J_duo < J_id


def test_no_activation_sparsity_is_sparsegpt():
    W, X = _layer(12, 8, 40, 120)
    out = R.prune_layer(W, X, 0.0, 0.5, B=16)
    Ws, ks = R.sparsegpt_layer(W, X, 0.0, 0.5, B=16)
    assert np.array_equal(out["keep"], ks)
    np.testing.assert_allclose(out["W_hat"], Ws, rtol=0, atol=1e-15)
    assert np.all(out["D"] == 0.0)


@pytest.mark.parametrize("B", [1, 3, 8, 16, 64])
def test_lazy_equals_eager(B):
    W, X = _layer(20 + B, 9, 45, 150, outliers=2)
    H, G, a = R.hessian_terms(X, 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    We, ke = R.sweep_eager(W, L, D, fac, 0.5, B)
    Wb, kb = R.sweep_blocked(W, L, D, fac, 0.5, B)
    assert np.array_equal(ke, kb)
    np.testing.assert_allclose(Wb, We, rtol=0, atol=1e-12 * np.abs(We).max())
    # forced mask: the result no longer depends on the block size
    W1, _ = R.sweep_blocked(W, L, D, fac, 0.5, 5, mask_in=ke)
    np.testing.assert_allclose(W1, We, rtol=0, atol=1e-12 * np.abs(We).max())


def test_lazy_uses_preprune_values():
    """Reading R-lazy is what makes blocked == eager; the post-prune reading
    (lazy update fed with the pruned columns) does not match."""
    W, X = _layer(31, 6, 32, 120)
    H, G, a = R.hessian_terms(X, 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    We, ke = R.sweep_eager(W, L, D, fac, 0.5, 8)
    # post-prune variant, written out here only to show the difference
    Wp = W.copy()
    for j0 in range(0, 32, 8):
        j1 = j0 + 8
        E = np.zeros((6, 8))
        for j in range(j0, j1):
            w0 = Wp[:, j].copy()
            p = w0 * ke[:, j]
            E[:, j - j0] = (w0 - p) / L[j, j]
            Wp[:, j] = p
            Wp[:, j + 1:j1] -= np.outer(E[:, j - j0], L[j + 1:j1, j]) - np.outer(w0, D[j, j + 1:j1])
        Wp[:, j1:] -= E @ L[j1:, j0:j1].T - Wp[:, j0:j1] @ D[j0:j1, j1:]
    assert np.max(np.abs(Wp * ke - We)) > 1e-6


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_objective_below_magnitude(seed):
    W, X = _layer(40 + seed, 16, 64, 256, scale_sigma=1.0, outliers=2)
    out = R.prune_layer(W, X, 0.5, 0.5, B=16)
    Wm, _ = R.magnitude_layer(W, 0.5, B=16)
    J_duo = R.objective(W, out["W_hat"], X, 0.5)
    J_mag = R.objective(W, Wm, X, 0.5)
    assert J_duo < J_mag


def test_beats_single_mask_bruteforce_bound():
    """Tiny layer, two weights removed from one row: the greedy sweep cannot
    beat the exhaustive optimum over all masks (each solved by least squares
    with the same ridge term), and it should not be far from it."""
    rng = np.random.default_rng(77)
    k, m = 6, 30
    X = rng.standard_normal((m, k)) * np.exp(0.5 * rng.standard_normal(k))
    W = rng.standard_normal((1, k))
    out = R.prune_layer(W, X, 0.5, 2.0 / k, damp=0.01, B=k)
    Xh, _ = R.sparsify_tokens(X, 0.5)
    lam = out["lam"]
    J_sweep = float(np.sum((X @ W[0] - Xh @ out["W_hat"][0]) ** 2))
    best = np.inf
    for pair in itertools.combinations(range(k), 2):
        free = [j for j in range(k) if j not in pair]
        v, _ = _ridge(Xh[:, free], X @ W[0], lam)
        wnew = np.zeros(k)
        wnew[free] = v
        best = min(best, float(np.sum((X @ W[0] - Xh @ wnew) ** 2)))
    assert J_sweep >= best * (1 - 1e-9)
    assert J_sweep <= 20.0 * best


def test_input_scale_invariance():
    W, X = _layer(50, 10, 48, 160)
    a = R.prune_layer(W, X, 0.5, 0.5, B=16)
    b = R.prune_layer(W, 4.0 * X, 0.5, 0.5, B=16)
    assert np.array_equal(a["keep"], b["keep"])
    np.testing.assert_allclose(b["W_hat"], a["W_hat"], rtol=1e-9, atol=1e-13)


def test_row_permutation_equivariance():
    W, X = _layer(51, 10, 48, 160)
    perm = np.random.default_rng(0).permutation(10)
    a = R.prune_layer(W, X, 0.5, 0.5, B=16)
    b = R.prune_layer(W[perm], X, 0.5, 0.5, B=16)
    assert np.array_equal(a["keep"][perm], b["keep"])
    np.testing.assert_allclose(b["W_hat"], a["W_hat"][perm], rtol=1e-12, atol=1e-15)


def test_two_stream_residual():
    """Multi-layer case (Sec. 4.2): X_src (pruned model's input) differs from
    X_dense.  H depends only on the sparsified X_src; dX = X_dense - Xh; the
    last-column closed form becomes fac_{k-1} = |X_dense_{k-1}|^2 + lam."""
    rng = np.random.default_rng(60)
    k, m = 9, 50
    Xd = rng.standard_normal((m, k))
    Xs = Xd + 0.1 * rng.standard_normal((m, k))
    H, G, a = R.hessian_terms(Xs, 0.5, Xd)
    Xh, _ = R.sparsify_tokens(Xs, 0.5)
    np.testing.assert_allclose(H, Xh.T @ Xh)
    np.testing.assert_allclose(G, (Xd - Xh).T @ Xh)
    L, lam = R.inverse_cholesky(H, 0.05)
    fac, D, _ = R.score_terms(G, L, a)
    assert abs(fac[-1] - (Xd[:, -1] @ Xd[:, -1] + lam)) < 1e-9 * fac[-1]
    for p in range(k):
        v, val = _ridge(Xh[:, p + 1:], Xd[:, p], lam)
        assert abs(fac[p] - (lam + val)) <= 1e-8 * fac[p]


@pytest.mark.parametrize("m,k,p_x", [(300, 37, 0.5), (200, 64, 0.0), (100, 20, 1.0), (257, 129, 0.6)])
def test_hessian_entries_match_full_terms(m, k, p_x):
    """Reading R-act through a selection (hessian_entries) and through a
    stable sort (hessian_terms) give the same stage-1 entries, with planted
    magnitude ties and signed zeros; token ranges add up."""
    rng = np.random.default_rng(k)
    X = np.round(rng.standard_normal((m, k)) * 4) / 4
    X[::5, ::3] = -0.0
    Xd = X + 0.1 * rng.standard_normal((m, k))
    H, G, a = R.hessian_terms(X, p_x, Xd)
    idx = np.sort(rng.choice(k, min(k, 9), replace=False))
    e = R.hessian_entries(X, p_x, idx, Xd)
    np.testing.assert_allclose(e["H"], H[np.ix_(idx, idx)], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(e["G"], G[np.ix_(idx, idx)], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(e["a"], a, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(e["diag"], np.diag(H), rtol=1e-12, atol=1e-12)
    lo = R.hessian_entries(X, p_x, idx, Xd, 0, m // 2)
    hi = R.hessian_entries(X, p_x, idx, Xd, m // 2, m)
    np.testing.assert_allclose(lo["H"] + hi["H"], e["H"], rtol=1e-12, atol=1e-12)
    rows = idx[::2]
    er = R.hessian_entries(X, p_x, idx, Xd, rows=rows)
    np.testing.assert_allclose(er["G_rows"], G[rows], rtol=1e-12, atol=1e-12)


def test_objective_candidates_and_token_ranges():
    """The objective of several candidates at once equals the single calls,
    and objectives over disjoint token ranges add up (Sec. 4.2: a sum over
    tokens of squared output errors)."""
    W, X = _layer(31, 6, 20, 300)
    W1 = W * (np.arange(20) % 3 != 0)
    W2 = 0.9 * W
    J = R.objective(W, [W1, W2], X, 0.5)
    assert J == [R.objective(W, W1, X, 0.5), R.objective(W, W2, X, 0.5)]
    Jlo = R.objective(W, W1, X[:110], 0.5)
    Jhi = R.objective(W, W1, X[110:], 0.5)
    assert abs(Jlo + Jhi - J[0]) <= 1e-12 * J[0]
    # the definition by hand on one token
    Xh, _ = R.sparsify_tokens(X[:1], 0.5)
    r = W @ X[0] - W1 @ Xh[0]
    assert abs(R.objective(W, W1, X[:1], 0.5) - r @ r) <= 1e-12 * (r @ r)


@pytest.mark.parametrize("t", [1, 5, 16])
def test_window_terms_trailing_block(t):
    """Trailing-window self-containment (the UL structure of Sec. 4.3's
    Cholesky of the inverse): L, fac and D on the last t columns follow from
    the window's H, G, a and the global lambda alone.  Checked against the
    full-matrix oracle and, independently, against the ridge characterisation
    fac_p = lambda + min |v Xh_{>p} - X_dense_p|^2 + lambda |v|^2 (App. A)."""
    W, X = _layer(70 + t, 1, 24, 120)
    Xd = X + 0.05 * np.random.default_rng(t).standard_normal(X.shape)
    H, G, a = R.hessian_terms(X, 0.5, Xd)
    L, lam = R.inverse_cholesky(H, 0.05)
    fac, D, _ = R.score_terms(G, L, a)
    k = H.shape[0]
    T = slice(k - t, k)
    Lw, facw, Dw = R.window_terms(H[T, T], G[T, T], a[T], lam)
    np.testing.assert_allclose(Lw, L[T, T], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(facw, fac[T], rtol=1e-9)
    np.testing.assert_allclose(Dw, D[T, T], rtol=1e-8, atol=1e-10)
    Xh, _ = R.sparsify_tokens(X, 0.5)
    for i, p in enumerate(range(k - t, k)):
        _, val = _ridge(Xh[:, p + 1:], Xd[:, p], lam)
        assert abs(facw[i] - (lam + val)) <= 1e-8 * facw[i]


# ---------------------------------------------------------------------------
# act_order (App. B, calibration settings): channels by decreasing diag(H)
# ---------------------------------------------------------------------------

def test_act_order_perm_direction_and_ties():
    """Closed form: largest diagonal first, equal diagonals in channel order."""
    H = np.diag([1.0, 3.0, 3.0, 0.0, 2.0, 3.0])
    H[0, 1] = H[1, 0] = 0.5  # off-diagonal entries play no part
    assert R.act_order_perm(H).tolist() == [1, 2, 5, 4, 0, 3]


def test_act_order_is_identity_for_sorted_diagonal():
    """When diag(H) already decreases, act_order changes nothing (bitwise)."""
    rng = np.random.default_rng(70)
    k, n, m = 40, 12, 256
    X = rng.standard_normal((m, k))
    X *= np.sqrt((k - np.arange(k)) / np.sum(X * X, axis=0))  # column c: |x_c|^2 = k - c
    W = 0.02 * rng.standard_normal((n, k))
    H, _, _ = R.hessian_terms(X, 0.0)
    assert np.all(np.diff(np.diag(H)) < 0)  # precondition of the pin
    a = R.prune_layer(W, X, 0.0, 0.5, B=8)
    b = R.prune_layer(W, X, 0.0, 0.5, B=8, act_order=True)
    assert b["perm"].tolist() == list(range(k))
    assert np.array_equal(a["keep"], b["keep"])
    assert np.array_equal(a["W_hat"], b["W_hat"])


@pytest.mark.parametrize("seed", [71, 72])
def test_act_order_channel_permutation_invariance(seed):
    """With act_order the result no longer depends on how the input channels
    are numbered (no ties): relabelling the channels of W and X relabels the
    output the same way.  Without act_order the result does depend on it."""
    W, X = _layer(seed, 10, 48, 200, scale_sigma=1.0)
    pi = np.random.default_rng(seed + 100).permutation(48)
    a = R.prune_layer(W, X, 0.5, 0.5, B=16, act_order=True)
    b = R.prune_layer(W[:, pi], X[:, pi], 0.5, 0.5, B=16, act_order=True)
    assert np.array_equal(a["keep"][:, pi], b["keep"])
    np.testing.assert_allclose(b["W_hat"], a["W_hat"][:, pi], rtol=1e-9, atol=1e-12)
    c = R.prune_layer(W, X, 0.5, 0.5, B=16)
    d = R.prune_layer(W[:, pi], X[:, pi], 0.5, 0.5, B=16)
    assert not np.allclose(d["W_hat"], c["W_hat"][:, pi], rtol=1e-6, atol=1e-9)


def test_act_order_lazy_equals_eager():
    W, X = _layer(73, 9, 40, 180, scale_sigma=1.0)
    a = R.prune_layer(W, X, 0.5, 0.5, B=8, act_order=True)
    b = R.prune_layer(W, X, 0.5, 0.5, B=8, act_order=True, blocked=False)
    assert np.array_equal(a["keep"], b["keep"])
    np.testing.assert_allclose(a["W_hat"], b["W_hat"], rtol=1e-9, atol=1e-13)


def test_act_order_forced_mask_follows_channels():
    """A forced mask is given in the original channel order."""
    W, X = _layer(74, 8, 32, 160, scale_sigma=1.0)
    a = R.prune_layer(W, X, 0.5, 0.5, B=8, act_order=True)
    b = R.prune_layer(W, X, 0.5, 0.5, B=8, act_order=True, mask_in=a["keep"])
    assert np.array_equal(a["keep"], b["keep"])
    np.testing.assert_allclose(a["W_hat"], b["W_hat"], rtol=1e-12, atol=1e-15)


def test_act_order_equals_plain_method_on_reordered_channels():
    """act_order = the plain method (pinned above) run on the channels listed
    in act_order_perm order, relabelled back."""
    W, X = _layer(75, 10, 48, 200, scale_sigma=1.0)
    a = R.prune_layer(W, X, 0.5, 0.5, B=16, act_order=True)
    H, _, _ = R.hessian_terms(X, 0.5)
    perm = R.act_order_perm(H)
    assert np.array_equal(a["perm"], perm)
    b = R.prune_layer(W[:, perm], X[:, perm], 0.5, 0.5, B=16)
    inv = np.argsort(perm)
    assert np.array_equal(a["keep"], b["keep"][:, inv])
    np.testing.assert_allclose(a["W_hat"], b["W_hat"][:, inv], rtol=1e-9, atol=1e-12)


# ---------------------------------------------------------------------------
# N:M semi-structured variant (App. B: mask selection and pruning over every
# group of 4 consecutive columns)
# ---------------------------------------------------------------------------

def test_nm_selection_closed_form():
    S = np.array([[3.0, 1.0, 2.0, 1.0], [0.0, 0.0, 0.0, 0.0], [4.0, 3.0, 2.0, 1.0]])
    keep = R.select_nm_mask(S, 2)
    assert keep.tolist() == [[True, False, True, False], [False, False, True, True], [True, True, False, False]]
    assert R.select_nm_mask(S, 0).all() and not R.select_nm_mask(S, 4).any()


def test_nm_orthogonal_inputs_closed_form():
    """Orthogonal input channels and no activation sparsity: H is diagonal, so
    L is diagonal, G = 0, D = 0 and nothing is compensated; the 2:4 result is
    W with the two lowest w^2 (|x_j|^2 + lambda) of every row and group of 4
    removed."""
    rng = np.random.default_rng(80)
    n, k, m, damp = 6, 24, 64, 0.01
    Q, _ = np.linalg.qr(rng.standard_normal((m, k)))
    s = np.exp(rng.standard_normal(k))
    X = Q * s
    W = rng.standard_normal((n, k))
    out = R.prune_layer(W, X, 0.0, 0.5, damp=damp, B=8, nm=(2, 4))
    lam = damp * np.mean(s * s)
    S = W * W * (s * s + lam)
    keep = np.concatenate([R.select_nm_mask(S[:, g:g + 4], 2) for g in range(0, k, 4)], axis=1)
    assert np.array_equal(out["keep"], keep)
    np.testing.assert_allclose(out["W_hat"], W * keep, rtol=1e-9, atol=1e-12)


@pytest.mark.parametrize("nm", [(2, 4), (1, 4), (3, 4)])
def test_nm_counts_and_lowest_scores(nm):
    W, X = _layer(81, 12, 64, 256, scale_sigma=1.0)
    scores = []
    out = R.prune_layer(W, X, 0.5, 0.5, B=16, nm=nm, scores_out=scores)
    keep = out["keep"]
    N, M = nm
    assert np.all((~keep).reshape(12, -1, M).sum(axis=2) == N)
    S = np.concatenate(scores, axis=1)
    for g in range(0, 64, M):
        assert np.array_equal(keep[:, g:g + M], R.select_nm_mask(S[:, g:g + M], N))
    assert np.all(out["W_hat"][~keep] == 0)


def test_nm_lazy_equals_eager():
    W, X = _layer(82, 10, 48, 200, scale_sigma=1.0)
    a = R.prune_layer(W, X, 0.5, 0.5, B=16, nm=(2, 4))
    b = R.prune_layer(W, X, 0.5, 0.5, B=16, nm=(2, 4), blocked=False)
    assert np.array_equal(a["keep"], b["keep"])
    np.testing.assert_allclose(a["W_hat"], b["W_hat"], rtol=1e-9, atol=1e-13)


def test_nm_uses_current_values_and_compensates():
    """The group mask is chosen from the values the sweep has updated so far,
    not from the dense weights, and the kept weights are compensated: the
    result has a lower objective than pruning the dense 2:4 magnitude mask."""
    W, X = _layer(83, 16, 64, 400, scale_sigma=1.0)
    out = R.prune_layer(W, X, 0.5, 0.5, B=16, nm=(2, 4))
    H, G, a = R.hessian_terms(X, 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, _, _ = R.score_terms(G, L, a)
    S0 = W * W * fac
    keep0 = np.concatenate([R.select_nm_mask(S0[:, g:g + 4], 2) for g in range(0, 64, 4)], axis=1)
    assert not np.array_equal(out["keep"], keep0)  # later groups see compensated values
    J = R.objective(W, out["W_hat"], X, 0.5)
    assert J < R.objective(W, W * keep0, X, 0.5)


def test_nm_with_act_order_is_refused():
    W, X = _layer(84, 4, 16, 64)
    with pytest.raises(ValueError):
        R.prune_layer(W, X, 0.5, 0.5, B=8, nm=(2, 4), act_order=True)


# ---------------------------------------------------------------------------
# Joint pruning and RTN quantisation (Table 4: channel-wise uniform integer,
# group size 128, inside the sweep)
# ---------------------------------------------------------------------------

def test_quant_grid_closed_form():
    # range [-1, 2] in 3 steps of 1.0 (2 bits); zero code 1
    assert R.quant_grid(np.array([-1.0, 0.5, 2.0]), 2) == (1.0, 1.0)
    # positive values: the range still includes 0; 4 bits: 15 steps of 0.2
    s, z = R.quant_grid(np.array([1.0, 3.0]), 4)
    assert abs(s - 0.2) < 1e-15 and z == 0.0
    # empty range -> [-1, 1]
    assert R.quant_grid(np.zeros(4), 8) == (2.0 / 255, 128.0)
    x = np.array([-1.2, -0.5, 0.49, 0.51, 1.5, 2.6])
    np.testing.assert_array_equal(R.quantize(x, 1.0, 1.0, 2), [-1.0, -0.0, 0.0, 1.0, 2.0, 2.0])
    assert R.quantize(np.array([0.0]), 0.3, 5.0, 4)[0] == 0.0  # 0 is on every grid


def test_quant_orthogonal_inputs_is_plain_rtn():
    """Orthogonal channels, no activation sparsity, no pruning: nothing is
    compensated, so the result is plain round-to-nearest of W with one grid
    per row and group of the dense weights."""
    rng = np.random.default_rng(90)
    n, k, m = 5, 32, 64
    Q, _ = np.linalg.qr(rng.standard_normal((m, k)))
    X = Q * np.exp(rng.standard_normal(k))
    W = rng.standard_normal((n, k))
    for bits, group in ((4, 8), (8, 16), (3, 4)):
        out = R.prune_layer(W, X, 0.0, 0.0, B=16, quant=(bits, group))
        want = np.empty_like(W)
        for r in range(n):
            for g in range(0, k, group):
                s, z = R.quant_grid(W[r, g:g + group], bits)
                want[r, g:g + group] = R.quantize(W[r, g:g + group], s, z, bits)
        assert out["keep"].all()
        np.testing.assert_allclose(out["W_hat"], want, rtol=0, atol=1e-12)


@pytest.mark.parametrize("bits,group", [(4, 16), (8, 32), (4, 8)])
def test_quant_values_on_grids_fixed_at_group_start(bits, group):
    W, X = _layer(91, 8, 64, 256, scale_sigma=1.0)
    qp = []
    out = R.prune_layer(W, X, 0.5, 0.5, B=32, quant=(bits, group), qparams_out=qp)
    assert len(qp) == 64 // group
    Wh, keep = out["W_hat"], out["keep"]
    assert np.all(Wh[~keep] == 0)
    for gi, (s, z, _) in enumerate(qp):
        cols = slice(gi * group, (gi + 1) * group)
        codes = Wh[:, cols] / s[:, None] + z[:, None]
        assert np.allclose(codes, np.round(codes), atol=1e-9)          # on the grid
        assert np.all(np.round(codes) >= -1e-9) and np.all(np.round(codes) <= 2 ** bits - 1 + 1e-9)
    # grids come from the values the sweep has compensated so far, not the dense W
    s0, _ = R.quant_grid(W[0, group:2 * group], bits)
    assert abs(qp[1][0][0] - s0) > 1e-12


def test_quant_lazy_equals_eager():
    W, X = _layer(92, 9, 48, 200, scale_sigma=1.0)
    a = R.prune_layer(W, X, 0.5, 0.5, B=16, quant=(4, 8))
    b = R.prune_layer(W, X, 0.5, 0.5, B=16, quant=(4, 8), blocked=False)
    assert np.array_equal(a["keep"], b["keep"])
    np.testing.assert_allclose(a["W_hat"], b["W_hat"], rtol=1e-9, atol=1e-12)


@pytest.mark.parametrize("quant", [None, (4, 4), (8, 8), (3, 2)])
def test_quant_last_column_is_ridge_optimum_given_frozen_prefix(quant):
    """Without activation sparsity the sweep leaves the last column at the
    damped least-squares optimum given every earlier column's final (pruned
    or quantised) value, v* = (r.x + lambda w) / (x.x + lambda) with r the
    target minus the prefix's contribution; the column then keeps the grid
    value of v* (or 0 where pruned).  This pins the compensation of the
    quantisation error, which the pruning pins do not see."""
    rng = np.random.default_rng(94)
    n, k, m, damp = 6, 24, 200, 0.01
    X = rng.standard_normal((m, k)) * np.exp(rng.standard_normal(k))
    W = 0.02 * rng.standard_normal((n, k))
    qp = []
    out = R.prune_layer(W, X, 0.0, 0.5, damp=damp, B=8, quant=quant, qparams_out=qp)
    Wh, keep = out["W_hat"], out["keep"][:, k - 1]
    lam = damp * np.mean(np.sum(X * X, axis=0))
    r = W @ X.T - Wh[:, :k - 1] @ X[:, :k - 1].T
    x = X[:, k - 1]
    v = (r @ x + lam * W[:, k - 1]) / (x @ x + lam)
    if quant is not None:
        sc, z, _ = qp[-1]
        v = sc * (np.clip(np.round(v / sc) + z, 0, 2 ** quant[0] - 1) - z)
    np.testing.assert_allclose(Wh[:, k - 1], np.where(keep, v, 0.0), rtol=0, atol=1e-12)


def test_forced_values_hook_reproduces_the_run():
    """values_in (a test hook, like mask_in) fed with a run's own output
    reproduces that run, and w0_out holds the values the grids rounded."""
    W, X = _layer(95, 8, 64, 256, scale_sigma=1.0)
    H, G, a = R.hessian_terms(X, 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    qp, w0 = [], np.zeros((8, 64))
    Wh, keep = R.sweep_blocked(W, L, D, fac, 0.5, 32, quant=(4, 16), qparams_out=qp, w0_out=w0)
    Wf, _ = R.sweep_blocked(W, L, D, fac, 0.5, 32, mask_in=keep, quant=(4, 16), values_in=Wh)
    np.testing.assert_array_equal(Wf, Wh)
    for gi, (sc, z, _) in enumerate(qp):
        cols = slice(16 * gi, 16 * gi + 16)
        want = sc[:, None] * (np.clip(np.round(w0[:, cols] / sc[:, None]) + z[:, None], 0, 15) - z[:, None])
        np.testing.assert_array_equal(np.where(keep[:, cols], want, 0.0), Wh[:, cols])


# ---------------------------------------------------------------------------
# Readings that decide discrete outcomes: the (S, column, row) tie order of the
# block mask and round-half-to-even on the quantisation grid.  Both are pinned
# on inputs where the floating-point values are exact, so the tie or the
# halfway case really occurs.
# ---------------------------------------------------------------------------

def _disjoint_channels(k, reps, norms):
    """Token-major X whose channels live on disjoint tokens: X^T X is exactly
    diagonal (every off-diagonal sum is a sum of exact zeros), so the damped
    inverse, its Cholesky factor and the update coefficients L[j', j] are
    exactly diagonal and no column compensates another."""
    X = np.zeros((k * reps, k))
    for c in range(k):
        X[c * reps:(c + 1) * reps, c] = norms[c] / np.sqrt(reps)
    return X


def test_block_tie_order_column_before_row():
    """Caption of Alg. 1 / mask line: equal scores are pruned lowest column
    first, then lowest row (reading R-mask).  With S[0, 1] == S[1, 0] and one
    weight to prune, (row 1, column 0) goes; row-major order would prune
    (row 0, column 1)."""
    S = np.array([[5.0, 1.0], [1.0, 5.0]])
    keep = R.select_block_mask(S, 1)
    np.testing.assert_array_equal(keep, [[True, True], [False, True]])
    # three-way tie spread over rows and columns: columns first, rows within
    # (column 0, row 2) and (column 1, row 0) go; row-major order would take
    # (row 0, column 1) and (row 1, column 1)
    S = np.array([[9.0, 2.0, 9.0], [9.0, 2.0, 9.0], [2.0, 9.0, 9.0]])
    np.testing.assert_array_equal(~R.select_block_mask(S, 2), [[False, True, False], [False, False, False],
                                                                [True, False, False]])
    # magnitude pruning orders |w| the same way
    _, keep_m = R.magnitude_layer(np.array([[1.0, -0.5], [0.5, 1.0]]), 0.25, B=2)
    np.testing.assert_array_equal(keep_m, [[True, True], [False, True]])


def test_block_tie_order_inside_the_sweep():
    """The same tie decided by the whole layer: channels with equal norms on
    disjoint tokens give equal score factors, so |W[0, 1]| == |W[1, 0]| is an
    exact tie in S; the sweep prunes (row 1, column 0)."""
    X = _disjoint_channels(2, 4, [2.0, 2.0])
    W = np.array([[1.0, 0.5], [0.5, 1.0]])
    scores = []
    out = R.prune_layer(W, X, 0.0, 0.25, damp=0.01, B=2, scores_out=scores)
    assert scores[0][0, 1] == scores[0][1, 0]
    np.testing.assert_array_equal(out["keep"], [[True, True], [False, True]])
    np.testing.assert_array_equal(out["W_hat"], [[1.0, 0.5], [0.0, 1.0]])


def test_quant_rounds_half_to_even():
    """Kept weights take the nearest grid value, halfway cases to the even
    integer code (Table 4's RTN; reading R20).  2 bits over [-1, 2]: step 1,
    zero code 1.  x/s = 0.5 -> 0, 1.5 -> 2, -0.5 -> 0, 2.5 -> 2 (clamped code
    3 either way), exactly on the grid otherwise."""
    x = np.array([-1.0, 2.0, 0.5, 1.5, -0.5, 0.25])
    s, z = R.quant_grid(x, 2)
    assert (s, z) == (1.0, 1.0)
    np.testing.assert_array_equal(R.quantize(x, s, z, 2), [-1.0, 2.0, 0.0, 2.0, 0.0, 0.0])
    np.testing.assert_array_equal(R.quantize(np.array([2.5, -2.5, 4.5]), 1.0, 3.0, 3),
                                  [2.0, -2.0, 4.0])


def test_quant_half_to_even_inside_the_sweep():
    """Same halfway cases decided by the sweep (the value a kept weight takes,
    not the stand-alone grid helper): exactly diagonal H, no activation or
    weight sparsity, so every column keeps RTN of its dense value."""
    k = 8
    X = _disjoint_channels(k, 2, np.arange(1.0, k + 1.0))
    W = np.array([[-1.0, 2.0, 0.5, 1.5, -0.5, 0.25, 1.0, -0.75],
                  [0.5, -1.5, 2.5, 3.5, -2.5, 0.0, 4.0, -3.0]])
    out = R.prune_layer(W, X, 0.0, 0.0, damp=0.01, B=8, quant=(2, 8))
    # row 0: grid [-1, 2], step 1, zero 1.  row 1: grid [-3, 4], step 7/3,
    # zero 1 (rint(3 / (7/3)) = rint(1.2857)).
    assert out["keep"].all()
    np.testing.assert_array_equal(out["W_hat"][0], [-1.0, 2.0, 0.0, 2.0, 0.0, 0.0, 1.0, -1.0])
    s1 = 7.0 / 3.0
    want1 = s1 * (np.clip(np.round(W[1] / s1) + 1.0, 0, 3) - 1.0)
    np.testing.assert_array_equal(out["W_hat"][1], want1)
