"""The Y form of the sweep is Algorithm 1's sweep with its residual term
carried differently (float64, CPU).

With V the values the columns have when they are processed and D = U L^T
(U strictly upper), the residual terms owed to column c sum to
(V D)_c = sum_{i <= c} L_ci y_i, y = V U, where y_i depends only on the
columns before i.  The sweep can therefore carry Y (the earlier blocks' part
of y) instead of forming D: a column before its block starts holds
W_c + sum_{i < block} (y_i - e_i) L_ci; at the block's start
W[:, blk] += Y[:, blk] L[blk, blk]^T; inside the block
w_c += (y_J - e_J) L_cJ and y_c += v_J U_Jc after column J, with
v_J = w_J + y_J L_JJ; the lazy products are W += (Y - E) L^T and Y += V U.
N:4 groups are chosen from the columns' current values, which in this form
are w_c + sum_{i=J..c} L_ci y_i for the group's columns c = J .. J + 3 (the y
terms the column would still receive inside the block before it is
processed); a quantisation grid fixed at a block's first column sees W[:, blk]
right after the start product, which already holds Algorithm 1's values.
This file writes that form out with numpy and checks it against the oracle's
blocked sweep (the definition up to rounding): the masks are the same and the
weights agree to rounding.  The HIP path's Y form (duo_prune_layer) is
compared with the oracle in the GPU parity tests.
"""

import numpy as np
import pytest

from oracle import duo_ref as R


def _y_form(W, L, U, fac, p_w, B, S, mask_in=None, start_term=True, nm=None, quant=None, rebuild=True):
    n, k = W.shape
    W = W.copy()
    Y = np.zeros((n, k))
    keep = np.ones((n, k), dtype=bool)
    counts = R.block_prune_counts(n, k, p_w, B)
    pend = []
    for bi, j0 in enumerate(range(0, k, B)):
        j1 = min(k, j0 + B)
        sb0 = j0 // S * S
        sb1 = min(k, sb0 + S)
        if start_term:
            W[:, j0:j1] += Y[:, j0:j1] @ L[j0:j1, j0:j1].T
        Sc = W[:, j0:j1] ** 2 * fac[j0:j1]
        if mask_in is not None:
            keep[:, j0:j1] = mask_in[:, j0:j1]
        elif nm is None:
            keep[:, j0:j1] = R.select_block_mask(Sc, counts[bi])
        if quant is not None:  # one grid per row and block, from the values after the start product
            grids = [R.quant_grid(W[r, j0:j1], quant) for r in range(n)]
            qs = np.array([g[0] for g in grids])
            qz = np.array([g[1] for g in grids])
        w = W[:, j0:j1].copy()
        y = np.zeros_like(w)
        E = np.zeros_like(w)
        V = np.zeros_like(w)
        for j in range(j1 - j0):
            ljj = L[j0 + j, j0 + j]
            if nm is not None and j % 4 == 0 and mask_in is None:
                val = w[:, j:j + 4].copy()
                if rebuild:
                    for c in range(val.shape[1]):
                        for i in range(c + 1):
                            val[:, c] += L[j0 + j + c, j0 + j + i] * y[:, j + i]
                keep[:, j0 + j:j0 + j + 4] = R.select_nm_mask(val ** 2 * fac[j0 + j:j0 + j + 4], nm)
            v = w[:, j] + y[:, j] * ljj
            kept = v if quant is None else R.quantize(v, qs, qz, quant)
            p = np.where(keep[:, j0 + j], kept, 0.0)
            e = (v - p) / ljj
            w[:, j] = p
            w[:, j + 1:] += np.outer(y[:, j] - e, L[j0 + j + 1:j1, j0 + j])
            y[:, j + 1:] += np.outer(v, U[j0 + j, j0 + j + 1:j1])
            E[:, j] = e
            V[:, j] = v
        W[:, j0:j1] = w
        Z = Y[:, j0:j1] + y - E
        W[:, j1:sb1] += Z @ L[j1:sb1, j0:j1].T
        Y[:, j1:sb1] += V @ U[j0:j1, j1:sb1]
        pend.append((j0, j1, Z, V))
        if j1 == sb1:
            if sb1 < k:
                for c0, c1, Zb, Vb in pend:
                    W[:, sb1:] += Zb @ L[sb1:, c0:c1].T
                    Y[:, sb1:] += Vb @ U[c0:c1, sb1:]
            pend = []
    return W * keep, keep


@pytest.mark.parametrize("n,k,B,S,p_w", [(48, 640, 128, 256, 0.6), (30, 200, 48, 96, 0.5), (20, 96, 16, 64, 0.45),
                                         (12, 70, 1, 8, 0.5)])
def test_y_form_equals_blocked_sweep(n, k, B, S, p_w):
    rng = np.random.default_rng(n + k)
    X = rng.standard_normal((4 * k, k)) * rng.uniform(0.2, 2.0, k)
    W = rng.standard_normal((n, k))
    H, G, a = R.hessian_terms(X, 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    U = np.triu(G @ L, 1)
    Wr, keep_r = R.sweep_blocked(W, L, D, fac, p_w, B)
    Wy, keep_y = _y_form(W, L, U, fac, p_w, B, S)
    assert np.array_equal(keep_y, keep_r)
    assert np.linalg.norm(Wy - Wr) <= 1e-12 * np.linalg.norm(Wr)


def test_y_form_needs_the_block_start_term():
    """Without W[:, blk] += Y[:, blk] L[blk, blk]^T (the residual terms of the
    block's own columns owed by the earlier blocks) the result differs: the
    identity is not satisfied trivially."""
    rng = np.random.default_rng(5)
    n, k, B = 16, 256, 64
    X = rng.standard_normal((4 * k, k))
    W = rng.standard_normal((n, k))
    H, G, a = R.hessian_terms(X, 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    U = np.triu(G @ L, 1)
    Wr, keep = R.sweep_blocked(W, L, D, fac, 0.5, B)
    Wy, _ = _y_form(W, L, U, fac, 0.5, B, 128, mask_in=keep)
    assert np.linalg.norm(Wy - Wr) <= 1e-12 * np.linalg.norm(Wr)
    Wbad, _ = _y_form(W, L, U, fac, 0.5, B, 128, mask_in=keep, start_term=False)
    assert np.linalg.norm(Wbad - Wr) > 1e-6 * np.linalg.norm(Wr)


def _terms(n, k, seed):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((4 * k, k)) * rng.uniform(0.2, 2.0, k)
    W = rng.standard_normal((n, k))
    H, G, a = R.hessian_terms(X, 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    return W, L, D, fac, np.triu(G @ L, 1)


@pytest.mark.parametrize("n,k,B,S,N", [(40, 256, 64, 128, 2), (24, 192, 16, 64, 1), (18, 96, 32, 64, 3)])
def test_y_form_nm_equals_blocked_sweep(n, k, B, S, N):
    """N:4 groups chosen from the rebuilt values give the oracle's masks and
    weights; without the y terms in the rebuilt values the masks differ."""
    W, L, D, fac, U = _terms(n, k, 3 * n + k)
    Wr, keep_r = R.sweep_blocked(W, L, D, fac, 0.5, B, nm=(N, 4))
    Wy, keep_y = _y_form(W, L, U, fac, 0.5, B, S, nm=N)
    assert np.array_equal(keep_y, keep_r)
    assert np.linalg.norm(Wy - Wr) <= 1e-12 * np.linalg.norm(Wr)
    _, keep_bad = _y_form(W, L, U, fac, 0.5, B, S, nm=N, rebuild=False)
    assert not np.array_equal(keep_bad, keep_r)


@pytest.mark.parametrize("n,k,B,S,bits", [(32, 256, 64, 128, 4), (20, 160, 32, 64, 3), (16, 96, 16, 32, 8)])
def test_y_form_quant_equals_blocked_sweep(n, k, B, S, bits):
    """Joint quantisation with one grid per row and block: grids fixed after
    the block's start product give the oracle's masks and weights."""
    W, L, D, fac, U = _terms(n, k, 5 * n + k + bits)
    Wr, keep_r = R.sweep_blocked(W, L, D, fac, 0.5, B, quant=(bits, B))
    Wy, keep_y = _y_form(W, L, U, fac, 0.5, B, S, quant=bits)
    assert np.array_equal(keep_y, keep_r)
    assert np.linalg.norm(Wy - Wr) <= 1e-12 * np.linalg.norm(Wr)
