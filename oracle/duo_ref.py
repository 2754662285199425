"""Float64 reference ("oracle") for DuoGPT's layer-wise calibration solver.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke entry point and the
CPU-baseline leg of the benchmark may import this module.  The product path
(the HIP library and its Python binding) never calls it and shares no code with
it.

Everything here is plain numpy in float64, written from the DuoGPT paper
(arXiv 2506.20194) to be checked against the paper by eye:

* activation sparsification, section "Preliminaries / Activation Sparsity";
* the asymmetric objective and its Lagrangian, section 4.2, Eq. 2;
* the single-weight closed form (loss and update), Eq. 3, proof in App. A.1;
* the decomposed score and its a, b, c terms, Eq. 5-7, App. A.2-A.4;
* Algorithm 1 (blocked column sweep with lazy batch updates).

Notation follows the paper: W is n x k (out x in), the paper's calibration
matrix X is k x m.  In memory (and in this module) activations are stored
token-major, m x k, i.e. the transpose of the paper's X.  X_dense is the
paper's X-tilde (dense stream), Xh is X-hat (the sparsified stream) and
dX = X_dense - Xh is the paper's Delta X.

Readings taken where the paper is silent or ambiguous (each is listed in the
design notes of the repository):

R-act   exactly floor(p_x*k + 0.5) activations are zeroed per token, those with
        the smallest (|x|, channel index) key; -0.0 counts as 0.
R-damp  lambda = damp * mean(diag(H)) with H = Xh^T Xh undamped; H + lambda*I
        replaces H everywhere (equivalently, a ridge term lambda*|dw|^2 is
        added to the layer objective).
R-mask  the weight mask of each B-column block is chosen globally over the
        n x B block; the count uses cumulative rounding so that blocks 0..b
        hold floor(p_w*n*(j0+B_b) + 0.5) zeros in total; ties in the score are
        broken by (score, column, row) ascending.
R-lazy  the residual-correction term of the lazy batch update uses the value
        each column had when it was processed (before it was pruned).  This is
        the only reading under which the blocked sweep equals the column-by-
        column (eager) sweep.
R-sign  the residual is R = W (X_dense - Xh); Eq. 4 prints the opposite sign,
        which contradicts Eq. 3 and the update rule of Algorithm 1.
R-order act_order (App. B) processes the channels by decreasing diag(H) of the
        sparse stream, equal values in channel order; off unless asked for
        (Algorithm 1 does not include it).
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "act_zero_count",
    "sparsify_tokens",
    "hessian_terms",
    "hessian_entries",
    "inverse_cholesky",
    "score_terms",
    "window_terms",
    "block_prune_counts",
    "select_block_mask",
    "select_nm_mask",
    "quant_grid",
    "quantize",
    "sweep_eager",
    "sweep_blocked",
    "act_order_perm",
    "prune_layer",
    "objective",
    "sparsegpt_layer",
    "magnitude_layer",
    "obs_closed_form",
    "obs_bruteforce",
]

_TOKEN_CHUNK = 8192


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# Activation sparsification (Preliminaries, "Activation Sparsity")
# ---------------------------------------------------------------------------

def act_zero_count(k: int, p_x: float) -> int:
    """Number of activations zeroed per token (reading R-act)."""
    return int(np.floor(p_x * k + 0.5))


def sparsify_tokens(X, p_x: float):
    """Per-token magnitude sparsification.

    Each token (a column of the paper's X, a row here) keeps all but the
    ``act_zero_count(k, p_x)`` entries of smallest |x|; equal magnitudes are
    ordered by channel index, so the lower channel is zeroed first.

    Returns (Xh, keep) with Xh = X * keep, both m x k.
    """
    X = _f64(X)
    m, k = X.shape
    z = act_zero_count(k, p_x)
    keep = np.ones((m, k), dtype=bool)
    if z > 0:
        for t0 in range(0, m, _TOKEN_CHUNK):
            t1 = min(m, t0 + _TOKEN_CHUNK)
            # stable sort: ascending |x|, equal keys stay in channel order
            order = np.argsort(np.abs(X[t0:t1]), axis=1, kind="stable")
            rows = np.arange(t1 - t0)[:, None]
            keep[t0:t1][rows, order[:, :z]] = False
    return np.where(keep, X, 0.0), keep


# ---------------------------------------------------------------------------
# Hessian and residual terms (Alg. 1 first two lines; Sec. 4.3 "a")
# ---------------------------------------------------------------------------

def hessian_terms(X_src, p_x: float, X_dense=None):
    """H = Xh Xh^T, G = dX Xh^T and a = diag(dX dX^T) in the paper's orientation.

    X_src is the stream that gets sparsified (the pruned model's input); X_dense
    is the dense model's input (defaults to X_src, the single-layer case).
    All inputs are token-major m x k.  Returns (H, G, a) with H, G k x k.
    """
    X_src = _f64(X_src)
    X_dense = X_src if X_dense is None else _f64(X_dense)
    m, k = X_src.shape
    H = np.zeros((k, k))
    G = np.zeros((k, k))
    a = np.zeros(k)
    for t0 in range(0, m, _TOKEN_CHUNK):
        t1 = min(m, t0 + _TOKEN_CHUNK)
        Xh, _ = sparsify_tokens(X_src[t0:t1], p_x)
        dX = X_dense[t0:t1] - Xh
        H += Xh.T @ Xh          # sum_t xh_t^T xh_t
        G += dX.T @ Xh          # G[p, q] = sum_t dX[t, p] * Xh[t, q]
        a += np.sum(dX * dX, axis=0)
    return H, G, a


def _token_keep(X, z: int):
    """Keep-mask of reading R-act for a block of tokens, through selection
    rather than a full sort: the z-th smallest magnitude v of each token is
    found; entries below v are zeroed, and of the entries equal to v the
    lowest-channel ones are zeroed until z entries are gone."""
    m, k = X.shape
    if z <= 0:
        return np.ones((m, k), dtype=bool)
    if z >= k:
        return np.zeros((m, k), dtype=bool)
    mag = np.abs(X)
    v = np.partition(mag, z - 1, axis=1)[:, z - 1:z]
    below = mag < v
    tied = mag == v
    need = z - np.sum(below, axis=1, keepdims=True)      # zeros still to place among the ties
    zero_tied = tied & (np.cumsum(tied, axis=1) <= need)   # channel order
    return ~(below | zero_tied)


def hessian_entries(X_src, p_x: float, idx, X_dense=None, t0: int = 0, t1: int | None = None, rows=None):
    """Selected entries of the stage-1 terms, summed over tokens t0..t1-1.

    Returns dict(H=H[idx][:, idx], G=G[idx][:, idx], a=a (all k), diag=diag(H)
    (all k)) with the same definitions as ``hessian_terms``, for layers whose
    full k x k terms are too large to form in float64; with ``rows`` also
    G_rows = G[rows, :] (whole rows).  Tokens are taken in chunks; results over
    disjoint token ranges add up.
    """
    idx = np.asarray(idx)
    m, k = X_src.shape
    t1 = m if t1 is None else t1
    z = act_zero_count(k, p_x)
    s = len(idx)
    H = np.zeros((s, s))
    G = np.zeros((s, s))
    a = np.zeros(k)
    diag = np.zeros(k)
    G_rows = None if rows is None else np.zeros((len(rows), k))
    for c0 in range(t0, t1, 1024):
        c1 = min(t1, c0 + 1024)
        Xs = _f64(X_src[c0:c1])
        Xd = Xs if X_dense is None else _f64(X_dense[c0:c1])
        Xh = np.where(_token_keep(Xs, z), Xs, 0.0)
        dX = Xd - Xh
        H += Xh[:, idx].T @ Xh[:, idx]
        G += dX[:, idx].T @ Xh[:, idx]
        a += np.sum(dX * dX, axis=0)
        diag += np.sum(Xh * Xh, axis=0)
        if G_rows is not None:
            G_rows += dX[:, rows].T @ Xh
    out = dict(H=H, G=G, a=a, diag=diag)
    if G_rows is not None:
        out["G_rows"] = G_rows
    return out


# ---------------------------------------------------------------------------
# Damped inverse Cholesky (Sec. 4.3, Alg. 1 "Inverse_Cholesky")
# ---------------------------------------------------------------------------

def inverse_cholesky(H, damp: float):
    """L lower-triangular with L L^T = (H + lambda I)^-1, lambda = damp*mean(diag H).

    The plain route: explicit inverse, symmetrised, then a Cholesky
    factorisation.  Returns (L, lambda).
    """
    H = _f64(H)
    k = H.shape[0]
    lam = damp * float(np.mean(np.diag(H)))
    Hl = H + lam * np.eye(k)
    Hinv = np.linalg.inv(Hl)
    Hinv = 0.5 * (Hinv + Hinv.T)
    L = np.linalg.cholesky(Hinv)
    return L, lam


# ---------------------------------------------------------------------------
# Score factor and residual-update matrix (Eq. 7; App. A.2-A.4)
# ---------------------------------------------------------------------------

def score_terms(G, L, a):
    """Precompute of Alg. 1: Q = G L, U = Q * M_u (strictly upper),
    b = diag(U U^T), c = diag(Q) / diag(L), D = U L^T and the per-column score
    factor fac = 1/diag(L)^2 + a - b + 2c (Eq. 7), so that S = W^2 * fac.

    Returns (fac, D, (a, b, c)).
    """
    G = _f64(G)
    L = _f64(L)
    a = _f64(a)
    Q = G @ L
    U = np.triu(Q, 1)
    b = np.sum(U * U, axis=1)
    dL = np.diag(L)
    c = np.diag(Q) / dL
    D = U @ L.T
    fac = 1.0 / dL ** 2 + a - b + 2.0 * c
    return fac, D, (a, b, c)


def window_terms(H_win, G_win, a_win, lam: float):
    """L, fac and D restricted to a trailing window of columns T = [k-t, k).

    Write H + lambda I = V V^T with V = L^-T upper triangular.  Because V is
    upper triangular, the trailing t x t block satisfies
    (H + lambda I)[T, T] = V[T, T] V[T, T]^T, so L[T, T] is the inverse
    Cholesky factor of that block alone.  Q = G L, b, c and D = U L^T restricted
    to T only involve L[T, T] and G[T, T] (L is lower, U strictly upper), so the
    window is self-contained once lambda (from the whole diagonal) is known.
    Returns (L_win, fac_win, D_win).
    """
    H_win = _f64(H_win)
    t = H_win.shape[0]
    Hinv = np.linalg.inv(H_win + lam * np.eye(t))
    L = np.linalg.cholesky(0.5 * (Hinv + Hinv.T))
    fac, D, _ = score_terms(G_win, L, a_win)
    return L, fac, D


# ---------------------------------------------------------------------------
# Weight-mask selection (Alg. 1, mask line; caption: each block p_w sparse)
# ---------------------------------------------------------------------------

def block_prune_counts(n: int, k: int, p_w: float, B: int):
    """Zeros per block under cumulative rounding (reading R-mask)."""
    counts = []
    prev = 0
    for j0 in range(0, k, B):
        j1 = min(k, j0 + B)
        cum = int(np.floor(p_w * n * j1 + 0.5))
        counts.append(cum - prev)
        prev = cum
    return counts


def select_block_mask(S, z: int):
    """Keep-mask of an n x Bb score block with the z lowest scores removed.

    Order: ascending score, then column, then row (reading R-mask).
    """
    S = _f64(S)
    n, Bb = S.shape
    flat = S.T.reshape(-1)                  # index = column * n + row
    order = np.argsort(flat, kind="stable")
    keep = np.ones(n * Bb, dtype=bool)
    keep[order[:z]] = False
    return keep.reshape(Bb, n).T


def select_nm_mask(S, N: int):
    """Keep-mask of an n x M score group with the N lowest scores of every row
    removed, equal scores in column order (the N:M variant of App. B)."""
    S = _f64(S)
    order = np.argsort(S, axis=1, kind="stable")
    keep = np.ones(S.shape, dtype=bool)
    keep[np.arange(S.shape[0])[:, None], order[:, :N]] = False
    return keep


def quant_grid(w, bits: int):
    """Round-to-nearest grid of one row group (Table 4: b-bit uniform integer,
    channel-wise, asymmetric): the range [min(0, min w), max(0, max w)] (or
    [-1, 1] when it is empty) split into 2^b - 1 steps; zero is the integer
    code of 0.  Returns (scale, zero)."""
    w = _f64(w)
    maxq = 2 ** bits - 1
    lo, hi = min(0.0, float(np.min(w))), max(0.0, float(np.max(w)))
    if lo == hi:
        lo, hi = -1.0, 1.0
    scale = (hi - lo) / maxq
    return scale, float(np.round(-lo / scale))


def quantize(x, scale: float, zero: float, bits: int):
    """Value of x on the grid: scale * (clamp(round(x / scale) + zero, 0,
    2^b - 1) - zero), round half to even."""
    q = np.clip(np.round(_f64(x) / scale) + zero, 0, 2 ** bits - 1)
    return scale * (q - zero)


def _check_quant(quant, B: int):
    if quant is None:
        return None
    bits, group = quant
    assert 2 <= bits <= 8 and group >= 1 and B % group == 0, "quantisation groups must divide the block"
    return bits, group


def _check_nm(nm, k: int, B: int):
    if nm is None:
        return None
    N, M = nm
    assert 0 <= N <= M and k % M == 0 and B % M == 0, "N:M needs M | k and M | B"
    return N, M


# ---------------------------------------------------------------------------
# Column sweep: definition (eager) and Algorithm 1 (blocked, lazy batches)
# ---------------------------------------------------------------------------

def _group_grids(Wg, bits: int, qparams_out):
    n = Wg.shape[0]
    qs, qz = np.empty(n), np.empty(n)
    for r in range(n):
        qs[r], qz[r] = quant_grid(Wg[r], bits)
    if qparams_out is not None:
        qparams_out.append((qs.copy(), qz.copy(), _f64(Wg).copy()))
    return qs, qz


def _kept_value(w0, keep_j, quant, qs, qz):
    """The value a processed column keeps: w0 (or its grid value) where kept, 0 where pruned."""
    if quant is None:
        return w0 * keep_j
    q = np.clip(np.round(w0 / qs) + qz, 0, 2 ** quant[0] - 1)
    return np.where(keep_j, qs * (q - qz), 0.0)

def _check_mask_in(mask_in, n, k):
    if mask_in is None:
        return None
    mask_in = np.asarray(mask_in, dtype=bool)
    assert mask_in.shape == (n, k)
    return mask_in


def _sweep(W, L, D, fac, p_w, B, lazy, mask_in, scores_out, nm, quant, qparams_out, values_in, w0_out):
    """The column sweep, in either of its two equivalent forms.

    Processing column j leaves it at the value p it keeps (w0, or its grid
    value, where kept; 0 where pruned), w0 being its value at that moment, and
    records what every later column j' owes it: the compensation of its
    error, e * L[j', j] with e = (w0 - p) / L_jj, minus its residual term
    w0 * D[j, j'] (Eq. 7; App. A.4).
      lazy=False: the debt is paid to every later column at once (the
        definition, column by column);
      lazy=True: it is paid at once only inside the block; the columns after
        the block receive the debts of the whole block together as one product
        E L[rest, blk]^T - W0 D[blk, rest], E and W0 collecting the block's e and
        w0 (Alg. 1, lazy batch updates; reading R-lazy: W0 holds the values
        before pruning).  The two forms give the same result up to rounding.
    The mask of each block is chosen when the sweep reaches the block, from
    S = W[:, blk]^2 * fac[blk] (select_block_mask); with nm = (N, M) it is
    instead chosen per row for each group of M columns when the sweep reaches
    the group (select_nm_mask).  quant = (bits, group): a grid per row and
    group is fixed from the group's current values when the sweep reaches it
    (quant_grid)."""
    W = _f64(W).copy()
    L = _f64(L)
    D = _f64(D)
    fac = _f64(fac)
    n, k = W.shape
    mask_in = _check_mask_in(mask_in, n, k)
    nm = _check_nm(nm, k, B)
    quant = _check_quant(quant, B)
    keep = np.ones((n, k), dtype=bool)
    counts = block_prune_counts(n, k, p_w, B)
    qs = qz = None
    for bi, j0 in enumerate(range(0, k, B)):
        j1 = min(k, j0 + B)
        S = W[:, j0:j1] ** 2 * fac[j0:j1]
        if nm is None:
            keep[:, j0:j1] = select_block_mask(S, counts[bi]) if mask_in is None else mask_in[:, j0:j1]
        elif mask_in is not None:
            keep[:, j0:j1] = mask_in[:, j0:j1]
        E = np.zeros((n, j1 - j0))
        W0 = np.zeros((n, j1 - j0))
        reach = j1 if lazy else k  # columns paid at once
        for j in range(j0, j1):
            if nm is not None and j % nm[1] == 0:
                S[:, j - j0:j - j0 + nm[1]] = W[:, j:j + nm[1]] ** 2 * fac[j:j + nm[1]]
                if mask_in is None:
                    keep[:, j:j + nm[1]] = select_nm_mask(S[:, j - j0:j - j0 + nm[1]], nm[0])
            if quant is not None and j % quant[1] == 0:
                qs, qz = _group_grids(W[:, j:min(j + quant[1], j1)], quant[0], qparams_out)
            w0 = W[:, j].copy()
            p = _kept_value(w0, keep[:, j], quant, qs, qz)
            if values_in is not None:
                p = np.where(keep[:, j], _f64(values_in[:, j]), 0.0)
            if w0_out is not None:
                w0_out[:, j] = w0
            e = (w0 - p) / L[j, j]
            W[:, j] = p
            W[:, j + 1:reach] -= np.outer(e, L[j + 1:reach, j]) - np.outer(w0, D[j, j + 1:reach])
            E[:, j - j0] = e
            W0[:, j - j0] = w0
        if reach < k:
            W[:, reach:] -= E @ L[reach:, j0:j1].T - W0 @ D[j0:j1, reach:]
        if scores_out is not None:
            scores_out.append(S.copy())
    return W * keep, keep


def sweep_eager(W, L, D, fac, p_w: float, B: int, mask_in=None, scores_out=None, nm=None, quant=None,
                qparams_out=None, values_in=None, w0_out=None):
    """Column sweep by definition: every column's update reaches all later
    columns at once (see _sweep).  qparams_out (a list) receives, per
    quantisation group, the (scale, zero) arrays of shape (n,) and the
    n x group values the grids were fixed from.  Test hooks: values_in
    (n x k) replaces the value every kept weight takes (as mask_in replaces
    the mask); w0_out (n x k) receives each column's value when it was
    processed.  Returns (W_hat, keep)."""
    return _sweep(W, L, D, fac, p_w, B, False, mask_in, scores_out, nm, quant, qparams_out, values_in, w0_out)


def sweep_blocked(W, L, D, fac, p_w: float, B: int, mask_in=None, scores_out=None, nm=None, quant=None,
                  qparams_out=None, values_in=None, w0_out=None):
    """Column sweep with the lazy batch update of Algorithm 1 (see _sweep):
    one product per block carries the block's debts to the later columns.
    Arguments as in sweep_eager; scores_out receives, per block, the scores
    each weight's selection used.  Returns (W_hat, keep)."""
    return _sweep(W, L, D, fac, p_w, B, True, mask_in, scores_out, nm, quant, qparams_out, values_in, w0_out)


# ---------------------------------------------------------------------------
# Whole layer, objective and comparators
# ---------------------------------------------------------------------------

def act_order_perm(H):
    """act_order (App. B, calibration settings): the columns are processed in
    the order of decreasing Hessian diagonal, H = Xh^T Xh of the sparse stream
    (reading R-order: largest first, as in the SparseGPT option the paper
    names; equal diagonals keep their channel order).  Returns perm with
    perm[i] = the channel processed i-th."""
    d = np.diag(_f64(H))
    k = d.shape[0]
    return np.lexsort((np.arange(k), -d))


def prune_layer(W, X_src, p_x: float, p_w: float, damp: float = 0.01, B: int = 128,
                X_dense=None, mask_in=None, blocked: bool = True, scores_out=None,
                act_order: bool = False, nm=None, quant=None, qparams_out=None):
    """DuoGPT on one linear layer: Alg. 1 end to end.  Returns a dict.

    act_order=True permutes the channels by act_order_perm(H) before the
    inverse Cholesky: W's columns, H's and G's rows and columns, a and a
    forced mask all follow the permutation; blocks are formed in that order.
    W_hat and keep come back in the original channel order; the returned H,
    G, a are the unpermuted ones, while L, D, fac, b, c and the block scores
    appended to scores_out belong to the permuted problem (perm alongside).

    nm = (N, M): the N:M semi-structured variant (App. B: mask selection and
    pruning over every group of M consecutive columns); p_w is then unused.
    It is not combined with act_order, whose permuted groups would not be
    groups of the layer's own consecutive columns.

    quant = (bits, group): joint pruning and RTN quantisation (Table 4), see
    sweep_eager; with act_order the groups are formed in the permuted order."""
    if act_order and nm is not None:
        raise ValueError("act_order and N:M groups are not combined")
    H, G, a = hessian_terms(X_src, p_x, X_dense)
    W = _f64(W)
    perm = None
    Hs, Gs, As, Ws, Ms = H, G, a, W, _check_mask_in(mask_in, W.shape[0], W.shape[1])
    if act_order:
        perm = act_order_perm(H)
        Hs, Gs, As, Ws = H[np.ix_(perm, perm)], G[np.ix_(perm, perm)], a[perm], W[:, perm]
        if Ms is not None:
            Ms = Ms[:, perm]
    L, lam = inverse_cholesky(Hs, damp)
    fac, D, (_, b, c) = score_terms(Gs, L, As)
    sweep = sweep_blocked if blocked else sweep_eager
    W_hat, keep = sweep(Ws, L, D, fac, p_w, B, mask_in=Ms, scores_out=scores_out, nm=nm, quant=quant,
                        qparams_out=qparams_out)
    if act_order:
        inv = np.argsort(perm)
        W_hat, keep = W_hat[:, inv], keep[:, inv]
    return dict(W_hat=W_hat, keep=keep, H=H, G=G, a=a, b=b, c=c, L=L, lam=lam, fac=fac, D=D, perm=perm)


def objective(W, W_hat, X_src, p_x: float, X_dense=None):
    """Layer objective |W X_dense - W_hat Xh|_F^2 (Sec. 4.2), undamped, f64.

    W_hat may be a list of candidate weights; the objective of each is then
    returned as a list (the tokens are sparsified once).  The sum runs over
    the given tokens, so objectives over disjoint token ranges add up."""
    many = isinstance(W_hat, (list, tuple))
    W = _f64(W)
    W_hats = [_f64(w) for w in (W_hat if many else [W_hat])]
    m = X_src.shape[0]
    totals = [0.0] * len(W_hats)
    for t0 in range(0, m, _TOKEN_CHUNK):
        t1 = min(m, t0 + _TOKEN_CHUNK)
        Xs = _f64(X_src[t0:t1])
        Xd = Xs if X_dense is None else _f64(X_dense[t0:t1])
        Xh, _ = sparsify_tokens(Xs, p_x)
        Y = Xd @ W.T
        for i, Wh in enumerate(W_hats):
            R = Y - Xh @ Wh.T
            totals[i] += float(np.sum(R * R))
    return totals if many else totals[0]


def sparsegpt_layer(W, X_src, p_x: float, p_w: float, damp: float = 0.01, B: int = 128):
    """Comparator: the same sweep on the same sparse Hessian without the
    residual terms (a = b = c = 0, D = 0), i.e. the OBS update of Eq. 1."""
    W = _f64(W)
    H, _, _ = hessian_terms(X_src, p_x)
    L, _ = inverse_cholesky(H, damp)
    k = W.shape[1]
    fac = 1.0 / np.diag(L) ** 2
    W_hat, keep = sweep_blocked(W, L, np.zeros((k, k)), fac, p_w, B)
    return W_hat, keep


def magnitude_layer(W, p_w: float, B: int = 128):
    """Comparator: magnitude pruning with the same per-block counts and tie
    order (|w|, column, row); no weight update."""
    W = _f64(W)
    n, k = W.shape
    keep = np.ones((n, k), dtype=bool)
    for bi, (j0, z) in enumerate(zip(range(0, k, B), block_prune_counts(n, k, p_w, B))):
        j1 = min(k, j0 + B)
        keep[:, j0:j1] = select_block_mask(np.abs(W[:, j0:j1]), z)
    return W * keep, keep


# ---------------------------------------------------------------------------
# Single-weight closed form (Eq. 3) and its brute-force counterpart
# ---------------------------------------------------------------------------

def obs_closed_form(w, Xh, X_dense, lam: float, p: int):
    """Eq. 3 for one row w (length k) and candidate p, with H = Xh^T Xh + lam I.

    r = w (X_dense - Xh) is the row's output residual (a length-m vector here).
    Returns (L_p, dw) with
      L_p = w_p^2/h + r r^T - r Xh^T H^-1_{-p} Xh r^T + (2 w_p / h) r Xh^T H^-1_{:,p}
      dw  = -(w_p / h) H^-1_{p,:} + r Xh^T H^-1_{-p}
    where h = [H^-1]_pp and H^-1_{-p} is the Gaussian-eliminated inverse.
    """
    w = _f64(w)
    Xh = _f64(Xh)
    X_dense = _f64(X_dense)
    k = w.shape[0]
    Hinv = np.linalg.inv(Xh.T @ Xh + lam * np.eye(k))
    h = Hinv[p, p]
    Hm = Hinv - np.outer(Hinv[:, p], Hinv[p, :]) / h
    r = (X_dense - Xh) @ w
    rX = Xh.T @ r
    Lp = w[p] ** 2 / h + r @ r - rX @ Hm @ rX + 2.0 * w[p] / h * (rX @ Hinv[:, p])
    dw = -(w[p] / h) * Hinv[p, :] + rX @ Hm
    return float(Lp), dw


def obs_bruteforce(w, Xh, X_dense, lam: float, p: int, frozen=()):
    """Direct constrained ridge least squares for removing weight p of row w:
    minimise |dw Xh - r|^2 + lam |dw|^2 subject to dw_p = -w_p and dw_f = 0 for
    every frozen index f.  Returns (loss, dw).  No closed form is used."""
    w = _f64(w)
    Xh = _f64(Xh)
    X_dense = _f64(X_dense)
    k = w.shape[0]
    r = (X_dense - Xh) @ w
    free = [j for j in range(k) if j != p and j not in set(frozen)]
    target = r + w[p] * Xh[:, p]            # residual left after dw_p = -w_p
    A = np.vstack([Xh[:, free], np.sqrt(lam) * np.eye(len(free))])
    t = np.concatenate([target, np.zeros(len(free))])
    dw = np.zeros(k)
    dw[p] = -w[p]
    if free:
        v, *_ = np.linalg.lstsq(A, t, rcond=None)
        dw[free] = v
    loss = float(np.sum((Xh @ dw - r) ** 2) + lam * np.sum(dw * dw))
    return loss, dw
