"""Parity of the HIP path (through the C ABI) with the float64 oracle.

Sizes span several 128-wide tiles and end in ragged tails; the oracle
finishes each case in seconds.  Tolerances (derived in the design notes):

* activation masks: bit-exact (integer keys on both sides);
* H, G, a: bf16 products are exact and sums are fp32, so each entry is within
  2e-5 * sqrt(H_ii H_jj) (resp. sqrt(a_p H_qq)) of the f64 value;
* L, D, fac: fp32 factorisation of a matrix with condition number up to ~1e5;
  compared in relative Frobenius norm;
* sweep / whole layer: mask agreement >= 99.9 % with every disagreement at a
  near-tie (|S - T_b| / T_b < 1e-5 in the oracle run forced to the GPU mask),
  W within 1e-3 relative Frobenius, objective within 1e-3 relative.
"""

import numpy as np
import pytest
import torch

from oracle import duo_ref as R
from workloads import synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def duo(duo_lib):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return duo_lib


def say(*a):
    print("[case]", *a, flush=True)


def f64(t):
    return t.detach().cpu().double().numpy()


def relfro(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def inputs(n, k, m, dtype, seed, kind="lognormal", sigma=1.0, outliers=0):
    W, X = synth.layer_inputs(n, k, m, dtype, dtype, seed=seed, device="cpu", kind=kind, sigma=sigma,
                              outliers=outliers)
    return W, X


# ---------------------------------------------------------------------------
# stage 1
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("m,k,p_x", [(300, 200, 0.5), (257, 4096, 0.5), (64, 11008, 0.6), (100, 129, 0.0),
                                     (50, 33, 1.0), (70, 1, 0.5), (40, 8200, 0.5), (33, 12296, 0.3),
                                     (20, 16392, 0.7), (17, 28672, 0.5), (9, 32768, 0.5), (12, 9000, 0.0),
                                     (12, 9000, 1.0)])
def test_act_mask_bit_exact(duo, dtype, m, k, p_x):
    say("act_mask", dtype, m, k, p_x)
    _, X = inputs(1, k, m, dtype, seed=k + m)
    if dtype == torch.bfloat16:  # plant many exact magnitude ties and signed zeros
        X[:, ::3] = X[:, ::3].sign() * 0.5
        X[::7, ::5] = -0.0
    mask = duo.unpack_mask(duo.duo_act_sparsify_mask(X.to(DEV), p_x), k).cpu().numpy()
    _, keep = R.sparsify_tokens(X.float().numpy(), p_x)
    assert np.array_equal(mask, keep)


def _check_gram(H, G, a, Hr, Gr, ar, tol, g_full=False):
    """H and a against the oracle; G on the entries stage 1 accumulates
    without g_full (p / 256 <= q / 256: its upper triangle and the diagonal
    256 x 256 tiles), the rest left as the caller set it (zero), or all of G
    with g_full.  H is returned exactly symmetric (its lower triangle mirrors
    the upper one)."""
    dH = np.sqrt(np.maximum(np.diag(Hr), 0))
    bound_H = tol * np.outer(dH, dH) + 1e-30
    assert np.all(np.abs(H - Hr) <= bound_H), float(np.max(np.abs(H - Hr) / bound_H))
    assert np.array_equal(H, H.T)
    if G is not None:
        bound_G = tol * np.outer(np.sqrt(np.maximum(ar, 0)), dH) + 1e-30
        tb = np.arange(G.shape[0]) // 256
        part = np.ones_like(G, dtype=bool) if g_full else tb[:, None] <= tb[None, :]
        err = np.where(part, np.abs(G - Gr), 0.0)
        assert np.all(err <= bound_G), float(np.max(err / bound_G))
        assert np.all(G[~part] == 0.0)
        assert np.all(np.abs(a - ar) <= tol * ar + 1e-30)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("m,k", [(1000, 300), (4096, 512), (2500, 640), (33, 130), (600, 1800)])
@pytest.mark.parametrize("g_full", [False, True])
def test_hessian_terms(duo, dtype, m, k, g_full):
    say("hessian", dtype, m, k, g_full)
    _, X = inputs(1, k, m, dtype, seed=3 * k + m, outliers=2)
    Xd = X.to(DEV)
    H = torch.zeros((k, k), device=DEV)
    G = torch.zeros((k, k), device=DEV)
    a = torch.zeros(k, device=DEV)
    duo.duo_hessian_accum(Xd, H, 0.5, G=G, a=a, g_full=g_full)
    torch.cuda.synchronize()
    Hr, Gr, ar = R.hessian_terms(X.float().numpy(), 0.5)
    _check_gram(f64(H), f64(G), f64(a), Hr, Gr, ar, 2e-5, g_full)


def test_hessian_accumulates_over_chunks(duo):
    say("hessian chunks")
    k, m = 384, 3000
    _, X = inputs(1, k, m, torch.bfloat16, seed=5)
    Xd = X.to(DEV)
    H = torch.zeros((k, k), device=DEV)
    G = torch.zeros((k, k), device=DEV)
    a = torch.zeros(k, device=DEV)
    for t0 in range(0, m, 1000):
        duo.duo_hessian_accum(Xd[t0:t0 + 1000], H, 0.5, G=G, a=a)
    Hr, Gr, ar = R.hessian_terms(X.float().numpy(), 0.5)
    _check_gram(f64(H), f64(G), f64(a), Hr, Gr, ar, 2e-5)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_two_stream_residual(duo, dtype):
    """Multi-layer case: the sparsified stream differs from the dense one."""
    say("two-stream", dtype)
    k, m = 260, 1500
    _, Xd_ = inputs(1, k, m, torch.float32, seed=11)
    Xs_ = (Xd_ + 0.3 * torch.randn(Xd_.shape, generator=torch.Generator().manual_seed(1))).to(dtype)
    Xd_ = Xd_.to(dtype)
    H = torch.zeros((k, k), device=DEV)
    G = torch.zeros((k, k), device=DEV)
    a = torch.zeros(k, device=DEV)
    duo.duo_hessian_accum(Xs_.to(DEV), H, 0.5, X_dense=Xd_.to(DEV), G=G, a=a, g_full=True)
    Hr, Gr, ar = R.hessian_terms(Xs_.float().numpy(), 0.5, Xd_.float().numpy())
    _check_gram(f64(H), f64(G), f64(a), Hr, Gr, ar, 2e-5 if dtype == torch.float32 else 6e-5, g_full=True)
    # the residual-only entry point gives the same G and a, in either form
    for g_full in (True, False):
        G2 = torch.zeros((k, k), device=DEV)
        a2 = torch.zeros(k, device=DEV)
        duo.duo_residual_term(Xd_.to(DEV), G2, a2, 0.5, X_src=Xs_.to(DEV), g_full=g_full)
        assert torch.equal(a2, a)
        tb = torch.arange(k, device=DEV) // 256
        assert torch.equal(G2, G if g_full else torch.where(tb[:, None] <= tb[None, :], G, 0.0))


# ---------------------------------------------------------------------------
# stage 2 and the precompute
# ---------------------------------------------------------------------------

def _oracle_stage(k, m, seed, p_x=0.5, damp=0.01, dtype=torch.bfloat16):
    _, X = inputs(1, k, m, dtype, seed=seed, outliers=2)
    H, G, a = R.hessian_terms(X.float().numpy(), p_x)
    return X, H, G, a


# 576 and 1344: the 64-tile products with 128-grid tiles half outside the
# matrix, a ragged last group of diagonal blocks and a merge level with a tail
# node; 2048: merges over several column tiles of the 128 grid
@pytest.mark.parametrize("k", [1, 100, 128, 300, 512, 576, 1000, 1344, 2048])
def test_chol_inv(duo, k):
    say("chol_inv", k)
    # k = 1 with p_x = 0.5 drops the only channel (H = 0): use dense input there
    _, H, _, _ = _oracle_stage(k, 4 * k + 64, seed=k, p_x=0.0 if k == 1 else 0.5)
    Hd = torch.tensor(H, dtype=torch.float32, device=DEV)
    lam, fail = duo.duo_chol_inv(Hd, 0.01)
    L = f64(Hd)
    Lr, lamr = R.inverse_cholesky(H.astype(np.float32).astype(np.float64), 0.01)
    assert fail == -1
    assert abs(lam - lamr) <= 1e-6 * lamr
    assert np.all(np.triu(L, 1) == 0.0)
    assert np.all(np.diag(L) > 0)
    assert relfro(L, Lr) < 2e-4, relfro(L, Lr)
    # the defining property, in f64 on the GPU's factor
    Hl = H + lamr * np.eye(k)
    E = L.T @ Hl @ L - np.eye(k)
    assert np.max(np.abs(E)) < 2e-3


def test_chol_inv_reports_not_pd(duo):
    say("chol_inv not pd")
    k = 200
    _, H, _, _ = _oracle_stage(k, 600, seed=1)
    H[:, 17] = 0.0
    H[17, :] = 0.0           # a dead channel; without damping H is singular
    Hd = torch.tensor(H, dtype=torch.float32, device=DEV)
    with pytest.raises(duo.DuoError) as e:
        duo.duo_chol_inv(Hd, 0.0)
    assert e.value.status == duo.DUO_ERR_NOT_PD
    # with damping the same matrix factors
    Hd = torch.tensor(H, dtype=torch.float32, device=DEV)
    lam, fail = duo.duo_chol_inv(Hd, 0.01)
    assert fail == -1 and lam > 0
    Hz = torch.zeros((64, 64), device=DEV)
    with pytest.raises(duo.DuoError) as e:
        duo.duo_chol_inv(Hz, 0.01)
    assert e.value.status == duo.DUO_ERR_NOT_PD


@pytest.mark.parametrize("k", [64, 300, 512, 576, 700, 1344])
def test_score_terms(duo, k):
    say("score_terms", k)
    _, H, G, a = _oracle_stage(k, 4 * k, seed=2 * k)
    L, _ = R.inverse_cholesky(H, 0.01)
    L32, G32, a32 = (x.astype(np.float32) for x in (L, G, a))
    fac_r, D_r, _ = R.score_terms(G32.astype(np.float64), L32.astype(np.float64), a32.astype(np.float64))
    D, fac = duo.duo_score_terms(torch.tensor(L32, device=DEV), torch.tensor(G32, device=DEV),
                                 torch.tensor(a32, device=DEV))
    D = f64(D)
    assert relfro(f64(fac), fac_r) < 1e-5
    assert relfro(np.triu(D, 1), D_r) < 1e-4, relfro(np.triu(D, 1), D_r)


# ---------------------------------------------------------------------------
# sweep
# ---------------------------------------------------------------------------

def _sweep_inputs(n, k, m, seed, dtype=torch.bfloat16):
    W, X = inputs(n, k, m, dtype, seed=seed, outliers=2)
    H, G, a = R.hessian_terms(X.float().numpy(), 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    L32, D32, f32 = (np.ascontiguousarray(x.astype(np.float32)) for x in (L, D, fac))
    return W, X, L32, D32, f32


def _mask_words(keep):
    n, k = keep.shape
    words = (k + 31) // 32
    pad = np.zeros((n, words * 32), dtype=np.uint64)
    pad[:, :k] = keep
    w = (pad.reshape(n, words, 32) << np.arange(32, dtype=np.uint64)).sum(-1)
    return torch.tensor(w.astype(np.uint32).view(np.int32))


@pytest.mark.parametrize("n,k,B", [(100, 300, 128), (64, 256, 64), (37, 200, 48), (16, 64, 1), (300, 130, 128)])
def test_sweep_forced_mask(duo, n, k, B):
    say("sweep forced", n, k, B)
    W, X, L, D, fac = _sweep_inputs(n, k, 3 * k, seed=n + k)
    Wr, keep = R.sweep_blocked(W.float().numpy(), L, D, fac, 0.5, B)
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, _ = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), 0.5, B, mask_in=_mask_words(keep).to(DEV))
    assert np.array_equal(duo.unpack_mask(mask, k).cpu().numpy(), keep)
    assert relfro(f64(W_out), Wr) < 1e-5, relfro(f64(W_out), Wr)
    assert np.all(f64(W_out)[~keep] == 0.0)


def _attribute(W, L, D, fac, p_w, B, gpu_keep, tol=1e-5):
    """Oracle run forced to the GPU mask; every block's GPU selection must be a
    valid lowest-z selection up to relative near-ties `tol`."""
    scores = []
    R.sweep_blocked(W, L, D, fac, p_w, B, mask_in=gpu_keep, scores_out=scores)
    n, k = W.shape
    counts = R.block_prune_counts(n, k, p_w, B)
    for bi, j0 in enumerate(range(0, k, B)):
        S = scores[bi]
        kb = gpu_keep[:, j0:j0 + B]
        assert (~kb).sum() == counts[bi]
        if kb.all() or (~kb).all():
            continue
        T = np.sort(S.T.reshape(-1), kind="stable")[counts[bi] - 1]
        assert S[~kb].max() <= T * (1 + tol) + 1e-300
        assert S[kb].min() >= T * (1 - tol) - 1e-300


@pytest.mark.parametrize("n,k,B,p_w", [(128, 512, 128, 0.5), (200, 300, 64, 0.6), (33, 129, 128, 0.37),
                                       (64, 256, 32, 0.0), (20, 64, 16, 1.0)])
def test_sweep_select(duo, n, k, B, p_w):
    say("sweep select", n, k, B, p_w)
    W, X, L, D, fac = _sweep_inputs(n, k, 3 * k, seed=7 * n + k)
    Wr, keep_r = R.sweep_blocked(W.float().numpy(), L, D, fac, p_w, B)
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, _ = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), p_w, B)
    keep = duo.unpack_mask(mask, k).cpu().numpy()
    assert (~keep).sum() == (~keep_r).sum()
    assert np.mean(keep == keep_r) >= 0.999
    _attribute(W.float().numpy(), L, D, fac, p_w, B, keep)
    if np.array_equal(keep, keep_r):
        assert relfro(f64(W_out), Wr) < 1e-5


@pytest.mark.parametrize("n,k,B,p_w", [(200, 336, 128, 0.5), (300, 1152, 128, 0.55), (150, 640, 64, 0.5),
                                       (90, 544, 16, 0.45), (4200, 256, 128, 0.5), (8200, 128, 128, 0.6),
                                       (50, 160, 32, 0.0), (40, 96, 16, 1.0),
                                       # n, k multiples of 64 but not of 128: the trailing
                                       # products on 64 tiles with 128-grid tiles half outside
                                       (192, 576, 128, 0.5), (320, 1728, 64, 0.5),
                                       # three 1024-column super-blocks, the last one ragged
                                       (64, 2304, 128, 0.5), (40, 2200, 16, 0.45)])
def test_sweep_select_shapes(duo, n, k, B, p_w):
    """Rows and the last block ragged, several 1024-column super-blocks, 8 and
    64 blocks per super-block, row counts of several selection workgroups'
    batches, and no or every weight pruned."""
    say("sweep select shapes", n, k, B, p_w)
    W, X, L, D, fac = _sweep_inputs(n, k, 3 * k, seed=5 * n + k)
    Wr, keep_r = R.sweep_blocked(W.float().numpy(), L, D, fac, p_w, B)
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, _ = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), p_w, B)
    keep = duo.unpack_mask(mask, k).cpu().numpy()
    assert np.isfinite(f64(W_out)).all()
    assert (~keep).sum() == (~keep_r).sum()
    assert np.mean(keep == keep_r) >= 0.999
    _attribute(W.float().numpy(), L, D, fac, p_w, B, keep)
    if np.array_equal(keep, keep_r):
        assert relfro(f64(W_out), Wr) < 1e-5, relfro(f64(W_out), Wr)


def test_sweep_ties_large_bucket(duo):
    """A bucket of equal scores larger than the gathered-candidate capacity
    (the threshold is then resolved from the block itself); ties broken by
    (column, row)."""
    say("sweep ties, large bucket")
    n, k, B = 1024, 256, 128
    W = torch.ones((n, k), dtype=torch.float32)
    W[::3] = 2.0
    L = np.eye(k, dtype=np.float32)
    D = np.zeros((k, k), dtype=np.float32)
    fac = np.ones(k, dtype=np.float32)
    Wr, keep_r = R.sweep_blocked(W.numpy(), L, D, fac, 0.5, B)
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, _ = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), 0.5, B)
    assert np.array_equal(duo.unpack_mask(mask, k).cpu().numpy(), keep_r)
    assert np.array_equal(f64(W_out), Wr)


def test_sweep_ties(duo):
    """Many exactly equal scores: ties are broken by (column, row)."""
    say("sweep ties")
    n, k, B = 40, 96, 32
    W = torch.ones((n, k), dtype=torch.float32)
    W[::3] = 2.0
    L = np.eye(k, dtype=np.float32)
    D = np.zeros((k, k), dtype=np.float32)
    fac = np.ones(k, dtype=np.float32)
    Wr, keep_r = R.sweep_blocked(W.numpy(), L, D, fac, 0.5, B)
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, _ = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), 0.5, B)
    assert np.array_equal(duo.unpack_mask(mask, k).cpu().numpy(), keep_r)
    assert np.array_equal(f64(W_out), Wr)


# ---------------------------------------------------------------------------
# stage 3 through duo_prune_layer in both residual forms (D formed, or the
# sweep carrying Y = W0 U instead)
# ---------------------------------------------------------------------------

def _layer_terms(n, k, m, seed):
    W, X = inputs(n, k, m, torch.bfloat16, seed=seed, outliers=2)
    H, G, a = R.hessian_terms(X.float().numpy(), 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    L32, G32, a32 = (np.ascontiguousarray(x.astype(np.float32)) for x in (L, G, a))
    fac, D, _ = R.score_terms(G32.astype(np.float64), L32.astype(np.float64), a32.astype(np.float64))
    return W, L32, G32, a32, D, fac


@pytest.mark.parametrize("form", ["d", "y"])
@pytest.mark.parametrize("n,k,B", [(100, 300, 128), (64, 256, 64), (37, 200, 48), (16, 64, 1), (300, 130, 128),
                                   (96, 1152, 128), (80, 1344, 64), (192, 576, 128), (48, 2304, 128),
                                   (40, 2200, 32)])
def test_prune_layer_forced_mask_forms(duo, n, k, B, form):
    say("prune_layer forced", n, k, B, form)
    W, L, G, a, D, fac = _layer_terms(n, k, 3 * k, seed=n + 3 * k)
    Wf = W.float().numpy()
    _, keep = R.sweep_blocked(Wf, L, D, fac, 0.5, B)
    Wr, _ = R.sweep_blocked(Wf, L, D, fac, 0.5, B, mask_in=keep)
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, _ = duo.duo_prune_layer(W.to(DEV), t(L), t(G), t(a), 0.5, B, mask_in=_mask_words(keep).to(DEV),
                                            form=form)
    assert np.array_equal(duo.unpack_mask(mask, k).cpu().numpy(), keep)
    assert relfro(f64(W_out), Wr) < 1e-5, relfro(f64(W_out), Wr)
    assert np.all(f64(W_out)[~keep] == 0.0)


@pytest.mark.parametrize("form", ["d", "y"])
@pytest.mark.parametrize("n,k,B,p_w", [(200, 336, 128, 0.5), (300, 1152, 128, 0.55), (150, 640, 64, 0.5),
                                       (90, 544, 16, 0.45), (4200, 256, 128, 0.5), (50, 160, 32, 0.0),
                                       (40, 96, 16, 1.0), (320, 1728, 64, 0.5), (64, 2304, 128, 0.5),
                                       (40, 2200, 16, 0.45)])
def test_prune_layer_select_forms(duo, n, k, B, p_w, form):
    """Whole stage 3 (Q, fac, selection, sweep) against the oracle's sweep on
    the same L, G, a; several super-blocks, ragged rows and blocks."""
    say("prune_layer select", n, k, B, p_w, form)
    W, L, G, a, D, fac = _layer_terms(n, k, 3 * k, seed=11 * n + k)
    Wf = W.float().numpy()
    Wr, keep_r = R.sweep_blocked(Wf, L, D, fac, p_w, B)
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, _ = duo.duo_prune_layer(W.to(DEV), t(L), t(G), t(a), p_w, B, form=form)
    keep = duo.unpack_mask(mask, k).cpu().numpy()
    assert np.isfinite(f64(W_out)).all()
    assert (~keep).sum() == (~keep_r).sum()
    assert np.mean(keep == keep_r) >= 0.999
    _attribute(Wf, L, D, fac, p_w, B, keep)
    if np.array_equal(keep, keep_r):
        assert relfro(f64(W_out), Wr) < 1e-5, relfro(f64(W_out), Wr)


@pytest.mark.parametrize("n,k,B", [(200, 1152, 128), (75, 1000, 64)])
def test_prune_layer_forms_scores_and_lowp(duo, n, k, B):
    """The block scores the selection used (S = W^2 fac of the values when a
    block starts: in the Y form after its start product) and the bf16 copy, in
    both forms, against the oracle run forced to the GPU's mask; ragged n and
    k (the dual lazy launch splits into two launches off the fast path)."""
    say("prune_layer forms: scores, bf16 copy", n, k, B)
    W, L, G, a, D, fac = _layer_terms(n, k, 3 * k, seed=n * k + 5)
    Wf = W.float().numpy()
    t = lambda x: torch.tensor(x, device=DEV)
    for form in ("d", "y"):
        W_out, lowp, mask, sc = duo.duo_prune_layer(W.to(DEV), t(L), t(G), t(a), 0.5, B, want_lowp=True,
                                                    want_scores=True, form=form)
        keep = duo.unpack_mask(mask, k).cpu().numpy()
        scores = []
        Wr, _ = R.sweep_blocked(Wf, L, D, fac, 0.5, B, mask_in=keep, scores_out=scores)
        S_ref = np.concatenate(scores, axis=1)
        assert relfro(f64(sc), S_ref) < 1e-5, (form, relfro(f64(sc), S_ref))
        assert relfro(f64(W_out), Wr) < 1e-5, (form, relfro(f64(W_out), Wr))
        assert torch.equal(lowp.cpu(), W_out.cpu().to(torch.bfloat16))
        _attribute(Wf, L, D, fac, 0.5, B, keep)


def test_prune_layer_forms_agree(duo):
    """The two forms on one layer: the same mask and weights within fp32
    rounding (k = 2048, 2 super-blocks of 1024)."""
    say("prune_layer forms agree")
    n, k, B = 256, 2048, 128
    W, L, G, a, D, fac = _layer_terms(n, k, 3 * k, seed=77)
    t = lambda x: torch.tensor(x, device=DEV)
    Wd, _, md, _ = duo.duo_prune_layer(W.to(DEV), t(L), t(G), t(a), 0.6, B, form="d")
    Wy, _, my, _ = duo.duo_prune_layer(W.to(DEV), t(L), t(G), t(a), 0.6, B, form="y")
    kd, ky = (duo.unpack_mask(x, k).cpu().numpy() for x in (md, my))
    assert np.mean(kd == ky) >= 0.999
    if np.array_equal(kd, ky):
        assert relfro(f64(Wy), f64(Wd)) < 1e-5


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------

def _layer_case(duo, W, X, p_x, p_w, B, damp=0.01, form=None):
    out = duo.prune_linear(W.to(DEV), X.to(DEV), p_x, p_w, damp=damp, block=B, form=form)
    torch.cuda.synchronize()
    ref = R.prune_layer(W.float().numpy(), X.float().numpy(), p_x, p_w, damp=damp, B=B)
    keep = out["mask"].cpu().numpy()
    Wg = f64(out["W_out"])
    agree = float(np.mean(keep == ref["keep"]))
    J_g = R.objective(W.float().numpy(), Wg, X.float().numpy(), p_x)
    J_r = R.objective(W.float().numpy(), ref["W_hat"], X.float().numpy(), p_x)
    return out, ref, keep, Wg, agree, J_g, J_r


def test_layer_tiny_linear_config(duo):
    """The 256 x 512 fp32 layer with 2048 tokens (the smallest benchmark config)."""
    c = synth.CONFIGS["tiny_linear"]
    say("layer tiny_linear")
    W, X = synth.config_inputs("tiny_linear")
    out, ref, keep, Wg, agree, J_g, J_r = _layer_case(duo, W, X, c["p_x"], c["p_w"], c["block"], c["damp"])
    assert (~keep).sum() == (~ref["keep"]).sum() == int(np.floor(c["p_w"] * c["n"] * c["k"] + 0.5))
    assert agree >= 0.999, agree
    assert relfro(Wg, ref["W_hat"]) < 1e-3
    assert abs(J_g - J_r) <= 1e-3 * J_r
    assert abs(out["lam"] - ref["lam"]) <= 1e-5 * ref["lam"]


@pytest.mark.parametrize("form", [None, "y"])
@pytest.mark.parametrize("n,k,m,B", [(192, 384, 1536, 128), (100, 200, 700, 64)])
def test_layer_bf16(duo, n, k, m, B, form):
    say("layer bf16", n, k, m, B, form)
    W, X = inputs(n, k, m, torch.bfloat16, seed=n * k, outliers=3)
    out, ref, keep, Wg, agree, J_g, J_r = _layer_case(duo, W, X, 0.5, 0.5, B, form=form)
    assert agree >= 0.999, agree
    assert relfro(Wg, ref["W_hat"]) < 1e-3
    assert abs(J_g - J_r) <= 1e-3 * J_r
    # bf16 copy is the round-to-nearest-even of the fp32 result
    assert torch.equal(out["W_lowp"].cpu(), out["W_out"].cpu().to(torch.bfloat16))
    Wm, _ = R.magnitude_layer(W.float().numpy(), 0.5, B)
    assert J_g < R.objective(W.float().numpy(), Wm, X.float().numpy(), 0.5)


@pytest.mark.parametrize("form", [None, "y"])
def test_zero_sparsity_returns_weights_unchanged(duo, form):
    say("zero sparsity", form)
    W, X = inputs(64, 256, 800, torch.bfloat16, seed=3)
    out = duo.prune_linear(W.to(DEV), X.to(DEV), 0.0, 0.0, block=64, form=form)
    assert torch.equal(out["W_out"].cpu(), W.float())
    assert out["mask"].all()


def test_deterministic(duo):
    say("determinism")
    W, X = inputs(96, 320, 900, torch.bfloat16, seed=4)
    a = duo.prune_linear(W.to(DEV), X.to(DEV), 0.5, 0.5, block=64)
    b = duo.prune_linear(W.to(DEV), X.to(DEV), 0.5, 0.5, block=64)
    assert torch.equal(a["W_out"], b["W_out"]) and torch.equal(a["mask"], b["mask"])


@pytest.mark.parametrize("k,dtype", [(96, torch.float32), (4096, torch.bfloat16), (11008, torch.bfloat16),
                                     (300, torch.bfloat16)])
def test_nonfinite_input_is_reported(duo, k, dtype):
    """Stage 1 flags NaN and inf calibration inputs (DUO_ERR_NONFINITE from
    the status check) and not finite ones, for the sparse and the dense
    stream; the largest finite bf16 magnitude is not flagged."""
    say("non-finite input", k, dtype)
    m = 40
    _, X = inputs(1, k, m, dtype, seed=k)
    X = X.to(DEV)
    H = torch.zeros((k, k), dtype=torch.float32, device=DEV)
    G = torch.zeros_like(H)
    a = torch.zeros(k, dtype=torch.float32, device=DEV)
    ws = duo.workspace(duo.DUO_OP_HESSIAN, 0, k, m, 0, DEV)
    big = X.clone()
    big[3, 5] = torch.finfo(dtype).max
    duo.duo_hessian_accum(big, H, 0.5, G=G, a=a, ws=ws, check=True)      # finite: no error
    for val, where in ((float("nan"), "src"), (float("inf"), "src"), (float("-inf"), "dense")):
        bad = X.clone()
        bad[m - 1, k - 1] = val
        H.zero_(), G.zero_(), a.zero_()
        with pytest.raises(duo.DuoError) as e:
            if where == "src":
                duo.duo_hessian_accum(bad, H, 0.5, G=G, a=a, ws=ws, check=True)
            else:
                duo.duo_hessian_accum(X, H, 0.5, X_dense=bad, G=G, a=a, ws=ws, check=True)
        assert e.value.status == duo.DUO_ERR_NONFINITE
        # the flag belongs to the last call: a clean call clears it
        duo.duo_hessian_accum(X, H, 0.5, G=G, a=a, ws=ws, check=True)
    # the activation-mask hook records it too
    bad = X.clone()
    bad[0, 0] = float("nan")
    duo.duo_act_sparsify_mask(bad, 0.5, ws=ws)
    assert duo.lib().duo_hessian_status(duo._ptr(ws), ws.numel(), duo._stream(DEV)) == duo.DUO_ERR_NONFINITE
