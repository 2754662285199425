"""N:4 semi-structured variant (App. B: mask selection and pruning over every
group of 4 consecutive columns) on the HIP path against the oracle.

Bars: exact per-row, per-group counts; the GPU's selection valid against the
scores it reports (the N lowest of every group, equal scores in column order:
integer decisions taken on the kernel's own fp32 scores, compared exactly);
agreement with the oracle's mask >= 99.9 %, each disagreement a near-tie in the
oracle run forced to the GPU mask (relative gap < 1e-5); W within 1e-5
relative Frobenius when the masks agree (sweep alone) and 1e-3 for the whole
layer, objective within 1e-3.
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


def _stage(n, k, m, seed):
    W, X = synth.layer_inputs(n, k, m, torch.bfloat16, torch.bfloat16, seed=seed, device="cpu", sigma=1.0,
                              outliers=2)
    H, G, a = R.hessian_terms(X.float().numpy(), 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    L32, D32, f32 = (np.ascontiguousarray(x.astype(np.float32)) for x in (L, D, fac))
    return W, X, L32, D32, f32


def _groups_valid(keep, S, N):
    """Every group's pruned entries are its N lowest scores, ties by column."""
    n, k = keep.shape
    for g in range(0, k, 4):
        assert np.array_equal(keep[:, g:g + 4], R.select_nm_mask(S[:, g:g + 4], N))


def _near_ties(W, L, D, fac, B, N, gpu_keep, tol=1e-5):
    """Oracle forced to the GPU mask: each group of the GPU mask is a valid
    N-lowest choice of the oracle's scores up to relative near-ties."""
    scores = []
    R.sweep_blocked(W, L, D, fac, 0.5, B, mask_in=gpu_keep, scores_out=scores, nm=(N, 4))
    S = np.concatenate(scores, axis=1)
    n, k = gpu_keep.shape
    for g in range(0, k, 4):
        kb, Sg = gpu_keep[:, g:g + 4], S[:, g:g + 4]
        ref = R.select_nm_mask(Sg, N)
        for r in np.nonzero(np.any(kb != ref, axis=1))[0]:
            T = np.sort(Sg[r])[N - 1] if N > 0 else 0.0
            assert Sg[r][~kb[r]].max() <= T * (1 + tol) + 1e-300
            assert Sg[r][kb[r]].min() >= T * (1 - tol) - 1e-300


@pytest.mark.parametrize("n,k,B,N", [(128, 512, 128, 2), (200, 300, 64, 2), (33, 132, 128, 1), (64, 256, 32, 3),
                                     (20, 64, 16, 4), (40, 96, 8, 2)])
def test_sweep_nm(duo, n, k, B, N):
    say("sweep nm", n, k, B, N)
    W, X, L, D, fac = _stage(n, k, 3 * k, seed=11 * n + k)
    Wn = W.float().numpy()
    Wr, keep_r = R.sweep_blocked(Wn, L, D, fac, 0.5, B, nm=(N, 4))
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, scores = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), 0.5, B, want_scores=True, nm_n=N)
    keep = duo.unpack_mask(mask, k).cpu().numpy()
    assert np.all((~keep).reshape(n, -1, 4).sum(axis=2) == N)
    _groups_valid(keep, f64(scores), N)
    assert np.mean(keep == keep_r) >= 0.999
    _near_ties(Wn, L, D, fac, B, N, keep)
    # the scores each group's selection used, against the oracle forced to the GPU's mask
    S_ref = []
    R.sweep_blocked(Wn, L, D, fac, 0.5, B, mask_in=keep, scores_out=S_ref, nm=(N, 4))
    assert relfro(f64(scores), np.concatenate(S_ref, axis=1)) < 1e-5
    assert np.all(f64(W_out)[~keep] == 0.0)
    if np.array_equal(keep, keep_r):
        assert relfro(f64(W_out), Wr) < 1e-5, relfro(f64(W_out), Wr)


def test_sweep_nm_forced_mask_wins(duo):
    """A forced mask replaces the group selection."""
    say("sweep nm forced")
    n, k, B = 48, 128, 64
    W, X, L, D, fac = _stage(n, k, 3 * k, seed=5)
    keep = np.random.default_rng(0).random((n, k)) < 0.7
    Wr, _ = R.sweep_blocked(W.float().numpy(), L, D, fac, 0.5, B, mask_in=keep)
    words = np.zeros((n, 4), dtype=np.uint64)
    for c in range(k):
        words[:, c // 32] |= keep[:, c].astype(np.uint64) << np.uint64(c % 32)
    t = lambda x: torch.tensor(x, device=DEV)
    mi = torch.tensor(words.astype(np.uint32).view(np.int32)).to(DEV)
    W_out, _, mask, _ = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), 0.5, B, mask_in=mi, nm_n=2)
    assert np.array_equal(duo.unpack_mask(mask, k).cpu().numpy(), keep)
    assert relfro(f64(W_out), Wr) < 1e-5


@pytest.mark.parametrize("n,k,m,B", [(192, 384, 1536, 128), (100, 200, 700, 64)])
def test_layer_two_four(duo, n, k, m, B):
    say("layer 2:4", n, k, m, B)
    W, X = synth.layer_inputs(n, k, m, torch.bfloat16, torch.bfloat16, seed=n + k + 3, device="cpu", sigma=1.0,
                              outliers=3)
    out = duo.prune_linear(W.to(DEV), X.to(DEV), 0.5, 0.5, block=B, nm=(2, 4))
    torch.cuda.synchronize()
    Wn, Xn = W.float().numpy(), X.float().numpy()
    ref = R.prune_layer(Wn, Xn, 0.5, 0.5, B=B, nm=(2, 4))
    keep = out["mask"].cpu().numpy()
    Wg = f64(out["W_out"])
    assert np.all((~keep).reshape(n, -1, 4).sum(axis=2) == 2)
    assert np.mean(keep == ref["keep"]) >= 0.999
    assert relfro(Wg, ref["W_hat"]) < 1e-3
    J_g, J_r = R.objective(Wn, Wg, Xn, 0.5), R.objective(Wn, ref["W_hat"], Xn, 0.5)
    assert abs(J_g - J_r) <= 1e-3 * J_r
    assert torch.equal(out["W_lowp"].cpu(), out["W_out"].cpu().to(torch.bfloat16))


@pytest.mark.parametrize("n,k,B,N", [(48, 2304, 128, 2), (40, 2200, 64, 1), (33, 132, 128, 3)])
def test_prune_layer_nm_forms(duo, n, k, B, N):
    """Stage 3 with N:4 groups in both residual forms (in the Y form a group's
    values are rebuilt from w and y before its selection): the mask a valid
    N-lowest choice of the GPU's own scores, those scores and W against the
    oracle forced to the GPU's mask, every difference from the oracle's own
    choice a near-tie; several super-blocks, ragged rows and blocks."""
    say("prune_layer N:4 forms", n, k, B, N)
    W, X = synth.layer_inputs(n, k, 3 * k, torch.bfloat16, torch.bfloat16, seed=n + k + 9, device="cpu", sigma=1.0,
                              outliers=2)
    H, G, a = R.hessian_terms(X.float().numpy(), 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    L32, D32, f32, G32, a32 = (np.ascontiguousarray(x.astype(np.float32)) for x in (L, D, fac, G, a))
    Wf = W.float().numpy()
    t = lambda x: torch.tensor(x, device=DEV)
    outs = {}
    for form in ("d", "y"):
        W_out, _, mask, sc = duo.duo_prune_layer(W.to(DEV), t(L32), t(G32), t(a32), 0.5, B, want_scores=True,
                                                 nm_n=N, form=form)
        keep = duo.unpack_mask(mask, k).cpu().numpy()
        S_g = f64(sc)
        assert np.all((~keep).reshape(n, -1, 4).sum(axis=2) == N), form
        _groups_valid(keep, S_g, N)
        scores = []
        Wr, _ = R.sweep_blocked(Wf, L32, D32, f32, 0.5, B, mask_in=keep, scores_out=scores, nm=(N, 4))
        S_ref = np.concatenate(scores, axis=1)
        assert relfro(S_g, S_ref) < 1e-5, (form, relfro(S_g, S_ref))
        assert relfro(f64(W_out), Wr) < 1e-5, (form, relfro(f64(W_out), Wr))
        _near_ties(Wf, L32, D32, f32, B, N, keep)
        outs[form] = (keep, f64(W_out))
    assert np.mean(outs["d"][0] == outs["y"][0]) >= 0.999
    if np.array_equal(outs["d"][0], outs["y"][0]):
        assert relfro(outs["y"][1], outs["d"][1]) < 1e-5


def test_nm_refuses_bad_shapes(duo):
    say("nm shapes")
    W = torch.zeros((8, 30), dtype=torch.float32, device=DEV)
    L = torch.eye(30, device=DEV)
    with pytest.raises(duo.DuoError):
        duo.duo_sweep(W, L, torch.zeros((30, 30), device=DEV), torch.ones(30, device=DEV), 0.5, 8, nm_n=2)
