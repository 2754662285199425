"""Parity at the full layer sizes of the LLaMA-shaped workloads, with the same
entry points, workspaces and launch configuration that bench.py times.

A float64 oracle cannot form k x k terms over 131072 tokens for these layers
in test time (k up to 28672), so each case compares what the oracle can
compute exactly at full size and checks the rest through properties that
hold at any size:

* activation masks bit-exact on sampled tokens (the oracle's per-token rule);
* H and G on a sampled set of channels (random channels plus a trailing
  window), and all of a and diag(H), summed by the oracle over every token;
  fp32 sums of exact bf16 products: each entry within 4e-5 * sqrt(H_ii H_jj)
  (resp. sqrt(a_i H_jj)), the worst-case relative error of a recursive fp32
  sum of ~600 partial sums (u = 6e-8);
* lambda, and L, fac, D on the trailing window of columns from the oracle's
  window terms (the window is self-contained given lambda; see
  oracle.duo_ref.window_terms), at the same relative-Frobenius bars as the
  small-size factorisation and score tests (2e-4 for L, 1e-4 for fac and D);
* the sweep: exact per-block prune counts (cumulative rounding), the mask a
  valid (score, column, row) selection of the scores the kernel selected on,
  W_hat zero exactly where pruned, the bf16 copy equal to RNE(W_out), sampled
  rows of W_hat equal to the column recurrence of Algorithm 1 evaluated in
  float64 on the kernel's own L, D and mask (1e-3 relative, the tolerance on
  pruned weights), and the layer objective below magnitude pruning's on a
  token sample.
"""

from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

from oracle import duo_ref as R
from workloads import synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
WINDOW = 512        # trailing window of columns checked against the oracle
N_RAND = 64         # further random channels in the sampled H/G set
N_TOK = 48          # sampled tokens for the activation mask
N_ROWS = 6          # sampled weight rows for the sweep recurrence

CASES = ["llama2_7b_q_proj", "llama2_7b_down_proj", "llama2_70b_down_proj"]


def say(*a):
    print("[case]", *a, flush=True)


def relfro(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.fixture(scope="module", params=CASES)
def run(request, duo_lib):
    """One full layer through the bench.py call sequence; keeps host copies of
    what the checks need."""
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    duo = duo_lib
    name = request.param
    c = synth.CONFIGS[name]
    n, k, m, B = c["n"], c["k"], c["m"], c["block"]
    say("full-size layer", name, n, k, m)
    W, X = synth.config_inputs(name, device=DEV)
    rng = np.random.default_rng(k)
    win = np.arange(k - WINDOW, k)
    rand = np.sort(rng.choice(k - WINDOW, N_RAND, replace=False))
    idx = np.concatenate([rand, win])
    idx_t = torch.tensor(idx, device=DEV)

    H = torch.zeros((k, k), dtype=torch.float32, device=DEV)
    G = torch.zeros((k, k), dtype=torch.float32, device=DEV)
    a = torch.zeros(k, dtype=torch.float32, device=DEV)
    ws_h = duo.workspace(duo.DUO_OP_HESSIAN, 0, k, m, 0, DEV)
    ws_c = duo.workspace(duo.DUO_OP_CHOL_INV, 0, k, 0, 0, DEV)
    ws_p = duo.workspace(duo.DUO_OP_PRUNE_LAYER, n, k, 0, B, DEV)
    duo.duo_hessian_accum(X, H, c["p_x"], G=G, a=a, ws=ws_h)
    out = dict(name=name, c=c, idx=idx, nwin=WINDOW)
    out["H_s"] = H[idx_t][:, idx_t].double().cpu().numpy()
    out["G_s"] = G[idx_t][:, idx_t].double().cpu().numpy()
    out["a"] = a.double().cpu().numpy()
    out["diag"] = H.diagonal().double().cpu().numpy()
    lam, fail = duo.duo_chol_inv(H, c["damp"], ws=ws_c, sync=True)
    out["lam"], out["fail"] = lam, fail
    W_out, lowp, mask, scores = duo.duo_prune_layer(W, H, G, a, c["p_w"], B, ws=ws_p, want_lowp=True,
                                                    want_scores=True)
    # the separate score-terms entry point on the same L, G, a (same kernels)
    D, fac = duo.duo_score_terms(H, G, a)
    torch.cuda.synchronize()
    del ws_h, ws_c, ws_p, G
    w = torch.tensor(win, device=DEV)
    out["L_win"] = H[w][:, w].double().cpu().numpy()
    out["D_win"] = D[w][:, w].double().cpu().numpy()
    out["fac"] = fac.double().cpu().numpy()
    out["LT"] = H.t().contiguous().cpu().numpy()          # row j = column j of L
    out["D"] = D.cpu().numpy()
    del H, D
    out["W"] = W.float().cpu().numpy()
    out["W_out"] = W_out.cpu().numpy()
    out["lowp_ok"] = bool(torch.equal(lowp, W_out.to(W.dtype)))
    out["keep"] = duo_lib.unpack_mask(mask, k).cpu().numpy()
    out["scores"] = scores.cpu().numpy()
    del W_out, lowp, mask, scores
    act = duo.duo_act_sparsify_mask(X, c["p_x"])
    tok = np.sort(np.concatenate([[0, m - 1], rng.choice(m, N_TOK, replace=False)]))
    tok_t = torch.tensor(tok, device=DEV)
    out["tok"] = tok
    out["act_keep"] = duo.unpack_mask(act[tok_t], k).cpu().numpy()
    out["X"] = X.float().cpu().numpy()
    del act, W, X
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    yield out


def _stage1_oracle(run):
    """Oracle H/G entries on the sampled channels and all of a, diag(H), over
    every token (token ranges summed in parallel threads)."""
    if "ref1" not in run:
        X, p_x, idx = run["X"], run["c"]["p_x"], run["idx"]
        m = X.shape[0]
        step = 8192
        with ThreadPoolExecutor(8) as ex:
            parts = list(ex.map(lambda t0: R.hessian_entries(X, p_x, idx, t0=t0, t1=min(m, t0 + step)),
                                range(0, m, step)))
        run["ref1"] = {key: sum(p[key] for p in parts) for key in parts[0]}
    return run["ref1"]


def test_fullsize_activation_mask(run):
    say("full-size act mask", run["name"])
    _, keep = R.sparsify_tokens(run["X"][run["tok"]], run["c"]["p_x"])
    assert np.array_equal(run["act_keep"], keep)


def test_fullsize_stage1_entries(run):
    say("full-size stage 1", run["name"])
    ref = _stage1_oracle(run)
    tol = 4e-5
    idx = run["idx"]
    dH = np.sqrt(ref["diag"][idx])
    bound = tol * np.outer(dH, dH) + 1e-30
    assert np.all(np.abs(run["H_s"] - ref["H"]) <= bound), float(np.max(np.abs(run["H_s"] - ref["H"]) / bound))
    bound_G = tol * np.outer(np.sqrt(ref["a"][idx]), dH) + 1e-30
    assert np.all(np.abs(run["G_s"] - ref["G"]) <= bound_G), float(np.max(np.abs(run["G_s"] - ref["G"]) / bound_G))
    assert np.all(np.abs(run["a"] - ref["a"]) <= tol * ref["a"] + 1e-30)
    assert np.all(np.abs(run["diag"] - ref["diag"]) <= tol * ref["diag"] + 1e-30)


def test_fullsize_factor_and_scores_window(run):
    say("full-size window", run["name"])
    ref = _stage1_oracle(run)
    c = run["c"]
    t = run["nwin"]
    lam = c["damp"] * float(np.mean(ref["diag"]))
    assert run["fail"] == -1
    assert abs(run["lam"] - lam) <= 5e-5 * lam
    w = slice(len(run["idx"]) - t, len(run["idx"]))
    Lr, facr, Dr = R.window_terms(ref["H"][w, w], ref["G"][w, w], ref["a"][-t:], lam)
    L = run["L_win"]
    assert np.all(np.triu(L, 1) == 0.0) and np.all(np.diag(L) > 0)
    eL, efac, eD = relfro(L, Lr), relfro(run["fac"][-t:], facr), relfro(np.triu(run["D_win"], 1), Dr)
    say("window errors L %.2e fac %.2e D %.2e" % (eL, efac, eD))
    assert eL < 2e-4 and efac < 1e-4 and eD < 1e-4


def test_fullsize_sweep_properties(run):
    say("full-size sweep", run["name"])
    c = run["c"]
    n, k, B, p_w = c["n"], c["k"], c["block"], c["p_w"]
    keep, W_out, S = run["keep"], run["W_out"], run["scores"]
    counts = R.block_prune_counts(n, k, p_w, B)
    assert (~keep).sum() == int(np.floor(p_w * n * k + 0.5))
    assert np.all(W_out[~keep] == 0.0)
    assert run["lowp_ok"]
    for bi, j0 in enumerate(range(0, k, B)):
        kb = keep[:, j0:j0 + B]
        assert (~kb).sum() == counts[bi], bi
        if kb.all() or (~kb).all():
            continue
        # valid lowest-z selection by (score, column, row): the largest pruned
        # key precedes the smallest kept key (flat index column * n + row)
        fS = S[:, j0:j0 + B].T.ravel()
        fK = kb.T.ravel()
        ip, ik = np.nonzero(~fK)[0], np.nonzero(fK)[0]
        smax = fS[ip].max()
        smin = fS[ik].min()
        last_pruned = (float(smax), int(ip[fS[ip] == smax].max()))
        first_kept = (float(smin), int(ik[fS[ik] == smin].min()))
        assert last_pruned < first_kept, (bi, last_pruned, first_kept)


def test_fullsize_sweep_rows(run):
    """Sampled rows follow the column recurrence of Algorithm 1 (the eager
    form, equal to the lazy one) on the kernel's own L, D and mask."""
    say("full-size sweep rows", run["name"])
    n, k = run["W"].shape
    rows = np.sort(np.random.default_rng(n).choice(n, N_ROWS, replace=False))
    Wr = run["W"][rows].astype(np.float64)
    keep = run["keep"][rows]
    LT, D = run["LT"], run["D"]
    for j in range(k):
        w0 = Wr[:, j].copy()
        p = w0 * keep[:, j]
        e = (w0 - p) / float(LT[j, j])
        Wr[:, j] = p
        if j + 1 < k:
            Wr[:, j + 1:] -= np.outer(e, LT[j, j + 1:]) - np.outer(w0, D[j, j + 1:])
    for i, r in enumerate(rows):
        assert relfro(run["W_out"][r], Wr[i]) < 1e-3, (r, relfro(run["W_out"][r], Wr[i]))


def test_fullsize_objective_below_magnitude(run):
    """Sec. 5: the asymmetric calibration beats plain magnitude pruning; on a
    sample of 1024 tokens the layer objective of W_hat is below that of
    magnitude pruning with the same per-block counts."""
    c = run["c"]
    if c["k"] > 12000:
        pytest.skip("magnitude comparator at k > 12000 exceeds the test's time budget")
    say("full-size objective", run["name"])
    X = run["X"][:1024]
    W = run["W"]
    Wm, _ = R.magnitude_layer(W, c["p_w"], c["block"])
    J = R.objective(W, run["W_out"], X, c["p_x"])
    Jm = R.objective(W, Wm, X, c["p_x"])
    say("objective %.4e magnitude %.4e" % (J, Jm))
    assert J < Jm
