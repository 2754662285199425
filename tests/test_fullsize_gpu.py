"""Parity at the full layer sizes of the LLaMA-shaped workloads, with the same
entry points, workspaces and launch configuration that bench.py times.

A float64 oracle cannot form k x k terms over 131072 tokens for these layers
in test time (k up to 28672), so each case compares what the oracle can
compute exactly at full size and checks the rest through properties that
hold at any size:

* activation masks bit-exact on sampled tokens (the oracle's per-token rule);
* H and G on a sampled set of channels (random channels plus a trailing
  window; G on and above its diagonal, the part stage 1 accumulates), and
  all of a and diag(H), summed by the oracle over every token;
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
    # columns for the defining property of L and rows for fac/D: column 0 and
    # k - 1 plus three per 1024 columns (every group of eight blocks the UL
    # factorisation updates together), and the first row of every such group
    cols = [0, k - 1]
    for g0 in range(0, k, 1024):
        g1 = min(k, g0 + 1024)
        cols += [g0, int(rng.integers(g0, g1)), g1 - 1]
    out["pcols"] = np.unique(np.array(cols))
    out["prows"] = np.unique(np.array([0, 1] + list(range(0, k, 1024)) + [int(rng.integers(0, 512))]))
    out["H_full"] = H.cpu().numpy()             # the matrix the factorisation is given
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
        rows = run["prows"]
        with ThreadPoolExecutor(8) as ex:
            parts = list(ex.map(lambda t0: R.hessian_entries(X, p_x, idx, t0=t0, t1=min(m, t0 + step), rows=rows),
                                range(0, m, step)))
        run["ref1"] = {key: sum(p[key] for p in parts) for key in parts[0]}
    return run["ref1"]


def test_fullsize_inverse_factor_property(run):
    """Defining property of the damped inverse Cholesky factor (Sec. 4.3,
    App. A.2): L^T (H + lambda I) L = I, evaluated in float64 on the sampled
    columns j (every group of eight blocks, column 0 included) for the fp32
    H the factorisation was given.  Bar on each column's residual norm:
    16 sqrt(k) u (u = 2^-24): the random-walk size of the k rounding errors of
    an fp32 inner-product chain, with a factor 16 for the chains of the
    factorisation and of the triangular inverse and for margin.  LAPACK's fp32
    factorisation along the same route (UL Cholesky of H + lambda I, then the
    triangular inverse V^-1 = L^T) of the same matrix is evaluated beside it
    and reported as the yardstick."""
    import scipy.linalg as sl

    say("full-size L property", run["name"])
    Hf, LT, lam = run["H_full"], run["LT"], run["lam"]
    k = Hf.shape[0]
    J = run["pcols"]
    Lj = LT[J].T.astype(np.float64)                        # k x |J|: columns j of L
    M = np.empty((k, len(J)))
    for r0 in range(0, k, 2048):
        r1 = min(k, r0 + 2048)
        M[r0:r1] = Hf[r0:r1].astype(np.float64) @ Lj + lam * Lj[r0:r1]
    Rg = np.empty((k, len(J)))
    for r0 in range(0, k, 2048):
        r1 = min(k, r0 + 2048)
        Rg[r0:r1] = LT[r0:r1].astype(np.float64) @ M
    Rg[J, np.arange(len(J))] -= 1.0
    res_gpu = np.linalg.norm(Rg, axis=0)
    # float32 LAPACK along the same route: H + lambda I = V V^T (V upper, from
    # the reversed lower Cholesky factor), L = V^-T by the triangular inverse
    Hl = Hf.copy()
    Hl[np.diag_indices(k)] += np.float32(lam)
    C = np.linalg.cholesky(Hl[::-1, ::-1])                 # float32
    del Hl
    V = np.ascontiguousarray(C[::-1, ::-1])
    del C
    Vinv, info = sl.lapack.strtri(V, lower=0)               # = L_ref^T, float32
    assert info == 0 and Vinv.dtype == np.float32
    del V
    Lr = Vinv[J].T.astype(np.float64)                       # columns j of L_ref
    Mr = np.empty((k, len(J)))
    for r0 in range(0, k, 2048):
        r1 = min(k, r0 + 2048)
        Mr[r0:r1] = Hf[r0:r1].astype(np.float64) @ Lr + lam * Lr[r0:r1]
    Rr = np.empty((k, len(J)))
    for r0 in range(0, k, 2048):
        r1 = min(k, r0 + 2048)
        Rr[r0:r1] = np.triu(Vinv[r0:r1], r0).astype(np.float64) @ Mr
    del Vinv
    Rr[J, np.arange(len(J))] -= 1.0
    res_ref = np.linalg.norm(Rr, axis=0)
    bar = 16.0 * np.sqrt(k) * 2.0 ** -24
    worst = int(np.argmax(res_gpu))
    say("L^T H L - I, worst column %d: GPU %.2e (LAPACK fp32 %.2e); median GPU %.2e, LAPACK %.2e; bar %.1e" %
        (J[worst], res_gpu[worst], res_ref[worst], float(np.median(res_gpu)), float(np.median(res_ref)), bar))
    assert np.all(res_gpu <= bar), (J[worst], res_gpu[worst], res_ref[worst])


def test_fullsize_score_terms_leading_rows(run):
    """fac_p and row p of D (Eq. 7, App. A.3-A.4) recomputed in float64 for
    sampled leading rows p from the oracle's G row over all tokens, its a_p,
    and the kernel's L: Q_p = G_p L, b_p = sum_{i>p} Q_pi^2, c_p = Q_pp / L_pp,
    D_p = U_p L^T.  fac within 1e-4 relative per row, D rows within 1e-4
    relative Frobenius (the window bars)."""
    say("full-size leading score rows", run["name"])
    ref = _stage1_oracle(run)
    LT = run["LT"]
    k = LT.shape[0]
    for i, p in enumerate(run["prows"]):
        g = ref["G_rows"][i]
        Q = np.empty(k)
        for r0 in range(0, k, 4096):
            r1 = min(k, r0 + 4096)
            Q[r0:r1] = LT[r0:r1].astype(np.float64) @ g          # Q_p,j = sum_l G_pl L_lj
        Lpp = float(LT[p, p])
        U = Q.copy()
        U[:p + 1] = 0.0
        fac = 1.0 / Lpp ** 2 + ref["a"][p] - float(U @ U) + 2.0 * Q[p] / Lpp
        D = np.empty(k)
        for r0 in range(0, k, 4096):
            r1 = min(k, r0 + 4096)
            D[r0:r1] = LT[:, r0:r1].T.astype(np.float64) @ U        # D_pj = sum_i U_pi L_ji
        D[:p + 1] = 0.0
        ef = abs(run["fac"][p] - fac) / abs(fac)
        eD = relfro(np.where(np.arange(k) > p, run["D"][p], 0.0), D) if p < k - 1 else 0.0
        say(f"row {p}: fac {ef:.2e}, D row {eD:.2e}")
        assert ef < 1e-4 and eD < 1e-4, (p, ef, eD)


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
    # stage 1 accumulates G on and above its diagonal 256-tiles (all the solver reads); below them G stays zero
    up = idx[:, None] // 256 <= idx[None, :] // 256
    errG = np.where(up, np.abs(run["G_s"] - ref["G"]), 0.0)
    assert np.all(errG <= bound_G), float(np.max(errG / bound_G))
    assert np.all(run["G_s"][~up] == 0.0)
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
    say("full-size objective", run["name"])
    X = run["X"][:1024]
    W = run["W"]
    Wm, _ = R.magnitude_layer(W, c["p_w"], c["block"])
    J, Jm = R.objective(W, [run["W_out"], Wm], X, c["p_x"])
    say("objective %.4e magnitude %.4e" % (J, Jm))
    assert J < Jm
