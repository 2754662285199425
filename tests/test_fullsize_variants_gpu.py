"""Full-size parity of the solver's options at the benchmark shape (LLaMA-2-7B
q_proj: n = k = 4096, 131072 bf16 tokens), through the call sequence that
bench.py times with --act-order, --nm 2 and --quant 4.

* act_order: the fp64 diagonal over every token against the oracle's
  (each square exact; sums in different orders: 1e-12 relative), the channel
  order bit-identical to the oracle's, and the outputs exactly the permuted
  run's outputs gathered back;
* 2:4 (both residual forms): exact per-group counts, each group's choice the two lowest of the
  scores the kernel selected on (ties by column), sampled rows equal to the
  column recurrence of Algorithm 1 in float64 on the kernel's own L, D and
  mask (1e-3 relative);
* INT4, groups of 128 (both residual forms): every kept weight exactly on its reported grid;
  sampled rows run through the same recurrence with the kernel's kept values
  forced, whose values at quantisation time must round to the kernel's codes
  except within 1e-3 of a step of a rounding boundary.
"""

from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

from oracle import duo_ref as R
from workloads import synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
NAME = "llama2_7b_q_proj"
N_ROWS = 6


def say(*a):
    print("[case]", *a, flush=True)


def relfro(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.fixture(scope="module")
def base(duo_lib):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    c = synth.CONFIGS[NAME]
    say("full-size variants", NAME)
    W, X = synth.config_inputs(NAME, device=DEV)
    return dict(duo=duo_lib, c=c, W=W, X=X)


def _stage12(b, hdiag=None):
    duo, c, W, X = b["duo"], b["c"], b["W"], b["X"]
    n, k, m = c["n"], c["k"], c["m"]
    H = torch.zeros((k, k), dtype=torch.float32, device=DEV)
    G = torch.zeros((k, k), dtype=torch.float32, device=DEV)
    a = torch.zeros(k, dtype=torch.float32, device=DEV)
    duo.duo_hessian_accum(X, H, c["p_x"], G=G, a=a, hdiag=hdiag)
    return H, G, a


def _recurrence(W, keep, LT, D, rows, values=None):
    """Eager column recurrence of Algorithm 1 in float64 on given L (as L^T
    rows), D and mask; values (optional) forces each kept weight's value.
    Returns (W_rows, w0_rows): final rows and each column's value when it was
    processed."""
    k = W.shape[1]
    Wr = W[rows].astype(np.float64)
    kp = keep[rows]
    w0s = np.zeros_like(Wr)
    for j in range(k):
        w0 = Wr[:, j].copy()
        w0s[:, j] = w0
        p = np.where(kp[:, j], w0 if values is None else values[rows, j], 0.0)
        e = (w0 - p) / float(LT[j, j])
        Wr[:, j] = p
        if j + 1 < k:
            Wr[:, j + 1:] -= np.outer(e, LT[j, j + 1:]) - np.outer(w0, D[j, j + 1:])
    return Wr, w0s


def test_fullsize_act_order(base):
    duo, c = base["duo"], base["c"]
    n, k, m, B = c["n"], c["k"], c["m"], c["block"]
    say("full-size act_order")
    hdiag = torch.zeros(k, dtype=torch.float64, device=DEV)
    H, G, a = _stage12(base, hdiag)
    perm, inv = duo.duo_act_order(hdiag)
    Hp, Gp = duo.duo_permute(H, perm, perm), duo.duo_permute(G, perm, perm)
    ap = duo.duo_permute(a.view(1, k), None, perm).view(k)
    Wp = duo.duo_permute(base["W"], None, perm)
    del H, G, a
    lam, fail = duo.duo_chol_inv(Hp, c["damp"], sync=True)
    assert fail == -1
    W_out_p, lowp_p, mask_p, _ = duo.duo_prune_layer(Wp, Hp, Gp, ap, c["p_w"], B, want_lowp=True)
    W_out = duo.duo_permute(W_out_p, None, inv)
    mask = duo.duo_permute_mask(mask_p, k, inv)
    torch.cuda.synchronize()
    # the diagonal and the order against the oracle's, over every token
    X = base["X"]
    step = 8192
    with ThreadPoolExecutor(8) as ex:
        parts = list(ex.map(lambda t0: R.hessian_entries(X[t0:t0 + step].float().cpu().numpy(), c["p_x"],
                                                         np.arange(2)), range(0, m, step)))
    diag = sum(p["diag"] for p in parts)
    hd = hdiag.cpu().numpy()
    assert np.all(np.abs(hd - diag) <= 1e-12 * diag + 1e-300), float(np.max(np.abs(hd - diag) / diag))
    ref_perm = np.lexsort((np.arange(k), -diag))
    assert np.array_equal(perm.cpu().numpy(), ref_perm)
    # outputs gathered back: exactly the permuted run's columns
    pm = perm.long().cpu()
    assert torch.equal(W_out.cpu()[:, pm], W_out_p.cpu())
    keep, keep_p = duo.unpack_mask(mask, k).cpu(), duo.unpack_mask(mask_p, k).cpu()
    assert torch.equal(keep[:, pm], keep_p)
    assert int((~keep).sum()) == int(np.floor(c["p_w"] * n * k + 0.5))
    # sampled rows of the permuted problem follow the recurrence on its own L, D
    D, _ = duo.duo_score_terms(Hp, Gp, ap)
    LT, Dn = Hp.t().contiguous().cpu().numpy(), D.cpu().numpy()
    rows = np.sort(np.random.default_rng(1).choice(n, N_ROWS, replace=False))
    Wr, _ = _recurrence(Wp.float().cpu().numpy(), keep_p.numpy(), LT, Dn, rows)
    Wo = W_out_p.cpu().numpy()
    for i, r in enumerate(rows):
        assert relfro(Wo[r], Wr[i]) < 1e-3, (r, relfro(Wo[r], Wr[i]))


@pytest.mark.parametrize("form", [None, "y"])
def test_fullsize_two_four(base, form):
    """form None: the automatic choice (the D form at k = 4096); "y": the Y
    form, whose group selections rebuild the values from w and y."""
    duo, c = base["duo"], base["c"]
    n, k, B = c["n"], c["k"], c["block"]
    say("full-size 2:4", form)
    H, G, a = _stage12(base)
    lam, fail = duo.duo_chol_inv(H, c["damp"], sync=True)
    assert fail == -1
    W_out, lowp, mask, scores = duo.duo_prune_layer(base["W"], H, G, a, c["p_w"], B, want_lowp=True,
                                                    want_scores=True, nm_n=2, form=form)
    D, _ = duo.duo_score_terms(H, G, a)
    torch.cuda.synchronize()
    keep = duo.unpack_mask(mask, k).cpu().numpy()
    S = scores.cpu().numpy()
    Wo = W_out.cpu().numpy()
    assert np.all((~keep).reshape(n, -1, 4).sum(axis=2) == 2)
    assert np.all(Wo[~keep] == 0.0)
    assert torch.equal(lowp, W_out.to(lowp.dtype))
    # each group: the two lowest kernel scores (ties by column)
    g = S.reshape(n, -1, 4)
    order = np.argsort(g, axis=2, kind="stable")
    want = np.ones_like(g, dtype=bool)
    np.put_along_axis(want, order[:, :, :2], False, axis=2)
    assert np.array_equal(want.reshape(n, k), keep)
    LT, Dn = H.t().contiguous().cpu().numpy(), D.cpu().numpy()
    rows = np.sort(np.random.default_rng(2).choice(n, N_ROWS, replace=False))
    Wr, _ = _recurrence(base["W"].float().cpu().numpy(), keep, LT, Dn, rows)
    for i, r in enumerate(rows):
        assert relfro(Wo[r], Wr[i]) < 1e-3, (r, relfro(Wo[r], Wr[i]))


@pytest.mark.parametrize("form", [None, "y"])
def test_fullsize_int4(base, form):
    duo, c = base["duo"], base["c"]
    n, k, B = c["n"], c["k"], c["block"]
    bits, group = 4, 128
    say("full-size int4", form)
    H, G, a = _stage12(base)
    lam, fail = duo.duo_chol_inv(H, c["damp"], sync=True)
    assert fail == -1
    W_out, _, mask, _, qs, qz = duo.duo_prune_layer(base["W"], H, G, a, c["p_w"], B, quant=(bits, group),
                                                    form=form)
    D, _ = duo.duo_score_terms(H, G, a)
    torch.cuda.synchronize()
    keep = duo.unpack_mask(mask, k).cpu().numpy()
    Wq, qs, qz = W_out.cpu().numpy(), qs.cpu().numpy(), qz.cpu().numpy()
    assert int((~keep).sum()) == int(np.floor(c["p_w"] * n * k + 0.5))
    cols = np.arange(k) // group
    s, z = qs[:, cols], qz[:, cols]
    code = np.rint(Wq / s) + z
    assert np.all(Wq[~keep] == 0) and np.all(z == np.rint(z))
    assert np.all((code >= 0) & (code <= 2 ** bits - 1))
    assert np.array_equal((s * (code.astype(np.float32) - z)).astype(np.float32)[keep], Wq[keep])
    LT, Dn = H.t().contiguous().cpu().numpy(), D.cpu().numpy()
    rows = np.sort(np.random.default_rng(3).choice(n, N_ROWS, replace=False))
    _, w0 = _recurrence(base["W"].float().cpu().numpy(), keep, LT, Dn, rows, values=Wq.astype(np.float64))
    t = w0 / s[rows]
    code_r = np.clip(np.round(t) + z[rows], 0, 2 ** bits - 1)
    kr = keep[rows]
    diff = kr & (code_r != code[rows])
    frac = np.abs(t - np.floor(t) - 0.5)
    say("int4 sampled rows: %d of %d codes differ" % (int(diff.sum()), int(kr.sum())))
    assert np.all(frac[diff] < 1e-3), float(frac[diff].max())
