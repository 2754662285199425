"""Joint pruning and RTN quantisation (Table 4) on the HIP path.

The kept weights are integer codes on per-row, per-group grids; each code is
an integer decided from fp32 values, so the checks separate what is exact from
what is floating point:

* structure (exact): pruned weights are 0; every kept weight equals
  s * (c - z) computed in fp32 with an integer code c in [0, 2^b - 1], for
  the grid (s, z) the kernel reports;
* parity without cascades: the oracle is run forced to the GPU's mask and
  kept values, so both sides compensate the same errors; then the oracle's
  grids match the GPU's (scale within 1e-5 relative, zero codes equal) and
  every GPU code is the rounding of the oracle's value at quantisation time,
  except where that value lies within 1e-3 of a step of a rounding boundary
  (fp32 against fp64 evaluation of the same sums: about 1e-6 relative to the
  weight, i.e. below 2.6e-4 of a step even at 8 bits);
* the unforced layer agrees with the oracle's mask to 99.9 %.
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


def _stage(n, k, m, seed):
    W, X = synth.layer_inputs(n, k, m, torch.bfloat16, torch.bfloat16, seed=seed, device="cpu", sigma=1.0,
                              outliers=2)
    H, G, a = R.hessian_terms(X.float().numpy(), 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    L32, D32, f32 = (np.ascontiguousarray(x.astype(np.float32)) for x in (L, D, fac))
    return W, X, L32, D32, f32


def _structure(Wq, keep, qs, qz, bits, group):
    """Exact: pruned = 0, kept = fp32 s * (c - z) with integer c in range."""
    n, k = Wq.shape
    cols = np.arange(k) // group
    s, z = qs[:, cols], qz[:, cols]
    assert np.all(Wq[~keep] == 0)
    assert np.all(z == np.round(z)) and np.all(s > 0)
    c = np.rint(Wq / s) + z
    assert np.all((c >= 0) & (c <= 2 ** bits - 1))
    rebuilt = (s * (c.astype(np.float32) - z)).astype(np.float32)
    assert np.array_equal(rebuilt[keep], Wq[keep])
    return c


def _forced_parity(W, L, D, fac, B, bits, group, Wq, keep, qs, qz, nm=None, tol=1e-3):
    """Oracle forced to the GPU's mask and kept values (no cascade).  tol:
    the distance from a rounding boundary, in steps, within which the two
    sides may round differently."""
    qp = []
    w0 = np.zeros(W.shape)
    R.sweep_blocked(W, L, D, fac, 0.5, B, mask_in=keep, quant=(bits, group), qparams_out=qp, w0_out=w0,
                    values_in=Wq.astype(np.float64), nm=nm)
    s_r = np.stack([p[0] for p in qp], axis=1)
    z_r = np.stack([p[1] for p in qp], axis=1)
    assert np.all(np.abs(s_r - qs) <= 1e-5 * s_r), float(np.max(np.abs(s_r - qs) / s_r))
    # a zero code may differ only where -min / s lies within tol of a rounding
    # boundary (the same fp32-against-fp64 margin as the codes below)
    lo = np.stack([np.minimum(0.0, p[2].min(axis=1)) for p in qp], axis=1)
    zr = -lo / s_r
    zdiff = z_r != qz
    assert np.all(np.abs(z_r - qz) <= 1)
    assert np.all(np.abs(zr - np.floor(zr) - 0.5)[zdiff] < tol), zr[zdiff]
    cols = np.arange(W.shape[1]) // group
    s, z = qs[:, cols].astype(np.float64), qz[:, cols].astype(np.float64)
    t = w0 / s
    code_r = np.clip(np.round(t) + z, 0, 2 ** bits - 1)
    code_g = np.rint(Wq / qs[:, cols]) + z
    diff = keep & (code_r != code_g)
    frac = np.abs(t - np.floor(t) - 0.5)            # distance from a rounding boundary, in steps
    assert np.all(frac[diff] < tol), float(frac[diff].max())
    assert diff.sum() <= 2 * tol * keep.sum() + 2
    return diff.sum()


@pytest.mark.parametrize("n,k,B,bits,group,nm", [(128, 512, 128, 4, 128, 0), (200, 384, 64, 8, 32, 0),
                                                 (64, 256, 128, 4, 16, 2), (33, 130, 128, 3, 64, 0),
                                                 (48, 256, 32, 2, 32, 0)])
def test_sweep_quant(duo, n, k, B, bits, group, nm):
    say("sweep quant", n, k, B, bits, group, nm)
    W, X, L, D, fac = _stage(n, k, 3 * k, seed=13 * n + k + bits)
    t = lambda x: torch.tensor(x, device=DEV)
    W_out, _, mask, _, qs, qz = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), 0.5, B, nm_n=nm, quant=(bits, group))
    Wq = W_out.cpu().numpy()
    keep = duo.unpack_mask(mask, k).cpu().numpy()
    qs, qz = qs.cpu().numpy(), qz.cpu().numpy()
    assert qs.shape == (n, (k + group - 1) // group)
    _structure(Wq, keep, qs, qz, bits, group)
    if nm:
        assert np.all((~keep).reshape(n, -1, 4).sum(axis=2) == nm)
    Wn = W.float().numpy()
    _forced_parity(Wn, L, D, fac, B, bits, group, Wq, keep, qs, qz, nm=(nm, 4) if nm else None)
    _, keep_r = R.sweep_blocked(Wn, L, D, fac, 0.5, B, quant=(bits, group), nm=(nm, 4) if nm else None)
    assert np.mean(keep == keep_r) >= 0.999


@pytest.mark.parametrize("bits", [4, 8])
def test_layer_quant(duo, bits):
    n, k, m, B = 192, 384, 1536, 128
    say("layer quant", bits)
    W, X = synth.layer_inputs(n, k, m, torch.bfloat16, torch.bfloat16, seed=n + k + bits, device="cpu",
                              sigma=1.0, outliers=3)
    out = duo.prune_linear(W.to(DEV), X.to(DEV), 0.5, 0.5, block=B, quant=(bits, 128))
    torch.cuda.synchronize()
    Wq = out["W_out"].cpu().numpy()
    keep = out["mask"].cpu().numpy()
    qs, qz = out["q_scale"].cpu().numpy(), out["q_zero"].cpu().numpy()
    _structure(Wq, keep, qs, qz, bits, 128)
    ref = R.prune_layer(W.float().numpy(), X.float().numpy(), 0.5, 0.5, B=B, quant=(bits, 128))
    assert np.mean(keep == ref["keep"]) >= 0.999
    # forced parity on the oracle's own stage-2 terms: the GPU compensated with
    # its fp32 L, D, fac (about 1e-5 relative from the oracle's), which moves
    # the values at quantisation time by up to ~5e-4 of a step at 8 bits
    H, G, a = R.hessian_terms(X.float().numpy(), 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    _forced_parity(W.float().numpy(), L, D, fac, B, bits, 128, Wq, keep, qs, qz, tol=5e-3)


def test_quant_wider_bits_approach_unquantised(duo):
    """With the same mask, 8-bit grids move the pruned layer by a few steps
    per weight at most (each weight's own rounding plus the compensation of
    the earlier columns' roundings)."""
    say("quant vs none")
    n, k, B = 96, 256, 128
    W, X, L, D, fac = _stage(n, k, 3 * k, seed=3)
    t = lambda x: torch.tensor(x, device=DEV)
    Wa, _, ma, _ = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), 0.5, B)
    Wb, _, mb, _, qs, _ = duo.duo_sweep(W.to(DEV), t(L), t(D), t(fac), 0.5, B, mask_in=ma, quant=(8, 128))
    assert torch.equal(ma, mb)
    a, b = Wa.cpu().numpy(), Wb.cpu().numpy()
    rel = np.linalg.norm(a - b) / np.linalg.norm(a)
    step = float(qs.max().cpu())
    assert rel < 0.05 and np.max(np.abs(a - b)) < 20 * step


@pytest.mark.parametrize("n,k,B,bits,group,nm", [(48, 2304, 128, 4, 128, 0), (40, 1000, 64, 8, 64, 0),
                                                 (64, 1152, 128, 4, 128, 2)])
def test_prune_layer_quant_forms(duo, n, k, B, bits, group, nm):
    """Stage 3 with one grid per row and block (group == block) in both
    residual forms: in the Y form a grid is fixed right after the block's
    start product, where W[:, blk] holds Algorithm 1's values; structure
    exact, grids and codes against the oracle forced to the GPU's mask and
    values on the same L, D, fac; several super-blocks, ragged rows and
    blocks, and N:4 with quantisation."""
    say("prune_layer quant forms", n, k, B, bits, group, nm)
    W, X = synth.layer_inputs(n, k, 3 * k, torch.bfloat16, torch.bfloat16, seed=n + k + bits + 17, device="cpu",
                              sigma=1.0, outliers=2)
    H, G, a = R.hessian_terms(X.float().numpy(), 0.5)
    L, _ = R.inverse_cholesky(H, 0.01)
    fac, D, _ = R.score_terms(G, L, a)
    L32, D32, f32, G32, a32 = (np.ascontiguousarray(x.astype(np.float32)) for x in (L, D, fac, G, a))
    Wn = W.float().numpy()
    t = lambda x: torch.tensor(x, device=DEV)
    keeps = {}
    for form in ("d", "y"):
        W_out, _, mask, _, qs, qz = duo.duo_prune_layer(W.to(DEV), t(L32), t(G32), t(a32), 0.5, B, nm_n=nm,
                                                        quant=(bits, group), form=form)
        Wq = W_out.cpu().numpy()
        keep = duo.unpack_mask(mask, k).cpu().numpy()
        qs, qz = qs.cpu().numpy(), qz.cpu().numpy()
        _structure(Wq, keep, qs, qz, bits, group)
        if nm:
            assert np.all((~keep).reshape(n, -1, 4).sum(axis=2) == nm)
        else:
            assert (~keep).sum() == sum(R.block_prune_counts(n, k, 0.5, B))
        # the GPU's fac and U come from its own Q = G L (about 1e-6 relative
        # from the oracle's), which moves values at quantisation time slightly
        _forced_parity(Wn, L32, D32, f32, B, bits, group, Wq, keep, qs, qz, nm=(nm, 4) if nm else None, tol=5e-3)
        keeps[form] = keep
    assert np.mean(keeps["d"] == keeps["y"]) >= 0.999
