"""Dual-sparse decode on the HIP path against oracle/decode_ref.py.

* compressed storage: integer and bit work, compared bit for bit with the
  oracle's compression of the same pruned weights and mask;
* the active channel set: the calibration rule's integer keys, so the GEMV
  uses exactly the oracle's channels;
* y: each product of a bf16 weight and an fp32 activation is rounded once in
  fp32 and the |A| terms of a row are summed in fp32, so every entry lies
  within (|A| + 2) 2^-24 sum_i |w_ri x_i| of the float64 value (recursive
  summation bound; |A| = number of active channels).
"""

import numpy as np
import pytest
import torch

from oracle import decode_ref as DR
from workloads import synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def duo(duo_lib):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return duo_lib


def say(*a):
    print("[case]", *a, flush=True)


def _mask_words(keep):
    n, k = keep.shape
    words = (k + 31) // 32
    pad = np.zeros((n, words * 32), dtype=np.uint64)
    pad[:, :k] = keep
    w = (pad.reshape(n, words, 32) << np.arange(32, dtype=np.uint64)).sum(-1)
    return torch.tensor(w.astype(np.uint32).view(np.int32))


def _layer(n, k, density, seed, dtype):
    g = torch.Generator().manual_seed(seed)
    keep = (torch.rand((n, k), generator=g) < density).numpy()
    W = (0.02 * torch.randn((n, k), generator=g)).to(dtype)
    W = torch.where(torch.tensor(keep), W, torch.zeros((), dtype=dtype))
    return W, keep


def _bits(W):
    if W.dtype == torch.bfloat16:
        return W.view(torch.int16).numpy().view(np.uint16)
    return DR._bf16_bits(W.numpy())


@pytest.mark.parametrize("n,k,density,dtype", [(300, 17, 0.5, torch.bfloat16), (513, 40, 0.1, torch.float32),
                                               (4096, 256, 0.5, torch.bfloat16), (257, 65, 1.0, torch.bfloat16),
                                               (64, 33, 0.0, torch.float32)])
def test_compress_bit_exact(duo, n, k, density, dtype):
    say("dsc compress", n, k, density, dtype)
    W, keep = _layer(n, k, density, n + k, dtype)
    comp = duo.dsc_compress(W.to(DEV), _mask_words(keep).to(DEV))
    ref = DR.compress(_bits(W), keep)
    assert np.array_equal(comp["col_ptr"].cpu().numpy(), ref["col_ptr"])
    assert np.array_equal(comp["maskT"].cpu().numpy().view(np.uint32), ref["mask"])
    assert np.array_equal(comp["chunk_off"].cpu().numpy().view(np.uint16), ref["chunk_off"])
    nnz = int(ref["col_ptr"][-1])
    assert np.array_equal(comp["values"].cpu().numpy().view(np.uint16)[:nnz], ref["values"])


def _check_gemv(y, Wb, x, p_x):
    xh, act = DR.active_channels(x, p_x)
    ref = Wb[:, act] @ xh[act]
    bound = (len(act) + 2) * 2.0 ** -24 * (np.abs(Wb[:, act]) @ np.abs(xh[act])) + 1e-30
    err = np.abs(y - ref)
    assert np.all(err <= bound), float(np.max(err / bound))


@pytest.mark.parametrize("n,k,p_x,xdtype", [(300, 17, 0.5, torch.float32), (4096, 4096, 0.5, torch.bfloat16),
                                            (1000, 700, 0.0, torch.bfloat16), (257, 129, 1.0, torch.float32),
                                            (8192, 3000, 0.6, torch.float32)])
def test_gemv_matches_definition(duo, n, k, p_x, xdtype):
    say("dsc gemv", n, k, p_x, xdtype)
    W, keep = _layer(n, k, 0.5, 3 * n + k, torch.bfloat16)
    comp = duo.dsc_compress(W.to(DEV), _mask_words(keep).to(DEV))
    g = torch.Generator().manual_seed(k)
    for t in range(3):
        x = (torch.randn(k, generator=g) * torch.exp(torch.randn(k, generator=g))).to(xdtype)
        y = duo.dsc_gemv(comp, x.to(DEV), p_x).cpu().numpy().astype(np.float64)
        Wb = W.float().numpy().astype(np.float64)
        _check_gemv(y, Wb, x.float().numpy().astype(np.float64), p_x)


def test_gemv_pruned_layer(duo):
    """On a layer pruned by the solver: compress its bf16 output and mask."""
    say("dsc gemv pruned layer")
    n, k, m = 384, 512, 2048
    W, X = synth.layer_inputs(n, k, m, torch.bfloat16, torch.bfloat16, seed=9, device="cpu", sigma=1.0)
    out = duo.prune_linear(W.to(DEV), X.to(DEV), 0.5, 0.5, block=128)
    keep = out["mask"].cpu().numpy()
    comp = duo.dsc_compress(out["W_lowp"], _mask_words(keep).to(DEV))
    Wb = out["W_lowp"].float().cpu().numpy().astype(np.float64)
    for t in range(4):
        x = X[t].float()
        y = duo.dsc_gemv(comp, X[t].to(DEV), 0.5).cpu().numpy().astype(np.float64)
        _check_gemv(y, Wb, x.numpy().astype(np.float64), 0.5)


def test_gemv_full_size_70b_down_proj(duo):
    """LLaMA-2-70B down_proj shape (n = 8192, k = 28672), 60 % weight and 50 %
    activation sparsity, a uniform random mask standing in for a calibrated
    one; every output row checked."""
    say("dsc gemv 70b down")
    n, k = 8192, 28672
    W, keep = _layer(n, k, 0.4, 70, torch.bfloat16)
    comp = duo.dsc_compress(W.to(DEV), _mask_words(keep).to(DEV))
    g = torch.Generator().manual_seed(1)
    x = (torch.randn(k, generator=g) * torch.exp(torch.randn(k, generator=g))).to(torch.bfloat16)
    y = duo.dsc_gemv(comp, x.to(DEV), 0.5).cpu().numpy().astype(np.float64)
    _check_gemv(y, W.float().numpy().astype(np.float64), x.float().numpy().astype(np.float64), 0.5)


@pytest.mark.parametrize("k,p_x,xdtype", [(4096, 0.5, torch.bfloat16), (1000, 0.3, torch.float32),
                                          (28672, 0.5, torch.bfloat16), (77, 0.9, torch.float32)])
def test_gemv_activation_ties(duo, k, p_x, xdtype):
    """Many equal magnitudes (and exact zeros) at the selection threshold:
    the calibration rule drops them in channel order."""
    say("dsc gemv ties", k, p_x, xdtype)
    n = 512
    W, keep = _layer(n, k, 0.5, k + 1, torch.bfloat16)
    comp = duo.dsc_compress(W.to(DEV), _mask_words(keep).to(DEV))
    g = torch.Generator().manual_seed(k)
    levels = torch.tensor([0.0, 0.5, 1.0, -1.0, 2.0, -0.5])
    x = levels[torch.randint(0, len(levels), (k,), generator=g)].to(xdtype)
    y = duo.dsc_gemv(comp, x.to(DEV), p_x).cpu().numpy().astype(np.float64)
    _check_gemv(y, W.float().numpy().astype(np.float64), x.float().numpy().astype(np.float64), p_x)
