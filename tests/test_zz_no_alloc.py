"""The allocation-free decode GEMV (duo_dsc_gemv_noalloc) through the C ABI:
bit-identical to duo_dsc_gemv (same kernels, same partition of the work,
fixed summation order), on two calls in a row with the second one smaller,
so a stale partial from the first call would show; and its size limit is an
error returned on the host."""

import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def say(*a):
    print("[case]", *a, flush=True)


def _layer(duo, n, k, seed):
    g = torch.Generator().manual_seed(seed)
    keep = torch.rand((n, k), generator=g) < 0.45
    W = torch.where(keep, (0.02 * torch.randn((n, k), generator=g)).to(torch.bfloat16),
                    torch.zeros((), dtype=torch.bfloat16))
    words = (k + 31) // 32
    pad = np.zeros((n, words * 32), dtype=np.uint64)
    pad[:, :k] = keep.numpy()
    mw = (pad.reshape(n, words, 32) << np.arange(32, dtype=np.uint64)).sum(-1).astype(np.uint32).view(np.int32)
    comp = duo.dsc_compress(W.to(DEV), torch.tensor(mw).to(DEV))
    x = (torch.randn(k, generator=g) * torch.exp(torch.randn(k, generator=g))).to(torch.bfloat16)
    return comp, x.to(DEV)


def test_noalloc_gemv_matches_workspace_gemv(duo_lib):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    duo = duo_lib
    # large first (every partial row of the array in use), then smaller
    for n, k, p_x, seed in ((8192, 28672, 0.5, 1), (300, 70, 0.6, 2), (4096, 4096, 0.5, 3), (65, 33, 0.0, 4)):
        say("noalloc gemv", n, k, p_x)
        comp, x = _layer(duo, n, k, seed)
        ref = duo.dsc_gemv(comp, x, p_x)
        y = torch.full((n,), float("nan"), dtype=torch.float32, device=DEV)
        duo.dsc_gemv_noalloc(comp, x, p_x, out=y)
        torch.cuda.synchronize()
        assert torch.equal(y, ref), (n, k, float((y - ref).abs().max()))
        # and again on the same inputs: the array keeps nothing that matters
        y2 = duo.dsc_gemv_noalloc(comp, x, p_x)
        assert torch.equal(y2, ref)


def test_noalloc_gemv_rejects_sizes_beyond_its_limit(duo_lib):
    """n > 32768 is refused on the host, before any launch."""
    duo = duo_lib
    L = duo.lib()
    dummy = torch.zeros(16, dtype=torch.int64, device=DEV)
    p = ctypes.c_void_p(dummy.data_ptr())
    st = L.duo_dsc_gemv_noalloc(p, duo.DUO_BF16, 32769, 8, duo.act_rule(0.5), p, p, p, p, p, None)
    assert st == duo.DUO_ERR_UNSUPPORTED
    st = L.duo_dsc_gemv_noalloc(p, duo.DUO_BF16, 64, 32769, duo.act_rule(0.5), p, p, p, p, p, None)
    assert st == duo.DUO_ERR_UNSUPPORTED
    st = L.duo_dsc_gemv_noalloc(None, duo.DUO_BF16, 64, 8, duo.act_rule(0.5), p, p, p, p, p, None)
    assert st == duo.DUO_ERR_INVALID_ARG
