"""Seeded synthetic inputs shaped like the DuoGPT paper's calibration workloads.

This module only draws random numbers and lays them out.  It holds none of the
method's arithmetic, so both the oracle and the HIP path may use it.

The paper calibrates LLaMA-2/3 layers on 128 x 2048 tokens of C4 text (Sec. 5,
"Experimental setup").  Neither the text nor the trained weights are available
here; these generators stand in for them with the same shapes:

* weights: N(0, 0.02^2) per entry, stored in the layer's dtype;
* "lognormal" activations: x[t, c] = s_c * N(0, 1) with per-channel scales
  s_c = exp(sigma * N(0, 1)), optionally a few outlier channels scaled by 20
  (the heavy-tailed channel structure of LLM hidden states);
* "silu_gated" activations (the input of a down projection): x = SiLU(a) * b
  with a = s^a_c N(0,1), b = s^b_c N(0,1) and independent lognormal channel
  scales s^a, s^b.

Values are produced in fp32 and rounded once (round to nearest even) to the
storage dtype.  Generation runs on the requested device with torch's seeded
generator; the same seed and device always give the same bytes.
"""

from __future__ import annotations

import numpy as np
import torch

CONFIGS = {
    # tiny single linear layer, fp32, 2048 tokens
    "tiny_linear": dict(n=256, k=512, m=2048, w_dtype=torch.float32, x_dtype=torch.float32, kind="lognormal",
                        sigma=0.5, outliers=0, p_x=0.5, p_w=0.5, block=128, damp=0.01, seed=1000),
    # LLaMA-2-7B q_proj shape, 64 x 2048 tokens
    "llama2_7b_q_proj": dict(n=4096, k=4096, m=131072, w_dtype=torch.bfloat16, x_dtype=torch.bfloat16,
                             kind="lognormal", sigma=1.0, outliers=8, p_x=0.5, p_w=0.5, block=128, damp=0.01,
                             seed=2000),
    # LLaMA-2-7B down_proj shape
    "llama2_7b_down_proj": dict(n=4096, k=11008, m=131072, w_dtype=torch.bfloat16, x_dtype=torch.bfloat16,
                                kind="silu_gated", sigma=1.0, outliers=0, p_x=0.6, p_w=0.5, block=128, damp=0.01,
                                seed=3000),
    # LLaMA-2-70B down_proj shape
    "llama2_70b_down_proj": dict(n=8192, k=28672, m=131072, w_dtype=torch.bfloat16, x_dtype=torch.bfloat16,
                                 kind="silu_gated", sigma=1.0, outliers=0, p_x=0.5, p_w=0.6, block=128, damp=0.01,
                                 seed=5000),
}

_CHUNK = 8192


def channel_scales(k: int, sigma: float, outliers: int, seed: int) -> np.ndarray:
    """Per-channel scales exp(sigma * N(0,1)); `outliers` channels x 20."""
    rng = np.random.default_rng(seed)
    s = np.exp(sigma * rng.standard_normal(k))
    if outliers:
        s[rng.choice(k, min(outliers, k), replace=False)] *= 20.0
    return s.astype(np.float32)


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def make_weight(n: int, k: int, dtype=torch.bfloat16, seed: int = 0, device="cpu", std: float = 0.02):
    g = _gen(device, seed)
    w = torch.randn((n, k), generator=g, device=device, dtype=torch.float32) * std
    return w.to(dtype)


def make_activations(m: int, k: int, dtype=torch.bfloat16, seed: int = 0, device="cpu", kind: str = "lognormal",
                     sigma: float = 1.0, outliers: int = 0):
    """Token-major m x k activations (the transpose of the paper's X)."""
    X = torch.empty((m, k), dtype=dtype, device=device)
    g = _gen(device, seed + 1)
    if kind == "lognormal":
        s = torch.from_numpy(channel_scales(k, sigma, outliers, seed + 2)).to(device)
        for t0 in range(0, m, _CHUNK):
            t1 = min(m, t0 + _CHUNK)
            x = torch.randn((t1 - t0, k), generator=g, device=device, dtype=torch.float32) * s
            X[t0:t1] = x.to(dtype)
    elif kind == "silu_gated":
        sa = torch.from_numpy(channel_scales(k, sigma, 0, seed + 3)).to(device)
        sb = torch.from_numpy(channel_scales(k, sigma, 0, seed + 4)).to(device)
        for t0 in range(0, m, _CHUNK):
            t1 = min(m, t0 + _CHUNK)
            a = torch.randn((t1 - t0, k), generator=g, device=device, dtype=torch.float32) * sa
            b = torch.randn((t1 - t0, k), generator=g, device=device, dtype=torch.float32) * sb
            X[t0:t1] = (torch.nn.functional.silu(a) * b).to(dtype)
    else:
        raise ValueError(kind)
    return X


def layer_inputs(n, k, m, x_dtype=torch.bfloat16, w_dtype=torch.bfloat16, seed=0, device="cpu", kind="lognormal",
                 sigma=1.0, outliers=0):
    W = make_weight(n, k, w_dtype, seed=seed, device=device)
    X = make_activations(m, k, x_dtype, seed=seed + 10, device=device, kind=kind, sigma=sigma, outliers=outliers)
    return W, X


def config_inputs(name: str, device="cpu", m: int | None = None):
    c = CONFIGS[name]
    return layer_inputs(c["n"], c["k"], c["m"] if m is None else m, c["x_dtype"], c["w_dtype"], seed=c["seed"],
                        device=device, kind=c["kind"], sigma=c["sigma"], outliers=c["outliers"])


# LLaMA-style decoder blocks for the block harness: hidden size d, MLP width
# ffn, heads x head_dim attention, nseq sequences of seq_len tokens.  The
# block input has the lognormal channel structure (8 outlier channels x20 at
# full size); every weight is N(0, 0.02^2) in bf16.
BLOCKS = {
    # LLaMA-2-7B block shape on 128 x 2048 tokens
    "llama2_7b_block": dict(d=4096, ffn=11008, heads=32, head_dim=128, seq_len=2048, nseq=128, sigma=1.0,
                            outliers=8, p_x=0.5, p_w=0.5, block=128, damp=0.01, theta=1e4, eps=1e-5, seed=4000),
    # the same structure at a size the float64 oracle runs end to end
    "tiny_block": dict(d=128, ffn=352, heads=2, head_dim=64, seq_len=256, nseq=4, sigma=1.0, outliers=2,
                       p_x=0.5, p_w=0.5, block=32, damp=0.01, theta=1e4, eps=1e-5, seed=4100),
}

BLOCK_LINEARS = ("q", "k", "v", "o", "gate", "up", "down")


def block_shapes(c):
    d, f = c["d"], c["ffn"]
    return dict(q=(d, d), k=(d, d), v=(d, d), o=(d, d), gate=(f, d), up=(f, d), down=(d, f))


def block_inputs(name: str, device="cpu", nseq: int | None = None):
    """(h, weights) of a block workload; h is (nseq*seq_len) x d bf16."""
    c = BLOCKS[name]
    nseq = c["nseq"] if nseq is None else nseq
    h = make_activations(nseq * c["seq_len"], c["d"], torch.bfloat16, seed=c["seed"], device=device,
                         kind="lognormal", sigma=c["sigma"], outliers=c["outliers"])
    weights = {nm: make_weight(n, k, torch.bfloat16, seed=c["seed"] + 10 * (i + 1), device=device)
               for i, (nm, (n, k)) in enumerate(block_shapes(c).items())}
    return h, weights


def block_cfg(name: str, nseq: int | None = None):
    c = BLOCKS[name]
    return dict(heads=c["heads"], head_dim=c["head_dim"], seq_len=c["seq_len"],
                nseq=c["nseq"] if nseq is None else nseq, theta=c["theta"], eps=c["eps"])
