"""Pins of the decoder-block reference (oracle/block_ref.py) against facts
that do not come from it: torch's bfloat16 rounding, the complex-number form
of the rotary embedding, causality and closed forms of attention, and the
zero-sparsity reduction of the two-stream block pruning (Sec. 4.2)."""

import numpy as np
import pytest
import torch

from oracle import block_ref as BR
from oracle import duo_ref as R
from workloads import synth


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def test_bf16_rounding_matches_torch():
    x = np.concatenate([_rand(20000, 0, 3.0), _rand(2000, 1, 1e-3), _rand(2000, 2, 1e4)])
    x32 = x.astype(np.float32).astype(np.float64)   # values torch can hold exactly as fp32
    ref = torch.tensor(x32, dtype=torch.float32).to(torch.bfloat16).double().numpy()
    assert np.array_equal(BR.bf16(x32), ref)
    # ties go to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    assert BR.bf16(1.0 + 2.0 ** -8) == 1.0
    assert BR.bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    assert BR.bf16(-(1.0 + 3 * 2.0 ** -8)) == -(1.0 + 2.0 ** -6)
    assert BR.bf16(0.0) == 0.0


def test_rmsnorm_unit_rms_and_scale_invariance():
    x = BR.bf16(_rand((7, 96), 3, 2.0))
    y = BR.rmsnorm(x, eps=0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=1)), 1.0, rtol=2 ** -7)
    assert np.array_equal(BR.rmsnorm(4.0 * x, eps=0.0), y)      # power-of-two scale is exact


def test_rope_is_complex_rotation():
    """Each pair (x_i, x_{i+d/2}) is multiplied by exp(i * pos * theta^(-2i/d))."""
    heads, hd, L = 3, 16, 5
    x = BR.bf16(_rand((2 * L, heads * hd), 4))
    y = BR.rope(x, heads, hd, L, theta=1e4)
    pos = np.arange(2 * L) % L
    for h in range(heads):
        z = x[:, h * hd:h * hd + hd // 2] + 1j * x[:, h * hd + hd // 2:(h + 1) * hd]
        w = z * np.exp(1j * pos[:, None] * 1e4 ** (-2.0 * np.arange(hd // 2) / hd))
        ref = np.concatenate([BR.bf16(w.real), BR.bf16(w.imag)], axis=1)
        assert np.allclose(y[:, h * hd:(h + 1) * hd], ref, rtol=2 ** -7, atol=1e-12)
    # position 0 is the identity
    assert np.array_equal(y[0], x[0]) and np.array_equal(y[L], x[L])


def test_attention_causal_and_closed_forms():
    nseq, L, heads, hd = 2, 6, 2, 8
    q, k, v = (BR.bf16(_rand((nseq * L, heads * hd), s)) for s in (5, 6, 7))
    o = BR.attention(q, k, v, nseq, L, heads, hd)
    # the first token of a sequence attends only to itself
    assert np.array_equal(o[0], BR.bf16(v[0])) and np.array_equal(o[L], BR.bf16(v[L]))
    # future tokens do not change earlier outputs
    k2, v2 = k.copy(), v.copy()
    k2[L - 1] += 5.0
    v2[L - 1] -= 3.0
    o2 = BR.attention(q, k2, v2, nseq, L, heads, hd)
    assert np.array_equal(o2[:L - 1], o[:L - 1]) and np.array_equal(o2[L:], o[L:])
    # equal scores: the output is the (bf16-rounded-weight) mean of the prefix values
    oz = BR.attention(np.zeros_like(q), k, v, nseq, L, heads, hd)
    for t in range(L):
        ref = BR.bf16(BR.bf16(np.full(t + 1, 1.0 / (t + 1))) @ v[:t + 1])
        assert np.array_equal(oz[t], ref)


def test_silu_mul_closed_forms():
    g = np.array([0.0, 30.0, -30.0, 1.0])
    u = np.array([5.0, 2.0, 2.0, 1.0])
    y = BR.silu_mul(g, u)
    assert y[0] == 0.0 and y[1] == 60.0 and abs(y[2]) < 1e-10
    assert y[3] == BR.bf16(1.0 / (1.0 + np.exp(-1.0)))


def _tiny():
    h, w = synth.block_inputs("tiny_block")
    h = h.float().numpy().astype(np.float64)
    w = {k: v.float().numpy().astype(np.float64) for k, v in w.items()}
    return h, w, synth.block_cfg("tiny_block"), synth.BLOCKS["tiny_block"]


def test_block_without_sparsity_keeps_weights_and_streams_equal():
    """p_x = p_w = 0: nothing is pruned, both streams coincide, every group's
    residual input is zero and the solver returns W bit-unchanged (Sec. 4.2
    with dX = 0 reduces to SparseGPT with nothing to prune)."""
    h, w, cfg, c = _tiny()
    out = BR.prune_block(h, w, cfg, 0.0, 0.0, damp=c["damp"], B=c["block"])
    for nm in synth.BLOCK_LINEARS:
        assert out["keep"][nm].all()
        assert np.array_equal(out["W_hat"][nm], w[nm])
    s, d = out["h3"]
    assert np.array_equal(s, d)
    for xs, xd in out["inputs"].values():
        assert np.array_equal(xs, xd)


def test_block_groups_share_inputs_and_counts():
    """Group members see the same two streams; every linear hits its exact
    prune count; the first group's streams coincide (same block input) while
    later groups' differ (pruning changed the sparse stream)."""
    h, w, cfg, c = _tiny()
    out = BR.prune_block(h, w, cfg, c["p_x"], c["p_w"], damp=c["damp"], B=c["block"])
    for nm in synth.BLOCK_LINEARS:
        n, k = w[nm].shape
        assert (~out["keep"][nm]).sum() == sum(R.block_prune_counts(n, k, c["p_w"], c["block"]))
    xs, xd = out["inputs"][("q", "k", "v")]
    assert np.array_equal(xs, xd)
    xs, xd = out["inputs"][("down",)]
    assert not np.array_equal(xs, xd)
    # the group solve equals a direct prune_layer on the recorded streams
    r = R.prune_layer(w["up"], *out["inputs"][("gate", "up")][:1], c["p_x"], c["p_w"], damp=c["damp"],
                      B=c["block"], X_dense=out["inputs"][("gate", "up")][1])
    assert np.array_equal(r["keep"], out["keep"]["up"])
