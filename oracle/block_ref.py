"""Float64 reference of the decoder-block harness: a LLaMA-style block carried
in two activation streams and pruned group by group with the layer oracle.

TEST INFRASTRUCTURE ONLY (like duo_ref): imported by tests only, shares no
code with the HIP path.

DuoGPT prunes a model layer by layer with two inputs per layer (Sec. 4.2,
multi-layer case): the dense model's activations X-tilde and the pruned
model's own activations, sparsified per token.  Within a LLaMA decoder block
(Sec. 5 evaluates LLaMA-2/3) the linears are pruned in groups that share one
Hessian: [q, k, v], then o, then [gate, up], then down; each group's two
streams are computed with the block's earlier groups already pruned.

Model (LLaMA-2 style, unit RMSNorm gains, no biases): x1 = rmsnorm(h);
q, k, v = x1 W^T; rotary embedding of q and k (rotate-half pairs (i, i+d/2),
angle = position * theta^(-2i/d)); causal softmax attention per sequence and
head; h2 = h + attn Wo^T; x2 = rmsnorm(h2); m = SiLU(x2 Wg^T) * (x2 Wu^T);
h3 = h2 + m Wd^T.  The sparse stream uses the pruned weights (rounded to
bf16) and sparsifies every linear input with the per-token rule.

Rounding points: activations are stored in bf16 after every operation
(round to nearest even, from the float64 value), and the attention
probabilities are rounded to bf16 before the product with V; the harness
stores them at exactly these points, so the reference mirrors them.  All
arithmetic between storage points is float64.
"""

from __future__ import annotations

import numpy as np

from . import duo_ref as R

GROUPS = (("q", "k", "v"), ("o",), ("gate", "up"), ("down",))


def bf16(x):
    """Round float64 values to the nearest bfloat16 (8 significant bits),
    ties to even; returned as float64."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m * 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0), e - 8)


def rmsnorm(x, eps=1e-5):
    x = np.asarray(x, dtype=np.float64)
    return bf16(x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + eps))


def linear(x, W, residual=None):
    y = np.asarray(x, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T
    if residual is not None:
        y = y + residual
    return bf16(y)


def rope(x, heads, head_dim, seq_len, theta=1e4):
    x = np.asarray(x, dtype=np.float64).copy()
    m = x.shape[0]
    half = head_dim // 2
    pos = (np.arange(m) % seq_len)[:, None].astype(np.float64)
    ang = pos * theta ** (-2.0 * np.arange(half) / head_dim)[None, :]
    c, s = np.cos(ang), np.sin(ang)
    for h in range(heads):
        a = x[:, h * head_dim:h * head_dim + half].copy()
        b = x[:, h * head_dim + half:(h + 1) * head_dim].copy()
        x[:, h * head_dim:h * head_dim + half] = a * c - b * s
        x[:, h * head_dim + half:(h + 1) * head_dim] = b * c + a * s
    return bf16(x)


def attention(q, k, v, nseq, seq_len, heads, head_dim):
    out = np.zeros((nseq * seq_len, heads * head_dim))
    causal = np.tril(np.ones((seq_len, seq_len), dtype=bool))
    for sq in range(nseq):
        rows = slice(sq * seq_len, (sq + 1) * seq_len)
        for h in range(heads):
            cols = slice(h * head_dim, (h + 1) * head_dim)
            S = q[rows, cols] @ k[rows, cols].T / np.sqrt(head_dim)
            S = np.where(causal, S, -np.inf)
            P = np.exp(S - S.max(axis=1, keepdims=True))
            P = bf16(P / P.sum(axis=1, keepdims=True))
            out[rows, cols] = P @ v[rows, cols]
    return bf16(out)


def silu_mul(g, u):
    g = np.asarray(g, dtype=np.float64)
    return bf16(g / (1.0 + np.exp(-g)) * u)


def sparsify(x, p_x):
    return R.sparsify_tokens(x, p_x)[0]


def prune_block(h, weights, cfg, p_x, p_w, damp=0.01, B=128):
    """Prune one decoder block group by group.

    h: token-major block input (bf16 values), shared by both streams.
    weights: dict name -> W (n x k, bf16 values) for q, k, v, o, gate, up, down.
    cfg: dict(heads, head_dim, seq_len, nseq, theta, eps).
    Returns dict(W_hat, keep, bf16 pruned weights, group inputs of both
    streams, and the block outputs h3 of both streams).
    """
    H, D_, L, S_, th, eps = (cfg["heads"], cfg["head_dim"], cfg["seq_len"], cfg["nseq"], cfg["theta"],
                             cfg["eps"])
    out = dict(W_hat={}, keep={}, W_lowp={}, inputs={})

    def group(names, x_sparse, x_dense):
        out["inputs"][names] = (x_sparse, x_dense)
        for nm in names:
            r = R.prune_layer(weights[nm], x_sparse, p_x, p_w, damp=damp, B=B, X_dense=x_dense)
            out["W_hat"][nm] = r["W_hat"]
            out["keep"][nm] = r["keep"]
            out["W_lowp"][nm] = bf16(r["W_hat"])

    def both(x_s, x_d, nm, res_s=None, res_d=None):
        return (linear(sparsify(x_s, p_x), out["W_lowp"][nm], res_s),
                linear(x_d, weights[nm], res_d))

    hs = hd = np.asarray(h, dtype=np.float64)
    x1s, x1d = rmsnorm(hs, eps), rmsnorm(hd, eps)
    group(("q", "k", "v"), x1s, x1d)
    qs, qd = both(x1s, x1d, "q")
    ks, kd = both(x1s, x1d, "k")
    vs, vd = both(x1s, x1d, "v")
    qs, qd, ks, kd = (rope(t, H, D_, L, th) for t in (qs, qd, ks, kd))
    a_s = attention(qs, ks, vs, S_, L, H, D_)
    a_d = attention(qd, kd, vd, S_, L, H, D_)
    group(("o",), a_s, a_d)
    h2s, h2d = both(a_s, a_d, "o", hs, hd)
    x2s, x2d = rmsnorm(h2s, eps), rmsnorm(h2d, eps)
    group(("gate", "up"), x2s, x2d)
    gs, gd = both(x2s, x2d, "gate")
    us, ud = both(x2s, x2d, "up")
    ms, md = silu_mul(gs, us), silu_mul(gd, ud)
    group(("down",), ms, md)
    out["h3"] = both(ms, md, "down", h2s, h2d)
    return out
