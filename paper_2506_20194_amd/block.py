"""Prune one LLaMA-style decoder block group by group on the device.

Two activation streams run through the block (the multi-layer case of
Sec. 4.2): the dense stream (dense weights, no activation sparsity) and the
sparse stream (the block's pruned weights, every linear input sparsified per
token).  The linears are pruned in groups that share one Hessian -- [q, k, v],
then o, then [gate, up], then down -- and each group's solver input is the
pair (sparse stream, dense stream) at that point, computed with the earlier
groups already pruned.  Every step runs in libduo's own kernels (the block's
products included: bf16 MFMA linears and causal attention); this module only
sequences the calls.
"""

from __future__ import annotations

import torch

from . import duo

GROUPS = (("q", "k", "v"), ("o",), ("gate", "up"), ("down",))


def _event(stream):
    e = torch.cuda.Event(enable_timing=True)
    e.record(stream)
    return e


def prune_block(h, weights, cfg, p_x, p_w, damp=0.01, block=128, keep_inputs=False, timing=False):
    """h: (nseq*seq_len) x d bf16 block input (both streams start from it).
    weights: dict name -> n x k bf16 tensor for q, k, v, o, gate, up, down.
    cfg: dict(heads, head_dim, seq_len, nseq, theta, eps).
    Returns dict(W_out fp32, W_lowp bf16, mask (packed words), lam per group,
    h3 = (sparse, dense) block outputs, optional group inputs and per-phase
    device milliseconds when timing=True)."""
    dev = h.device
    stream = torch.cuda.current_stream(dev)
    heads, hd, L, nseq = cfg["heads"], cfg["head_dim"], cfg["seq_len"], cfg["nseq"]
    theta, eps = cfg["theta"], cfg["eps"]
    m = h.shape[0]
    if m != nseq * L:
        raise ValueError("prune_block: h must hold nseq * seq_len tokens")
    ws_lin = duo.block_workspace(duo.DUO_BOP_LINEAR, 0, 0, 0, dev)
    ws_att = duo.block_workspace(duo.DUO_BOP_ATTENTION, 0, L, heads, dev)
    ws_act = duo.block_workspace(duo.DUO_BOP_ACT_SPARSIFY, m, 0, 0, dev)
    out = dict(W_out={}, W_lowp={}, mask={}, lam={}, inputs={}, ms={})
    marks = []

    def mark(name):
        if timing:
            marks.append((name, _event(stream)))

    def group(names, xs, xd):
        k = xs.shape[1]
        H = torch.zeros((k, k), dtype=torch.float32, device=dev)
        G = torch.zeros((k, k), dtype=torch.float32, device=dev)
        a = torch.zeros(k, dtype=torch.float32, device=dev)
        duo.duo_hessian_accum(xs, H, p_x, X_dense=xd, G=G, a=a)
        lam, fail = duo.duo_chol_inv(H, damp, sync=True)
        if fail != -1:
            raise duo.DuoError(duo.DUO_ERR_NOT_PD, f"prune_block group {names}")
        out["lam"][names] = lam
        if keep_inputs:
            out["inputs"][names] = (xs, xd)
        for nm in names:
            W = weights[nm]
            W_out, lowp, mask, _ = duo.duo_prune_layer(W, H, G, a, p_w, block, want_lowp=True)
            out["W_out"][nm], out["W_lowp"][nm], out["mask"][nm] = W_out, lowp, mask
        del H, G, a

    def both(xs, xd, nm, rs=None, rd=None):
        x_hat = duo.duo_act_sparsify(xs, p_x, ws=ws_act)
        ys = duo.duo_linear(x_hat, out["W_lowp"][nm], R=rs, ws=ws_lin)
        del x_hat
        yd = duo.duo_linear(xd, weights[nm], R=rd, ws=ws_lin)
        return ys, yd

    mark("start")
    x1s = duo.duo_rmsnorm(h, eps)
    x1d = x1s.clone()          # both streams start from the same block input
    mark("forward")
    group(("q", "k", "v"), x1s, x1d)
    mark("solve_qkv")
    qs, qd = both(x1s, x1d, "q")
    ks, kd = both(x1s, x1d, "k")
    vs, vd = both(x1s, x1d, "v")
    if not keep_inputs:
        del x1s, x1d
    for t in (qs, qd, ks, kd):
        duo.duo_rope(t, heads, hd, L, theta)
    a_s = duo.duo_attention(qs, ks, vs, nseq, L, heads, hd, ws=ws_att)
    a_d = duo.duo_attention(qd, kd, vd, nseq, L, heads, hd, ws=ws_att)
    del qs, qd, ks, kd, vs, vd
    mark("forward")
    group(("o",), a_s, a_d)
    mark("solve_o")
    h2s, h2d = both(a_s, a_d, "o", h, h)
    if not keep_inputs:
        del a_s, a_d
    x2s, x2d = duo.duo_rmsnorm(h2s, eps), duo.duo_rmsnorm(h2d, eps)
    mark("forward")
    group(("gate", "up"), x2s, x2d)
    mark("solve_gate_up")
    gs, gd = both(x2s, x2d, "gate")
    us, ud = both(x2s, x2d, "up")
    if not keep_inputs:
        del x2s, x2d
    ms, md = duo.duo_silu_mul(gs, us), duo.duo_silu_mul(gd, ud)
    del gs, gd, us, ud
    mark("forward")
    group(("down",), ms, md)
    mark("solve_down")
    out["h3"] = both(ms, md, "down", h2s, h2d)
    mark("forward")
    if timing:
        torch.cuda.synchronize(dev)
        for (_, e0), (name, e1) in zip(marks[:-1], marks[1:]):
            out["ms"][name] = out["ms"].get(name, 0.0) + e0.elapsed_time(e1)
    return out
