"""Host-side checks of the C ABI (no GPU needed): every symbol declared in
include/duo.h is exported, workspace sizes are sane, and argument errors are
rejected before any device work (a call with valid arguments reports
DUO_ERR_NO_DEVICE here, proving it got past validation)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "duo.h")
FAKE = ctypes.c_void_p(1 << 20)      # never dereferenced on the host
WS = ctypes.c_void_p(256 << 20)      # 256-byte aligned fake workspace


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(duo_[a-z_]+)\s*\(", text)))


def test_header_declares_the_named_entry_points():
    names = declared_functions()
    for n in ("duo_hessian_accum", "duo_residual_term", "duo_chol_inv", "duo_prune_layer"):
        assert n in names


def test_every_declared_symbol_is_exported(duo_lib):
    L = duo_lib.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
    assert set(duo_lib.EXPORTED) == set(declared_functions())


def test_status_strings_and_version(duo_lib):
    for s in range(8):
        assert duo_lib.status_string(s) not in ("", "unknown status")
    assert duo_lib.status_string(99) == "unknown status"
    assert "gfx950" in duo_lib.version()


def test_workspace_sizes(duo_lib):
    ws = duo_lib.duo_workspace_size
    assert ws(duo_lib.DUO_OP_HESSIAN, 0, 512, 2048, 0) > 0
    assert ws(duo_lib.DUO_OP_HESSIAN, 0, 4096, 131072, 0) >= ws(duo_lib.DUO_OP_HESSIAN, 0, 4096, 1024, 0)
    assert ws(duo_lib.DUO_OP_CHOL_INV, 0, 4096, 0, 0) >= 4096 * 4096 // 4 * 4
    assert ws(duo_lib.DUO_OP_PRUNE_LAYER, 4096, 4096, 0, 128) > ws(duo_lib.DUO_OP_SWEEP, 4096, 4096, 0, 128)
    assert ws(duo_lib.DUO_OP_SWEEP, 16, 16, 0, 0) == 0          # bad block
    assert ws(duo_lib.DUO_OP_SWEEP, 16, 16, 0, 129) == 0
    assert ws(duo_lib.DUO_OP_CHOL_INV, 0, 0, 0, 0) == 0         # bad k
    assert ws(duo_lib.DUO_OP_CHOL_INV, 0, 40000, 0, 0) == 0     # beyond the k limit
    assert ws(99, 1, 1, 1, 1) == 0


def _rule(p=0.5, kind=1):
    from paper_2506_20194_amd.duo import ActRule

    return ActRule(kind, p)


def test_hessian_argument_errors(duo_lib):
    L = duo_lib.lib()
    E, NODEV = duo_lib.DUO_ERR_INVALID_ARG, duo_lib.DUO_ERR_NO_DEVICE
    big = 10 ** 10

    def call(X=FAKE, Xd=None, dt=1, m=64, k=32, ldx=32, rule=None, H=FAKE, ldh=32, G=None, ldg=32, a=None, ws=WS,
             wsb=big, hdiag=None, gp=0):
        return L.duo_hessian_accum(X, Xd, dt, m, k, ldx, rule or _rule(), H, ldh, G, ldg, gp, a, hdiag, ws, wsb, None)

    assert call() == NODEV
    assert call(X=None) == E
    assert call(H=None) == E
    assert call(dt=7) == E
    assert call(m=-1) == E
    assert call(k=0) == E
    assert call(k=40000, ldx=40000, ldh=40000) == duo_lib.DUO_ERR_UNSUPPORTED
    assert call(ldx=31) == E
    assert call(ldh=31) == E
    assert call(G=FAKE) == E                     # G without a
    assert call(G=FAKE, a=FAKE, ldg=8) == E
    assert call(rule=_rule(1.5)) == E
    assert call(rule=_rule(float("nan"))) == E
    assert call(rule=_rule(0.5, kind=9)) == E
    assert call(ws=None) == duo_lib.DUO_ERR_WORKSPACE
    assert call(wsb=16) == duo_lib.DUO_ERR_WORKSPACE
    assert call(ws=ctypes.c_void_p((256 << 20) + 8)) == duo_lib.DUO_ERR_WORKSPACE
    assert call(m=0) == duo_lib.DUO_OK           # nothing to do, nothing enqueued
    assert call(hdiag=FAKE) == NODEV
    assert call(G=FAKE, a=FAKE, gp=1) == NODEV   # all of G
    assert call(G=FAKE, a=FAKE, gp=2) == E       # no such G part
    assert L.duo_residual_term(None, None, 1, 64, 32, 32, _rule(), FAKE, 32, 0, FAKE, WS, big, None) == E
    assert L.duo_residual_term(FAKE, None, 1, 64, 32, 32, _rule(), FAKE, 32, 0, FAKE, WS, big, None) == NODEV
    assert L.duo_residual_term(FAKE, None, 1, 64, 32, 32, _rule(), FAKE, 32, 1, FAKE, WS, big, None) == NODEV
    assert L.duo_residual_term(FAKE, None, 1, 64, 32, 32, _rule(), FAKE, 32, 2, FAKE, WS, big, None) == E


def test_chol_and_sweep_argument_errors(duo_lib):
    L = duo_lib.lib()
    E, NODEV = duo_lib.DUO_ERR_INVALID_ARG, duo_lib.DUO_ERR_NO_DEVICE
    big = 10 ** 10
    assert L.duo_chol_inv(FAKE, 64, 64, 0.01, None, WS, big, None) == NODEV
    assert L.duo_chol_inv(None, 64, 64, 0.01, None, WS, big, None) == E
    assert L.duo_chol_inv(FAKE, 64, 63, 0.01, None, WS, big, None) == E
    assert L.duo_chol_inv(FAKE, 64, 64, -1.0, None, WS, big, None) == E
    assert L.duo_chol_inv(FAKE, 64, 64, float("inf"), None, WS, big, None) == E
    assert L.duo_chol_inv(FAKE, 64, 64, 0.01, None, WS, 8, None) == duo_lib.DUO_ERR_WORKSPACE
    assert L.duo_score_terms(FAKE, 64, FAKE, 64, FAKE, 64, FAKE, 64, FAKE, WS, big, None) == NODEV
    assert L.duo_score_terms(FAKE, 64, None, 64, FAKE, 64, FAKE, 64, FAKE, WS, big, None) == E

    from paper_2506_20194_amd.duo import SweepOpts

    def sweep(W=FAKE, dt=1, n=32, k=64, ldw=64, p=0.5, B=16, Wo=FAKE, fn=L.duo_sweep, nm=0, qb=0, qg=0, form=0):
        o = ctypes.byref(SweepOpts(nm, qb, qg, None, None, form)) if (nm or qb or qg or form) else None
        return fn(W, dt, n, k, ldw, FAKE, 64, FAKE, 64, FAKE, p, o, B, None, Wo, None, None, None, WS, big, None)

    # residual form: 0 automatic, 1 D, 2 Y (duo_prune_layer only; with quantisation only for q_group == block)
    assert sweep(form=1) == NODEV
    assert sweep(form=2) == E
    assert sweep(form=3) == E
    assert sweep(form=-1) == E
    P = L.duo_prune_layer
    assert sweep(fn=P, form=1) == NODEV
    assert sweep(fn=P, form=2) == NODEV
    assert sweep(fn=P, form=3) == E
    assert sweep(fn=P, form=2, nm=2) == NODEV
    assert sweep(fn=P, form=2, qb=4, qg=16, B=32) == duo_lib.DUO_ERR_UNSUPPORTED  # groups inside a block
    assert sweep(fn=P, form=2, qb=4, qg=16, B=16) == NODEV  # one grid per row and block

    for fn in (L.duo_sweep, L.duo_prune_layer):
        assert sweep(fn=fn) == NODEV
        assert sweep(W=None, fn=fn) == E
        assert sweep(Wo=None, fn=fn) == E
        assert sweep(n=0, fn=fn) == E
        assert sweep(ldw=60, fn=fn) == E
        assert sweep(p=-0.1, fn=fn) == E
        assert sweep(p=1.01, fn=fn) == E
        assert sweep(B=0, fn=fn) == E
        assert sweep(B=129, fn=fn) == E
        assert sweep(dt=3, fn=fn) == E
        assert sweep(nm=2, fn=fn) == NODEV         # N:4 with k, B multiples of 4
        assert sweep(nm=5, fn=fn) == E
        assert sweep(nm=-1, fn=fn) == E
        assert sweep(nm=2, B=18, fn=fn) == E       # B not a multiple of 4
        assert sweep(nm=2, k=62, ldw=64, fn=fn) == E
        assert sweep(qb=4, qg=16, fn=fn) == NODEV  # quantisation grids of 16 columns in blocks of 16
        assert sweep(qb=4, qg=16, B=32, nm=2, fn=fn) == NODEV
        assert sweep(qb=1, qg=16, fn=fn) == E      # bits outside 2..8
        assert sweep(qb=9, qg=16, fn=fn) == E
        assert sweep(qb=4, qg=24, B=48, fn=fn) == E   # group not 16/32/64/128
        assert sweep(qb=4, qg=32, B=16, fn=fn) == E   # group does not divide the block
        assert sweep(qg=7, fn=fn) == NODEV         # the group is ignored without bits


def test_binding_refuses_host_tensors(duo_lib):
    import torch

    H = torch.zeros((8, 8))
    with pytest.raises(ValueError):
        duo_lib.duo_chol_inv(H, 0.01, ws=torch.zeros(1 << 20, dtype=torch.uint8))
    with pytest.raises(ValueError):
        duo_lib.prune_linear(torch.zeros(4, 8), torch.zeros(16, 8), 0.5, 0.5)


def test_block_harness_argument_errors(duo_lib):
    """The decoder-block calls validate before touching the device."""
    L = duo_lib.lib()
    E, W_, NODEV = duo_lib.DUO_ERR_INVALID_ARG, duo_lib.DUO_ERR_WORKSPACE, duo_lib.DUO_ERR_NO_DEVICE
    UNS = duo_lib.DUO_ERR_UNSUPPORTED
    big = 10 ** 12
    assert L.duo_rmsnorm(FAKE, 8, 64, 64, 1e-5, FAKE, 64, None) == NODEV
    assert L.duo_rmsnorm(FAKE, 8, 64, 63, 1e-5, FAKE, 64, None) == E
    assert L.duo_rmsnorm(None, 8, 64, 64, 1e-5, FAKE, 64, None) == E
    assert L.duo_rmsnorm(FAKE, 8, 64, 64, -1.0, FAKE, 64, None) == E
    assert L.duo_rmsnorm(None, 0, 64, 64, 1e-5, None, 64, None) == duo_lib.DUO_OK   # nothing to do
    assert L.duo_act_sparsify(FAKE, 8, 64, 64, _rule(), FAKE, 64, WS, big, None) == NODEV
    assert L.duo_act_sparsify(FAKE, 8, 64, 64, _rule(1.5), FAKE, 64, WS, big, None) == E
    assert L.duo_act_sparsify(FAKE, 8, 64, 64, _rule(), FAKE, 64, WS, 4, None) == W_
    assert L.duo_act_sparsify(FAKE, 8, 40000, 40000, _rule(), FAKE, 40000, WS, big, None) == E
    assert L.duo_linear(FAKE, 8, 64, 64, FAKE, 32, 64, None, 0, FAKE, 32, WS, big, None) == NODEV
    assert L.duo_linear(FAKE, 8, 64, 64, FAKE, 32, 63, None, 0, FAKE, 32, WS, big, None) == E
    assert L.duo_linear(FAKE, 8, 64, 64, FAKE, 32, 64, FAKE, 31, FAKE, 32, WS, big, None) == E
    # no scratch memory: a NULL workspace is fine
    assert L.duo_block_workspace_size(duo_lib.DUO_BOP_LINEAR, 0, 0, 0) == 0
    assert L.duo_linear(FAKE, 8, 64, 64, FAKE, 32, 64, None, 0, FAKE, 32, None, 0, None) == NODEV
    assert L.duo_rope(FAKE, 8, 2, 64, 128, 4, 1e4, None) == NODEV
    assert L.duo_rope(FAKE, 8, 2, 63, 128, 4, 1e4, None) == E          # odd head_dim
    assert L.duo_rope(FAKE, 8, 2, 64, 127, 4, 1e4, None) == E
    assert L.duo_rope(FAKE, 8, 2, 64, 128, 4, 0.0, None) == E
    assert L.duo_block_workspace_size(duo_lib.DUO_BOP_ATTENTION, 0, 16, 2) == 0
    assert L.duo_attention(FAKE, FAKE, FAKE, 128, 2, 16, 2, 64, FAKE, 128, None, 0, None) == NODEV
    assert L.duo_attention(FAKE, FAKE, FAKE, 127, 2, 16, 2, 64, FAKE, 128, None, 0, None) == E
    assert L.duo_attention(FAKE, FAKE, FAKE, 192, 2, 16, 2, 96, FAKE, 192, None, 0, None) == UNS  # head_dim
    assert L.duo_attention(FAKE, FAKE, FAKE, 132, 2, 16, 2, 64, FAKE, 128, None, 0, None) == UNS  # ld % 8
    assert L.duo_silu_mul(FAKE, FAKE, 8, 64, 64, FAKE, 64, None) == NODEV
    assert L.duo_silu_mul(FAKE, FAKE, 8, 64, 32, FAKE, 64, None) == E
    assert L.duo_block_workspace_size(99, 1, 1, 1) == 0
    assert L.duo_block_workspace_size(duo_lib.DUO_BOP_ACT_SPARSIFY, 100, 0, 0) >= 800


def test_act_order_argument_errors(duo_lib):
    L = duo_lib.lib()
    E, NODEV = duo_lib.DUO_ERR_INVALID_ARG, duo_lib.DUO_ERR_NO_DEVICE
    assert L.duo_act_order(FAKE, 64, FAKE, None, None) == NODEV
    assert L.duo_act_order(None, 64, FAKE, None, None) == E
    assert L.duo_act_order(FAKE, 64, None, None, None) == E
    assert L.duo_act_order(FAKE, 0, FAKE, None, None) == E
    assert L.duo_act_order(FAKE, 40000, FAKE, None, None) == duo_lib.DUO_ERR_UNSUPPORTED
    OTHER = ctypes.c_void_p(FAKE.value + (1 << 20))

    def perm(src=FAKE, dt=0, sr=8, sc=16, lds=16, ri=None, ci=None, r=8, c=16, dst=OTHER, ldd=16):
        return L.duo_permute(src, dt, sr, sc, lds, ri, ci, r, c, dst, ldd, None)

    assert perm() == NODEV
    assert perm(ri=FAKE, ci=FAKE, r=100, c=100, ldd=100) == NODEV  # gathers may change the shape
    assert perm(dt=5) == E
    assert perm(lds=15) == E
    assert perm(ldd=15) == E
    assert perm(r=9) == E                      # more rows than the source without an index
    assert perm(c=17, ldd=17) == E
    assert perm(dst=FAKE) == E                 # in place
    assert perm(src=None) == E
    assert perm(r=0) == duo_lib.DUO_OK
    assert perm(ri=FAKE, r=70000) == duo_lib.DUO_ERR_UNSUPPORTED
    assert L.duo_permute_mask(FAKE, 8, 64, FAKE, OTHER, None) == NODEV
    assert L.duo_permute_mask(FAKE, 8, 64, None, OTHER, None) == E
    assert L.duo_permute_mask(FAKE, 8, 64, FAKE, FAKE, None) == E
    assert L.duo_permute_mask(FAKE, -1, 64, FAKE, OTHER, None) == E
    assert L.duo_permute_mask(FAKE, 0, 64, FAKE, OTHER, None) == duo_lib.DUO_OK


def test_decode_argument_errors(duo_lib):
    L = duo_lib.lib()
    E, NODEV = duo_lib.DUO_ERR_INVALID_ARG, duo_lib.DUO_ERR_NO_DEVICE
    ws = L.duo_dsc_workspace_size(4096, 4096)
    assert ws >= 4096 * 8 and L.duo_dsc_workspace_size(70000, 16) == 0 and L.duo_dsc_workspace_size(0, 16) == 0
    big = 10 ** 10
    assert L.duo_dsc_layout(FAKE, 64, 32, FAKE, FAKE, FAKE, WS, big, None) == NODEV
    assert L.duo_dsc_layout(None, 64, 32, FAKE, FAKE, FAKE, WS, big, None) == E
    assert L.duo_dsc_layout(FAKE, 0, 32, FAKE, FAKE, FAKE, WS, big, None) == E
    assert L.duo_dsc_layout(FAKE, 70000, 32, FAKE, FAKE, FAKE, WS, big, None) == duo_lib.DUO_ERR_UNSUPPORTED
    assert L.duo_dsc_layout(FAKE, 64, 32, FAKE, FAKE, FAKE, WS, 8, None) == duo_lib.DUO_ERR_WORKSPACE
    assert L.duo_dsc_pack(FAKE, 1, 64, 32, 32, FAKE, FAKE, FAKE, FAKE, None) == NODEV
    assert L.duo_dsc_pack(FAKE, 1, 64, 32, 31, FAKE, FAKE, FAKE, FAKE, None) == E
    assert L.duo_dsc_pack(FAKE, 4, 64, 32, 32, FAKE, FAKE, FAKE, FAKE, None) == E
    assert L.duo_dsc_gemv(FAKE, 1, 64, 32, _rule(), FAKE, FAKE, FAKE, FAKE, FAKE, WS, big, None) == NODEV
    assert L.duo_dsc_gemv(FAKE, 1, 64, 32, _rule(1.5), FAKE, FAKE, FAKE, FAKE, FAKE, WS, big, None) == E
    assert L.duo_dsc_gemv(FAKE, 1, 64, 32, _rule(), FAKE, FAKE, FAKE, None, FAKE, WS, big, None) == E
    assert L.duo_dsc_gemv(FAKE, 1, 64, 32, _rule(), FAKE, FAKE, FAKE, FAKE, FAKE, WS, 16, None) == \
        duo_lib.DUO_ERR_WORKSPACE
