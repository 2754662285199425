"""Thin Python binding of libduo.so (the gfx950 DuoGPT layer solver).

The functions carry the names of the C entry points in include/duo.h and only
marshal arguments: tensors become device pointers, the current torch stream
becomes the HIP stream, workspaces are allocated from torch's caching
allocator.  Every computation happens in the HIP library; if the library is
missing or no gfx950 device is present the calls raise.
"""

from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libduo.so")

DUO_OK, DUO_ERR_INVALID_ARG, DUO_ERR_UNSUPPORTED, DUO_ERR_WORKSPACE = 0, 1, 2, 3
DUO_ERR_NOT_PD, DUO_ERR_NONFINITE, DUO_ERR_HIP, DUO_ERR_NO_DEVICE = 4, 5, 6, 7
DUO_F32, DUO_BF16 = 0, 1
DUO_ACT_NONE, DUO_ACT_TOPK_MAG_PER_TOKEN = 0, 1
DUO_OP_HESSIAN, DUO_OP_CHOL_INV, DUO_OP_SCORE_TERMS, DUO_OP_SWEEP, DUO_OP_PRUNE_LAYER = 0, 1, 2, 3, 4
DUO_G_UPPER, DUO_G_FULL = 0, 1

EXPORTED = (
    "duo_workspace_size", "duo_status_string", "duo_version", "duo_act_sparsify_mask",
    "duo_hessian_accum", "duo_residual_term", "duo_chol_inv", "duo_score_terms", "duo_sweep",
    "duo_prune_layer", "duo_profile_enable", "duo_profile_read", "duo_block_workspace_size", "duo_rmsnorm",
    "duo_act_sparsify", "duo_linear", "duo_rope", "duo_attention", "duo_silu_mul", "duo_act_order",
    "duo_permute", "duo_permute_mask", "duo_dsc_workspace_size", "duo_dsc_layout", "duo_dsc_pack",
    "duo_dsc_gemv", "duo_dsc_gemv_noalloc", "duo_hessian_status",
)
PROF = dict(gram=0, hessian=1, chol=2, score=3, sweep=4, inblock=5, trail=6, select=7, decode=8)
DUO_BOP_ACT_SPARSIFY, DUO_BOP_LINEAR, DUO_BOP_ATTENTION = 0, 1, 2


class DuoError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


class ActRule(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("sparsity", ctypes.c_double)]


class SweepOpts(ctypes.Structure):
    _fields_ = [("nm_n", ctypes.c_int32), ("q_bits", ctypes.c_int32), ("q_group", ctypes.c_int32),
                ("q_scale_out", ctypes.c_void_p), ("q_zero_out", ctypes.c_void_p),
                ("residual_form", ctypes.c_int32)]


# residual_form of duo_prune_layer: None / "auto", "d", "y"
FORMS = {None: 0, "auto": 0, "d": 1, "y": 2}


class CholInfo(ctypes.Structure):
    _fields_ = [("lam", ctypes.c_double), ("fail_index", ctypes.c_int64), ("status", ctypes.c_int32)]


_lib = None
P = ctypes.c_void_p
I64 = ctypes.c_int64
I32 = ctypes.c_int32
F64 = ctypes.c_double
SZ = ctypes.c_size_t


def lib():
    """The loaded library (raises when libduo.so has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.duo_workspace_size.restype = SZ
        L.duo_workspace_size.argtypes = [I32, I64, I64, I64, I32]
        L.duo_status_string.restype = ctypes.c_char_p
        L.duo_status_string.argtypes = [I32]
        L.duo_version.restype = ctypes.c_char_p
        L.duo_version.argtypes = []
        L.duo_act_sparsify_mask.restype = I32
        L.duo_act_sparsify_mask.argtypes = [P, I32, I64, I64, I64, ActRule, P, P, SZ, P]
        L.duo_hessian_accum.restype = I32
        L.duo_hessian_accum.argtypes = [P, P, I32, I64, I64, I64, ActRule, P, I64, P, I64, I32, P, P, P, SZ, P]
        L.duo_hessian_status.restype = I32
        L.duo_hessian_status.argtypes = [P, SZ, P]
        L.duo_residual_term.restype = I32
        L.duo_residual_term.argtypes = [P, P, I32, I64, I64, I64, ActRule, P, I64, I32, P, P, SZ, P]
        L.duo_chol_inv.restype = I32
        L.duo_chol_inv.argtypes = [P, I64, I64, F64, ctypes.POINTER(CholInfo), P, SZ, P]
        L.duo_score_terms.restype = I32
        L.duo_score_terms.argtypes = [P, I64, P, I64, P, I64, P, I64, P, P, SZ, P]
        L.duo_sweep.restype = I32
        L.duo_sweep.argtypes = [P, I32, I64, I64, I64, P, I64, P, I64, P, F64, ctypes.POINTER(SweepOpts), I32, P, P,
                                P, P, P, P, SZ, P]
        L.duo_prune_layer.restype = I32
        L.duo_prune_layer.argtypes = [P, I32, I64, I64, I64, P, I64, P, I64, P, F64, ctypes.POINTER(SweepOpts), I32,
                                      P, P, P, P, P, P, SZ, P]
        L.duo_block_workspace_size.restype = SZ
        L.duo_block_workspace_size.argtypes = [I32, I64, I64, I64]
        L.duo_rmsnorm.restype = I32
        L.duo_rmsnorm.argtypes = [P, I64, I64, I64, F64, P, I64, P]
        L.duo_act_sparsify.restype = I32
        L.duo_act_sparsify.argtypes = [P, I64, I64, I64, ActRule, P, I64, P, SZ, P]
        L.duo_linear.restype = I32
        L.duo_linear.argtypes = [P, I64, I64, I64, P, I64, I64, P, I64, P, I64, P, SZ, P]
        L.duo_rope.restype = I32
        L.duo_rope.argtypes = [P, I64, I64, I64, I64, I64, F64, P]
        L.duo_attention.restype = I32
        L.duo_attention.argtypes = [P, P, P, I64, I64, I64, I64, I64, P, I64, P, SZ, P]
        L.duo_silu_mul.restype = I32
        L.duo_silu_mul.argtypes = [P, P, I64, I64, I64, P, I64, P]
        L.duo_act_order.restype = I32
        L.duo_act_order.argtypes = [P, I64, P, P, P]
        L.duo_permute.restype = I32
        L.duo_permute.argtypes = [P, I32, I64, I64, I64, P, P, I64, I64, P, I64, P]
        L.duo_permute_mask.restype = I32
        L.duo_permute_mask.argtypes = [P, I64, I64, P, P, P]
        L.duo_dsc_workspace_size.restype = SZ
        L.duo_dsc_workspace_size.argtypes = [I64, I64]
        L.duo_dsc_layout.restype = I32
        L.duo_dsc_layout.argtypes = [P, I64, I64, P, P, P, P, SZ, P]
        L.duo_dsc_pack.restype = I32
        L.duo_dsc_pack.argtypes = [P, I32, I64, I64, I64, P, P, P, P, P]
        L.duo_dsc_gemv.restype = I32
        L.duo_dsc_gemv.argtypes = [P, I32, I64, I64, ActRule, P, P, P, P, P, P, SZ, P]
        L.duo_dsc_gemv_noalloc.restype = I32
        L.duo_dsc_gemv_noalloc.argtypes = [P, I32, I64, I64, ActRule, P, P, P, P, P, P]
        L.duo_profile_enable.restype = I32
        L.duo_profile_enable.argtypes = [I32]
        L.duo_profile_read.restype = I32
        L.duo_profile_read.argtypes = [I32, ctypes.POINTER(F64), ctypes.POINTER(I64)]
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().duo_status_string(int(status)).decode()


def version() -> str:
    return lib().duo_version().decode()


def _check(status: int, where: str):
    if status != DUO_OK:
        raise DuoError(status, where)


def _dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return DUO_F32
    if t.dtype == torch.bfloat16:
        return DUO_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _ld(t: torch.Tensor) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a 2-d tensor with unit column stride")
    return t.stride(0)


def _stream(device) -> ctypes.c_void_p:
    if torch.device(device).type != "cuda":
        raise ValueError("duo: tensors must live on a CUDA (HIP) device")
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _same_device(*ts):
    devs = {t.device for t in ts if t is not None}
    if len(devs) != 1 or next(iter(devs)).type != "cuda":
        raise ValueError("duo: all tensors must be on one CUDA (HIP) device")


def _shape(t, shape, name):
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"duo: {name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _contig(t, name):
    if t is not None and not t.is_contiguous():
        raise ValueError(f"duo: {name} must be contiguous")


def act_rule(sparsity: float | None) -> ActRule:
    if sparsity is None:
        return ActRule(DUO_ACT_NONE, 0.0)
    return ActRule(DUO_ACT_TOPK_MAG_PER_TOKEN, float(sparsity))


def duo_workspace_size(op: int, n: int, k: int, m: int, block: int) -> int:
    return int(lib().duo_workspace_size(op, n, k, m, block))


def workspace(op: int, n: int, k: int, m: int, block: int, device) -> torch.Tensor:
    """A workspace tensor for `op` (256-byte aligned by torch's allocator)."""
    nbytes = duo_workspace_size(op, n, k, m, block)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def duo_act_sparsify_mask(X, act_sparsity, mask_out=None, ws=None):
    m, k = X.shape
    _same_device(X, mask_out, ws)
    _shape(mask_out, (m, (k + 31) // 32), "mask_out")
    _contig(mask_out, "mask_out")
    if mask_out is None:
        mask_out = torch.empty((m, (k + 31) // 32), dtype=torch.int32, device=X.device)
    if ws is None:
        ws = workspace(DUO_OP_HESSIAN, 0, k, m, 0, X.device)
    st = lib().duo_act_sparsify_mask(_ptr(X), _dtype(X), m, k, _ld(X), act_rule(act_sparsity), _ptr(mask_out),
                                     _ptr(ws), ws.numel(), _stream(X.device))
    _check(st, "duo_act_sparsify_mask")
    return mask_out


def duo_hessian_accum(X_src, H, act_sparsity, X_dense=None, G=None, a=None, ws=None, hdiag=None, check=False,
                      g_full=None):
    """Stage 1 (H, and G and a when given).  check=True waits for the stream
    and raises DuoError(DUO_ERR_NONFINITE) if the inputs held NaN or inf.
    g_full: accumulate all of G (True) or only its upper triangle, diagonal
    included, which is all the solver reads (False); by default all of G
    exactly when hdiag is given (act_order permutes G afterwards)."""
    if g_full is None:
        g_full = hdiag is not None
    m, k = X_src.shape
    _same_device(X_src, X_dense, H, G, a, ws, hdiag)
    _shape(H, (k, k), "H")
    _shape(G, (k, k), "G")
    _shape(a, (k,), "a")
    _contig(a, "a")
    _shape(hdiag, (k,), "hdiag")
    _contig(hdiag, "hdiag")
    if hdiag is not None and hdiag.dtype != torch.float64:
        raise TypeError("hdiag must be float64")
    if ws is None:
        ws = workspace(DUO_OP_HESSIAN, 0, k, m, 0, X_src.device)
    if X_dense is not None and (X_dense.shape != X_src.shape or X_dense.stride() != X_src.stride()):
        raise ValueError("X_dense must have the shape and strides of X_src")
    st = lib().duo_hessian_accum(_ptr(X_src), _ptr(X_dense), _dtype(X_src), m, k, _ld(X_src), act_rule(act_sparsity),
                                 _ptr(H), _ld(H), _ptr(G), _ld(G) if G is not None else k,
                                 DUO_G_FULL if g_full else DUO_G_UPPER, _ptr(a), _ptr(hdiag),
                                 _ptr(ws), ws.numel(), _stream(X_src.device))
    _check(st, "duo_hessian_accum")
    if check and m > 0:
        _check(lib().duo_hessian_status(_ptr(ws), ws.numel(), _stream(X_src.device)), "duo_hessian_accum")


def duo_residual_term(X_dense, G, a, act_sparsity, X_src=None, ws=None, g_full=False):
    m, k = X_dense.shape
    _same_device(X_dense, X_src, G, a, ws)
    _shape(X_src, (m, k), "X_src")
    _shape(G, (k, k), "G")
    _shape(a, (k,), "a")
    _contig(a, "a")
    if X_src is not None and X_src.stride() != X_dense.stride():
        raise ValueError("X_src must have the strides of X_dense")
    if ws is None:
        ws = workspace(DUO_OP_HESSIAN, 0, k, m, 0, X_dense.device)
    st = lib().duo_residual_term(_ptr(X_dense), _ptr(X_src), _dtype(X_dense), m, k, _ld(X_dense),
                                 act_rule(act_sparsity), _ptr(G), _ld(G), DUO_G_FULL if g_full else DUO_G_UPPER,
                                 _ptr(a), _ptr(ws), ws.numel(),
                                 _stream(X_dense.device))
    _check(st, "duo_residual_term")


def duo_chol_inv(H, damp, ws=None, sync=True):
    """In place: H becomes L.  Returns (lambda, fail_index) when sync, else None."""
    k = H.shape[0]
    _same_device(H, ws)
    _shape(H, (k, k), "H")
    if ws is None:
        ws = workspace(DUO_OP_CHOL_INV, 0, k, 0, 0, H.device)
    info = CholInfo()
    st = lib().duo_chol_inv(_ptr(H), k, _ld(H), float(damp), ctypes.byref(info) if sync else None, _ptr(ws),
                            ws.numel(), _stream(H.device))
    _check(st, "duo_chol_inv")
    return (info.lam, info.fail_index) if sync else None


def duo_score_terms(L, G, a, D=None, fac=None, ws=None):
    k = L.shape[0]
    _same_device(L, G, a, D, fac, ws)
    for t, nm in ((L, "L"), (G, "G"), (D, "D")):
        _shape(t, (k, k), nm)
    _shape(a, (k,), "a")
    _shape(fac, (k,), "fac")
    _contig(a, "a")
    _contig(fac, "fac")
    if D is None:
        D = torch.zeros((k, k), dtype=torch.float32, device=L.device)
    if fac is None:
        fac = torch.empty(k, dtype=torch.float32, device=L.device)
    if ws is None:
        ws = workspace(DUO_OP_SCORE_TERMS, 0, k, 0, 0, L.device)
    _shape(D, (k, k), "D")
    _shape(fac, (k,), "fac")
    st = lib().duo_score_terms(_ptr(L), _ld(L), _ptr(G), _ld(G), _ptr(a), k, _ptr(D), _ld(D), _ptr(fac), _ptr(ws),
                               ws.numel(), _stream(L.device))
    _check(st, "duo_score_terms")
    return D, fac


def _check_outputs(out, W):
    n, k = W.shape
    W_out, lowp, mask, scores = out
    _same_device(W, W_out, lowp, mask, scores)
    _shape(W_out, (n, k), "W_out")
    _shape(lowp, (n, k), "W_out_lowp")
    _shape(mask, (n, (k + 31) // 32), "mask_out")
    _shape(scores, (n, k), "block_scores_out")
    for t, nm in ((W_out, "W_out"), (lowp, "W_out_lowp"), (mask, "mask_out"), (scores, "block_scores_out")):
        _contig(t, nm)
    if W_out is None or W_out.dtype != torch.float32 or (lowp is not None and lowp.dtype != W.dtype):
        raise ValueError("duo: W_out must be fp32 and W_out_lowp in W's dtype")


def _sweep_outputs(W, want_lowp, want_mask, want_scores):
    n, k = W.shape
    dev = W.device
    W_out = torch.empty((n, k), dtype=torch.float32, device=dev)
    lowp = torch.empty((n, k), dtype=W.dtype, device=dev) if want_lowp else None
    mask = torch.empty((n, (k + 31) // 32), dtype=torch.int32, device=dev) if want_mask else None
    scores = torch.empty((n, k), dtype=torch.float32, device=dev) if want_scores else None
    return W_out, lowp, mask, scores


def _opts(W, nm_n, quant, form=None):
    """(SweepOpts or None, q_scale, q_zero) for the sweep; quant = (bits, group);
    form: the residual form (FORMS)."""
    if form not in FORMS:
        raise ValueError(f"form must be one of {list(FORMS)}")
    if not nm_n and quant is None and not FORMS[form]:
        return None, None, None
    n, k = W.shape
    qs = qz = None
    bits, group = (0, 0) if quant is None else (int(quant[0]), int(quant[1]))
    if bits:
        ng = (k + group - 1) // group
        qs = torch.empty((n, ng), dtype=torch.float32, device=W.device)
        qz = torch.empty((n, ng), dtype=torch.float32, device=W.device)
    o = SweepOpts(int(nm_n), bits, group, qs.data_ptr() if qs is not None else None,
                  qz.data_ptr() if qz is not None else None, FORMS[form])
    return o, qs, qz


def duo_sweep(W, L, D, fac, w_sparsity, block=128, mask_in=None, want_lowp=False, want_mask=True,
              want_scores=False, ws=None, out=None, nm_n=0, quant=None):
    """Returns (W_out, W_lowp, mask, scores), plus (q_scale, q_zero) when
    quant = (bits, group) is given."""
    n, k = W.shape
    _same_device(W, L, D, fac, mask_in, ws)
    _shape(L, (k, k), "L")
    _shape(D, (k, k), "D")
    _shape(fac, (k,), "fac")
    _contig(fac, "fac")
    _shape(mask_in, (n, (k + 31) // 32), "mask_in")
    _contig(mask_in, "mask_in")
    if ws is None:
        ws = workspace(DUO_OP_SWEEP, n, k, 0, block, W.device)
    W_out, lowp, mask, scores = out if out is not None else _sweep_outputs(W, want_lowp, want_mask, want_scores)
    _check_outputs((W_out, lowp, mask, scores), W)
    o, qs, qz = _opts(W, nm_n, quant)
    st = lib().duo_sweep(_ptr(W), _dtype(W), n, k, _ld(W), _ptr(L), _ld(L), _ptr(D), _ld(D), _ptr(fac),
                         float(w_sparsity), ctypes.byref(o) if o is not None else None, int(block), _ptr(mask_in),
                         _ptr(W_out), _ptr(lowp), _ptr(mask), _ptr(scores), _ptr(ws), ws.numel(),
                         _stream(W.device))
    _check(st, "duo_sweep")
    if quant is not None:
        return W_out, lowp, mask, scores, qs, qz
    return W_out, lowp, mask, scores


def duo_prune_layer(W, L, G, a, w_sparsity, block=128, mask_in=None, want_lowp=False, want_mask=True,
                    want_scores=False, ws=None, out=None, nm_n=0, quant=None, form=None):
    """Returns (W_out, W_lowp, mask, scores), plus (q_scale, q_zero) when
    quant = (bits, group) is given.  form: residual form, None (automatic),
    "d" or "y"."""
    n, k = W.shape
    _same_device(W, L, G, a, mask_in, ws)
    _shape(L, (k, k), "L")
    _shape(G, (k, k), "G")
    _shape(a, (k,), "a")
    _contig(a, "a")
    _shape(mask_in, (n, (k + 31) // 32), "mask_in")
    _contig(mask_in, "mask_in")
    if ws is None:
        ws = workspace(DUO_OP_PRUNE_LAYER, n, k, 0, block, W.device)
    W_out, lowp, mask, scores = out if out is not None else _sweep_outputs(W, want_lowp, want_mask, want_scores)
    _check_outputs((W_out, lowp, mask, scores), W)
    o, qs, qz = _opts(W, nm_n, quant, form)
    st = lib().duo_prune_layer(_ptr(W), _dtype(W), n, k, _ld(W), _ptr(L), _ld(L), _ptr(G), _ld(G), _ptr(a),
                               float(w_sparsity), ctypes.byref(o) if o is not None else None, int(block),
                               _ptr(mask_in), _ptr(W_out), _ptr(lowp), _ptr(mask), _ptr(scores), _ptr(ws),
                               ws.numel(), _stream(W.device))
    _check(st, "duo_prune_layer")
    if quant is not None:
        return W_out, lowp, mask, scores, qs, qz
    return W_out, lowp, mask, scores


def duo_profile_enable(on: bool = True):
    _check(lib().duo_profile_enable(1 if on else 0), "duo_profile_enable")


def duo_profile_read(kernel: str):
    """(total milliseconds, launches) of a tracked kernel since the last read."""
    ms, n = F64(), I64()
    _check(lib().duo_profile_read(PROF[kernel], ctypes.byref(ms), ctypes.byref(n)), "duo_profile_read")
    return ms.value, n.value


def unpack_mask(words: torch.Tensor, k: int) -> torch.Tensor:
    """Bit-packed (rows x ceil(k/32) int32) mask -> bool rows x k (device-side
    bit extraction by torch; used for inspection only)."""
    w = words.to(torch.int64) & 0xFFFFFFFF
    bits = (w.unsqueeze(-1) >> torch.arange(32, device=words.device)) & 1
    return bits.reshape(words.shape[0], -1)[:, :k].bool()


def duo_act_order(hdiag):
    """act_order channel order from duo_hessian_accum's fp64 diagonal:
    returns (perm, inv_perm), int32 on hdiag's device."""
    k = hdiag.shape[0]
    if hdiag.dtype != torch.float64 or hdiag.dim() != 1:
        raise TypeError("hdiag must be a 1-D float64 tensor")
    _contig(hdiag, "hdiag")
    perm = torch.empty(k, dtype=torch.int32, device=hdiag.device)
    inv = torch.empty(k, dtype=torch.int32, device=hdiag.device)
    _check(lib().duo_act_order(_ptr(hdiag), k, _ptr(perm), _ptr(inv), _stream(hdiag.device)), "duo_act_order")
    return perm, inv


def _idx(t, n, name):
    if t is None:
        return None
    if t.dtype != torch.int32 or t.dim() != 1 or t.shape[0] != n:
        raise ValueError(f"{name} must be int32 of length {n}")
    _contig(t, name)
    return t


def duo_permute(src, row_idx=None, col_idx=None, out=None):
    """out[i][j] = src[row_idx[i]][col_idx[j]] (either index may be None =
    identity) for a 2-D fp32 or bf16 tensor with unit column stride."""
    if src.dim() != 2 or src.stride(1) != 1:
        raise ValueError("src must be 2-D with unit column stride")
    rows = row_idx.shape[0] if row_idx is not None else src.shape[0]
    cols = col_idx.shape[0] if col_idx is not None else src.shape[1]
    _idx(row_idx, rows, "row_idx")
    _idx(col_idx, cols, "col_idx")
    if out is None:
        out = torch.empty((rows, cols), dtype=src.dtype, device=src.device)
    _shape(out, (rows, cols), "out")
    _same_device(src, row_idx, col_idx, out)
    st = lib().duo_permute(_ptr(src), _dtype(src), src.shape[0], src.shape[1], _ld(src), _ptr(row_idx),
                           _ptr(col_idx), rows, cols, _ptr(out), _ld(out), _stream(src.device))
    _check(st, "duo_permute")
    return out


def duo_permute_mask(words, k, col_idx, out=None):
    """Column gather of a bit-packed n x ceil(k/32) mask (int32 words)."""
    n = words.shape[0]
    _idx(col_idx, k, "col_idx")
    _contig(words, "mask")
    if out is None:
        out = torch.empty_like(words)
    _same_device(words, col_idx, out)
    _check(lib().duo_permute_mask(_ptr(words), n, k, _ptr(col_idx), _ptr(out), _stream(words.device)),
           "duo_permute_mask")
    return out


def prune_linear(W, X, act_sparsity, w_sparsity, damp=0.01, block=128, X_dense=None, want_lowp=True,
                 act_order=False, nm=None, quant=None, form=None):
    """DuoGPT on one linear layer (stages 1-3 on the device).

    W: n x k (out x in), X: m x k token-major calibration input of the pruned
    stream (sparsified per token), X_dense: the dense stream (defaults to X).
    act_order: process the channels by decreasing Hessian diagonal (App. B);
    the outputs are returned in the original channel order.
    nm: None, or (N, 4) for the N:4 semi-structured variant (App. B), in which
    w_sparsity is not used; not combined with act_order.
    quant: None, or (bits, group) for joint RTN quantisation (Table 4); the
    grids (q_scale, q_zero: n x ceil(k / group)) are returned too (in the
    permuted channel order when act_order is set, as their groups are).
    form: residual form of the sweep (duo_prune_layer), None for automatic.
    Returns dict(W_out fp32, W_lowp in W's dtype, mask (bool n x k), lam, and
    perm when act_order).
    """
    n, k = W.shape
    dev = W.device
    nm_n = 0
    if nm is not None:
        if tuple(nm)[1] != 4 or act_order:
            raise ValueError("nm must be (N, 4) and is not combined with act_order")
        nm_n = int(nm[0])
    H = torch.zeros((k, k), dtype=torch.float32, device=dev)
    G = torch.zeros((k, k), dtype=torch.float32, device=dev)
    a = torch.zeros(k, dtype=torch.float32, device=dev)
    hdiag = torch.zeros(k, dtype=torch.float64, device=dev) if act_order else None
    duo_hessian_accum(X, H, act_sparsity, X_dense=X_dense, G=G, a=a, hdiag=hdiag, check=True)
    perm = None
    if act_order:
        perm, inv = duo_act_order(hdiag)
        H = duo_permute(H, perm, perm)
        G = duo_permute(G, perm, perm)
        a = duo_permute(a.view(1, k), None, perm).view(k)
        W = duo_permute(W, None, perm)
    lam, _ = duo_chol_inv(H, damp)
    res = duo_prune_layer(W, H, G, a, w_sparsity, block, want_lowp=want_lowp, nm_n=nm_n, quant=quant, form=form)
    W_out, lowp, mask = res[0], res[1], res[2]
    if act_order:
        W_out = duo_permute(W_out, None, inv)
        lowp = duo_permute(lowp, None, inv) if lowp is not None else None
        mask = duo_permute_mask(mask, k, inv)
    out = dict(W_out=W_out, W_lowp=lowp, mask=unpack_mask(mask, k), lam=lam, perm=perm)
    if quant is not None:
        out["q_scale"], out["q_zero"] = res[4], res[5]
    return out


# ---------------------------------------------------------------------------
# dual-sparse decode (compressed columns, activation-sparse GEMV)
# ---------------------------------------------------------------------------

def dsc_workspace(n: int, k: int, device) -> torch.Tensor:
    nbytes = int(lib().duo_dsc_workspace_size(n, k))
    if nbytes == 0:
        raise DuoError(DUO_ERR_UNSUPPORTED, "duo_dsc_workspace_size")
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def dsc_compress(W, mask, ws=None):
    """Compressed decode storage of a pruned layer: W (n x k fp32 or bf16, the
    pruned weights) and its bit mask (n x ceil(k/32) words as the sweep writes
    it).  Returns dict(col_ptr, maskT, chunk_off, values, n, k)."""
    n, k = W.shape
    _shape(mask, (n, (k + 31) // 32), "mask")
    _contig(mask, "mask")
    dev = W.device
    _same_device(W, mask, ws)
    if ws is None:
        ws = dsc_workspace(n, k, dev)
    col_ptr = torch.empty(k + 1, dtype=torch.int64, device=dev)
    maskT = torch.empty((k, (n + 31) // 32), dtype=torch.int32, device=dev)
    chunk_off = torch.empty((k, (n + 255) // 256), dtype=torch.int16, device=dev)
    st = lib().duo_dsc_layout(_ptr(mask), n, k, _ptr(col_ptr), _ptr(maskT), _ptr(chunk_off), _ptr(ws), ws.numel(),
                              _stream(dev))
    _check(st, "duo_dsc_layout")
    nnz = int(col_ptr[k].item())
    values = torch.zeros(nnz + 8, dtype=torch.int16, device=dev)  # + 8: the GEMV reads aligned 16-byte windows
    st = lib().duo_dsc_pack(_ptr(W), _dtype(W), n, k, _ld(W), _ptr(col_ptr), _ptr(maskT), _ptr(chunk_off),
                            _ptr(values), _stream(dev))
    _check(st, "duo_dsc_pack")
    return dict(col_ptr=col_ptr, maskT=maskT, chunk_off=chunk_off, values=values, n=n, k=k)


def dsc_gemv(comp, x, act_sparsity, ws=None, out=None):
    """One decode step y = W (x * m^x) over the compressed columns: x (k,)
    fp32 or bf16, sparsified with the calibration rule; y (n,) fp32."""
    n, k = comp["n"], comp["k"]
    if x.dim() != 1 or x.shape[0] != k:
        raise ValueError(f"x must have shape ({k},)")
    _contig(x, "x")
    dev = x.device
    if ws is None:
        ws = dsc_workspace(n, k, dev)
    y = out if out is not None else torch.empty(n, dtype=torch.float32, device=dev)
    _same_device(x, y, ws, comp["values"])
    st = lib().duo_dsc_gemv(_ptr(x), _dtype(x), n, k, act_rule(act_sparsity), _ptr(comp["col_ptr"]),
                            _ptr(comp["maskT"]), _ptr(comp["chunk_off"]), _ptr(comp["values"]), _ptr(y), _ptr(ws),
                            ws.numel(), _stream(dev))
    _check(st, "duo_dsc_gemv")
    return y


def dsc_gemv_noalloc(comp, x, act_sparsity, out=None):
    """dsc_gemv through the allocation-free entry point: no workspace; the
    library's per-GPU partial rows are used (calls on one GPU must not
    overlap).  `out` (n,) fp32 is written in place when given."""
    n, k = comp["n"], comp["k"]
    if x.dim() != 1 or x.shape[0] != k:
        raise ValueError(f"x must have shape ({k},)")
    _contig(x, "x")
    dev = x.device
    y = out if out is not None else torch.empty(n, dtype=torch.float32, device=dev)
    _same_device(x, y, comp["values"])
    st = lib().duo_dsc_gemv_noalloc(_ptr(x), _dtype(x), n, k, act_rule(act_sparsity), _ptr(comp["col_ptr"]),
                                    _ptr(comp["maskT"]), _ptr(comp["chunk_off"]), _ptr(comp["values"]), _ptr(y),
                                    _stream(dev))
    _check(st, "duo_dsc_gemv_noalloc")
    return y


# ---------------------------------------------------------------------------
# decoder-block harness (bf16 activations, token-major)
# ---------------------------------------------------------------------------

def _bf16_rows(t, name):
    if t.dtype != torch.bfloat16:
        raise TypeError(f"duo: {name} must be bfloat16")
    return _ld(t)


def block_workspace(op: int, m: int, seq_len: int, heads: int, device) -> torch.Tensor:
    nbytes = int(lib().duo_block_workspace_size(op, m, seq_len, heads))
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def duo_rmsnorm(X, eps=1e-5, out=None):
    m, d = X.shape
    Y = torch.empty_like(X) if out is None else out
    _same_device(X, Y)
    _shape(Y, (m, d), "Y")
    _check(lib().duo_rmsnorm(_ptr(X), m, d, _bf16_rows(X, "X"), float(eps), _ptr(Y), _bf16_rows(Y, "Y"),
                             _stream(X.device)), "duo_rmsnorm")
    return Y


def duo_act_sparsify(X, act_sparsity, out=None, ws=None):
    m, k = X.shape
    Y = torch.empty_like(X) if out is None else out
    _same_device(X, Y, ws)
    _shape(Y, (m, k), "Y")
    if ws is None:
        ws = block_workspace(DUO_BOP_ACT_SPARSIFY, m, 0, 0, X.device)
    _check(lib().duo_act_sparsify(_ptr(X), m, k, _bf16_rows(X, "X"), act_rule(act_sparsity), _ptr(Y),
                                  _bf16_rows(Y, "Y"), _ptr(ws), ws.numel(), _stream(X.device)), "duo_act_sparsify")
    return Y


def duo_linear(X, W, R=None, out=None, ws=None):
    """Y = X W^T (+ R), bf16."""
    m, k = X.shape
    n = W.shape[0]
    _shape(W, (n, k), "W")
    _shape(R, (m, n), "R")
    Y = torch.empty((m, n), dtype=torch.bfloat16, device=X.device) if out is None else out
    _same_device(X, W, R, Y, ws)
    _shape(Y, (m, n), "Y")
    if ws is None:
        ws = block_workspace(DUO_BOP_LINEAR, 0, 0, 0, X.device)
    _check(lib().duo_linear(_ptr(X), m, k, _bf16_rows(X, "X"), _ptr(W), n, _bf16_rows(W, "W"), _ptr(R),
                            _bf16_rows(R, "R") if R is not None else 0, _ptr(Y), _bf16_rows(Y, "Y"), _ptr(ws),
                            ws.numel(), _stream(X.device)), "duo_linear")
    return Y


def duo_rope(X, heads, head_dim, seq_len, theta=1e4):
    """In place."""
    m = X.shape[0]
    if X.shape[1] < heads * head_dim:
        raise ValueError("duo: X is narrower than heads * head_dim")
    _same_device(X)
    _check(lib().duo_rope(_ptr(X), m, heads, head_dim, _bf16_rows(X, "X"), seq_len, float(theta),
                          _stream(X.device)), "duo_rope")
    return X


def duo_attention(Q, K, V, nseq, seq_len, heads, head_dim, out=None, ws=None):
    m = nseq * seq_len
    for t, nm in ((Q, "Q"), (K, "K"), (V, "V")):
        if t.shape[0] < m or t.shape[1] < heads * head_dim:
            raise ValueError(f"duo: {nm} is smaller than nseq*seq_len x heads*head_dim")
    if not (Q.stride(0) == K.stride(0) == V.stride(0)):
        raise ValueError("duo: Q, K and V must share their row stride")
    O = torch.empty((m, heads * head_dim), dtype=torch.bfloat16, device=Q.device) if out is None else out
    _same_device(Q, K, V, O, ws)
    if ws is None:
        ws = block_workspace(DUO_BOP_ATTENTION, 0, seq_len, heads, Q.device)
    _check(lib().duo_attention(_ptr(Q), _ptr(K), _ptr(V), _bf16_rows(Q, "Q"), nseq, seq_len, heads, head_dim,
                               _ptr(O), _bf16_rows(O, "O"), _ptr(ws), ws.numel(), _stream(Q.device)),
           "duo_attention")
    return O


def duo_silu_mul(G, U, out=None):
    m, n = G.shape
    _shape(U, (m, n), "U")
    if G.stride(0) != U.stride(0):
        raise ValueError("duo: G and U must share their row stride")
    Y = torch.empty_like(G) if out is None else out
    _same_device(G, U, Y)
    _check(lib().duo_silu_mul(_ptr(G), _ptr(U), m, n, _bf16_rows(G, "G"), _ptr(Y), _bf16_rows(Y, "Y"),
                              _stream(G.device)), "duo_silu_mul")
    return Y
