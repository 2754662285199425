"""Float64 reference ("oracle") for the dual-sparse decode GEMV.

TEST INFRASTRUCTURE ONLY: the test-suite and the benchmark's CPU-baseline leg
may import this module; the HIP library never calls it and shares no code
with it.

Preliminaries ("Activation Sparsity") and Sec. 4.1 of the DuoGPT paper: at
decoding time a linear layer computes y = W (x * m^x), the sum of the weight
columns W[:, i] whose activation x_i survives, times x_i; only those columns
are fetched from HBM, and with dual sparsity each fetched column is stored
compressed.  The paper has no kernel for this (it leaves the spMspV kernel to
future work), so the storage below is this library's own definition:

  per input channel i (a column of the n x k weight matrix W):
    mask[i]      ceil(n / 32) uint32 words, bit r % 32 of word r // 32 set
                 when weight W[r, i] is kept;
    values       the kept weights of column i in row order (bf16 bits), at
                 values[col_ptr[i] : col_ptr[i + 1]];
    chunk_off[i] ceil(n / 256) uint16: the number of kept weights of column
                 i in rows [0, 256 c), so that row r's value (when kept) sits
                 at col_ptr[i] + chunk_off[i][r // 256] + (kept rows in
                 [256 (r // 256), r)).

The activation rule is the calibration one (Preliminaries): the z =
floor(p_x k + 0.5) entries with the smallest (|x|, channel) are zeroed.
"""

from __future__ import annotations

import numpy as np

from . import duo_ref as R

__all__ = ["CHUNK", "compress", "decompress", "gemv", "active_channels", "fetched_bytes"]

CHUNK = 256  # rows per chunk offset


def _bf16_bits(W):
    """Round-to-nearest-even bf16 bit patterns of W (as uint16)."""
    b = np.ascontiguousarray(np.asarray(W, dtype=np.float32)).view(np.uint32).astype(np.uint64)
    lsb = (b >> 16) & 1
    return ((b + 0x7FFF + lsb) >> 16).astype(np.uint16)


def compress(W_bits, keep):
    """W_bits: n x k bf16 bit patterns (uint16) of the pruned weights; keep:
    n x k bool.  Returns dict(col_ptr (k+1,) int64, mask (k, ceil(n/32))
    uint32, chunk_off (k, ceil(n/256)) uint16, values (nnz,) uint16)."""
    W_bits = np.asarray(W_bits, dtype=np.uint16)
    keep = np.asarray(keep, dtype=bool)
    n, k = keep.shape
    words, chunks = (n + 31) // 32, (n + CHUNK - 1) // CHUNK
    mask = np.zeros((k, words), dtype=np.uint32)
    chunk_off = np.zeros((k, chunks), dtype=np.uint16)
    col_ptr = np.zeros(k + 1, dtype=np.int64)
    vals = []
    for i in range(k):
        rows = np.nonzero(keep[:, i])[0]
        for r in rows:
            mask[i, r // 32] |= np.uint32(1) << np.uint32(r % 32)
        for c in range(chunks):
            chunk_off[i, c] = np.sum(rows < CHUNK * c)
        vals.append(W_bits[rows, i])
        col_ptr[i + 1] = col_ptr[i] + len(rows)
    values = np.concatenate(vals) if vals else np.zeros(0, dtype=np.uint16)
    return dict(col_ptr=col_ptr, mask=mask, chunk_off=chunk_off, values=values.astype(np.uint16))


def decompress(comp, n):
    """The dense n x k bf16 bit matrix the compressed form stands for (0 where
    not kept), reading each value through the chunk offsets."""
    mask, off, ptr, values = comp["mask"], comp["chunk_off"], comp["col_ptr"], comp["values"]
    k = mask.shape[0]
    out = np.zeros((n, k), dtype=np.uint16)
    for i in range(k):
        for r in range(n):
            w, b = divmod(r, 32)
            if (int(mask[i, w]) >> b) & 1:
                c0 = CHUNK * (r // CHUNK)
                before = sum((int(mask[i, q // 32]) >> (q % 32)) & 1 for q in range(c0, r))
                out[r, i] = values[ptr[i] + int(off[i, r // CHUNK]) + before]
    return out


def active_channels(x, p_x: float):
    """x_hat of one token (the calibration rule) and the indices of its
    nonzero entries in channel order."""
    x = np.asarray(x, dtype=np.float64).reshape(1, -1)
    xh, keep = R.sparsify_tokens(x, p_x)
    xh = xh[0]
    return xh, np.nonzero(xh != 0.0)[0]


def gemv(W_hat, x, p_x: float):
    """y = W_hat x_hat (float64), the definition of the dual-sparse GEMV."""
    xh, _ = active_channels(x, p_x)
    return np.asarray(W_hat, dtype=np.float64) @ xh


def fetched_bytes(comp, active, n):
    """Bytes an implementation that reads only the active channels must move:
    mask words, chunk offsets and kept values of those channels."""
    ptr = comp["col_ptr"]
    words, chunks = (n + 31) // 32, (n + CHUNK - 1) // CHUNK
    nnz = int(np.sum(ptr[np.asarray(active) + 1] - ptr[np.asarray(active)]))
    return len(active) * (4 * words + 2 * chunks) + 2 * nnz
