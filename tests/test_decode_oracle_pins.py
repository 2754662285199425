"""Pins of the dual-sparse decode oracle (oracle/decode_ref.py): the
compressed storage by a hand-worked example and by round trips, and the
GEMV by its dense definition and the dual-sparse property (inactive columns
are never needed)."""

import numpy as np
import pytest

from oracle import decode_ref as DR
from oracle import duo_ref as R


def test_compress_hand_example():
    n, k = 300, 3
    keep = np.zeros((n, k), dtype=bool)
    keep[[0, 5, 260, 299], 0] = True
    keep[250:260, 2] = True
    W = (np.arange(n * k, dtype=np.uint16).reshape(n, k) + 1).astype(np.uint16)
    c = DR.compress(W, keep)
    assert c["col_ptr"].tolist() == [0, 4, 4, 14]
    m = c["mask"]
    assert m.shape == (3, 10)
    assert m[0].tolist() == [0x21, 0, 0, 0, 0, 0, 0, 0, 0x10, 0x800]
    assert not m[1].any()
    assert m[2].tolist() == [0, 0, 0, 0, 0, 0, 0, 0xFC000000, 0xF, 0]
    assert c["chunk_off"].tolist() == [[0, 2], [0, 0], [0, 6]]
    want = [W[0, 0], W[5, 0], W[260, 0], W[299, 0]] + [W[r, 2] for r in range(250, 260)]
    assert c["values"].tolist() == want


@pytest.mark.parametrize("n,k,density", [(300, 17, 0.5), (513, 8, 0.1), (64, 5, 1.0), (40, 3, 0.0)])
def test_compress_round_trip(n, k, density):
    rng = np.random.default_rng(n + k)
    keep = rng.random((n, k)) < density
    W = rng.integers(1, 65535, size=(n, k)).astype(np.uint16)
    c = DR.compress(W, keep)
    assert c["col_ptr"][-1] == keep.sum()
    assert np.array_equal(DR.decompress(c, n), np.where(keep, W, 0))


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -9], dtype=np.float32)
    b = DR._bf16_bits(x)
    back = (b.astype(np.uint32) << 16).view(np.float32)
    assert back.tolist() == [1.0, 1.0, 1.0 + 2 ** -6, -2.5, 1.0]


def test_gemv_is_the_dense_product_over_active_columns():
    rng = np.random.default_rng(5)
    n, k, p_x = 96, 64, 0.5
    keep = rng.random((n, k)) < 0.5
    W = rng.standard_normal((n, k)) * keep
    x = rng.standard_normal(k)
    xh, act = DR.active_channels(x, p_x)
    assert len(act) == k - R.act_zero_count(k, p_x)
    y = DR.gemv(W, x, p_x)
    np.testing.assert_allclose(y, W[:, act] @ x[act], rtol=1e-12, atol=1e-14)
    # the dual-sparse property: the inactive columns' stored data plays no part
    bits = DR._bf16_bits(W)
    c = DR.compress(bits, keep)
    Wb = (DR.decompress(c, n).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    c2 = {key: v.copy() for key, v in c.items()}
    inactive = np.setdiff1d(np.arange(k), act)
    for i in inactive:
        c2["values"][c2["col_ptr"][i]:c2["col_ptr"][i + 1]] = 0x7FC0  # NaN
    Wb2 = (DR.decompress(c2, n).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    np.testing.assert_array_equal(Wb2[:, act] @ xh[act], Wb[:, act] @ xh[act])
    assert np.isnan(Wb2[:, inactive]).any() or keep[:, inactive].sum() == 0


def test_fetched_bytes_counts_active_channels_only():
    rng = np.random.default_rng(6)
    n, k = 520, 12
    keep = rng.random((n, k)) < 0.5
    c = DR.compress(np.ones((n, k), dtype=np.uint16), keep)
    act = np.array([1, 4, 7])
    want = 3 * (4 * 17 + 2 * 3) + 2 * int(keep[:, act].sum())
    assert DR.fetched_bytes(c, act, n) == want
