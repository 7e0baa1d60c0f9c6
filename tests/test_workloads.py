"""The synthetic input generators (no method arithmetic): shapes, seeding and
the shifted-window mask layout."""
import numpy as np

import workloads as W


def test_shifted_window_mask_regions():
    """14 x 14 tokens, 7 x 7 windows, shift 3: the first window lies in one
    region, the two edge windows in two (28 and 21 tokens), the corner window
    in four (16, 12, 12 and 9 tokens)."""
    m = W.shifted_window_mask(14, 7, 3, -7)
    assert m.shape == (4, 49, 49) and m.dtype == np.int32
    assert set(np.unique(m)) <= {0, -7}
    for w in range(4):
        assert np.array_equal(m[w], m[w].T)
        assert np.all(np.diag(m[w]) == 0)
    masked = [int((m[w] != 0).sum()) for w in range(4)]
    assert masked == [0, 2 * 28 * 21, 2 * 28 * 21, 49 * 49 - (16 ** 2 + 12 ** 2 + 12 ** 2 + 9 ** 2)]


def test_generators_are_seeded():
    a = W.attn_inputs(4, 20, 20, 8, seed=3, heads=2, bias=True)
    b = W.attn_inputs(4, 20, 20, 8, seed=3, heads=2, bias=True)
    c = W.attn_inputs(4, 20, 20, 8, seed=4, heads=2, bias=True)
    assert all(np.array_equal(a[k], b[k]) for k in ("logits", "v", "bias"))
    assert not np.array_equal(a["logits"], c["logits"])
    q = W.qk_inputs(3, 16, 16, 32, 32, seed=5, zp_q=4, zp_k=-3)
    assert q["q"].shape == (3, 16, 32) and q["k"].dtype == np.int8
