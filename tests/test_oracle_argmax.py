"""Pins of the oracle's greedy decoding of watermarked logits (Eq. 2 then argmax).

The fused definition must equal numpy's argmax (first maximum, NaN counts as the
maximum, -0 == +0) applied to the oracle's watermarked logits, whose own pins are
in test_oracle_pins; plus the tie, NaN and signed-zero cases written out.
"""
import numpy as np
import pytest

import oracle
import workloads

KEY = oracle.PAPER_KEY


def _np_argmax(x):
    if x.dtype == np.uint16:
        x = (x.astype(np.uint32) << 16).view(np.float32)
    idx = np.argmax(x, axis=1)
    return idx.astype(np.int32), x[np.arange(x.shape[0]), idx]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
def test_argmax_equals_numpy_argmax_of_the_watermarked_logits(dtype, seeding, width):
    rng = np.random.default_rng(60 + width)
    B, V = 6, 4099
    x = rng.standard_normal((B, V)).astype(np.float32)
    x[1, 17] = np.nan            # a NaN row
    x[1, 900] = np.nan
    x[2, :] = 0.0                # all equal: the first green token wins after the bias
    x[3, ::2] = -0.0             # signed zeros
    x[4, 5] = np.inf
    if dtype == "bf16":
        x = workloads.f32_to_bf16_bits(x)
    ctx = workloads.context_tokens(B, width, V, rng)
    for delta in (2.0, 0.0, -3.0):
        tok, val = oracle.watermark_argmax(x, ctx, KEY, 0.25, delta, seeding)
        wm = oracle.watermark_w(x, ctx, KEY, 0.25, delta, seeding)
        e_tok, e_val = _np_argmax(wm)
        assert np.array_equal(tok, e_tok), delta
        both_nan = np.isnan(val) & np.isnan(e_val)
        assert np.array_equal(val.view(np.uint32)[~both_nan], e_val.view(np.uint32)[~both_nan])


def test_argmax_ties_nans_and_zeros():
    # gamma = 0: nothing is green, so the argmax is plain argmax of the input
    x = np.array([[1.0, 3.0, 3.0, 2.0],
                  [-0.0, 0.0, -1.0, -0.0],
                  [1.0, np.nan, 5.0, np.nan],
                  [-np.inf, -np.inf, -np.inf, -np.inf]], dtype=np.float32)
    prev = np.zeros(4, np.int32)
    tok, val = oracle.watermark_argmax(x, prev, KEY, 0.0, 1.0)
    assert list(tok) == [1, 0, 1, 0]
    assert val[0] == 3.0 and val[1] == 0.0 and np.isnan(val[2]) and val[3] == -np.inf
    # gamma = 1: everything gets +delta, same winners
    tok1, val1 = oracle.watermark_argmax(x, prev, KEY, 1.0, 1.0)
    assert list(tok1) == [1, 0, 1, 0] and val1[0] == 4.0
