"""The bounds on the Gumbel noise that the sampling kernel uses to skip tokens.

The kernel bounds a token's noise from the number c of leading one bits of its
32-bit draw (capped at 23) instead of evaluating the two logarithms: from above by
c ln 2 + (ln 2 + margin), and, for c >= 2, from below by that bound minus a fixed
gap.  A wrong bound would make the kernel skip a token that can win, so both are
checked here against the oracle's noise for every one of the 2^23 values the
uniform variate takes, with the constants read from the kernel's header and the
bound computed in fp32 the way the kernel computes it (one fused multiply-add).
"""
import pathlib
import re

import numpy as np
import pytest

import oracle

HEADER = pathlib.Path(__file__).resolve().parents[1] / "paper_2609_03844_amd" / "csrc" / "sbw_device.hpp"


def header_constants():
    text = HEADER.read_text()
    out = {}
    for name, value in re.findall(r"constexpr float (k\w+) = ([-+0-9.eE]+)f;", text):
        out[name] = np.float32(float(value))
    return out


@pytest.fixture(scope="module")
def every_draw():
    x = np.arange(1 << 23, dtype=np.uint32) << np.uint32(9)   # the low 9 bits do not enter u
    return x, oracle.gumbel_of_draws(x).astype(np.float64)


def leading_ones_capped(x):
    """clz(~x | 2^8), counted bit by bit."""
    y = (~x) | np.uint32(0x100)
    c = np.zeros(x.shape, dtype=np.int64)
    running = np.ones(x.shape, dtype=bool)
    for b in range(31, -1, -1):
        running &= ((y >> np.uint32(b)) & np.uint32(1)) == 0
        c += running
    return c


def fma32(a, b, c):
    # a * b + c is exact in double for these magnitudes, so one rounding to fp32 is the fma
    return (np.float64(a) * np.float64(b) + np.float64(c)).astype(np.float32).astype(np.float64)


def test_upper_bound_holds_for_every_draw(every_draw):
    x, g = every_draw
    k = header_constants()
    c = leading_ones_capped(x)
    assert c.min() == 0 and c.max() == 23
    offset = np.float32(k["kLn2f"] + k["kGumbelMargin"])     # constexpr sum, rounded to fp32
    upper = fma32(c.astype(np.float32), k["kLn2f"], offset)
    assert np.all(g <= upper), (g - upper).max()
    assert (upper - g).min() > 0.0005                        # room for the fp32 logarithm
    assert k["kLn2f"] >= np.log(2.0)


def test_gap_below_the_upper_bound_for_c_at_least_2(every_draw):
    x, g = every_draw
    k = header_constants()
    c = leading_ones_capped(x)
    offset = np.float32(k["kLn2f"] + k["kGumbelMargin"])
    upper = fma32(c.astype(np.float32), k["kLn2f"], offset)
    sel = c >= 2
    assert np.all(g[sel] >= upper[sel] - np.float64(k["kGumbelGap"]))
    assert (g[sel] - (upper[sel] - np.float64(k["kGumbelGap"]))).min() > 0.005
    # the gap would not hold for c = 1: that is why the kernel leaves those tokens out
    assert np.any(g[c == 1] < upper[c == 1] - np.float64(k["kGumbelGap"]))


def test_overall_range(every_draw):
    _, g = every_draw
    k = header_constants()
    assert k["kGumbelLo"] < g.min() and g.max() < k["kGumbelHi"]
