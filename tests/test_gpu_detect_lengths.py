"""GPU parity of detection at every text length around the pass boundaries.

A detection launch picks 1, 2, 4 or 8 positions per lane from the longest text (up to
64, 128, 256 or more scored positions), and a text longer than a pass takes several
passes.  Within a pass, the in-range lanes of each chunk form a mask (full chunks, one
partial chunk, empty chunks), and the self-salt hash of a position's window token is
handed from chunk to chunk and from pass to pass.  Each case below gives one launch
texts of every length from 0 to L (one text per length), so every remainder of the
scored positions modulo 64, and every chunk boundary, occurs in one batch; widths 1
and 4, both seedings.  Counts and scored counts bit-exact, z within 1e-6 relative,
against the oracle.
"""
import numpy as np
import pytest

import oracle
from test_gpu_detect_ex import assert_ex_equal, run_detect_ex
from test_gpu_parity import WIDE, env, say  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
@pytest.mark.parametrize("L", [65, 130, 258, 600, 1100])
def test_detect_every_length(env, seeding, width, L):
    rng = np.random.default_rng(300 + L + width)
    N = L + 1
    tok = rng.integers(0, 128256, (N, L)).astype(np.int32)
    lengths = np.arange(N, dtype=np.int32)          # text n holds n tokens
    say(f"detect every length {seeding} h={width} L={L}")
    got = run_detect_ex(env, tok, width, WIDE, 0.25, seeding, lengths, pad=5)
    expect = oracle.detect_ex(tok, width, WIDE, 0.25, seeding, lengths=lengths)
    assert_ex_equal(got, expect, f"{seeding}/{width}/L={L}")
