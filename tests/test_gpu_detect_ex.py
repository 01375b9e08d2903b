"""GPU parity of sbw_detect_ex: texts of different lengths, and each distinct
(width+1)-gram scored once.

Green counts and scored counts bit-exact, z within 1e-6 relative, against the
oracle: lengths in and out of [0, L], widths 1, 4 and 8, both seedings, small
vocabularies (repeats everywhere), copied spans and constant texts, padded rows,
the 4096-position limit of the repeat rule, graph replay, and the c5 batch at full
size with lengths drawn in [L/2, L].
"""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_parity import KEY, WIDE, Z_RTOL, env, say  # noqa: F401

pytestmark = pytest.mark.gpu


def run_detect_ex(env, tok, width, key, gamma, seeding, lengths=None, ignore=False, pad=0):
    torch, sbw, dev = env
    N, L = tok.shape
    host = np.full((N, L + pad), 7, dtype=np.int32)
    host[:, :L] = tok
    t = torch.from_numpy(host).to(dev)[:, :L]
    lens = None if lengths is None else torch.from_numpy(np.ascontiguousarray(lengths, np.int32)).to(dev)
    counts, scored, z = sbw.detect_ex(t, key, gamma, seeding, width=width, lengths=lens,
                                      ignore_repeated=ignore)
    torch.cuda.synchronize()
    return counts.cpu().numpy(), scored.cpu().numpy(), z.cpu().numpy()


def assert_ex_equal(got, expect, what=""):
    gc, gs, gz = got
    ec, es, ez = expect
    assert np.array_equal(gc, ec), f"{what}: counts differ at {np.flatnonzero(gc != ec)[:5]}"
    assert np.array_equal(gs, es), f"{what}: scored differ at {np.flatnonzero(gs != es)[:5]}"
    assert np.array_equal(np.isnan(gz), np.isnan(ez)), what
    ok = ~np.isnan(ez)
    np.testing.assert_allclose(gz[ok], ez[ok], rtol=Z_RTOL, atol=Z_RTOL, err_msg=what)


def texts(rng, N, L, V):
    tok = rng.integers(0, V, (N, L)).astype(np.int32)
    if N >= 3 and L >= 40:
        tok[1, L // 2:L // 2 + 15] = tok[1, 3:18]      # a copied span
        tok[2, :] = 11                                  # one token throughout
    return tok


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4, 8])
@pytest.mark.parametrize("ignore", [False, True])
@pytest.mark.parametrize("N,L,V", [(1, 0, 10), (3, 1, 10), (5, 9, 3), (6, 130, 5), (9, 700, 50),
                                   (4, 3000, 128256)])
def test_detect_ex_small(env, seeding, width, ignore, N, L, V):
    rng = np.random.default_rng(200 + width + N * 3 + L)
    tok = texts(rng, N, L, V)
    lengths = rng.integers(-2, L + 3, N).astype(np.int32)
    if N > 1:
        lengths[0] = L
    for lens in (None, lengths):
        say(f"detect_ex {seeding} h={width} ignore={ignore} N={N} L={L} V={V} lengths={lens is not None}")
        got = run_detect_ex(env, tok, width, WIDE, 0.25, seeding, lens, ignore, pad=3)
        expect = oracle.detect_ex(tok, width, WIDE, 0.25, seeding, lengths=lens, ignore_repeated=ignore)
        assert_ex_equal(got, expect, f"{seeding}/{width}/{ignore}/{N}x{L}")


@pytest.mark.parametrize("width", [1, 4])
def test_detect_ex_repeat_rule_at_its_limit(env, width):
    rng = np.random.default_rng(210)
    L = 4096 + width                                   # 4096 scored positions
    tok = texts(rng, 3, L, 40)
    say(f"detect_ex limit h={width}")
    got = run_detect_ex(env, tok, width, KEY, 0.5, "self_salt", ignore=True)
    assert_ex_equal(got, oracle.detect_ex(tok, width, KEY, 0.5, "self_salt", ignore_repeated=True))


def test_detect_ex_graph_replay(env):
    torch, sbw, dev = env
    rng = np.random.default_rng(220)
    tok = texts(rng, 64, 300, 20)
    lengths = rng.integers(0, 301, 64).astype(np.int32)
    expect = oracle.detect_ex(tok, 4, KEY, 0.25, "context", lengths=lengths, ignore_repeated=True)
    t = torch.from_numpy(tok).to(dev)
    lens = torch.from_numpy(lengths).to(dev)
    counts = torch.empty(64, dtype=torch.int32, device=dev)
    scored = torch.empty(64, dtype=torch.int32, device=dev)
    z = torch.empty(64, dtype=torch.float64, device=dev)
    sbw.detect_ex(t, KEY, 0.25, "context", width=4, lengths=lens, ignore_repeated=True,
                  counts=counts, scored=scored, z=z)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sbw.detect_ex(t, KEY, 0.25, "context", width=4, lengths=lens, ignore_repeated=True,
                      counts=counts, scored=scored, z=z)
    for replay in range(4):
        counts.fill_(-1); scored.fill_(-1); z.fill_(0.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert_ex_equal((counts.cpu().numpy(), scored.cpu().numpy(), z.cpu().numpy()), expect,
                        f"replay {replay}")


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("ignore", [False, True])
def test_detect_ex_c5_full_size(env, seeding, ignore):
    c = workloads.C5
    tok = workloads.detect_inputs(c["N"], c["L"], c["V"], c["gamma"], c["delta"], seeding,
                                  lambda p, v: oracle.is_green_many(KEY, p, v, c["gamma"], seeding))
    lengths = workloads.rng_for("c5", salt=9).integers(c["L"] // 2, c["L"] + 1, c["N"]).astype(np.int32)
    say(f"detect_ex c5 {seeding} ignore={ignore}")
    got = run_detect_ex(env, tok, 1, KEY, c["gamma"], seeding, lengths, ignore)
    expect = oracle.detect_ex(tok, 1, KEY, c["gamma"], seeding, lengths=lengths, ignore_repeated=ignore)
    assert_ex_equal(got, expect, f"c5 {seeding} {ignore}")
    # the watermarked half is still detected with shorter texts
    assert np.nanmin(got[2][c["N"] // 2:]) > 4.0
