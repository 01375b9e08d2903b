"""GPU parity of the fused watermark + greedy decoding (sbw_watermark_argmax).

Tokens must equal the oracle's exactly and the values bit for bit (NaN as NaN),
over ragged shapes, both dtypes and seedings, windows, the gamma = 0 and 1
extremes, ties, NaN rows and signed zeros, unaligned rows, graph replay, and the
c4 workload at full size.
"""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_parity import KEY, WIDE, env, say, special_logits, _to_device  # noqa: F401

pytestmark = pytest.mark.gpu


def run_argmax(env, x, ctx, key, gamma, delta, seeding, offset=0, stride_pad=0, workspace=None):
    torch, sbw, dev = env
    B, V = x.shape
    stride = V + stride_pad
    base = np.zeros(offset + B * stride + 8, dtype=x.dtype)
    np.lib.stride_tricks.as_strided(base[offset:], shape=(B, V),
                                    strides=(stride * x.itemsize, x.itemsize))[...] = x
    tb = _to_device(torch, dev, base)
    t = tb[offset:offset + B * stride].view(B, stride)[:, :V]
    c = torch.from_numpy(np.ascontiguousarray(ctx, dtype=np.int32)).to(dev)
    tokens, values = sbw.watermark_argmax(t, c, key, gamma, delta, seeding, workspace=workspace)
    torch.cuda.synchronize()
    assert np.array_equal(tb.cpu().numpy().view(np.uint8) if x.dtype != np.uint16 else
                          tb.view(torch.int16).cpu().numpy().view(np.uint8),
                          base.view(np.uint8)), "logits were modified"
    return tokens.cpu().numpy(), values.cpu().numpy()


def assert_argmax_equal(got, expect, what=""):
    gt, gv = got
    et, ev = expect
    assert np.array_equal(gt, et), f"{what}: tokens differ at rows {np.flatnonzero(gt != et)[:5]}"
    nan = np.isnan(ev)
    assert np.array_equal(np.isnan(gv), nan), what
    assert np.array_equal(gv.view(np.uint32)[~nan], ev.view(np.uint32)[~nan]), what


def hard_rows(rng, B, V, dtype):
    x = special_logits(rng, B, V, "f32")
    if B >= 4:
        x[0, :] = 1.5                     # all equal: ties everywhere
        x[1, 3] = np.nan                  # NaN rows (first NaN wins)
        x[1, V // 2] = np.nan
        x[2, :] = -0.0                    # signed zeros
        x[2, ::3] = 0.0
        x[3, :] = -np.inf
    if dtype == "bf16":
        return workloads.f32_to_bf16_bits(x)
    return x


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
@pytest.mark.parametrize("B,V", [(1, 1), (4, 7), (5, 1000), (6, 4097), (4, 40001)])
def test_argmax_small(env, dtype, seeding, width, B, V):
    rng = np.random.default_rng(70 + width * 3 + B * 11 + V)
    x = hard_rows(rng, B, V, dtype)
    ctx = workloads.context_tokens(B, width, max(V, 2), rng)
    for gamma, delta in [(0.25, 2.0), (0.5, -1.0), (0.0, 3.0), (1.0, 0.5)]:
        say(f"argmax {dtype} {seeding} h={width} B={B} V={V} gamma={gamma}")
        assert_argmax_equal(run_argmax(env, x, ctx, WIDE, gamma, delta, seeding),
                            oracle.watermark_argmax(x, ctx, WIDE, gamma, delta, seeding),
                            f"{dtype}/{seeding}/{B}x{V}/{gamma}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("offset,stride_pad", [(1, 0), (0, 3), (8, 8), (0, 7)])   # 9008: aligned in both dtypes
def test_argmax_layouts(env, dtype, seeding, offset, stride_pad):
    rng = np.random.default_rng(80 + offset + stride_pad)
    B, V = 5, 9001
    x = hard_rows(rng, B, V, dtype)
    prev = rng.integers(0, V, B).astype(np.int32)
    say(f"argmax layout {dtype} {seeding} offset={offset} pad={stride_pad}")
    assert_argmax_equal(run_argmax(env, x, prev, KEY, 0.25, 2.0, seeding, offset, stride_pad),
                        oracle.watermark_argmax(x, prev, KEY, 0.25, 2.0, seeding))


def test_argmax_reuses_a_larger_workspace(env):
    torch, sbw, dev = env
    need = max(sbw.argmax_workspace_size(40, 3000), sbw.argmax_workspace_size(7, 50000))
    ws = torch.full((need + 5,), -1, dtype=torch.int64, device=dev)   # contents must not matter
    rng = np.random.default_rng(90)
    for B, V in [(40, 3000), (7, 50000), (40, 3000)]:
        x = rng.standard_normal((B, V)).astype(np.float32)
        prev = rng.integers(0, V, B).astype(np.int32)
        say(f"argmax workspace reuse B={B} V={V}")
        assert_argmax_equal(run_argmax(env, x, prev, KEY, 0.25, 2.0, "self_salt", workspace=ws),
                            oracle.watermark_argmax(x, prev, KEY, 0.25, 2.0, "self_salt"))


def test_argmax_graph_replay(env):
    torch, sbw, dev = env
    rng = np.random.default_rng(91)
    B, V = 16, 50003
    x = rng.standard_normal((B, V)).astype(np.float32)
    ctx = workloads.context_tokens(B, 4, V, rng)
    t = torch.from_numpy(x).to(dev)
    c = torch.from_numpy(ctx).to(dev)
    tokens = torch.empty(B, dtype=torch.int32, device=dev)
    values = torch.empty(B, dtype=torch.float32, device=dev)
    ws = torch.empty(sbw.argmax_workspace_size(B, V), dtype=torch.int64, device=dev)
    expect = oracle.watermark_argmax(x, ctx, KEY, 0.25, 2.0, "self_salt")
    sbw.watermark_argmax(t, c, KEY, 0.25, 2.0, "self_salt", tokens=tokens, values=values,
                         workspace=ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sbw.watermark_argmax(t, c, KEY, 0.25, 2.0, "self_salt", tokens=tokens, values=values,
                             workspace=ws)
    for replay in range(4):
        tokens.fill_(-7)
        values.fill_(0.0)
        ws.fill_(123)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert_argmax_equal((tokens.cpu().numpy(), values.cpu().numpy()), expect, f"replay {replay}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_argmax_c4_full_size(env, seeding, dtype):
    c = workloads.C4
    x, prev = workloads.watermark_inputs("c4")
    if dtype == "bf16":
        x = workloads.f32_to_bf16_bits(x)
    say(f"argmax c4 {seeding} {dtype}")
    got = run_argmax(env, x, prev, KEY, c["gamma"], c["delta"], seeding)
    expect = oracle.watermark_argmax(x, prev, KEY, c["gamma"], c["delta"], seeding)
    assert_argmax_equal(got, expect, f"c4 {seeding}")
    # the bias moves the argmax: most rows now pick a green token
    green = oracle.is_green_many(KEY, prev, expect[0], c["gamma"], seeding)
    assert green.mean() > 0.5


def bound_rows(rng, V, dtype):
    """Rows aimed at the pass's skip test, which leaves out elements whose logit and
    whose green value both lie below the largest logit m of a wave's share (or below
    m + delta when delta < 0): elements whose green value lands exactly on m, earlier
    and later than m; NaN and +inf after a spike; a single finite value among -inf;
    a row of equal values; a bf16 row where x + delta rounds (to even) onto m."""
    rows = []
    base = (0.05 * rng.standard_normal(V)).astype(np.float32)
    r = base.copy(); r[V - 5] = 4.0; r[7:V:977] = 2.0; rows.append(r)          # 2 + 2 == 4
    r = base.copy(); r[3] = 4.0; r[100:V:613] = 2.0; rows.append(r)           # m first
    r = base.copy(); r[V // 3] = 5.0; r[11:V:501] = 4.0; rows.append(r)       # delta < 0: 5 - 1 == 4
    r = base.copy(); r[50] = 9.0; r[V - 2] = np.nan; rows.append(r)           # NaN after a spike
    r = base.copy(); r[50] = 9.0; r[V // 2] = np.inf; rows.append(r)
    r = np.full(V, -np.inf, dtype=np.float32); r[V - 9] = -3.0; rows.append(r)
    rows.append(np.full(V, 2.0, dtype=np.float32))
    r = base.copy(); r[V - 100] = 256.0; r[13:V:389] = 254.0; rows.append(r)  # bf16: 254 + 1.5 -> 256
    x = np.stack(rows)
    return workloads.f32_to_bf16_bits(x) if dtype == "bf16" else x


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_argmax_skip_bound_edges(env, dtype, seeding):
    rng = np.random.default_rng(92)
    V = 40001
    x = bound_rows(rng, V, dtype)
    B = x.shape[0]
    ctx = workloads.context_tokens(B, 1, V, rng)[:, 0].copy()
    for gamma, delta in [(0.25, 2.0), (0.5, 2.0), (1.0, 2.0), (0.5, -1.0), (1.0, -1.0),
                         (0.5, 1.5), (1.0, 1.5), (0.0, 2.0)]:
        say(f"argmax bound edges {dtype} {seeding} gamma={gamma} delta={delta}")
        assert_argmax_equal(run_argmax(env, x, ctx, WIDE, gamma, delta, seeding),
                            oracle.watermark_argmax(x, ctx, WIDE, gamma, delta, seeding),
                            f"{dtype}/{seeding}/{gamma}/{delta}")


# Launches whose grid would hold fewer than this many workgroups take the decode kernel
# with half the vectors per lane; the bound-edge rows are run on both sides of it.
SMALL_DECODE_GRID = 900


def decode_segment(dtype, sample):
    """Logits per full-width decode segment, read from the kernel source's launch knobs
    (16-byte vectors per lane x 256 lanes), and the small-grid threshold, so that a
    retune of either keeps these tests honest about which kernel they run."""
    import os
    import re
    src = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                            "paper_2609_03844_amd", "csrc", "sbw_kernels.hip")).read()

    def knob(name):
        return int(re.search(rf"#define {name} (\d+)", src).group(1))
    threshold = int(re.search(r"kSmallDecodeGrid = (\d+);", src).group(1))
    assert threshold == SMALL_DECODE_GRID
    name = {("f32", False): "SBW_DECODE_VECS_F32_GREEDY", ("f32", True): "SBW_DECODE_VECS_F32",
            ("bf16", False): "SBW_DECODE_VECS_BF16",
            ("bf16", True): "SBW_DECODE_VECS_BF16_SAMPLE"}[(dtype, sample)]
    return (4 if dtype == "f32" else 8) * 256 * knob(name)



@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_argmax_both_launch_shapes(env, dtype, seeding):
    """The bound-edge rows tiled to 256 rows (the full-width kernel: more than 900
    workgroups) and to 8 rows (the half-width kernel for small grids)."""
    rng = np.random.default_rng(93)
    V = 40001
    edge = bound_rows(rng, V, dtype)
    seg = decode_segment(dtype, sample=False)      # logits per full-width segment
    for B in (8, 256):
        x = np.concatenate([edge] * (-(-B // edge.shape[0])))[:B].copy()
        ctx = workloads.context_tokens(B, 1, V, rng)[:, 0].copy()
        big = B * (-(-V // seg)) >= SMALL_DECODE_GRID
        assert big == (B == 256), (B, seg)         # both launch shapes are exercised
        for gamma, delta in [(0.25, 2.0), (0.5, -1.0)]:
            say(f"argmax launch shapes {dtype} {seeding} B={B} big={big} gamma={gamma}")
            assert_argmax_equal(run_argmax(env, x, ctx, WIDE, gamma, delta, seeding),
                                oracle.watermark_argmax(x, ctx, WIDE, gamma, delta, seeding),
                                f"{dtype}/{seeding}/B={B}/{gamma}")
