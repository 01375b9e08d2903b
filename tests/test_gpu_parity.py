"""GPU parity: the HIP path against the CPU oracle, element by element.

Watermarked logits, green masks and green counts must be bit-identical; z-scores
agree within 1e-6 relative (both NaN where T = 0).  Small cases span several
workgroup tiles and ragged tails; the five workload configurations run at their
full sizes through the same entry points and launch shapes the benchmark uses.
"""
import math
import sys

import numpy as np
import pytest

import oracle
import workloads

pytestmark = pytest.mark.gpu

KEY = workloads.PAPER_KEY
WIDE = workloads.WIDE_KEY
Z_RTOL = 1e-6


def say(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch
    import paper_2609_03844_amd as sbw
    assert torch.cuda.is_available()
    torch.cuda.init()
    return torch, sbw, torch.device("cuda:0")


def _to_device(torch, dev, x: np.ndarray):
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16).copy()).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev)


def _from_device(torch, t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _nan_mask(x: np.ndarray) -> np.ndarray:
    if x.dtype == np.uint16:
        return np.isnan((x.astype(np.uint32) << 16).view(np.float32))
    return np.isnan(x)


def assert_logits_equal(got: np.ndarray, expect: np.ndarray, what=""):
    assert got.shape == expect.shape and got.dtype == expect.dtype
    gn, en = _nan_mask(got), _nan_mask(expect)
    assert np.array_equal(gn, en), f"{what}: NaN positions differ"
    bits = np.uint16 if got.dtype == np.uint16 else np.uint32
    g, e = got.view(bits)[~gn], expect.view(bits)[~en]
    if not np.array_equal(g, e):
        bad = np.flatnonzero(g != e)
        raise AssertionError(f"{what}: {bad.size} elements differ, first at {bad[:5]}")


def run_watermark(env, x, prev, key, gamma, delta, seeding, stride=None, offset=0):
    """x [B, V] on the host -> GPU watermark -> host array.  `stride` pads rows;
    `offset` shifts the first element (for unaligned row starts)."""
    torch, sbw, dev = env
    B, V = x.shape
    stride = stride or V
    base = np.zeros((offset + B * stride + 8,), dtype=x.dtype)
    view = np.lib.stride_tricks.as_strided(base[offset:], shape=(B, V),
                                           strides=(stride * x.itemsize, x.itemsize))
    view[...] = x
    tb = _to_device(torch, dev, base)
    t = tb[offset:offset + B * stride].view(B, stride)[:, :V] if B > 0 else tb[:0].view(0, V)
    p = torch.from_numpy(np.ascontiguousarray(prev, dtype=np.int32)).to(dev)
    sbw.watermark(t, p, key, gamma, delta, seeding)
    torch.cuda.synchronize()
    out_base = _from_device(torch, tb)
    # elements outside the [B, V] window must be untouched
    untouched = np.ones(out_base.shape, bool)
    for b in range(B):
        untouched[offset + b * stride: offset + b * stride + V] = False
    assert np.array_equal(out_base[untouched].view(np.uint8), base[untouched].view(np.uint8))
    return np.lib.stride_tricks.as_strided(out_base[offset:], shape=(B, V),
                                           strides=(stride * x.itemsize, x.itemsize)).copy()


def run_mask(env, B, V, prev, key, gamma, seeding):
    torch, sbw, dev = env
    p = torch.from_numpy(np.ascontiguousarray(prev, dtype=np.int32)).to(dev)
    out = sbw.green_mask(p, V, key, gamma, seeding)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint32)


def run_detect(env, tok, key, gamma, seeding, stride=None):
    torch, sbw, dev = env
    N, L = tok.shape
    stride = stride or max(L, 1)
    host = np.zeros((N, stride), dtype=np.int32)
    host[:, :L] = tok
    t = torch.from_numpy(host).to(dev)[:, :L]
    counts, z = sbw.detect(t, key, gamma, seeding)
    torch.cuda.synchronize()
    return counts.cpu().numpy(), z.cpu().numpy()


def assert_detect_equal(got, expect):
    gc, gz = got
    ec, ez = expect
    assert np.array_equal(gc, ec), f"counts differ at {np.flatnonzero(gc != ec)[:5]}"
    assert np.array_equal(np.isnan(gz), np.isnan(ez))
    ok = ~np.isnan(ez)
    np.testing.assert_allclose(gz[ok], ez[ok], rtol=Z_RTOL, atol=Z_RTOL)


def special_logits(rng, B, V, dtype):
    x = rng.standard_normal((B, V)).astype(np.float32) * np.float32(4)
    flat = x.reshape(-1)
    specials = np.array([np.nan, -np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-45, -1e-45, 1e-39,
                         3.4e38, -3.4e38, 1.17549435e-38], dtype=np.float32)
    payload_nan = np.array([0x7F800001, 0xFFC00123, 0x7FBFFFFF], dtype=np.uint32).view(np.float32)
    specials = np.concatenate([specials, payload_nan])
    idx = rng.choice(flat.size, size=min(flat.size, 4 * specials.size), replace=False)
    flat[idx] = np.resize(specials, idx.size)
    if dtype == "bf16":
        return workloads.f32_to_bf16_bits(x)
    return x


# --- small cases: tiles, ragged tails, layouts, special values ----------------------

SHAPES = [(1, 1), (1, 3), (2, 5), (3, 31), (2, 32), (2, 33), (4, 1000), (3, 4097), (2, 32001),
          (5, 1024 * 4 * 2 + 7)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("B,V", SHAPES)
def test_watermark_small(env, dtype, seeding, B, V):
    rng = np.random.default_rng(1000 + B * 7 + V)
    x = special_logits(rng, B, V, dtype)
    prev = rng.integers(0, max(V, 2), B).astype(np.int32)
    for gamma, delta, key in [(0.25, 2.0, KEY), (0.5, -1.5, WIDE), (0.3, 1e-3, KEY)]:
        say(f"watermark {dtype} {seeding} B={B} V={V} gamma={gamma} delta={delta}")
        got = run_watermark(env, x, prev, key, gamma, delta, seeding)
        assert_logits_equal(got, oracle.watermark(x, prev, key, gamma, delta, seeding),
                            f"{dtype}/{seeding}/{B}x{V}/{gamma}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("stride_pad,offset", [(1, 0), (3, 0), (8, 0), (0, 1), (5, 3), (0, 8),
                                               (5, 0), (13, 8)])
def test_watermark_layouts(env, dtype, seeding, stride_pad, offset):
    # padded rows, unaligned row starts (element kernel) and aligned-but-offset starts;
    # strides of 5008 and 5016 keep rows 16-byte aligned in both dtypes (the vector
    # kernels with a 3-token row tail)
    rng = np.random.default_rng(77 + stride_pad * 10 + offset)
    B, V = 6, 5003
    x = special_logits(rng, B, V, dtype)
    prev = rng.integers(0, V, B).astype(np.int32)
    say(f"layout {dtype} {seeding} stride=V+{stride_pad} offset={offset}")
    got = run_watermark(env, x, prev, KEY, 0.25, 2.0, seeding, stride=V + stride_pad, offset=offset)
    assert_logits_equal(got, oracle.watermark(x, prev, KEY, 0.25, 2.0, seeding))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("gamma,delta", [(0.0, 2.0), (1.0, 2.0), (1.0, -0.0), (0.5, 0.0),
                                         (0.25, 3e38), (0.25, -3e38), (0.25, 1e-45),
                                         (5e-324, 1.0), (0.9999999999, 1.0)])
def test_watermark_degenerate_parameters(env, dtype, gamma, delta):
    rng = np.random.default_rng(5)
    B, V = 3, 2051
    x = special_logits(rng, B, V, dtype)
    prev = np.array([0, -1, 2 ** 31 - 1], dtype=np.int32)  # 0, 0xFFFFFFFF, ids >= V
    for seeding in ("context", "self_salt"):
        say(f"degenerate {dtype} {seeding} gamma={gamma} delta={delta}")
        got = run_watermark(env, x, prev, WIDE, gamma, delta, seeding)
        assert_logits_equal(got, oracle.watermark(x, prev, WIDE, gamma, delta, seeding))


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("B,V", [(1, 1), (2, 31), (2, 32), (3, 33), (4, 4097), (2, 128256)])
def test_green_mask(env, seeding, B, V):
    rng = np.random.default_rng(B * 13 + V)
    prev = rng.integers(-5, V + 5, B).astype(np.int32)
    for gamma in (0.0, 0.25, 0.5, 0.3, 1.0):
        say(f"mask {seeding} B={B} V={V} gamma={gamma}")
        got = run_mask(env, B, V, prev, WIDE, gamma, seeding)
        assert np.array_equal(got, oracle.green_mask(B, V, prev, WIDE, gamma, seeding))


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("N,L", [(1, 0), (3, 1), (2, 2), (5, 63), (5, 64), (5, 65), (7, 200),
                                 (9, 256), (9, 257), (9, 258), (4, 2049),
                                 (300, 129), (3, 5000)])
def test_detect_small(env, seeding, N, L):
    rng = np.random.default_rng(N * 31 + L)
    tok = rng.integers(-(1 << 31), 1 << 31, (N, L), dtype=np.int64).astype(np.int32)
    tok[:, ::3] = rng.integers(0, 100, tok[:, ::3].shape)  # repeated small ids too
    for gamma in (0.25, 0.5, 0.3):
        say(f"detect {seeding} N={N} L={L} gamma={gamma}")
        got = run_detect(env, tok, WIDE, gamma, seeding, stride=L + 3)
        assert_detect_equal(got, oracle.detect(tok, WIDE, gamma, seeding))


def test_deterministic_and_on_a_side_stream(env):
    torch, sbw, dev = env
    rng = np.random.default_rng(8)
    x = rng.standard_normal((16, 40000)).astype(np.float32)
    prev = rng.integers(0, 40000, 16).astype(np.int32)
    expect = oracle.watermark(x, prev, KEY, 0.25, 2.0, "self_salt")
    say("determinism + side stream")
    s = torch.cuda.Stream()
    outs = []
    for _ in range(2):
        with torch.cuda.stream(s):
            t = torch.from_numpy(x).to(dev, non_blocking=False)
            p = torch.from_numpy(prev).to(dev)
            sbw.watermark(t, p, KEY, 0.25, 2.0, "self_salt")
        s.synchronize()
        outs.append(t.cpu().numpy())
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    assert_logits_equal(outs[0], expect)


def test_no_device_memory_is_allocated(env):
    torch, sbw, dev = env
    x = torch.randn(64, 128256, device=dev)
    p = torch.randint(0, 128256, (64,), dtype=torch.int32, device=dev)
    tok = torch.randint(0, 128256, (256, 512), dtype=torch.int32, device=dev)
    counts = torch.empty(256, dtype=torch.int32, device=dev)
    z = torch.empty(256, dtype=torch.float64, device=dev)
    say("zero allocation")
    for seeding in ("context", "self_salt"):  # warm every kernel once
        sbw.watermark(x, p, KEY, 0.25, 2.0, seeding)
        sbw.detect(tok, KEY, 0.25, seeding, counts=counts, z=z)
    torch.cuda.synchronize()
    alloc0, free0 = torch.cuda.memory_allocated(), torch.cuda.mem_get_info()[0]
    for seeding in ("context", "self_salt"):
        sbw.watermark(x, p, KEY, 0.25, 2.0, seeding)
        sbw.detect(tok, KEY, 0.25, seeding, counts=counts, z=z)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == alloc0
    assert torch.cuda.mem_get_info()[0] == free0


# --- the five workload configurations at full size ---------------------------------

def test_config_c1(env):
    x, prev = workloads.watermark_inputs("c1")
    c = workloads.C1
    say("c1 watermark")
    got = run_watermark(env, x, prev, KEY, c["gamma"], c["delta"], c["seeding"])
    assert_logits_equal(got, oracle.watermark(x, prev, KEY, c["gamma"], c["delta"], c["seeding"]))
    tok = workloads.uniform_tokens(c["detect_N"], c["detect_L"], c["V"], workloads.rng_for("c1", 1))
    for seeding in ("context", "self_salt"):
        say(f"c1 detect {seeding}")
        assert_detect_equal(run_detect(env, tok, KEY, c["gamma"], seeding),
                            oracle.detect(tok, KEY, c["gamma"], seeding))


def test_config_c2_sweep(env):
    x, prev = workloads.watermark_inputs("c2")
    c = workloads.C2
    for gamma, delta in c["sweep"]:
        say(f"c2 bf16 gamma={gamma} delta={delta}")
        got = run_watermark(env, x, prev, KEY, gamma, delta, c["seeding"])
        assert_logits_equal(got, oracle.watermark(x, prev, KEY, gamma, delta, c["seeding"]),
                            f"c2 {gamma} {delta}")


def test_config_c3(env):
    x, prev = workloads.watermark_inputs("c3")
    c = workloads.C3
    say("c3 self-salt")
    got = run_watermark(env, x, prev, KEY, c["gamma"], c["delta"], c["seeding"])
    assert_logits_equal(got, oracle.watermark(x, prev, KEY, c["gamma"], c["delta"], c["seeding"]))


@pytest.mark.parametrize("seeding", ["self_salt", "context"])
@pytest.mark.parametrize("large", [False, True])
def test_config_c4(env, seeding, large):
    c = workloads.C4
    B = c["B_large"] if large else c["B"]
    x, prev = workloads.watermark_inputs("c4", B=B)
    say(f"c4 B={B} {seeding}")
    got = run_watermark(env, x, prev, KEY, c["gamma"], c["delta"], seeding)
    expect = oracle.watermark(x, prev, KEY, c["gamma"], c["delta"], seeding)
    assert_logits_equal(got, expect, f"c4 B={B} {seeding}")


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_config_c5(env, seeding):
    c = workloads.C5

    def member(p, v):
        return oracle.is_green_many(KEY, p, v, c["gamma"], seeding)

    tok = workloads.detect_inputs(c["N"], c["L"], c["V"], c["gamma"], c["delta"], seeding, member)
    say(f"c5 detect {seeding}")
    got = run_detect(env, tok, KEY, c["gamma"], seeding)
    expect = oracle.detect(tok, KEY, c["gamma"], seeding)
    assert_detect_equal(got, expect)
    # the watermarked half is detected, the null half is not
    z = expect[1]
    assert np.median(z[c["N"] // 2:]) > 15 and abs(np.median(z[: c["N"] // 2])) < 1


BF16_DELTAS = [2.0 ** -149, -(2.0 ** -149), 1e-40, -3e-39, 1e-38, 1e-30, -1e-20, 1e-10, 3e-5,
               -1e-3, 0.0078125, 0.1, -0.3, 0.5, 1.0, -1.0, 1.5, 2.0, 3.0, -7.0, 8.0, 10.0,
               100.0, -1e3, 12345.678, 1e6, -3e7, 1e10, 1e20, -1e30, 3e38, -3e38, 0.0, -0.0,
               1 / 3, 2 / 3, math.pi, -math.e, math.sqrt(2)]


@pytest.mark.parametrize("layout", ["vector", "unaligned"])
def test_bf16_rounding_every_pattern(env, layout):
    # Every bf16 bit pattern, all green (gamma = 1), one fp32 add and one rounding to
    # bf16 per element, for deltas from the smallest subnormal to 3e38: covers ties,
    # carries into the exponent, overflow to infinity, subnormal sums and NaN inputs.
    x = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(1, -1)
    prev = np.array([7], dtype=np.int32)
    for delta in BF16_DELTAS:
        say(f"bf16 rounding {layout} delta={delta!r}")
        if layout == "vector":
            got = run_watermark(env, x, prev, KEY, 1.0, delta, "context")
        else:
            got = run_watermark(env, x, prev, KEY, 1.0, delta, "context", offset=1)
        assert_logits_equal(got, oracle.watermark(x, prev, KEY, 1.0, delta, "context"),
                            f"bf16 delta={delta!r}")


@pytest.mark.parametrize("dtype,B,V", [
    ("f32", 512, 131075),     # 268.4 MB of logits, just past 256 MiB: whole rows per XCD
    ("bf16", 1024, 131075),   # the same bytes in bf16
    ("f32", 515, 1000),       # not a multiple of 8 rows: the plain order
])
def test_context_xcd_rows(env, dtype, B, V):
    """Context-seeded launches of at least 512 rows, a multiple of 8, and more logit
    bytes than the Infinity Cache holds renumber their workgroups so that each XCD takes
    whole rows; rows padded to 16 bytes so that the vector kernel takes them."""
    rng = np.random.default_rng(5120 + B + V)
    x = special_logits(rng, B, V, dtype)
    prev = rng.integers(0, 1 << 31, B).astype(np.int32)
    say(f"context xcd rows {dtype} B={B} V={V}")
    torch, sbw, dev = env
    stride = -(-V // 8) * 8
    t = torch.zeros((B, stride), dtype=torch.bfloat16 if dtype == "bf16" else torch.float32,
                    device=dev)
    t[:, :V] = _to_device(torch, dev, x)
    sbw.watermark(t[:, :V], torch.from_numpy(prev).to(dev), WIDE, 0.25, 2.0, "context")
    torch.cuda.synchronize()
    out = _from_device(torch, t)
    assert_logits_equal(out[:, :V], oracle.watermark(x, prev, WIDE, 0.25, 2.0, "context"),
                        f"{dtype} B={B} V={V}")
    assert not out[:, V:].any(), "the padding columns were written"


@pytest.mark.parametrize("dtype,B,V,width,rows", [
    ("f32", 75, 152063, 1, 4),      # 149 tiles x 19 / 20 groups of 4 rows, last group of 3 / 1;
    ("f32", 77, 152061, 1, 4),      #   6-row slabs would make 13 x 149 < 2000 workgroups
    ("bf16", 151, 152063, 1, 2),    # bf16 takes at most 2 rows; 4 groups per workgroup (the
                                    #   next one loaded while the current one is drawn)
    ("f32", 221, 151937, 4, 1),     # width 4 (SBW-ss-V) keeps one row per workgroup
    ("f32", 63, 128256, 1, 4),      # c3's launch, last group of 3
    ("f32", 33, 128256, 1, 4),      # last group of 1
    ("bf16", 67, 128256, 1, 2),     # 2-row groups, two per workgroup, last group of 1
])
def test_self_salt_row_groups(env, dtype, B, V, width, rows):
    """Self-salt launches of the sizes at which a workgroup shares the candidate terms
    across `rows` rows (width 1 with enough workgroups), with a partial last vector
    (rows padded to a multiple of 16 bytes, so that the vector kernels take them) and a
    partial last row group."""
    rng = np.random.default_rng(230 + B + width)
    x = special_logits(rng, B, V, dtype)
    ctx = workloads.context_tokens(B, width, V, rng)
    say(f"self-salt row groups {dtype} B={B} V={V} h={width} rows={rows}")
    torch, sbw, dev = env
    stride = -(-V // 8) * 8
    t = torch.zeros((B, stride), dtype=torch.bfloat16 if dtype == "bf16" else torch.float32,
                    device=dev)
    t[:, :V] = _to_device(torch, dev, x)
    c = torch.from_numpy(ctx).to(dev)
    sbw.watermark(t[:, :V], c if width > 1 else c[:, 0].contiguous(), WIDE, 0.25, 2.0, "self_salt")
    torch.cuda.synchronize()
    expect = oracle.watermark_w(x, ctx, WIDE, 0.25, 2.0, "self_salt")
    out = _from_device(torch, t)
    assert_logits_equal(out[:, :V], expect, f"{dtype} B={B} V={V} h={width}")
    assert not out[:, V:].any(), "the padding columns were written"
