"""GPU parity of the self-salt split-term slab kernel (fp32 and bf16, window of one token).

Large self-salt launches take a kernel that draws each column's self-term block once
per slab of 12 rows (8, then 6, for launches that taller slabs would leave with too few
workgroups) and queues in LDS only the (row, token) pairs whose row term is the
smaller one.  Every case here is sized to take that kernel (the launch rule is
mirrored in `slab_rows` and asserted), and is compared with the oracle bit for bit:
  * slabs cut short (B not a multiple of 12), a row tail (V mod 4 != 0), the last
    workgroup tile partly past the row, padded rows;
  * special values (NaNs with payloads, infinities, signed zeros, subnormals);
  * gamma from tiny to 1 (every token green), both key shapes, both signs of delta;
  * a vocabulary shard whose first token id is a multiple of 4, as one of 8
    tensor-parallel heads of the 152064-token vocabulary holds it;
  * two launches back to back, the second smaller (nothing a launch leaves in LDS
    changes the next one);
  * more slabs than the grid's y dimension holds (workgroups that take two).
The c4 configurations at full size (B = 256 and 1024) take this kernel too and are
checked in test_gpu_parity.py.
"""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_parity import (KEY, WIDE, _from_device, _to_device, assert_logits_equal, env,  # noqa: F401
                             say, special_logits)

pytestmark = pytest.mark.gpu

SLAB_ROWS = 12
MIN_GROUPS_12 = 3000  # workgroups below which 12-row slabs give way to 8-row ones
MIN_GROUPS = 2000     # workgroups below which 8- and 6-row slabs give way


def slab_rows(B, V, dtype="f32"):
    """The launch rule of the self-salt watermark, window of one token (rows 16-byte
    aligned): the slab height the launch takes, or 0 for the row-group kernel."""
    per = 4 if dtype == "f32" else 8     # tokens in a 16-byte vector
    tiles = -(-(-(-V // per)) // 256)
    if tiles * -(-B // 12) >= MIN_GROUPS_12:
        return 12
    for rows in (8, 6):
        if tiles * -(-B // rows) >= MIN_GROUPS:
            return rows
    return 0


def takes_slab(B, V):
    return slab_rows(B, V) == SLAB_ROWS


def run(env, x, prev, key, gamma, delta, stride=None, v_offset=None):
    """Watermarks x in a device buffer of rows `stride` elements apart: by default V when
    that keeps every row 16-byte aligned, else V rounded up to a multiple of 8 (rows that
    are not aligned take the element-wise kernel instead)."""
    torch, sbw, dev = env
    B, V = x.shape
    if stride is None and (V * x.itemsize) % 16 != 0:
        stride = -(-V // 8) * 8
    if stride is None:
        t = _to_device(torch, dev, x)
        view = t
    else:
        dt = torch.bfloat16 if x.dtype == np.uint16 else torch.float32
        t = torch.zeros((B, stride), dtype=dt, device=dev)
        t[:, :V] = _to_device(torch, dev, x)
        view = t[:, :V]
    p = torch.from_numpy(prev).to(dev)
    if v_offset is None:
        sbw.watermark(view, p, key, gamma, delta, "self_salt")
    else:
        sbw.watermark_shard(view, p, v_offset, key, gamma, delta, "self_salt")
    torch.cuda.synchronize()
    out = _from_device(torch, t)
    return out if stride is None else out[:, :V], (None if stride is None else out[:, V:])


@pytest.mark.parametrize("B,V,stride", [
    (4501, 8195, None),      # slab of 1 row at the end, V mod 4 = 3, 2049 vectors (tile of 1)
    (3600, 10241, 10248),    # whole slabs, padded rows, V mod 4 = 1
    (2125, 16386, None),     # V mod 4 = 2, last tile partly past the row
    (893, 40000, 40004),     # whole vectors, padded rows, slab of 5 rows at the end
])
def test_slab_shapes(env, B, V, stride):
    assert takes_slab(B, V)
    rng = np.random.default_rng(77 + B + V)
    x = special_logits(rng, B, V, "f32")
    prev = rng.integers(0, 1 << 31, B).astype(np.int32)
    prev[:3] = [0, -1, 2**31 - 1]
    say(f"slab shapes B={B} V={V} stride={stride}")
    got, pad = run(env, x, prev, WIDE, 0.25, 2.0, stride)
    assert_logits_equal(got, oracle.watermark(x, prev, WIDE, 0.25, 2.0, "self_salt"),
                        f"B={B} V={V}")
    if pad is not None:
        assert not pad.any(), "the padding columns were written"


@pytest.mark.parametrize("gamma,delta,key", [
    (0.25, 2.0, KEY),
    (0.5, -3.0, WIDE),
    (1e-9, 8.0, WIDE),       # almost no token green
    (1.0 - 1e-10, 1.0, KEY),
    (1.0, 4.0, WIDE),        # every token green
])
def test_slab_parameters(env, gamma, delta, key):
    B, V = 2762, 12292
    assert takes_slab(B, V)
    rng = np.random.default_rng(int(gamma * 1e6) + int(delta * 10) + 5)
    x = rng.standard_normal((B, V)).astype(np.float32)
    prev = rng.integers(0, V, B).astype(np.int32)
    say(f"slab parameters gamma={gamma} delta={delta}")
    got, _ = run(env, x, prev, key, gamma, delta)
    assert_logits_equal(got, oracle.watermark(x, prev, key, gamma, delta, "self_salt"),
                        f"gamma={gamma} delta={delta}")


def test_slab_shard(env):
    """Columns [57024, 57024 + 19008) of a 152064-token vocabulary (one of 8 shards) at
    B = 1900: token ids from 57024, the draws those of the full row."""
    a, n, V, B = 57024, 19008, 152064, 1900
    assert takes_slab(B, n)
    rng = np.random.default_rng(4242)
    x = rng.standard_normal((B, n)).astype(np.float32) * np.float32(3)
    prev = rng.integers(0, V, B).astype(np.int32)
    say("slab shard 57024+19008, B=1900")
    got, _ = run(env, x, prev, WIDE, 0.25, 2.0, v_offset=a)
    # the oracle's membership of tokens a .. a+n-1 in each row, and its fp32 bias
    green = oracle.is_green_many(WIDE, np.repeat(prev, n), np.tile(np.arange(a, a + n), B), 0.25,
                                 "self_salt").reshape(B, n)
    expect = np.where(green, oracle.bias_f32_many(x, 2.0), x)
    assert_logits_equal(got, expect, "shard")


def test_slab_twice_in_a_row(env):
    """Two launches back to back, the second smaller, on fresh inputs each: nothing a
    launch leaves in LDS or in the logits changes the next one's result."""
    rng = np.random.default_rng(99)
    for B, V in ((3000, 12300), (2900, 12299)):
        assert takes_slab(B, V)
        x = rng.standard_normal((B, V)).astype(np.float32)
        prev = rng.integers(0, V, B).astype(np.int32)
        say(f"slab twice B={B} V={V}")
        got, _ = run(env, x, prev, KEY, 0.25, 2.0)
        assert_logits_equal(got, oracle.watermark(x, prev, KEY, 0.25, 2.0, "self_salt"),
                            f"B={B} V={V}")


def test_slab_grid_stride(env):
    """More slabs than the 65535 workgroups of the grid's y dimension: some workgroups
    take a second slab (and 800003 rows of 6 logits: a 2-logit row tail, a last slab of
    11 rows)."""
    B, V = 800003, 6
    assert takes_slab(B, V) and -(-B // SLAB_ROWS) > 65535
    rng = np.random.default_rng(5150)
    x = rng.standard_normal((B, V)).astype(np.float32)
    prev = rng.integers(0, 1 << 20, B).astype(np.int32)
    say(f"slab grid stride B={B} V={V}")
    got, _ = run(env, x, prev, WIDE, 0.25, 2.0)
    assert_logits_equal(got, oracle.watermark(x, prev, WIDE, 0.25, 2.0, "self_salt"), "grid stride")


@pytest.mark.parametrize("B,V", [
    (128, 128256),    # whole 8-row slabs
    (131, 128255),    # a last slab of 3 rows, V mod 4 = 3
])
def test_slab_eight_rows(env, B, V):
    """Launches that 12-row slabs would leave with too few workgroups (here under 2000;
    below 3000 as well) take 8-row ones."""
    assert slab_rows(B, V) == 8
    rng = np.random.default_rng(808 + B)
    x = special_logits(rng, B, V, "f32")
    prev = rng.integers(0, V, B).astype(np.int32)
    say(f"slab 8 rows B={B} V={V}")
    got, _ = run(env, x, prev, WIDE, 0.25, 2.0)
    assert_logits_equal(got, oracle.watermark(x, prev, WIDE, 0.25, 2.0, "self_salt"),
                        f"B={B} V={V}")


@pytest.mark.parametrize("B,V", [
    (96, 128256),     # whole 6-row slabs
    (101, 128255),    # a last slab of 5 rows, V mod 4 = 3
    (80, 152064),
])
def test_slab_six_rows(env, B, V):
    """Launches that 8-row slabs would leave with too few workgroups take 6-row ones."""
    assert slab_rows(B, V) == 6
    rng = np.random.default_rng(606 + B)
    x = special_logits(rng, B, V, "f32")
    prev = rng.integers(0, V, B).astype(np.int32)
    say(f"slab 6 rows B={B} V={V}")
    got, _ = run(env, x, prev, KEY, 0.5, -2.0)
    assert_logits_equal(got, oracle.watermark(x, prev, KEY, 0.5, -2.0, "self_salt"),
                        f"B={B} V={V}")


@pytest.mark.parametrize("B,V,stride,rows", [
    (3600, 20483, None, 12),      # V mod 8 = 3, a tile of 1 vector at the end
    (3607, 20480, 20488, 12),     # padded rows, a last slab of 7 rows
    (256, 152064, None, 8),       # the c4 shape in bf16: 8-row slabs
    (263, 152061, None, 8),       # a last slab of 7 rows, V mod 8 = 5
    (192, 152064, None, 6),       # 6-row slabs
    (197, 152061, None, 6),       # a last slab of 5 rows, V mod 8 = 5
])
def test_slab_bf16(env, B, V, stride, rows):
    """bf16 logits: 8 tokens a vector, two Philox counters a lane, 8 map bytes a row."""
    assert slab_rows(B, V, "bf16") == rows
    rng = np.random.default_rng(1616 + B + V)
    x = special_logits(rng, B, V, "bf16")
    prev = rng.integers(0, 1 << 31, B).astype(np.int32)
    prev[:2] = [0, -1]
    say(f"slab bf16 B={B} V={V} stride={stride}")
    got, pad = run(env, x, prev, WIDE, 0.25, 2.0, stride)
    assert_logits_equal(got, oracle.watermark(x, prev, WIDE, 0.25, 2.0, "self_salt"),
                        f"bf16 B={B} V={V}")
    if pad is not None:
        assert not pad.any(), "the padding columns were written"


def test_slab_bf16_shard(env):
    """A bf16 vocabulary shard whose first token id is a multiple of 8 (not of 16)."""
    a, n, V, B = 57024 + 8, 19000, 152064, 3600
    assert slab_rows(B, n, "bf16") == 12
    rng = np.random.default_rng(4343)
    x = workloads.f32_to_bf16_bits(rng.standard_normal((B, n)).astype(np.float32) * np.float32(2))
    prev = rng.integers(0, V, B).astype(np.int32)
    say("slab bf16 shard 57032+19000, B=3600")
    got, _ = run(env, x, prev, KEY, 0.5, -1.5, v_offset=a)
    green = oracle.is_green_many(KEY, np.repeat(prev, n), np.tile(np.arange(a, a + n), B), 0.5,
                                 "self_salt").reshape(B, n)
    expect = np.where(green, oracle.bias_bf16_many(x, -1.5), x)
    assert_logits_equal(got, expect, "bf16 shard")


def test_launch_rule_cases():
    """The c4 configurations take 12-row slabs, B = 160-240 of 152064 tokens and B = 128
    of 128256 8-row ones, B = 96 6-row ones; c3 and small batches take the row-group
    kernel."""
    assert slab_rows(256, 152064) == 12 and slab_rows(1024, 152064) == 12
    assert slab_rows(160, 152064) == 8 and slab_rows(240, 152064) == 8
    assert slab_rows(128, 128256) == 8 and slab_rows(96, 128256) == 6
    assert slab_rows(64, 128256) == 0 and slab_rows(16, 152064) == 0
    assert slab_rows(256, 152064, "bf16") == 8 and slab_rows(1024, 152064, "bf16") == 12
    assert slab_rows(192, 152064, "bf16") == 6 and slab_rows(151, 152063, "bf16") == 0
