"""GPU parity of the context-window entry points (width h; SBW-4 and SBW-ss-V).

Watermarked logits, masks and green counts bit-identical to the oracle; z within
1e-6 relative.  Widths 1..8, ragged shapes, both dtypes and seedings, and the
paper's width-4 schemes at the c4 (B=256, V=152064) and c5 (4096 x 512) sizes.
"""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_parity import (KEY, WIDE, assert_detect_equal, assert_logits_equal, env,  # noqa: F401
                             say, special_logits, _to_device, _from_device)

pytestmark = pytest.mark.gpu


def run_watermark_w(env, x, ctx, key, gamma, delta, seeding):
    torch, sbw, dev = env
    t = _to_device(torch, dev, x)
    c = torch.from_numpy(np.ascontiguousarray(ctx, dtype=np.int32)).to(dev)
    sbw.watermark(t, c, key, gamma, delta, seeding)
    torch.cuda.synchronize()
    return _from_device(torch, t)


def run_detect_w(env, tok, width, key, gamma, seeding):
    torch, sbw, dev = env
    t = torch.from_numpy(np.ascontiguousarray(tok)).to(dev)
    counts, z = sbw.detect(t, key, gamma, seeding, width=width)
    torch.cuda.synchronize()
    return counts.cpu().numpy(), z.cpu().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 2, 4, 8])
@pytest.mark.parametrize("B,V", [(1, 5), (3, 33), (4, 4097), (2, 32001)])
def test_watermark_window(env, dtype, seeding, width, B, V):
    rng = np.random.default_rng(width * 1000 + B * 7 + V)
    x = special_logits(rng, B, V, dtype)
    ctx = workloads.context_tokens(B, width, max(V, 2), rng)
    ctx[0, 0] = -1  # a 32-bit pattern outside the vocabulary
    for gamma, delta, key in [(0.25, 2.0, KEY), (0.5, -1.5, WIDE)]:
        say(f"window watermark {dtype} {seeding} h={width} B={B} V={V} gamma={gamma}")
        got = run_watermark_w(env, x, ctx, key, gamma, delta, seeding)
        assert_logits_equal(got, oracle.watermark_w(x, ctx, key, gamma, delta, seeding),
                            f"{dtype}/{seeding}/h={width}/{B}x{V}")


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [2, 3, 4, 8])
def test_green_mask_window(env, seeding, width):
    torch, sbw, dev = env
    rng = np.random.default_rng(50 + width)
    B, V = 5, 4129
    ctx = workloads.context_tokens(B, width, V, rng)
    for gamma in (0.25, 0.5, 1.0, 0.0):
        say(f"window mask {seeding} h={width} gamma={gamma}")
        out = sbw.green_mask(torch.from_numpy(ctx).to(dev), V, WIDE, gamma, seeding)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().view(np.uint32),
                              oracle.green_mask_w(B, V, ctx, WIDE, gamma, seeding))


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 2, 4, 5, 8])
@pytest.mark.parametrize("N,L", [(3, 0), (3, 4), (4, 5), (5, 9), (6, 69), (7, 200), (5, 600)])
def test_detect_window(env, seeding, width, N, L):
    rng = np.random.default_rng(width * 97 + N * 31 + L)
    tok = rng.integers(-(1 << 31), 1 << 31, (N, L), dtype=np.int64).astype(np.int32)
    tok[:, ::2] = rng.integers(0, 50, tok[:, ::2].shape)
    for gamma in (0.25, 0.5):
        say(f"window detect {seeding} h={width} N={N} L={L} gamma={gamma}")
        assert_detect_equal(run_detect_w(env, tok, width, WIDE, gamma, seeding),
                            oracle.detect_w(tok, width, WIDE, gamma, seeding))


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_paper_width4_schemes_at_c4_size(env, seeding):
    # SBW-4 (context) and SBW-ss-V (self-salt) at B=256, V=152064 fp32.
    c = workloads.C4
    x, _ = workloads.watermark_inputs("c4")
    ctx = workloads.context_tokens(c["B"], 4, c["V"], workloads.rng_for("c4", 3))
    say(f"c4 width-4 {seeding}")
    got = run_watermark_w(env, x, ctx, KEY, c["gamma"], c["delta"], seeding)
    assert_logits_equal(got, oracle.watermark_w(x, ctx, KEY, c["gamma"], c["delta"], seeding),
                        f"c4 h=4 {seeding}")


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_paper_width4_detect_at_c5_size(env, seeding):
    c = workloads.C5

    def member(window, v):
        return oracle.is_green_w_many(KEY, window, v, c["gamma"], seeding)

    tok = workloads.detect_inputs(c["N"], c["L"], c["V"], c["gamma"], c["delta"], seeding, member,
                                  width=4)
    say(f"c5 width-4 detect {seeding}")
    got = run_detect_w(env, tok, 4, KEY, c["gamma"], seeding)
    expect = oracle.detect_w(tok, 4, KEY, c["gamma"], seeding)
    assert_detect_equal(got, expect)
    z = expect[1]
    assert np.median(z[c["N"] // 2:]) > 15 and abs(np.median(z[: c["N"] // 2])) < 1
