"""sbw_watermark_argmax_noalloc (the greedy decoding call for callers that cannot
allocate) against sbw_watermark_argmax with a caller workspace, through the C ABI:
tokens equal and values bit-equal on consecutive calls whose sizes shrink, so the
second call runs on a scratch array that still holds the first call's partials."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import workloads

pytestmark = pytest.mark.gpu

KEY = workloads.PAPER_KEY
SEEDINGS = {"context": 0, "self_salt": 1}


@pytest.fixture(scope="module")
def sbw():
    import paper_2609_03844_amd as sbw
    return sbw


def _args(logits, context):
    dtype = 0 if logits.dtype == torch.float32 else 1
    B, V = logits.shape
    width = 1 if context.dim() == 1 else context.shape[1]
    stride = logits.stride(0) if B > 1 else max(V, logits.stride(0))
    return dtype, B, V, stride, width


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def noalloc(lib, logits, context, gamma, delta, seeding):
    dtype, B, V, stride, width = _args(logits, context)
    tokens = torch.full((B,), -7, dtype=torch.int32, device=logits.device)
    values = torch.full((B,), 1.5, dtype=torch.float32, device=logits.device)
    st = lib.sbw_watermark_argmax_noalloc(logits.data_ptr(), dtype, B, V, stride,
                                          context.data_ptr(), width, KEY, gamma, delta,
                                          SEEDINGS[seeding], tokens.data_ptr(),
                                          values.data_ptr(), _stream())
    assert st == 0, lib.sbw_strerror(st)
    return tokens, values


def with_workspace(lib, logits, context, gamma, delta, seeding):
    dtype, B, V, stride, width = _args(logits, context)
    tokens = torch.full((B,), -9, dtype=torch.int32, device=logits.device)
    values = torch.full((B,), -2.5, dtype=torch.float32, device=logits.device)
    ws = torch.empty(max(1, lib.sbw_watermark_argmax_workspace(B, V)), dtype=torch.int64,
                     device=logits.device)
    st = lib.sbw_watermark_argmax(logits.data_ptr(), dtype, B, V, stride, context.data_ptr(),
                                  width, KEY, gamma, delta, SEEDINGS[seeding], tokens.data_ptr(),
                                  values.data_ptr(), ws.data_ptr(), _stream())
    assert st == 0, lib.sbw_strerror(st)
    return tokens, values


def _same(a, b):
    ta, va = a
    tb, vb = b
    torch.cuda.synchronize()
    assert torch.equal(ta.cpu(), tb.cpu())
    assert np.array_equal(va.cpu().numpy().view(np.uint32), vb.cpu().numpy().view(np.uint32))


def _logits(B, V, dtype, seed, pad=0, offset=0):
    rng = np.random.default_rng(seed)
    x = (3.0 * rng.standard_normal((B, V + pad + offset))).astype(np.float32)
    x[rng.random(x.shape) < 0.05] += 8.0
    t = torch.from_numpy(x).cuda()
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t[:, offset:offset + V]


CASES = [
    # (B, V, dtype, width, seeding, gamma, delta, pad, offset): each later case is smaller
    (256, 152064, "f32", 1, "self_salt", 0.25, 2.0, 0, 0),
    (37, 32001, "bf16", 4, "context", 0.5, 4.0, 0, 0),
    (5, 6000, "f32", 1, "context", 0.25, -3.0, 3, 1),      # unaligned rows: element path
    (1, 7, "bf16", 2, "self_salt", 1.0, 2.0, 0, 0),
]


def test_noalloc_matches_workspace_call_on_shrinking_inputs(sbw):
    lib = sbw.raw()
    rng = np.random.default_rng(11)
    for i, (B, V, dt, width, seeding, gamma, delta, pad, off) in enumerate(CASES):
        print(f"case {i}: B={B} V={V} {dt} width={width} {seeding}", flush=True)
        x = _logits(B, V, dt, 100 + i, pad, off)
        ctx = torch.from_numpy(workloads.context_tokens(B, width, V, rng)).cuda()
        if width == 1:
            ctx = ctx[:, 0].contiguous()
        got = noalloc(lib, x, ctx, gamma, delta, seeding)
        _same(got, with_workspace(lib, x, ctx, gamma, delta, seeding))
        # the same call again, after the workspace call: the scratch holds the same partials
        _same(noalloc(lib, x, ctx, gamma, delta, seeding), got)


def test_noalloc_second_call_smaller_against_the_oracle(sbw):
    lib = sbw.raw()
    rng = np.random.default_rng(12)
    for B, V in ((64, 40000), (3, 9001)):
        x = rng.standard_normal((B, V)).astype(np.float32)
        prev = rng.integers(0, V, B).astype(np.int32)
        t, p = torch.from_numpy(x).cuda(), torch.from_numpy(prev).cuda()
        for seeding in ("context", "self_salt"):
            tok, val = noalloc(lib, t, p, 0.25, 2.0, seeding)
            et, ev = oracle.watermark_argmax(x, prev, KEY, 0.25, 2.0, seeding)
            torch.cuda.synchronize()
            assert np.array_equal(tok.cpu().numpy(), et)
            assert np.array_equal(val.cpu().numpy().view(np.uint32), ev.view(np.uint32))


def test_noalloc_at_its_size_limit(sbw):
    lib = sbw.raw()
    V = 152064
    B = 262144 // 75          # 3495 rows: 262125 partials, the most that fit
    assert lib.sbw_watermark_argmax_workspace(B, V) <= sbw.NOALLOC_SCRATCH_ELEMS
    assert lib.sbw_watermark_argmax_workspace(B + 1, V) > sbw.NOALLOC_SCRATCH_ELEMS
    x = _logits(B, V, "f32", 7)
    prev = torch.from_numpy(np.random.default_rng(13).integers(0, V, B).astype(np.int32)).cuda()
    for seeding in ("context", "self_salt"):
        _same(noalloc(lib, x, prev, 0.25, 2.0, seeding),
              with_workspace(lib, x, prev, 0.25, 2.0, seeding))
    # one row more is refused before any HIP call (every buffer is sized for it anyway)
    del x
    y = torch.zeros((B + 1, V), dtype=torch.float32, device="cuda")
    prev1 = torch.zeros(B + 1, dtype=torch.int32, device="cuda")
    tok1 = torch.full((B + 1,), -7, dtype=torch.int32, device="cuda")
    st = lib.sbw_watermark_argmax_noalloc(y.data_ptr(), 0, B + 1, V, V, prev1.data_ptr(), 1,
                                          KEY, 0.25, 2.0, 0, tok1.data_ptr(), None, _stream())
    assert st == 4   # SBW_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((tok1 == -7).all())


def test_noalloc_allocates_no_device_memory(sbw):
    lib = sbw.raw()
    x = _logits(64, 152064, "f32", 3)
    prev = torch.from_numpy(np.arange(64, dtype=np.int32)).cuda()
    tokens = torch.empty(64, dtype=torch.int32, device="cuda")
    values = torch.empty(64, dtype=torch.float32, device="cuda")

    def call():
        st = lib.sbw_watermark_argmax_noalloc(x.data_ptr(), 0, 64, 152064, 152064,
                                              prev.data_ptr(), 1, KEY, 0.25, 2.0, 1,
                                              tokens.data_ptr(), values.data_ptr(), _stream())
        assert st == 0
    call()
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    alloc0 = torch.cuda.memory_allocated()
    for _ in range(20):
        call()
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] == free0
    assert torch.cuda.memory_allocated() == alloc0


def test_noalloc_binding(sbw):
    rng = np.random.default_rng(14)
    x = rng.standard_normal((9, 20000)).astype(np.float32)
    prev = rng.integers(0, 20000, 9).astype(np.int32)
    t, p = torch.from_numpy(x).cuda(), torch.from_numpy(prev).cuda()
    for seeding in ("context", "self_salt"):
        a = sbw.watermark_argmax_noalloc(t, p, KEY, 0.25, 2.0, seeding)
        b = sbw.watermark_argmax(t, p, KEY, 0.25, 2.0, seeding)
        _same(a, b)
