"""The C ABI on the CPU: the library loads, exports what include/sbw.h declares,
and rejects bad arguments on the host before any HIP call.

No test here launches a kernel: calls that would pass validation are only made
where no GPU is visible (they must then return SBW_ERR_NO_DEVICE).
"""
import ctypes
import math
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sbw.h")

OK, INVALID, GAMMA, DELTA, UNSUPPORTED, NO_DEVICE, HIP = range(7)


@pytest.fixture(scope="module")
def sbw():
    import paper_2609_03844_amd as sbw
    return sbw


@pytest.fixture(scope="module")
def lib(sbw):
    return sbw.raw()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(sbw_[a-z_0-9]+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    assert _declared() == ["sbw_detect", "sbw_detect_ex", "sbw_detect_window", "sbw_green_mask",
                           "sbw_green_mask_window", "sbw_last_hip_error", "sbw_strerror",
                           "sbw_version", "sbw_watermark", "sbw_watermark_argmax",
                           "sbw_watermark_argmax_noalloc", "sbw_watermark_argmax_shard",
                           "sbw_watermark_argmax_workspace",
                           "sbw_watermark_candidates", "sbw_watermark_sample",
                           "sbw_watermark_sample_shard", "sbw_watermark_shard",
                           "sbw_watermark_window"]


def test_library_exports_every_declared_symbol(sbw, lib):
    out = subprocess.run(["nm", "-D", "--defined-only", sbw.library_path()], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(sbw_\w+)$", out, re.M))
    for name in _declared():
        assert name in exported, name
        assert hasattr(lib, name)
    assert set(sbw.EXPORTED) == set(_declared())


def test_library_is_gfx950_code():
    # the device code bundled into the library targets gfx950
    import paper_2609_03844_amd as sbw
    sections = subprocess.run(["readelf", "-S", "-W", sbw.library_path()], capture_output=True,
                              text=True, check=True).stdout
    assert ".hip_fatbin" in sections
    assert b"amdgcn-amd-amdhsa--gfx950" in open(sbw.library_path(), "rb").read()


def test_strerror_and_version(lib, sbw):
    for code in range(7):
        s = lib.sbw_strerror(code)
        assert s and len(s) > 3
    assert lib.sbw_strerror(99) == b"unknown status"
    assert re.fullmatch(r"\d+\.\d+\.\d+", sbw.version())
    assert lib.sbw_last_hip_error().startswith(b"hip")


# A dummy non-null pointer; validation rejects the call before it could be used.
DUMMY = ctypes.c_void_p(0x1000)
NULL = None
KEY = 15485863


def wm(lib, logits=DUMMY, dtype=0, B=2, V=8, stride=8, prev=DUMMY, gamma=0.25, delta=2.0,
       seeding=0):
    return lib.sbw_watermark(logits, dtype, B, V, stride, prev, KEY, gamma, delta, seeding, None)


def gm(lib, bits=DUMMY, B=2, V=8, prev=DUMMY, gamma=0.25, seeding=0):
    return lib.sbw_green_mask(bits, B, V, prev, KEY, gamma, seeding, None)


def det(lib, tokens=DUMMY, N=2, L=8, stride=8, gamma=0.25, seeding=0, counts=DUMMY, z=DUMMY):
    return lib.sbw_detect(tokens, N, L, stride, KEY, gamma, seeding, counts, z, None)


def test_watermark_rejects_bad_arguments(lib):
    assert wm(lib, B=-1) == INVALID
    assert wm(lib, V=-1) == INVALID
    assert wm(lib, stride=7) == INVALID
    assert wm(lib, logits=NULL) == INVALID
    assert wm(lib, prev=NULL) == INVALID
    assert wm(lib, dtype=2) == UNSUPPORTED
    assert wm(lib, dtype=-1) == UNSUPPORTED
    assert wm(lib, seeding=2) == UNSUPPORTED
    for g in (-0.1, 1.0000001, math.nan, math.inf, -math.inf):
        assert wm(lib, gamma=g) == GAMMA, g
    for d in (math.inf, -math.inf, math.nan):
        assert wm(lib, delta=d) == DELTA, d
    assert wm(lib, V=1 << 32, stride=1 << 32) == UNSUPPORTED
    assert wm(lib, B=1 << 62, V=8, stride=1 << 20) == UNSUPPORTED


def test_watermark_empty_and_noop_calls_succeed_without_hip(lib):
    assert wm(lib, B=0) == OK
    assert wm(lib, V=0, stride=0) == OK
    assert wm(lib, B=0, logits=NULL, prev=NULL) == OK
    # gamma = 0: nothing is green, nothing to do
    assert wm(lib, gamma=0.0) == OK


def test_green_mask_rejects_bad_arguments(lib):
    assert gm(lib, B=-1) == INVALID
    assert gm(lib, V=-1) == INVALID
    assert gm(lib, bits=NULL) == INVALID
    assert gm(lib, prev=NULL) == INVALID
    assert gm(lib, seeding=7) == UNSUPPORTED
    assert gm(lib, gamma=1.5) == GAMMA
    assert gm(lib, gamma=math.nan) == GAMMA
    assert gm(lib, V=1 << 32) == UNSUPPORTED
    assert gm(lib, B=0) == OK
    assert gm(lib, V=0) == OK


def test_detect_rejects_bad_arguments(lib):
    assert det(lib, N=-1) == INVALID
    assert det(lib, L=-1) == INVALID
    assert det(lib, stride=7) == INVALID
    assert det(lib, tokens=NULL) == INVALID
    assert det(lib, counts=NULL) == INVALID
    assert det(lib, z=NULL) == INVALID
    assert det(lib, seeding=3) == UNSUPPORTED
    for g in (0.0, 1.0, -0.5, 2.0, math.nan):
        assert det(lib, gamma=g) == GAMMA, g
    assert det(lib, L=1 << 31, stride=1 << 31) == UNSUPPORTED
    assert det(lib, N=0) == OK
    assert det(lib, N=0, tokens=NULL, counts=NULL, z=NULL) == OK


def _gpu_visible():
    import torch
    return torch.cuda.is_available()


def test_no_device_is_reported():
    import paper_2609_03844_amd as sbw
    if _gpu_visible():
        pytest.skip("a GPU is visible; the no-device path cannot be exercised")
    lib = sbw.raw()
    assert wm(lib) == NO_DEVICE
    assert gm(lib) == NO_DEVICE
    assert det(lib) == NO_DEVICE
    assert det(lib, L=0, tokens=NULL, stride=0) == NO_DEVICE
    assert lib.sbw_last_hip_error() != b"hipSuccess"


def test_python_binding_validates_before_the_c_abi():
    import torch
    import paper_2609_03844_amd as sbw
    with pytest.raises(ValueError):
        sbw.watermark(torch.zeros(3), torch.zeros(1, dtype=torch.int32), KEY, 0.25, 2.0)
    with pytest.raises(TypeError):
        sbw.watermark(torch.zeros(1, 3, dtype=torch.float16), torch.zeros(1, dtype=torch.int32),
                      KEY, 0.25, 2.0)
    with pytest.raises(ValueError):
        sbw.watermark(torch.zeros(2, 3), torch.zeros(2, dtype=torch.int64), KEY, 0.25, 2.0)
    with pytest.raises(ValueError):
        sbw.detect(torch.zeros(2, 3, dtype=torch.int64), KEY, 0.25)
    with pytest.raises(KeyError):
        sbw.watermark(torch.zeros(2, 3), torch.zeros(2, dtype=torch.int32), KEY, 0.25, 2.0,
                      seeding="bogus")


def test_error_codes_surface_as_exceptions():
    import paper_2609_03844_amd as sbw
    with pytest.raises(sbw.SbwError) as e:
        sbw._check(GAMMA)
    assert e.value.code == "SBW_ERR_GAMMA"


def test_status_and_enum_values_match_the_header():
    text = open(HEADER).read()
    enums = dict((k, int(v)) for k, v in re.findall(r"(SBW_[A-Z0-9_]+)\s*=\s*(\d+)", text))
    import paper_2609_03844_amd as sbw
    assert enums["SBW_SEED_CONTEXT"] == sbw.SEED_CONTEXT
    assert enums["SBW_SEED_SELF_SALT"] == sbw.SEED_SELF_SALT
    assert enums["SBW_F32"] == sbw.F32 and enums["SBW_BF16"] == sbw.BF16
    for code, name in sbw._STATUS.items():
        assert enums[name] == code
    # the oracle's scheme codes agree with the library's by value (no shared header)
    import oracle
    assert oracle.SEED_CONTEXT == sbw.SEED_CONTEXT and oracle.SEED_SELF_SALT == sbw.SEED_SELF_SALT


def wmw(lib, width=4, context=DUMMY, **kw):
    a = dict(logits=DUMMY, dtype=0, B=2, V=8, stride=8, gamma=0.25, delta=2.0, seeding=0)
    a.update(kw)
    return lib.sbw_watermark_window(a["logits"], a["dtype"], a["B"], a["V"], a["stride"], context,
                                    width, KEY, a["gamma"], a["delta"], a["seeding"], None)


def test_window_entry_points_reject_bad_arguments(lib):
    for fn in (lambda **k: wmw(lib, **k),
               lambda width=4, context=DUMMY: lib.sbw_green_mask_window(
                   DUMMY, 2, 8, context, width, KEY, 0.25, 0, None),
               lambda width=4, context=DUMMY: lib.sbw_detect_window(
                   context, 2, 8, 8, width, KEY, 0.25, 0, DUMMY, DUMMY, None)):
        assert fn(width=0) == INVALID
        assert fn(width=-3) == INVALID
        assert fn(width=9) == UNSUPPORTED
        assert fn(context=NULL) == INVALID
    assert wmw(lib, B=0) == OK
    assert wmw(lib, seeding=5) == UNSUPPORTED
    assert wmw(lib, gamma=1.5) == GAMMA
    assert lib.sbw_detect_window(DUMMY, 0, 8, 8, 4, KEY, 0.25, 0, NULL, NULL, None) == OK


def test_window_no_device_is_reported():
    import paper_2609_03844_amd as sbw
    if _gpu_visible():
        pytest.skip("a GPU is visible; the no-device path cannot be exercised")
    lib = sbw.raw()
    assert wmw(lib, width=8) == NO_DEVICE
    assert lib.sbw_detect_window(DUMMY, 2, 8, 8, 1, KEY, 0.25, 1, DUMMY, DUMMY, None) == NO_DEVICE


def test_python_binding_window_shapes():
    import torch
    import paper_2609_03844_amd as sbw
    with pytest.raises(ValueError):
        sbw.watermark(torch.zeros(2, 3), torch.zeros(3, 4, dtype=torch.int32), KEY, 0.25, 2.0)
    with pytest.raises(ValueError):
        sbw.watermark(torch.zeros(2, 3), torch.zeros(2, 4, 1, dtype=torch.int32), KEY, 0.25, 2.0)


def am(lib, logits=DUMMY, dtype=0, B=2, V=8, stride=8, context=DUMMY, width=1, gamma=0.25,
       delta=2.0, seeding=0, tokens=DUMMY, values=DUMMY, workspace=DUMMY):
    return lib.sbw_watermark_argmax(logits, dtype, B, V, stride, context, width, KEY, gamma, delta,
                                    seeding, tokens, values, workspace, None)


def test_argmax_rejects_bad_arguments(lib):
    assert am(lib, V=0, stride=0) == INVALID       # no token to choose
    assert am(lib, B=-1) == INVALID
    assert am(lib, stride=7) == INVALID
    for name in ("logits", "context", "tokens", "workspace"):
        assert am(lib, **{name: NULL}) == INVALID, name
    assert am(lib, width=0) == INVALID
    assert am(lib, width=9) == UNSUPPORTED
    assert am(lib, dtype=3) == UNSUPPORTED
    assert am(lib, gamma=-1.0) == GAMMA
    assert am(lib, delta=math.inf) == DELTA
    assert am(lib, B=0) == OK
    if not _gpu_visible():
        assert am(lib, values=NULL) == NO_DEVICE   # values may be NULL


def amn(lib, logits=DUMMY, dtype=0, B=2, V=8, stride=8, context=DUMMY, width=1, gamma=0.25,
        delta=2.0, seeding=0, tokens=DUMMY, values=DUMMY):
    return lib.sbw_watermark_argmax_noalloc(logits, dtype, B, V, stride, context, width, KEY,
                                            gamma, delta, seeding, tokens, values, None)


def test_argmax_noalloc_rejects_bad_arguments(lib, sbw):
    assert sbw.NOALLOC_SCRATCH_ELEMS == 262144
    assert re.search(r"#define SBW_NOALLOC_SCRATCH_ELEMS 262144\b", open(HEADER).read())
    assert amn(lib, V=0, stride=0) == INVALID
    assert amn(lib, B=-1) == INVALID
    assert amn(lib, stride=7) == INVALID
    for name in ("logits", "context", "tokens"):
        assert amn(lib, **{name: NULL}) == INVALID, name
    assert amn(lib, width=9) == UNSUPPORTED
    assert amn(lib, dtype=3) == UNSUPPORTED
    assert amn(lib, seeding=2) == UNSUPPORTED
    assert amn(lib, gamma=2.0) == GAMMA
    assert amn(lib, delta=math.nan) == DELTA
    assert amn(lib, B=0) == OK
    # the partials must fit the static array: B * ceil(V / 2048) <= 262144
    V = 152064
    assert lib.sbw_watermark_argmax_workspace(3495, V) <= 262144 < \
        lib.sbw_watermark_argmax_workspace(3496, V)
    assert amn(lib, B=3496, V=V, stride=V) == UNSUPPORTED
    assert amn(lib, B=262145, V=1, stride=1) == UNSUPPORTED
    assert amn(lib, B=1 << 40, V=1 << 20, stride=1 << 20) == UNSUPPORTED
    if not _gpu_visible():
        # within the limit, validation passes and the device lookup reports its absence
        assert amn(lib, B=3495, V=V, stride=V) == NO_DEVICE
        assert amn(lib, B=262144, V=2048, stride=2048) == NO_DEVICE
        assert amn(lib, values=NULL) == NO_DEVICE


def test_argmax_workspace_size(lib):
    assert lib.sbw_watermark_argmax_workspace(0, 10) == 0
    assert lib.sbw_watermark_argmax_workspace(3, 0) == 0
    assert lib.sbw_watermark_argmax_workspace(1, 1) == 1
    assert lib.sbw_watermark_argmax_workspace(256, 152064) == 256 * 75
    assert lib.sbw_watermark_argmax_workspace(2, 2048) == 2
    assert lib.sbw_watermark_argmax_workspace(2, 2049) == 4


def wc(lib, logits=DUMMY, dtype=0, B=2, V=8, stride=8, cand=DUMMY, k=3, context=DUMMY, width=4,
       gamma=0.25, delta=2.0, seeding=1):
    return lib.sbw_watermark_candidates(logits, dtype, B, V, stride, cand, k, context, width, KEY,
                                        gamma, delta, seeding, None)


def test_candidates_rejects_bad_arguments(lib):
    assert wc(lib, k=-1) == INVALID
    assert wc(lib, B=-1) == INVALID
    assert wc(lib, stride=7) == INVALID
    for name in ("logits", "cand", "context"):
        assert wc(lib, **{name: NULL}) == INVALID, name
    assert wc(lib, k=1025) == UNSUPPORTED
    assert wc(lib, width=9) == UNSUPPORTED
    assert wc(lib, dtype=2) == UNSUPPORTED
    assert wc(lib, seeding=5) == UNSUPPORTED
    assert wc(lib, gamma=1.5) == GAMMA
    assert wc(lib, delta=math.nan) == DELTA
    # no-ops succeed without a device: nothing to do
    assert wc(lib, k=0, cand=NULL) == OK
    assert wc(lib, B=0) == OK
    assert wc(lib, gamma=0.0) == OK
    if not _gpu_visible():
        assert wc(lib) == NO_DEVICE
        assert wc(lib, k=1024) == NO_DEVICE


def dx(lib, tokens=DUMMY, N=2, L=8, stride=8, lengths=NULL, width=1, gamma=0.25, seeding=0,
       flags=0, counts=DUMMY, scored=NULL, z=DUMMY):
    return lib.sbw_detect_ex(tokens, N, L, stride, lengths, width, KEY, gamma, seeding, flags,
                             counts, scored, z, None)


def test_detect_ex_rejects_bad_arguments(lib):
    assert dx(lib, N=-1) == INVALID
    assert dx(lib, stride=7) == INVALID
    for name in ("tokens", "counts", "z"):
        assert dx(lib, **{name: NULL}) == INVALID, name
    assert dx(lib, flags=2) == UNSUPPORTED
    assert dx(lib, width=9) == UNSUPPORTED
    assert dx(lib, seeding=2) == UNSUPPORTED
    assert dx(lib, gamma=0.0) == GAMMA and dx(lib, gamma=1.0) == GAMMA
    # the repeat rule holds up to 4096 scored positions
    assert dx(lib, flags=1, L=4098, stride=4098, width=1) == UNSUPPORTED
    assert dx(lib, N=0, flags=1, L=4097, stride=4097) == OK
    assert dx(lib, N=0) == OK
    if not _gpu_visible():
        assert dx(lib, flags=1, L=4097, stride=4097) == NO_DEVICE
        assert dx(lib, lengths=DUMMY, scored=DUMMY) == NO_DEVICE


def test_binding_rejects_tensors_off_the_device(sbw):
    # a host pointer would reach a kernel: the binding refuses before any HIP call
    import torch
    x = torch.zeros(2, 8)
    prev = torch.zeros(2, dtype=torch.int32)
    with pytest.raises(ValueError, match="current HIP device"):
        sbw.watermark(x, prev, KEY, 0.25, 2.0)
    with pytest.raises(ValueError, match="current HIP device"):
        sbw.watermark_candidates(x, prev, torch.zeros(2, 3, dtype=torch.int32), KEY, 0.25, 2.0)
    with pytest.raises(ValueError, match="current HIP device"):
        sbw.watermark_argmax(x, prev, KEY, 0.25, 2.0, tokens=torch.zeros(2, dtype=torch.int32),
                             values=torch.zeros(2), workspace=torch.zeros(4, dtype=torch.int64))
    with pytest.raises(ValueError, match="current HIP device"):
        sbw.green_mask(prev, 8, KEY, 0.25, out=torch.zeros(2, 1, dtype=torch.int32))
    tok = torch.zeros(2, 5, dtype=torch.int32)
    with pytest.raises(ValueError, match="current HIP device"):
        sbw.detect(tok, KEY, 0.25, counts=torch.zeros(2, dtype=torch.int32),
                   z=torch.zeros(2, dtype=torch.float64))
    with pytest.raises(ValueError, match="current HIP device"):
        sbw.detect_ex(tok, KEY, 0.25)


def ws_(lib, logits=DUMMY, dtype=0, B=2, V=8, stride=8, context=DUMMY, width=1, gamma=0.25,
        delta=2.0, seeding=0, seeds=DUMMY, inv_t=1.0, tokens=DUMMY, scores=DUMMY, workspace=DUMMY):
    return lib.sbw_watermark_sample(logits, dtype, B, V, stride, context, width, KEY, gamma, delta,
                                    seeding, seeds, inv_t, tokens, scores, workspace, None)


def test_sample_rejects_bad_arguments(lib):
    for inv_t in (0.0, -1.0, math.inf, math.nan):
        assert ws_(lib, inv_t=inv_t) == INVALID, inv_t
    for name in ("logits", "context", "seeds", "tokens", "workspace"):
        assert ws_(lib, **{name: NULL}) == INVALID, name
    assert ws_(lib, V=0, stride=0) == INVALID
    assert ws_(lib, gamma=2.0) == GAMMA
    assert ws_(lib, delta=math.inf) == DELTA
    assert ws_(lib, seeding=7) == UNSUPPORTED
    assert ws_(lib, B=0, seeds=NULL) == OK
    if not _gpu_visible():
        assert ws_(lib, scores=NULL) == NO_DEVICE


def test_shard_entry_points_reject_bad_offsets(lib):
    """v_offset >= 0 and v_offset + V <= 2^32 (token ids are 32-bit); every other check
    is the unsharded call's."""
    def wsh(v_offset, V=8, **kw):
        a = dict(logits=DUMMY, B=2, stride=max(V, 8))
        a.update(kw)
        return lib.sbw_watermark_shard(a["logits"], 0, a["B"], V, a["stride"], DUMMY, 1, v_offset,
                                       KEY, 0.25, 2.0, 0, None)

    def ash(v_offset, V=8, **kw):
        return lib.sbw_watermark_argmax_shard(DUMMY, 1, 2, V, max(V, 8), DUMMY, 1, v_offset, KEY,
                                              0.25, 2.0, 1, DUMMY, DUMMY, DUMMY, None)

    def ssh(v_offset, V=8, inv_t=1.0):
        return lib.sbw_watermark_sample_shard(DUMMY, 0, 2, V, max(V, 8), DUMMY, 1, v_offset, KEY,
                                              0.25, 2.0, 0, DUMMY, inv_t, DUMMY, DUMMY, DUMMY,
                                              None)

    for fn in (wsh, ash, ssh):
        assert fn(-1) == INVALID
        assert fn(-(1 << 40)) == INVALID
        assert fn((1 << 32) - 7) == UNSUPPORTED          # last id would be 2^32
        assert fn((1 << 32) + 1, V=0) == UNSUPPORTED
    assert ssh(0, inv_t=0.0) == INVALID
    assert wsh(5, B=0) == OK
    assert wsh(1 << 32, V=0) == OK                         # an empty shard: nothing to do
    assert ash(0, V=0) == INVALID                          # no token to choose
    assert ssh(1 << 32, V=0) == INVALID
    if not _gpu_visible():
        for fn in (wsh, ash, ssh):
            assert fn((1 << 32) - 8) == NO_DEVICE          # last id 2^32 - 1 is allowed
            assert fn(12345) == NO_DEVICE


def test_binding_shard_calls_validate_before_the_c_abi(sbw):
    import torch
    x = torch.zeros(2, 8)
    prev = torch.zeros(2, dtype=torch.int32)
    with pytest.raises(ValueError, match="current HIP device"):
        sbw.watermark_shard(x, prev, 16, KEY, 0.25, 2.0)
    with pytest.raises(ValueError, match="current HIP device"):
        sbw.watermark_argmax_shard(x, prev, 16, KEY, 0.25, 2.0,
                                   tokens=torch.zeros(2, dtype=torch.int32), values=torch.zeros(2),
                                   workspace=torch.zeros(4, dtype=torch.int64))
