"""Stateless Bernoulli Watermarking on MI355X (gfx950): Python binding of libsbw.

A thin ctypes layer over the C ABI in ``include/sbw.h``; it only marshals
arguments (device pointers, sizes, the current HIP stream).  Every step of the
watermark and detect path runs in the HIP kernels of ``libsbw.so``.  There is no
fallback: if the library is missing this module raises on import.

    watermark(logits, prev_tokens, key, gamma, delta, seeding="context")   in place
    watermark_argmax(logits, prev_tokens, key, gamma, delta) -> (tokens [B], values [B])
    watermark_argmax_noalloc(...)  the same with the library's static scratch array
    watermark_sample(logits, prev_tokens, key, gamma, delta, seeds) -> (tokens [B], scores [B])
    green_mask(prev_tokens, V, key, gamma, seeding="context") -> int32 [B, ceil(V/32)]
    detect(tokens, key, gamma, seeding="context") -> (counts int32 [N], z float64 [N])

Tensors are torch tensors on the current HIP device; torch provides the memory
and the stream, nothing else.

The three logits calls take ``v_offset``: the logits are then one vocabulary shard,
column c being token v_offset + c (``sbw_*_shard`` in the C ABI); ``watermark_shard``,
``watermark_argmax_shard`` and ``watermark_sample_shard`` are the same calls.
"""
from __future__ import annotations

import ctypes
import functools
import os

import torch  # loads torch's HIP runtime first, so libsbw binds to the same one

from ._build import LIBRARY, build  # noqa: F401  (build is re-exported)

__all__ = ["watermark", "watermark_argmax", "watermark_argmax_noalloc", "watermark_sample",
           "watermark_shard",
           "watermark_argmax_shard", "watermark_sample_shard", "watermark_candidates",
           "green_mask", "detect", "detect_ex", "SbwError", "version", "library_path",
           "SEED_CONTEXT", "SEED_SELF_SALT"]

SEED_CONTEXT = 0
SEED_SELF_SALT = 1
F32 = 0
BF16 = 1

_STATUS = {
    0: "SBW_OK",
    1: "SBW_ERR_INVALID_ARG",
    2: "SBW_ERR_GAMMA",
    3: "SBW_ERR_DELTA",
    4: "SBW_ERR_UNSUPPORTED",
    5: "SBW_ERR_NO_DEVICE",
    6: "SBW_ERR_HIP",
}

EXPORTED = ("sbw_watermark", "sbw_green_mask", "sbw_detect", "sbw_watermark_window",
            "sbw_green_mask_window", "sbw_detect_window", "sbw_watermark_argmax",
            "sbw_watermark_argmax_workspace", "sbw_watermark_candidates", "sbw_detect_ex",
            "sbw_watermark_sample", "sbw_watermark_shard", "sbw_watermark_argmax_shard",
            "sbw_watermark_sample_shard", "sbw_watermark_argmax_noalloc",
            "sbw_strerror", "sbw_last_hip_error", "sbw_version")
NOALLOC_SCRATCH_ELEMS = 262144   # SBW_NOALLOC_SCRATCH_ELEMS
DETECT_IGNORE_REPEATED = 1
MAX_UNIQUE_POSITIONS = 4096
MAX_CANDIDATES = 1024
MAX_WIDTH = 8


class SbwError(RuntimeError):
    def __init__(self, status: int, message: str, hip_error: str | None = None):
        self.status = status
        self.code = _STATUS.get(status, str(status))
        self.hip_error = hip_error
        text = f"{self.code}: {message}"
        if hip_error and hip_error != "hipSuccess":
            text += f" ({hip_error})"
        super().__init__(text)


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIBRARY):
        raise ImportError(f"libsbw.so not built at {LIBRARY}; run __graft_entry__.build() "
                          "or python -m paper_2609_03844_amd._build")
    lib = ctypes.CDLL(LIBRARY)
    P, i64, u64, f64, f32, i32 = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                  ctypes.c_double, ctypes.c_float, ctypes.c_int)
    lib.sbw_watermark.restype = i32
    lib.sbw_watermark.argtypes = [P, i32, i64, i64, i64, P, u64, f64, f32, i32, P]
    lib.sbw_green_mask.restype = i32
    lib.sbw_green_mask.argtypes = [P, i64, i64, P, u64, f64, i32, P]
    lib.sbw_detect.restype = i32
    lib.sbw_detect.argtypes = [P, i64, i64, i64, u64, f64, i32, P, P, P]
    lib.sbw_watermark_window.restype = i32
    lib.sbw_watermark_window.argtypes = [P, i32, i64, i64, i64, P, i64, u64, f64, f32, i32, P]
    lib.sbw_green_mask_window.restype = i32
    lib.sbw_green_mask_window.argtypes = [P, i64, i64, P, i64, u64, f64, i32, P]
    lib.sbw_detect_window.restype = i32
    lib.sbw_detect_window.argtypes = [P, i64, i64, i64, i64, u64, f64, i32, P, P, P]
    lib.sbw_watermark_argmax.restype = i32
    lib.sbw_watermark_argmax.argtypes = [P, i32, i64, i64, i64, P, i64, u64, f64, f32, i32, P, P,
                                         P, P]
    lib.sbw_watermark_sample.restype = i32
    lib.sbw_watermark_sample.argtypes = [P, i32, i64, i64, i64, P, i64, u64, f64, f32, i32, P, f32,
                                         P, P, P, P]
    lib.sbw_watermark_shard.restype = i32
    lib.sbw_watermark_shard.argtypes = [P, i32, i64, i64, i64, P, i64, i64, u64, f64, f32, i32, P]
    lib.sbw_watermark_argmax_shard.restype = i32
    lib.sbw_watermark_argmax_shard.argtypes = [P, i32, i64, i64, i64, P, i64, i64, u64, f64, f32,
                                               i32, P, P, P, P]
    lib.sbw_watermark_sample_shard.restype = i32
    lib.sbw_watermark_sample_shard.argtypes = [P, i32, i64, i64, i64, P, i64, i64, u64, f64, f32,
                                               i32, P, f32, P, P, P, P]
    lib.sbw_detect_ex.restype = i32
    lib.sbw_detect_ex.argtypes = [P, i64, i64, i64, P, i64, u64, f64, i32, ctypes.c_uint32, P, P,
                                  P, P]
    lib.sbw_watermark_candidates.restype = i32
    lib.sbw_watermark_candidates.argtypes = [P, i32, i64, i64, i64, P, i64, P, i64, u64, f64, f32,
                                             i32, P]
    lib.sbw_watermark_argmax_noalloc.restype = i32
    lib.sbw_watermark_argmax_noalloc.argtypes = [P, i32, i64, i64, i64, P, i64, u64, f64, f32, i32,
                                                 P, P, P]
    lib.sbw_watermark_argmax_workspace.restype = i64
    lib.sbw_watermark_argmax_workspace.argtypes = [i64, i64]
    lib.sbw_strerror.restype = ctypes.c_char_p
    lib.sbw_strerror.argtypes = [i32]
    lib.sbw_last_hip_error.restype = ctypes.c_char_p
    lib.sbw_last_hip_error.argtypes = []
    lib.sbw_version.restype = ctypes.c_char_p
    lib.sbw_version.argtypes = []
    return lib


_lib = _load()


def library_path() -> str:
    return LIBRARY


def version() -> str:
    return _lib.sbw_version().decode()


def raw() -> ctypes.CDLL:
    """The ctypes handle of libsbw (the C ABI itself)."""
    return _lib


def _check(status: int) -> None:
    if status != 0:
        hip = _lib.sbw_last_hip_error().decode() if status == 6 else None
        raise SbwError(status, _lib.sbw_strerror(status).decode(), hip)


def _seeding(s) -> int:
    if isinstance(s, str):
        return {"context": SEED_CONTEXT, "self_salt": SEED_SELF_SALT}[s]
    return int(s)


# The current device and its current stream straight from torch's C layer: building a
# torch.cuda.Stream object per call costs about 3 us, more than a small launch.
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_get_device = getattr(torch._C, "_cuda_getDevice", None)


def _current_device() -> int:
    return _get_device() if _get_device is not None else torch.cuda.current_device()


def _stream(stream) -> int:
    if stream is None:
        if _raw_stream is not None:
            return _raw_stream(_current_device())
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _key(key: int) -> int:
    return int(key) & 0xFFFFFFFFFFFFFFFF


def _on_device(**tensors) -> None:
    """Every tensor argument must live on the current HIP device: the kernels
    dereference the pointers, and a host or peer pointer would fault the GPU."""
    dev = None
    for name, t in tensors.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the current HIP device, got {t.device}")
        if dev is None:
            dev = _current_device()
        if t.get_device() != dev:
            raise ValueError(f"{name} must be on the current HIP device (cuda:{dev}), "
                             f"got {t.device}")


def _window(context: torch.Tensor, B: int):
    """[B] (the previous token) or [B, h] (the h tokens before the step) -> (tensor, h)."""
    if context.dtype != torch.int32:
        raise ValueError("the context tokens must be int32")
    if context.dim() == 1:
        if context.shape[0] != B:
            raise ValueError("prev_tokens must be int32 [B]")
        width = 1
    elif context.dim() == 2 and context.shape[0] == B:
        width = context.shape[1]
    else:
        raise ValueError("context must be int32 [B] or [B, width]")
    if B > 0 and not context.is_contiguous():
        raise ValueError("the context tokens must be contiguous")
    return context, width


def watermark(logits: torch.Tensor, prev_tokens: torch.Tensor, key: int, gamma: float,
              delta: float, seeding="context", stream=None, v_offset: int = 0) -> torch.Tensor:
    """Adds delta to the green logits of every row, in place; returns ``logits``.

    logits: [B, V] float32 or bfloat16 on the GPU, unit stride along V (rows may be
    padded: stride(0) >= V).  prev_tokens: int32 [B] (the previous token of each row)
    or int32 [B, h] (the h tokens before the step, context width h <= 8).  v_offset:
    the token id of column 0 when the logits are one shard of the vocabulary.
    """
    if logits.dim() != 2:
        raise ValueError("logits must be [B, V]")
    if logits.dtype == torch.float32:
        dtype = F32
    elif logits.dtype == torch.bfloat16:
        dtype = BF16
    else:
        raise TypeError("logits must be float32 or bfloat16")
    B, V = logits.shape
    if B > 0 and V > 0 and logits.stride(1) != 1:
        raise ValueError("logits must have unit stride along the vocabulary")
    context, width = _window(prev_tokens, B)
    row_stride = logits.stride(0) if B > 1 else max(V, logits.stride(0))
    seed_kind = _seeding(seeding)
    _on_device(logits=logits, prev_tokens=context)
    if v_offset == 0:
        _check(_lib.sbw_watermark_window(logits.data_ptr(), dtype, B, V, row_stride,
                                         context.data_ptr(), width, _key(key), float(gamma),
                                         float(delta), seed_kind, _stream(stream)))
    else:
        _check(_lib.sbw_watermark_shard(logits.data_ptr(), dtype, B, V, row_stride,
                                        context.data_ptr(), width, int(v_offset), _key(key),
                                        float(gamma), float(delta), seed_kind, _stream(stream)))
    return logits


def watermark_candidates(logits: torch.Tensor, prev_tokens: torch.Tensor,
                         candidates: torch.Tensor, key: int, gamma: float, delta: float,
                         seeding="self_salt", stream=None) -> torch.Tensor:
    """The watermark restricted to candidates [B, k] int32 (k <= 1024), in place; the
    top-k self-salt scheme (SBW-ss) with its top-k ids as candidates.  Ids outside
    [0, V) are ignored, a repeated id is biased once; returns ``logits``."""
    if logits.dim() != 2:
        raise ValueError("logits must be [B, V]")
    if logits.dtype == torch.float32:
        dtype = F32
    elif logits.dtype == torch.bfloat16:
        dtype = BF16
    else:
        raise TypeError("logits must be float32 or bfloat16")
    B, V = logits.shape
    if B > 0 and V > 0 and logits.stride(1) != 1:
        raise ValueError("logits must have unit stride along the vocabulary")
    if (candidates.dim() != 2 or candidates.shape[0] != B or candidates.dtype != torch.int32
            or not candidates.is_contiguous()):
        raise ValueError("candidates must be contiguous int32 [B, k]")
    context, width = _window(prev_tokens, B)
    row_stride = logits.stride(0) if B > 1 else max(V, logits.stride(0))
    _on_device(logits=logits, prev_tokens=context, candidates=candidates)
    _check(_lib.sbw_watermark_candidates(logits.data_ptr(), dtype, B, V, row_stride,
                                         candidates.data_ptr(), candidates.shape[1],
                                         context.data_ptr(), width, _key(key), float(gamma),
                                         float(delta), _seeding(seeding), _stream(stream)))
    return logits


def watermark_argmax(logits: torch.Tensor, prev_tokens: torch.Tensor, key: int, gamma: float,
                     delta: float, seeding="context", tokens: torch.Tensor | None = None,
                     values: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                     with_values: bool = True, stream=None, v_offset: int = 0):
    """Greedy decoding of the watermarked logits in one read-only pass.

    Returns (tokens int32 [B], values float32 [B] or None).  ``workspace`` is an int64
    scratch tensor of at least argmax_workspace_size(B, V) elements (allocated here
    when not given).  With v_offset the logits are a vocabulary shard and the tokens
    global ids."""
    if logits.dim() != 2:
        raise ValueError("logits must be [B, V]")
    if logits.dtype == torch.float32:
        dtype = F32
    elif logits.dtype == torch.bfloat16:
        dtype = BF16
    else:
        raise TypeError("logits must be float32 or bfloat16")
    B, V = logits.shape
    if B > 0 and V > 0 and logits.stride(1) != 1:
        raise ValueError("logits must have unit stride along the vocabulary")
    context, width = _window(prev_tokens, B)
    dev = logits.device
    if tokens is None:
        tokens = torch.empty(B, dtype=torch.int32, device=dev)
    if values is None and with_values:
        values = torch.empty(B, dtype=torch.float32, device=dev)
    need = argmax_workspace_size(B, V)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.int64, device=dev)
    if tokens.shape != (B,) or tokens.dtype != torch.int32 or not tokens.is_contiguous():
        raise ValueError("tokens must be contiguous int32 [B]")
    if (workspace.dtype != torch.int64 or not workspace.is_contiguous()
            or workspace.numel() < need):
        raise ValueError(f"workspace must be contiguous int64 with >= {need} elements")
    if values is not None and (values.shape != (B,) or values.dtype != torch.float32
                               or not values.is_contiguous()):
        raise ValueError("values must be contiguous float32 [B]")
    row_stride = logits.stride(0) if B > 1 else max(V, logits.stride(0))
    _on_device(logits=logits, prev_tokens=context, tokens=tokens, values=values,
               workspace=workspace)
    vptr = values.data_ptr() if values is not None else None
    if v_offset == 0:
        _check(_lib.sbw_watermark_argmax(logits.data_ptr(), dtype, B, V, row_stride,
                                         context.data_ptr(), width, _key(key), float(gamma),
                                         float(delta), _seeding(seeding), tokens.data_ptr(), vptr,
                                         workspace.data_ptr(), _stream(stream)))
    else:
        _check(_lib.sbw_watermark_argmax_shard(logits.data_ptr(), dtype, B, V, row_stride,
                                               context.data_ptr(), width, int(v_offset),
                                               _key(key), float(gamma), float(delta),
                                               _seeding(seeding), tokens.data_ptr(), vptr,
                                               workspace.data_ptr(), _stream(stream)))
    return tokens, values


def watermark_argmax_noalloc(logits: torch.Tensor, prev_tokens: torch.Tensor, key: int,
                             gamma: float, delta: float, seeding="context",
                             tokens: torch.Tensor | None = None,
                             values: torch.Tensor | None = None, with_values: bool = True,
                             stream=None):
    """watermark_argmax() without a workspace: the library keeps the partials in a static
    device array (``sbw_watermark_argmax_noalloc``), so with ``tokens`` (and ``values``)
    given nothing is allocated.  Calls on one device share that array: keep them ordered.
    Returns (tokens int32 [B], values float32 [B] or None)."""
    if logits.dim() != 2:
        raise ValueError("logits must be [B, V]")
    if logits.dtype == torch.float32:
        dtype = F32
    elif logits.dtype == torch.bfloat16:
        dtype = BF16
    else:
        raise TypeError("logits must be float32 or bfloat16")
    B, V = logits.shape
    if B > 0 and V > 0 and logits.stride(1) != 1:
        raise ValueError("logits must have unit stride along the vocabulary")
    context, width = _window(prev_tokens, B)
    dev = logits.device
    if tokens is None:
        tokens = torch.empty(B, dtype=torch.int32, device=dev)
    if values is None and with_values:
        values = torch.empty(B, dtype=torch.float32, device=dev)
    if tokens.shape != (B,) or tokens.dtype != torch.int32 or not tokens.is_contiguous():
        raise ValueError("tokens must be contiguous int32 [B]")
    if values is not None and (values.shape != (B,) or values.dtype != torch.float32
                               or not values.is_contiguous()):
        raise ValueError("values must be contiguous float32 [B]")
    row_stride = logits.stride(0) if B > 1 else max(V, logits.stride(0))
    _on_device(logits=logits, prev_tokens=context, tokens=tokens, values=values)
    _check(_lib.sbw_watermark_argmax_noalloc(logits.data_ptr(), dtype, B, V, row_stride,
                                             context.data_ptr(), width, _key(key), float(gamma),
                                             float(delta), _seeding(seeding), tokens.data_ptr(),
                                             values.data_ptr() if values is not None else None,
                                             _stream(stream)))
    return tokens, values


def watermark_sample(logits: torch.Tensor, prev_tokens: torch.Tensor, key: int, gamma: float,
                     delta: float, seeds: torch.Tensor, seeding="context",
                     inv_temperature: float = 1.0, tokens: torch.Tensor | None = None,
                     scores: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                     with_scores: bool = True, stream=None, v_offset: int = 0):
    """One draw per row from softmax(watermarked logits * inv_temperature), fused
    (Gumbel-max with noise from seeds, uint64 [B] as an int64 tensor).  Returns (tokens
    int32 [B], scores float32 [B] or None); the workspace and v_offset are as for
    watermark_argmax."""
    if logits.dim() != 2:
        raise ValueError("logits must be [B, V]")
    if logits.dtype == torch.float32:
        dtype = F32
    elif logits.dtype == torch.bfloat16:
        dtype = BF16
    else:
        raise TypeError("logits must be float32 or bfloat16")
    B, V = logits.shape
    if B > 0 and V > 0 and logits.stride(1) != 1:
        raise ValueError("logits must have unit stride along the vocabulary")
    if seeds.shape != (B,) or seeds.dtype not in (torch.int64, torch.uint64) or not seeds.is_contiguous():
        raise ValueError("seeds must be contiguous 64-bit integers [B]")
    context, width = _window(prev_tokens, B)
    dev = logits.device
    if tokens is None:
        tokens = torch.empty(B, dtype=torch.int32, device=dev)
    if scores is None and with_scores:
        scores = torch.empty(B, dtype=torch.float32, device=dev)
    need = argmax_workspace_size(B, V)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.int64, device=dev)
    if tokens.shape != (B,) or tokens.dtype != torch.int32 or not tokens.is_contiguous():
        raise ValueError("tokens must be contiguous int32 [B]")
    if (workspace.dtype != torch.int64 or not workspace.is_contiguous()
            or workspace.numel() < need):
        raise ValueError(f"workspace must be contiguous int64 with >= {need} elements")
    if scores is not None and (scores.shape != (B,) or scores.dtype != torch.float32
                               or not scores.is_contiguous()):
        raise ValueError("scores must be contiguous float32 [B]")
    row_stride = logits.stride(0) if B > 1 else max(V, logits.stride(0))
    seed_kind = _seeding(seeding)
    _on_device(logits=logits, prev_tokens=context, seeds=seeds, tokens=tokens, scores=scores,
               workspace=workspace)
    sptr = scores.data_ptr() if scores is not None else None
    if v_offset == 0:
        _check(_lib.sbw_watermark_sample(logits.data_ptr(), dtype, B, V, row_stride,
                                         context.data_ptr(), width, _key(key), float(gamma),
                                         float(delta), seed_kind, seeds.data_ptr(),
                                         float(inv_temperature), tokens.data_ptr(), sptr,
                                         workspace.data_ptr(), _stream(stream)))
    else:
        _check(_lib.sbw_watermark_sample_shard(logits.data_ptr(), dtype, B, V, row_stride,
                                               context.data_ptr(), width, int(v_offset),
                                               _key(key), float(gamma), float(delta), seed_kind,
                                               seeds.data_ptr(), float(inv_temperature),
                                               tokens.data_ptr(), sptr, workspace.data_ptr(),
                                               _stream(stream)))
    return tokens, scores


def watermark_shard(logits: torch.Tensor, prev_tokens: torch.Tensor, v_offset: int, key: int,
                    gamma: float, delta: float, seeding="context", stream=None) -> torch.Tensor:
    """watermark() of one vocabulary shard: column c of logits is token v_offset + c."""
    return watermark(logits, prev_tokens, key, gamma, delta, seeding, stream, v_offset=v_offset)


def watermark_argmax_shard(logits: torch.Tensor, prev_tokens: torch.Tensor, v_offset: int,
                           key: int, gamma: float, delta: float, seeding="context", **kw):
    """watermark_argmax() of one vocabulary shard; the tokens are global ids."""
    return watermark_argmax(logits, prev_tokens, key, gamma, delta, seeding, v_offset=v_offset,
                            **kw)


def watermark_sample_shard(logits: torch.Tensor, prev_tokens: torch.Tensor, v_offset: int,
                           key: int, gamma: float, delta: float, seeds: torch.Tensor,
                           seeding="context", inv_temperature: float = 1.0, **kw):
    """watermark_sample() of one vocabulary shard; the tokens are global ids."""
    return watermark_sample(logits, prev_tokens, key, gamma, delta, seeds, seeding,
                            inv_temperature, v_offset=v_offset, **kw)


@functools.lru_cache(maxsize=1024)
def argmax_workspace_size(B: int, V: int) -> int:
    """uint64 elements of scratch that watermark_argmax needs for B rows of V logits."""
    return int(_lib.sbw_watermark_argmax_workspace(int(B), int(V)))


def green_mask(prev_tokens: torch.Tensor, V: int, key: int, gamma: float, seeding="context",
               out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Green lists as bit sets: int32 [B, ceil(V/32)], bit v%32 of word v//32.
    prev_tokens: int32 [B] or [B, h] as for watermark()."""
    if prev_tokens.dim() not in (1, 2):
        raise ValueError("prev_tokens must be int32 [B] or [B, width]")
    B = prev_tokens.shape[0]
    context, width = _window(prev_tokens, B)
    words = (int(V) + 31) // 32
    if out is None:
        out = torch.empty((B, words), dtype=torch.int32, device=prev_tokens.device)
    elif out.shape != (B, words) or out.dtype != torch.int32 or not out.is_contiguous():
        raise ValueError("out must be contiguous int32 [B, ceil(V/32)]")
    _on_device(prev_tokens=context, out=out)
    _check(_lib.sbw_green_mask_window(out.data_ptr(), B, int(V), context.data_ptr(), width,
                                      _key(key), float(gamma), _seeding(seeding),
                                      _stream(stream)))
    return out


def detect(tokens: torch.Tensor, key: int, gamma: float, seeding="context",
           counts: torch.Tensor | None = None, z: torch.Tensor | None = None, stream=None,
           width: int = 1):
    """Green count and z-score per sequence of tokens [N, L] int32 (unit stride along L).
    Positions width..L-1 are scored under the `width` tokens before each (T = L - width)."""
    if tokens.dtype != torch.int32 or tokens.dim() != 2:
        raise ValueError("tokens must be int32 [N, L]")
    N, L = tokens.shape
    if N > 0 and L > 0 and tokens.stride(1) != 1:
        raise ValueError("tokens must have unit stride along L")
    dev = tokens.device
    if counts is None:
        counts = torch.empty(N, dtype=torch.int32, device=dev)
    if z is None:
        z = torch.empty(N, dtype=torch.float64, device=dev)
    if counts.shape != (N,) or counts.dtype != torch.int32 or not counts.is_contiguous():
        raise ValueError("counts must be contiguous int32 [N]")
    if z.shape != (N,) or z.dtype != torch.float64 or not z.is_contiguous():
        raise ValueError("z must be contiguous float64 [N]")
    row_stride = tokens.stride(0) if N > 1 else max(L, tokens.stride(0))
    _on_device(tokens=tokens, counts=counts, z=z)
    _check(_lib.sbw_detect_window(tokens.data_ptr() if L > 0 else None, N, L, row_stride,
                                  int(width), _key(key), float(gamma), _seeding(seeding),
                                  counts.data_ptr(), z.data_ptr(), _stream(stream)))
    return counts, z


def detect_ex(tokens: torch.Tensor, key: int, gamma: float, seeding="context", width: int = 1,
              lengths: torch.Tensor | None = None, ignore_repeated: bool = False,
              counts: torch.Tensor | None = None, scored: torch.Tensor | None = None,
              z: torch.Tensor | None = None, stream=None):
    """Detection of texts of different lengths: tokens int32 [N, L] (L the longest),
    lengths int32 [N] or None (clamped to [0, L]); with ignore_repeated, each distinct
    (width+1)-gram of a text is scored once (L - width <= 4096).  Returns (green
    counts int32 [N], scored positions int32 [N], z float64 [N])."""
    if tokens.dtype != torch.int32 or tokens.dim() != 2:
        raise ValueError("tokens must be int32 [N, L]")
    N, L = tokens.shape
    if N > 0 and L > 0 and tokens.stride(1) != 1:
        raise ValueError("tokens must have unit stride along L")
    dev = tokens.device
    if lengths is not None and (lengths.shape != (N,) or lengths.dtype != torch.int32
                                or not lengths.is_contiguous()):
        raise ValueError("lengths must be contiguous int32 [N]")
    counts = torch.empty(N, dtype=torch.int32, device=dev) if counts is None else counts
    scored = torch.empty(N, dtype=torch.int32, device=dev) if scored is None else scored
    z = torch.empty(N, dtype=torch.float64, device=dev) if z is None else z
    for name, t, dt in (("counts", counts, torch.int32), ("scored", scored, torch.int32),
                        ("z", z, torch.float64)):
        if t.shape != (N,) or t.dtype != dt or not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous {dt} [N]")
    row_stride = tokens.stride(0) if N > 1 else max(L, tokens.stride(0))
    _on_device(tokens=tokens, lengths=lengths, counts=counts, scored=scored, z=z)
    _check(_lib.sbw_detect_ex(tokens.data_ptr(), N, L, row_stride,
                              lengths.data_ptr() if lengths is not None else None, int(width),
                              _key(key), float(gamma), _seeding(seeding),
                              DETECT_IGNORE_REPEATED if ignore_repeated else 0, counts.data_ptr(),
                              scored.data_ptr(), z.data_ptr(), _stream(stream)))
    return counts, scored, z
