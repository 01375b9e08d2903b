"""CPU oracle for Stateless Bernoulli Watermarking -- TEST INFRASTRUCTURE ONLY.

Python access (ctypes + numpy) to the plain C definitions in ``sbw_oracle.c``.
Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
in ``paper_2609_03844_amd`` and neither imports the other.

The C source states which passage of the paper each function follows and the
readings taken where the paper is silent.  ``jenkins32`` is "parity unpinned":
it is checked only through its properties.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "sbw_oracle.c")
LIBRARY = os.path.join(HERE, "liboracle.so")

SEED_CONTEXT = 0
SEED_SELF_SALT = 1
_SEEDING = {"context": SEED_CONTEXT, "self_salt": SEED_SELF_SALT}

# The paper's hash key (App. C, reproducibility).
PAPER_KEY = 15485863


def build() -> str:
    """Compile the oracle with plain gcc: no FMA contraction, no fast-math."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
           "-ffp-contract=off", "-fno-fast-math", "-o", LIBRARY + ".tmp", SOURCE, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(LIBRARY + ".tmp", LIBRARY)
    return LIBRARY


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY) or os.path.getmtime(LIBRARY) < os.path.getmtime(SOURCE):
            build()
        _lib = _declare(ctypes.CDLL(LIBRARY))
    return _lib


def _declare(l: ctypes.CDLL) -> ctypes.CDLL:
    P = ctypes.c_void_p
    i64, u64, u32, i32 = ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int
    f64, f32 = ctypes.c_double, ctypes.c_float
    sig = {
        "oracle_philox4x32_10": (None, [P, P, P]),
        "oracle_cbrng": (u32, [u32, u64]),
        "oracle_threshold": (u64, [f64]),
        "oracle_jenkins32": (u32, [u32]),
        "oracle_seed_context": (u64, [u64, u32]),
        "oracle_seed_self_salt": (u64, [u64, u32, u32]),
        "oracle_is_green_many": (None, [u64, P, P, i64, f64, i32, P]),
        "oracle_watermark_f32": (None, [P, i64, i64, i64, P, u64, f64, f32, i32]),
        "oracle_watermark_bf16": (None, [P, i64, i64, i64, P, u64, f64, f32, i32]),
        "oracle_green_mask": (None, [P, i64, i64, P, u64, f64, i32]),
        "oracle_z_score": (f64, [i64, i64, f64]),
        "oracle_detect": (None, [P, i64, i64, i64, u64, f64, i32, P, P]),
        "oracle_cbrng_many": (None, [P, P, i64, P]),
        "oracle_jenkins32_many": (None, [P, i64, P]),
        "oracle_seed_many": (None, [u64, P, P, i64, i32, P]),
        "oracle_bias_f32_many": (None, [P, i64, f32, P]),
        "oracle_bias_bf16_many": (None, [P, i64, f32, P]),
        "oracle_f32_to_bf16_many": (None, [P, i64, P]),
        "oracle_seed_context_w": (u64, [u64, P, i64]),
        "oracle_seed_self_salt_w": (u64, [u64, P, i64, u32]),
        "oracle_watermark_f32_w": (None, [P, i64, i64, i64, P, i64, u64, f64, f32, i32]),
        "oracle_watermark_bf16_w": (None, [P, i64, i64, i64, P, i64, u64, f64, f32, i32]),
        "oracle_green_mask_w": (None, [P, i64, i64, P, i64, u64, f64, i32]),
        "oracle_detect_w": (None, [P, i64, i64, i64, i64, u64, f64, i32, P, P]),
        "oracle_seed_w_many": (None, [u64, P, i64, P, i64, i32, P]),
        "oracle_is_green_w_many": (None, [u64, P, i64, P, i64, f64, i32, P]),
        "oracle_watermark_argmax_f32_w": (None, [P, i64, i64, i64, P, i64, u64, f64, f32, i32, P, P]),
        "oracle_watermark_argmax_bf16_w": (None, [P, i64, i64, i64, P, i64, u64, f64, f32, i32, P, P]),
        "oracle_watermark_candidates_f32_w": (None, [P, i64, i64, i64, P, i64, P, i64, u64, f64, f32, i32]),
        "oracle_detect_ex": (None, [P, i64, i64, i64, P, i64, u64, f64, i32, i32, P, P, P]),
        "oracle_sample_log": (f32, [f32]),
        "oracle_gumbel": (f32, [u32, u64]),
        "oracle_sample_log_many": (None, [P, i64, P]),
        "oracle_gumbel_many": (None, [P, P, i64, P]),
        "oracle_gumbel_of_draws": (None, [P, i64, P]),
        "oracle_watermark_sample_f32_w": (None, [P, i64, i64, i64, P, i64, u64, f64, f32, i32, P, f32, P, P]),
        "oracle_watermark_sample_bf16_w": (None, [P, i64, i64, i64, P, i64, u64, f64, f32, i32, P, f32, P, P]),
        "oracle_watermark_candidates_bf16_w": (None, [P, i64, i64, i64, P, i64, P, i64, u64, f64, f32, i32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(l, name)
        fn.restype = res
        fn.argtypes = args
    return l


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _seeding(s) -> int:
    return _SEEDING[s] if isinstance(s, str) else int(s)


# --- scalar definitions ------------------------------------------------------

def philox4x32_10(counter, key) -> np.ndarray:
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def cbrng(v: int, r: int) -> int:
    return int(lib().oracle_cbrng(v & 0xFFFFFFFF, r & 0xFFFFFFFFFFFFFFFF))


def threshold(gamma: float) -> int:
    return int(lib().oracle_threshold(float(gamma)))


def jenkins32(a: int) -> int:
    return int(lib().oracle_jenkins32(a & 0xFFFFFFFF))


def seed_context(key: int, prev: int) -> int:
    return int(lib().oracle_seed_context(key, prev & 0xFFFFFFFF))


def seed_self_salt(key: int, prev: int, cand: int) -> int:
    return int(lib().oracle_seed_self_salt(key, prev & 0xFFFFFFFF, cand & 0xFFFFFFFF))


def z_score(green_count: int, T: int, gamma: float) -> float:
    return float(lib().oracle_z_score(int(green_count), int(T), float(gamma)))


# --- array forms --------------------------------------------------------------

def cbrng_many(v, r) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.uint32)
    r = np.ascontiguousarray(np.broadcast_to(np.asarray(r, dtype=np.uint64), v.shape))
    out = np.empty(v.shape, dtype=np.uint32)
    lib().oracle_cbrng_many(_ptr(v), _ptr(r), v.size, _ptr(out))
    return out


def jenkins32_many(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.uint32)
    out = np.empty(a.shape, dtype=np.uint32)
    lib().oracle_jenkins32_many(_ptr(a), a.size, _ptr(out))
    return out


def seed_many(key: int, prev, cand, seeding) -> np.ndarray:
    prev = np.ascontiguousarray(prev, dtype=np.int32)
    cand = np.ascontiguousarray(np.broadcast_to(np.asarray(cand, dtype=np.int32), prev.shape))
    out = np.empty(prev.shape, dtype=np.uint64)
    lib().oracle_seed_many(key, _ptr(prev), _ptr(cand), prev.size, _seeding(seeding), _ptr(out))
    return out


def is_green_many(key: int, prev, cand, gamma: float, seeding) -> np.ndarray:
    prev = np.ascontiguousarray(prev, dtype=np.int32)
    cand = np.ascontiguousarray(cand, dtype=np.int32)
    assert prev.shape == cand.shape
    out = np.empty(prev.shape, dtype=np.uint8)
    lib().oracle_is_green_many(key, _ptr(prev), _ptr(cand), prev.size, float(gamma),
                               _seeding(seeding), _ptr(out))
    return out.astype(bool)


def bias_f32_many(x, delta: float) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    lib().oracle_bias_f32_many(_ptr(x), x.size, float(delta), _ptr(out))
    return out


def bias_bf16_many(x_bits, delta: float) -> np.ndarray:
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    out = np.empty_like(x)
    lib().oracle_bias_bf16_many(_ptr(x), x.size, float(delta), _ptr(out))
    return out


def f32_to_bf16_many(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().oracle_f32_to_bf16_many(_ptr(x), x.size, _ptr(out))
    return out


# --- the hot-path definitions ---------------------------------------------------

def watermark(logits: np.ndarray, prev, key: int, gamma: float, delta: float,
              seeding="context") -> np.ndarray:
    """Returns a biased copy of ``logits`` ([B, V]; float32, or uint16 holding bf16
    bit patterns).  Row stride is taken from the array's first stride."""
    out = np.array(logits, copy=True, order="C")
    if out.ndim != 2:
        raise ValueError("logits must be [B, V]")
    B, V = out.shape
    prev = np.ascontiguousarray(prev, dtype=np.int32)
    if prev.shape != (B,):
        raise ValueError("prev must be [B]")
    if out.dtype == np.float32:
        fn = lib().oracle_watermark_f32
    elif out.dtype == np.uint16:
        fn = lib().oracle_watermark_bf16
    else:
        raise TypeError("logits must be float32 or uint16 (bf16 bits)")
    fn(_ptr(out), B, V, V, _ptr(prev), key, float(gamma), float(delta), _seeding(seeding))
    return out


def green_mask(B: int, V: int, prev, key: int, gamma: float, seeding="context") -> np.ndarray:
    prev = np.ascontiguousarray(prev, dtype=np.int32)
    if prev.shape != (B,):
        raise ValueError("prev must be [B]")
    out = np.empty((B, (V + 31) // 32), dtype=np.uint32)
    lib().oracle_green_mask(_ptr(out), B, V, _ptr(prev), key, float(gamma), _seeding(seeding))
    return out


def detect(tokens: np.ndarray, key: int, gamma: float, seeding="context"):
    """tokens [N, L] int32 -> (green_counts int32 [N], z float64 [N])."""
    tok = np.ascontiguousarray(tokens, dtype=np.int32)
    if tok.ndim != 2:
        raise ValueError("tokens must be [N, L]")
    N, L = tok.shape
    counts = np.empty(N, dtype=np.int32)
    z = np.empty(N, dtype=np.float64)
    lib().oracle_detect(_ptr(tok), N, L, L, key, float(gamma), _seeding(seeding),
                        _ptr(counts), _ptr(z))
    return counts, z


# --- context width h (window of the h tokens before each position) ----------------

def _context(context, rows: int | None = None) -> np.ndarray:
    c = np.ascontiguousarray(context, dtype=np.int32)
    if c.ndim == 1:
        c = c.reshape(-1, 1)
    if c.ndim != 2 or (rows is not None and c.shape[0] != rows):
        raise ValueError("context must be [rows, width]")
    return c


def seed_w_many(key: int, context, cand, seeding) -> np.ndarray:
    c = _context(context)
    cand = np.ascontiguousarray(np.broadcast_to(np.asarray(cand, dtype=np.int32), (c.shape[0],)))
    out = np.empty(c.shape[0], dtype=np.uint64)
    lib().oracle_seed_w_many(key, _ptr(c), c.shape[1], _ptr(cand), c.shape[0], _seeding(seeding),
                             _ptr(out))
    return out


def is_green_w_many(key: int, context, cand, gamma: float, seeding) -> np.ndarray:
    c = _context(context)
    cand = np.ascontiguousarray(cand, dtype=np.int32)
    assert cand.shape == (c.shape[0],)
    out = np.empty(c.shape[0], dtype=np.uint8)
    lib().oracle_is_green_w_many(key, _ptr(c), c.shape[1], _ptr(cand), c.shape[0], float(gamma),
                                 _seeding(seeding), _ptr(out))
    return out.astype(bool)


def watermark_w(logits: np.ndarray, context, key: int, gamma: float, delta: float,
                seeding="context") -> np.ndarray:
    """Width-h watermark: context [B, h] holds the h tokens before this step per row."""
    out = np.array(logits, copy=True, order="C")
    B, V = out.shape
    c = _context(context, B)
    fn = lib().oracle_watermark_f32_w if out.dtype == np.float32 else lib().oracle_watermark_bf16_w
    if out.dtype not in (np.float32, np.uint16):
        raise TypeError("logits must be float32 or uint16 (bf16 bits)")
    fn(_ptr(out), B, V, V, _ptr(c), c.shape[1], key, float(gamma), float(delta), _seeding(seeding))
    return out


def green_mask_w(B: int, V: int, context, key: int, gamma: float, seeding="context") -> np.ndarray:
    c = _context(context, B)
    out = np.empty((B, (V + 31) // 32), dtype=np.uint32)
    lib().oracle_green_mask_w(_ptr(out), B, V, _ptr(c), c.shape[1], key, float(gamma),
                              _seeding(seeding))
    return out


def detect_w(tokens: np.ndarray, width: int, key: int, gamma: float, seeding="context"):
    """Width-h detect: positions h..L-1, each under the h tokens before it (T = L - h)."""
    tok = np.ascontiguousarray(tokens, dtype=np.int32)
    N, L = tok.shape
    counts = np.empty(N, dtype=np.int32)
    z = np.empty(N, dtype=np.float64)
    lib().oracle_detect_w(_ptr(tok), N, L, L, int(width), key, float(gamma), _seeding(seeding),
                          _ptr(counts), _ptr(z))
    return counts, z


def watermark_argmax(logits: np.ndarray, context, key: int, gamma: float, delta: float,
                     seeding="context"):
    """Greedy decoding of the watermarked logits: (tokens int32 [B], values float32 [B]).
    context: [B] previous tokens or [B, h] windows.  Ties -> smallest index; NaN is
    the largest value (first NaN wins); -0 == +0; bf16 values are widened to fp32."""
    x = np.ascontiguousarray(logits)
    B, V = x.shape
    c = _context(context, B)
    tokens = np.empty(B, dtype=np.int32)
    values = np.empty(B, dtype=np.float32)
    if x.dtype == np.float32:
        fn = lib().oracle_watermark_argmax_f32_w
    elif x.dtype == np.uint16:
        fn = lib().oracle_watermark_argmax_bf16_w
    else:
        raise TypeError("logits must be float32 or uint16 (bf16 bits)")
    fn(_ptr(x), B, V, V, _ptr(c), c.shape[1], key, float(gamma), float(delta), _seeding(seeding),
       _ptr(tokens), _ptr(values))
    return tokens, values


def watermark_candidates(logits: np.ndarray, candidates, context, key: int, gamma: float,
                         delta: float, seeding="self_salt") -> np.ndarray:
    """Watermark restricted to candidate ids [B, k] (SBW-ss: top-k candidates, the rest
    of the row unbiased).  Ids outside [0, V) are ignored; a repeated id is biased once."""
    out = np.array(logits, copy=True, order="C")
    B, V = out.shape
    cand = np.ascontiguousarray(candidates, dtype=np.int32)
    if cand.ndim != 2 or cand.shape[0] != B:
        raise ValueError("candidates must be [B, k]")
    c = _context(context, B)
    if out.dtype == np.float32:
        fn = lib().oracle_watermark_candidates_f32_w
    elif out.dtype == np.uint16:
        fn = lib().oracle_watermark_candidates_bf16_w
    else:
        raise TypeError("logits must be float32 or uint16 (bf16 bits)")
    fn(_ptr(out), B, V, V, _ptr(cand), cand.shape[1], _ptr(c), c.shape[1], key, float(gamma),
       float(delta), _seeding(seeding))
    return out


def detect_ex(tokens: np.ndarray, width: int, key: int, gamma: float, seeding="context",
              lengths=None, ignore_repeated: bool = False):
    """Detection with per-sequence lengths (clamped to [0, L]; None = all L) and,
    optionally, each distinct (width+1)-gram scored once.  Returns (green counts,
    scored positions T, z)."""
    tok = np.ascontiguousarray(tokens, dtype=np.int32)
    N, L = tok.shape
    lens = None if lengths is None else np.ascontiguousarray(lengths, dtype=np.int32)
    if lens is not None and lens.shape != (N,):
        raise ValueError("lengths must be [N]")
    counts = np.empty(N, dtype=np.int32)
    scored = np.empty(N, dtype=np.int32)
    z = np.empty(N, dtype=np.float64)
    lib().oracle_detect_ex(_ptr(tok), N, L, L, None if lens is None else _ptr(lens), int(width),
                           key, float(gamma), _seeding(seeding), int(bool(ignore_repeated)),
                           _ptr(counts), _ptr(scored), _ptr(z))
    return counts, scored, z


def sample_log(x) -> np.ndarray:
    """The sampler's fp32 logarithm, elementwise (finite normal x > 0)."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(a)
    lib().oracle_sample_log_many(_ptr(a), a.size, _ptr(out))
    return out


def gumbel_many(v, seed) -> np.ndarray:
    """Gumbel noise G(v, seed) = -log(-log(u)), u from CBRNG(v, seed)."""
    v = np.ascontiguousarray(v, dtype=np.uint32)
    s = np.ascontiguousarray(np.broadcast_to(np.asarray(seed, dtype=np.uint64), v.shape))
    out = np.empty(v.shape, dtype=np.float32)
    lib().oracle_gumbel_many(_ptr(v), _ptr(s), v.size, _ptr(out))
    return out


def gumbel_of_draws(x) -> np.ndarray:
    """The noise G = -log(-log u) of raw 32-bit draws x, u = ((x >> 9) + 1/2) * 2^-23."""
    x = np.ascontiguousarray(x, dtype=np.uint32)
    out = np.empty(x.shape, dtype=np.float32)
    lib().oracle_gumbel_of_draws(_ptr(x), x.size, _ptr(out))
    return out


def watermark_sample(logits: np.ndarray, context, key: int, gamma: float, delta: float,
                     seeding, seeds, inv_temperature: float = 1.0):
    """Gumbel-max draw from softmax(watermarked logits * inv_temperature), one per row:
    (tokens int32 [B], scores float32 [B]); seeds uint64 [B] drive the noise.  Ties,
    NaN and signed zeros follow watermark_argmax."""
    x = np.ascontiguousarray(logits)
    B, V = x.shape
    c = _context(context, B)
    sd = np.ascontiguousarray(seeds, dtype=np.uint64)
    if sd.shape != (B,):
        raise ValueError("seeds must be uint64 [B]")
    tokens = np.empty(B, dtype=np.int32)
    scores = np.empty(B, dtype=np.float32)
    if x.dtype == np.float32:
        fn = lib().oracle_watermark_sample_f32_w
    elif x.dtype == np.uint16:
        fn = lib().oracle_watermark_sample_bf16_w
    else:
        raise TypeError("logits must be float32 or uint16 (bf16 bits)")
    fn(_ptr(x), B, V, V, _ptr(c), c.shape[1], key, float(gamma), float(delta), _seeding(seeding),
       _ptr(sd), float(inv_temperature), _ptr(tokens), _ptr(scores))
    return tokens, scores
