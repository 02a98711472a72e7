"""fp64 CPU oracle for paged attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the GPU
library and never imports it.

The arithmetic lives in ``pa_oracle.c`` (plain C, fp64, Neumaier sums); this
module only marshals arrays through ctypes.  What it computes is the plain
definition of causal grouped-query attention over a paged KV cache
(arxiv 2511.11581, Sec. 4.1 Eq. 1-2, Sec. 4.2, Sec. 4.3); the segment/merge
helpers restate the parallel tiled softmax of Sec. 4.5 in fp64.

Pins (see ``tests/test_oracle_pins.py``): dense fp64 SDPA from torch,
block-permutation invariance, single-key and constant-V special cases,
weight row sums, uniform attention, two-key closed forms, split/merge
identity, decode == last prefill row, chunked == whole prefill,
GQA == repeated-head MHA, the fp8 decode table against torch, and the
paper's 32-tile / 4-segment partition example (Fig. 4).

``cache_write`` is the step before the path (new tokens' K/V into their
slots, with fp8 quantisation; Sec. 4.2 / Sec. 4.3 take it as done), pinned
in ``tests/test_oracle_cache_write.py``: its e4m3fn encoder against torch's
conversion and an exhaustive round trip, write-then-gather identity, skipped
slots, and the half-step error bound.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pa_oracle.c")
_LIB = os.path.join(_HERE, "libpa_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``pa_oracle.c`` with gcc into ``libpa_oracle.so``."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
               "-o", _LIB + ".tmp", _SRC, "-lpthread", "-lm"]
        subprocess.check_call(cmd)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("PA_ORACLE_LIB")  # a test-built variant (mutation tests)
    if not path:
        path = _LIB
        if not os.path.exists(_LIB):
            build(force=True)
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I = ctypes.c_int64
    D = ctypes.c_double
    prob = [P, P, P, ctypes.c_int, D, D, P, I, P, P, I, I, I, I, I, I, I, D]
    lib.pa_oracle_forward.argtypes = prob + [P, P, ctypes.c_int]
    lib.pa_oracle_forward.restype = ctypes.c_int
    lib.pa_oracle_rows.argtypes = prob + [P, I, P, P, P, I]
    lib.pa_oracle_rows.restype = ctypes.c_int
    lib.pa_oracle_segment.argtypes = prob + [I, I, I, I, P, P, P]
    lib.pa_oracle_segment.restype = ctypes.c_int
    lib.pa_oracle_merge.argtypes = [P, P, P, I, I, P]
    lib.pa_oracle_merge.restype = ctypes.c_int
    lib.pa_oracle_gather.argtypes = [P, P, I, P, I, P, I, I, I, I, I, P, P]
    lib.pa_oracle_gather.restype = ctypes.c_int
    lib.pa_oracle_segment_ranges.argtypes = [I, I, P, I]
    lib.pa_oracle_segment_ranges.restype = ctypes.c_int64
    lib.pa_oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.pa_oracle_bf16_to_f64.restype = D
    lib.pa_oracle_fp8e4m3_to_f64.argtypes = [ctypes.c_uint8]
    lib.pa_oracle_fp8e4m3_to_f64.restype = D
    lib.pa_oracle_f32_to_fp8e4m3.argtypes = [ctypes.c_float]
    lib.pa_oracle_f32_to_fp8e4m3.restype = ctypes.c_uint8
    lib.pa_oracle_cache_write.argtypes = [P, P, I, I, I, I, I, I, I, P, P, P, I, I, ctypes.c_int,
                                          ctypes.c_float, ctypes.c_float]
    lib.pa_oracle_cache_write.restype = ctypes.c_int
    lib.pa_oracle_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


class OracleError(RuntimeError):
    pass


def _bits(t):
    """A CPU torch tensor or numpy array -> contiguous numpy array of its stored bits."""
    try:
        import torch
    except ImportError:  # pragma: no cover
        torch = None
    if torch is not None and isinstance(t, torch.Tensor):
        t = t.detach().cpu().contiguous()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16), False
        if t.dtype == getattr(torch, "float8_e4m3fn", None):
            return t.view(torch.uint8).numpy(), True
        if t.dtype == torch.int32:
            return t.numpy(), False
        if t.dtype == torch.uint8:
            return t.numpy(), True
        raise TypeError(f"unsupported tensor dtype {t.dtype}")
    a = np.ascontiguousarray(t)
    return a, a.dtype == np.uint8


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc):
    if rc != 0:
        raise OracleError(_load().pa_oracle_last_error().decode())


def _problem(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale,
             k_scale, v_scale):
    qb, _ = _bits(q)
    kb, kfp8 = _bits(k_cache)
    vb, vfp8 = _bits(v_cache)
    if kfp8 != vfp8:
        raise TypeError("k_cache and v_cache must share a dtype")
    bt, _ = _bits(block_table)
    sl, _ = _bits(seq_lens)
    qsl, _ = _bits(query_start_loc)
    bt = np.ascontiguousarray(bt, dtype=np.int32)
    sl = np.ascontiguousarray(sl, dtype=np.int32)
    qsl = np.ascontiguousarray(qsl, dtype=np.int32)
    T, Hq, d = qb.shape
    NB, bs, Hkv, d2 = kb.shape
    if d2 != d or vb.shape != kb.shape:
        raise ValueError("cache shapes disagree with q")
    S = sl.shape[0]
    MB = bt.shape[1] if bt.ndim == 2 else 0
    if qsl.shape[0] != S + 1 or bt.shape[0] != S:
        raise ValueError("metadata shapes disagree")
    keep = (qb, kb, vb, bt, sl, qsl)
    args = [_ptr(qb), _ptr(kb), _ptr(vb), int(kfp8), float(k_scale), float(v_scale),
            _ptr(bt), MB, _ptr(sl), _ptr(qsl), S, T, NB, bs, Hq, Hkv, d, float(scale)]
    return args, keep, (T, Hq, d)


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


def forward(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale,
            k_scale=1.0, v_scale=1.0, threads=None, with_lse=False):
    """Full fp64 forward.  Returns out [T, Hq, d] (rows past query_start_loc[S]
    are NaN), and lse [T, Hq] if ``with_lse``."""
    lib = _load()
    args, keep, (T, Hq, d) = _problem(q, k_cache, v_cache, block_table, seq_lens,
                                      query_start_loc, scale, k_scale, v_scale)
    out = np.full((T, Hq, d), np.nan, dtype=np.float64)
    lse = np.full((T, Hq), np.nan, dtype=np.float64) if with_lse else None
    nt = threads if threads is not None else default_threads()
    _check(lib.pa_oracle_forward(*args, _ptr(out), _ptr(lse) if lse is not None else None, nt))
    del keep
    return (out, lse) if with_lse else out


def rows(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale, row_ids,
         k_scale=1.0, v_scale=1.0, with_lse=False, max_keys=0):
    """fp64 result of selected (token, head) rows.  ``row_ids`` is int [n, 2].
    With ``max_keys`` > 0 also returns the normalised weights [n, max_keys]."""
    lib = _load()
    args, keep, (T, Hq, d) = _problem(q, k_cache, v_cache, block_table, seq_lens,
                                      query_start_loc, scale, k_scale, v_scale)
    r = np.ascontiguousarray(np.asarray(row_ids, dtype=np.int64).reshape(-1, 2))
    n = r.shape[0]
    out = np.zeros((n, d), dtype=np.float64)
    lse = np.zeros((n,), dtype=np.float64)
    w = np.zeros((n, max_keys), dtype=np.float64) if max_keys > 0 else None
    _check(lib.pa_oracle_rows(*args, _ptr(r), n, _ptr(out), _ptr(lse),
                              _ptr(w) if w is not None else None, max_keys))
    del keep
    res = [out]
    if with_lse:
        res.append(lse)
    if w is not None:
        res.append(w)
    return res[0] if len(res) == 1 else tuple(res)


def segment(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale,
            token, head, k0, k1, k_scale=1.0, v_scale=1.0):
    """(acc [d], m, l) partials of one row over keys [k0, k1) (Sec. 4.5)."""
    lib = _load()
    args, keep, (T, Hq, d) = _problem(q, k_cache, v_cache, block_table, seq_lens,
                                      query_start_loc, scale, k_scale, v_scale)
    acc = np.zeros((d,), dtype=np.float64)
    m = ctypes.c_double()
    l = ctypes.c_double()
    _check(lib.pa_oracle_segment(*args, int(token), int(head), int(k0), int(k1), _ptr(acc),
                                 ctypes.byref(m), ctypes.byref(l)))
    del keep
    return acc, m.value, l.value


def merge(acc, m, l):
    """Merge segment partials acc [n, d], m [n], l [n] into one row [d]."""
    lib = _load()
    acc = np.ascontiguousarray(acc, dtype=np.float64)
    m = np.ascontiguousarray(m, dtype=np.float64)
    l = np.ascontiguousarray(l, dtype=np.float64)
    n, d = acc.shape
    out = np.zeros((d,), dtype=np.float64)
    _check(lib.pa_oracle_merge(_ptr(acc), _ptr(m), _ptr(l), n, d, _ptr(out)))
    return out


def segment_ranges(n_tiles, tiles_per_segment):
    """Tile ranges [(begin, end)] of the segments of a row (Sec. 4.5, Fig. 4)."""
    lib = _load()
    cap = max(1, (int(n_tiles) + int(tiles_per_segment) - 1) // max(1, int(tiles_per_segment)))
    buf = np.zeros((cap, 2), dtype=np.int64)
    n = lib.pa_oracle_segment_ranges(int(n_tiles), int(tiles_per_segment), _ptr(buf), cap)
    if n < 0:
        raise OracleError("invalid segment partition request")
    return [tuple(int(x) for x in buf[k]) for k in range(n)]


def gather(k_cache, v_cache, block_table, seq_lens, fill=0):
    """Stored K/V bytes in logical order: two uint8 arrays
    [S, MB*bs, Hkv, d*elem_bytes]; positions >= seq_len keep ``fill``."""
    lib = _load()
    kb, fp8 = _bits(k_cache)
    vb, _ = _bits(v_cache)
    bt, _ = _bits(block_table)
    sl, _ = _bits(seq_lens)
    bt = np.ascontiguousarray(bt, dtype=np.int32)
    sl = np.ascontiguousarray(sl, dtype=np.int32)
    NB, bs, Hkv, d = kb.shape
    eb = 1 if fp8 else 2
    S, MB = bt.shape
    kd = np.full((S, MB * bs, Hkv, d * eb), fill, dtype=np.uint8)
    vd = np.full((S, MB * bs, Hkv, d * eb), fill, dtype=np.uint8)
    _check(lib.pa_oracle_gather(_ptr(kb), _ptr(vb), eb, _ptr(bt), MB, _ptr(sl), S, NB, bs,
                                Hkv, d, _ptr(kd), _ptr(vd)))
    return kd, vd


def bf16_to_f64(bits: int) -> float:
    return _load().pa_oracle_bf16_to_f64(int(bits))


def fp8e4m3_to_f64(bits: int) -> float:
    return _load().pa_oracle_fp8e4m3_to_f64(int(bits))


def f32_to_fp8e4m3(x: float) -> int:
    """e4m3fn code of the fp32 value x (limited to +-448, nearest, ties to even)."""
    return int(_load().pa_oracle_f32_to_fp8e4m3(float(x)))


def cache_write(key, value, slot_mapping, k_cache, v_cache, k_scale=1.0, v_scale=1.0):
    """The caches after writing row t of key / value ([T, Hkv, d] bf16) into
    slot slot_mapping[t] (= block * block_size + offset; slots outside the
    cache are skipped).  fp8 caches store the e4m3fn code of value / scale
    (the division in fp32).  Returns two new numpy arrays of the caches'
    stored bits (uint16 for bf16, uint8 for fp8); the inputs are not changed."""
    lib = _load()
    kb, _ = _bits(key)
    vb, _ = _bits(value)
    sm, _ = _bits(slot_mapping)
    sm = np.ascontiguousarray(sm, dtype=np.int32)
    kc, fp8 = _bits(k_cache)
    vc, _ = _bits(v_cache)
    kc = kc.copy()
    vc = vc.copy()
    T, Hkv, d = kb.shape
    NB, bs = kc.shape[0], kc.shape[1]
    _check(lib.pa_oracle_cache_write(_ptr(kb), _ptr(vb), T, Hkv, d, Hkv * d, d, Hkv * d, d,
                                     _ptr(sm), _ptr(kc), _ptr(vc), NB, bs, 1 if fp8 else 0,
                                     float(k_scale), float(v_scale)))
    return kc, vc
