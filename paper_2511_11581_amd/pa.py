"""ctypes binding of libpa.so (declared in include/pa.h).

Argument marshalling only: torch tensors are described by ``pa_tensor``
(device pointer, dtype, shape, strides) and the current HIP stream is
passed through.  Every attention step runs in the library's HIP kernels;
there is no fallback: if ``libpa.so`` is missing or fails to load, the first
call raises.

The functions keep the C names (``EXPORTS`` lists every entry point of the
header, from ``pa_workspace_bytes`` and ``pa_create`` to ``pa_forward``,
``pa_forward_hinted``, ``pa_forward_noalloc`` and ``pa_cache_write``).
``PagedAttention`` bundles a handle with a workspace allocated through
torch.
"""
from __future__ import annotations

import ctypes
import os
import struct
import threading
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpa.so")

PA_OK = 0
PA_ERR_INVALID_ARG = 1
PA_ERR_UNSUPPORTED = 2
PA_ERR_WORKSPACE = 3
PA_ERR_DEVICE = 4
STATUS_NAMES = {0: "PA_OK", 1: "PA_ERR_INVALID_ARG", 2: "PA_ERR_UNSUPPORTED",
                3: "PA_ERR_WORKSPACE", 4: "PA_ERR_DEVICE"}

PA_DTYPE_BF16 = 0
PA_DTYPE_FP8_E4M3 = 1
PA_DTYPE_I32 = 2
PA_DTYPE_F32 = 3
PA_FLAG_VALIDATE = 1
PA_FLAG_PROFILE = 2
PA_FLAG_NO_SPLIT_KV = 4
PA_KERNEL_KINDS = 4
KERNEL_NAMES = ("decode", "merge", "prefill", "plan")
PA_MAX_DIMS = 4

# Every function declared in include/pa.h.
EXPORTS = ("pa_workspace_bytes", "pa_create", "pa_forward", "pa_forward_hinted", "pa_forward_noalloc",
           "pa_forward_baseline", "pa_cache_write", "pa_debug_gather", "pa_plan",
           "pa_decode_pieces", "pa_profile_read", "pa_destroy", "pa_last_error")


class pa_tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * PA_MAX_DIMS), ("stride", ctypes.c_int64 * PA_MAX_DIMS)]


class pa_config(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int32), ("k_scale", ctypes.c_float),
                ("v_scale", ctypes.c_float), ("flags", ctypes.c_uint32),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_uint64)]


class pa_plan_info(ctypes.Structure):
    _fields_ = [("decode_launch", ctypes.c_int32), ("decode_step", ctypes.c_int32),
                ("decode_waves", ctypes.c_int32), ("decode_workers", ctypes.c_int32),
                ("decode_min_steps", ctypes.c_int32), ("decode_unit_heads", ctypes.c_int32),
                ("decode_whole_units", ctypes.c_int32),
                ("merge_launch", ctypes.c_int32), ("prefill_qmin", ctypes.c_int32),
                ("prefill_launch", ctypes.c_int32), ("block_m", ctypes.c_int32),
                ("block_q", ctypes.c_int32), ("prefill_tile", ctypes.c_int32),
                ("decode_grid", ctypes.c_int64 * 3), ("merge_grid", ctypes.c_int64 * 3),
                ("prefill_grid", ctypes.c_int64 * 3), ("prefill_units", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_uint64)]

    def as_dict(self):
        d = {}
        for name, _ in self._fields_:
            v = getattr(self, name)
            d[name] = list(v) if hasattr(v, "__len__") else int(v)
        return d


class pa_batch_hint(ctypes.Structure):
    _fields_ = [("num_decode_seqs", ctypes.c_int32), ("max_query_len", ctypes.c_int32)]


class pa_decode_piece(ctypes.Structure):
    _fields_ = [("seq", ctypes.c_int32), ("kv_head", ctypes.c_int32), ("worker", ctypes.c_int32),
                ("first_key", ctypes.c_int32), ("end_key", ctypes.c_int32), ("slot", ctypes.c_int32)]


class pa_profile(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64 * PA_KERNEL_KINDS),
                ("total_ms", ctypes.c_double * PA_KERNEL_KINDS)]


class PaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libpa.so; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2511_11581_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    T = ctypes.POINTER(pa_tensor)
    C = ctypes.POINTER(pa_config)
    lib.pa_workspace_bytes.argtypes = [C, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                       ctypes.POINTER(ctypes.c_uint64)]
    lib.pa_create.argtypes = [C, ctypes.POINTER(P)]
    lib.pa_forward.argtypes = [P, T, T, T, T, T, T, ctypes.c_float, T, P]
    lib.pa_forward_noalloc.argtypes = [P, T, T, T, T, T, T, ctypes.c_float, T, P]
    lib.pa_forward_hinted.argtypes = [P, T, T, T, T, T, T, ctypes.c_float, T,
                                      ctypes.POINTER(pa_batch_hint), P]
    lib.pa_forward_baseline.argtypes = [P, T, T, T, T, T, T, ctypes.c_float, T, P]
    lib.pa_debug_gather.argtypes = [P, T, T, T, T, T, ctypes.c_int64, T, T, P]
    lib.pa_cache_write.argtypes = [P, T, T, T, T, T, P]
    lib.pa_plan.argtypes = [P, C, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                            ctypes.POINTER(pa_batch_hint), ctypes.POINTER(pa_plan_info)]
    I32P = ctypes.POINTER(ctypes.c_int32)
    lib.pa_decode_pieces.argtypes = [P, C, ctypes.c_int32, I32P, I32P, ctypes.c_int64,
                                     ctypes.c_int64, ctypes.c_int64,
                                     ctypes.POINTER(pa_decode_piece), ctypes.c_int64,
                                     ctypes.POINTER(ctypes.c_int64)]
    lib.pa_profile_read.argtypes = [P, ctypes.POINTER(pa_profile), ctypes.c_int]
    lib.pa_destroy.argtypes = [P]
    lib.pa_destroy.restype = None
    lib.pa_last_error.argtypes = []
    lib.pa_last_error.restype = ctypes.c_char_p
    for name in ("pa_workspace_bytes", "pa_create", "pa_forward", "pa_forward_hinted", "pa_forward_noalloc",
                 "pa_forward_baseline", "pa_cache_write", "pa_debug_gather", "pa_plan",
                 "pa_decode_pieces", "pa_profile_read"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def pa_last_error() -> str:
    return load_library().pa_last_error().decode()


def _check(st: int):
    if st != PA_OK:
        raise PaError(st, pa_last_error())


_DTYPES = {torch.bfloat16: PA_DTYPE_BF16, torch.float8_e4m3fn: PA_DTYPE_FP8_E4M3,
           torch.int32: PA_DTYPE_I32, torch.float32: PA_DTYPE_F32}


def describe(t: torch.Tensor) -> pa_tensor:
    """pa_tensor descriptor of a torch tensor (no copy)."""
    if t.dim() > PA_MAX_DIMS:
        raise ValueError("at most 4 dimensions")
    d = pa_tensor()
    d.data = t.data_ptr() if t.numel() > 0 else 0
    d.dtype = _DTYPES.get(t.dtype, -1)
    d.ndim = t.dim()
    for i in range(t.dim()):
        d.shape[i] = t.shape[i]
        d.stride[i] = t.stride(i)
    return d


# The per-call path packs the descriptors with struct into one array per
# thread (the same bytes as describe(), ~1.3 us per tensor against ~3.8 us
# for field-by-field ctypes assignment, which dominated small calls).
_PACK = struct.Struct("=Qii4q4q")
assert _PACK.size == ctypes.sizeof(pa_tensor)
_ZEROS = ((), (0,), (0, 0), (0, 0, 0), (0, 0, 0, 0))
_tls = threading.local()


def _descs(*tensors):
    """Pointers to descriptors of `tensors`, valid until this thread's next call."""
    arr = getattr(_tls, "arr", None)
    if arr is None:
        arr = _tls.arr = (pa_tensor * 8)()
        _tls.refs = tuple(ctypes.byref(arr[i]) for i in range(8))   # views of arr's buffer
    for i, t in enumerate(tensors):
        sh = t.shape
        n = len(sh)
        if n > PA_MAX_DIMS:
            raise ValueError("at most 4 dimensions")
        z = _ZEROS[PA_MAX_DIMS - n]
        _PACK.pack_into(arr, i * _PACK.size, t.data_ptr() if t.numel() > 0 else 0,
                        _DTYPES.get(t.dtype, -1), n, *sh, *z, *t.stride(), *z)
    return _tls.refs[:len(tensors)]


def make_config(num_q_heads, num_kv_heads, head_dim, block_size=16, kv_dtype=PA_DTYPE_BF16,
                k_scale=1.0, v_scale=1.0, flags=0, workspace=0, workspace_bytes=0) -> pa_config:
    c = pa_config()
    c.num_q_heads, c.num_kv_heads, c.head_dim, c.block_size = (num_q_heads, num_kv_heads,
                                                              head_dim, block_size)
    c.kv_dtype = kv_dtype
    c.k_scale, c.v_scale = k_scale, v_scale
    c.flags = flags
    c.workspace = workspace
    c.workspace_bytes = workspace_bytes
    return c


def pa_workspace_bytes(cfg: pa_config, max_tokens: int, max_seqs: int,
                       max_blocks_per_seq: int) -> int:
    out = ctypes.c_uint64()
    _check(load_library().pa_workspace_bytes(ctypes.byref(cfg), max_tokens, max_seqs,
                                             max_blocks_per_seq, ctypes.byref(out)))
    return int(out.value)


def pa_create(cfg: pa_config) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    _check(load_library().pa_create(ctypes.byref(cfg), ctypes.byref(h)))
    return h


def pa_destroy(h) -> None:
    if h:
        load_library().pa_destroy(h)


def pa_plan(h=None, cfg: Optional[pa_config] = None, num_cus: int = 0, num_tokens: int = 0,
            num_seqs: int = 0, max_blocks_per_seq: int = 0, hint=None) -> dict:
    """hint: optional (num_decode_seqs, max_query_len), as for forward."""
    info = pa_plan_info()
    hp = ctypes.byref(pa_batch_hint(int(hint[0]), int(hint[1]))) if hint is not None else None
    _check(load_library().pa_plan(h, ctypes.byref(cfg) if cfg is not None else None, num_cus,
                                  num_tokens, num_seqs, max_blocks_per_seq, hp, ctypes.byref(info)))
    return info.as_dict()


def pa_decode_pieces(h=None, cfg: Optional[pa_config] = None, num_cus: int = 0, seq_lens=(),
                     query_start_loc=(), num_tokens: int = 0, max_blocks_per_seq: int = 0) -> list:
    """The decode partition of a batch whose metadata is given on the host:
    a list of dicts {seq, kv_head, worker, first_key, end_key, slot}."""
    lib = load_library()
    sl = (ctypes.c_int32 * max(1, len(seq_lens)))(*[int(x) for x in seq_lens])
    qsl = (ctypes.c_int32 * max(1, len(query_start_loc)))(*[int(x) for x in query_start_loc])
    cfgp = ctypes.byref(cfg) if cfg is not None else None
    n = ctypes.c_int64()
    _check(lib.pa_decode_pieces(h, cfgp, num_cus, sl, qsl, len(seq_lens), num_tokens,
                                max_blocks_per_seq, None, 0, ctypes.byref(n)))
    buf = (pa_decode_piece * max(1, n.value))()
    _check(lib.pa_decode_pieces(h, cfgp, num_cus, sl, qsl, len(seq_lens), num_tokens,
                                max_blocks_per_seq, buf, n.value, ctypes.byref(n)))
    return [{k: int(getattr(buf[i], k)) for k, _ in pa_decode_piece._fields_} for i in range(n.value)]


def pa_profile_read(h, reset: bool = True) -> dict:
    """{kernel: (launches, total_ms)} recorded under PA_FLAG_PROFILE."""
    prof = pa_profile()
    _check(load_library().pa_profile_read(h, ctypes.byref(prof), int(reset)))
    return {KERNEL_NAMES[k]: (int(prof.launches[k]), float(prof.total_ms[k]))
            for k in range(PA_KERNEL_KINDS)}


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(stream)


def pa_forward(h, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale, out,
               stream=None) -> None:
    d = _descs(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, out)
    _check(load_library().pa_forward(h, *d[:6], float(scale), d[6], _stream(stream)))


def pa_forward_hinted(h, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale, out,
                      num_decode_seqs=-1, max_query_len=-1, stream=None) -> None:
    """pa_forward with the host's knowledge of the batch (-1: unknown): no
    decode rows skips the decode + merge launches, max_query_len <= 1 the
    Q-block launch."""
    d = _descs(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, out)
    hint = pa_batch_hint(int(num_decode_seqs), int(max_query_len))
    _check(load_library().pa_forward_hinted(h, *d[:6], float(scale), d[6], ctypes.byref(hint),
                                            _stream(stream)))


def pa_forward_noalloc(h, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale, out,
                       stream=None) -> None:
    """pa_forward with the library's static device scratch instead of a
    workspace (for callers that cannot allocate)."""
    d = _descs(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, out)
    _check(load_library().pa_forward_noalloc(h, *d[:6], float(scale), d[6], _stream(stream)))


def pa_forward_baseline(h, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, scale,
                        out, stream=None) -> None:
    d = _descs(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, out)
    _check(load_library().pa_forward_baseline(h, *d[:6], float(scale), d[6], _stream(stream)))


def pa_debug_gather(h, k_cache, v_cache, block_table, seq_lens, query_start_loc, num_tokens,
                    k_dense, v_dense, stream=None) -> None:
    d = _descs(k_cache, v_cache, block_table, seq_lens, query_start_loc, k_dense, v_dense)
    _check(load_library().pa_debug_gather(h, *d[:5], int(num_tokens), *d[5:], _stream(stream)))


def pa_cache_write(h, key, value, slot_mapping, k_cache, v_cache, stream=None) -> None:
    d = _descs(key, value, slot_mapping, k_cache, v_cache)
    _check(load_library().pa_cache_write(h, *d, _stream(stream)))


class PagedAttention:
    """A handle plus a torch-allocated workspace sized for the given maxima."""

    def __init__(self, num_q_heads: int, num_kv_heads: int, head_dim: int, block_size: int = 16,
                 kv_dtype: torch.dtype = torch.bfloat16, k_scale: float = 1.0,
                 v_scale: float = 1.0, max_tokens: int = 1, max_seqs: int = 1,
                 max_blocks_per_seq: int = 1, validate: bool = False, profile: bool = False,
                 no_split_kv: bool = False, device="cuda"):
        """no_split_kv: ablation only, single-token rows through the Q-block
        kernel (PA_FLAG_NO_SPLIT_KV)."""
        kvd = _DTYPES.get(kv_dtype, -1)
        flags = ((PA_FLAG_VALIDATE if validate else 0) | (PA_FLAG_PROFILE if profile else 0)
                 | (PA_FLAG_NO_SPLIT_KV if no_split_kv else 0))
        cfg = make_config(num_q_heads, num_kv_heads, head_dim, block_size, kvd, k_scale, v_scale,
                          flags)
        nbytes = pa_workspace_bytes(cfg, max_tokens, max_seqs, max_blocks_per_seq)
        self._ws_raw = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        base = self._ws_raw.data_ptr()
        cfg.workspace = (base + 255) & ~255
        cfg.workspace_bytes = nbytes
        self.cfg = cfg
        self.handle = pa_create(cfg)

    def plan(self, num_tokens: int, num_seqs: int, max_blocks_per_seq: int, hint=None) -> dict:
        return pa_plan(self.handle, None, 0, num_tokens, num_seqs, max_blocks_per_seq, hint)

    def forward(self, q, k_cache, v_cache, block_table, seq_lens, query_start_loc,
                scale: Optional[float] = None, out: Optional[torch.Tensor] = None, stream=None,
                hint=None):
        """hint: optional (num_decode_seqs, max_query_len) known on the host
        (pa_forward_hinted); None calls pa_forward."""
        if out is None:
            out = torch.empty_like(q)
        if scale is None:
            scale = q.shape[-1] ** -0.5
        if hint is None:
            pa_forward(self.handle, q, k_cache, v_cache, block_table, seq_lens, query_start_loc,
                       scale, out, stream)
        else:
            pa_forward_hinted(self.handle, q, k_cache, v_cache, block_table, seq_lens,
                              query_start_loc, scale, out, hint[0], hint[1], stream)
        return out

    def forward_baseline(self, q, k_cache, v_cache, block_table, seq_lens, query_start_loc,
                         scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                         stream=None):
        """The same attention with the paper's baseline decomposition (ablation only)."""
        if out is None:
            out = torch.empty_like(q)
        if scale is None:
            scale = q.shape[-1] ** -0.5
        pa_forward_baseline(self.handle, q, k_cache, v_cache, block_table, seq_lens,
                            query_start_loc, scale, out, stream)
        return out

    def profile(self, reset: bool = True) -> dict:
        return pa_profile_read(self.handle, reset)

    def cache_write(self, key, value, slot_mapping, k_cache, v_cache, stream=None):
        """Write new tokens' K/V (bf16 [T, Hkv, d]) into their slots of the caches."""
        pa_cache_write(self.handle, key, value, slot_mapping, k_cache, v_cache, stream)

    def gather(self, k_cache, v_cache, block_table, seq_lens, query_start_loc, num_tokens,
               stream=None):
        """The K/V bytes the attention loaders read for this batch (debug):
        dense [S, MB * bs, Hkv, d] tensors, zero where nothing is read."""
        S, MB = block_table.shape
        shape = (S, MB * k_cache.shape[1], k_cache.shape[2], k_cache.shape[3])
        kd = torch.zeros(shape, dtype=k_cache.dtype, device=k_cache.device)
        vd = torch.zeros(shape, dtype=v_cache.dtype, device=v_cache.device)
        pa_debug_gather(self.handle, k_cache, v_cache, block_table, seq_lens, query_start_loc,
                        num_tokens, kd, vd, stream)
        return kd, vd

    def close(self):
        if getattr(self, "handle", None):
            pa_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
