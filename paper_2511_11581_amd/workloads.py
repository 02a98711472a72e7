"""Seeded synthetic batches for paged attention.

This module only draws inputs; it holds none of the attention arithmetic and
is the one piece of code that both the GPU library's callers and the oracle's
callers use.  A batch is a list of sequences, each with a context length
(tokens already cached) and a query length (new tokens); the sequence length
is their sum (arxiv 2511.11581, Sec. 4.2).  The KV cache is a pool of
physical blocks of ``block_size`` token slots addressed through a block table
(Sec. 4.3).

Draw order (fixed): lengths -> block permutation -> Q -> K -> V.  Lengths and
the permutation come from a CPU ``torch.Generator`` seeded with ``seed``;
values come from a generator on the target device seeded with ``seed + 1``.
Values are N(0, 1) drawn in fp32 and rounded to bf16.  For fp8 caches the
fp32 draws are quantised per tensor with ``scale = amax / 448`` to OCP
e4m3fn.  Slots past a sequence's length in its last block and blocks no
sequence references are NaN-poisoned (``poison=True``); table entries past a
sequence's last block hold -1.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import torch

FP8 = torch.float8_e4m3fn
FP8_MAX = 448.0

# The five benchmark batches.  Each is (description, builder).
CONFIG_NAMES = {
    1: "tiny-decode: 4 seqs ctx {17,64,100,255} q=1, Hq 8 / Hkv 2, d 64, bf16, pool 64 blocks",
    2: "llama3-8b-decode: 64 seqs ctx U[512,8192] q=1, Hq 32 / Hkv 8, d 128, bf16",
    3: "varlen-prefill: q {2048,1024,3000,517} ctx 0, Hq 32 / Hkv 8, d 128, bf16",
    4: "mixed: 8 x (ctx U[0,4096], q 512) + 120 x (ctx U[1024,16384], q 1), Hq 32 / Hkv 8, d 128, bf16",
    5: "llama3-70b-long-decode: 16 seqs ctx U[32768,131072] q=1, Hq 64 / Hkv 8, d 128, fp8 e4m3 KV",
}


@dataclasses.dataclass
class Workload:
    name: str
    q: torch.Tensor                 # bf16 [T, Hq, d]
    k_cache: torch.Tensor           # bf16 or float8_e4m3fn [NB, bs, Hkv, d]
    v_cache: torch.Tensor
    block_table: torch.Tensor       # int32 [S, MB]
    seq_lens: torch.Tensor          # int32 [S]
    query_start_loc: torch.Tensor   # int32 [S + 1]
    scale: float
    k_scale: float
    v_scale: float
    ctx_lens: List[int]
    q_lens: List[int]
    seed: int

    @property
    def num_seqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def num_tokens(self) -> int:
        return int(self.q.shape[0])

    @property
    def num_q_heads(self) -> int:
        return int(self.q.shape[1])

    @property
    def head_dim(self) -> int:
        return int(self.q.shape[2])

    @property
    def num_kv_heads(self) -> int:
        return int(self.k_cache.shape[2])

    @property
    def block_size(self) -> int:
        return int(self.k_cache.shape[1])

    @property
    def num_blocks(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def kv_fp8(self) -> bool:
        return self.k_cache.dtype == FP8

    @property
    def seq_len_list(self) -> List[int]:
        return [c + q for c, q in zip(self.ctx_lens, self.q_lens)]

    def to(self, device) -> "Workload":
        f = lambda t: t.to(device)
        return dataclasses.replace(
            self, q=f(self.q), k_cache=f(self.k_cache), v_cache=f(self.v_cache),
            block_table=f(self.block_table), seq_lens=f(self.seq_lens),
            query_start_loc=f(self.query_start_loc))


def _fill_normal(shape, gen, device, out_dtype, chunk=1 << 26, mult=1.0):
    """N(0,1) fp32 draws (times ``mult``) rounded to ``out_dtype``, drawn in chunks."""
    n = math.prod(shape)
    out = torch.empty(n, dtype=out_dtype, device=device)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        x = torch.randn(e - s, generator=gen, device=device, dtype=torch.float32)
        if mult != 1.0:
            x = x * mult
        out[s:e] = x.to(out_dtype)
    return out.view(*shape)


def _fill_fp8(shape, gen, device, chunk=1 << 26, plant=None):
    """N(0,1) fp32 draws quantised per tensor to e4m3fn; returns (tensor, scale).
    ``plant`` may overwrite rows of the fp32 draws (viewed with ``shape``)
    before the scale is taken."""
    n = math.prod(shape)
    x = torch.empty(n, dtype=torch.float32, device=device)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        x[s:e] = torch.randn(e - s, generator=gen, device=device, dtype=torch.float32)
    if plant is not None:
        plant(x.view(*shape))
    amax = float(x.abs().max()) if n else 1.0
    scale = amax / FP8_MAX if amax > 0 else 1.0
    out = torch.empty(n, dtype=FP8, device=device)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        out[s:e] = (x[s:e] / scale).clamp_(-FP8_MAX, FP8_MAX).to(FP8)
    del x
    return out.view(*shape), scale


def make_batch(seqs: Sequence[Tuple[int, int]], num_q_heads: int, num_kv_heads: int,
               head_dim: int, kv_dtype: str = "bf16", block_size: int = 16, seed: int = 0,
               pool_blocks: Optional[int] = None, poison: bool = True, device="cpu",
               table_width: Optional[int] = None, token_pad: int = 0,
               name: str = "custom", scale: Optional[float] = None,
               q_scale: float = 1.0, spikes: Sequence[Tuple[int, int, int, float]] = (),
               _gen: Optional[torch.Generator] = None) -> Workload:
    """Build a paged batch from explicit (context_len, query_len) pairs.

    ``pool_blocks`` defaults to the blocks the batch needs; ``table_width``
    defaults to the longest sequence's block count; ``token_pad`` appends
    query rows past ``query_start_loc[S]`` that no sequence owns.

    Large logits: ``q_scale`` multiplies the fp32 Q draws before rounding.
    ``spikes`` plants keys aligned with a query: for (i, p, j, c), key
    position p of sequence i gets, in every kv head g, c times the mean of
    the G query rows of token j of sequence i in that group, so those rows
    score it far above the rest (set before rounding / quantisation)."""
    gen = _gen if _gen is not None else torch.Generator().manual_seed(seed)
    ctx = [int(c) for c, _ in seqs]
    ql = [int(q) for _, q in seqs]
    L = [c + q for c, q in zip(ctx, ql)]
    S = len(seqs)
    nblk = [(x + block_size - 1) // block_size for x in L]
    need = sum(nblk)
    NB = pool_blocks if pool_blocks is not None else max(need, 1)
    if NB < need:
        raise ValueError(f"pool of {NB} blocks cannot hold {need}")
    MB = table_width if table_width is not None else max(nblk + [1])
    if MB < max(nblk + [0]):
        raise ValueError("table_width too small")
    perm = torch.randperm(NB, generator=gen)
    table = torch.full((S, MB), -1, dtype=torch.int32)
    off = 0
    for i, nb in enumerate(nblk):
        table[i, :nb] = perm[off:off + nb].to(torch.int32)
        off += nb
    qsl = torch.zeros(S + 1, dtype=torch.int32)
    if S:
        qsl[1:] = torch.cumsum(torch.tensor(ql, dtype=torch.int64), 0).to(torch.int32)
    T = int(qsl[-1]) + token_pad

    vgen = torch.Generator(device=device).manual_seed(seed + 1)
    q = _fill_normal((T, num_q_heads, head_dim), vgen, device, torch.bfloat16, mult=q_scale)
    shape = (NB, block_size, num_kv_heads, head_dim)
    G = num_q_heads // num_kv_heads

    def plant(kx):
        # kx: [NB, bs, Hkv, d] (fp32 draws or the bf16 cache)
        for (i, p, j, c) in spikes:
            if not (0 <= p < L[i] and 0 <= j < ql[i]):
                raise ValueError(f"spike {(i, p, j)} outside sequence {i}")
            page, slot = int(table[i, p // block_size]), p % block_size
            qrow = q[int(qsl[i]) + j].float().view(num_kv_heads, G, head_dim).mean(1)
            kx[page, slot] = (c * qrow).to(kx.dtype)

    if kv_dtype == "bf16":
        k = _fill_normal(shape, vgen, device, torch.bfloat16)
        v = _fill_normal(shape, vgen, device, torch.bfloat16)
        if spikes:
            plant(k)
        ks = vs = 1.0
    elif kv_dtype == "fp8":
        k, ks = _fill_fp8(shape, vgen, device, plant=plant if spikes else None)
        v, vs = _fill_fp8(shape, vgen, device)
    else:
        raise ValueError(f"unknown kv_dtype {kv_dtype}")

    if poison:
        used = torch.zeros(NB * block_size, dtype=torch.bool)
        for i in range(S):
            if L[i] == 0:
                continue
            blocks = table[i, :nblk[i]].to(torch.int64)
            slots = (blocks[:, None] * block_size + torch.arange(block_size)[None, :]).reshape(-1)
            used[slots[:L[i]]] = True
        unused = (~used).to(device)
        if kv_dtype == "bf16":
            nan_bits = torch.tensor(0x7FC0, dtype=torch.int16).item()
            for c in (k, v):
                c.view(torch.int16).view(NB * block_size, -1)[unused] = nan_bits
        else:
            for c in (k, v):
                c.view(torch.uint8).view(NB * block_size, -1)[unused] = 0x7F
        if token_pad:
            q.view(torch.int16)[T - token_pad:] = torch.tensor(0x7FC0, dtype=torch.int16).item()

    return Workload(
        name=name, q=q, k_cache=k, v_cache=v, block_table=table.to(device),
        seq_lens=torch.tensor(L, dtype=torch.int32).to(device), query_start_loc=qsl.to(device),
        scale=float(scale if scale is not None else 1.0 / math.sqrt(head_dim)),
        k_scale=float(ks), v_scale=float(vs), ctx_lens=ctx, q_lens=ql, seed=seed)


def _randint(gen, lo, hi, n):
    """n integers uniform on [lo, hi] inclusive."""
    return [int(x) for x in torch.randint(lo, hi + 1, (n,), generator=gen)]


def config_seqs(k: int, seed: Optional[int] = None):
    """(seqs, heads/dims kwargs, generator) for benchmark batch k (1..5)."""
    seed = 11581 + k if seed is None else seed
    gen = torch.Generator().manual_seed(seed)
    if k == 1:
        seqs = [(c, 1) for c in (17, 64, 100, 255)]
        kw = dict(num_q_heads=8, num_kv_heads=2, head_dim=64, pool_blocks=64)
    elif k == 2:
        seqs = [(c, 1) for c in _randint(gen, 512, 8192, 64)]
        kw = dict(num_q_heads=32, num_kv_heads=8, head_dim=128)
    elif k == 3:
        seqs = [(0, q) for q in (2048, 1024, 3000, 517)]
        kw = dict(num_q_heads=32, num_kv_heads=8, head_dim=128)
    elif k == 4:
        pre = [(c, 512) for c in _randint(gen, 0, 4096, 8)]
        dec = [(c, 1) for c in _randint(gen, 1024, 16384, 120)]
        seqs = dec + pre  # decode-first order
        kw = dict(num_q_heads=32, num_kv_heads=8, head_dim=128)
    elif k == 5:
        seqs = [(c, 1) for c in _randint(gen, 32768, 131072, 16)]
        kw = dict(num_q_heads=64, num_kv_heads=8, head_dim=128, kv_dtype="fp8")
    else:
        raise ValueError(f"no benchmark batch {k}")
    return seqs, kw, gen, seed


def make_config(k: int, seed: Optional[int] = None, device="cpu", poison: bool = True,
                shuffle: bool = False) -> Workload:
    """Benchmark batch k (1..5), seeded with 11581 + k unless ``seed`` is given.
    ``shuffle`` permutes the sequence order (same lengths)."""
    seqs, kw, gen, seed = config_seqs(k, seed)
    if shuffle:
        order = torch.randperm(len(seqs), generator=gen).tolist()
        seqs = [seqs[i] for i in order]
    return make_batch(seqs, seed=seed, device=device, poison=poison,
                      name=f"config{k}", _gen=gen, **kw)
