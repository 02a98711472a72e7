"""Pins of the oracle's KV-cache write (new tokens' K/V into their slots; the
paper's kernels take this step as done, Sec. 4.2 / Sec. 4.3) and of its fp8
e4m3fn encoder.  CPU only."""
import numpy as np
import pytest
import torch

import oracle

FP8 = torch.float8_e4m3fn


def _codes(x):
    return np.array([oracle.f32_to_fp8e4m3(float(v)) for v in x], dtype=np.uint8)


def test_fp8_encoder_matches_torch_rounding_in_range():
    # Library pin: torch's e4m3fn conversion rounds to nearest, ties to even.
    g = torch.Generator().manual_seed(7)
    x = torch.cat([torch.randn(3000, generator=g) * s for s in (1e-3, 0.05, 1.0, 30.0, 200.0)])
    # every code's value and every midpoint between neighbouring codes (the ties)
    vals = torch.tensor([oracle.fp8e4m3_to_f64(c) for c in range(0x7F)], dtype=torch.float64)
    mids = (vals[1:] + vals[:-1]) / 2
    x = torch.cat([x, vals.float(), mids.float(), -vals.float(), -mids.float()])
    x = x.clamp(-448, 448).float()
    ref = x.to(FP8).view(torch.uint8).numpy()
    assert np.array_equal(_codes(x.numpy()), ref)


def test_fp8_encoder_saturates_and_round_trips():
    assert oracle.f32_to_fp8e4m3(1e6) == 0x7E and oracle.f32_to_fp8e4m3(-1e6) == 0xFE
    assert oracle.f32_to_fp8e4m3(464.0) == 0x7E      # above the last midpoint: still limited to 448
    assert oracle.f32_to_fp8e4m3(float("nan")) & 0x7F == 0x7F
    for c in range(0x7F):                             # every finite code decodes and re-encodes to itself
        v = oracle.fp8e4m3_to_f64(c)
        assert oracle.f32_to_fp8e4m3(v) == c
        assert oracle.f32_to_fp8e4m3(-v) == (c | 0x80)


def _batch(T=37, Hkv=2, d=16, NB=11, bs=16, seed=3):
    g = torch.Generator().manual_seed(seed)
    key = torch.randn(T, Hkv, d, generator=g).to(torch.bfloat16)
    value = torch.randn(T, Hkv, d, generator=g).to(torch.bfloat16)
    slots = torch.randperm(NB * bs, generator=g)[:T].to(torch.int32)
    return key, value, slots


def test_bf16_write_then_gather_returns_the_rows():
    # Invariant through the oracle's independent gather: a sequence whose block
    # table lists the blocks in order reads back exactly the rows written to
    # its positions.
    T, Hkv, d, NB, bs = 40, 2, 16, 6, 16
    key, value, _ = _batch(T, Hkv, d, NB, bs)
    g = torch.Generator().manual_seed(9)
    blocks = torch.randperm(NB, generator=g)[:3].to(torch.int32)   # a 3-block sequence, 40 tokens
    slots = (blocks[torch.arange(T) // bs] * bs + torch.arange(T) % bs).to(torch.int32)
    kc = torch.zeros(NB, bs, Hkv, d, dtype=torch.bfloat16)
    vc = torch.zeros_like(kc)
    k2, v2 = oracle.cache_write(key, value, slots, kc, vc)
    bt = torch.full((1, 4), -1, dtype=torch.int32)
    bt[0, :3] = blocks
    kd, vd = oracle.gather(torch.from_numpy(k2.view(np.int16)).view(torch.bfloat16),
                           torch.from_numpy(v2.view(np.int16)).view(torch.bfloat16),
                           bt, torch.tensor([T], dtype=torch.int32))
    assert np.array_equal(kd[0, :T].view(np.uint16), key.view(torch.int16).numpy().view(np.uint16))
    assert np.array_equal(vd[0, :T].view(np.uint16), value.view(torch.int16).numpy().view(np.uint16))


def test_skipped_slots_and_untouched_cache():
    key, value, slots = _batch()
    slots[::5] = -1                          # padding tokens
    slots[3] = 11 * 16                       # one past the cache: skipped
    kc = torch.randn(11, 16, 2, 16).to(torch.bfloat16)
    vc = torch.randn(11, 16, 2, 16).to(torch.bfloat16)
    k2, v2 = oracle.cache_write(key, value, slots, kc, vc)
    written = np.zeros(11 * 16, dtype=bool)
    for t, s in enumerate(slots.tolist()):
        if 0 <= s < 11 * 16:
            written[s] = True
            assert np.array_equal(k2.reshape(-1, 2, 16)[s], key[t].view(torch.int16).numpy().view(np.uint16))
    kb = kc.view(torch.int16).numpy().view(np.uint16).reshape(-1, 2, 16)
    assert np.array_equal(k2.reshape(-1, 2, 16)[~written], kb[~written])


def test_fp8_write_is_within_half_a_step_of_the_value():
    # Error bound: the stored code times the scale is the nearest e4m3 value
    # of value / scale, so it lies within half of the local code spacing.
    key, value, slots = _batch(seed=5)
    kc = torch.zeros(11, 16, 2, 16, dtype=torch.uint8)
    vc = torch.zeros_like(kc)
    ks, vs = 0.02, 0.015
    k2, v2 = oracle.cache_write(key, value, slots, kc, vc, ks, vs)
    table = np.array([oracle.fp8e4m3_to_f64(c) for c in range(256)])
    for t, s in enumerate(slots.tolist()):
        x = (key[t].float() / ks).numpy().astype(np.float64)
        got = table[k2.reshape(-1, 2, 16)[s]]
        xa = np.clip(np.abs(x), 0, 448)
        step = np.where(xa < 2.0 ** -6, 2.0 ** -9, 2.0 ** (np.floor(np.log2(np.maximum(xa, 2.0 ** -6))) - 3))
        assert np.all(np.abs(np.abs(got) - xa) <= step / 2 + 1e-12)
        ref = torch.from_numpy((key[t].float() / ks).numpy()).clamp(-448, 448).to(FP8).view(torch.uint8).numpy()
        assert np.array_equal(k2.reshape(-1, 2, 16)[s], ref)


def test_fp8_v_half_uses_v_scale():
    # Library pin of the V branch: the stored V codes are torch's e4m3fn
    # conversion of value / v_scale (fp32 division, limited to +-448), with
    # v_scale different from k_scale, so a swapped or shared scale fails.
    key, value, slots = _batch(seed=6)
    kc = torch.zeros(11, 16, 2, 16, dtype=torch.uint8)
    vc = torch.zeros_like(kc)
    ks, vs = 0.02, 0.0037
    k2, v2 = oracle.cache_write(key, value, slots, kc, vc, ks, vs)
    for t, s in enumerate(slots.tolist()):
        vref = (value[t].float() / vs).clamp(-448, 448).to(FP8).view(torch.uint8).numpy()
        kref = (key[t].float() / ks).clamp(-448, 448).to(FP8).view(torch.uint8).numpy()
        assert np.array_equal(v2.reshape(-1, 2, 16)[s], vref)
        assert np.array_equal(k2.reshape(-1, 2, 16)[s], kref)
    # large values saturate to the largest finite code on the V side too
    big = value.clone()
    big[0] = 1000.0
    _, v3 = oracle.cache_write(key, big, slots, kc, vc, ks, vs)
    row = v3.reshape(-1, 2, 16)[int(slots[0])]
    assert np.all((row & 0x7F) == 0x7E)


def test_duplicate_slots_are_rejected():
    # Every new token owns its own slot (Sec. 4.3); a mapping that names one
    # slot twice has no single result and is refused.  Skipped (negative or
    # out-of-range) slots may repeat.
    key, value, slots = _batch(T=8)
    kc = torch.zeros(11, 16, 2, 16).to(torch.bfloat16)
    slots[5] = slots[2]
    with pytest.raises(oracle.OracleError, match="same slot"):
        oracle.cache_write(key, value, slots, kc, kc.clone())
    slots[5] = -1
    slots[6] = -1
    slots[7] = 11 * 16 + 3
    oracle.cache_write(key, value, slots, kc, kc.clone())
