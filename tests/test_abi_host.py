"""Host-side tests of the C ABI: the library loads and exports every function
declared in include/pa.h, the header is plain C whose struct layout matches
the binding, and the launch planner's decisions (no GPU needed)."""
import ctypes
import itertools
import os
import re
import subprocess

import pytest
import torch

from paper_2511_11581_amd import pa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pa.h")
GOLDEN = os.path.join(ROOT, "tests", "golden")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pa_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = pa.load_library()
    declared = header_functions()
    assert sorted(pa.EXPORTS) == declared
    for name in declared:
        assert hasattr(lib, name), name


def test_header_is_plain_c_and_matches_binding_layout(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(r'''
#include <stddef.h>
#include <stdio.h>
#include "pa.h"
int main(void) {
  printf("%zu %zu %zu %zu\n", sizeof(pa_tensor), offsetof(pa_tensor, shape), offsetof(pa_tensor, stride), sizeof(pa_config));
  printf("%zu %zu %zu %zu\n", offsetof(pa_config, workspace), offsetof(pa_config, workspace_bytes), sizeof(pa_plan_info), offsetof(pa_plan_info, decode_grid));
  printf("%zu\n", offsetof(pa_plan_info, workspace_bytes));
  return 0;
}
''')
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(HEADER),
                           str(src), "-o", str(exe)])
    vals = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    expect = [ctypes.sizeof(pa.pa_tensor), pa.pa_tensor.shape.offset, pa.pa_tensor.stride.offset,
              ctypes.sizeof(pa.pa_config), pa.pa_config.workspace.offset,
              pa.pa_config.workspace_bytes.offset, ctypes.sizeof(pa.pa_plan_info),
              pa.pa_plan_info.decode_grid.offset, pa.pa_plan_info.workspace_bytes.offset]
    assert vals == expect


def cfg(Hq=32, Hkv=8, d=128, bs=16, kv=pa.PA_DTYPE_BF16):
    return pa.make_config(Hq, Hkv, d, bs, kv)


def plan(c, cus=256, T=1, S=1, MB=1):
    return pa.pa_plan(None, c, cus, T, S, MB)


def segment_ranges(n_keys, seg_len, tile):
    """The decode kernel's partition of one row: segment k covers keys
    [k * seg_len, min((k + 1) * seg_len, n_keys)), returned in tiles."""
    out = []
    k = 0
    while k * seg_len < n_keys:
        a, b = k * seg_len, min((k + 1) * seg_len, n_keys)
        out.append((a // tile, -(-b // tile)))
        k += 1
    return out


def test_plan_reproduces_the_papers_partition_example():
    # Fig. 4 (Sec. 4.5): 32 tiles distributed over 4 segments of 8 tiles.
    line = [x for x in open(os.path.join(GOLDEN, "fig4_segments.txt")).read().splitlines()
            if x and not x.startswith("#")][0]
    head, tail = line.split("|")
    n_tiles, tps = (int(x) for x in head.split())
    expect = [tuple(int(x) for x in part.split()) for part in tail.split(";")]
    p = plan(cfg(), cus=256, T=64, S=64, MB=n_tiles * 32 // 16)
    assert p["decode_tile"] == 32
    assert p["segment_len"] == tps * p["decode_tile"]
    assert p["max_splits"] == len(expect)
    assert segment_ranges(n_tiles * p["decode_tile"], p["segment_len"], p["decode_tile"]) == expect


def test_plan_decode_splits_fill_the_gpu():
    # Llama-3-8B decode shape: 64 sequences up to 8193 tokens.
    p = plan(cfg(), cus=256, T=64, S=64, MB=513)
    assert p["decode_launch"] == 1 and p["merge_launch"] == 1
    assert p["segment_len"] % (p["decode_tile"] * p["decode_waves"]) == 0
    assert p["max_splits"] * p["segment_len"] >= 513 * 16
    assert 64 * 8 * p["max_splits"] >= 8 * 256 * 0.9
    assert p["decode_grid"] == [p["max_splits"], 64, 8]
    # 70B-style long decode: 16 sequences, 8 kv heads, up to 131088 tokens.
    p = plan(cfg(64, 8), cus=256, T=16, S=16, MB=8193)
    assert p["max_splits"] >= 16 and p["segment_len"] >= 256


def test_plan_short_batches_do_not_split():
    p = plan(cfg(8, 2, 64), cus=256, T=4, S=4, MB=16)
    assert p["max_splits"] == 1 and p["merge_launch"] == 0
    assert p["workspace_bytes"] < 4096  # no split partials; header + prefill work list only


def test_plan_prefill_grid_bounds_the_q_blocks():
    p = plan(cfg(), cus=256, T=6589, S=4, MB=188)
    assert p["prefill_launch"] == 1
    assert p["block_m"] == 128 and p["block_q"] == 32
    # sum ceil(q_i / BLOCK_Q) <= ceil(T / BLOCK_Q) + S
    qs = [2048, 1024, 3000, 517]
    need = sum(-(-q // 32) for q in qs)
    assert p["prefill_grid"][0] >= need * 8
    p1 = plan(cfg(), T=1, S=1, MB=4)
    assert p1["prefill_launch"] == 0


@pytest.mark.parametrize("Hq,Hkv,d,bs,kv,status", [
    (32, 8, 128, 16, pa.PA_DTYPE_BF16, pa.PA_OK),
    (12, 4, 128, 16, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),   # G = 3
    (64, 2, 128, 16, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),   # G = 32
    (32, 8, 96, 16, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),
    (32, 8, 128, 8, pa.PA_DTYPE_BF16, pa.PA_ERR_UNSUPPORTED),
    (30, 8, 128, 16, pa.PA_DTYPE_BF16, pa.PA_ERR_INVALID_ARG),
    (32, 8, 128, 16, pa.PA_DTYPE_F32, pa.PA_ERR_UNSUPPORTED),
    (32, 8, 128, 32, pa.PA_DTYPE_FP8_E4M3, pa.PA_OK),
])
def test_config_validation(Hq, Hkv, d, bs, kv, status):
    c = cfg(Hq, Hkv, d, bs, kv)
    info = pa.pa_plan_info()
    st = pa.load_library().pa_plan(None, ctypes.byref(c), 256, 10, 2, 4, ctypes.byref(info))
    assert st == status, pa.pa_last_error()
    if st != pa.PA_OK:
        assert pa.pa_last_error()


def test_workspace_bound_covers_every_plan():
    for Hq, Hkv, d in [(32, 8, 128), (8, 2, 64), (64, 8, 128), (16, 16, 128)]:
        c = cfg(Hq, Hkv, d)
        for S_max, MB_max in [(1, 1), (4, 16), (64, 513), (16, 8193), (128, 1025), (300, 40)]:
            bound = pa.pa_workspace_bytes(c, 10 * S_max, S_max, MB_max)
            for S, MB, cus in itertools.product(sorted({1, 2, 3, S_max // 2 or 1, S_max}),
                                                sorted({1, MB_max // 3 or 1, MB_max}),
                                                (1, 80, 256)):
                p = plan(c, cus=cus, T=S, S=S, MB=MB)
                assert p["workspace_bytes"] <= bound, (Hq, Hkv, d, S, MB, cus)


def test_create_without_a_gpu_reports_a_device_error():
    if torch.cuda.is_available():
        pytest.skip("a GPU is visible")
    c = cfg()
    h = ctypes.c_void_p()
    st = pa.load_library().pa_create(ctypes.byref(c), ctypes.byref(h))
    assert st == pa.PA_ERR_DEVICE
    assert "hip" in pa.pa_last_error().lower()
