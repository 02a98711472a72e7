"""The oracle's pins must be strong enough to catch plausible mistakes.

Each case plants one mistake in a temporary copy of ``oracle/pa_oracle.c``
(a dropped term, a wrong sign or index, a transposed operand, a wrong GQA
map, a missing scale ...), builds it with gcc into a temporary library and
runs the pin suite against it in a child process (``PA_ORACLE_LIB``).  The
suite must fail for every mutant.  The committed oracle is never modified.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "pa_oracle.c")
PINS = [os.path.join(ROOT, "tests", "test_oracle_pins.py"),
        os.path.join(ROOT, "tests", "test_oracle_cache_write.py")]

# (name, original text, planted text, occurrences replaced)
MUTANTS = [
    ("gqa_map_modulo", "int64_t g = h / (P->Hq / P->Hkv);", "int64_t g = h % P->Hkv;", 2),
    ("diagonal_dropped", "row_attend(P, i, t, h, c + j + 1,", "row_attend(P, i, t, h, c + j + (j > 0),", 1),
    ("top_left_causal", "row_attend(P, i, t, h, c + j + 1,", "row_attend(P, i, t, h, j + 1 + (c > 0),", 1),
    ("exp_sign_flipped", "s[p] = exp(s[p] - m); /* s now holds w_p */",
     "s[p] = exp(m - s[p]); /* s now holds w_p */", 1),
    ("cache_index_transposed", "((blk * P->bs + slot) * P->Hkv + g) * P->d + x",
     "((blk * P->Hkv + g) * P->bs + slot) * P->d + x", 1),
    ("scale_missing", "s[p] = P->scale * acc_get(&a);", "s[p] = acc_get(&a);", 1),
    ("fp8_bias_off_by_one", "ldexp(1.0 + m / 8.0, e - 7)", "ldexp(1.0 + m / 8.0, e - 8)", 1),
    ("fp8_subnormal_wrong", "ldexp((double)m, -9)", "ldexp((double)m, -10)", 1),
    ("bf16_shift_wrong", "((uint32_t)bits) << 16", "((uint32_t)bits) << 15", 1),
    ("v_scale_missing", "kv_at(P, P->v_cache, P->v_scale,", "kv_at(P, P->v_cache, 1.0,", 1),
    ("k_scale_on_v", "kv_at(P, P->v_cache, P->v_scale,", "kv_at(P, P->v_cache, P->k_scale,", 1),
    ("normalisation_missing", "out[x] = acc_get(&o[x]) / lsum;", "out[x] = acc_get(&o[x]);", 1),
    ("lse_not_logged", "*lse = m + log(lsum);", "*lse = m + lsum;", 1),
    ("table_row_stride", "P->block_table[i * P->MB + p / P->bs]", "P->block_table[i * P->bs + p / P->bs]", 2),
    ("slot_index", "int64_t slot = p % P->bs;", "int64_t slot = (p + 1) % P->bs;", 1),
    ("v_uses_k_cache", "acc_add(&o[x], s[p] * kv_at(P, P->v_cache, P->v_scale,",
     "acc_add(&o[x], s[p] * kv_at(P, P->k_cache, P->v_scale,", 1),
    ("q_head_transposed", "P->q + (t * P->Hq + h) * P->d", "P->q + (h * P->T + t) * P->d", 1),
    ("merge_weight_dropped", "acc_add(&den, exp(m[k] - M) * l[k]);", "acc_add(&den, l[k]);", 1),
    ("merge_numerator_unscaled", "acc_add(&num, exp(m[k] - M) * acc[k * d + x]);",
     "acc_add(&num, acc[k * d + x]);", 1),
    ("segment_sum_unshifted", "for (int64_t p = k0; p < k1; ++p) acc_add(&l, exp(s[p] - m));",
     "for (int64_t p = k0; p < k1; ++p) acc_add(&l, exp(s[p]));", 1),
    ("segment_last_clamp", "(k + 1) * tps < n_tiles ? (k + 1) * tps : n_tiles",
     "(k + 1) * tps", 1),
    ("validate_block_upper", "if (blk < 0 || blk >= P->NB) return fail(\"block id out of range\", i, blk);",
     "if (blk < 0) return fail(\"block id out of range\", i, blk);", 1),
    ("gather_slot", "int64_t src = ((int64_t)blk * block_size + p % block_size) * row;",
     "int64_t src = ((int64_t)blk * block_size + p / block_size) * row;", 1),
    ("cache_write_v_uses_k_scale", "float vf = (float)pa_oracle_bf16_to_f64(vb) / v_scale;",
     "float vf = (float)pa_oracle_bf16_to_f64(vb) / k_scale;", 1),
    ("cache_write_v_unscaled", "float vf = (float)pa_oracle_bf16_to_f64(vb) / v_scale;",
     "float vf = (float)pa_oracle_bf16_to_f64(vb);", 1),
    ("cache_write_duplicates_accepted", "if (slot_mapping[u] == slot) return fail(",
     "if (slot_mapping[u] == slot && 0) return fail(", 1),
    ("fp8_encoder_ties_to_odd", "(err == best_err && (c & 1) == 0)", "(err == best_err && (c & 1) == 1)", 1),
]


def _plant(src, old, new, count):
    assert src.count(old) == count, (old, src.count(old))
    return src.replace(old, new)


def _run_mutant(tmp, name, old, new, count):
    src = _plant(open(SRC).read(), old, new, count)
    c = os.path.join(tmp, f"{name}.c")
    so = os.path.join(tmp, f"lib{name}.so")
    open(c, "w").write(src)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-o", so, c,
                           "-lpthread", "-lm"])
    env = dict(os.environ, PA_ORACLE_LIB=so)
    r = subprocess.run([sys.executable, "-m", "pytest", *PINS, "-x", "-q", "-p", "no:cacheprovider"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    return name, r.returncode, r.stdout[-400:]


def test_unmodified_copy_passes_the_pins(tmp_path):
    src = open(SRC).read()
    _, rc, tail = _run_mutant(str(tmp_path), "identity", src[:40], src[:40], 1)
    assert rc == 0, tail


def test_every_planted_mistake_fails_a_pin(tmp_path):
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda m: _run_mutant(str(tmp_path), *m), MUTANTS))
    survivors = [(name, tail) for name, rc, tail in results if rc == 0]
    assert not survivors, survivors
    # A mutant must fail on an assertion, not on a crash or collection error.
    for name, rc, tail in results:
        assert rc == 1, (name, rc, tail)
