"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check
that the pins catch every one of them."""
import os
import subprocess

import pytest

import oracle_pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                   "sp_attn_oracle.c")

# (name, original text, mutated text)
MUTANTS = [
    ("visible_off_by_one", "int64_t visible = (int64_t)prefix_lens[b] + i + 1;",
     "int64_t visible = (int64_t)prefix_lens[b] + i;"),
    ("top_left_alignment", "int64_t visible = (int64_t)prefix_lens[b] + i + 1;",
     "int64_t visible = i + 1;"),
    ("gqa_modulo_mapping", "h / G != g", "h % Hkv != g"),
    ("scale_dropped", "double sigma = sm_scale > 0.0 ? sm_scale : 1.0 / sqrt((double)d);",
     "double sigma = sm_scale > 0.0 ? sm_scale : 1.0;"),
    ("lse_without_max", "*lse = m + log(l);", "*lse = log(l);"),
    ("exp_without_max", "double w = exp(scores[j] - m);", "double w = exp(scores[j]);"),
    ("no_normalisation", "o[e] /= l;", "o[e] /= 1.0;"),
    ("wrong_slot", "return page * page_size + t % page_size;",
     "return page * page_size + (page_size - 1 - t % page_size);"),
    ("v_layout_untransposed", "return ((page * Hkv + g) * d + e) * page_size + slot;",
     "return ((page * Hkv + g) * page_size + slot) * d + e;"),
    ("transposed_k", "dot += qrow[e] * K[j * d + e];", "dot += qrow[e] * K[e * n + j];"),
    ("k_v_swapped", "krow[e] = c->k_pool[k_index(page, slot, g, e, c->Hkv, c->page_size, c->d)];\n        vrow[e] = c->v_pool[v_index(page, slot, g, e, c->Hkv, c->page_size, c->d)];",
     "krow[e] = c->v_pool[k_index(page, slot, g, e, c->Hkv, c->page_size, c->d)];\n        vrow[e] = c->k_pool[v_index(page, slot, g, e, c->Hkv, c->page_size, c->d)];"),
    ("append_ignores_seq_offset", "int64_t src = ((off + i) * Hkv + g) * d + e;",
     "int64_t src = (i * Hkv + g) * d + e;"),
    ("gather_misses_last_token", "int64_t n = (int64_t)prefix_lens[b] + suffix_lens[b];\n        for (int64_t t = 0; t < n; ++t) {\n            if",
     "int64_t n = (int64_t)prefix_lens[b] + suffix_lens[b];\n        for (int64_t t = 0; t + 1 < n; ++t) {\n            if"),
    ("gather_head_mixup", "int64_t dst = ((off + t) * Hkv + g) * d + e;",
     "int64_t dst = ((off + t) * Hkv + (Hkv - 1 - g)) * d + e;"),
    ("sign_flip_dot", "scores[j] = sigma * dot;", "scores[j] = -sigma * dot;"),
    # Row-subset mode: the row list ignored, and output k written to slot r.
    # The pin's first list is a permutation of every row, so the second
    # mutant stays in bounds until that list's check fails.
    ("rows_list_ignored", "int64_t r = rows ? rows[k] : k;", "int64_t r = k;"),
    ("rows_output_slot", "o + k * d, lse + k);", "o + r * d, lse + r);"),
]


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("mutants")


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(name, old, new, mutant_dir):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new)
    c_path = mutant_dir / f"{name}.c"
    so_path = mutant_dir / f"{name}.so"
    c_path.write_text(mutated)
    subprocess.run(["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", str(so_path),
                    str(c_path), "-lm"], check=True)
    failed = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(str(so_path))
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"no pin caught mutant {name}"
