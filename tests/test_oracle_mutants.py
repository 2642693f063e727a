"""The oracle's pins catch plausible mistakes in it (CPU only).

Each mutant is a copy of the C oracle with one planted mistake (a wrong index,
a dropped term, a flipped sign, a transposed operand), compiled to a library of
its own.  The pins of test_oracle_pins.py run against it, and at least one of
them must fail.  An unmodified copy built the same way passes every pin, so a
failure is the mistake's doing.
"""

import os
import subprocess

import pytest

import oracle
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "paged_attention_ref.c")

# name -> (text, replacement, which occurrence of the text, 0-based)
MUTANTS = {
    "gqa_head_modulo": ("const int g = h / G;", "const int g = h % L->num_kv_heads;", 0),
    "scale_dropped": ("s[t] = scale * acc;", "s[t] = acc;", 0),
    "weights_not_normalised": ("const double w = s[t] / Z;", "const double w = s[t];", 0),
    "softmax_sign": ("s[t] = exp(s[t] - m);", "s[t] = exp(m - s[t]);", 0),
    "k_tile_token_major": ("idx = ((long)(d / x) * L->page_size + t) * x + (d % x);",
                           "idx = (long)t * L->head_dim + d;", 0),
    "v_tile_token_major": ("idx = (long)d * L->page_size + t;", "idx = (long)t * L->head_dim + d;", 0),
    "v_read_from_k_tile": ("oracle_elem_offset(L, page, layer, g, 1, t % P, i)",
                           "oracle_elem_offset(L, page, layer, g, 0, t % P, i)", 0),
    "v_slot_off_by_one": ("oracle_elem_offset(L, page, layer, g, 1, t % P, i)",
                          "oracle_elem_offset(L, page, layer, g, 1, (t + 1) % P, i)", 0),
    "v_page_of_next_token": ("page_table[(long)b * pt_stride + t / P]",
                             "page_table[(long)b * pt_stride + (t + 1) / P]", 1),
    "layer_ignored": ("((long)(layer * L->num_kv_heads + head) * 2 + kind)", "((long)head * 2 + kind)", 0),
    "kv_tiles_swapped": ("((long)(layer * L->num_kv_heads + head) * 2 + kind)",
                         "((long)(layer * L->num_kv_heads + head) * 2 + (1 - kind))", 0),
    "bf16_low_half": ("uint32_t bits = (uint32_t)h << 16;", "uint32_t bits = (uint32_t)h;", 0),
    "query_of_wrong_row": ("qb + ((long)row * D + i) * e", "qb + ((long)b * D + i) * e", 0),
    "last_token_dropped": ("for (int t = 0; t < Lb && !bad; ++t) {", "for (int t = 0; t < Lb - 1 && !bad; ++t) {", 0),
}


def _battery():
    """Every pin of test_oracle_pins.py, as (name, call)."""
    calls = []
    for dtype in (oracle.BF16, oracle.F32):
        for d in (64, 128):
            for hkv, g in ((1, 1), (1, 4), (2, 2), (4, 8)):
                calls.append(("p1 %d %d %d %d" % (dtype, d, hkv, g),
                              lambda a=(dtype, d, hkv, g): pins.test_p1_brute_force_dense(*a)))
        calls.append(("p2 %d" % dtype, lambda a=dtype: pins.test_p2_single_token_returns_v(a)))
        calls.append(("p4 %d" % dtype, lambda a=dtype: pins.test_p4_weights_sum_to_one(a)))
        calls.append(("p6 %d" % dtype, lambda a=dtype: pins.test_p6_poison_outside_valid_tokens(a)))
    for where in ("first", "page_end", "page_start", "last", "random"):
        calls.append(("p5 " + where, lambda a=where: pins.test_p5_needle(a)))
    for name in ("test_p1_other_layers_untouched", "test_p3_identical_keys_give_mean_of_v",
                 "test_two_token_closed_form", "test_p9_key_shift_invariance",
                 "test_zero_length_gives_zero_and_bad_page_rejected", "test_layout_offsets_hand_computed",
                 "test_pack_pool_matches_accessor", "test_p12_paper_shape_numbers"):
        calls.append((name, getattr(pins, name)))
    return calls


def _build(tmp_path, name, text=None, repl=None, nth=0):
    src = open(SRC).read()
    if text is not None:
        at = -1
        for _ in range(nth + 1):
            at = src.index(text, at + 1)
        src = src[:at] + repl + src[at + len(text):]
    c = tmp_path / (name + ".c")
    c.write_text(src)
    so = tmp_path / (name + ".so")
    subprocess.check_call(["gcc", "-O1", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-o", str(so), str(c), "-lm"])
    return oracle.load_library(str(so))


def _failing_pins(monkeypatch, lib):
    monkeypatch.setattr(oracle, "_lib", lib)
    failed = []
    for name, call in _battery():
        try:
            call()
        except Exception:  # an assertion, or the oracle refusing its input
            failed.append(name)
    return failed


def test_unmodified_copy_passes_every_pin(tmp_path, monkeypatch):
    assert _failing_pins(monkeypatch, _build(tmp_path, "control")) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(tmp_path, monkeypatch, name):
    text, repl, nth = MUTANTS[name]
    failed = _failing_pins(monkeypatch, _build(tmp_path, name, text, repl, nth))
    assert failed, "mutant %s passes every pin" % name
