"""The work-split oracle's pins catch plausible mistakes in it (CPU only).

Each mutant is oracle/partition.py with one planted mistake, loaded as a module
of its own; the pins of test_partition_oracle.py run against it and at least
one must fail.  The unmodified source loaded the same way passes them all.
"""

import sys
import types

import pytest

import oracle.partition as real
import test_partition_oracle as pins

# name -> [(text, replacement)]
MUTANTS = {
    "bounds_rounded_up": [("bounds = [(k * T) // workers for k in range(workers + 1)]",
                           "bounds = [-((-k * T) // workers) for k in range(workers + 1)]")],
    "slot_without_segment": [("out.append(((k + s) * L + w,", "out.append(((k) * L + w,")],
    "slot_segment_not_scaled": [("out.append(((k + s) * L + w,", "out.append((k * L + s + w,")],
    "head_of_wave_reversed": [("k * L + w, b, hg * L + w,", "k * L + w, b, hg * L + (L - 1 - w),")],
    "units_ordered_page_then_head": [
        ("        for hg in range(groups):\n            for i in range(n):\n                units.append((b, hg, i))",
         "        for i in range(n):\n            for hg in range(groups):\n                units.append((b, hg, i))")],
    "group_of_four_always": [("return 4 if num_kv_heads % 4 == 0 and waves % 4 == 0 else 1",
                              "return 4 if num_kv_heads % 4 == 0 else 1")],
    "group_width_one_always": [("return 4 if num_kv_heads % 4 == 0 and waves % 4 == 0 else 1", "return 1")],
    "empty_rows_get_a_page": [("if int(length) > 0 else 0", "if int(length) > 0 else 1")],
    "page_end_exclusive_off_by_one": [("i0, units[v - 1][2] + 1))", "i0, units[v - 1][2]))")],
}


def _load(name, edits):
    src = open(real.__file__).read()
    for text, repl in edits:
        assert text in src, "mutation text not found: %r" % text[:60]
        src = src.replace(text, repl, 1)
    mod = types.ModuleType("partition_" + name)
    sys.modules[mod.__name__] = mod
    try:
        exec(compile(src, "<%s>" % name, "exec"), mod.__dict__)
    finally:
        del sys.modules[mod.__name__]
    return mod


def _battery():
    calls = [("group_width_rule", pins.test_group_width_rule),
             ("closed_form", pins.test_closed_form_matches_enumeration),
             ("small_examples", pins.test_slot_table_small_examples)]
    calls += [("cover_%d" % s, lambda s=s: pins.test_exact_cover_and_balance(s)) for s in range(10)]
    return calls


def _failing_pins(monkeypatch, mod):
    monkeypatch.setattr(pins, "partition", mod)
    failed = []
    for name, call in _battery():
        try:
            call()
        except Exception:
            failed.append(name)
    return failed


def test_unmodified_source_passes_every_pin(monkeypatch):
    assert _failing_pins(monkeypatch, _load("control", [])) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(monkeypatch, name):
    failed = _failing_pins(monkeypatch, _load(name, MUTANTS[name]))
    assert failed, "mutant %s passes every pin" % name
