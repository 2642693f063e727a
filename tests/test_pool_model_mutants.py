"""The pool model's pins catch plausible mistakes in it (CPU only).

Each mutant is the oracle's pool model with one planted mistake in its policy
or bookkeeping, loaded as a module of its own; the pins of test_pool_model.py
run against it and at least one must fail.  The unmodified source loaded the
same way passes every pin.
"""

import sys
import types

import pytest

import oracle.pool_model as real
import test_pool_model as pins

SRC = real.__file__

# name -> [(text, replacement), ...]
MUTANTS = {
    "allocation_highest_first": [("return sorted(free)[:n]", "return sorted(free, reverse=True)[:n]")],
    "lru_newest_first": [("for _stamp, sid in order:", "for _stamp, sid in reversed(order):")],
    "resume_evicts_its_own_pages": [("self._plan(need, exclude=set(sids), fresh_spill=False)",
                                     "self._plan(need, exclude=set(), fresh_spill=False)")],
    "resume_refetches_resident_pages": [("need += sum(1 for p in s.hot if p < 0)", "need += len(s.hot)")],
    "evict_rewrites_valid_copies": [
        ("dirty += sum(1 for c in s.cold if c < 0)", "dirty += len(s.cold)"),
        ("                if s.cold[i] < 0:\n                    c = next(fresh)",
         "                if True:\n                    if s.cold[i] >= 0:\n"
         "                        self._release_cold(s.cold[i])\n                    c = next(fresh)")],
    "written_page_keeps_its_cold_copy": [
        ("            if s.hot[i] >= 0 and s.cold[i] >= 0:\n                self._release_cold(s.cold[i])\n"
         "                s.cold[i] = -1", "            pass")],
    "extend_keeps_tail_cold_copy": [
        ("        if tail >= 0 and s.hot[tail] >= 0 and s.cold[tail] >= 0:", "        if False:")],
    "extend_writes_shared_spilled_tail": [
        ("        if tail >= 0 and s.hot[tail] < 0 and self.cold_ref[s.cold[tail]] > 1:", "        if False:")],
    "destroy_keeps_cold_references": [
        ("        for c in s.cold:\n            if c >= 0:\n                self._release_cold(c)\n"
         "        self.sessions[sid] = _Session()", "        self.sessions[sid] = _Session()")],
    "pause_keeps_old_lru_stamp": [("        s.state = PAUSED\n        s.stamp = self._tick()\n\n    def evict_pages",
                                   "        s.state = PAUSED\n\n    def evict_pages")],
}


def _load(name, edits):
    src = open(SRC).read()
    for text, repl in edits:
        assert src.count(text) >= 1, "mutation text not found: %r" % text[:60]
        src = src.replace(text, repl, 1)
    mod = types.ModuleType("pool_model_" + name)
    sys.modules[mod.__name__] = mod       # dataclasses look their module up while decorating
    try:
        exec(compile(src, "<%s>" % name, "exec"), mod.__dict__)
    finally:
        del sys.modules[mod.__name__]
    return mod


def _battery():
    calls = []
    for name in sorted(dir(pins)):
        if not name.startswith("test_"):
            continue
        fn = getattr(pins, name)
        if name == "test_spill_invariants_on_random_sequences":
            calls += [(name + str(s), lambda f=fn, s=s: f(s)) for s in range(3)]
        else:
            calls.append((name, fn))
    return calls


def _failing_pins(monkeypatch, mod):
    monkeypatch.setattr(pins, "PoolModel", mod.PoolModel)
    monkeypatch.setattr(pins, "ModelError", mod.ModelError)
    failed = []
    for name, call in _battery():
        try:
            call()
        except (Exception, pytest.fail.Exception):   # pytest.raises reports DID NOT RAISE this way
            failed.append(name)
    return failed


def test_unmodified_source_passes_every_pin(monkeypatch):
    assert _failing_pins(monkeypatch, _load("control", [])) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(monkeypatch, name):
    failed = _failing_pins(monkeypatch, _load(name, MUTANTS[name]))
    assert failed, "mutant %s passes every pin" % name
