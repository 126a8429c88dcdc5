"""Mutation check of the reference-selection pins: each case plants one
plausible mistake in a copy of oracle/spans.py and runs the pins against it;
at least one pin must fail."""
from __future__ import annotations

import importlib.util
import os

import pytest

import oracle.spans as spans_mod
from tests import test_oracle_spans as pins

MUTANTS = [
    ("recency_prefers_older", "if best is None or cand > best:", "if best is None or cand[0] > best[0]:"),
    ("no_occurrence_limit", "            if len(lst) > keep:\n", "            if False:\n"),
    ("drops_newest_not_oldest", "lst.pop(0)", "lst.pop()"),
    ("scan_steps_by_one", "        i += L\n", "        i += 1\n"),
    ("no_forward_extension", "L += 1", "break"),
    ("older_position_wins_inside_a_request", "cand = (L, r, j)", "cand = (L, r, -j)"),
    ("rows_from_request_start", "out[i + o] = history[r][1] + j + o", "out[i + o] = history[r][1] + o"),
]
PINS = [getattr(pins, n) for n in dir(pins) if n.startswith("test_")]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(tmp_path, monkeypatch, name, old, new):
    src = open(spans_mod.__file__).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    path = tmp_path / "spans_mutant.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("spans_mutant", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    monkeypatch.setattr(pins, "select_spans", mod.select_spans)
    caught = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, IndexError, KeyError):
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutant {name}"
