"""The CPU oracle against its pins (hand-worked examples, closed forms, brute
force, library routines and the paper's invariants)."""
import pytest

import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


@pytest.mark.parametrize("name,seeds", [("tiny", range(20)), ("int8", (0,)), ("paper1m", (0, 1))])
def test_planted_chunks_always_kept(name, seeds):
    P.pin_planted_selected(name, seeds)
