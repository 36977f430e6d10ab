"""The gradient oracle against autograd, brute force and a closed form, plus
planted mistakes that the pins must catch."""
import importlib.util
import os

import pytest

from oracle import backward as ob
from tests import oracle_pins
from tests.conftest import ROOT


@pytest.mark.parametrize("pin", oracle_pins.BWD_PINS, ids=lambda f: f.__name__)
def test_backward_pin(pin):
    pin(ob.attention_backward)


MUTANTS = [
    ("D from the wrong row sum", "big_d = (gh[rows] * out).sum(axis=-1, keepdims=True)",
     "big_d = (gh[rows] * out).sum(axis=0, keepdims=True)"),
    ("missing scale on dk", "dk[b, h, cols] += scale * (ds.T @ qh[rows])", "dk[b, h, cols] += (ds.T @ qh[rows])"),
    ("dv from dS instead of P", "dv[b, h, cols] += p.T @ gh[rows]", "dv[b, h, cols] += ds.T @ gh[rows]"),
    ("dq from V instead of K", "dq[b, h, rows] += scale * (ds @ kh[cols])", "dq[b, h, rows] += scale * (ds @ vh[cols])"),
    ("dP transposed operands", "dp = gh[rows] @ vh[cols].T", "dp = qh[rows] @ vh[cols].T"),
]


def _load_mutant(old, new):
    src = open(os.path.join(ROOT, "oracle", "backward.py")).read()
    assert src.count(old) == 1, old
    src = src.replace(old, new).replace("from .attention import", "from oracle.attention import")
    spec = importlib.util.spec_from_loader("oracle_backward_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src, "oracle_backward_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_backward_pins_catch_planted_mistake(name, old, new):
    mutant = _load_mutant(old, new)
    failures = 0
    for pin in oracle_pins.BWD_PINS:
        try:
            pin(mutant.attention_backward)
        except Exception:
            failures += 1
    assert failures > 0, f"no pin caught: {name}"
