"""The gradient oracle against autograd, brute force and a closed form, plus
planted mistakes that the pins must catch."""
import importlib.util
import os

import numpy as np
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


def test_rows_variant_matches_full_gradients():
    """attention_backward_rows is the same computation restricted to chosen rows: it
    must agree with the pinned attention_backward at every row, per-head masks, empty
    rows and columns and several query chunks included."""
    rng = np.random.default_rng(23)
    B, H, F, T, d = 2, 2, 4, 7, 5
    q, k, v, g = (rng.standard_normal((B, H, F * T, d)) for _ in range(4))
    masks = (rng.random((H, F, F)) < 0.5).astype(np.uint8)
    masks[0, 1, :] = 0
    masks[1, :, 2] = 0
    masks[1, 3, :] = 1
    full = ob.attention_backward(q, k, v, g, masks, T, 0.4)
    bb, hh, ss = np.meshgrid(np.arange(B), np.arange(H), np.arange(F * T), indexing="ij")
    bb, hh, ss = bb.ravel(), hh.ravel(), ss.ravel()
    dq, dk, dv = ob.attention_backward_rows(q, k, v, g, masks, T, 0.4, bb, hh, ss, bb, hh, ss, chunk=3)
    for got, ref in zip((dq, dk, dv), full):
        assert np.max(np.abs(got - ref[bb, hh, ss])) < 1e-12
