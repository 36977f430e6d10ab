"""The MM-DiT oracle against SDPA with the token mask, dense attention, brute force and
invariants, plus planted mistakes that the pins must catch."""
import importlib.util
import os

import numpy as np
import pytest

from oracle import attention as oa
from oracle import mmdit as om
from tests import oracle_pins
from tests.conftest import ROOT


@pytest.mark.parametrize("pin", oracle_pins.MMDIT_PINS, ids=lambda f: f.__name__)
def test_mmdit_pin(pin):
    pin(om.attention_mmdit)


def test_mmdit_lse_pin():
    oracle_pins.pin_mmdit_lse(om.attention_mmdit_lse)


def test_mmdit_without_text_is_the_plain_form():
    rng = np.random.default_rng(35)
    B, H, F, T, d = 1, 2, 4, 3, 5
    q, k, v = (rng.standard_normal((B, H, F * T, d)) for _ in range(3))
    masks = (rng.random((H, F, F)) < 0.5).astype(np.uint8)
    assert np.max(np.abs(om.attention_mmdit(q, k, v, masks, T, 0, 0.6) -
                         oa.attention(q, k, v, masks, T, 0.6))) < 1e-12


def test_mmdit_rows_variant_matches():
    rng = np.random.default_rng(36)
    B, H, F, T, P, d = 2, 2, 3, 4, 5, 6
    q, k, v = (rng.standard_normal((B, H, P + F * T, d)) for _ in range(3))
    masks = (rng.random((H, F, F)) < 0.5).astype(np.uint8)
    full = om.attention_mmdit(q, k, v, masks, T, P, 0.4)
    bb, hh, ss = np.meshgrid(np.arange(B), np.arange(H), np.arange(P + F * T), indexing="ij")
    rows = om.attention_mmdit_rows(q, k, v, masks, T, P, 0.4, bb.ravel(), hh.ravel(), ss.ravel())
    assert np.max(np.abs(rows - full[bb.ravel(), hh.ravel(), ss.ravel()])) < 1e-12


MUTANTS = [
    ("text queries follow mask row 0", "        return np.arange(P + F * T)",
     "        i = 0"),
    ("video queries skip the text", "    parts = [text_tokens(P)] + [video_frame_tokens",
     "    parts = [text_tokens(0)] + [video_frame_tokens"),
    ("video tokens not offset by P", "    return np.arange(P + j * T, P + (j + 1) * T)",
     "    return np.arange(j * T, (j + 1) * T)"),
]


def _load_mutant(old, new):
    src = open(os.path.join(ROOT, "oracle", "mmdit.py")).read()
    assert src.count(old) == 1, old
    src = src.replace(old, new).replace("from .attention import", "from oracle.attention import")
    spec = importlib.util.spec_from_loader("oracle_mmdit_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src, "oracle_mmdit_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mmdit_pins_catch_planted_mistake(name, old, new):
    mutant = _load_mutant(old, new)
    failures = 0
    for pin in oracle_pins.MMDIT_PINS:
        try:
            pin(mutant.attention_mmdit)
        except Exception:
            failures += 1
    assert failures > 0, f"no pin caught: {name}"


@pytest.mark.parametrize("pin", oracle_pins.MMDIT_BWD_PINS, ids=lambda f: f.__name__)
def test_mmdit_bwd_pin(pin):
    pin(om.attention_backward_mmdit)


def test_mmdit_bwd_without_text_is_the_plain_form():
    from oracle import backward as ob
    rng = np.random.default_rng(42)
    B, H, F, T, d = 1, 2, 3, 4, 5
    q, k, v, g = (rng.standard_normal((B, H, F * T, d)) for _ in range(4))
    masks = (rng.random((H, F, F)) < 0.5).astype(np.uint8)
    for a, b in zip(om.attention_backward_mmdit(q, k, v, g, masks, T, 0, 0.5),
                    ob.attention_backward(q, k, v, g, masks, T, 0.5)):
        assert np.max(np.abs(a - b)) < 1e-12


def test_mmdit_bwd_rows_variant_matches():
    rng = np.random.default_rng(43)
    B, H, F, T, P, d = 1, 2, 3, 4, 5, 6
    q, k, v, g = (rng.standard_normal((B, H, P + F * T, d)) for _ in range(4))
    masks = (rng.random((H, F, F)) < 0.5).astype(np.uint8)
    masks[1, :, 0] = 0
    full = om.attention_backward_mmdit(q, k, v, g, masks, T, P, 0.45)
    bb, hh, ss = (x.ravel() for x in np.meshgrid(np.arange(B), np.arange(H), np.arange(P + F * T), indexing="ij"))
    rows = om.attention_backward_mmdit_rows(q, k, v, g, masks, T, P, 0.45, bb, hh, ss, bb, hh, ss, chunk=3)
    for a, r in zip(rows, full):
        assert np.max(np.abs(a - r[bb, hh, ss])) < 1e-12


BWD_MUTANTS = [
    ("text keys get no dk", "                dk[b, h, cols] += scale * (ds.T @ qh[rows])",
     "                dk[b, h, cols[cols >= P]] += scale * (ds.T @ qh[rows])[cols >= P]"),
    ("delta without the text", "                ds = p * (gh[rows] @ vh[cols].T - (gh[rows] * out).sum(axis=-1, keepdims=True))",
     "                ds = p * (gh[rows] @ vh[cols].T - (gh[rows] * (p[:, P:] @ vh[cols][P:])).sum(axis=-1, keepdims=True))"),
]


@pytest.mark.parametrize("name,old,new", BWD_MUTANTS, ids=[m[0] for m in BWD_MUTANTS])
def test_mmdit_bwd_pins_catch_planted_mistake(name, old, new):
    mutant = _load_mutant(old, new)
    failures = 0
    for pin in oracle_pins.MMDIT_BWD_PINS:
        try:
            pin(mutant.attention_backward_mmdit)
        except Exception:
            failures += 1
    assert failures > 0, f"no pin caught: {name}"
