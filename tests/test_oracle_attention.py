"""Pins of the float64 attention oracle (CPU only)."""
import importlib.util
import os

import numpy as np
import pytest

import oracle.attention as oa
from tests import oracle_pins
from tests.conftest import ROOT


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(oa.attention)


def _rows_as_full(q, k, v, mask, T, scale):
    B, H, S, d = q.shape
    bb, hh, ss = np.meshgrid(np.arange(B), np.arange(H), np.arange(S), indexing="ij")
    rows = oa.attention_rows(q, k, v, mask, T, scale, bb.ravel(), hh.ravel(), ss.ravel())
    return rows.reshape(B, H, S, d)


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_rows_pin(pin):
    """The row-sampled oracle meets the same pins."""
    pin(_rows_as_full)


def test_bf16_bits_widen_exactly():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x4049, 0x7F7F, 0x0001], dtype=np.uint16)
    vals = oa.as_f64(bits)
    assert vals[0] == 1.0 and vals[1] == -1.0 and vals[2] == 0.0
    assert vals[3] == 3.140625
    assert vals[4] == float.fromhex("0x1.fep127")
    assert vals[5] == float.fromhex("0x1p-133")


def test_uint16_input_equals_float_input():
    rng = np.random.default_rng(0)
    bits = rng.integers(0x3000, 0x4000, size=(3, 1, 2, 8, 4)).astype(np.uint16)
    mask = np.array([[1, 0], [1, 1]], np.uint8)
    a = oa.attention(*bits, mask, 4, 0.5)
    b = oa.attention(*(oa.as_f64(x) for x in bits), mask, 4, 0.5)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("pin", oracle_pins.LSE_PINS, ids=lambda f: f.__name__)
def test_oracle_lse_pin(pin):
    pin(oa.attention_lse)


def test_lse_matches_attention_normaliser():
    """The same weights normalise the output: with V = e_j (one-hot columns) the output is
    the softmax itself, whose log at the max logit equals max - lse."""
    rng = np.random.default_rng(13)
    F, T, d = 3, 4, 5
    mask = np.array([[1, 1, 0], [0, 1, 1], [1, 0, 1]], np.uint8)
    q, k = rng.standard_normal((2, 1, 1, F * T, d))
    lse = oa.attention_lse(q, k, mask, T, 0.7)
    for s in range(F * T):
        kept = [t for t in range(F * T) if mask[s // T][t // T]]
        logits = [0.7 * float(q[0, 0, s] @ k[0, 0, t]) for t in kept]
        assert abs(sum(np.exp(np.array(logits) - lse[0, 0, s])) - 1.0) < 1e-12


# Planted mistakes: each mutant of the oracle source must fail at least one pin.
MUTANTS = [
    ("transposed mask", "mask[i, j]", "mask[j, i]"),
    ("dropped scale", "logits = scale * (qh[rows] @ kh[cols].T)", "logits = (qh[rows] @ kh[cols].T)"),
    ("dropped normalisation", "return (w @ vk) / z", "return (w @ vk)"),
    ("last token of each frame dropped", "np.arange(j * T, (j + 1) * T)", "np.arange(j * T, (j + 1) * T - 1)"),
    ("wrong exponent sign", "w = np.exp(logits - m)", "w = np.exp(m - logits)"),
    ("K used as V", "out[b, h, rows] = _softmax_rows_times_v(logits, vh[cols])",
     "out[b, h, rows] = _softmax_rows_times_v(logits, kh[cols])"),
    ("query rows of the wrong frame", "rows = frame_tokens(i, T)", "rows = frame_tokens((i + 1) % F, T)"),
    ("query and key swapped", "logits = scale * (qh[rows] @ kh[cols].T)", "logits = scale * (kh[rows] @ qh[cols].T)"),
    ("mask of head 0 for every head", "return mask if mask.ndim == 2 else mask[h]",
     "return mask if mask.ndim == 2 else mask[0]"),
    ("log2 in the log-sum-exp", "m + np.log(np.exp(logits - m)", "m + np.log2(np.exp(logits - m)"),
    ("lse without the max shift", "lse[b, h, rows] = (m + np.log(", "lse[b, h, rows] = (np.log("),
]


def _load_mutant(old, new):
    path = os.path.join(ROOT, "oracle", "attention.py")
    src = open(path).read()
    assert src.count(old) >= 1, f"mutation target {old!r} not found"
    spec = importlib.util.spec_from_loader("oracle_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(name, old, new):
    mutant = _load_mutant(old, new)
    failures = 0
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(mutant.attention)
        except Exception:
            failures += 1
    for pin in oracle_pins.LSE_PINS:
        try:
            pin(mutant.attention_lse)
        except Exception:
            failures += 1
    assert failures > 0, f"no pin caught the planted mistake: {name}"
