"""The fused-operation oracle against its pins, and planted mistakes in a
private copy of it (on the CPU) that the pins must catch."""

import inspect
import types

import pytest

import fused_pins
from oracle import fused_oracle


@pytest.mark.parametrize("pin", fused_pins.ALL_PINS, ids=[p.__name__ for p in fused_pins.ALL_PINS])
def test_fused_oracle_pin(pin):
    pin(fused_oracle)


MUTANTS = [
    ("RMSNorm without the root", "return x / np.sqrt(ms + eps) * g", "return x / (ms + eps) * g"),
    ("RMSNorm sum instead of mean", "ms = np.mean(x * x)", "ms = np.sum(x * x)"),
    ("RMSNorm eps outside the root", "return x / np.sqrt(ms + eps) * g", "return x / (np.sqrt(ms) + eps) * g"),
    ("RMSNorm without the weight", "return x / np.sqrt(ms + eps) * g", "return x / np.sqrt(ms + eps)"),
    ("RMSNorm mean of |x|", "ms = np.mean(x * x)", "ms = np.mean(np.abs(x)) ** 2"),
    ("SiLU with exp(+a)", "return a / (1.0 + np.exp(-a)) * b", "return a / (1.0 + np.exp(a)) * b"),
    ("sigmoid instead of SiLU", "return a / (1.0 + np.exp(-a)) * b", "return 1.0 / (1.0 + np.exp(-a)) * b"),
    ("gate and up swapped", "a, b = x[:k], x[k:]", "b, a = x[:k], x[k:]"),
    ("halves interleaved", "a, b = x[:k], x[k:]", "a, b = x[0::2], x[1::2]"),
    ("residual subtracted", "y64 = y64 + r.astype(np.float64)", "y64 = y64 - r.astype(np.float64)"),
    ("linear rounded before the residual", "y64 = y64 + r.astype(np.float64)",
     "y64 = y64.astype(np.float16).astype(np.float64) + r.astype(np.float64)"),
    ("prologue not rounded to fp16", "return rmsnorm_f64(x, g, eps).astype(np.float16)",
     "return rmsnorm_f64(x, g, eps).astype(np.float32)"),
    ("argmax takes the last maximum", "if y[i] > y[best]:", "if y[i] >= y[best]:"),
    ("argmax is argmin", "if y[i] > y[best]:", "if y[i] < y[best]:"),
    ("tolerance 2e-2", "FUSED_REL_TOL = 2e-3", "FUSED_REL_TOL = 2e-2"),
    ("tolerance ignores the residual", "v = v + np.abs(np.asarray(residual, dtype=np.float16).astype(np.float64))",
     "v = v"),
    ("NaN accepted", "return np.isfinite(a) & (np.abs(a - b) <= bound)", "return ~(np.abs(a - b) > bound)"),
]


def _mutant(old, new):
    src = inspect.getsource(fused_oracle)
    assert src.count(old) == 1, f"mutation site not unique or missing: {old!r}"
    src = src.replace(old, new).replace("from . import wq_oracle", "from oracle import wq_oracle")
    mod = types.ModuleType("fused_oracle_mutant")
    exec(compile(src, "<fused oracle mutant>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_fused_pins_catch_planted_mistake(name, old, new):
    orc = _mutant(old, new)
    failed = []
    for pin in fused_pins.ALL_PINS:
        try:
            pin(orc)
        except Exception:  # AssertionError, or a crash caused by the mutation
            failed.append(pin.__name__)
    assert failed, f"no pin caught the planted mistake: {name}"


def test_unmutated_fused_copy_passes_every_pin():
    orc = _mutant("FUSED_ABS_TOL = 1e-5", "FUSED_ABS_TOL = 1e-5")
    for pin in fused_pins.ALL_PINS:
        pin(orc)
