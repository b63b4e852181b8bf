"""The decode-attention oracle against its pins, and planted mistakes in a
private copy of it (on the CPU) that the pins must catch."""

import inspect
import types

import pytest

import attn_pins
from oracle import attn_oracle


@pytest.mark.parametrize("pin", attn_pins.ALL_PINS, ids=[p.__name__ for p in attn_pins.ALL_PINS])
def test_attention_oracle_pin(pin):
    pin(attn_oracle)


MUTANTS = [
    ("kv head h % HKV instead of h // G", "kvh = h // group", "kvh = h % hkv"),
    ("scale dropped", "a = scale * (kk @ qq)", "a = kk @ qq"),
    ("scale squared", "a = scale * (kk @ qq)", "a = scale * scale * (kk @ qq)"),
    ("scores negated", "a = scale * (kk @ qq)", "a = -scale * (kk @ qq)"),
    ("maximum not subtracted", "e = np.exp(a - np.max(a))", "e = np.exp(a)"),
    ("normalised by L", "w = e / np.sum(e)", "w = e / len(e)"),
    ("values taken from the keys", "vv = values[:, kvh, :]", "vv = keys[:, kvh, :]"),
    ("page and slot swapped", "pages = table_row[t // page_size]\n    slots = t % page_size",
     "pages = table_row[t % page_size]\n    slots = t // page_size"),
    ("next page", "pages = table_row[t // page_size]", "pages = table_row[t // page_size + 1]"),
    ("slot counted from the page end", "slots = t % page_size", "slots = page_size - 1 - t % page_size"),
    ("last token dropped", "t = np.arange(length)", "t = np.arange(length - 1)"),
    ("query of the kv head", "qq = q[s, h].astype(np.float64)", "qq = q[s, kvh].astype(np.float64)"),
    ("double rounding through fp32", "return o64.astype(np.float16)",
     "return o64.astype(np.float32).astype(np.float16)"),
    ("empty sequence gives the mean of nothing", "        if length == 0:\n            continue\n", ""),
    ("weights without abs in the bound", "wabs[s, h] = w @ np.abs(vv)", "wabs[s, h] = w @ vv"),
    ("tolerance 2e-2", "ATTN_REL_TOL = 2e-3", "ATTN_REL_TOL = 2e-2"),
    ("NaN accepted", "return np.isfinite(a) & (diff <= attn_tol_bound(wabs))",
     "return ~(diff > attn_tol_bound(wabs))"),
    ("page range not checked", "if np.any(used < 0) or np.any(used >= num_pages):",
     "if np.any(used < 0):"),
    ("score bound from signed scores", "smax[s, h] = abs(scale) * np.max(np.abs(kk) @ np.abs(qq))",
     "smax[s, h] = scale * np.max(kk @ qq)"),
    ("score bound without abs(scale)", "smax[s, h] = abs(scale) * np.max(np.abs(kk) @ np.abs(qq))",
     "smax[s, h] = scale * np.max(np.abs(kk) @ np.abs(qq))"),
    ("score bound from |signed scores|", "smax[s, h] = abs(scale) * np.max(np.abs(kk) @ np.abs(qq))",
     "smax[s, h] = abs(scale) * np.max(np.abs(kk @ qq))"),
]


def _mutant(old, new):
    src = inspect.getsource(attn_oracle)
    assert src.count(old) == 1, f"mutation site not unique or missing: {old!r}"
    mod = types.ModuleType("attn_oracle_mutant")
    exec(compile(src.replace(old, new), "<attention oracle mutant>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_attention_pins_catch_planted_mistake(name, old, new):
    orc = _mutant(old, new)
    failed = []
    for pin in attn_pins.ALL_PINS:
        try:
            pin(orc)
        except Exception:  # AssertionError, or a crash caused by the mutation
            failed.append(pin.__name__)
    assert failed, f"no pin caught the planted mistake: {name}"


def test_unmutated_attention_copy_passes_every_pin():
    orc = _mutant("ATTN_ABS_TOL = 1e-6", "ATTN_ABS_TOL = 1e-6")
    for pin in attn_pins.ALL_PINS:
        pin(orc)
