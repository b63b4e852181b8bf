"""Plant plausible mistakes in a private copy of the oracle (on the CPU) and
check that the pin suite catches every one of them.  This is what makes the
pins worth trusting: a dropped term, a wrong sign, an index or bit-order slip,
the wrong rounding mode or the wrong scale reading each fail at least one pin.
"""

import inspect
import types

import pytest

import oracle_pins
from oracle import wq_oracle

MUTANTS = [
    ("pack nibble order reversed", "packed |= q[:, i::CODES_PER_WORD].astype(np.uint32) << np.uint32(4 * i)",
     "packed |= q[:, i::CODES_PER_WORD].astype(np.uint32) << np.uint32(4 * (7 - i))"),
    ("unpack nibble order reversed", "(packed >> np.uint32(4 * i)) & np.uint32(0xF)",
     "(packed >> np.uint32(4 * (7 - i))) & np.uint32(0xF)"),
    ("dequant offset 7 instead of 8", "(q.astype(np.float32) - np.float32(ZERO_CODE))",
     "(q.astype(np.float32) - np.float32(7))"),
    ("dequant sign flipped", "(q.astype(np.float32) - np.float32(ZERO_CODE))",
     "(np.float32(ZERO_CODE) - q.astype(np.float32))"),
    ("zero code 7 everywhere", "ZERO_CODE = 8 ", "ZERO_CODE = 7 "),
    ("divide by unrounded fp32 scale", "divisor = s16.astype(np.float32)", "divisor = s32"),
    ("round half away from zero", "rounded = np.rint(r).astype(np.int64)",
     "rounded = np.trunc(r + np.copysign(np.float32(0.5), r)).astype(np.int64)"),
    ("round half up", "rounded = np.rint(r).astype(np.int64)",
     "rounded = np.floor(r + np.float32(0.5)).astype(np.int64)"),
    ("scale divisor 7.5", "SCALE_DIVISOR = 7 ", "SCALE_DIVISOR = 7.5 "),
    ("amax without abs", "amax = np.max(np.abs(wg), axis=2)", "amax = np.max(wg, axis=2)"),
    ("scale truncated to fp16", "s16 = s32.astype(np.float16)",
     "s16 = np.where(np.abs(s32.astype(np.float16).astype(np.float32)) > np.abs(s32), "
     "np.nextafter(s32.astype(np.float16), np.float16(0)), s32.astype(np.float16))"),
    ("zero scale gives code 0", "q = np.full((n, ngroups, group), ZERO_CODE, dtype=np.int64)",
     "q = np.full((n, ngroups, group), 0, dtype=np.int64)"),
    ("clamp low end at 1", "np.clip(rounded + ZERO_CODE, 0, QMAX_CODE)", "np.clip(rounded + ZERO_CODE, 1, QMAX_CODE)"),
    ("scale index tiled not repeated", "np.repeat(s16.astype(np.float32), group, axis=1)",
     "np.tile(s16.astype(np.float32), (1, group))"),
    ("x reversed along K", "y64[mi, r0:r1] = np.sum(w_hat * x64[mi][None, :], axis=1)",
     "y64[mi, r0:r1] = np.sum(w_hat * x64[mi][None, ::-1], axis=1)"),
    ("first K term dropped", "y64[mi, r0:r1] = np.sum(w_hat * x64[mi][None, :], axis=1)",
     "y64[mi, r0:r1] = np.sum((w_hat * x64[mi][None, :])[:, 1:], axis=1)"),
    ("sum in fp32", "y64[mi, r0:r1] = np.sum(w_hat * x64[mi][None, :], axis=1)",
     "y64[mi, r0:r1] = np.sum((w_hat * x64[mi][None, :]).astype(np.float32), axis=1)"),
    ("double rounding through fp32", "return gemv_f64(packed, scales, x, n, k, group).astype(np.float16)",
     "return gemv_f64(packed, scales, x, n, k, group).astype(np.float32).astype(np.float16)"),
    ("tolerance without abs", "w_abs = np.abs(dequant(", "w_abs = (dequant("),
    ("tolerance 1e-2", "REL_TOL = 1e-3", "REL_TOL = 1e-2"),
    ("tolerance without absolute term", "return REL_TOL * out + ABS_TOL", "return REL_TOL * out"),
    ("NaN accepted", "return (a == b) | (np.isfinite(diff) & (diff <= bound))",
     "return (a == b) | ~(diff > bound)"),
]


def _mutant(old, new):
    src = inspect.getsource(wq_oracle)
    assert src.count(old) == 1, f"mutation site not unique or missing: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "<oracle mutant>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(name, old, new):
    orc = _mutant(old, new)
    failed = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(orc)
        except Exception:  # AssertionError, or a crash caused by the mutation
            failed.append(pin.__name__)
    assert failed, f"no pin caught the planted mistake: {name}"


def test_unmutated_copy_passes_every_pin():
    orc = _mutant("GROUP = 32 ", "GROUP = 32 ")
    for pin in oracle_pins.ALL_PINS:
        pin(orc)
