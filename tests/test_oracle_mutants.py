"""Every planted mistake in the oracle must trip at least one pin (CPU only).

The mutants are compile-time variants of the oracle source (ORACLE_MUTANT):
1 e0 left out of the minimum, 2 sign error in the difference, 3 wrong
normaliser, 4 coordinates paired in reverse, 5 last set member skipped,
6 difference of losses reversed, 7 maximum instead of minimum, 8 distance not
squared.
"""
import pytest

import oracle
from oracle_pins import PINS

MUTANTS = list(range(1, 9))


@pytest.mark.parametrize("mutant", MUTANTS)
def test_mutant_is_caught(mutant, tmp_path):
    o = oracle.load_mutant(mutant, str(tmp_path))
    caught = []
    for pin in PINS:
        try:
            pin(o)
        except AssertionError as e:
            caught.append(pin.__name__)
        except Exception as e:  # a crash or NaN-driven error also counts
            caught.append(f"{pin.__name__}:{type(e).__name__}")
    assert caught, f"mutant {mutant} passed every pin"
