"""Planted mistakes in the oracle must each trip at least one pin.

Every mutant is the oracle source compiled with one ``-DGDO_MUTANT_*`` define
(a dropped term, a wrong sign, a reversed order, an off-by-one k, ...).  This
shows the pins in ``pins.py`` are strong enough to catch the plausible ways
of getting the definition wrong.  Mutants exist only in the test build; the
oracle library used everywhere else is compiled without any of them.
"""
import pytest

import oracle
from pins import ALL_PINS

MUTANTS = [
    "GDO_MUTANT_SIGNED_KEY",
    "GDO_MUTANT_CEIL_K",
    "GDO_MUTANT_GLOBAL_K_PER_TENSOR",
    "GDO_MUTANT_NO_RESIDUAL",
    "GDO_MUTANT_STRICT_ONLY",
    "GDO_MUTANT_TIES_HIGH_INDEX",
    "GDO_MUTANT_KEPT_RESIDUAL_KEEPS_ACC",
    "GDO_MUTANT_SWAP_CENTRES",
    "GDO_MUTANT_BITS_MSB_FIRST",
    "GDO_MUTANT_APPLY_REVERSE_CLIENTS",
    "GDO_MUTANT_APPLY_ADD",
    "GDO_MUTANT_DELTA_REVERSED",
    "GDO_MUTANT_SAMPLED_KTH",
    "GDO_MUTANT_SAMPLED_GE",
    "GDO_MUTANT_SAMPLED_NO_CAPACITY",
    "GDO_MUTANT_SPLITMIX_SHIFT",
    "GDO_MUTANT_SAMPLE_WHOLE_SEGMENT",
    "GDO_MUTANT_THRESHOLD_MAX",
    "GDO_MUTANT_GLOBAL_MEAN_PER_TENSOR",
    "GDO_MUTANT_COLUMN_IS_ROW",
    "GDO_MUTANT_PULL_ADDS_ZERO",
    "GDO_MUTANT_PULL_COPY_IS_P",
    "GDO_MUTANT_DECODE_BITS_MSB",
]


def first_failing_pin(lib):
    """Name of the first pin (in ALL_PINS order) that the library fails, or None."""
    for pin in ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError, IndexError):
            return pin.__name__
    return None


@pytest.mark.parametrize("mutant", MUTANTS)
def test_mutant_is_caught(mutant):
    lib = oracle.build_variant([mutant])
    assert first_failing_pin(lib), f"{mutant} passed every pin"
