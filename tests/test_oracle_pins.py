"""The CPU oracle against library routines, closed forms, invariants and brute force."""
import pytest

import oracle
from oracle_pins import ALL_PINS


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_pin(pin, lib):
    pin(lib)


def test_bf16_rounding_recipe():
    """The generator's bf16 rounding is round-to-nearest-even on the bit pattern."""
    import numpy as np
    from paper_2607_27735_amd.workloads import f32_to_bf16_bits, bf16_bits_to_f32
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(200000).astype(np.float32) * 10.0 ** rng.integers(-8, 8, 200000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -2.5e-39],
                                 dtype=np.float32)]).astype(np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    ref = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    assert np.array_equal(f32_to_bf16_bits(x), ref)
    assert np.array_equal(bf16_bits_to_f32(ref), (ref.astype(np.uint32) << 16).view(np.float32))
    # ties go to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    assert f32_to_bf16_bits(np.array([1.00390625], np.float32))[0] == 0x3F80
    assert f32_to_bf16_bits(np.array([1.01171875], np.float32))[0] == 0x3F82
