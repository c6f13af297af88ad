"""The oracle against its pins (CPU only), and proof that the pins catch
plausible mistakes planted in the oracle."""
import pytest

import oracle
import oracle_pins

# Planted mistakes compiled into oracle variants (see ORACLE_PLANT in
# oracle/rfq_oracle.c): 1 Eq. 3 without the -2 offset, 2 offset off by one,
# 3 ties away from zero, 4 sign of zero dropped, 5 nibble order swapped,
# 6 residual taken of x instead of x - q, 7 weight scaled by the activation
# scale, 8 residual term dropped from the product, 9 bf16 truncation,
# 10 sign error in silu, 11 weight index shifted by one, 12 phi tile width
# halved, 13 strict comparison in the scale-threshold phi rule; in
# oracle/hif4_oracle.c: 14 HiF4 macro scale sized for a 6 instead of 7
# maximum, 15 shared 8-element micro-exponent set too eagerly, 16 E6M2 bias
# 47, 17 HiF4 element ties away from zero.
PLANTS = list(range(1, 18))


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(orc, pin):
    pin(orc)


@pytest.mark.parametrize("plant", PLANTS)
def test_planted_mistake_is_caught(plant, tmp_path):
    bad = oracle.variant(["-DORACLE_PLANT=%d" % plant], "plant%d" % plant)
    failed = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(bad)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, "no pin caught planted mistake %d" % plant
