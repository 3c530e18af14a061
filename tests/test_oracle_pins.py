"""The oracle against its pins (CPU only)."""
import numpy as np
import pytest

import oracle
import oracle_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(pins.real_handle())


def test_thread_count_does_not_change_results():
    rng = np.random.default_rng(3)
    c = pins.rand_case(rng, N=2, M=3, D=4, shapes=((9, 7), (4, 5)), Lq=40, P=3)
    args = (c["value"], c["shapes"], c["starts"], c["loc"], c["attn"])
    o1 = oracle.forward(*args, threads=1)
    o4 = oracle.forward(*args, threads=4)
    assert np.array_equal(o1, o4)
    b1 = oracle.backward(*args, c["g"], threads=1)
    b4 = oracle.backward(*args, c["g"], threads=3)
    for x, y in zip(b1, b4):
        assert np.array_equal(x, y)
