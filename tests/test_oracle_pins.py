"""The oracle against its pins (closed forms, invariants, an independent
library implementation); see tests/oracle_pins.py for what each pins."""
import pytest

import oracle
from oracle_pins import PINS


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("name", sorted(PINS))
def test_pin(name, lib):
    PINS[name](lib)


def test_rejects_invalid_shapes(lib):
    import numpy as np
    from paper_2504_17577_amd import gen
    q, k, v = gen.random_problem(1, 3, 2, 4, 4, 8, seed=0)   # Hq % Hkv != 0
    with pytest.raises(oracle.OracleError):
        oracle.attn_fwd(q, k, v, False, 1.0, lib=lib)
    q, k, v = gen.random_problem(1, 2, 2, 6, 4, 8, seed=0)   # causal with Sq > Sk
    with pytest.raises(oracle.OracleError):
        oracle.attn_fwd(q, k, v, True, 1.0, lib=lib)
    with pytest.raises(oracle.OracleError):
        oracle.attn_rows(q, k, v, False, 1.0, [(0, 2, 0)], lib=lib)
    o, lse = oracle.attn_fwd(q, k, v, False, 1.0, lib=lib)
    assert np.isfinite(o).all() and np.isfinite(lse).all()
