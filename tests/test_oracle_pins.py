"""The fp64 oracle against its pins (brute force, closed forms, invariants, paper bounds)."""
import pytest

import oracle_pins


@pytest.mark.parametrize("check", oracle_pins.ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check()


def test_oracle_rejects_nonfinite():
    import numpy as np
    import oracle
    from paper_2609_36301_amd.inputs import make_inputs

    inp = make_inputs(4, 16, 16, 8, seed=0)
    x = inp.x.copy()
    x[1, 3] = 0x7FC0  # bf16 NaN
    with pytest.raises(ValueError):
        oracle.route_lowrank(x, inp.R1, inp.R2, 2)
    R2 = inp.R2.copy()
    R2[0, 0] = 0x7F80  # bf16 +inf
    with pytest.raises(ValueError):
        oracle.route_lowrank(inp.x, inp.R1, R2, 2)
    with pytest.raises(ValueError):
        oracle.route_lowrank(inp.x, inp.R1, inp.R2, 9)  # k > M


def test_oracle_rows_subset_matches_full():
    import numpy as np
    import oracle
    from paper_2609_36301_amd.inputs import make_inputs

    inp = make_inputs(50, 32, 16, 40, seed=4)
    full = oracle.route_lowrank(inp.x, inp.R1, inp.R2, 4)
    rows = np.array([49, 0, 17, 17, 3])
    sub = oracle.route_lowrank(inp.x, inp.R1, inp.R2, 4, rows=rows)
    assert np.array_equal(sub.idx, full.idx[rows])
    assert np.array_equal(sub.gate, full.gate[rows])
