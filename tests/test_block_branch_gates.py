"""The block's branch gates have teeth (CPU only, small shapes).

Planted in the oracle: the oldest history chunk dropped from every node that
reads history, that chunk's level off by one, and the queries left
unrotated.  Each must fail the branch gate on the attention output o and on
the attention branch a = o Wo^T (q without RoPE also on q), for every node,
on the same inputs the GPU block tests use; rounding the exact values to
bf16 must use well under the gate.  Eq. 6 (only the selected states are
visible) and Sec. 3.2 ("Effective context and visibility").
"""
import numpy as np
import pytest

from block_inputs import (PLANTED, X_SMALL, BlockInputs, branch_ratio, oracle_traces,
                          planted_must_fail)
from synth import bf16_round
from synth.configs import SMALL

CASES = [
    ("prog", [(6, 1), (7, 2), (8, 3), (9, 4)], [(c, 0) for c in range(6)]),
    ("prog", [(6, 0), (7, 1), (8, 2), (9, 3), (10, 4)], [(c, 0) for c in range(6)]),
    ("same", [(6 + i, 3) for i in range(4)], [(c, 3) for c in range(6)]),
    ("clean", [(6, 4)], [(c, 0) for c in range(6)]),
]


@pytest.mark.parametrize("x_small", [False, True], ids=["x", "x-small-w_down-0"])
@pytest.mark.parametrize("kind,pack,resident", CASES, ids=["prog4", "prog5", "same", "clean"])
def test_planted_mistakes_fail_the_branch_gates(kind, pack, resident, x_small):
    inp = BlockInputs(SMALL, kind, pack, resident, seed=11, x_scale=X_SMALL if x_small else 1.0,
                      zero_down=x_small)
    tr = oracle_traces(inp, rows=None)
    worst = planted_must_fail(tr)
    assert set(worst) == set(PLANTED)
    for i, t in tr["exact"].items():
        for key in ("q", "o", "a"):
            rnd = bf16_round(t[key].astype(np.float32)).astype(np.float64)
            assert branch_ratio(rnd, t[key]) < 0.5, (pack[i], key)


def test_small_x_branch_is_y_minus_x():
    """With w_down = 0 the block output is x + a exactly (fp64 oracle), so
    y - x measured on a GPU output is the attention branch; at x of scale
    2^-8 the bf16 rounding of x + a is small against a."""
    inp = BlockInputs(SMALL, *CASES[0], seed=11, x_scale=X_SMALL, zero_down=True)
    tr = {}
    y, _ = inp.oracle(rows=None, trace=tr)
    for i in range(len(inp.pack)):
        np.testing.assert_allclose(y[i] - inp.x[i], tr[i]["a"], rtol=0, atol=1e-15)
        rounded = bf16_round((inp.x[i] + tr[i]["a"]).astype(np.float32)).astype(np.float64)
        assert branch_ratio(rounded - inp.x[i], tr[i]["a"]) < 0.5
