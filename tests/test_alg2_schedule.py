"""Pins of the model of the paper's MatMul 2 work split and of its gain formula.  CPU only.

The worked constants are derived from Algorithm 2's integer formulas at the paper's MatMul 2 shape
(golden/alg2_worked_example.json); the gain formula is checked against the numbers printed in the
Evaluation section and Table II (golden/mean_gain.json).
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import alg2_schedule as a2
import synthetic as syn

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# the golden file names each quantity by the paper's symbol; the model names it in its own terms
SYMBOLS = {"fractalSize": "col_block", "kSplitSize": "k_slice", "kParts": "n_slices",
           "fractalNum": "n_col_blocks", "S": "n_blocks", "V": "n_units", "nPart_W": "blocks_per_unit",
           "groupSize": "units_per_slice"}


def test_worked_constants_of_matmul2():
    g = _gold("alg2_worked_example.json")
    p = a2.partition(g["K"], g["N"], g["P"])
    for sym, field in SYMBOLS.items():
        assert getattr(p, field) == g[sym], sym
    per_unit = p.blocks_per_unit * p.k_slice * p.col_block * 2
    assert per_unit == g["bytes_per_executor"]
    assert p.n_units * per_unit == g["weight_bytes"] == g["K"] * g["N"] * 2


@pytest.mark.parametrize("N", [576, 2112])
def test_every_block_is_computed_exactly_once(N):
    p = a2.partition(7168, N)
    seen = [b for u in range(p.n_units) for b in p.blocks_of(u)]
    assert sorted(seen) == list(range(p.n_blocks))
    cells = {p.slice_and_cols(b) for b in seen}
    assert cells == {(s, c) for s in range(p.n_slices) for c in range(p.n_col_blocks)}


def test_one_token_offset_per_unit_holds_at_576_but_not_2112():
    # the reading of the section's indexing: at N = 576 every unit's run lies in one row slice,
    # so one token offset per unit (its slice) describes it; at N = 2112 some runs straddle two
    p = a2.partition(7168, 576)
    assert all(len(p.slices_of(u)) == 1 for u in range(p.n_units))
    assert [min(p.slices_of(u)) for u in range(p.n_units)] == [u // p.units_per_slice for u in range(p.n_units)]
    q = a2.partition(7168, 2112)
    assert (q.n_units, q.n_slices, q.units_per_slice) == (44, 7, 6)
    assert max(u // q.units_per_slice for u in range(q.n_units)) >= q.n_slices    # past the token's end
    assert any(len(q.slices_of(u)) > 1 for u in range(q.n_units))


@pytest.mark.parametrize("N", [576, 2112])
def test_split_result_matches_plain_product(N):
    c = syn.down_projection(n=N)
    p = a2.partition(c.K, c.N)
    total, partials = a2.evaluate(c.x, c.W, p, oracle.decode)
    assert not np.isnan(partials).any()
    y, a = oracle.gemv(c.x, c.W, c.dt)
    assert oracle.within_tolerance(total, y[0], a[0]).all()
    # the output cast to bf16 stays within one bf16 rounding of the fp32 result
    out = oracle.decode(oracle.round_bf16(total), syn.BF16)
    assert np.all(np.abs(out - total) <= np.abs(total) * 2.0 ** -8)


def test_mean_gain_formula_matches_printed_numbers():
    from bench import mean_gain
    g = _gold("mean_gain.json")
    e = g["evaluation"]
    G = mean_gain(e["E_T_opt"], e["E_T_base"])
    assert abs(G - 0.2020) < 5e-4 and round(100 * G) == e["G_percent_printed"]
    for row in g["table2"]:
        assert round(100 * mean_gain(row["optimized"], row["baseline"])) in (
            row["speedup_percent_printed"], row["speedup_percent_printed"] + 1)
