"""Pins of the paper's Algorithm 2 partition model and of its gain formula.  CPU only.

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


def test_worked_constants_of_matmul2():
    g = _gold("alg2_worked_example.json")
    p = a2.plan(g["K"], g["N"], g["P"])
    for key in ("fractalSize", "kSplitSize", "kParts", "fractalNum", "S", "V", "nPart_W", "groupSize"):
        assert getattr(p, key) == g[key], key
    per_exec = p.nPart_W * p.kSplitSize * p.fractalSize * 2
    assert per_exec == g["bytes_per_executor"]
    assert p.V * per_exec == g["weight_bytes"] == g["K"] * g["N"] * 2


@pytest.mark.parametrize("N", [576, 2112])
def test_every_block_is_computed_exactly_once(N):
    p = a2.plan(7168, N)
    seen = [fid for v in range(p.V) for fid in p.frac_ids(v)]
    assert sorted(seen) == list(range(p.S))
    blocks = {p.block(f) for f in seen}
    assert blocks == {(kp, cf) for kp in range(p.kParts) for cf in range(p.fractalNum)}


def test_printed_token_offset_holds_at_576_but_not_2112():
    p = a2.plan(7168, 576)
    for v in range(p.V):
        for f in p.frac_ids(v):
            assert p.block(f)[0] * p.kSplitSize == p.literal_off_T(v)
    q = a2.plan(7168, 2112)
    assert (q.V, q.kParts, q.groupSize) == (44, 7, 6)
    assert max(q.literal_off_T(v) for v in range(q.V)) >= 7168     # would read past T
    straddle = [v for v in range(q.V) if len({q.block(f)[0] for f in q.frac_ids(v)}) > 1]
    assert straddle, "under the reading, some executors' blocks span two k-parts"


@pytest.mark.parametrize("N", [576, 2112])
def test_alg2_result_matches_plain_product(N):
    c = syn.down_projection(n=N)
    p = a2.plan(c.K, c.N)
    acc, tmp = a2.run(c.x, c.W, p, oracle.decode)
    assert not np.isnan(tmp).any()
    y, a = oracle.gemv(c.x, c.W, c.dt)
    assert oracle.within_tolerance(acc, y[0], a[0]).all()
    # the output cast of Algorithm 2 (bf16) stays within one bf16 rounding of the fp32 result
    out = oracle.decode(oracle.round_bf16(acc), syn.BF16)
    assert np.all(np.abs(out - acc) <= np.abs(acc) * 2.0 ** -8)


def test_mean_gain_formula_matches_printed_numbers():
    from bench import mean_gain
    g = _gold("mean_gain.json")
    e = g["evaluation"]
    G = mean_gain(e["E_T_opt"], e["E_T_base"])
    assert abs(G - 0.2020) < 5e-4 and round(100 * G) == e["G_percent_printed"]
    for row in g["table2"]:
        assert round(100 * mean_gain(row["optimized"], row["baseline"])) in (
            row["speedup_percent_printed"], row["speedup_percent_printed"] + 1)
