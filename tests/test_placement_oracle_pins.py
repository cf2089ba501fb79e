"""Pins of the placement-model oracle (Sec. VI: Eq. 1-5 and the LP relaxation).

Every expected value comes from another route than the oracle's own code: a
hand derivation of Eq. 1-4 on a three-expert example, a placement whose
optimality follows from the construction, closed forms of the relaxation
(perfect fractional balance; a single GPU), and the relaxation bound against
brute force on tiny random inputs.
"""
import json
import os

import numpy as np
import pytest

from oracle import placement as op

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "placement_hand_example.json")


def test_hand_worked_example_of_eq1_to_eq4():
    g = json.load(open(GOLDEN))
    W, P, G, d = g["W"], g["P"], g["G"], g["d"]
    lin = [(1.0, 0.0)]
    assert op.loads(W[0], P[0], G) == g["lambda"]
    assert op.volumes(W[0], P[0], G, d) == g["D"]
    assert op.latency(W, P, G, d, lin, lin) == g["T_linear"]
    # f_comp(z) = max(z, 2z - 5), f_comm(z) = max(1, z): hand-evaluated in the fixture
    assert op.latency(W, P, G, d, [(1.0, 0.0), (2.0, -5.0)], [(0.0, 1.0), (1.0, 0.0)]) == g["T_pwl"]


def test_hand_worked_example_with_active_experts():
    """f_comp of the load and the number of active experts, hand-evaluated in the
    fixture; an expert with no tokens does not count as active."""
    g = json.load(open(GOLDEN))
    W, P, G, d = g["W"], g["P"], g["G"], g["d"]
    f2 = [tuple(p) for p in g["f_comp_2d"]]
    lin = [(1.0, 0.0)]
    assert op.active(W[0], P[0], G) == g["active"]
    assert op.latency(W, P, G, d, f2, lin) == g["T_2d"]
    W4 = [[row + [0] for row in W[0]]]                 # a fourth expert, no tokens, on GPU 1
    assert op.active(W4[0], P[0] + [1], G) == g["active"]
    assert op.latency(W4, [P[0] + [1]], G, d, f2, lin) == g["T_2d"]
    # pieces with no active-expert slope are the one-variable model
    assert op.latency(W, P, G, d, [(1.0, 0.0, 0.0)], lin) == g["T_linear"]


def test_lp_optimum_prices_active_experts_on_one_gpu():
    """One GPU hosts every expert: lambda = the whole demand, a = the experts with
    tokens; tau_comp = max(z + 4a, 2a) at z = 16, a = 2 (one expert has none) -> 24."""
    W = [[[3, 0, 13]]]
    beta, x = op.lp_optimum(W, 1, 3, 1.0, [(1.0, 4.0, 0.0), (0.0, 2.0, 0.0)], [(1.0, 0.0)])
    assert beta == pytest.approx(24.0, abs=1e-9)


def test_exhaustive_finds_the_placement_that_is_optimal_by_construction():
    # GPU 0's tokens go only to experts 0, 1 and GPU 1's only to 2, 3, with equal
    # demand: hosting {0,1} on GPU 0 and {2,3} on GPU 1 balances the load exactly
    # and sends nothing, so no placement can do better.
    W = [[[5, 5, 0, 0], [0, 0, 5, 5]]]
    lin = [(1.0, 0.0)]
    P, T = op.exhaustive(W, 2, 2, 1.0, lin, lin)
    assert P == [[0, 0, 1, 1]]
    assert T == 10.0


def test_lp_optimum_is_perfect_fractional_balance_without_communication_cost():
    rng = np.random.default_rng(3)
    G, E = 3, 5
    W = [rng.integers(0, 20, size=(G, E)).tolist()]
    total = float(np.sum(W))
    beta, x = op.lp_optimum(W, G, E, 1.0, [(1.0, 0.0)], [(0.0, 0.0)])
    assert beta == pytest.approx(total / G, rel=1e-9, abs=1e-9)
    assert np.all(x.sum(axis=2) >= 1 - 1e-9)


def test_lp_optimum_on_one_gpu_is_f_comp_of_the_whole_demand():
    W = [[[3, 9, 4]]]
    f_comp = [(1.0, 0.0), (3.0, -10.0)]          # max(z, 3z - 10) at z = 16 -> 38
    beta, x = op.lp_optimum(W, 1, 3, 1.0, f_comp, [(1.0, 0.0)])
    assert beta == pytest.approx(38.0, abs=1e-9)
    assert np.allclose(x, 1.0)


@pytest.mark.parametrize("seed", range(6))
def test_relaxation_never_exceeds_the_integer_optimum(seed):
    rng = np.random.default_rng(100 + seed)
    L, G, E = 1 + seed % 2, 2 + seed % 2, 4
    W = rng.integers(0, 30, size=(L, G, E)).tolist()
    f_comp = [(1.0, 0.0), (2.0, -40.0)]
    f_comm = [(0.5, 0.0)]
    C_max = 2 + seed % 2
    P, T = op.exhaustive(W, G, C_max, 1.0, f_comp, f_comm)
    beta, _ = op.lp_optimum(W, G, C_max, 1.0, f_comp, f_comm)
    assert beta <= T + 1e-9
    # the enumerated optimum respects the capacity and hosts every expert once
    for P_l in P:
        assert len(P_l) == E and max(P_l.count(j) for j in range(G)) <= C_max
