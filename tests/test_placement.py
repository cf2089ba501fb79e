"""The placement optimizer (Sec. VI-C, Alg. 1) against the plain oracle.

Parity: the exact latency of a placement (Eq. 1-4) matches the oracle's loops;
the budget found by the binary search matches the optimum of the LP relaxation
minimised directly; the integral placement respects the problem's constraints
(Eq. 5) and, on inputs small enough to enumerate, lands at or just above the
exhaustive optimum.
"""
import numpy as np
import pytest

from oracle import placement as op
from paper_2607_08782_amd import placement as pl

F_COMP = [(1.0, 0.0), (2.0, -40.0)]
F_COMM = [(0.3, 2.0)]


def _tiny(seed):
    rng = np.random.default_rng(seed)
    L, G, E = 1 + seed % 2, 2 + seed % 3, 4 + seed % 3
    W = rng.integers(0, 40, size=(L, G, E))
    return W, G, max(2, (E + G - 1) // G)


def _zipf_workload(E, G, T, k, s, seed):
    """Tokens per (GPU, expert): Zipf popularity with a per-GPU Dirichlet skew."""
    rng = np.random.default_rng(seed)
    p = np.arange(1, E + 1) ** (-s)
    p = (p / p.sum())[rng.permutation(E)]
    return np.stack([rng.multinomial(T * k, rng.dirichlet(p * 50)) for _ in range(G)])


def _assert_valid(P, L, E, G, C_max):
    P = np.asarray(P)
    assert P.shape == (L, E)
    assert P.min() >= 0 and P.max() < G
    for l in range(L):
        assert np.bincount(P[l], minlength=G).max() <= C_max


@pytest.mark.parametrize("seed", range(5))
def test_latency_matches_the_oracle(seed):
    rng = np.random.default_rng(seed)
    L, G, E = 2, 3, 7
    W = rng.integers(0, 50, size=(L, G, E))
    P = rng.integers(0, G, size=(L, E))
    ours = pl.total_latency(W, P, 3.0, F_COMP, F_COMM)
    ref = op.latency(W.tolist(), P.tolist(), G, 3.0, F_COMP, F_COMM)
    assert ours == pytest.approx(ref, rel=1e-12)


F_COMP_2D = [(1.0, 6.0, 0.0), (0.2, 20.0, 5.0)]     # load and active experts


@pytest.mark.parametrize("seed", range(4))
def test_active_expert_model_matches_the_oracle(seed):
    """f_comp of the load and the active-expert count: exact latency as the oracle's
    loops (some experts get no tokens), and the binary search's budget at the LP
    optimum minimised directly; the integral placement is valid."""
    rng = np.random.default_rng(50 + seed)
    L, G, E = 1 + seed % 2, 3, 6
    W = rng.integers(0, 30, size=(L, G, E))
    W[:, :, rng.integers(0, E)] = 0                       # an expert nobody routes to
    P = rng.integers(0, G, size=(L, E))
    ours = pl.total_latency(W, P, 2.0, F_COMP_2D, F_COMM)
    ref = op.latency(W.tolist(), P.tolist(), G, 2.0, F_COMP_2D, F_COMM)
    assert ours == pytest.approx(ref, rel=1e-12)
    C_max = 3
    res = pl.place(W, G, C_max, 2.0, F_COMP_2D, F_COMM, seed=seed)
    beta, _ = op.lp_optimum(W.tolist(), G, C_max, 2.0, F_COMP_2D, F_COMM)
    assert res.beta_star == pytest.approx(beta, rel=2e-3)
    _assert_valid(res.P, L, E, G, C_max)
    assert res.latency == pytest.approx(
        op.latency(W.tolist(), res.P.tolist(), G, 2.0, F_COMP_2D, F_COMM), rel=1e-12)


def test_two_variable_fit_reproduces_a_roofline_and_passes_under_the_points():
    """f(lambda, a) = max(20 + 15 a, 10 + 0.05 lambda + 2 a), the shape of a step bound
    by streaming a experts' weights or by the rows' arithmetic: the fit reproduces
    it on the grid; with noise added it stays at or under every point."""
    from paper_2607_08782_amd.fcomp import fit_convex_pwl2
    pts = [(lam, a, max(20 + 15 * a, 10 + 0.05 * lam + 2 * a)) for a in (1, 2, 4, 6, 8)
           for lam in (8, 16, 64, 256, 1024, 4096) if lam >= a]
    planes = fit_convex_pwl2(pts)
    got = pl.comp_eval(planes, [p[0] for p in pts], [p[1] for p in pts])
    assert np.allclose(got, [p[2] for p in pts], rtol=1e-9)
    rng = np.random.default_rng(1)
    noisy = [(lam, a, t * (1 + 0.05 * rng.random())) for lam, a, t in pts]
    planes = fit_convex_pwl2(noisy)
    got = pl.comp_eval(planes, [p[0] for p in noisy], [p[1] for p in noisy])
    assert np.all(got <= np.array([p[2] for p in noisy]) * (1 + 1e-9))
    assert all(a >= 0 and c >= 0 for a, c, _ in planes)


def test_convex_fit_reproduces_a_convex_function_and_underestimates_otherwise():
    z = np.array([0, 16, 64, 128, 512, 1024, 4096], float)
    f = [(0.0, 190.0), (0.3, 0.0)]                       # max(190, 0.3 z)
    t = pl.pwl_eval(f, z)
    got = pl.fit_convex_pwl(z, t)
    assert np.allclose(pl.pwl_eval(got, z), t)
    # a bump at z = 128 is not convex: the fit passes under it and stays convex
    t2 = t.copy()
    t2[3] += 50.0
    got2 = pl.fit_convex_pwl(z, t2)
    assert np.all(pl.pwl_eval(got2, z) <= t2 + 1e-9)
    slopes = [a for a, _ in got2]
    assert slopes == sorted(slopes)


@pytest.mark.parametrize("seed", range(8))
def test_binary_search_budget_matches_the_lp_optimum(seed):
    W, G, C = _tiny(seed)
    res = pl.place(W, G, C, 1.0, F_COMP, F_COMM, eps=1e-4, seed=seed)
    beta, _ = op.lp_optimum(W.tolist(), G, C, 1.0, F_COMP, F_COMM)
    assert beta * (1 - 1e-9) <= res.beta_star <= beta * (1 + 2e-4) + 1e-9


@pytest.mark.parametrize("seed", range(12))
def test_placement_is_feasible_and_close_to_exhaustive(seed):
    W, G, C = _tiny(seed)
    L, _, E = W.shape
    res = pl.place(W, G, C, 1.0, F_COMP, F_COMM, seed=seed)
    _assert_valid(res.P, L, E, G, C)
    assert np.array_equal(res.x.argmax(axis=2), res.P) and np.all(res.x.sum(axis=2) == 1)
    _, best = op.exhaustive(W.tolist(), G, C, 1.0, F_COMP, F_COMM)
    assert res.latency == pytest.approx(op.latency(W.tolist(), res.P.tolist(), G, 1.0, F_COMP, F_COMM), rel=1e-12)
    assert best - 1e-9 <= res.latency <= 1.05 * best


@pytest.mark.parametrize("seed", range(3))
def test_mixtral_sized_placement_within_half_percent_of_exhaustive(seed):
    # 8 experts on 4 GPUs, 2 per GPU; f_comp = max(190 us, 0.3 us/token),
    # f_comm = 5 us + bytes / 153 GB/s (one xGMI link), d = 4096 bf16 values
    W = _zipf_workload(8, 4, 1024, 2, 1.0, seed)[None]
    f_comp, f_comm, d = [(0.0, 190.0), (0.3, 0.0)], [(1e6 / 153e9, 5.0)], 8192.0
    res = pl.place(W, 4, 2, d, f_comp, f_comm, seed=seed)
    _assert_valid(res.P, 1, 8, 4, 2)
    _, best = op.exhaustive(W.tolist(), 4, 2, d, f_comp, f_comm)
    assert best - 1e-9 <= res.latency <= 1.005 * best
    assert res.beta_star <= best + 1e-9


def test_rounding_without_polish_is_feasible_and_deterministic():
    W = _zipf_workload(16, 4, 512, 2, 1.2, 7)[None]
    a = pl.place(W, 4, 5, 8192.0, F_COMP, F_COMM, polish=False, seed=3)
    b = pl.place(W, 4, 5, 8192.0, F_COMP, F_COMM, polish=False, seed=3)
    _assert_valid(a.P, 1, 16, 4, 5)
    assert np.array_equal(a.P, b.P) and a.latency == b.latency
    assert a.latency >= a.beta_star * (1 - 1e-9)


def test_walk_stays_inside_the_polytope():
    W = _zipf_workload(12, 3, 256, 2, 1.0, 11).astype(float)[None]
    lp = pl._build_lp(W, 1.0, 5, F_COMP, F_COMM)
    x0, full = pl._feasible(lp, 1e9)
    rng = np.random.default_rng(0)
    # constraints on x alone with the auxiliaries fixed at a generous value
    aux = np.full(lp.nv - lp.nx, 1e6)
    aux[:2] = 1e7                      # tau_comp, tau_comm above the sum of their pair terms
    A = lp.A.tocsr()
    b = lp.b.copy()
    b[0] = 1e12
    b_in = b - A[:, lp.nx:] @ aux
    Ax = A[:, :lp.nx]
    start = np.full(lp.nx, 1.0 / 3)
    x, stats = pl._walk(start, Ax, b_in, rng, alpha=2.0, gamma=0.25, t_micro=200, max_macro=6)
    assert np.all(Ax @ x <= b_in + 1e-7)
    assert np.all((x >= -1e-12) & (x <= 1 + 1e-12))
    assert stats["fractional_end"] < stats["fractional_start"]


def test_capacity_too_small_is_rejected():
    with pytest.raises(ValueError):
        pl.place(np.ones((1, 2, 9)), 2, 4, 1.0, F_COMP, F_COMM)
