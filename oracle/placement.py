"""Plain reference of Director's placement model -- TEST INFRASTRUCTURE.

Only ``tests/`` may import this module; the product's optimizer
(``paper_2607_08782_amd/placement.py``) never does, and this module imports
nothing from the product.  Everything here is written for checking by eye
against the paper (arXiv 2607.08782, Sec. VI), with plain loops:

* ``loads``        -- Eq. 1: lambda_j = sum_i [P(i) = j] sum_k W[k][i]
* ``volumes``      -- Eq. 3: D[j][k] = sum_{i : P(i) = k} d * W[j][i]
* ``latency``      -- Eq. 2 + Eq. 4: sum over layers of the straggler GPU's
                      f_comp(lambda_j) plus the straggler's sum over k != j of
                      f_comm(D[j][k])
* ``exhaustive``   -- the problem of Eq. 5 solved by enumerating every map
                      expert -> GPU that respects C_max (one host per expert,
                      as in the paper's exhaustive study, Sec. III); tiny inputs
* ``lp_optimum``   -- the LP relaxation of Sec. VI-C (x in [0,1], every expert
                      hosted at least once, at most C_max experts per GPU, the
                      max operators and the piecewise-linear latencies written
                      in epigraph form), minimised directly in one LP.  Its
                      optimum is the beta* that the paper's binary search over
                      the budget converges to.

Latency functions are convex piecewise-linear, given as a list of pieces
(slope, intercept): f(z) = max over pieces of slope * z + intercept (the
"standard piecewise linear approximation" of Sec. VI-C, read as convex so that
the epigraph constraints are exact).  f_comp may also be given as pieces
(slope, slope_active, intercept) of the GPU's load lambda_j and its number of
active experts a_j (hosted experts with at least one token): Eq. 2 prices the
computation by the load alone, but a decode-sized step streams the weights of
every active expert, so its time grows with a_j, which is as linear in the
placement as lambda_j is.

Workload tensors are W[l][j][i]: tokens on GPU j routed to expert i in layer l
(Sec. VI-A).  A placement is an integer array P[l][i] = host GPU of expert i.
"""
from __future__ import annotations

import itertools

import numpy as np


def pwl(pieces, z):
    """f(z) = max over (slope, intercept) pieces."""
    return max(a * z + b for a, b in pieces)


def comp(pieces, lam, act):
    """f_comp of a GPU with load lam and act active experts: (slope, intercept)
    pieces price the load alone, (slope, slope_active, intercept) pieces both."""
    if len(pieces[0]) == 2:
        return pwl(pieces, lam)
    return max(a * lam + c * act + b for a, c, b in pieces)


def active(W_l, P_l, G):
    """Active experts of every GPU: hosted experts with a non-zero demand."""
    act = [0] * G
    for i in range(len(P_l)):
        demand = 0.0
        for k in range(G):
            demand += W_l[k][i]
        if demand != 0:
            act[P_l[i]] += 1
    return act


def loads(W_l, P_l, G):
    """Eq. 1 for one layer: computational load of every GPU."""
    E = len(P_l)
    lam = [0.0] * G
    for i in range(E):
        demand = 0.0
        for k in range(G):
            demand += W_l[k][i]
        lam[P_l[i]] += demand
    return lam


def volumes(W_l, P_l, G, d):
    """Eq. 3 for one layer: data volume sent from GPU j to GPU k."""
    E = len(P_l)
    D = [[0.0] * G for _ in range(G)]
    for j in range(G):
        for i in range(E):
            D[j][P_l[i]] += d * W_l[j][i]
    return D


def latency(W, P, G, d, f_comp, f_comm):
    """Eq. 2 + Eq. 4: total computation plus communication latency."""
    total_comp = 0.0
    total_comm = 0.0
    for l in range(len(W)):
        lam = loads(W[l], P[l], G)
        act = active(W[l], P[l], G)
        total_comp += max(comp(f_comp, lam[j], act[j]) for j in range(G))
        D = volumes(W[l], P[l], G, d)
        worst = None
        for j in range(G):
            s = 0.0
            for k in range(G):
                if k != j:
                    s += pwl(f_comm, D[j][k])
            worst = s if worst is None else max(worst, s)
        total_comm += worst
    return total_comp + total_comm


def exhaustive(W, G, C_max, d, f_comp, f_comm):
    """Best one-host-per-expert placement by enumeration (layers are independent
    in Eq. 2 and Eq. 4, so each layer is enumerated on its own)."""
    best_P = []
    best_T = 0.0
    for l in range(len(W)):
        E = len(W[l][0])
        lay_best, lay_T = None, None
        for P_l in itertools.product(range(G), repeat=E):
            if max(P_l.count(j) for j in range(G)) > C_max:
                continue
            T = latency([W[l]], [list(P_l)], G, d, f_comp, f_comm)
            if lay_T is None or T < lay_T:
                lay_best, lay_T = list(P_l), T
        best_P.append(lay_best)
        best_T += lay_T
    return best_P, best_T


def lp_optimum(W, G, C_max, d, f_comp, f_comm):
    """Minimum of sum_l (tau_comp^l + tau_comm^l) over the LP relaxation.

    Variables, in order: x[l][i][j] (L*E*G), tau_comp[l], tau_comm[l], and
    u[l][j][k] for k != j (the epigraph of f_comm per GPU pair).
    Returns (beta_star, x as an array [L][E][G]).
    """
    from scipy.optimize import linprog

    L = len(W)
    E = len(W[0][0])
    nx = L * E * G
    ix = lambda l, i, j: (l * E + i) * G + j
    itc = lambda l: nx + l
    itm = lambda l: nx + L + l
    pairs = [(j, k) for j in range(G) for k in range(G) if k != j]
    iu = lambda l, p: nx + 2 * L + l * len(pairs) + p
    nv = nx + 2 * L + L * len(pairs)

    c = np.zeros(nv)
    for l in range(L):
        c[itc(l)] = 1.0
        c[itm(l)] = 1.0
    A, b = [], []
    for l in range(L):
        demand = [sum(W[l][k][i] for k in range(G)) for i in range(E)]
        for j in range(G):
            # tau_comp >= slope * lambda_j(x) [+ slope_active * a_j(x)] + intercept
            for piece in f_comp:
                a, c_act, b0 = piece if len(piece) == 3 else (piece[0], 0.0, piece[1])
                row = np.zeros(nv)
                for i in range(E):
                    row[ix(l, i, j)] = a * demand[i] + (c_act if demand[i] != 0 else 0.0)
                row[itc(l)] = -1.0
                A.append(row)
                b.append(-b0)
            # tau_comm >= sum_{k != j} u[j][k]
            row = np.zeros(nv)
            for p, (jj, k) in enumerate(pairs):
                if jj == j:
                    row[iu(l, p)] = 1.0
            row[itm(l)] = -1.0
            A.append(row)
            b.append(0.0)
        # u[j][k] >= slope * D_jk(x) + intercept
        for p, (j, k) in enumerate(pairs):
            for a, b0 in f_comm:
                row = np.zeros(nv)
                for i in range(E):
                    row[ix(l, i, k)] = a * d * W[l][j][i]
                row[iu(l, p)] = -1.0
                A.append(row)
                b.append(-b0)
        # every expert hosted at least once: -sum_j x <= -1
        for i in range(E):
            row = np.zeros(nv)
            for j in range(G):
                row[ix(l, i, j)] = -1.0
            A.append(row)
            b.append(-1.0)
        # at most C_max experts per GPU
        for j in range(G):
            row = np.zeros(nv)
            for i in range(E):
                row[ix(l, i, j)] = 1.0
            A.append(row)
            b.append(float(C_max))
    bounds = [(0.0, 1.0)] * nx + [(None, None)] * (nv - nx)
    res = linprog(c, A_ub=np.array(A), b_ub=np.array(b), bounds=bounds, method="highs")
    if res.status != 0:
        raise RuntimeError("LP failed: %s" % res.message)
    return float(res.fun), np.asarray(res.x[:nx]).reshape(L, E, G)
