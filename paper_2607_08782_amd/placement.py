"""Director's relaxation-based expert placement (Sec. VI, Alg. 1), host side.

Given the predicted workload W[l][j][i] (tokens on GPU j routed to expert i in
layer l; per GPU this is what ``moe_expert_histogram`` returns), the per-token
bytes d, the per-GPU capacity C_max and latency models f_comp / f_comm, find a
placement minimising T_comp + T_comm (Eq. 2, Eq. 4, problem of Eq. 5):

1. LP relaxation (Sec. VI-C, Eq. 6a-6f): x[l][i][j] in [0, 1]; every expert
   hosted at least once; at most C_max experts per GPU; the max operators and
   the piecewise-linear latencies in epigraph form (auxiliary tau_comp^l,
   tau_comm^l and one u per GPU pair for f_comm); the budget
   sum_l (tau_comp^l + tau_comm^l) <= beta.  Solved with HiGHS through SciPy,
   as the paper solves its LP with SciPy.
2. Binary search on the budget beta (Alg. 1) between a lower bound (straggler
   load at least the average load; every GPU pays f_comm(0) per peer) and the
   latency of a feasible greedy placement, until the bracket is within a
   relative epsilon; the tightest feasible beta is beta*.
3. Iterative rounding (Sec. VI-C): the LP is solved again at the slack budget
   (1 + eps_round / 2) * beta*, and macro-iterations of a constrained random
   walk drive fractional variables to 0 or 1.  Each macro-iteration gives every
   fractional variable a scale s = 2^-k (min(x, 1-x) in (2^-(k+1), 2^-k]),
   bounds its distance from its integer by alpha * s, keeps the sum of each
   scale class fixed, and takes steps gamma * S g with g a Gaussian direction
   projected (in scaled coordinates) onto the null space of the tight
   constraints; a variable that reaches 0 or 1 is fixed there.
4. The result is made integral with one host per expert: experts the walk left
   fractional (or hosted more than once) are assigned, largest demand first,
   to the candidate GPU (x > 0, capacity left) that adds the least latency.
5. Optional polish (not part of the paper's procedure): single-expert moves
   and pairwise swaps while they strictly lower the exact latency; the
   polished greedy placement is returned instead if it is better.

Latency functions are convex piecewise-linear: pieces (slope, intercept),
f(z) = max over pieces.  ``fit_convex_pwl`` builds one from profiled points.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np
import scipy.sparse as sp
from scipy.optimize import linprog

Pieces = Sequence[Tuple[float, float]]


# ----------------------------------------------------------------------------- model
def pwl_eval(pieces: Pieces, z):
    z = np.asarray(z, dtype=np.float64)
    return np.max([a * z + b for a, b in pieces], axis=0)


def comp_pieces(f_comp):
    """f_comp as (slope of the load, slope of the active-expert count, intercept)
    triples: (slope, intercept) pieces price the load alone."""
    return [(p[0], 0.0, p[1]) if len(p) == 2 else (p[0], p[1], p[2]) for p in f_comp]


def comp_eval(f_comp, lam, act):
    """f_comp of a GPU with load lam and act active experts (hosted experts with
    at least one token): a decode-sized step streams every active expert's
    weights, so its time grows with act as well as with the load (Eq. 2 extended;
    pieces of the load alone give Eq. 2 itself)."""
    lam = np.asarray(lam, dtype=np.float64)
    act = np.asarray(act, dtype=np.float64)
    return np.max([a * lam + c * act + b for a, c, b in comp_pieces(f_comp)], axis=0)


def fit_convex_pwl(z, t) -> List[Tuple[float, float]]:
    """Convex, non-decreasing piecewise-linear model through the lower convex hull of (z, t)."""
    pts = sorted(zip(np.asarray(z, float).tolist(), np.asarray(t, float).tolist()))
    hull: List[Tuple[float, float]] = []
    for p in pts:
        if hull and p[0] == hull[-1][0]:
            if p[1] >= hull[-1][1]:
                continue
            hull.pop()
        while len(hull) >= 2:
            (x1, y1), (x2, y2) = hull[-2], hull[-1]
            if (y2 - y1) * (p[0] - x1) >= (p[1] - y1) * (x2 - x1):   # hull[-1] above the chord
                hull.pop()
            else:
                break
        hull.append(p)
    if len(hull) == 1:
        return [(0.0, hull[0][1])]
    pieces = []
    for (x1, y1), (x2, y2) in zip(hull[:-1], hull[1:]):
        a = (y2 - y1) / (x2 - x1)
        pieces.append((a, y1 - a * x1))
    # a latency does not fall as the load grows: a falling start of the hull
    # (measurement noise at small loads) becomes a flat piece at its minimum
    if pieces[0][0] < 0:
        floor = min(y for _, y in hull)
        pieces = [(0.0, floor)] + [p for p in pieces if p[0] >= 0]
    return pieces


def layer_latencies(W: np.ndarray, P: np.ndarray, d: float, f_comp: Pieces, f_comm: Pieces):
    """Per-layer (comp, comm) latency of an integer placement P[l][i] (Eq. 1-4)."""
    L, G, E = W.shape
    onehot = np.zeros((L, E, G))
    onehot[np.arange(L)[:, None], np.arange(E)[None, :], P] = 1.0
    demand = W.sum(axis=1)                                   # [L][E]
    lam = np.einsum("le,leg->lg", demand, onehot)            # Eq. 1
    act = np.einsum("le,leg->lg", (demand != 0).astype(np.float64), onehot)
    D = d * np.einsum("lje,lek->ljk", W, onehot)             # Eq. 3
    comp = comp_eval(f_comp, lam, act).max(axis=1)
    fc = pwl_eval(f_comm, D)
    fc[:, np.arange(G), np.arange(G)] = 0.0
    comm = fc.sum(axis=2).max(axis=1)
    return comp, comm


def total_latency(W, P, d, f_comp, f_comm) -> float:
    comp, comm = layer_latencies(np.asarray(W, np.float64), np.asarray(P), d, f_comp, f_comm)
    return float(comp.sum() + comm.sum())


# ----------------------------------------------------------------------------- LP
@dataclass
class _LP:
    A: sp.csr_matrix          # A_ub (budget row first)
    b: np.ndarray             # b_ub with the budget entry to be filled in
    nx: int
    nv: int
    bounds: list
    rows_assign: slice
    rows_cap: slice


def _build_lp(W: np.ndarray, d: float, C_max: int, f_comp: Pieces, f_comm: Pieces) -> _LP:
    L, G, E = W.shape
    nx = L * E * G
    pairs = [(j, k) for j in range(G) for k in range(G) if k != j]
    npair = len(pairs)
    itc = nx + np.arange(L)
    itm = nx + L + np.arange(L)
    iu0 = nx + 2 * L
    nv = iu0 + L * npair
    xi = lambda l, i, j: (l * E + i) * G + j
    rows, cols, vals, rhs = [], [], [], []
    r = 0
    # budget: sum_l tau_comp + tau_comm <= beta
    for l in range(L):
        rows += [r, r]; cols += [itc[l], itm[l]]; vals += [1.0, 1.0]
    rhs.append(0.0); r += 1
    demand = W.sum(axis=1)
    for l in range(L):
        for j in range(G):
            for a, c_act, b0 in comp_pieces(f_comp):   # a lambda_j + c a_j + b0 <= tau_comp
                for i in range(E):
                    v = a * demand[l, i] + (c_act if demand[l, i] != 0 else 0.0)
                    if v != 0:
                        rows.append(r); cols.append(xi(l, i, j)); vals.append(v)
                rows.append(r); cols.append(itc[l]); vals.append(-1.0)
                rhs.append(-b0); r += 1
            for p, (jj, k) in enumerate(pairs):        # sum_k u_jk <= tau_comm
                if jj == j:
                    rows.append(r); cols.append(iu0 + l * npair + p); vals.append(1.0)
            rows.append(r); cols.append(itm[l]); vals.append(-1.0)
            rhs.append(0.0); r += 1
        for p, (j, k) in enumerate(pairs):             # slope*D_jk + b0 <= u_jk
            for a, b0 in f_comm:
                for i in range(E):
                    if W[l, j, i] != 0 and a != 0:
                        rows.append(r); cols.append(xi(l, i, k)); vals.append(a * d * W[l, j, i])
                rows.append(r); cols.append(iu0 + l * npair + p); vals.append(-1.0)
                rhs.append(-b0); r += 1
    a0 = r
    for l in range(L):                                  # -sum_j x <= -1
        for i in range(E):
            for j in range(G):
                rows.append(r); cols.append(xi(l, i, j)); vals.append(-1.0)
            rhs.append(-1.0); r += 1
    c0 = r
    for l in range(L):                                  # sum_i x <= C_max
        for j in range(G):
            for i in range(E):
                rows.append(r); cols.append(xi(l, i, j)); vals.append(1.0)
            rhs.append(float(C_max)); r += 1
    A = sp.csr_matrix((vals, (rows, cols)), shape=(r, nv))
    bounds = [(0.0, 1.0)] * nx + [(None, None)] * (nv - nx)
    return _LP(A, np.array(rhs), nx, nv, bounds, slice(a0, c0), slice(c0, r))


def _feasible(lp: _LP, beta: float, c: Optional[np.ndarray] = None):
    """A point of the LP at budget beta, or (None, None) when there is none.  If the
    solver cannot decide (numerical trouble), the interior-point method is tried;
    a budget still undecided is treated as infeasible, which only keeps the binary
    search's upper end at a budget known to be feasible."""
    b = lp.b.copy()
    b[0] = beta
    obj = np.zeros(lp.nv) if c is None else c
    for method in ("highs", "highs-ipm"):
        res = linprog(obj, A_ub=lp.A, b_ub=b, bounds=lp.bounds, method=method)
        if res.status == 0:
            return np.clip(res.x[:lp.nx], 0.0, 1.0), res.x
        if res.status == 2:
            return None, None
    return None, None


# ----------------------------------------------------------------------------- rounding
def _scales(v):
    m = np.minimum(v, 1.0 - v)
    k = np.floor(-np.log2(np.maximum(m, 1e-300)))
    return np.exp2(-np.maximum(k, 1.0))


def _walk(x0: np.ndarray, A_in: sp.csr_matrix, b_in: np.ndarray, rng: np.random.Generator,
          alpha: float, gamma: float, t_micro: int, max_macro: int, tol: float = 1e-9):
    """Constrained random walk on x subject to A_in x <= b_in and 0 <= x <= 1."""
    x = x0.copy()
    n = x.size
    fixed = (x <= tol) | (x >= 1.0 - tol)
    x[fixed] = np.round(x[fixed])
    A = A_in.tocsc()
    stats = {"macro": 0, "steps": 0, "fractional_start": int((~fixed).sum())}
    for _ in range(max_macro):
        F = np.flatnonzero(~fixed)
        if F.size == 0:
            break
        stats["macro"] += 1
        s = np.ones(n)
        s[F] = _scales(x[F])
        near_one = x > 0.5
        kcls = np.round(-np.log2(s)).astype(int)
        classes = {k: np.flatnonzero((~fixed) & (kcls == k)) for k in np.unique(kcls[F])}
        for _ in range(t_micro):
            F = np.flatnonzero(~fixed)
            if F.size == 0:
                break
            xF = x[F]
            AF = A[:, F].tocsr()
            slack = b_in - A @ x
            tight = np.flatnonzero(slack <= 1e-9 * (1.0 + np.abs(b_in)))
            # variables pinned at their scale bound cannot move further out
            dist = np.where(near_one[F], 1.0 - xF, xF)
            movable = dist < alpha * s[F] - 1e-12
            rowsC = [AF[tight].toarray()] if tight.size else []
            for k, idx in classes.items():
                row = np.zeros(F.size)
                row[np.isin(F, idx)] = 1.0
                if row.any():
                    rowsC.append(row[None, :])
            C = np.vstack(rowsC) if rowsC else np.zeros((0, F.size))
            sF = s[F] * movable
            if not sF.any():
                break
            CS = C * sF[None, :]
            r = rng.standard_normal(F.size) * (sF > 0)
            if CS.shape[0]:
                # orthonormal basis of the tight normals (scaled coordinates)
                u, sv, _ = np.linalg.svd(CS.T, full_matrices=False)
                u = u[:, sv > 1e-10 * max(1.0, sv[0] if sv.size else 1.0)]
                r = r - u @ (u.T @ r)
            g = sF * r
            if np.linalg.norm(g) < 1e-12:
                break
            # largest step in (0, gamma] that keeps every constraint (tight rows
            # are orthogonal to g and are left out of the ratio test)
            t = gamma
            Ag = AF @ g
            pos = Ag > 1e-15
            pos[tight] = False
            if pos.any():
                t = min(t, float(np.min(np.maximum(slack[pos], 0.0) / Ag[pos])))
            up, dn = g > 0, g < 0
            if up.any():
                t = min(t, float(np.min((1.0 - xF[up]) / g[up])))
            if dn.any():
                t = min(t, float(np.min(xF[dn] / -g[dn])))
            # scale bounds: distance from the integer at most alpha * s
            away = np.where(near_one[F], -g, g)
            grow = away > 0
            if grow.any():
                t = min(t, float(np.min(np.maximum(alpha * s[F][grow] - dist[grow], 0.0) / away[grow])))
            x[F] = xF + t * g
            stats["steps"] += 1
            hit0 = x[F] <= tol
            hit1 = x[F] >= 1.0 - tol
            x[F[hit0]] = 0.0
            x[F[hit1]] = 1.0
            fixed[F[hit0 | hit1]] = True
    stats["fractional_end"] = int((~fixed).sum())
    return x, stats


def _min_aux(xl: np.ndarray, W: np.ndarray, d, f_comp, f_comm) -> np.ndarray:
    """Smallest auxiliaries (tau_comp, tau_comm, u per GPU pair) for a fractional x."""
    L, E, G = xl.shape
    demand = W.sum(axis=1)
    lam = np.einsum("le,leg->lg", demand, xl)
    act = np.einsum("le,leg->lg", (demand != 0).astype(np.float64), xl)
    D = d * np.einsum("lje,lek->ljk", W, xl)
    u = pwl_eval(f_comm, D)
    off = ~np.eye(G, dtype=bool)
    tau_c = comp_eval(f_comp, lam, act).max(axis=1)
    tau_m = np.where(off[None], u, 0.0).sum(axis=2).max(axis=1)
    u_pairs = u[:, off]                                       # (j, k != j), j-major
    return np.concatenate([tau_c, tau_m, u_pairs.reshape(-1)])


def _complete(xl: np.ndarray, W: np.ndarray, d, C_max, f_comp, f_comm) -> np.ndarray:
    """Integral placement with one host per expert from a (partly) rounded x."""
    L, E, G = xl.shape
    P = np.full((L, E), -1, dtype=np.int64)
    for l in range(L):
        used = np.zeros(G, dtype=np.int64)
        ones = xl[l] >= 1.0 - 1e-9
        for i in range(E):
            if ones[i].sum() == 1:
                j = int(np.argmax(ones[i]))
                P[l, i] = j
                used[j] += 1
        demand = W[l].sum(axis=0)
        for i in sorted(np.flatnonzero(P[l] < 0), key=lambda i: -demand[i]):
            cand = [j for j in range(G) if xl[l, i, j] > 1e-9 and used[j] < C_max]
            if not cand:
                cand = [j for j in range(G) if used[j] < C_max]
            best, best_t = None, None
            for j in cand:
                P[l, i] = j
                part = P[l] >= 0
                Wp = W[l][:, part][None]
                c, m = layer_latencies(Wp, P[l][part][None], d, f_comp, f_comm)
                if best_t is None or c[0] + m[0] < best_t:
                    best, best_t = j, c[0] + m[0]
            P[l, i] = best
            used[best] += 1
    return P


def _polish(P: np.ndarray, W: np.ndarray, d, C_max, f_comp, f_comm, max_passes: int = 50):
    """Local descent on the exact latency: move one expert, or swap two, while
    that strictly lowers the layer's T_comp + T_comm."""
    L, G, E = W.shape
    P = P.copy()
    moves = 0
    for l in range(L):
        Wl = W[l][None]
        def cur():
            c, m = layer_latencies(Wl, P[l][None], d, f_comp, f_comm)
            return float(c[0] + m[0])
        best = cur()
        for _ in range(max_passes):
            improved = False
            used = np.bincount(P[l], minlength=G)
            for i in range(E):
                src = P[l, i]
                for j in range(G):
                    if j == src or used[j] >= C_max:
                        continue
                    P[l, i] = j
                    t = cur()
                    if t < best - 1e-12:
                        best, improved = t, True
                        used[src] -= 1
                        used[j] += 1
                        src = j
                        moves += 1
                    else:
                        P[l, i] = src
            for i in range(E):
                for k in range(i + 1, E):
                    if P[l, i] == P[l, k]:
                        continue
                    P[l, i], P[l, k] = P[l, k], P[l, i]
                    t = cur()
                    if t < best - 1e-12:
                        best, improved = t, True
                        moves += 1
                    else:
                        P[l, i], P[l, k] = P[l, k], P[l, i]
            if not improved:
                break
    return P, moves


def _greedy(W: np.ndarray, d, C_max, f_comp, f_comm) -> np.ndarray:
    L, G, E = W.shape
    return _complete(np.ones((L, E, G)) * 0.5, W, d, C_max, f_comp, f_comm)


# ----------------------------------------------------------------------------- driver
@dataclass
class PlacementResult:
    P: np.ndarray                     # [L][E] host GPU of each expert
    x: np.ndarray                     # [L][E][G] uint8 placement map (moe_permute's form)
    beta_star: float                  # LP optimum found by the binary search
    latency: float                    # T_comp + T_comm of P (Eq. 2 + Eq. 4)
    info: dict = field(default_factory=dict)


def place(W, G: int, C_max: int, d: float, f_comp: Pieces, f_comm: Pieces, eps: float = 1e-3,
          eps_round: float = 0.05, alpha: float = 2.0, gamma: float = 0.25,
          t_micro: Optional[int] = None, max_macro: Optional[int] = None,
          n_starts: int = 4, polish: bool = True, seed: int = 0) -> PlacementResult:
    """Alg. 1: binary search on the LP budget, then iterative rounding."""
    t0 = time.perf_counter()
    W = np.asarray(W, dtype=np.float64)
    if W.ndim == 2:
        W = W[None]
    L, G_, E = W.shape
    if G_ != G:
        raise ValueError("W must be [L][G][E]")
    if C_max * G < E:
        raise ValueError("C_max * G < E: some expert cannot be hosted")
    lp = _build_lp(W, d, C_max, f_comp, f_comm)
    P0 = _greedy(W, d, C_max, f_comp, f_comm)
    hi = total_latency(W, P0, d, f_comp, f_comm)
    demand = W.sum(axis=(1, 2))
    if all(c >= 0 for _, c, _ in comp_pieces(f_comp)):
        # the straggler's f_comp is at least f_comp of the mean load and of the mean
        # active-expert count (convex and non-decreasing in the count), every
        # expert with tokens being active somewhere
        n_act = (W.sum(axis=1) != 0).sum(axis=1)
        lo = float(np.sum(comp_eval(f_comp, demand / G, n_act / G)) +
                   L * (G - 1) * float(pwl_eval(f_comm, 0.0)))
    else:
        lo = 0.0
    lo = min(lo, hi) * (1.0 - 1e-12)
    x_best, _ = _feasible(lp, hi)
    if x_best is None:
        raise RuntimeError("the greedy placement's latency should be a feasible budget")
    solves = 1
    while hi - lo > eps * hi:
        mid = 0.5 * (lo + hi)
        x, _ = _feasible(lp, mid)
        solves += 1
        if x is None:
            lo = mid
        else:
            hi, x_best = mid, x
    beta_star = hi
    t_search = time.perf_counter() - t0
    # rounding starts from the LP at the slack budget (1 + eps_round / 2) * beta*
    beta_r = (1.0 + 0.5 * eps_round) * beta_star
    # start the walk inside the feasible set rather than at a vertex (where the
    # tight constraints leave no direction to move in): the mean of vertices
    # reached from random objectives over x is feasible and mostly fractional
    rng = np.random.default_rng(seed)
    x_r, full = _feasible(lp, beta_r)
    solves += 1
    n_avg = 1
    for _ in range(n_starts):
        c = np.zeros(lp.nv)
        c[:lp.nx] = rng.standard_normal(lp.nx)
        xv, fv = _feasible(lp, beta_r, c)
        solves += 1
        x_r, full, n_avg = x_r + xv, full + fv, n_avg + 1
    x_r, full = x_r / n_avg, full / n_avg
    # freeze the auxiliaries: spread the budget slack over the latency terms so
    # the walk runs in x alone inside {A_x x <= b - A_aux aux}
    aux = _min_aux(x_r.reshape(L, E, G), W, d, f_comp, f_comm)
    nx = lp.nx
    A = lp.A.tocsc()
    Ax, Aaux = A[:, :nx].tocsr(), A[:, nx:].tocsr()
    spent = float(aux[:2 * L].sum())
    if spent > 0:
        scale = beta_r / spent        # >= 1: x_r is feasible at beta_r
        aux[:2 * L] *= scale
        aux[2 * L:] *= scale          # per-pair terms under tau_comm grow with it
    b_in = lp.b.copy()
    b_in[0] = beta_r
    b_in = b_in - Aaux @ aux
    keep = np.ones(lp.A.shape[0], bool)
    keep[0] = False                       # the budget row only involves auxiliaries
    nvars = int(np.sum((x_r > 1e-9) & (x_r < 1 - 1e-9)))
    x_w, stats = _walk(x_r, Ax[keep], b_in[keep], rng, alpha, gamma,
                       t_micro if t_micro is not None else max(50, 4 * nvars),
                       max_macro if max_macro is not None else max(1, int(np.ceil(2 * np.log2(max(nvars, 2))))))
    P = _complete(x_w.reshape(L, E, G), W, d, C_max, f_comp, f_comm)
    T_rounded = total_latency(W, P, d, f_comp, f_comm)
    moves = 0
    source = "rounding"
    if polish:
        P, moves = _polish(P, W, d, C_max, f_comp, f_comm)
        # safeguard: the polished greedy placement if it happens to be better
        Pg, _ = _polish(P0, W, d, C_max, f_comp, f_comm)
        if total_latency(W, Pg, d, f_comp, f_comm) < total_latency(W, P, d, f_comp, f_comm):
            P, source = Pg, "greedy"
    xmap = np.zeros((L, E, G), dtype=np.uint8)
    xmap[np.arange(L)[:, None], np.arange(E)[None, :], P] = 1
    T = total_latency(W, P, d, f_comp, f_comm)
    info = {"lp_solves": solves, "beta_greedy": float(total_latency(W, P0, d, f_comp, f_comm)),
            "beta_rounding": beta_r, "latency_rounded": T_rounded, "polish_moves": moves,
            "source": source,
            "search_s": t_search, "total_s": time.perf_counter() - t0, "walk": stats}
    return PlacementResult(P=P, x=xmap, beta_star=beta_star, latency=T, info=info)
