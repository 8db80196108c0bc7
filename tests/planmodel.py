"""Test-side model of the paper's formulation (Section 4.2), written
independently of the oracle: constraints C1-C5, the objective of Eqs. 5-8,
brute-force optima on tiny instances, and an enumerator of refinement
candidates (Section 4.3, Eq. 10) that checks one committed move at a time.

Arrays use the paper's indices: omega[s, e], x[e, r], q[s, e, r].
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass

import numpy as np


@dataclass
class Topo:
    R: int
    G: int
    E: int
    cI: int
    cX: int
    S: int
    W: int
    N: int
    C: object = None      # general cost matrix [R, R] (the full model of Sec. 4.1), or None
    Wvec: object = None   # ||W_e|| per expert [E], or None (W for every expert)

    @property
    def M(self):
        return self.R // self.G

    @property
    def P(self):
        return self.E // self.R

    def dom(self, r):
        return r // self.G

    def main(self, e):
        return e // self.P

    def w(self, e):
        return int(self.Wvec[e]) if self.Wvec is not None else self.W

    def cost_matrix(self):
        if self.C is not None:
            return np.asarray(self.C, np.int64)
        r = np.arange(self.R)
        same = (r[:, None] // self.G) == (r[None, :] // self.G)
        C = np.where(same, self.cI, self.cX).astype(np.int64)
        np.fill_diagonal(C, 0)
        return C


# ---------------------------------------------------------------- constraints

def check_constraints(t: Topo, omega, x, q, D=None):
    """C1-C5 of Section 4.2.  Raises AssertionError naming the violated one."""
    omega = np.asarray(omega, np.int64)
    x = np.asarray(x, bool)
    q = np.asarray(q, np.int64)
    assert (q >= 0).all(), "q must be nonnegative"
    # C1 token conservation
    assert (q.sum(axis=2) == omega).all(), "C1 violated"
    # C2 instance reachability: q[s,e,r] <= omega[s,e] x[e,r]
    assert (q <= omega[:, :, None] * x[None, :, :]).all(), "C2 violated"
    # C3 replica capacity
    mains = np.zeros_like(x)
    mains[np.arange(t.E), np.arange(t.E) // t.P] = True
    assert ((x & ~mains).sum(axis=0) <= t.N).all(), "C3 violated"
    # C4 cross-domain replica criterion ||W|| < 2 D S
    if D is None:
        D = domain_demand(t, omega)
    for e in range(t.E):
        for r in range(t.R):
            if x[e, r] and t.dom(r) != t.dom(t.main(e)):
                assert t.w(e) < 2 * int(D[t.dom(r), e]) * t.S, "C4 violated"
    # C5 fixed main placement
    assert x[np.arange(t.E), np.arange(t.E) // t.P].all(), "C5 violated"


def domain_demand(t: Topo, omega):
    """Eq. 4 via a reshape-sum (numpy reduction), independent of the oracle."""
    return np.asarray(omega, np.int64).reshape(t.M, t.G, t.E).sum(axis=1)


def loads(q):
    """L_r = sum_s sum_e q[s,e,r]."""
    return np.asarray(q, np.int64).sum(axis=(0, 1))


def objective(t: Topo, x, q, t_ffn=0):
    """Eqs. 5-8: t_FFN L_max + 2 S sum c q + sum_{r != main(e)} c(main(e), r) W x."""
    C = t.cost_matrix()
    q = np.asarray(q, np.int64)
    x = np.asarray(x, bool)
    T_comp = t_ffn * int(loads(q).max()) if q.size else 0
    T_tok = 2 * t.S * int((C[:, None, :] * q).sum())
    T_rep = 0
    for e in range(t.E):
        me = t.main(e)
        for r in range(t.R):
            if r != me and x[e, r]:
                T_rep += int(C[me, r]) * t.w(e)
    return T_comp + T_tok + T_rep


def cross_domain_assignments(t: Topo, q):
    q = np.asarray(q, np.int64)
    r = np.arange(t.R)
    cross = (r[:, None] // t.G) != (r[None, :] // t.G)   # [s, r]
    return int((q * cross[:, None, :]).sum())


# ---------------------------------------------------------------- brute force

def brute_force_opt_no_compute(t: Topo, omega):
    """Exact minimum of Eq. 8 with t_FFN = 0 by enumerating every placement x
    that satisfies C3-C5; for a fixed x the best q sends each assignment to
    its cheapest reachable instance."""
    omega = np.asarray(omega, np.int64)
    C = t.cost_matrix()
    D = domain_demand(t, omega)
    pairs = [(e, r) for e in range(t.E) for r in range(t.R) if r != t.main(e)]
    best = None
    for mask in range(1 << len(pairs)):
        x = np.zeros((t.E, t.R), bool)
        x[np.arange(t.E), np.arange(t.E) // t.P] = True
        ok = True
        for i, (e, r) in enumerate(pairs):
            if mask >> i & 1:
                if t.dom(r) != t.dom(t.main(e)) and not (t.w(e) < 2 * int(D[t.dom(r), e]) * t.S):
                    ok = False
                    break
                x[e, r] = True
        if not ok or ((x.sum(axis=0) - np.bincount(np.arange(t.E) // t.P, minlength=t.R)) > t.N).any():
            continue
        tok = 0
        for s in range(t.R):
            for e in range(t.E):
                if omega[s, e]:
                    tok += int(omega[s, e]) * int(C[s, x[e]].min())
        rep = sum(int(C[t.main(e), r]) * t.w(e) for e in range(t.E) for r in range(t.R)
                  if r != t.main(e) and x[e, r])
        val = 2 * t.S * tok + rep
        if best is None or val < best:
            best = val
    return best


def stage1_best_benefit(t: Topo, D, d):
    """Maximum of sum b over subsets (size <= G N) of the domain's admissible
    candidates (remote main, b > 0): the exact optimum the greedy must hit."""
    bs = []
    for e in range(t.E):
        if t.dom(t.main(e)) == d:
            continue
        b = 2 * int(D[d, e]) * t.S - t.w(e)
        if b > 0:
            bs.append(b)
    cap = t.G * t.N
    best = 0
    for size in range(0, min(cap, len(bs)) + 1):
        for comb in itertools.combinations(bs, size):
            best = max(best, sum(comb))
    return best


# ---------------------------------------------------------------- refinement

def _splits(avail, delta):
    """Every integer vector m with 0 <= m_s <= avail_s and sum m = delta."""
    def rec(i, left):
        if i == len(avail):
            if left == 0:
                yield ()
            return
        for v in range(0, min(avail[i], left) + 1):
            for rest in rec(i + 1, left - v):
                yield (v,) + rest
    yield from rec(0, delta)


def enumerate_candidates(t: Topo, x, q, used, d, brute_split=True):
    """All refinement candidates of domain d in the given state.

    Returns (rb, list of dicts(e, rt, delta, load_t, hosts, dcost, m)).  The
    cost change is measured as objective(after) - objective(before) with
    t_FFN = 0, minimised over every admissible split when ``brute_split``;
    ``m`` is the minimum-cost split that takes as much as possible from
    sources earlier in (c(s,rt) - c(s,rb), s) order.
    """
    q = np.asarray(q, np.int64)
    x = np.asarray(x, bool)
    C = t.cost_matrix()
    L = loads(q)
    ranks = list(range(d * t.G, (d + 1) * t.G))
    rb = max(ranks, key=lambda r: (L[r], -r))
    U = q.sum(axis=0)   # [e, r]
    out = []
    for e in range(t.E):
        if U[e, rb] <= 0:
            continue
        for rt in ranks:
            if rt == rb:
                continue
            hosts = bool(x[e, rt])
            if not hosts and used[rt] >= t.N:
                continue
            delta = min(int(U[e, rb]), (int(L[rb]) - int(L[rt])) // 2)
            if delta < 1:
                continue
            avail = [int(q[s, e, rb]) for s in range(t.R)]
            diff = [int(C[s, rt] - C[s, rb]) for s in range(t.R)]
            rep = 0 if hosts else int(C[t.main(e), rt]) * t.w(e)
            if brute_split:
                best = None
                order = sorted(range(t.R), key=lambda s: (diff[s], s))
                for m in _splits(avail, delta):
                    c = 2 * t.S * sum(m[s] * diff[s] for s in range(t.R)) + rep
                    tieb = tuple(-m[s] for s in order)
                    if best is None or (c, tieb) < best[0]:
                        best = ((c, tieb), m)
                dcost, m = best[0][0], best[1]
            else:
                order = sorted(range(t.R), key=lambda s: (diff[s], s))
                m = [0] * t.R
                left = delta
                for s in order:
                    m[s] = min(left, avail[s])
                    left -= m[s]
                dcost = 2 * t.S * sum(m[s] * diff[s] for s in range(t.R)) + rep
            out.append(dict(e=e, rt=rt, delta=delta, load_t=int(L[rt]), hosts=hosts,
                            dcost=dcost, m=list(m)))
    return rb, out


def best_candidate(cands):
    if not cands:
        return None
    return min(cands, key=lambda c: (-c["delta"], c["load_t"], c["dcost"], c["e"], c["rt"]))
