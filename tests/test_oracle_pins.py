"""Pins of the oracle against the mathematics of the paper's formulation
(Section 4.2) and solver (Section 4.3), on seeded random tiny instances.

Each check uses something other than the oracle's own code: numpy library
routines (bincount, reshape-sum, stable argsort), the constraints C1-C5, the
objective of Eqs. 5-8 evaluated on dense arrays, brute-force optima and an
independent enumerator of refinement candidates.
"""
import itertools

import numpy as np
import pytest

import oracle
from planmodel import (Topo, best_candidate, brute_force_opt_no_compute, check_constraints,
                       cross_domain_assignments, domain_demand, enumerate_candidates, loads,
                       objective, stage1_best_benefit)


def random_instance(seed, R=None, G=None, P=None, N=None, k=None, big=False, general=False):
    """A tiny instance whose every rank's top-k array is simulated; with
    general, a random symmetric cost matrix (zero diagonal) and a random
    size per expert (the full model of Section 4.1)."""
    rng = np.random.default_rng(seed)
    if G is None:
        G = int(rng.choice([1, 2, 3, 4]))
    if R is None:
        R = G * int(rng.choice([1, 2, 3]))
    if P is None:
        P = int(rng.choice([1, 2, 3]))
    E = R * P
    if N is None:
        N = int(rng.integers(0, 4))
    if k is None:
        k = int(rng.integers(1, min(E, 3) + 1))
    cI = int(rng.integers(0, 3))
    cX = int(rng.integers(cI, 7))
    S = int(rng.integers(1, 5))
    # skewed popularity, some experts hot
    pop = rng.dirichlet(np.full(E, 0.3))
    topks = []
    for s in range(R):
        T = int(rng.integers(0, 40 if big else 14))
        ids = rng.choice(E, size=(T, k), p=pop).astype(np.int32)
        topks.append(ids)
    omega = np.stack([np.bincount(t.ravel(), minlength=E) for t in topks]).astype(np.int32)
    Dmax = max(1, int(domain_demand(Topo(R, G, E, cI, cX, S, 0, N), omega).max()))
    W = int(rng.integers(0, 2 * S * Dmax + 2))
    t = Topo(R, G, E, cI, cX, S, W, N)
    if general:
        C = np.triu(rng.integers(0, 9, size=(R, R)), 1)
        t.C = (C + C.T).astype(np.int32)
        t.Wvec = rng.integers(0, 2 * S * Dmax + 2, size=E).astype(np.int64)
    return t, omega, topks


def run(t, omega, topk, self_rank, **kw):
    topo = oracle.topology(t.R, t.G, t.E, self_rank, t.cI, t.cX, t.S, t.W)
    return oracle.plan_ref(topo, omega, topk, t.N, cost_matrix=t.C, expert_bytes=t.Wvec, **kw)


SEEDS = list(range(60))


@pytest.mark.parametrize("seed", SEEDS)
def test_histogram_and_demand(seed):
    t, omega, topks = random_instance(seed)
    s = seed % t.R
    out = run(t, omega, topks[s], s, debug=True, move_cap=1000)
    assert out["status"] == 0
    assert (out["hist"] == np.bincount(topks[s].ravel(), minlength=t.E)).all()
    D = domain_demand(t, omega)
    assert (out["demand"] == D).all()
    assert (D.sum(axis=0) == omega.sum(axis=0)).all()


@pytest.mark.parametrize("general", [False, True])
@pytest.mark.parametrize("seed", SEEDS)
def test_stage1_placement(seed, general):
    """Inter-node placement (Eq. 9): greedy sum of b is the subset optimum, the
    ranks follow 'least occupied rank with a free slot', C3-C5 hold."""
    t, omega, topks = random_instance(seed, N=int(np.random.default_rng(seed).integers(0, 3)), general=general)
    out = run(t, omega, topks[0], 0, debug=True, move_cap=1000)
    x1 = out["x_stage1"].astype(bool)
    D = domain_demand(t, omega)
    mains = np.zeros_like(x1)
    mains[np.arange(t.E), np.arange(t.E) // t.P] = True
    reps = x1 & ~mains
    for d in range(t.M):
        ranks = range(d * t.G, (d + 1) * t.G)
        chosen = [e for e in range(t.E) if reps[e, list(ranks)].any()]
        # at most one replica per (domain, expert), only remote mains with b > 0
        for e in chosen:
            assert reps[e, list(ranks)].sum() == 1
            assert t.dom(t.main(e)) != d
            assert 2 * int(D[d, e]) * t.S - t.w(e) > 0
        total_b = sum(2 * int(D[d, e]) * t.S - t.w(e) for e in chosen)
        assert total_b == stage1_best_benefit(t, D, d)
        # closed form of 'fewest used slots, ties to the lowest rank': the i-th
        # chosen candidate in (b desc, e asc) order lands on rank dG + i mod G,
        # slot i div G
        order = sorted(chosen, key=lambda e: (-(2 * int(D[d, e]) * t.S - t.w(e)), e))
        for i, e in enumerate(order):
            r = d * t.G + i % t.G
            assert reps[e, r]
            assert out["replica_slots"][r, i // t.G] == e
    check_constraints(t, omega, x1, out["q_routed"])


@pytest.mark.parametrize("seed", SEEDS)
def test_routing_construction(seed):
    """Routing after stage 1: C1/C2, same-domain preference, even split with
    the remainder on the lowest ranks."""
    t, omega, topks = random_instance(seed)
    out = run(t, omega, topks[0], 0, debug=True, move_cap=1000)
    x1 = out["x_stage1"].astype(bool)
    q = out["q_routed"].astype(np.int64)
    check_constraints(t, omega, x1, q)
    for s in range(t.R):
        for e in range(t.E):
            w = int(omega[s, e])
            hosts = np.nonzero(x1[e])[0]
            local = [r for r in hosts if t.dom(r) == t.dom(s)]
            sel = local if local else list(hosts)
            got = q[s, e]
            assert got[[r for r in range(t.R) if r not in sel]].sum() == 0
            share = got[sel]
            n = len(sel)
            assert share.tolist() == [w // n + (1 if i < w % n else 0) for i in range(n)]
    assert (loads(q) == out["load_routed"]).all()


@pytest.mark.parametrize("general", [False, True])
@pytest.mark.parametrize("seed", SEEDS)
def test_refinement_steps(seed, general):
    """Replay every committed move of the intra-node refinement (Eq. 10)
    against an independent enumerator: the chosen candidate is the key
    minimum, its split is a minimum-cost split, its cost change equals the
    change of Eqs. 6-7, and the invariants of Section 4.3 hold."""
    rng = np.random.default_rng(1000 + seed)
    t, omega, topks = random_instance(1000 + seed, N=int(rng.integers(1, 4)), big=True, general=general)
    out = run(t, omega, topks[0], 0, debug=True, move_cap=10000)
    assert out["n_moves"] <= 10000
    x = out["x_stage1"].astype(bool).copy()
    q = out["q_routed"].astype(np.int64).copy()
    mains = np.zeros_like(x)
    mains[np.arange(t.E), np.arange(t.E) // t.P] = True
    used = (x & ~mains).sum(axis=0)
    cross0 = cross_domain_assignments(t, q)
    D = domain_demand(t, omega)
    i = 0
    for d in range(t.M):
        for _ in range(int(out["iters"][d])):
            dd, rb, rt, e, delta, created = out["moves"][i].tolist()
            assert dd == d
            avail = [int(q[s, e, rb]) for s in range(t.R)]
            small = np.prod([a + 1 for a in avail], dtype=float) <= 5000
            rb_e, cands = enumerate_candidates(t, x, q, used, d, brute_split=small)
            assert rb_e == rb
            best = best_candidate(cands)
            assert best is not None
            assert (best["e"], best["rt"], best["delta"], best["hosts"]) == (e, rt, delta, not created)
            m = out["move_m"][i].astype(np.int64)
            assert m.tolist() == best["m"]
            assert m.sum() == delta and (m >= 0).all()
            L_pre = loads(q)
            pre = objective(t, x, q)
            if created:
                assert not x[e, rt] and used[rt] < t.N
                x[e, rt] = True
                used[rt] += 1
            q[:, e, rb] -= m
            q[:, e, rt] += m
            post = objective(t, x, q)
            assert post - pre == int(out["move_dcost"][i]) == best["dcost"]
            L = loads(q)
            assert L[rb] >= L[rt]                                  # order not reversed
            assert (L.astype(np.int64) ** 2).sum() < (L_pre.astype(np.int64) ** 2).sum()
            assert cross_domain_assignments(t, q) == cross0        # no new cross-domain routes
            check_constraints(t, omega, x, q, D)
            i += 1
        # stop rule: the busiest rank of the domain has no candidate left
        _, cands = enumerate_candidates(t, x, q, used, d, brute_split=False)
        assert best_candidate(cands) is None
    assert i == out["n_moves"]
    # the second status word reports the same count (each iteration commits one move)
    assert out["move_count"] == out["n_moves"] == int(out["iters"].sum())
    assert (q == out["q_final"]).all()
    assert (x == out["x_final"].astype(bool)).all()
    assert (loads(q) == out["load_final"]).all()


def _stable_dest(t, topk, q_self):
    """Destinations by the stable-argsort construction: occurrences of each
    expert in row-major order, sliced by the per-instance counts in ascending
    rank order."""
    ids = topk.ravel()
    dest = np.full(ids.size, -1, np.int64)
    order = np.argsort(ids, kind="stable")
    start = 0
    for e in range(t.E):
        cnt = int((ids == e).sum())
        seq = np.repeat(np.arange(t.R), q_self[e].astype(np.int64))
        assert seq.size == cnt
        dest[order[start:start + cnt]] = seq
        start += cnt
    return dest.reshape(topk.shape)


@pytest.mark.parametrize("seed", SEEDS)
def test_rerouting_and_cross_rank(seed):
    """Every rank derives the same replica slots; each rank's destinations
    follow the stable construction; send counts add up to the rank loads."""
    t, omega, topks = random_instance(2000 + seed, big=True)
    slots0 = None
    total = np.zeros(t.R, np.int64)
    for s in range(t.R):
        out = run(t, omega, topks[s], s, debug=True, move_cap=10000)
        assert out["status"] == 0
        if slots0 is None:
            slots0 = out["replica_slots"].copy()
            L = out["load_final"]
        assert (out["replica_slots"] == slots0).all()
        q_self = out["q_final"][s]
        dest = out["token_dest"]
        assert (dest == _stable_dest(t, topks[s], q_self)).all()
        assert (np.bincount(dest.ravel(), minlength=t.R) == out["send_counts"]).all()
        assert out["send_counts"].sum() == topks[s].size
        # every destination hosts its expert
        xf = out["x_final"].astype(bool)
        assert xf[topks[s].ravel(), dest.ravel()].all() if dest.size else True
        total += out["send_counts"]
    assert (total == L).all()


@pytest.mark.parametrize("seed", range(20))
def test_static_ep_without_slots(seed):
    """N = 0: no replicas, every assignment goes to its expert's main."""
    t, omega, topks = random_instance(3000 + seed, N=0)
    out = run(t, omega, topks[0], 0)
    assert (out["replica_slots"].size == 0)
    assert (out["token_dest"] == topks[0] // t.P).all()


@pytest.mark.parametrize("seed", range(20))
def test_single_domain_has_no_stage1(seed):
    """M = 1: every main is inside the only domain, stage 1 places nothing."""
    rng = np.random.default_rng(seed)
    G = int(rng.choice([2, 3, 4]))
    t, omega, topks = random_instance(4000 + seed, R=G, G=G, N=int(rng.integers(1, 3)))
    out = run(t, omega, topks[0], 0, debug=True, move_cap=1000)
    x1 = out["x_stage1"].astype(bool)
    assert x1.sum() == t.E


@pytest.mark.parametrize("seed", range(40))
def test_one_gpu_per_node_reaches_the_optimum(seed):
    """G = 1 and t_FFN = 0: refinement has nothing to do and the plan's
    objective (Eqs. 6-8) equals the brute-force optimum over all placements."""
    rng = np.random.default_rng(5000 + seed)
    R = int(rng.choice([2, 3]))
    P = 1 if R == 3 else int(rng.choice([1, 2]))
    t, omega, topks = random_instance(5000 + seed, R=R, G=1, P=P, N=int(rng.integers(0, 2)))
    out = run(t, omega, topks[0], 0, debug=True, move_cap=1000)
    assert out["n_moves"] == 0
    got = objective(t, out["x_final"], out["q_final"])
    assert got == brute_force_opt_no_compute(t, omega)


@pytest.mark.parametrize("seed", range(20))
def test_balanced_static_plan_is_kept(seed):
    """Equal rank loads and no profitable replica: the plan is static EP,
    which is optimal (L_max equals the mean, no transfer)."""
    rng = np.random.default_rng(6000 + seed)
    G = int(rng.choice([1, 2, 4]))
    R = G * int(rng.choice([1, 2]))
    P = int(rng.choice([1, 2]))
    E = R * P
    per = int(rng.integers(1, 6))
    omega = np.zeros((R, E), np.int32)
    # every source sends 'per' assignments to each expert of its own rank only
    for s in range(R):
        omega[s, s * P:(s + 1) * P] = per
    S = 2
    W = 2 * per * G * S  # b <= 0 for every remote (d, e): D <= per * G
    t = Topo(R, G, E, 1, 3, S, W, int(rng.integers(0, 3)))
    topk = np.repeat(np.arange(P, dtype=np.int32), per).reshape(-1, 1)
    out = run(t, omega, topk, 0, debug=True, move_cap=100)
    assert (out["replica_slots"] == -1).all()
    assert out["n_moves"] == 0
    assert objective(t, out["x_final"], out["q_final"]) == 0


# ---------------------------------------------------------------- dispatch layout

@pytest.mark.parametrize("seed", SEEDS)
def test_receive_counts_match_every_senders_plan(seed):
    """Every rank makes the same plan, so what rank r expects from rank s
    (its receive count) is what rank s's own plan sends to r; the counts a
    rank receives add up to its final load."""
    t, omega, topks = random_instance(5000 + seed, big=True)
    outs = [run(t, omega, topks[s], s, debug=True) for s in range(t.R)]
    for r in range(t.R):
        assert outs[r]["status"] == 0
        for s in range(t.R):
            assert outs[r]["recv_counts"][s] == outs[s]["send_counts"][r], (r, s)
        assert outs[r]["recv_counts"].sum() == outs[r]["load_final"][r]


def _layout_by_sort(R, dest, send_counts):
    """The send buffer by a stable argsort on the destination: position of
    each assignment in that order, -1 for a non-rank destination."""
    d = dest.ravel().astype(np.int64)
    ok = (d >= 0) & (d < R)
    key = np.where(ok, d, R)              # invalid ones sort last
    order = np.argsort(key, kind="stable")
    slot = np.empty(d.size, np.int64)
    slot[order] = np.arange(d.size)
    slot[~ok] = -1
    offs = np.concatenate([[0], np.cumsum(np.bincount(d[ok], minlength=R))])
    return offs, slot.reshape(dest.shape)


@pytest.mark.parametrize("seed", SEEDS)
def test_dispatch_layout_is_the_stable_sort_by_destination(seed):
    t, omega, topks = random_instance(6000 + seed, big=True)
    s = seed % t.R
    out = run(t, omega, topks[s], s)
    offs, slot = oracle.layout_ref(t.R, out["token_dest"], out["send_counts"])
    ref_offs, ref_slot = _layout_by_sort(t.R, out["token_dest"], out["send_counts"])
    assert (offs == ref_offs).all()
    assert (slot == ref_slot).all()
    # every slot of [0, T k) is used once
    assert np.array_equal(np.sort(slot.ravel()), np.arange(slot.size))


def test_dispatch_layout_special_cases():
    # destinations that are not ranks keep slot -1 and take no room
    dest = np.array([[2, -1], [0, 2], [5, 0]], np.int32)
    offs, slot = oracle.layout_ref(3, dest, np.array([2, 0, 2], np.int32))
    assert offs.tolist() == [0, 2, 2, 4]
    assert slot.tolist() == [[2, -1], [0, 3], [-1, 1]]
    # one destination: the slot is the row-major index
    dest = np.zeros((5, 3), np.int32)
    offs, slot = oracle.layout_ref(4, dest, np.array([15, 0, 0, 0], np.int32))
    assert offs.tolist() == [0, 15, 15, 15, 15]
    assert (slot.ravel() == np.arange(15)).all()
    # empty batch
    offs, slot = oracle.layout_ref(2, np.zeros((0, 2), np.int32), np.zeros(2, np.int32))
    assert offs.tolist() == [0, 0, 0] and slot.shape == (0, 2)


def test_receive_counts_without_a_plan():
    t, omega, topks = random_instance(77, big=True)
    om = omega.copy()
    om[0, 0] = -1
    out = run(t, om, topks[0], 0)
    assert out["status"] & oracle.ST_NEG_LOAD
    assert (out["recv_counts"] == 0).all()


# ---------------------------------------------------------------- replica-slot gather

def test_gather_matches_fancy_indexing_and_keeps_other_slots():
    """The gather against numpy fancy indexing, on parameters whose every
    row encodes its expert id, with empty slots and unchanged slots."""
    rng = np.random.default_rng(4)
    R, E, N, W = 6, 12, 3, 40
    params = (np.arange(E, dtype=np.int64)[:, None] * 1000 + np.arange(W)).astype(np.int32)
    slots = rng.integers(-1, E, size=(R, N)).astype(np.int32)
    slots[2] = [5, -1, 11]
    before = rng.integers(-9, 0, size=(N, W)).astype(np.int32)
    out = oracle.gather_ref(slots, 2, params, before)
    assert (out[0] == params[5]).all() and (out[2] == params[11]).all()
    assert (out[1] == before[1]).all()              # empty slot untouched
    assert (out[0] // 1000 == 5).all()
    filled = slots[2] >= 0
    assert (out[filled] == params[slots[2][filled]]).all()
    # a slot whose expert is unchanged is not copied
    out2 = oracle.gather_ref(slots, 2, params, before, prev_slots=np.array([5, 7, 3], np.int32))
    assert (out2[0] == before[0]).all() and (out2[2] == params[11]).all()


# ---------------------------------------------------------------- general cost model

@pytest.mark.parametrize("seed", range(30))
def test_general_model_with_two_level_costs_is_the_two_level_plan(seed):
    """The two-level matrix and one size for every expert, given explicitly,
    give exactly the plan of the two-level parameters."""
    t, omega, topks = random_instance(3300 + seed, big=True)
    s = seed % t.R
    a = run(t, omega, topks[s], s)
    t.C = t.cost_matrix().astype(np.int32)
    t.Wvec = np.full(t.E, t.W, np.int64)
    b = run(t, omega, topks[s], s)
    for key in ("replica_slots", "token_dest", "send_counts", "recv_counts"):
        assert (a[key] == b[key]).all(), key
    assert (a["status"], a["move_count"]) == (b["status"], b["move_count"])


@pytest.mark.parametrize("seed", range(20))
def test_general_model_conservation_and_receive_counts(seed):
    """C1-C5 on the final plan and every rank's receive counts against every
    sender's own plan, under a general cost matrix and per-expert sizes."""
    t, omega, topks = random_instance(3400 + seed, big=True, general=True)
    outs = [run(t, omega, topks[s], s, debug=True) for s in range(t.R)]
    for r in range(t.R):
        assert outs[r]["status"] == 0
        assert (outs[r]["replica_slots"] == outs[0]["replica_slots"]).all()
        for s in range(t.R):
            assert outs[r]["recv_counts"][s] == outs[s]["send_counts"][r]
    check_constraints(t, omega, outs[0]["x_final"], outs[0]["q_final"])


def test_invalid_cost_model_makes_no_plan():
    t, omega, topks = random_instance(77, big=True, general=True)
    good = t.C.copy()
    bad_cases = []
    c = good.copy(); c[0, 1] += 1; bad_cases.append(("asymmetric", c, t.Wvec))
    c = good.copy(); c[1, 1] = 2; bad_cases.append(("diagonal", c, t.Wvec))
    c = good.copy(); c[0, 1] = c[1, 0] = -1; bad_cases.append(("negative", c, t.Wvec))
    w = t.Wvec.copy(); w[3] = -5; bad_cases.append(("negative size", good, w))
    for what, C, W in bad_cases:
        t.C, t.Wvec = C, W
        out = run(t, omega, topks[0], 0)
        assert out["status"] & oracle.ST_COST, what
        assert (out["replica_slots"] == -1).all() and (out["send_counts"] == 0).all(), what
        assert (out["token_dest"] == -1).all() and (out["recv_counts"] == 0).all(), what
