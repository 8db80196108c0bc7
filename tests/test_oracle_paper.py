"""Pins of the oracle against numbers the paper prints.

* The two-stage worked example of Section 4.3 (golden/worked_example.json).
* The placement-cost example of Section 2.3 and the benefit of Eq. 9 at its
  sign boundary (golden/placement_cost.json).
"""
import json
import os

import numpy as np
import pytest

import oracle
from planmodel import Topo, check_constraints, cross_domain_assignments

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _topk_from_row(row):
    ids = []
    for e, c in enumerate(row):
        ids += [e] * int(c)
    return np.array(ids, np.int32).reshape(-1, 1)


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


@pytest.mark.parametrize("self_rank", [0, 1, 2, 3])
def test_worked_example(self_rank):
    g = _load("worked_example.json")
    tp, exp = g["topology"], g["expected"]
    omega = np.array(g["omega"], np.int32)
    topo = oracle.topology(tp["R"], tp["G"], tp["E"], self_rank, tp["c_intra"], tp["c_inter"],
                           tp["S"], tp["W"])
    out = oracle.plan_ref(topo, omega, _topk_from_row(omega[self_rank]), tp["N"], debug=True,
                          move_cap=16)
    assert out["status"] == 0
    # stage 1: E4' on GPU 0 and nothing else
    x1 = out["x_stage1"].astype(bool)
    reps = [(e, r) for e in range(tp["E"]) for r in range(tp["R"])
            if x1[e, r] and r != e // (tp["E"] // tp["R"])]
    assert reps == [tuple(p) for p in exp["stage1_replicas"]]
    assert out["load_routed"][:2].tolist() == exp["loads_after_stage1_gpu0_gpu1"]
    # refinement: one move, E4 from GPU 0 to a new replica on GPU 1, four assignments
    assert out["n_moves"] == len(exp["refinement_moves"])
    assert out["move_count"] == len(exp["refinement_moves"])
    d, rb, rt, e, delta, created = out["moves"][0].tolist()
    mv = exp["refinement_moves"][0]
    assert (e, rb, rt, delta, bool(created)) == (mv["e"], mv["from"], mv["to"], mv["delta"], mv["created"])
    assert out["load_final"][:2].tolist() == exp["loads_final_gpu0_gpu1"]
    assert out["replica_slots"].tolist() == exp["replica_slots"]
    t = Topo(tp["R"], tp["G"], tp["E"], tp["c_intra"], tp["c_inter"], tp["S"], tp["W"], tp["N"])
    assert cross_domain_assignments(t, out["q_routed"]) == 0
    # before stage 1 (static placement) the eight E4 assignments of GPU 0 cross domains
    q_static = np.zeros((4, 8, 4), np.int64)
    for s in range(4):
        for ee in range(8):
            q_static[s, ee, ee // 2] = omega[s, ee]
    assert cross_domain_assignments(t, q_static) == exp["cross_domain_assignments_before"]
    assert cross_domain_assignments(t, out["q_final"]) == exp["cross_domain_assignments_after"]
    assert out["send_counts"].tolist() == exp["send_counts_by_self"][str(self_rank)]
    check_constraints(t, omega, out["x_final"], out["q_final"])
    if self_rank == 0:
        # the first four E4 occurrences stay on GPU 0, the next four go to GPU 1
        dest = out["token_dest"].ravel()
        e4 = dest[_topk_from_row(omega[0]).ravel() == 4]
        assert e4.tolist() == [0, 0, 0, 0, 1, 1, 1, 1]


def test_placement_cost_example():
    g = _load("placement_cost.json")["printed_by_paper"]
    n_tok = g["tokens_per_node"]
    S = g["hidden"] * g["bytes_per_value"]
    W = g["expert_bytes_mib"] * 2**20
    MiB = 2**20
    # forward + backward, dispatch + combine: 4 D S bytes of remote token traffic
    assert 4 * n_tok * S == g["token_traffic_mib_replica_on_main_node"] * MiB
    # two parameter fetches plus one gradient return
    assert 2 * W == g["param_traffic_mib_replica_on_demand_node"] * MiB
    assert W == g["grad_traffic_mib_replica_on_demand_node"] * MiB
    ratio = (4 * n_tok * S) / (3 * W)
    assert round(ratio, 1) == g["rdma_reduction_factor_approx"]
    # Eq. 9 benefit of replicating on the demanding node is positive
    assert 2 * n_tok * S - W == 24117248 > 0

    # The oracle places that replica on the demanding node (placement (b)).
    # Two nodes, one rank each; expert 1 has its main on node 1; both nodes
    # send n_tok assignments to it.
    omega = np.array([[0, n_tok], [0, n_tok]], np.int32)
    topo = oracle.topology(2, 1, 2, 0, 1, 4, S, W)
    tk = np.ones((n_tok, 1), np.int32)
    out = oracle.plan_ref(topo, omega, tk, 1, debug=True, move_cap=4)
    assert out["status"] == 0
    assert out["replica_slots"].tolist() == [[1], [-1]]
    assert out["load_final"].tolist() == [n_tok, n_tok] and out["load_final"].max() == g["lmax_both_placements"]
    assert (out["token_dest"] == 0).all()
    t = Topo(2, 1, 2, 1, 4, S, W, 1)
    assert cross_domain_assignments(t, out["q_final"]) == 0


@pytest.mark.parametrize("delta_w, expect_replica", [(0, False), (-1, True), (1, False)])
def test_benefit_sign_boundary(delta_w, expect_replica):
    """Eq. 9 / C4: a replica outside the main's domain needs W < 2 D S strictly."""
    D = 37
    S = 4096
    W = 2 * D * S + delta_w
    omega = np.array([[0, D], [0, 5]], np.int32)
    topo = oracle.topology(2, 1, 2, 0, 1, 4, S, W)
    tk = np.ones((D, 1), np.int32)
    out = oracle.plan_ref(topo, omega, tk, 1)
    assert (out["replica_slots"][0, 0] == 1) == expect_replica
