"""The plan-quality metrics of the report (CPU): rank loads from every
rank's send counts equal the oracle's final loads; the inter-node and
replica-served fractions equal their definitions on the oracle's q and
destinations."""
import numpy as np
import pytest

import oracle
from paper_2609_35481_amd import report
from test_oracle_pins import random_instance


@pytest.mark.parametrize("seed", range(12))
def test_metrics_match_the_plans_own_state(seed):
    t, omega, topks = random_instance(8200 + seed, big=True)
    outs = []
    for s in range(t.R):
        topo = oracle.topology(t.R, t.G, t.E, s, t.cI, t.cX, t.S, t.W)
        outs.append(oracle.plan_ref(topo, omega, topks[s], t.N, debug=True))
    sends = [o["send_counts"] for o in outs]
    L = report.rank_loads(sends)
    assert (L == outs[0]["load_final"]).all()
    q = outs[0]["q_final"]                              # [s][e][r], the same plan on every rank
    dom = np.arange(t.R) // t.G
    cross = sum(int(q[s, :, r].sum()) for s in range(t.R) for r in range(t.R) if dom[s] != dom[r])
    total = int(q.sum())
    assert report.inter_node_fraction(sends, t.G) == pytest.approx(cross / total if total else 0.0)
    P = t.E // t.R
    away = sum(int(q[s, e, r]) for s in range(t.R) for e in range(t.E) for r in range(t.R) if r != e // P)
    frac = report.replica_served_fraction([o["token_dest"] for o in outs], topks, P)
    assert frac == pytest.approx(away / total if total else 0.0)


def test_max_to_mean():
    assert report.max_to_mean([2, 2, 2, 2]) == 1.0
    assert report.max_to_mean([8, 0, 0, 0]) == 4.0
    assert report.max_to_mean([0, 0]) == 0.0
