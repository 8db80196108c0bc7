"""GPU parity under the full cost model of Section 4.1 (a general symmetric
cost matrix and one size per expert, topoep_plan_costs), against the
oracle, bit for bit: replica slots, destinations, send counts, status and
move count.

Cases: random tiny instances with random matrices and sizes (every self
rank class), the two-level matrix given explicitly, sizes alone, invalid
models, and full-size workloads with a three-level (rack) cost and varied
expert sizes, up to 256 ranks.
"""
import numpy as np
import pytest

import oracle
import workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_35481_amd import topoep  # noqa: E402
from test_oracle_pins import random_instance  # noqa: E402

DEV = torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)


def both(R, G, E, s, cI, cX, S, W, N, gl, tk, C=None, We=None, what=""):
    say("case", what)
    topo = topoep.topology(R, G, E, s, cI, cX, S, W)
    T, k = tk.shape
    Cd = torch.from_numpy(np.array(C, np.int32)).to(DEV) if C is not None else None
    Wd = torch.from_numpy(np.array(We, np.int64)).to(DEV) if We is not None else None
    p = topoep.CostPlanner(topo, T, k, N, cost=Cd, expert_bytes=Wd, device=DEV)
    outs = p.plan(torch.from_numpy(np.array(gl, np.int32)).to(DEV), torch.from_numpy(np.array(tk, np.int32)).to(DEV))
    torch.cuda.synchronize()
    got = {"replica_slots": outs[0].cpu().numpy(), "token_dest": outs[1].cpu().numpy(),
           "send_counts": outs[2].cpu().numpy(), "status": int(outs[3][0].item()),
           "move_count": int(outs[3][1].item())}
    ref = oracle.plan_ref(oracle.topology(R, G, E, s, cI, cX, S, W), gl, tk, N, cost_matrix=C, expert_bytes=We)
    assert got["status"] == ref["status"], (what, got["status"], ref["status"])
    assert got["move_count"] == ref["move_count"], (what, got["move_count"], ref["move_count"])
    for key in ("replica_slots", "send_counts", "token_dest"):
        a, b = got[key], ref[key]
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)
            raise AssertionError("%s: %s differs at %d places, first %s: gpu %s oracle %s" % (
                what, key, len(bad), bad[0].tolist(), a[tuple(bad[0])], b[tuple(bad[0])]))
    return got, ref


@pytest.mark.parametrize("seed", range(80))
def test_random_tiny_general(seed):
    t, omega, topks = random_instance(9500 + seed, big=bool(seed % 2), general=True)
    s = seed % t.R
    tk = topks[s]
    if tk.ndim != 2 or tk.shape[0] == 0:
        tk = np.zeros((0, 1), np.int32)
    both(t.R, t.G, t.E, s, t.cI, t.cX, t.S, t.W, t.N, omega, tk, C=t.C, We=t.Wvec, what="tiny seed %d" % seed)


@pytest.mark.parametrize("seed", range(20))
def test_sizes_alone_and_two_level_matrix(seed):
    t, omega, topks = random_instance(9700 + seed, big=True, general=True)
    s = seed % t.R
    both(t.R, t.G, t.E, s, t.cI, t.cX, t.S, t.W, t.N, omega, topks[s], We=t.Wvec, what="sizes %d" % seed)
    C2 = t.cost_matrix() if t.C is None else None
    t.C = None
    C2 = t.cost_matrix().astype(np.int32)
    got, _ = both(t.R, t.G, t.E, s, t.cI, t.cX, t.S, t.W, t.N, omega, topks[s], C=C2, what="two-level %d" % seed)
    # the same plan as the two-level entry point
    topo = topoep.topology(t.R, t.G, t.E, s, t.cI, t.cX, t.S, t.W)
    slots, dest, sc, st = topoep.plan(topo, torch.from_numpy(omega).to(DEV), torch.from_numpy(topks[s]).to(DEV),
                                      t.N)
    torch.cuda.synchronize()
    assert np.array_equal(slots.cpu().numpy(), got["replica_slots"])
    assert np.array_equal(dest.cpu().numpy(), got["token_dest"])
    assert int(st[1].item()) == got["move_count"]


def test_invalid_models():
    t, omega, topks = random_instance(77, big=True, general=True)
    good = t.C.copy()
    cases = []
    c = good.copy(); c[0, 1] += 1; cases.append(("asymmetric", c, t.Wvec))
    c = good.copy(); c[1, 1] = 2; cases.append(("diagonal", c, t.Wvec))
    c = good.copy(); c[0, 1] = c[1, 0] = -1; cases.append(("negative", c, t.Wvec))
    w = t.Wvec.copy(); w[3] = -5; cases.append(("negative size", good, w))
    for what, C, W in cases:
        got, _ = both(t.R, t.G, t.E, 0, t.cI, t.cX, t.S, t.W, t.N, omega, topks[0], C=C, We=W, what=what)
        assert got["status"] & topoep.ST_COST
        assert (got["replica_slots"] == -1).all() and (got["token_dest"] == -1).all()


def rack_costs(R, G, racks_of, c_node=1, c_rack=4, c_far=12):
    """Three-level cost: same node, same rack (racks_of nodes), elsewhere."""
    r = np.arange(R)
    node = r // G
    rack = node // racks_of
    C = np.where(node[:, None] == node[None, :], c_node, np.where(rack[:, None] == rack[None, :], c_rack, c_far))
    np.fill_diagonal(C, 0)
    return C.astype(np.int32)


@pytest.mark.parametrize("name,budget", [("qwen3", 2), ("dsv3", 2), ("dsv3", 5), ("mixtral", 1), ("stress", 4)])
def test_workloads_with_rack_costs(name, budget):
    cfg = workload.get(name)
    gl, tk = workload.make_layer(cfg, 3, 0, 0)
    rng = np.random.default_rng(5)
    C = rack_costs(cfg.R, cfg.G, racks_of=2)
    We = (cfg.W * rng.uniform(0.25, 1.75, size=cfg.E)).astype(np.int64)
    both(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W, budget, gl, tk, C=C, We=We,
         what="%s N=%d" % (name, budget))
