"""GPU parity: every output of the HIP planner (replica_slots, token_dest,
send_counts, status bits and refinement move count) equals the oracle's bit
for bit, through the C ABI.

Integer work throughout, so the bar is exact equality.  Cases: the paper's
worked example, seeded random tiny instances (ragged sizes, every topology
shape), mid-size random instances (up to 96 ranks, domains of up to 16),
the five workload configurations at full size, larger replica
budgets that keep the refinement busy at scale, edge cases, launch-shape
and repeat determinism, HIP-graph replay, and the single-stage entry point.
"""
import json
import os

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
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def say(*a):
    print(*a, flush=True)


def gpu_plan(R, G, E, self_rank, cI, cX, S, W, N, gl, tk, launch=None):
    topo = topoep.topology(R, G, E, self_rank, cI, cX, S, W)
    T, k = tk.shape
    p = topoep.Planner(topo, T, k, N, device=DEV, launch=launch)
    gl_d = torch.from_numpy(np.ascontiguousarray(gl, dtype=np.int32)).to(DEV)
    tk_d = torch.from_numpy(np.ascontiguousarray(tk, dtype=np.int32)).to(DEV)
    slots, dest, sc, st = p.plan(gl_d, tk_d)
    torch.cuda.synchronize()
    return dict(replica_slots=slots.cpu().numpy(), token_dest=dest.cpu().numpy(),
                send_counts=sc.cpu().numpy(), status=int(st[0].item()), move_count=int(st[1].item()))


def ref_plan(R, G, E, self_rank, cI, cX, S, W, N, gl, tk):
    topo = oracle.topology(R, G, E, self_rank, cI, cX, S, W)
    return oracle.plan_ref(topo, gl, tk, N)


def assert_same(got, ref, what=""):
    assert got["status"] == ref["status"], (what, got["status"], ref["status"])
    assert got["move_count"] == ref["move_count"], (what, got["move_count"], ref["move_count"])
    for key in ("replica_slots", "send_counts", "token_dest"):
        a, b = got[key], ref[key]
        assert a.shape == b.shape, (what, key, a.shape, b.shape)
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)
            raise AssertionError("%s: %s differs at %d places, first %s: gpu %s oracle %s" % (
                what, key, len(bad), bad[0].tolist(), a[tuple(bad[0])], b[tuple(bad[0])]))


def both(*args, launch=None, what=""):
    say("case", what)
    got = gpu_plan(*args, launch=launch)
    ref = ref_plan(*args)
    assert_same(got, ref, what)
    return got, ref


def cfg_args(cfg, self_rank, gl, tk, N=None):
    return (cfg.R, cfg.G, cfg.E, self_rank, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W,
            cfg.N if N is None else N, gl, tk)


# ---------------------------------------------------------------- paper example

@pytest.mark.parametrize("self_rank", [0, 1, 2, 3])
def test_worked_example(self_rank):
    g = json.load(open(os.path.join(GOLD, "worked_example.json")))
    tp = g["topology"]
    om = np.array(g["omega"], np.int32)
    tk = np.repeat(np.arange(tp["E"], dtype=np.int32), om[self_rank]).reshape(-1, 1)
    got, _ = both(tp["R"], tp["G"], tp["E"], self_rank, tp["c_intra"], tp["c_inter"], tp["S"], tp["W"],
                  tp["N"], om, tk, what="worked example self=%d" % self_rank)
    assert got["replica_slots"].tolist() == g["expected"]["replica_slots"]


# ---------------------------------------------------------------- random tiny

SOLVERS = {"single": (0, 0, 0, 0, 1), "perdomain": (0, 0, 0, 0, 2), "fused": (0, 0, 0, 0, 3)}


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("seed", range(150))
def test_random_tiny(seed, solver):
    rng = np.random.default_rng(7000 + seed)
    t, omega, topks = random_instance(7000 + seed, big=bool(seed % 2))
    s = int(rng.integers(t.R))
    tk = topks[s]
    if tk.shape[0] == 0:
        tk = np.zeros((0, topks[0].shape[1] if topks[0].ndim == 2 else 1), np.int32)
    both(t.R, t.G, t.E, s, t.cI, t.cX, t.S, t.W, t.N, omega, tk, launch=SOLVERS[solver],
         what="tiny seed %d %s" % (seed, solver))


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("seed", range(40))
def test_random_refinement_heavy(seed, solver):
    """Several slots per rank, one hot expert per domain: long refinement."""
    rng = np.random.default_rng(9000 + seed)
    G = int(rng.choice([2, 4, 8]))
    M = int(rng.choice([1, 2, 4]))
    R = G * M
    P = int(rng.choice([1, 2, 4]))
    E = R * P
    k = int(rng.integers(1, min(E, 4) + 1))
    N = int(rng.integers(1, 5))
    pop = rng.dirichlet(np.full(E, 0.2))
    topks = [rng.choice(E, size=(int(rng.integers(50, 400)), k), p=pop).astype(np.int32) for _ in range(R)]
    omega = np.stack([np.bincount(x.ravel(), minlength=E) for x in topks]).astype(np.int32)
    cI = int(rng.integers(0, 3))
    cX = int(rng.integers(cI, 9))
    S = int(rng.integers(1, 64))
    W = int(rng.integers(1, 2 * S * 400))
    s = int(rng.integers(R))
    both(R, G, E, s, cI, cX, S, W, N, omega, topks[s], launch=SOLVERS[solver],
         what="refine seed %d %s" % (seed, solver))


def random_mid_instance(seed):
    """A mid-size instance: up to 96 ranks in domains of 1..16, up to 8
    experts per rank, top-1..8, 0..3000 local tokens, 0..5 replica slots,
    popularity from flat to one hot expert, and in one case of ten a row self
    of Omega that is not the histogram of the ids."""
    rng = np.random.default_rng(50000 + seed)
    G = int(rng.choice([1, 2, 3, 4, 6, 8, 16]))
    M = int(rng.choice([1, 2, 3, 4, 8]))
    if G * M > 96:
        M = max(1, 96 // G)
    R = G * M
    P = int(rng.choice([1, 2, 3, 4, 8]))
    E = R * P
    k = int(rng.integers(1, min(E, 8) + 1))
    N = int(rng.integers(0, 6))
    pop = rng.dirichlet(np.full(E, float(rng.choice([0.05, 0.2, 1.0, 5.0]))))
    T = int(rng.choice([0, 1, 7, 64, 500, 3000]))
    topks = [rng.choice(E, size=(int(rng.integers(0, 2 * T + 2)), k), p=pop).astype(np.int32) for _ in range(R)]
    s = int(rng.integers(R))
    topks[s] = rng.choice(E, size=(T, k), p=pop).astype(np.int32)
    omega = np.stack([np.bincount(x.ravel(), minlength=E) for x in topks]).astype(np.int32)
    if rng.random() < 0.1:
        omega[s] = rng.integers(0, 50, size=E)
    cI = int(rng.integers(0, 3))
    cX = int(rng.integers(cI, 12))
    S = int(rng.integers(1, 9))
    D = int(omega.reshape(M, G, E).sum(1).max())
    W = int(rng.integers(0, 2 * S * max(D, 1) + 2))
    return (R, G, E, s, cI, cX, S, W, N, omega, topks[s])


@pytest.mark.parametrize("solver", sorted(SOLVERS))
def test_random_mid(solver):
    """300 mid-size instances per solver (one test each: a failure names its
    seed); a shape beyond the solver's LDS limit is skipped."""
    done = 0
    for seed in range(300):
        args = random_mid_instance(seed)
        try:
            got = gpu_plan(*args, launch=SOLVERS[solver])
        except topoep.TopoepError as ex:
            if ex.rc == topoep.ELIMIT:
                continue
            raise
        R, G, E, s, _, _, _, _, N, _, tk = args
        assert_same(got, ref_plan(*args), "mid seed %d %s R%d G%d E%d k%d T%d N%d" % (
            seed, solver, R, G, E, tk.shape[1], tk.shape[0], N))
        done += 1
    say("mid", solver, done, "instances")
    assert done >= 200


# ---------------------------------------------------------------- configurations

CONFIG_CASES = [("tiny", 0, 0), ("mixtral", 0, 0), ("mixtral", 7, 0), ("qwen3", 0, 0), ("qwen3", 5, 3),
                ("dsv3", 0, 0), ("dsv3", 57, 0), ("stress", 0, 0)]


@pytest.mark.parametrize("name,layer,mb", CONFIG_CASES)
def test_config_full_size(name, layer, mb):
    cfg = workload.get(name)
    gl, tk = workload.make_layer(cfg, layer, mb, 0)
    both(*cfg_args(cfg, 0, gl, tk), what="%s layer %d mb %d" % (name, layer, mb))


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("name,layer", [("tiny", 0), ("mixtral", 3), ("qwen3", 2), ("dsv3", 1)])
def test_config_both_solvers(name, layer, solver):
    cfg = workload.get(name)
    gl, tk = workload.make_layer(cfg, layer, 0, 0)
    both(*cfg_args(cfg, 0, gl, tk, N=cfg.N + 2), launch=SOLVERS[solver],
         what="%s layer %d %s" % (name, layer, solver))


@pytest.mark.parametrize("name,N", [("dsv3", 4), ("dsv3", 8), ("qwen3", 6), ("mixtral", 3), ("stress", 8)])
def test_config_larger_budget(name, N):
    """More slots than stage 1 can fill: the refinement commits many moves."""
    cfg = workload.get(name)
    gl, tk = workload.make_layer(cfg, 1, 0, 0)
    both(*cfg_args(cfg, 0, gl, tk, N=N), what="%s N=%d" % (name, N))


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("R,E,N", [(8, 640, 2), (8, 512, 6), (16, 640, 4), (8, 64, 1), (4, 320, 3)])
def test_many_instances_per_rank(R, E, N, solver):
    """The solver-scaling rows: up to 80 main experts per rank (more than one
    wavefront of instances on the busiest rank) and tens of refinement moves
    per layer."""
    cfg = workload.Config("scale", 6, R=R, G=min(R, 8), E=E, k=8, T=4096, N=N, c_intra=1, c_inter=8,
                          S=2048 * 2, W=3 * 2048 * 768 * 2, layers=1, microbatches=1, zipf_s=1.0)
    gl, tk = workload.make_layer(cfg, 0, 0, 0)
    both(*cfg_args(cfg, 0, gl, np.ascontiguousarray(tk)), launch=SOLVERS[solver],
         what="R=%d E=%d N=%d %s" % (R, E, N, solver))


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("G,M,P,N", [(16, 1, 2, 3), (32, 2, 1, 4), (64, 1, 1, 2), (24, 2, 3, 4), (32, 4, 2, 4), (64, 2, 1, 2)])
def test_large_nodes(G, M, P, N, solver):
    """Nodes of 16 to 64 ranks: rank reductions over the whole wavefront,
    hosting masks of up to 64 ranks, long refinement."""
    rng = np.random.default_rng(9700 + G * 10 + M * 3 + N)
    R = G * M
    E = R * P
    k = 4
    pop = rng.dirichlet(np.full(E, 0.3))
    topks = [np.stack([rng.choice(E, size=k, replace=False, p=pop) for _ in range(int(rng.integers(100, 300)))])
             .astype(np.int32) for _ in range(R)]
    omega = np.stack([np.bincount(x.ravel(), minlength=E) for x in topks]).astype(np.int32)
    s = int(rng.integers(R))
    ref = ref_plan(R, G, E, s, 1, 8, 64, 1000, N, omega, topks[s])
    assert ref["move_count"] > 0
    try:
        topoep.Planner(topoep.topology(R, G, E, s, 1, 8, 64, 1000), topks[s].shape[0], k, N, device=DEV,
                       launch=SOLVERS[solver])
    except topoep.TopoepError as ex:
        if ex.rc != topoep.ELIMIT:
            raise
        pytest.skip("the %s solver's state does not fit one workgroup's LDS here" % solver)
    both(R, G, E, s, 1, 8, 64, 1000, N, omega, topks[s], launch=SOLVERS[solver],
         what="G=%d M=%d P=%d N=%d %s" % (G, M, P, N, solver))


@pytest.mark.parametrize("seed", range(30))
def test_refinement_equal_loads(seed):
    """Receivers tied on load: every token count a multiple of a large unit,
    so many ranks share one load level and the cost change and rank order
    break the ties."""
    rng = np.random.default_rng(9500 + seed)
    G = int(rng.choice([4, 8]))
    M = int(rng.choice([1, 2]))
    R, P = G * M, int(rng.choice([1, 2, 3]))
    E = R * P
    k = int(rng.integers(1, min(E, 3) + 1))
    N = int(rng.integers(2, 6))
    hot = rng.choice(E, size=max(1, E // 4), replace=False)
    pop = np.full(E, 1.0)
    pop[hot] = 8.0
    pop /= pop.sum()
    T = int(rng.integers(16, 64)) * 4
    topks = [np.stack([rng.choice(E, size=k, replace=False, p=pop) for _ in range(T)]).astype(np.int32)
             for _ in range(R)]
    omega = np.stack([np.bincount(x.ravel(), minlength=E) for x in topks]).astype(np.int32)
    omega = (omega // 4) * 4
    s = int(rng.integers(R))
    tk = topks[s]
    omega[s] = np.bincount(tk.ravel(), minlength=E)
    cI = int(rng.integers(0, 2))
    both(R, G, E, s, cI, cI + int(rng.integers(0, 6)), int(rng.integers(1, 9)), int(rng.integers(1, 200)), N,
         omega, tk, launch=SOLVERS[["single", "perdomain", "fused"][seed % 3]],
         what="equal loads seed %d" % seed)


@pytest.mark.parametrize("name", ["tiny"])
def test_every_self_rank_agrees(name):
    """Every rank derives the same replica slots; send counts add up to the
    rank loads of the plan (Section 3.1: no coordinator, no broadcast)."""
    cfg = workload.get(name)
    allr = workload.all_rank_topk(cfg, 0, 0)
    gl, _ = workload.make_layer(cfg, 0, 0, 0)
    slots = None
    total = np.zeros(cfg.R, np.int64)
    ranks = range(cfg.R) if cfg.R <= 8 else [0, 1, 7, 8, 15, 16, 31]
    for s in ranks:
        got, _ = both(*cfg_args(cfg, s, gl, np.ascontiguousarray(allr[s])), what="%s self=%d" % (name, s))
        if slots is None:
            slots = got["replica_slots"]
        assert np.array_equal(got["replica_slots"], slots)
        total += got["send_counts"]
    if cfg.R <= 8:
        ref = oracle.plan_ref(oracle.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W),
                              gl, allr[0], cfg.N, debug=True, move_cap=10000)
        assert np.array_equal(total, ref["load_final"])


# ---------------------------------------------------------------- edge cases

def _tiny():
    cfg = workload.get("tiny")
    gl, tk = workload.make_layer(cfg, 0, 0, 0)
    return cfg, gl, tk


def test_empty_local_batch():
    cfg, gl, _ = _tiny()
    gl = gl.copy()
    gl[0] = 0
    both(*cfg_args(cfg, 0, gl, np.zeros((0, cfg.k), np.int32)), what="T=0")


def test_static_ep_budget_zero():
    cfg, gl, tk = _tiny()
    got, _ = both(*cfg_args(cfg, 0, gl, tk, N=0), what="N=0")
    assert np.array_equal(got["token_dest"], tk // cfg.P)


def test_budget_beyond_experts():
    cfg, gl, tk = _tiny()
    both(*cfg_args(cfg, 0, gl, tk, N=40), what="N=40")


def test_k1_and_ragged():
    rng = np.random.default_rng(3)
    E, R, G = 24, 6, 3
    tk = rng.integers(0, E, size=(1237, 1)).astype(np.int32)
    gl = rng.integers(0, 300, size=(R, E)).astype(np.int32)
    gl[2] = np.bincount(tk.ravel(), minlength=E)
    both(R, G, E, 2, 1, 5, 33, 5000, 2, gl, tk, what="k=1 ragged")


def test_one_gpu_per_node_and_single_domain():
    cfg, gl, tk = _tiny()
    both(cfg.R, 1, cfg.E, 0, 1, 4, cfg.S, cfg.W, 2, gl, tk, what="G=1")
    both(cfg.R, cfg.R, cfg.E, 0, 1, 4, cfg.S, cfg.W, 2, gl, tk, what="M=1")


def test_zero_intra_cost():
    cfg, gl, tk = _tiny()
    both(cfg.R, cfg.G, cfg.E, 0, 0, 4, cfg.S, cfg.W, 3, gl, tk, what="c_intra=0")


def test_bad_id():
    cfg, gl, tk = _tiny()
    tk = tk.copy()
    tk[100, 1] = cfg.E + 3
    got, _ = both(*cfg_args(cfg, 0, gl, tk), what="bad id")
    assert got["status"] & topoep.ST_BAD_ID
    tk[100, 1] = -5
    both(*cfg_args(cfg, 0, gl, tk), what="negative id")


def test_negative_load_and_mismatch():
    cfg, gl, tk = _tiny()
    g2 = gl.copy()
    g2[3, 5] = -2
    got, _ = both(*cfg_args(cfg, 0, g2, tk), what="negative load")
    assert got["status"] == topoep.ST_NEG_LOAD
    g3 = gl.copy()
    g3[0, 1] += 5
    got, _ = both(*cfg_args(cfg, 0, g3, tk), what="self row mismatch")
    assert got["status"] == topoep.ST_SELF_DIFF


def _self_row_cases():
    """Omega's row self against the histogram of local_topk (self = 2 of the
    tiny configuration): the one-launch plan is first made from Omega as
    gathered and kept only when that row equals the histogram."""
    cfg, gl, tk = _tiny()
    s = 2
    tk = tk.copy()
    hist = np.bincount(tk.ravel(), minlength=cfg.E).astype(np.int64)
    gl = gl.copy()
    gl[s] = hist
    out = [("equal rows", gl, tk)]
    g = gl.copy()
    g[s] = np.roll(hist, 5) * 3        # a different demand: a different plan
    out.append(("row self differs", g, tk))
    g = gl.copy()
    g[s, 0] = 2**31 - 1                # Omega out of range, Omega' in range
    out.append(("range only before", g, tk))
    g = gl.copy()
    g[s] = 0
    rest = int(g.astype(np.int64).sum())
    g[(s + 1) % cfg.R, 0] += 2**31 - 1 - rest - int(hist.sum()) + 1   # Omega' just out of range
    out.append(("range only after", g, tk))
    g = gl.copy()
    g[s, 3] = -1                       # a negative load in row self only
    out.append(("negative in row self", g, tk))
    g = gl.copy()
    g[(s + 3) % cfg.R, 1] = -4         # refused Omega, equal rows
    out.append(("negative elsewhere", g, tk))
    t2 = tk.copy()
    t2[7, 1] = cfg.E + 2               # a bad id; the valid ids' histogram is row self
    g = gl.copy()
    g[s] = np.bincount(t2[(t2 >= 0) & (t2 < cfg.E)], minlength=cfg.E)
    out.append(("bad id", g, t2))
    return cfg, s, out


@pytest.mark.parametrize("solver", sorted(SOLVERS))
def test_self_row_against_histogram(solver):
    cfg, s, cases = _self_row_cases()
    for what, g, t in cases:
        assert int(g.max()) < 2**31 and int(g.min()) >= -2**31
        both(cfg.R, cfg.G, cfg.E, s, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W, cfg.N,
             g.astype(np.int32), t, launch=SOLVERS[solver], what="%s (%s)" % (what, solver))


def test_range_bit():
    cfg, gl, tk = _tiny()
    got, _ = both(cfg.R, cfg.G, cfg.E, 0, 1, 1 << 10, 1 << 50, cfg.W, 1, gl, tk, what="range S")
    assert got["status"] & topoep.ST_RANGE
    got, _ = both(cfg.R, cfg.G, cfg.E, 0, 1, 4, cfg.S, 1 << 61, 1, gl, tk, what="range W")
    assert got["status"] & topoep.ST_RANGE


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("W", [0, 3 << 40])
def test_range_threshold(solver, W):
    """Both sides of the exact-range limit 4 S total c + c W < 2^62: the
    largest S that keeps a plan in range, and one more (RANGE), against the
    oracle's own overflow-checked products."""
    cfg, gl, tk = _tiny()
    g = gl.astype(np.int64).copy()
    g[0] = np.bincount(tk[(tk >= 0) & (tk < cfg.E)], minlength=cfg.E)   # row self of Omega'
    total = int(g[g > 0].sum())
    cI, cX = 1, 4
    x = 4 * cX * total
    s_in = ((1 << 62) - cX * W - 1) // x
    got, _ = both(cfg.R, cfg.G, cfg.E, 0, cI, cX, s_in, W, 1, gl, tk, launch=SOLVERS[solver],
                  what="range threshold, S in range (%s)" % solver)
    assert not got["status"] & topoep.ST_RANGE
    got, _ = both(cfg.R, cfg.G, cfg.E, 0, cI, cX, s_in + 1, W, 1, gl, tk, launch=SOLVERS[solver],
                  what="range threshold, S one past (%s)" % solver)
    assert got["status"] & topoep.ST_RANGE


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("W", [1 << 60, (1 << 60) - 1])
def test_range_expert_bytes_at_the_bound(solver, W):
    """c W at 2^62 (every plan out of range, whatever S) and just below it
    (every plan with a positive load out of range: the bound leaves room
    for no assignment), against the oracle."""
    cfg, gl, tk = _tiny()
    got, _ = both(cfg.R, cfg.G, cfg.E, 0, 1, 4, 1, W, 1, gl, tk, launch=SOLVERS[solver],
                  what="range at the expert-bytes bound W=%d (%s)" % (W, solver))
    assert got["status"] & topoep.ST_RANGE


def test_many_domains_more_than_solver_groups():
    """M = 256 domains (G = 1): solver workgroups loop over several domains."""
    rng = np.random.default_rng(11)
    R, G, E = 256, 1, 256
    tk = rng.integers(0, E, size=(300, 2)).astype(np.int32)
    gl = rng.integers(0, 20, size=(R, E)).astype(np.int32)
    gl[5] = np.bincount(tk.ravel(), minlength=E)
    both(R, G, E, 5, 1, 4, 64, 1500, 2, gl, tk, what="M=256")


# ---------------------------------------------------------------- determinism

LAUNCHES = [(1, 64, 0, 64, 2), (2, 128, 1, 128, 1), (4, 256, 0, 256, 2), (8, 256, 2, 512, 1),
            (8, 1024, 0, 1024, 2), (1, 1024, 3, 64, 1), (4, 512, 1, 256, 0),
            (1, 0, 0, 1024, 3), (2, 0, 0, 1024, 3), (4, 0, 0, 512, 3), (4, 0, 0, 1024, 3), (8, 0, 0, 512, 3),
            (8, 0, 0, 256, 3), (4, 0, 0, 128, 3)]


@pytest.mark.parametrize("launch", LAUNCHES)
@pytest.mark.parametrize("name", ["mixtral", "dsv3"])
def test_launch_shapes_are_bitwise_identical(name, launch):
    cfg = workload.get(name)
    gl, tk = workload.make_layer(cfg, 2, 0, 0)
    N = cfg.N + 2
    both(*cfg_args(cfg, 0, gl, tk, N=N), launch=launch, what="%s launch %s" % (name, launch))


def test_repeated_runs_identical():
    cfg = workload.get("dsv3")
    gl, tk = workload.make_layer(cfg, 3, 0, 0)
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    p = topoep.Planner(topo, cfg.T, cfg.k, 4, device=DEV)
    gl_d = torch.from_numpy(gl).to(DEV)
    tk_d = torch.from_numpy(tk).to(DEV)
    first = None
    for i in range(50):
        out = [x.clone() for x in p.plan(gl_d, tk_d)]
        if first is None:
            first = out
        else:
            for a, b in zip(out, first):
                assert torch.equal(a, b), i
    ref = ref_plan(*cfg_args(cfg, 0, gl, tk, N=4))
    torch.cuda.synchronize()
    assert np.array_equal(first[1].cpu().numpy(), ref["token_dest"])


@pytest.mark.parametrize("solver", sorted(SOLVERS))
def test_graph_replay_matches_eager(solver):
    """The enqueue is captured in a HIP graph and replayed with eager work in
    between; every replay equals the oracle."""
    say("case graph replay", solver)
    cfg = workload.get("qwen3")
    gl, tk = workload.make_layer(cfg, 4, 1, 0)
    ref = ref_plan(*cfg_args(cfg, 0, gl, tk))
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    p = topoep.Planner(topo, cfg.T, cfg.k, cfg.N, device=DEV, launch=SOLVERS[solver])
    gl_d = torch.from_numpy(gl).to(DEV)
    tk_d = torch.from_numpy(tk).to(DEV)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        p.plan(gl_d, tk_d)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        p.plan(gl_d, tk_d)
    for i in range(5):
        p.token_dest.fill_(-9)
        p.send_counts.fill_(-9)
        junk = torch.randn(1 << 16, device=DEV).sum()
        g.replay()
        torch.cuda.synchronize()
        got = dict(replica_slots=p.replica_slots.cpu().numpy(), token_dest=p.token_dest.cpu().numpy(),
                   send_counts=p.send_counts.cpu().numpy(), status=int(p.status[0].item()),
                   move_count=int(p.status[1].item()))
        assert_same(got, ref, "graph replay %d" % i)
        del junk


def test_single_stages_repeat():
    """After one plan, re-running each stage alone reproduces the outputs."""
    cfg = workload.get("tiny")
    gl, tk = workload.make_layer(cfg, 0, 0, 0)
    ref = ref_plan(*cfg_args(cfg, 0, gl, tk))
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    p = topoep.Planner(topo, cfg.T, cfg.k, cfg.N, device=DEV, launch=SOLVERS["single"])
    assert p.shape.kernels == 3
    gl_d = torch.from_numpy(gl).to(DEV)
    tk_d = torch.from_numpy(tk).to(DEV)
    p.plan(gl_d, tk_d)
    for stage in (2, 1, 2, 0, 1, 2):
        p.token_dest.fill_(-9)
        p.stage(stage, gl_d, tk_d)
        if stage != 2:
            p.stage(2, gl_d, tk_d)
        torch.cuda.synchronize()
        assert np.array_equal(p.token_dest.cpu().numpy(), ref["token_dest"]), stage


def test_one_launch_stage_and_control_words():
    """With one kernel, stage 0 is the whole plan; stages 1 and 2 are
    rejected.  Between plans the one-launch plan's hand-over words hold its
    generation: word 10 advances by one per plan and the 64-bit arrival
    count (words 8..9) is that generation times the chunk count, so a plan
    on a reused workspace needs no clearing."""
    cfg = workload.get("dsv3")
    gl, tk = workload.make_layer(cfg, 5, 0, 0)
    ref = ref_plan(*cfg_args(cfg, 0, gl, tk))
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    p = topoep.Planner(topo, cfg.T, cfg.k, cfg.N, device=DEV, launch=SOLVERS["fused"])
    assert p.shape.kernels == 1 and p.shape.solver == topoep.SOLVER_FUSED
    nb = p.shape.chunk_blocks
    gl_d = torch.from_numpy(gl).to(DEV)
    tk_d = torch.from_numpy(tk).to(DEV)
    for i in range(4):
        p.token_dest.fill_(-9)
        if i % 2:
            p.stage(0, gl_d, tk_d)
        else:
            p.plan(gl_d, tk_d)
        torch.cuda.synchronize()
        assert np.array_equal(p.token_dest.cpu().numpy(), ref["token_dest"]), i
        ctrl = p.workspace_view()[:256].cpu().numpy()
        gen = int(ctrl.view(np.uint32)[10])
        arrivals = int(ctrl[32:40].view(np.uint64)[0])
        assert gen == i + 1 and arrivals == gen * nb, (i, gen, arrivals)
    for stage in (1, 2):
        with pytest.raises(topoep.TopoepError):
            p.stage(stage, gl_d, tk_d)


def _planner_for(cfg, solver, N=None):
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    return topoep.Planner(topo, cfg.T, cfg.k, cfg.N if N is None else N, device=DEV, launch=SOLVERS[solver])


def _got(p):
    torch.cuda.synchronize()
    return dict(replica_slots=p.replica_slots.cpu().numpy(), token_dest=p.token_dest.cpu().numpy(),
                send_counts=p.send_counts.cpu().numpy(), status=int(p.status[0].item()),
                move_count=int(p.status[1].item()))


@pytest.mark.parametrize("solver", ["fused", "perdomain"])
def test_wait_that_gives_up_leaves_nothing_behind(solver):
    """Every bounded wait of the plan is made to give up from the host
    (spin_limit -1: no poll at all; every kernel still runs to its end):
    the plan reports SYNC.  The next plans on the same workspace, without
    clearing it, equal the oracle, also when their inputs differ from the
    plan that gave up and when one of them must be redone (row self of Omega
    differing from the histogram)."""
    cfg = workload.get("qwen3" if solver == "fused" else "stress")
    layers = [workload.make_layer(cfg, l, 0, 0) for l in (0, 1)]
    p = _planner_for(cfg, solver)
    give_up = tuple(SOLVERS[solver]) + (-1, 0)
    dev = [(torch.from_numpy(g).to(DEV), torch.from_numpy(t).to(DEV)) for g, t in layers]
    refs = [ref_plan(*cfg_args(cfg, 0, g, t)) for g, t in layers]
    # a row self that differs from the histogram: the one-launch plan redoes it
    g_diff = layers[1][0].copy()
    g_diff[0] = np.roll(g_diff[0], 3)
    ref_diff = ref_plan(*cfg_args(cfg, 0, g_diff, layers[1][1]))
    g_diff_d = torch.from_numpy(g_diff).to(DEV)
    for rnd in range(3):
        say("give up", solver, "round", rnd)
        p.plan(*dev[0])
        assert_same(_got(p), refs[0], "%s before, round %d" % (solver, rnd))
        p.token_dest.fill_(-9)
        p.plan(*dev[1], launch=give_up)
        got = _got(p)
        assert got["status"] & topoep.ST_SYNC, got["status"]
        assert (got["token_dest"] == -1).all()
        p.plan(*dev[1])
        assert_same(_got(p), refs[1], "%s after, round %d" % (solver, rnd))
        p.plan(g_diff_d, dev[1][1], launch=give_up)
        assert _got(p)["status"] & topoep.ST_SYNC
        p.plan(g_diff_d, dev[1][1])
        assert_same(_got(p), ref_diff, "%s redo after, round %d" % (solver, rnd))


def test_single_stages_repeat_per_domain_solver():
    """The per-domain solver restores its own control words: its stage
    repeated alone, many times after one full plan, reproduces every output
    and the status words (moves, no RANGE) each time."""
    cfg = workload.get("stress")
    gl, tk = workload.make_layer(cfg, 0, 0, 0)
    ref = ref_plan(*cfg_args(cfg, 0, gl, tk, N=8))
    p = _planner_for(cfg, "perdomain", N=8)
    assert p.shape.kernels == 3 and p.shape.solver == topoep.SOLVER_PER_DOMAIN
    gl_d = torch.from_numpy(gl).to(DEV)
    tk_d = torch.from_numpy(tk).to(DEV)
    p.plan(gl_d, tk_d)
    assert_same(_got(p), ref, "per-domain full plan")
    assert ref["move_count"] > 0
    for rep in range(70):
        p.token_dest.fill_(-9)
        p.replica_slots.fill_(-9)
        p.status.fill_(-9)
        p.stage(1, gl_d, tk_d)
        p.stage(2, gl_d, tk_d)
        if rep % 10 == 9:
            assert_same(_got(p), ref, "per-domain stage repeat %d" % rep)


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("limit", [1, 2, 5])
def test_refinement_iteration_bound(solver, limit):
    """A domain that still has a move after iter_limit committed moves stops
    with ITER; the oracle applies the same bound, so the plans are equal."""
    cfg = workload.get("mixtral")
    gl, tk = workload.make_layer(cfg, 3, 0, 0)
    args = cfg_args(cfg, 0, gl, tk, N=3)
    full = ref_plan(*args)
    assert full["move_count"] > limit
    topo = oracle.topology(*args[:8])
    ref = oracle.plan_ref(topo, gl, tk, 3, iter_limit=limit)
    assert ref["status"] & oracle.ST_ITER and ref["move_count"] == limit
    got = gpu_plan(*args, launch=tuple(SOLVERS[solver]) + (0, limit))
    assert_same(got, ref, "iter limit %d %s" % (limit, solver))


@pytest.mark.parametrize("solver", sorted(SOLVERS))
def test_launch_floor_writes_nothing(solver):
    """The launch-floor stage runs empty kernels of the plan's shapes."""
    cfg = workload.get("qwen3")
    gl, tk = workload.make_layer(cfg, 0, 0, 0)
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    p = topoep.Planner(topo, cfg.T, cfg.k, cfg.N, device=DEV, launch=SOLVERS[solver])
    gl_d = torch.from_numpy(gl).to(DEV)
    tk_d = torch.from_numpy(tk).to(DEV)
    for t in (p.token_dest, p.send_counts, p.replica_slots, p.status):
        t.fill_(-9)
    p.stage(topoep.STAGE_FLOOR, gl_d, tk_d)
    torch.cuda.synchronize()
    for t in (p.token_dest, p.send_counts, p.replica_slots, p.status):
        assert bool((t == -9).all())


@pytest.mark.parametrize("solver", sorted(SOLVERS))
@pytest.mark.parametrize("N", [0, 1, 3])
def test_single_rank_single_expert(solver, N):
    """R = G = E = 1: one rank, one expert, no replica possible (the
    solver's scratch must still fit every wave's share)."""
    rng = np.random.default_rng(N)
    tk = np.zeros((int(rng.integers(1, 40)), 1), np.int32)
    gl = np.array([[tk.shape[0]]], np.int32)
    both(1, 1, 1, 0, 0, 6, 2, 25, N, gl, tk, launch=SOLVERS[solver], what="R=G=E=1 N=%d %s" % (N, solver))
