"""GPU parity of the dispatch side of a plan through the C ABI: receive
counts (what every rank sends to this one under the replicated plan), send
offsets and the send-buffer slot of every assignment, against the oracle,
bit for bit.

Cases: the workload configurations at full size (every plan output too),
seeded random tiny instances for every self rank, and the layout kernel
alone on synthetic destinations: ragged sizes, many workgroups (look-back
across several windows of predecessors), non-rank destinations, one rank,
the largest rank count, an empty batch, and back-to-back calls on one
workspace.
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


def dispatch_gpu(R, G, E, s, cI, cX, S, W, N, gl, tk):
    topo = topoep.topology(R, G, E, s, cI, cX, S, W)
    T, k = tk.shape
    p = topoep.DispatchPlanner(topo, T, k, N, device=DEV)
    gl_d = torch.from_numpy(np.array(gl, np.int32)).to(DEV)
    tk_d = torch.from_numpy(np.array(tk, np.int32)).to(DEV)
    outs = p.plan(gl_d, tk_d)
    torch.cuda.synchronize()
    names = ("replica_slots", "token_dest", "send_counts", "recv_counts", "send_offsets", "token_slot")
    got = {n: o.cpu().numpy() for n, o in zip(names, outs[:6])}
    got["status"] = int(outs[6][0].item())
    got["move_count"] = int(outs[6][1].item())
    return got


def dispatch_ref(R, G, E, s, cI, cX, S, W, N, gl, tk):
    ref = oracle.plan_ref(oracle.topology(R, G, E, s, cI, cX, S, W), gl, tk, N)
    ref["send_offsets"], ref["token_slot"] = oracle.layout_ref(R, ref["token_dest"], ref["send_counts"])
    return ref


def check(args, what):
    say("case", what)
    got = dispatch_gpu(*args)
    ref = dispatch_ref(*args)
    assert got["status"] == ref["status"], (what, got["status"], ref["status"])
    assert got["move_count"] == ref["move_count"], what
    for key in ("replica_slots", "send_counts", "token_dest", "recv_counts", "send_offsets", "token_slot"):
        a, b = got[key], ref[key]
        assert a.shape == b.shape, (what, key)
        if not np.array_equal(a, b):
            bad = np.argwhere(a != b)
            raise AssertionError("%s: %s differs at %d places, first %s: gpu %s oracle %s" % (
                what, key, len(bad), bad[0].tolist(), a[tuple(bad[0])], b[tuple(bad[0])]))
    return got


def cfg_args(cfg, s, gl, tk, N=None):
    return (cfg.R, cfg.G, cfg.E, s, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W, cfg.N if N is None else N, gl, tk)


@pytest.mark.parametrize("name", ["tiny", "mixtral", "qwen3", "dsv3", "stress"])
def test_workloads(name):
    cfg = workload.get(name)
    gl, tk = workload.make_layer(cfg, 1, 0, 0)
    check(cfg_args(cfg, 0, gl, tk), name)


@pytest.mark.parametrize("name", ["tiny", "qwen3", "dsv3"])
def test_workloads_other_self_rank_and_budget(name):
    """A self rank in another domain, and budgets that leave slots free (the
    refinement moves load, so receive counts come from refined q)."""
    cfg = workload.get(name)
    s = cfg.R - 3
    tops = workload.make_layer(cfg, 2, 0, 0)
    gl, _ = tops
    # this rank's ids: simulate them from its own row of Omega
    row = gl[s].astype(np.int64)
    ids = np.repeat(np.arange(cfg.E, dtype=np.int32), row)
    rng = np.random.default_rng(5)
    rng.shuffle(ids)
    k = cfg.k
    T = ids.size // k
    tk = ids[:T * k].reshape(T, k)
    gl = gl.copy()
    gl[s] = np.bincount(tk.ravel(), minlength=cfg.E)
    for N in (cfg.N, cfg.N + 3):
        check(cfg_args(cfg, s, gl, tk, N=N), "%s self=%d N=%d" % (name, s, N))


@pytest.mark.parametrize("seed", range(60))
def test_random_tiny(seed):
    t, omega, topks = random_instance(9100 + seed, big=bool(seed % 2))
    s = seed % t.R
    tk = topks[s]
    if tk.ndim != 2 or tk.shape[0] == 0:
        tk = np.zeros((0, 1), np.int32)
    check((t.R, t.G, t.E, s, t.cI, t.cX, t.S, t.W, t.N, omega, tk), "tiny seed %d" % seed)


def test_many_ids_three_kernels():
    """4 M assignments: too many for the one-launch plan, so the histogram,
    solver and reroute kernels run, each reroute workgroup over several
    tiles (the slot counts before each tile come from its running per-expert
    offsets)."""
    cfg = workload.get("dsv3")
    rng = np.random.default_rng(17)
    T, k = 1 << 19, 8
    p = workload.generate.zipf_weights(cfg.E, 1.0)
    tk = rng.choice(cfg.E, size=(T, k), p=p).astype(np.int32)
    gl = rng.integers(0, 2000, size=(cfg.R, cfg.E)).astype(np.int32)
    gl[0] = np.bincount(tk.ravel(), minlength=cfg.E)
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    assert topoep.plan_shape(topo, T, k, cfg.N).kernels == 3
    check((cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W, cfg.N, gl, tk), "4M ids")


def test_refused_plan_has_no_receive_counts():
    cfg = workload.get("tiny")
    gl, tk = workload.make_layer(cfg, 0, 0, 0)
    gl = gl.copy()
    gl[3, 2] = -1
    got = check(cfg_args(cfg, 0, gl, tk), "negative load")
    assert (got["recv_counts"] == 0).all() and (got["token_slot"] == -1).all()


# ---------------------------------------------------------------- layout kernel alone

def layout_gpu(R, dest, send, reps=1, planner=None):
    T, k = dest.shape
    topo = topoep.topology(R, 1, R, 0, 1, 1, 1, 0)
    p = planner or topoep.LayoutPlanner(topo, T, k, device=DEV)
    d = torch.from_numpy(np.ascontiguousarray(dest, np.int32)).to(DEV)
    sc = torch.from_numpy(np.ascontiguousarray(send, np.int32)).to(DEV)
    for _ in range(reps):
        offs, slot = p.layout(d, sc)
    torch.cuda.synchronize()
    assert int(p.status[0].item()) == 0
    return offs.cpu().numpy(), slot.cpu().numpy(), p


def layout_case(R, n, rng, k=8, invalid=0.0, skew=None):
    T = -(-n // k)
    if skew is None:
        dest = rng.integers(0, R, size=(T, k))
    else:
        p = np.arange(1, R + 1, dtype=np.float64) ** -skew
        dest = rng.choice(R, size=(T, k), p=p / p.sum())
    if invalid:
        bad = rng.random((T, k)) < invalid
        dest[bad] = rng.choice([-1, R, R + 7, -100], size=int(bad.sum()))
    dest = dest.astype(np.int32)
    valid = dest[(dest >= 0) & (dest < R)]
    send = np.bincount(valid, minlength=R).astype(np.int32)
    return dest, send


@pytest.mark.parametrize("R,n,invalid,skew", [
    (32, 65536, 0.0, 1.0),          # DeepSeek-V3-like size
    (8, 8192, 0.0, None),
    (256, 131072, 0.0, 1.4),        # Stress-like
    (32, 65536 + 8 * 37, 0.05, None),   # ragged, some non-rank destinations
    (1, 5000, 0.0, None),
    (1024, 200000, 0.01, 0.8),      # the most ranks
    (64, (1 << 20) + 24, 0.0, 1.2),   # 256 workgroups: look-back across windows
    (7, 8 * 3, 0.0, None),          # smaller than one wave
    (32, 5000000, 0.01, 1.0),       # 2 tiles per workgroup: counts first, ranks after the look-back
    (256, (1 << 24) + 8 * 13, 0.0, 1.4),   # 5 tiles per workgroup, ragged last tile
    (512, (1 << 22) + 8 * 5, 0.01, 1.1),   # several tiles, two copies of the counts
    (1024, (1 << 22) + 8 * 3, 0.0, 0.9),   # several tiles, one copy (the most ranks)
])
def test_layout_alone(R, n, invalid, skew):
    say("layout R=%d n=%d" % (R, n))
    rng = np.random.default_rng(R * 1000 + n % 997)
    dest, send = layout_case(R, n, rng, invalid=invalid, skew=skew)
    offs, slot, _ = layout_gpu(R, dest, send)
    ref_offs, ref_slot = oracle.layout_ref(R, dest, send)
    assert np.array_equal(offs, ref_offs)
    assert np.array_equal(slot, ref_slot)


def test_layout_unaligned_destinations():
    """Destinations that start 4 bytes past a 16-byte boundary, long chunks:
    the first pass loads them one by one instead of four at a time."""
    R, n = 32, 5000000
    say("layout unaligned R=%d n=%d" % (R, n))
    rng = np.random.default_rng(4242)
    dest, send = layout_case(R, n, rng, skew=1.0)
    T, k = dest.shape
    big = torch.zeros(T * k + 1, dtype=torch.int32, device=DEV)
    big[1:] = torch.from_numpy(dest.ravel()).to(DEV)
    d = big[1:].view(T, k)
    assert d.data_ptr() % 16 != 0
    topo = topoep.topology(R, 1, R, 0, 1, 1, 1, 0)
    p = topoep.LayoutPlanner(topo, T, k, device=DEV)
    offs, slot = p.layout(d, torch.from_numpy(send).to(DEV))
    torch.cuda.synchronize()
    assert int(p.status[0].item()) == 0
    ref_offs, ref_slot = oracle.layout_ref(R, dest, send)
    assert np.array_equal(offs.cpu().numpy(), ref_offs)
    assert np.array_equal(slot.cpu().numpy(), ref_slot)


def test_layout_empty_batch():
    offs, slot, _ = layout_gpu(4, np.zeros((0, 2), np.int32), np.zeros(4, np.int32))
    assert offs.tolist() == [0, 0, 0, 0, 0] and slot.shape == (0, 2)


def test_layout_back_to_back_on_one_workspace():
    """Every call leaves the workspace's flags and ticket zero, so calls in
    a row on one workspace (different inputs, same sizes) stay exact."""
    rng = np.random.default_rng(3)
    R, n = 32, (1 << 19)
    planner = None
    for i in range(4):
        dest, send = layout_case(R, n, rng, skew=0.5 * i)
        offs, slot, planner = layout_gpu(R, dest, send, reps=1 + i % 2, planner=planner)
        ref_offs, ref_slot = oracle.layout_ref(R, dest, send)
        assert np.array_equal(offs, ref_offs) and np.array_equal(slot, ref_slot), i
    # the control word and the per-workgroup flags (the workspace's first
    # two regions) are zero again; the counts stay, later calls overwrite them
    off = planner.ws_ptr - planner._ws.data_ptr()
    nb = -(-n // (1024 * 4))
    head = 256 + -(-nb * 4 // 256) * 256
    ws = planner._ws.cpu().numpy()[off:off + head]
    assert not ws.any()
