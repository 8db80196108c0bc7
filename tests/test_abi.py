"""The C ABI library loads, exports every function include/topoep.h declares,
and validates host arguments (no GPU work: only host-side paths are called)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "topoep.h")


@pytest.fixture(scope="module")
def tp():
    from paper_2609_35481_amd import topoep
    return topoep


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*int\s+(topoep_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    assert "topoep_plan" in names and "topoep_workspace_bytes" in names
    assert len(names) == 14


def test_library_exports_every_declared_symbol(tp):
    lib = ctypes.CDLL(tp.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) == set(tp.EXPORTS)


def test_struct_layout_matches_header(tp):
    assert ctypes.sizeof(tp.Topology) == 6 * 4 + 2 * 8
    assert tp.Topology.tok_bytes.offset == 24
    assert ctypes.sizeof(tp.Launch) == 7 * 4
    assert tp.Launch.spin_limit.offset == 20 and tp.Launch.iter_limit.offset == 24
    assert ctypes.sizeof(tp.Shape) == 13 * 4


def base(tp, **kw):
    args = dict(R=8, G=4, E=16, self_rank=0, c_intra=1, c_inter=4, S=4096, W=1 << 20)
    args.update(kw)
    return tp.topology(args["R"], args["G"], args["E"], args["self_rank"], args["c_intra"],
                       args["c_inter"], args["S"], args["W"])


def test_workspace_bytes_ok(tp):
    n = tp.workspace_bytes(base(tp), 512, 2, 1)
    assert n > 0 and n % 256 == 0
    assert tp.workspace_bytes(base(tp), 0, 1, 0) > 0


@pytest.mark.parametrize("kw,T,k,N,rc", [
    (dict(R=0), 8, 1, 1, -1), (dict(G=3), 8, 1, 1, -1), (dict(E=12), 8, 1, 1, -1),
    (dict(self_rank=8), 8, 1, 1, -1), (dict(self_rank=-1), 8, 1, 1, -1),
    (dict(c_intra=-1), 8, 1, 1, -1), (dict(c_inter=-1), 8, 1, 1, -1), (dict(S=0), 8, 1, 1, -1),
    (dict(W=-1), 8, 1, 1, -1), ({}, -1, 1, 1, -1), ({}, 8, 0, 1, -1), ({}, 8, 17, 1, -1),
    ({}, 8, 1, -1, -1), ({}, 1 << 30, 4, 1, -1),
    (dict(R=128, G=128, E=128), 8, 1, 1, -4),
])
def test_workspace_bytes_rejects(tp, kw, T, k, N, rc):
    R = kw.get("R", 8)
    t = base(tp, **kw)
    got, _ = tp.raw_workspace_bytes(t, T, k, N)
    assert got == rc


def test_lds_limit_is_reported(tp):
    # one domain of 64 ranks x 64 instances x 256 sources cannot sit in LDS
    t = base(tp, R=256, G=64, E=256 * 60)
    got, _ = tp.raw_workspace_bytes(t, 16, 1, 4)
    assert got == tp.ELIMIT


def test_plan_rejects_null_and_small_workspace_without_launching(tp):
    t = base(tp)
    ws = tp.workspace_bytes(t, 16, 2, 1)
    # null global_load
    assert tp.raw_plan(ctypes.byref(t), None, 256, 16, 2, 1, 512, 1024, 2048, 4096, 8192, ws, None) == tp.EINVAL
    # misaligned workspace
    assert tp.raw_plan(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, 4096, 8192 + 4, ws,
                       None) == tp.EWORKSPACE
    # too small
    assert tp.raw_plan(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, 4096, 8192, ws - 256,
                       None) == tp.EWORKSPACE
    # bad launch shape
    with pytest.raises(tp.TopoepError):
        tp.workspace_bytes(t, 16, 2, 1, launch=(3, 256, 0, 256))
    with pytest.raises(tp.TopoepError):
        tp.workspace_bytes(t, 16, 2, 1, launch=(4, 96, 0, 256))
    # wait and refinement bounds: -1 (give up at once) is the only negative spin limit
    assert tp.workspace_bytes(t, 16, 2, 1, launch=(0, 0, 0, 0, 0, -1, 5)) == ws
    with pytest.raises(tp.TopoepError):
        tp.workspace_bytes(t, 16, 2, 1, launch=(0, 0, 0, 0, 0, -2, 0))
    with pytest.raises(tp.TopoepError):
        tp.workspace_bytes(t, 16, 2, 1, launch=(0, 0, 0, 0, 0, 0, -1))


def test_plan_shape_choices(tp):
    """One launch when the single-workgroup solver fits and the ids fit 128
    workgroups; three kernels otherwise (host-side choice only)."""
    t = tp.topology(32, 8, 256, 0, 1, 8, 14336, 88080384)
    sh = tp.plan_shape(t, 8192, 8, 2)
    # the fewest ids per thread that keep to 32 chunks: two
    assert sh.kernels == 1 and sh.solver == tp.SOLVER_FUSED and sh.chunk_blocks == 32
    assert sh.grid[0] == 33 and sh.block[0] == 1024 and sh.items_per_thread == 2
    sh = tp.plan_shape(t, 8192, 8, 2, launch=(4, 0, 0, 0, 3))
    assert sh.chunk_blocks == 16 and sh.items_per_thread == 4
    # 512 threads, 8 ids each: 16 chunks
    sh = tp.plan_shape(t, 8192, 8, 2, launch=(8, 0, 0, 512, 3))
    assert sh.chunk_blocks == 16 and sh.block[0] == 512
    # 128 threads, 4 ids each: 128 chunks, the most one launch takes
    sh = tp.plan_shape(t, 8192, 8, 2, launch=(4, 0, 0, 128, 3))
    assert sh.chunk_blocks == 128 and sh.grid[0] == 129
    # 64 threads, 8 ids each would need 128 chunks of 512 ids: still one launch
    assert tp.plan_shape(t, 8192, 8, 2, launch=(8, 0, 0, 64, 3)).chunk_blocks == 128
    with pytest.raises(tp.TopoepError):   # 64 threads, 4 ids: 256 chunks
        tp.plan_shape(t, 8192, 8, 2, launch=(4, 0, 0, 64, 3))
    sh = tp.plan_shape(t, 8192, 8, 2, launch=(0, 0, 0, 0, 1))
    assert sh.kernels == 3 and sh.solver == tp.SOLVER_SINGLE
    # too many ids for 128 one-launch workgroups: three kernels
    sh = tp.plan_shape(t, 1 << 20, 8, 2)
    assert sh.kernels == 3
    with pytest.raises(tp.TopoepError):
        tp.plan_shape(t, 1 << 20, 8, 2, launch=(0, 0, 0, 0, 3))
    # a solver state too large for one workgroup: per-domain solver
    big = tp.topology(256, 8, 512, 0, 1, 16, 4096, 9 << 20)
    sh = tp.plan_shape(big, 16384, 8, 4)
    assert sh.kernels == 3 and sh.solver == tp.SOLVER_PER_DOMAIN
    with pytest.raises(tp.TopoepError):
        tp.plan_shape(t, 8192, 8, 2, launch=(0, 0, 0, 0, 4))


def _no_gpu():
    """True only when this host certainly has no GPU: no /dev/kfd (the ROCm
    kernel driver's node) and torch reports none.  Any doubt, an exception
    included, counts as a GPU, so the placeholder-pointer launches below are
    skipped rather than run where a kernel could start."""
    if os.path.exists("/dev/kfd"):
        return False
    try:
        import torch
        return not torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.skipif(not _no_gpu(), reason="launches on placeholder pointers: only where no GPU is present")
@pytest.mark.parametrize("solver", [0, 1, 2, 3])
def test_valid_calls_reach_the_launch(tp, solver):
    """With no GPU present a valid call passes every host check and fails at
    the launch (EHIP): argument validation accepts every stage the plan has."""
    t = base(tp)
    launch = tp.Launch(0, 0, 0, 0, solver)
    ws = tp.workspace_bytes(t, 16, 2, 1, launch=launch)
    args = (ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, 4096, 8192, ws, None)
    assert tp._lib.topoep_plan_ex(*args, ctypes.byref(launch)) == tp.EHIP
    kernels = tp.plan_shape(t, 16, 2, 1, launch=launch).kernels
    for stage in range(kernels):
        assert tp._lib.topoep_plan_stage(stage, *args, ctypes.byref(launch)) == tp.EHIP, stage
    assert tp._lib.topoep_plan_stage(tp.STAGE_FLOOR, *args, ctypes.byref(launch)) == tp.EHIP
    for stage in range(kernels, 3):
        assert tp._lib.topoep_plan_stage(stage, *args, ctypes.byref(launch)) == tp.EINVAL, stage
    assert tp._lib.topoep_plan_stage(4, *args, ctypes.byref(launch)) == tp.EINVAL


def test_dispatch_workspace_and_host_checks(tp):
    t = base(tp)
    lw = tp.layout_workspace_bytes(t, 512, 2)
    assert lw > 0 and lw % 256 == 0
    assert tp.layout_workspace_bytes(t, 0, 2) > 0
    pw = tp.workspace_bytes(t, 512, 2, 1)
    assert tp.dispatch_workspace_bytes(t, 512, 2, 1) == pw
    out = ctypes.c_size_t(0)
    assert tp._lib.topoep_layout_workspace_bytes(ctypes.byref(t), -1, 2, ctypes.byref(out)) == tp.EINVAL
    assert tp._lib.topoep_layout_workspace_bytes(ctypes.byref(t), 8, 0, ctypes.byref(out)) == tp.EINVAL
    big = base(tp, R=2048, G=8, E=2048)
    assert tp._lib.topoep_layout_workspace_bytes(ctypes.byref(big), 8, 1, ctypes.byref(out)) == tp.ELIMIT
    # layout: null send counts / offsets / workspace, small or misaligned workspace
    L = tp._lib.topoep_dispatch_layout
    assert L(ctypes.byref(t), 256, 512, 2, None, 1024, 2048, None, 4096, lw, None) == tp.EINVAL
    assert L(ctypes.byref(t), 256, 512, 2, 512, None, 2048, None, 4096, lw, None) == tp.EINVAL
    assert L(ctypes.byref(t), None, 512, 2, 512, 1024, 2048, None, 4096, lw, None) == tp.EINVAL
    assert L(ctypes.byref(t), 256, 512, 2, 512, 1024, 2048, None, None, lw, None) == tp.EINVAL
    assert L(ctypes.byref(t), 256, 512, 2, 512, 1024, 2048, None, 4096, lw - 256, None) == tp.EWORKSPACE
    assert L(ctypes.byref(t), 256, 512, 2, 512, 1024, 2048, None, 4096 + 8, lw, None) == tp.EWORKSPACE
    # plan + dispatch: nothing asked beyond the plan, a half-given layout, a small workspace
    D = tp._lib.topoep_plan_dispatch
    dw = tp.dispatch_workspace_bytes(t, 16, 2, 1)
    assert D(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, None, None, None, 4096, 8192, dw,
             None) == tp.EINVAL
    assert D(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, None, 3072, None, 4096, 8192, dw,
             None) == tp.EINVAL
    assert D(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, 2560, 3072, 3584, 4096, 8192, dw - 256,
             None) == tp.EWORKSPACE


@pytest.mark.skipif(not _no_gpu(), reason="launches on placeholder pointers: only where no GPU is present")
def test_valid_dispatch_calls_reach_the_launch(tp):
    t = base(tp)
    lw = tp.layout_workspace_bytes(t, 512, 2)
    assert tp._lib.topoep_dispatch_layout(ctypes.byref(t), 256, 512, 2, 512, 1024, 2048, None, 4096, lw,
                                          None) == tp.EHIP
    dw = tp.dispatch_workspace_bytes(t, 16, 2, 1)
    assert tp._lib.topoep_plan_dispatch(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, 2560, 3072, 3584,
                                        4096, 8192, dw, None) == tp.EHIP
    # receive counts only
    assert tp._lib.topoep_plan_dispatch(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, 2560, None, None,
                                        4096, 8192, dw, None) == tp.EHIP


def test_gather_host_checks(tp):
    t = base(tp)
    G = tp._lib.topoep_gather_replicas
    assert G(None, 1, 256, None, 512, 64, 1024, None) == tp.EINVAL
    assert G(ctypes.byref(t), -1, 256, None, 512, 64, 1024, None) == tp.EINVAL
    assert G(ctypes.byref(t), 1, None, None, 512, 64, 1024, None) == tp.EINVAL
    assert G(ctypes.byref(t), 1, 256, None, None, 64, 1024, None) == tp.EINVAL
    assert G(ctypes.byref(t), 1, 256, None, 512, 64, None, None) == tp.EINVAL
    assert G(ctypes.byref(t), 1, 256, None, 512, 60, 1024, None) == tp.EINVAL     # not a multiple of 16
    assert G(ctypes.byref(t), 1, 256, None, 520, 64, 1024, None) == tp.EINVAL     # misaligned
    assert G(ctypes.byref(base(tp, self_rank=9)), 1, 256, None, 512, 64, 1024, None) == tp.EINVAL
    assert G(ctypes.byref(t), 1 << 17, 256, None, 512, 64, 1024, None) == tp.ELIMIT
    # nothing to copy: no launch, OK even on placeholder pointers
    assert G(ctypes.byref(t), 0, None, None, None, 64, None, None) == tp.OK
    assert G(ctypes.byref(t), 2, 256, None, 512, 0, 1024, None) == tp.OK


def test_costs_workspace_and_shape(tp):
    t = base(tp)
    n = tp.costs_workspace_bytes(t, 512, 2, 1)
    assert n > 0 and n % 256 == 0
    out = ctypes.c_size_t(0)
    # a domain too large for one workgroup's LDS with the cost tables
    big = base(tp, R=256, G=64, E=256 * 60)
    assert tp._lib.topoep_costs_workspace_bytes(ctypes.byref(big), 16, 1, 4, ctypes.byref(out)) == tp.ELIMIT
    assert tp._lib.topoep_costs_workspace_bytes(ctypes.byref(t), -1, 1, 1, ctypes.byref(out)) == tp.EINVAL


@pytest.mark.skipif(not _no_gpu(), reason="launches on placeholder pointers: only where no GPU is present")
def test_valid_costs_call_reaches_the_launch(tp):
    t = base(tp)
    ws = tp.costs_workspace_bytes(t, 16, 2, 1)
    c = tp.Costs(4096, 8192)
    assert tp._lib.topoep_plan_costs(ctypes.byref(t), ctypes.byref(c), 256, 256, 16, 2, 1, 512, 1024, 2048,
                                     2560, 8192 * 2, ws, None) == tp.EHIP
    assert tp._lib.topoep_plan_costs(ctypes.byref(t), None, 256, 256, 16, 2, 1, 512, 1024, 2048,
                                     2560, 8192 * 2, ws, None) == tp.EHIP
    assert tp._lib.topoep_plan_costs(ctypes.byref(t), ctypes.byref(c), None, 256, 16, 2, 1, 512, 1024, 2048,
                                     2560, 8192 * 2, ws, None) == tp.EINVAL


def test_noalloc_host_checks(tp):
    """topoep_plan_noalloc refuses bad arguments and shapes beyond its array
    before any device call (placeholder pointers are never launched on)."""
    t = base(tp)
    P = tp._lib.topoep_plan_noalloc
    assert P(None, 256, 256, 16, 2, 1, 512, 1024, 2048, 4096, None) == tp.EINVAL
    assert P(ctypes.byref(t), None, 256, 16, 2, 1, 512, 1024, 2048, 4096, None) == tp.EINVAL
    assert P(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, None, 4096, None) == tp.EINVAL
    big = tp.topology(32, 8, 256, 0, 1, 8, 14336, 88080384)
    assert tp.workspace_bytes(big, 1 << 20, 8, 2) > tp.NOALLOC_SCRATCH_BYTES
    assert P(ctypes.byref(big), 256, 256, 1 << 20, 8, 2, 512, 1024, 2048, 4096, None) == tp.EWORKSPACE


@pytest.mark.skipif(not _no_gpu(), reason="only where no GPU is present")
def test_noalloc_without_a_device_is_a_hip_error(tp):
    t = base(tp)
    assert tp._lib.topoep_plan_noalloc(ctypes.byref(t), 256, 256, 16, 2, 1, 512, 1024, 2048, 4096, None) == tp.EHIP
