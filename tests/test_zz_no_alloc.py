"""The no-allocation entry point through the C ABI: topoep_plan_noalloc's
outputs equal topoep_plan's on the same inputs, call after call, each call
smaller than the one before (the library's scratch array keeps the previous
call's contents, of another shape), on the one-launch and the three-kernel
paths; a shape that needs more than the array is refused."""
import ctypes

import numpy as np
import pytest

import workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_35481_amd import topoep  # noqa: E402

DEV = torch.device("cuda:0")


def _noalloc(topo, gl_d, tk_d, N, outs):
    T, k = tk_d.shape
    slots, dest, sc, st = outs
    return topoep._lib.topoep_plan_noalloc(
        ctypes.byref(topo), gl_d.data_ptr(), tk_d.data_ptr() if T > 0 else None, T, k, N,
        slots.data_ptr() if slots.numel() else None, dest.data_ptr() if T > 0 else None, sc.data_ptr(),
        st.data_ptr(), torch.cuda.current_stream(DEV).cuda_stream)


def _case(name, layer, N=None):
    cfg = workload.get(name)
    N = cfg.N if N is None else N
    gl, tk = workload.make_layer(cfg, layer, 0, 0)
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    print("case no-alloc", name, "layer", layer, "N", N, "workspace", topoep.workspace_bytes(topo, cfg.T, cfg.k, N),
          flush=True)
    gl_d = torch.from_numpy(gl.copy()).to(DEV)
    tk_d = torch.from_numpy(tk.copy()).to(DEV)
    p = topoep.Planner(topo, cfg.T, cfg.k, N, device=DEV)
    want = [x.clone() for x in p.plan(gl_d, tk_d)]
    outs = [torch.full_like(x, -9) for x in want]
    assert _noalloc(topo, gl_d, tk_d, N, outs) == topoep.OK
    torch.cuda.synchronize()
    for what, a, b in zip(("replica_slots", "token_dest", "send_counts", "status"), outs, want):
        assert torch.equal(a, b), (name, layer, what)
    return p.shape.kernels


def test_noalloc_matches_plan_call_after_call():
    kernels = [_case("stress", 2), _case("dsv3", 4), _case("qwen3", 7), _case("tiny", 0), _case("dsv3", 4),
               _case("mixtral", 5, N=3)]
    assert 3 in kernels and 1 in kernels


def test_noalloc_refuses_a_shape_beyond_its_array():
    topo = topoep.topology(32, 8, 256, 0, 1, 8, 14336, 88080384)
    T, k = 1 << 20, 8
    assert topoep.workspace_bytes(topo, T, k, 2) > topoep.NOALLOC_SCRATCH_BYTES
    gl = torch.zeros((32, 256), dtype=torch.int32, device=DEV)
    tk = torch.zeros((T, k), dtype=torch.int32, device=DEV)
    outs = [torch.empty((32, 2), dtype=torch.int32, device=DEV), torch.empty((T, k), dtype=torch.int32, device=DEV),
            torch.empty((32,), dtype=torch.int32, device=DEV), torch.empty((2,), dtype=torch.int32, device=DEV)]
    assert _noalloc(topo, gl, tk, 2, outs) == topoep.EWORKSPACE
