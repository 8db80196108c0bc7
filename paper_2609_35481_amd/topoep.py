"""Thin Python binding of the planner's C ABI (include/topoep.h).

Argument marshalling only: torch provides device memory and the current
stream; every step of the plan runs in the HIP kernels of libtopoep.so.
Importing this module fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# TOPOEP_STAMPS=1 loads the instrumented build (phase stamps in the
# workspace's control words; bench.py --phases) instead of the product one.
LIB_PATH = os.path.join(_HERE, "libtopoep_stamps.so" if os.environ.get("TOPOEP_STAMPS") == "1" else "libtopoep.so")

OK = 0
EINVAL = -1
EWORKSPACE = -2
EHIP = -3
ELIMIT = -4

ST_BAD_ID = 1
ST_NEG_LOAD = 2
ST_SELF_DIFF = 4
ST_RANGE = 8
ST_SYNC = 16
ST_ITER = 32
ST_COST = 64

STAGE_HIST = 0
STAGE_SOLVE = 1
STAGE_REROUTE = 2
STAGE_FLOOR = 3

SOLVER_AUTO = 0
SOLVER_SINGLE = 1
SOLVER_PER_DOMAIN = 2
SOLVER_FUSED = 3


class Topology(ctypes.Structure):
    """topoep_topology: R ranks, G per node, E experts, this rank, costs, S_tok, ||W||."""
    _fields_ = [("num_ranks", ctypes.c_int32), ("ranks_per_node", ctypes.c_int32),
                ("num_experts", ctypes.c_int32), ("self_rank", ctypes.c_int32),
                ("cost_intra", ctypes.c_int32), ("cost_inter", ctypes.c_int32),
                ("tok_bytes", ctypes.c_int64), ("expert_bytes", ctypes.c_int64)]


class Launch(ctypes.Structure):
    """topoep_launch: launch shape (results do not depend on it), and the
    bounds of the in-kernel waits (spin_limit: 0 default, -1 give up at
    once) and of the refinement (iter_limit: 0 default).  A tuple of up to
    seven values fills the fields in order."""
    _fields_ = [("items_per_thread", ctypes.c_int32), ("block_threads", ctypes.c_int32),
                ("tiles_per_block", ctypes.c_int32), ("solve_threads", ctypes.c_int32),
                ("solver", ctypes.c_int32), ("spin_limit", ctypes.c_int32),
                ("iter_limit", ctypes.c_int32)]


class Shape(ctypes.Structure):
    """topoep_shape: the kernels one plan enqueues (count, grid, threads, LDS)."""
    _fields_ = [("kernels", ctypes.c_int32), ("solver", ctypes.c_int32),
                ("items_per_thread", ctypes.c_int32), ("chunk_blocks", ctypes.c_int32),
                ("grid", ctypes.c_int32 * 3), ("block", ctypes.c_int32 * 3),
                ("lds_bytes", ctypes.c_int32 * 3)]

    def as_dict(self):
        n = self.kernels
        return {"kernels": n, "solver": self.solver, "items_per_thread": self.items_per_thread,
                "chunk_blocks": self.chunk_blocks, "grid": list(self.grid)[:n],
                "block": list(self.block)[:n], "lds_bytes": list(self.lds_bytes)[:n]}


class Costs(ctypes.Structure):
    """topoep_costs: a general cost matrix [R, R] int32 and per-expert sizes
    [E] int64 (device pointers; 0 = the topology's two-level values)."""
    _fields_ = [("cost", ctypes.c_void_p), ("expert_bytes", ctypes.c_void_p)]


class TopoepError(RuntimeError):
    def __init__(self, fn, rc):
        super().__init__("%s returned %d" % (fn, rc))
        self.rc = rc


if not os.path.exists(LIB_PATH):
    raise ImportError("libtopoep.so is not built (run __graft_entry__.build() or "
                      "python -m paper_2609_35481_amd.build): " + LIB_PATH)

_lib = ctypes.CDLL(LIB_PATH)
_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_lib.topoep_workspace_bytes_ex.restype = ctypes.c_int
_lib.topoep_workspace_bytes_ex.argtypes = [ctypes.POINTER(Topology), _i32, _i32, _i32,
                                           ctypes.POINTER(Launch), ctypes.POINTER(ctypes.c_size_t)]
_lib.topoep_workspace_bytes.restype = ctypes.c_int
_lib.topoep_workspace_bytes.argtypes = [ctypes.POINTER(Topology), _i32, _i32, _i32,
                                        ctypes.POINTER(ctypes.c_size_t)]
_PLAN_ARGS = [ctypes.POINTER(Topology), _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp,
              ctypes.c_size_t, _vp]
_lib.topoep_plan.restype = ctypes.c_int
_lib.topoep_plan.argtypes = _PLAN_ARGS
_lib.topoep_plan_ex.restype = ctypes.c_int
_lib.topoep_plan_ex.argtypes = _PLAN_ARGS + [ctypes.POINTER(Launch)]
_lib.topoep_plan_stage.restype = ctypes.c_int
_lib.topoep_plan_stage.argtypes = [_i32] + _PLAN_ARGS + [ctypes.POINTER(Launch)]
_lib.topoep_plan_shape.restype = ctypes.c_int
_lib.topoep_plan_shape.argtypes = [ctypes.POINTER(Topology), _i32, _i32, _i32, ctypes.POINTER(Launch),
                                   ctypes.POINTER(Shape)]

_lib.topoep_layout_workspace_bytes.restype = ctypes.c_int
_lib.topoep_layout_workspace_bytes.argtypes = [ctypes.POINTER(Topology), _i32, _i32,
                                               ctypes.POINTER(ctypes.c_size_t)]
_lib.topoep_dispatch_layout.restype = ctypes.c_int
_lib.topoep_dispatch_layout.argtypes = [ctypes.POINTER(Topology), _vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp,
                                        ctypes.c_size_t, _vp]
_lib.topoep_dispatch_workspace_bytes.restype = ctypes.c_int
_lib.topoep_dispatch_workspace_bytes.argtypes = [ctypes.POINTER(Topology), _i32, _i32, _i32,
                                                 ctypes.POINTER(ctypes.c_size_t)]
_lib.topoep_plan_dispatch.restype = ctypes.c_int
_lib.topoep_plan_dispatch.argtypes = [ctypes.POINTER(Topology), _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp,
                                      _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]

_lib.topoep_costs_workspace_bytes.restype = ctypes.c_int
_lib.topoep_costs_workspace_bytes.argtypes = [ctypes.POINTER(Topology), _i32, _i32, _i32,
                                              ctypes.POINTER(ctypes.c_size_t)]
_lib.topoep_plan_costs.restype = ctypes.c_int
_lib.topoep_plan_costs.argtypes = [ctypes.POINTER(Topology), ctypes.POINTER(Costs), _vp, _vp, _i32, _i32, _i32,
                                   _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
_lib.topoep_gather_replicas.restype = ctypes.c_int
_lib.topoep_gather_replicas.argtypes = [ctypes.POINTER(Topology), _i32, _vp, _vp, _vp, ctypes.c_int64, _vp, _vp]

_lib.topoep_plan_noalloc.restype = ctypes.c_int
_lib.topoep_plan_noalloc.argtypes = [ctypes.POINTER(Topology), _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp]
NOALLOC_SCRATCH_BYTES = 4 << 20

EXPORTS = ("topoep_workspace_bytes", "topoep_workspace_bytes_ex", "topoep_plan",
           "topoep_plan_ex", "topoep_plan_stage", "topoep_plan_shape",
           "topoep_layout_workspace_bytes", "topoep_dispatch_layout",
           "topoep_dispatch_workspace_bytes", "topoep_plan_dispatch", "topoep_gather_replicas",
           "topoep_costs_workspace_bytes", "topoep_plan_costs", "topoep_plan_noalloc")


def topology(R, G, E, self_rank, c_intra, c_inter, S, W) -> Topology:
    return Topology(R, G, E, self_rank, c_intra, c_inter, S, W)


def _launch_ptr(launch):
    if launch is None:
        return None
    if isinstance(launch, Launch):
        return ctypes.byref(launch)
    return ctypes.byref(Launch(*launch))


def workspace_bytes(topo: Topology, T: int, k: int, replica_budget: int, launch=None) -> int:
    out = ctypes.c_size_t(0)
    rc = _lib.topoep_workspace_bytes_ex(ctypes.byref(topo), T, k, replica_budget,
                                        _launch_ptr(launch), ctypes.byref(out))
    if rc != OK:
        raise TopoepError("topoep_workspace_bytes", rc)
    return out.value


def plan_shape(topo: Topology, T: int, k: int, replica_budget: int, launch=None) -> Shape:
    out = Shape()
    rc = _lib.topoep_plan_shape(ctypes.byref(topo), T, k, replica_budget, _launch_ptr(launch),
                                ctypes.byref(out))
    if rc != OK:
        raise TopoepError("topoep_plan_shape", rc)
    return out


def layout_workspace_bytes(topo: Topology, T: int, k: int) -> int:
    out = ctypes.c_size_t(0)
    rc = _lib.topoep_layout_workspace_bytes(ctypes.byref(topo), T, k, ctypes.byref(out))
    if rc != OK:
        raise TopoepError("topoep_layout_workspace_bytes", rc)
    return out.value


def dispatch_workspace_bytes(topo: Topology, T: int, k: int, replica_budget: int) -> int:
    out = ctypes.c_size_t(0)
    rc = _lib.topoep_dispatch_workspace_bytes(ctypes.byref(topo), T, k, replica_budget, ctypes.byref(out))
    if rc != OK:
        raise TopoepError("topoep_dispatch_workspace_bytes", rc)
    return out.value


def _aligned_workspace(nbytes, dev):
    """A zero-filled byte tensor and the 256-byte aligned address inside it."""
    ws = torch.zeros(nbytes + 256, dtype=torch.uint8, device=dev)
    return ws, (ws.data_ptr() + 255) & ~255


def _stream_ptr(stream, dev):
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev_i32(t, name, shape=None):
    if not isinstance(t, torch.Tensor) or t.dtype != torch.int32 or not t.is_cuda:
        raise TypeError("%s must be a CUDA int32 tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    return t


def _same_device(dev, **tensors):
    """Every given tensor (None skipped) lives where the outputs and the
    workspace do."""
    for name, t in tensors.items():
        if t is not None and t.device != dev:
            raise ValueError("%s is on %s, the planner's memory on %s" % (name, t.device, dev))


class Planner:
    """Holds the output tensors and workspace of one (topology, T, k, N)
    problem so repeated plans allocate nothing (and can be graph-captured)."""

    def __init__(self, topo: Topology, T: int, k: int, replica_budget: int, device=None, launch=None):
        self.topo = topo
        self.T, self.k, self.N = int(T), int(k), int(replica_budget)
        self.launch = launch
        dev = torch.device(device if device is not None else "cuda")
        R = topo.num_ranks
        self.ws_bytes = workspace_bytes(topo, self.T, self.k, self.N, launch)
        self.shape = plan_shape(topo, self.T, self.k, self.N, launch)
        # 256-byte aligned workspace carved from a byte tensor, zero-filled
        # once (every plan leaves its control words zero again)
        self._ws = torch.zeros(self.ws_bytes + 256, dtype=torch.uint8, device=dev)
        base = self._ws.data_ptr()
        self.ws_ptr = (base + 255) & ~255
        self.replica_slots = torch.empty((R, self.N), dtype=torch.int32, device=dev)
        self.token_dest = torch.empty((self.T, self.k), dtype=torch.int32, device=dev)
        self.send_counts = torch.empty((R,), dtype=torch.int32, device=dev)
        # status[0] = TOPOEP_ST_* bits, status[1] = refinement moves committed
        self.status = torch.empty((2,), dtype=torch.int32, device=dev)

    def _args(self, global_load, local_topk, stream):
        R, E = self.topo.num_ranks, self.topo.num_experts
        _dev_i32(global_load, "global_load", (R, E))
        if self.T > 0:
            _dev_i32(local_topk, "local_topk", (self.T, self.k))
        _same_device(self._ws.device, global_load=global_load, local_topk=local_topk if self.T > 0 else None)
        if stream is None:
            stream = torch.cuda.current_stream(global_load.device)
        sp = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        return (ctypes.byref(self.topo), global_load.data_ptr(),
                local_topk.data_ptr() if self.T > 0 else None, self.T, self.k, self.N,
                self.replica_slots.data_ptr() if self.replica_slots.numel() else None,
                self.token_dest.data_ptr() if self.T > 0 else None,
                self.send_counts.data_ptr(), self.status.data_ptr(), self.ws_ptr,
                self.ws_bytes, sp)

    def plan(self, global_load, local_topk, stream=None, launch=None):
        """Enqueue topoep_plan_ex; returns (replica_slots, token_dest, send_counts, status).
        ``launch`` overrides the planner's launch for this call; it must keep
        the same shape (only spin_limit and iter_limit may differ)."""
        if launch is not None and plan_shape(self.topo, self.T, self.k, self.N, launch).as_dict() != \
                self.shape.as_dict():
            raise ValueError("a per-call launch must keep the planner's shape")
        rc = _lib.topoep_plan_ex(*self._args(global_load, local_topk, stream),
                                 _launch_ptr(self.launch if launch is None else launch))
        if rc != OK:
            raise TopoepError("topoep_plan", rc)
        return self.replica_slots, self.token_dest, self.send_counts, self.status

    def stage(self, stage: int, global_load, local_topk, stream=None):
        """Enqueue one kernel of the plan (three kernels: 0 hist, 1 solve,
        2 reroute; one kernel: 0), or STAGE_FLOOR: the plan's kernels with
        empty bodies."""
        rc = _lib.topoep_plan_stage(stage, *self._args(global_load, local_topk, stream),
                                    _launch_ptr(self.launch))
        if rc != OK:
            raise TopoepError("topoep_plan_stage", rc)

    def workspace_view(self) -> torch.Tensor:
        off = self.ws_ptr - self._ws.data_ptr()
        return self._ws[off:off + self.ws_bytes]


def costs_workspace_bytes(topo: Topology, T: int, k: int, replica_budget: int) -> int:
    out = ctypes.c_size_t(0)
    rc = _lib.topoep_costs_workspace_bytes(ctypes.byref(topo), T, k, replica_budget, ctypes.byref(out))
    if rc != OK:
        raise TopoepError("topoep_costs_workspace_bytes", rc)
    return out.value


class CostPlanner:
    """Plans under the full cost model of Section 4.1 (topoep_plan_costs): a
    general cost matrix (CUDA int32 [R, R]) and/or per-expert sizes (CUDA
    int64 [E]); None keeps the topology's value."""

    def __init__(self, topo: Topology, T: int, k: int, replica_budget: int, cost=None, expert_bytes=None,
                 device=None):
        self.topo = topo
        self.T, self.k, self.N = int(T), int(k), int(replica_budget)
        dev = torch.device(device if device is not None else "cuda")
        R, E = topo.num_ranks, topo.num_experts
        if cost is not None:
            _dev_i32(cost, "cost", (R, R))
        if expert_bytes is not None:
            if expert_bytes.dtype != torch.int64 or not expert_bytes.is_cuda or tuple(expert_bytes.shape) != (E,):
                raise TypeError("expert_bytes must be a CUDA int64 tensor of shape [E]")
        self.cost, self.expert_bytes = cost, expert_bytes
        self.costs = Costs(cost.data_ptr() if cost is not None else None,
                           expert_bytes.data_ptr() if expert_bytes is not None else None)
        self.ws_bytes = costs_workspace_bytes(topo, self.T, self.k, self.N)
        self._ws, self.ws_ptr = _aligned_workspace(self.ws_bytes, dev)
        self.replica_slots = torch.empty((R, self.N), dtype=torch.int32, device=dev)
        self.token_dest = torch.empty((self.T, self.k), dtype=torch.int32, device=dev)
        self.send_counts = torch.empty((R,), dtype=torch.int32, device=dev)
        self.status = torch.empty((2,), dtype=torch.int32, device=dev)

    def plan(self, global_load, local_topk, stream=None):
        """Enqueue topoep_plan_costs; returns (replica_slots, token_dest, send_counts, status)."""
        R, E = self.topo.num_ranks, self.topo.num_experts
        _dev_i32(global_load, "global_load", (R, E))
        t = self.T > 0
        if t:
            _dev_i32(local_topk, "local_topk", (self.T, self.k))
        _same_device(self._ws.device, global_load=global_load, local_topk=local_topk if t else None,
                     cost=self.cost, expert_bytes=self.expert_bytes)
        rc = _lib.topoep_plan_costs(
            ctypes.byref(self.topo), ctypes.byref(self.costs), global_load.data_ptr(),
            local_topk.data_ptr() if t else None, self.T, self.k, self.N,
            self.replica_slots.data_ptr() if self.replica_slots.numel() else None,
            self.token_dest.data_ptr() if t else None, self.send_counts.data_ptr(), self.status.data_ptr(),
            self.ws_ptr, self.ws_bytes, _stream_ptr(stream, global_load.device))
        if rc != OK:
            raise TopoepError("topoep_plan_costs", rc)
        return self.replica_slots, self.token_dest, self.send_counts, self.status


class DispatchPlanner:
    """Plan plus its dispatch side (receive counts, send offsets, send-buffer
    slot of every assignment) with preallocated outputs and workspace."""

    def __init__(self, topo: Topology, T: int, k: int, replica_budget: int, device=None):
        self.topo = topo
        self.T, self.k, self.N = int(T), int(k), int(replica_budget)
        dev = torch.device(device if device is not None else "cuda")
        R = topo.num_ranks
        self.ws_bytes = dispatch_workspace_bytes(topo, self.T, self.k, self.N)
        self._ws, self.ws_ptr = _aligned_workspace(self.ws_bytes, dev)
        self.replica_slots = torch.empty((R, self.N), dtype=torch.int32, device=dev)
        self.token_dest = torch.empty((self.T, self.k), dtype=torch.int32, device=dev)
        self.send_counts = torch.empty((R,), dtype=torch.int32, device=dev)
        self.recv_counts = torch.empty((R,), dtype=torch.int32, device=dev)
        self.send_offsets = torch.empty((R + 1,), dtype=torch.int32, device=dev)
        self.token_slot = torch.empty((self.T, self.k), dtype=torch.int32, device=dev)
        self.status = torch.empty((2,), dtype=torch.int32, device=dev)

    def plan(self, global_load, local_topk, stream=None):
        """Enqueue topoep_plan_dispatch; returns (replica_slots, token_dest,
        send_counts, recv_counts, send_offsets, token_slot, status)."""
        R, E = self.topo.num_ranks, self.topo.num_experts
        _dev_i32(global_load, "global_load", (R, E))
        if self.T > 0:
            _dev_i32(local_topk, "local_topk", (self.T, self.k))
        t = self.T > 0
        _same_device(self._ws.device, global_load=global_load, local_topk=local_topk if t else None)
        rc = _lib.topoep_plan_dispatch(
            ctypes.byref(self.topo), global_load.data_ptr(), local_topk.data_ptr() if t else None,
            self.T, self.k, self.N, self.replica_slots.data_ptr() if self.replica_slots.numel() else None,
            self.token_dest.data_ptr() if t else None, self.send_counts.data_ptr(),
            self.recv_counts.data_ptr(), self.send_offsets.data_ptr(), self.token_slot.data_ptr() if t else None,
            self.status.data_ptr(), self.ws_ptr, self.ws_bytes, _stream_ptr(stream, global_load.device))
        if rc != OK:
            raise TopoepError("topoep_plan_dispatch", rc)
        return (self.replica_slots, self.token_dest, self.send_counts, self.recv_counts, self.send_offsets,
                self.token_slot, self.status)


class LayoutPlanner:
    """The send-buffer layout alone (topoep_dispatch_layout) for a fixed
    number of assignments, with preallocated outputs and workspace."""

    def __init__(self, topo: Topology, T: int, k: int, device=None):
        self.topo = topo
        self.T, self.k = int(T), int(k)
        dev = torch.device(device if device is not None else "cuda")
        R = topo.num_ranks
        self.ws_bytes = layout_workspace_bytes(topo, self.T, self.k)
        self._ws, self.ws_ptr = _aligned_workspace(self.ws_bytes, dev)
        self.send_offsets = torch.empty((R + 1,), dtype=torch.int32, device=dev)
        self.token_slot = torch.empty((self.T, self.k), dtype=torch.int32, device=dev)
        self.status = torch.zeros((1,), dtype=torch.int32, device=dev)

    def layout(self, token_dest, send_counts, stream=None):
        """Enqueue topoep_dispatch_layout; returns (send_offsets, token_slot)."""
        R = self.topo.num_ranks
        _dev_i32(send_counts, "send_counts", (R,))
        t = self.T > 0
        if t:
            _dev_i32(token_dest, "token_dest", (self.T, self.k))
        _same_device(self._ws.device, send_counts=send_counts, token_dest=token_dest if t else None)
        rc = _lib.topoep_dispatch_layout(
            ctypes.byref(self.topo), token_dest.data_ptr() if t else None, self.T, self.k, send_counts.data_ptr(),
            self.send_offsets.data_ptr(), self.token_slot.data_ptr() if t else None, self.status.data_ptr(),
            self.ws_ptr, self.ws_bytes, _stream_ptr(stream, send_counts.device))
        if rc != OK:
            raise TopoepError("topoep_dispatch_layout", rc)
        return self.send_offsets, self.token_slot


def plan_noalloc(topo: Topology, global_load, local_topk, replica_budget: int, replica_slots, token_dest,
                 send_counts, status, stream=None):
    """Enqueue topoep_plan_noalloc into caller-given outputs (nothing is
    allocated, here or in the library); raises TopoepError on a nonzero
    return code."""
    R, E = topo.num_ranks, topo.num_experts
    _dev_i32(global_load, "global_load", (R, E))
    T, k = (local_topk.shape[0], local_topk.shape[1]) if local_topk is not None else (0, 1)
    if T > 0:
        _dev_i32(local_topk, "local_topk", (T, k))
        _dev_i32(token_dest, "token_dest", (T, k))
    _dev_i32(send_counts, "send_counts", (R,))
    _dev_i32(status, "status", (2,))
    if replica_slots.numel():
        _dev_i32(replica_slots, "replica_slots", (R, replica_budget))
    rc = _lib.topoep_plan_noalloc(
        ctypes.byref(topo), global_load.data_ptr(), local_topk.data_ptr() if T > 0 else None, T, k,
        int(replica_budget), replica_slots.data_ptr() if replica_slots.numel() else None,
        token_dest.data_ptr() if T > 0 else None, send_counts.data_ptr(), status.data_ptr(),
        _stream_ptr(stream, global_load.device))
    if rc != OK:
        raise TopoepError("topoep_plan_noalloc", rc)


def gather_replicas(topo: Topology, replica_slots, expert_params, slot_params, prev_slots=None, stream=None):
    """Enqueue topoep_gather_replicas: slot j of rank topo.self_rank receives
    expert_params[replica_slots[self, j]] (empty or unchanged slots are not
    written).  expert_params [E, ...] and slot_params [N, ...] are CUDA
    tensors of one dtype and one per-expert shape."""
    R, E = topo.num_ranks, topo.num_experts
    _dev_i32(replica_slots, "replica_slots")
    if replica_slots.dim() != 2 or replica_slots.shape[0] != R:
        raise ValueError("replica_slots must be [R, N]")
    N = int(replica_slots.shape[1])
    if not (expert_params.is_cuda and slot_params.is_cuda) or expert_params.dtype != slot_params.dtype:
        raise TypeError("expert_params and slot_params must be CUDA tensors of one dtype")
    if not (expert_params.is_contiguous() and slot_params.is_contiguous()):
        raise ValueError("expert_params and slot_params must be contiguous")
    if expert_params.shape[0] != E or slot_params.shape[0] != N or expert_params.shape[1:] != slot_params.shape[1:]:
        raise ValueError("expert_params must be [E, ...] and slot_params [N, ...] with the same per-expert shape")
    per = expert_params[0].numel() * expert_params.element_size() if E else 0
    if prev_slots is not None:
        _dev_i32(prev_slots, "prev_slots", (N,))
    rc = _lib.topoep_gather_replicas(
        ctypes.byref(topo), N, replica_slots.data_ptr(), prev_slots.data_ptr() if prev_slots is not None else None,
        expert_params.data_ptr(), per, slot_params.data_ptr(), _stream_ptr(stream, replica_slots.device))
    if rc != OK:
        raise TopoepError("topoep_gather_replicas", rc)
    return slot_params


def plan(topo: Topology, global_load, local_topk, replica_budget: int, stream=None, launch=None):
    """One-shot plan: allocates outputs and workspace, enqueues topoep_plan.

    Returns (replica_slots [R, N], token_dest [T, k], send_counts [R], status [2])
    as CUDA int32 tensors, valid once the stream reaches them.
    """
    T, k = (int(local_topk.shape[0]), int(local_topk.shape[1])) if local_topk is not None else (0, 1)
    p = Planner(topo, T, k, replica_budget, device=global_load.device, launch=launch)
    # The workspace returns to torch's caching allocator with the Planner;
    # reuse of that memory is ordered after these kernels on the same stream.
    return p.plan(global_load, local_topk, stream)


def raw_plan(*args):
    """Direct call of topoep_plan with raw pointers (for ABI tests)."""
    return _lib.topoep_plan(*args)


def raw_workspace_bytes(topo, T, k, N):
    out = ctypes.c_size_t(0)
    rc = _lib.topoep_workspace_bytes(ctypes.byref(topo), T, k, N, ctypes.byref(out))
    return rc, out.value
