"""CPU oracle of the TopoEP planner -- test infrastructure only.

Plain single-threaded C (``topoep_oracle.c``) following the paper's
Section 4 step by step, loaded through ctypes.  Only the tests, the smoke
check and the benchmark's CPU baseline may import this package; the GPU
library never does, and the two share no code.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "topoep_oracle.c")
_LIB = os.path.join(_HERE, "libtopoep_oracle.so")

ST_BAD_ID = 1
ST_NEG_LOAD = 2
ST_SELF_DIFF = 4
ST_RANGE = 8
ST_ITER = 32
ST_COST = 64
ITER_LIMIT = 1 << 22


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, no vector intrinsics)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class RefTopology(ctypes.Structure):
    _fields_ = [("num_ranks", ctypes.c_int32), ("ranks_per_node", ctypes.c_int32),
                ("num_experts", ctypes.c_int32), ("self_rank", ctypes.c_int32),
                ("cost_intra", ctypes.c_int32), ("cost_inter", ctypes.c_int32),
                ("tok_bytes", ctypes.c_int64), ("expert_bytes", ctypes.c_int64)]


_P32 = ctypes.POINTER(ctypes.c_int32)
_P64 = ctypes.POINTER(ctypes.c_int64)
_P8 = ctypes.POINTER(ctypes.c_uint8)


class RefDebug(ctypes.Structure):
    _fields_ = [("hist", _P32), ("demand", _P32), ("x_stage1", _P8), ("q_routed", _P32),
                ("load_routed", _P32), ("x_final", _P8), ("q_final", _P32), ("load_final", _P32),
                ("iters", _P32), ("move_cap", ctypes.c_int32), ("moves", _P32),
                ("move_dcost", _P64), ("move_m", _P32), ("n_moves", ctypes.c_int32)]


_lib = None


def load_library(path: str):
    """Load an oracle shared library (the default one, or a test-built
    variant) and make it the one ``plan_ref`` calls."""
    global _lib
    lib = ctypes.CDLL(path)
    lib.topoep_plan_ref.restype = ctypes.c_int
    lib.topoep_plan_ref.argtypes = [ctypes.POINTER(RefTopology), _P32, _P32, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_int32, _P32, _P32, _P32, _P32,
                                    ctypes.POINTER(RefDebug)]
    lib.topoep_plan_ref_ex.restype = ctypes.c_int
    lib.topoep_plan_ref_ex.argtypes = [ctypes.POINTER(RefTopology), _P32, _P32, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_int32, _P32, _P32, _P32, _P32, _P32,
                                       ctypes.POINTER(RefDebug)]
    lib.topoep_plan_ref_general.restype = ctypes.c_int
    lib.topoep_plan_ref_general.argtypes = [ctypes.POINTER(RefTopology), _P32, _P64, _P32, _P32, ctypes.c_int32,
                                            ctypes.c_int32, ctypes.c_int32, _P32, _P32, _P32, _P32, _P32,
                                            ctypes.POINTER(RefDebug)]
    lib.topoep_plan_ref_capped.restype = ctypes.c_int
    lib.topoep_plan_ref_capped.argtypes = [ctypes.POINTER(RefTopology), _P32, _P64, _P32, _P32, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_int32, _P32, _P32, _P32, _P32, _P32,
                                           ctypes.POINTER(RefDebug), ctypes.c_int32]
    lib.topoep_layout_ref.restype = ctypes.c_int
    lib.topoep_layout_ref.argtypes = [ctypes.c_int32, _P32, ctypes.c_int64, _P32, _P32, _P32]
    _lib = lib
    return lib


def _load():
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        load_library(_LIB)
    return _lib


def _ptr(a, ty=_P32):
    return a.ctypes.data_as(ty) if a is not None else None


def topology(R, G, E, self_rank, c_intra, c_inter, S, W) -> RefTopology:
    return RefTopology(R, G, E, self_rank, c_intra, c_inter, S, W)


def plan_ref(topo: RefTopology, global_load, local_topk, replica_budget: int,
             debug: bool = False, move_cap: int = 0, raw_rc: bool = False, cost_matrix=None,
             expert_bytes=None, iter_limit: int = ITER_LIMIT):
    """Run the oracle.  Returns a dict of numpy arrays.

    cost_matrix ([R, R] int32) and expert_bytes ([E] int64) select the full
    model of Section 4.1 (a general cost and per-expert sizes).  iter_limit
    bounds the refinement moves of each domain (ST_ITER when a domain still
    had a move after that many).

    Keys: replica_slots [R, N], token_dest [T, k], send_counts [R],
    recv_counts [R] (what each rank sends to this one under the same plan),
    status (the bits), move_count (refinement moves committed), and with
    ``debug``: hist, demand, x_stage1, q_routed, load_routed, x_final,
    q_final, load_final, iters, moves, move_dcost, move_m, n_moves.
    """
    lib = _load()
    gl = np.ascontiguousarray(global_load, dtype=np.int32)
    tk = np.ascontiguousarray(local_topk, dtype=np.int32)
    R, E = topo.num_ranks, topo.num_experts
    T, k = tk.shape if tk.ndim == 2 else (0, 1)
    N = int(replica_budget)
    G = topo.ranks_per_node
    M = R // G if G > 0 and R % G == 0 else 1
    slots = np.full((R, max(N, 0)), -7, dtype=np.int32)
    dest = np.full((T, k), -7, dtype=np.int32)
    sc = np.full(R, -7, dtype=np.int32)
    rcv = np.full(R, -7, dtype=np.int32)
    st = np.zeros(2, dtype=np.int32)
    out = {}
    dbgp = None
    if debug:
        out["hist"] = np.zeros(E, np.int32)
        out["demand"] = np.zeros((M, E), np.int32)
        out["x_stage1"] = np.zeros((E, R), np.uint8)
        out["q_routed"] = np.zeros((R, E, R), np.int32)
        out["load_routed"] = np.zeros(R, np.int32)
        out["x_final"] = np.zeros((E, R), np.uint8)
        out["q_final"] = np.zeros((R, E, R), np.int32)
        out["load_final"] = np.zeros(R, np.int32)
        out["iters"] = np.zeros(M, np.int32)
        out["moves"] = np.zeros((max(move_cap, 1), 6), np.int32)
        out["move_dcost"] = np.zeros(max(move_cap, 1), np.int64)
        out["move_m"] = np.zeros((max(move_cap, 1), R), np.int32)
        dbg = RefDebug(_ptr(out["hist"]), _ptr(out["demand"]), _ptr(out["x_stage1"], _P8),
                       _ptr(out["q_routed"]), _ptr(out["load_routed"]), _ptr(out["x_final"], _P8),
                       _ptr(out["q_final"]), _ptr(out["load_final"]), _ptr(out["iters"]),
                       int(move_cap), _ptr(out["moves"]), _ptr(out["move_dcost"], _P64),
                       _ptr(out["move_m"]), 0)
        dbgp = ctypes.byref(dbg)
    cm = np.ascontiguousarray(cost_matrix, dtype=np.int32) if cost_matrix is not None else None
    wb = np.ascontiguousarray(expert_bytes, dtype=np.int64) if expert_bytes is not None else None
    rc = lib.topoep_plan_ref_capped(ctypes.byref(topo), _ptr(cm), _ptr(wb, _P64), _ptr(gl),
                                    _ptr(tk) if T > 0 else None, T, k, N, _ptr(slots),
                                    _ptr(dest) if T > 0 else None, _ptr(sc), _ptr(rcv), _ptr(st), dbgp,
                                    int(iter_limit))
    if raw_rc:
        return rc
    if rc != 0:
        raise ValueError("topoep_plan_ref returned %d" % rc)
    out.update(replica_slots=slots, token_dest=dest, send_counts=sc, recv_counts=rcv, status=int(st[0]),
               move_count=int(st[1]))
    if debug:
        out["n_moves"] = dbg.n_moves
        nm = min(dbg.n_moves, move_cap)
        out["moves"] = out["moves"][:nm]
        out["move_dcost"] = out["move_dcost"][:nm]
        out["move_m"] = out["move_m"][:nm]
    return out


def layout_ref(R: int, token_dest, send_counts):
    """Dispatch layout of a plan's destinations: (send_offsets [R + 1],
    token_slot with token_dest's shape)."""
    lib = _load()
    td = np.ascontiguousarray(token_dest, dtype=np.int32)
    sc = np.ascontiguousarray(send_counts, dtype=np.int32)
    offs = np.full(R + 1, -7, dtype=np.int32)
    slot = np.full(td.shape, -7, dtype=np.int32)
    rc = lib.topoep_layout_ref(int(R), _ptr(td) if td.size else None, int(td.size), _ptr(sc), _ptr(offs),
                               _ptr(slot) if td.size else None)
    if rc != 0:
        raise ValueError("topoep_layout_ref returned %d" % rc)
    return offs, slot


def gather_ref(replica_slots, self_rank: int, expert_params, slot_params, prev_slots=None):
    """Replica-slot parameter gather (Section 3.2), its plain definition:
    slot j of rank self receives the parameters of expert
    replica_slots[self, j]; an empty slot (-1, or any id outside [0, E)) and,
    with prev_slots, a slot whose expert is unchanged keep their contents.
    Returns a new array; the inputs are not modified."""
    out = np.array(slot_params, copy=True)
    E = expert_params.shape[0]
    for j, e in enumerate(np.asarray(replica_slots)[self_rank]):
        if not 0 <= e < E:
            continue
        if prev_slots is not None and prev_slots[j] == e:
            continue
        out[j] = expert_params[e]
    return out


def plan_cfg(cfg, global_load, local_topk, self_rank: int = 0, **kw):
    """Convenience: oracle plan for a ``workload.Config``."""
    topo = topology(cfg.R, cfg.G, cfg.E, self_rank, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    return plan_ref(topo, global_load, local_topk, cfg.N, **kw)
