"""Oracle edge cases: argument errors, status bits, empty batches, k = 1,
duplicates inside one token."""
import numpy as np
import pytest

import oracle


def topo(R=4, G=2, E=8, self_rank=0, cI=1, cX=4, S=1, W=10):
    return oracle.topology(R, G, E, self_rank, cI, cX, S, W)


def base():
    gl = np.zeros((4, 8), np.int32)
    gl[0, [0, 1, 4]] = [3, 3, 8]
    gl[1, [2, 3]] = 3
    gl[2, [4, 5]] = 3
    gl[3, [6, 7]] = 3
    tk = np.repeat(np.arange(8, dtype=np.int32), gl[0]).reshape(-1, 1)
    return gl, tk


@pytest.mark.parametrize("kw", [dict(R=0), dict(G=3), dict(E=6), dict(self_rank=4), dict(self_rank=-1),
                                dict(cI=-1), dict(cX=-2), dict(S=0), dict(W=-1)])
def test_invalid_topology(kw):
    gl, tk = base()
    t = topo(**kw)
    R = max(t.num_ranks, 1)
    E = max(t.num_experts, 1)
    rc = oracle.plan_ref(t, np.zeros((R, E), np.int32), tk, 1, raw_rc=True)
    assert rc == -1


def test_invalid_k_and_budget():
    gl, tk = base()
    assert oracle.plan_ref(topo(), gl, np.zeros((2, 9), np.int32), 1, raw_rc=True) == -1
    assert oracle.plan_ref(topo(), gl, tk, -1, raw_rc=True) == -1


def test_bad_id_sets_status_and_blank_outputs():
    gl, tk = base()
    tk = tk.copy()
    tk[3, 0] = 8
    out = oracle.plan_ref(topo(), gl, tk, 1)
    assert out["status"] & oracle.ST_BAD_ID
    assert (out["replica_slots"] == -1).all()
    assert (out["send_counts"] == 0).all()
    assert (out["token_dest"] == -1).all()


def test_negative_load_sets_status():
    gl, tk = base()
    gl = gl.copy()
    gl[2, 1] = -1
    out = oracle.plan_ref(topo(), gl, tk, 1)
    assert out["status"] == oracle.ST_NEG_LOAD
    assert (out["token_dest"] == -1).all()


def test_self_row_mismatch_is_informational():
    gl, tk = base()
    gl2 = gl.copy()
    gl2[0, 4] = 1   # the plan must still use the histogram of local_topk
    a = oracle.plan_ref(topo(), gl, tk, 1)
    b = oracle.plan_ref(topo(), gl2, tk, 1)
    assert b["status"] == oracle.ST_SELF_DIFF
    for key in ("replica_slots", "token_dest", "send_counts"):
        assert (a[key] == b[key]).all()


def test_range_bit():
    gl, tk = base()
    # 4 S total c + c W >= 2^62
    out = oracle.plan_ref(topo(S=2**50, cX=2**10), gl, tk, 1)
    assert out["status"] & oracle.ST_RANGE
    out = oracle.plan_ref(topo(W=2**61), gl, tk, 1)
    assert out["status"] & oracle.ST_RANGE
    out = oracle.plan_ref(topo(W=2**55), gl, tk, 1)
    assert out["status"] == 0


def test_empty_local_batch():
    gl, tk = base()
    gl = gl.copy()
    gl[0] = 0
    out = oracle.plan_ref(topo(), gl, np.zeros((0, 1), np.int32), 1)
    assert out["status"] == 0
    assert out["token_dest"].shape == (0, 1)
    assert (out["send_counts"] == 0).all()


def test_duplicates_inside_a_token_count_independently():
    gl = np.zeros((2, 2), np.int32)
    tk = np.array([[1, 1], [1, 0]], np.int32)
    gl[0] = np.bincount(tk.ravel(), minlength=2)
    t = oracle.topology(2, 2, 2, 0, 1, 4, 1, 10)
    out = oracle.plan_ref(t, gl, tk, 1, debug=True, move_cap=8)
    assert out["hist"].tolist() == [1, 3]
    assert out["send_counts"].sum() == 4
