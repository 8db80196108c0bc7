"""The seeded generator: deterministic, distinct ids per token, consistent
global_load, and the skew features of each configuration."""
import numpy as np
import pytest

import workload
from workload import generate


@pytest.mark.parametrize("name", ["tiny", "mixtral", "qwen3", "dsv3"])
def test_shapes_and_consistency(name):
    cfg = workload.get(name)
    gl, tk = workload.make_layer(cfg, 0, 0, 0)
    assert gl.shape == (cfg.R, cfg.E) and gl.dtype == np.int32
    assert tk.shape == (cfg.T, cfg.k) and tk.dtype == np.int32
    assert ((tk >= 0) & (tk < cfg.E)).all()
    srt = np.sort(tk, axis=1)
    assert (np.diff(srt, axis=1) != 0).all()           # without replacement
    assert (gl.sum(axis=1) == cfg.T * cfg.k).all()
    assert (gl[0] == np.bincount(tk.ravel(), minlength=cfg.E)).all()
    gl2, tk2 = workload.make_layer(cfg, 0, 0, 0)
    assert (gl == gl2).all() and (tk == tk2).all()


def test_layers_differ_and_self_rank_slices():
    cfg = workload.get("tiny")
    g0, t0 = workload.make_layer(cfg, 0, 0, 0)
    g1, t1 = workload.make_layer(cfg, 0, 0, 3)
    assert (g0 == g1).all()
    assert (g1[3] == np.bincount(t1.ravel(), minlength=cfg.E)).all()
    cfg2 = workload.get("mixtral")
    a, _ = workload.make_layer(cfg2, 0)
    b, _ = workload.make_layer(cfg2, 1)
    assert not (a == b).all()


def test_drift_changes_a_tenth_of_the_order():
    cfg = workload.get("qwen3")
    o0 = generate.expert_order(cfg, 0, 0)
    o1 = generate.expert_order(cfg, 0, 1)
    changed = (o0 != o1).sum()
    assert 0 < changed <= cfg.drift_positions
    assert sorted(o1.tolist()) == list(range(cfg.E))


def test_successive_sampling_matches_exact_probabilities():
    """First-k-distinct of iid draws is sampling without replacement: check
    the inclusion probability of a 3-expert, k=2 case against the closed form
    P(e in top-2) = p_e + sum_{f != e} p_f p_e / (1 - p_f)."""
    p = np.array([0.6, 0.3, 0.1])
    rng = np.random.Generator(np.random.PCG64(7))
    ids = generate._successive_sample(rng, p, 200000, np.full(200000, 2))
    freq = np.bincount(ids.ravel(), minlength=3) / 200000
    exact = [p[e] + sum(p[f] * p[e] / (1 - p[f]) for f in range(3) if f != e) for e in range(3)]
    assert np.allclose(freq, exact, atol=0.005)


def test_node_limited_sampling_restricts_nodes():
    cfg = workload.Config("nl", 9, R=8, G=1, E=16, k=4, T=256, N=1, c_intra=1, c_inter=8,
                          S=2, W=10, layers=1, microbatches=1, zipf_s=1.0, node_limit=2)
    allr = workload.all_rank_topk(cfg, 0, 0)
    nodes = allr // (cfg.G * cfg.P)
    for tok in nodes.reshape(-1, cfg.k):
        assert len(set(tok.tolist())) <= 2


def test_adversarial_experts_first():
    cfg = workload.Config("adv", 8, R=4, G=2, E=32, k=8, T=512, N=1, c_intra=1, c_inter=8,
                          S=2, W=10, layers=1, microbatches=1, zipf_s=1.4,
                          adversarial=(0, 1, 2, 3), adv_p=0.6)
    _, tk = workload.make_layer(cfg)
    adv = tk < 4
    # adversarial ids occupy a prefix of the row, in ascending order
    for row, a in zip(tk, adv):
        n = a.sum()
        assert a[:n].all() and not a[n:].any()
        assert (np.diff(row[:n]) > 0).all()
    share = adv.mean()
    assert abs(share - 0.3) < 0.03
