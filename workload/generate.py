"""Seeded synthetic routing for the TopoEP planner.

Stands in for the natural routing of the paper's MoE models (Section 2.2
reports per-layer max/mean expert load of about 7 and 16-20 % churn of the
hottest experts between microbatches; Section 6.4 adds a synthetic
``router_skew`` generator).  Neither the paper's datasets nor its trained
routers are used; every array here is drawn from a seeded PCG64 stream.

Recipe (all steps deterministic in (config, layer, microbatch)):

* Expert popularity is Zipf(s) over a per-layer permutation of the experts:
  the expert at position i of the order has weight (i + 1) ** -s.
* A token's top-k ids are drawn without replacement by successive sampling:
  draws with replacement by inverse CDF, keeping the first k distinct ids in
  draw order (exactly sequential sampling without replacement).
* Drift (Qwen3-like): at microbatch m > 0 the order of microbatch m - 1 has
  the experts at ``drift_positions`` seeded positions shuffled among
  themselves.
* Node limit (DeepSeek-V3-like): each token first picks at most
  ``node_limit`` nodes without replacement, weighted by the Zipf mass of
  the experts whose main instance is on that node, then samples experts
  only from those nodes.  When the topology has no more nodes than the
  limit every node is picked and the restriction is vacuous, so no node
  draw is made.
* Adversarial experts (Stress): each listed expert is included in a token
  independently with probability ``adv_p`` and listed first in ascending
  id; the remaining slots are successive Zipf draws over the other experts.
* Every simulated rank's routing is drawn; ``global_load[s, :]`` is the
  count of expert ids in rank s's top-k array (the all-gathered routing
  matrix a rank would receive), and ``local_topk`` is rank ``self_rank``'s
  array.

This module holds no step of the planner; both the oracle tests and the
GPU path read the arrays it returns.
"""
from __future__ import annotations

import functools

import numpy as np

from .configs import Config

SEED_TAG = 0x70E9


def zipf_weights(n: int, s: float) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


def base_order(cfg: Config, layer: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_TAG, cfg.cfg_id, layer, 0xFFFF])))
    return rng.permutation(cfg.E).astype(np.int64)


@functools.lru_cache(maxsize=256)
def expert_order(cfg: Config, layer: int, mb: int) -> np.ndarray:
    """Popularity order: order[i] is the expert with the i-th largest weight."""
    order = base_order(cfg, layer)
    for m in range(1, mb + 1):
        if cfg.drift_positions <= 0:
            break
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([SEED_TAG, cfg.cfg_id, layer, m, 0xD1F7])))
        pos = rng.choice(cfg.E, size=cfg.drift_positions, replace=False)
        order = order.copy()
        order[pos] = order[pos[rng.permutation(len(pos))]]
    order.setflags(write=False)
    return order


def expert_probs(cfg: Config, layer: int, mb: int, exclude=()) -> np.ndarray:
    """Per-expert probability (indexed by expert id) under the layer's Zipf order."""
    order = expert_order(cfg, layer, mb)
    keep = np.ones(cfg.E, dtype=bool)
    keep[list(exclude)] = False
    order = order[keep[order]]
    p = np.zeros(cfg.E, dtype=np.float64)
    p[order] = zipf_weights(len(order), cfg.zipf_s)
    return p


def _first_distinct(draws: np.ndarray, need: np.ndarray, valid: np.ndarray | None = None,
                    n_values: int | None = None):
    """For each row keep the first need[row] distinct (valid) values in draw order.

    Returns (out[n, max_need] filled with -1 beyond need, got[n]).
    """
    n, m = draws.shape
    if n_values is None:
        n_values = int(draws.max()) + 1 if draws.size else 1
    kmax = int(need.max()) if n else 0
    out = np.full((n, kmax), -1, dtype=np.int64)
    got = np.zeros(n, dtype=np.int64)
    seen = np.zeros((n, n_values), dtype=bool)
    rows = np.arange(n)
    for j in range(m):
        v = draws[:, j]
        fresh = ~seen[rows, v] & (got < need)
        if valid is not None:
            fresh &= valid[:, j]
        seen[rows, v] |= fresh
        r = rows[fresh]
        out[r, got[r]] = v[r]
        got += fresh
    return out, got


def _successive_sample(rng, p: np.ndarray, n: int, need: np.ndarray, allowed: np.ndarray | None = None):
    """Successive sampling without replacement: need[i] ids for token i.

    ``allowed[i, e]`` (optional) restricts token i to a subset of experts; draws
    outside the subset are rejected, which samples from the renormalised
    restriction.
    """
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    kmax = int(need.max()) if n else 0
    out = np.full((n, kmax), -1, dtype=np.int64)
    if kmax == 0:
        return out
    m = max(2 * kmax, 4)
    pending = np.arange(n)
    # Rows that do not reach need[i] distinct values get more draws appended
    # to their own stream, so each token sees one continuous sequence.
    acc = {}
    while pending.size:
        u = rng.random((pending.size, m))
        d = np.searchsorted(cdf, u, side="right")
        d = np.minimum(d, len(p) - 1)
        prev = acc.get("d")
        if prev is None:
            cur = d
        else:
            cur = np.concatenate([prev, d], axis=1)
        valid = None
        if allowed is not None:
            valid = allowed[pending[:, None], cur]
        res, got = _first_distinct(cur, need[pending], valid, len(p))
        done = got >= need[pending]
        out[pending[done], :res.shape[1]] = res[done]
        acc["d"] = cur[~done]
        pending = pending[~done]
    return out


@functools.lru_cache(maxsize=8)
def _layer_all_ranks(cfg: Config, layer: int, mb: int) -> np.ndarray:
    """Top-k ids of every simulated rank: int32 array [R, T, k]."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_TAG, cfg.cfg_id, layer, mb])))
    R, T, k, E = cfg.R, cfg.T, cfg.k, cfg.E
    out = np.empty((R, T, k), dtype=np.int32)
    P = cfg.P
    G = cfg.G
    M = cfg.M
    chunk = max(1, (1 << 19) // max(1, T * k))   # ranks per generation chunk
    for r0 in range(0, R, chunk):
        r1 = min(R, r0 + chunk)
        n = (r1 - r0) * T
        if cfg.adversarial:
            adv = np.array(sorted(cfg.adversarial), dtype=np.int64)
            inc = rng.random((n, len(adv))) < cfg.adv_p
            a_cnt = inc.sum(axis=1)
            p = expert_probs(cfg, layer, mb, exclude=tuple(adv))
            rest = _successive_sample(rng, p, n, k - a_cnt)
            # included adversarial ids first, ascending, then the successive draws
            big = np.iinfo(np.int64).max
            adv_sorted = np.sort(np.where(inc, adv[None, :], big), axis=1)
            ids = np.empty((n, k), dtype=np.int64)
            rows = np.arange(n)
            for j in range(k):
                from_adv = j < a_cnt
                aj = adv_sorted[:, min(j, len(adv) - 1)]
                rj = rest[rows, np.clip(j - a_cnt, 0, rest.shape[1] - 1)]
                ids[:, j] = np.where(from_adv, aj, rj)
        elif cfg.node_limit and M > cfg.node_limit:
            p = expert_probs(cfg, layer, mb)
            node_mass = p.reshape(M, G * P).sum(axis=1)
            nodes = _successive_sample(rng, node_mass, n, np.full(n, cfg.node_limit))
            allowed_nodes = np.zeros((n, M), dtype=bool)
            allowed_nodes[np.arange(n)[:, None], nodes] = True
            allowed = np.repeat(allowed_nodes, G * P, axis=1)
            ids = _successive_sample(rng, p, n, np.full(n, k), allowed)
        else:
            p = expert_probs(cfg, layer, mb)
            ids = _successive_sample(rng, p, n, np.full(n, k))
        out[r0:r1] = ids.reshape(r1 - r0, T, k).astype(np.int32)
    out.setflags(write=False)
    return out


def make_layer(cfg: Config, layer: int = 0, mb: int = 0, self_rank: int = 0):
    """Inputs of one plan: (global_load[R, E] int32, local_topk[T, k] int32)."""
    allr = _layer_all_ranks(cfg, layer, mb)
    gl = np.empty((cfg.R, cfg.E), dtype=np.int32)
    for s in range(cfg.R):
        gl[s] = np.bincount(allr[s].ravel(), minlength=cfg.E)
    return gl, np.ascontiguousarray(allr[self_rank])


def all_rank_topk(cfg: Config, layer: int = 0, mb: int = 0) -> np.ndarray:
    """Top-k arrays of every simulated rank, [R, T, k] int32 (read-only)."""
    return _layer_all_ranks(cfg, layer, mb)


def _make_layer_job(args):
    cfg, layer, mb, self_rank = args
    return make_layer(cfg, layer, mb, self_rank)


def make_layers(cfg: Config, keys, self_rank: int = 0, workers: int = 8):
    """make_layer for every (layer, microbatch) of keys, in a pool of fresh
    interpreter processes (spawned, so a caller that holds a GPU does not
    hand it to them); returns the inputs in the order of keys."""
    jobs = [(cfg, layer, mb, self_rank) for layer, mb in keys]
    if workers <= 1 or len(jobs) <= 1:
        return [_make_layer_job(j) for j in jobs]
    import multiprocessing as mp
    with mp.get_context("spawn").Pool(min(workers, len(jobs))) as pool:
        return pool.map(_make_layer_job, jobs)
