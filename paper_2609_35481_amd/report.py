"""Plan-quality and solver-scaling report of the GPU planner.

Quality (the balance study of Section 6.2): on a synthetic 32-rank,
640-expert, top-8 workload, every rank plans from the same Omega with its
own ids (the all-rank sweep), and the plans give
  * the rank loads L[r] = sum over ranks s of send_counts_s[r] (the
    assignments rank r executes) and their maximum-to-mean ratio, per
    replica budget N_slot = 0..4 (0 is static expert parallelism);
  * the fraction of assignments that cross nodes (dom(s) != dom(r));
  * the fraction served by a replica (destination != main(e)).
Scaling (the solver study of Section 6.3): plan latency per layer with the
expert count fixed at 640 and EP 8..128 ranks (8 per node), and with EP 32
and 64..1024 experts.  The latency is the whole plan (histogram, solver,
rerouting), timed as a HIP graph of back-to-back layers.

The inputs are seeded and synthetic (the paper's routing traces are not
available): top-k ids drawn without replacement from a Zipf distribution
over a seed-permuted expert order, every rank simulated.

    python -m paper_2609_35481_amd.report [--quality] [--scaling] [--json]
"""
from __future__ import annotations

import argparse
import dataclasses
import json

import numpy as np

import workload

QUALITY_BASE = workload.Config("quality-640", 6, R=32, G=8, E=640, k=8, T=4096, N=0, c_intra=1, c_inter=8,
                               S=2048 * 2, W=3 * 2048 * 768 * 2, layers=4, microbatches=1, zipf_s=1.0)


# ---------------------------------------------------------------- metrics (plain numpy)

def rank_loads(send_all):
    """L[r] = sum_s send_counts of rank s to r (send_all: [R_self, R])."""
    return np.asarray(send_all, dtype=np.int64).sum(axis=0)


def max_to_mean(loads):
    loads = np.asarray(loads, dtype=np.float64)
    return float(loads.max() / loads.mean()) if loads.mean() > 0 else 0.0


def inter_node_fraction(send_all, G):
    """Share of assignments whose destination sits in another node."""
    send = np.asarray(send_all, dtype=np.int64)
    R = send.shape[1]
    dom = np.arange(R) // G
    cross = dom[:, None] != dom[None, :]
    total = send.sum()
    return float(send[cross].sum() / total) if total else 0.0


def replica_served_fraction(dests, topks, P):
    """Share of assignments executed away from their expert's main rank."""
    served = total = 0
    for d, t in zip(dests, topks):
        d = np.asarray(d).ravel()
        t = np.asarray(t).ravel()
        ok = d >= 0
        served += int((d[ok] != t[ok] // P).sum())
        total += int(ok.sum())
    return served / total if total else 0.0


# ---------------------------------------------------------------- GPU runs

def _topo(topoep, cfg, s):
    return topoep.topology(cfg.R, cfg.G, cfg.E, s, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)


def quality(budgets=(0, 1, 2, 3, 4), zipf=(1.0, 1.2), layers=2):
    import torch
    from paper_2609_35481_amd import topoep
    dev = torch.device("cuda:0")
    rows = []
    for s_z in zipf:
        cfg = dataclasses.replace(QUALITY_BASE, zipf_s=s_z)
        for N in budgets:
            acc = {"max_mean": [], "inter_node": [], "replica_served": [], "moves": 0}
            for layer in range(layers):
                allr = workload.all_rank_topk(cfg, layer, 0)
                gl = np.stack([np.bincount(allr[s].ravel(), minlength=cfg.E) for s in range(cfg.R)]).astype(np.int32)
                gl_d = torch.from_numpy(gl).to(dev)
                sends, dests = [], []
                for s in range(cfg.R):
                    p = topoep.Planner(_topo(topoep, cfg, s), cfg.T, cfg.k, N, device=dev)
                    _, dest, send, st = p.plan(gl_d, torch.from_numpy(np.array(allr[s])).to(dev))
                    torch.cuda.synchronize()
                    if int(st[0].item()) & ~topoep.ST_SELF_DIFF:
                        raise RuntimeError("plan status %d" % int(st[0].item()))
                    sends.append(send.cpu().numpy())
                    dests.append(dest.cpu().numpy())
                    if s == 0:
                        acc["moves"] += int(st[1].item())
                acc["max_mean"].append(max_to_mean(rank_loads(sends)))
                acc["inter_node"].append(inter_node_fraction(sends, cfg.G))
                acc["replica_served"].append(replica_served_fraction(dests, allr, cfg.P))
            rows.append({"zipf": s_z, "N_slot": N, "max_to_mean": float(np.mean(acc["max_mean"])),
                         "inter_node_fraction": float(np.mean(acc["inter_node"])),
                         "replica_served_fraction": float(np.mean(acc["replica_served"])),
                         "refinement_moves_per_layer": acc["moves"] / layers})
    return rows


def _latency(topoep, torch, cfg, layers=4, reps=50):
    dev = torch.device("cuda:0")
    ins = []
    for layer in range(layers):
        gl, tk = workload.make_layer(cfg, layer, 0, 0)
        ins.append((torch.from_numpy(gl).to(dev), torch.from_numpy(np.array(tk)).to(dev)))
    pls = [topoep.Planner(_topo(topoep, cfg, 0), cfg.T, cfg.k, cfg.N, device=dev) for _ in range(layers)]
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        for p, (g, t) in zip(pls, ins):
            p.plan(g, t, stream=stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            for p, (g, t) in zip(pls, ins):
                p.plan(g, t, stream=stream)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for _ in range(5):
            graph.replay()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            graph.replay()
        b.record(stream)
    torch.cuda.synchronize()
    st = torch.stack([p.status for p in pls]).cpu().numpy()
    if (st[:, 0] & ~topoep.ST_SELF_DIFF).any():
        raise RuntimeError("plan status %s" % np.unique(st[:, 0]))
    return a.elapsed_time(b) * 1e3 / (reps * layers), pls[0].shape.as_dict(), float(st[:, 1].mean())


def scaling(ranks=(8, 16, 32, 64, 128), experts=(64, 128, 256, 512, 1024), N=2):
    import torch
    from paper_2609_35481_amd import topoep
    rows = []
    for R in ranks:
        cfg = dataclasses.replace(QUALITY_BASE, name="scale-R%d" % R, cfg_id=7, R=R, N=N)
        us, shape, moves = _latency(topoep, torch, cfg)
        rows.append({"sweep": "EP size, E=640", "R": R, "E": cfg.E, "us_per_layer": us,
                     "kernels": shape["kernels"], "solver": shape["solver"], "moves_per_layer": moves})
    for E in experts:
        cfg = dataclasses.replace(QUALITY_BASE, name="scale-E%d" % E, cfg_id=8, E=E, N=N)
        us, shape, moves = _latency(topoep, torch, cfg)
        rows.append({"sweep": "experts, EP 32", "R": cfg.R, "E": E, "us_per_layer": us,
                     "kernels": shape["kernels"], "solver": shape["solver"], "moves_per_layer": moves})
    return rows


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--quality", action="store_true")
    ap.add_argument("--scaling", action="store_true")
    ap.add_argument("--json", action="store_true")
    args = ap.parse_args()
    both = not (args.quality or args.scaling)
    out = {}
    if args.quality or both:
        out["quality"] = quality()
    if args.scaling or both:
        out["scaling"] = scaling()
    if args.json:
        print(json.dumps(out))
        return
    if "quality" in out:
        print("| Zipf s | N_slot | max/mean rank load | inter-node | replica-served | moves/layer |")
        print("|---|---|---|---|---|---|")
        for r in out["quality"]:
            print("| %.1f | %d | %.2f | %.1f %% | %.1f %% | %.1f |" % (
                r["zipf"], r["N_slot"], r["max_to_mean"], 100 * r["inter_node_fraction"],
                100 * r["replica_served_fraction"], r["refinement_moves_per_layer"]))
    if "scaling" in out:
        print("| sweep | R | E | plan us/layer | kernels | solver | moves/layer |")
        print("|---|---|---|---|---|---|---|")
        for r in out["scaling"]:
            print("| %s | %d | %d | %.1f | %d | %d | %.1f |" % (r["sweep"], r["R"], r["E"], r["us_per_layer"],
                                                              r["kernels"], r["solver"], r["moves_per_layer"]))


if __name__ == "__main__":
    main()
