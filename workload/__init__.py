"""Seeded synthetic inputs for the TopoEP planner (no planner arithmetic here)."""
from .configs import CONFIGS, Config, get  # noqa: F401
from .generate import all_rank_topk, expert_order, make_layer, make_layers  # noqa: F401
