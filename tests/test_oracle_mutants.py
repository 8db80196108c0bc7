"""The pins catch plausible mistakes: each mutant is the oracle's C source
with one planted error (a dropped factor, a flipped order, a wrong index, an
off-by-one), compiled on the CPU into a temporary library.  The pin battery
(paper fixtures, brute force, invariants, the refinement enumerator) must
fail on every mutant.  A mutant that runs past the time limit also counts as
caught.  Nothing here touches the GPU.
"""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "topoep_oracle.c")

MUTANTS = [
    ("benefit without the factor 2",
     "int64_t b = 2 * D[(size_t)d * E + e] * m.S - wexp(&m, e);", "int64_t b = D[(size_t)d * E + e] * m.S - wexp(&m, e);"),
    ("benefit test not strict", "if (b > 0) {", "if (b >= 0) {"),
    ("candidates in ascending benefit",
     "if (a->b != b->b) return a->b > b->b ? -1 : 1;", "if (a->b != b->b) return a->b < b->b ? -1 : 1;"),
    ("stage-1 slot ties to the highest rank",
     "if (best < 0 || used[r] < used[best]) best = r;", "if (best < 0 || used[r] <= used[best]) best = r;"),
    ("demand summed over the wrong domain",
     "D[(size_t)dom(&m, s) * E + e] += omega", "D[(size_t)dom(&m, (s + m.G) % m.R) * E + e] += omega"),
    ("remainder to the highest ranks",
     "Q(s, e, inst[i]) = w / n + (i < w % n ? 1 : 0);", "Q(s, e, inst[i]) = w / n + (i >= n - w % n ? 1 : 0);"),
    ("no same-domain preference",
     "if (X(e, r) && dom(&m, r) == dom(&m, s)) inst[n++] = r;", "if (0) inst[n++] = r;"),
    ("refinement moves more than half the gap", "int64_t delta = gap / 2;", "int64_t delta = (gap + 1) / 2;"),
    ("target load descending",
     "if (a->load_t != b->load_t) return a->load_t < b->load_t;",
     "if (a->load_t != b->load_t) return a->load_t > b->load_t;"),
    ("cost change ascending ignored",
     "if (a->dcost != b->dcost) return a->dcost < b->dcost;", "if (0) return 0;"),
    ("busiest-rank ties to the highest rank", "if (L[r] > L[rb]) rb = r;", "if (L[r] >= L[rb]) rb = r;"),
    ("sources walked in descending cost order",
     "if (a->diff != b->diff) return a->diff < b->diff ? -1 : 1;",
     "if (a->diff != b->diff) return a->diff > b->diff ? -1 : 1;"),
    ("replica transfer cost dropped",
     "(hosts ? 0 : cost(&m, main_rank(&m, e), rt) * wexp(&m, e))", "0"),
    ("token cost change with the wrong sign", "int64_t dcost = 2 * m.S * dtok +", "int64_t dcost = -2 * m.S * dtok +"),
    ("rerouting off by one", "if (rho < prefix + c) {", "if (rho <= prefix + c) {"),
    ("send counts read the wrong index",
     "for (int e = 0; e < E; ++e) sc += Q(m.self, e, r);", "for (int e = 0; e < E; ++e) sc += Q(r, e, m.self);"),
    ("histogram not used as row self", "omega[(size_t)m.self * E + e] = hist[e];", "(void)0;"),
    ("full slots still accept replicas", "if (!hosts && used[rt] >= N) continue;", "if (!hosts && used[rt] > N) continue;"),
    ("one expert size for every expert",
     "static int64_t wexp(const model *m, int e) { return m->We ? m->We[e] : m->W; }",
     "static int64_t wexp(const model *m, int e) { (void)e; return m->W; }"),
    ("replica cost from the target's own expert size",
     "(hosts ? 0 : cost(&m, main_rank(&m, e), rt) * wexp(&m, e))",
     "(hosts ? 0 : cost(&m, main_rank(&m, e), rt) * wexp(&m, rt % m.E))"),
    ("general cost read as the two-level one",
     "  if (m->C) return m->C[(size_t)s * m->R + r];\n", ""),
    ("asymmetric matrix accepted",
     "if (c < 0 || c != m.C[(size_t)r * R + s] || (s == r && c != 0)) st |= REF_ST_COST;",
     "if (c < 0 || (s == r && c != 0)) st |= REF_ST_COST;"),
]


def _battery():
    """Run the pin checks once; exit 1 on the first failure, 0 if all pass."""
    sys.path.insert(0, HERE)
    sys.path.insert(0, ROOT)
    import oracle
    oracle.load_library(sys.argv[1])
    import test_oracle_paper as tp
    import test_oracle_pins as pins
    import test_oracle_edges as edges
    checks = [lambda: tp.test_worked_example(0), lambda: tp.test_worked_example(2),
              tp.test_placement_cost_example,
              edges.test_self_row_mismatch_is_informational]
    for s in pins.SEEDS[:30]:
        checks += [lambda s=s: pins.test_histogram_and_demand(s),
                   lambda s=s: pins.test_stage1_placement(s, False),
                   lambda s=s: pins.test_stage1_placement(s, True),
                   lambda s=s: pins.test_routing_construction(s),
                   lambda s=s: pins.test_refinement_steps(s, False),
                   lambda s=s: pins.test_refinement_steps(s, True),
                   lambda s=s: pins.test_rerouting_and_cross_rank(s)]
    checks += [pins.test_invalid_cost_model_makes_no_plan]
    for s in range(20):
        checks += [lambda s=s: pins.test_one_gpu_per_node_reaches_the_optimum(s)]
    for c in checks:
        try:
            c()
        except Exception:
            sys.exit(1)
    sys.exit(0)


def _build(tmp_path, text, name):
    src = tmp_path / (name + ".c")
    src.write_text(text)
    lib = tmp_path / (name + ".so")
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-I",
                           os.path.join(ROOT, "oracle"), "-o", str(lib), str(src)])
    return str(lib)


def _run_battery(lib):
    try:
        return subprocess.run([sys.executable, __file__, lib], timeout=120,
                              capture_output=True).returncode
    except subprocess.TimeoutExpired:
        return "timeout"


def test_unmutated_oracle_passes_the_battery(tmp_path):
    with open(SRC) as f:
        text = f.read()
    assert _run_battery(_build(tmp_path, text, "orig")) == 0


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) == 1, "mutation site not found: " + name
    rc = _run_battery(_build(tmp_path, text.replace(old, new), "mutant"))
    assert rc != 0, "pins did not catch: " + name


if __name__ == "__main__":
    _battery()
