/*
 * TopoEP planner, CPU oracle (test infrastructure; see topoep_oracle.h).
 *
 * Follows the paper's Section 4 step by step, in its notation:
 *   O0  histogram of local_topk -> row self of Omega   (Section 3.1, Eq. 3)
 *   O1  domain demand D                                 (Section 4.1, Eq. 4)
 *   O2  inter-node placement with b = 2 D S - W_e       (Section 4.3, Eq. 9)
 *   O3  routing construction q, U, L                    (Section 4.3)
 *   O4  intra-node refinement, delta of Eq. 10          (Section 4.3)
 *   O5  send counts and per-assignment destinations     (Section 4.2, q)
 *
 * The cost c(s, r) is the two-level one of the topology (0, cost_intra,
 * cost_inter) or, in topoep_plan_ref_general, any symmetric nonnegative
 * matrix with a zero diagonal (the full model of Section 4.1), and ||W_e||
 * one size for every expert or one per expert.
 *
 * Where the paper leaves a choice open, the readings below are used; each is
 * repeated at the step it concerns.
 *   - main(e) = e / (E/R) (main instances evenly and contiguously spread);
 *     dom(r) = r / G.
 *   - The plan uses the histogram of local_topk as row self of Omega.
 *   - Stage 1: only b > 0 (strict) for experts whose main is outside the
 *     domain; candidates in (b descending, e ascending) order; each goes to
 *     the domain rank with the fewest used replica slots among those with a
 *     free slot, ties to the lowest rank; at most one replica per (domain,
 *     expert); candidates beyond the domain's free slots are dropped.
 *   - Routing: the selected instances are those of e in dom(s) (the main one
 *     included), else all instances of e; w is split as floor(w/n), the first
 *     (w mod n) instances in ascending rank order taking one more.
 *   - Refinement: busiest rank of the domain with ties to the lowest rank;
 *     experts "contributing to its load" are those with U[e][rb] > 0;
 *     candidates ranked by (delta desc, L[rt] asc, cost change asc, e asc,
 *     rt asc); the moved assignments are taken from sources in ascending
 *     (c(s,rt) - c(s,rb), s) order, which minimises the token-cost change
 *     for that delta; the cost change is the change of Eq. 6 plus Eq. 7; the
 *     loop stops when the busiest rank has no candidate with delta >= 1;
 *     replicas whose load falls to zero keep their slot.
 *   - Slot j of rank r holds the j-th replica created on r (stage 1 first,
 *     then refinement in commit order).
 *   - Rerouting: the rho-th occurrence (0-based, row-major order) of expert e
 *     in local_topk goes to the instance r_i whose range
 *     [p_i, p_i + q[self][e][r_i]) contains rho, instances in ascending rank.
 */
#include "topoep_oracle.h"

#include <stdlib.h>
#include <string.h>

typedef struct {
  int R, G, M, E, P, N, self;
  int64_t cI, cX, S, W;
  const int32_t *C;    /* general cost matrix [R][R], or NULL (two-level) */
  const int64_t *We;   /* ||W_e|| per expert, or NULL (W for every expert) */
} model;

/* Communication cost per byte c(s, r) (Section 4.1): the given symmetric
 * matrix, or the two-level model (0 on the diagonal, cI inside a domain, cX
 * across). */
static int64_t cost(const model *m, int s, int r) {
  if (m->C) return m->C[(size_t)s * m->R + r];
  if (s == r) return 0;
  return (s / m->G == r / m->G) ? m->cI : m->cX;
}

/* Parameter size of expert e, ||W_e||. */
static int64_t wexp(const model *m, int e) { return m->We ? m->We[e] : m->W; }

static int dom(const model *m, int r) { return r / m->G; }
static int main_rank(const model *m, int e) { return e / m->P; }

/* Lexicographic candidate key of the refinement (smaller is better). */
typedef struct {
  int64_t neg_delta, load_t, dcost, e, rt;
} cand_key;

static int key_less(const cand_key *a, const cand_key *b) {
  if (a->neg_delta != b->neg_delta) return a->neg_delta < b->neg_delta;
  if (a->load_t != b->load_t) return a->load_t < b->load_t;
  if (a->dcost != b->dcost) return a->dcost < b->dcost;
  if (a->e != b->e) return a->e < b->e;
  return a->rt < b->rt;
}

/* Stage-1 candidate (expert, benefit). */
typedef struct {
  int e;
  int64_t b;
} stage1_cand;

static int stage1_cmp(const void *pa, const void *pb) {
  const stage1_cand *a = (const stage1_cand *)pa, *b = (const stage1_cand *)pb;
  if (a->b != b->b) return a->b > b->b ? -1 : 1; /* b descending */
  return a->e < b->e ? -1 : (a->e > b->e);       /* then e ascending */
}

/* Sources ordered for a move from rb to rt. */
typedef struct {
  int64_t diff;
  int s;
} src_order;

static int src_cmp(const void *pa, const void *pb) {
  const src_order *a = (const src_order *)pa, *b = (const src_order *)pb;
  if (a->diff != b->diff) return a->diff < b->diff ? -1 : 1;
  return a->s < b->s ? -1 : (a->s > b->s);
}

int topoep_plan_ref(const ref_topology *topo, const int32_t *global_load,
                    const int32_t *local_topk, int32_t T, int32_t k,
                    int32_t replica_budget, int32_t *replica_slots,
                    int32_t *token_dest, int32_t *send_counts,
                    int32_t *status, ref_debug *dbg) {
  return topoep_plan_ref_ex(topo, global_load, local_topk, T, k, replica_budget, replica_slots,
                            token_dest, send_counts, NULL, status, dbg);
}

int topoep_plan_ref_ex(const ref_topology *topo, const int32_t *global_load,
                       const int32_t *local_topk, int32_t T, int32_t k,
                       int32_t replica_budget, int32_t *replica_slots,
                       int32_t *token_dest, int32_t *send_counts,
                       int32_t *recv_counts, int32_t *status, ref_debug *dbg) {
  return topoep_plan_ref_general(topo, NULL, NULL, global_load, local_topk, T, k, replica_budget,
                                 replica_slots, token_dest, send_counts, recv_counts, status, dbg);
}

int topoep_plan_ref_general(const ref_topology *topo, const int32_t *cost_matrix,
                            const int64_t *expert_bytes, const int32_t *global_load,
                            const int32_t *local_topk, int32_t T, int32_t k,
                            int32_t replica_budget, int32_t *replica_slots,
                            int32_t *token_dest, int32_t *send_counts,
                            int32_t *recv_counts, int32_t *status, ref_debug *dbg) {
  return topoep_plan_ref_capped(topo, cost_matrix, expert_bytes, global_load, local_topk, T, k,
                                replica_budget, replica_slots, token_dest, send_counts, recv_counts,
                                status, dbg, REF_ITER_LIMIT);
}

int topoep_plan_ref_capped(const ref_topology *topo, const int32_t *cost_matrix,
                           const int64_t *expert_bytes, const int32_t *global_load,
                           const int32_t *local_topk, int32_t T, int32_t k,
                           int32_t replica_budget, int32_t *replica_slots,
                           int32_t *token_dest, int32_t *send_counts,
                           int32_t *recv_counts, int32_t *status, ref_debug *dbg,
                           int32_t iter_limit) {
  if (!topo || !global_load || !replica_slots || !send_counts || !status) return REF_EINVAL;
  if (iter_limit < 0) return REF_EINVAL;
  if (T < 0 || k < 1 || replica_budget < 0) return REF_EINVAL;
  if (T > 0 && (!local_topk || !token_dest)) return REF_EINVAL;
  model m;
  m.R = topo->num_ranks;
  m.G = topo->ranks_per_node;
  m.E = topo->num_experts;
  m.self = topo->self_rank;
  if (m.R <= 0 || m.G <= 0 || m.E <= 0 || m.R % m.G != 0 || m.E % m.R != 0) return REF_EINVAL;
  if (k > m.E || m.self < 0 || m.self >= m.R) return REF_EINVAL;
  if (topo->cost_intra < 0 || topo->cost_inter < 0 || topo->tok_bytes <= 0 || topo->expert_bytes < 0)
    return REF_EINVAL;
  if ((int64_t)T * k > INT32_MAX) return REF_EINVAL;
  m.M = m.R / m.G;
  m.P = m.E / m.R;
  m.N = replica_budget;
  m.cI = topo->cost_intra;
  m.cX = topo->cost_inter;
  m.S = topo->tok_bytes;
  m.W = topo->expert_bytes;
  m.C = cost_matrix;
  m.We = expert_bytes;
  const int R = m.R, G = m.G, M = m.M, E = m.E, N = m.N;
  const int64_t n_assign = (int64_t)T * k;

  int32_t *hist = calloc((size_t)E, sizeof(int32_t));
  int32_t *omega = malloc((size_t)R * E * sizeof(int32_t));
  int64_t *D = calloc((size_t)M * E, sizeof(int64_t));
  uint8_t *x = calloc((size_t)E * R, 1);
  int32_t *used = calloc((size_t)R, sizeof(int32_t));
  int32_t *slots = malloc((size_t)R * (N > 0 ? N : 1) * sizeof(int32_t));
  int32_t *q = calloc((size_t)R * E * R, sizeof(int32_t));
  int32_t *U = calloc((size_t)E * R, sizeof(int32_t));
  int32_t *L = calloc((size_t)R, sizeof(int32_t));
  int32_t *mv = calloc((size_t)R, sizeof(int32_t));
  int32_t *best_mv = calloc((size_t)R, sizeof(int32_t));
  src_order *order = malloc((size_t)R * sizeof(src_order));
  stage1_cand *cand = malloc((size_t)E * sizeof(stage1_cand));
  int32_t *inst = malloc((size_t)R * sizeof(int32_t));
  int64_t *seen = calloc((size_t)E, sizeof(int64_t));
  if (!hist || !omega || !D || !x || !used || !slots || !q || !U || !L || !mv || !best_mv || !order ||
      !cand || !inst || !seen) {
    free(hist); free(omega); free(D); free(x); free(used); free(slots); free(q); free(U); free(L);
    free(mv); free(best_mv); free(order); free(cand); free(inst); free(seen);
    return REF_ENOMEM;
  }
#define Q(s, e, r) q[((size_t)(s) * E + (e)) * R + (r)]
#define X(e, r) x[(size_t)(e) * R + (r)]
#define UU(e, r) U[(size_t)(e) * R + (r)]

  uint32_t st = 0;

  /* O0: histogram of the local top-k ids; it replaces row self of Omega
   * (the row the EP all-gather of Section 3.1 would carry for this rank). */
  for (int64_t i = 0; i < n_assign; ++i) {
    int e = local_topk[i];
    if (e < 0 || e >= E) st |= REF_ST_BAD_ID;
    else hist[e]++;
  }
  memcpy(omega, global_load, (size_t)R * E * sizeof(int32_t));
  for (int e = 0; e < E; ++e) {
    if (global_load[(size_t)m.self * E + e] != hist[e]) st |= REF_ST_SELF_DIFF;
    omega[(size_t)m.self * E + e] = hist[e];
  }
  for (size_t i = 0; i < (size_t)R * E; ++i)
    if (global_load[i] < 0) st |= REF_ST_NEG_LOAD;

  /* A general cost matrix must be a cost: symmetric, nonnegative, zero on
   * the diagonal (Section 4.1); expert sizes nonnegative. */
  int64_t cmax = m.cI > m.cX ? m.cI : m.cX, wmax = m.W;
  if (m.C) {
    cmax = 0;
    for (int s = 0; s < R; ++s)
      for (int r = 0; r < R; ++r) {
        int32_t c = m.C[(size_t)s * R + r];
        if (c < 0 || c != m.C[(size_t)r * R + s] || (s == r && c != 0)) st |= REF_ST_COST;
        if (c > cmax) cmax = c;
      }
  }
  if (m.We) {
    wmax = 0;
    for (int e = 0; e < E; ++e) {
      if (m.We[e] < 0) st |= REF_ST_COST;
      if (m.We[e] > wmax) wmax = m.We[e];
    }
  }

  /* Exact-arithmetic range: counts are int32 and cost terms int64.  The
   * total load must fit int32 and 4 S total max(c,1) + max(c,1) max(W) <
   * 2^62 bounds every benefit b and every cost change of a move. */
  {
    int64_t total = 0;
    for (size_t i = 0; i < (size_t)R * E; ++i)
      if (omega[i] > 0) total += omega[i];
    int64_t cm = cmax;
    if (cm < 1) cm = 1;
    unsigned __int128 bound = (unsigned __int128)4 * (unsigned __int128)m.S *
                                  (unsigned __int128)total * (unsigned __int128)cm +
                              (unsigned __int128)cm * (unsigned __int128)(wmax > 0 ? wmax : 0);
    if (total > INT32_MAX || bound >= ((unsigned __int128)1 << 62)) st |= REF_ST_RANGE;
  }

  if (st & (REF_ST_BAD_ID | REF_ST_NEG_LOAD | REF_ST_RANGE | REF_ST_COST)) {
    for (int i = 0; i < R * N; ++i) replica_slots[i] = -1;
    for (int r = 0; r < R; ++r) send_counts[r] = 0;
    if (recv_counts)
      for (int r = 0; r < R; ++r) recv_counts[r] = 0;
    for (int64_t i = 0; i < n_assign; ++i) token_dest[i] = -1;
    status[0] = (int32_t)st;
    status[1] = 0;
    if (dbg) {
      dbg->n_moves = 0;
      if (dbg->hist) memcpy(dbg->hist, hist, (size_t)E * sizeof(int32_t));
    }
    free(hist); free(omega); free(D); free(x); free(used); free(slots); free(q); free(U); free(L);
    free(mv); free(best_mv); free(order); free(cand); free(inst); free(seen);
    return REF_OK;
  }

  /* O1: demand of domain d for expert e, D[d][e] = sum of omega[s][e] over
   * the sources s of domain d (Eq. 4). */
  for (int s = 0; s < R; ++s)
    for (int e = 0; e < E; ++e) D[(size_t)dom(&m, s) * E + e] += omega[(size_t)s * E + e];

  /* O2: fixed main instances (C5), empty replica slots. */
  for (int e = 0; e < E; ++e) X(e, main_rank(&m, e)) = 1;
  for (int i = 0; i < R * (N > 0 ? N : 1); ++i) slots[i] = -1;

  /* Inter-node placement (Eq. 9).  Each domain independently: candidates are
   * experts whose main instance lies outside the domain with b > 0, taken in
   * (b descending, e ascending) order; each is placed on the domain rank with
   * the fewest used replica slots among those with a free slot (ties to the
   * lowest rank). */
  for (int d = 0; d < M; ++d) {
    int nc = 0;
    for (int e = 0; e < E; ++e) {
      if (dom(&m, main_rank(&m, e)) == d) continue;
      int64_t b = 2 * D[(size_t)d * E + e] * m.S - wexp(&m, e);
      if (b > 0) {
        cand[nc].e = e;
        cand[nc].b = b;
        nc++;
      }
    }
    qsort(cand, (size_t)nc, sizeof(stage1_cand), stage1_cmp);
    for (int i = 0; i < nc; ++i) {
      int best = -1;
      for (int r = d * G; r < (d + 1) * G; ++r) {
        if (used[r] >= N) continue;
        if (best < 0 || used[r] < used[best]) best = r;
      }
      if (best < 0) break; /* no free slot left in this domain */
      int e = cand[i].e;
      slots[(size_t)best * N + used[best]] = e;
      used[best]++;
      X(e, best) = 1;
    }
  }
  if (dbg && dbg->x_stage1) memcpy(dbg->x_stage1, x, (size_t)E * R);
  if (dbg && dbg->demand)
    for (int i = 0; i < M * E; ++i) dbg->demand[i] = (int32_t)D[i];
  if (dbg && dbg->hist) memcpy(dbg->hist, hist, (size_t)E * sizeof(int32_t));

  /* O3: routing construction.  For every (s, e) with w > 0: the instances of
   * e inside dom(s) if any, otherwise every instance of e, ascending rank;
   * w is split as evenly as integers allow, lower ranks taking the
   * remainder. */
  for (int s = 0; s < R; ++s) {
    for (int e = 0; e < E; ++e) {
      int32_t w = omega[(size_t)s * E + e];
      if (w <= 0) continue;
      int n = 0;
      for (int r = 0; r < R; ++r)
        if (X(e, r) && dom(&m, r) == dom(&m, s)) inst[n++] = r;
      if (n == 0)
        for (int r = 0; r < R; ++r)
          if (X(e, r)) inst[n++] = r;
      for (int i = 0; i < n; ++i) Q(s, e, inst[i]) = w / n + (i < w % n ? 1 : 0);
    }
  }
  /* Per-instance loads U[e][r] and rank loads L[r] (load metric of Section 4.2). */
  for (int s = 0; s < R; ++s)
    for (int e = 0; e < E; ++e)
      for (int r = 0; r < R; ++r) UU(e, r) += Q(s, e, r);
  for (int e = 0; e < E; ++e)
    for (int r = 0; r < R; ++r) L[r] += UU(e, r);
  if (dbg && dbg->q_routed) memcpy(dbg->q_routed, q, (size_t)R * E * R * sizeof(int32_t));
  if (dbg && dbg->load_routed) memcpy(dbg->load_routed, L, (size_t)R * sizeof(int32_t));

  /* O4: intra-node refinement, every domain independently. */
  int32_t n_moves = 0;
  for (int d = 0; d < M; ++d) {
    int32_t iters = 0;
    for (;;) {
      /* busiest rank of the domain, ties to the lowest rank */
      int rb = d * G;
      for (int r = d * G + 1; r < (d + 1) * G; ++r)
        if (L[r] > L[rb]) rb = r;
      int have = 0;
      cand_key best = {0, 0, 0, 0, 0};
      int best_e = -1, best_rt = -1, best_created = 0;
      int32_t best_delta = 0;
      for (int e = 0; e < E; ++e) {
        if (UU(e, rb) <= 0) continue;
        for (int rt = d * G; rt < (d + 1) * G; ++rt) {
          if (rt == rb) continue;
          int hosts = X(e, rt);
          if (!hosts && used[rt] >= N) continue; /* needs a free slot */
          int64_t gap = (int64_t)L[rb] - L[rt];
          if (gap < 2) continue;                  /* floor(gap/2) < 1 */
          int64_t delta = gap / 2;
          if (UU(e, rb) < delta) delta = UU(e, rb);
          /* sources in ascending (c(s,rt) - c(s,rb), s) order */
          for (int s = 0; s < R; ++s) {
            order[s].diff = cost(&m, s, rt) - cost(&m, s, rb);
            order[s].s = s;
          }
          qsort(order, (size_t)R, sizeof(src_order), src_cmp);
          int64_t remaining = delta, dtok = 0;
          for (int i = 0; i < R; ++i) {
            int s = order[i].s;
            int64_t take = Q(s, e, rb);
            if (take > remaining) take = remaining;
            mv[s] = (int32_t)take;
            remaining -= take;
            dtok += take * order[i].diff;
          }
          int64_t dcost = 2 * m.S * dtok + (hosts ? 0 : cost(&m, main_rank(&m, e), rt) * wexp(&m, e));
          cand_key key = {-delta, L[rt], dcost, e, rt};
          if (!have || key_less(&key, &best)) {
            have = 1;
            best = key;
            best_e = e;
            best_rt = rt;
            best_delta = (int32_t)delta;
            best_created = !hosts;
            memcpy(best_mv, mv, (size_t)R * sizeof(int32_t));
          }
        }
      }
      if (!have) break;
      /* The paper's loop has no bound: it ends because sum_r L_r^2 falls by
       * at least 2 with every move, which still allows up to total^2 / 2
       * moves.  A domain that has committed iter_limit moves and still has
       * one stops here with ITER (the plan stays valid), so every plan's work
       * is bounded; the GPU path applies the same rule. */
      if (iters >= iter_limit) {
        st |= REF_ST_ITER;
        break;
      }
      /* commit the selected move */
      int e = best_e, rt = best_rt;
      if (!X(e, rt)) {
        X(e, rt) = 1;
        slots[(size_t)rt * N + used[rt]] = e;
        used[rt]++;
      }
      for (int s = 0; s < R; ++s) {
        Q(s, e, rb) -= best_mv[s];
        Q(s, e, rt) += best_mv[s];
      }
      UU(e, rb) -= best_delta;
      UU(e, rt) += best_delta;
      L[rb] -= best_delta;
      L[rt] += best_delta;
      if (dbg && n_moves < dbg->move_cap) {
        if (dbg->moves) {
          int32_t *mm = dbg->moves + (size_t)n_moves * 6;
          mm[0] = d; mm[1] = rb; mm[2] = rt; mm[3] = e; mm[4] = best_delta; mm[5] = best_created;
        }
        if (dbg->move_dcost) dbg->move_dcost[n_moves] = best.dcost;
        if (dbg->move_m) memcpy(dbg->move_m + (size_t)n_moves * R, best_mv, (size_t)R * sizeof(int32_t));
      }
      n_moves++;
      iters++;
    }
    if (dbg && dbg->iters) dbg->iters[d] = iters;
  }
  if (dbg) {
    dbg->n_moves = n_moves;
    if (dbg->x_final) memcpy(dbg->x_final, x, (size_t)E * R);
    if (dbg->q_final) memcpy(dbg->q_final, q, (size_t)R * E * R * sizeof(int32_t));
    if (dbg->load_final) memcpy(dbg->load_final, L, (size_t)R * sizeof(int32_t));
  }

  /* O5: outputs.  replica_slots; send_counts[r] = sum_e q[self][e][r]; the
   * rho-th occurrence of e in local_topk (row-major) goes to the instance
   * whose prefix range over ascending ranks contains rho. */
  for (int i = 0; i < R * N; ++i) replica_slots[i] = slots[i];
  for (int r = 0; r < R; ++r) {
    int64_t sc = 0;
    for (int e = 0; e < E; ++e) sc += Q(m.self, e, r);
    send_counts[r] = (int32_t)sc;
  }
  /* Receive counts: every rank makes the same plan, so what source s sends
   * to this rank is its share q[s][e][self] summed over the experts (the
   * count the dispatch of Section 4.3 needs on the receiving side). */
  if (recv_counts)
    for (int s2 = 0; s2 < R; ++s2) {
      int64_t rc = 0;
      for (int e = 0; e < E; ++e) rc += Q(s2, e, m.self);
      recv_counts[s2] = (int32_t)rc;
    }
  for (int64_t i = 0; i < n_assign; ++i) {
    int e = local_topk[i];
    int64_t rho = seen[e]++;
    int64_t prefix = 0;
    int dest = -1;
    for (int r = 0; r < R; ++r) {
      int32_t c = Q(m.self, e, r);
      if (c <= 0) continue;
      if (rho < prefix + c) {
        dest = r;
        break;
      }
      prefix += c;
    }
    token_dest[i] = dest;
  }
  status[0] = (int32_t)st;
  status[1] = n_moves;
#undef Q
#undef X
#undef UU
  free(hist); free(omega); free(D); free(x); free(used); free(slots); free(q); free(U); free(L);
  free(mv); free(best_mv); free(order); free(cand); free(inst); free(seen);
  return REF_OK;
}

/* Dispatch layout: the send buffer holds the assignments grouped by
 * destination rank, ranks ascending, and inside one destination in
 * row-major (token, k) order.  send_offsets[r] = sum of send_counts[r'] for
 * r' < r (R + 1 entries); token_slot[i] = send_offsets[dest] + the number of
 * earlier assignments with the same destination, -1 when token_dest[i] is
 * not a rank. */
int topoep_layout_ref(int32_t R, const int32_t *token_dest, int64_t n, const int32_t *send_counts,
                      int32_t *send_offsets, int32_t *token_slot) {
  if (R <= 0 || n < 0 || !send_counts || !send_offsets || (n > 0 && (!token_dest || !token_slot)))
    return REF_EINVAL;
  int64_t acc = 0;
  for (int r = 0; r < R; ++r) {
    send_offsets[r] = (int32_t)acc;
    acc += send_counts[r];
  }
  send_offsets[R] = (int32_t)acc;
  int64_t *seen = calloc((size_t)R, sizeof(int64_t));
  if (!seen) return REF_ENOMEM;
  for (int64_t i = 0; i < n; ++i) {
    const int d = token_dest[i];
    if (d < 0 || d >= R) {
      token_slot[i] = -1;
      continue;
    }
    token_slot[i] = (int32_t)(send_offsets[d] + seen[d]);
    seen[d]++;
  }
  free(seen);
  return REF_OK;
}
