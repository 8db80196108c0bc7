/*
 * TopoEP planner, CPU oracle (test infrastructure).
 *
 * A plain, slow, single-threaded C implementation of the per-layer,
 * per-microbatch plan of "TopoEP: Topology-Aware Load Balancing for
 * Expert-Parallel MoE Training", Section 4: routing matrix and domain demand
 * (Section 4.1, Eqs. 3-4), inter-node placement (Section 4.3, Eq. 9), routing
 * construction (Section 4.3), intra-node refinement (Section 4.3, Eq. 10) and
 * the per-assignment rerouting that turns the per-instance counts q into a
 * destination for every (token, k) assignment.
 *
 * It exists only to check the GPU path.  It shares no code, header, table or
 * helper with the GPU library; only the tests, the smoke check and the CPU
 * baseline of the benchmark may load it.  Dense arrays (x[E][R],
 * q[R][E][R]) are used on purpose so that every step reads like the paper.
 */
#ifndef TOPOEP_ORACLE_H
#define TOPOEP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Two-level instance of the paper's system model (Section 4.1): R ranks in
 * M = R / G domains of G consecutive ranks; E experts with main(e) = e / (E/R);
 * c(s,r) = 0 if s == r, cost_intra inside a domain, cost_inter across. */
typedef struct {
  int32_t num_ranks;
  int32_t ranks_per_node;
  int32_t num_experts;
  int32_t self_rank;
  int32_t cost_intra;
  int32_t cost_inter;
  int64_t tok_bytes;     /* S_tok */
  int64_t expert_bytes;  /* ||W_e||, equal for every expert */
} ref_topology;

/* Optional intermediate state; every pointer may be NULL. */
typedef struct {
  int32_t *hist;         /* [E]      histogram of local_topk                   */
  int32_t *demand;       /* [M*E]    D[d][e]                                    */
  uint8_t *x_stage1;     /* [E*R]    placement after inter-node placement       */
  int32_t *q_routed;     /* [R*E*R]  q[s][e][r] after routing construction      */
  int32_t *load_routed;  /* [R]      L after routing construction               */
  uint8_t *x_final;      /* [E*R]    placement after refinement                 */
  int32_t *q_final;      /* [R*E*R]  q after refinement                         */
  int32_t *load_final;   /* [R]                                                 */
  int32_t *iters;        /* [M]      committed refinement moves per domain      */
  int32_t move_cap;      /* capacity of the move log                            */
  int32_t *moves;        /* [move_cap*6] d, rb, rt, e, delta, created           */
  int64_t *move_dcost;   /* [move_cap]   cost change of the move                */
  int32_t *move_m;       /* [move_cap*R] assignments moved per source           */
  int32_t n_moves;       /* out: moves committed (may exceed move_cap)          */
} ref_debug;

/* Return codes (same meaning as the GPU library's). */
#define REF_OK 0
#define REF_EINVAL (-1)
#define REF_ENOMEM (-5)

/* Status bits. */
#define REF_ST_BAD_ID 1u      /* an id in local_topk outside [0, E)               */
#define REF_ST_NEG_LOAD 2u    /* a negative entry in global_load                  */
#define REF_ST_SELF_DIFF 4u   /* global_load[self] differs from the histogram     */
#define REF_ST_RANGE 8u       /* loads or costs exceed the exact integer range    */
#define REF_ST_ITER 32u       /* a domain still had a refinement move after       */
                              /* iter_limit of them (the plan stays valid)         */
#define REF_ST_COST 64u       /* a general cost matrix is not symmetric, has a    */
                              /* nonzero diagonal or a negative entry, or an      */
                              /* expert size is negative                          */

/*
 * All pointers are host pointers, row-major.  Outputs: replica_slots[R*N]
 * (slot j of rank r = the j-th replica created on r, -1 if empty),
 * token_dest[T*k], send_counts[R], status[2]: status[0] = REF_ST_* bits,
 * status[1] = refinement moves committed, summed over domains (each
 * iteration of the Eq. 10 loop commits one).  When status[0] has BAD_ID,
 * NEG_LOAD or RANGE set, no plan is made: replica_slots = -1,
 * send_counts = 0, token_dest = -1, status[1] = 0.
 */
int topoep_plan_ref(const ref_topology *topo, const int32_t *global_load,
                    const int32_t *local_topk, int32_t T, int32_t k,
                    int32_t replica_budget, int32_t *replica_slots,
                    int32_t *token_dest, int32_t *send_counts,
                    int32_t *status, ref_debug *dbg);

/* The same plan plus recv_counts[R] (may be NULL): recv_counts[s] = sum over
 * e of q[s][e][self], what rank s sends to this rank under the replicated
 * plan (0 when no plan is made). */
int topoep_plan_ref_ex(const ref_topology *topo, const int32_t *global_load,
                       const int32_t *local_topk, int32_t T, int32_t k,
                       int32_t replica_budget, int32_t *replica_slots,
                       int32_t *token_dest, int32_t *send_counts,
                       int32_t *recv_counts, int32_t *status, ref_debug *dbg);

/* The full model of Section 4.1: cost_matrix [R*R] (c(s,r), row-major) or
 * NULL for the topology's two-level cost; expert_bytes [E] (||W_e||) or
 * NULL for topo->expert_bytes for every expert.  An invalid matrix or a
 * negative size sets REF_ST_COST and no plan is made. */
int topoep_plan_ref_general(const ref_topology *topo, const int32_t *cost_matrix,
                            const int64_t *expert_bytes, const int32_t *global_load,
                            const int32_t *local_topk, int32_t T, int32_t k,
                            int32_t replica_budget, int32_t *replica_slots,
                            int32_t *token_dest, int32_t *send_counts,
                            int32_t *recv_counts, int32_t *status, ref_debug *dbg);

/* Committed refinement moves per domain after which a domain that still
 * has a move stops with REF_ST_ITER (the entry points above use it). */
#define REF_ITER_LIMIT (1 << 22)

/* topoep_plan_ref_general with an explicit bound iter_limit >= 0 on the
 * refinement moves of each domain. */
int topoep_plan_ref_capped(const ref_topology *topo, const int32_t *cost_matrix,
                           const int64_t *expert_bytes, const int32_t *global_load,
                           const int32_t *local_topk, int32_t T, int32_t k,
                           int32_t replica_budget, int32_t *replica_slots,
                           int32_t *token_dest, int32_t *send_counts,
                           int32_t *recv_counts, int32_t *status, ref_debug *dbg,
                           int32_t iter_limit);

/* Dispatch layout of the rerouted assignments: send_offsets[R + 1] is the
 * exclusive prefix of send_counts; token_slot[n] = send_offsets[dest] + the
 * number of earlier assignments (row-major) with the same destination, or
 * -1 when token_dest is not a rank. */
int topoep_layout_ref(int32_t R, const int32_t *token_dest, int64_t n, const int32_t *send_counts,
                      int32_t *send_offsets, int32_t *token_slot);

#ifdef __cplusplus
}
#endif

#endif
