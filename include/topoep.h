/*
 * topoep.h -- C ABI of the TopoEP per-layer planner on one MI355X (gfx950).
 *
 * The planner turns one EP rank's routing result into a topology-aware plan
 * (TopoEP, Sections 3.1 and 4):
 *   1. the per-expert histogram of the rank's top-k ids, which is this
 *      rank's row of the routing matrix Omega (Eq. 3);
 *   2. the domain demand D (Eq. 4) and inter-node replica placement driven by
 *      the benefit b = 2 D S_tok - ||W_e|| (Section 4.3, Eq. 9);
 *   3. routing construction q, U, L (Section 4.3) and intra-node refinement
 *      with the transfer amount of Eq. 10;
 *   4. rerouting of every (token, k) assignment to an expert instance, and
 *      per-destination send counts (the q[self][e][r] of Section 4.2 expanded
 *      to assignments).
 *
 * Conventions shared by every entry point:
 *   - All counts are int32; all arrays are row-major and densely packed.
 *   - "device" pointers are HIP device memory of the current device; the
 *     caller owns every buffer (inputs, outputs, workspace).  The library
 *     keeps no state between calls and never allocates or frees device
 *     memory during a call.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is only enqueued: a call returns before the GPU finishes, with no
 *     host-device synchronisation and no device-to-host copy, so an enqueue
 *     may be captured in a HIP graph.  Outputs are valid once the stream
 *     reaches them.
 *   - One workspace serves one plan at a time: plans that share a workspace
 *     must be ordered on one stream.  A workspace serves one problem shape:
 *     the topology, T, k, N_slot and the launch shape (its layout and its
 *     hand-over words depend on all of them).  It is zero-filled before the
 *     first plan of a shape (e.g. hipMemset after allocation, or again
 *     before another shape reuses the memory); after that no clearing is
 *     needed between plans, including after a plan that reported
 *     TOPOEP_ST_SYNC: the words that order the kernels' hand-overs carry a
 *     plan generation the kernels advance themselves, so nothing a plan
 *     leaves behind can satisfy a later plan's wait.
 *   - main(e) = e / (E/R) (main instances spread contiguously and evenly,
 *     Section 3.2); dom(r) = r / G.  Cost c(s,r) = 0 if s == r, cost_intra
 *     inside a domain, cost_inter across domains (a two-level instance of
 *     the symmetric cost matrix C of Section 4.1).
 */
#ifndef TOPOEP_H
#define TOPOEP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* System model of Section 4.1, passed by host pointer and copied into the
 * kernel arguments. */
typedef struct topoep_topology {
  int32_t num_ranks;      /* R > 0                                              */
  int32_t ranks_per_node; /* G > 0, G divides R (G <= 64)                       */
  int32_t num_experts;    /* E > 0, R divides E                                 */
  int32_t self_rank;      /* rank whose local_topk is passed, 0 <= self < R     */
  int32_t cost_intra;     /* c(s,r) for s != r in one domain, >= 0              */
  int32_t cost_inter;     /* c(s,r) across domains, >= 0                        */
  int64_t tok_bytes;      /* S_tok, bytes of one routed activation, > 0         */
  int64_t expert_bytes;   /* ||W_e||, bytes of one expert (all equal), >= 0     */
} topoep_topology;

/* Optional launch shape.  Every valid shape gives bitwise-identical results;
 * it only changes speed.  NULL selects the default. */
typedef struct topoep_launch {
  int32_t items_per_thread; /* 1, 2, 4 or 8 ids per thread per tile              */
  int32_t block_threads;    /* 64..1024, multiple of 64, for histogram/reroute    */
  int32_t tiles_per_block;  /* >= 1; 0 = choose from the problem size             */
  int32_t solve_threads;    /* 64..1024, multiple of 64, for the solver           */
  int32_t solver;           /* 0 = choose (3 when it fits, else 1, else 2);       */
                            /* 1 = three kernels (histogram, solver, reroute)    */
                            /*     with one solver workgroup for all domains     */
                            /*     (its whole state in LDS);                     */
                            /* 2 = three kernels, one solver workgroup per       */
                            /*     domain with a bounded grid barrier;           */
                            /* 3 = one kernel: the solver workgroup of 1 plus at */
                            /*     most 128 workgroups of solve_threads threads  */
                            /*     holding items_per_thread ids each, which      */
                            /*     count, wait (bounded) for the solver and      */
                            /*     reroute; block_threads and tiles_per_block    */
                            /*     are ignored                                   */
  int32_t spin_limit;       /* polls of each bounded in-kernel wait before it    */
                            /* gives up with TOPOEP_ST_SYNC; 0 = the default     */
                            /* (2^24), -1 = every such wait gives up at once     */
                            /* (for testing the error path; the kernels still    */
                            /* run to completion)                                */
  int32_t iter_limit;       /* refinement moves per domain after which a domain  */
                            /* that still has a move stops with TOPOEP_ST_ITER;  */
                            /* 0 = the default (2^22)                            */
} topoep_launch;

/* Launch shape a plan will use (topoep_plan_shape). */
typedef struct topoep_shape {
  int32_t kernels;          /* kernels one plan enqueues: 1 (solver 3) or 3     */
  int32_t solver;           /* 1, 2 or 3 as in topoep_launch.solver              */
  int32_t items_per_thread; /* ids per thread of the histogram/reroute work      */
  int32_t chunk_blocks;     /* workgroups holding ids                            */
  int32_t grid[3];          /* workgroups of each kernel, in launch order        */
  int32_t block[3];         /* threads per workgroup of each kernel              */
  int32_t lds_bytes[3];     /* dynamic LDS of each kernel                        */
} topoep_shape;

/* topoep_plan_stage: the plan's kernels with empty bodies (launch floor). */
#define TOPOEP_STAGE_FLOOR 3

/* Host return codes. */
#define TOPOEP_OK 0
#define TOPOEP_EINVAL (-1)     /* bad argument (see topoep_plan)                   */
#define TOPOEP_EWORKSPACE (-2) /* workspace smaller than required, or misaligned  */
#define TOPOEP_EHIP (-3)       /* a HIP launch failed (hipGetLastError)            */
#define TOPOEP_ELIMIT (-4)     /* per-domain solver state exceeds on-chip memory  */

/* Device status bits, written by the plan into *status. */
#define TOPOEP_ST_BAD_ID 1u      /* an id of local_topk is outside [0, E)            */
#define TOPOEP_ST_NEG_LOAD 2u    /* global_load holds a negative entry               */
#define TOPOEP_ST_SELF_DIFF 4u   /* global_load[self] differs from the histogram of  */
                                 /* local_topk (informational: the plan always uses  */
                                 /* the histogram as row self of Omega)              */
#define TOPOEP_ST_RANGE 8u       /* sum of loads > INT32_MAX, or                     */
                                 /* 4 S total max(c,1) + max(c,1) W >= 2^62, so the  */
                                 /* integer cost terms would not be exact            */
#define TOPOEP_ST_SYNC 16u       /* a bounded in-kernel wait gave up (outputs wrong) */
#define TOPOEP_ST_ITER 32u       /* a domain still had a refinement move after its   */
                                 /* iteration bound (the plan is valid, less        */
                                 /* refined; the CPU oracle applies the same bound)  */
#define TOPOEP_ST_COST 64u       /* (topoep_plan_costs) the cost matrix is not        */
                                 /* symmetric, nonnegative and zero on its diagonal, */
                                 /* or an expert size is negative                    */
/* With BAD_ID, NEG_LOAD, RANGE or COST no plan is made: replica_slots = -1,
 * send_counts = 0, token_dest = -1, status[1] = 0. */

/*
 * Bytes of device workspace topoep_plan needs for these sizes (default
 * launch shape).  Returns TOPOEP_OK, TOPOEP_EINVAL for invalid sizes, or
 * TOPOEP_ELIMIT when one domain's solver state cannot fit in LDS.
 */
int topoep_workspace_bytes(const topoep_topology *topo, int32_t T, int32_t k,
                           int32_t replica_budget, size_t *bytes_out);

/* Same for an explicit launch shape (NULL = default). */
int topoep_workspace_bytes_ex(const topoep_topology *topo, int32_t T, int32_t k,
                              int32_t replica_budget, const topoep_launch *launch,
                              size_t *bytes_out);

/* The launch shape topoep_plan_ex would use for these sizes (host only;
 * same return codes as topoep_workspace_bytes_ex). */
int topoep_plan_shape(const topoep_topology *topo, int32_t T, int32_t k, int32_t replica_budget,
                      const topoep_launch *launch, topoep_shape *out);

/*
 * Enqueue one plan (Sections 3.1 and 4.3).
 *
 *   global_load    device int32 [R, E]: Omega as the EP all-gather delivers
 *                  it (row s = assignments of rank s per expert).  Row
 *                  self_rank is replaced by the histogram of local_topk.
 *   local_topk     device int32 [T, k]: this rank's top-k expert ids.  May be
 *                  NULL when T == 0.  Duplicate ids in one token count
 *                  independently.
 *   replica_budget N_slot >= 0 replica slots per rank (Section 4.1).  Budgets
 *                  above E - E/R are legal; the extra slots stay empty.
 *   replica_slots  device int32 out [R, N_slot]: slot j of rank r holds the
 *                  expert of the j-th replica created on r (inter-node
 *                  placement first, then refinement in commit order), -1 if
 *                  empty.
 *   token_dest     device int32 out [T, k]: the rank that executes each
 *                  assignment.  The rho-th occurrence (row-major) of expert e
 *                  goes to instance r_i, instances of e with a nonzero share
 *                  of this rank's assignments in ascending rank, where
 *                  sum_{j<i} q[self][e][r_j] <= rho < sum_{j<=i} q[self][e][r_j].
 *                  May be NULL when T == 0.
 *   send_counts    device int32 out [R]: sum_e q[self][e][r].
 *   status         device int32 out [2]: [0] = TOPOEP_ST_* bits; [1] = the
 *                  number of refinement moves committed (Eq. 10 transfers,
 *                  summed over domains).
 *   workspace      device memory of at least topoep_workspace_bytes bytes,
 *                  256-byte aligned, zero-filled before its first plan (see
 *                  above); it holds the plan's intermediate state.
 *
 * Host checks (TOPOEP_EINVAL): null pointers; R <= 0; G <= 0 or G does not
 * divide R; R does not divide E; k < 1 or k > E; T < 0 or T * k > INT32_MAX;
 * N_slot < 0; self_rank outside [0, R); negative costs; S_tok <= 0;
 * ||W|| < 0.  TOPOEP_ELIMIT: G > 64 or a domain's state exceeds LDS.
 * TOPOEP_EWORKSPACE: workspace too small or not 256-byte aligned.
 * TOPOEP_EHIP: a kernel launch failed.
 */
int topoep_plan(const topoep_topology *topo, const int32_t *global_load,
                const int32_t *local_topk, int32_t T, int32_t k, int32_t replica_budget,
                int32_t *replica_slots, int32_t *token_dest, int32_t *send_counts,
                int32_t *status, void *workspace, size_t workspace_bytes, void *stream);

/* topoep_plan with an explicit launch shape (NULL = default). */
int topoep_plan_ex(const topoep_topology *topo, const int32_t *global_load,
                   const int32_t *local_topk, int32_t T, int32_t k, int32_t replica_budget,
                   int32_t *replica_slots, int32_t *token_dest, int32_t *send_counts,
                   int32_t *status, void *workspace, size_t workspace_bytes, void *stream,
                   const topoep_launch *launch);

/*
 * Enqueue one kernel of the plan, for measurement.  With three kernels:
 * stage 0 = histogram (Eq. 3 row), 1 = solver (Eqs. 4, 9, 10 and routing),
 * 2 = reroute; a stage reads the workspace state the earlier stages left for
 * the same inputs, so it may be repeated after one full plan and gives the
 * same outputs.  With one kernel (solver 3), stage 0 is the whole plan.
 * TOPOEP_STAGE_FLOOR enqueues every kernel of the plan with an empty body
 * and the same grid, threads and dynamic LDS (writes nothing).  The
 * arguments are those of topoep_plan_ex.  TOPOEP_EINVAL for any other stage.
 */
int topoep_plan_stage(int32_t stage, const topoep_topology *topo, const int32_t *global_load,
                      const int32_t *local_topk, int32_t T, int32_t k, int32_t replica_budget,
                      int32_t *replica_slots, int32_t *token_dest, int32_t *send_counts,
                      int32_t *status, void *workspace, size_t workspace_bytes, void *stream,
                      const topoep_launch *launch);

/*
 * Dispatch side of a plan (Section 4.3: the expert-parallel dispatch
 * consumes the per-destination counts q of the plan).  Every rank makes the
 * same plan from the same Omega, so what a rank receives follows from the
 * plan without communication, and the send buffer can be laid out before
 * the all-to-all.
 *
 * Send-buffer layout: the assignments grouped by destination rank, ranks
 * ascending, row-major (token, k) order inside one destination.
 */

/* Bytes of device workspace topoep_dispatch_layout needs (TOPOEP_EINVAL for
 * invalid sizes, TOPOEP_ELIMIT for R > 1024). */
int topoep_layout_workspace_bytes(const topoep_topology *topo, int32_t T, int32_t k, size_t *bytes_out);

/*
 * Enqueue the send-buffer layout of a plan's destinations (one kernel).
 *
 *   token_dest    device int32 [T, k]: destinations from a plan (values
 *                 outside [0, R) take no slot).  May be NULL when T == 0.
 *   send_counts   device int32 [R]: the same plan's send counts (the number
 *                 of assignments per destination).
 *   send_offsets  device int32 out [R + 1]: exclusive prefix of send_counts
 *                 ([R] = the total).
 *   token_slot    device int32 out [T, k]: send_offsets[dest] + the number of
 *                 earlier assignments (row-major) with the same destination;
 *                 -1 where token_dest is not a rank.  May be NULL when T == 0.
 *   status        device int32 [1] or NULL: TOPOEP_ST_SYNC is ORed in if a
 *                 bounded wait gave up (slots then wrong; zero-fill the
 *                 workspace again before the next call).
 *   workspace     at least topoep_layout_workspace_bytes bytes, 256-byte
 *                 aligned, zero-filled before its first call; every call
 *                 leaves it zero again.  Calls sharing a workspace must be
 *                 ordered on one stream.
 *
 * Only topo->num_ranks is read from the topology.  Host checks as
 * topoep_plan (TOPOEP_EINVAL for null pointers or invalid sizes,
 * TOPOEP_EWORKSPACE, TOPOEP_EHIP, TOPOEP_ELIMIT for R > 1024).
 */
int topoep_dispatch_layout(const topoep_topology *topo, const int32_t *token_dest, int32_t T, int32_t k,
                           const int32_t *send_counts, int32_t *send_offsets, int32_t *token_slot,
                           int32_t *status, void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of device workspace topoep_plan_dispatch needs (the plan's, default
 * launch shape: the layout is computed inside the plan's kernels). */
int topoep_dispatch_workspace_bytes(const topoep_topology *topo, int32_t T, int32_t k,
                                    int32_t replica_budget, size_t *bytes_out);

/*
 * Enqueue one plan (as topoep_plan, default launch shape) with its dispatch
 * side computed by the same kernels:
 *   recv_counts   device int32 out [R] or NULL: recv_counts[s] =
 *                 sum_e q[s][e][self], the assignments rank s sends to this
 *                 rank under the same plan (0 when no plan is made).
 *   send_offsets, token_slot: as topoep_dispatch_layout (both NULL to skip
 *                 the layout; recv_counts and the layout may not both be
 *                 skipped).  The slot count before each chunk of ids comes
 *                 from the chunk's per-expert offsets and this rank's
 *                 instance list (each expert's occurrences are dealt to its
 *                 instances in occurrence order), so no second pass over
 *                 the destinations is needed.
 * The workspace is one buffer of topoep_dispatch_workspace_bytes bytes
 * (256-byte aligned, zero-filled before its first call).  Return codes as
 * topoep_plan.
 */
int topoep_plan_dispatch(const topoep_topology *topo, const int32_t *global_load, const int32_t *local_topk,
                         int32_t T, int32_t k, int32_t replica_budget, int32_t *replica_slots,
                         int32_t *token_dest, int32_t *send_counts, int32_t *recv_counts,
                         int32_t *send_offsets, int32_t *token_slot, int32_t *status, void *workspace,
                         size_t workspace_bytes, void *stream);

/*
 * Replica-slot parameter gather (Section 3.2): once the plan names the
 * expert of each of this rank's replica slots, the slot receives a copy of
 * that expert's parameters.  On one GPU the parameters of every expert sit
 * in one buffer and the gather is a device copy in slot order (one kernel,
 * HBM-bound).
 *
 *   topo           R, E and self_rank are read.
 *   replica_budget N_slot (the plan's).
 *   replica_slots  device int32 [R, N_slot]: a plan's replica slots; row
 *                  self_rank is used, -1 = empty (left untouched).
 *   prev_slots     device int32 [N_slot] or NULL: the experts the slots held
 *                  before; a slot whose expert is unchanged is not copied.
 *   expert_params  device [E, bytes_per_expert] (any element type), 16-byte
 *                  aligned.
 *   bytes_per_expert  ||W_e|| in bytes, a multiple of 16 (0 copies nothing).
 *   slot_params    device out [N_slot, bytes_per_expert], 16-byte aligned;
 *                  slot j receives expert_params[replica_slots[self][j]].
 *
 * Host checks: TOPOEP_EINVAL for null pointers, R <= 0, E <= 0, self_rank
 * outside [0, R), N_slot < 0, a size that is not a multiple of 16 or a
 * misaligned buffer; TOPOEP_ELIMIT for N_slot > 65535; TOPOEP_EHIP when the
 * launch fails.  Slots holding an id outside [0, E) are left untouched.
 */
int topoep_gather_replicas(const topoep_topology *topo, int32_t replica_budget, const int32_t *replica_slots,
                           const int32_t *prev_slots, const void *expert_params, int64_t bytes_per_expert,
                           void *slot_params, void *stream);

/*
 * The full model of Section 4.1: a general symmetric cost matrix C and one
 * parameter size per expert, in place of the topology's two-level cost
 * (cost_intra, cost_inter) and single expert_bytes.  Both enter the
 * stage-1 benefit b = 2 D S_tok - ||W_e|| (Eq. 9), the refinement's cost
 * change and the order in which a move takes assignments from the sources
 * (ascending c(s,rt) - c(s,rb), then s), and the exact-range bound (the
 * largest entry of C and the largest size).  Domains stay G consecutive
 * ranks.  Such plans run the three-kernel shape with the per-domain solver.
 */
typedef struct topoep_costs {
  const int32_t *cost;          /* device int32 [R, R] c(s, r) row-major, or NULL:     */
                                /* the topology's two-level cost                       */
  const int64_t *expert_bytes;  /* device int64 [E] ||W_e||, or NULL: the topology's   */
                                /* expert_bytes for every expert                       */
} topoep_costs;

/* Bytes of device workspace topoep_plan_costs needs (TOPOEP_ELIMIT when a
 * domain's state with the cost tables cannot fit in LDS). */
int topoep_costs_workspace_bytes(const topoep_topology *topo, int32_t T, int32_t k, int32_t replica_budget,
                                 size_t *bytes_out);

/*
 * topoep_plan under the full cost model (costs may be NULL, or either of
 * its pointers, for the topology's values).  The matrix is checked on the
 * device: an asymmetric matrix, a nonzero diagonal or a negative entry, or
 * a negative size, sets TOPOEP_ST_COST and no plan is made.  Other
 * arguments, outputs and return codes as topoep_plan; the workspace is
 * topoep_costs_workspace_bytes bytes.
 */
int topoep_plan_costs(const topoep_topology *topo, const topoep_costs *costs, const int32_t *global_load,
                      const int32_t *local_topk, int32_t T, int32_t k, int32_t replica_budget,
                      int32_t *replica_slots, int32_t *token_dest, int32_t *send_counts, int32_t *status,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * topoep_plan for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * It takes no workspace: the plan runs in a device array of
 * TOPOEP_NOALLOC_SCRATCH_BYTES held by the library, one per GPU it runs
 * on, until the process ends.  Each call first clears what the plan needs
 * zero there with a small kernel on `stream` (no hipMemset, no allocation,
 * no host synchronisation), then enqueues the plan of topoep_plan with the
 * default launch shape; successive calls may use different shapes.
 *
 * All calls on one GPU share that GPU's array, which keeps the last call's
 * contents: calls that overlap on one GPU (two streams, or two threads
 * without ordering) race and give wrong outputs; order them on one stream.
 *
 * Arguments, outputs and status bits as topoep_plan.  TOPOEP_EWORKSPACE:
 * the plan needs more than TOPOEP_NOALLOC_SCRATCH_BYTES of workspace
 * (topoep_workspace_bytes; every workload size up to that runs).
 * TOPOEP_EHIP: the array's device address could not be obtained, or a
 * launch failed.  Other return codes as topoep_plan.
 */
#define TOPOEP_NOALLOC_SCRATCH_BYTES (4u << 20)
int topoep_plan_noalloc(const topoep_topology *topo, const int32_t *global_load, const int32_t *local_topk,
                        int32_t T, int32_t k, int32_t replica_budget, int32_t *replica_slots, int32_t *token_dest,
                        int32_t *send_counts, int32_t *status, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* TOPOEP_H */
