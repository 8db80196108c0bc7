// TopoEP per-layer planner for MI355X (gfx950): HIP kernels and the C ABI
// declared in include/topoep.h.
//
// Three kernels per plan, enqueued back to back on one stream:
//
//   hist     one block per contiguous chunk of the flattened [T, k] ids.
//            LDS-privatised histogram; within a wave the lanes holding the
//            same expert are found with ballots over the id bits, and only
//            the lowest such lane adds the group's popcount.  Writes the
//            block's partial histogram (this rank's row of the routing
//            matrix Omega, Eq. 3, Section 3.1).
//   solve    the placement solver, in one of two shapes:
//            - one workgroup for every domain when the whole state fits in
//              the 160 KB of LDS: Omega, every domain's instances and their
//              q columns live on one CU, and each domain's refinement runs
//              on its own wavefront;
//            - one workgroup per domain (NVLink/xGMI node) otherwise, with a
//              bounded grid barrier that publishes the inter-node placement
//              of every domain and a last-workgroup step that assembles
//              this rank's instance list.
//            Either way: domain demand D (Eq. 4), inter-node placement by
//            the benefit b = 2 D S - W (Eq. 9), routing construction q, U, L
//            (Section 4.3) and intra-node refinement (Eq. 10) with wave64
//            reductions and no barrier per iteration.  Extra workgroups of
//            the same launch compute each histogram block's exclusive
//            per-expert offsets for the reroute, off the solver's path.
//   reroute  same chunking as hist.  Stable rank of every assignment among
//            the earlier assignments of its expert (ballot peer masks inside
//            a wave, per-wave counts scanned across waves, block offsets),
//            then the instance whose prefix range holds it.
//
// All arithmetic is integer; no atomic decides an order or a placement
// (LDS/global integer atomics only accumulate commutative counts, masks and
// barrier tickets, or pick list slots whose order is re-established by a
// key), so results are bitwise reproducible across runs and launch shapes.
// Divisions by launch-time constants use a multiply and a shift (fastdiv.h).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <climits>
#include <mutex>
#include <vector>

#include "fastdiv.h"
#include "topoep.h"
#include "wave.h"

namespace {

using namespace topoep_dev;

// ---------------------------------------------------------------- constants

constexpr int kCtrlBytes = 256;
constexpr int kCtrlBar = 0;      // grid-barrier arrivals
constexpr int kCtrlTicket = 1;   // finish tickets of the solver workgroups
constexpr int kCtrlStatus = 2;   // status bits accumulated during the plan
constexpr int kCtrlFinal = 3;    // final status of the plan (read by reroute)
constexpr int kCtrlTotal = 4;    // uint64 at words 4..5: sum of positive loads
constexpr int kCtrlMoves = 6;    // refinement moves of the per-domain solver
constexpr int kCtrlHelpers = 7;  // offset helpers that have published their experts' totals
// one-launch plan.  Every word a wait reads carries the plan's generation g,
// so a word left over by an earlier plan (one whose bounded wait gave up)
// never satisfies a later wait, and no word needs clearing between plans:
//   words 8..9   arrivals of the chunk workgroups, 64-bit, never reset: nb per
//                plan, so the chunk that moves it from g nb + c learns g and
//                whether it is the last (c = nb - 1);
//   word 10      g itself, read by the solver at its start and advanced by it
//                at its end (arrivals = g nb holds between plans);
//   word 11      the last chunk's verdict ((g + 1) << 2) | v (the tag g + 1
//                so that a zero-filled word is no generation's): v =
//                kVerdictSame when the histogram equals row self of Omega and
//                no id is bad, kVerdictRedo otherwise;
//   flags[b]     word 0: g + 1 once the solver's plan is ready; word 1: g + 1
//                once every chunk's counts are written;
//   ghist[g & 1] the histogram of plan g (atomic adds of the chunks), cleared
//                for plan g + 1 by the solver of plan g at its start.
constexpr int kCtrlArrive = 8;
constexpr int kCtrlGen = 10;
constexpr int kCtrlVerdict = 11;
constexpr uint32_t kVerdictSame = 1;
constexpr uint32_t kVerdictRedo = 2;
// words 16..63: phase stamps of the instrumented build (TOPOEP_STAMPS)
constexpr int kCtrlStamps = 16;

constexpr uint32_t kNoPlan = TOPOEP_ST_BAD_ID | TOPOEP_ST_NEG_LOAD | TOPOEP_ST_RANGE | TOPOEP_ST_COST;
constexpr int kLdsLimit = 160 * 1024;   // LDS per workgroup on gfx950
constexpr int kMaxSolveGroups = 128;    // co-resident by a wide margin (256 CUs)
constexpr int kMinBlocks = 2048;        // histogram/reroute blocks to aim for, at least
constexpr int kMaxBlocks = 8192;        // and at most
constexpr int kOffsetExperts = 64;      // experts per offset workgroup
// chunk workgroups the single-launch plan aims for: each chunk reads the
// instance list and up to nb / 2 rows of the other chunks' counts, so 32
// rather than 64 cut the DeepSeek-V3-like plan's HBM traffic from 1.16 to
// 0.97 MB for 0.16 us more latency (two ids per thread)
constexpr int kFusedBlocks = 32;
constexpr int kMaxFusedBlocks = 128;    // and at most (all co-resident: 256 CUs)
constexpr int kFlagStride = 32;         // words between ready flags (one 128-byte line each)
constexpr uint32_t kSpinLimit = 1u << 24;    // polls of a bounded wait before it gives up
constexpr uint32_t kHelperSpin = 1u << 12;   // polls of the offset helpers' counter before summing alone
constexpr int kListRegs = 4;   // instances per thread the instance list keeps in registers
constexpr uint32_t kIterLimit = 1u << 22;    // refinement moves per domain before ITER

// ---------------------------------------------------------------- plan

struct Plan {
  int R, G, M, E, P, N, Neff, PN, I, self, MW, RW, nbits, rbits, cap1, nent_cap, QS;
  int cI, cX;
  int64_t S, W;
  uint64_t tot_max;   // two-level model: the least total load out of the exact range (see out_of_range)
  int64_t n, chunk;
  int nb, n_solvers, n_helpers;
  int rchunks_all, rchunks_dom;   // routing: source-domain chunks (divisors of M)
  uint32_t spin_limit;   // polls of a bounded wait (0: every such wait gives up at once)
  uint32_t iter_limit;   // committed refinement moves per domain before ITER
  FastDiv fE, fG, fGP, fP, fI, fPN, fCap, fN, fMI;
  const int32_t *gl, *topk;
  int32_t *slots_out, *dest_out, *send_out, *status_out;
  int32_t *recv_out;   // receive counts [R], or null
  const int32_t *Cm;   // general cost matrix [R, R] (with general), else null
  const int64_t *We;   // ||W_e|| per expert [E] (with general), else null
  int general;         // the full model of Section 4.1 (per-domain solver only)
  int32_t *slot_out;   // send-buffer slot of every assignment [n], or null
  int32_t *offs_out;   // send offsets [R + 1] (given with slot_out)
  uint32_t *ctrl;
  int32_t *partials, *offsets, *blk_err, *repl1, *seg_e, *seg_q, *csr_ptr, *csr_r, *csr_end;
  int32_t *htot;   // three-kernel plan: each expert's count over the histogram blocks [E]
  // one-launch plan: each chunk's per-expert counts [nb][E] (16 bits: a
  // chunk holds at most 1024 x 8 ids), the histogram of the ids with a
  // bad-id count [2][E + 1] (one buffer per generation parity), one flag
  // line per chunk (kFlagStride words apart)
  uint16_t *pub;
  uint32_t *ghist, *flags;
};


// Phase stamps of the instrumented build (compiled with -DTOPOEP_STAMPS into
// a separate library for measurement; the product library has none):
// thread 0 of the calling workgroup keeps the low word of the 100 MHz
// constant clock (STAMP) or of the core clock (STAMP_CLK) for slot i (0..47)
// in LDS, and STAMP_FLUSH copies slots [lo, hi) to the control words 16..63
// at the end of the role.  Stamps stay out of global memory until then: on
// gfx9 a wait for any load also waits for every earlier store, so a store
// per stamp would delay the phase that follows it.
#ifdef TOPOEP_STAMPS
__shared__ uint32_t stamp_lds[48];
#define STAMP(p, i)                                                          \
  do {                                                                       \
    if (threadIdx.x == 0) stamp_lds[(i)] = (uint32_t)__builtin_readsteadycounter(); \
  } while (0)
#define STAMP_CLK(p, i)                                                      \
  do {                                                                       \
    if (threadIdx.x == 0) stamp_lds[(i)] = (uint32_t)__builtin_amdgcn_s_memtime(); \
  } while (0)
#define STAMP_FLUSH(p, lo, hi)                                               \
  do {                                                                       \
    if (threadIdx.x == 0)                                                    \
      for (int s_ = (lo); s_ < (hi); ++s_) (p).ctrl[kCtrlStamps + s_] = stamp_lds[s_]; \
  } while (0)
#define STAMP_CLEAR(lo, hi)                                       \
  do {                                                            \
    if (threadIdx.x == 0)                                         \
      for (int s_ = (lo); s_ < (hi); ++s_) stamp_lds[s_] = 0;     \
  } while (0)
__device__ inline void stamp_nc(int nc) { stamp_lds[17] = (uint32_t)nc; }
// Core-clock cycles of the refinement loop of domain 0 by section, summed
// over its iterations (slots 32..37, the iteration count in slot 38).
#define RSECT_DECL(d)           \
  const bool rs_on_ = (d) == 0; \
  uint64_t rs_last_ = __builtin_amdgcn_s_memtime();
#define RSECT(k)                                                                     \
  do {                                                                               \
    if (rs_on_) {                                                                    \
      const uint64_t n_ = __builtin_amdgcn_s_memtime();                              \
      if (lane_id() == 0) atomicAdd(&stamp_lds[32 + (k)], (uint32_t)(n_ - rs_last_)); \
      rs_last_ = n_;                                                                 \
    }                                                                                \
  } while (0)
#define RSECT_END(iters)                                           \
  do {                                                             \
    if (rs_on_ && lane_id() == 0) atomicAdd(&stamp_lds[38], (iters)); \
  } while (0)
#else
#define STAMP(p, i) \
  do {              \
  } while (0)
#define STAMP_CLK(p, i) \
  do {                  \
  } while (0)
#define STAMP_FLUSH(p, lo, hi) \
  do {                         \
  } while (0)
#define STAMP_CLEAR(lo, hi) \
  do {                      \
  } while (0)
__device__ inline void stamp_nc(int) {}
#define RSECT_DECL(d)
#define RSECT(k) \
  do {           \
  } while (0)
#define RSECT_END(iters) \
  do {                   \
  } while (0)
#endif

// The solvers hold more uniform values (sizes, divisors, LDS offsets,
// pointers) than the scalar register file takes; the spilled ones come back
// lane by lane (v_readlane) all over the solver.  A value passed through
// vgpr() is kept in a vector register instead (LDS addresses and the
// divisions' multiplies take vector operands anyway).
__device__ inline int vgpr(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// The plan with its divisors in vector registers (see vgpr).
__device__ inline Plan solver_plan(Plan q) {
  FastDiv *fds[] = {&q.fE, &q.fG, &q.fGP, &q.fP, &q.fI, &q.fPN, &q.fCap, &q.fN, &q.fMI};
  for (FastDiv *f : fds) {
    f->m = (uint32_t)vgpr((int)f->m);
    f->sh = (uint32_t)vgpr((int)f->sh);
  }
  return q;
}

typedef const __attribute__((address_space(4))) Plan KernargPlan;

// The plan's fields for one role of the one-launch kernel, loaded after the
// role's branch from an opaque pointer to the kernel arguments: otherwise
// the compiler loads every field either role uses at the kernel's entry and
// keeps them all live, and the solver's scalar registers spill.  (The host
// pass only type-checks this function.)
__device__ inline Plan role_plan(const Plan &p) {
#if __HIP_DEVICE_COMPILE__
  (void)p;
  KernargPlan *k = (KernargPlan *)(__builtin_amdgcn_kernarg_segment_ptr());
  asm volatile("" : "+s"(k));
  return *k;
#else
  return p;
#endif
}

// Scratch words of the histogram reduction (hist_from_partials, load_fast)
// for up to 1024 threads: max(E, 4 * threads).
__host__ __device__ inline int hist_scratch_words(const Plan &p) { return imax(p.E, 4 * 1024); }

// LDS layout of the one-workgroup-per-domain solver, in int32 words.
struct DomainLds {
  int ck, fdt, hs, rows, mask, slots, used, L, e_of, U, misc, qcol, ord, ccol, wx, words;
};

// The general cost model's per-domain tables in LDS (see domain_lds).
struct GenCost {
  const uint16_t *ord;
  const int *ccol;
  const int64_t *wx;
};

__host__ __device__ inline DomainLds domain_lds(const Plan &p) {
  DomainLds l;
  int o = 0;
  l.ck = o;    o += 2 * p.E;                 // uint64 stage-1 candidate keys
  l.fdt = o;   o += 2 * (p.M + 1);           // divisors 1..M
  l.hs = o;    o += p.E;                     // row self of Omega (histogram)
  l.rows = o;  o += p.G * p.E;               // Omega rows of the domain's sources
  l.mask = o;  o += p.E * p.MW;              // per expert: domains hosting it
  l.slots = o; o += p.G * imax(p.Neff, 1);   // replica slots of the domain's ranks
  l.used = o;  o += p.G;
  l.L = o;     o += p.G;                     // rank loads
  l.e_of = o;  o += p.I;                     // expert of each instance (-1 empty)
  l.U = o;     o += p.I;                     // instance loads
  o = (o + 3) & ~3;
  l.misc = o;  o += 64;
  l.qcol = o;                                // q[s][e][r] of the domain's instances
  o += imax(p.I * p.QS, imax(p.E + 2 + p.E * p.RW + 64 + p.nent_cap, hist_scratch_words(p)));
  // general cost model: per (busiest, target) pair of the domain's ranks the
  // sources in (c(s,rt) - c(s,rb), s) order (16-bit), the costs to the
  // domain's ranks, ||W_e||
  l.ord = o;   o += p.general ? (p.G * p.G * p.R + 1) / 2 : 0;
  l.ccol = o;  o += p.general ? p.G * p.R : 0;
  o = (o + 1) & ~1;
  l.wx = o;    o += p.general ? 2 * p.E : 0;
  l.words = o;
  return l;
}

// LDS layout of the single-workgroup solver: every domain's state at once.
struct SingleLds {
  int ck, em, fdt, hs, cnt, dfree, mask, bm, sendl, wt, repl, slots, used, L, e_of, U, misc, om, qcol, words;
};

__host__ __device__ inline SingleLds single_lds(const Plan &p) {
  SingleLds l;
  int o = 0;
  l.ck = o;    o += 2 * p.M * ((p.E + 15) & ~15);   // uint64 stage-1 candidate keys per domain (stride E rounded to 16)
  l.em = o;    o += 2 * p.M * p.E;            // uint64 per domain and expert: local ranks hosting it
  l.fdt = o;   o += 2 * (p.M + 1);            // divisors 1..M
  l.hs = o;    o += p.E;                      // histogram of local_topk
  l.cnt = o;   o += p.M;                      // candidates per domain
  l.dfree = o; o += p.M;                      // 1: a rank of the domain has a free slot
  l.mask = o;  o += p.E * p.MW;               // per expert: hosting domains
  l.bm = o;    o += p.E * p.RW;               // per expert: ranks in this rank's instance list
  l.sendl = o; o += p.R;                      // send counts being summed
  l.wt = o;    o += imax(32, (p.E + 63) / 64);   // per-wave totals of a scan (and their sum), or per 64 experts
  l.repl = o;  o += p.M * imax(p.cap1, 1);    // stage-1 replicas per domain
  l.slots = o; o += p.R * imax(p.Neff, 1);    // replica slots of every rank
  l.used = o;  o += p.R;
  l.L = o;     o += p.R;                      // rank loads
  l.e_of = o;  o += p.M * p.I;                // expert of each instance
  l.U = o;     o += p.M * p.I;                // instance loads
  o = (o + 3) & ~3;
  l.misc = o;  o += 64;
  l.om = o;                                   // Omega' [R][E], then list scratch
  o += p.R * p.E;
  o = (o + 3) & ~3;
  l.qcol = o;                                 // partial-sum scratch, then q columns
  o += imax(p.M * p.I * p.QS, hist_scratch_words(p));
  l.words = o;
  return l;
}

// LDS layout of a chunk workgroup of the single-launch plan (nt threads).
struct ChunkLds {
  int wc, run, ptr, ent, gs, so, flag, words;
};

__host__ __device__ inline ChunkLds chunk_lds(const Plan &p, int nt) {
  ChunkLds l;
  int o = 0;
  l.wc = o;   o += (nt >> 6) * p.E;          // per-wave counts, then offsets in the block
  l.run = o;  o += p.E;                      // offset of the block per expert
  l.ptr = o;  o += p.E + 1;                  // instance list: first entry per expert
  o = (o + 1) & ~1;
  l.ent = o;  o += 2 * p.nent_cap;           //   (cumulative share, instance rank) per entry
  l.gs = o;   o += imax(nt, p.E);            // partial sums of the chunk's offsets, then counts per rank
  l.so = o;   o += p.R + 1 + (nt >> 6) + 1;  // send offsets and their scan scratch
  l.flag = o; o += 4;
  l.words = o;
  return l;
}

// Global -> LDS copy by the whole workgroup, four 16-byte loads in flight
// per thread when source, destination and length allow.
__device__ void copy_to_lds(int *dst, const int *src, int n) {
  const int tid = threadIdx.x, nt = blockDim.x;
  if (((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15) == 0 && (n & 3) == 0) {
    const int n4 = n >> 2;
    const int4 *s4 = reinterpret_cast<const int4 *>(src);
    int4 *d4 = reinterpret_cast<int4 *>(dst);
    int base = tid;
    for (; base + 3 * nt < n4; base += 4 * nt) {
      const int4 a = s4[base], b = s4[base + nt], c = s4[base + 2 * nt], d = s4[base + 3 * nt];
      d4[base] = a;
      d4[base + nt] = b;
      d4[base + 2 * nt] = c;
      d4[base + 3 * nt] = d;
    }
    for (; base < n4; base += nt) d4[base] = s4[base];
  } else {
    int base = tid;
    for (; base + 3 * nt < n; base += 4 * nt) {
      const int a = src[base], b = src[base + nt], c = src[base + 2 * nt], d = src[base + 3 * nt];
      dst[base] = a;
      dst[base + nt] = b;
      dst[base + 2 * nt] = c;
      dst[base + 3 * nt] = d;
    }
    for (; base < n; base += nt) dst[base] = src[base];
  }
}

// make_fastdiv on the device without a 64-bit integer division: for
// d < 2^21 the quotient 2^(31+l) / d is formed in double precision and
// corrected to the exact floor with integer arithmetic.
__device__ inline FastDiv make_fastdiv_dev(uint32_t d) {
  if (d >= (1u << 21)) return make_fastdiv(d);
  const uint32_t l = d <= 1 ? 0u : 32u - (uint32_t)__clz(d - 1);
  const uint64_t x = 1ull << (31 + l);
  uint64_t q = (uint64_t)((double)x / (double)d);
  int64_t r = (int64_t)(x - q * d);
  while (r < 0) {
    --q;
    r += d;
  }
  while (r >= (int64_t)d) {
    ++q;
    r -= d;
  }
  FastDiv f;
  f.m = (uint32_t)(q + (r != 0));
  f.sh = 31 + l;
  return f;
}

// x / d with one high multiply (x < 2^31): m < 2^32 and sh >= 32 except for
// d = 1, where the quotient is x.
__device__ inline uint32_t fdiv_hi(uint32_t x, FastDiv f) {
  const uint32_t hi = __umulhi(x, f.m) >> ((f.sh - 32u) & 31u);   // computed for every lane: a select, no branch
  return f.sh >= 32 ? hi : x;
}

// Histogram of local_topk (row self of Omega) as the sum of the histogram
// blocks' partials: thread (e, g) sums its share of the blocks with eight
// loads in flight; scratch needs hist_scratch_words(p) = max(E, 4 * blockDim)
// words (the int4 path keeps blockDim int4 partial sums).
__device__ void hist_from_partials(const Plan &p, int *hs, int *scratch) {
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E, nb = p.nb;
  if ((E & 3) == 0) {
    // thread (e4, g): four experts, a share of the blocks, 16-byte loads
    const int E4 = E >> 2;
    const int groups = imax(1, nt / E4);
    const int per = (nb + groups - 1) / groups;
    const int4 *part4 = reinterpret_cast<const int4 *>(p.partials);
    int4 *scr4 = reinterpret_cast<int4 *>(scratch);
    for (int t = tid; t < groups * E4; t += nt) {
      const int g = t / E4, e4 = t - g * E4;
      const int b0 = g * per, b1 = imin(nb, b0 + per);
      int4 run = make_int4(0, 0, 0, 0);
      for (int b = b0; b < b1; b += 8) {
        int4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = b + u < b1 ? part4[(int64_t)(b + u) * E4 + e4] : make_int4(0, 0, 0, 0);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          run.x += v[u].x;
          run.y += v[u].y;
          run.z += v[u].z;
          run.w += v[u].w;
        }
      }
      scr4[t] = run;
    }
    lds_barrier();
    for (int e = tid; e < E; e += nt) {
      int sum = 0;
      for (int g = 0; g < groups; ++g) sum += scratch[g * E + e];
      hs[e] = sum;
    }
    lds_barrier();
    return;
  }
  const int groups = imax(1, nt / E);
  const int per = (nb + groups - 1) / groups;
  for (int t = tid; t < groups * E; t += nt) {
    const int g = (int)fdiv((uint32_t)t, p.fE), e = t - g * E;
    const int b0 = g * per, b1 = imin(nb, b0 + per);
    int run = 0;
    for (int b = b0; b < b1; b += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = b + u < b1 ? p.partials[(int64_t)(b + u) * E + e] : 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) run += v[u];
    }
    scratch[t] = run;
  }
  lds_barrier();
  for (int e = tid; e < E; e += nt) {
    int sum = 0;
    for (int g = 0; g < groups; ++g) sum += scratch[g * E + e];
    hs[e] = sum;
  }
  lds_barrier();
}

// Load phase of the single-workgroup solver when the sizes are small
// (E % 4 == 0, Omega at most 4 int4 and the partials at most 8 int4 per
// thread): every global load (the histogram blocks' partials, Omega and the
// blocks' error flags) is issued before any is used, branch-free with
// clamped indices.  Fills om (Omega, row self replaced by the histogram) and
// hs, and accumulates status bits and the total load in misc.
__device__ inline bool load_fast_ok(const Plan &p) {
  const int nt = blockDim.x, E4 = p.E >> 2;
  if ((p.E & 3) || E4 > nt || ((reinterpret_cast<uintptr_t>(p.gl)) & 15)) return false;
  const int G4 = nt / E4;
  return (p.R * p.E) / 4 <= 4 * nt && (p.nb + G4 - 1) / G4 <= 8 && p.nb <= nt;
}

__device__ void load_fast(const Plan &p, int *om, int *hs, int *scratch, int *misc) {
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E, R = p.R, nb = p.nb;
  const int E4 = E >> 2, G4 = nt / E4;
  const int n4 = (R * E) >> 2;
  const int g = tid / E4, e4 = tid - g * E4;
  const int4 *part4 = reinterpret_cast<const int4 *>(p.partials);
  const int4 *gl4 = reinterpret_cast<const int4 *>(p.gl);
  const int4 z = make_int4(0, 0, 0, 0);
  int4 pv[8], ov[4];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int b = g + u * G4;
    pv[u] = part4[(int64_t)imin(b, nb - 1) * E4 + e4];
    if (b >= nb || g >= G4) pv[u] = z;
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) ov[u] = gl4[imin(tid + u * nt, n4 - 1)];
  const int be = p.blk_err[imin(tid, nb - 1)];
  // Omega to LDS; negative entries and the total of positive loads
  int4 *om4 = reinterpret_cast<int4 *>(om);
  bool neg = false;
  uint64_t tot = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = tid + u * nt;
    if (i < n4) {
      om4[i] = ov[u];
      neg |= (ov[u].x | ov[u].y | ov[u].z | ov[u].w) < 0;
      tot += (uint64_t)(ov[u].x > 0 ? ov[u].x : 0) + (uint64_t)(ov[u].y > 0 ? ov[u].y : 0) +
             (uint64_t)(ov[u].z > 0 ? ov[u].z : 0) + (uint64_t)(ov[u].w > 0 ? ov[u].w : 0);
    }
  }
  int4 s = z;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    s.x += pv[u].x;
    s.y += pv[u].y;
    s.z += pv[u].z;
    s.w += pv[u].w;
  }
  if (g < G4) reinterpret_cast<int4 *>(scratch)[g * E4 + e4] = s;
  lds_barrier();
  // histogram; row self of Omega := histogram
  bool diff = false;
  for (int e = tid; e < E; e += nt) {
    int h = 0;
    for (int gg = 0; gg < G4; ++gg) h += scratch[gg * E + e];
    hs[e] = h;
    const int gself = om[p.self * E + e];
    diff |= gself != h;
    if (gself > 0) tot -= (uint64_t)gself;
    if (h > 0) tot += (uint64_t)h;
    om[p.self * E + e] = h;
  }
  tot = wave_sum_u64(tot);
  const uint64_t any_neg = __ballot(neg), any_diff = __ballot(diff), any_bad = __ballot(tid < nb && be != 0);
  if (lane_id() == 0) {
    const uint32_t w = (any_neg ? TOPOEP_ST_NEG_LOAD : 0u) | (any_diff ? TOPOEP_ST_SELF_DIFF : 0u) |
                       (any_bad ? TOPOEP_ST_BAD_ID : 0u);
    if (w) atomicOr(reinterpret_cast<unsigned *>(&misc[0]), w);
    if (tot) atomicAdd(reinterpret_cast<unsigned long long *>(misc + 8), (unsigned long long)tot);
  }
  lds_barrier();
}

// Exclusive per-expert offset of every histogram block, for the reroute
// (offset workgroup h of n_helpers handles kOffsetExperts experts at a time),
// and each expert's count over all blocks (htot, the histogram of
// local_topk), announced by one increment of the helpers' counter as soon
// as the totals are written: the offsets follow in a second pass (only the
// next launch reads them).  scratch: nw x 64 words per expert group of this
// workgroup (one group when n_helpers covers E, as the host sets it).
__device__ void block_offsets(const Plan &p, int h, int *scratch, bool announce) {
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6, E = p.E, nb = p.nb;
  const int el = tid & 63, g = tid >> 6;
  const int per = (nb + nw - 1) / nw;
  const int b0 = g * per, b1 = imin(nb, b0 + per);
  const int gstride = p.n_helpers * kOffsetExperts;
  // pass 1: each wave's sum over its blocks, per expert of every group
  int grp = 0;
  for (int e0 = h * kOffsetExperts; e0 < E; e0 += gstride, ++grp) {
    const int e = e0 + el;
    int run = 0;
    if (e < E) {
      for (int b = b0; b < b1; b += 8) {
        int v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = b + u < b1 ? p.partials[(int64_t)(b + u) * E + e] : 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) run += v[u];
      }
    }
    scratch[(grp * nw + g) * 64 + el] = run;
  }
  __syncthreads();
  // the totals (the expert's count over every block), then the announcement
  grp = 0;
  for (int e0 = h * kOffsetExperts; e0 < E; e0 += gstride, ++grp) {
    const int e = e0 + el;
    if (g == nw - 1 && e < E) {
      int tot = 0;
      for (int g2 = 0; g2 < nw; ++g2) tot += scratch[(grp * nw + g2) * 64 + el];
      p.htot[e] = tot;
    }
  }
  if (announce) {
    // publish: every total written before the count of finished helpers
    // (only the per-domain solver reads it)
    drain_then_barrier();
    if (tid == 0) __hip_atomic_fetch_add(&p.ctrl[kCtrlHelpers], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
  // pass 2: the blocks' exclusive offsets
  grp = 0;
  for (int e0 = h * kOffsetExperts; e0 < E; e0 += gstride, ++grp) {
    const int e = e0 + el;
    if (e >= E) continue;
    int base = 0;
    for (int g2 = 0; g2 < g; ++g2) base += scratch[(grp * nw + g2) * 64 + el];
    for (int b = b0; b < b1; b += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = b + u < b1 ? p.partials[(int64_t)(b + u) * E + e] : 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (b + u < b1) p.offsets[(int64_t)(b + u) * E + e] = base;
        base += v[u];
      }
    }
  }
}

// The histogram of local_topk (row self of Omega) for the per-domain
// solver: the offset helpers' totals once all of them have published, else
// the sum of the blocks' counts made here.  The helpers normally finish in
// a few microseconds beside the solver workgroups; the wait is bounded by
// kHelperSpin polls (~0.2 ms), not by the hang guard, so a dispatch whose
// helpers start late costs little.  flag: one LDS word.
__device__ void row_self(const Plan &p, int *hs, int *scratch, int *flag) {
  if (threadIdx.x == 0) {
    uint32_t it = 0;
    int ok = 1;
    while (__hip_atomic_load(&p.ctrl[kCtrlHelpers], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
           (uint32_t)p.n_helpers) {
      if (++it > kHelperSpin) {
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    *flag = ok;
  }
  __syncthreads();
  if (*flag) {
    for (int e = threadIdx.x; e < p.E; e += blockDim.x) hs[e] = p.htot[e];
    lds_barrier();
  } else {
    hist_from_partials(p, hs, scratch);
  }
}

// Exact-range check: the total load fits int32 and 4 S total c + c W < 2^62
// (c = max(c_intra, c_inter, 1)), so every benefit and cost change is exact.
__device__ inline bool out_of_range_cw(const Plan &p, uint64_t total, uint64_t cmax, uint64_t wmax) {
  const uint64_t lim = 1ull << 62;
  const uint64_t cm = cmax > 1 ? cmax : 1;
  if (total > 0x7FFFFFFFull) return true;
  // 4 S total cm and cm W with overflow checks (every factor is nonnegative)
  uint64_t tok = 0, rep = 0;
  if (__builtin_mul_overflow((uint64_t)p.S, 4ull * total, &tok)) return true;
  if (__builtin_mul_overflow(tok, cm, &tok)) return true;
  if (__builtin_mul_overflow(wmax, cm, &rep)) return true;
  if (tok >= lim || rep >= lim) return true;
  return tok + rep >= lim;
}

// The same check for the two-level model, whose c and W the host knows: with
// k = 4 S c, 4 S total c + c W >= 2^62 holds exactly when c W >= 2^62 or
// total >= ceil((2^62 - c W) / k), the threshold the host stores in tot_max
// (0 when c W >= 2^62); two compares instead of overflow-checked products.
__device__ inline bool out_of_range(const Plan &p, uint64_t total) {
  return total > 0x7FFFFFFFull || total >= p.tot_max;
}

// Grid barrier of the per-domain solver workgroups: all of them are
// resident (at most kMaxSolveGroups), and the wait is bounded so the kernel
// always exits.
__device__ bool grid_barrier(uint32_t *count, uint32_t groups, uint32_t spin_limit, int *flag) {
  drain_then_barrier();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(count, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    int ok = 0;
    for (uint32_t it = 0; it < spin_limit; ++it) {
      if (it > 0) __builtin_amdgcn_s_sleep(1);
      if (__hip_atomic_load(count, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) >= groups) {
        ok = 1;
        break;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    *flag = ok;
  }
  __syncthreads();
  return *flag != 0;
}

// ---------------------------------------------------------------- histogram

template <int IPT>
__global__ __launch_bounds__(1024) void hist_kernel(Plan p) {
  extern __shared__ int smem_h[];
  int *h = smem_h;
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  for (int e = tid; e < p.E; e += nt) h[e] = 0;
  __syncthreads();
  const int64_t lo = (int64_t)b * p.chunk;
  const int64_t hi = lo + p.chunk < p.n ? lo + p.chunk : p.n;
  const int64_t tile = (int64_t)nt * IPT;
  int bad = 0;
  for (int64_t base = lo; base < hi; base += tile) {
    const int64_t wbase = base + (int64_t)wave * 64 * IPT + lane;
    int ev[IPT];
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = wbase + i * 64;
      ev[i] = idx < hi ? p.topk[idx] : -1;
    }
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = wbase + i * 64;
      const bool inr = idx < hi;
      const bool valid = inr && (unsigned)ev[i] < (unsigned)p.E;
      bad |= (inr && !valid) ? 1 : 0;
      if (valid) atomicAdd(&h[ev[i]], 1);
    }
  }
  bad = __syncthreads_or(bad);
  for (int e = tid; e < p.E; e += nt) p.partials[(int64_t)b * p.E + e] = h[e];
  if (tid == 0) p.blk_err[b] = bad;
}

// ---------------------------------------------------------------- solver steps

// Routing construction (Section 4.3) for NI instances, instance i of domain
// dom_of(i) holding expert e_of[i] (-1 = empty).  The unique instance of e
// inside dom(s) takes all of omega[s][e]; sources of a domain without an
// instance of e split omega[s][e] evenly over every instance of e (one per
// hosting domain, so an instance's position in ascending rank order is the
// number of hosting domains below its own), the lowest positions taking the
// remainder; sources of another domain that hosts e send it nothing.  The
// case is decided once per source domain.  Thread t handles source domains
// [c * M / chunks, (c + 1) * M / chunks) of instance t % NI, c = t / NI
// (chunks divides M); omega[s][e] of instance i is src_of(i, e)[s * stride];
// qcol[i * QS + s] = q[s][e][r_i] (may be the source itself: every value is
// read before it is written); U[i] += sum_s q (U must be zero on entry).
struct RouteCase {
  FastDiv fn;
  int n, below, keep, take;
};

template <int B>
__device__ inline int route_batch(const int *src, int stride, int *dst, const RouteCase &rc) {
  int w[B];
#pragma unroll
  for (int u = 0; u < B; ++u) w[u] = src[u * stride];
  int sum = 0;
#pragma unroll
  for (int u = 0; u < B; ++u) {
    const int qq = (int)fdiv_hi((uint32_t)w[u], rc.fn);
    const int split = qq + (rc.below < w[u] - qq * rc.n ? 1 : 0);
    const int q = (w[u] & rc.keep) + (split & rc.take);   // local: w; hosting domain: 0; else the split
    dst[u] = q;
    sum += q;
  }
  return sum;
}

// q[s][e][r] of an instance of e in domain d for one source s of domain ds,
// w = omega[s][e]: the routing rule of route_instances for a single source
// (the whole load to the instance in the source's own domain, nothing when
// another instance sits there, else the even split over the hosting
// domains, the remainder to the lowest ones).
__device__ inline int route_q(const Plan &p, int d, int e, int w, int ds, const uint32_t *mask, const FastDiv *fdt) {
  if (ds == d) return w;                                   // the instance inside dom(s)
  const uint32_t *me = mask + e * p.MW;
  if ((me[ds >> 5] >> (ds & 31)) & 1u) return 0;           // dom(s) hosts e itself
  int n = 0, below = 0;
  for (int wd = 0; wd < p.MW; ++wd) {
    const uint32_t bits = me[wd];
    n += __popc(bits);
    const int lo = wd * 32;
    if (d >= lo + 32) below += __popc(bits);
    else if (d > lo) below += __popc(bits & ((1u << (d - lo)) - 1u));
  }
  const FastDiv fn = fdt[n];
  const int qq = (int)fdiv_hi((uint32_t)w, fn);
  return qq + (below < w - qq * n ? 1 : 0);
}

__device__ inline int route_self_q(const Plan &p, int d, int e, int w, const uint32_t *mask, const FastDiv *fdt) {
  return route_q(p, d, e, w, (int)fdiv((uint32_t)p.self, p.fG), mask, fdt);
}

// Receive counts: recv[s] = sum over the instances on rank self (instance
// indices i0 .. i0 + PN - 1, expert e_of[i], column qcol + i * QS) of
// q[s][e][self].  With full, every source's q of those instances is in
// qcol (and reflects the refinement); otherwise the routing rule gives it
// from omega(s, e).
// One thread per (source, instance); acc: R words of LDS scratch.
template <class OmegaOf>
__device__ void write_recv_counts(const Plan &p, int i0, const int *e_of, const int *qcol, bool full,
                                  const uint32_t *mask, const FastDiv *fdt, OmegaOf omega_of, int *acc) {
  const int tid = threadIdx.x, nt = blockDim.x, R = p.R, PN = p.PN;
  const int ds = (int)fdiv((uint32_t)p.self, p.fG);
  for (int s = tid; s < R; s += nt) acc[s] = 0;
  lds_barrier();
  for (int x = tid; x < R * PN; x += nt) {
    const int s = (int)fdiv((uint32_t)x, p.fPN), i = i0 + x - s * PN, e = e_of[i];
    if (e < 0) continue;
    const int q = full ? qcol[i * p.QS + s]
                       : route_q(p, ds, e, omega_of(s, e), (int)fdiv((uint32_t)s, p.fG), mask, fdt);
    if (q) atomicAdd(&acc[s], q);
  }
  lds_barrier();
  for (int s = tid; s < R; s += nt) p.recv_out[s] = acc[s];
}

// full(d): whether every source's q is needed for domain d's instances.  A
// domain whose refinement cannot move anything (no free slot) only needs
// q[self] (send counts and this rank's instance list read nothing else, and
// instance loads feed the refinement only): the chunk holding dom(self)
// writes that one value, then calls on_self(i, d, e, q); the other sources
// of the column are left unset.
template <class SrcOf, class DomOf, class Full, class OnSelf>
__device__ void route_instances(const Plan &p, int NI, FastDiv fNI, int chunks, const int *e_of,
                                const uint32_t *mask, const FastDiv *fdt, int *qcol, int *U, SrcOf src_of,
                                int stride, DomOf dom_of, Full full, OnSelf on_self) {
  const int tid = threadIdx.x, nt = blockDim.x, G = p.G;
  const int dpc = p.M / chunks;
  const int c_self = (int)fdiv((uint32_t)p.self, p.fG) / dpc;
  for (int t = tid; t < NI * chunks; t += nt) {
    const int c = (int)fdiv((uint32_t)t, fNI), i = t - c * NI;
    const int e = e_of[i];
    const int ds0 = c * dpc, ds1 = ds0 + dpc;
    int *row = qcol + i * p.QS;
    const int d = dom_of(i);
    if (!full(d)) {
      if (c == c_self) {
        const int q = e < 0 ? 0 : route_self_q(p, d, e, src_of(i, e)[p.self * stride], mask, fdt);
        row[p.self] = q;
        on_self(i, d, e, q);
      }
      continue;
    }
    if (e < 0) {
      for (int s = ds0 * G; s < ds1 * G; ++s) row[s] = 0;
      continue;
    }
    const uint32_t *me = mask + e * p.MW;
    RouteCase rc;
    rc.n = 0;
    rc.below = 0;
    for (int wd = 0; wd < p.MW; ++wd) {
      const uint32_t bits = me[wd];
      rc.n += __popc(bits);
      const int lo = wd * 32;
      if (d >= lo + 32) rc.below += __popc(bits);
      else if (d > lo) rc.below += __popc(bits & ((1u << (d - lo)) - 1u));
    }
    rc.fn = fdt[rc.n];
    const int *col = src_of(i, e);
    int usum = 0;
    for (int ds = ds0; ds < ds1; ++ds) {
      const bool local = ds == d;
      const bool zero = !local && ((me[ds >> 5] >> (ds & 31)) & 1u);
      rc.keep = local ? -1 : 0;
      rc.take = (local || zero) ? 0 : -1;
      const int *src = col + ds * G * stride;
      int *dst = row + ds * G;
      int j = 0;
      for (; j + 8 <= G; j += 8) usum += route_batch<8>(src + j * stride, stride, dst + j, rc);
      for (; j + 4 <= G; j += 4) usum += route_batch<4>(src + j * stride, stride, dst + j, rc);
      for (; j < G; ++j) usum += route_batch<1>(src + j * stride, stride, dst + j, rc);
    }
    if (usum) atomicAdd(&U[i], usum);
  }
}

// Divisors 1..M (hosting-domain counts) for the routing's even splits,
// built once per workgroup into fdt[0..M].
__device__ inline void build_divisors(int M, FastDiv *fdt) {
  for (int n = threadIdx.x; n <= M; n += blockDim.x) fdt[n] = make_fastdiv_dev((uint32_t)(n > 0 ? n : 1));
}

// Instance index of expert e on local rank j of domain d, or -1.
__device__ inline int instance_of(const Plan &p, int d, int j, int e, const int *slots,
                                  const int *used) {
  const int rank = d * p.G + j;
  if ((int)fdiv((uint32_t)e, p.fP) == rank) return j * p.PN + (e - rank * p.P);
  const int u = used[j];
  for (int t = 0; t < u; ++t)
    if (slots[j * p.Neff + t] == e) return j * p.PN + p.P + t;
  return -1;
}

// Forms of the refinement loop: the register form where the domain fits it
// (refine_in_registers), scoring (instance, target) pairs when a rank has
// at most four instances (refine_in_pairs; one-launch kernel only), else
// the LDS form; a kernel that knows its form carries only that one's code.
constexpr int kRefineAny = 0, kRefineReg = 1, kRefineLds = 2, kRefinePairs = 3;
__host__ __device__ inline bool refine_in_registers(int G, int I, int PN) { return G <= 16 && I <= 128 && PN <= 64; }
// the register form scoring (instance, target) pairs: at most four instances
// per rank (a row of 16 lanes each)
__host__ __device__ inline bool refine_in_pairs(int G, int I, int PN) { return refine_in_registers(G, I, PN) && PN <= 4; }
__host__ __device__ inline int refine_form(int G, int I, int PN) {
  return refine_in_pairs(G, I, PN) ? kRefinePairs : (refine_in_registers(G, I, PN) ? kRefineReg : kRefineLds);
}

// Minimum over each row of 16 lanes, left in every lane of the row.
__device__ inline uint32_t row_min_all_u32(uint32_t v) {
  uint32_t o;
  o = dpp_mov<0x128>(v); v = o < v ? o : v;
  o = dpp_mov<0x124>(v); v = o < v ? o : v;
  o = dpp_mov<0x122>(v); v = o < v ? o : v;
  o = dpp_mov<0x121>(v); v = o < v ? o : v;
  return v;
}
__device__ inline uint64_t row_min_all_u64(uint64_t v) {
  uint64_t o;
  o = dpp_mov64<0x128>(v); v = o < v ? o : v;
  o = dpp_mov64<0x124>(v); v = o < v ? o : v;
  o = dpp_mov64<0x122>(v); v = o < v ? o : v;
  o = dpp_mov64<0x121>(v); v = o < v ? o : v;
  return v;
}
// Lane l's value in a vector register (the same in every lane), and a lane
// predicate as 0 or 1 in a vector register.  A single wave pays about 20
// cycles each time the scalar unit consumes a vector result (a lane mask
// combined with s_and, a branch on a compare, arithmetic on a readlane), and
// plain bool logic lives in scalar lane masks; values passed through these
// keep such logic in vector instructions (selects, ands) instead.
__device__ inline int vlane(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ inline uint64_t vlane64(uint64_t v, int l) {
  return ((uint64_t)(uint32_t)vlane((int)(v >> 32), l) << 32) | (uint32_t)vlane((int)v, l);
}
__device__ inline int vb(bool b) { return b ? 1 : 0; }
__device__ inline int row_max_all_i32(int v) {
  int o;
  o = (int)dpp_mov<0x128>((uint32_t)v); v = o > v ? o : v;
  o = (int)dpp_mov<0x124>((uint32_t)v); v = o > v ? o : v;
  o = (int)dpp_mov<0x122>((uint32_t)v); v = o > v ? o : v;
  o = (int)dpp_mov<0x121>((uint32_t)v); v = o > v ? o : v;
  return v;
}

// Register form of the refinement loop below (two-level cost, G <= GM <= 16
// ranks, I <= 128 instances, PN <= 64): lane l keeps instances l and l + 64
// (expert, load, the domain ranks hosting that expert) and lane j < G rank
// j's load and used slots; only the q columns stay in LDS.  It makes the
// same moves in the same order as the LDS form (the busiest rank rb, lowest
// index on ties; one lane per instance of rb scoring its lightest
// receivers, or with at most four instances per rank one row of 16 lanes
// per instance, a lane per target rank; the minimum of (delta descending,
// L[rt], cost change, e, rt);
// the transfer from rt's own assignments, then the other sources
// ascending, rb's own last), as straight-line vector code with few scalar
// hand-overs (see vlane and vb).  e_of, U, Lr, used, slots, em and the q
// columns hold the final state on return.
template <int GM, bool Pairs>
__device__ uint32_t refine_domain_reg(const Plan &p, int d, int *e_of, int *U, int *qcol, int *slots, int *used,
                                      int *Lr, uint64_t *em, uint32_t *flags) {
  const int lane = lane_id();
  const int G = p.G, PN = p.PN, R = p.R, P = p.P, Neff = p.Neff, QS = p.QS, I = p.I;
  const int r0 = d * G;
  const bool two_level = p.cI > 0;
  const int64_t tokc = 2 * p.S * (int64_t)p.cI;
  const int64_t repI = (int64_t)p.cI * p.W, repX = (int64_t)p.cX * p.W;
  // rb's instances one per lane, or (at most four of them, pairs) one per
  // row of 16 lanes, a lane per target rank
  constexpr bool pairs = Pairs;
  const bool one_row = pairs ? PN <= 1 : PN <= 16;
  const int vl = vgpr(lane);
  const int rank_lane = vb(vl < G), rb_lane = vb(vl < PN), src_lane = vb(vl < R);
  // instance registers: lane l holds instances l and l + 64
  int ie0 = vl < I ? e_of[vl] : -1, ie1 = vl + 64 < I ? e_of[vl + 64] : -1;
  int iu0 = vl < I ? U[vl] : 0, iu1 = vl + 64 < I ? U[vl + 64] : 0;
  uint32_t ih0 = ie0 >= 0 ? (uint32_t)em[ie0] : 0u, ih1 = ie1 >= 0 ? (uint32_t)em[ie1] : 0u;
  // rank registers (lanes >= G: never the busiest, never a receiver)
  int lj = rank_lane ? Lr[vl] : -1;
  int uj = rank_lane ? used[vl] : Neff;
  uint32_t it = 0;
  RSECT_DECL(d);
  for (;; ++it) {
    // ---- busiest rank rb: the largest L, lowest index on ties
    const int Lrb = vlane(row_max_all_i32(lj), 0);
    const int rbj_s = __ffsll((long long)__ballot(rank_lane && lj == Lrb)) - 1;
    const int rbj = vgpr(rbj_s);
    const int rb = r0 + rbj;
    // ---- receivers: L[rt] <= L[rb] - 2; the lightest with a free slot form
    // one level (lf, tfm); hosting receivers matter up to that level (lightm)
    const int low = rank_lane & vb(vl != rbj) & vb(Lrb - lj >= 2);
    const int fr = low & vb(uj < Neff);
    const uint32_t lf = (uint32_t)vlane((int)row_min_all_u32(fr ? (uint32_t)lj : ~0u), 0);
    const uint32_t tfm = (uint32_t)vgpr((int)(uint32_t)__ballot(fr & vb((uint32_t)lj == lf)));
    const uint32_t lightm = (uint32_t)vgpr((int)(uint32_t)__ballot(low & vb((uint32_t)lj <= lf)));
    RSECT(0);
    // ---- the candidates: a scored lane's instance of rb (expert e, load u,
    // hosting mask hm), its lightest receiver level lm, delta, and its best
    // target bj with that target's cost change bc and q column word bq
    int e, u, valid, delta, bj, bq;
    uint32_t hm, lm;
    int64_t bc;
    if constexpr (pairs) {
      // lane 16 c + j: rb's instance c (a = rbj PN + c) against local rank
      // j; the row of 16 lanes of instance c keeps its lightest receivers
      // (low ranks with a free slot or already hosting e), which are its
      // targets, each scored by one lane
      const uint32_t lowm = (uint32_t)vgpr((int)(uint32_t)__ballot(low)), frm = (uint32_t)vgpr((int)(uint32_t)__ballot(fr));
      const int c = vl >> 4, jj = vl & 15;
      const int a = rbj * PN + c;
      const int src = (a & 63) << 2;
      const int e0 = __builtin_amdgcn_ds_bpermute(src, ie0), e1 = __builtin_amdgcn_ds_bpermute(src, ie1);
      const int u0 = __builtin_amdgcn_ds_bpermute(src, iu0), u1 = __builtin_amdgcn_ds_bpermute(src, iu1);
      const int h0 = __builtin_amdgcn_ds_bpermute(src, (int)ih0), h1 = __builtin_amdgcn_ds_bpermute(src, (int)ih1);
      const int Lq = __builtin_amdgcn_ds_bpermute(jj << 2, lj);   // rank jj's load (-1 from G on)
      const int *qa = qcol + (c < PN ? a : 0) * QS;
      const int qrb = two_level ? qa[rb] : 0;
      const int qt = two_level ? qa[r0 + (jj < G ? jj : 0)] : 0;
      const int hi = vb(a >= 64);
      e = hi ? e1 : e0;
      u = hi ? u1 : u0;
      hm = (uint32_t)(hi ? h1 : h0);
      const int cand = vb(c < PN) & vb(e >= 0) & vb(u > 0);
      const int hostj = (int)((hm >> jj) & 1u);
      const int ok = cand & (int)((lowm >> jj) & 1u) & ((int)((frm >> jj) & 1u) | hostj);
      lm = row_min_all_u32(ok ? (uint32_t)Lq : ~0u);
      valid = ok & vb((uint32_t)Lq == lm);
      delta = imin(u, (Lrb - (int)lm) >> 1);
      int64_t dc = 0;
      if (two_level) {
        const int m_rt = imin(delta, qt);
        const int rest = delta - m_rt;
        const int m_rb = rest - imin(rest, u - qt - qrb);
        dc = tokc * (int64_t)(m_rb - m_rt);
      }
      bc = hostj ? dc : dc + (((int)fdiv((uint32_t)e, p.fGP) == d) ? repI : repX);
      bj = jj;
      bq = qt;
    } else {
      // ---- lane c < PN: rb's instance a = rbj PN + c, its fields from the lane
      // holding it
      const int a = rbj * PN + vl;
      const int src = (a & 63) << 2;
      const int e0 = __builtin_amdgcn_ds_bpermute(src, ie0), e1 = __builtin_amdgcn_ds_bpermute(src, ie1);
      const int u0 = __builtin_amdgcn_ds_bpermute(src, iu0), u1 = __builtin_amdgcn_ds_bpermute(src, iu1);
      const int h0 = __builtin_amdgcn_ds_bpermute(src, (int)ih0), h1 = __builtin_amdgcn_ds_bpermute(src, (int)ih1);
      const int *qa = qcol + (rb_lane ? a : 0) * QS;
      const int qrb = two_level ? qa[rb] : 0;
      const int hi = vb(a >= 64);
      e = hi ? e1 : e0;
      u = hi ? u1 : u0;
      hm = (uint32_t)(hi ? h1 : h0);
      const int cand = rb_lane & vb(e >= 0) & vb(u > 0);
      // the lightest receivers hosting e, no heavier than the free level
      const uint32_t hl = cand ? hm & lightm : 0u;
      uint32_t lh = ~0u, th = 0u;
      if (__ballot(hl != 0u)) {
#pragma unroll
        for (int j = 0; j < GM; ++j) {
          const uint32_t Lj = (uint32_t)__builtin_amdgcn_readlane(lj, j);
          const uint32_t c = (hl >> j) & 1u ? Lj : ~0u;
          th = c < lh ? 1u << j : (c == lh ? th | (1u << j) : th);
          lh = c < lh ? c : lh;
        }
      }
      lm = lf < lh ? lf : lh;
      valid = cand & vb(lm != ~0u);
      const uint32_t tset = valid ? ((lf == lm ? tfm : 0u) | (lh == lm ? th : 0u)) : 0u;
      delta = imin(u, (Lrb - (int)lm) >> 1);
      // ---- cost change at each target of tset, lowest (cost, rt) kept
      auto cost_at = [&](int jt, int &qt) {
        int64_t dc = 0;
        qt = 0;
        if (two_level) {
          qt = qa[r0 + jt];
          const int m_rt = imin(delta, qt);
          const int rest = delta - m_rt;
          const int m_rb = rest - imin(rest, u - qt - qrb);
          dc = tokc * (int64_t)(m_rb - m_rt);
        }
        const int64_t rep = ((int)fdiv((uint32_t)e, p.fGP) == d) ? repI : repX;
        return ((hm >> jt) & 1u) ? dc : dc + rep;
      };
      bj = valid ? __ffs(tset) - 1 : 0;
      bc = cost_at(bj, bq);
      const uint32_t more = tset & (tset - 1u);
      if (__ballot(more != 0u)) {
        for (uint32_t t = more; t; t &= t - 1u) {
          const int jt = __ffs(t) - 1;
          int qt;
          const int64_t dc = cost_at(jt, qt);
          if (dc < bc) {
            bc = dc;
            bj = jt;
            bq = qt;
          }
        }
      }
    }
    RSECT(1);
    // ---- minimum key: (delta descending, L[rt]) first, then cost, e, rt
    const uint64_t k1 = valid ? ((uint64_t)(uint32_t)(0x7FFFFFFF - delta) << 32) | lm : ~0ull;
    uint64_t m1 = row_min_all_u64(k1);
    if (!one_row) {
      const uint64_t x1 = vlane64(m1, 16), x2 = vlane64(m1, 32), x3 = vlane64(m1, 48);
      m1 = vlane64(m1, 0);
      m1 = x1 < m1 ? x1 : m1;
      m1 = x2 < m1 ? x2 : m1;
      m1 = x3 < m1 ? x3 : m1;
    } else {
      m1 = vlane64(m1, 0);
    }
    if (m1 == ~0ull) break;
    if (it >= p.iter_limit) {
      if (lane == 0) *flags |= TOPOEP_ST_ITER;
      break;
    }
    uint64_t win = __ballot(k1 == m1);
    if (__popcll(win) != 1) {
      const bool in2 = k1 == m1;
      const uint64_t kc = in2 ? (uint64_t)bc ^ (1ull << 63) : ~0ull;
      const uint64_t m3 = wave_min_u64(kc);
      win &= __ballot(kc == m3);
      if (__popcll(win) != 1) {
        const bool in3 = ((win >> lane) & 1ull) != 0;
        const uint64_t ke = in3 ? ((uint64_t)(uint32_t)e << 32) | (uint32_t)(r0 + bj) : ~0ull;
        const uint64_t m4 = wave_min_u64(ke);
        win &= __ballot(ke == m4);
      }
    }
    const int wl = __ffsll((long long)win) - 1;
    const int dw = vlane(delta, wl);
    const int Lrt = vlane((int)lm, wl);
    const int ew = vlane(e, wl);
    const int rtj_s = __builtin_amdgcn_readlane(bj, wl);
    const int rtj = vgpr(rtj_s);
    const int rt = r0 + rtj;
    const int uw = vlane(u, wl);
    const int qrt = vlane(bq, wl);
    const uint32_t hw = (uint32_t)vlane((int)hm, wl);
    const int aw_s = rbj_s * PN + (pairs ? wl >> 4 : wl);
    const int aw = vgpr(aw_s);
    const int fresh = vb(((hw >> rtj) & 1u) == 0u);
    RSECT(2);
    // ---- rt's instance of e: the one it holds (rt's instances are rtj PN ..
    // rtj PN + PN - 1), or its first free slot
    const int base = rtj * PN;
    const uint64_t f0 = __ballot(vb(ie0 == ew) & vb((uint32_t)(vl - base) < (uint32_t)PN));
    const uint64_t f1 = __ballot(vb(ie1 == ew) & vb((uint32_t)(vl + 64 - base) < (uint32_t)PN));
    const int held = f0 ? __ffsll((long long)f0) - 1 : 64 + __ffsll((long long)f1) - 1;
    const int a2 = fresh ? base + P + vlane(uj, rtj_s) : vgpr(held);
    RSECT(3);
    // ---- the transfer of dw assignments from aw's column to a2's
    int *qw = qcol + aw_s * QS;
    int *qb = qcol + a2 * QS;
    if (R <= 64) {
      // one pass: rt's own first, the other sources ascending, rb's own last;
      // lanes >= R take the spare word after the sources (QS > R)
      const int sv = src_lane ? vl : R;
      const int av = src_lane ? qw[sv] : 0;
      int excl;
      if (two_level) {
        const int is_rt = vb(vl == rt), is_rb = vb(vl == rb);
        const int other = (is_rt | is_rb) ? 0 : av;
        const int incl = wave_incl_scan(other);
        const int tot = vlane(incl, 63);
        excl = is_rt ? 0 : (is_rb ? qrt + tot : qrt + incl - other);
      } else {
        excl = wave_incl_scan(av) - av;
      }
      int m = dw - excl;
      m = m < 0 ? 0 : (m > av ? av : m);
      qw[sv] = av - m;
      atomicAdd(&qb[sv], m);
    } else {
      int rest = dw;
      int m_rt = 0;
      if (two_level) {
        m_rt = imin(rest, qrt);
        rest -= m_rt;
      }
      for (int s0 = 0; s0 < R && rest > 0; s0 += 64) {
        const int sv = s0 + lane;
        int av = 0;
        if (sv < R && (!two_level || (sv != rt && sv != rb))) av = qw[sv];
        const int incl = wave_incl_scan(av);
        const int excl = incl - av;
        int m = rest - excl;
        m = m < 0 ? 0 : (m > av ? av : m);
        if (m) {
          qw[sv] = av - m;
          atomicAdd(&qb[sv], m);
        }
        const int total = readlane_i32(incl, 63);
        rest -= total < rest ? total : rest;
      }
      if (lane == 0) {
        if (m_rt) {
          atomicSub(&qw[rt], m_rt);
          atomicAdd(&qb[rt], m_rt);
        }
        if (rest > 0) {
          atomicSub(&qw[rb], rest);
          atomicAdd(&qb[rb], rest);
        }
      }
    }
    RSECT(4);
    // ---- registers: the two instances' loads, a new replica's expert and the
    // hosting mask of its expert, the two ranks
    const uint32_t hn = hw | (1u << rtj);
    const int at0 = vb(vl == a2), at1 = vb(vl + 64 == a2);
    iu0 = vl == aw ? uw - dw : iu0;
    iu1 = vl + 64 == aw ? uw - dw : iu1;
    iu0 = at0 ? iu0 + dw : iu0;
    iu1 = at1 ? iu1 + dw : iu1;
    ie0 = (fresh & at0) ? ew : ie0;
    ie1 = (fresh & at1) ? ew : ie1;
    ih0 = (fresh & vb(ie0 == ew)) ? hn : ih0;
    ih1 = (fresh & vb(ie1 == ew)) ? hn : ih1;
    lj = vl == rbj ? Lrb - dw : (vl == rtj ? Lrt + dw : lj);
    uj = (fresh & vb(vl == rtj)) ? uj + 1 : uj;
    RSECT(5);
  }
  RSECT_END(it);
  // final state: instances, their slots, the hosting masks, the ranks
  auto put = [&](int a, int ex, int ux, uint32_t hx) {
    if (a < I) {
      e_of[a] = ex;
      U[a] = ux;
      const int j = (int)fdiv((uint32_t)a, p.fPN), pos = a - j * PN;
      if (pos >= P) slots[j * Neff + pos - P] = ex;
      if (ex >= 0) em[ex] = (uint64_t)hx;
    }
  };
  put(vl, ie0, iu0, ih0);
  put(vl + 64, ie1, iu1, ih1);
  if (rank_lane) {
    Lr[vl] = lj;
    used[vl] = uj;
  }
  wave_sync();
  return it;
}

// Intra-node refinement of domain d (Section 4.3, Eq. 10), by one wave.
// e_of/U/qcol/slots/used/Lr point at the domain's own state; em (E words of
// 64 bits, scratch) receives, per expert, the mask of the domain's local
// ranks hosting it.  Each iteration picks the busiest rank rb (ties to the
// lowest rank), takes the best (instance of rb, other rank of the domain)
// candidate by key (delta desc, L[rt] asc, cost change asc, e asc, rt asc)
// and commits it: each lane takes an instance of rb and scores only its
// lightest receivers (the others cannot win).  Domains that fit it run the
// register form (refine_domain_reg); Form pins one form at compile time.
// The moved assignments come from sources in ascending (c(s,rt) - c(s,rb),
// s) order: with the two-level cost that is rt
// itself, then the other sources ascending, then rb (or plain ascending when
// the intra-domain cost is zero).  The loop ends when no candidate has
// delta >= 1.  Returns the number of moves committed (at once 0 when no rank
// of the domain has a free slot).  With prepared, em already holds the masks
// and the wave sums the rank loads Lr itself; otherwise Lr is given and em is
// scratch filled here.  With General (the full model of Section 4.1) the
// moved assignments come from the sources in the precomputed (c(s,rt) -
// c(s,rb), s) order of gc, and the cost change uses the cost matrix and
// ||W_e||.
template <bool General = false, int Form = kRefineAny>
__device__ uint32_t refine_domain(const Plan &p, int d, int *e_of, int *U, int *qcol, int *slots, int *used,
                                  int *Lr, uint64_t *em, uint32_t *flags, bool prepared, GenCost gc = GenCost{}) {
  static_assert(!(General && (Form == kRefineReg || Form == kRefinePairs)),
                "the register form scores the two-level cost only");
  const int lane = lane_id();
  const int G = p.G, PN = p.PN, R = p.R, P = p.P, Neff = p.Neff, QS = p.QS, E = p.E, I = p.I;
  if (G < 2) return 0;
  const int r0 = d * G;
  // At the start of refinement every expert has at most one instance in the
  // domain (stage 1 places one replica per domain and expert, never in the
  // main's own domain), so a candidate's target must have a free slot:
  // without one anywhere in the domain no candidate ever exists.
  {
    const bool free_slot = lane < G && used[lane] < Neff;
    if (__ballot(free_slot) == 0) return 0;
  }
  if (prepared) {
    // em already holds the hosting masks; the rank loads are summed here
    if (lane < G) {
      int l = 0;
      for (int pos = 0; pos < PN; ++pos) l += U[lane * PN + pos];
      Lr[lane] = l;
    }
  } else {
    // hosting masks per expert
    for (int e = lane; e < E; e += 64) em[e] = 0;
    wave_sync();
    for (int a = lane; a < I; a += 64) {
      const int e = e_of[a];
      if (e >= 0) atomicOr(reinterpret_cast<unsigned long long *>(&em[e]), 1ull << (uint32_t)fdiv((uint32_t)a, p.fPN));
    }
  }
  wave_sync();
  // (the pairs variant only where the kernel was built for it: the
  // one-launch plan's; the three-kernel solvers keep one register variant)
  if constexpr (!General && Form == kRefinePairs) {
    return G <= 8 ? refine_domain_reg<8, true>(p, d, e_of, U, qcol, slots, used, Lr, em, flags)
                  : refine_domain_reg<16, true>(p, d, e_of, U, qcol, slots, used, Lr, em, flags);
  }
  if constexpr (!General && (Form == kRefineReg || Form == kRefineAny)) {
    if (Form == kRefineReg || refine_in_registers(G, I, PN)) {
      return G <= 8 ? refine_domain_reg<8, false>(p, d, e_of, U, qcol, slots, used, Lr, em, flags)
                    : refine_domain_reg<16, false>(p, d, e_of, U, qcol, slots, used, Lr, em, flags);
    }
  }
  if constexpr (Form == kRefineReg || Form == kRefinePairs) {
    return 0;   // (not reached: the host picks the register form only where it applies)
  } else {
  // One lane per instance of rb.  Among the targets an instance may move to
  // (the domain's other ranks with L[rt] <= L[rb] - 2 that host its expert
  // or have a free slot) delta = min(u, (L[rb] - L[rt]) / 2) only grows as
  // L[rt] falls, so the instance's best keys all sit at its lightest
  // targets: the lane scores just those (usually one rank) instead of all
  // G - 1, and the wave keeps the overall minimum of the same key.
  const int rounds = (PN + 63) >> 6;
  // with at most 16 ranks the reductions over ranks stay in the first row
  // of 16 lanes
  const bool rank_row = G <= 16;
  auto min_u32 = [&](uint32_t v) { return rows_min_u32(v, rank_row); };
  const int64_t tokc = 2 * p.S * (int64_t)p.cI;   // cost change per moved assignment and unit of (m_rb - m_rt)
  const int64_t repI = (int64_t)p.cI * p.W, repX = (int64_t)p.cX * p.W;
  // lane j < G keeps rank j's load and used slots in registers (and the
  // LDS copies current for the other lanes' reads)
  int lj = 0, uj = 0;
  if (lane < G) {
    lj = Lr[lane];
    uj = used[lane];
  }
  uint32_t it = 0;
  RSECT_DECL(d);
  for (;; ++it) {
    // busiest rank, lowest index on ties
    const int Lrb = (int)~min_u32(lane < G ? ~(uint32_t)lj : ~0u);
    const int rbj = __ffsll((long long)__ballot(lane < G && lj == Lrb)) - 1;
    const int rb = r0 + rbj;
    // receivers: delta >= 1 needs L[rt] <= L[rb] - 2; those with a free slot
    // take any expert, and the lightest of them form one level (lf, tf)
    const bool low = lane < G && lane != rbj && (int64_t)Lrb - lj >= 2;
    const uint64_t lowm = __ballot(low);
    if (lowm == 0) break;
    const bool fr = low && uj < Neff;
    uint32_t lf = ~0u;
    uint64_t tf = 0;
    if (__ballot(fr)) {
      lf = min_u32(fr ? (uint32_t)lj : ~0u);
      tf = __ballot(fr && (uint32_t)lj == lf);
    }
    // the first rank of the free level: its q is read with the instance's
    // own words (it is usually the one target scored)
    const int jf = tf ? __ffsll((long long)tf) - 1 : 0;
    RSECT(0);
    uint64_t k1 = ~0ull, k2 = ~0ull, k3 = ~0ull, best_hm = 0;
    int best_a = 0, best_u = 0, best_q = 0;
    const bool two_level = !General && p.cI > 0;
    // instance a of rb (expert e, load u, q[rb] and q[r0 + jf] of its
    // column, hosting mask hmf of e) scored against its lightest receivers
    auto score = [&](int a, int e, int u, int qrb, int qf, uint64_t hmf) {
      const int *qa = qcol + a * QS;
      // the lightest receivers already hosting e (no slot needed)
      uint32_t lh = ~0u;
      uint64_t th = 0;
      for (uint64_t h = hmf & lowm; h; h &= h - 1) {
        const int j = __ffsll((long long)h) - 1;
        const uint32_t L = (uint32_t)Lr[j];
        if (L < lh) {
          lh = L;
          th = 0;
        }
        if (L == lh) th |= 1ull << j;
      }
      const uint32_t lm = lf < lh ? lf : lh;
      if (lm == ~0u) return;
      const uint64_t tset = (lf == lm ? tf : 0) | (lh == lm ? th : 0);
      const int delta = imin(u, (Lrb - (int)lm) >> 1);
      // lowest (cost change, rt) among the lightest receivers
      int64_t bc = INT64_MAX;
      int bj = 0, bq = 0;
      for (uint64_t t = tset; t; t &= t - 1) {
        const int rtj = __ffsll((long long)t) - 1;
        const bool hosts = (hmf >> rtj) & 1ull;
        const int rt = r0 + rtj;
        int64_t dcost = 0;
        int qrt = 0;
        if constexpr (General) {
          // fill delta from the sources in (c(s,rt) - c(s,rb), s) order
          const uint16_t *o = gc.ord + (rbj * G + rtj) * R;
          const int *ct = gc.ccol + rtj * R, *cb = gc.ccol + rbj * R;
          int rest = delta;
          int64_t dt = 0;
          for (int k = 0; k < R && rest > 0; ++k) {
            const int s2 = o[k];
            const int take = imin(rest, qa[s2]);
            dt += (int64_t)take * (ct[s2] - cb[s2]);
            rest -= take;
          }
          dcost = 2 * p.S * dt;
          if (!hosts) dcost += (int64_t)gc.ccol[rtj * R + (int)fdiv((uint32_t)e, p.fP)] * gc.wx[e];
        } else {
          if (p.cI > 0) {
            qrt = rtj == jf ? qf : qa[rt];
            const int m_rt = imin(delta, qrt);
            const int rest = delta - m_rt;
            const int m_rb = rest - imin(rest, u - qrt - qrb);
            dcost = tokc * (int64_t)(m_rb - m_rt);
          }
          if (!hosts) dcost += ((int)fdiv((uint32_t)e, p.fGP) == d) ? repI : repX;
        }
        if (dcost < bc) {
          bc = dcost;
          bj = rtj;
          bq = qrt;
        }
      }
      const uint64_t c1 = ((uint64_t)(uint32_t)(0x7FFFFFFF - delta) << 32) | lm;
      const uint64_t c2 = (uint64_t)bc ^ (1ull << 63);
      const uint64_t c3 = ((uint64_t)(uint32_t)e << 32) | (uint32_t)(r0 + bj);
      // (c1, c2, c3) < (k1, k2, k3), with no branches
      const bool lt = (c1 < k1) | ((c1 == k1) & ((c2 < k2) | ((c2 == k2) & (c3 < k3))));
      k1 = lt ? c1 : k1;
      k2 = lt ? c2 : k2;
      k3 = lt ? c3 : k3;
      best_a = lt ? a : best_a;
      best_u = lt ? u : best_u;
      best_hm = lt ? hmf : best_hm;
      best_q = lt ? bq : best_q;
    };
    // one lane per instance, two instances (rounds of 64) at a time: the
    // pair's words and hosting masks are read before either is scored, so
    // their LDS round trips overlap (a lane's instances hold distinct
    // experts, so the order it scores them in does not matter)
    for (int rd = 0; rd < rounds; rd += 2) {
      const int ai0 = lane + rd * 64, ai1 = ai0 + 64;
      const bool v0 = ai0 < PN, v1 = ai1 < PN;
      const int a0 = rbj * PN + (v0 ? ai0 : 0), a1 = rbj * PN + (v1 ? ai1 : 0);
      const int *qa0 = qcol + a0 * QS, *qa1 = qcol + a1 * QS;
      const int e0 = v0 ? e_of[a0] : -1, e1 = v1 ? e_of[a1] : -1;
      const int u0 = v0 ? U[a0] : 0, u1 = v1 ? U[a1] : 0;
      const int qrb0 = two_level ? qa0[rb] : 0, qf0 = two_level ? qa0[r0 + jf] : 0;
      const int qrb1 = two_level && v1 ? qa1[rb] : 0, qf1 = two_level && v1 ? qa1[r0 + jf] : 0;
      const uint64_t hm0 = e0 >= 0 ? em[e0] : 0, hm1 = e1 >= 0 ? em[e1] : 0;
      if (e0 >= 0 && u0 > 0) score(a0, e0, u0, qrb0, qf0, hm0);
      if (e1 >= 0 && u1 > 0) score(a1, e1, u1, qrb1, qf1, hm1);
    }
    RSECT(1);
    const uint64_t m1 = wave_min_u64(k1);
    if (m1 == ~0ull) break;
    // a move is still available after iter_limit of them: stop with ITER
    if (it >= p.iter_limit) {
      if (lane == 0) *flags |= TOPOEP_ST_ITER;
      break;
    }
    uint64_t win = __ballot(k1 == m1);
    if (__popcll(win) != 1) {
      const uint64_t m2 = wave_min_u64(k1 == m1 ? k2 : ~0ull);
      win &= __ballot(k2 == m2);
      if (__popcll(win) != 1) {
        const uint64_t m3 = wave_min_u64((k1 == m1 && k2 == m2) ? k3 : ~0ull);
        win &= __ballot(k3 == m3);
      }
    }
    const int wl = __ffsll((long long)win) - 1;
    const uint64_t kw1 = readlane64(k1, wl);
    const int delta = 0x7FFFFFFF - (int)(kw1 >> 32);
    const int Lrt = (int)(uint32_t)kw1;
    const uint64_t kw = readlane64(k3, wl);
    const int e = (int)(kw >> 32);
    const int rt = (int)(uint32_t)kw;
    const int rtj = rt - r0;
    const int a = readlane_i32(best_a, wl);
    const int ua = readlane_i32(best_u, wl);
    const int qrt = readlane_i32(best_q, wl);
    const bool hosts = (readlane64(best_hm, wl) >> rtj) & 1ull;
    RSECT(2);
    // rt's instance of e: its main expert, the replica slot holding it, or a
    // new replica in rt's first free slot
    int a2 = -1;
    bool fresh = false;
    if (!hosts) {
      a2 = rtj * PN + P + readlane_i32(uj, rtj);
      fresh = true;
    } else if ((int)fdiv((uint32_t)e, p.fP) == rt) {
      a2 = rtj * PN + (e - rt * P);
    } else {
      const int ut = readlane_i32(uj, rtj);
      for (int t0 = 0; t0 < ut && a2 < 0; t0 += 64) {
        const uint64_t hit = __ballot(t0 + lane < ut && slots[rtj * Neff + t0 + lane] == e);
        if (hit) a2 = rtj * PN + P + t0 + __ffsll((long long)hit) - 1;
      }
    }
    RSECT(3);
    int *qa = qcol + a * QS;
    int *qb = qcol + a2 * QS;
    int rest = delta;
    int m_rt = 0;
    if constexpr (General) {
      // the sources in the pair's order, 64 at a time
      const uint16_t *o = gc.ord + (rbj * G + rtj) * R;
      for (int k0 = 0; k0 < R && rest > 0; k0 += 64) {
        const int k = k0 + lane;
        const int s = k < R ? o[k] : 0;
        const int av = k < R ? qa[s] : 0;
        const int incl = wave_incl_scan(av);
        const int excl = incl - av;
        int m = rest - excl;
        m = m < 0 ? 0 : (m > av ? av : m);
        if (m) {
          qa[s] = av - m;
          atomicAdd(&qb[s], m);
        }
        const int total = readlane_i32(incl, 63);
        rest -= total < rest ? total : rest;
      }
    } else {
      // rt's own assignments first, then the other sources ascending (rb's
      // own are taken last, below)
      if (p.cI > 0) {
        m_rt = imin(rest, qrt);
        rest -= m_rt;
      }
      for (int s0 = 0; s0 < R && rest > 0; s0 += 64) {
        const int s = s0 + lane;
        int av = 0;
        if (s < R && (p.cI == 0 || (s != rt && s != rb))) av = qa[s];
        const int incl = wave_incl_scan(av);
        const int excl = incl - av;
        int m = rest - excl;
        m = m < 0 ? 0 : (m > av ? av : m);
        if (m) {
          qa[s] = av - m;
          atomicAdd(&qb[s], m);
        }
        const int total = readlane_i32(incl, 63);
        rest -= total < rest ? total : rest;
      }
    }
    RSECT(4);
    // (the sources above exclude rt and rb, so these words are disjoint
    // from the lanes' updates; LDS atomics without return need no wait)
    if (lane == 0) {
      if (fresh) {
        slots[rtj * Neff + (a2 - rtj * PN - P)] = e;
        used[rtj] = a2 - rtj * PN - P + 1;
        e_of[a2] = e;
        atomicOr(reinterpret_cast<unsigned long long *>(&em[e]), 1ull << rtj);
      }
      if (m_rt) {
        atomicSub(&qa[rt], m_rt);
        atomicAdd(&qb[rt], m_rt);
      }
      if (rest > 0) {   // the rest comes from rb itself (two-level cost, taken last)
        atomicSub(&qa[rb], rest);
        atomicAdd(&qb[rb], rest);
      }
      U[a] = ua - delta;
      atomicAdd(&U[a2], delta);
      Lr[rbj] = Lrb - delta;
      Lr[rtj] = Lrt + delta;
    }
    if (lane == rbj) lj = Lrb - delta;
    if (lane == rtj) {
      lj = Lrt + delta;
      uj += fresh ? 1 : 0;
    }
    wave_sync();
    RSECT(5);
  }
  RSECT_END(it);
  return it;   // one move per completed iteration
  }
}

// Stage-1 candidate key: (D descending, e ascending) as one unsigned
// 64-bit value, smaller first.  This is the order of the benefit
// b = 2 D S - W descending (S > 0), ties to the lower expert id.
__device__ inline uint64_t cand_key(int D, int e) {
  return ((uint64_t)(uint32_t)(0x7FFFFFFF - D) << 32) | (uint32_t)e;
}

// Rank of candidate c among the nc keys of its domain (keys are distinct);
// the first cap ranks name the domain's stage-1 replicas.
__device__ inline void rank_candidates(int c, int nc, int cap, const uint64_t *keys, int *out) {
  const uint64_t kc = keys[c];
  int rank = 0;
  int c2 = 0;
  for (; c2 + 8 <= nc; c2 += 8) {
    uint64_t k[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) k[u] = keys[c2 + u];
#pragma unroll
    for (int u = 0; u < 8; ++u) rank += k[u] < kc;
  }
  for (; c2 < nc; ++c2) rank += keys[c2] < kc;
  if (rank < cap) out[rank] = (int)(uint32_t)kc;
}

// Rank of candidate c by (benefit b descending, expert ascending) among nc
// candidates with benefits bs[] and experts es[] (the general model, where
// ||W_e|| differs per expert so b does not follow D); the first cap ranks
// name the domain's stage-1 replicas.
__device__ inline void rank_candidates_b(int c, int nc, int cap, const uint64_t *bs, const int *es, int *out) {
  const uint64_t bc = bs[c];
  const int ec = es[c];
  int rank = 0;
  for (int c2 = 0; c2 < nc; ++c2) {
    const uint64_t b2 = bs[c2];
    rank += b2 > bc || (b2 == bc && es[c2] < ec);
  }
  if (rank < cap) out[rank] = ec;
}

// Stage 1 (Eq. 9) candidates of domain d, by one wave: the experts whose
// main is outside d with benefit b = 2 D S - W > 0 (D from om, Omega with
// row self already the histogram when dom(self) = d), compacted with ballots
// into keys ck_d; returns their count on every lane.
__device__ int stage1_candidates_wave(const Plan &p, int d, const int *om, uint64_t *ck_d) {
  const int lane = lane_id(), E = p.E, G = p.G;
  int nc = 0;
  for (int e0 = 0; e0 < E; e0 += 64) {
    const int e = e0 + lane;
    bool cand = false;
    uint64_t key = 0;
    if (e < E && (int)fdiv((uint32_t)e, p.fGP) != d) {
      int D = 0;
#pragma unroll 8
      for (int j = 0; j < G; ++j) D += om[(d * G + j) * E + e];
      cand = (int64_t)2 * D * p.S > p.W;
      key = cand_key(D, e);
    }
    const uint64_t m = __ballot(cand);
    if (cand) ck_d[nc + __popcll(m & lanemask_lt())] = key;
    nc += __popcll(m);
  }
  wave_sync();
  return nc;
}

// Stage 1 of domain d by one wave: candidates, then each ranked by key; the
// first cap ranks fill repl_d (pre-filled with -1) and ccnt[d] = the count.
__device__ void stage1_domain_wave(const Plan &p, int d, const int *om, uint64_t *ck_d, int *ccnt, int *repl_d) {
  const int nc = stage1_candidates_wave(p, d, om, ck_d);
  if (d == 0) STAMP(p, 22);
  for (int c = lane_id(); c < nc; c += 64) rank_candidates(c, nc, p.cap1, ck_d, repl_d);
  if (lane_id() == 0) ccnt[d] = nc;
}


// Stage 1 (Eq. 9) of every domain by the whole workgroup.  Item (d, e):
// D[d][e] summed over the domain's rows of Omega; an expert whose main lies
// outside d with b = 2 D S - W > 0 is a candidate and takes a slot of
// ck + d E16 (E16 = E rounded up to 16; the keys were set to ~0, which sorts
// after every candidate) from the domain's LDS counter ccnt[d] (the slots'
// order is arbitrary).  Each candidate's rank among its domain's candidates
// by key (D descending, e ascending; keys are distinct) is then counted in
// parts of 16 keys: the workgroup's threads are split into one block per
// domain (whole waves; one domain after another when there are more domains
// than waves), a block's items being (candidate c, part h) with Hp parts
// per candidate (ceil(nc / 16) rounded up to a power of two).  rk[d E + c]
// = the rank of the domain's candidate in slot c.  The ranks below cap1
// name the domain's stage-1 replicas.  rk: M E words.
__device__ __forceinline__ void stage1_ranks(const Plan &p, const int *om, uint64_t *ck, int *ccnt, int *rk) {
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E, G = p.G, M = p.M, E16 = (E + 15) & ~15;
  // item idx = d E + e, walked with (d, e) kept as the index advances
  const int dstep = (int)fdiv((uint32_t)nt, p.fE), estep = nt - dstep * E;
  int d = (int)fdiv((uint32_t)tid, p.fE), e = tid - d * E;
  for (int idx = tid; idx < M * E; idx += nt, d += dstep, e += estep) {
    if (e >= E) {
      e -= E;
      ++d;
    }
    rk[idx] = 0;
    if ((int)fdiv((uint32_t)e, p.fGP) == d) continue;   // main inside the domain
    const int *col = om + d * G * E + e;
    int D = 0;
#pragma unroll 8
    for (int j = 0; j < G; ++j) D += col[j * E];
    if ((int64_t)2 * D * p.S > p.W) {
      const int pos = atomicAdd(&ccnt[d], 1);
      ck[d * E16 + pos] = cand_key(D, e);
    }
  }
  lds_barrier();
  STAMP(p, 24);
  const int nw = nt >> 6;
  const int wpd = M <= nw ? nw / M : 0;
  const int d0 = wpd ? (tid >> 6) / wpd : 0;
  const int tpd = wpd ? wpd * 64 : nt;
  const int lt = wpd ? tid - d0 * tpd : tid;
  for (d = d0; d < (wpd ? imin(d0 + 1, M) : M); ++d) {
    const int nc = uniform_i32(ccnt[d]);   // (d is the same in the whole wave)
    const int parts = (nc + 15) >> 4;
    const int lh = parts <= 1 ? 0 : 32 - __clz(parts - 1);
    const uint64_t *kd = ck + d * E16;
    for (int v = lt; v < (nc << lh); v += tpd) {
      const int c = v >> lh, h = v & ((1 << lh) - 1);
      if (16 * h >= nc) continue;
      const uint64_t kc = kd[c];
      const uint64_t *kp = kd + 16 * h;
      uint64_t k[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) k[i] = kp[i];
      int below = 0;
#pragma unroll
      for (int i = 0; i < 16; ++i) below += k[i] < kc ? 1 : 0;
      if (below) atomicAdd(&rk[d * E + c], below);
    }
  }
  lds_barrier();
  STAMP(p, 26);
}

// The stage-1 replica lists from the ranks: repl[d cap1 + rank] = e for the
// ranks below cap1 (repl holds -1 elsewhere).  Ends with a barrier.
__device__ __forceinline__ void stage1_lists(const Plan &p, const uint64_t *ck, const int *ccnt, const int *rk,
                                             int *repl) {
  for (int idx = threadIdx.x; idx < p.M * p.E; idx += blockDim.x) {
    const int d = (int)fdiv((uint32_t)idx, p.fE), c = idx - d * p.E;
    if (c < ccnt[d] && rk[idx] < p.cap1) repl[d * p.cap1 + rk[idx]] = (int)(uint32_t)ck[d * ((p.E + 15) & ~15) + c];
  }
  lds_barrier();
}

// This rank's per-expert instance list: bm[e * RW ...] marks the ranks
// whose instance of e has a nonzero share q[self][e][r].  Thread t takes
// experts [t * K, (t + 1) * K), K = ceil(E / blockDim): it counts their
// ranks; a wave scan plus the totals of the waves before (one barrier) give
// each expert's first entry; then it walks the ranks in ascending order
// writing (rank, cumulative share).  qcol and e_of address instance (d, a)
// as d * I + a; slots/used are every rank's; tmp holds blockDim / 64 words.
__device__ void emit_instance_list(const Plan &p, const int *qcol, const int *slots, const int *used,
                                   const uint32_t *bm, int *tmp) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int E = p.E, RW = p.RW, K = (E + nt - 1) / nt;
  const int e0 = imin(E, tid * K), e1 = imin(E, e0 + K);
  int cnt = 0;
  for (int e = e0; e < e1; ++e)
    for (int w = 0; w < RW; ++w) cnt += __popc(bm[e * RW + w]);
  const int incl = wave_incl_scan(cnt);
  if (lane == 63) tmp[wave] = incl;
  __syncthreads();
  int pos = incl - cnt;
  for (int w = 0; w < wave; ++w) pos += tmp[w];
  if (tid == nt - 1) p.csr_ptr[E] = pos + cnt;
  for (int e = e0; e < e1; ++e) {
    p.csr_ptr[e] = pos;
    int run = 0;
    for (int w = 0; w < RW; ++w) {
      uint32_t bits = bm[e * RW + w];
      while (bits) {
        const int r = w * 32 + __ffs(bits) - 1;
        bits &= bits - 1u;
        const int d = (int)fdiv((uint32_t)r, p.fG), j = r - d * p.G;
        const int a = instance_of(p, d, j, e, slots + d * p.G * p.Neff, used + d * p.G);
        if (a >= 0) run += qcol[(d * p.I + a) * p.QS + p.self];   // a >= 0: bm marks hosts only
        p.csr_r[pos] = r;
        p.csr_end[pos] = run;
        ++pos;
      }
    }
  }
}

// Status bits and the sum of positive loads of Omega' (row self replaced by
// the histogram hs) over rows [r0, r1) held at rows[(s - r0) * E + e];
// wave-reduced, then one LDS atomic per wave into misc[0] (bits) and
// misc[8..9] (total).  Called by every thread of the workgroup.
__device__ void scan_rows(const Plan &p, int r0, int r1, const int *rows, const int *hs, int *misc) {
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E;
  bool neg = false, diff = false;
  uint64_t tot = 0;
  const int n = (r1 - r0) * E;
  for (int i = tid; i < n; i += nt) {
    const int g = rows[i];
    neg |= g < 0;
    if (g > 0) tot += (uint64_t)g;
  }
  if (p.self >= r0 && p.self < r1) {
    // row self: the plan uses the histogram instead of the gathered row
    for (int e = tid; e < E; e += nt) {
      const int g = rows[(p.self - r0) * E + e];
      if (g > 0) tot -= (uint64_t)g;
      if (hs[e] > 0) tot += (uint64_t)hs[e];
      diff |= g != hs[e];
    }
  }
  tot = wave_sum_u64(tot);
  const uint64_t any_neg = __ballot(neg);
  const uint64_t any_diff = __ballot(diff);
  if (lane_id() == 0) {
    const uint32_t w = (any_neg ? TOPOEP_ST_NEG_LOAD : 0u) | (any_diff ? TOPOEP_ST_SELF_DIFF : 0u);
    if (w) atomicOr(reinterpret_cast<unsigned *>(&misc[0]), w);
    if (tot) atomicAdd(reinterpret_cast<unsigned long long *>(misc + 8), (unsigned long long)tot);
  }
}

// ---------------------------------------------------------------- general cost model

// The full model of Section 4.1 on the device: whether the cost matrix is a
// cost (symmetric, nonnegative, zero diagonal) and every size nonnegative,
// and the largest entry and size for the exact-range bound.  misc[16..23]
// are scratch; returns the COST bit or 0 (the same on every thread).
__device__ uint32_t general_check(const Plan &p, int *misc, uint64_t *cmax, uint64_t *wmax) {
  const int tid = threadIdx.x, nt = blockDim.x, R = p.R;
  if (tid < 8) misc[16 + tid] = 0;
  lds_barrier();
  bool bad = false;
  uint32_t cm = 0;
  uint64_t wm = 0;
  if (p.Cm) {
    for (int i = tid; i < R * R; i += nt) {
      const int s = i / R, r = i - s * R;
      const int c = p.Cm[i];
      bad |= c < 0 || (s == r && c != 0) || c != p.Cm[(int64_t)r * R + s];
      if (c > 0 && (uint32_t)c > cm) cm = (uint32_t)c;
    }
  } else {
    cm = (uint32_t)imax(p.cI, p.cX);
  }
  if (p.We) {
    for (int e = tid; e < p.E; e += nt) {
      const int64_t w = p.We[e];
      bad |= w < 0;
      if (w > 0 && (uint64_t)w > wm) wm = (uint64_t)w;
    }
  } else {
    wm = (uint64_t)p.W;
  }
  if (bad) misc[16] = 1;
  atomicMax(reinterpret_cast<unsigned *>(&misc[17]), cm);
  atomicMax(reinterpret_cast<unsigned long long *>(misc + 18), (unsigned long long)wm);
  lds_barrier();
  *cmax = (uint32_t)misc[17];
  *wmax = *reinterpret_cast<const unsigned long long *>(misc + 18);
  const uint32_t st = misc[16] ? TOPOEP_ST_COST : 0u;
  lds_barrier();
  return st;
}

// Cost tables of domain d for its refinement: ccol[j][s] = c(s, dG + j),
// ||W_e|| and, per ordered pair (jb, jt) of the domain's ranks, the sources
// in ascending (c(s,rt) - c(s,rb), s) order.
__device__ GenCost general_tables(const Plan &p, int d, int *sm, const DomainLds &lay) {
  const int tid = threadIdx.x, nt = blockDim.x, R = p.R, G = p.G;
  uint16_t *ord = reinterpret_cast<uint16_t *>(sm + lay.ord);
  int *ccol = sm + lay.ccol;
  int64_t *wx = reinterpret_cast<int64_t *>(sm + lay.wx);
  for (int i = tid; i < G * R; i += nt) {
    const int j = i / R, s = i - j * R, r = d * G + j;
    ccol[i] = p.Cm ? p.Cm[(int64_t)s * R + r] : (s == r ? 0 : (s / G == r / G ? p.cI : p.cX));
  }
  for (int e = tid; e < p.E; e += nt) wx[e] = p.We ? p.We[e] : p.W;
  lds_barrier();
  for (int x = tid; x < G * G * R; x += nt) {
    const int pair = x / R, s = x - pair * R, jb = pair / G, jt = pair - jb * G;
    if (jb == jt) continue;
    const int *cb = ccol + jb * R, *ct = ccol + jt * R;
    const int ds = ct[s] - cb[s];
    int rank = 0;
    for (int s2 = 0; s2 < R; ++s2) {
      const int d2 = ct[s2] - cb[s2];
      rank += d2 < ds || (d2 == ds && s2 < s);
    }
    ord[pair * R + rank] = (uint16_t)s;
  }
  lds_barrier();
  GenCost gc;
  gc.ord = ord;
  gc.ccol = ccol;
  gc.wx = wx;
  return gc;
}

// ---------------------------------------------------------------- solver: one workgroup per domain
//
// Workgroups 0 .. n_solvers-1 each take the domains d = wg, wg + n_solvers,
// ...; the n_helpers after them compute the histogram blocks' offsets for
// the reroute and each expert's total (row self of Omega).  Per domain:
// stage 1 (Eq. 9) from the domain's rows of Omega, then a bounded grid
// barrier publishes every domain's replicas; the hosting masks, the
// domain's instances, routing (Section 4.3), refinement (Eq. 10) and the
// domain's outputs follow.  The last solver workgroup to finish (a ticket)
// lists this rank's instances per expert for the reroute and writes the
// final status.  NT: the most threads per workgroup (launch bounds): the
// usual 512-thread launch gets twice the registers a 1024-thread one may use.
template <int NT>
__global__ __launch_bounds__(NT) void solve_kernel(Plan p0) {
  extern __shared__ int64_t smem_s[];
  int *sm = reinterpret_cast<int *>(smem_s);
  if ((int)blockIdx.x >= p0.n_solvers) {
    block_offsets(p0, blockIdx.x - p0.n_solvers, sm, true);
    return;
  }
  const Plan p = solver_plan(p0);
  DomainLds lay = domain_lds(p);
  int *offs[] = {&lay.ck, &lay.fdt, &lay.hs, &lay.rows, &lay.mask, &lay.slots, &lay.used, &lay.L,
                 &lay.e_of, &lay.U, &lay.misc, &lay.qcol, &lay.ord, &lay.ccol, &lay.wx};
  for (int *o : offs) *o = vgpr(*o);
  uint64_t *ck = reinterpret_cast<uint64_t *>(sm + lay.ck);
  FastDiv *fdt = reinterpret_cast<FastDiv *>(sm + lay.fdt);
  int *hs = sm + lay.hs;
  int *rows = sm + lay.rows;
  uint32_t *mask = reinterpret_cast<uint32_t *>(sm + lay.mask);
  int *slots = sm + lay.slots;
  int *used = sm + lay.used;
  int *Lr = sm + lay.L;
  int *e_of = sm + lay.e_of;
  int *U = sm + lay.U;
  int *misc = sm + lay.misc;
  int *qcol = sm + lay.qcol;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int wg = blockIdx.x, nwg = p.n_solvers;
  const int E = p.E, G = p.G, R = p.R, M = p.M, I = p.I, P = p.P, PN = p.PN, Neff = p.Neff;
  const int cap = p.cap1;

  if (wg == 0) STAMP(p, 0);
  if (tid < 16) misc[tid] = 0;
  build_divisors(M, fdt);
  uint64_t cmax = (uint64_t)imax(p.cI, p.cX), wmax = (uint64_t)p.W;
  if (p.general) {
    const uint32_t cst = general_check(p, misc, &cmax, &wmax);
    if (tid == 0 && cst) atomicOr(reinterpret_cast<unsigned *>(&misc[0]), cst);
  }
  // ---- row self of Omega: the histogram of local_topk, from the offset
  // helpers; the workgroup of the domain holding self needs it for its
  // stage 1 (it waits once its rows of Omega are loaded), the others only
  // after the grid barrier (by then the helpers are done)
  const int dself = (int)fdiv((uint32_t)p.self, p.fG);
  const bool has_self = dself < M && dself % nwg == wg;
  if (wg == 0)
    for (int b = tid; b < p.nb; b += nt)
      if (p.blk_err[b]) atomicOr(reinterpret_cast<unsigned *>(&misc[0]), TOPOEP_ST_BAD_ID);

  // ---- inter-node placement (Eq. 9), each domain independently
  for (int d = wg; d < M; d += nwg) {
    const Plan p = solver_plan(role_plan(p0));   // (reloaded: see the domain loop below)
    copy_to_lds(rows, p.gl + (int64_t)d * G * E, G * E);
    if (wg == 0) STAMP(p, 14);
    if (d == dself) row_self(p, hs, qcol, &misc[10]);
    if (wg == 0) STAMP(p, 15);
    if (tid == 0) misc[1] = 0;
    lds_barrier();
    scan_rows(p, d * G, (d + 1) * G, rows, hs, misc);
    for (int e = tid; e < E; e += nt) {
      if ((int)fdiv((uint32_t)e, p.fGP) == d) continue;   // main inside the domain
      int D = 0;
#pragma unroll 8
      for (int j = 0; j < G; ++j) {
        const int s = d * G + j;
        D += s == p.self ? hs[e] : rows[j * E + e];
      }
      const int64_t we = p.general && p.We ? p.We[e] : p.W;
      if ((int64_t)2 * D * p.S > we) {
        const int pos = atomicAdd(&misc[1], 1);
        if (p.general) {
          // sizes differ per expert: rank by the benefit itself (qcol is
          // free until the routing and holds the experts)
          ck[pos] = (uint64_t)((int64_t)2 * D * p.S - we);
          qcol[pos] = e;
        } else {
          ck[pos] = cand_key(D, e);
        }
      }
    }
    lds_barrier();
    if (wg == 0) STAMP(p, 16);
    const int nc = misc[1];
    if (wg == 0 && tid == 0) stamp_nc(nc);
    for (int c = tid; c < nc; c += nt) {
      if (p.general) rank_candidates_b(c, nc, cap, ck, qcol, p.repl1 + (int64_t)d * cap);
      else rank_candidates(c, nc, cap, ck, p.repl1 + (int64_t)d * cap);
    }
    for (int i = imin(nc, cap) + tid; i < cap; i += nt) p.repl1[(int64_t)d * cap + i] = -1;
    lds_barrier();
  }
  if (tid == 0) {
    if (misc[0]) atomicOr(&p.ctrl[kCtrlStatus], (uint32_t)misc[0]);
    const unsigned long long t = *reinterpret_cast<unsigned long long *>(misc + 8);
    if (t) atomicAdd(reinterpret_cast<unsigned long long *>(p.ctrl + kCtrlTotal), t);
  }

  // ---- every domain's replicas are needed by every routing construction
  if (wg == 0) STAMP(p, 1);
  const bool synced = grid_barrier(&p.ctrl[kCtrlBar], (uint32_t)nwg, p.spin_limit, &misc[2]);
  if (wg == 0) STAMP(p, 2);
  uint32_t gst = __hip_atomic_load(&p.ctrl[kCtrlStatus], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t total = __hip_atomic_load(reinterpret_cast<unsigned long long *>(p.ctrl + kCtrlTotal),
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (out_of_range_cw(p, total, cmax, wmax)) gst |= TOPOEP_ST_RANGE;
  if (!synced) gst |= TOPOEP_ST_SYNC;
  const bool noplan = (gst & kNoPlan) != 0 || !synced;

  if (!has_self && !noplan) row_self(p, hs, qcol, &misc[10]);

  // ---- domains hosting each expert: the main's domain plus stage-1 replicas
  const bool one_domain = M <= nwg;
  if (!noplan) {
    for (int i = tid; i < E * p.MW; i += nt) mask[i] = 0;
    __syncthreads();
    for (int e = tid; e < E; e += nt) {
      const int dm = (int)fdiv((uint32_t)e, p.fGP);
      atomicOr(&mask[e * p.MW + (dm >> 5)], 1u << (dm & 31));
    }
    for (int i = tid; i < M * cap; i += nt) {
      const int e = p.repl1[i];
      const int dd = (int)fdiv((uint32_t)i, p.fCap);
      // a workgroup of one domain keeps that domain's list (rows is free
      // after stage 1: cap = G Neff <= G E words)
      if (one_domain && dd == wg) rows[i - dd * cap] = e;
      if ((unsigned)e < (unsigned)E) atomicOr(&mask[e * p.MW + (dd >> 5)], 1u << (dd & 31));
    }
  }
  __syncthreads();
  if (wg == 0) STAMP(p, 3);

  uint32_t flags = 0;
  for (int d = wg; d < M; d += nwg) {
    // the plan's fields load again in every iteration (see role_plan): the
    // loop usually runs once, and invariants hoisted out of it would only
    // crowd the scalar registers
    const Plan p = solver_plan(role_plan(p0));
    if (noplan) {
      for (int i = tid; i < G * p.N; i += nt) p.slots_out[(int64_t)d * G * p.N + i] = -1;
      for (int j = tid; j < G; j += nt) p.send_out[d * G + j] = 0;
      if (p.recv_out && d == (int)fdiv((uint32_t)p.self, p.fG))
        for (int r = tid; r < R; r += nt) p.recv_out[r] = 0;
      for (int a = tid; a < I; a += nt) {
        p.seg_e[(int64_t)d * I + a] = -1;
        p.seg_q[(int64_t)d * I + a] = 0;
      }
      continue;
    }
    // stage-1 slots of the domain's ranks: candidate i sits on local rank
    // i mod G, slot i / G; the chosen ones are a prefix of the list, in
    // rows (kept there by the mask loop when the workgroup holds one domain)
    int *sel = rows;
    if (!one_domain) {
      for (int c = tid; c < cap; c += nt) sel[c] = p.repl1[(int64_t)d * cap + c];
      lds_barrier();
    }
    if (tid < 64) {
      // the chosen ones: the prefix before the first empty entry
      int nsel = cap;
      for (int c0 = 0; c0 < cap; c0 += 64) {
        const int c = c0 + tid;
        const uint64_t m = __ballot(c < cap && (unsigned)sel[c] >= (unsigned)E);
        if (m) {
          nsel = c0 + __ffsll((long long)m) - 1;
          break;
        }
      }
      if (tid == 0) misc[3] = nsel;
    }
    lds_barrier();
    const int nsel = misc[3];
    for (int j = tid; j < G; j += nt) {
      const int u = nsel > j ? (int)fdiv((uint32_t)(nsel - j + G - 1), p.fG) : 0;
      used[j] = u;
      for (int t = 0; t < Neff; ++t) slots[j * Neff + t] = t < u ? sel[t * G + j] : -1;
    }
    lds_barrier();
    for (int a = tid; a < I; a += nt) {
      const int j = (int)fdiv((uint32_t)a, p.fPN), pos = a - j * PN;
      int e;
      if (pos < P) e = (d * G + j) * P + pos;
      else e = (pos - P) < used[j] ? slots[j * Neff + pos - P] : -1;
      e_of[a] = e;
      U[a] = 0;
    }
    lds_barrier();
    if (wg == 0) STAMP(p, 4);
    // whether the domain can refine at all (a rank with a free slot); if not,
    // only the q[self] column is needed, else the columns omega[s][e] of the
    // domain's instances, then q in place
    if (tid < 64) {
      const bool fr = __ballot(tid < G && used[tid] < Neff) != 0;   // G <= 64
      if (tid == 0) misc[5] = fr ? 1 : 0;
    }
    lds_barrier();
    const bool full = misc[5] != 0;
    if (full) {
      for (int t = tid; t < I * R; t += nt) {
        const int s = (int)fdiv((uint32_t)t, p.fI), a = t - s * I;
        const int e = e_of[a];
        qcol[a * p.QS + s] = e < 0 ? 0 : (s == p.self ? hs[e] : p.gl[(int64_t)s * E + e]);
      }
    } else {
      for (int a = tid; a < I; a += nt) {
        const int e = e_of[a];
        qcol[a * p.QS + p.self] = e < 0 ? 0 : hs[e];
      }
    }
    lds_barrier();
    if (wg == 0) STAMP(p, 5);
    route_instances(
        p, I, p.fI, p.rchunks_dom, e_of, mask, fdt, qcol, U, [&](int i, int) { return qcol + i * p.QS; }, 1,
        [&](int) { return d; }, [&](int) { return full; }, [](int, int, int, int) {});
    lds_barrier();
    for (int j = tid; j < G; j += nt) {
      int l = 0;
      for (int pos = 0; pos < PN; ++pos) l += U[j * PN + pos];
      Lr[j] = l;
    }
    lds_barrier();
    if (wg == 0) STAMP(p, 6);
    if (p.general && full) {
      const GenCost gc = general_tables(p, d, sm, lay);
      if (tid < 64) {
        const uint32_t mv = refine_domain<true>(p, d, e_of, U, qcol, slots, used, Lr, ck, &flags, false, gc);
        if (tid == 0 && mv) atomicAdd(&p.ctrl[kCtrlMoves], mv);
      }
    } else if (tid < 64) {
      const uint32_t mv = refine_domain(p, d, e_of, U, qcol, slots, used, Lr, ck, &flags, false);
      if (tid == 0 && mv) atomicAdd(&p.ctrl[kCtrlMoves], mv);
    }
    lds_barrier();
    if (wg == 0) STAMP(p, 7);
    // outputs of the domain's ranks
    for (int i = tid; i < G * p.N; i += nt) {
      const int j = (int)fdiv((uint32_t)i, p.fN), t = i - j * p.N;
      p.slots_out[(int64_t)(d * G + j) * p.N + t] = (t < used[j]) ? slots[j * Neff + t] : -1;
    }
    for (int j = tid; j < G; j += nt) {
      int sc = 0;
      for (int pos = 0; pos < PN; ++pos) sc += qcol[(j * PN + pos) * p.QS + p.self];
      p.send_out[d * G + j] = sc;
    }
    for (int a = tid; a < I; a += nt) {
      p.seg_e[(int64_t)d * I + a] = e_of[a];
      p.seg_q[(int64_t)d * I + a] = e_of[a] >= 0 ? qcol[a * p.QS + p.self] : 0;
    }
    if (p.recv_out && d == (int)fdiv((uint32_t)p.self, p.fG))
      write_recv_counts(p, (p.self - d * G) * PN, e_of, qcol, full, mask, fdt,
                        [&](int s, int e) { return s == p.self ? hs[e] : p.gl[(int64_t)s * E + e]; },
                        reinterpret_cast<int *>(ck));
    lds_barrier();
  }
  if (tid == 0 && (flags || !synced)) atomicOr(&p.ctrl[kCtrlStatus], flags | (synced ? 0u : TOPOEP_ST_SYNC));

  // ---- the last workgroup to finish lists this rank's instances per expert
  if (wg == 0) STAMP(p, 8);
  drain_then_barrier();
  if (wg == 0) STAMP(p, 9);
  if (wg == 0) STAMP_FLUSH(p, 0, 10);
  if (wg == 0) STAMP_FLUSH(p, 14, 18);
  if (tid == 0) {
    const uint32_t t = __hip_atomic_fetch_add(&p.ctrl[kCtrlTicket], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    misc[4] = t == (uint32_t)nwg - 1;
  }
  __syncthreads();
  if (!misc[4]) return;
  STAMP(p, 10);
  int *cnt = qcol;                                            // E + 1
  uint32_t *bm = reinterpret_cast<uint32_t *>(qcol + E + 2);  // E * RW
  int *tmp = qcol + E + 2 + E * p.RW;                         // scan scratch (64)
  int *cv = tmp + 64;                                         // nent_cap: shares, then their prefix
  for (int e = tid; e <= E; e += nt) cnt[e] = 0;
  for (int i = tid; i < E * p.RW; i += nt) bm[i] = 0;
  __syncthreads();
  // the domains' instances (expert, share of self): the first kListRegs per
  // thread are read once and kept in registers for the second pass
  auto count = [&](int idx, int e, int q) {
    if ((unsigned)e < (unsigned)E && q > 0) {
      const int d = (int)fdiv((uint32_t)idx, p.fI), a = idx - d * I;
      const int r = d * G + (int)fdiv((uint32_t)a, p.fPN);
      atomicAdd(&cnt[e], 1);
      atomicOr(&bm[e * p.RW + (r >> 5)], 1u << (r & 31));
    }
  };
  auto place = [&](int idx, int e, int q) {
    if ((unsigned)e < (unsigned)E && q > 0) {
      const int d = (int)fdiv((uint32_t)idx, p.fI), a = idx - d * I;
      const int r = d * G + (int)fdiv((uint32_t)a, p.fPN);
      const uint32_t *row = bm + e * p.RW;
      int pos = 0;
      for (int w = 0; w < (r >> 5); ++w) pos += __popc(row[w]);
      pos += __popc(row[r >> 5] & ((1u << (r & 31)) - 1u));
      const int j = cnt[e] + pos;
      p.csr_r[j] = r;
      cv[j] = q;
    }
  };
  int se[kListRegs], sq[kListRegs];
#pragma unroll
  for (int u = 0; u < kListRegs; ++u) {
    const int idx = tid + u * nt;
    se[u] = idx < M * I ? p.seg_e[idx] : -1;
    sq[u] = idx < M * I ? p.seg_q[idx] : 0;
  }
#pragma unroll
  for (int u = 0; u < kListRegs; ++u) count(tid + u * nt, se[u], sq[u]);
  for (int idx = tid + kListRegs * nt; idx < M * I; idx += nt) count(idx, p.seg_e[idx], p.seg_q[idx]);
  __syncthreads();
  STAMP(p, 11);
  block_excl_scan(cnt, E + 1, tmp);
  for (int e = tid; e <= E; e += nt) p.csr_ptr[e] = cnt[e];
#pragma unroll
  for (int u = 0; u < kListRegs; ++u) place(tid + u * nt, se[u], sq[u]);
  for (int idx = tid + kListRegs * nt; idx < M * I; idx += nt) place(idx, p.seg_e[idx], p.seg_q[idx]);
  __syncthreads();
  // cumulative shares per expert, in LDS, then out
  for (int e = tid; e < E; e += nt) {
    int run = 0;
    for (int j = cnt[e]; j < cnt[e + 1]; ++j) {
      run += cv[j];
      cv[j] = run;
    }
  }
  __syncthreads();
  STAMP(p, 12);
  for (int j = tid; j < cnt[E]; j += nt) p.csr_end[j] = cv[j];
  __syncthreads();
  STAMP(p, 13);
  STAMP_FLUSH(p, 10, 14);
  if (tid == 0) {
    uint32_t fin = __hip_atomic_load(&p.ctrl[kCtrlStatus], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    fin |= gst & TOPOEP_ST_RANGE;
    p.ctrl[kCtrlFinal] = fin;
    p.status_out[0] = (int32_t)fin;
    p.status_out[1] = (fin & (kNoPlan | TOPOEP_ST_SYNC))
                          ? 0
                          : (int32_t)__hip_atomic_load(&p.ctrl[kCtrlMoves], __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
    // every solver workgroup has taken its ticket, so the words it
    // accumulated are final: restore them for the next solve (which may be
    // this stage again, without a histogram kernel before it); the helpers'
    // count goes back by their number (one still running adds its own last)
    p.ctrl[kCtrlBar] = 0;
    p.ctrl[kCtrlTicket] = 0;
    p.ctrl[kCtrlStatus] = 0;
    p.ctrl[kCtrlMoves] = 0;
    *reinterpret_cast<unsigned long long *>(p.ctrl + kCtrlTotal) = 0ull;
    __hip_atomic_fetch_sub(&p.ctrl[kCtrlHelpers], (uint32_t)p.n_helpers, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ---------------------------------------------------------------- solver: one workgroup for every domain

// LDS state of the single-workgroup solver.
struct SingleState {
  uint64_t *ck, *em;
  FastDiv *fdt;
  int *hs, *ccnt, *dfree, *repl, *slots, *used, *Lr, *e_of, *U, *misc, *om, *qcol;
  uint32_t *mask, *bm;
  int *sendl, *wt;
};

__device__ inline SingleState single_state(const Plan &p, int *sm) {
  SingleLds lay = single_lds(p);
  lay.ck = vgpr(lay.ck);
  lay.em = vgpr(lay.em);
  lay.fdt = vgpr(lay.fdt);
  lay.hs = vgpr(lay.hs);
  lay.cnt = vgpr(lay.cnt);
  lay.dfree = vgpr(lay.dfree);
  lay.mask = vgpr(lay.mask);
  lay.bm = vgpr(lay.bm);
  lay.sendl = vgpr(lay.sendl);
  lay.wt = vgpr(lay.wt);
  lay.repl = vgpr(lay.repl);
  lay.slots = vgpr(lay.slots);
  lay.used = vgpr(lay.used);
  lay.L = vgpr(lay.L);
  lay.e_of = vgpr(lay.e_of);
  lay.U = vgpr(lay.U);
  lay.misc = vgpr(lay.misc);
  lay.om = vgpr(lay.om);
  lay.qcol = vgpr(lay.qcol);
  SingleState t;
  t.ck = reinterpret_cast<uint64_t *>(sm + lay.ck);
  t.em = reinterpret_cast<uint64_t *>(sm + lay.em);
  t.fdt = reinterpret_cast<FastDiv *>(sm + lay.fdt);
  t.hs = sm + lay.hs;
  t.ccnt = sm + lay.cnt;
  t.dfree = sm + lay.dfree;
  t.mask = reinterpret_cast<uint32_t *>(sm + lay.mask);
  t.bm = reinterpret_cast<uint32_t *>(sm + lay.bm);
  t.sendl = sm + lay.sendl;
  t.wt = sm + lay.wt;
  t.repl = sm + lay.repl;
  t.slots = sm + lay.slots;
  t.used = sm + lay.used;
  t.Lr = sm + lay.L;
  t.e_of = sm + lay.e_of;
  t.U = sm + lay.U;
  t.misc = sm + lay.misc;
  t.om = sm + lay.om;
  t.qcol = sm + lay.qcol;
  return t;
}

// misc[0] status bits, misc[2] wait flag, misc[8..9] total load, misc[12]
// refinement moves, misc[14] a domain with a free slot; candidate counts,
// hosting-domain masks, local hosting masks, instance-list bitmaps and send
// counts zero; stage-1 replica lists empty; the divisor table.
__device__ inline void single_init(const Plan &p, const SingleState &t) {
  const int tid = threadIdx.x, nt = blockDim.x;
  if (tid < 16) t.misc[tid] = 0;
  for (int d = tid; d < p.M; d += nt) {
    t.ccnt[d] = 0;
    t.dfree[d] = 0;
  }
  for (int i = tid; i < p.E * p.MW; i += nt) t.mask[i] = 0;
  for (int i = tid; i < p.E * p.RW; i += nt) t.bm[i] = 0;
  for (int i = tid; i < p.R; i += nt) t.sendl[i] = 0;
  for (int i = tid; i < p.M * p.cap1; i += nt) t.repl[i] = -1;
  for (int i = tid; i < p.M * p.E; i += nt) t.em[i] = 0;
  // candidate keys: ~0 sorts after every candidate (stage1_ranks reads
  // whole parts of 16)
  for (int i = tid; i < p.M * ((p.E + 15) & ~15); i += nt) t.ck[i] = ~0ull;
  build_divisors(p.M, t.fdt);
}

// The rest of the plan when no domain can refine: every domain's replica
// slots are all taken by stage 1 (or a domain holds one rank).  Every expert
// then has at most one instance per domain (stage 1 places one replica per
// domain and expert, never in the main's own domain), a refinement move
// needs a free slot on its target, so none is committed; and this rank's
// share of expert e follows from the routing rule of Section 4.3 alone: all
// of w = omega[self][e] to the instance in dom(self) if there is one, else
// the even split over the n instances, one per hosting domain in ascending
// order: the i-th takes floor(w / n) + [i < w mod n].  The instances with a
// nonzero share are then the first min(n, w), and the i-th of them ends at
// the cumulative share (i + 1) floor(w / n) + min(i + 1, w mod n).
// Phases: the stage-1 lists with the hosting domains and instance ranks;
// per expert its number of entries, scanned within each wave; per (expert,
// domain) the entry of that domain's instance, the send counts and the
// replica slots.  rr: M E words (rank of e's instance in domain d); ex:
// E words (each expert's first entry inside its wave).  Sets misc[15].
__device__ __forceinline__ void fast_finish(const Plan &p, const SingleState &t, const uint64_t *ck, const int *rk,
                                            int *rr, int *ex) {
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E, G = p.G, M = p.M, R = p.R, cap = p.cap1;
  const int E16 = (E + 15) & ~15, lane = tid & 63, wave = tid >> 6, nw = nt >> 6;
  const int *om = t.om, *ccnt = t.ccnt;
  int *repl = t.repl;
  uint32_t *mask = t.mask;
  int *sendl = t.sendl, *misc = t.misc, *wt = t.wt;
  const int ds = (int)fdiv((uint32_t)p.self, p.fG);
  if (tid == 0) misc[15] = 1;   // (single_recv_counts: the plan came from here; barriers follow)
  // the stage-1 lists, hosting domains and the rank of each instance
  for (int e = tid; e < E; e += nt) {
    const int dm = (int)fdiv((uint32_t)e, p.fGP);
    atomicOr(&mask[e * p.MW + (dm >> 5)], 1u << (dm & 31));
    rr[dm * E + e] = (int)fdiv((uint32_t)e, p.fP);
  }
  // items idx = d E + c, walked with (d, c) kept as the index advances
  const int dstep = (int)fdiv((uint32_t)nt, p.fE), estep = nt - dstep * E;
  const int dfirst = (int)fdiv((uint32_t)tid, p.fE), efirst = tid - dfirst * E;
  int d = dfirst, c = efirst;
  for (int idx = tid; idx < M * E; idx += nt, d += dstep, c += estep) {
    if (c >= E) {
      c -= E;
      ++d;
    }
    const int rank = rk[idx];
    if (c >= ccnt[d] || rank >= cap) continue;
    const int e = (int)(uint32_t)ck[d * E16 + c];
    repl[d * cap + rank] = e;
    atomicOr(&mask[e * p.MW + (d >> 5)], 1u << (d & 31));
    rr[d * E + e] = d * G + (rank - (int)fdiv_hi((uint32_t)rank, p.fG) * G);
  }
  lds_barrier();
  STAMP(p, 27);
  // per expert: its entries, scanned inside the wave; the waves' totals
  // (experts e and e + blockDim ... take rounds; wt holds 16 totals a round)
  const int rounds = (E + nt - 1) / nt;
  for (int r0 = 0; r0 < rounds; ++r0) {
    const int e = r0 * nt + tid;
    int c = 0;
    if (e < E) {
      const int w = om[p.self * E + e];
      const uint32_t *me = mask + e * p.MW;
      int n = 0;
      for (int wd = 0; wd < p.MW; ++wd) n += __popc(me[wd]);
      c = w <= 0 ? 0 : (((me[ds >> 5] >> (ds & 31)) & 1u) ? 1 : imin(n, w));
    }
    const int incl = wave_incl_scan(c);
    if (e < E) ex[e] = incl - c;
    if (lane == 63 && r0 * nt + wave * 64 < E) wt[r0 * nw + wave] = incl;   // per block of 64 experts
  }
  lds_barrier();
  STAMP(p, 28);
  // per (expert, domain): the entry of the domain's instance
  d = dfirst;
  int e = efirst;
  for (int idx = tid; idx < M * E; idx += nt, d += dstep, e += estep) {
    if (e >= E) {
      e -= E;
      ++d;
    }
    const uint32_t *me = mask + e * p.MW;
    const int w = om[p.self * E + e];
    // the expert's first entry: its place in its wave plus the totals of the
    // waves (and rounds) before it
    int first = ex[e];
    for (int b = 0; b < (e >> 6); ++b) first += wt[b];
    if (d == 0) p.csr_ptr[e] = first;
    if (w <= 0 || !((me[d >> 5] >> (d & 31)) & 1u)) continue;
    const bool local = (me[ds >> 5] >> (ds & 31)) & 1u;
    int i = 0, q = w, end = w;
    if (local) {
      if (d != ds) continue;   // all of w to the instance in dom(self)
    } else {
      int n = 0;
      for (int wd = 0; wd < p.MW; ++wd) {
        n += __popc(me[wd]);
        const int lo = wd * 32;
        if (d >= lo + 32) i += __popc(me[wd]);
        else if (d > lo) i += __popc(me[wd] & ((1u << (d - lo)) - 1u));
      }
      const FastDiv fn = t.fdt[n];
      const int qq = (int)fdiv_hi((uint32_t)w, fn), rem = w - qq * n;
      q = qq + (i < rem ? 1 : 0);
      if (q <= 0) continue;
      end = (i + 1) * qq + imin(i + 1, rem);
    }
    const int r = rr[d * E + e];
    p.csr_r[first + i] = r;
    p.csr_end[first + i] = end;
    atomicAdd(&sendl[r], q);
  }
  if (tid == 0) {
    int all = 0;
    for (int b = 0; b < (E + 63) >> 6; ++b) all += wt[b];
    p.csr_ptr[E] = all;
  }
  lds_barrier();
  STAMP(p, 30);
}

// The lean finish's replica slots and send counts, for the caller alone (no
// chunk reads them, so they go out after the flags): slot t of local rank j
// of domain d holds stage-1 entry t G + j (entries are a prefix of the
// domain's list).
__device__ __forceinline__ void fast_outputs(const Plan &p, const SingleState &t) {
  const int tid = threadIdx.x, nt = blockDim.x, G = p.G, R = p.R, cap = p.cap1;
  for (int i = tid; i < R * p.N; i += nt) {
    const int r = (int)fdiv((uint32_t)i, p.fN), s2 = i - r * p.N;
    const int d = (int)fdiv((uint32_t)r, p.fG), j = r - d * G;
    p.slots_out[i] = s2 < p.Neff ? t.repl[d * cap + s2 * G + j] : -1;
  }
  for (int r = tid; r < R; r += nt) p.send_out[r] = t.sendl[r];
}

// Every step after the load: with Omega' in om (row self = the histogram hs)
// and the status bits gst, plans all domains (Eq. 9 placement, routing,
// Eq. 10 refinement) and writes replica_slots, send_counts, this rank's
// instance list and the final status (ctrl word and status_out).  With
// BAD_ID, NEG_LOAD, RANGE or SYNC in gst only the blank outputs are written.
struct NoHook {
  __device__ void operator()() const {}
};
template <class H> struct IsNoHook { static constexpr bool value = false; };
template <> struct IsNoHook<NoHook> { static constexpr bool value = true; };

template <int Form = kRefineAny, class Published = NoHook>
__device__ __forceinline__ void single_plan(const Plan &p, const SingleState &t, uint32_t gst, bool or_status,
                                            Published published = NoHook{}) {
  uint64_t *ck = t.ck, *em = t.em;
  FastDiv *fdt = t.fdt;
  int *hs = t.hs, *ccnt = t.ccnt, *dfree = t.dfree, *repl = t.repl, *slots = t.slots, *used = t.used;
  int *Lr = t.Lr, *e_of = t.e_of, *U = t.U, *misc = t.misc, *om = t.om, *qcol = t.qcol;
  uint32_t *mask = t.mask;
  (void)hs;
  const int tid = threadIdx.x, nt = blockDim.x, wave = tid >> 6, nw = nt >> 6;
  const int E = p.E, G = p.G, R = p.R, M = p.M, I = p.I, P = p.P, PN = p.PN, Neff = p.Neff;
  const int cap = p.cap1;
  if (gst & (kNoPlan | TOPOEP_ST_SYNC)) {
    for (int i = tid; i < R * p.N; i += nt) p.slots_out[i] = -1;
    for (int r = tid; r < R; r += nt) p.send_out[r] = 0;
    if (p.recv_out)
      for (int r = tid; r < R; r += nt) p.recv_out[r] = 0;
    if (tid == 0) {
      p.ctrl[kCtrlFinal] = gst;
      if (or_status) atomicOr(reinterpret_cast<unsigned *>(p.status_out), gst);
      else p.status_out[0] = (int32_t)gst;
      p.status_out[1] = 0;
    }
    return;
  }
  lds_barrier();
  STAMP(p, 23);

  // ---- inter-node placement (Eq. 9), every domain by the whole workgroup
  // (qcol is free until the routing)
  stage1_ranks(p, om, ck, ccnt, qcol);

  // ---- no domain can refine (all slots taken, or one rank per domain):
  // the routing rule alone gives this rank's shares
  {
    bool full = true;
    for (int d = 0; d < M && full; ++d) full = uniform_i32(ccnt[d]) >= cap;
    if (full || G < 2) {
      fast_finish(p, t, ck, qcol, reinterpret_cast<int *>(em), U);
      STAMP(p, 7);
      if (tid == 0) {
        const uint32_t fin = (uint32_t)misc[0] | (gst & TOPOEP_ST_RANGE);
        p.ctrl[kCtrlFinal] = fin;
        misc[45] = (int)fin;   // (kept in LDS past the hook)
      }
      published();
      // the caller's outputs (no chunk reads them)
      fast_outputs(p, t);
      if (tid == 0) {
        const uint32_t fin = (uint32_t)misc[45];
        if (or_status) atomicOr(reinterpret_cast<unsigned *>(p.status_out), fin);
        else p.status_out[0] = (int32_t)fin;
        p.status_out[1] = 0;
      }
      return;
    }
  }
  stage1_lists(p, ck, ccnt, qcol, repl);
  STAMP(p, 2);

  // ---- hosting domains per expert; every rank's slots and instances, and
  // the local ranks hosting each expert in its domain (one pass: stage-1
  // replica i of domain d sits on local rank i mod G, slot i / G, so rank j
  // uses ceil((n_sel - j) / G) slots)
  // (four independent loops over one index space, so each thread runs one
  // loop body instead of one of each)
  {
    const int n1 = M * I, n2 = n1 + E, n3 = n2 + M * cap, n4 = n3 + R;
    for (int v = tid; v < n4; v += nt) {
      if (v < n1) {
        const int idx = v;
        const int d = (int)fdiv((uint32_t)idx, p.fI), a = idx - d * I;
        const int j = (int)fdiv((uint32_t)a, p.fPN), pos = a - j * PN;
        int e;
        if (pos < P) {
          e = (d * G + j) * P + pos;
        } else {
          const int ns = imin(ccnt[d], cap);
          const int u = ns > j ? (int)fdiv((uint32_t)(ns - j + G - 1), p.fG) : 0;
          e = (pos - P) < u ? repl[d * cap + (pos - P) * G + j] : -1;
        }
        e_of[idx] = e;
        U[idx] = 0;
        if (e >= 0) atomicOr(reinterpret_cast<unsigned long long *>(&em[d * E + e]), 1ull << (uint32_t)j);
      } else if (v < n2) {
        const int e = v - n1;
        const int dm = (int)fdiv((uint32_t)e, p.fGP);
        atomicOr(&mask[e * p.MW + (dm >> 5)], 1u << (dm & 31));
      } else if (v < n3) {
        const int i = v - n2;
        const int e = repl[i];
        if (e >= 0) {
          const int dd = (int)fdiv((uint32_t)i, p.fCap);
          atomicOr(&mask[e * p.MW + (dd >> 5)], 1u << (dd & 31));
        }
      } else {
        const int r = v - n3;
        const int d = (int)fdiv((uint32_t)r, p.fG), j = r - d * G;
        const int ns = imin(ccnt[d], cap);
        const int u = ns > j ? (int)fdiv((uint32_t)(ns - j + G - 1), p.fG) : 0;
        used[r] = u;
        for (int t = 0; t < Neff; ++t) slots[r * Neff + t] = t < u ? repl[d * cap + t * G + j] : -1;
        if (u < Neff) {
          dfree[d] = 1;
          misc[14] = 1;
        }
      }
    }
  }
  lds_barrier();

  STAMP(p, 3);
  // ---- routing construction (Section 4.3) for every domain's instances;
  // instances of domains that cannot refine enter this rank's instance-list
  // bitmaps and send counts at once
  uint32_t *bm = t.bm;
  int *sendl = t.sendl;
  auto mark = [&](int i, int d, int e, int q) {
    if (q > 0) {
      const int r = d * G + (int)fdiv((uint32_t)(i - d * I), p.fPN);
      atomicOr(&bm[e * p.RW + (r >> 5)], 1u << (r & 31));
      atomicAdd(&sendl[r], q);
    }
  };
  route_instances(
      p, M * I, p.fMI, p.rchunks_all, e_of, mask, fdt, qcol, U, [&](int, int e) { return om + e; }, E,
      [&](int i) { return (int)fdiv((uint32_t)i, p.fI); }, [&](int d) { return dfree[d] != 0; }, mark);
  lds_barrier();
  STAMP(p, 4);

  if (misc[14]) {
    // ---- intra-node refinement (Eq. 10): one wave per domain (it sums its
    // ranks' loads first; a domain without a free slot returns at once)
    uint32_t flags = 0, moves = 0;
    for (int d = wave; d < M; d += nw)
      moves += refine_domain<false, Form>(p, d, e_of + d * I, U + d * I, qcol + d * I * p.QS, slots + d * G * Neff,
                             used + d * G, Lr + d * G, em + (int64_t)d * E, &flags, true);
    if (lane_id() == 0) {
      if (flags) atomicOr(reinterpret_cast<unsigned *>(&misc[0]), flags);
      if (moves) atomicAdd(reinterpret_cast<unsigned *>(&misc[12]), moves);
    }
    lds_barrier();
    // ---- the refined domains' instances enter the bitmaps and send counts
    for (int idx = tid; idx < M * I; idx += nt) {
      const int d = (int)fdiv((uint32_t)idx, p.fI);
      const int e = e_of[idx];
      if (dfree[d] && e >= 0) mark(idx, d, e, qcol[idx * p.QS + p.self]);
    }
    lds_barrier();
  }

  STAMP(p, 5);
  // ---- outputs: replica slots, send counts, this rank's instance list and
  // the final status.  With a hook (the one-launch plan, whose chunks read
  // only the list and the final status word) the caller's outputs wait
  // until the hook has released the chunks.
  constexpr bool defer = !IsNoHook<Published>::value;
  auto caller_outputs = [&]() {
    for (int i = tid; i < R * p.N; i += nt) {
      const int r = (int)fdiv((uint32_t)i, p.fN), t2 = i - r * p.N;
      p.slots_out[i] = t2 < used[r] ? slots[r * Neff + t2] : -1;
    }
    for (int r = tid; r < R; r += nt) p.send_out[r] = sendl[r];
    if (tid == 0) {
      const uint32_t fin = (uint32_t)misc[45];
      if (or_status) atomicOr(reinterpret_cast<unsigned *>(p.status_out), fin);
      else p.status_out[0] = (int32_t)fin;
      p.status_out[1] = misc[12];
    }
  };
  if constexpr (!defer) {
    for (int i = tid; i < R * p.N; i += nt) {
      const int r = (int)fdiv((uint32_t)i, p.fN), t2 = i - r * p.N;
      p.slots_out[i] = t2 < used[r] ? slots[r * Neff + t2] : -1;
    }
    for (int r = tid; r < R; r += nt) p.send_out[r] = sendl[r];
  }
  STAMP(p, 6);
  emit_instance_list(p, qcol, slots, used, bm, t.wt);
  STAMP(p, 7);
  if (tid == 0) {
    const uint32_t fin = (uint32_t)misc[0] | (gst & TOPOEP_ST_RANGE);
    p.ctrl[kCtrlFinal] = fin;
    misc[45] = (int)fin;   // (kept in LDS past the hook)
    if constexpr (!defer) {
      if (or_status) atomicOr(reinterpret_cast<unsigned *>(p.status_out), fin);
      else p.status_out[0] = (int32_t)fin;
      p.status_out[1] = misc[12];
    }
  }
  published();
  if constexpr (defer) caller_outputs();
}

// Receive counts from the single-workgroup solver's final LDS state (after
// single_plan made a plan): the instances on rank self, full columns when
// its domain was routed for every source.  A plan of fast_finish (misc[15])
// kept no instance state: rank self's instances are its mains and its
// stage-1 replicas (slot t = entry t G + j of its domain's list), and the
// routing rule gives every source's share.
__device__ __forceinline__ void single_recv_counts(const Plan &p, const SingleState &t) {
  const int ds = (int)fdiv((uint32_t)p.self, p.fG), E = p.E;
  const int *om = t.om;
  if (t.misc[15]) {
    int *selfe = t.U;
    const int js = p.self - ds * p.G;
    for (int a = threadIdx.x; a < p.PN; a += blockDim.x)
      selfe[a] = a < p.P ? p.self * p.P + a : t.repl[ds * p.cap1 + (a - p.P) * p.G + js];
    lds_barrier();
    write_recv_counts(p, 0, selfe, nullptr, false, t.mask, t.fdt, [&](int s, int e) { return om[s * E + e]; },
                      t.hs);
    return;
  }
  // (hs, the histogram, is no longer needed: it is the scratch)
  write_recv_counts(p, ds * p.I + (p.self - ds * p.G) * p.PN, t.e_of, t.qcol, t.dfree[ds] != 0, t.mask, t.fdt,
                    [&](int s, int e) { return om[s * E + e]; }, t.hs);
}

// Send offsets of the one-launch plan (exclusive prefix of the send counts
// sendl, total at [R]) by wave 0, for the caller and for the chunks.
__device__ __forceinline__ void solver_send_offsets(const Plan &p, const int *sendl) {
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x, R = p.R;
  const int per = (R + 63) / 64, lo = imin(R, lane * per), hi = imin(R, lo + per);
  int sum = 0;
  for (int r = lo; r < hi; ++r) sum += sendl[r];
  int run = wave_incl_scan(sum) - sum;
  for (int r = lo; r < hi; ++r) {
    p.offs_out[r] = run;
    run += sendl[r];
  }
  if (lane == 63) p.offs_out[R] = run;
}

// The same steps with every domain's state in the LDS of one CU; each
// domain's refinement runs on its own wave.  Used when Omega and all q
// columns fit in LDS.  Workgroups beyond the first compute the histogram
// blocks' offsets for the reroute.
__global__ __launch_bounds__(1024) void solve_single_kernel(Plan p0) {
  extern __shared__ int64_t smem_1[];
  int *sm = reinterpret_cast<int *>(smem_1);
  if (blockIdx.x > 0) {
    block_offsets(p0, blockIdx.x - 1, sm, false);
    return;
  }
  const Plan p = solver_plan(p0);
  const SingleState t = single_state(p, sm);
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E, R = p.R;
  single_init(p, t);
  // ---- Omega to LDS; histogram of local_topk from the blocks' partials
  lds_barrier();
  if (load_fast_ok(p)) {
    load_fast(p, t.om, t.hs, t.qcol, t.misc);
  } else {
    copy_to_lds(t.om, p.gl, R * E);
    hist_from_partials(p, t.hs, t.qcol);
    for (int b = tid; b < p.nb; b += nt)
      if (p.blk_err[b]) atomicOr(reinterpret_cast<unsigned *>(&t.misc[0]), TOPOEP_ST_BAD_ID);
    scan_rows(p, 0, R, t.om, t.hs, t.misc);
    lds_barrier();
    for (int e = tid; e < E; e += nt) t.om[p.self * E + e] = t.hs[e];
  }
  uint32_t gst = (uint32_t)t.misc[0];
  if (out_of_range(p, *reinterpret_cast<unsigned long long *>(t.misc + 8))) gst |= TOPOEP_ST_RANGE;
  single_plan(p, t, gst, false);
  if (p.recv_out && !(gst & kNoPlan)) single_recv_counts(p, t);
}

// ---------------------------------------------------------------- send-buffer slots
//
// The send buffer groups the assignments by destination (ranks ascending,
// row-major order inside one destination).  An assignment's slot is
// offs[d] + (assignments to d before its tile) + (those of earlier waves of
// the tile) + (its rank among its wave's earlier assignments to d).  The
// count before a tile follows from the per-expert counts before it, with no
// pass over earlier ids: expert e's occurrences are dealt to its instances
// in occurrence order, instance j taking [end(j-1), end(j)), so
// clamp(run[e] - end(j-1), 0, end(j) - end(j-1)) of them went to j's rank.

// offs[0..R) holds the send counts: it becomes their exclusive prefix with
// the total at offs[R] (tmp: blockDim/64 + 1 words); `first` writes it out.
__device__ void slot_offsets(const Plan &p, int *offs, int *tmp, bool first) {
  lds_barrier();
  offs[p.R] = block_excl_scan(offs, p.R, tmp);
  if (first && p.offs_out)
    for (int r = threadIdx.x; r <= p.R; r += blockDim.x) p.offs_out[r] = offs[r];
}

// excl[r] = assignments to rank r before the tile (run[e]: occurrences of e
// before it; ptr/er/eend: this rank's instance list).  Ends with a barrier.
__device__ void slot_before(const Plan &p, const int *run, const int *ptr, const int2 *ent, int *excl) {
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int r = tid; r < p.R; r += nt) excl[r] = 0;
  lds_barrier();
  for (int e = tid; e < p.E; e += nt) {
    const int re = run[e], j1 = ptr[e + 1];
    int start = 0;
    for (int j = ptr[e]; j < j1; ++j) {
      const int2 en = ent[j];   // (cumulative share, rank)
      const int c = imin(imax(re - start, 0), en.x - start);
      if (c > 0 && (unsigned)en.y < (unsigned)p.R) atomicAdd(&excl[en.y], c);
      start = en.x;
    }
  }
  lds_barrier();
}

// Per-wave counts to offsets, one column per key: wc[(w * ws + k) * S] (w <
// nw <= 16 waves, k < n keys, ws > n odd so a column's words sit in distinct
// banks; S: words per element) becomes base[k] + the counts of waves
// 0..w-1, and base[k] grows by the column's total (base may be null:
// offsets from 0).  Beyond four waves a group of g lanes (g = nw rounded up
// to a power of two) per key scans the column in registers instead of
// walking it with nw dependent LDS round trips.
template <int S = 1>
__device__ inline void scan_wave_columns(int *wc, int ws, int n, int nw, int *base) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63;
  if (nw <= 4) {
    // short columns: one thread walks each
    for (int k = tid; k < n; k += nt) {
      int run = base ? base[k] : 0;
      for (int w = 0; w < nw; ++w) {
        const int t = wc[(w * ws + k) * S];
        wc[(w * ws + k) * S] = run;
        run += t;
      }
      if (base) base[k] = run;
    }
    return;
  }
  const int lg = nw <= 1 ? 0 : 32 - __clz(nw - 1);   // log2 of the group size
  const int g = 1 << lg, w = lane & (g - 1);
  for (int k = tid >> lg; k < n; k += nt >> lg) {
    const int v = w < nw ? wc[(w * ws + k) * S] : 0;
    int x = v;
    // inclusive scan inside the group (row shifts; a group never crosses a row)
    int y;
    y = (int)dpp_mov<0x111>((uint32_t)x); x += w >= 1 ? y : 0;
    y = (int)dpp_mov<0x112>((uint32_t)x); x += w >= 2 ? y : 0;
    y = (int)dpp_mov<0x114>((uint32_t)x); x += w >= 4 ? y : 0;
    y = (int)dpp_mov<0x118>((uint32_t)x); x += w >= 8 ? y : 0;
    const int tot = __shfl(x, lane | (g - 1));
    const int b0 = base ? base[k] : 0;
    if (w < nw) wc[(w * ws + k) * S] = b0 + x - v;
    if (base && w == 0) base[k] = b0 + tot;
  }
}

// Slots of one tile (destinations dv in registers; index order: wave, then
// i, then lane); wcd: blockDim/64 * (R | 1) words of scratch.
template <int IPT>
__device__ void slot_write(const Plan &p, const int (&dv)[IPT], int64_t wbase, int64_t hi, const int *offs,
                           const int *excl, int *wcd) {
  const int nt = blockDim.x, nw = nt >> 6, lane = threadIdx.x & 63, wave = threadIdx.x >> 6, R = p.R;
  const int ws = R | 1;
  int *mw = wcd + wave * ws;
  for (int r = lane; r < R; r += 64) mw[r] = 0;
  wave_sync();
  int lr[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    // (dv is -1 past the end)
    lr[i] = wave_rank(dv[i], (unsigned)dv[i] < (unsigned)R, p.rbits, mw);
  }
  lds_barrier();
  scan_wave_columns(wcd, ws, R, nw, nullptr);
  lds_barrier();
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int64_t idx = wbase + i * 64;
    if (idx < hi) {
      const int d = dv[i];
      p.slot_out[idx] = (unsigned)d < (unsigned)R ? offs[d] + excl[d] + mw[d] + lr[i] : -1;
    }
  }
}

// ---------------------------------------------------------------- reroute

template <int IPT>
__global__ __launch_bounds__(1024) void reroute_kernel(Plan p) {
  extern __shared__ int smem_r[];
  const int nt = blockDim.x, nw = nt >> 6;
  const int E = p.E, ws = E | 1;
  int2 *ent = reinterpret_cast<int2 *>(smem_r);   // nent_cap + 1: (cumulative share, rank) per entry
  int2 *cur = ent + p.nent_cap + 1;  // E: (entry holding the next occurrence, end of e's entries)
  int2 *wc = cur + E;                // nw * ws: per wave and expert the count, then (offset, entry)
  int *run = reinterpret_cast<int *>(wc + nw * ws);   // E: running offset per expert
  int *ptr = run + E;                // E + 1
  int *wcd = ptr + E + 1;            // nw * (R | 1): send-buffer slots: per-wave counts
  int *excl = wcd + nw * (p.R | 1);  // R: assignments per rank before the tile
  int *so = excl + p.R;              // R + 1 + nw + 1: send offsets, scan scratch
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  const int64_t lo = (int64_t)b * p.chunk;
  const int64_t hi = lo + p.chunk < p.n ? lo + p.chunk : p.n;
  const uint32_t fin = p.ctrl[kCtrlFinal];
  if (fin & (kNoPlan | TOPOEP_ST_SYNC)) {
    for (int64_t i = lo + tid; i < hi; i += nt) p.dest_out[i] = -1;
    if (p.slot_out)
      for (int64_t i = lo + tid; i < hi; i += nt) p.slot_out[i] = -1;
    if (b == 0 && p.offs_out)
      for (int r = tid; r <= p.R; r += nt) p.offs_out[r] = 0;
    return;
  }
  // the first tile's ids are on their way while the block reads its offsets
  // and the instance list
  const int64_t tile = (int64_t)nt * IPT;
  int evn[IPT];
  auto load_tile = [&](int64_t base) {
    const int64_t wbase = base + (int64_t)wave * 64 * IPT + lane;
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = wbase + i * 64;
      evn[i] = idx < hi ? p.topk[idx] : -1;
    }
  };
  load_tile(lo);
  if (p.offs_out) {
    for (int r = tid; r < p.R; r += nt) so[r] = p.send_out[r];
    slot_offsets(p, so, so + p.R + 1, b == 0);
  }
  for (int e = tid; e < E; e += nt) run[e] = p.offsets[(int64_t)b * E + e];
  for (int e = tid; e <= E; e += nt) {
    const int v = p.csr_ptr[e];
    ptr[e] = v < 0 ? 0 : (v > p.nent_cap ? p.nent_cap : v);
  }
  __syncthreads();
  const int nent = ptr[E];
  for (int j = tid; j < nent; j += nt) ent[j] = make_int2(p.csr_end[j], p.csr_r[j]);
  // past the last entry: a sentinel no occurrence lies below
  if (tid == 0) ent[p.nent_cap] = make_int2(INT_MIN, -1);
  __syncthreads();
  // run[e] counts e's occurrences before the chunk: each expert's cursor
  // starts at the entry holding occurrence run[e], the first of [ptr[e],
  // ptr[e + 1]) whose cumulative share exceeds it (shares ascend: a binary
  // search); each tile moves it on past its own occurrences.  (The thread
  // that sets a cursor is the one that walks it below: no barrier.)
  for (int e = tid; e < E; e += nt) {
    const int re = run[e], j1 = ptr[e + 1];
    int lo2 = ptr[e], hi2 = j1;
    while (lo2 < hi2) {
      const int mid = (lo2 + hi2) >> 1;
      if (ent[mid].x <= re) lo2 = mid + 1;
      else hi2 = mid;
    }
    cur[e] = make_int2(lo2, j1);
  }
  int2 *mywc = wc + wave * ws;
  for (int64_t base = lo; base < hi; base += tile) {
    int ev[IPT];
#pragma unroll
    for (int i = 0; i < IPT; ++i) ev[i] = evn[i];
    // the next tile's ids load while this one is ranked (the barriers below
    // order LDS only, so they do not wait for these loads)
    if (base + tile < hi) load_tile(base + tile);
    if (p.slot_out) slot_before(p, run, ptr, ent, excl);
    for (int e = lane; e < E; e += 64) mywc[e].x = 0;
    wave_sync();
    const int64_t wbase = base + (int64_t)wave * 64 * IPT + lane;
    // ids of this lane left in the chunk (the stores' bound)
    const int lim = (int)(hi - wbase < 64 * IPT ? hi - wbase : 64 * IPT);
    int lr[IPT];
#pragma unroll
    for (int i = 0; i < IPT; ++i)   // (ev is -1 past the end)
      lr[i] = wave_rank<2>(ev[i], (unsigned)ev[i] < (unsigned)E, p.nbits, reinterpret_cast<int *>(mywc));
    lds_barrier();
    // each wave's offset of e, and the entry holding that first occurrence
    // (the sentinel when it lies past e's entries), found from e's cursor
    // (offsets grow with the wave), which then moves past the tile: up to
    // four waves one thread walks each expert's column once, else the
    // columns are scanned first
    // (the current entry's share end stays in a register: LDS is read only
    // when the walk moves on)
    auto entry_of = [&](int2 c, int &j, int &ej, int off) {
      while (j < c.y && ej <= off) {
        ++j;
        ej = j < c.y ? ent[j].x : INT_MAX;
      }
      return j < c.y ? j : p.nent_cap;
    };
    if (nw <= 4) {
      for (int e = tid; e < E; e += nt) {
        const int2 c = cur[e];
        int j = c.x, r = run[e];
        int ej = j < c.y ? ent[j].x : INT_MAX;
        for (int w = 0; w < nw; ++w) {
          int2 *x = wc + w * ws + e;
          const int t = x->x;
          *x = make_int2(r, entry_of(c, j, ej, r));
          r += t;
        }
        run[e] = r;
        entry_of(c, j, ej, r);
        if (j != c.x) cur[e].x = j;
      }
    } else {
      scan_wave_columns<2>(reinterpret_cast<int *>(wc), ws, E, nw, run);
      lds_barrier();
      for (int e = tid; e < E; e += nt) {
        const int2 c = cur[e];
        int j = c.x;
        int ej = j < c.y ? ent[j].x : INT_MAX;
        for (int w = 0; w < nw; ++w) {
          int2 *x = wc + w * ws + e;
          x->y = entry_of(c, j, ej, x->x);
        }
        entry_of(c, j, ej, run[e]);
        if (j != c.x) cur[e].x = j;
      }
    }
    lds_barrier();
    int dv[IPT];
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      // occurrence rho of e: the entry of the wave's first occurrence holds
      // it unless the wave's occurrences run past that instance's share
      // (then the entries after it, or none past e's last)
      const int e = ev[i];
      const bool valid = (unsigned)e < (unsigned)E;
      const int2 r = mywc[valid ? e : 0];
      const int rho = r.x + lr[i];
      const int2 en = ent[r.y];
      const bool hit = rho < en.x;
      int dest = valid && hit ? en.y : -1;
      const bool slow = valid && !hit;
      if (slow) {   // (skipped when no lane of the wave needs it)
        const int j1 = ptr[e + 1];
        for (int j = r.y + 1; j < j1; ++j) {
          const int2 en2 = ent[j];
          if (rho < en2.x) {
            dest = en2.y;
            break;
          }
        }
      }
      if (i * 64 < lim) p.dest_out[wbase + i * 64] = dest;
      dv[i] = dest;
    }
    if (p.slot_out) slot_write<IPT>(p, dv, wbase, hi, so, excl, wcd);
    lds_barrier();
  }
}

// ---------------------------------------------------------------- single-launch plan
//
// Workgroup 0 solves; workgroups 1..nb each hold one chunk of ids.  The
// plan's generation g orders the hand-overs (control words 8..11 above):
//   chunk -> everyone: chunk b writes its count of every expert to
//     pub[b][e] and adds it to the histogram ghist[g & 1][e] with an
//     agent-scope atomic (integer adds commute: the sum does not depend on
//     their order; word E counts bad ids), then makes one release increment
//     of the 64-bit arrival counter; the value it moves the counter from,
//     g nb + c, gives g and tells the last arrival (c = nb - 1).  A chunk
//     reads g from word 10 to pick the histogram buffer before it arrives;
//     that read can only be stale when the solver has already given up on
//     this plan, and the chunk then takes its adds back.
//   last chunk -> chunks: word 1 of every chunk's flag line = g + 1
//     (release): every count is written.  Chunk b then sums its first
//     occurrence index of each expert from the counts of the chunks before
//     it, or from the histogram less the counts of the chunks from b on,
//     whichever reads fewer rows (at most nb / 2).
//   last chunk -> solver: the histogram against row self of Omega, released
//     as the verdict ((g + 1) << 2) | v.  Only the solver polls that word.
//   solver -> chunk b: word 0 of chunk b's flag line = g + 1 (release) once
//     the outputs, this rank's instance list and the final status are
//     written.  Chunk b polls only its own 128-byte flag line, acquires, and
//     reads the instance list in one round trip.
// No word is cleared between plans except the other histogram buffer (by
// the solver, before any chunk of the next plan can use it): a workspace is
// zero-filled before its first plan, and a plan whose bounded wait gave up
// (SYNC) leaves nothing that a later plan's waits could mistake for its own.

// Omega to LDS with its status bits and total load (row self included as
// gathered; the caller swaps in the histogram later).  `between` runs on
// every thread once the first loads are issued (LDS set-up that overlaps
// their latency); the status words are written after a barrier behind it.
template <typename Between>
__device__ __forceinline__ void load_omega(const Plan &p, int *om, int *misc, Between between) {
  const int tid = threadIdx.x, nt = blockDim.x, n = p.R * p.E;
  bool neg = false;
  uint64_t tot = 0;
  if ((p.E & 3) == 0 && (reinterpret_cast<uintptr_t>(p.gl) & 15) == 0) {
    const int n4 = n >> 2;
    const int4 *g4 = reinterpret_cast<const int4 *>(p.gl);
    int4 *o4 = reinterpret_cast<int4 *>(om);
    int4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = g4[imin(tid + u * nt, n4 - 1)];
    between();
    for (int i = tid; i < n4; i += 4 * nt) {
      if (i != tid) {
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = g4[imin(i + u * nt, n4 - 1)];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (i + u * nt < n4) {
          o4[i + u * nt] = v[u];
          neg |= (v[u].x | v[u].y | v[u].z | v[u].w) < 0;
          tot += (uint64_t)(v[u].x > 0 ? v[u].x : 0) + (uint64_t)(v[u].y > 0 ? v[u].y : 0) +
                 (uint64_t)(v[u].z > 0 ? v[u].z : 0) + (uint64_t)(v[u].w > 0 ? v[u].w : 0);
        }
      }
    }
  } else {
    between();
    for (int i = tid; i < n; i += nt) {
      const int g = p.gl[i];
      om[i] = g;
      neg |= g < 0;
      if (g > 0) tot += (uint64_t)g;
    }
  }
  tot = wave_sum_u64(tot);
  const uint64_t any_neg = __ballot(neg);
  lds_barrier();
  if (lane_id() == 0) {
    if (any_neg) atomicOr(reinterpret_cast<unsigned *>(&misc[0]), TOPOEP_ST_NEG_LOAD);
    if (tot) atomicAdd(reinterpret_cast<unsigned long long *>(misc + 8), (unsigned long long)tot);
  }
}

// Solver side of a redo: hs[e] = the histogram of local_topk, gh[e] (every
// chunk's adds, acquired with the last chunk's verdict), BAD_ID from gh[E].
__device__ __forceinline__ void read_histogram(const Plan &p, const uint32_t *gh, int *hs, int *misc) {
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E;
  bool bad = false;
  for (int e = tid; e <= E; e += nt) {
    const uint32_t v = gh[e];
    if (e < E) hs[e] = (int)v;
    else bad = v != 0;
  }
  const uint64_t any_bad = __ballot(bad);
  if (lane_id() == 0 && any_bad) atomicOr(reinterpret_cast<unsigned *>(&misc[0]), TOPOEP_ST_BAD_ID);
  __syncthreads();
}

// Solver role (workgroup 0): Omega goes to LDS and the whole plan is made
// from it while the chunks count; once the last chunk has compared the
// histogram with row self of Omega, that plan stands (equal rows, so Omega'
// = Omega) or is made again from Omega' on fresh state; then every chunk's
// flag is set to g + 1 and the generation advances.
template <int Form>
__device__ __forceinline__ void fused_solver(const Plan &p, int *sm) {
  const SingleState t = single_state(p, sm);
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E;
  // this plan's generation (stored by the previous plan's solver); wave 0
  // waits for the verdict and sets the flags
  uint32_t gen = 0;
  if (tid < 64) {
    gen = __hip_atomic_load(&p.ctrl[kCtrlGen], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // the next plan's histogram buffer starts from zero (stored long before
    // this plan ends, which is when that plan's chunks may start)
    uint32_t *other = p.ghist + ((gen + 1u) & 1u) * (p.E + 1);
    for (int e = tid; e <= p.E; e += 64) __hip_atomic_store(other + e, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  STAMP(p, 0);
  STAMP_CLK(p, 20);
  STAMP_CLEAR(32, 39);
  if (tid == 0) p.status_out[0] = 0;   // chunks may OR SYNC into it
  load_omega(p, t.om, t.misc, [&] { single_init(p, t); });
  if (tid == 0) {
    t.misc[40] = (int)gen;   // (single_init clears words 0..15 only)
    t.misc[44] = 0;          // the speculative plan went out early
  }
  lds_barrier();
  STAMP(p, 1);
  // Omega's status (single_plan starts with a barrier before any thread
  // writes these words again)
  const uint64_t total0 = uniform_u64(*reinterpret_cast<const unsigned long long *>(t.misc + 8));
  const uint32_t gst0 = ((uint32_t)uniform_i32(t.misc[0]) & TOPOEP_ST_NEG_LOAD) |
                        (out_of_range(p, total0) ? TOPOEP_ST_RANGE : 0u);
  const uint32_t neg0 = gst0 & TOPOEP_ST_NEG_LOAD;
  // Speculative plan from Omega as gathered while the chunks count: it is
  // the plan whenever the histogram equals row self (the gathered row is
  // this rank's own count), else it is redone below; nothing reads the
  // outputs before the flags say the plan is ready.
  const bool spec = !(gst0 & kNoPlan);
  // the flags: every output the chunks read (the instance list, the final
  // status, the send offsets) drained first, then released
  auto release_flags = [&]() {
    STAMP(p, 10);
    STAMP_CLK(p, 21);
    if (tid < 64)
      for (int b = tid; b < p.nb; b += 64)
        __hip_atomic_store(p.flags + (int64_t)b * kFlagStride, gen + 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  };
  auto set_flags = [&]() {
    drain_then_barrier();
    release_flags();
  };
  // as soon as the speculative plan's list and status are written: when the
  // verdict is already in and says the plan stands (the usual case), the
  // flags go out at once
  auto publish_early = [&]() {
    if (tid == 0) {
      const uint32_t v = __hip_atomic_load(&p.ctrl[kCtrlVerdict], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      t.misc[44] = ((v >> 2) == ((gen + 1u) & 0x3FFFFFFFu) && (v & 3u) == kVerdictSame) ? 1 : 0;
    }
    lds_barrier();
    if (t.misc[44]) {
      if (p.offs_out) solver_send_offsets(p, t.sendl);
      set_flags();
    }
  };
  if (spec) single_plan<Form>(p, t, gst0, true, publish_early);   // (with its status: it usually stands)
  STAMP(p, 8);
  const bool early = t.misc[44] != 0;
  // the last chunk's verdict on this generation: its first read overlaps
  // the drain of the speculative outputs
  uint32_t w = 0;
  if (!early && tid == 0) w = __hip_atomic_load(&p.ctrl[kCtrlVerdict], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (!early) drain_then_barrier();
  if (early) {
    if (tid == 0) {
      t.misc[2] = 1;
      t.misc[3] = (int)kVerdictSame;
    }
  } else if (tid == 0) {
    const uint32_t want = (gen + 1u) & 0x3FFFFFFFu;
    bool ok = false;
    for (uint32_t it = 0; it < p.spin_limit; ++it) {
      if (it > 0) {
        __builtin_amdgcn_s_sleep(1);
        w = __hip_atomic_load(&p.ctrl[kCtrlVerdict], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      if ((w >> 2) == want) {
        ok = true;
        break;
      }
    }
    // acquire: the histogram of a redo, and (passed on by the flags' release)
    // the chunks' counts
    if (ok) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    t.misc[2] = ok;
    t.misc[3] = (int)(w & 3u);
  }
  __syncthreads();
  STAMP(p, 9);
  const bool synced = t.misc[2] != 0;
  const uint32_t verdict = (uint32_t)t.misc[3];
  const bool stands = synced && verdict == kVerdictSame && spec;
  bool planned = stands;
  // a plan that does not stand: its status bits go (a chunk's SYNC stays)
  if (spec && !stands && tid == 0) atomicAnd(reinterpret_cast<unsigned *>(p.status_out), TOPOEP_ST_SYNC);
  if (stands) {
    // the speculative plan stands (Omega' = Omega) with its status
  } else if (synced && verdict == kVerdictSame) {
    single_plan<Form>(p, t, gst0, true);   // Omega itself refused: blank outputs
  } else if (synced) {
    // row self differs from the histogram, or a bad id: plan again from
    // Omega' (row self = the histogram) on fresh state
    single_init(p, t);
    lds_barrier();
    read_histogram(p, p.ghist + (int64_t)(t.misc[40] & 1) * (E + 1), t.hs, t.misc);
    bool diff = false;
    int64_t adj = 0;
    for (int e = tid; e < E; e += nt) {
      const int h = t.hs[e], g = t.om[p.self * E + e];
      diff |= g != h;
      adj += (int64_t)(h > 0 ? h : 0) - (int64_t)(g > 0 ? g : 0);
      t.om[p.self * E + e] = h;
    }
    adj = (int64_t)wave_sum_u64((uint64_t)adj);
    const uint64_t any_diff = __ballot(diff);
    if (lane_id() == 0) {
      atomicOr(reinterpret_cast<unsigned *>(&t.misc[0]), (any_diff ? TOPOEP_ST_SELF_DIFF : 0u) | neg0);
      if (adj) atomicAdd(reinterpret_cast<unsigned long long *>(t.misc + 8), (unsigned long long)adj);
    }
    lds_barrier();
    uint32_t gst = (uint32_t)t.misc[0];
    if (out_of_range(p, total0 + *reinterpret_cast<const unsigned long long *>(t.misc + 8))) gst |= TOPOEP_ST_RANGE;
    single_plan<Form>(p, t, gst, true);
    planned = !(gst & kNoPlan);
  } else {
    single_plan<Form>(p, t, TOPOEP_ST_SYNC, true);
  }
  if (!early) {
    if (planned && p.offs_out) solver_send_offsets(p, t.sendl);
    set_flags();
  }
  // the next generation
  if (tid == 0) __hip_atomic_store(&p.ctrl[kCtrlGen], gen + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  STAMP_FLUSH(p, 0, 12);
  STAMP_FLUSH(p, 20, 39);
  // receive counts of a plan that was made (a refused one wrote zeros):
  // for the caller only, so they are summed while the chunks route
  if (planned && p.recv_out) single_recv_counts(p, t);
}

// x / d for x < 2^52 and 0 < d < 2^31: the quotient formed in double
// precision (within one of the exact one there), then corrected to the floor.
__device__ inline uint64_t div_u64_small(uint64_t x, uint32_t d) {
  uint64_t q = (uint64_t)((double)x / (double)d);
  int64_t r = (int64_t)(x - q * d);
  while (r < 0) {
    --q;
    r += d;
  }
  while (r >= (int64_t)d) {
    ++q;
    r -= d;
  }
  return q;
}

// The last chunk to arrive (every chunk's counts are in pub and in
// ghist[g & 1]): word 1 of every chunk's flag line (the chunks start summing
// their offsets), then the histogram against row self of Omega and the
// bad-id count, released as the verdict of generation g.
__device__ __forceinline__ void last_arrival(const Plan &p, uint32_t g) {
  const int tid = threadIdx.x, E = p.E;
  if (tid < 64)
    for (int c = tid; c < p.nb; c += 64)
      __hip_atomic_store(p.flags + (int64_t)c * kFlagStride + 1, g + 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t *gh = p.ghist + (g & 1u) * (E + 1);
  bool diff = false;
  for (int e = tid; e <= E; e += blockDim.x) {
    const uint32_t v = gh[e];
    diff |= e < E ? (int)v != p.gl[(int64_t)p.self * E + e] : v != 0u;
  }
  const bool redo = __syncthreads_or(diff) != 0;
  if (tid == 0)
    __hip_atomic_store(&p.ctrl[kCtrlVerdict], (((g + 1u) & 0x3FFFFFFFu) << 2) | (redo ? kVerdictRedo : kVerdictSame),
                       __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded wait of chunk b's workgroup until word w of its flag line holds
// `target` (the plan's generation + 1), at most spin_limit polls.  Thread 0
// polls (more pollers per chunk slow every agent-coherent load down), then
// acquires (the L1 and L2 invalidations cover the whole CU).  Returns false
// (on every thread) if the wait gave up.
__device__ __forceinline__ bool wait_flag(const Plan &p, int b, int w, uint32_t target, int *flag) {
  if (threadIdx.x == 0) {
    uint32_t *f = p.flags + (int64_t)b * kFlagStride + w;
    int ok = 0;
    for (uint32_t it = 0; it < p.spin_limit; ++it) {
      if (it > 0) __builtin_amdgcn_s_sleep(2);
      if (__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == target) {
        ok = 1;
        break;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    *flag = ok;
  }
  __syncthreads();
  return *flag != 0;
}

// Chunk b's first occurrence index of every expert (run[e]) once every
// count is written: the sum of the counts of chunks 0 .. b - 1, or the
// histogram gh less the counts of chunks b .. nb - 1 when that reads fewer
// rows.  Thread (grp, e) sums its share of the rows with eight loads in
// flight; gs: blockDim words of partial sums.
__device__ __forceinline__ void chunk_offsets(const Plan &p, int b, const uint32_t *gh, int *run, int *gs) {
  const int tid = threadIdx.x, nt = blockDim.x, E = p.E, nb = p.nb;
  const bool from_start = 2 * b <= nb;
  const int r0 = from_start ? 0 : b, cnt = from_start ? b : nb - b;
  const int groups = imax(1, nt / E);
  const int per = (cnt + groups - 1) / groups;
  for (int t = tid; t < groups * E; t += nt) {
    const int g = (int)fdiv((uint32_t)t, p.fE), e = t - g * E;
    const int b0 = r0 + g * per, n = imax(0, imin(r0 + cnt, b0 + per) - b0);
    int sum = 0;
    for (int j0 = 0; j0 < n; j0 += 8) {
      uint32_t w[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) w[u] = p.pub[(int64_t)(b0 + imin(j0 + u, n - 1)) * E + e];   // (16-bit loads)
#pragma unroll
      for (int u = 0; u < 8; ++u) sum += j0 + u < n ? (int)w[u] : 0;
    }
    gs[t] = sum;
  }
  __syncthreads();
  for (int e = tid; e < E; e += nt) {
    int sum = 0;
    for (int g = 0; g < groups; ++g) sum += gs[g * E + e];
    run[e] = from_start ? sum : (int)gh[e] - sum;
  }
}

// Send-buffer slots of a chunk of the one-launch plan, with three barriers:
// the counts per rank before the chunk (from run[e] and the instance list,
// into excl, zeroed with the instance-list load) and each wave's ranks by
// destination (its own row of wc, stride E, which only it read before) are
// made together; the wave offsets per rank come from one 16-lane scan per
// rank (lane w of a row holds wave w's count); then the slots.  offs: the
// send offsets.
template <int IPT>
__device__ __forceinline__ void chunk_slots(const Plan &p, const int (&dv)[IPT], int64_t wbase, int64_t hi,
                                            const int *run, const int *ptr, const int2 *ent,
                                            const int *offs, int *excl, int *wc) {
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6, lane = tid & 63, wave = tid >> 6;
  const int R = p.R, E = p.E;
  for (int e = tid; e < E; e += nt) {
    const int re = run[e], j1 = ptr[e + 1];
    int start = 0;
    for (int j = ptr[e]; j < j1; ++j) {
      const int end = ent[j].x, rk = ent[j].y;
      const int c = imin(imax(re - start, 0), end - start);
      if (c > 0 && (unsigned)rk < (unsigned)R) atomicAdd(&excl[rk], c);
      start = end;
    }
  }
  int *mw = wc + wave * E;
  wave_sync();
  for (int r = lane; r < R; r += 64) mw[r] = 0;
  wave_sync();
  int lr[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    // (dv is -1 past the end)
    lr[i] = wave_rank(dv[i], (unsigned)dv[i] < (unsigned)R, p.rbits, mw);
  }
  lds_barrier();
  // lane w of the row of rank r: wave w's count, scanned across the row
  const int rows = R * 16, span = (rows + 63) & ~63;
  for (int t = tid; t < span; t += nt) {
    const int r = t >> 4, w = t & 15;
    const bool in = t < rows && w < nw;
    const int c = in ? wc[w * E + r] : 0;
    const int incl = row16_incl_scan(c);
    if (in) wc[w * E + r] = incl - c;
  }
  lds_barrier();
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int64_t idx = wbase + i * 64;
    if (idx < hi) {
      const int d = dv[i];
      p.slot_out[idx] = (unsigned)d < (unsigned)R ? offs[d] + excl[d] + mw[d] + lr[i] : -1;
    }
  }
}

// Chunk role (workgroup 1 + b): ids [b * chunk, (b + 1) * chunk) stay in
// registers for the whole plan.  Each wave ranks its ids among equal ids
// (row-major order); the workgroup writes its counts, adds them to the
// histogram and arrives (the last to arrive announces that every count is
// written and sends the verdict); it then sums its first occurrence index
// per expert; once the plan is ready each id's occurrence index rho =
// (offset of the chunk) + (offset of the wave in the chunk) + (rank in the
// wave) picks the instance from this rank's instance list.  A bounded wait
// that gives up writes -1 and SYNC.
template <int IPT>
__device__ __forceinline__ void fused_chunk(const Plan &p, int b, int *sm) {
  const ChunkLds l = chunk_lds(p, blockDim.x);
  int *wc = sm + l.wc, *run = sm + l.run, *ptr = sm + l.ptr;
  int2 *ent = reinterpret_cast<int2 *>(sm + l.ent);
  int *gs = sm + l.gs, *so = sm + l.so, *flag = sm + l.flag;
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6, lane = tid & 63, wave = tid >> 6;
  const int E = p.E;
  const int64_t lo = (int64_t)b * p.chunk;
  const int64_t hi = lo + p.chunk < p.n ? lo + p.chunk : p.n;
  const int64_t wbase = lo + (int64_t)wave * 64 * IPT + lane;
  int ev[IPT], lr[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int64_t idx = wbase + i * 64;
    ev[i] = idx < hi ? p.topk[idx] : -1;
  }
  // the generation as the solver left it: the histogram buffer to add to
  const uint32_t gread = __hip_atomic_load(&p.ctrl[kCtrlGen], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  int *mywc = wc + wave * E;
  for (int e = lane; e < E; e += 64) mywc[e] = 0;
  wave_sync();
  int bad = 0;
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int64_t idx = wbase + i * 64;
    const bool inr = idx < hi;
    const bool valid = (unsigned)ev[i] < (unsigned)E;   // (ev is -1 past the end)
    bad |= (inr && !valid) ? 1 : 0;
    lr[i] = wave_rank(ev[i], valid, p.nbits, mywc);
  }
  bad = __syncthreads_or(bad);
  // publish the chunk's counts; wc becomes each wave's offset in the chunk
  uint32_t *gh = p.ghist + (gread & 1u) * (E + 1);
  for (int e = tid; e < E; e += nt) {
    int sum = 0;
    for (int w = 0; w < nw; ++w) {
      const int c = wc[w * E + e];
      wc[w * E + e] = sum;
      sum += c;
    }
    p.pub[(int64_t)b * E + e] = (uint16_t)sum;
    if (sum) atomicAdd(gh + e, (uint32_t)sum);
  }
  if (tid == 0 && bad) atomicAdd(gh + E, 1u);
  drain_then_barrier();
  if (tid == 0) {
    const uint64_t before = __hip_atomic_fetch_add(reinterpret_cast<unsigned long long *>(p.ctrl + kCtrlArrive), 1ull,
                                                   __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t g = div_u64_small(before, (uint32_t)p.nb);
    const bool last = before - g * (uint64_t)p.nb == (uint64_t)(p.nb - 1);
    // the last arrival acquires every other chunk's counts
    if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    flag[1] = last;
    flag[2] = (int)(uint32_t)g;
  }
  __syncthreads();
  if (b == 0) STAMP(p, 12);
  const uint32_t gen = (uint32_t)flag[2];
  if (gen != gread) {
    // the solver has already given up on this plan and moved on: take the
    // adds back out of the next plan's buffer (it starts after this kernel)
    for (int e = tid; e < E; e += nt) {
      const uint32_t c = p.pub[(int64_t)b * E + e];
      if (c) atomicSub(gh + e, c);
    }
    if (tid == 0 && bad) atomicSub(gh + E, 1u);
  }
  if (flag[1]) {
    STAMP(p, 19);
    last_arrival(p, gen);
    STAMP(p, 13);
    STAMP_FLUSH(p, 13, 14);
    STAMP_FLUSH(p, 19, 20);
  }
  // every count is written: this chunk's first occurrence index per expert
  bool ok = wait_flag(p, b, 1, gen + 1u, flag);
  if (ok) chunk_offsets(p, b, p.ghist + (gen & 1u) * (E + 1), run, gs);
  if (b == 0) STAMP(p, 16);
  // each id's occurrence index rho = chunk offset + wave offset + rank in
  // the wave, while the plan is still being made
  __syncthreads();
  int rho[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int e = (unsigned)ev[i] < (unsigned)E ? ev[i] : 0;
    rho[i] = run[e] + wc[wave * E + e] + lr[i];
  }
  // the plan is ready
  ok = ok && wait_flag(p, b, 0, gen + 1u, flag);
  if (b == 0) STAMP(p, 14);
  uint32_t fin = 0;
  if (ok) {
    // the instance list and the final status in one round trip: every load
    // of a pass issued before any is used
    fin = __hip_atomic_load(&p.ctrl[kCtrlFinal], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int n_ld = imax(E + 1, p.nent_cap);
    for (int i = tid; i < n_ld; i += nt) {
      const int pv = p.csr_ptr[imin(i, E)];
      const int rv = p.csr_r[imin(i, p.nent_cap - 1)];
      const int xv = p.csr_end[imin(i, p.nent_cap - 1)];
      if (i <= E) ptr[i] = pv < 0 ? 0 : (pv > p.nent_cap ? p.nent_cap : pv);
      if (i < p.nent_cap) ent[i] = make_int2(xv, rv);
    }
    if (p.slot_out) {
      // the send offsets (the solver wrote them) in the same round trip;
      // the per-rank counts before this chunk start from zero
      for (int r = tid; r < p.R; r += nt) {
        so[r] = p.offs_out[r];
        gs[r] = 0;
      }
    }
  }
  if (!ok || (fin & (kNoPlan | TOPOEP_ST_SYNC))) {
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = wbase + i * 64;
      if (idx < hi) {
        p.dest_out[idx] = -1;
        if (p.slot_out) p.slot_out[idx] = -1;
      }
    }
    if (b == 0 && p.offs_out)
      for (int r = tid; r <= p.R; r += nt) p.offs_out[r] = 0;
    if (!ok && tid == 0) atomicOr(reinterpret_cast<unsigned *>(p.status_out), TOPOEP_ST_SYNC);
    return;
  }
  __syncthreads();
  int dv[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int64_t idx = wbase + i * 64;
    int dest = -1;
    if (idx < hi) {
      if ((unsigned)ev[i] < (unsigned)E) {
        const int j1 = ptr[ev[i] + 1];
        for (int j = ptr[ev[i]]; j < j1; ++j) {
          const int2 en = ent[j];
          if (rho[i] < en.x) {
            dest = en.y;
            break;
          }
        }
      }
      p.dest_out[idx] = dest;
    }
    dv[i] = dest;
  }
  if (p.slot_out) chunk_slots<IPT>(p, dv, wbase, hi, run, ptr, ent, so, gs, wc);
  if (b == 0) {
    STAMP(p, 15);
    STAMP_FLUSH(p, 12, 13);
    STAMP_FLUSH(p, 14, 17);
  }
}

// The whole plan in one launch: workgroup 0 solves, workgroups 1..nb hold
// the ids; all are resident at once (nb <= kMaxFusedBlocks) and every wait
// is bounded.
// Form: the refinement's form for the shape (refine_form: registers with
// (instance, target) pairs, registers, or LDS); one instantiation each keeps
// the others' registers out.
template <int IPT, int Form>
__global__ __launch_bounds__(1024) void plan_fused_kernel(Plan p) {
  extern __shared__ int64_t smem_f[];
  int *sm = reinterpret_cast<int *>(smem_f);
  (void)p;
  if (blockIdx.x == 0) {
    const Plan q = solver_plan(role_plan(p));
    fused_solver<Form>(q, sm);
  } else {
    const Plan q = role_plan(p);
    fused_chunk<IPT>(q, blockIdx.x - 1, sm);
  }
}

// Same launch shape, empty body: the launch floor of a plan's kernel.
__global__ __launch_bounds__(1024) void empty_kernel(Plan p) { (void)p; }

// ---------------------------------------------------------------- host side

struct Shape {
  int ipt, bt, st;
  size_t zero_bytes;   // workspace prefix that must be zero before a first plan
  int mode;       // 1 single-workgroup solver, 2 per-domain solver (three kernels each), 3 one launch
  size_t lds_hist, lds_solve, lds_reroute, lds_fused;
  int solve_groups;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int ceil_log2(int v) {
  int b = 0;
  while ((1 << b) < v) ++b;
  return b;
}

template <typename K>
void allow_lds(K kernel) {
  (void)hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, kLdsLimit);
}

void set_attrs();

// Workgroups of one kernel shape that the current device keeps resident at
// once: its compute units times the shape's occupancy per unit.  Kernels
// whose workgroups wait on each other (the one-launch plan, the per-domain
// solver's grid barrier) are only chosen when every workgroup fits.  A
// device that cannot be queried (no GPU: sizes only) counts as gfx950's
// 256 compute units with one workgroup each, which every shape within the
// LDS and thread limits checked here reaches.  Results are cached.
int resident_capacity(const void *fn, int threads, size_t lds) {
  struct Entry {
    int dev;
    const void *fn;
    int threads;
    size_t lds;
    int cap;
  };
  static std::mutex mu;
  static std::vector<Entry> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return 256;
  }
  {
    std::lock_guard<std::mutex> lock(mu);
    for (const Entry &e : cache)
      if (e.dev == dev && e.fn == fn && e.threads == threads && e.lds == lds) return e.cap;
  }
  set_attrs();
  int cus = 0, occ = 0;
  int cap = 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0 &&
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, threads, lds) == hipSuccess)
    cap = cus * occ;
  (void)hipGetLastError();   // a failed query is not the caller's error
  std::lock_guard<std::mutex> lock(mu);
  cache.push_back(Entry{dev, fn, threads, lds, cap});
  return cap;
}

const void *fused_fn(int ipt, int form);

// Validate the arguments and fill the plan's sizes, launch shape and
// workspace layout (pointers are offsets when ws == nullptr).
int setup(const topoep_topology *t, int32_t T, int32_t k, int32_t N, const topoep_launch *lc, Plan *p,
          Shape *sh, size_t *ws_bytes, char *ws, bool general = false) {
  if (!t) return TOPOEP_EINVAL;
  const int R = t->num_ranks, G = t->ranks_per_node, E = t->num_experts;
  if (R <= 0 || G <= 0 || E <= 0 || R % G != 0 || E % R != 0) return TOPOEP_EINVAL;
  if (k < 1 || k > E || T < 0 || (int64_t)T * k > 0x7FFFFFFF || N < 0) return TOPOEP_EINVAL;
  if (t->self_rank < 0 || t->self_rank >= R) return TOPOEP_EINVAL;
  if (t->cost_intra < 0 || t->cost_inter < 0 || t->tok_bytes <= 0 || t->expert_bytes < 0) return TOPOEP_EINVAL;
  if (G > 64) return TOPOEP_ELIMIT;
  Plan q = {};
  q.R = R;
  q.G = G;
  q.M = R / G;
  q.E = E;
  q.P = E / R;
  q.N = N;
  q.Neff = imin(N, E - q.P);
  q.PN = q.P + q.Neff;
  q.I = G * q.PN;
  q.self = t->self_rank;
  q.MW = (q.M + 31) / 32;
  q.RW = (R + 31) / 32;
  q.nbits = ceil_log2(E);
  q.rbits = ceil_log2(R);
  q.cap1 = G * q.Neff;
  q.nent_cap = E + R * q.Neff;
  // odd row stride of the q columns (no LDS bank conflicts) with at least
  // one spare word after the R sources
  q.QS = (R + 1) | 1;
  q.cI = t->cost_intra;
  q.cX = t->cost_inter;
  q.S = t->tok_bytes;
  q.W = t->expert_bytes;
  {
    // the two-level model's range threshold (out_of_range): exact in 128 bits
    const unsigned __int128 lim = (unsigned __int128)1 << 62;
    const uint64_t cm = (uint64_t)imax(imax(q.cI, q.cX), 1);
    const unsigned __int128 rep = (unsigned __int128)(uint64_t)q.W * cm;
    const unsigned __int128 kk = (unsigned __int128)4 * (uint64_t)q.S * cm;
    q.tot_max = rep >= lim ? 0 : (uint64_t)((lim - rep + kk - 1) / kk);
  }
  q.n = (int64_t)T * k;
  q.spin_limit = kSpinLimit;
  q.iter_limit = kIterLimit;
  if (lc) {
    if (lc->spin_limit < -1 || lc->iter_limit < 0) return TOPOEP_EINVAL;
    if (lc->spin_limit == -1) q.spin_limit = 0;   // every bounded wait gives up at once
    else if (lc->spin_limit > 0) q.spin_limit = (uint32_t)lc->spin_limit;
    if (lc->iter_limit > 0) q.iter_limit = (uint32_t)lc->iter_limit;
  }
  q.general = general ? 1 : 0;
  if (general && R > 65535) return TOPOEP_ELIMIT;
  if ((int64_t)q.M * q.I * q.QS >= (1 << 30) || (int64_t)R * E >= (1 << 30)) return TOPOEP_ELIMIT;
  q.fE = make_fastdiv((uint32_t)E);
  q.fG = make_fastdiv((uint32_t)G);
  q.fGP = make_fastdiv((uint32_t)(G * q.P));
  q.fP = make_fastdiv((uint32_t)q.P);
  q.fI = make_fastdiv((uint32_t)q.I);
  q.fPN = make_fastdiv((uint32_t)q.PN);
  q.fCap = make_fastdiv((uint32_t)imax(q.cap1, 1));
  q.fN = make_fastdiv((uint32_t)imax(N, 1));
  q.fMI = make_fastdiv((uint32_t)(q.M * q.I));

  Shape s;
  const int ipt_req = lc ? lc->items_per_thread : 0;
  s.ipt = ipt_req ? ipt_req : (q.n >= ((int64_t)1 << 24) ? 8 : 4);   // 8 ids per thread measured ~3 % faster from 2^24 on
  s.bt = lc && lc->block_threads ? lc->block_threads : 256;
  s.st = lc && lc->solve_threads ? lc->solve_threads : 0;
  const int solver = lc ? lc->solver : 0;
  if (solver < 0 || solver > 3) return TOPOEP_EINVAL;
  if (!(s.ipt == 1 || s.ipt == 2 || s.ipt == 4 || s.ipt == 8)) return TOPOEP_EINVAL;
  if (s.bt < 64 || s.bt > 1024 || s.bt % 64) return TOPOEP_EINVAL;
  if (s.st != 0 && (s.st < 64 || s.st > 1024 || s.st % 64)) return TOPOEP_EINVAL;
  if (lc && lc->tiles_per_block < 0) return TOPOEP_EINVAL;

  // the single-workgroup solver when its whole state fits in LDS
  const int64_t single_words = (int64_t)single_lds(q).words;
  const int64_t multi_words = (int64_t)domain_lds(q).words;
  const bool single_fits = single_words * 4 <= kLdsLimit;
  const bool multi_fits = multi_words * 4 <= kLdsLimit;

  // one launch: the single-workgroup solver plus at most kMaxFusedBlocks
  // chunk workgroups of st threads holding ipt ids per thread
  {
    const int st = s.st ? s.st : 1024;
    int ipt = 0;
    int64_t nbf = 0;
    for (int c = 1; c <= 8; c *= 2) {
      if (ipt_req && c != ipt_req) continue;
      const int64_t nbc = q.n > 0 ? (q.n + (int64_t)st * c - 1) / ((int64_t)st * c) : 1;
      if (nbc <= kMaxFusedBlocks && (ipt == 0 || nbf > kFusedBlocks)) {
        ipt = c;
        nbf = nbc;
      }
    }
    const int64_t chunk_words = (int64_t)chunk_lds(q, st).words;
    // (1 KiB left for the kernel's static LDS, which __syncthreads_or uses)
    const int64_t fused_words = single_words > chunk_words ? single_words : chunk_words;
    bool fused_ok = single_fits && ipt > 0 && fused_words * 4 + 1024 <= kLdsLimit;
    // every workgroup of the launch resident at once (they wait on each other)
    if (fused_ok)
      fused_ok = nbf + 1 <= resident_capacity(fused_fn(ipt, refine_form(q.G, q.I, q.PN)), st, (size_t)fused_words * 4);
    if (solver == 3 && !fused_ok) return TOPOEP_ELIMIT;
    if (general && solver == 3) return TOPOEP_EINVAL;   // the general model runs the per-domain solver
    if (fused_ok && !general && (solver == 3 || solver == 0)) {
      s.mode = 3;
      s.ipt = ipt;
      s.st = st;
      q.chunk = (int64_t)st * ipt;
      q.nb = (int)nbf;
      q.n_solvers = 1;
      q.n_helpers = 0;
      s.solve_groups = 1;
      s.lds_hist = s.lds_solve = s.lds_reroute = 0;
      s.lds_fused = (size_t)fused_words * 4;
    } else {
      s.mode = 0;
    }
  }

  if (s.mode != 3) {
  const int64_t tile = (int64_t)s.bt * s.ipt;
  const int64_t tiles = (q.n + tile - 1) / tile;
  // about 16 K ids per block, 2048..8192 blocks: every CU keeps eight
  // 256-thread blocks resident with work to spare, while the solver's
  // per-block offset scan (nb words per expert) stays short
  const int64_t want = q.n / 16384;
  const int64_t target = want < kMinBlocks ? kMinBlocks : (want > kMaxBlocks ? kMaxBlocks : want);
  int64_t tpb = lc && lc->tiles_per_block > 0 ? lc->tiles_per_block : (tiles + target - 1) / target;
  if (tpb < 1) tpb = 1;
  q.chunk = tpb * tile;
  const int64_t nb = q.n > 0 ? (q.n + q.chunk - 1) / q.chunk : 1;
  if (nb > (1 << 24)) return TOPOEP_ELIMIT;
  q.nb = (int)nb;
  q.n_helpers = (E + kOffsetExperts - 1) / kOffsetExperts;
  if (general) {
    if (solver == 1) return TOPOEP_EINVAL;
    if (!multi_fits) return TOPOEP_ELIMIT;
    s.mode = 2;
  } else if (solver == 1) {
    if (!single_fits) return TOPOEP_ELIMIT;
    s.mode = 1;
  } else if (solver == 2) {
    if (!multi_fits) return TOPOEP_ELIMIT;
    s.mode = 2;
  } else {
    if (!single_fits && !multi_fits) return TOPOEP_ELIMIT;
    s.mode = single_fits ? 1 : 2;
  }
  if (s.st == 0) s.st = s.mode == 1 ? 1024 : 512;
  s.lds_solve = (size_t)(s.mode == 1 ? single_words : multi_words) * 4;
  q.n_solvers = s.mode == 1 ? 1 : imin(q.M, kMaxSolveGroups);
  // the per-domain solver's workgroups meet at a grid barrier: all resident
  if (s.mode == 2 && q.n_solvers > resident_capacity(s.st <= 512 ? reinterpret_cast<const void *>(solve_kernel<512>)
                                                                  : reinterpret_cast<const void *>(solve_kernel<1024>),
                                                     s.st, s.lds_solve))
    return TOPOEP_ELIMIT;
  s.solve_groups = q.n_solvers + q.n_helpers;
  s.lds_hist = (size_t)E * 4;
  // instance entries, cursors, per-wave (count, entry) pairs, run, ptr,
  // per-wave rank counts, counts before the tile, send offsets and scratch
  s.lds_reroute = (2 * ((size_t)q.nent_cap + 1) + 2 * (size_t)E + 2 * (size_t)(E | 1) * (s.bt / 64) + (size_t)E +
                   (size_t)E + 1 + (size_t)(R | 1) * (s.bt / 64) + (size_t)R + (size_t)R + 1 + s.bt / 64 + 1) * 4;
  s.lds_fused = 0;
  if (s.lds_reroute > (size_t)kLdsLimit) return TOPOEP_ELIMIT;
  }

  // routing: the largest divisor c of M with (instances routed at once) * c
  // <= solver threads, so every thread routes whole source domains
  auto chunks_for = [&](int64_t ni) {
    int best = 1;
    for (int c = 1; c <= q.M; ++c)
      if (q.M % c == 0 && ni * c <= s.st) best = c;
    return best;
  };
  q.rchunks_all = chunks_for((int64_t)q.M * q.I);
  q.rchunks_dom = chunks_for(q.I);

  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  // every word a plan needs zero before its first use sits in the prefix
  // [0, zero_bytes): the control words, then (one launch) the ready flags
  const bool one = s.mode == 3;
  const bool three = !one;
  const size_t o_ctrl = take(kCtrlBytes);
  const size_t o_flg = take(one ? (size_t)q.nb * kFlagStride * 4 : 0);
  const size_t o_gh = take(one ? (size_t)2 * (E + 1) * 4 : 0);
  s.zero_bytes = off;
  const size_t o_part = take(three ? (size_t)q.nb * E * 4 : 0);
  const size_t o_offs = take(three ? (size_t)q.nb * E * 4 : 0);
  const size_t o_berr = take(three ? (size_t)q.nb * 4 : 0);
  const size_t o_repl = take(s.mode == 2 ? (size_t)q.M * imax(q.cap1, 1) * 4 : 0);
  const size_t o_sege = take(s.mode == 2 ? (size_t)q.M * q.I * 4 : 0);
  const size_t o_segq = take(s.mode == 2 ? (size_t)q.M * q.I * 4 : 0);
  const size_t o_cptr = take((size_t)(E + 1) * 4);
  const size_t o_cr = take((size_t)q.nent_cap * 4);
  const size_t o_ce = take((size_t)q.nent_cap * 4);
  const size_t o_ht = take(three ? (size_t)E * 4 : 0);
  const size_t o_pub = take(one ? (size_t)q.nb * E * 2 : 0);
  *ws_bytes = off;
  if (ws) {
    auto at = [&](size_t o, bool have) { return have ? reinterpret_cast<int32_t *>(ws + o) : nullptr; };
    auto atu = [&](size_t o, bool have) { return have ? reinterpret_cast<uint32_t *>(ws + o) : nullptr; };
    q.ctrl = atu(o_ctrl, true);
    q.partials = at(o_part, three);
    q.offsets = at(o_offs, three);
    q.blk_err = at(o_berr, three);
    q.repl1 = at(o_repl, s.mode == 2);
    q.seg_e = at(o_sege, s.mode == 2);
    q.seg_q = at(o_segq, s.mode == 2);
    q.csr_ptr = at(o_cptr, true);
    q.csr_r = at(o_cr, true);
    q.csr_end = at(o_ce, true);
    q.htot = at(o_ht, three);
    q.flags = atu(o_flg, one);
    q.pub = one ? reinterpret_cast<uint16_t *>(ws + o_pub) : nullptr;
    q.ghist = atu(o_gh, one);
  }
  *p = q;
  *sh = s;
  return TOPOEP_OK;
}

std::atomic<bool> g_attrs_set{false};

template <int IPT>
const void *fused_fn_ipt(int form) {
  return form == kRefinePairs ? reinterpret_cast<const void *>(plan_fused_kernel<IPT, kRefinePairs>)
         : form == kRefineReg ? reinterpret_cast<const void *>(plan_fused_kernel<IPT, kRefineReg>)
                              : reinterpret_cast<const void *>(plan_fused_kernel<IPT, kRefineLds>);
}

const void *fused_fn(int ipt, int form) {
  switch (ipt) {
    case 1: return fused_fn_ipt<1>(form);
    case 2: return fused_fn_ipt<2>(form);
    case 4: return fused_fn_ipt<4>(form);
    default: return fused_fn_ipt<8>(form);
  }
}

void set_attrs() {
  if (g_attrs_set) return;
  allow_lds(hist_kernel<1>);
  allow_lds(hist_kernel<2>);
  allow_lds(hist_kernel<4>);
  allow_lds(hist_kernel<8>);
  allow_lds(reroute_kernel<1>);
  allow_lds(reroute_kernel<2>);
  allow_lds(reroute_kernel<4>);
  allow_lds(reroute_kernel<8>);
  allow_lds(solve_kernel<512>);
  allow_lds(solve_kernel<1024>);
  allow_lds(solve_single_kernel);
  allow_lds(plan_fused_kernel<1, kRefineLds>);
  allow_lds(plan_fused_kernel<1, kRefineReg>);
  allow_lds(plan_fused_kernel<1, kRefinePairs>);
  allow_lds(plan_fused_kernel<2, kRefineLds>);
  allow_lds(plan_fused_kernel<2, kRefineReg>);
  allow_lds(plan_fused_kernel<2, kRefinePairs>);
  allow_lds(plan_fused_kernel<4, kRefineLds>);
  allow_lds(plan_fused_kernel<4, kRefineReg>);
  allow_lds(plan_fused_kernel<4, kRefinePairs>);
  allow_lds(plan_fused_kernel<8, kRefineLds>);
  allow_lds(plan_fused_kernel<8, kRefineReg>);
  allow_lds(plan_fused_kernel<8, kRefinePairs>);
  allow_lds(empty_kernel);
  // (an attribute a kernel refuses must not linger as the caller's error)
  (void)hipGetLastError();
  g_attrs_set = true;
}

void launch_hist(const Plan &p, const Shape &s, hipStream_t st) {
  const dim3 g(p.nb), b(s.bt);
  switch (s.ipt) {
    case 1: hipLaunchKernelGGL(hist_kernel<1>, g, b, s.lds_hist, st, p); break;
    case 2: hipLaunchKernelGGL(hist_kernel<2>, g, b, s.lds_hist, st, p); break;
    case 4: hipLaunchKernelGGL(hist_kernel<4>, g, b, s.lds_hist, st, p); break;
    default: hipLaunchKernelGGL(hist_kernel<8>, g, b, s.lds_hist, st, p); break;
  }
}

void launch_reroute(const Plan &p, const Shape &s, hipStream_t st) {
  const dim3 g(p.nb), b(s.bt);
  switch (s.ipt) {
    case 1: hipLaunchKernelGGL(reroute_kernel<1>, g, b, s.lds_reroute, st, p); break;
    case 2: hipLaunchKernelGGL(reroute_kernel<2>, g, b, s.lds_reroute, st, p); break;
    case 4: hipLaunchKernelGGL(reroute_kernel<4>, g, b, s.lds_reroute, st, p); break;
    default: hipLaunchKernelGGL(reroute_kernel<8>, g, b, s.lds_reroute, st, p); break;
  }
}

void launch_solve(const Plan &p, const Shape &s, hipStream_t st) {
  if (s.mode == 1) hipLaunchKernelGGL(solve_single_kernel, dim3(s.solve_groups), dim3(s.st), s.lds_solve, st, p);
  else if (s.st <= 512) hipLaunchKernelGGL(solve_kernel<512>, dim3(s.solve_groups), dim3(s.st), s.lds_solve, st, p);
  else hipLaunchKernelGGL(solve_kernel<1024>, dim3(s.solve_groups), dim3(s.st), s.lds_solve, st, p);
}

template <int IPT>
void launch_fused_ipt(int form, dim3 g, dim3 b, size_t lds, hipStream_t st, const Plan &p) {
  if (form == kRefinePairs) hipLaunchKernelGGL((plan_fused_kernel<IPT, kRefinePairs>), g, b, lds, st, p);
  else if (form == kRefineReg) hipLaunchKernelGGL((plan_fused_kernel<IPT, kRefineReg>), g, b, lds, st, p);
  else hipLaunchKernelGGL((plan_fused_kernel<IPT, kRefineLds>), g, b, lds, st, p);
}

void launch_fused(const Plan &p, const Shape &s, hipStream_t st) {
  const dim3 g(p.nb + 1), b(s.st);
  const int form = refine_form(p.G, p.I, p.PN);
  switch (s.ipt) {
    case 1: launch_fused_ipt<1>(form, g, b, s.lds_fused, st, p); break;
    case 2: launch_fused_ipt<2>(form, g, b, s.lds_fused, st, p); break;
    case 4: launch_fused_ipt<4>(form, g, b, s.lds_fused, st, p); break;
    default: launch_fused_ipt<8>(form, g, b, s.lds_fused, st, p); break;
  }
}

// Kernels of one plan in launch order: grid, threads, dynamic LDS.
int plan_kernels(const Plan &p, const Shape &s, int grid[3], int block[3], size_t lds[3]) {
  if (s.mode == 3) {
    grid[0] = p.nb + 1;
    block[0] = s.st;
    lds[0] = s.lds_fused;
    return 1;
  }
  grid[0] = p.nb;
  block[0] = s.bt;
  lds[0] = s.lds_hist;
  grid[1] = s.solve_groups;
  block[1] = s.st;
  lds[1] = s.lds_solve;
  grid[2] = p.nb;
  block[2] = s.bt;
  lds[2] = s.lds_reroute;
  return 3;
}

constexpr int kFloorMask = 8;

int enqueue(int stage_mask, const topoep_topology *topo, const int32_t *global_load,
            const int32_t *local_topk, int32_t T, int32_t k, int32_t N, int32_t *replica_slots,
            int32_t *token_dest, int32_t *send_counts, int32_t *status, void *workspace,
            size_t workspace_bytes, void *stream, const topoep_launch *launch,
            int32_t *recv_counts = nullptr, int32_t *send_offsets = nullptr, int32_t *token_slot = nullptr,
            const topoep_costs *costs = nullptr) {
  Plan p;
  Shape s;
  size_t need = 0;
  const bool general = costs != nullptr;
  int rc = setup(topo, T, k, N, launch, &p, &s, &need, nullptr, general);
  if (rc != TOPOEP_OK) return rc;
  if (!global_load || !send_counts || !status || !workspace) return TOPOEP_EINVAL;
  if ((int64_t)topo->num_ranks * N > 0 && !replica_slots) return TOPOEP_EINVAL;
  if (T > 0 && (!local_topk || !token_dest)) return TOPOEP_EINVAL;
  if (workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return TOPOEP_EWORKSPACE;
  rc = setup(topo, T, k, N, launch, &p, &s, &need, static_cast<char *>(workspace), general);
  if (rc != TOPOEP_OK) return rc;
  p.Cm = general ? costs->cost : nullptr;
  p.We = general ? costs->expert_bytes : nullptr;
  p.gl = global_load;
  p.topk = local_topk;
  p.slots_out = replica_slots;
  p.dest_out = token_dest;
  p.send_out = send_counts;
  p.status_out = status;
  p.recv_out = recv_counts;
  p.offs_out = send_offsets;
  p.slot_out = send_offsets ? token_slot : nullptr;   // (null when T == 0: offsets only)
  set_attrs();
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (stage_mask == kFloorMask) {
    int grid[3], block[3];
    size_t lds[3];
    const int nk = plan_kernels(p, s, grid, block, lds);
    for (int i = 0; i < nk; ++i) hipLaunchKernelGGL(empty_kernel, dim3(grid[i]), dim3(block[i]), lds[i], st, p);
  } else if (s.mode == 3) {
    if (stage_mask != 7 && stage_mask != 1) return TOPOEP_EINVAL;   // one kernel: the plan, or stage 0
    launch_fused(p, s, st);
  } else {
    if (stage_mask & 1) launch_hist(p, s, st);
    if (stage_mask & 2) launch_solve(p, s, st);
    if (stage_mask & 4) launch_reroute(p, s, st);
  }
  return hipGetLastError() == hipSuccess ? TOPOEP_OK : TOPOEP_EHIP;
}

// ---------------------------------------------------------------- no-allocation entry point
//
// topoep_plan_noalloc plans into `scratch`, a device array of fixed size in
// place of a caller's workspace: one copy per GPU the library runs on, held
// until the process ends.  In host code the array's name is only a
// host-side stand-in; kernels and the clearing launch get the device
// address hipGetSymbolAddress returns for the current device, looked up
// once per device and kept.

constexpr size_t kScratchBytes = TOPOEP_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

int scratch_address(void **out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return TOPOEP_EHIP;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) {
      (void)hipGetLastError();
      return TOPOEP_EHIP;
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return TOPOEP_OK;
}

// Zero n words (the workspace prefix a first plan needs zero): a kernel, so
// that the clearing can be captured in a HIP graph like the plan itself.
__global__ __launch_bounds__(256) void zero_words(uint32_t *w, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    w[i] = 0u;
}

}  // namespace

extern "C" {

int topoep_plan_noalloc(const topoep_topology *topo, const int32_t *global_load, const int32_t *local_topk,
                        int32_t T, int32_t k, int32_t replica_budget, int32_t *replica_slots, int32_t *token_dest,
                        int32_t *send_counts, int32_t *status, void *stream) {
  Plan p;
  Shape s;
  size_t need = 0;
  int rc = setup(topo, T, k, replica_budget, nullptr, &p, &s, &need, nullptr);
  if (rc != TOPOEP_OK) return rc;
  // the argument checks of topoep_plan, before anything is enqueued
  if (!global_load || !send_counts || !status) return TOPOEP_EINVAL;
  if ((int64_t)topo->num_ranks * replica_budget > 0 && !replica_slots) return TOPOEP_EINVAL;
  if (T > 0 && (!local_topk || !token_dest)) return TOPOEP_EINVAL;
  if (need > kScratchBytes) return TOPOEP_EWORKSPACE;
  void *ws = nullptr;
  rc = scratch_address(&ws);
  if (rc != TOPOEP_OK) return rc;
  // the previous call may have been another shape: clear what this plan
  // needs zero (control words, flags, histogram buffers)
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const int64_t words = (int64_t)(s.zero_bytes / 4);
  hipLaunchKernelGGL(zero_words, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, st, static_cast<uint32_t *>(ws),
                     words);
  if (hipGetLastError() != hipSuccess) return TOPOEP_EHIP;
  return enqueue(7, topo, global_load, local_topk, T, k, replica_budget, replica_slots, token_dest, send_counts,
                 status, ws, kScratchBytes, stream, nullptr);
}

int topoep_workspace_bytes_ex(const topoep_topology *topo, int32_t T, int32_t k, int32_t replica_budget,
                              const topoep_launch *launch, size_t *bytes_out) {
  if (!bytes_out) return TOPOEP_EINVAL;
  Plan p;
  Shape s;
  size_t need = 0;
  const int rc = setup(topo, T, k, replica_budget, launch, &p, &s, &need, nullptr);
  if (rc == TOPOEP_OK) *bytes_out = need;
  return rc;
}

int topoep_workspace_bytes(const topoep_topology *topo, int32_t T, int32_t k, int32_t replica_budget,
                           size_t *bytes_out) {
  return topoep_workspace_bytes_ex(topo, T, k, replica_budget, nullptr, bytes_out);
}

int topoep_plan_ex(const topoep_topology *topo, const int32_t *global_load, const int32_t *local_topk,
                   int32_t T, int32_t k, int32_t replica_budget, int32_t *replica_slots,
                   int32_t *token_dest, int32_t *send_counts, int32_t *status, void *workspace,
                   size_t workspace_bytes, void *stream, const topoep_launch *launch) {
  return enqueue(7, topo, global_load, local_topk, T, k, replica_budget, replica_slots, token_dest,
                 send_counts, status, workspace, workspace_bytes, stream, launch);
}

int topoep_plan_shape(const topoep_topology *topo, int32_t T, int32_t k, int32_t replica_budget,
                      const topoep_launch *launch, topoep_shape *out) {
  if (!out) return TOPOEP_EINVAL;
  Plan p;
  Shape s;
  size_t need = 0;
  const int rc = setup(topo, T, k, replica_budget, launch, &p, &s, &need, nullptr);
  if (rc != TOPOEP_OK) return rc;
  int grid[3] = {0, 0, 0}, block[3] = {0, 0, 0};
  size_t lds[3] = {0, 0, 0};
  topoep_shape o = {};
  o.kernels = plan_kernels(p, s, grid, block, lds);
  o.solver = s.mode;
  o.items_per_thread = s.ipt;
  o.chunk_blocks = p.nb;
  for (int i = 0; i < 3; ++i) {
    o.grid[i] = grid[i];
    o.block[i] = block[i];
    o.lds_bytes[i] = (int32_t)lds[i];
  }
  *out = o;
  return TOPOEP_OK;
}

int topoep_plan(const topoep_topology *topo, const int32_t *global_load, const int32_t *local_topk,
                int32_t T, int32_t k, int32_t replica_budget, int32_t *replica_slots, int32_t *token_dest,
                int32_t *send_counts, int32_t *status, void *workspace, size_t workspace_bytes,
                void *stream) {
  return enqueue(7, topo, global_load, local_topk, T, k, replica_budget, replica_slots, token_dest,
                 send_counts, status, workspace, workspace_bytes, stream, nullptr);
}

int topoep_dispatch_workspace_bytes(const topoep_topology *topo, int32_t T, int32_t k, int32_t replica_budget,
                                    size_t *bytes_out) {
  return topoep_workspace_bytes_ex(topo, T, k, replica_budget, nullptr, bytes_out);
}

int topoep_plan_dispatch(const topoep_topology *topo, const int32_t *global_load, const int32_t *local_topk,
                         int32_t T, int32_t k, int32_t replica_budget, int32_t *replica_slots,
                         int32_t *token_dest, int32_t *send_counts, int32_t *recv_counts, int32_t *send_offsets,
                         int32_t *token_slot, int32_t *status, void *workspace, size_t workspace_bytes,
                         void *stream) {
  const bool layout = send_offsets != nullptr || token_slot != nullptr;
  if (layout && (!send_offsets || (T > 0 && !token_slot))) return TOPOEP_EINVAL;
  if (!recv_counts && !layout) return TOPOEP_EINVAL;
  return enqueue(7, topo, global_load, local_topk, T, k, replica_budget, replica_slots, token_dest, send_counts,
                 status, workspace, workspace_bytes, stream, nullptr, recv_counts, send_offsets, token_slot);
}

int topoep_costs_workspace_bytes(const topoep_topology *topo, int32_t T, int32_t k, int32_t replica_budget,
                                 size_t *bytes_out) {
  if (!bytes_out) return TOPOEP_EINVAL;
  Plan p;
  Shape s;
  size_t need = 0;
  const int rc = setup(topo, T, k, replica_budget, nullptr, &p, &s, &need, nullptr, true);
  if (rc == TOPOEP_OK) *bytes_out = need;
  return rc;
}

int topoep_plan_costs(const topoep_topology *topo, const topoep_costs *costs, const int32_t *global_load,
                      const int32_t *local_topk, int32_t T, int32_t k, int32_t replica_budget,
                      int32_t *replica_slots, int32_t *token_dest, int32_t *send_counts, int32_t *status,
                      void *workspace, size_t workspace_bytes, void *stream) {
  const topoep_costs none = {nullptr, nullptr};
  return enqueue(7, topo, global_load, local_topk, T, k, replica_budget, replica_slots, token_dest, send_counts,
                 status, workspace, workspace_bytes, stream, nullptr, nullptr, nullptr, nullptr,
                 costs ? costs : &none);
}

int topoep_plan_stage(int32_t stage, const topoep_topology *topo, const int32_t *global_load,
                      const int32_t *local_topk, int32_t T, int32_t k, int32_t replica_budget,
                      int32_t *replica_slots, int32_t *token_dest, int32_t *send_counts, int32_t *status,
                      void *workspace, size_t workspace_bytes, void *stream, const topoep_launch *launch) {
  if (stage < 0 || stage > TOPOEP_STAGE_FLOOR) return TOPOEP_EINVAL;
  return enqueue(1 << stage, topo, global_load, local_topk, T, k, replica_budget, replica_slots,
                 token_dest, send_counts, status, workspace, workspace_bytes, stream, launch);
}

}  // extern "C"
