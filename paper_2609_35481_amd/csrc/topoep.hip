// TopoEP per-layer planner for MI355X (gfx950): HIP kernels and the C ABI
// declared in include/topoep.h.
//
// Three kernels per plan, enqueued back to back on one stream:
//
//   hist     one block per contiguous chunk of the flattened [T, k] ids.
//            LDS-privatised histogram; within a wave the lanes holding the
//            same expert are found with ballots over the id bits, and only
//            the lowest such lane adds the group's popcount.  Writes the
//            block's partial histogram (routing-matrix row of this rank,
//            Eq. 3, Section 3.1).
//   solve    one workgroup per domain (NVLink/xGMI node).  Sums the block
//            partials (row self of Omega and the per-block offsets for the
//            reroute), computes the domain demand D (Eq. 4) and the
//            inter-node placement by the benefit b = 2 D S - W (Eq. 9); a
//            bounded grid barrier publishes every domain's replicas; each
//            workgroup then builds its instances' routing q (Section 4.3,
//            routing construction) in LDS and runs the intra-node refinement
//            (Eq. 10) on one wavefront with wave64 reductions and no
//            barriers per iteration.  The last workgroup to finish turns this
//            rank's q row into a per-expert instance list.
//   reroute  same chunking as hist.  Stable rank of every assignment among
//            the earlier assignments of its expert (ballot peer masks inside
//            a wave, per-wave counts scanned across waves, block offsets from
//            the solver), then the instance whose prefix range holds it.
//
// All arithmetic is integer; no atomic decides an order or a placement
// (LDS/global integer atomics only accumulate commutative counts, masks and
// a grid-barrier ticket), so results are bitwise reproducible across runs
// and launch shapes.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "topoep.h"

namespace {

// ---------------------------------------------------------------- constants

constexpr int kCtrlBytes = 256;
constexpr int kCtrlBar = 0;      // grid-barrier arrivals
constexpr int kCtrlTicket = 1;   // finish tickets of the solver workgroups
constexpr int kCtrlStatus = 2;   // status bits accumulated during the plan
constexpr int kCtrlFinal = 3;    // final status of the plan (read by reroute)
constexpr int kCtrlTotal = 4;    // uint64 at words 4..5: sum of positive loads

constexpr uint32_t kNoPlan = TOPOEP_ST_BAD_ID | TOPOEP_ST_NEG_LOAD | TOPOEP_ST_RANGE;
constexpr int kLdsLimit = 160 * 1024;   // LDS per workgroup on gfx950
constexpr int kMaxSolveGroups = 128;    // co-resident by a wide margin (256 CUs)
constexpr int kTargetBlocks = 256;      // histogram/reroute blocks to aim for
constexpr uint32_t kSpinLimit = 1u << 24;
constexpr uint32_t kIterLimit = 1u << 22;

// ---------------------------------------------------------------- plan

struct Plan {
  int R, G, M, E, P, N, Neff, PN, I, self, MW, RW, nbits, cap1, nent_cap;
  int cI, cX;
  int64_t S, W;
  int64_t n, chunk;
  int nb;
  uint32_t spin_limit, iter_limit;
  const int32_t *gl, *topk;
  int32_t *slots_out, *dest_out, *send_out, *status_out;
  uint32_t *ctrl;
  int32_t *partials, *offsets, *blk_err, *hist, *repl1, *seg_e, *seg_q, *csr_ptr, *csr_r, *csr_end;
};

// LDS layout of the solver, in int32 words (shared by host sizing and device).
struct SolveLds {
  int cb, hs, ce, mask, slots, used, L, e_of, U, misc, qcol, words;
};

__host__ __device__ inline int imax(int a, int b) { return a > b ? a : b; }
__host__ __device__ inline int imin(int a, int b) { return a < b ? a : b; }

__host__ __device__ inline SolveLds solve_lds(const Plan &p) {
  SolveLds l;
  int o = 0;
  l.cb = o;    o += 2 * p.E;                 // int64 benefits of stage-1 candidates
  l.hs = o;    o += p.E;                     // row self of Omega (histogram)
  l.ce = o;    o += p.E;                     // stage-1 candidate experts
  l.mask = o;  o += p.E * p.MW;              // per expert: domains hosting it
  l.slots = o; o += p.G * imax(p.Neff, 1);   // replica slots of the domain's ranks
  l.used = o;  o += p.G;
  l.L = o;     o += p.G;                     // rank loads
  l.e_of = o;  o += p.I;                     // expert of each instance (-1 empty)
  l.U = o;     o += p.I;                     // instance loads
  o = (o + 3) & ~3;
  l.misc = o;  o += 64;
  l.qcol = o;                                // q[s][e][r] of the domain's instances
  o += imax(p.I * p.R, 2 * p.E + 2 + p.E * p.RW + 64);
  l.words = o;
  return l;
}

// ---------------------------------------------------------------- wave helpers

__device__ inline int lane_id() { return threadIdx.x & 63; }

__device__ inline uint64_t lanemask_lt() { return (1ull << lane_id()) - 1ull; }

// Lanes of this wave holding the same (valid) value: one ballot per id bit.
__device__ inline uint64_t peer_mask(int v, bool valid, int nbits) {
  uint64_t m = __ballot(valid);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (v >> b) & 1;
    const uint64_t on = __ballot(bit);
    m &= bit ? on : ~on;
  }
  return m;
}

// Order LDS traffic of the lanes of one wave (the refinement runs on one
// wave and needs no workgroup barrier).
__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

__device__ inline bool lex_less(uint64_t a1, uint64_t a2, uint64_t a3, uint64_t b1, uint64_t b2,
                                uint64_t b3) {
  if (a1 != b1) return a1 < b1;
  if (a2 != b2) return a2 < b2;
  return a3 < b3;
}

__device__ inline void wave_argmin3(uint64_t &k1, uint64_t &k2, uint64_t &k3) {
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o1 = __shfl_xor(k1, off), o2 = __shfl_xor(k2, off), o3 = __shfl_xor(k3, off);
    if (lex_less(o1, o2, o3, k1, k2, k3)) {
      k1 = o1;
      k2 = o2;
      k3 = o3;
    }
  }
}

__device__ inline uint64_t wave_max_u64(uint64_t v) {
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off);
    v = o > v ? o : v;
  }
  return v;
}

__device__ inline int wave_incl_scan(int x) {
  const int lane = lane_id();
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

// Exclusive scan of a[0..n) in place by the whole workgroup; returns the total.
// tmp needs blockDim/64 + 1 words.
__device__ int block_excl_scan(int *a, int n, int *tmp) {
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6, lane = tid & 63, wave = tid >> 6;
  const int per = (n + nt - 1) / nt;
  const int lo = imin(n, tid * per), hi = imin(n, lo + per);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += a[i];
  const int incl = wave_incl_scan(s);
  if (lane == 63) tmp[wave] = incl;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int w = 0; w < nw; ++w) {
      const int t = tmp[w];
      tmp[w] = run;
      run += t;
    }
    tmp[nw] = run;
  }
  __syncthreads();
  int run = tmp[wave] + incl - s;
  for (int i = lo; i < hi; ++i) {
    const int t = a[i];
    a[i] = run;
    run += t;
  }
  const int total = tmp[nw];
  __syncthreads();
  return total;
}

// Grid barrier of the solver's workgroups: every workgroup is resident (at
// most kMaxSolveGroups), and the wait is bounded so the kernel always exits.
__device__ bool grid_barrier(uint32_t *count, uint32_t groups, uint32_t spin_limit, int *flag) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    __hip_atomic_fetch_add(count, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    uint32_t it = 0;
    int ok = 1;
    while (__hip_atomic_load(count, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < groups) {
      if (++it > spin_limit) {
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    __threadfence();
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
  if (b == 0 && tid == 0) {
    // Reset the solver's control words; it runs after this kernel.
    p.ctrl[kCtrlBar] = 0;
    p.ctrl[kCtrlTicket] = 0;
    p.ctrl[kCtrlStatus] = 0;
    p.ctrl[kCtrlFinal] = 0;
    *reinterpret_cast<unsigned long long *>(p.ctrl + kCtrlTotal) = 0ull;
  }
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
      const uint64_t peers = peer_mask(ev[i], valid, p.nbits);
      if (valid && (peers & lanemask_lt()) == 0) atomicAdd(&h[ev[i]], __popcll(peers));
    }
  }
  bad = __syncthreads_or(bad);
  for (int e = tid; e < p.E; e += nt) p.partials[(int64_t)b * p.E + e] = h[e];
  if (tid == 0) p.blk_err[b] = bad;
}

// ---------------------------------------------------------------- solver

// Instance index of expert e on local rank j of domain d, or -1.
__device__ inline int instance_of(const Plan &p, int d, int j, int e, const int *slots,
                                  const int *used) {
  const int rank = d * p.G + j;
  if (e / p.P == rank) return j * p.PN + (e - rank * p.P);
  const int u = used[j];
  for (int t = 0; t < u; ++t)
    if (slots[j * p.Neff + t] == e) return j * p.PN + p.P + t;
  return -1;
}

// Intra-node refinement of domain d (Section 4.3, Eq. 10), by wave 0.
// Each iteration picks the busiest rank rb (ties to the lowest rank), scores
// every (instance of rb, other rank of the domain) candidate with key
// (delta desc, L[rt] asc, cost change asc, e asc, rt asc), and commits the
// best one.  The moved assignments come from sources in ascending
// (c(s,rt) - c(s,rb), s) order: with the two-level cost that is rt itself,
// then the other sources ascending, then rb (or plain ascending when the
// intra-domain cost is zero).  The loop ends when no candidate has
// delta >= 1.
__device__ void refine_domain(const Plan &p, int d, int *e_of, int *U, int *qcol, int *slots, int *used,
                              int *Lr, uint32_t *flags) {
  const int lane = lane_id();
  const int G = p.G, PN = p.PN, R = p.R, P = p.P, Neff = p.Neff;
  if (G < 2) return;
  const int r0 = d * G;
  const int ncand = PN * (G - 1);
  const int64_t twoS = 2 * p.S;
  for (uint32_t it = 0;; ++it) {
    if (it >= p.iter_limit) {
      if (lane == 0) *flags |= TOPOEP_ST_ITER;
      break;
    }
    // busiest rank, lowest index on ties
    uint64_t bkey = 0;
    if (lane < G) bkey = ((uint64_t)(uint32_t)Lr[lane] << 32) | (uint32_t)(0xFFFFFFFFu - lane);
    bkey = wave_max_u64(bkey);
    const int rbj = (int)(0xFFFFFFFFu - (uint32_t)bkey);
    const int Lrb = (int)(bkey >> 32);
    const int rb = r0 + rbj;
    uint64_t k1 = ~0ull, k2 = ~0ull, k3 = ~0ull;
    for (int c = lane; c < ncand; c += 64) {
      const int ai = c / (G - 1), jj = c - ai * (G - 1);
      const int rtj = jj < rbj ? jj : jj + 1;
      const int a = rbj * PN + ai;
      const int e = e_of[a];
      const int u = U[a];
      if (e < 0 || u <= 0) continue;
      const int rt = r0 + rtj;
      const int me = e / P;
      bool hosts = me == rt;
      const int urt = used[rtj];
      for (int t = 0; t < urt && !hosts; ++t) hosts = slots[rtj * Neff + t] == e;
      if (!hosts && urt >= Neff) continue;
      const int Lrt = Lr[rtj];
      const int64_t gap = (int64_t)Lrb - Lrt;
      if (gap < 2) continue;
      const int delta = (int)((int64_t)u < gap / 2 ? (int64_t)u : gap / 2);
      int64_t dtok = 0;
      if (p.cI > 0) {
        const int qrt = qcol[a * R + rt], qrb = qcol[a * R + rb];
        const int m_rt = imin(delta, qrt);
        const int rest = delta - m_rt;
        const int m_oth = imin(rest, u - qrt - qrb);
        const int m_rb = rest - m_oth;
        dtok = (int64_t)p.cI * (int64_t)(m_rb - m_rt);
      }
      const int64_t crep = (me / G == d) ? p.cI : p.cX;   // me != rt when !hosts
      const int64_t dcost = twoS * dtok + (hosts ? 0 : crep * p.W);
      const uint64_t c1 = ((uint64_t)(uint32_t)(0x7FFFFFFF - delta) << 32) | (uint32_t)Lrt;
      const uint64_t c2 = (uint64_t)dcost ^ (1ull << 63);
      const uint64_t c3 = ((uint64_t)(uint32_t)e << 32) | (uint32_t)rt;
      if (lex_less(c1, c2, c3, k1, k2, k3)) {
        k1 = c1;
        k2 = c2;
        k3 = c3;
      }
    }
    wave_argmin3(k1, k2, k3);
    if (k1 == ~0ull) break;
    const int delta = 0x7FFFFFFF - (int)(k1 >> 32);
    const int e = (int)(k3 >> 32);
    const int rt = (int)(uint32_t)k3;
    const int rtj = rt - r0;
    const int a = instance_of(p, d, rbj, e, slots, used);
    int a2 = instance_of(p, d, rtj, e, slots, used);
    if (a < 0) {   // cannot happen: the candidate came from an instance of rb
      if (lane == 0) *flags |= TOPOEP_ST_ITER;
      break;
    }
    wave_sync();
    if (a2 < 0) {
      // new replica in the first free slot of rt
      const int t = used[rtj];
      a2 = rtj * PN + P + t;
      if (lane == 0) {
        slots[rtj * Neff + t] = e;
        used[rtj] = t + 1;
        e_of[a2] = e;
      }
    }
    wave_sync();
    int *qa = qcol + a * R;
    int *qb = qcol + a2 * R;
    int rest = delta;
    if (p.cI > 0) {
      const int m_rt = imin(rest, qa[rt]);
      wave_sync();
      if (lane == 0 && m_rt) {
        qa[rt] -= m_rt;
        qb[rt] += m_rt;
      }
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
        qa[s] -= m;
        qb[s] += m;
      }
      const int total = __shfl(incl, 63);
      rest -= total < rest ? total : rest;
    }
    wave_sync();
    if (lane == 0) {
      if (rest > 0) {   // the rest comes from rb itself (two-level cost, taken last)
        qa[rb] -= rest;
        qb[rb] += rest;
      }
      U[a] -= delta;
      U[a2] += delta;
      Lr[rbj] -= delta;
      Lr[rtj] += delta;
    }
    wave_sync();
  }
}

__global__ __launch_bounds__(1024) void solve_kernel(Plan p) {
  extern __shared__ int64_t smem_s[];
  int *sm = reinterpret_cast<int *>(smem_s);
  const SolveLds lay = solve_lds(p);
  int64_t *cb = reinterpret_cast<int64_t *>(sm + lay.cb);
  int *hs = sm + lay.hs;
  int *ce = sm + lay.ce;
  uint32_t *mask = reinterpret_cast<uint32_t *>(sm + lay.mask);
  int *slots = sm + lay.slots;
  int *used = sm + lay.used;
  int *Lr = sm + lay.L;
  int *e_of = sm + lay.e_of;
  int *U = sm + lay.U;
  int *misc = sm + lay.misc;
  int *qcol = sm + lay.qcol;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int wg = blockIdx.x, nwg = gridDim.x;
  const int E = p.E, G = p.G, R = p.R, M = p.M, I = p.I, P = p.P, PN = p.PN, Neff = p.Neff;
  const int cap = p.cap1;
  uint64_t *mtotal = reinterpret_cast<uint64_t *>(sm + lay.misc + 8);

  // ---- row self of Omega: the histogram of local_topk (sum of the block
  // partials); workgroup 0 also leaves the exclusive per-block offsets.
  for (int e = tid; e < E; e += nt) {
    int run = 0;
    for (int b = 0; b < p.nb; ++b) {
      const int v = p.partials[(int64_t)b * E + e];
      if (wg == 0) p.offsets[(int64_t)b * E + e] = run;
      run += v;
    }
    hs[e] = run;
    if (wg == 0) p.hist[e] = run;
  }
  if (tid == 0) {
    misc[0] = 0;
    *mtotal = 0;
  }
  __syncthreads();
  uint32_t st = 0;
  if (wg == 0) {
    for (int b = tid; b < p.nb; b += nt)
      if (p.blk_err[b]) st |= TOPOEP_ST_BAD_ID;
    for (int e = tid; e < E; e += nt)
      if (p.gl[(int64_t)p.self * E + e] != hs[e]) st |= TOPOEP_ST_SELF_DIFF;
  }
  uint64_t tot = 0;
  for (int d = wg; d < M; d += nwg) {
    for (int i = tid; i < G * E; i += nt) {
      const int s = d * G + i / E, e = i % E;
      const int g = p.gl[(int64_t)s * E + e];
      if (g < 0) st |= TOPOEP_ST_NEG_LOAD;
      const int w = s == p.self ? hs[e] : g;
      if (w > 0) tot += (uint64_t)w;
    }
  }
  if (st) atomicOr(reinterpret_cast<unsigned *>(&misc[0]), st);
  if (tot) atomicAdd(reinterpret_cast<unsigned long long *>(mtotal), (unsigned long long)tot);
  __syncthreads();
  if (tid == 0) {
    if (misc[0]) atomicOr(&p.ctrl[kCtrlStatus], (uint32_t)misc[0]);
    if (*mtotal)
      atomicAdd(reinterpret_cast<unsigned long long *>(p.ctrl + kCtrlTotal), (unsigned long long)*mtotal);
  }

  // ---- inter-node placement (Eq. 9), each domain independently.
  for (int d = wg; d < M; d += nwg) {
    __syncthreads();
    if (tid == 0) misc[1] = 0;
    __syncthreads();
    for (int e = tid; e < E; e += nt) {
      if ((e / P) / G == d) continue;   // main inside the domain: never a candidate
      uint64_t D = 0;
      for (int j = 0; j < G; ++j) {
        const int s = d * G + j;
        D += (uint64_t)(int64_t)(s == p.self ? hs[e] : p.gl[(int64_t)s * E + e]);
      }
      // wrapping arithmetic: out-of-range inputs are flagged later and get no plan
      const int64_t b = (int64_t)(2ull * D * (uint64_t)p.S - (uint64_t)p.W);
      if (b > 0) {
        const int pos = atomicAdd(&misc[1], 1);
        ce[pos] = e;
        cb[pos] = b;
      }
    }
    __syncthreads();
    const int nc = misc[1];
    // rank of each candidate in (b descending, e ascending) order; the i-th
    // goes to rank d G + (i mod G), slot i / G: the domain rank with the
    // fewest used slots, ties to the lowest rank
    for (int c = tid; c < nc; c += nt) {
      const int64_t bc = cb[c];
      const int ec = ce[c];
      int rank = 0;
      for (int c2 = 0; c2 < nc; ++c2) {
        const int64_t b2 = cb[c2];
        rank += (b2 > bc) || (b2 == bc && ce[c2] < ec);
      }
      if (rank < cap) p.repl1[(int64_t)d * cap + rank] = ec;
    }
    for (int i = imin(nc, cap) + tid; i < cap; i += nt) p.repl1[(int64_t)d * cap + i] = -1;
  }

  // ---- every domain's replicas are needed by every routing construction
  const bool synced = grid_barrier(&p.ctrl[kCtrlBar], (uint32_t)nwg, p.spin_limit, &misc[2]);
  uint32_t gst = __hip_atomic_load(&p.ctrl[kCtrlStatus], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t total =
      __hip_atomic_load(reinterpret_cast<unsigned long long *>(p.ctrl + kCtrlTotal), __ATOMIC_RELAXED,
                        __HIP_MEMORY_SCOPE_AGENT);
  {
    // exact-range check: total <= INT32_MAX and 4 S total c + c W < 2^62
    const uint64_t lim = 1ull << 62;
    const uint64_t cm = (uint64_t)imax(imax(p.cI, p.cX), 1);
    bool range = total > 0x7FFFFFFFull;
    uint64_t tokterm = 0;
    if (!range && total > 0) {
      uint64_t a = (uint64_t)p.S;
      if (a > lim / 4) range = true;
      else {
        a *= 4;
        if (a > lim / total) range = true;
        else {
          a *= total;
          if (a > lim / cm) range = true;
          else tokterm = a * cm;
        }
      }
    }
    if (!range) {
      const uint64_t w = (uint64_t)p.W;
      if (w > lim / cm) range = true;
      else if (tokterm + w * cm >= lim) range = true;
    }
    if (range) gst |= TOPOEP_ST_RANGE;
  }
  if (!synced) gst |= TOPOEP_ST_SYNC;
  const bool noplan = (gst & kNoPlan) != 0 || !synced;

  // ---- domains hosting each expert: the main's domain plus stage-1 replicas
  if (!noplan) {
    for (int i = tid; i < E * p.MW; i += nt) mask[i] = 0;
    __syncthreads();
    for (int e = tid; e < E; e += nt) {
      const int dm = (e / P) / G;
      atomicOr(&mask[e * p.MW + (dm >> 5)], 1u << (dm & 31));
    }
    for (int i = tid; i < M * cap; i += nt) {
      const int e = p.repl1[i];
      if ((unsigned)e < (unsigned)E) {
        const int dd = i / cap;
        atomicOr(&mask[e * p.MW + (dd >> 5)], 1u << (dd & 31));
      }
    }
  }
  __syncthreads();

  uint32_t flags = 0;
  for (int d = wg; d < M; d += nwg) {
    if (noplan) {
      for (int i = tid; i < G * p.N; i += nt) p.slots_out[(int64_t)d * G * p.N + i] = -1;
      for (int j = tid; j < G; j += nt) p.send_out[d * G + j] = 0;
      for (int a = tid; a < I; a += nt) {
        p.seg_e[(int64_t)d * I + a] = -1;
        p.seg_q[(int64_t)d * I + a] = 0;
      }
      continue;
    }
    // stage-1 slots of the domain's ranks: candidate i sits on local rank
    // i mod G, slot i / G; the chosen ones are a prefix of the list
    if (tid == 0) {
      int nsel = 0;
      while (nsel < cap && (unsigned)p.repl1[(int64_t)d * cap + nsel] < (unsigned)E) ++nsel;
      misc[3] = nsel;
    }
    __syncthreads();
    const int nsel = misc[3];
    for (int j = tid; j < G; j += nt) {
      const int u = nsel > j ? (nsel - j + G - 1) / G : 0;
      used[j] = u;
      for (int t = 0; t < Neff; ++t) slots[j * Neff + t] = t < u ? p.repl1[(int64_t)d * cap + t * G + j] : -1;
    }
    __syncthreads();
    for (int a = tid; a < I; a += nt) {
      const int j = a / PN, pos = a - j * PN;
      int e;
      if (pos < P) e = (d * G + j) * P + pos;
      else e = (pos - P) < used[j] ? slots[j * Neff + pos - P] : -1;
      e_of[a] = e;
      U[a] = 0;
    }
    __syncthreads();
    // routing construction: the unique instance of e inside dom(s) takes all
    // of omega[s][e]; sources of a domain without an instance split evenly
    // over every instance (one per hosting domain, so the position in
    // ascending rank order is the number of hosting domains below d)
    for (int idx = tid; idx < I * R; idx += nt) {
      const int s = idx / I, a = idx - s * I;
      const int e = e_of[a];
      int q = 0;
      if (e >= 0) {
        const int w = s == p.self ? hs[e] : p.gl[(int64_t)s * E + e];
        if (w > 0) {
          const int ds = s / G;
          const uint32_t *me = mask + e * p.MW;
          if (ds == d) {
            q = w;
          } else if (!((me[ds >> 5] >> (ds & 31)) & 1u)) {
            int n = 0, below = 0;
            for (int wd = 0; wd < p.MW; ++wd) {
              const uint32_t bits = me[wd];
              n += __popc(bits);
              const int lo = wd * 32;
              if (d >= lo + 32) below += __popc(bits);
              else if (d > lo) below += __popc(bits & ((1u << (d - lo)) - 1u));
            }
            q = w / n + (below < w % n ? 1 : 0);
          }
        }
      }
      qcol[a * R + s] = q;
      if (q) atomicAdd(&U[a], q);
    }
    __syncthreads();
    for (int j = tid; j < G; j += nt) {
      int l = 0;
      for (int pos = 0; pos < PN; ++pos) l += U[j * PN + pos];
      Lr[j] = l;
    }
    __syncthreads();
    if (tid < 64) refine_domain(p, d, e_of, U, qcol, slots, used, Lr, &flags);
    __syncthreads();
    // outputs of the domain's ranks
    for (int i = tid; i < G * p.N; i += nt) {
      const int j = i / p.N, t = i - j * p.N;
      p.slots_out[(int64_t)(d * G + j) * p.N + t] = (t < used[j]) ? slots[j * Neff + t] : -1;
    }
    for (int j = tid; j < G; j += nt) {
      int sc = 0;
      for (int pos = 0; pos < PN; ++pos) sc += qcol[(j * PN + pos) * R + p.self];
      p.send_out[d * G + j] = sc;
    }
    for (int a = tid; a < I; a += nt) {
      p.seg_e[(int64_t)d * I + a] = e_of[a];
      p.seg_q[(int64_t)d * I + a] = e_of[a] >= 0 ? qcol[a * R + p.self] : 0;
    }
    __syncthreads();
  }
  if (tid == 0 && (flags || !synced)) atomicOr(&p.ctrl[kCtrlStatus], flags | (synced ? 0u : TOPOEP_ST_SYNC));

  // ---- the last workgroup to finish lists this rank's instances per expert
  __syncthreads();
  if (tid == 0) {
    __threadfence();
    const uint32_t t = __hip_atomic_fetch_add(&p.ctrl[kCtrlTicket], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    misc[4] = t == (uint32_t)nwg - 1;
  }
  __syncthreads();
  if (!misc[4]) return;
  __threadfence();
  int *cnt = qcol;                                            // E + 1
  uint32_t *bm = reinterpret_cast<uint32_t *>(qcol + E + 2);  // E * RW
  int *tmp = qcol + E + 2 + E * p.RW;                         // scan scratch
  for (int e = tid; e <= E; e += nt) cnt[e] = 0;
  for (int i = tid; i < E * p.RW; i += nt) bm[i] = 0;
  __syncthreads();
  for (int idx = tid; idx < M * I; idx += nt) {
    const int e = p.seg_e[idx], q = p.seg_q[idx];
    if ((unsigned)e < (unsigned)E && q > 0) {
      const int d = idx / I, a = idx - d * I;
      const int r = d * G + a / PN;
      atomicAdd(&cnt[e], 1);
      atomicOr(&bm[e * p.RW + (r >> 5)], 1u << (r & 31));
    }
  }
  __syncthreads();
  const int nent = block_excl_scan(cnt, E + 1, tmp);
  (void)nent;
  for (int e = tid; e <= E; e += nt) p.csr_ptr[e] = cnt[e];
  for (int idx = tid; idx < M * I; idx += nt) {
    const int e = p.seg_e[idx], q = p.seg_q[idx];
    if ((unsigned)e < (unsigned)E && q > 0) {
      const int d = idx / I, a = idx - d * I;
      const int r = d * G + a / PN;
      const uint32_t *row = bm + e * p.RW;
      int pos = 0;
      for (int w = 0; w < (r >> 5); ++w) pos += __popc(row[w]);
      pos += __popc(row[r >> 5] & ((1u << (r & 31)) - 1u));
      const int j = cnt[e] + pos;
      p.csr_r[j] = r;
      p.csr_end[j] = q;
    }
  }
  __syncthreads();
  for (int e = tid; e < E; e += nt) {
    int run = 0;
    for (int j = cnt[e]; j < cnt[e + 1]; ++j) {
      run += p.csr_end[j];
      p.csr_end[j] = run;
    }
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t fin = __hip_atomic_load(&p.ctrl[kCtrlStatus], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    fin |= gst & TOPOEP_ST_RANGE;
    p.ctrl[kCtrlFinal] = fin;
    p.status_out[0] = (int32_t)fin;
    p.ctrl[kCtrlBar] = 0;
    p.ctrl[kCtrlTicket] = 0;
  }
}

// ---------------------------------------------------------------- reroute

template <int IPT>
__global__ __launch_bounds__(1024) void reroute_kernel(Plan p) {
  extern __shared__ int smem_r[];
  const int nt = blockDim.x, nw = nt >> 6;
  const int E = p.E;
  int *run = smem_r;                 // E: running offset per expert
  int *wc = run + E;                 // nw * E: per-wave counts, then offsets
  int *ptr = wc + nw * E;            // E + 1
  int *er = ptr + E + 1;             // nent_cap: instance rank
  int *eend = er + p.nent_cap;       // nent_cap: cumulative share
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  const int64_t lo = (int64_t)b * p.chunk;
  const int64_t hi = lo + p.chunk < p.n ? lo + p.chunk : p.n;
  const uint32_t fin = p.ctrl[kCtrlFinal];
  if (fin & (kNoPlan | TOPOEP_ST_SYNC)) {
    for (int64_t i = lo + tid; i < hi; i += nt) p.dest_out[i] = -1;
    return;
  }
  for (int e = tid; e < E; e += nt) run[e] = p.offsets[(int64_t)b * E + e];
  for (int e = tid; e <= E; e += nt) {
    const int v = p.csr_ptr[e];
    ptr[e] = v < 0 ? 0 : (v > p.nent_cap ? p.nent_cap : v);
  }
  __syncthreads();
  const int nent = ptr[E];
  for (int j = tid; j < nent; j += nt) {
    er[j] = p.csr_r[j];
    eend[j] = p.csr_end[j];
  }
  __syncthreads();
  int *mywc = wc + wave * E;
  const int64_t tile = (int64_t)nt * IPT;
  for (int64_t base = lo; base < hi; base += tile) {
    for (int e = lane; e < E; e += 64) mywc[e] = 0;
    wave_sync();
    const int64_t wbase = base + (int64_t)wave * 64 * IPT + lane;
    int ev[IPT], lr[IPT];
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = wbase + i * 64;
      ev[i] = idx < hi ? p.topk[idx] : -1;
    }
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = wbase + i * 64;
      const bool valid = idx < hi && (unsigned)ev[i] < (unsigned)E;
      const uint64_t peers = peer_mask(ev[i], valid, p.nbits);
      const int c = valid ? mywc[ev[i]] : 0;
      lr[i] = c + __popcll(peers & lanemask_lt());
      wave_sync();
      if (valid && (peers & lanemask_lt()) == 0) mywc[ev[i]] = c + __popcll(peers);
      wave_sync();
    }
    __syncthreads();
    for (int e = tid; e < E; e += nt) {
      int s = run[e];
      for (int w = 0; w < nw; ++w) {
        const int t = wc[w * E + e];
        wc[w * E + e] = s;
        s += t;
      }
      run[e] = s;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = wbase + i * 64;
      if (idx < hi) {
        int dest = -1;
        if ((unsigned)ev[i] < (unsigned)E) {
          const int rho = mywc[ev[i]] + lr[i];
          const int j1 = ptr[ev[i] + 1];
          for (int j = ptr[ev[i]]; j < j1; ++j) {
            if (rho < eend[j]) {
              dest = er[j];
              break;
            }
          }
        }
        p.dest_out[idx] = dest;
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- host side

struct Shape {
  int ipt, bt, st;
  size_t lds_hist, lds_solve, lds_reroute;
  int solve_groups;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int ceil_log2(int v) {
  int b = 0;
  while ((1 << b) < v) ++b;
  return b;
}

// Validate the arguments and fill the plan's sizes, launch shape and
// workspace layout (pointers are offsets when ws == nullptr).
int setup(const topoep_topology *t, int32_t T, int32_t k, int32_t N, const topoep_launch *lc, Plan *p,
          Shape *sh, size_t *ws_bytes, char *ws) {
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
  q.cap1 = G * q.Neff;
  q.nent_cap = E + R * q.Neff;
  q.cI = t->cost_intra;
  q.cX = t->cost_inter;
  q.S = t->tok_bytes;
  q.W = t->expert_bytes;
  q.n = (int64_t)T * k;
  q.spin_limit = kSpinLimit;
  q.iter_limit = kIterLimit;

  Shape s;
  s.ipt = lc && lc->items_per_thread ? lc->items_per_thread : 4;
  s.bt = lc && lc->block_threads ? lc->block_threads : 256;
  s.st = lc && lc->solve_threads ? lc->solve_threads : 256;
  if (!(s.ipt == 1 || s.ipt == 2 || s.ipt == 4 || s.ipt == 8)) return TOPOEP_EINVAL;
  if (s.bt < 64 || s.bt > 1024 || s.bt % 64 || s.st < 64 || s.st > 1024 || s.st % 64) return TOPOEP_EINVAL;
  const int64_t tile = (int64_t)s.bt * s.ipt;
  const int64_t tiles = (q.n + tile - 1) / tile;
  int64_t tpb = lc && lc->tiles_per_block > 0 ? lc->tiles_per_block
                                              : (tiles + kTargetBlocks - 1) / kTargetBlocks;
  if (lc && lc->tiles_per_block < 0) return TOPOEP_EINVAL;
  if (tpb < 1) tpb = 1;
  q.chunk = tpb * tile;
  const int64_t nb = q.n > 0 ? (q.n + q.chunk - 1) / q.chunk : 1;
  if (nb > (1 << 24)) return TOPOEP_ELIMIT;
  q.nb = (int)nb;

  const SolveLds lay = solve_lds(q);
  s.lds_solve = (size_t)lay.words * 4;
  s.lds_hist = (size_t)E * 4;
  s.lds_reroute = ((size_t)E * (2 + s.bt / 64) + 1 + 2 * (size_t)q.nent_cap) * 4;
  if (s.lds_solve > (size_t)kLdsLimit || s.lds_reroute > (size_t)kLdsLimit) return TOPOEP_ELIMIT;
  s.solve_groups = imin(q.M, kMaxSolveGroups);

  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t o_ctrl = take(kCtrlBytes);
  const size_t o_part = take((size_t)q.nb * E * 4);
  const size_t o_offs = take((size_t)q.nb * E * 4);
  const size_t o_berr = take((size_t)q.nb * 4);
  const size_t o_hist = take((size_t)E * 4);
  const size_t o_repl = take((size_t)q.M * imax(q.cap1, 1) * 4);
  const size_t o_sege = take((size_t)q.M * q.I * 4);
  const size_t o_segq = take((size_t)q.M * q.I * 4);
  const size_t o_cptr = take((size_t)(E + 1) * 4);
  const size_t o_cr = take((size_t)q.nent_cap * 4);
  const size_t o_ce = take((size_t)q.nent_cap * 4);
  *ws_bytes = off;
  if (ws) {
    q.ctrl = reinterpret_cast<uint32_t *>(ws + o_ctrl);
    q.partials = reinterpret_cast<int32_t *>(ws + o_part);
    q.offsets = reinterpret_cast<int32_t *>(ws + o_offs);
    q.blk_err = reinterpret_cast<int32_t *>(ws + o_berr);
    q.hist = reinterpret_cast<int32_t *>(ws + o_hist);
    q.repl1 = reinterpret_cast<int32_t *>(ws + o_repl);
    q.seg_e = reinterpret_cast<int32_t *>(ws + o_sege);
    q.seg_q = reinterpret_cast<int32_t *>(ws + o_segq);
    q.csr_ptr = reinterpret_cast<int32_t *>(ws + o_cptr);
    q.csr_r = reinterpret_cast<int32_t *>(ws + o_cr);
    q.csr_end = reinterpret_cast<int32_t *>(ws + o_ce);
  }
  *p = q;
  *sh = s;
  return TOPOEP_OK;
}

template <typename K>
void allow_lds(K kernel) {
  (void)hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, kLdsLimit);
}

bool g_attrs_set = false;

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
  allow_lds(solve_kernel);
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
  hipLaunchKernelGGL(solve_kernel, dim3(s.solve_groups), dim3(s.st), s.lds_solve, st, p);
}

int enqueue(int stage_mask, const topoep_topology *topo, const int32_t *global_load,
            const int32_t *local_topk, int32_t T, int32_t k, int32_t N, int32_t *replica_slots,
            int32_t *token_dest, int32_t *send_counts, int32_t *status, void *workspace,
            size_t workspace_bytes, void *stream, const topoep_launch *launch) {
  Plan p;
  Shape s;
  size_t need = 0;
  int rc = setup(topo, T, k, N, launch, &p, &s, &need, nullptr);
  if (rc != TOPOEP_OK) return rc;
  if (!global_load || !send_counts || !status || !workspace) return TOPOEP_EINVAL;
  if ((int64_t)topo->num_ranks * N > 0 && !replica_slots) return TOPOEP_EINVAL;
  if (T > 0 && (!local_topk || !token_dest)) return TOPOEP_EINVAL;
  if (workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return TOPOEP_EWORKSPACE;
  rc = setup(topo, T, k, N, launch, &p, &s, &need, static_cast<char *>(workspace));
  if (rc != TOPOEP_OK) return rc;
  p.gl = global_load;
  p.topk = local_topk;
  p.slots_out = replica_slots;
  p.dest_out = token_dest;
  p.send_out = send_counts;
  p.status_out = status;
  set_attrs();
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (stage_mask & 1) launch_hist(p, s, st);
  if (stage_mask & 2) launch_solve(p, s, st);
  if (stage_mask & 4) launch_reroute(p, s, st);
  return hipGetLastError() == hipSuccess ? TOPOEP_OK : TOPOEP_EHIP;
}

}  // namespace

extern "C" {

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

int topoep_plan(const topoep_topology *topo, const int32_t *global_load, const int32_t *local_topk,
                int32_t T, int32_t k, int32_t replica_budget, int32_t *replica_slots, int32_t *token_dest,
                int32_t *send_counts, int32_t *status, void *workspace, size_t workspace_bytes,
                void *stream) {
  return enqueue(7, topo, global_load, local_topk, T, k, replica_budget, replica_slots, token_dest,
                 send_counts, status, workspace, workspace_bytes, stream, nullptr);
}

int topoep_plan_stage(int32_t stage, const topoep_topology *topo, const int32_t *global_load,
                      const int32_t *local_topk, int32_t T, int32_t k, int32_t replica_budget,
                      int32_t *replica_slots, int32_t *token_dest, int32_t *send_counts, int32_t *status,
                      void *workspace, size_t workspace_bytes, void *stream, const topoep_launch *launch) {
  if (stage < 0 || stage > 2) return TOPOEP_EINVAL;
  return enqueue(1 << stage, topo, global_load, local_topk, T, k, replica_budget, replica_slots,
                 token_dest, send_counts, status, workspace, workspace_bytes, stream, launch);
}

}  // extern "C"
