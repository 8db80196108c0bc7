// Dispatch layout of the rerouted assignments on gfx950: the send buffer
// groups the assignments by destination rank (ranks ascending) and keeps
// row-major (token, k) order inside one destination, so each destination's
// assignments form one contiguous run that an all-to-all dispatch sends as
// is (the per-destination counts the dispatch consumes, Section 4.3).
//
// One launch; one pass over token_dest for a chunk of one tile per
// workgroup, two passes for longer chunks (at most 256 workgroups):
//   - a one-tile workgroup holds its assignments in registers and ranks
//     them among equal destinations inside each wave (ballots over the
//     destination bits give each lane its peers), then scans the per-wave
//     counts across waves in LDS; a longer chunk is cut into one contiguous
//     part per wave, each wave only counts its part's destinations here
//     (LDS atomics), and after the look-back ranks its part step by step
//     from its own running base, reading the assignments again, with no
//     workgroup barrier;
//   - it publishes its per-destination counts (flag 1), then looks back
//     over up to 64 predecessors at a time: wave 0 waits for their flags in
//     parallel and stops at the nearest one whose inclusive prefix is
//     published (flag 2), the whole workgroup sums their counts per
//     destination, and (when the grid is longer than one window plus
//     workgroup 0) the workgroup publishes its own inclusive prefix (flag
//     2).  Workgroup 0 publishes its counts as its inclusive prefix;
//   - slot = send_offsets[dest] + (earlier workgroups) + (earlier waves, or
//     their parts) + (earlier steps of the wave's part) + (rank in the
//     wave).
// The waits are bounded and only on lower workgroup indices, which are
// dispatched first.  The last workgroup to finish its look-back (a ticket)
// clears every flag, so the workspace is zero again for the next call.
// All arithmetic is integer and no atomic decides an order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "topoep.h"
#include "wave.h"

namespace {

using namespace topoep_dev;

constexpr int kLayoutThreads = 1024;
constexpr int kLayoutMaxRanks = 1024;   // per-wave counts of 16 waves fit 64 KB of LDS
constexpr int kLayoutWindow = 64;       // predecessors examined per look-back step
constexpr int kLayoutBlocks = 256;      // workgroups at most (longer chunks take several tiles)
constexpr uint32_t kLayoutSpin = 1u << 24;
constexpr int kLayoutCtrlBytes = 256;

struct Layout {
  int R, nbits, nb;
  int64_t n, chunk;
  const int32_t *dest;
  const int32_t *send;
  int32_t *offs_out;   // [R + 1]
  int32_t *slot_out;   // [n]
  int32_t *status;     // [1] or null: TOPOEP_ST_SYNC when a wait gave up
  uint32_t *agg;       // [nb][R] counts of each workgroup
  uint32_t *incl;      // [nb][R] inclusive prefixes over workgroups
  uint32_t *flags;     // [nb] 0, 1 counts published, 2 inclusive prefix published
  uint32_t *ctrl;      // [0] finish ticket
  uint32_t spin_limit;
};

// LDS words: per-wave counts (then offsets, then a long chunk's running
// slot bases) [nw][R], the workgroup's counts [R], the exclusive prefix over
// earlier workgroups [R], send offsets [R + 1], broadcast words, and the
// counting copies of a long chunk's first pass [nw][C][R] (C > 1).
struct LayoutLds {
  int wc, agg, excl, offs, misc, cnt, words;
};

// Copies of each wave's counts in the first pass of a long chunk: lane l
// counts into copy l % C, so equal destinations of one wave instruction
// meet fewer times on one LDS word (at most 64 KB of copies).
__host__ __device__ inline int layout_copies(int R) { return R <= 256 ? 4 : (R <= 512 ? 2 : 1); }

__host__ __device__ inline LayoutLds layout_lds(int R, int nt) {
  LayoutLds l;
  int o = 0;
  l.wc = o; o += (nt / 64) * R;
  l.agg = o; o += R;
  l.excl = o; o += R;
  l.offs = o; o += R + 1;
  l.misc = o; o += 8;
  l.cnt = o; o += layout_copies(R) > 1 ? (nt / 64) * layout_copies(R) * R : 0;
  l.words = o;
  return l;
}

// Rank of each of the wave's IPT x 64 assignments among the wave's earlier
// ones with the same destination (index order: i, then lane) into lr, and
// the wave's count of every destination into its row of wc.
template <int IPT>
__device__ inline void rank_wave(int R, int nbits, const int (&dv)[IPT], int (&lr)[IPT], int *mywc) {
  const int lane = lane_id();
  for (int r = lane; r < R; r += 64) mywc[r] = 0;
  wave_sync();
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    lr[i] = wave_rank(dv[i], (unsigned)dv[i] < (unsigned)R, nbits, mywc);
  }
}

// Per destination: the waves' counts in wc become their offsets (one 16-lane
// scan per rank, lane w holding wave w's count) and tot[r] the row's total.
__device__ inline void scan_waves(int R, int nw, int *wc, int *tot) {
  const int rows = R * 16, span = (rows + 63) & ~63;
  for (int t = threadIdx.x; t < span; t += blockDim.x) {
    const int r = t >> 4, w = t & 15;
    const bool in = t < rows && w < nw;
    const int c = in ? wc[w * R + r] : 0;
    const int incl = row16_incl_scan(c);
    if (in) wc[w * R + r] = incl - c;
    if (t < rows && w == 15) tot[r] = incl;
  }
}

template <int IPT>
__global__ __launch_bounds__(kLayoutThreads) void layout_kernel(Layout L) {
  extern __shared__ int lsm[];
  const int R = L.R, tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  const LayoutLds l = layout_lds(R, nt);
  int *wc = lsm + l.wc, *agg = lsm + l.agg, *excl = lsm + l.excl, *offs = lsm + l.offs;
  int *misc = lsm + l.misc;
  const int64_t lo = (int64_t)b * L.chunk;
  const int64_t hi = lo + L.chunk < L.n ? lo + L.chunk : L.n;
  const int64_t tile = (int64_t)nt * IPT;
  // a chunk of one tile keeps its ids and ranks in registers across the
  // look-back; a longer chunk counts its tiles first (pass 1) and ranks them
  // after the look-back (pass 2), reading the ids twice
  const bool multi = L.chunk > tile;
  const int64_t wofs = (int64_t)wave * 64 * IPT + lane;
  // a longer chunk: wave w owns the w-th of nw equal contiguous parts, in
  // steps of 64 IPT ids (the chunk is a whole number of tiles)
  const int64_t step = 64 * IPT, sub = L.chunk / nw;
  const int64_t wlo = lo + wave * sub, whi = wlo + sub < hi ? wlo + sub : hi;
  auto load_step = [&](int (&v)[IPT], int64_t base) {
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = base + lane + i * 64;
      v[i] = idx < whi ? L.dest[idx] : -1;
    }
  };
  // workgroups whose look-back window reaches workgroup 0 never need the
  // inclusive prefix of another one
  const bool publish_incl = L.nb > kLayoutWindow + 1;
  int *mywc = wc + wave * R;

  int dv[IPT], lr[IPT];
  for (int r = tid; r < R; r += nt) {
    offs[r] = L.send[r];
    excl[r] = 0;
  }
  if (tid < 8) misc[tid] = 0;
  if (!multi) {
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = lo + wofs + i * 64;
      dv[i] = idx < hi ? L.dest[idx] : -1;
    }
    rank_wave<IPT>(R, L.nbits, dv, lr, mywc);
  } else {
    // pass 1: each wave's count of every destination over its own part of
    // the chunk, one LDS atomic per assignment into the lane's copy of the
    // wave's counts (the order of the counting does not matter: a lane
    // loads four consecutive ids at once; the next step's loads are in
    // flight meanwhile), then the copies summed into the wave's row
    const int C = layout_copies(R);
    int *rows = C > 1 ? lsm + l.cnt + wave * C * R : mywc;
    for (int r = lane; r < C * R; r += 64) rows[r] = 0;
    wave_sync();
    int *myc = rows + (lane & (C - 1)) * R;
    // V loads of four ids per lane and step (256 V ids; parts start on
    // multiples of 64 ids, so a 16-byte aligned array keeps them aligned)
    constexpr int V = IPT >= 4 ? IPT / 4 : 1;
    const int64_t step1 = 256 * V;
    const bool vec = (reinterpret_cast<uintptr_t>(L.dest) & 15) == 0;
    auto load4 = [&](int4 (&v)[V], int64_t base) {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int64_t idx = base + (int64_t)(j * 64 + lane) * 4;
        if (vec && idx + 4 <= whi) {
          v[j] = *reinterpret_cast<const int4 *>(L.dest + idx);
        } else {
          v[j].x = idx < whi ? L.dest[idx] : -1;
          v[j].y = idx + 1 < whi ? L.dest[idx + 1] : -1;
          v[j].z = idx + 2 < whi ? L.dest[idx + 2] : -1;
          v[j].w = idx + 3 < whi ? L.dest[idx + 3] : -1;
        }
      }
    };
    int4 nx[V];
    load4(nx, wlo);
    for (int64_t base = wlo; base < whi; base += step1) {
      int4 cv[V];
#pragma unroll
      for (int j = 0; j < V; ++j) cv[j] = nx[j];
      if (base + step1 < whi) load4(nx, base + step1);
#pragma unroll
      for (int j = 0; j < V; ++j) {
        if ((unsigned)cv[j].x < (unsigned)R) atomicAdd(&myc[cv[j].x], 1);
        if ((unsigned)cv[j].y < (unsigned)R) atomicAdd(&myc[cv[j].y], 1);
        if ((unsigned)cv[j].z < (unsigned)R) atomicAdd(&myc[cv[j].z], 1);
        if ((unsigned)cv[j].w < (unsigned)R) atomicAdd(&myc[cv[j].w], 1);
      }
    }
    if (C > 1) {
      wave_sync();
      for (int r = lane; r < R; r += 64) {
        int sum = 0;
        for (int c = 0; c < C; ++c) sum += rows[c * R + r];
        mywc[r] = sum;
      }
    }
  }
  lds_barrier();
  scan_waves(R, nw, wc, agg);
  lds_barrier();
  for (int r = tid; r < R; r += nt) {
    L.agg[(int64_t)b * R + r] = (uint32_t)agg[r];
    if (b == 0) L.incl[r] = (uint32_t)agg[r];
  }
  // send offsets (exclusive prefix of the send counts) by wave 0
  if (wave == 0) {
    const int per = (R + 63) / 64, a0 = imin(R, lane * per), a1 = imin(R, a0 + per);
    int sum = 0;
    for (int r = a0; r < a1; ++r) sum += offs[r];
    int acc = wave_incl_scan(sum) - sum;
    for (int r = a0; r < a1; ++r) {
      const int c = offs[r];
      offs[r] = acc;
      acc += c;
    }
    if (lane == 63) offs[R] = acc;
  }
  drain_then_barrier();
  if (tid == 0)
    __hip_atomic_store(L.flags + b, b == 0 ? 2u : 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  if (b == 0 && L.offs_out)
    for (int r = tid; r <= R; r += nt) L.offs_out[r] = offs[r];

  // look-back over the workgroups before b
  bool ok = true;
  int jhi = b - 1;
  while (jhi >= 0) {
    if (wave == 0) {
      const int cnt = imin(kLayoutWindow, jhi + 1);
      const int j = jhi - lane;
      uint32_t f = 0;
      bool gave_up = false;
      if (lane < cnt) {
        uint32_t it = 0;
        while ((f = __hip_atomic_load(L.flags + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) == 0u) {
          if (++it > L.spin_limit) {
            gave_up = true;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      const uint64_t done = __ballot(lane < cnt && f == 2u);
      const bool bad = __ballot(gave_up) != 0;
      // the nearest predecessor with an inclusive prefix, else the window's end
      const int stop = done ? jhi - (__ffsll((long long)done) - 1) : jhi - cnt + 1;
      if (lane == 0) {
        misc[0] = stop;
        misc[1] = done != 0;
        misc[2] = bad;
      }
    }
    __syncthreads();
    const int stop = misc[0];
    const bool found = misc[1] != 0;
    if (misc[2]) {
      ok = false;
      break;
    }
    // excl[r] += counts of stop+1 .. jhi, plus the inclusive prefix (or the
    // counts) of stop
    const int span = jhi - stop + 1;
    for (int x = tid; x < span * R; x += nt) {
      const int jj = x / R, r = x - jj * R;
      const int j = stop + jj;
      const uint32_t v = (j == stop && found) ? L.incl[(int64_t)j * R + r] : L.agg[(int64_t)j * R + r];
      if (v) atomicAdd(&excl[r], (int)v);
    }
    lds_barrier();
    if (found) break;
    jhi = stop - 1;
  }
  if (b > 0 && publish_incl) {
    for (int r = tid; r < R; r += nt) L.incl[(int64_t)b * R + r] = (uint32_t)(excl[r] + agg[r]);
    drain_then_barrier();
    if (tid == 0)
      __hip_atomic_store(L.flags + b, 2u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (!multi) {
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int64_t idx = lo + wofs + i * 64;
      if (idx < hi) {
        const int d = dv[i];
        const bool valid = ok && (unsigned)d < (unsigned)R;
        L.slot_out[idx] = valid ? offs[d] + excl[d] + mywc[d] + lr[i] : -1;
      }
    }
  } else {
    // pass 2: the wave's row becomes its first slot per destination (send
    // offset + earlier workgroups + earlier waves), and each step's slots
    // are that running base plus the rank in the wave, which the rank
    // advances: no workgroup barrier
    for (int r = lane; r < R; r += 64) mywc[r] += offs[r] + excl[r];
    wave_sync();
    int nx[IPT];
    load_step(nx, wlo);
    for (int64_t base = wlo; base < whi; base += step) {
#pragma unroll
      for (int i = 0; i < IPT; ++i) dv[i] = nx[i];
      if (base + step < whi) load_step(nx, base + step);
#pragma unroll
      for (int i = 0; i < IPT; ++i) {
        const int d = dv[i];
        const bool valid = (unsigned)d < (unsigned)R;
        const int slot = wave_rank(d, valid, L.nbits, mywc);
        const int64_t idx = base + lane + i * 64;
        if (idx < whi) L.slot_out[idx] = ok && valid ? slot : -1;
      }
    }
  }
  // this workgroup has read every flag it needs: the last one to get here
  // clears them all for the next call
  if (tid == 0) {
    const uint32_t t = __hip_atomic_fetch_add(L.ctrl, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    misc[3] = t + 1u == (uint32_t)L.nb;
    if (!ok && L.status) atomicOr(reinterpret_cast<unsigned *>(L.status), TOPOEP_ST_SYNC);
  }
  __syncthreads();
  if (misc[3]) {
    for (int j = tid; j < L.nb; j += nt)
      __hip_atomic_store(L.flags + j, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (tid == 0) __hip_atomic_store(L.ctrl, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int ceil_log2(int v) {
  int b = 0;
  while ((1 << b) < v) ++b;
  return b;
}

struct LayoutShape {
  int ipt;
  size_t lds;
};

// Sizes, launch shape and workspace layout (pointers stay null when ws is).
int layout_setup(const topoep_topology *t, int32_t T, int32_t k, Layout *out, LayoutShape *sh,
                 size_t *ws_bytes, char *ws) {
  if (!t) return TOPOEP_EINVAL;
  const int R = t->num_ranks;
  if (R <= 0 || T < 0 || k < 1 || (int64_t)T * k > 0x7FFFFFFF) return TOPOEP_EINVAL;
  if (R > kLayoutMaxRanks) return TOPOEP_ELIMIT;
  Layout L = {};
  L.R = R;
  L.nbits = ceil_log2(R);
  L.n = (int64_t)T * k;
  // ids per thread, then whole tiles per workgroup so that the grid stays
  // within kLayoutBlocks workgroups, half that up to 2^21 ids (the look-back
  // chain grows with the grid; on MI355X these bounds measured fastest)
  const int ipt = L.n <= (int64_t)kLayoutThreads * 16 ? 1 : (L.n <= (int64_t)1 << 20 ? 4 : 8);
  const int64_t tile = (int64_t)kLayoutThreads * ipt;
  const int64_t tiles = L.n > 0 ? (L.n + tile - 1) / tile : 1;
  const int64_t max_blocks = L.n <= ((int64_t)1 << 21) ? kLayoutBlocks / 2 : kLayoutBlocks;
  L.chunk = tile * ((tiles + max_blocks - 1) / max_blocks);
  const int64_t nb = L.n > 0 ? (L.n + L.chunk - 1) / L.chunk : 1;
  if (nb > (1 << 20)) return TOPOEP_ELIMIT;
  L.nb = (int)nb;
  L.spin_limit = kLayoutSpin;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t o_ctrl = take(kLayoutCtrlBytes);
  const size_t o_flag = take((size_t)L.nb * 4);
  const size_t o_agg = take((size_t)L.nb * R * 4);
  const size_t o_incl = take((size_t)L.nb * R * 4);
  *ws_bytes = off;
  if (ws) {
    L.ctrl = reinterpret_cast<uint32_t *>(ws + o_ctrl);
    L.flags = reinterpret_cast<uint32_t *>(ws + o_flag);
    L.agg = reinterpret_cast<uint32_t *>(ws + o_agg);
    L.incl = reinterpret_cast<uint32_t *>(ws + o_incl);
  }
  sh->ipt = ipt;
  sh->lds = (size_t)layout_lds(R, kLayoutThreads).words * 4;
  *out = L;
  return TOPOEP_OK;
}

bool g_layout_attrs = false;

void layout_attrs() {
  if (g_layout_attrs) return;
  const void *ks[] = {reinterpret_cast<const void *>(layout_kernel<1>), reinterpret_cast<const void *>(layout_kernel<2>),
                      reinterpret_cast<const void *>(layout_kernel<4>), reinterpret_cast<const void *>(layout_kernel<8>)};
  for (const void *kf : ks) (void)hipFuncSetAttribute(kf, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  g_layout_attrs = true;
}

}  // namespace

extern "C" {

int topoep_layout_workspace_bytes(const topoep_topology *topo, int32_t T, int32_t k, size_t *bytes_out) {
  if (!bytes_out) return TOPOEP_EINVAL;
  Layout L;
  LayoutShape sh;
  size_t need = 0;
  const int rc = layout_setup(topo, T, k, &L, &sh, &need, nullptr);
  if (rc == TOPOEP_OK) *bytes_out = need;
  return rc;
}

int topoep_dispatch_layout(const topoep_topology *topo, const int32_t *token_dest, int32_t T, int32_t k,
                           const int32_t *send_counts, int32_t *send_offsets, int32_t *token_slot,
                           int32_t *status, void *workspace, size_t workspace_bytes, void *stream) {
  Layout L;
  LayoutShape sh;
  size_t need = 0;
  int rc = layout_setup(topo, T, k, &L, &sh, &need, nullptr);
  if (rc != TOPOEP_OK) return rc;
  if (!send_counts || !send_offsets || !workspace || (T > 0 && (!token_dest || !token_slot)))
    return TOPOEP_EINVAL;
  if (workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return TOPOEP_EWORKSPACE;
  rc = layout_setup(topo, T, k, &L, &sh, &need, static_cast<char *>(workspace));
  if (rc != TOPOEP_OK) return rc;
  L.dest = token_dest;
  L.send = send_counts;
  L.offs_out = send_offsets;
  L.slot_out = token_slot;
  L.status = status;
  layout_attrs();
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const dim3 g(L.nb), bl(kLayoutThreads);
  switch (sh.ipt) {
    case 1: hipLaunchKernelGGL(layout_kernel<1>, g, bl, sh.lds, st, L); break;
    case 2: hipLaunchKernelGGL(layout_kernel<2>, g, bl, sh.lds, st, L); break;
    case 4: hipLaunchKernelGGL(layout_kernel<4>, g, bl, sh.lds, st, L); break;
    default: hipLaunchKernelGGL(layout_kernel<8>, g, bl, sh.lds, st, L); break;
  }
  return hipGetLastError() == hipSuccess ? TOPOEP_OK : TOPOEP_EHIP;
}

}  // extern "C"
