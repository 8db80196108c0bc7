// Wave64 and workgroup helpers shared by the planner's kernels (gfx950):
// lane masks, ballot peer groups, DPP reductions and scans, LDS-only
// barriers and the drain-then-signal hand-over between workgroups.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace topoep_dev {

__host__ __device__ inline int imax(int a, int b) { return a > b ? a : b; }
__host__ __device__ inline int imin(int a, int b) { return a < b ? a : b; }

// ---------------------------------------------------------------- wave helpers

__device__ inline int lane_id() { return threadIdx.x & 63; }

__device__ inline uint64_t lanemask_lt() { return (1ull << lane_id()) - 1ull; }

// Order LDS traffic of the lanes of one wave (the refinement runs on one
// wave and needs no workgroup barrier).
__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Lanes of this wave holding the same value as this lane, among the lanes
// where valid holds: one ballot per value bit (nbits low bits).  The mask
// starts as the valid lanes and, per bit, keeps the lanes whose bit (read
// from that bit's ballot) equals this lane's: a bit-field extract, the
// ballot's compare and one three-input bit operation per mask half
// (v_bitop3 on gfx950).
__device__ inline uint64_t peer_mask(int v, bool valid, int nbits) {
  const uint64_t vm = __ballot(valid);
  uint32_t elo = (uint32_t)vm, ehi = (uint32_t)(vm >> 32);
  for (int b = 0; b < nbits; ++b) {
    const int sb = __builtin_amdgcn_sbfe(v, b, 1);   // bit b as 0 or all ones
    const uint64_t on = __ballot(sb != 0);
    elo &= ~((uint32_t)on ^ (uint32_t)sb);
    ehi &= ~((uint32_t)(on >> 32) ^ (uint32_t)sb);
  }
  return ((uint64_t)ehi << 32) | elo;
}

// c plus the number of lanes below this one in mask (v_mbcnt).
__device__ inline int count_below(uint64_t mask, int c) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, (uint32_t)c));
}

// Stable rank of this lane's value v among the wave's lanes: counts[v] (the
// wave's earlier occurrences of v, its own LDS row) plus the lanes below
// holding v; counts[v] then grows by the lanes holding v.  Every lane of a
// group stores the same new count, so no lane needs to be picked to store
// it.  Invalid lanes take no part (their result means nothing).
// (S: the counts lie S words apart.)
template <int S = 1>
__device__ inline int wave_rank(int v, bool valid, int nbits, int *counts) {
  const uint64_t peers = peer_mask(v, valid, nbits);
  const int c = valid ? counts[v * S] : 0;
  const int r = count_below(peers, c);
  wave_sync();
  if (valid) counts[v * S] = c + __popc((uint32_t)peers) + __popc((uint32_t)(peers >> 32));
  wave_sync();
  return r;
}

// Workgroup barrier that orders LDS only: it does not wait for outstanding
// global stores (the solver's outputs), unlike __syncthreads.
__device__ inline void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Cross-lane moves within rows of 16 lanes (DPP); every lane of the wave
// must be active.  0x121..0x12F = row_ror:1..15, 0x111..0x11F = row_shr,
// 0x142/0x143 = row_bcast:15/31.
template <int C>
__device__ inline uint32_t dpp_mov(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, C, 0xF, 0xF, true);
}
template <int C>
__device__ inline uint64_t dpp_mov64(uint64_t v) {
  return ((uint64_t)dpp_mov<C>((uint32_t)(v >> 32)) << 32) | dpp_mov<C>((uint32_t)v);
}
__device__ inline uint64_t readlane64(uint64_t v, int l) {
  return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(v >> 32), l) << 32) |
         (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}

// Wave-wide minimum / sum, the same value in every lane: rotations by 8, 4,
// 2, 1 inside each row of 16 lanes, then the four row results.
__device__ inline uint64_t wave_min_u64(uint64_t v) {
  uint64_t o;
  o = dpp_mov64<0x128>(v); v = o < v ? o : v;
  o = dpp_mov64<0x124>(v); v = o < v ? o : v;
  o = dpp_mov64<0x122>(v); v = o < v ? o : v;
  o = dpp_mov64<0x121>(v); v = o < v ? o : v;
  uint64_t a = readlane64(v, 0), b = readlane64(v, 16), c = readlane64(v, 32), d = readlane64(v, 48);
  a = b < a ? b : a;
  c = d < c ? d : c;
  return c < a ? c : a;
}

// 32-bit minimum, with the candidates known to sit in lanes 0..15 when
// rows1 (the other rows are then ignored): one readlane instead of four.
__device__ inline uint32_t rows_min_u32(uint32_t v, bool rows1) {
  uint32_t o;
  o = dpp_mov<0x128>(v); v = o < v ? o : v;
  o = dpp_mov<0x124>(v); v = o < v ? o : v;
  o = dpp_mov<0x122>(v); v = o < v ? o : v;
  o = dpp_mov<0x121>(v); v = o < v ? o : v;
  uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
  if (!rows1) {
    const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
    const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
    const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
    a = b < a ? b : a;
    a = c < a ? c : a;
    a = d < a ? d : a;
  }
  return a;
}

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
  v += dpp_mov64<0x128>(v);
  v += dpp_mov64<0x124>(v);
  v += dpp_mov64<0x122>(v);
  v += dpp_mov64<0x121>(v);
  return readlane64(v, 0) + readlane64(v, 16) + readlane64(v, 32) + readlane64(v, 48);
}

// Inclusive prefix sum over the 64 lanes (row shifts, then row broadcasts).
__device__ inline int wave_incl_scan(int x) {
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);
  return x;
}

// Inclusive prefix sum inside each row of 16 lanes.
__device__ inline int row16_incl_scan(int x) {
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);
  x += (int)__builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);
  return x;
}

__device__ inline int readlane_i32(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

// A value every lane of the wave holds alike (read from LDS, say), made
// scalar: work on it then runs once on the scalar unit instead of in every
// lane of every wave.
__device__ inline int uniform_i32(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ inline uint64_t uniform_u64(uint64_t v) {
  return ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(v >> 32)) << 32) |
         (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

__device__ inline bool lex_less(uint64_t a1, uint64_t a2, uint64_t a3, uint64_t b1, uint64_t b2,
                                uint64_t b3) {
  if (a1 != b1) return a1 < b1;
  if (a2 != b2) return a2 < b2;
  return a3 < b3;
}

// Exclusive scan of a[0..n) in place by the whole workgroup; returns the total.
// tmp needs blockDim/64 + 1 words.
__device__ inline int block_excl_scan(int *a, int n, int *tmp) {
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6, lane = tid & 63, wave = tid >> 6;
  const int per = (n + nt - 1) / nt;
  const int lo = imin(n, tid * per), hi = imin(n, lo + per);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += a[i];
  const int incl = wave_incl_scan(s);
  if (lane == 63) tmp[wave] = incl;
  lds_barrier();
  if (tid == 0) {
    int run = 0;
    for (int w = 0; w < nw; ++w) {
      const int t = tmp[w];
      tmp[w] = run;
      run += t;
    }
    tmp[nw] = run;
  }
  lds_barrier();
  int run = tmp[wave] + incl - s;
  for (int i = lo; i < hi; ++i) {
    const int t = a[i];
    a[i] = run;
    run += t;
  }
  const int total = tmp[nw];
  lds_barrier();
  return total;
}

// Hand-overs between workgroups.  A workgroup barrier orders the waves but
// does not wait for their global stores, and one wave's agent-scope release
// (an L2 write-back) only covers stores that have reached the L2.  So before
// the barrier that precedes a signal every wave waits for its own memory
// operations to complete (s_waitcnt, no cache operation); then one wave
// releases and signals.  On the waiting side one wave acquires (the L1 and
// L2 invalidations cover the whole CU) before the barrier that releases the
// other waves' loads.
__device__ inline void drain_then_barrier() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

}  // namespace topoep_dev
