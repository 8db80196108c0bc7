// Replica-slot parameter gather on gfx950 (Section 3.2: every rank holds
// N_slot replica slots beside its main experts; once the plan names the
// expert of each slot, the slot receives that expert's parameters).  On one
// GPU the main parameters of every expert sit in one buffer and the gather
// is a device copy into this rank's slots in slot order.
//
// One launch, HBM-bound: a 2-D grid of (chunk of the expert's bytes, slot).
// Each workgroup reads the slot's expert id once (uniform), skips empty
// slots and slots that already hold that expert (prev_slots), and streams
// its chunk with four 16-byte loads in flight per thread before the
// non-temporal stores, so the copy does not evict the caches' other data.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "topoep.h"

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));   // one 16-byte word

constexpr int kGatherThreads = 256;
constexpr int kGatherUnroll = 4;                                   // 16-byte words in flight per thread
// 16-byte words per workgroup (16 KB): one 9 MiB expert spans 576
// workgroups, so even two slots fill the 256 CUs several times over
constexpr int64_t kGatherChunk = (int64_t)kGatherThreads * kGatherUnroll;

struct Gather {
  int R, N, E, self;
  int64_t words;          // 16-byte words per expert
  const int32_t *slots;   // [R, N]
  const int32_t *prev;    // [N] or null
  const v4i *params;      // [E, words]
  v4i *out;               // [N, words]
};

__global__ __launch_bounds__(kGatherThreads) void gather_kernel(Gather g) {
  const int j = blockIdx.y;
  const int e = g.slots[(int64_t)g.self * g.N + j];
  if ((unsigned)e >= (unsigned)g.E) return;                 // empty slot (or not an expert)
  if (g.prev && g.prev[j] == e) return;                      // already holds that expert
  const v4i *src = g.params + (int64_t)e * g.words;
  v4i *dst = g.out + (int64_t)j * g.words;
  const int64_t base = (int64_t)blockIdx.x * kGatherChunk;
  const int64_t end = base + kGatherChunk < g.words ? base + kGatherChunk : g.words;
  for (int64_t i0 = base + threadIdx.x; i0 < end; i0 += (int64_t)kGatherThreads * kGatherUnroll) {
    v4i v[kGatherUnroll];
#pragma unroll
    for (int u = 0; u < kGatherUnroll; ++u) {
      const int64_t i = i0 + (int64_t)u * kGatherThreads;
      if (i < end) v[u] = __builtin_nontemporal_load(src + i);
    }
#pragma unroll
    for (int u = 0; u < kGatherUnroll; ++u) {
      const int64_t i = i0 + (int64_t)u * kGatherThreads;
      if (i < end) __builtin_nontemporal_store(v[u], dst + i);
    }
  }
}

}  // namespace

extern "C" {

int topoep_gather_replicas(const topoep_topology *topo, int32_t replica_budget, const int32_t *replica_slots,
                           const int32_t *prev_slots, const void *expert_params, int64_t bytes_per_expert,
                           void *slot_params, void *stream) {
  if (!topo) return TOPOEP_EINVAL;
  const int R = topo->num_ranks, E = topo->num_experts, self = topo->self_rank;
  if (R <= 0 || E <= 0 || self < 0 || self >= R || replica_budget < 0) return TOPOEP_EINVAL;
  if (bytes_per_expert < 0 || (bytes_per_expert & 15)) return TOPOEP_EINVAL;
  if (replica_budget == 0 || bytes_per_expert == 0) return TOPOEP_OK;   // nothing to copy
  if (!replica_slots || !expert_params || !slot_params) return TOPOEP_EINVAL;
  if (((reinterpret_cast<uintptr_t>(expert_params) | reinterpret_cast<uintptr_t>(slot_params)) & 15) != 0)
    return TOPOEP_EINVAL;
  if (replica_budget > 65535) return TOPOEP_ELIMIT;
  Gather g;
  g.R = R;
  g.N = replica_budget;
  g.E = E;
  g.self = self;
  g.words = bytes_per_expert / 16;
  g.slots = replica_slots;
  g.prev = prev_slots;
  g.params = static_cast<const v4i *>(expert_params);
  g.out = static_cast<v4i *>(slot_params);
  const int64_t chunks = (g.words + kGatherChunk - 1) / kGatherChunk;
  if (chunks > 0x7FFFFFFF) return TOPOEP_ELIMIT;
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)chunks, (unsigned)replica_budget), dim3(kGatherThreads), 0, st,
                     g);
  return hipGetLastError() == hipSuccess ? TOPOEP_OK : TOPOEP_EHIP;
}

}  // extern "C"
