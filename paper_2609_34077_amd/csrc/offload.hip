// Offloaded decode of one MoE layer, batch 1 (Section 1 and Section 3.1: the experts live in host
// memory, a layer keeps B of them in GPU memory, and every selected expert that is not cached is
// fetched over PCIe, evicting one cached expert under the policy when the cache is full;
// Section 4.1 for LRU, LFU and FIFO).
//
// The cache decision and the transfer run on the GPU, in stream order, with no host round trip:
// offload_cache_kernel applies the policy step of the trace replay (cache_step.hpp) to the
// token's selected experts and assigns each fetched expert a slot of the device pool (the slot
// its victim frees, else the lowest free one); offload_fetch_kernel then copies the fetched
// experts' weights from pinned host memory, read through its device mapping, into their slots.
// The few-token expert kernels read routed experts' weights through the slot map.
//
// Cache state of a layer (int32 [B + 2E], device): the cached experts oldest first (-1 = empty;
// the layout of the trace replay's state), the LFU access counts, and the slot of each expert
// (-1 when not cached). A state that is not self-consistent is reported and replaced by an
// empty cache, so the slots read afterwards always hold the experts the map names.

#include <limits.h>

#include "cache_step.hpp"
#include "common.hpp"
#include "kernels.hpp"

namespace maskmoe {
namespace {

constexpr int kFetchThreads = 256, kFetchUnroll = 4;

template <int POLICY>
__global__ __launch_bounds__(64) void offload_cache_kernel(const int32_t* __restrict__ idx, int E, int K, int B,
                                                           int32_t* __restrict__ state, int32_t* __restrict__ fetch,
                                                           int64_t* __restrict__ counters,
                                                           int32_t* __restrict__ dev_error) {
  const int lane = threadIdx.x;
  int32_t* order = state;
  int32_t* counts = state + B;
  int32_t* slot_of = state + B + E;
  bool cached = false, bad = false;
  int stamp = INT_MAX, count = 0, ncached = 0;
  int slot = lane < E ? slot_of[lane] : -1;
  if (lane < E) count = counts[lane];
  for (int s = 0; s < B; ++s) {   // oldest first
    const int e = order[s];      // wave-uniform
    if (e < 0) continue;
    if (e >= E || ((__ballot(cached) >> e) & 1ull)) {
      bad = true;
      continue;
    }
    if (lane == e) {
      cached = true;
      stamp = s;
    }
    ++ncached;
  }
  // every cached expert holds a distinct slot in [0, B); no other expert holds one
  if (__ballot(lane < E && (cached ? (slot < 0 || slot >= B) : slot != -1))) bad = true;
  uint64_t free_slots = B == 64 ? ~0ull : ((1ull << B) - 1);
  for (int s = 0; s < B; ++s) {
    const uint64_t m = __ballot(cached && slot == s);
    if (__popcll(m) > 1) bad = true;
    if (m) free_slots &= ~(1ull << s);
  }
  if (bad) {   // start from an empty cache
    cached = false;
    stamp = INT_MAX;
    slot = -1;
    ncached = 0;
    free_slots = B == 64 ? ~0ull : ((1ull << B) - 1);
  }
  uint64_t sel = 0;
  for (int k = 0; k < K; ++k) {
    const int e = idx[k];
    if (e < 0 || e >= E || ((sel >> e) & 1ull)) bad = true;
    else sel |= 1ull << e;
  }
  int clock = B, nf = 0;
  const int h = cache_step<POLICY>(sel, B, lane, cached, stamp, count, ncached, clock, [&](int e, int victim) {
    int s_new;
    if (victim >= 0) {
      s_new = __shfl(slot, victim, kWave);   // the victim's slot is freed for e
      if (lane == victim) slot = -1;
    } else {
      s_new = __ffsll(static_cast<unsigned long long>(free_slots)) - 1;
      free_slots &= free_slots - 1;
    }
    if (lane == e) slot = s_new;
    if (lane == 0) {
      fetch[1 + nf] = e;
      fetch[1 + K + nf] = s_new;
    }
    ++nf;
  });
  if (lane < E) {
    counts[lane] = count;
    slot_of[lane] = slot;
  }
  const int rank = cache_rank(cached, stamp);
  const int nc = __popcll(__ballot(cached));
  for (int s = lane; s < B; s += 64)
    if (s >= nc) order[s] = -1;
  if (cached) order[rank] = lane;
  if (lane == 0) {
    fetch[0] = nf;
    if (counters) {
      counters[0] += nf;
      counters[1] += h;
    }
    if (bad && dev_error) *dev_error = 1;
  }
}

// Copies fetch j (blockIdx.y) from host to its slot: both weight matrices of one expert as
// 16-byte units, kFetchUnroll loads in flight per thread.
__global__ __launch_bounds__(kFetchThreads) void offload_fetch_kernel(const int32_t* __restrict__ fetch, int K, int E,
                                                                      int B, const u32x4* __restrict__ host_gu,
                                                                      const u32x4* __restrict__ host_dn,
                                                                      u32x4* __restrict__ slots_gu,
                                                                      u32x4* __restrict__ slots_dn, size_t n_gu,
                                                                      size_t n_dn) {
  const int j = blockIdx.y;
  if (j >= fetch[0]) return;
  const int e = fetch[1 + j], s = fetch[1 + K + j];
  if (e < 0 || e >= E || s < 0 || s >= B) return;
  const u32x4* src_gu = host_gu + static_cast<size_t>(e) * n_gu;
  const u32x4* src_dn = host_dn + static_cast<size_t>(e) * n_dn;
  u32x4* dst_gu = slots_gu + static_cast<size_t>(s) * n_gu;
  u32x4* dst_dn = slots_dn + static_cast<size_t>(s) * n_dn;
  const size_t n = n_gu + n_dn;
  const size_t stride = static_cast<size_t>(gridDim.x) * kFetchThreads;
  size_t i = static_cast<size_t>(blockIdx.x) * kFetchThreads + threadIdx.x;
  for (; i + (kFetchUnroll - 1) * stride < n; i += kFetchUnroll * stride) {
    u32x4 v[kFetchUnroll];
#pragma unroll
    for (int u = 0; u < kFetchUnroll; ++u) {
      const size_t q = i + u * stride;
      v[u] = q < n_gu ? src_gu[q] : src_dn[q - n_gu];
    }
#pragma unroll
    for (int u = 0; u < kFetchUnroll; ++u) {
      const size_t q = i + u * stride;
      if (q < n_gu) dst_gu[q] = v[u];
      else dst_dn[q - n_gu] = v[u];
    }
  }
  for (; i < n; i += stride) {
    if (i < n_gu) dst_gu[i] = src_gu[i];
    else dst_dn[i - n_gu] = src_dn[i - n_gu];
  }
}

}  // namespace

hipError_t launch_offload_cache(int policy, const int32_t* idx, int E, int K, int B, int32_t* state, int32_t* fetch,
                                int64_t* counters, int32_t* dev_error, hipStream_t stream) {
  if (policy == 1)
    hipLaunchKernelGGL(offload_cache_kernel<1>, dim3(1), dim3(64), 0, stream, idx, E, K, B, state, fetch, counters,
                       dev_error);
  else if (policy == 2)
    hipLaunchKernelGGL(offload_cache_kernel<2>, dim3(1), dim3(64), 0, stream, idx, E, K, B, state, fetch, counters,
                       dev_error);
  else
    hipLaunchKernelGGL(offload_cache_kernel<0>, dim3(1), dim3(64), 0, stream, idx, E, K, B, state, fetch, counters,
                       dev_error);
  return hipGetLastError();
}

hipError_t launch_offload_fetch(const int32_t* fetch, int K, int E, int B, int d, int F, const void* host_gu,
                                const void* host_dn, void* slots_gu, void* slots_dn, hipStream_t stream) {
  const size_t n_gu = static_cast<size_t>(2) * F * d * 2 / 16, n_dn = static_cast<size_t>(d) * F * 2 / 16;
  hipLaunchKernelGGL(offload_fetch_kernel, dim3(kOffloadFetchBlocks, K), dim3(kFetchThreads), 0, stream, fetch, K, E,
                     B, static_cast<const u32x4*>(host_gu), static_cast<const u32x4*>(host_dn),
                     static_cast<u32x4*>(slots_gu), static_cast<u32x4*>(slots_dn), n_gu, n_dn);
  return hipGetLastError();
}

}  // namespace maskmoe
