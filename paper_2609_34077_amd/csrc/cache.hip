// Per-layer expert cache replay behind the hit rate and fetches-per-token metrics.
//
// Section 4.1 (Simulation): every layer keeps a cache of B routed experts; caches start
// empty (or from a given state), initial fills are misses, each miss is one fetch and,
// when the cache is full, one eviction under LRU, LFU or FIFO. Eq. 5: h_{l,t} = selected
// experts already cached, f_{l,t} = K - h_{l,t}; HR = sum h / (N L K), Fetches/tok = sum f / N.
//
// One wavefront replays one (layer, stream) trace; lane e owns expert e (E <= 64) and keeps
// a cached flag, a stamp (last use for LRU and LFU, insertion time for FIFO) and, for LFU,
// its access count. A step is a handful of wave-uniform bitmask operations: ballot the
// cached set, intersect with the selected set for the hits, count the accesses (LFU), stamp
// the hits in ascending expert order (LRU, LFU), then insert the misses in ascending order,
// each evicting, among the cached experts not selected at this step, the smallest stamp
// (LRU, FIFO) or the smallest (count, stamp) (LFU). The trace is read 64 entries at a time,
// coalesced; once per chunk, lane j turns the entries of step j into that step's selected-set
// bitmask (and flags invalid entries), and each step then reads its mask back as one
// wave-uniform value (readlane). Per-step miss counts are gathered in lanes and written 64
// bytes at a time.

#include <limits.h>

#include "cache_step.hpp"
#include "common.hpp"
#include "kernels.hpp"

namespace maskmoe {
namespace {

constexpr int kCacheWavesPerBlock = 4;

template <int POLICY>  // 0 LRU, 1 LFU, 2 FIFO
__global__ __launch_bounds__(64 * kCacheWavesPerBlock) void cache_kernel(
    const int32_t* __restrict__ trace, int L, int S, int N, int K, int E, int B,
    int32_t* __restrict__ state, int32_t* __restrict__ counts, int64_t* __restrict__ fetches,
    int64_t* __restrict__ hits, uint8_t* __restrict__ f_per_step, int32_t* __restrict__ dev_error) {
  const int lane = threadIdx.x & 63;
  const long stream = static_cast<long>(blockIdx.x) * kCacheWavesPerBlock + (threadIdx.x >> 6);
  if (stream >= static_cast<long>(L) * S) return;  // whole wavefront exits together
  const int32_t* tr = trace + stream * static_cast<long>(N) * K;

  bool cached = false;
  int stamp = INT_MAX;
  int count = 0;
  int ncached = 0;
  int clock = 0;
  bool bad = false;

  if (POLICY == 1 && counts && lane < E) count = counts[stream * E + lane];
  if (state) {  // slots are listed oldest first
    const int32_t* st = state + stream * B;
    for (int s = 0; s < B; ++s) {
      const int e = st[s];  // wave-uniform
      if (e < 0) continue;
      const bool dup = e < E && ((__ballot(cached) >> e) & 1ull);
      if (e >= E || dup) {
        bad = true;
        continue;
      }
      if (lane == e) {
        cached = true;
        stamp = s;
      }
      ++ncached;
    }
    clock = B;
  }

  long tot_f = 0, tot_h = 0;
  const int chunk = 64 / K;  // steps per 64-entry load
  // entries of the steps n0 .. n0 + ns - 1 in lanes 0 .. ns K - 1; the next chunk's load is
  // issued before the current chunk is replayed
  auto load_chunk = [&](int n0) {
    const int ns = min(chunk, N - n0);
    return (n0 < N && lane < ns * K) ? tr[static_cast<long>(n0) * K + lane] : -1;
  };
  int v_next = load_chunk(0);
  for (int n0 = 0; n0 < N; n0 += chunk) {
    const int ns = min(chunk, N - n0);
    const int v = v_next;
    v_next = load_chunk(n0 + chunk);
    // lane j < ns builds the selected set of step n0 + j from its K entries, once per chunk
    uint64_t my_sel = 0;
    bool my_bad = false;
    for (int k = 0; k < K; ++k) {
      const int e = __shfl(v, (lane * K + k) & 63, kWave);
      if (lane < ns) {
        if (e < 0 || e >= E || ((my_sel >> e) & 1ull)) my_bad = true;
        else my_sel |= 1ull << e;
      }
    }
    if (__ballot(my_bad)) bad = true;
    const int sel_lo = static_cast<int>(my_sel & 0xffffffffull);
    const int sel_hi = static_cast<int>(my_sel >> 32);
    int my_f = 0;
    for (int j = 0; j < ns; ++j) {
      // the step's set, read back as a wave-uniform (scalar) value
      const uint64_t sel = (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readlane(sel_hi, j))) << 32) |
                           static_cast<uint32_t>(__builtin_amdgcn_readlane(sel_lo, j));
      const int h = cache_step<POLICY>(sel, B, lane, cached, stamp, count, ncached, clock, [](int, int) {});
      const int f = __popcll(sel) - h;
      tot_h += h;
      tot_f += f;
      if (lane == j) my_f = f;
    }
    if (f_per_step && lane < ns) f_per_step[stream * N + n0 + lane] = static_cast<uint8_t>(my_f);
  }

  if (lane == 0) {
    fetches[stream] = tot_f;
    hits[stream] = tot_h;
    if (bad && dev_error) *dev_error = 1;
  }
  if (POLICY == 1 && counts && lane < E) counts[stream * E + lane] = count;
  if (state) {
    const int rank = cache_rank(cached, stamp);   // its position, oldest first
    int32_t* st = state + stream * B;
    const int nc = __popcll(__ballot(cached));
    for (int s = lane; s < B; s += 64)
      if (s >= nc) st[s] = -1;
    if (cached) st[rank] = lane;
  }
}

}  // namespace

hipError_t launch_cache(int policy, const int32_t* trace, int L, int S, int N, int K, int E, int B,
                        int32_t* state, int32_t* counts, int64_t* fetches, int64_t* hits,
                        uint8_t* f_per_step, int32_t* dev_error, hipStream_t stream) {
  const long streams = static_cast<long>(L) * S;
  if (streams == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((streams + kCacheWavesPerBlock - 1) / kCacheWavesPerBlock));
  const dim3 block(64 * kCacheWavesPerBlock);
  if (policy == 1)
    hipLaunchKernelGGL(cache_kernel<1>, grid, block, 0, stream, trace, L, S, N, K, E, B, state, counts, fetches,
                       hits, f_per_step, dev_error);
  else if (policy == 2)
    hipLaunchKernelGGL(cache_kernel<2>, grid, block, 0, stream, trace, L, S, N, K, E, B, state, counts, fetches,
                       hits, f_per_step, dev_error);
  else
    hipLaunchKernelGGL(cache_kernel<0>, grid, block, 0, stream, trace, L, S, N, K, E, B, state, counts, fetches,
                       hits, f_per_step, dev_error);
  return hipGetLastError();
}

}  // namespace maskmoe
