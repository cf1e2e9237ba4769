// One step of the per-layer expert cache (Section 4.1, Simulation; Eq. 5), shared by the trace
// replay (cache.hip) and the offloaded decode (offload.hip), so both apply the same policy.
//
// Wavefront layout: lane e owns expert e (E <= 64) and holds `cached`, `stamp` (last use for LRU
// and LFU, insertion time for FIFO; INT_MAX when not cached) and, for LFU, `count` (accesses of
// the stream so far). `ncached` and `clock` are wave-uniform. A step with selected set `sel`:
// count the accesses (LFU); the hits become the most recently used in ascending expert order
// (LRU, LFU); then every miss, in ascending expert order, evicts when the cache is full the
// cached expert not selected at this step with the smallest stamp (LRU, FIFO) or the smallest
// (count, stamp) (LFU), and is inserted with the next stamp. on_insert(e, victim) runs for each
// miss before e is marked cached (victim = -1 when nothing was evicted; the victim lane is
// already cleared). Returns the hits; the misses are popc(sel) - hits.
#pragma once

#include <limits.h>

#include "common.hpp"

namespace maskmoe {

template <int POLICY, class OnInsert>   // POLICY: 0 LRU, 1 LFU, 2 FIFO
__device__ __forceinline__ int cache_step(uint64_t sel, int B, int lane, bool& cached, int& stamp, int& count,
                                          int& ncached, int& clock, OnInsert&& on_insert) {
  const bool mine = (sel >> lane) & 1ull;
  if (POLICY == 1 && mine) ++count;
  const uint64_t cmask = __ballot(cached);
  const uint64_t hitm = sel & cmask;
  uint64_t missm = sel & ~cmask;
  const int h = __popcll(hitm);
  if (POLICY != 2) {  // a hit becomes the most recently used
    if ((hitm >> lane) & 1ull) stamp = clock + __popcll(hitm & lanemask_lt(lane));
    clock += h;
  }
  while (missm) {
    const int e = __ffsll(static_cast<unsigned long long>(missm)) - 1;
    missm &= missm - 1;
    int victim = -1;
    if (ncached >= B) {
      const bool eligible = cached && !mine;
      int key;
      if (POLICY == 1) {  // lowest count first, then oldest stamp
        const int low = wave_min_int(eligible ? count : INT_MAX);
        key = (eligible && count == low) ? stamp : INT_MAX;
      } else {
        key = eligible ? stamp : INT_MAX;
      }
      const int mn = wave_min_int(key);
      const uint64_t vm = __ballot(eligible && key == mn);
      victim = __ffsll(static_cast<unsigned long long>(vm)) - 1;
      if (lane == victim) {
        cached = false;
        stamp = INT_MAX;
      }
      --ncached;
    }
    on_insert(e, victim);
    if (lane == e) {
      cached = true;
      stamp = clock;
    }
    ++clock;
    ++ncached;
  }
  return h;
}

// Slot of each cached expert in a list ordered by stamp (oldest first): the number of cached
// experts with a smaller stamp.
__device__ __forceinline__ int cache_rank(bool cached, int stamp) {
  int rank = 0;
  for (int o = 0; o < 64; ++o) {
    const int so = __shfl(cached ? stamp : INT_MAX, o, kWave);
    if (cached && so < stamp) ++rank;
  }
  return rank;
}

}  // namespace maskmoe
