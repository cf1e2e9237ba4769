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
//
// Few experts (E <= 16): the same step on 64 / W streams per wavefront (cache_seg_kernel,
// W = 8 or 16 lanes per stream, lane sl of segment g owning expert sl of stream g), so that
// the 16-lane SIMDs do not spend 4 cycles per instruction on 56 idle lanes. Bitmasks are the
// segment's bits of the ballots, and the stream-uniform values (selected set, clock, cache
// fill) are kept in every lane of the segment. A step's evictions are taken at once: the
// victims of its misses are the eligible experts of smallest key, each expert's rank among the
// segment's keys coming from DPP lane exchanges, which keeps the step free of a chain of
// reductions per miss. The selected sets of kSegChunk steps of every stream are first built in
// LDS (an LDS OR per valid entry); a set of fewer than K experts flags an invalid or repeated
// entry.

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

  const int chunk = 64 / K;  // steps per 64-entry load
  // entries of the steps n0 .. n0 + ns - 1 in lanes 0 .. ns K - 1; the next chunk's load is
  // issued before the current chunk is replayed (the first one before the state is read)
  auto load_chunk = [&](int n0) {
    const int ns = min(chunk, N - n0);
    return (n0 < N && lane < ns * K) ? tr[static_cast<long>(n0) * K + lane] : -1;
  };
  int v_next = load_chunk(0);

  if (POLICY == 1 && counts && lane < E) count = counts[stream * E + lane];
  if (state) {  // slots are listed oldest first; 64 slots per load, taken in order from the lanes
    const int32_t* st = state + stream * B;
    for (int s0 = 0; s0 < B; s0 += 64) {
      const int sv = s0 + lane < B ? st[s0 + lane] : -1;
      const int ns = min(64, B - s0);
      for (int i = 0; i < ns; ++i) {
        const int e = __builtin_amdgcn_readlane(sv, i);   // slot s0 + i
        if (e < 0) continue;
        const bool dup = e < E && ((__ballot(cached) >> e) & 1ull);
        if (e >= E || dup) {
          bad = true;
          continue;
        }
        if (lane == e) {
          cached = true;
          stamp = s0 + i;
        }
        ++ncached;
      }
    }
    clock = B;
  }

  long tot_f = 0, tot_h = 0;
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

constexpr int kSegChunk = 512;
constexpr int kSegBatch = 32;
constexpr int kSegMinSteps = 64;

// The value of lane (lane ^ x) for x = 1..W-1 within each aligned group of W lanes (W = 8 or
// 16), by DPP: quad permutations give x = 1..3, the half-row mirror x = 7 (and with a quad
// permutation after it x = 4..6), the row mirror x = 15 (and after it x = 8..14).
__device__ __forceinline__ int dpp_xor_quad(int v, int x) {   // x = 1, 2, 3
  return x == 1 ? __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false)    // quad_perm [1,0,3,2]
       : x == 2 ? __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false)    // quad_perm [2,3,0,1]
                : __builtin_amdgcn_update_dpp(v, v, 0x1B, 0xF, 0xF, false);   // quad_perm [3,2,1,0]
}

// Rank of each lane's key within its group of W lanes: the number of lanes of the group
// whose key is smaller. Every lane of the wavefront must be active.
template <int W>
__device__ __forceinline__ int seg_rank(int key) {
  int rank = 0;
  auto add8 = [&](int v) {   // the 8 lanes (lane ^ x), x = 0..7, of v
    const int m = __builtin_amdgcn_update_dpp(v, v, 0x141, 0xF, 0xF, false);   // row_half_mirror: x = 7
#pragma unroll
    for (int x = 1; x <= 3; ++x) {
      rank += dpp_xor_quad(v, x) < key ? 1 : 0;
      rank += dpp_xor_quad(m, x) < key ? 1 : 0;
    }
    rank += m < key ? 1 : 0;
  };
  add8(key);
  if (W == 16) {
    const int r = __builtin_amdgcn_update_dpp(key, key, 0x140, 0xF, 0xF, false);   // row_mirror: x = 15
    rank += r < key ? 1 : 0;
    add8(r);   // x = 15 ^ 1 .. 15 ^ 7 = 14 .. 8
  }
  return rank;
}

// The same rank for 64-bit keys given as (hi, lo), compared as (signed hi, unsigned lo).
template <int W>
__device__ __forceinline__ int seg_rank(int hi, int lo) {
  int rank = 0;
  auto less = [&](int h, int l) { return (h < hi || (h == hi && static_cast<uint32_t>(l) < static_cast<uint32_t>(lo))) ? 1 : 0; };
  auto add8 = [&](int vh, int vl) {
    const int mh = __builtin_amdgcn_update_dpp(vh, vh, 0x141, 0xF, 0xF, false);
    const int ml = __builtin_amdgcn_update_dpp(vl, vl, 0x141, 0xF, 0xF, false);
#pragma unroll
    for (int x = 1; x <= 3; ++x) {
      rank += less(dpp_xor_quad(vh, x), dpp_xor_quad(vl, x));
      rank += less(dpp_xor_quad(mh, x), dpp_xor_quad(ml, x));
    }
    rank += less(mh, ml);
  };
  add8(hi, lo);
  if (W == 16) {
    const int rh = __builtin_amdgcn_update_dpp(hi, hi, 0x140, 0xF, 0xF, false);
    const int rl = __builtin_amdgcn_update_dpp(lo, lo, 0x140, 0xF, 0xF, false);
    rank += less(rh, rl);
    add8(rh, rl);
  }
  return rank;
}

template <int W>
__device__ __forceinline__ uint32_t seg_bits(uint64_t ballot, int g) {
  return static_cast<uint32_t>(ballot >> (g * W)) & ((1u << W) - 1u);
}

template <int POLICY, int W>   // E <= W
__global__ __launch_bounds__(64) void cache_seg_kernel(
    const int32_t* __restrict__ trace, int L, int S, int N, int K, int E, int B,
    int32_t* __restrict__ state, int32_t* __restrict__ counts, int64_t* __restrict__ fetches,
    int64_t* __restrict__ hits, uint8_t* __restrict__ f_per_step, int32_t* __restrict__ dev_error) {
  constexpr int G = 64 / W;
  constexpr int LD = kSegChunk + 1;   // odd row stride: the segments' reads of one step fall on distinct banks
  __shared__ uint32_t sel_lds[G * LD];
  constexpr int FLD = kSegChunk + 4;   // f_lds rows one bank apart
  __shared__ uint8_t f_lds[G * FLD];
  const int lane = threadIdx.x, g = lane / W, sl = lane % W;
  const long nstreams = static_cast<long>(L) * S;
  const long stream0 = static_cast<long>(blockIdx.x) * G;
  const long stream = stream0 + g;
  const bool live = stream < nstreams;

  bool cached = false;
  int stamp = INT_MAX;
  int count = 0;
  int ncached = 0;
  int clock = 0;
  bool bad = false;

  if (POLICY == 1 && counts && live && sl < E) count = counts[stream * E + sl];
  if (state) {  // slots are listed oldest first
    for (int s = 0; s < B; ++s) {
      const int e = live ? state[stream * B + s] : -1;   // the same in every lane of the segment
      const uint32_t cm = seg_bits<W>(__ballot(cached), g);
      const bool use = e >= 0 && e < E && !((cm >> (e & (W - 1))) & 1u);
      bad = bad || (e >= 0 && !use);
      cached = cached || (use && sl == e);
      stamp = (use && sl == e) ? s : stamp;
      ncached += use ? 1 : 0;
    }
    clock = B;
  }

  long tot_f = 0, tot_h = 0;
  const float rk = 1.0f / static_cast<float>(K);
  for (int n0 = 0; n0 < N; n0 += kSegChunk) {
    const int ns = min(kSegChunk, N - n0);
    for (int i = lane; i < G * LD; i += 64) sel_lds[i] = 0;
    lds_sync();
    // each segment ORs its stream's valid entries into the steps' sets, kSegBatch loads in
    // flight per lane; invalid and repeated entries show up as sets of fewer than K experts
    if (live) {
      const int per = ns * K;
      const int32_t* tr = trace + (stream * N + n0) * static_cast<long>(K);
      for (int q0 = 0; q0 < per; q0 += W * kSegBatch) {
        int v[kSegBatch];
#pragma unroll
        for (int u = 0; u < kSegBatch; ++u) {
          const int q = q0 + u * W + sl;
          v[u] = q < per ? tr[q] : -1;
        }
#pragma unroll
        for (int u = 0; u < kSegBatch; ++u) {
          const int q = q0 + u * W + sl;
          // q / K in single precision: exact, the quotient being below 2^13 and K <= 16
          const int step = static_cast<int>((static_cast<float>(q) + 0.5f) * rk);
          if (v[u] >= 0 && v[u] < E) atomicOr(&sel_lds[g * LD + step], 1u << v[u]);
        }
      }
    }
    lds_sync();
    int chunk_f = 0, chunk_h = 0;
    uint32_t sel_next = sel_lds[g * LD];
    for (int j = 0; j < ns; ++j) {
      const uint32_t sel = sel_next;   // 0 for a segment without a stream
      sel_next = sel_lds[g * LD + j + 1];   // j + 1 <= kSegChunk < LD: inside the row
      const bool mine = (sel >> sl) & 1u;
      if (POLICY == 1) count += mine ? 1 : 0;
      const uint32_t cmask = seg_bits<W>(__ballot(cached), g);
      const uint32_t hitm = sel & cmask;
      const uint32_t missm = sel & ~cmask;
      const int h = __popc(hitm), nmiss = __popc(missm);
      const uint32_t below = (1u << sl) - 1u;
      if (POLICY != 2) {  // a hit becomes the most recently used
        stamp = ((hitm >> sl) & 1u) ? clock + __popc(hitm & below) : stamp;
        clock += h;
      }
      // The first B - ncached misses fill free slots; each later one evicts the eligible expert
      // (cached, not selected at this step) of smallest key. Inserted experts are selected, so
      // never eligible, and the eligible keys do not change during the step: the victims are
      // the nevict eligible experts of smallest key, found by rank (keys are distinct).
      const int nevict = max(0, ncached + nmiss - B);
      if (__ballot(nevict > 0)) {
        const bool eligible = cached && !mine;
        int rank;
        if (POLICY == 1) {  // lowest count first, then oldest stamp
          const long key = eligible ? static_cast<long>(count) * (1l << 32) + stamp : LONG_MAX;
          rank = seg_rank<W>(static_cast<int>(key >> 32), static_cast<int>(key & 0xffffffffl));
        } else {
          rank = seg_rank<W>(eligible ? stamp : INT_MAX);
        }
        const bool evict = eligible && rank < nevict;
        cached = cached && !evict;
        stamp = evict ? INT_MAX : stamp;
      }
      const bool insert = (missm >> sl) & 1u;   // misses take stamps in ascending expert order
      stamp = insert ? clock + __popc(missm & below) : stamp;
      cached = cached || insert;
      clock += nmiss;
      ncached += nmiss - nevict;
      bad = bad || (live && h + nmiss != K);
      chunk_h += h;
      chunk_f += nmiss;
      if (f_per_step) f_lds[g * FLD + j] = static_cast<uint8_t>(nmiss);   // the segment's lanes store the same byte
    }
    tot_h += chunk_h;
    tot_f += chunk_f;
    lds_sync();
    if (f_per_step) {
      for (int gg = 0; gg < G; ++gg) {
        if (stream0 + gg >= nstreams) break;
        for (int j = lane; j < ns; j += 64) f_per_step[(stream0 + gg) * N + n0 + j] = f_lds[gg * FLD + j];
      }
    }
  }

  if (__ballot(bad) && lane == 0 && dev_error) *dev_error = 1;
  if (!live) return;   // after the last cross-lane operation
  if (sl == 0) {
    fetches[stream] = tot_f;
    hits[stream] = tot_h;
  }
  if (POLICY == 1 && counts && sl < E) counts[stream * E + sl] = count;
  if (state) {
    int rank = 0;   // position of this cached expert, oldest first
    int nc = 0;
    for (int o = 0; o < W; ++o) {
      const int so = __shfl(cached ? stamp : INT_MAX, g * W + o, kWave);
      nc += so != INT_MAX ? 1 : 0;
      if (cached && so < stamp) ++rank;
    }
    int32_t* st = state + stream * B;
    for (int s = sl; s < B; s += W)
      if (s >= nc) st[s] = -1;
    if (cached) st[rank] = sl;
  }
}

template <int POLICY>
void launch_cache_policy(const int32_t* trace, int L, int S, int N, int K, int E, int B, int32_t* state,
                         int32_t* counts, int64_t* fetches, int64_t* hits, uint8_t* f_per_step, int32_t* dev_error,
                         hipStream_t stream) {
  const long streams = static_cast<long>(L) * S;
  // Short replays (a decode step's single step per stream) are dominated by the segmented
  // kernel's set-up (clearing its LDS sets); the one-wavefront kernel starts faster.
  if (N < kSegMinSteps) {
    const dim3 grid(static_cast<unsigned>((streams + kCacheWavesPerBlock - 1) / kCacheWavesPerBlock));
    hipLaunchKernelGGL(cache_kernel<POLICY>, grid, dim3(64 * kCacheWavesPerBlock), 0, stream, trace, L, S, N, K, E,
                       B, state, counts, fetches, hits, f_per_step, dev_error);
  } else if (E <= 8) {
    const dim3 grid(static_cast<unsigned>((streams + 7) / 8));
    hipLaunchKernelGGL((cache_seg_kernel<POLICY, 8>), grid, dim3(64), 0, stream, trace, L, S, N, K, E, B, state,
                       counts, fetches, hits, f_per_step, dev_error);
  } else if (E <= 16) {
    const dim3 grid(static_cast<unsigned>((streams + 3) / 4));
    hipLaunchKernelGGL((cache_seg_kernel<POLICY, 16>), grid, dim3(64), 0, stream, trace, L, S, N, K, E, B, state,
                       counts, fetches, hits, f_per_step, dev_error);
  } else {
    const dim3 grid(static_cast<unsigned>((streams + kCacheWavesPerBlock - 1) / kCacheWavesPerBlock));
    hipLaunchKernelGGL(cache_kernel<POLICY>, grid, dim3(64 * kCacheWavesPerBlock), 0, stream, trace, L, S, N, K, E,
                       B, state, counts, fetches, hits, f_per_step, dev_error);
  }
}

}  // namespace

hipError_t launch_cache(int policy, const int32_t* trace, int L, int S, int N, int K, int E, int B,
                        int32_t* state, int32_t* counts, int64_t* fetches, int64_t* hits,
                        uint8_t* f_per_step, int32_t* dev_error, hipStream_t stream) {
  const long streams = static_cast<long>(L) * S;
  if (streams == 0) return hipSuccess;
  if (policy == 1)
    launch_cache_policy<1>(trace, L, S, N, K, E, B, state, counts, fetches, hits, f_per_step, dev_error, stream);
  else if (policy == 2)
    launch_cache_policy<2>(trace, L, S, N, K, E, B, state, counts, fetches, hits, f_per_step, dev_error, stream);
  else
    launch_cache_policy<0>(trace, L, S, N, K, E, B, state, counts, fetches, hits, f_per_step, dev_error, stream);
  return hipGetLastError();
}

}  // namespace maskmoe
