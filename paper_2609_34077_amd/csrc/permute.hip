// Token permutation by expert for many tokens (the layout of permute_block.hpp: stable
// grouping of the T*K (token, slot) entries by expert, n_shared groups of all tokens appended),
// spread over the chip in three passes over chunks of kPermChunk entries:
//   1. permute_count_kernel: one workgroup per chunk counts its entries per expert;
//   2. permute_scan_kernel: one workgroup turns the counts into each chunk's first row per
//      expert (a prefix over chunks) and the group offsets, tile offsets and active list;
//   3. permute_scatter_kernel: one workgroup per chunk places its entries, ranked among equal
//      experts in entry order (ballots within a wavefront, per-wavefront counts in LDS).
// Integer only, no global atomics: the result is the same as the single-workgroup version.

#include "permute_block.hpp"

namespace maskmoe {
namespace {

constexpr int kPermThreads = 1024;   // one entry per thread and chunk

__global__ __launch_bounds__(kPermThreads) void permute_count_kernel(const int32_t* __restrict__ idx, int n, int E,
                                                                    int32_t* __restrict__ counts) {
  __shared__ int hist[kPermMaxGroups];
  const int tid = threadIdx.x, c = blockIdx.x;
  for (int g = tid; g < E; g += kPermThreads) hist[g] = 0;
  __syncthreads();
  const int j = c * kPermChunk + tid;
  if (j < n) {
    const int e = idx[j];
    if (e >= 0 && e < E) atomicAdd(&hist[e], 1);   // LDS integer counts: order-independent
  }
  __syncthreads();
  for (int g = tid; g < E; g += kPermThreads) counts[static_cast<size_t>(c) * E + g] = hist[g];
}

__global__ __launch_bounds__(kPermThreads) void permute_scan_kernel(int32_t* __restrict__ counts, int n_chunks, int T,
                                                                   int E, int n_shared, int tile_rows,
                                                                   PermBuffers pb) {
  __shared__ int total[kPermMaxGroups];
  const int tid = threadIdx.x;
  const int G = E + n_shared;
  constexpr int U = 16;   // chunk counts loaded together: a few memory round trips, not one per chunk
  for (int g = tid; g < E; g += kPermThreads) {   // counts -> first row of each chunk within group g
    int run = 0;
    for (int c0 = 0; c0 < n_chunks; c0 += U) {
      int v[U];
#pragma unroll
      for (int i = 0; i < U; ++i) v[i] = c0 + i < n_chunks ? counts[static_cast<size_t>(c0 + i) * E + g] : 0;
#pragma unroll
      for (int i = 0; i < U; ++i) {
        if (c0 + i < n_chunks) counts[static_cast<size_t>(c0 + i) * E + g] = run;
        run += v[i];
      }
    }
    total[g] = run;
  }
  lds_sync();
  if (tid < kWave) {   // one wavefront: lane l takes groups l*PG .. l*PG + PG - 1 in order
    constexpr int PG = (kPermMaxGroups + kWave - 1) / kWave;
    const int g0 = tid * PG;
    int cnt[PG], til[PG], sc = 0, st = 0, sa = 0;
#pragma unroll
    for (int i = 0; i < PG; ++i) {
      const int g = g0 + i;
      cnt[i] = g < G ? (g < E ? total[g] : T) : 0;
      til[i] = (cnt[i] + tile_rows - 1) / tile_rows;
      sc += cnt[i];
      st += til[i];
      sa += cnt[i] > 0 ? 1 : 0;
    }
    int off = wave_inclusive_sum(sc) - sc, toff = wave_inclusive_sum(st) - st, na = wave_inclusive_sum(sa) - sa;
#pragma unroll
    for (int i = 0; i < PG; ++i) {
      const int g = g0 + i;
      if (g <= G) {   // offsets[G], tile_off[G]: the totals
        pb.offsets[g] = off;
        pb.tile_off[g] = toff;
      }
      if (g < G && cnt[i] > 0) pb.active[na++] = g;
      off += cnt[i];
      toff += til[i];
    }
    if (tid == kWave - 1) pb.n_active[0] = na;
  }
}

__global__ __launch_bounds__(kPermThreads) void permute_scatter_kernel(const int32_t* __restrict__ idx, int T, int K,
                                                                      int E, int n_shared,
                                                                      const int32_t* __restrict__ counts,
                                                                      PermBuffers pb) {
  __shared__ int wcnt[kPermThreads / kWave][kPermMaxGroups];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, c = blockIdx.x;
  const int n = T * K;
  // shared-expert rows: token t of shared expert s sits at row n + s*T + t
  for (int r = c * kPermThreads + tid; r < n_shared * T; r += gridDim.x * kPermThreads) pb.row_tok[n + r] = r % T;
  const int j = c * kPermChunk + tid;
  const int e = j < n ? idx[j] : -1;
  const bool valid = e >= 0 && e < E;
  uint64_t same = __ballot(valid);   // lanes of this wavefront holding the same expert
#pragma unroll
  for (int b = 0; b < 9; ++b) {
    const uint64_t bb = __ballot(valid && ((e >> b) & 1));
    same &= ((e >> b) & 1) ? bb : ~bb;
  }
  for (int g = lane; g < E; g += kWave) wcnt[wave][g] = 0;
  lds_sync();
  const uint64_t lower = same & lanemask_lt(lane);
  if (valid && lower == 0) wcnt[wave][e] = __popcll(same);
  __syncthreads();
  if (valid) {
    int pos = pb.offsets[e] + counts[static_cast<size_t>(c) * E + e] + __popcll(lower);
    for (int w = 0; w < wave; ++w) pos += wcnt[w][e];
    pb.perm[pos] = j;
    pb.inv[j] = pos;
    pb.row_tok[pos] = j / K;
  }
}

}  // namespace

hipError_t launch_permute(const int32_t* idx, int T, int K, int E, int n_shared, int tile_rows,
                          const PermBuffers& pb, int32_t* chunk_counts, hipStream_t stream) {
  const int n = T * K;
  const int n_chunks = permute_chunks(T, K);
  if (n_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(permute_count_kernel, dim3(n_chunks), dim3(kPermThreads), 0, stream, idx, n, E, chunk_counts);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(permute_scan_kernel, dim3(1), dim3(kPermThreads), 0, stream, chunk_counts, n_chunks, T, E,
                     n_shared, tile_rows, pb);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(permute_scatter_kernel, dim3(n_chunks), dim3(kPermThreads), 0, stream, idx, T, K, E, n_shared,
                     chunk_counts, pb);
  return hipGetLastError();
}

}  // namespace maskmoe
