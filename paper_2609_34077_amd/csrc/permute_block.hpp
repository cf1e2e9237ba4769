// Token permutation by expert, run by one workgroup of `nthreads` threads (the launch's block
// size, a multiple of 64, <= 1024).
//
// The combine of Eq. 1 (Section 3.1) sums, for every token, the outputs of the experts it
// selected. To run each expert as one dense GEMM over the tokens that chose it, the T*K
// (token, slot) entries j = t*K + k are grouped by expert, keeping entry order inside a
// group (a stable counting sort), and n_shared groups holding every token are appended
// for the shared experts (Section 3.1). Outputs, with G = E + n_shared groups:
//   offsets[g]   first row of group g (offsets[G] = T*(K + n_shared))
//   tile_off[g]  first row-tile of group g in units of `tile_rows` (tile_off[G] = total)
//   active[i]    the i-th non-empty group, n_active[0] their count
//   perm[pos]    entry j placed at row pos (routed rows only), inv[j] = pos
//   row_tok[pos] token of row pos (routed and shared rows)
// LDS histogram, scan, then a chunked stable scatter where the rank of an entry among equal
// experts inside a wavefront comes from ballots on the expert id bits. Integer only,
// deterministic. `idx` may have been written by this workgroup just before the call, after
// a barrier that orders it (lds_sync for LDS, __syncthreads for global memory). The threads
// exchange data through LDS only; the outputs are written, never read back.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace maskmoe {

constexpr int kPermMaxWaves = 16;
constexpr int kPermMaxGroups = 256 + 8;

struct PermLds {
  int hist[kPermMaxGroups];
  int running[kPermMaxGroups];
  int wcnt[kPermMaxWaves][kPermMaxGroups];
};

__device__ inline void permute_block(const int32_t* idx, int T, int K, int E, int n_shared, int tile_rows,
                                     const PermBuffers& pb, PermLds& s, int nthreads) {
  const int nwaves = nthreads / kWave;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = T * K;
  const int G = E + n_shared;

  for (int g = tid; g < G; g += nthreads) s.hist[g] = 0;
  lds_sync();
  for (int j = tid; j < n; j += nthreads) {
    const int e = idx[j];
    if (e >= 0 && e < E) atomicAdd(&s.hist[e], 1);  // LDS integer counts: order-independent
  }
  lds_sync();
  if (tid == 0) {
    int off = 0, toff = 0, na = 0;
    for (int g = 0; g < G; ++g) {
      const int c = g < E ? s.hist[g] : T;
      pb.offsets[g] = off;
      pb.tile_off[g] = toff;
      s.running[g] = off;
      if (c > 0) pb.active[na++] = g;
      off += c;
      toff += (c + tile_rows - 1) / tile_rows;
    }
    pb.offsets[G] = off;
    pb.tile_off[G] = toff;
    pb.n_active[0] = na;
  }
  // shared-expert rows: token t of shared expert s sits at row n + s*T + t
  for (int r = tid; r < n_shared * T; r += nthreads) pb.row_tok[n + r] = r % T;
  lds_sync();

  for (int base = 0; base < n; base += nthreads) {
    const int j = base + tid;
    const int e = (j < n) ? idx[j] : -1;
    const bool valid = e >= 0 && e < E;
    // lanes of this wavefront holding the same expert
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 9; ++b) {
      const uint64_t bb = __ballot(valid && ((e >> b) & 1));
      same &= ((e >> b) & 1) ? bb : ~bb;
    }
    for (int g = lane; g < G; g += kWave) s.wcnt[wave][g] = 0;
    lds_sync();
    const uint64_t lower = same & lanemask_lt(lane);
    if (valid && lower == 0) s.wcnt[wave][e] = __popcll(same);
    lds_sync();
    if (valid) {
      int pos = s.running[e] + __popcll(lower);
      for (int w = 0; w < wave; ++w) pos += s.wcnt[w][e];
      pb.perm[pos] = j;
      pb.inv[j] = pos;
      pb.row_tok[pos] = j / K;
    }
    lds_sync();
    for (int g = tid; g < E; g += nthreads) {
      int sum = 0;
      for (int w = 0; w < nwaves; ++w) sum += s.wcnt[w][g];
      s.running[g] += sum;
    }
    lds_sync();
  }
}

// Inclusive prefix sum over the 64 lanes with DPP lane shifts: within each 16-lane row by
// shifts of 1, 2, 4, 8 (lanes shifted in from outside the row add 0), then the last lane of
// rows 0 and 2 is added to rows 1 and 3 (row_bcast:15) and lane 31 to rows 2 and 3
// (row_bcast:31).
__device__ __forceinline__ int wave_inclusive_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);   // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);   // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);   // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);   // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);   // row_bcast:15 into rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);   // row_bcast:31 into rows 2, 3
  return v;
}

// The same layout computed by one wavefront, for n = T*K <= 64 entries and G = E + n_shared < 64
// groups: lane j holds entry j and lane g group g. Group sizes come from a pass over the
// entries, first rows and row-tiles from lane prefix sums, the rank of an entry among equal
// experts from ballots on the expert id bits; no LDS passes and no barriers. Same outputs as
// permute_block (and the same contract for `idx`).
__device__ inline void permute_wave(const int32_t* idx, int T, int K, int E, int n_shared, int tile_rows,
                                    const PermBuffers& pb) {
  const int lane = threadIdx.x & 63;
  const int n = T * K, G = E + n_shared;
  const int e = lane < n ? idx[lane] : -1;
  const bool valid = e >= 0 && e < E;
  uint64_t same = __ballot(valid);   // lanes holding the same expert (E < 64: six id bits)
#pragma unroll
  for (int b = 0; b < 6; ++b) {
    const uint64_t bb = __ballot(valid && ((e >> b) & 1));
    same &= ((e >> b) & 1) ? bb : ~bb;
  }
  int c = 0;   // entries of expert `lane` (an invalid entry matches no lane below E)
  for (int j = 0; j < n; ++j) c += __builtin_amdgcn_readlane(e, j) == lane ? 1 : 0;
  if (lane >= E) c = lane < G ? T : 0;   // shared groups hold every token; none past G
  const int tiles = (c + tile_rows - 1) / tile_rows;
  int off = wave_inclusive_sum(c), toff = wave_inclusive_sum(tiles);
  off -= c;   // first row and row-tile of group `lane`; lane G: the totals
  toff -= tiles;
  if (lane <= G) {
    pb.offsets[lane] = off;
    pb.tile_off[lane] = toff;
  }
  const uint64_t act = __ballot(lane < G && c > 0);
  if (lane < G && c > 0) pb.active[__popcll(act & lanemask_lt(lane))] = lane;
  if (lane == 0) pb.n_active[0] = __popcll(act);
  // shared-expert rows: token t of shared expert s sits at row n + s*T + t
  for (int r = lane; r < n_shared * T; r += kWave) pb.row_tok[n + r] = r % T;
  const int first = __shfl(off, valid ? e : 0);
  if (valid) {
    const int pos = first + __popcll(same & lanemask_lt(lane));
    pb.perm[pos] = lane;
    pb.inv[lane] = pos;
    pb.row_tok[pos] = lane / K;
  }
}

}  // namespace maskmoe
