// The 256 x 256 x 64 bf16 MFMA tile pipeline shared by the expert GEMMs (forward, dgrad and
// wgrad): acc += A_tile * B_tile^T for 256 rows of A and 256 rows of B, both K-contiguous.
//
// 512 threads in 8 waves (2 along A rows x 4 along B rows); each wave owns 4 x 2 fragments of
// v_mfma_f32_32x32x16_bf16 (128 A rows x 64 B rows). Thread tid loads 16-byte chunks of rows
// (tid >> 3) + 64 i (i < 4) of each operand; LDS slot u = tid + 512 i (row u >> 3, physical
// chunk u & 7) receives the logical chunk (u & 7) ^ lds_swizzle(row), which keeps the operand
// reads free of bank conflicts. Pipeline: k-tile kt sits in LDS buffer kt & 1 and tile kt + 1 in
// registers; right after the first k16 step of tile kt the registers go to the other buffer and
// are refilled with tile kt + 2, so every global load has a whole k-tile of MFMA work to
// arrive. Operand fragments of the next k16 step are read while the current one multiplies.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace maskmoe {

constexpr int kTileM = 256, kTileN = 256, kTileK = 64, kTileThreads = 512;
constexpr int kTileU = kTileM * 8 / kTileThreads;   // 16-byte units per thread, operand and stage
constexpr int kTileTM = 4, kTileTN = 2;             // 32x32 fragments per wave

// Row r0 = tid >> 3 of a thread's first unit and its swizzled chunk offset (elements).
__device__ __forceinline__ int tile_load_row() { return threadIdx.x >> 3; }
__device__ __forceinline__ int tile_load_chunk() {
  return ((threadIdx.x & 7) ^ lds_swizzle(threadIdx.x >> 3)) * 8;
}

// One more k-tile ahead of the main operands: its rows of A at xa + xaoffs[i], of B at
// xb + xboffs[i] (64 elements each, chunk included). The low-rank adapters use it: A' = [U | X],
// B' = [s B | W] turns W x + s B (A x) into one product. It is the first tile, so only the
// prologue loads it and the steady-state loop is the same as without it.
struct TileExtra {
  const uint16_t* xa;
  const uint16_t* xb;
  int xaoffs[kTileU];
  int xboffs[kTileU];
};

// aoffs / boffs: element offsets from abase / bbase of the thread's unit i rows, chunk included
// (rows r0 + 64 i of the tile); aoff / boff: 16-byte LDS slot offsets of the wave's fragment
// rows (row * 8). nk: k-tiles of 64 of the main operands (none and no extra tile leaves acc
// unchanged). BSTEP: elements between consecutive k-tiles of a B row (kTileK row-major,
// kPackBlock in the packed weight layout).
template <bool EXTRA = false, int BSTEP = kTileK>
__device__ __forceinline__ void gemm_tile_mainloop(const uint16_t* __restrict__ abase, const int (&aoffs)[kTileU],
                                                   const uint16_t* __restrict__ bbase, const int (&boffs)[kTileU],
                                                   const int (&aoff)[kTileTM], const int (&boff)[kTileTN], int nk,
                                                   f32x16 (&acc)[kTileTM][kTileTN], u32x4 (*lds_a)[kTileM * 8],
                                                   u32x4 (*lds_b)[kTileN * 8], const TileExtra* extra = nullptr) {
  constexpr int U = kTileU, TM = kTileTM, TN = kTileTN, BK = kTileK, NT = kTileThreads;
  constexpr int X = EXTRA ? 1 : 0;   // pipeline tile kt holds main tile kt - X
  const int ntot = nk + X;
  if (ntot <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int sw = lds_swizzle(lane);   // fragment rows are a multiple of 32 plus (lane & 31)
  u32x4 ra[U], rb[U];
  auto gload = [&](int t) {   // main tile t
#pragma unroll
    for (int i = 0; i < U; ++i) {
      ra[i] = *reinterpret_cast<const u32x4*>(abase + (aoffs[i] + t * BK));
      rb[i] = *reinterpret_cast<const u32x4*>(bbase + (boffs[i] + t * BSTEP));
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < U; ++i) {
      lds_a[buf][tid + NT * i] = ra[i];
      lds_b[buf][tid + NT * i] = rb[i];
    }
  };
  u32x4 af[2][TM], bf[2][TN];
  auto read_frags = [&](int buf, int kk, int slot) {
    const int ch = (kk * 2 + (lane >> 5)) ^ sw;
#pragma unroll
    for (int i = 0; i < TM; ++i) af[slot][i] = lds_a[buf][aoff[i] + ch];
#pragma unroll
    for (int j = 0; j < TN; ++j) bf[slot][j] = lds_b[buf][boff[j] + ch];
  };

  if (EXTRA) {
#pragma unroll
    for (int i = 0; i < U; ++i) {
      ra[i] = *reinterpret_cast<const u32x4*>(extra->xa + extra->xaoffs[i]);
      rb[i] = *reinterpret_cast<const u32x4*>(extra->xb + extra->xboffs[i]);
    }
  } else {
    gload(0);
  }
  lstore(0);
  gload(min(1 - X, nk - 1));
  __syncthreads();
  read_frags(0, 0, 0);
  // The loop body has no branches, so that LDS stores and global loads can be interleaved
  // with the MFMAs (LLVM's MFMA/DS interleaving strategy 0): past the end, the last main tile is
  // loaded again and stored into the idle buffer, which nothing reads afterwards (every LDS
  // access of the loop has completed at its last barrier).
  for (int kt = 0; kt < ntot; ++kt) {
    const int buf = kt & 1;
    __builtin_amdgcn_iglp_opt(0);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int cur = kk & 1;
      if (kk + 1 < BK / 16) read_frags(buf, kk + 1, cur ^ 1);
      if (kk == 0) {
        lstore(buf ^ 1);
        gload(min(kt + 2 - X, nk - 1));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma_32x32x16(af[cur][i], bf[cur][j], acc[i][j]);
    }
    __syncthreads();
    read_frags(buf ^ 1, 0, 0);
  }
}

// XCD-aware tile order: the hardware deals workgroup ids round-robin over the 8 XCDs, so ids
// are remapped to give each XCD a contiguous range of logical tiles; logical tiles come in
// groups of 4 column tiles, the column tile varying fastest, so the ~32 workgroups an XCD runs
// at once cover about 8 row tiles x 4 column tiles and share both operands in its L2.
// Returns the logical tile id of this workgroup when the first nwg workgroups of the grid are
// the live ones (nwg = gridDim.x by default).
__device__ __forceinline__ int xcd_tile_id(int nwg) {
  const int bid = blockIdx.x;
  const int xcd = bid & 7, local = bid >> 3, q = nwg >> 3, rem = nwg & 7;
  return xcd < rem ? xcd * (q + 1) + local : rem * (q + 1) + (xcd - rem) * q + local;
}
__device__ __forceinline__ int xcd_tile_id() { return xcd_tile_id(static_cast<int>(gridDim.x)); }

__device__ __forceinline__ void grouped_tile_coords(int lid, int mt_max, int n_tiles, int& mt, int& nt) {
  constexpr int GN = 4;
  const int per_group = GN * mt_max;
  const int first_n = (lid / per_group) * GN;
  const int gsize = min(n_tiles - first_n, GN);
  const int within = lid % per_group;
  nt = first_n + within % gsize;
  mt = within / gsize;
}

// Tail split. The hardware deals workgroups round-robin over the 8 XCDs; XCD x takes a
// contiguous range of the live tiles (the partition of xcd_tile_id) and runs cu_xcd of them at
// a time. All tiles cost the same, so the r tiles of an XCD's last, partial round would leave
// most of its CUs idle; instead each of them is split into s reduction slices (the largest
// power of two <= kTailMaxSplit with r * s <= min(cu_xcd, kTailSlotsPerXcd), s dividing the
// k-tiles and leaving >= kTailMinK per slice), so the last round is short and full. A slice
// writes its partial tile to a slot (tail_store_partial); a fix-up kernel adds a tile's slices
// in slice order (tail_sum_partials) and applies the GEMM's epilogue, so results stay
// deterministic.
constexpr int kTailSlotsPerXcd = kTailSlots / 8;
constexpr int kTailMaxSplit = 8, kTailMinK = 16;
// a split into two slices is possible: nk even, >= kTailMinK k-tiles each
__host__ __device__ constexpr bool tail_splittable(int nk) { return nk % 2 == 0 && nk / 2 >= kTailMinK; }

struct TileJob {
  int lid;    // logical tile (grouped_tile_coords order)
  int z, s;   // reduction slice z of s (s == 1: the whole tile)
  int slot;   // partial-tile slot when s > 1
};

struct XcdShare {
  int base, full, r, s;   // first tile, tiles run whole, tail tiles, their slices
};

__device__ __forceinline__ XcdShare xcd_share(int xcd, int live, int cu_xcd, int nk, bool split_ok) {
  XcdShare x;
  const int q = live >> 3, rem = live & 7;
  const int count = q + (xcd < rem ? 1 : 0);
  x.base = xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q;
  x.full = count / cu_xcd * cu_xcd;
  x.r = count - x.full;
  const int cap = min(cu_xcd, kTailSlotsPerXcd);
  x.s = 1;
  if (split_ok && x.r > 0)
    for (int s = 2; s <= kTailMaxSplit; s *= 2)
      if (x.r * s <= cap && nk % s == 0 && nk / s >= kTailMinK) x.s = s;
  return x;
}

// The job of workgroup bid, or false when it has none.
__device__ __forceinline__ bool tile_job(int bid, int live, int cu_xcd, int nk, bool split_ok, TileJob& j) {
  const int xcd = bid & 7, local = bid >> 3;
  const XcdShare x = xcd_share(xcd, live, cu_xcd, nk, split_ok);
  if (local < x.full || x.s == 1) {
    if (local >= x.full + x.r) return false;
    j.lid = x.base + local;
    j.z = 0;
    j.s = 1;
    j.slot = -1;
    return true;
  }
  const int t = local - x.full;   // tail unit
  if (t >= x.r * x.s) return false;
  j.lid = x.base + x.full + t / x.s;
  j.z = t % x.s;
  j.s = x.s;
  j.slot = xcd * kTailSlotsPerXcd + t;
  return true;
}

// Partial-tile slot layout: float4 e of thread tid at [e][tid] (coalesced for both sides).
constexpr int kTailTileFloats = kTileM * kTileN;

__device__ __forceinline__ void tail_store_partial(float* part, int slot, const f32x16 (&acc)[kTileTM][kTileTN]) {
  float4* dst = reinterpret_cast<float4*>(part + static_cast<size_t>(slot) * kTailTileFloats);
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < kTileTM; ++i)
#pragma unroll
    for (int j = 0; j < kTileTN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        dst[((i * kTileTN + j) * 4 + q) * kTileThreads + tid] =
            make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
}

// acc = the sum, in slice order, of the s partial tiles in slots slot0 .. slot0 + s - 1.
__device__ __forceinline__ void tail_sum_partials(const float* part, int slot0, int s,
                                                  f32x16 (&acc)[kTileTM][kTileTN]) {
  const float4* src = reinterpret_cast<const float4*>(part) + static_cast<size_t>(slot0) * (kTailTileFloats / 4);
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < kTileTM; ++i)
#pragma unroll
    for (int j = 0; j < kTileTN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const size_t e = static_cast<size_t>((i * kTileTN + j) * 4 + q) * kTileThreads + tid;
        float4 v = src[e];
        for (int z = 1; z < s; ++z) {
          const float4 u = src[static_cast<size_t>(z) * (kTailTileFloats / 4) + e];
          v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
        }
        acc[i][j][4 * q] = v.x;
        acc[i][j][4 * q + 1] = v.y;
        acc[i][j][4 * q + 2] = v.z;
        acc[i][j][4 * q + 3] = v.w;
      }
}

}  // namespace maskmoe
