// The 256 x 256 x 64 bf16 MFMA tile pipeline shared by the expert GEMMs (forward, dgrad and
// wgrad): acc += A_tile * B_tile^T for 256 rows of A and 256 rows of B, both K-contiguous.
//
// 512 threads in 8 waves; wave w belongs to group g = w / 4 (A rows 128 g .. 128 g + 127) and
// owns 4 x 2 fragments of v_mfma_f32_32x32x16_bf16 (128 A rows x 64 B rows). The two waves that
// share a SIMD (w and w + 4) alternate roles in phases of one 32-wide k step, separated by one
// workgroup barrier: while one multiplies on operands it already holds in registers, the other
// issues its share of the global loads of a later k-tile and reads its next operands from LDS.
// The matrix unit therefore never waits for a load or an LDS read, and a load has at least two
// phases to arrive. Global loads go straight to LDS (global_load_lds_dwordx4, 1 KB per
// instruction: 8 rows x one 128-byte line), spread over the phases so that the texture unit is
// never flooded. LDS (160 KB): each group's 128-row A half double-buffered (16 KB each), the
// 256-row B tile triple-buffered (32 KB each), rows of 128 bytes with a 16-byte XOR swizzle
// (bank-conflict free for the fragment reads). Group 0 issues its A half of tile m + 1 in its
// first phase of tile m and its B half of tile m + 2 in its second; group 1 the same one phase
// later. Each wave waits for its own loads (vmcnt) before the barrier that precedes their first
// reader; a barrier never waits on the other group's loads.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace maskmoe {

constexpr int kTileM = 256, kTileN = 256, kTileK = 64, kTileThreads = 512;
constexpr int kTileTM = 4, kTileTN = 2;   // 32x32 fragments per wave

struct TileLds {
  u32x4 a[2][2][128 * 8];   // [group][buffer][row * 8 + chunk]
  u32x4 b[3][256 * 8];      // [buffer][row * 8 + chunk]
};

// Tile row (0..255) of this lane's i-th 16-byte piece of each operand per k-tile (i < 4), and
// the piece's logical chunk (its physical LDS chunk is lane & 7).
__device__ __forceinline__ int tile_dma_row(int i) {
  const int wave = threadIdx.x >> 6;
  return (wave >> 2) * 128 + 8 * (4 * (wave & 3) + i) + ((threadIdx.x & 63) >> 3);
}
__device__ __forceinline__ int tile_dma_chunk(int i) { return (threadIdx.x & 7) ^ lds_swizzle(tile_dma_row(i)); }

// Operands of one tile: byte bases at the first k-tile (wave-uniform) and this lane's byte
// offsets of its four rows (tile_dma_row(i), chunk included) of each; A k-tiles are 128 bytes
// apart, B k-tiles b_step bytes apart (128 row-major, the block size in the packed layout).
struct TileOps {
  const char* a;
  const char* b;
  uint32_t aoff[4];
  uint32_t boff[4];
  uint32_t b_step;
};

// A K-major operand (the contraction index strided in storage): element (k, m) of the tile's
// k-range at base + k * ld + 2 m bytes. k-rows at or beyond krows read as zeros; columns at or
// beyond mcols (a multiple of 8) are clamped to the last valid 8-column piece, whose products
// land in columns that are never stored. Loaded with buffer loads whose range is the krows
// valid rows (out-of-range lanes return zeros), ld >= 512 and krows * ld < 2^32.
struct TileKm {
  const char* base;
  int ld;
  int krows;
  int mcols;
};

// K-major operands sit in LDS as [128-row half][64 k][128 m] with 256-byte k-rows of 16
// 16-byte units; unit u of k-row kr is stored at unit u ^ 4 (kr & 3). A transposing read
// (ds_read_b64_tr_b16) has each 32 lanes touch 4 consecutive k-rows x 4 adjacent units; the
// swizzle puts those 16 units in distinct banks (with u ^ 2 (kr & 3) they pair up: 2-way
// conflicts on every read, measured).
__device__ __forceinline__ int km_unit(int u, int kr) { return u ^ (4 * (kr & 3)); }

typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
__device__ __forceinline__ uint32_t lds_offset(const u32x4* p) {
  return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<size_t>((lds_u32x4*)p)));
}
// 16 bytes per lane from gbase + voff straight into LDS at m0v + 16 * lane. The M0 write needs
// one wait state before the load.
__device__ __forceinline__ void dma16(uint32_t m0v, const void* gbase, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(m0v), "v"(voff), "s"(gbase)
               : "memory", "m0");
}
// The same through a buffer resource (K-major operands): 16 bytes at offset voff of the buffer
// described by rsrc, zeros where voff is past its size. (Full 64-bit per-lane addresses halve the
// texture unit's load rate.)
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void dma16b(uint32_t m0v, i32x4 rsrc, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(m0v), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
// A raw buffer resource over [p, p + bytes): base, stride 0, size, and the gfx9 data format word.
__device__ __forceinline__ i32x4 buffer_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  i32x4 r;
  r.x = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(a)));
  r.y = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(a >> 32) & 0xffffu));
  r.z = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes));
  r.w = 0x00020000;
  return r;
}
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
// One MFMA operand (8 consecutive k of one row) from a K-major half buffer: two transposing
// reads of 4 k-rows each. ds_read_b64_tr_b16 hands lane i of each 16-lane group element i % 4 of
// the 8 bytes read by lane 4 c + i / 4 of the group as its element c; lane j therefore reads 4
// adjacent columns (rbase + 16 (G & 1) + 4 (j & 3)) of k-row kk*16 + 8 (G >> 1) + j / 4, and
// lane i ends up with column rbase + 16 (G & 1) + i of 4 consecutive k-rows: row rbase + (lane
// & 31) of the operand, k-values 8 (lane >> 5) .. + 7 of k step kk, as the MFMA expects.
__device__ __forceinline__ u32x4 read_km_operand(const u32x4* half, int rbase, int kk) {
  const int lane = threadIdx.x & 63, G = lane >> 4, j = lane & 15;
  const int m = rbase + 16 * (G & 1) + 4 * (j & 3);
  const int kr = kk * 16 + 8 * (G >> 1) + (j >> 2);
  const char* p = reinterpret_cast<const char*>(half) + kr * 256 + km_unit(m >> 3, kr) * 16 + (m & 7) * 2;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * 256));
  const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
  return u32x4{a.x, a.y, b.x, b.y};
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }
__device__ __forceinline__ void wait_lgkmcnt0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// A workgroup barrier without the memory fence of __syncthreads (which would also wait for
// every load still in flight); LDS ordering is made explicit with the waits above.
__device__ __forceinline__ void tile_barrier() { asm volatile("s_barrier" ::: "memory"); }

// acc += A B^T over nk k-tiles (nk >= 1). EXTRA: one more k-tile first, from the operands in
// *x (its b_step is unused); the low-rank adapters use it: [U | X] [s B | W]^T turns
// W x + s B (A x) into one product. AKM / BKM: operand A / B is K-major (*akm / *bkm; the
// matching TileOps fields are unused). bfrag[j]: tile row of B fragment j for this lane (a
// multiple of 32 plus lane & 31); A fragment i is tile row 128 g + 32 i + (lane & 31).
template <bool EXTRA = false, bool AKM = false, bool BKM = false>
__device__ __forceinline__ void gemm_tile_mainloop(const TileOps& o, int nk, const int (&bfrag)[kTileTN],
                                                   f32x16 (&acc)[kTileTM][kTileTN], TileLds& L,
                                                   const TileOps* x = nullptr, const TileKm* akm = nullptr,
                                                   const TileKm* bkm = nullptr) {
  static_assert(!(EXTRA && (AKM || BKM)), "the extra k-tile is K-contiguous");
  constexpr int X = EXTRA ? 1 : 0;
  if (nk <= 0) return;
  const int ntot = nk + X;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int g = wave >> 2, q = wave & 3;
  const uint32_t la0 = lds_offset(&L.a[g][0][0]) + q * 4 * 1024;
  const uint32_t lb0 = lds_offset(&L.b[0][0]) + (g * 16 + q * 4) * 1024;
  // K-major pieces of this lane: k-row 4 (4 q + i) + lane / 16 of the group's half, the
  // 8 columns of its physical slot lane & 15; byte offsets at k-tile 0
  uint32_t akoff[4], bkoff[4];
  i32x4 arsrc{}, brsrc{};
  if (AKM) arsrc = buffer_rsrc(akm->base, static_cast<uint32_t>(akm->krows) * static_cast<uint32_t>(akm->ld));
  if (BKM) brsrc = buffer_rsrc(bkm->base, static_cast<uint32_t>(bkm->krows) * static_cast<uint32_t>(bkm->ld));
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int kr = 4 * (4 * q + i) + (lane >> 4);
    const int col = g * 128 + 8 * km_unit(lane & 15, kr);
    if (AKM) akoff[i] = static_cast<uint32_t>(kr * akm->ld + min(col, akm->mcols - 8) * 2);
    if (BKM) bkoff[i] = static_cast<uint32_t>(kr * bkm->ld + min(col, bkm->mcols - 8) * 2);
  }
  auto dma_km = [&](i32x4 rsrc, const uint32_t (&off)[4], int ld, uint32_t lbase, int tt) {
    const uint32_t step = static_cast<uint32_t>(tt) * 64u * static_cast<uint32_t>(ld);
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16b(lbase + static_cast<uint32_t>(i * 1024), rsrc, off[i] + step);
  };
  // Loads of pipeline tile t (main k-tile t - X), clamped to the last one: past the end they
  // refill a buffer that nothing reads again, which keeps every wait count the same.
  auto dma_a = [&](int t) {
    const int tt = min(t, ntot - 1) - X;
    if (AKM) {
      dma_km(arsrc, akoff, akm->ld, la0 + static_cast<uint32_t>((t & 1) * 16384), tt);
    } else {
      const char* ga = o.a + static_cast<size_t>(tt) * 128;
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16(la0 + static_cast<uint32_t>((t & 1) * 16384 + i * 1024), ga, o.aoff[i]);
    }
  };
  auto dma_b = [&](int t) {
    const int tt = min(t, ntot - 1) - X;
    if (BKM) {
      dma_km(brsrc, bkoff, bkm->ld, lb0 + static_cast<uint32_t>((t % 3) * 32768), tt);
    } else {
      const char* gb = o.b + static_cast<size_t>(tt) * o.b_step;
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16(lb0 + static_cast<uint32_t>((t % 3) * 32768 + i * 1024), gb, o.boff[i]);
    }
  };
  const int sw = lds_swizzle(lane & 31);
  u32x4 af[2][kTileTM], bf[2][kTileTN];
  auto read_half = [&](int t, int h) {   // operands of k steps 2h, 2h + 1 of pipeline tile t
    const u32x4* pa = &L.a[g][t & 1][0];
    const u32x4* pb = &L.b[t % 3][0];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int ch = (4 * h + 2 * kk + (lane >> 5)) ^ sw;
#pragma unroll
      for (int i = 0; i < kTileTM; ++i)
        af[kk][i] = AKM ? read_km_operand(pa, i * 32, 2 * h + kk) : pa[(i * 32 + (lane & 31)) * 8 + ch];
#pragma unroll
      for (int j = 0; j < kTileTN; ++j) {
        const int r0 = bfrag[j] & ~31;   // the fragment's first tile row
        bf[kk][j] = BKM ? read_km_operand(pb + (r0 >> 7) * 1024, r0 & 127, 2 * h + kk) : pb[bfrag[j] * 8 + ch];
      }
    }
  };
  auto compute = [&]() {
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int i = 0; i < kTileTM; ++i)
#pragma unroll
        for (int j = 0; j < kTileTN; ++j) acc[i][j] = mfma_32x32x16(af[kk][i], bf[kk][j], acc[i][j]);
    __builtin_amdgcn_s_setprio(0);
  };

  // prologue: this wave's A piece of tile 0 and B pieces of tiles 0 and 1
  if (EXTRA) {
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16(la0 + static_cast<uint32_t>(i * 1024), x->a, x->aoff[i]);
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16(lb0 + static_cast<uint32_t>(i * 1024), x->b, x->boff[i]);
  } else {
    dma_a(0);
    dma_b(0);
  }
  dma_b(1);
  wait_vmcnt<0>();
  tile_barrier();
  // group 1 runs one phase behind group 0: one extra barrier first (group 0 adds it at the end)
  if (g == 1) tile_barrier();
  for (int m = 0; m < ntot; ++m) {
    __builtin_amdgcn_sched_barrier(0);
    dma_a(m + 1);
    read_half(m, 0);
    __builtin_amdgcn_sched_barrier(0);
    wait_lgkmcnt0();
    tile_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compute();
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<4>();
    tile_barrier();
    __builtin_amdgcn_sched_barrier(0);
    dma_b(m + 2);
    read_half(m, 1);
    __builtin_amdgcn_sched_barrier(0);
    wait_lgkmcnt0();
    tile_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compute();
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<4>();
    tile_barrier();
  }
  if (g == 0) tile_barrier();
  wait_vmcnt<0>();
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
// in slice order (tail_fixup_part) and applies the GEMM's epilogue, so results stay
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

// Fix-up of split tail tiles, spread over kTailFixParts workgroups per tile: part p adds, in
// slice order, the partial-tile units of the fragment rows (i, q) = (iq / 4, iq % 4) for
// iq = kTailPairsPerPart p .., both column fragments j (unit e = (i * kTileTN + j) * 4 + q of
// thread tid holds acc[i][j][4 q .. 4 q + 3]: tile rows wm*128 + i*32 + 8q + 4 (lane >> 5) + (0..3)
// of fragment column j), and hands the sums to st(i, q, sum_j0, sum_j1). All slices of a unit
// are loaded before any is added.
constexpr int kTailFixParts = 8, kTailPairsPerPart = kTileTM * 4 / kTailFixParts;
static_assert(kTileTN == 2, "the fix-up hands over two column fragments");

template <class Store>
__device__ __forceinline__ void tail_fixup_part(const float* part, int slot0, int s, int p, Store st) {
  const float4* src = reinterpret_cast<const float4*>(part) + static_cast<size_t>(slot0) * (kTailTileFloats / 4);
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < kTailPairsPerPart; ++u) {
    const int iq = p * kTailPairsPerPart + u, i = iq >> 2, q = iq & 3;
    float4 v[kTileTN][kTailMaxSplit];
#pragma unroll
    for (int j = 0; j < kTileTN; ++j)
#pragma unroll
      for (int z = 0; z < kTailMaxSplit; ++z)
        if (z < s)
          v[j][z] = src[static_cast<size_t>(z) * (kTailTileFloats / 4) +
                        static_cast<size_t>((i * kTileTN + j) * 4 + q) * kTileThreads + tid];
    float4 a[kTileTN];
#pragma unroll
    for (int j = 0; j < kTileTN; ++j) {
      a[j] = v[j][0];
#pragma unroll
      for (int z = 1; z < kTailMaxSplit; ++z)
        if (z < s) {
          a[j].x += v[j][z].x; a[j].y += v[j][z].y; a[j].z += v[j][z].z; a[j].w += v[j][z].w;
        }
    }
    st(i, q, a[0], a[1]);
  }
}

}  // namespace maskmoe
