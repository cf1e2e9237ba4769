// Expert FFNs and the gate-weighted combine of the masked MoE layer.
//
// Eq. 1 (Section 3.1): y = sum_{i in A} g_i F_i(x), plus the shared experts' outputs
// with weight 1. Each expert is the SwiGLU FFN F(x) = W_down (SiLU(W_gate x) * W_up x).
// After the permutation every expert group is a dense row block, so the FFN is a grouped
// GEMM pair:
//   H_g = SiLU(X_g W_gate,g^T) * (X_g W_up,g^T)   (rows gathered from x through row_tok)
//   O_g = H_g W_down,g^T
// followed by y_t = sum_k g_{t,k} O[inv(t,k)] + sum_s O[shared row of t].
//
// bf16, many tokens: 256x256x64 block tiles on v_mfma_f32_32x32x16_bf16, 8 waves (2 x 4),
// 128x64 per wave, A and B double-buffered in LDS (128 KB) with a 16-byte XOR swizzle so
// that the MFMA operand reads are bank-conflict free; global loads run two k-tiles ahead.
// The gate/up GEMM holds matching 128-column slices of W_gate and W_up in one tile and
// applies SwiGLU in registers (H rounded once to bf16). Tiles are enumerated expert-tile
// fastest so the workgroups that share a weight slice run together, and the linear block
// id is remapped so each XCD (L2) receives a contiguous range of tiles.
//
// bf16, few tokens (decode): the work is reading each selected expert's weights once; the
// kernels stream weight rows through LDS in cache-line-sized row segments (see the decode
// section below); both projections split their reduction dimension when few experts are
// active so that every CU keeps streaming. MFMA 16x16x32 with the token rows padded to 16.
//
// f32: plain fp32 loops (no MFMA), one thread per output element.

#include <algorithm>
#include <cmath>
#include <cstdlib>

#include <type_traits>

#include "common.hpp"
#include "gemm_tile.hpp"
#include "kernels.hpp"

namespace maskmoe {
namespace {

// ------------------------------------------------------------------ bf16 grouped GEMM

constexpr int BM = kGemmBM, BN = kTileN, BK = kTileK, GEMM_THREADS = kTileThreads;
static_assert(BM == kTileM, "tile mapping assumes 256-row tiles");

struct GemmArgs {
  const uint16_t* a;        // EPI 0: x [T, d] (rows via row_tok); EPI 1: H [rows, F]
  const int32_t* row_tok;
  const uint16_t* w;        // routed weights: EPI 0 [E, 2F, d], EPI 1 [E, d, F]
  const uint16_t* ws;       // shared weights, same layout with n_shared experts
  const int32_t* offsets;   // [G+1]
  const int32_t* tile_off;  // [G+1]
  void* out;                // EPI 0: H bf16 [rows, F]; EPI 1: O bf16 [rows, d]
  uint16_t* ab;             // EPI 0, training: gate / up pre-activations bf16 [rows, 2F], or null
  const uint16_t* lora_u;   // LORA: rank-r projections of this GEMM's A rows, bf16 [rows, 64]
  const uint16_t* lora_b;   // LORA: (alpha / r) B rows matching the B operand, bf16 [G, N rows, 64]
  float* part;              // partial tiles of split tail tiles, kTailSlots x [64 x 512 x 4] fp32
  int G, E, F, d;
  int mt_max;               // bound on row tiles (the grid is sized for mt_max * n_tiles tiles)
  int n_tiles;              // column tiles
  int cu_xcd;               // workgroups an XCD runs at once (one per CU)
};

// Only the down GEMM splits its tail tiles (tile_job in gemm_tile.hpp): its long reductions
// amortise a slice's fixed costs, and the gate/up GEMM's epilogue needs whole sums. Measured,
// slices shorter than 16 k-tiles and splits of the gate/up tiles (with SwiGLU applied in the
// fix-up) gained nothing over the partial round they save.
__host__ __device__ constexpr bool tail_can_split(int epi, int nk) { return epi == 1 && tail_splittable(nk); }

__device__ __forceinline__ int find_group(const int32_t* tile_off, int G, int mt) {
  int lo = 0, hi = G;  // tile_off[lo] <= mt < tile_off[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tile_off[mid] <= mt) lo = mid; else hi = mid;
  }
  return lo;
}

// Epilogue of a finished tile: rows [row0, row_end) of one group, columns from n0. EPI 0:
// SwiGLU of the gate / up column pairs into H (bf16; the pre-activations into ab when given);
// EPI 1: O, each expert output rounded to bf16 (the layer's dtype; the combine adds them in
// fp32). acc[i][j][4*jj+ii] is row wm*128 + i*32 + 8*jj + 4*(lane>>5) + ii, column (lane & 31)
// of fragment j. The bf16 tile is staged in LDS (free after the k-loop; rows padded by 16
// bytes, conflict-free) and stored eight columns per 16-byte access: a lane holds one column
// of each row it owns, and 2-byte stores kept the texture-address path busy for several
// percent of a tile.
template <int COLS>   // columns of the staged tile: LDS row pitch COLS + 8 elements
__device__ __forceinline__ void store_staged(const uint16_t* stg, uint16_t* out, size_t ld, int row0, int row_end,
                                             int col0, int ncol) {
  constexpr int G = COLS / 8;   // 8-column groups per row
  for (int u = threadIdx.x; u < 256 * G; u += kTileThreads) {
    const int lr = u / G, cg = (u % G) * 8;
    const int row = row0 + lr, col = col0 + cg;
    if (row >= row_end || col >= ncol) continue;
    const uint16_t* src = stg + lr * (COLS + 8) + cg;
    uint16_t* dst = out + static_cast<size_t>(row) * ld + col;
    if (col + 8 <= ncol) {   // ld and col are multiples of 8: 16-byte aligned
      *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
    } else {
      for (int e = 0; e < ncol - col; ++e) dst[e] = src[e];
    }
  }
}

template <int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& p, const f32x16 (&acc)[kTileTM][kTileTN], int row0,
                                              int row_end, int n0, TileLds& L) {
  constexpr int WN = 4, TM = kTileTM, TN = kTileTN;
  constexpr int COLS = EPI == 0 ? BN / 2 : BN, PITCH = COLS + 8;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  uint16_t* stg = reinterpret_cast<uint16_t*>(&L);
  static_assert((EPI == 0 ? 2 : 1) * 256 * PITCH * 2 <= sizeof(TileLds), "the staged tiles fit in LDS");
  wait_lgkmcnt0();
  tile_barrier();   // every wave is past the k-loop's LDS reads and DMA writes
  // this lane's rows of the tile: row_of(i, r)
  auto row_of = [&](int i, int r) { return wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); };
  if (EPI == 0) {   // H, and the gate pre-activations when kept (the up ones follow)
    const int c = wn * 32 + (lane & 31);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) stg[row_of(i, r) * PITCH + c] = f32_to_bf16(silu(acc[i][0][r]) * acc[i][1][r]);
    if (p.ab)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) stg[256 * PITCH + row_of(i, r) * PITCH + c] = f32_to_bf16(acc[i][0][r]);
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r)
#pragma unroll
        for (int j = 0; j < TN; ++j) stg[row_of(i, r) * PITCH + wn * 64 + j * 32 + (lane & 31)] = f32_to_bf16(acc[i][j][r]);
  }
  wait_lgkmcnt0();
  tile_barrier();
  uint16_t* out = static_cast<uint16_t*>(p.out);
  if (EPI == 0) {
    store_staged<COLS>(stg, out, p.F, row0, row_end, n0, p.F);
    if (p.ab) {
      store_staged<COLS>(stg + 256 * PITCH, p.ab, 2 * static_cast<size_t>(p.F), row0, row_end, n0, p.F);
      wait_lgkmcnt0();
      tile_barrier();   // the staged tiles are read: stage the up pre-activations
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) stg[row_of(i, r) * PITCH + wn * 32 + (lane & 31)] = f32_to_bf16(acc[i][1][r]);
      wait_lgkmcnt0();
      tile_barrier();
      store_staged<COLS>(stg, p.ab + p.F, 2 * static_cast<size_t>(p.F), row0, row_end, n0, p.F);
    }
  } else {
    store_staged<COLS>(stg, out, p.d, row0, row_end, n0, p.d);
  }
}

// PACKED: the expert matrices are in the packed layout (kPackRows x kPackCols blocks).
template <int EPI, bool LORA = false, bool PACKED = false>
__global__ __launch_bounds__(GEMM_THREADS) void grouped_gemm_bf16(const GemmArgs p) {
  constexpr int WN = 4;                 // waves: 2 along rows x 4 along columns
  constexpr int TM = kTileTM, TN = kTileTN;
  __shared__ TileLds lds;

  // The grid covers the most tiles any routing can need plus the tail slices; tile_job gives
  // each XCD's workgroups that XCD's share of the live tiles (their count read on the device),
  // so every XCD gets an equal share however many tiles are live.
  const int mt_live = p.tile_off[p.G];
  const int live = mt_live * p.n_tiles;
  const int Kdim = EPI == 0 ? p.d : p.F;
  TileJob job;
  if (!tile_job(static_cast<int>(blockIdx.x), live, p.cu_xcd, Kdim / BK, tail_can_split(EPI, Kdim / BK), job)) return;
  int mt, nt;
  grouped_tile_coords(job.lid, mt_live, p.n_tiles, mt, nt);
  const int z = job.z;
  const int g = find_group(p.tile_off, p.G, mt);
  const int row0 = p.offsets[g] + (mt - p.tile_off[g]) * BM;
  const int row_end = p.offsets[g + 1];
  const int n0 = nt * (EPI == 0 ? BN / 2 : BN);
  const int nks = Kdim / BK / job.s;   // k-tiles of this slice
  const int k0 = z * nks * BK;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wn = wave % WN;

  // This lane's four rows of the A and B tiles (tile_dma_row in gemm_tile.hpp). B tile rows
  // 0..127 of the gate/up GEMM are W_gate rows n0.., rows 128..255 the matching W_up rows.
  const uint16_t* wg = g < p.E ? p.w + static_cast<size_t>(g) * (EPI == 0 ? 2 * p.F : p.d) * Kdim
                               : p.ws + static_cast<size_t>(g - p.E) * (EPI == 0 ? 2 * p.F : p.d) * Kdim;
  TileOps ops;
  ops.a = reinterpret_cast<const char*>(p.a + k0);
  ops.b = reinterpret_cast<const char*>(wg + (PACKED ? static_cast<size_t>(k0 / kPackCols) * kPackBlock : k0));
  ops.b_step = PACKED ? kPackBlock * 2 : BK * 2;
  int brows[4];   // the pieces' B rows within the matrix
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = tile_dma_row(i);
    const int chunk = tile_dma_chunk(i) * 8;
    const int row = min(row0 + r, row_end - 1);
    ops.aoff[i] = static_cast<uint32_t>((EPI == 0 ? p.row_tok[row] : row) * Kdim + chunk) * 2u;
    int brow, grp, rig;   // row in the matrix; its packed group and row within the group
    if (EPI == 0) {
      const int n = min(n0 + (r & 127), p.F - 1);
      brow = r < 128 ? n : p.F + n;
      grp = n / 64;
      rig = n % 64 + (r < 128 ? 0 : 64);
    } else {
      brow = min(n0 + r, p.d - 1);
      grp = brow / kPackRows;
      rig = brow % kPackRows;
    }
    brows[i] = brow;
    ops.boff[i] = static_cast<uint32_t>(PACKED ? grp * kPackRows * Kdim + rig * kPackCols + chunk : brow * Kdim + chunk) * 2u;
  }

  // B fragment rows: EPI 0 -> gate wn*32 + ... and the matching up row 128 + wn*32 + ...;
  // EPI 1 -> wn*64 + j*32 + ...
  int bfrag[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) bfrag[j] = (EPI == 0 ? (j == 0 ? 0 : 128) + wn * 32 : wn * 64 + j * 32) + (lane & 31);

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  if (LORA && z == 0) {   // the adapters' term as one more k-tile: A' = [U | rows], B' = [s B | W]
    TileOps ex;
    ex.a = reinterpret_cast<const char*>(p.lora_u);
    ex.b = reinterpret_cast<const char*>(p.lora_b + static_cast<size_t>(g) * (EPI == 0 ? 2 * p.F : p.d) * 64);
    ex.b_step = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int chunk = tile_dma_chunk(i) * 8;
      ex.aoff[i] = static_cast<uint32_t>(min(row0 + tile_dma_row(i), row_end - 1) * 64 + chunk) * 2u;
      ex.boff[i] = static_cast<uint32_t>(brows[i] * 64 + chunk) * 2u;
    }
    gemm_tile_mainloop<true>(ops, nks, bfrag, acc, lds, &ex);
  } else {
    gemm_tile_mainloop<false>(ops, nks, bfrag, acc, lds);
  }
  if (job.s > 1) {   // a slice of a split tail tile: its partial tile goes to the slot
    tail_store_partial(p.part, job.slot, acc);
    return;
  }
  gemm_epilogue<EPI>(p, acc, row0, row_end, n0, lds);
}

// Adds the slices of each split tail tile of the down GEMM (grouped_gemm_bf16<1>) in slice order
// and stores its rows of O; kTailFixParts workgroups per possible tail tile, grid
// 8 x kTailSlotsPerXcd x kTailFixParts.
__global__ __launch_bounds__(GEMM_THREADS) void grouped_tail_fixup(const GemmArgs p) {
  const int mt_live = p.tile_off[p.G];
  const int live = mt_live * p.n_tiles;
  const int nk = p.F / BK;
  const int b = blockIdx.x, xcd = b & 7, t = (b >> 3) % kTailSlotsPerXcd, part = b / (8 * kTailSlotsPerXcd);
  const XcdShare x = xcd_share(xcd, live, p.cu_xcd, nk, tail_can_split(1, nk));
  if (x.s == 1 || t >= x.r) return;
  int mt, nt;
  grouped_tile_coords(x.base + x.full + t, mt_live, p.n_tiles, mt, nt);
  const int g = find_group(p.tile_off, p.G, mt);
  const int row0 = p.offsets[g] + (mt - p.tile_off[g]) * BM, row_end = p.offsets[g + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wm = wave / 4, wn = wave % 4;
  const int c0 = nt * BN + wn * 64 + (lane & 31);
  uint16_t* out = static_cast<uint16_t*>(p.out);
  tail_fixup_part(p.part, xcd * kTailSlotsPerXcd + t * x.s, x.s, part, [&](int i, int q, float4 a0, float4 a1) {
    const float v0[4] = {a0.x, a0.y, a0.z, a0.w}, v1[4] = {a1.x, a1.y, a1.z, a1.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = row0 + wm * 128 + i * 32 + 8 * q + 4 * (lane >> 5) + u;
      if (row >= row_end) continue;
      const size_t o = static_cast<size_t>(row) * p.d + c0;
      if (c0 < p.d) out[o] = f32_to_bf16(v0[u]);
      if (c0 + 32 < p.d) out[o + 32] = f32_to_bf16(v1[u]);
    }
  });
}

// y_t = sum_k gate[t,k] * O[inv[t*K+k]] + sum_s O[T*K + s*T + t]; fp32 sum in k order, one
// rounding at the end. O holds `split` partial slices [split, rows, d] that are added first,
// in slice order. One workgroup per token.
// Each expert output of a bf16 layer is rounded to bf16 (the layer's dtype) before the gated
// sum: the grouped path stores O in bf16; the few-token path rounds its fp32 slice sums.
__device__ __forceinline__ float4 round_bf16x4(float4 v) {
  return make_float4(bf16_to_f32(f32_to_bf16(v.x)), bf16_to_f32(f32_to_bf16(v.y)), bf16_to_f32(f32_to_bf16(v.z)),
                     bf16_to_f32(f32_to_bf16(v.w)));
}

// Four consecutive expert-output values at element offset off of O: fp32, or (OB) bf16.
template <bool OB>
__device__ __forceinline__ float4 load_o4(const void* O, size_t off) {
  if (OB) {
    const uint2 u = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(O) + off);
    return make_float4(bf16_to_f32(static_cast<uint16_t>(u.x & 0xffffu)), bf16_to_f32(static_cast<uint16_t>(u.x >> 16)),
                       bf16_to_f32(static_cast<uint16_t>(u.y & 0xffffu)), bf16_to_f32(static_cast<uint16_t>(u.y >> 16)));
  }
  return *reinterpret_cast<const float4*>(static_cast<const float*>(O) + off);
}

// Sum of the `split` slices at offset off, added in slice order; groups of four loads are
// issued together so that a long split costs a few memory round trips, not one per slice.
__device__ __forceinline__ float4 sum_slices(const float* O, int split, size_t slice, size_t off) {
  if (split <= kDecodeMaxSplit) {   // every slice's load in flight at once
    float4 u[kDecodeMaxSplit];
#pragma unroll
    for (int z = 0; z < kDecodeMaxSplit; ++z)
      if (z < split) u[z] = *reinterpret_cast<const float4*>(O + z * slice + off);
    float4 v = u[0];
#pragma unroll
    for (int z = 1; z < kDecodeMaxSplit; ++z)
      if (z < split) {
        v.x += u[z].x; v.y += u[z].y; v.z += u[z].z; v.w += u[z].w;
      }
    return v;
  }
  float4 v = *reinterpret_cast<const float4*>(O + off);
  int z = 1;
  for (; z + 3 < split; z += 4) {
    float4 u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) u[i] = *reinterpret_cast<const float4*>(O + (z + i) * slice + off);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v.x += u[i].x; v.y += u[i].y; v.z += u[i].z; v.w += u[i].w;
    }
  }
  for (; z < split; ++z) {
    const float4 u = *reinterpret_cast<const float4*>(O + z * slice + off);
    v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
  }
  return v;
}

// y[t, c] = sum_k gate[t, k] O[inv[t K + k], c] + sum over shared experts of their rows, with
// O's slices added first; when eo is given, eo[t, k, c] also receives the slice sum of row
// inv[t K + k] (the selected expert's output before gating). One workgroup of 256 threads
// per (token, block of kCombineCols columns), token-major in a 1-D grid.
constexpr int kCombineCols = 1024;
constexpr int kCombineColsOB = 2048;   // the bf16-O instances with K known: 8 columns per thread
constexpr int kMaxSharedCombine = 8;   // the API's limit on shared experts

// KC: K known at compile time with one slice (the grouped path): every row's index, gate and
// O values are loaded before any is added (same additions, same order). OB: O holds bf16
// values (one slice); the sums are still formed in fp32. KC and OB together: a thread takes
// eight columns (16-byte loads of every row, grid by kCombineColsOB).
template <bool BF16, int KC = 0, bool OB = false>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ Ov,
                                                       const int32_t* __restrict__ inv,
                                                       const float* __restrict__ gate, int T, int K,
                                                       int n_shared, int d, void* y, int split,
                                                       float* __restrict__ eo) {
  const float* O = static_cast<const float*>(Ov);
  if (BF16 && KC > 0 && OB) {   // eight columns per thread: 16-byte loads of every bf16 row; d % 8 == 0
    constexpr int KA = KC > 0 ? KC : 1;
    const int nb8 = (d + kCombineColsOB - 1) / kCombineColsOB;
    const int t = blockIdx.x / nb8, c = (blockIdx.x % nb8) * kCombineColsOB + threadIdx.x * 8;
    if (c >= d) return;
    int row[KA];
    float gk[KA];
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      row[k] = inv[t * KC + k];
      gk[k] = gate[t * KC + k];
    }
    const uint16_t* O16 = static_cast<const uint16_t*>(Ov);
    u32x4 v[KA], vs[kMaxSharedCombine];
#pragma unroll
    for (int k = 0; k < KC; ++k) v[k] = *reinterpret_cast<const u32x4*>(O16 + static_cast<size_t>(row[k]) * d + c);
#pragma unroll
    for (int sh = 0; sh < kMaxSharedCombine; ++sh)
      if (sh < n_shared)
        vs[sh] = *reinterpret_cast<const u32x4*>(
            O16 + (static_cast<size_t>(T) * KC + static_cast<size_t>(sh) * T + t) * d + c);
    // element e of a 16-byte piece: bf16 number e (little-endian halves of the four words)
    auto el = [](const u32x4& u, int e) {
      const uint32_t w = u[e >> 1];
      return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
    };
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = 0.0f;
#pragma unroll
    for (int k = 0; k < KC; ++k) {
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += gk[k] * el(v[k], e);
      if (eo) {
        float* dst = eo + (static_cast<size_t>(t) * KC + k) * d + c;
        *reinterpret_cast<float4*>(dst) = make_float4(el(v[k], 0), el(v[k], 1), el(v[k], 2), el(v[k], 3));
        *reinterpret_cast<float4*>(dst + 4) = make_float4(el(v[k], 4), el(v[k], 5), el(v[k], 6), el(v[k], 7));
      }
    }
#pragma unroll
    for (int sh = 0; sh < kMaxSharedCombine; ++sh)
      if (sh < n_shared)
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] += el(vs[sh], e);
    u32x4 packed;
#pragma unroll
    for (int q = 0; q < 4; ++q) packed[q] = f32x2_to_bf16x2(s[2 * q], s[2 * q + 1]);
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(y) + static_cast<size_t>(t) * d + c) = packed;
    return;
  }
  const int nb = (d + kCombineCols - 1) / kCombineCols;
  const int t = blockIdx.x / nb, cb = blockIdx.x % nb;
  if (BF16 && KC > 0) {  // d % 4 == 0, split == 1, K == KC, n_shared <= kMaxSharedCombine
    const int c = cb * kCombineCols + threadIdx.x * 4;
    if (c >= d) return;
    constexpr int KA = KC > 0 ? KC : 1;   // array extent of the generic instance (branch not taken)
    int row[KA];
    float gk[KA];
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      row[k] = inv[t * KC + k];
      gk[k] = gate[t * KC + k];
    }
    float4 v[KA], vs[kMaxSharedCombine];
#pragma unroll
    for (int k = 0; k < KC; ++k) v[k] = load_o4<OB>(Ov, static_cast<size_t>(row[k]) * d + c);
#pragma unroll
    for (int sh = 0; sh < kMaxSharedCombine; ++sh)
      if (sh < n_shared)
        vs[sh] = load_o4<OB>(Ov, (static_cast<size_t>(T) * KC + static_cast<size_t>(sh) * T + t) * d + c);
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      s.x += gk[k] * v[k].x; s.y += gk[k] * v[k].y; s.z += gk[k] * v[k].z; s.w += gk[k] * v[k].w;
      if (eo) *reinterpret_cast<float4*>(eo + (static_cast<size_t>(t) * KC + k) * d + c) = v[k];
    }
#pragma unroll
    for (int sh = 0; sh < kMaxSharedCombine; ++sh)
      if (sh < n_shared) {
        s.x += vs[sh].x; s.y += vs[sh].y; s.z += vs[sh].z; s.w += vs[sh].w;
      }
    uint2 packed;
    packed.x = f32x2_to_bf16x2(s.x, s.y);
    packed.y = f32x2_to_bf16x2(s.z, s.w);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(y) + static_cast<size_t>(t) * d + c) = packed;
  } else if (BF16) {  // d % 4 == 0
    const size_t slice = static_cast<size_t>(T) * (K + n_shared) * d;
    const int c = cb * kCombineCols + threadIdx.x * 4;
    if (c >= d) return;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int k = 0; k < K; ++k) {
      const float gk = gate[t * K + k];
      const size_t off = static_cast<size_t>(inv[t * K + k]) * d + c;
      const float4 v = OB ? load_o4<true>(Ov, off) : round_bf16x4(sum_slices(O, split, slice, off));
      s.x += gk * v.x; s.y += gk * v.y; s.z += gk * v.z; s.w += gk * v.w;
      if (eo) *reinterpret_cast<float4*>(eo + (static_cast<size_t>(t) * K + k) * d + c) = v;
    }
    for (int sh = 0; sh < n_shared; ++sh) {
      const size_t off = (static_cast<size_t>(T) * K + static_cast<size_t>(sh) * T + t) * d + c;
      const float4 v = OB ? load_o4<true>(Ov, off) : round_bf16x4(sum_slices(O, split, slice, off));
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
    uint2 packed;
    packed.x = f32x2_to_bf16x2(s.x, s.y);
    packed.y = f32x2_to_bf16x2(s.z, s.w);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(y) + static_cast<size_t>(t) * d + c) = packed;
  } else {
    for (int c = cb * kCombineCols + threadIdx.x; c < d && c < (cb + 1) * kCombineCols; c += 256) {
      float s = 0.0f;
      for (int k = 0; k < K; ++k) {
        const float v = O[static_cast<size_t>(inv[t * K + k]) * d + c];
        s += gate[t * K + k] * v;
        if (eo) eo[(static_cast<size_t>(t) * K + k) * d + c] = v;
      }
      for (int sh = 0; sh < n_shared; ++sh) s += O[(static_cast<size_t>(T) * K + static_cast<size_t>(sh) * T + t) * d + c];
      static_cast<float*>(y)[static_cast<size_t>(t) * d + c] = s;
    }
  }
}

static dim3 combine_grid(int T, int d, int cols = kCombineCols) { return dim3(T * ((d + cols - 1) / cols)); }

// ------------------------------------------------------------------ bf16 decode kernels
//
// With few tokens the FFN is a weight stream: each selected expert's matrices are read once
// and every row meets at most 16 token rows. A workgroup owns DEC_NT tiles of 16 weight rows
// (gate/up kernel: DEC_NT gate tiles and the DEC_NT matching up tiles) and walks the
// reduction dimension in chunks of DEC_CK values. Each chunk is loaded with 16-byte loads in
// which a wavefront covers whole 128-byte row segments (full cache lines), stored to LDS with
// a 16-byte row pad (conflict-free MFMA operand reads), and multiplied on MFMA 16x16x32 with
// the token rows padded to 16. The next two chunks' loads (weights and token operands) are in
// flight while the current one is multiplied. Both projections split their reduction dimension into slices when few experts
// are active, so that enough workgroups stream at once: the gate/up slices are added by a
// small SwiGLU pass, the down slices by the combine, always in slice order. (Letting the
// last workgroup of a column slab do the combine needs a device-scope release per
// workgroup, which on this multi-XCD part costs more than the separate small launch.)

constexpr int DEC_NT = 4;        // 16-row weight tiles per operand per workgroup
constexpr int DEC_CK = 64;       // reduction values per chunk (128 bytes per row)
constexpr int DEC_THREADS = 256;
// Down workgroups that build their H rows from the gate/up partial sums (decode_down_kernel
// SWIGLU): LDS bytes for the rows, four-column groups per thread (their loads issued together).
constexpr int kFusedSwigluLds = 8192;
constexpr int kFusedItems = 2;

struct DecodeArgs {
  const uint16_t* x;
  const int32_t* row_tok;
  const int32_t* offsets;
  const int32_t* active;
  const int32_t* n_active;
  const uint16_t* w_gate_up;
  const uint16_t* w_down;
  const uint16_t* ws_gate_up;
  const uint16_t* ws_down;
  uint16_t* H;        // [rows, F] bf16
  float* P;           // [split_gu, rows, 2F] fp32 partial gate/up sums (split_gu > 1)
  float* O;           // [split, rows, d] fp32
  const int32_t* slot_of;   // routed expert -> weight block (offloaded decode), or null
  int T, d, F, E, K, rows, split, split_gu, n_slots;
};

// Weight block of routed expert g: g itself, or its slot in the pool of an offloaded decode
// (clamped into the pool, which the cache step guarantees anyway).
__device__ __forceinline__ int weight_block(const DecodeArgs& p, int g) {
  return p.slot_of ? min(max(p.slot_of[g], 0), p.n_slots - 1) : g;
}

// Token-row operand of stream_rows: the 8 bf16 values of row (lane & 15) at k = base +
// c * DEC_CK + ks * 32 + (lane >> 4) * 8 for chunk c of the stream, `ap` pointing at base +
// (lane >> 4) * 8 of the row. IN_LDS: the rows sit in LDS (written before the stream's first
// barrier) and are read where they are used; otherwise they are global and are loaded two
// chunks ahead, with the weights.
template <bool IN_LDS>
struct RowOperand {
  const uint16_t* ap;
  __device__ __forceinline__ u32x4 operator()(int c, int ks) const {
    return *reinterpret_cast<const u32x4*>(ap + c * DEC_CK + ks * 32);
  }
};

// Streams R = 16 * NTILE weight rows over k in [k0, k0 + klen) and accumulates tile
// (wave + 4q) of A(16 x k) * W^T into acc[q]; `arow` gives the A operand (RowOperand, its
// chunks counted from k0). Row r's values k .. k + 63 of chunk k / 64 start at wrow(r) +
// (k / 64) * CSTRIDE: CSTRIDE = DEC_CK for row-major weights, kPackBlock for packed ones
// (where the R rows of a chunk are one contiguous block). `prologue` runs once the first two
// weight chunks are in flight, before the first barrier.
template <int NTILE, int CSTRIDE, bool A_LDS, class RowPtr, class Prologue>
__device__ __forceinline__ void stream_rows(const RowPtr& wrow, const RowOperand<A_LDS>& arow, int k0, int klen,
                                            unsigned char (*lds)[16 * NTILE * (DEC_CK * 2 + 16)],
                                            f32x4* acc, const Prologue& prologue) {
  constexpr int R = 16 * NTILE;
  constexpr int PITCH = DEC_CK * 2 + 16;
  constexpr int UPR = DEC_CK * 2 / 16;
  constexpr int PER = R * UPR / DEC_THREADS;
  constexpr int TPW = (NTILE + 3) / 4;
  static_assert(R * UPR % DEC_THREADS == 0, "chunk must split evenly over the threads");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint16_t* src[PER];
  int dst[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int u = tid + DEC_THREADS * i;
    const int r = u / UPR, piece = u % UPR;
    src[i] = wrow(r) + (CSTRIDE == DEC_CK ? k0 : (k0 / DEC_CK) * CSTRIDE) + piece * 8;
    dst[i] = r * PITCH + piece * 16;
  }
  const int nc = klen / DEC_CK;
  // Weight chunks c + 1 and c + 2 are in flight in registers while chunk c is multiplied from
  // LDS; the token rows' operands travel with them (a wait on a load issued after the weight
  // loads would also wait for those).
  constexpr int KS = DEC_CK / 32;
  u32x4 reg[2][PER], areg[2][KS];
  auto load_w = [&](int c, u32x4* r) {
#pragma unroll
    for (int i = 0; i < PER; ++i) r[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src[i] + c * CSTRIDE));
  };
  auto load_a = [&](int c, u32x4* r) {
    if (!A_LDS) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) r[ks] = arow(c, ks);
    }
  };
  auto store = [&](int buf, const u32x4* r) {
#pragma unroll
    for (int i = 0; i < PER; ++i) *reinterpret_cast<u32x4*>(&lds[buf][dst[i]]) = r[i];
  };
  // The loop is straight-line in its loads and stores (the tail steps are peeled), so the
  // compiler's wait counts stay exact: a wait for chunk c + 1 never waits for chunk c + 2.
  load_w(0, reg[0]);
  load_a(0, areg[0]);
  load_w(min(1, nc - 1), reg[1]);   // nc == 1 (d or F of 64) reloads chunk 0
  load_a(min(1, nc - 1), areg[1]);
  prologue();
  store(0, reg[0]);
  __syncthreads();
  // one chunk; BUF = c & 1 is a compile-time index so that the staging stays in registers;
  // LOAD: chunk c + 2 exists; STORE: chunk c + 1 exists
  auto step = [&](int c, auto buf_c, auto load_c, auto store_c) {
    constexpr int buf = decltype(buf_c)::value;
    if (decltype(load_c)::value) load_w(c + 2, reg[buf]);   // reg[buf] held chunk c, already in LDS
    __builtin_amdgcn_sched_barrier(0);   // keep the loads first and the LDS stores last
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 a = A_LDS ? arow(c, ks) : areg[buf][ks];
#pragma unroll
      for (int q = 0; q < TPW; ++q) {
        const int tile = wave + 4 * q;
        if (NTILE % 4 == 0 || tile < NTILE) {
          const int r = tile * 16 + (lane & 15);
          const u32x4 b = *reinterpret_cast<const u32x4*>(&lds[buf][r * PITCH + ks * 64 + (lane >> 4) * 16]);
          acc[q] = mfma_16x16x32(a, b, acc[q]);
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (decltype(load_c)::value) load_a(c + 2, areg[buf]);
    if (decltype(store_c)::value) store(buf ^ 1, reg[buf ^ 1]);
    __syncthreads();
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using Y = std::true_type;
  using N = std::false_type;
  int c = 0;
  for (; c + 3 < nc; c += 2) {
    step(c, B0{}, Y{}, Y{});
    step(c + 1, B1{}, Y{}, Y{});
  }
  if (nc - c == 3) {
    step(c, B0{}, Y{}, Y{});
    step(c + 1, B1{}, N{}, Y{});
    step(c + 2, B0{}, N{}, N{});
  } else if (nc - c == 2) {
    step(c, B0{}, N{}, Y{});
    step(c + 1, B1{}, N{}, N{});
  } else {
    step(c, B0{}, N{}, N{});
  }
}

// H[row0 + r, n0 + j] = SiLU(x_r . W_gate[n0 + j]) * (x_r . W_up[n0 + j]) for the rows of one
// active expert; grid (F / (16 * DEC_NT), max active experts, split_gu). With split_gu > 1
// each workgroup covers one slice of d and writes its partial dot products to P instead;
// decode_swiglu_kernel then adds the slices and applies SwiGLU.
template <bool PACKED>
__global__ __launch_bounds__(DEC_THREADS) void decode_gate_up_kernel(const DecodeArgs p) {
  constexpr int NTILE = 2 * DEC_NT;
  constexpr int TPW = (NTILE + 3) / 4;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][16 * NTILE * (DEC_CK * 2 + 16)];
  const int slot = blockIdx.y;
  if (slot >= p.n_active[0]) return;
  const int g = p.active[slot];
  const int row0 = p.offsets[g];
  const int nrows = p.offsets[g + 1] - row0;   // 1..16
  const int n0 = blockIdx.x * 16 * DEC_NT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint16_t* wg = g < p.E ? p.w_gate_up + static_cast<size_t>(weight_block(p, g)) * 2 * p.F * p.d
                               : p.ws_gate_up + static_cast<size_t>(g - p.E) * 2 * p.F * p.d;
  const int F = p.F, d = p.d;
  static_assert(16 * DEC_NT * 2 == kPackRows, "a workgroup's rows are one packed group");
  auto wrow = [=](int r) {  // rows 0..16*DEC_NT-1: W_gate, then the matching W_up rows
    if (PACKED) return wg + static_cast<size_t>(blockIdx.x) * kPackRows * d + r * kPackCols;
    const int n = n0 + (r % (16 * DEC_NT));
    return wg + static_cast<size_t>(r < 16 * DEC_NT ? n : F + n) * d;
  };
  const uint16_t* arow = p.x + static_cast<size_t>(p.row_tok[row0 + min(lane & 15, nrows - 1)]) * p.d;
  f32x4 acc[TPW];
#pragma unroll
  for (int q = 0; q < TPW; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int klen = p.d / p.split_gu, z = blockIdx.z;
  const RowOperand<false> aop{arow + z * klen + (lane >> 4) * 8};
  stream_rows<NTILE, PACKED ? kPackBlock : DEC_CK>(wrow, aop, z * klen, klen, lds, acc, [] {});
  if (p.split_gu > 1) {  // partial sums: wave w holds tiles w and w + 4 (gate tile j, up tile j)
#pragma unroll
    for (int q = 0; q < TPW; ++q) {
      const int tile = wave + 4 * q;
      const int col = n0 + (tile % DEC_NT) * 16 + (lane & 15) + (tile < DEC_NT ? 0 : F);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 4 * (lane >> 4) + i;
        if (row < nrows) p.P[(static_cast<size_t>(z) * p.rows + row0 + row) * 2 * F + col] = acc[q][i];
      }
    }
    return;
  }
  // gate tile j pairs with up tile j + DEC_NT: exchange through LDS
  f32x4* ex = reinterpret_cast<f32x4*>(&lds[0][0]);
#pragma unroll
  for (int q = 0; q < TPW; ++q) {
    const int tile = wave + 4 * q;
    if (tile < NTILE) ex[tile * 64 + lane] = acc[q];
  }
  __syncthreads();
  const int j = tid >> 6, l = tid & 63;   // DEC_NT = 4 gate tiles over 256 threads
  const f32x4 gs = ex[j * 64 + l], us = ex[(j + DEC_NT) * 64 + l];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * (l >> 4) + i;
    if (row < nrows)
      p.H[static_cast<size_t>(row0 + row) * p.F + n0 + j * 16 + (l & 15)] = f32_to_bf16(silu(gs[i]) * us[i]);
  }
}

// Four H values from the gate/up partial sums: SiLU(sum_z P[z, r, c]) * (sum_z P[z, r, F + c])
// for c = c0 .. c0 + 3, the slices added in order; `src` is &P[0, r, c0], `slice` the stride
// of z. The loads of all slices are issued together. Packed bf16, columns in order.
__device__ __forceinline__ uint2 swiglu_from_partials(const float* src, size_t slice, int F, int split) {
  float4 g[kDecodeMaxSplitGateUp], u[kDecodeMaxSplitGateUp];
#pragma unroll
  for (int z = 0; z < kDecodeMaxSplitGateUp; ++z) {
    if (z < split) {
      g[z] = *reinterpret_cast<const float4*>(src + z * slice);
      u[z] = *reinterpret_cast<const float4*>(src + z * slice + F);
    }
  }
  float4 gs = g[0], us = u[0];
#pragma unroll
  for (int z = 1; z < kDecodeMaxSplitGateUp; ++z) {
    if (z < split) {
      gs.x += g[z].x; gs.y += g[z].y; gs.z += g[z].z; gs.w += g[z].w;
      us.x += u[z].x; us.y += u[z].y; us.z += u[z].z; us.w += u[z].w;
    }
  }
  uint2 packed;
  packed.x = f32x2_to_bf16x2(silu(gs.x) * us.x, silu(gs.y) * us.y);
  packed.y = f32x2_to_bf16x2(silu(gs.z) * us.z, silu(gs.w) * us.w);
  return packed;
}

// H[r, c] = SiLU(sum_z P[z, r, c]) * (sum_z P[z, r, F + c]), slices added in order. One
// thread per four columns (F % 64 == 0).
__global__ __launch_bounds__(256) void decode_swiglu_kernel(const float* __restrict__ P, uint16_t* __restrict__ H,
                                                            int rows, int F, int split) {
  const int i = blockIdx.x * 256 + threadIdx.x;   // index of a group of four columns
  const int per_row = F / 4;
  if (i >= rows * per_row) return;
  const int r = i / per_row, c = (i - r * per_row) * 4;
  const size_t slice = static_cast<size_t>(rows) * 2 * F;
  *reinterpret_cast<uint2*>(H + static_cast<size_t>(r) * F + c) =
      swiglu_from_partials(P + static_cast<size_t>(r) * 2 * F + c, slice, F, split);
}

// O[z, row0 + r, n0 + j] = sum over k in slice z of H[row0 + r, k] * W_down[n0 + j, k];
// grid (d / (16 * DEC_NT), max active experts, split).
// SWIGLU: H is not materialised; the prologue builds the workgroup's H rows of slice z in LDS
// from the gate/up partial sums P with the arithmetic of decode_swiglu_kernel, so the bits are
// the same. The host takes this path when every group's rows of one slice fit in
// kFusedSwigluLds and take at most kFusedItems four-column groups per thread.
template <int NTILE, bool PACKED, bool SWIGLU = false>   // NTILE: 16-row W_down tiles per workgroup (4 or 8)
__global__ __launch_bounds__(DEC_THREADS) void decode_down_kernel(const DecodeArgs p) {
  static_assert(!PACKED || 16 * NTILE == kPackRows, "a workgroup's rows are one packed group");
  constexpr int TPW = (NTILE + 3) / 4;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][16 * NTILE * (DEC_CK * 2 + 16)];
  const int slot = blockIdx.y;
  if (slot >= p.n_active[0]) return;
  const int g = p.active[slot];
  const int row0 = p.offsets[g];
  const int nrows = p.offsets[g + 1] - row0;
  const int n0 = blockIdx.x * 16 * NTILE;
  const int z = blockIdx.z;
  const int klen = p.F / p.split;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint16_t* wd = g < p.E ? p.w_down + static_cast<size_t>(weight_block(p, g)) * p.d * p.F
                               : p.ws_down + static_cast<size_t>(g - p.E) * p.d * p.F;
  const int F = p.F;
  auto wrow = [=](int r) {
    return PACKED ? wd + static_cast<size_t>(n0) * F + r * kPackCols : wd + static_cast<size_t>(n0 + r) * F;
  };
  f32x4 acc[TPW];
#pragma unroll
  for (int q = 0; q < TPW; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (SWIGLU) {
    __shared__ __attribute__((aligned(16))) uint16_t hs[kFusedSwigluLds / 2];
    const int pitch = klen + 8;   // 16 bytes past a multiple of 128: rows start on different banks
    const RowOperand<true> aop{hs + min(lane & 15, nrows - 1) * pitch + (lane >> 4) * 8};
    auto prologue = [&] {
      const int per_row = klen / 4, items = nrows * per_row;
      const size_t slice = static_cast<size_t>(p.rows) * 2 * F;
#pragma unroll
      for (int i = 0; i < kFusedItems; ++i) {
        const int it = threadIdx.x + i * DEC_THREADS;
        if (it < items) {
          const int r = it / per_row, c = (it - r * per_row) * 4;
          *reinterpret_cast<uint2*>(hs + r * pitch + c) = swiglu_from_partials(
              p.P + static_cast<size_t>(row0 + r) * 2 * F + z * klen + c, slice, F, p.split_gu);
        }
      }
    };
    stream_rows<NTILE, PACKED ? kPackBlock : DEC_CK>(wrow, aop, z * klen, klen, lds, acc, prologue);
  } else {
    const uint16_t* arow = p.H + static_cast<size_t>(row0 + min(lane & 15, nrows - 1)) * p.F;
    const RowOperand<false> aop{arow + z * klen + (lane >> 4) * 8};
    stream_rows<NTILE, PACKED ? kPackBlock : DEC_CK>(wrow, aop, z * klen, klen, lds, acc, [] {});
  }
  // wave w holds tiles w, w + 4: rows 4*(lane>>4)+i, column lane & 15
#pragma unroll
  for (int q = 0; q < TPW; ++q)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * (lane >> 4) + i;
      if (row < nrows)
        p.O[(static_cast<size_t>(z) * p.rows + row0 + row) * p.d + n0 + (wave + 4 * q) * 16 + (lane & 15)] = acc[q][i];
    }
}

// ------------------------------------------------------------------ f32 kernels

__device__ __forceinline__ int group_of_row(const int32_t* offsets, int G, int pos) {
  int lo = 0, hi = G;  // offsets[lo] <= pos < offsets[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (offsets[mid] <= pos) lo = mid; else hi = mid;
  }
  return lo;
}

struct F32Args {
  const float* x;
  const int32_t* row_tok;
  const int32_t* offsets;
  const float* w_gate_up;
  const float* w_down;
  const float* ws_gate_up;
  const float* ws_down;
  float* H;
  float* O;
  int rows, d, F, E, G;
};

__global__ __launch_bounds__(256) void f32_gate_up_kernel(const F32Args p) {
  const size_t id = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= static_cast<size_t>(p.rows) * p.F) return;
  const int pos = static_cast<int>(id / p.F), n = static_cast<int>(id % p.F);
  const int g = group_of_row(p.offsets, p.G, pos);
  const float* w = g < p.E ? p.w_gate_up + static_cast<size_t>(g) * 2 * p.F * p.d
                           : p.ws_gate_up + static_cast<size_t>(g - p.E) * 2 * p.F * p.d;
  const float* xr = p.x + static_cast<size_t>(p.row_tok[pos]) * p.d;
  const float* wg = w + static_cast<size_t>(n) * p.d;
  const float* wu = w + static_cast<size_t>(p.F + n) * p.d;
  float a = 0.0f, b = 0.0f;
  for (int k = 0; k < p.d; ++k) {
    a = fmaf(xr[k], wg[k], a);
    b = fmaf(xr[k], wu[k], b);
  }
  p.H[id] = (a / (1.0f + expf(-a))) * b;
}

__global__ __launch_bounds__(256) void f32_down_kernel(const F32Args p) {
  const size_t id = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= static_cast<size_t>(p.rows) * p.d) return;
  const int pos = static_cast<int>(id / p.d), n = static_cast<int>(id % p.d);
  const int g = group_of_row(p.offsets, p.G, pos);
  const float* w = g < p.E ? p.w_down + static_cast<size_t>(g) * p.d * p.F
                           : p.ws_down + static_cast<size_t>(g - p.E) * p.d * p.F;
  const float* h = p.H + static_cast<size_t>(pos) * p.F;
  const float* wr = w + static_cast<size_t>(n) * p.F;
  float a = 0.0f;
  for (int k = 0; k < p.F; ++k) a = fmaf(h[k], wr[k], a);
  p.O[id] = a;
}

}  // namespace

int device_cus_per_xcd() {
  int dev = 0, cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu < 8)
    cu = 256;
  return cu / 8;
}

// Grid of a grouped GEMM: 8 XCDs x (their largest share of tiles + tail slices).
static dim3 grouped_grid(int max_tiles, int n_tiles) {
  const long per_xcd = (static_cast<long>(max_tiles) * n_tiles + 7) / 8 + kTailSlotsPerXcd;
  return dim3(static_cast<unsigned>(8 * per_xcd));
}

template <int EPI>
static void launch_grouped(bool lora, bool packed, dim3 grid, const GemmArgs& g, hipStream_t stream) {
  if (lora && packed)
    hipLaunchKernelGGL((grouped_gemm_bf16<EPI, true, true>), grid, dim3(GEMM_THREADS), 0, stream, g);
  else if (lora)
    hipLaunchKernelGGL((grouped_gemm_bf16<EPI, true>), grid, dim3(GEMM_THREADS), 0, stream, g);
  else if (packed)
    hipLaunchKernelGGL((grouped_gemm_bf16<EPI, false, true>), grid, dim3(GEMM_THREADS), 0, stream, g);
  else
    hipLaunchKernelGGL((grouped_gemm_bf16<EPI>), grid, dim3(GEMM_THREADS), 0, stream, g);
}

hipError_t launch_experts_bf16(const ExpertArgs& a, const PermBuffers& pb, uint16_t* H, float* O, float* part,
                               void* y, int max_tiles, hipStream_t stream, hipEvent_t* marks, uint16_t* ab,
                               const LoraArgs* lora) {
  const int G = a.E + a.n_shared;
  GemmArgs g{};
  g.ab = ab;
  g.part = part;
  g.cu_xcd = device_cus_per_xcd();
  const dim3 fixup_grid(8 * kTailSlotsPerXcd * kTailFixParts);
  hipError_t err;
  if (lora) {
    err = launch_lora_pack(*lora, G, a.E, a.F, a.d, stream);
    if (err != hipSuccess) return err;
    err = launch_lora_down(static_cast<const uint16_t*>(a.x), pb.row_tok, a.d, lora->a_gate_up,
                           lora->as_gate_up, 2 * lora->rank, G, a.E, pb, max_tiles, lora->u, stream);
    if (err != hipSuccess) return err;
    g.lora_u = lora->u;
    g.lora_b = lora->bp_gate_up;
  }
  g.row_tok = pb.row_tok;
  g.offsets = pb.offsets;
  g.tile_off = pb.tile_off;
  g.G = G; g.E = a.E; g.F = a.F; g.d = a.d;
  g.mt_max = max_tiles;

  g.a = static_cast<const uint16_t*>(a.x);
  g.w = static_cast<const uint16_t*>(a.w_gate_up);
  g.ws = static_cast<const uint16_t*>(a.ws_gate_up);
  g.out = H;
  const int nt1 = (a.F + BN / 2 - 1) / (BN / 2);
  g.n_tiles = nt1;
  launch_grouped<0>(lora != nullptr, a.packed, grouped_grid(max_tiles, nt1), g, stream);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  record_mark(marks, 0, stream);
  if (lora) {
    err = launch_lora_down(H, nullptr, a.F, lora->a_down, lora->as_down, lora->rank, G, a.E, pb, max_tiles, lora->v,
                           stream);
    if (err != hipSuccess) return err;
    g.lora_u = lora->v;
    g.lora_b = lora->bp_down;
  }

  g.ab = nullptr;
  g.a = H;
  g.w = static_cast<const uint16_t*>(a.w_down);
  g.ws = static_cast<const uint16_t*>(a.ws_down);
  g.out = O;
  const int nt2 = (a.d + BN - 1) / BN;
  g.n_tiles = nt2;
  launch_grouped<1>(lora != nullptr, a.packed, grouped_grid(max_tiles, nt2), g, stream);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (tail_can_split(1, a.F / BK)) {
    hipLaunchKernelGGL(grouped_tail_fixup, fixup_grid, dim3(GEMM_THREADS), 0, stream, g);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  record_mark(marks, 1, stream);

  // O holds bf16 expert outputs; with K known, eight columns per thread
  const dim3 cgrid = combine_grid(a.T, a.d), cgrid8 = combine_grid(a.T, a.d, kCombineColsOB), cblk(256);
  if (a.K == 2)
    hipLaunchKernelGGL((combine_kernel<true, 2, true>), cgrid8, cblk, 0, stream, O, pb.inv, a.gate, a.T, a.K,
                       a.n_shared, a.d, y, 1, a.expert_out);
  else if (a.K == 6)
    hipLaunchKernelGGL((combine_kernel<true, 6, true>), cgrid8, cblk, 0, stream, O, pb.inv, a.gate, a.T, a.K,
                       a.n_shared, a.d, y, 1, a.expert_out);
  else
    hipLaunchKernelGGL((combine_kernel<true, 0, true>), cgrid, cblk, 0, stream, O, pb.inv, a.gate, a.T, a.K,
                       a.n_shared, a.d, y, 1, a.expert_out);
  err = hipGetLastError();
  record_mark(marks, 2, stream);
  return err;
}

// Slices of the reduction dimension for the two streaming kernels. Measured on MI355X (a sweep
// of the target at 1, 4 and 16 tokens), the gate/up stream runs best with about 1800
// workgroups in flight and the down stream with about 1300 (fewer slices also shorten the
// combine, which adds them), as long as each slice keeps at
// least 16 chunks (shorter slices lose more to their start-up than the extra workgroups
// gain): fewer workgroups leave HBM channels idle, and a count just past one full residency
// wave leaves a ragged second wave. The split is the power of two (dividing the chunk count,
// keeping >= kDecodeMinChunks per slice) whose workgroup count is closest to the target, for
// the number of experts a batch of T tokens is expected to activate under uniform routing,
// E (1 - (1 - K/E)^T), plus the shared experts. The grid is still sized for the most experts
// that can be active; the estimate only picks the split.
constexpr int kDecodeTargetWGsGateUp = 1792, kDecodeTargetWGsDown = 1280, kDecodeMinChunks = 16;
constexpr int kDecodeDownTiles = 8;

static int best_split(int per_slice_wgs, int chunks, int max_split, int target) {
  if (per_slice_wgs <= 0) return 1;  // no tokens: nothing is launched
  int best = 1, best_gap = 1 << 30;
  for (int s = 1; s <= max_split; s *= 2) {
    if (chunks % s || (s > 1 && chunks / s < kDecodeMinChunks)) break;
    const int gap = std::abs(per_slice_wgs * s - target);
    if (gap < best_gap) {
      best_gap = gap;
      best = s;
    }
  }
  return best;
}

static int max_active_groups(int T, int E, int K, int n_shared) {
  return (T * K < E ? T * K : E) + n_shared;
}

static int expected_active_groups(int T, int E, int K, int n_shared) {
  if (T <= 0) return 0;
  const double routed = E * (1.0 - std::pow(1.0 - static_cast<double>(K) / E, T));
  int a = static_cast<int>(std::lround(routed));
  a = std::max(a, K);
  a = std::min(a, T * K < E ? T * K : E);
  return a + n_shared;
}

// W_down rows per decode workgroup: 16 * decode_down_tiles(d).
static int decode_down_tiles(int d) { return d % (16 * kDecodeDownTiles) == 0 ? kDecodeDownTiles : DEC_NT; }

int decode_split(int T, int d, int F, int E, int K, int n_shared) {
  return best_split(d / (16 * decode_down_tiles(d)) * expected_active_groups(T, E, K, n_shared), F / DEC_CK,
                    kDecodeMaxSplit, kDecodeTargetWGsDown);
}

int decode_split_gate_up(int T, int d, int F, int E, int K, int n_shared) {
  return best_split(F / (16 * DEC_NT) * expected_active_groups(T, E, K, n_shared), d / DEC_CK,
                    kDecodeMaxSplitGateUp, kDecodeTargetWGsGateUp);
}

hipError_t launch_experts_bf16_decode(const ExpertArgs& a, const PermBuffers& pb, uint16_t* H, float* P, float* O,
                                      void* y, hipStream_t stream, hipEvent_t* marks) {
  DecodeArgs p;
  p.x = static_cast<const uint16_t*>(a.x);
  p.row_tok = pb.row_tok;
  p.offsets = pb.offsets;
  p.active = pb.active;
  p.n_active = pb.n_active;
  p.w_gate_up = static_cast<const uint16_t*>(a.w_gate_up);
  p.w_down = static_cast<const uint16_t*>(a.w_down);
  p.ws_gate_up = static_cast<const uint16_t*>(a.ws_gate_up);
  p.ws_down = static_cast<const uint16_t*>(a.ws_down);
  p.H = H;
  p.P = P;
  p.O = O;
  p.slot_of = a.slot_of;
  p.n_slots = a.n_slots;
  p.T = a.T; p.d = a.d; p.F = a.F; p.E = a.E; p.K = a.K;
  p.rows = a.T * (a.K + a.n_shared);
  p.split = decode_split(a.T, a.d, a.F, a.E, a.K, a.n_shared);
  p.split_gu = decode_split_gate_up(a.T, a.d, a.F, a.E, a.K, a.n_shared);
  const int max_active = max_active_groups(a.T, a.E, a.K, a.n_shared);
  const dim3 gu_grid(a.F / (16 * DEC_NT), max_active, p.split_gu);
  if (a.packed)
    hipLaunchKernelGGL(decode_gate_up_kernel<true>, gu_grid, dim3(DEC_THREADS), 0, stream, p);
  else
    hipLaunchKernelGGL(decode_gate_up_kernel<false>, gu_grid, dim3(DEC_THREADS), 0, stream, p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  record_mark(marks, 0, stream);
  // A group holds at most T rows (a token picks an expert once; a shared expert takes all T).
  const int klen_down = p.F / p.split;
  const bool fuse = p.split_gu > 1 && a.T * (klen_down + 8) * 2 <= kFusedSwigluLds &&
                    a.T * (klen_down / 4) <= kFusedItems * DEC_THREADS;
  if (p.split_gu > 1 && !fuse) {  // timed with the down stage
    const int groups = p.rows * (p.F / 4);   // rows <= 16 (K + n_shared): no overflow
    const unsigned blocks = static_cast<unsigned>((groups + 255) / 256);
    hipLaunchKernelGGL(decode_swiglu_kernel, dim3(blocks), dim3(256), 0, stream, P, H, p.rows, p.F, p.split_gu);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  const dim3 dn_grid8(a.d / 128, max_active, p.split), dn_grid4(a.d / (16 * DEC_NT), max_active, p.split);
  if (a.packed && fuse)   // d % kPackRows == 0, so decode_down_tiles(d) == 8
    hipLaunchKernelGGL((decode_down_kernel<8, true, true>), dn_grid8, dim3(DEC_THREADS), 0, stream, p);
  else if (a.packed)
    hipLaunchKernelGGL((decode_down_kernel<8, true>), dn_grid8, dim3(DEC_THREADS), 0, stream, p);
  else if (decode_down_tiles(a.d) == 8 && fuse)
    hipLaunchKernelGGL((decode_down_kernel<8, false, true>), dn_grid8, dim3(DEC_THREADS), 0, stream, p);
  else if (decode_down_tiles(a.d) == 8)
    hipLaunchKernelGGL((decode_down_kernel<8, false>), dn_grid8, dim3(DEC_THREADS), 0, stream, p);
  else if (fuse)
    hipLaunchKernelGGL((decode_down_kernel<DEC_NT, false, true>), dn_grid4, dim3(DEC_THREADS), 0, stream, p);
  else
    hipLaunchKernelGGL((decode_down_kernel<DEC_NT, false>), dn_grid4, dim3(DEC_THREADS), 0, stream, p);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  record_mark(marks, 1, stream);
  hipLaunchKernelGGL(combine_kernel<true>, combine_grid(a.T, a.d), dim3(256), 0, stream, O, pb.inv, a.gate, a.T, a.K,
                     a.n_shared, a.d, y, p.split, a.expert_out);
  err = hipGetLastError();
  record_mark(marks, 2, stream);
  return err;
}

// ------------------------------------------------------------------ packed weight layout
//
// One thread per 16-byte piece of the packed output, in output order: piece u of block
// ((e * groups + q) * chunks + c) is row i = (u % 1024) / 8 of the block, columns
// 8 * (u % 8) .. + 7 of chunk c. gate_up: block row i < 64 is W_gate row 64 q + i, the rest
// the matching W_up rows F + 64 q + i - 64; otherwise block row i is row kPackRows q + i.
// Reads are 128-byte row pieces, writes are contiguous.
__global__ __launch_bounds__(256) void pack_weights_kernel(const uint16_t* __restrict__ src,
                                                           uint16_t* __restrict__ dst, int n, int rows, int cols,
                                                           bool gate_up, int F) {
  const size_t pieces = static_cast<size_t>(n) * rows * cols / 8;
  const int chunks = cols / kPackCols, groups = rows / kPackRows;
  for (size_t u = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; u < pieces;
       u += static_cast<size_t>(gridDim.x) * 256) {
    const size_t blk = u / (kPackBlock / 8);
    const int within = static_cast<int>(u % (kPackBlock / 8));
    const int i = within / 8, j = (within % 8) * 8;
    const int c = static_cast<int>(blk % chunks);
    const size_t eq = blk / chunks;
    const int q = static_cast<int>(eq % groups);
    const size_t e = eq / groups;
    const int row = gate_up ? (i < 64 ? q * 64 + i : F + q * 64 + (i - 64)) : q * kPackRows + i;
    const u32x4 v = *reinterpret_cast<const u32x4*>(src + (e * rows + row) * cols + static_cast<size_t>(c) * kPackCols + j);
    *reinterpret_cast<u32x4*>(dst + u * 8) = v;
  }
}

hipError_t launch_pack_weights(const uint16_t* w_gate_up, const uint16_t* w_down, uint16_t* p_gate_up,
                               uint16_t* p_down, int n, int d, int F, hipStream_t stream) {
  const size_t pieces = static_cast<size_t>(n) * 2 * F * d / 8;   // gate/up; down has half
  const dim3 grid(static_cast<unsigned>(std::min<size_t>((pieces + 255) / 256, 16384)));
  if (w_gate_up) {
    hipLaunchKernelGGL(pack_weights_kernel, grid, dim3(256), 0, stream, w_gate_up, p_gate_up, n, 2 * F, d, true, F);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  if (w_down) {
    hipLaunchKernelGGL(pack_weights_kernel, grid, dim3(256), 0, stream, w_down, p_down, n, d, F, false, F);
    return hipGetLastError();
  }
  return hipSuccess;
}

hipError_t launch_experts_f32(const ExpertArgs& a, const PermBuffers& pb, float* H, float* O,
                              void* y, hipStream_t stream, hipEvent_t* marks) {
  F32Args p;
  p.x = static_cast<const float*>(a.x);
  p.row_tok = pb.row_tok;
  p.offsets = pb.offsets;
  p.w_gate_up = static_cast<const float*>(a.w_gate_up);
  p.w_down = static_cast<const float*>(a.w_down);
  p.ws_gate_up = static_cast<const float*>(a.ws_gate_up);
  p.ws_down = static_cast<const float*>(a.ws_down);
  p.H = H;
  p.O = O;
  p.rows = a.T * (a.K + a.n_shared);
  p.d = a.d; p.F = a.F; p.E = a.E; p.G = a.E + a.n_shared;
  const size_t n1 = static_cast<size_t>(p.rows) * a.F, n2 = static_cast<size_t>(p.rows) * a.d;
  hipLaunchKernelGGL(f32_gate_up_kernel, dim3((n1 + 255) / 256), dim3(256), 0, stream, p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  record_mark(marks, 0, stream);
  hipLaunchKernelGGL(f32_down_kernel, dim3((n2 + 255) / 256), dim3(256), 0, stream, p);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  record_mark(marks, 1, stream);
  hipLaunchKernelGGL(combine_kernel<false>, combine_grid(a.T, a.d), dim3(256), 0, stream, O, pb.inv, a.gate, a.T,
                     a.K, a.n_shared, a.d, y, 1, a.expert_out);
  err = hipGetLastError();
  record_mark(marks, 2, stream);
  return err;
}

}  // namespace maskmoe
