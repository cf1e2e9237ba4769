// Expert-side backward of the masked MoE layer: the SwiGLU experts' weight gradients and their
// share of dL/dx, with the routing held fixed.
//
// The routers and experts update at every step (Section 3.2, Stage 1; Stage 2 continues with
// them). By Eq. 1, routed expert e receives dL/dF = g dy on the tokens that chose it and a
// shared expert dy on every token. Through F(x) = W_down (SiLU(W_gate x) * W_up x), with
// a = x W_gate^T, b = x W_up^T, h = SiLU(a) * b kept by the training forward:
//   dh = dO W_down               da = dh * b * SiLU'(a),  db = dh * SiLU(a)
//   dX = da W_gate + db W_up     dW_down = dO^T h,  dW_gate = da^T x,  dW_up = db^T x
// per expert, over the permuted rows of the forward (one row per (token, slot), shared
// experts' rows after them).
//
// Every product is run as C = A B^T on the 256x256x64 MFMA tile of gemm_tile.hpp. Operands whose
// contraction index is strided in storage are read in place as K-major operands (loaded by rows
// of the contraction index, turned into MFMA operands by transposing LDS reads): the weights
// of the dgrads, and both operands of the weight gradients, whose contraction runs over each
// expert's own rows of dO, h, [da db] and the gathered x (rows past the group's end read as
// zeros; an expert no token chose gets zeros).
// Rounding (bf16 layers): dO = g dy and [da db] are rounded to bf16 before their GEMMs;
// accumulation is fp32; dX, dW are fp32.

#include <mutex>

#include "common.hpp"
#include "gemm_tile.hpp"
#include "kernels.hpp"

namespace maskmoe {
namespace {

constexpr int kBwdThreads = 256;

__device__ __forceinline__ uint32_t scale_pair(uint32_t v, float w) {
  const float lo = bf16_to_f32(static_cast<uint16_t>(v & 0xffffu)) * w;
  const float hi = bf16_to_f32(static_cast<uint16_t>(v >> 16)) * w;
  return f32x2_to_bf16x2(lo, hi);
}

// dO[r, :] = bf16(w_r dy[row_tok[r], :]): w_r the gate of the (token, slot) entry at routed row
// r, 1 for shared-expert rows. One workgroup per row; d % 8 == 0.
__global__ __launch_bounds__(kBwdThreads) void build_dout_kernel(const uint16_t* __restrict__ dy,
                                                                 const float* __restrict__ gate,
                                                                 const int32_t* __restrict__ perm,
                                                                 const int32_t* __restrict__ row_tok, int TK, int d,
                                                                 uint16_t* __restrict__ dout) {
  const int r = blockIdx.x;
  const float w = r < TK ? gate[perm[r]] : 1.0f;
  const uint16_t* src = dy + static_cast<size_t>(row_tok[r]) * d;
  uint16_t* dst = dout + static_cast<size_t>(r) * d;
  for (int c = threadIdx.x * 8; c < d; c += kBwdThreads * 8) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(src + c);
    u32x4 o;
#pragma unroll
    for (int h = 0; h < 4; ++h) o[h] = scale_pair(v[h], w);
    *reinterpret_cast<u32x4*>(dst + c) = o;
  }
}

// xg[r, :] = x[row_tok[r], :] (the gathered tokens of the weight gradient of gate/up, read in
// place as a K-major operand). One workgroup per row; d % 8 == 0.
__global__ __launch_bounds__(kBwdThreads) void gather_rows_kernel(const uint16_t* __restrict__ x,
                                                                  const int32_t* __restrict__ row_tok, int d,
                                                                  uint16_t* __restrict__ xg) {
  const int r = blockIdx.x;
  const uint16_t* src = x + static_cast<size_t>(row_tok[r]) * d;
  uint16_t* dst = xg + static_cast<size_t>(r) * d;
  for (int c = threadIdx.x * 8; c < d; c += kBwdThreads * 8)
    *reinterpret_cast<u32x4*>(dst + c) = *reinterpret_cast<const u32x4*>(src + c);
}

struct NtArgs {
  const uint16_t* a;          // ROWS: [rows, K] (lda), K-contiguous; KSPLIT: K-major [rows, M] (lda)
  const uint16_t* b;          // ROWS: per routed expert K-major [K, N] matrices (ldb = N); KSPLIT: K-major [rows, N]
  const uint16_t* bs;         // ROWS: the shared experts' [K, N] matrices
  const int32_t* offsets;     // [G+1] rows of each group
  const int32_t* tile_off;    // [G+1] row tiles of each group (ROWS)
  const int32_t* active;      // KSPLIT: the non-empty groups, n_active[0] of them
  const int32_t* n_active;
  const uint16_t* ab;         // SWIGLU_BWD: saved pre-activations [rows, 2N]
  void* c;                    // ROWS: [rows, ldc]; KSPLIT: routed groups' [M, N] matrices
  void* cs;                   // KSPLIT: shared groups' [M, N] matrices
  float* part;                // ROWS, fp32 output: partial tiles of split tail tiles (tile_job)
  int G, E, M, N, K, lda, ldb, ldc, mt_max, n_tiles;
  int cu_xcd;                 // workgroups an XCD runs at once
};

// ROWS with fp32 output may split each XCD's last-round tiles (see tile_job).
__host__ __device__ constexpr bool nt_tail_split(int mode, int epi, int nk) {
  return mode == 0 && epi == 1 && tail_splittable(nk);
}

// Stores a finished ROWS tile of fp32 output: rows [row0, row_end), columns from n0.
// Staged fp32 tiles: 128 rows x 256 columns at a pitch of 264 floats (the two 32-lane halves of
// a wavefront, four rows apart, then write different banks).
constexpr int kStgPitch = 264;
static_assert(128 * kStgPitch * 4 <= sizeof(TileLds), "a staged half tile fits in LDS");

// Half h (0, 1) of the tile into LDS: acc[2h + ii] of every wave, as staged row
// wm*64 + ii*32 + (row within the 32-row block). Staged row pr is tile row
// (pr >> 6) * 128 + 64 h + (pr & 63).
__device__ __forceinline__ void stage_half(float* stg, const f32x16 (&acc)[kTileTM][kTileTN], int h) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / 4, wn = wave % 4;
#pragma unroll
  for (int ii = 0; ii < 2; ++ii)
#pragma unroll
    for (int r = 0; r < 16; ++r)
#pragma unroll
      for (int j = 0; j < kTileTN; ++j)
        stg[(wm * 64 + ii * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * kStgPitch + wn * 64 + j * 32 +
            (lane & 31)] = (h == 0 ? acc[ii][j][r] : acc[2 + ii][j][r]);
}

// The fp32 tile (rows row0.., columns n0..) into out (row stride ld), through LDS in two halves
// so that it leaves in 16-byte stores: one 4-byte store per value and lane kept the
// texture-address path busy for ~10 us at the end of every tile. ncol % 4 == 0.
__device__ __forceinline__ void nt_store_staged(const f32x16 (&acc)[kTileTM][kTileTN], float* out, size_t ld, int row0,
                                                int row_end, int n0, int ncol, TileLds& L) {
  float* stg = reinterpret_cast<float*>(&L);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    wait_lgkmcnt0();
    tile_barrier();   // the k-loop's (or the previous half's) LDS reads are done
    stage_half(stg, acc, h);
    wait_lgkmcnt0();
    tile_barrier();
#pragma unroll 4
    for (int q = 0; q < 16; ++q) {   // 8192 float4 per half: 64 per staged row
      const int u = static_cast<int>(threadIdx.x) + kTileThreads * q;
      const int pr = u >> 6, c = (u & 63) * 4;
      const int row = row0 + (pr >> 6) * 128 + 64 * h + (pr & 63), col = n0 + c;
      if (row < row_end && col < ncol)
        *reinterpret_cast<float4*>(out + static_cast<size_t>(row) * ld + col) =
            *reinterpret_cast<const float4*>(&stg[pr * kStgPitch + c]);
    }
  }
}

enum { kNtRows = 0, kNtKSplit = 1 };
enum { kEpiSwigluBwd = 0, kEpiF32 = 1 };

// ROWS (dgrad): group g's rows offsets[g]..offsets[g+1] of A (K-contiguous) times its own
// K-major [K, N] matrix, row tiles enumerated by tile_off as in the forward. KSPLIT (wgrad): for
// every non-empty group g the full [M, N] product over its rows offsets[g]..offsets[g+1] of the
// K-major A [rows, M] and B [rows, N]; the grid is sized for all groups and the live tiles
// (n_active x tiles per group) are spread over the XCDs.
template <int MODE, int EPI>
__global__ __launch_bounds__(kTileThreads) void gemm_nt_kernel(const NtArgs p) {
  constexpr int TM = kTileTM, TN = kTileTN, WN = 4;
  __shared__ TileLds lds;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave % WN;
  int mt, nt, g, row0, row_end, nk;
  TileJob job{0, 0, 1, -1};
  TileOps ops{};
  TileKm akm{}, bkm{};
  if (MODE == kNtRows) {   // each XCD's share of the live row tiles (tile_job)
    const int mt_live = p.tile_off[p.G];
    const int live = mt_live * p.n_tiles;
    const int nkf = p.K / kTileK;
    if (!tile_job(static_cast<int>(blockIdx.x), live, p.cu_xcd, nkf, nt_tail_split(MODE, EPI, nkf), job)) return;
    grouped_tile_coords(job.lid, mt_live, p.n_tiles, mt, nt);
    int lo = 0, hi = p.G;   // tile_off[lo] <= mt < tile_off[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (p.tile_off[mid] <= mt) lo = mid; else hi = mid;
    }
    g = lo;
    row0 = p.offsets[g] + (mt - p.tile_off[g]) * kTileM;
    row_end = p.offsets[g + 1];
    nk = nkf / job.s;
    const int k0 = job.z * nk * kTileK;
    const int n0 = nt * kTileN;
    ops.a = reinterpret_cast<const char*>(p.a + k0);
#pragma unroll
    for (int i = 0; i < 4; ++i)   // element offsets < 2^31 (checked by the host)
      ops.aoff[i] = static_cast<uint32_t>(min(row0 + tile_dma_row(i), row_end - 1) * p.lda + tile_dma_chunk(i) * 8) * 2u;
    const uint16_t* bm = g < p.E ? p.b + static_cast<size_t>(g) * p.N * p.K : p.bs + static_cast<size_t>(g - p.E) * p.N * p.K;
    bkm.base = reinterpret_cast<const char*>(bm + static_cast<size_t>(k0) * p.ldb + n0);
    bkm.ld = p.ldb * 2;
    bkm.krows = nk * kTileK;
    bkm.mcols = p.N - n0;
  } else {
    const int per = p.mt_max * p.n_tiles;
    const int live = p.n_active[0] * per;
    if (static_cast<int>(blockIdx.x) >= live) return;
    const int lid = xcd_tile_id(live);
    g = p.active[lid / per];
    grouped_tile_coords(lid % per, p.mt_max, p.n_tiles, mt, nt);
    row0 = mt * kTileM;
    row_end = p.M;
    const int r0 = p.offsets[g], nrows = p.offsets[g + 1] - r0;
    nk = (nrows + kTileK - 1) / kTileK;
    akm.base = reinterpret_cast<const char*>(p.a + static_cast<size_t>(r0) * p.lda + row0);
    akm.ld = p.lda * 2;
    akm.krows = nrows;
    akm.mcols = p.M - row0;
    bkm.base = reinterpret_cast<const char*>(p.b + static_cast<size_t>(r0) * p.ldb + nt * kTileN);
    bkm.ld = p.ldb * 2;
    bkm.krows = nrows;
    bkm.mcols = p.N - nt * kTileN;
  }
  const int n0 = nt * kTileN;
  int bfrag[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) bfrag[j] = wn * 64 + j * 32 + (lane & 31);
  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  gemm_tile_mainloop<false, MODE == kNtKSplit, true>(ops, nk, bfrag, acc, lds, nullptr, &akm, &bkm);
  if (MODE == kNtRows && EPI == kEpiF32) {
    if (job.s > 1) tail_store_partial(p.part, job.slot, acc);   // a slice of a split tail tile
    else nt_store_staged(acc, static_cast<float*>(p.c), p.ldc, row0, row_end, nt * kTileN, p.N, lds);
    return;
  }

  // acc[i][j][4 jj + ii] is row wm*128 + i*32 + 8 jj + 4 (lane >> 5) + ii, column
  // wn*64 + j*32 + (lane & 31) of the tile.
  if (EPI == kEpiSwigluBwd) {
    // v = dh; da, db (bf16) into [rows, 2N]. The tile goes through LDS (free after the k-loop)
    // in two halves of 128 rows x 256 columns, so that each thread then reads a, b and writes
    // da, db eight columns at a time: 16-byte accesses instead of one 2-byte access per value
    // and operand, which kept the texture-address path busy for a fifth of the kernel. A half's
    // a and b are loaded before it is staged, all in flight together. N % 64 == 0 (checked by
    // the host), so a group of eight columns is either whole or past N.
    float* stg = reinterpret_cast<float*>(&lds);
    uint16_t* o = static_cast<uint16_t*>(p.c);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      u32x4 a8[8], b8[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {   // 4096 groups of 8 columns: 32 per staged row
        const int u = tid + kTileThreads * q;
        const int pr = u >> 5, col = n0 + (u & 31) * 8;
        const int row = row0 + (pr >> 6) * 128 + 64 * h + (pr & 63);
        if (row < row_end && col < p.N) {
          const uint16_t* src = p.ab + static_cast<size_t>(row) * 2 * p.N + col;
          a8[q] = *reinterpret_cast<const u32x4*>(src);
          b8[q] = *reinterpret_cast<const u32x4*>(src + p.N);
        }
      }
      wait_lgkmcnt0();
      tile_barrier();   // the k-loop's (or the previous half's) LDS reads are done
      stage_half(stg, acc, h);
      wait_lgkmcnt0();
      tile_barrier();
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int u = tid + kTileThreads * q;
        const int pr = u >> 5, cg = (u & 31) * 8, col = n0 + cg;
        const int row = row0 + (pr >> 6) * 128 + 64 * h + (pr & 63);
        if (row >= row_end || col >= p.N) continue;
        float v[8];
        *reinterpret_cast<float4*>(&v[0]) = *reinterpret_cast<const float4*>(&stg[pr * kStgPitch + cg]);
        *reinterpret_cast<float4*>(&v[4]) = *reinterpret_cast<const float4*>(&stg[pr * kStgPitch + cg + 4]);
        const uint16_t* av8 = reinterpret_cast<const uint16_t*>(&a8[q]);
        const uint16_t* bv8 = reinterpret_cast<const uint16_t*>(&b8[q]);
        uint16_t da8[8], db8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float av = bf16_to_f32(av8[e]), bv = bf16_to_f32(bv8[e]);
          const float s = sigmoid(av);
          da8[e] = f32_to_bf16(v[e] * bv * (s * (1.0f + av * (1.0f - s))));
          db8[e] = f32_to_bf16(v[e] * av * s);
        }
        uint16_t* dst = o + static_cast<size_t>(row) * 2 * p.N + col;
        *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(da8);
        *reinterpret_cast<u32x4*>(dst + p.N) = *reinterpret_cast<const u32x4*>(db8);
      }
    }
    return;
  }
  float* cf = g < p.E ? static_cast<float*>(p.c) + static_cast<size_t>(g) * p.M * p.N
                      : static_cast<float*>(p.cs) + static_cast<size_t>(g - p.E) * p.M * p.N;
  nt_store_staged(acc, cf, p.N, row0, row_end, n0, p.N, lds);
}

// Adds the slices of each split tail tile of the ROWS fp32 product in slice order and stores
// it; kTailFixParts workgroups per possible tail tile, grid 8 x kTailSlotsPerXcd x kTailFixParts.
__global__ __launch_bounds__(kTileThreads) void nt_tail_fixup(const NtArgs p) {
  const int mt_live = p.tile_off[p.G];
  const int live = mt_live * p.n_tiles;
  const int nk = p.K / kTileK;
  const int b = blockIdx.x, xcd = b & 7, t = (b >> 3) % kTailSlotsPerXcd, part = b / (8 * kTailSlotsPerXcd);
  const XcdShare x = xcd_share(xcd, live, p.cu_xcd, nk, nt_tail_split(kNtRows, kEpiF32, nk));
  if (x.s == 1 || t >= x.r) return;
  int mt, nt;
  grouped_tile_coords(x.base + x.full + t, mt_live, p.n_tiles, mt, nt);
  int lo = 0, hi = p.G;   // tile_off[lo] <= mt < tile_off[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (p.tile_off[mid] <= mt) lo = mid; else hi = mid;
  }
  const int row0 = p.offsets[lo] + (mt - p.tile_off[lo]) * kTileM, row_end = p.offsets[lo + 1], n0 = nt * kTileN;
  float* out = static_cast<float*>(p.c);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wm = wave / 4, wn = wave % 4;
  tail_fixup_part(p.part, xcd * kTailSlotsPerXcd + t * x.s, x.s, part, [&](int i, int q, float4 a0, float4 a1) {
    const float v0[4] = {a0.x, a0.y, a0.z, a0.w}, v1[4] = {a1.x, a1.y, a1.z, a1.w};
    const int c0 = n0 + wn * 64 + (lane & 31);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = row0 + wm * 128 + i * 32 + 8 * q + 4 * (lane >> 5) + u;
      if (row >= row_end) continue;
      if (c0 < p.N) out[static_cast<size_t>(row) * p.ldc + c0] = v0[u];
      if (c0 + 32 < p.N) out[static_cast<size_t>(row) * p.ldc + c0 + 32] = v1[u];
    }
  });
}

// dx[t, c] = sum_k dXr[inv[t K + k], c] + sum_s dXr[T K + s T + t, c], in that order.
__global__ __launch_bounds__(kBwdThreads) void dx_combine_kernel(const float* __restrict__ dxr,
                                                                 const int32_t* __restrict__ inv, int T, int K, int S,
                                                                 int d, float* __restrict__ dx) {
  const int t = blockIdx.x;
  for (int c = threadIdx.x * 4; c < d; c += kBwdThreads * 4) {
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int k = 0; k < K + S; ++k) {
      const size_t row = k < K ? static_cast<size_t>(inv[t * K + k]) : static_cast<size_t>(T) * K + (k - K) * T + t;
      const float4 v = *reinterpret_cast<const float4*>(dxr + row * d + c);
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
    *reinterpret_cast<float4*>(dx + static_cast<size_t>(t) * d + c) = s;
  }
}

// Zero the [M, N] gradient matrices of the groups that no row reached (offsets[g+1] ==
// offsets[g]). Grid (G, chunks); float4 stores; M N % 4 == 0.
__global__ __launch_bounds__(kBwdThreads) void zero_unused_kernel(const int32_t* __restrict__ offsets, int E,
                                                                  size_t mn, float* __restrict__ c,
                                                                  float* __restrict__ cs) {
  const int g = blockIdx.x;
  if (offsets[g + 1] > offsets[g]) return;
  float4* dst = reinterpret_cast<float4*>(g < E ? c + g * mn : cs + (g - E) * mn);
  const size_t n4 = mn / 4;
  for (size_t i = static_cast<size_t>(blockIdx.y) * kBwdThreads + threadIdx.x; i < n4;
       i += static_cast<size_t>(gridDim.y) * kBwdThreads)
    dst[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

#define MASKMOE_TRY(x)               \
  do {                               \
    const hipError_t e_ = (x);       \
    if (e_ != hipSuccess) return e_; \
  } while (0)

// A second stream per device (default priority, created on first use and kept until the
// process ends) on which the backward writes the zero gradients of unchosen experts while the
// GEMMs run on the caller's stream. Ordered with the caller's stream by two events created per
// call.
constexpr int kMaxDevices = 64;
hipError_t side_stream(hipStream_t* out) {
  static std::mutex mu;
  static hipStream_t streams[kMaxDevices] = {};
  int dev = 0;
  MASKMOE_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!streams[dev]) MASKMOE_TRY(hipStreamCreateWithFlags(&streams[dev], hipStreamNonBlocking));
  *out = streams[dev];
  return hipSuccess;
}

}  // namespace

BwdLayout backward_layout(int T, int d, int F, int E, int K, int S) {
  BwdLayout w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) / 256 * 256;
    return o;
  };
  (void)E;
  const size_t R = static_cast<size_t>(T) * (K + S);
  w.dout = take(R * d * 2);
  w.dab = take(R * 2 * F * 2);
  w.dxr = take(R * d * 4);
  w.xg = take(R * d * 2);
  w.part = take(kTailPartBytes);
  w.total = off;
  return w;
}

// The ROWS grid: 8 XCDs x (their largest share of the tiles + tail slices).
static dim3 rows_grid(int mt_max, int n_tiles) {
  return dim3(static_cast<unsigned>(8 * ((static_cast<long>(mt_max) * n_tiles + 7) / 8 + kTailSlotsPerXcd)));
}

// The zero gradients of the experts no token chose depend on nothing but the routing; they are
// written on a second stream beside the GEMMs, forked after the row gathers: the fill is bound
// by HBM writes like the gathers, and next to them it slowed both (gathers 0.08 -> 0.66 ms on
// the Mixtral fine-tuning layer).
hipError_t launch_layer_backward(const BwdArgs& a, hipStream_t s) {
  const int G = a.E + a.S, T = a.T, d = a.d, F = a.F, K = a.K;
  const int R = T * (K + a.S);
  const size_t FD = static_cast<size_t>(F) * d;
  const BwdLayout& w = a.lay;
  char* ws = static_cast<char*>(a.workspace);
  uint16_t* dout = reinterpret_cast<uint16_t*>(ws + w.dout);
  uint16_t* dab = reinterpret_cast<uint16_t*>(ws + w.dab);
  float* dxr = reinterpret_cast<float*>(ws + w.dxr);
  uint16_t* xg = reinterpret_cast<uint16_t*>(ws + w.xg);

  hipStream_t side;
  MASKMOE_TRY(side_stream(&side));
  hipEvent_t fork, join;
  MASKMOE_TRY(hipEventCreateWithFlags(&fork, hipEventDisableTiming));
  hipError_t e = hipEventCreateWithFlags(&join, hipEventDisableTiming);
  if (e != hipSuccess) {
    (void)hipEventDestroy(fork);
    return e;
  }
  bool forked = false;
  auto fill = [&]() {   // fork the zero fill off the caller's stream
    if (e == hipSuccess) e = hipEventRecord(fork, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(side, fork, 0);
    if (e != hipSuccess) return;
    hipLaunchKernelGGL(zero_unused_kernel, dim3(G, 512), dim3(kBwdThreads), 0, side, a.pb.offsets, a.E, FD,
                       a.d_w_down, a.d_ws_down);
    hipLaunchKernelGGL(zero_unused_kernel, dim3(G, 512), dim3(kBwdThreads), 0, side, a.pb.offsets, a.E, 2 * FD,
                       a.d_w_gate_up, a.d_ws_gate_up);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipEventRecord(join, side);
    forked = e == hipSuccess;
  };
  auto check = [&]() {
    if (e == hipSuccess) e = hipGetLastError();
  };

  // dO and the gathered tokens
  hipLaunchKernelGGL(build_dout_kernel, dim3(R), dim3(kBwdThreads), 0, s, a.dy, a.gate, a.pb.perm, a.pb.row_tok, T * K,
                     d, dout);
  hipLaunchKernelGGL(gather_rows_kernel, dim3(R), dim3(kBwdThreads), 0, s, a.x, a.pb.row_tok, d, xg);
  check();
  fill();
  // dgrad of the down projection with the SwiGLU backward: [da db] (bf16)
  NtArgs n{};
  n.offsets = a.pb.offsets;
  n.tile_off = a.pb.tile_off;
  n.G = G; n.E = a.E;
  n.mt_max = a.max_tiles;
  n.a = dout; n.lda = d;
  n.b = a.w_down; n.bs = a.ws_down; n.N = F; n.K = d; n.ldb = F;   // W_down [d, F]: K-major
  n.ab = a.ab;
  n.c = dab;
  n.n_tiles = (F + kTileN - 1) / kTileN;
  n.cu_xcd = device_cus_per_xcd();
  n.part = reinterpret_cast<float*>(ws + w.part);
  if (e == hipSuccess) {
    hipLaunchKernelGGL((gemm_nt_kernel<kNtRows, kEpiSwigluBwd>), rows_grid(n.mt_max, n.n_tiles), dim3(kTileThreads),
                       0, s, n);
    check();
  }
  // dgrad of gate/up: dX rows = [da db] W_gate_up, then the token sums
  if (e == hipSuccess) {
    n.a = dab; n.lda = 2 * F;
    n.b = a.w_gate_up; n.bs = a.ws_gate_up; n.N = d; n.K = 2 * F; n.ldb = d;   // W_gate_up [2F, d]: K-major
    n.ab = nullptr;
    n.c = dxr; n.ldc = d;
    n.n_tiles = (d + kTileN - 1) / kTileN;
    hipLaunchKernelGGL((gemm_nt_kernel<kNtRows, kEpiF32>), rows_grid(n.mt_max, n.n_tiles), dim3(kTileThreads), 0, s,
                       n);
    if (nt_tail_split(kNtRows, kEpiF32, n.K / kTileK))
      hipLaunchKernelGGL(nt_tail_fixup, dim3(8 * kTailSlotsPerXcd * kTailFixParts), dim3(kTileThreads), 0, s, n);
    hipLaunchKernelGGL(dx_combine_kernel, dim3(T), dim3(kBwdThreads), 0, s, dxr, a.pb.inv, T, K, a.S, d, a.d_x);
    check();
  }
  // weight gradients over each expert's own rows
  NtArgs m{};
  m.offsets = a.pb.offsets;
  m.active = a.pb.active;
  m.n_active = a.pb.n_active;
  m.G = G; m.E = a.E;
  if (e == hipSuccess) {   // dW_down [d, F] = dO^T h
    m.a = dout; m.lda = d; m.b = a.h; m.ldb = F; m.M = d; m.N = F;
    m.c = a.d_w_down; m.cs = a.d_ws_down;
    m.mt_max = (d + kTileM - 1) / kTileM;
    m.n_tiles = (F + kTileN - 1) / kTileN;
    hipLaunchKernelGGL((gemm_nt_kernel<kNtKSplit, kEpiF32>), dim3(G * m.mt_max * m.n_tiles), dim3(kTileThreads), 0, s,
                       m);
    check();
  }
  if (e == hipSuccess) {   // dW_gate_up [2F, d] = [da db]^T x
    m.a = dab; m.lda = 2 * F; m.b = xg; m.ldb = d; m.M = 2 * F; m.N = d;
    m.c = a.d_w_gate_up; m.cs = a.d_ws_gate_up;
    m.mt_max = (2 * F + kTileM - 1) / kTileM;
    m.n_tiles = (d + kTileN - 1) / kTileN;
    hipLaunchKernelGGL((gemm_nt_kernel<kNtKSplit, kEpiF32>), dim3(G * m.mt_max * m.n_tiles), dim3(kTileThreads), 0, s,
                       m);
    check();
  }
  if (forked) {   // the caller's stream sees the fill done
    const hipError_t je = hipStreamWaitEvent(s, join, 0);
    if (e == hipSuccess) e = je;
  }
  (void)hipEventDestroy(fork);   // released once their waits are done
  (void)hipEventDestroy(join);
  return e;
}

}  // namespace maskmoe
