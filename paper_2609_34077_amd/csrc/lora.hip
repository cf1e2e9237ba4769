// Low-rank adapters of the experts (Stage 2 of the fine-tuning, Section 3.2; rank 8, alpha 16
// in Appendix B; routed and shared experts): an adapted projection computes
// W x + s B (A x), s = alpha / r, for the gate, up and down projections of every expert.
//
// The adapter term rides in the expert GEMMs as one more 64-wide k-tile (gemm_tile.hpp):
// A' = [U | rows] with U = rows A^T (r or 2r values, zero-padded to 64, bf16) and
// B' = [s B | W] (the matching s B row, zero-padded, bf16). For gate/up, U holds A_gate x in
// columns 0..r-1 and A_up x in r..2r-1, and a gate row of B' carries s B_gate in columns
// 0..r-1, an up row s B_up in r..2r-1, so the two adapters stay apart in one product.
// lora_pack_kernel builds B'; lora_down_kernel computes U (gate/up: from the gathered token
// rows) and V = h A_down^T (down: from the SwiGLU rows) with v_mfma_f32_16x16x32_bf16,
// 16 rows per workgroup, per expert group.

#include "common.hpp"
#include "kernels.hpp"

namespace maskmoe {
namespace {

constexpr int kLoraThreads = 256;

// B' rows: [G, rows, 64] from b [G, rows, r] (shared groups from bs), scaled by s and padded;
// one thread per 8 columns of a row (one 16-byte store).
// gate_up (UPSPLIT): rows < F carry columns 0..r-1, rows >= F columns r..2r-1.
template <bool UPSPLIT>
__global__ __launch_bounds__(kLoraThreads) void lora_pack_kernel(const uint16_t* __restrict__ b,
                                                                 const uint16_t* __restrict__ bs, int E, int rows,
                                                                 int F, int r, float s, uint16_t* __restrict__ out) {
  const int g = blockIdx.y;
  const uint16_t* src = g < E ? b + static_cast<size_t>(g) * rows * r : bs + static_cast<size_t>(g - E) * rows * r;
  u32x4* dst = reinterpret_cast<u32x4*>(out + static_cast<size_t>(g) * rows * 64);
  const int n = rows * 8;
  for (int i = blockIdx.x * kLoraThreads + threadIdx.x; i < n; i += gridDim.x * kLoraThreads) {
    const int row = i >> 3, c8 = (i & 7) * 8;
    const int c0 = (UPSPLIT && row >= F) ? r : 0;   // first column of this row's adapter
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t pair = 0;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = c8 + 2 * j + h;
        float v = 0.0f;
        if (c >= c0 && c < c0 + r) v = s * bf16_to_f32(src[static_cast<size_t>(row) * r + (c - c0)]);
        pair |= static_cast<uint32_t>(f32_to_bf16(v)) << (16 * h);
      }
      w[j] = pair;
    }
    dst[i] = u32x4{w[0], w[1], w[2], w[3]};
  }
}

// out[row, 0..63] = bf16(src_row . A_g[q]) for q < nq (A_g the [nq, K] adapter matrix of the
// row's group), 0 for q >= nq. One workgroup per 16 rows of a group (16 per 256-row tile of the
// permutation); its 4 wavefronts take contiguous quarters of K, 8 k-steps of loads in flight,
// and their partial sums are added in LDS in wave order.
constexpr int kLoraRows = 16, kLoraWaves = kLoraThreads / 64, kLoraUnroll = 8;
__global__ __launch_bounds__(kLoraThreads) void lora_down_kernel(const uint16_t* __restrict__ src,
                                                                 const int32_t* __restrict__ row_tok, int K,
                                                                 const uint16_t* __restrict__ a,
                                                                 const uint16_t* __restrict__ as, int nq, int G, int E,
                                                                 const int32_t* __restrict__ offsets,
                                                                 const int32_t* __restrict__ tile_off,
                                                                 uint16_t* __restrict__ out) {
  __shared__ float part[kLoraWaves][kLoraRows][32];
  constexpr int kSub = kGemmBM / kLoraRows;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int mt = blockIdx.x / kSub, sub = blockIdx.x % kSub;
  if (mt >= tile_off[G]) return;
  int lo = 0, hi = G;   // tile_off[lo] <= mt < tile_off[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tile_off[mid] <= mt) lo = mid; else hi = mid;
  }
  const int g = lo;
  const int row0 = offsets[g] + (mt - tile_off[g]) * kGemmBM + sub * kLoraRows;
  const int row_end = offsets[g + 1];
  if (row0 >= row_end) return;   // the whole workgroup leaves together
  const int rr = min(row0 + (lane & 15), row_end - 1);
  const uint16_t* xrow = src + static_cast<size_t>(row_tok ? row_tok[rr] : rr) * K + (lane >> 4) * 8;
  const uint16_t* la = g < E ? a + static_cast<size_t>(g) * nq * K : as + static_cast<size_t>(g - E) * nq * K;
  const int n0 = lane & 15, n1 = n0 + 16;
  const uint16_t* b0 = la + static_cast<size_t>(min(n0, nq - 1)) * K + (lane >> 4) * 8;
  const uint16_t* b1 = la + static_cast<size_t>(min(n1, nq - 1)) * K + (lane >> 4) * 8;
  const bool two = nq > 16, has0 = n0 < nq, has1 = n1 < nq;
  const u32x4 zero = {0u, 0u, 0u, 0u};
  f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  const int steps = K / 32, per = (steps + kLoraWaves - 1) / kLoraWaves;
  const int s0 = min(wave * per, steps), s1 = min(s0 + per, steps);
  int s = s0;
  for (; s + kLoraUnroll <= s1; s += kLoraUnroll) {   // all loads of kLoraUnroll k-steps first
    u32x4 av[kLoraUnroll], bv0[kLoraUnroll], bv1[kLoraUnroll];
#pragma unroll
    for (int u = 0; u < kLoraUnroll; ++u) {
      const int k = (s + u) * 32;
      av[u] = *reinterpret_cast<const u32x4*>(xrow + k);
      bv0[u] = has0 ? *reinterpret_cast<const u32x4*>(b0 + k) : zero;
      bv1[u] = has1 ? *reinterpret_cast<const u32x4*>(b1 + k) : zero;
    }
#pragma unroll
    for (int u = 0; u < kLoraUnroll; ++u) {
      acc0 = mfma_16x16x32(av[u], bv0[u], acc0);
      if (two) acc1 = mfma_16x16x32(av[u], bv1[u], acc1);
    }
  }
  for (; s < s1; ++s) {
    const int k = s * 32;
    const u32x4 av = *reinterpret_cast<const u32x4*>(xrow + k);
    acc0 = mfma_16x16x32(av, has0 ? *reinterpret_cast<const u32x4*>(b0 + k) : zero, acc0);
    if (two) acc1 = mfma_16x16x32(av, has1 ? *reinterpret_cast<const u32x4*>(b1 + k) : zero, acc1);
  }
  // acc[i] is row 4 (lane >> 4) + i, column lane & 15 (second tile: + 16)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    part[wave][4 * (lane >> 4) + i][n0] = acc0[i];
    part[wave][4 * (lane >> 4) + i][n1] = acc1[i];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < kLoraRows * 64; e += kLoraThreads) {
    const int r = e / 64, c = e % 64, row = row0 + r;
    if (row >= row_end) continue;
    float v = 0.0f;
    if (c < 32) {
#pragma unroll
      for (int w = 0; w < kLoraWaves; ++w) v += part[w][r][c];
    }
    out[static_cast<size_t>(row) * 64 + c] = f32_to_bf16(v);
  }
}

}  // namespace

hipError_t launch_lora_pack(const LoraArgs& l, int G, int E, int F, int d, hipStream_t stream) {
  hipLaunchKernelGGL(lora_pack_kernel<true>, dim3(256, G), dim3(kLoraThreads), 0, stream, l.b_gate_up, l.bs_gate_up,
                     E, 2 * F, F, l.rank, l.scale, l.bp_gate_up);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(lora_pack_kernel<false>, dim3(256, G), dim3(kLoraThreads), 0, stream, l.b_down, l.bs_down, E, d,
                     F, l.rank, l.scale, l.bp_down);
  return hipGetLastError();
}

hipError_t launch_lora_down(const uint16_t* src, const int32_t* row_tok, int K, const uint16_t* a, const uint16_t* as,
                            int nq, int G, int E, const PermBuffers& pb, int max_tiles, uint16_t* out,
                            hipStream_t stream) {
  hipLaunchKernelGGL(lora_down_kernel, dim3((kGemmBM / kLoraRows) * max_tiles), dim3(kLoraThreads), 0, stream, src,
                     row_tok, K, a, as, nq, G, E, pb.offsets, pb.tile_off, out);
  return hipGetLastError();
}

}  // namespace maskmoe
