// Router logits + softmax + hard-mask / soft-prior Top-K + gates, fused in one kernel.
//
// Section 3.1 (Eq. 1): z = W x, p = softmax(z), A = Top-K(p), gates g_i = p_i or
// p_i / sum_{j in A} p_j. Section 3.2, Stage 1 (Eq. 2): A = Top-K(p * m) with a binary
// mask m; the gates computed from p * m equal those of p on A. Section 3.2, inference
// (Eq. 4): A = Top-K(p * pi) with a prior pi > 0; gates stay those of p.
//
// Experts are ranked on log-domain keys z_i + c_i, with c_i = 0 (plain), 0 or -inf
// (mask), log pi_i (prior); softmax is monotone with a shared normaliser, so these order
// experts exactly as the products do and avoid ties from exp underflow. Equal keys go to
// the lower expert index.
//
// bf16 logits use v_mfma_f32_16x16x32_bf16 (route_bf16_kernel): a workgroup computes a tile of
// (16*MB tokens) x (16*NB*WN outputs), where outputs are the rows of [L*E, d] router
// weights of whole layers; its WN*WK waves split the outputs (WN) and the k-steps (WK)
// and the WK partial tiles are summed in LDS in a fixed order. Small token counts
// (decode) use WK = 8..16 so all of d is in flight at once; large token counts stream x.
// Many tokens routed through many layers at once use route_gemm_kernel instead, which stages
// both operands through LDS.
// The selection runs one thread per (token, layer) on the fp32 logits in LDS.

#include <limits.h>
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"
#include "permute_block.hpp"

namespace maskmoe {
namespace {

constexpr int kMaxK = 16;
constexpr int kMaxModeParams = 512;
// Selection by one thread per (token, layer) pair up to this many experts, by one wavefront
// (a lane per expert) above it when E <= 64. The softmax normaliser over all E experts (g = p)
// is summed in expert order for E <= kSelThreadE and E > 64; for kSelThreadE < E <= 64 in the
// order of a 64-lane butterfly: lane e with lane e ^ 32, then ^ 16, ..., ^ 1, experts past E
// counting as 0. The wavefront selection sums that way in six steps (a serial sum over the
// lanes took ~5 us of the 4096-token selection kernel), the per-thread selection replays the
// same tree, so every path gives the same bits.
constexpr int kSelThreadE = 16;
// The LDS-tiled router GEMM (route_gemm_kernel) pays off once a launch has many tokens and
// enough router outputs to fill its 256-wide tile.
constexpr int kRouteGemmMinT = 1024;
constexpr int kRouteGemmMinOutputs = 128;

struct RouteParams {
  const void* x;
  const void* w;       // [L, E, d] router weights of this launch's first layer
  int32_t* idx;        // [L, T, K]
  float* gate;         // [L, T, K]
  float* margin;       // [L, T] or null
  float* logits;       // [L, T, E] fp32 router logits or null
  int T, d, E, K, L, lpw, mode, gate_mode;
  PermBuffers pb;               // fused permutation (single-workgroup launches only)
  int n_shared, tile_rows;
  float modep[kMaxModeParams];  // [L, E]: mask (0/1) or prior values of this launch
};

__device__ __forceinline__ float key_offset(int mode, float v) {
  if (mode == 1) return v != 0.0f ? 0.0f : -INFINITY;  // hard mask
  if (mode == 2) return logf(v);                        // soft prior
  return 0.0f;                                          // plain
}

// Selection, gates and outputs of one (token, layer) pair: z the E fp32 logits, o the E key
// offsets, obase the pair's index in the [L, T] outputs. write_logits: also store z in p.logits.
// EC: the expert count when known at compile time (0: p.E); the arithmetic is the same.
template <int EC = 0>
__device__ __forceinline__ void select_pair(const RouteParams& p, const float* z, const float* o, size_t obase,
                                            bool write_logits) {
  const int E = EC ? EC : p.E, K = p.K;
  uint64_t tk0 = 0, tk1 = 0, tk2 = 0, tk3 = 0;
  int sel[kMaxK];
  float selz[kMaxK];
  float kth = -INFINITY, nxt = -INFINITY;
#pragma unroll
  for (int j = 0; j <= kMaxK; ++j) {
    if (j <= K) {
      float best = -INFINITY;
      int bi = -1;
      for (int e = 0; e < E; ++e) {
        const uint64_t word = e < 64 ? tk0 : e < 128 ? tk1 : e < 192 ? tk2 : tk3;
        if ((word >> (e & 63)) & 1ull) continue;
        const float key = z[e] + o[e];
        if (key > best) {
          best = key;
          bi = e;
        }
      }
      if (j < K) {
        if (bi < 0) {  // only reachable with non-finite logits: keep the output well formed
          for (int e = 0; e < E && bi < 0; ++e) {
            const uint64_t word = e < 64 ? tk0 : e < 128 ? tk1 : e < 192 ? tk2 : tk3;
            if (!((word >> (e & 63)) & 1ull)) bi = e;
          }
        }
        const uint64_t bit = 1ull << (bi & 63);
        if (bi < 64) tk0 |= bit; else if (bi < 128) tk1 |= bit; else if (bi < 192) tk2 |= bit; else tk3 |= bit;
        sel[j] = bi;
        selz[j] = z[bi];
        kth = best;
      } else {
        nxt = best;
      }
    }
  }

  float zref, norm = 0.0f;
  if (p.gate_mode == 0) {  // g = p_i: full softmax over all E experts
    zref = z[0];
    for (int e = 1; e < E; ++e) zref = fmaxf(zref, z[e]);
    if (E > kSelThreadE && E <= kWave) {   // the butterfly's tree (kSelThreadE)
      float a[kWave / 2];
#pragma unroll
      for (int i = 0; i < kWave / 2; ++i)
        a[i] = (i < E ? expf(z[i] - zref) : 0.0f) + (i + kWave / 2 < E ? expf(z[i + kWave / 2] - zref) : 0.0f);
#pragma unroll
      for (int w = kWave / 4; w >= 1; w >>= 1)
#pragma unroll
        for (int i = 0; i < w; ++i) a[i] = a[i] + a[i + w];
      norm = a[0];
    } else {
      for (int e = 0; e < E; ++e) norm += expf(z[e] - zref);
    }
  } else {  // g = p_i / sum_{j in A} p_j
    zref = selz[0];
#pragma unroll
    for (int j = 1; j < kMaxK; ++j)
      if (j < K) zref = fmaxf(zref, selz[j]);
#pragma unroll
    for (int j = 0; j < kMaxK; ++j)
      if (j < K) norm += expf(selz[j] - zref);
  }
  const float inv = 1.0f / norm;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < K) {
      p.idx[obase * K + j] = sel[j];
      p.gate[obase * K + j] = expf(selz[j] - zref) * inv;
    }
  }
  if (p.margin) p.margin[obase] = (nxt == -INFINITY) ? INFINITY : (kth - nxt);
  if (write_logits && p.logits)
    for (int e = 0; e < E; ++e) p.logits[obase * E + e] = z[e];
}

// Selection and gates for every (token, layer) pair of the tile. logits[tt * ld + lw*E + e]
// are the fp32 router logits, lo[lw*E + e] the key offsets. TOKEN_FASTEST: consecutive threads
// take consecutive tokens of one layer (conflict-free LDS reads when ld is odd, coalesced
// stores); otherwise consecutive layers of one token.
template <bool TOKEN_FASTEST = false>
__device__ void route_finalize(const RouteParams& p, const float* logits, int ld, const float* lo,
                               int t0, int TT, int lg0, int nl, int nthreads) {
  const int E = p.E;
  for (int pi = threadIdx.x; pi < TT * nl; pi += nthreads) {
    const int tt = TOKEN_FASTEST ? pi % TT : pi / nl;
    const int lw = TOKEN_FASTEST ? pi / TT : pi - tt * nl;
    const int t = t0 + tt;
    if (t >= p.T) continue;
    const float* z = logits + tt * ld + lw * E;
    const float* o = lo + lw * E;
    const size_t obase = (static_cast<size_t>(lg0 + lw) * p.T + t);

    select_pair(p, z, o, obase, true);
  }
}

// Split routing: the logits of every (token, layer) pair are first written to p.logits
// ([L, T, E] fp32, the caller's output or workspace) by the logit kernels, then selected here at
// full occupancy (the selection otherwise runs after the logit GEMM at the GEMM's occupancy).
// Pairs are taken token-fastest: pair q is (layer q / T, token q % T), its logits at q * E.
constexpr int kSelThreads = 256;

// E <= kSelThreadE: one thread per pair, the block's logits staged in LDS (odd row stride) so
// the per-pair selection reads them without bank conflicts.
template <int EC>
__global__ __launch_bounds__(kSelThreads) void route_select_kernel(const RouteParams p) {
  constexpr int EMAX = EC ? EC : kSelThreadE;
  __shared__ float zs[kSelThreads * (EMAX + 1)];
  __shared__ float lo[kMaxModeParams];
  const int E = EC ? EC : p.E;
  const uint32_t pairs = static_cast<uint32_t>(p.L) * p.T;   // < 2^31
  const uint32_t q0 = blockIdx.x * kSelThreads;
  for (int i = threadIdx.x; i < p.L * E; i += kSelThreads) lo[i] = key_offset(p.mode, p.modep[i]);
  const int rows = pairs - q0 < kSelThreads ? static_cast<int>(pairs - q0) : kSelThreads;
  const float* src = p.logits + static_cast<size_t>(q0) * E;
  if ((E & 3) == 0) {   // 16-byte loads; a 4-float unit never straddles two rows
    for (int i = threadIdx.x; i < rows * E / 4; i += kSelThreads) {
      const f32x4 v = reinterpret_cast<const f32x4*>(src)[i];
      const int r = (4 * i) / E, c = 4 * i - r * E;
      float* d = zs + r * (E + 1) + c;
      d[0] = v[0];
      d[1] = v[1];
      d[2] = v[2];
      d[3] = v[3];
    }
  } else {
    for (int i = threadIdx.x; i < rows * E; i += kSelThreads) {
      const int r = i / E;
      zs[r * (E + 1) + i - r * E] = src[i];
    }
  }
  __syncthreads();
  const uint32_t q = q0 + threadIdx.x;
  if (q >= pairs) return;
  const int l = static_cast<int>(q / static_cast<uint32_t>(p.T));
  select_pair<EC>(p, zs + threadIdx.x * (E + 1), lo + l * E, q, false);
}

// Lane exchanges within a 16-lane row (DPP): lane e of the row receives lane (e - R) mod 16.
template <int R>
__device__ __forceinline__ int row_ror(int v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x120 + R, 0xF, 0xF, false);
}

// Adds to `rank` the number of the row's keys src_key (of experts src_idx, one per lane,
// rotated by R .. 15 lanes within the row; R = 0 is the lane's own source) that rank above
// (key, idx): valid (above -inf, not NaN) and larger, or equal with a lower index. Branch-free.
template <int R>
__device__ __forceinline__ void rank_from_row(float src_key, int src_idx, float key, int idx, int& rank) {
  if constexpr (R < 16) {
    const float kf = R == 0 ? src_key : __int_as_float(row_ror<R == 0 ? 1 : R>(__float_as_int(src_key)));
    const int f = R == 0 ? src_idx : row_ror<R == 0 ? 1 : R>(src_idx);
    rank += static_cast<int>(kf > -INFINITY) &
            (static_cast<int>(kf > key) | (static_cast<int>(kf == key) & static_cast<int>(f < idx)));
    rank_from_row<R + 1>(src_key, src_idx, key, idx, rank);
  }
}

// One (token, layer) pair on one wavefront, lane e holding expert e (E <= 64): z its logit,
// key its log-domain key (z + offset). Each expert's rank (the number of valid keys larger, or
// equal with a lower index; -inf and NaN keys are not valid) is its position in the successive
// picks of select_pair, so both give the same selection, margin and gate bits (the normalisers
// are summed in the same order). Writes the pair's outputs at obase; returns, in lanes j < K,
// pick j.
__device__ __forceinline__ int wave_select_pair(const RouteParams& p, float z, float key, bool in, size_t obase) {
  const int lane = threadIdx.x & 63;
  const int E = p.E, K = p.K;
  const bool valid = in && key > -INFINITY;   // false for NaN too
  // rank over the 64 lanes (lanes past E hold -inf): the lane's own row by DPP rotations, the
  // other three rows through one lane exchange each
  int rank = 0;
  rank_from_row<1>(key, lane, key, lane, rank);
#pragma unroll
  for (int ro = 16; ro < 64; ro += 16) rank_from_row<0>(__shfl_xor(key, ro, kWave), lane ^ ro, key, lane, rank);
  const uint64_t vmask = __ballot(valid);
  const int n_valid = __popcll(vmask);
  // picks in order: valid experts by rank, then (fewer than K valid keys) the lowest others
  uint64_t taken = 0;
  int my_sel = 0;
  float my_selz = 0.0f, kth = -INFINITY, nxt = -INFINITY;
  for (int j = 0; j < K; ++j) {
    int e;
    if (j < n_valid) {
      e = __ffsll(static_cast<unsigned long long>(__ballot(valid && rank == j))) - 1;
      kth = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(key), e));
    } else {
      e = __ffsll(static_cast<unsigned long long>(~taken & (E == 64 ? ~0ull : ((1ull << E) - 1)))) - 1;
      kth = -INFINITY;
    }
    taken |= 1ull << e;
    const float ze = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(z), e));
    if (lane == j) {
      my_sel = e;
      my_selz = ze;
    }
  }
  if (K < n_valid) {
    const int e = __ffsll(static_cast<unsigned long long>(__ballot(valid && rank == K))) - 1;
    nxt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(key), e));
  }
  float zref, norm = 0.0f;
  if (p.gate_mode == 0) {   // softmax over all E
    // the largest logit: fmaxf drops NaN operands (lanes past E hold NaN), so the reduction
    // order does not change the value (the largest non-NaN logit, NaN if all are NaN)
    zref = in ? z : __builtin_nanf("");
#pragma unroll
    for (int m = kWave / 2; m >= 1; m >>= 1) zref = fmaxf(zref, __shfl_xor(zref, m, kWave));
    float ex = in ? expf(z - zref) : 0.0f;
    if (E > kSelThreadE) {   // the butterfly's tree (kSelThreadE)
#pragma unroll
      for (int m = kWave / 2; m >= 1; m >>= 1) ex += __shfl_xor(ex, m, kWave);
      norm = ex;
    } else {   // expert order, as the per-thread selection for E <= kSelThreadE
      for (int e = 0; e < E; ++e) norm += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ex), e));
    }
  } else {   // renormalised over the picks, in pick order
    zref = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_selz), 0));
    for (int j = 1; j < K; ++j) zref = fmaxf(zref, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_selz), j)));
    for (int j = 0; j < K; ++j)
      norm += expf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_selz), j)) - zref);
  }
  const float inv = 1.0f / norm;
  if (lane < K) {
    p.idx[obase * K + lane] = my_sel;
    p.gate[obase * K + lane] = expf(my_selz - zref) * inv;
  }
  if (lane == 0 && p.margin) p.margin[obase] = (nxt == -INFINITY) ? INFINITY : (kth - nxt);
  return my_sel;
}

// kSelThreadE < E <= 64: one wavefront per pair (wave_select_pair).
__global__ __launch_bounds__(kSelThreads) void route_select_wave_kernel(const RouteParams p) {
  const int lane = threadIdx.x & 63;
  const int E = p.E, T = p.T;
  const uint32_t q = blockIdx.x * (kSelThreads / 64) + (threadIdx.x >> 6);
  if (q >= static_cast<uint32_t>(p.L) * T) return;   // the whole wavefront leaves (L * T < 2^31)
  const int l = static_cast<int>(q / static_cast<uint32_t>(T));
  const bool in = lane < E;
  const float z = in ? p.logits[static_cast<size_t>(q) * E + lane] : 0.0f;
  const float key = in ? z + key_offset(p.mode, p.modep[l * E + lane]) : -INFINITY;
  wave_select_pair(p, z, key, in, q);
}

// The same selection and gates for the single-workgroup launch (one layer, tokens 0..T-1), one
// wavefront per token: lane e holds the keys of experts e, e + 64, ...; each of the K + 1 picks
// is a wave reduction (largest key, then lowest index), and the softmax normaliser is summed in
// expert order (selection order for the renormalised rule), as in route_finalize, so both give
// the same bits. The selections are also left in sel_lds [T, K] for the permutation.
__device__ void route_finalize_wave(const RouteParams& p, const float* logits, int ld, const float* lo, int TT,
                                    int32_t* sel_lds, int nwaves) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int E = p.E, K = p.K;
  if (E <= 64) {   // one expert per lane: rank-based picks, no cross-lane reductions
    for (int t = wave; t < TT && t < p.T; t += nwaves) {
      const bool in = lane < E;
      const float z = in ? logits[t * ld + lane] : 0.0f;
      const float key = in ? z + lo[lane] : -INFINITY;
      const int my_sel = wave_select_pair(p, z, key, in, t);
      if (lane < K) sel_lds[t * K + lane] = my_sel;
      if (p.logits && in) p.logits[static_cast<size_t>(t) * E + lane] = z;
    }
    return;
  }
  constexpr int Q = 4;   // experts per lane, E <= 256
  for (int t = wave; t < TT && t < p.T; t += nwaves) {
    const float* z = logits + t * ld;
    float key[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int e = lane + 64 * q;
      key[q] = e < E ? z[e] + lo[e] : -INFINITY;
    }
    uint32_t taken = 0;   // bit q: expert lane + 64 q is selected
    int my_sel = 0;
    float my_selz = 0.0f, kth = -INFINITY, nxt = -INFINITY;
    for (int j = 0; j <= K; ++j) {
      float bv = -INFINITY;
      int bi = -1;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int e = lane + 64 * q;
        if (e < E && !((taken >> q) & 1u) && key[q] > bv) {
          bv = key[q];
          bi = e;
        }
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        const float ov = __shfl_xor(bv, m, kWave);
        const int oi = __shfl_xor(bi, m, kWave);
        if (oi >= 0 && (bi < 0 || ov > bv || (ov == bv && oi < bi))) {
          bv = ov;
          bi = oi;
        }
      }
      if (j < K) {
        if (bi < 0) {   // only reachable with non-finite logits: the lowest expert not taken
          int lowest = INT_MAX;
#pragma unroll
          for (int q = 0; q < Q; ++q) {
            const int e = lane + 64 * q;
            if (e < E && !((taken >> q) & 1u)) lowest = min(lowest, e);
          }
          bi = wave_min_int(lowest);
        }
        if (lane == (bi & 63)) taken |= 1u << (bi >> 6);
        const float zb = z[bi];
        if (lane == j) {
          my_sel = bi;
          my_selz = zb;
        }
        kth = bv;
      } else {
        nxt = bv;
      }
    }
    float zref, norm = 0.0f;
    if (p.gate_mode == 0) {   // g = p_i: softmax over all E experts
      float m = -INFINITY;
#pragma unroll
      for (int q = 0; q < Q; ++q)
        if (lane + 64 * q < E) m = fmaxf(m, z[lane + 64 * q]);
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));
      zref = m;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const float ex = lane + 64 * q < E ? expf(z[lane + 64 * q] - zref) : 0.0f;
        const int n_q = min(64, E - 64 * q);
        for (int l = 0; l < n_q; ++l) norm += __shfl(ex, l, kWave);   // expert order
      }
    } else {   // g = p_i / sum_{j in A} p_j, in selection order
      zref = __shfl(my_selz, 0, kWave);
      for (int j = 1; j < K; ++j) zref = fmaxf(zref, __shfl(my_selz, j, kWave));
      for (int j = 0; j < K; ++j) norm += expf(__shfl(my_selz, j, kWave) - zref);
    }
    const float inv = 1.0f / norm;
    if (lane < K) {
      p.idx[static_cast<size_t>(t) * K + lane] = my_sel;
      p.gate[static_cast<size_t>(t) * K + lane] = expf(my_selz - zref) * inv;
      sel_lds[t * K + lane] = my_sel;
    }
    if (lane == 0 && p.margin) p.margin[t] = (nxt == -INFINITY) ? INFINITY : (kth - nxt);
    if (p.logits)
      for (int e = lane; e < E; e += 64) p.logits[static_cast<size_t>(t) * E + e] = z[e];
  }
}

// fmaxf over the 16 lanes of the row, in every lane. fmaxf drops NaN operands, so any order
// of the reduction gives the same value (the largest non-NaN, NaN if all are NaN).
__device__ __forceinline__ float row_max(float v) {
  v = fmaxf(v, __int_as_float(row_ror<8>(__float_as_int(v))));
  v = fmaxf(v, __int_as_float(row_ror<4>(__float_as_int(v))));
  v = fmaxf(v, __int_as_float(row_ror<2>(__float_as_int(v))));
  v = fmaxf(v, __int_as_float(row_ror<1>(__float_as_int(v))));
  return v;
}

// E <= 16 experts, the tokens of the single-workgroup launch (4 per wavefront, every wavefront
// calls this: it holds a barrier): token t is selected by 16-lane row t % 4 of wavefront t / 4,
// lane e of the row holding expert e. An expert's rank among the valid keys (larger, or equal
// with a lower index; -inf and NaN keys are not valid) is its position in select_pair's
// successive picks; with fewer than K valid keys the lowest other experts follow in index
// order. Each picked lane writes its own outputs. The maxima are order-free; the normalisers
// are summed through LDS (`sc`, [16 tokens][16]) in select_pair's order (picks for the
// renormalised rule, experts for the softmax), so both give the same bits. The picks are also
// left in sel_lds [T, K] for the permutation.
__device__ void route_select_rows(const RouteParams& p, const float* logits, int ld, const float* lo, float* sc,
                                  int32_t* sel_lds) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int E = p.E, K = p.K, rb = lane & 48, e = lane & 15;
  const int t = 4 * wave + (lane >> 4);
  const bool act = 4 * wave < p.T;   // wavefronts without tokens only take part in the barrier
  const bool live = t < p.T;         // p.T <= 16
  const bool in = live && e < E;
  const bool soft_all = p.gate_mode == 0;   // g = p_i (softmax over all E), else renormalised over the picks
  float z = 0.0f, key = -INFINITY, ex = 0.0f, zref = 0.0f, kth = -INFINITY, nxt = -INFINITY;
  int pos = 0;
  bool pick = false;
  if (act) {
    z = in ? logits[t * ld + e] : 0.0f;
    key = in ? z + lo[e] : -INFINITY;
    const bool valid = key > -INFINITY;   // false for NaN too
    int rank = 0;
    rank_from_row<1>(key, e, key, e, rank);
    const uint32_t vbits = static_cast<uint32_t>(__ballot(valid) >> rb) & 0xffffu;
    const uint32_t ibits = static_cast<uint32_t>(__ballot(in && !valid) >> rb) & 0xffffu;
    pos = valid ? rank : __popc(vbits) + __popc(ibits & ((1u << e) - 1u));
    pick = in && pos < K;
    kth = row_max(pick && valid && pos == K - 1 ? key : -INFINITY);
    nxt = row_max(valid && rank == K ? key : -INFINITY);
    const bool term = soft_all ? in : pick;
    zref = row_max(term ? z : __builtin_nanf(""));
    ex = expf(z - zref);
    if (term) sc[t * 16 + (soft_all ? e : pos)] = ex;
  }
  lds_sync();
  if (!act) return;
  float norm = 0.0f;
  const int nterms = soft_all ? E : K;
  if (live)
    for (int i = 0; i < nterms; ++i) norm += sc[t * 16 + i];
  const float inv = 1.0f / norm;
  if (pick) {
    p.idx[static_cast<size_t>(t) * K + pos] = e;
    p.gate[static_cast<size_t>(t) * K + pos] = ex * inv;
    sel_lds[t * K + pos] = e;
  }
  if (live && e == 0 && p.margin) p.margin[t] = (nxt == -INFINITY) ? INFINITY : (kth - nxt);
  if (in && p.logits) p.logits[static_cast<size_t>(t) * E + e] = z;
}

// FUSE: the grid is one workgroup holding every token of one layer; after the selection it
// also groups the (token, slot) pairs by expert (permute_wave for few entries, else
// permute_block).
// SPLIT (not with FUSE): the tile's logits go to p.logits and route_select_kernel selects.
// Kernel parameters not needed before the epilogue, read at the start so that their loads
// share the first memory round trip: the argument block is fetched from memory at each
// launch, and a parameter first read after the k-loop would cost a round trip of its own.
template <typename V>
__device__ __forceinline__ void load_now(V v) {
  asm volatile("" ::"s"(v));
}

template <int MB, int NB, int WN, int WK, bool FUSE, bool SPLIT = false>
__global__ __launch_bounds__(64 * WN * WK) void route_bf16_kernel(const RouteParams p) {
  constexpr int TT = 16 * MB, NO = 16 * NB * WN, NT = 64 * WN * WK;
  // FUSE with one 16-wide output tile: the E <= 16 key parameters of the single layer are
  // loaded as scalars with the others.
  constexpr bool kScalarModep = FUSE && NO <= 16;
  __shared__ float red[WK * TT * NO];
  __shared__ float lo[NO];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wn = wave % WN, wk = wave / WN;
  const int t0 = blockIdx.x * TT;
  const int lg0 = blockIdx.y * p.lpw;
  const int nl = min(p.lpw, p.L - lg0);
  const int nout = nl * p.E;
  const uint16_t* x = static_cast<const uint16_t*>(p.x);
  const uint16_t* w = static_cast<const uint16_t*>(p.w) + static_cast<size_t>(lg0) * p.E * p.d;
  const int ksteps = p.d >> 5;
  const int kg = (lane >> 4) * 8;
  float mp[16];
  if (FUSE) {
    load_now(p.idx); load_now(p.gate); load_now(p.logits);
    load_now(p.K); load_now(p.mode); load_now(p.gate_mode); load_now(p.n_shared); load_now(p.tile_rows);
    load_now(p.pb.offsets); load_now(p.pb.tile_off); load_now(p.pb.active); load_now(p.pb.n_active);
    load_now(p.pb.perm); load_now(p.pb.inv); load_now(p.pb.row_tok);
  }
  if (kScalarModep) {   // lg0 == 0; 16 <= kMaxModeParams
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      mp[i] = p.modep[i];
      load_now(mp[i]);
    }
  }

  // Rows past the last token / output are clamped onto valid rows and not loaded (zeros):
  // their results are never written, and MFMA rows and columns do not mix.
  const uint16_t* ap[MB];
  const uint16_t* bp[NB];
  bool arow[MB], brow[NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int t = min(t0 + mb * 16 + (lane & 15), p.T - 1);
    ap[mb] = x + static_cast<size_t>(t) * p.d + kg;
    arow[mb] = t0 + mb * 16 + (lane & 15) < p.T;
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int o = min((wn * NB + nb) * 16 + (lane & 15), nout - 1);
    bp[nb] = w + static_cast<size_t>(o) * p.d + kg;
    brow[nb] = (wn * NB + nb) * 16 + (lane & 15) < nout;
  }
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  f32x4 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // k-steps wk, wk+WK, ...; groups of U steps are loaded before any is multiplied. Each wave
  // accumulates its steps in increasing order on every path below.
  constexpr int U = (MB + NB) <= 2 ? 8 : 4;
  int s = wk;
  // Few tokens in the fused launch: their rows are read once into LDS (all lanes of a row
  // tile share them) and the A operands come from there, which halves the load instructions;
  // the first group's weight loads are issued before the rows are stored.
  constexpr bool kStageX = FUSE && NO <= 16 && MB == 1 && NB == 1;
  constexpr int kXsUnits = kStageX ? 2 * NT : 1;   // 16-byte units: 32 KB
  __shared__ u32x4 xs[kXsUnits];
  if (kStageX && p.T * p.d <= kXsUnits * 8) {
    const int units = p.T * p.d / 8;
    const int tr = lane & 15;   // token row of this lane's A operand (loaded when tr < T)
    u32x4 xr[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = threadIdx.x + i * NT;
      xr[i] = c < units ? reinterpret_cast<const u32x4*>(x)[c] : zero4;
    }
    u32x4 bv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int st = s + u * WK;
      bv[u] = brow[0] && st < ksteps ? *reinterpret_cast<const u32x4*>(bp[0] + (st << 5)) : zero4;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = threadIdx.x + i * NT;
      if (c < units) xs[c] = xr[i];
    }
    lds_sync();
    const u32x4* xa = xs + (tr * p.d + kg) / 8;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int st = s + u * WK;
      if (st < ksteps) acc[0][0] = mfma_16x16x32(arow[0] ? xa[st * 4] : zero4, bv[u], acc[0][0]);
    }
    for (s += U * WK; s < ksteps; s += WK) {
      const u32x4 b = brow[0] ? *reinterpret_cast<const u32x4*>(bp[0] + (s << 5)) : zero4;
      acc[0][0] = mfma_16x16x32(arow[0] ? xa[s * 4] : zero4, b, acc[0][0]);
    }
  }
  for (; s + (U - 1) * WK < ksteps; s += U * WK) {
    u32x4 av[U][MB], bv[U][NB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = (s + u * WK) << 5;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) av[u][mb] = arow[mb] ? *reinterpret_cast<const u32x4*>(ap[mb] + k) : zero4;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) bv[u][nb] = brow[nb] ? *reinterpret_cast<const u32x4*>(bp[nb] + k) : zero4;
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = mfma_16x16x32(av[u][mb], bv[u][nb], acc[mb][nb]);
  }
  for (; s < ksteps; s += WK) {
    const int k = s << 5;
    u32x4 av[MB], bv[NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) av[mb] = arow[mb] ? *reinterpret_cast<const u32x4*>(ap[mb] + k) : zero4;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) bv[nb] = brow[nb] ? *reinterpret_cast<const u32x4*>(bp[nb] + k) : zero4;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = mfma_16x16x32(av[mb], bv[nb], acc[mb][nb]);
  }

  float* r = red + wk * TT * NO;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        r[(mb * 16 + (lane >> 4) * 4 + i) * NO + (wn * NB + nb) * 16 + (lane & 15)] = acc[mb][nb][i];
  if (kScalarModep) {
    if (wave == 0) {   // lane i: expert i
      float v = mp[0];
#pragma unroll
      for (int i = 1; i < 16; ++i) v = lane == i ? mp[i] : v;
      if (lane < nout) lo[lane] = key_offset(p.mode, v);
    }
  } else {
    for (int i = threadIdx.x; i < nout; i += NT) lo[i] = key_offset(p.mode, p.modep[lg0 * p.E + i]);
  }
  lds_sync();
  if (WK > 1) {
    for (int i = threadIdx.x; i < TT * NO; i += NT) {
      float s = red[i];
#pragma unroll
      for (int q = 1; q < WK; ++q) s += red[q * TT * NO + i];
      red[i] = s;
    }
    lds_sync();
  }
  if (SPLIT) {   // [TT, nl * E] tile -> p.logits [L, T, E], consecutive threads on consecutive floats
    for (int i = threadIdx.x; i < TT * nout; i += NT) {
      const int lw = i / (TT * p.E), rem = i - lw * TT * p.E;
      const int tt = rem / p.E, e = rem - tt * p.E;
      if (t0 + tt < p.T)
        p.logits[(static_cast<size_t>(lg0 + lw) * p.T + t0 + tt) * p.E + e] = red[tt * NO + lw * p.E + e];
    }
  } else if (FUSE) {
    __shared__ PermLds plds;
    __shared__ int32_t sel_lds[kRouteOneBlockT * kMaxK];
    if (NO <= 16) {   // E <= 16
      static_assert(!FUSE || NO > 16 || (TT == 16 && NT >= 4 * 64), "four wavefronts of 4 rows hold the 16 tokens");
      __shared__ float sc[16 * 16];
      route_select_rows(p, red, NO, lo, sc, sel_lds);
    } else
      route_finalize_wave(p, red, NO, lo, TT, sel_lds, NT / 64);
    lds_sync();   // the selections left in sel_lds are read by other threads
    if (p.T * p.K <= kWave && p.E + p.n_shared < kWave) {
      if (wave == 0) permute_wave(sel_lds, p.T, p.K, p.E, p.n_shared, p.tile_rows, p.pb);
    } else {
      permute_block(sel_lds, p.T, p.K, p.E, p.n_shared, p.tile_rows, p.pb, plds, NT);
    }
  } else {
    route_finalize(p, red, NO, lo, t0, TT, lg0, nl, NT);
  }
}

// Many tokens and many router outputs (tens of layers routed from the same tokens): a
// 256-token x 256-output tile of whole layers, both operands staged through LDS in 64-wide
// k-steps (the same load pipeline and swizzle as the expert GEMM: every token row is read
// from HBM once, the router rows are shared by all workgroups through L2), accumulated on
// v_mfma_f32_32x32x16_bf16. After the k-loop the staging LDS holds the fp32 logits of one
// half of the tokens at a time, and the selection runs on them as in route_bf16_kernel.
constexpr int kRgBM = 256, kRgBN = 256, kRgBK = 64, kRgThreads = 512;

template <bool SPLIT>
__global__ __launch_bounds__(kRgThreads) void route_gemm_kernel(const RouteParams p) {
  constexpr int BM = kRgBM, BN = kRgBN, BK = kRgBK, NT = kRgThreads;
  constexpr int WN = 4;                        // waves: 2 along tokens x 4 along outputs
  constexpr int TM = 4, TN = 2;                // 32x32 fragments per wave: 128 tokens x 64 outputs
  constexpr int HALF = BM / 2;                 // token rows per selection phase (one wave row)
  constexpr int UA = BM * 8 / NT, UB = BN * 8 / NT;   // 16-byte units per thread and stage
  constexpr int SA = BM * 8, SB = BN * 8;             // 16-byte slots per stage
  constexpr int STAGING = 2 * (SA + SB) * 16;
  constexpr int LD = BN + 1;                   // logits row stride: odd, so token rows fall on distinct banks
  constexpr int LOGITS = HALF * LD * 4;
  __shared__ __attribute__((aligned(16))) unsigned char smem[STAGING > LOGITS ? STAGING : LOGITS];
  __shared__ float lo[BN];
  u32x4* lds_a = reinterpret_cast<u32x4*>(smem);   // [2][SA]
  u32x4* lds_b = lds_a + 2 * SA;                    // [2][SB]
  float* logits = reinterpret_cast<float*>(smem);   // [HALF][LD], after the k-loop

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int t0 = blockIdx.x * BM;
  const int lg0 = blockIdx.y * p.lpw;
  const int nl = min(p.lpw, p.L - lg0);
  const int nout = nl * p.E;
  const uint16_t* x = static_cast<const uint16_t*>(p.x);
  const uint16_t* w = static_cast<const uint16_t*>(p.w) + static_cast<size_t>(lg0) * p.E * p.d;

  // Thread tid loads rows (tid >> 3) + 64 i of each operand; rows past the last token or
  // output are clamped onto valid rows and their results never written.
  const int r0 = tid >> 3;
  const int chunk = ((tid & 7) ^ lds_swizzle(r0)) * 8;
  const uint16_t* asrc[UA];
  const uint16_t* bsrc[UB];
#pragma unroll
  for (int i = 0; i < UA; ++i) asrc[i] = x + static_cast<size_t>(min(t0 + r0 + 64 * i, p.T - 1)) * p.d + chunk;
#pragma unroll
  for (int i = 0; i < UB; ++i) bsrc[i] = w + static_cast<size_t>(min(r0 + 64 * i, nout - 1)) * p.d + chunk;
  int aoff[TM], boff[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) aoff[i] = (wm * 128 + i * 32 + (lane & 31)) * 8;
#pragma unroll
  for (int j = 0; j < TN; ++j) boff[j] = (wn * 64 + j * 32 + (lane & 31)) * 8;
  const int sw = lds_swizzle(lane);   // fragment rows are a multiple of 32 plus (lane & 31)

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  u32x4 ra[UA], rb[UB];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < UA; ++i) ra[i] = *reinterpret_cast<const u32x4*>(asrc[i] + kt * BK);
#pragma unroll
    for (int i = 0; i < UB; ++i) rb[i] = *reinterpret_cast<const u32x4*>(bsrc[i] + kt * BK);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < UA; ++i) lds_a[buf * SA + tid + NT * i] = ra[i];
#pragma unroll
    for (int i = 0; i < UB; ++i) lds_b[buf * SB + tid + NT * i] = rb[i];
  };
  u32x4 af[2][TM], bf[2][TN];
  auto read_frags = [&](int buf, int kk, int slot) {
    const int ch = (kk * 2 + (lane >> 5)) ^ sw;
#pragma unroll
    for (int i = 0; i < TM; ++i) af[slot][i] = lds_a[buf * SA + aoff[i] + ch];
#pragma unroll
    for (int j = 0; j < TN; ++j) bf[slot][j] = lds_b[buf * SB + boff[j] + ch];
  };

  // k-tile kt sits in LDS buffer kt & 1 and tile kt + 1 in registers; after the first k16 step
  // of tile kt the registers go to the other buffer and are refilled with tile kt + 2.
  // Branch-free body, interleaved by LLVM's MFMA/DS strategy as in the expert GEMM: past the end
  // the last tile is loaded again into the idle buffer, which nothing reads.
  const int nk = p.d / BK;
  gload(0);
  lstore(0);
  gload(min(1, nk - 1));
  __syncthreads();
  read_frags(0, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    __builtin_amdgcn_iglp_opt(0);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int cur = kk & 1;
      if (kk + 1 < BK / 16) read_frags(buf, kk + 1, cur ^ 1);
      if (kk == 0) {
        lstore(buf ^ 1);
        gload(min(kt + 2, nk - 1));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma_32x32x16(af[cur][i], bf[cur][j], acc[i][j]);
    }
    __syncthreads();
    read_frags(buf ^ 1, 0, 0);
  }

  // The last barrier of the loop ends every read of the staging buffers. Phase h: the waves
  // of token half h write their logits, then every thread selects for those tokens.
  // acc[i][j][4 jj + ii] is token row wm*128 + i*32 + 8 jj + 4 (lane >> 5) + ii, output
  // column wn*64 + j*32 + (lane & 31).
  for (int i = tid; i < nout; i += NT) lo[i] = key_offset(p.mode, p.modep[lg0 * p.E + i]);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (wm == h) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            logits[row * LD + wn * 64 + j * 32 + (lane & 31)] = acc[i][j][r];
          }
    }
    lds_sync();
    if (SPLIT) {   // this half's logits -> p.logits [L, T, E]: a thread per (token, layer), tokens fastest
      const int E = p.E;
      for (int i = tid; i < HALF * nl; i += NT) {
        const int tt = i % HALF, lw = i / HALF;
        const int t = t0 + h * HALF + tt;
        if (t >= p.T) continue;
        const float* src = logits + tt * LD + lw * E;   // odd LD: the lanes' reads fall on distinct banks
        float* dst = p.logits + (static_cast<size_t>(lg0 + lw) * p.T + t) * E;
        if ((E & 3) == 0) {   // rows are 16-byte aligned
          for (int e = 0; e < E; e += 4)
            *reinterpret_cast<f32x4*>(dst + e) = f32x4{src[e], src[e + 1], src[e + 2], src[e + 3]};
        } else {
          for (int e = 0; e < E; ++e) dst[e] = src[e];
        }
      }
    } else {
      route_finalize<true>(p, logits, LD, lo, t0 + h * HALF, HALF, lg0, nl, NT);
    }
    lds_sync();   // the next phase overwrites the logits
  }
}

// fp32 router: plain fp32 dot products (no MFMA), one thread per (token, output).
constexpr int kF32TT = 16;
__global__ __launch_bounds__(256) void route_f32_kernel(const RouteParams p) {
  __shared__ float logits[kF32TT * 256];
  __shared__ float lo[256];
  const int t0 = blockIdx.x * kF32TT;
  const int lg0 = blockIdx.y * p.lpw;
  const int nl = min(p.lpw, p.L - lg0);
  const int nout = nl * p.E;
  const float* x = static_cast<const float*>(p.x);
  const float* w = static_cast<const float*>(p.w) + static_cast<size_t>(lg0) * p.E * p.d;
  for (int i = threadIdx.x; i < kF32TT * nout; i += 256) {
    const int tt = i / nout, o = i - tt * nout;
    const int t = min(t0 + tt, p.T - 1);
    const float* xr = x + static_cast<size_t>(t) * p.d;
    const float* wr = w + static_cast<size_t>(o) * p.d;
    float s = 0.0f;
    for (int k = 0; k < p.d; ++k) s = fmaf(xr[k], wr[k], s);
    logits[tt * 256 + o] = s;
  }
  for (int i = threadIdx.x; i < nout; i += 256) lo[i] = key_offset(p.mode, p.modep[lg0 * p.E + i]);
  __syncthreads();
  route_finalize(p, logits, 256, lo, t0, kF32TT, lg0, nl, 256);
}

template <int MB, int NB, int WN, int WK, bool FUSE = false, bool SPLIT = false>
hipError_t launch_bf16(RouteParams& p, hipStream_t stream) {
  constexpr int TT = 16 * MB, NO = 16 * NB * WN;
  p.lpw = NO / p.E < 1 ? 1 : NO / p.E;
  if (p.lpw > p.L) p.lpw = p.L;
  dim3 grid((p.T + TT - 1) / TT, (p.L + p.lpw - 1) / p.lpw);
  if (FUSE && (grid.x != 1 || grid.y != 1)) return hipErrorInvalidValue;  // needs one workgroup
  hipLaunchKernelGGL((route_bf16_kernel<MB, NB, WN, WK, FUSE, SPLIT>), grid, dim3(64 * WN * WK), 0, stream, p);
  return hipGetLastError();
}

void fill_params(RouteParams& p, const void* x, const void* w_router, int T, int d, int E, int K, int L, int l0,
                 int mode, int gate_mode, const uint8_t* mask, const float* prior, int32_t* idx, float* gate,
                 float* margin, float* logits, size_t esz) {
  p.x = x;
  p.w = static_cast<const char*>(w_router) + static_cast<size_t>(l0) * E * d * esz;
  p.idx = idx + static_cast<size_t>(l0) * T * K;
  p.gate = gate + static_cast<size_t>(l0) * T * K;
  p.margin = margin ? margin + static_cast<size_t>(l0) * T : nullptr;
  p.logits = logits ? logits + static_cast<size_t>(l0) * T * E : nullptr;
  p.T = T; p.d = d; p.E = E; p.K = K;
  p.L = L;
  p.mode = mode; p.gate_mode = gate_mode;
  p.pb = PermBuffers{};
  p.n_shared = 0;
  p.tile_rows = 1;
  for (int i = 0; i < p.L * E; ++i) {
    const size_t gi = static_cast<size_t>(l0) * E + i;
    p.modep[i] = mode == 1 ? (mask[gi] ? 1.0f : 0.0f) : mode == 2 ? prior[gi] : 1.0f;
  }
}

}  // namespace

hipError_t launch_route(bool bf16, const void* x, const void* w_router, int T, int d, int E, int K,
                        int L, int mode, int gate_mode, const uint8_t* mask, const float* prior,
                        int32_t* idx, float* gate, float* margin, float* logits, float* split_ws,
                        hipStream_t stream) {
  if (T == 0 || L == 0) return hipSuccess;
  // Split routing needs an [L, T, E] fp32 buffer: the caller's logits output, else split_ws.
  float* zbuf = logits ? logits : split_ws;
  const bool split = route_splits(bf16, T, E) && zbuf;
  // Layers are processed in launches whose (layer, expert) parameters fit in the kernel
  // arguments; every launch covers whole layers.
  const int max_layers = kMaxModeParams / E;
  const size_t esz = bf16 ? 2 : 4;
  for (int l0 = 0; l0 < L; l0 += max_layers) {
    RouteParams p;
    fill_params(p, x, w_router, T, d, E, K, L - l0 < max_layers ? L - l0 : max_layers, l0, mode, gate_mode, mask,
                prior, idx, gate, margin, split ? zbuf : logits, esz);
    hipError_t err;
    if (!bf16) {
      p.lpw = 256 / E < 1 ? 1 : 256 / E;
      if (p.lpw > p.L) p.lpw = p.L;
      dim3 grid((T + kF32TT - 1) / kF32TT, (p.L + p.lpw - 1) / p.lpw);
      hipLaunchKernelGGL(route_f32_kernel, grid, dim3(256), 0, stream, p);
      err = hipGetLastError();
    } else if (T >= kRouteGemmMinT && d % kRgBK == 0 && p.L * E >= kRouteGemmMinOutputs) {
      p.lpw = kRgBN / E;
      if (p.lpw > p.L) p.lpw = p.L;
      dim3 grid((T + kRgBM - 1) / kRgBM, (p.L + p.lpw - 1) / p.lpw);
      if (split) hipLaunchKernelGGL(route_gemm_kernel<true>, grid, dim3(kRgThreads), 0, stream, p);
      else hipLaunchKernelGGL(route_gemm_kernel<false>, grid, dim3(kRgThreads), 0, stream, p);
      err = hipGetLastError();
    } else {
      const int need = p.L * E < 256 ? p.L * E : 256;
      const bool small = T <= 128;
      if (split) {   // T >= kRouteSplitMinT
        if (need <= 16) err = launch_bf16<1, 1, 1, 8, false, true>(p, stream);
        else if (need <= 64) err = launch_bf16<1, 4, 1, 8, false, true>(p, stream);
        else err = launch_bf16<2, 4, 4, 1, false, true>(p, stream);
      } else if (need <= 16) {   // the split launch's logit tiles for many tokens: the same bits
        err = small ? launch_bf16<1, 1, 1, 16>(p, stream) : launch_bf16<1, 1, 1, 8>(p, stream);
      } else if (need <= 64) {
        err = launch_bf16<1, 4, 1, 8>(p, stream);
      } else {
        err = small ? launch_bf16<1, 4, 4, 2>(p, stream) : launch_bf16<2, 4, 4, 1>(p, stream);
      }
    }
    if (err != hipSuccess) return err;
    if (split) {
      const size_t pairs = static_cast<size_t>(p.L) * T;
      if (E <= kSelThreadE) {
        dim3 grid(static_cast<unsigned>((pairs + kSelThreads - 1) / kSelThreads));
        if (E == 8) hipLaunchKernelGGL(route_select_kernel<8>, grid, dim3(kSelThreads), 0, stream, p);
        else if (E == 16) hipLaunchKernelGGL(route_select_kernel<16>, grid, dim3(kSelThreads), 0, stream, p);
        else hipLaunchKernelGGL(route_select_kernel<0>, grid, dim3(kSelThreads), 0, stream, p);
      } else {
        constexpr int per_block = kSelThreads / 64;
        dim3 grid(static_cast<unsigned>((pairs + per_block - 1) / per_block));
        hipLaunchKernelGGL(route_select_wave_kernel, grid, dim3(kSelThreads), 0, stream, p);
      }
      err = hipGetLastError();
      if (err != hipSuccess) return err;
    }
  }
  return hipSuccess;
}

hipError_t launch_route_permute(const void* x, const void* w_router, int T, int d, int E, int K, int mode,
                                int gate_mode, const uint8_t* mask, const float* prior, int32_t* idx,
                                float* gate, float* logits, int n_shared, int tile_rows, const PermBuffers& pb,
                                hipStream_t stream) {
  if (T == 0) return hipSuccess;
  if (T > kRouteOneBlockT) return hipErrorInvalidValue;
  RouteParams p;
  fill_params(p, x, w_router, T, d, E, K, 1, 0, mode, gate_mode, mask, prior, idx, gate, nullptr, logits, 2);
  p.pb = pb;
  p.n_shared = n_shared;
  p.tile_rows = tile_rows;
  if (E <= 16) return launch_bf16<1, 1, 1, 16, true>(p, stream);
  if (E <= 64) return launch_bf16<1, 4, 1, 8, true>(p, stream);
  return launch_bf16<1, 4, 4, 2, true>(p, stream);
}

}  // namespace maskmoe
