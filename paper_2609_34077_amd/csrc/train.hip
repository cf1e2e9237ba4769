// Stage 1 of masked co-adaptive fine-tuning: mask sampling and the gradients that reach the
// mask and the router through the gate values.
//
// Section 3.2, Stage 1 (Eq. 2): pi = softmax(m~); E' distinct experts drawn from pi without
// replacement form the binary mask m shared by every token of the batch; A = Top-K(p * m),
// gates computed from p * m. Mask optimization (Eq. 3): dL/dm sums every token's contribution
// through its active gates; the straight-through estimator passes it to pi and the softmax
// Jacobian to m~: dL/dm~ = (diag(pi) - pi pi^T) dL/dm, accumulated over steps by the caller's
// buffer.
//
// With dy the cotangent of y and F_i(x_t) the selected expert's output (Eq. 1), the gate
// cotangent is dg_{t,k} = <dy_t, F_{A_t[k]}(x_t)>. Holding A fixed and m = 1 on it:
//   g = p m            (g_i = p_i):  dL/dm_k += p_k dg_k, dz = p * (dp - <p, dp>), dp = dg on A;
//   g = p m / sum_A pm (renormalised): dL/dm_k += g_k (dg_k - gbar) and dz_k = g_k (dg_k - gbar)
//                                       on A (0 elsewhere), gbar = sum_A g_i dg_i.
// The router gradients follow from z = W x: dW = dz^T x and the router's share of dx = dz W.
//
// Kernels: gate_grad_kernel (one wavefront per token: the K dot products over d and the
// per-token dz and mask terms), mask_sum_kernel (one workgroup per expert: fixed-order sum over
// tokens) and mask_ste_kernel (Eq. 3), router_wgrad_vec_kernel / router_wgrad_kernel +
// slice_sum_kernel (dW in token slices, slices added in order), router_dgrad_kernel (dx). Every
// reduction has a fixed order, so results are deterministic.

#include <cmath>
#include <vector>

#include "common.hpp"
#include "kernels.hpp"

namespace maskmoe {
namespace {

constexpr int kTrainThreads = 256;
constexpr int kWaves = kTrainThreads / kWave;

__device__ __forceinline__ float load_f(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ float load_f(const uint16_t* p, size_t i) { return bf16_to_f32(p[i]); }

// Sum of v over the workgroup in a fixed order: within each wave by xor shuffles, then the
// wave sums in wave order. The result is returned to every thread.
__device__ float block_sum(float v, float* scratch) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();                     // scratch may still be read from a previous call
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  float s = scratch[0];
  for (int w = 1; w < kWaves; ++w) s += scratch[w];
  return s;
}

__device__ __forceinline__ float4 load4(const float* p, size_t i) { return *reinterpret_cast<const float4*>(p + i); }
__device__ __forceinline__ float4 load4(const uint16_t* p, size_t i) {
  const uint2 u = *reinterpret_cast<const uint2*>(p + i);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xffff0000u));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
  return v;
}

// One wavefront per token t (four tokens per workgroup; no workgroup barriers). The K dot
// products share one pass over d (four columns per lane and step when the rows allow vector
// loads) and are summed across lanes in a fixed order; lane l holds the softmax probability of
// experts l, l + 64, l + 128, l + 192 of the token's logits.
// KC: K when known at compile time (0: the runtime K), so that the K rows' loads of a step are
// issued together rather than behind one branch each.
template <typename TIn, int KC>
__global__ __launch_bounds__(kTrainThreads) void gate_grad_kernel(const TIn* __restrict__ dy,
                                                                  const float* __restrict__ eo,
                                                                  const float* __restrict__ logits,
                                                                  const int32_t* __restrict__ idx, int T, int d,
                                                                  int E, int K, int gate_mode, bool vec,
                                                                  float* __restrict__ dg_out, float* __restrict__ dz,
                                                                  float* __restrict__ dm_tok) {
  constexpr int PE = kMaxETrain / kWave;   // experts per lane
  static_assert(PE == 4, "p_of below selects among four registers");
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (t >= T) return;                      // the whole wavefront leaves together
  const TIn* dyt = dy + static_cast<size_t>(t) * d;
  const float* eot = eo + static_cast<size_t>(t) * K * d;
  float acc[kMaxKTrain];
#pragma unroll
  for (int k = 0; k < kMaxKTrain; ++k) acc[k] = 0.0f;
  constexpr int KL = KC ? KC : kMaxKTrain;
  if (vec) {   // d % 4 == 0, rows 16-byte (fp32) / 8-byte (bf16) aligned
#pragma unroll 4
    for (int c = lane * 4; c < d; c += kWave * 4) {
      const float4 a = load4(dyt, c);
#pragma unroll
      for (int k = 0; k < KL; ++k) {
        if (KC || k < K) {
          const float4 e = load4(eot, static_cast<size_t>(k) * d + c);
          acc[k] += a.x * e.x + a.y * e.y + a.z * e.z + a.w * e.w;
        }
      }
    }
  } else {
    for (int c = lane; c < d; c += kWave) {
      const float a = load_f(dyt, c);
#pragma unroll
      for (int k = 0; k < kMaxKTrain; ++k)
        if (k < K) acc[k] += a * eot[static_cast<size_t>(k) * d + c];
    }
  }
  float dg[kMaxKTrain];
#pragma unroll
  for (int k = 0; k < kMaxKTrain; ++k) dg[k] = k < K ? wave_sum(acc[k]) : 0.0f;
  if (dg_out && lane < K) {
    float v = 0.0f;
#pragma unroll
    for (int k = 0; k < kMaxKTrain; ++k)
      if (k == lane) v = dg[k];
    dg_out[static_cast<size_t>(t) * K + lane] = v;
  }
  // softmax of the logits
  const float* z = logits + static_cast<size_t>(t) * E;
  float pv[PE];
  float zmax = -INFINITY;
#pragma unroll
  for (int i = 0; i < PE; ++i) {
    const int e = lane + kWave * i;
    pv[i] = e < E ? z[e] : -INFINITY;
    zmax = fmaxf(zmax, pv[i]);
  }
  zmax = wave_max(zmax);
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < PE; ++i) {
    const int e = lane + kWave * i;
    pv[i] = e < E ? expf(pv[i] - zmax) : 0.0f;
    sum += pv[i];
  }
  sum = wave_sum(sum);
  const float inv = 1.0f / sum;
#pragma unroll
  for (int i = 0; i < PE; ++i) pv[i] *= inv;
  // p of expert e (wave-uniform e), fetched from the lane that owns it
  auto p_of = [&](int e) {
    const int i = e / kWave;
    const float v = i == 0 ? pv[0] : i == 1 ? pv[1] : i == 2 ? pv[2] : pv[3];
    return __shfl(v, e % kWave, kWave);
  };
  const int32_t* A = idx + static_cast<size_t>(t) * K;
  int a[kMaxKTrain];
  float pA = 0.0f, pdg = 0.0f;
#pragma unroll
  for (int k = 0; k < kMaxKTrain; ++k) {
    a[k] = k < K ? A[k] : -1;
    if (k < K) {
      const float pk = p_of(a[k]);
      pA += pk;
      pdg += pk * dg[k];
    }
  }
#pragma unroll
  for (int i = 0; i < PE; ++i) {
    const int e = lane + kWave * i;
    if (e >= E) continue;
    float dge = 0.0f;
    bool sel = false;
#pragma unroll
    for (int k = 0; k < kMaxKTrain; ++k)
      if (k < K && a[k] == e) {
        dge = dg[k];
        sel = true;
      }
    float zg, mg;
    if (gate_mode == 0) {        // g = p m
      mg = sel ? pv[i] * dge : 0.0f;
      zg = pv[i] * (dge - pdg);
    } else {                     // g = p m / sum_A p m: gbar = sum_A g dg = pdg / pA
      const float gbar = pdg / pA;
      mg = sel ? (pv[i] / pA) * (dge - gbar) : 0.0f;
      zg = mg;
    }
    dz[static_cast<size_t>(t) * E + e] = zg;
    dm_tok[static_cast<size_t>(t) * E + e] = mg;
  }
}

struct MaskPi {
  float v[kMaxETrain];   // pi = softmax(m~), computed on the host in double precision
};

// dL/dm_e = sum_t dm_tok[t, e]: workgroup e; thread j adds tokens j, j + 256, ... in order
// (eight loads in flight per step), then the fixed workgroup sum.
__global__ __launch_bounds__(kTrainThreads) void mask_sum_kernel(const float* __restrict__ dm_tok, int T, int E,
                                                                 float* __restrict__ dm) {
  __shared__ float scratch[kWaves];
  const int e = blockIdx.x, tid = threadIdx.x;
  constexpr int U = 8;
  float s = 0.0f;
  int t = tid;
  for (; t + (U - 1) * kTrainThreads < T; t += U * kTrainThreads) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dm_tok[static_cast<size_t>(t + u * kTrainThreads) * E + e];
#pragma unroll
    for (int u = 0; u < U; ++u) s += v[u];
  }
  for (; t < T; t += kTrainThreads) s += dm_tok[static_cast<size_t>(t) * E + e];
  s = block_sum(s, scratch);
  if (tid == 0) dm[e] = s;
}

// Eq. 3 into the accumulator: d_mask_logits += pi (dm - <pi, dm>). One workgroup.
__global__ __launch_bounds__(kTrainThreads) void mask_ste_kernel(const float* __restrict__ dm, int E,
                                                                 float* __restrict__ d_mask,
                                                                 float* __restrict__ d_mask_logits, const MaskPi pi) {
  float pidm = 0.0f;
  for (int e = 0; e < E; ++e) pidm += pi.v[e] * dm[e];
  for (int e = threadIdx.x; e < E; e += kTrainThreads) {
    if (d_mask) d_mask[e] = dm[e];
    if (d_mask_logits) d_mask_logits[e] += pi.v[e] * (dm[e] - pidm);
  }
}

// partial[s, e, c] = sum over tokens t of slice s of dz[t, e] x[t, c]. Grid (ceil(d / 256),
// ceil(E / kWgradEB), slices); thread c of a workgroup owns column c and kWgradEB experts;
// the dz rows of the slice are staged through LDS in chunks.
constexpr int kWgradEB = 8;
constexpr int kWgradRows = 64;

template <typename TIn>
__global__ __launch_bounds__(kTrainThreads) void router_wgrad_kernel(const TIn* __restrict__ x,
                                                                     const float* __restrict__ dz, int T, int d, int E,
                                                                     int rows_per_slice, float* __restrict__ partial) {
  __shared__ float dzs[kWgradRows][kWgradEB];
  const int c = blockIdx.x * kTrainThreads + threadIdx.x;
  const int e0 = blockIdx.y * kWgradEB;
  const int ne = min(kWgradEB, E - e0);
  const int t_begin = blockIdx.z * rows_per_slice;
  const int t_end = min(T, t_begin + rows_per_slice);
  float acc[kWgradEB];
#pragma unroll
  for (int q = 0; q < kWgradEB; ++q) acc[q] = 0.0f;
  for (int t0 = t_begin; t0 < t_end; t0 += kWgradRows) {
    const int nr = min(kWgradRows, t_end - t0);
    __syncthreads();
    for (int i = threadIdx.x; i < kWgradRows * kWgradEB; i += kTrainThreads) {
      const int r = i / kWgradEB, q = i % kWgradEB;
      dzs[r][q] = (r < nr && q < ne) ? dz[static_cast<size_t>(t0 + r) * E + e0 + q] : 0.0f;
    }
    __syncthreads();
    if (c < d) {
      for (int r = 0; r < nr; ++r) {
        const float xv = load_f(x, static_cast<size_t>(t0 + r) * d + c);
#pragma unroll
        for (int q = 0; q < kWgradEB; ++q) acc[q] += dzs[r][q] * xv;
      }
    }
  }
  if (c < d)
    for (int q = 0; q < ne; ++q)
      partial[(static_cast<size_t>(blockIdx.z) * E + e0 + q) * d + c] = acc[q];
}

// Vectorised form (rows of x 16-byte aligned, d a multiple of VEC = 16 bytes of elements):
// a workgroup covers 32 * VEC columns of a token slice; thread (rg, j) owns columns
// [j VEC, (j + 1) VEC) and the slice rows rg, rg + kRowGroups, ..., loading each with one
// 16-byte load; the kRowGroups partial sums are added in LDS in row-group order.
constexpr int kRowGroups = kTrainThreads / 32;

template <typename TIn>
__global__ __launch_bounds__(kTrainThreads) void router_wgrad_vec_kernel(const TIn* __restrict__ x,
                                                                         const float* __restrict__ dz, int T, int d,
                                                                         int E, int rows_per_slice,
                                                                         float* __restrict__ partial) {
  constexpr int VEC = 16 / sizeof(TIn);
  constexpr int COLS = 32 * VEC;
  __shared__ float dzs[kWgradRows][kWgradEB];
  __shared__ float sums[kRowGroups][kWgradEB][COLS];
  const int j = threadIdx.x & 31, rg = threadIdx.x >> 5;
  const int c0 = blockIdx.x * COLS + j * VEC;
  const bool live = c0 < d;
  const int e0 = blockIdx.y * kWgradEB;
  const int ne = min(kWgradEB, E - e0);
  const int t_begin = blockIdx.z * rows_per_slice;
  const int t_end = min(T, t_begin + rows_per_slice);
  float acc[kWgradEB][VEC];
#pragma unroll
  for (int q = 0; q < kWgradEB; ++q)
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[q][v] = 0.0f;
  for (int t0 = t_begin; t0 < t_end; t0 += kWgradRows) {
    const int nr = min(kWgradRows, t_end - t0);
    __syncthreads();
    for (int i = threadIdx.x; i < kWgradRows * kWgradEB; i += kTrainThreads) {
      const int r = i / kWgradEB, q = i % kWgradEB;
      dzs[r][q] = (r < nr && q < ne) ? dz[static_cast<size_t>(t0 + r) * E + e0 + q] : 0.0f;
    }
    __syncthreads();
    if (live) {
#pragma unroll 4
      for (int r = rg; r < nr; r += kRowGroups) {
        const TIn* row = x + static_cast<size_t>(t0 + r) * d + c0;
        float xv[VEC];
        if constexpr (VEC == 8) {
          const uint4 u = *reinterpret_cast<const uint4*>(row);
          const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            xv[2 * h] = __uint_as_float(w[h] << 16);
            xv[2 * h + 1] = __uint_as_float(w[h] & 0xffff0000u);
          }
        } else {
          const float4 f = *reinterpret_cast<const float4*>(row);
          xv[0] = f.x; xv[1] = f.y; xv[2] = f.z; xv[3] = f.w;
        }
#pragma unroll
        for (int q = 0; q < kWgradEB; ++q) {
          const float g = dzs[r][q];
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[q][v] += g * xv[v];
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < kWgradEB; ++q)
#pragma unroll
    for (int v = 0; v < VEC; ++v) sums[rg][q][j * VEC + v] = acc[q][v];
  __syncthreads();
  for (int i = threadIdx.x; i < kWgradEB * COLS; i += kTrainThreads) {
    const int q = i / COLS, col = i % COLS;
    const int c = blockIdx.x * COLS + col;
    if (q >= ne || c >= d) continue;
    float s = sums[0][q][col];
    for (int g = 1; g < kRowGroups; ++g) s += sums[g][q][col];
    partial[(static_cast<size_t>(blockIdx.z) * E + e0 + q) * d + c] = s;
  }
}

// out[i] = sum_s partial[s, i], s in order.
__global__ __launch_bounds__(kTrainThreads) void slice_sum_kernel(const float* __restrict__ partial, int slices,
                                                                  size_t n, float* __restrict__ out) {
  const size_t i = static_cast<size_t>(blockIdx.x) * kTrainThreads + threadIdx.x;
  if (i >= n) return;
  constexpr int U = 8;
  float s = partial[i];
  int z = 1;
  for (; z + U - 1 < slices; z += U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = partial[static_cast<size_t>(z + u) * n + i];
#pragma unroll
    for (int u = 0; u < U; ++u) s += v[u];
  }
  for (; z < slices; ++z) s += partial[static_cast<size_t>(z) * n + i];
  out[i] = s;
}

// dx[t, c] = sum_e dz[t, e] W[e, c]. Grid (ceil(d / 256), ceil(T / kDgradRows)); thread c owns
// a column and kDgradRows tokens, whose dz rows sit in LDS; W is read once per workgroup.
constexpr int kDgradRows = 16;

template <typename TIn>
__global__ __launch_bounds__(kTrainThreads) void router_dgrad_kernel(const TIn* __restrict__ w,
                                                                     const float* __restrict__ dz, int T, int d, int E,
                                                                     float* __restrict__ dx) {
  __shared__ float dzs[kDgradRows][kMaxETrain];
  const int c = blockIdx.x * kTrainThreads + threadIdx.x;
  const int t0 = blockIdx.y * kDgradRows;
  const int nr = min(kDgradRows, T - t0);
  for (int i = threadIdx.x; i < kDgradRows * E; i += kTrainThreads) {
    const int r = i / E, e = i % E;
    dzs[r][e] = r < nr ? dz[static_cast<size_t>(t0 + r) * E + e] : 0.0f;
  }
  __syncthreads();
  if (c >= d) return;
  float acc[kDgradRows];
#pragma unroll
  for (int r = 0; r < kDgradRows; ++r) acc[r] = 0.0f;
  for (int e = 0; e < E; ++e) {
    const float wv = load_f(w, static_cast<size_t>(e) * d + c);
#pragma unroll
    for (int r = 0; r < kDgradRows; ++r) acc[r] += dzs[r][e] * wv;
  }
  for (int r = 0; r < nr; ++r) dx[static_cast<size_t>(t0 + r) * d + c] = acc[r];
}

int wgrad_cols(bool vec, int elem_bytes) { return vec ? 32 * (16 / elem_bytes) : kTrainThreads; }

int wgrad_slices(int T, int d, int E, int cols) {
  const int blocks = ((d + cols - 1) / cols) * ((E + kWgradEB - 1) / kWgradEB);
  int s = (1024 + blocks - 1) / blocks;           // about 1024 workgroups
  const int max_s = (T + kWgradRows - 1) / kWgradRows;
  if (s > max_s) s = max_s;
  if (s > kMaxWgradSlices) s = kMaxWgradSlices;
  return s < 1 ? 1 : s;
}

template <typename TIn>
hipError_t launch_stage1(const Stage1Args& a, hipStream_t stream) {
  const TIn* dy = static_cast<const TIn*>(a.dy);
  const dim3 grid((a.T + kWaves - 1) / kWaves), block(kTrainThreads);
#define MASKMOE_GATE_GRAD(KC)                                                                                  \
  hipLaunchKernelGGL((gate_grad_kernel<TIn, KC>), grid, block, 0, stream, dy, a.expert_out, a.router_logits, a.idx, \
                     a.T, a.d, a.E, a.K, a.gate_mode, a.vec_rows, a.d_gate, a.dz, a.dm_tok)
  switch (a.K) {   // the two models' K, and a runtime-K instance for the rest
    case 2: MASKMOE_GATE_GRAD(2); break;
    case 6: MASKMOE_GATE_GRAD(6); break;
    default: MASKMOE_GATE_GRAD(0); break;
  }
#undef MASKMOE_GATE_GRAD
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(mask_sum_kernel, dim3(a.E), dim3(kTrainThreads), 0, stream, a.dm_tok, a.T, a.E, a.dm);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  MaskPi pi;
  for (int e = 0; e < a.E; ++e) pi.v[e] = static_cast<float>(a.pi[e]);
  hipLaunchKernelGGL(mask_ste_kernel, dim3(1), dim3(kTrainThreads), 0, stream, a.dm, a.E, a.d_mask,
                     a.d_mask_logits, pi);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int cols = wgrad_cols(a.vec_x, static_cast<int>(sizeof(TIn)));
  const int slices = wgrad_slices(a.T, a.d, a.E, cols);
  const int rows = (a.T + slices - 1) / slices;
  const dim3 wg((a.d + cols - 1) / cols, (a.E + kWgradEB - 1) / kWgradEB, slices);
  if (a.vec_x)
    hipLaunchKernelGGL((router_wgrad_vec_kernel<TIn>), wg, dim3(kTrainThreads), 0, stream,
                       static_cast<const TIn*>(a.x), a.dz, a.T, a.d, a.E, rows, a.wgrad_partial);
  else
    hipLaunchKernelGGL((router_wgrad_kernel<TIn>), wg, dim3(kTrainThreads), 0, stream, static_cast<const TIn*>(a.x),
                       a.dz, a.T, a.d, a.E, rows, a.wgrad_partial);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  const size_t n = static_cast<size_t>(a.E) * a.d;
  hipLaunchKernelGGL(slice_sum_kernel, dim3(static_cast<unsigned>((n + kTrainThreads - 1) / kTrainThreads)),
                     dim3(kTrainThreads), 0, stream, a.wgrad_partial, slices, n, a.d_w_router);
  err = hipGetLastError();
  if (err != hipSuccess || !a.d_x) return err;
  const dim3 dg((a.d + kTrainThreads - 1) / kTrainThreads, (a.T + kDgradRows - 1) / kDgradRows);
  hipLaunchKernelGGL((router_dgrad_kernel<TIn>), dg, dim3(kTrainThreads), 0, stream,
                     static_cast<const TIn*>(a.w_router), a.dz, a.T, a.d, a.E, a.d_x);
  return hipGetLastError();
}

}  // namespace

size_t stage1_workspace_bytes(int T, int d, int E) {
  // dz and dm_tok [T, E], the per-expert sums [E], then the dW slices of the load path with
  // the widest workgroup column coverage (fewest column blocks, so the most slices): 256
  // columns (the scalar path and 16-byte bf16 loads; 16-byte fp32 loads cover 128)
  static_assert(kTrainThreads >= 32 * 8, "no load path covers more than kTrainThreads columns");
  const size_t tok = (static_cast<size_t>(T) * E * 4 + 255) / 256 * 256;
  const size_t dm = (static_cast<size_t>(E) * 4 + 255) / 256 * 256;
  const size_t part = static_cast<size_t>(wgrad_slices(T, d, E, kTrainThreads)) * E * d * 4;
  return 2 * tok + dm + (part + 255) / 256 * 256;
}

hipError_t launch_stage1_backward(const Stage1Args& a, bool bf16, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  return bf16 ? launch_stage1<uint16_t>(a, stream) : launch_stage1<float>(a, stream);
}

void softmax_f64(const float* logits, int E, double* pi) {
  double mx = logits[0];
  for (int e = 1; e < E; ++e) mx = logits[e] > mx ? logits[e] : mx;
  double sum = 0.0;
  for (int e = 0; e < E; ++e) {
    pi[e] = std::exp(static_cast<double>(logits[e]) - mx);
    sum += pi[e];
  }
  for (int e = 0; e < E; ++e) pi[e] /= sum;
}

void sample_mask_host(const float* mask_logits, const double* uniforms, int E, int e_keep, uint8_t* mask) {
  std::vector<double> pi(E);
  softmax_f64(mask_logits, E, pi.data());
  std::vector<int> remaining(E);
  for (int e = 0; e < E; ++e) {
    remaining[e] = e;
    mask[e] = 0;
  }
  for (int s = 0; s < e_keep; ++s) {
    double total = 0.0;
    for (int i : remaining) total += pi[i];
    const double target = uniforms[s] * total;
    double run = 0.0;
    size_t pos = remaining.size() - 1;   // u * total below the full sum lands earlier
    for (size_t j = 0; j < remaining.size(); ++j) {
      run += pi[remaining[j]];
      if (target < run) {
        pos = j;
        break;
      }
    }
    mask[remaining[pos]] = 1;
    remaining.erase(remaining.begin() + static_cast<long>(pos));
  }
}

}  // namespace maskmoe
