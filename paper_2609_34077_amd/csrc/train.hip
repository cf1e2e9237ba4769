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
// Kernels: gate_grad_kernel (one workgroup per token: the K dot products over d and the
// per-token dz and mask terms), mask_reduce_kernel (fixed-order sum over tokens, then Eq. 3),
// router_wgrad_kernel + slice_sum_kernel (dW in token slices, slices added in order),
// router_dgrad_kernel (dx). Every reduction has a fixed order, so results are deterministic.

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

// One workgroup per token t.
template <typename TIn>
__global__ __launch_bounds__(kTrainThreads) void gate_grad_kernel(const TIn* __restrict__ dy,
                                                                  const float* __restrict__ eo,
                                                                  const float* __restrict__ logits,
                                                                  const int32_t* __restrict__ idx, int T, int d,
                                                                  int E, int K, int gate_mode, float* __restrict__ dg_out,
                                                                  float* __restrict__ dz, float* __restrict__ dm_tok) {
  __shared__ float scratch[kWaves];
  __shared__ float dg[kMaxKTrain];
  __shared__ float p[kMaxETrain];
  const int t = blockIdx.x, tid = threadIdx.x;
  const TIn* dyt = dy + static_cast<size_t>(t) * d;
  for (int k = 0; k < K; ++k) {
    const float* e = eo + (static_cast<size_t>(t) * K + k) * d;
    float s = 0.0f;
    for (int c = tid; c < d; c += kTrainThreads) s += load_f(dyt, c) * e[c];
    s = block_sum(s, scratch);
    if (tid == 0) dg[k] = s;
  }
  // softmax of the token's logits (one thread per expert, E <= kMaxETrain)
  const float* z = logits + static_cast<size_t>(t) * E;
  if (tid == 0) {
    float zmax = z[0];
    for (int e = 1; e < E; ++e) zmax = fmaxf(zmax, z[e]);
    float sum = 0.0f;
    for (int e = 0; e < E; ++e) sum += expf(z[e] - zmax);
    const float inv = 1.0f / sum;
    for (int e = 0; e < E; ++e) p[e] = expf(z[e] - zmax) * inv;
  }
  __syncthreads();
  if (tid == 0 && dg_out)
    for (int k = 0; k < K; ++k) dg_out[static_cast<size_t>(t) * K + k] = dg[k];
  const int32_t* A = idx + static_cast<size_t>(t) * K;
  // shared per-token scalars, computed redundantly by every thread in the same order
  float pA = 0.0f, pdg = 0.0f;
  for (int k = 0; k < K; ++k) {
    pA += p[A[k]];
    pdg += p[A[k]] * dg[k];
  }
  for (int e = tid; e < E; e += kTrainThreads) {
    int kpos = -1;
    for (int k = 0; k < K; ++k)
      if (A[k] == e) kpos = k;
    float zg, mg;
    if (gate_mode == 0) {        // g = p m
      mg = kpos >= 0 ? p[e] * dg[kpos] : 0.0f;
      zg = p[e] * ((kpos >= 0 ? dg[kpos] : 0.0f) - pdg);
    } else {                     // g = p m / sum_A p m: gbar = sum_A g dg = pdg / pA
      const float gbar = pdg / pA;
      mg = kpos >= 0 ? (p[e] / pA) * (dg[kpos] - gbar) : 0.0f;
      zg = mg;
    }
    dz[static_cast<size_t>(t) * E + e] = zg;
    dm_tok[static_cast<size_t>(t) * E + e] = mg;
  }
}

struct MaskPi {
  float v[kMaxETrain];   // pi = softmax(m~), computed on the host in double precision
};

// dL/dm_e = sum_t dm_tok[t, e] (threads take tokens tid, tid + 256, ... in order, then the
// fixed block sum), then Eq. 3 into the accumulator. One workgroup.
__global__ __launch_bounds__(kTrainThreads) void mask_reduce_kernel(const float* __restrict__ dm_tok, int T, int E,
                                                                    float* __restrict__ d_mask,
                                                                    float* __restrict__ d_mask_logits, const MaskPi pi) {
  __shared__ float scratch[kWaves];
  __shared__ float dm[kMaxETrain];
  const int tid = threadIdx.x;
  for (int e = 0; e < E; ++e) {
    float s = 0.0f;
    for (int t = tid; t < T; t += kTrainThreads) s += dm_tok[static_cast<size_t>(t) * E + e];
    s = block_sum(s, scratch);
    if (tid == 0) dm[e] = s;
  }
  __syncthreads();
  float pidm = 0.0f;
  for (int e = 0; e < E; ++e) pidm += pi.v[e] * dm[e];
  for (int e = tid; e < E; e += kTrainThreads) {
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

// out[i] = sum_s partial[s, i], s in order.
__global__ __launch_bounds__(kTrainThreads) void slice_sum_kernel(const float* __restrict__ partial, int slices,
                                                                  size_t n, float* __restrict__ out) {
  const size_t i = static_cast<size_t>(blockIdx.x) * kTrainThreads + threadIdx.x;
  if (i >= n) return;
  float s = partial[i];
  for (int z = 1; z < slices; ++z) s += partial[static_cast<size_t>(z) * n + i];
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

int wgrad_slices(int T, int d, int E) {
  const int blocks = ((d + kTrainThreads - 1) / kTrainThreads) * ((E + kWgradEB - 1) / kWgradEB);
  int s = (1024 + blocks - 1) / blocks;           // about 1024 workgroups
  const int max_s = (T + kWgradRows - 1) / kWgradRows;
  if (s > max_s) s = max_s;
  if (s > kMaxWgradSlices) s = kMaxWgradSlices;
  return s < 1 ? 1 : s;
}

template <typename TIn>
hipError_t launch_stage1(const Stage1Args& a, hipStream_t stream) {
  const TIn* dy = static_cast<const TIn*>(a.dy);
  hipLaunchKernelGGL((gate_grad_kernel<TIn>), dim3(a.T), dim3(kTrainThreads), 0, stream, dy, a.expert_out,
                     a.router_logits, a.idx, a.T, a.d, a.E, a.K, a.gate_mode, a.d_gate, a.dz, a.dm_tok);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  MaskPi pi;
  for (int e = 0; e < a.E; ++e) pi.v[e] = static_cast<float>(a.pi[e]);
  hipLaunchKernelGGL(mask_reduce_kernel, dim3(1), dim3(kTrainThreads), 0, stream, a.dm_tok, a.T, a.E, a.d_mask,
                     a.d_mask_logits, pi);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int slices = wgrad_slices(a.T, a.d, a.E);
  const int rows = (a.T + slices - 1) / slices;
  const dim3 wg((a.d + kTrainThreads - 1) / kTrainThreads, (a.E + kWgradEB - 1) / kWgradEB, slices);
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
  const size_t tok = (static_cast<size_t>(T) * E * 4 + 255) / 256 * 256;   // dz, dm_tok
  const size_t part = static_cast<size_t>(wgrad_slices(T, d, E)) * E * d * 4;
  return 2 * tok + (part + 255) / 256 * 256;
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
