// Token permutation by expert (see permute_block.hpp): one workgroup of 1024 threads.

#include "permute_block.hpp"

namespace maskmoe {
namespace {

constexpr int kPermThreads = 1024;

__global__ __launch_bounds__(kPermThreads) void permute_kernel(const int32_t* __restrict__ idx, int T, int K,
                                                              int E, int n_shared, int tile_rows,
                                                              PermBuffers pb) {
  __shared__ PermLds lds;
  permute_block(idx, T, K, E, n_shared, tile_rows, pb, lds);
}

}  // namespace

hipError_t launch_permute(const int32_t* idx, int T, int K, int E, int n_shared, int tile_rows,
                          const PermBuffers& pb, hipStream_t stream) {
  hipLaunchKernelGGL(permute_kernel, dim3(1), dim3(kPermThreads), 0, stream, idx, T, K, E, n_shared,
                     tile_rows, pb);
  return hipGetLastError();
}

}  // namespace maskmoe
