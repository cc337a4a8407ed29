// K3: delay-pattern de-interleave / interleave between a per-request stream
// buffer [T][K] (token of codebook k emitted at step t) and the frame grid
// [K][F] (Sec. 2.1: stream k is offset by d_k steps, so frame f of codebook k
// was emitted at step f + d_k).  One thread per output element; the grid side
// is written (de-interleave) or read (interleave) contiguously.
#include "mcd_internal.h"

namespace mcd {
namespace {

__global__ __launch_bounds__(256) void deinterleave_kernel(const int32_t *__restrict__ streams,
                                                           int32_t n_req, int32_t T, int32_t K,
                                                           Delays d, int32_t F,
                                                           int32_t *__restrict__ grid) {
  const size_t total = (size_t)n_req * K * F;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int32_t f = (int32_t)(i % F);
    const int32_t k = (int32_t)((i / F) % K);
    const size_t r = i / ((size_t)F * K);
    grid[i] = streams[(r * T + (size_t)(f + d.d[k])) * K + k];
  }
}

__global__ __launch_bounds__(256) void interleave_kernel(const int32_t *__restrict__ grid,
                                                         int32_t n_req, int32_t F, int32_t K,
                                                         Delays d, int32_t T, int32_t pad_id,
                                                         int32_t *__restrict__ streams) {
  const size_t total = (size_t)n_req * T * K;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int32_t k = (int32_t)(i % K);
    const int32_t t = (int32_t)((i / K) % T);
    const size_t r = i / ((size_t)K * T);
    const int32_t f = t - d.d[k];
    streams[i] = (f >= 0 && f < F) ? grid[(r * K + k) * F + f] : pad_id;
  }
}

unsigned blocks_for(size_t total) {
  size_t b = (total + 255) / 256;
  if (b > 65536) b = 65536;
  return (unsigned)(b ? b : 1);
}

}  // namespace

hipError_t launch_deinterleave(const int32_t *streams, int32_t n_req, int32_t T, int32_t K,
                               const Delays &d, int32_t F, int32_t *grid, hipStream_t st) {
  const size_t total = (size_t)n_req * K * F;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(deinterleave_kernel, dim3(blocks_for(total)), dim3(256), 0, st, streams,
                     n_req, T, K, d, F, grid);
  return hipGetLastError();
}

hipError_t launch_interleave(const int32_t *grid, int32_t n_req, int32_t F, int32_t K,
                             const Delays &d, int32_t T, int32_t pad_id, int32_t *streams,
                             hipStream_t st) {
  const size_t total = (size_t)n_req * T * K;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(interleave_kernel, dim3(blocks_for(total)), dim3(256), 0, st, grid, n_req,
                     F, K, d, T, pad_id, streams);
  return hipGetLastError();
}

}  // namespace mcd
