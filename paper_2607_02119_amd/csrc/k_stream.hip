// K1, weight-streaming path (at most 128 GEMM rows; also audio batches of
// more than 128 rows that do not fill the chip with 256 x 256 tiles, in
// 128-row tiles): codebook-head projection
// with the CFG merge and temperature fused into the epilogue, or the text-head
// projection with a fused (max, lowest argmax) epilogue.
//
//   logits[g][n] = sum_h hidden[row(g)][h] * W[n][h]         (Sec. 2.1, n = k*V + v)
//   pair p (GEMM rows 2p, 2p+1 = Main, Companion):
//     scores[p][n] = (w * l_main + (1 - w) * l_comp) / T    (Eq. 1, Sec. 2.4)
//   solo row j:  scores[n_pairs + j][n] = l / T;  T = 0 (greedy): no division
//   text rows:   per row and 32-column part, the largest logit and its lowest id.
#include "stream_tile.h"

namespace mcd {
namespace {

template <int BM, int BN, bool TEXT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void head_gemm_dma(
    HeadView hv, StepView sv) {
  __shared__ __attribute__((aligned(1024))) char lds[DmaShape<BM, BN>::kLds];
  dma_tile<BM, BN, TEXT>(hv, sv, blockIdx.x, lds);
}

template <int BM, int BN, bool TEXT>
hipError_t launch_dma(const HeadView &hv, const StepView &sv, int M, int N, hipStream_t st) {
  const int tm = (M + BM - 1) / BM, tn = (N + BN - 1) / BN;
  hipLaunchKernelGGL((head_gemm_dma<BM, BN, TEXT>), dim3(tm * tn), dim3(256), 0, st, hv, sv);
  return hipGetLastError();
}

template <int BM, bool TEXT>
hipError_t launch_rows(const HeadView &hv, const StepView &sv, int M, int N, hipStream_t st) {
  const int t128 = (N + 127) / 128;
  if (t128 < 256) return launch_dma<BM, 64, TEXT>(hv, sv, M, N, st);
  if (t128 == 256) return launch_dma<BM, 128, TEXT>(hv, sv, M, N, st);
  return launch_dma<BM, 256, TEXT>(hv, sv, M, N, st);
}

// Weight-streaming launch for M <= 128 rows: 64-column tiles when 128-column
// ones would leave compute units idle, 128-column tiles when they make exactly
// one round, and 256-column tiles (half the hidden-state bytes per weight
// byte) when there is more than one round.
template <bool TEXT>
hipError_t launch_skinny(const HeadView &hv, const StepView &sv, int M, int N, hipStream_t st) {
  if (M <= 32) return launch_rows<32, TEXT>(hv, sv, M, N, st);
  if (M <= 64) return launch_rows<64, TEXT>(hv, sv, M, N, st);
  return launch_rows<128, TEXT>(hv, sv, M, N, st);
}

}  // namespace

// Audio batches of more than 128 GEMM rows that make fewer than 256 tiles of
// 256 x 256 (the cfg workloads' 512 rows): 128 x 256 tiles, row tile by row
// tile.  Their 64-k slices read whole 128-byte row segments; the 256 x 128
// MFMA tiles' 32-k slices read half segments and took 5-12 % longer.
hipError_t launch_stream_rows(const HeadView &hv, const StepView &sv, hipStream_t st) {
  return launch_dma<128, 256, false>(hv, sv, sv.Mg, hv.N, st);
}

hipError_t launch_stream_gemm(const HeadView &hv, const StepView &sv, bool text,
                              hipStream_t st) {
  return text ? launch_skinny<true>(hv, sv, sv.n_text, hv.V_text, st)
              : launch_skinny<false>(hv, sv, sv.Mg, hv.N, st);
}

}  // namespace mcd
