// K1 for a mixed batch in one launch: the audio rows' projection with the CFG
// merge and temperature (Sec. 2.1, Eq. 1, Sec. 2.4) in 256 x 256 MFMA tiles,
// and the text rows' projection with its (max, lowest argmax) partials in
// weight-streaming tiles (Sec. 2.4: the text head takes no CFG).
//
// Workgroups [0, n_audio) run audio tiles, the rest text tiles.  Workgroups
// are dispatched in index order, so the longer audio tiles start first and
// the text tiles fill the compute units as they free up.  One launch on one
// stream replaces two concurrent launches on two streams, and with them the
// cross-stream fork and join of every step.  Every tile runs exactly the code
// of its own kernel, so the results are those of the two-launch path.
#include "mfma2_tile.h"
#include "stream_tile.h"

namespace mcd {
namespace {

template <int BNT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void head_gemm_mixed(
    HeadView hv, StepView sv, int n_audio) {
  constexpr int LA = M2Shape::kLds, LT = DmaShape<128, BNT>::kLds;
  __shared__ __attribute__((aligned(1024))) char lds[LA > LT ? LA : LT];
  const int b = blockIdx.x;
  if (b < n_audio) mfma2_tile(hv, sv, b, n_audio, lds);
  else dma_tile<128, BNT, true>(hv, sv, b - n_audio, lds);
}

template <int BNT>
hipError_t launch_mixed(const HeadView &hv, const StepView &sv, int n_audio, hipStream_t st) {
  const int n_text = (hv.V_text + BNT - 1) / BNT;   // one row tile of 128 text rows
  hipLaunchKernelGGL((head_gemm_mixed<BNT>), dim3((unsigned)(n_audio + n_text)), dim3(256), 0,
                     st, hv, sv, n_audio);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_mixed_gemm(const HeadView &hv, const StepView &sv, hipStream_t st,
                             bool *launched) {
  *launched = false;
  // audio rows in 256 x 256 tiles (at least one full round of them), text rows
  // in one row tile of 65..128 rows
  if (hv.dtype != MCD_BF16 || sv.Mg <= 128 || sv.n_text <= 64 || sv.n_text > 128) return hipSuccess;
  const int64_t n_audio = tiles_256(sv.Mg, hv.N);
  if (n_audio < 256 || n_audio > (1 << 20)) return hipSuccess;
  *launched = true;
  // the text tile width of the streaming launch for the same rows
  const int t128 = (hv.V_text + 127) / 128;
  if (t128 < 256) return launch_mixed<64>(hv, sv, (int)n_audio, st);
  if (t128 == 256) return launch_mixed<128>(hv, sv, (int)n_audio, st);
  return launch_mixed<256>(hv, sv, (int)n_audio, st);
}

}  // namespace mcd
