// K1 dispatch, and the fp32 path: codebook-head projection with the CFG merge
// and temperature fused into the epilogue, and the text-head projection with a
// fused (max, lowest argmax) epilogue.
//
//   logits[g][n] = sum_h hidden[row(g)][h] * W[n][h]         (Sec. 2.1, n = k*V + v)
//   pair p (GEMM rows 2p, 2p+1 = Main, Companion):
//     scores[p][n] = (w * l_main + (1 - w) * l_comp) / T    (Eq. 1, Sec. 2.4)
//   solo row j:  scores[n_pairs + j][n] = l / T;  T = 0 (greedy): no division
//   text rows:   per row and 32-column part, the largest logit and its lowest id.
//
// bf16 heads run on the streaming kernel (k_stream.hip) up to 128 GEMM rows and
// on the MFMA-regime kernel (k_mfma.hip) above; fp32 heads (true fp32
// products, for the fp32 parity workload) run on a plain FMA kernel here.
#include "gemm_common.h"

namespace mcd {
namespace {

// Epilogue of an audio tile for GEMM rows g (even) and g+1 at column n.
__device__ inline void emit_audio(const HeadView &hv, const StepView &sv, const int32_t *rows,
                                  int g, float v0, float v1, int n) {
  if (n >= hv.N || g >= sv.Mg) return;
  if (hv.bias) {
    const float b = hv.bias[n];
    v0 += b;
    v1 += b;
  }
  if (g < 2 * sv.n_pairs) {
    const int p = g >> 1;
    const int r = rows[g];
    if (r < 0 || r >= sv.R) return;
    const float w = sv.cfg_w[r];
    const float T = sv.temperature[r];
    float s = fmaf(w, v0, (1.0f - w) * v1);
    if (T > 0.0f) s = s * (1.0f / T);
    sv.scores[(size_t)p * hv.N + n] = s;
    return;
  }
  for (int q = 0; q < 2; ++q) {
    const int gg = g + q;
    if (gg >= sv.Mg) break;
    const int r = rows[gg];
    if (r < 0 || r >= sv.R) continue;
    const float T = sv.temperature[r];
    float s = q ? v1 : v0;
    if (T > 0.0f) s = s * (1.0f / T);
    sv.scores[(size_t)(sv.n_pairs + (gg - 2 * sv.n_pairs)) * hv.N + n] = s;
  }
}

// fp32 path (plain FMA, ascending h).  256 threads: 64 columns x 4 row lanes;
// thread (c, y) computes column n0 + c for GEMM row pairs y, y+4, ...
template <bool TEXT>
__global__ __launch_bounds__(256) void head_gemm_f32(HeadView hv, StepView sv) {
  if (!plan_ok(sv)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }
  const int32_t *rows = sv.plan + kPlanHeader + (TEXT ? sv.Mg : 0);
  const int M = TEXT ? sv.n_text : sv.Mg;
  const int N = TEXT ? hv.V_text : hv.N;
  const float *Wp = static_cast<const float *>(TEXT ? hv.W_text : hv.W);
  const float *X = static_cast<const float *>(sv.hidden);
  const int H = hv.H;
  const int c = threadIdx.x & 63, y = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + c;
  const bool col_ok = n < N;
  const float *wrow = Wp + (size_t)(col_ok ? n : 0) * H;
  auto dot = [&](int g) -> float {
    const int r = rows[g];
    if (r < 0 || r >= sv.R) {
      atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
      return 0.0f;
    }
    const float *x = X + (size_t)r * H;
    float acc = 0.0f;
    for (int h = 0; h < H; ++h) acc = fmaf(x[h], wrow[h], acc);
    return acc;
  };
  if constexpr (!TEXT) {
    for (int g = 2 * y; g < M; g += 8) {
      const float v0 = col_ok ? dot(g) : 0.0f;
      const float v1 = (col_ok && g + 1 < M) ? dot(g + 1) : 0.0f;
      emit_audio(hv, sv, rows, g, v0, v1, n);
    }
  } else {
    // two 32-column parts per block: lanes 0-31 and 32-63
    for (int g0 = 0; g0 < M; g0 += 4) {
      const int g = g0 + y;
      float bv = -INFINITY;
      int bi = INT32_MAX;
      if (g < M && col_ok) {
        bv = dot(g);
        bi = n;
      }
      for (int off = 1; off < 32; off <<= 1) {
        const float ov = __shfl_xor(bv, off);
        const int oi = __shfl_xor(bi, off);
        better(bv, bi, ov, oi);
      }
      const int part = blockIdx.x * 2 + (c >> 5);
      if ((c & 31) == 0 && g < M && part < sv.text_parts) {
        sv.text_val[(size_t)g * sv.text_parts + part] = bv;
        sv.text_idx[(size_t)g * sv.text_parts + part] = bi;
      }
    }
  }
}

}  // namespace

hipError_t launch_head_gemm_part(const HeadView &hv, const StepView &sv, bool text,
                                 hipStream_t st) {
  const int M = text ? sv.n_text : sv.Mg;
  if (M == 0) return hipSuccess;
  if (hv.dtype == MCD_F32) {
    const int N = text ? hv.V_text : hv.N;
    if (text) hipLaunchKernelGGL(head_gemm_f32<true>, dim3((N + 63) / 64), dim3(256), 0, st, hv, sv);
    else hipLaunchKernelGGL(head_gemm_f32<false>, dim3((N + 63) / 64), dim3(256), 0, st, hv, sv);
    return hipGetLastError();
  }
  return M <= 128 ? launch_stream_gemm(hv, sv, text, st) : launch_mfma_gemm(hv, sv, text, st);
}

hipError_t launch_head_gemm(const HeadView &hv, const StepView &sv, hipStream_t st) {
  hipError_t e = launch_head_gemm_part(hv, sv, false, st);
  if (e == hipSuccess) e = launch_head_gemm_part(hv, sv, true, st);
  return e;
}

}  // namespace mcd
