// Next-step input of the delay pattern (Sec. 2.1): the backbone's input for
// the next step aggregates the embeddings of the K tokens a row emitted at
// this step, one per stream, each for its own delayed frame.  Here:
//   out[r][h] = sum_k E[k][row_k][h],   row_k = tokens[r][k] (V for the pad id)
//   TEXT rows: out[r][h] = E_text[tokens[r][0]][h]
// summed in fp64 and rounded once to the table type.
//
// A gather-reduce bound by HBM: one workgroup per (row, 2048- or 1024-element
// column block), one thread per 16 bytes of output.  The table rows of a
// workgroup are uniform, so the tokens are read with scalar loads; the K
// 16-byte loads of a thread are issued eight at a time before any is summed.
#include "gemm_common.h"

namespace mcd {
namespace {

// The nearest bfloat16 of x (8 significant bits at x's own exponent, the step
// floored at the bf16 subnormal spacing 2^-133), ties to even, taken straight
// from the double: no intermediate fp32 rounding.
__device__ inline uint32_t bf16_bits_from_f64(double x) {
  if (x != x) return 0x7FC0u;
  const double ax = fabs(x);
  if (ax == 0.0 || ax == INFINITY) return __float_as_uint((float)x) >> 16;
  const int e = max(ilogb(ax), -126);
  const double up = ldexp(1.0, 7 - e), down = ldexp(1.0, e - 7);   // exact powers of two
  const double y = rint(x * up) * down;                            // nearest, ties to even
  const float f = fabs(y) >= 0x1p128 ? copysignf(INFINITY, (float)x) : (float)y;
  return __float_as_uint(f) >> 16;
}

template <bool BF16>
__device__ inline double elem_f64(const void *p, int64_t i) {
  if constexpr (BF16) return (double)__uint_as_float((uint32_t)static_cast<const uint16_t *>(p)[i] << 16);
  else return (double)static_cast<const float *>(p)[i];
}

template <bool BF16>
__global__ __launch_bounds__(256) void next_input_kernel(EmbedView ev) {
  constexpr int VEC = BF16 ? 8 : 4;        // elements per 16 bytes
  constexpr int G = 8;                     // table rows loaded before summing
  const int r = blockIdx.x;
  const int H = ev.H, K = ev.K;
  const int h0 = (blockIdx.y * 256 + threadIdx.x) * VEC;
  const bool text = ld_const(ev.row_kind, r) == MCD_ROW_TEXT;
  const int nsrc = text ? 1 : K;
  const void *tab = text ? ev.E_text : ev.E;
  const bool vec = (H % VEC == 0) && (h0 + VEC <= H);
  double acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.0;
  bool bad = false;
  for (int k0 = 0; k0 < nsrc; k0 += G) {
    int64_t base[G];
    bool use[G];
    static_for<0, G>([&](auto jc) __attribute__((always_inline)) {
      constexpr int j = decltype(jc)::value;
      const int k = k0 + j;
      use[j] = false;
      base[j] = 0;
      if (k < nsrc) {
        const int tok = ld_const(ev.tokens, r * K + k);
        int64_t row = -1;
        if (text) {
          if (ev.E_text && tok >= 0 && tok < ev.V_text) row = tok;
        } else if (tok == ev.pad_id) {
          row = (int64_t)k * (ev.V + 1) + ev.V;
        } else if (tok >= 0 && tok < ev.V) {
          row = (int64_t)k * (ev.V + 1) + tok;
        }
        bad |= row < 0;
        use[j] = row >= 0;
        base[j] = row < 0 ? 0 : row * H;
      }
    });
    if (vec) {
      u32x4 v[G];
      static_for<0, G>([&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value;
        v[j] = u32x4{0u, 0u, 0u, 0u};
        if (use[j]) {
          const char *p = static_cast<const char *>(tab) + (base[j] + h0) * (BF16 ? 2 : 4);
          v[j] = *reinterpret_cast<const u32x4 *>(p);
        }
      });
      static_for<0, G>([&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if constexpr (BF16) {
            acc[2 * w] += (double)__uint_as_float(v[j][w] << 16);
            acc[2 * w + 1] += (double)__uint_as_float(v[j][w] & 0xFFFF0000u);
          } else {
            acc[w] += (double)__uint_as_float(v[j][w]);
          }
        }
      });
    } else {
      static_for<0, G>([&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value;
        if (use[j]) {
#pragma unroll
          for (int e = 0; e < VEC; ++e)
            if (h0 + e < H) acc[e] += elem_f64<BF16>(tab, base[j] + h0 + e);
        }
      });
    }
  }
  if (bad && blockIdx.y == 0 && threadIdx.x == 0 && ev.status)
    atomicOr(ev.status, (uint32_t)MCD_DEV_BAD_TOKEN);
  if (h0 >= H) return;
  const int64_t o = (int64_t)r * H + h0;
  if (vec) {
    u32x4 w;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if constexpr (BF16) {
        w[q] = bad ? 0u : (bf16_bits_from_f64(acc[2 * q]) | (bf16_bits_from_f64(acc[2 * q + 1]) << 16));
      } else {
        w[q] = bad ? 0u : __float_as_uint((float)acc[q]);
      }
    }
    *reinterpret_cast<u32x4 *>(static_cast<char *>(ev.out) + o * (BF16 ? 2 : 4)) = w;
  } else {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      if (h0 + e >= H) break;
      if constexpr (BF16) {
        static_cast<uint16_t *>(ev.out)[o + e] = bad ? 0 : (uint16_t)bf16_bits_from_f64(acc[e]);
      } else {
        static_cast<float *>(ev.out)[o + e] = bad ? 0.0f : (float)acc[e];
      }
    }
  }
}

}  // namespace

hipError_t launch_next_input(const EmbedView &ev, bool bf16, hipStream_t st) {
  const int vec = bf16 ? 8 : 4;
  const int per_block = 256 * vec;
  const dim3 grid((unsigned)ev.R, (unsigned)((ev.H + per_block - 1) / per_block));
  if (bf16) hipLaunchKernelGGL(next_input_kernel<true>, grid, dim3(256), 0, st, ev);
  else hipLaunchKernelGGL(next_input_kernel<false>, grid, dim3(256), 0, st, ev);
  return hipGetLastError();
}

}  // namespace mcd
