// K1: codebook-head projection with the CFG merge and temperature fused into
// the epilogue, and the text-head projection with a fused (max, argmax) epilogue.
//
//   logits[g][n] = sum_h hidden[row(g)][h] * W[n][h]         (Sec. 2.1, n = k*V + v)
//   pair p (GEMM rows 2p, 2p+1 = Main, Companion):
//     scores[p][n] = (w * l_main + (1 - w) * l_comp) / T    (Eq. 1, Sec. 2.4)
//   solo row j:  scores[n_pairs + j][n] = l / T;  T = 0 (greedy): no division
//   text rows:   per row and 64-column part, the largest logit and its lowest id.
//
// The unmerged logits live only in accumulator registers: a pair's two rows sit
// in the same lane (rows 4q..4q+3 of a 16x16 MFMA block belong to one lane), so
// the merge is a per-lane FMA.
#include "mcd_internal.h"

namespace mcd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ inline bool plan_ok(const StepView &sv) {
  const int32_t *p = sv.plan;
  return p[kPlanMagicWord] == kPlanMagic && p[kPlanR] == sv.R && p[kPlanPairs] == sv.n_pairs &&
         p[kPlanSolo] == sv.n_solo && p[kPlanText] == sv.n_text;
}

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

__device__ inline void better(float &bv, int &bi, float v, int i) {
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA path.  256 threads = 4 waves in a 2x2 layout; tile BM x BN; the H
// loop runs in 64-wide slices staged through LDS (double-buffered, one barrier
// per slice).  Each wave owns a (BM/2) x (BN/2) sub-tile of 16x16 MFMA blocks
// (v_mfma_f32_16x16x32_bf16: lane l holds A row l%16 / B column l%16 with 8
// consecutive k; the 4 results of a lane are rows 4*(l/16)+0..3, column l%16).
constexpr int BK = 64;
constexpr int LDK = BK + 8;  // padded LDS row (elements) against bank conflicts

template <int BM, int BN, bool TEXT>
__global__ __launch_bounds__(256) void head_gemm_bf16(HeadView hv, StepView sv) {
  constexpr int MB = BM / 32;      // 16-row blocks per wave
  constexpr int NB = BN / 32;      // 16-col blocks per wave
  constexpr int ACH = BM * BK / 8 / 256;  // 16-byte chunks per thread (A tile)
  constexpr int BCH = BN * BK / 8 / 256;  // (B tile)
  static_assert(ACH >= 1 && BCH >= 1, "tile too small");

  __shared__ __attribute__((aligned(16))) __bf16 As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[2][BN * LDK];

  if (!plan_ok(sv)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }
  const int32_t *rows = sv.plan + kPlanHeader + (TEXT ? sv.Mg : 0);
  const int M = TEXT ? sv.n_text : sv.Mg;
  const int N = TEXT ? hv.V_text : hv.N;
  const __bf16 *Wp = static_cast<const __bf16 *>(TEXT ? hv.W_text : hv.W);
  const __bf16 *X = static_cast<const __bf16 *>(sv.hidden);
  const int H = hv.H;

  const int tiles_m = (M + BM - 1) / BM;
  const int tile_m = blockIdx.x % tiles_m;
  const int tile_n = blockIdx.x / tiles_m;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // global source pointers of this thread's chunks (nullptr: zero fill)
  const __bf16 *asrc[ACH];
  const __bf16 *bsrc[BCH];
  int aoff[ACH], boff[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + 256 * i, row = c >> 3, col = (c & 7) * 8;
    const int m = m0 + row;
    asrc[i] = nullptr;
    if (m < M) {
      const int r = rows[m];
      if (r >= 0 && r < sv.R) asrc[i] = X + (size_t)r * H + col;
      else atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    }
    aoff[i] = row * LDK + col;
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int c = tid + 256 * i, row = c >> 3, col = (c & 7) * 8;
    const int n = n0 + row;
    bsrc[i] = (n < N) ? Wp + (size_t)n * H + col : nullptr;
    boff[i] = row * LDK + col;
  }

  uint4 areg[ACH], breg[BCH];
  auto load = [&](int kt) {
#pragma unroll
    for (int i = 0; i < ACH; ++i)
      areg[i] = asrc[i] ? *reinterpret_cast<const uint4 *>(asrc[i] + kt * BK) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < BCH; ++i)
      breg[i] = bsrc[i] ? *reinterpret_cast<const uint4 *>(bsrc[i] + kt * BK) : make_uint4(0, 0, 0, 0);
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) *reinterpret_cast<uint4 *>(&As[buf][aoff[i]]) = areg[i];
#pragma unroll
    for (int i = 0; i < BCH; ++i) *reinterpret_cast<uint4 *>(&Bs[buf][boff[i]]) = breg[i];
  };

  floatx4 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int KT = H / BK;
  load(0);
  store(0);
  __syncthreads();
  const int frow = lane & 15, fk = (lane >> 4) * 8;
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) load(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 a[MB], b[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i)
        a[i] = *reinterpret_cast<const bf16x8 *>(
            &As[buf][(wm * (BM / 2) + i * 16 + frow) * LDK + ks * 32 + fk]);
#pragma unroll
      for (int j = 0; j < NB; ++j)
        b[j] = *reinterpret_cast<const bf16x8 *>(
            &Bs[buf][(wn * (BN / 2) + j * 16 + frow) * LDK + ks * 32 + fk]);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) store(buf ^ 1);
    __syncthreads();
  }

  const int rq = (lane >> 4) * 4;  // first of the lane's 4 rows in a block
  if constexpr (!TEXT) {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int g = m0 + wm * (BM / 2) + i * 16 + rq;
        const int n = n0 + wn * (BN / 2) + j * 16 + frow;
        emit_audio(hv, sv, rows, g, acc[i][j][0], acc[i][j][1], n);
        emit_audio(hv, sv, rows, g + 2, acc[i][j][2], acc[i][j][3], n);
      }
  } else {
    // each wave's column half is one 64-column part
    static_assert(BN / 2 == kTextPartCols, "text parts are 64 columns");
    const int part = (n0 + wn * (BN / 2)) / kTextPartCols;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float bv = -INFINITY;
        int bi = INT32_MAX;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int n = n0 + wn * (BN / 2) + j * 16 + frow;
          if (n < N) better(bv, bi, acc[i][j][q], n);
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) {
          const float ov = __shfl_xor(bv, off);
          const int oi = __shfl_xor(bi, off);
          better(bv, bi, ov, oi);
        }
        const int g = m0 + wm * (BM / 2) + i * 16 + rq + q;
        if (frow == 0 && g < M && part < sv.text_parts) {
          sv.text_val[(size_t)g * sv.text_parts + part] = bv;
          sv.text_idx[(size_t)g * sv.text_parts + part] = bi;
        }
      }
  }
}

// ---------------------------------------------------------------------------
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
    for (int g0 = 0; g0 < M; g0 += 4) {
      const int g = g0 + y;
      float bv = -INFINITY;
      int bi = INT32_MAX;
      if (g < M && col_ok) {
        bv = dot(g);
        bi = n;
      }
      for (int off = 1; off < 64; off <<= 1) {
        const float ov = __shfl_xor(bv, off);
        const int oi = __shfl_xor(bi, off);
        better(bv, bi, ov, oi);
      }
      if (c == 0 && g < M) {
        sv.text_val[(size_t)g * sv.text_parts + blockIdx.x] = bv;
        sv.text_idx[(size_t)g * sv.text_parts + blockIdx.x] = bi;
      }
    }
  }
}

template <int BM, int BN, bool TEXT>
hipError_t launch_bf16(const HeadView &hv, const StepView &sv, int M, int N, hipStream_t st) {
  const int tm = (M + BM - 1) / BM, tn = (N + BN - 1) / BN;
  hipLaunchKernelGGL((head_gemm_bf16<BM, BN, TEXT>), dim3(tm * tn), dim3(256), 0, st, hv, sv);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_head_gemm(const HeadView &hv, const StepView &sv, hipStream_t st) {
  hipError_t e = hipSuccess;
  if (hv.dtype == MCD_F32) {
    if (sv.Mg > 0) {
      hipLaunchKernelGGL(head_gemm_f32<false>, dim3((hv.N + 63) / 64), dim3(256), 0, st, hv, sv);
      e = hipGetLastError();
    }
    if (e == hipSuccess && sv.n_text > 0) {
      hipLaunchKernelGGL(head_gemm_f32<true>, dim3((hv.V_text + 63) / 64), dim3(256), 0, st, hv,
                         sv);
      e = hipGetLastError();
    }
    return e;
  }
  if (sv.Mg > 0) {
    if (sv.Mg <= 32) e = launch_bf16<32, 64, false>(hv, sv, sv.Mg, hv.N, st);
    else if (sv.Mg <= 64) e = launch_bf16<64, 128, false>(hv, sv, sv.Mg, hv.N, st);
    else e = launch_bf16<128, 128, false>(hv, sv, sv.Mg, hv.N, st);
  }
  if (e == hipSuccess && sv.n_text > 0) {
    if (sv.n_text <= 64) e = launch_bf16<64, 128, true>(hv, sv, sv.n_text, hv.V_text, st);
    else e = launch_bf16<128, 128, true>(hv, sv, sv.n_text, hv.V_text, st);
  }
  return e;
}

}  // namespace mcd
