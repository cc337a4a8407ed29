// Device helpers shared by the bf16 head-projection kernels (streaming and
// MFMA-regime paths): register vector types, compile-time loops, plan check,
// global->LDS copies with explicit waits, and the fused epilogue that turns a
// tile of sums staged in LDS into merged, temperature-divided scores (Eq. 1,
// Sec. 2.4) or text-head (max, lowest argmax) partials.
#pragma once

#include <type_traits>

#include "mcd_internal.h"

namespace mcd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // 16-byte chunk in registers

// Compile-time loop: f(integral_constant<int, I>) for I in [B, E).  Register
// arrays indexed only through it keep literal indices from the first
// optimisation pass on, so they are never demoted to scratch or LDS.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Uniform load through the constant address space: a scalar load, counted
// apart from the vector-memory counter, so it never waits for the global->LDS
// copies in flight.  Only for buffers that no kernel writes while it runs.
template <typename T>
__device__ __forceinline__ T ld_const(const T *p, int i) {
  return ((const __attribute__((address_space(4))) T *)p)[i];
}

// The plan header matches the step.  Scalar loads, every word read (no
// short-circuit), so that they go out together.
__device__ inline bool plan_ok(const StepView &sv) {
  const int32_t *p = sv.plan;
  const bool magic = ld_const(p, kPlanMagicWord) == kPlanMagic;
  const bool r = ld_const(p, kPlanR) == sv.R, pairs = ld_const(p, kPlanPairs) == sv.n_pairs;
  const bool solo = ld_const(p, kPlanSolo) == sv.n_solo, text = ld_const(p, kPlanText) == sv.n_text;
  return magic & r & pairs & solo & text;
}

__device__ inline void better(float &bv, int &bi, float v, int i) {
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

// s_waitcnt immediate: at most n outstanding vector-memory operations and no
// outstanding LDS operation (gfx9 encoding; export counter left free).
template <int n>
__device__ __forceinline__ void wait_vmem_and_lds() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  constexpr int imm = (n & 0xF) | (0x7 << 4) | (0x0 << 8) | (((n >> 4) & 3) << 14);
  __builtin_amdgcn_s_waitcnt(imm);
}

// 16-byte global->LDS copy per lane: lane i's 16 bytes land at LDS byte
// address lds_base + 16 * i (lds_base is wave-uniform and goes to M0).  Issued
// as inline assembly so that the compiler does not insert its own conservative
// waits for it; the kernel waits for these copies explicitly.
__device__ __forceinline__ void lds_copy16(const void *src, uint32_t lds_base) {
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(lds_base) : "memory");
}

// The same copy with the non-temporal hint, for data read exactly once (the
// weights): it is not kept in L2 at the expense of the hidden states, which
// every workgroup re-reads.
__device__ __forceinline__ void lds_copy16_stream(const void *src, uint32_t lds_base) {
  asm volatile("global_load_lds_dwordx4 %0, off nt" ::"v"(src), "{m0}"(lds_base) : "memory");
}

// Workgroup barrier that does not wait for outstanding global->LDS copies
// (__syncthreads would drain them all); compiler-only fences keep memory
// accesses on their side of it.
__device__ __forceinline__ void block_barrier_no_vmem_wait() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Epilogue parameters of GEMM rows g0 (even) and g0 + 1: {w, 1/T, out, -2} for
// a CFG pair (the Main row carries w and T), {1/T0, 1/T1, out0, out1} for solo
// rows (out -1: no such row).  In two halves: the loads (at clamped indices,
// no branch on the loaded parameters, so nothing waits for them yet), and the
// arithmetic, which may come much later.
struct PairLoads {
  float w, t0, t1;
  int g0;
  bool ok0, ok1;
};

// r0, r1: the plan rows of GEMM rows g0 and g0 + 1 (each index clamped to Mg - 1)
__device__ inline PairLoads pair_params_load(const StepView &sv, int g0, int r0, int r1) {
  const bool pair = g0 < 2 * sv.n_pairs;
  const bool ok0 = g0 < sv.Mg && r0 >= 0 && r0 < sv.R;
  const bool ok1 = !pair && g0 + 1 < sv.Mg && r1 >= 0 && r1 < sv.R;
  const int c0 = ok0 ? r0 : 0, c1 = ok1 ? r1 : 0;
  return PairLoads{sv.cfg_w[c0], sv.temperature[c0], sv.temperature[c1], g0, ok0, ok1};
}

__device__ inline float4 pair_params_finish(const StepView &sv, const PairLoads &p) {
  auto inv = [](float T) __attribute__((always_inline)) { return T > 0.0f ? 1.0f / T : 1.0f; };
  float4 pr = make_float4(0.0f, 1.0f, __int_as_float(-1), __int_as_float(-1));
  if (p.g0 < 2 * sv.n_pairs) {
    if (p.ok0) pr = make_float4(p.w, inv(p.t0), __int_as_float(p.g0 >> 1), __int_as_float(-2));
    return pr;
  }
  const int out0 = sv.n_pairs + (p.g0 - 2 * sv.n_pairs);
  if (p.ok0) {
    pr.x = inv(p.t0);
    pr.z = __int_as_float(out0);
  }
  if (p.ok1) {
    pr.y = inv(p.t1);
    pr.w = __int_as_float(out0 + 1);
  }
  return pr;
}

__device__ inline float4 pair_params(const StepView &sv, const int32_t *rows, int g0) {
  const int r0 = rows[min(g0, sv.Mg - 1)], r1 = rows[min(g0 + 1, sv.Mg - 1)];
  return pair_params_finish(sv, pair_params_load(sv, g0, r0, r1));
}

// Second phase of the LDS epilogue of a BM x BN tile whose sums sit in C
// (pitch CP floats; NH = 2: two k-half arrays BM * CP apart, added here).
// Audio: each thread owns a fixed 4-column chunk and walks row pairs, adds the
// bias, applies the CFG merge (Eq. 1) and 1/T, and stores 16 bytes per output
// row.  Text: each thread scans whole 32-column parts of rows and writes the
// (max, lowest argmax) partials.  Starts with a workgroup barrier.
template <int BM, int BN, int CP, bool TEXT, int NH, int NT = 256>
__device__ __forceinline__ void epilogue_from_lds(const HeadView &hv, const StepView &sv,
                                                  const float *C, const float4 *rowp, int m0,
                                                  int n0, int M, int N) {
  const int tid = threadIdx.x;
  auto sum4 = [&](const float *p) __attribute__((always_inline)) {
    floatx4 v = *reinterpret_cast<const floatx4 *>(p);
    if constexpr (NH == 2) v = v + *reinterpret_cast<const floatx4 *>(p + BM * CP);
    return v;
  };
  if constexpr (!TEXT) {
    constexpr int CH = BN / 4;
    constexpr int ITEMS = (BM / 2) * CH / NT;
    static_assert(ITEMS >= 1 && (BM / 2) * CH % NT == 0, "whole items per thread");
    const int c = tid % CH;
    const int nc = n0 + 4 * c;
    floatx4 bias = {0.0f, 0.0f, 0.0f, 0.0f};
    if (hv.bias) {
#pragma unroll
      for (int e = 0; e < 4; ++e) bias[e] = (nc + e < N) ? hv.bias[nc + e] : 0.0f;
    }
    // no global load may stay pending among the stores below
    wait_vmem_and_lds<0>();
    __syncthreads();
    const bool vec_ok = (N % 4 == 0) && (nc + 4 <= N);
    auto put = [&](int out, const floatx4 &v) __attribute__((always_inline)) {
      float *dst = sv.scores + (size_t)out * N + nc;
      if (vec_ok) {
        // streaming store: the scores are read once, by the sampler
        __builtin_nontemporal_store(v, reinterpret_cast<floatx4 *>(dst));
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (nc + e < N) dst[e] = v[e];
      }
    };
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int q = (it * NT + tid) / CH;
      if (m0 + 2 * q >= M || nc >= N) continue;
      const float *c0 = C + (2 * q) * CP + 4 * c;
      const floatx4 v0 = sum4(c0) + bias;
      const floatx4 v1 = sum4(c0 + CP) + bias;
      const float4 pr = rowp[q];
      const int o0 = __float_as_int(pr.z), o1 = __float_as_int(pr.w);
      if (o1 == -2) {
        floatx4 s;
#pragma unroll
        for (int e = 0; e < 4; ++e) s[e] = fmaf(pr.x, v0[e], (1.0f - pr.x) * v1[e]) * pr.y;
        put(o0, s);
      } else {
        if (o0 >= 0) put(o0, v0 * pr.x);
        if (o1 >= 0) put(o1, v1 * pr.y);
      }
    }
  } else {
    static_assert(kTextPartCols == 32 && BN % 32 == 0, "text parts are 32 columns");
    constexpr int PPR = BN / 32;
    __syncthreads();
    for (int item = tid; item < BM * PPR; item += NT) {
      const int row = item / PPR, p = item % PPR;
      const int g = m0 + row;
      const int part = (n0 + 32 * p) / kTextPartCols;
      if (g >= M || part >= sv.text_parts) continue;
      const float *c0 = C + row * CP + 32 * p;
      float bv = -INFINITY;
      int bi = INT32_MAX;
#pragma unroll
      for (int x4 = 0; x4 < 8; ++x4) {
        const floatx4 v = sum4(c0 + 4 * x4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int n = n0 + 32 * p + 4 * x4 + e;
          if (n < N) better(bv, bi, v[e], n);
        }
      }
      sv.text_val[(size_t)g * sv.text_parts + part] = bv;
      sv.text_idx[(size_t)g * sv.text_parts + part] = bi;
    }
  }
}

}  // namespace
}  // namespace mcd
