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
// Weight-streaming path for up to 128 rows, staged with direct global->LDS
// loads.  A workgroup owns all BM rows and BN columns.  Each k slice of SK = 64
// (128 bytes of every weight and hidden row) is copied into one of S LDS
// stages by global_load_lds_dwordx4 (64 lanes x 16 B, eight 128-byte row
// segments per instruction), S - 1 slices ahead of its use, without passing
// through registers.  Waves split the tile 2 x 2: column half (w & 1) and the
// k32 half (w >> 1) of every slice; the two k halves meet in LDS at the end.
//
// LDS layout of a slice: [rows][8 chunks of 16 B]; chunk c of row r is stored
// at position c ^ ((r >> 1) & 7), so the 16 rows of an MFMA fragment read hit
// 16 distinct bank groups.  The loop waits for the copies explicitly (vector
// memory counter: only these copies are outstanding in the loop); slices past
// the end re-load the last slice (clamped) so that every iteration issues the
// same count, and a copy only ever targets the stage read S - 1 iterations
// earlier, after a barrier that follows every wave's reads of it.
constexpr int kDmaSK = 64;                 // k per slice
constexpr int kDmaLdsBudget = 144 * 1024;  // bytes of LDS for the two rings

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
// rows (out -1: no such row).
__device__ inline float4 pair_params(const StepView &sv, const int32_t *rows, int g0) {
  float4 pr = make_float4(0.0f, 1.0f, __int_as_float(-1), __int_as_float(-1));
  if (g0 < 2 * sv.n_pairs) {
    const int r = rows[g0];
    if (r >= 0 && r < sv.R) {
      const float T = sv.temperature[r];
      pr = make_float4(sv.cfg_w[r], T > 0.0f ? 1.0f / T : 1.0f, __int_as_float(g0 >> 1),
                       __int_as_float(-2));
    }
    return pr;
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int g = g0 + h;
    if (g < sv.Mg) {
      const int r = rows[g];
      if (r >= 0 && r < sv.R) {
        const float T = sv.temperature[r];
        const float it = T > 0.0f ? 1.0f / T : 1.0f;
        const int out = sv.n_pairs + (g - 2 * sv.n_pairs);
        if (h == 0) {
          pr.x = it;
          pr.z = __int_as_float(out);
        } else {
          pr.y = it;
          pr.w = __int_as_float(out);
        }
      }
    }
  }
  return pr;
}

// Second phase of the LDS epilogue of a BM x BN tile whose sums sit in C
// (pitch CP floats; NH = 2: two k-half arrays BM * CP apart, added here).
// Audio: each thread owns a fixed 4-column chunk and walks row pairs, adds the
// bias, applies the CFG merge (Eq. 1) and 1/T, and stores 16 bytes per output
// row.  Text: each thread scans whole 32-column parts of rows and writes the
// (max, lowest argmax) partials.  Starts with a workgroup barrier.
template <int BM, int BN, int CP, bool TEXT, int NH>
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
    constexpr int ITEMS = (BM / 2) * CH / 256;
    static_assert(ITEMS >= 1 && (BM / 2) * CH % 256 == 0, "whole items per thread");
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
        *reinterpret_cast<floatx4 *>(dst) = v;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (nc + e < N) dst[e] = v[e];
      }
    };
#pragma unroll
    for (int it = 0; it < ITEMS; ++it) {
      const int q = (it * 256 + tid) / CH;
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
    for (int item = tid; item < BM * PPR; item += 256) {
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

template <int BM, int BN, bool TEXT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void head_gemm_dma(
    HeadView hv, StepView sv) {
  constexpr int SK = kDmaSK;
  constexpr int MB = BM / 32;              // 32-row MFMA blocks: all rows of the tile
  constexpr int WN = BN / 2;               // columns per wave
  constexpr int NB = WN / 32;              // 32-column MFMA blocks per wave
  constexpr int ROWB = SK * 2;             // bytes of one row segment (128)
  constexpr int WST = BN * ROWB, AST = BM * ROWB;
  // Waves 0-1 copy weight slices, waves 2-3 hidden-state slices.  Vector
  // memory operations of one wave complete in issue order, so a wave that
  // issued only weight copies can keep SW - 1 of them in flight without
  // waiting behind the (faster, L2-resident) hidden-state copies.
  constexpr int SA = 3;                                           // hidden-state stages
  constexpr int SW0 = (kDmaLdsBudget - SA * AST) / WST;
  constexpr int SW = SW0 > 8 ? 8 : SW0;                           // weight stages
  constexpr int WIW = WST / 1024 / 2;      // copy instructions per weight wave per slice
  constexpr int AIA = AST / 1024 / 2;      // per hidden-state wave per slice
  static_assert(SW >= 3 && WIW >= 1 && AIA >= 1 && MB >= 1 && NB >= 1, "tile shape");
  static_assert((SW - 2) * WIW < 64 && (SA - 2) * AIA < 64, "vmcnt range");

  __shared__ __attribute__((aligned(1024))) char lds[SW * WST + SA * AST];
  char *const wring = lds;                 // weight stages
  char *const aring = lds + SW * WST;      // hidden-state stages
  // per pair of GEMM rows (2q, 2q + 1): {w, 1/T, out, -2} for a CFG pair,
  // {1/T_0, 1/T_1, out_0, out_1} for two solo rows (out -1: no row)
  __shared__ float4 rowp[BM / 2];

  const int32_t *rows = sv.plan + kPlanHeader + (TEXT ? sv.Mg : 0);
  const int M = TEXT ? sv.n_text : sv.Mg;
  const int N = TEXT ? hv.V_text : hv.N;
  const __bf16 *Wp = static_cast<const __bf16 *>(TEXT ? hv.W_text : hv.W);
  const __bf16 *X = static_cast<const __bf16 *>(sv.hidden);
  const int H = hv.H;
  const int NST = H / SK;

  const int tiles_m = (M + BM - 1) / BM;
  const int tile_m = blockIdx.x % tiles_m;
  const int tile_n = blockIdx.x / tiles_m;
  const int m0 = tile_m * BM, n0 = tile_n * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ch = wave & 1, kh = wave >> 1;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const bool w_copier = wave_s < 2;        // wave-uniform role

  // Each tile walks the k slices starting at its own offset, so that at any
  // moment the workgroups read different offsets of their (8 KiB-strided)
  // weight rows and spread over the HBM channels instead of all hitting the
  // same ones.  The sum order per tile is fixed, so results stay deterministic.
  const int kskew = (int)(((unsigned)tile_n * 7u) % (unsigned)NST);
  const uint32_t wbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)wring;
  const uint32_t abase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)aring;
  const int seg_r = lane >> 3, seg_c = lane & 7;

  // Per-lane global sources of this wave's copy instructions (chunk-swizzled):
  // a weight wave copies rows (wave * WIW + q) * 8 .. +7 of the tile, a
  // hidden-state wave rows ((wave - 2) * AIA + q) * 8 .. +7.
  constexpr int QN = WIW > AIA ? WIW : AIA;
  const __bf16 *src[QN];
  // copy slice st (clamped to the last one) into its stage
  auto issue_w = [&](int st) __attribute__((always_inline)) {
    int ks = min(st, NST - 1) + kskew;
    ks = ks >= NST ? ks - NST : ks;
    const uint32_t sb = wbase + (uint32_t)((st % SW) * WST);
    static_for<0, WIW>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      lds_copy16_stream(src[q] + ks * SK, sb + (uint32_t)((wave_s * WIW + q) * 1024));
    });
  };
  auto issue_a = [&](int st) __attribute__((always_inline)) {
    int ks = min(st, NST - 1) + kskew;
    ks = ks >= NST ? ks - NST : ks;
    const uint32_t sb = abase + (uint32_t)((st % SA) * AST);
    static_for<0, AIA>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      lds_copy16(src[q] + ks * SK, sb + (uint32_t)(((wave_s - 2) * AIA + q) * 1024));
    });
  };

  // The weight waves start streaming at once: their copies depend on nothing
  // but the tile, and nothing else is outstanding in their counters until the
  // end of the loop.
  wait_vmem_and_lds<0>();
  if (w_copier) {
    static_for<0, QN>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      src[q] = nullptr;
      if (q < WIW) {
        const int r = (wave_s * WIW + q) * 8 + seg_r;
        const int n = min(n0 + r, N - 1);
        src[q] = Wp + (size_t)n * H + ((seg_c ^ ((r >> 1) & 7)) * 8);
      }
    });
#pragma unroll
    for (int st = 0; st < SW - 1; ++st) issue_w(st);
  }

  if (!plan_ok(sv)) {
    wait_vmem_and_lds<0>();  // no copy may still be landing in this workgroup's LDS
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }

  if (!w_copier) {
    // The hidden-state waves gather their rows through the plan, stage the
    // per-row epilogue parameters in LDS, and wait for all of it before their
    // first copy, so that only copies are outstanding in their loop counters.
    static_for<0, QN>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      src[q] = nullptr;
      if (q < AIA) {
        const int r = ((wave_s - 2) * AIA + q) * 8 + seg_r;
        int pr = rows[min(m0 + r, M - 1)];
        if (pr < 0 || pr >= sv.R) {
          atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
          pr = 0;
        }
        src[q] = X + (size_t)pr * H + ((seg_c ^ ((r >> 1) & 7)) * 8);
      }
    });
    const int q2 = tid - 128;
    if (!TEXT && q2 < BM / 2) rowp[q2] = pair_params(sv, rows, m0 + 2 * q2);
    wait_vmem_and_lds<0>();
#pragma unroll
    for (int st = 0; st < SA - 1; ++st) issue_a(st);
  }

  floatx16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Fragment byte offsets within a stage.  v_mfma_f32_32x32x16_bf16: lane l
  // holds row (or column) l % 32 and the 8 consecutive k of chunk l / 32 of the
  // k16 step; this wave covers k32 half kh of the slice (chunks 4kh .. 4kh+3).
  const int frow = lane & 31;
  int aoff[2][MB], woff[2][NB];
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const int c = 4 * kh + 2 * s2 + (lane >> 5);
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      const int r = i * 32 + frow;
      aoff[s2][i] = r * ROWB + ((c ^ ((r >> 1) & 7)) * 16);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int r = ch * WN + j * 32 + frow;
      woff[s2][j] = r * ROWB + ((c ^ ((r >> 1) & 7)) * 16);
    }
  }

  for (int st = 0; st < NST; ++st) {
    // this wave's copies of slice st have landed and its reads of slice st - 1
    // are done; the barrier extends both to the whole workgroup
    if (w_copier) wait_vmem_and_lds<(SW - 2) * WIW>();
    else wait_vmem_and_lds<(SA - 2) * AIA>();
    block_barrier_no_vmem_wait();
    if (w_copier) issue_w(st + SW - 1);
    else issue_a(st + SA - 1);
    const char *wsb = wring + (st % SW) * WST;
    const char *asb = aring + (st % SA) * AST;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      bf16x8 a[MB], b[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i) a[i] = *reinterpret_cast<const bf16x8 *>(asb + aoff[s2][i]);
#pragma unroll
      for (int j = 0; j < NB; ++j) b[j] = *reinterpret_cast<const bf16x8 *>(wsb + woff[s2][j]);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
  // the copies are invisible to the compiler: drain them before reusing LDS
  wait_vmem_and_lds<0>();
  __syncthreads();

  // Epilogue, in two phases through LDS (the rings are free now).
  // Phase 1: every wave writes its partial sums (its k half) to C[kh][row][col].
  // Phase 2: each thread takes 16-byte column chunks (audio) or 32-column text
  // parts of whole rows, adds the two k halves (a two-term sum: order-free),
  // and applies the fused epilogue with coalesced stores.  No global load is
  // left pending among the stores, so they never wait for each other.
  constexpr int CP = BN + 4;               // padded row pitch of C (floats)
  static_assert(2 * BM * CP * 4 <= SW * WST + SA * AST, "C fits the rings");
  float *C = reinterpret_cast<float *>(lds);
  static_for<0, MB * NB * 16>([&](auto fc) __attribute__((always_inline)) {
    constexpr int f = decltype(fc)::value;
    constexpr int i = f / (NB * 16), j = (f / 16) % NB, r = f % 16;
    const int row = i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
    C[(kh * BM + row) * CP + ch * WN + j * 32 + frow] = acc[i][j][r];
  });

  epilogue_from_lds<BM, BN, CP, TEXT, 2>(hv, sv, C, rowp, m0, n0, M, N);
}

// ---------------------------------------------------------------------------
// MFMA-regime path for more than 128 GEMM rows (bf16, H a multiple of 32).
// A workgroup owns a 256 x 128 output tile.  The waves split it by row half
// (wm = wave & 1) and k half (kh = wave >> 1): each wave accumulates a
// 128 x 128 block (4 x 4 blocks of v_mfma_f32_32x32x16_bf16, 256 accumulator
// registers) over its 16 k of every 32-k slice, so each MFMA costs half a
// fragment of LDS reads.  Slices are copied global->LDS like the streaming
// path: waves 0-1 copy weight slices into a deep ring (the weights come from
// HBM, once per XCD), waves 2-3 copy hidden-state slices into a shorter one
// (they are re-read from L2).  A slice row is 64 bytes, 4 chunks of 16 B;
// chunk c of row r is stored at position c ^ ((r >> 2) & 3), so the 16 rows
// of a 16-lane fragment read group hit all 64 banks once.
//
// Tile order is XCD-aware: workgroups are dealt to the 8 XCDs in turn, so the
// grid index is remapped to give each XCD a contiguous run of tiles, in which
// the row tiles of a column tile are neighbours and run at the same time:
// they share that column's weights through the XCD's L2.
constexpr int kMfmaBM = 256, kMfmaBN = 128, kMfmaSK = 32;
constexpr int kMfmaSA = 5, kMfmaSB = 8;

template <bool TEXT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void head_gemm_mfma(
    HeadView hv, StepView sv) {
  constexpr int BM = kMfmaBM, BN = kMfmaBN, SK = kMfmaSK;
  constexpr int SA = kMfmaSA, SB = kMfmaSB;
  constexpr int ROWB = SK * 2;                       // 64 bytes per row and slice
  constexpr int AST = BM * ROWB, BST = BN * ROWB;    // 16 KiB, 8 KiB per stage
  constexpr int AIA = AST / 1024 / 2, BIB = BST / 1024 / 2;  // copies per wave per slice
  constexpr int MB = 4, NB = 4;                      // 32x32 blocks per wave
  static_assert((SA - 1) * AIA < 64 && (SB - 1) * BIB < 64, "vmcnt range");
  // both copy roles keep the same number of copies in flight in the loop, so
  // that its one wait needs no branch (a branch makes the compiler's own
  // LDS-read waits conservative)
  constexpr int kLoopVm = (SA - 2) * AIA;
  static_assert((SB - 2) * BIB == kLoopVm, "equal in-flight copy counts");
  static_assert(MB * NB == 16 && AIA == 8 && BIB == 4, "copy slots of the slice schedule");
  constexpr int CP = BN + 4;                         // epilogue row pitch (floats)
  static_assert(BM * CP * 4 <= SA * AST + SB * BST, "epilogue tile fits the rings");

  __shared__ __attribute__((aligned(1024))) char lds[SA * AST + SB * BST];
  char *const aring = lds;
  char *const bring = lds + SA * AST;
  __shared__ float4 rowp[BM / 2];

  const int32_t *rows = sv.plan + kPlanHeader + (TEXT ? sv.Mg : 0);
  const int M = TEXT ? sv.n_text : sv.Mg;
  const int N = TEXT ? hv.V_text : hv.N;
  const __bf16 *Wp = static_cast<const __bf16 *>(TEXT ? hv.W_text : hv.W);
  const __bf16 *X = static_cast<const __bf16 *>(sv.hidden);
  const int H = hv.H;
  const int NST = H / SK;

  const int tiles_m = (M + BM - 1) / BM;
  int bx = blockIdx.x;
  if (gridDim.x % 8 == 0) bx = (bx % 8) * (gridDim.x / 8) + bx / 8;
  const int tile_m = bx % tiles_m, tile_n = bx / tiles_m;
  const int m0 = tile_m * BM, n0 = tile_n * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, kh = wave >> 1;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const bool b_copier = wave_s < 2;

  // the row tiles of one column tile walk k in the same order (they share the
  // weights in L2); different column tiles start at different k
  const int kskew = (int)(((unsigned)tile_n * 7u) % (unsigned)NST);
  const uint32_t abase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)aring;
  const uint32_t bbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)bring;
  // one copy instruction: 16 rows x 4 chunks; lane i -> row i / 4, position i % 4
  const int seg_r = lane >> 2, seg_p = lane & 3;
  constexpr int QN = AIA > BIB ? AIA : BIB;
  const __bf16 *src[QN];
  auto issue_b = [&](int st) __attribute__((always_inline)) {
    int ks = min(st, NST - 1) + kskew;
    ks = ks >= NST ? ks - NST : ks;
    const uint32_t sb = bbase + (uint32_t)((st % SB) * BST);
    static_for<0, BIB>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      lds_copy16(src[q] + ks * SK, sb + (uint32_t)((wave_s * BIB + q) * 1024));
    });
  };
  auto issue_a = [&](int st) __attribute__((always_inline)) {
    int ks = min(st, NST - 1) + kskew;
    ks = ks >= NST ? ks - NST : ks;
    const uint32_t sb = abase + (uint32_t)((st % SA) * AST);
    static_for<0, AIA>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      lds_copy16(src[q] + ks * SK, sb + (uint32_t)(((wave_s - 2) * AIA + q) * 1024));
    });
  };

  wait_vmem_and_lds<0>();
  if (b_copier) {
    static_for<0, QN>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      src[q] = nullptr;
      if (q < BIB) {
        const int r = (wave_s * BIB + q) * 16 + seg_r;
        const int n = min(n0 + r, N - 1);
        src[q] = Wp + (size_t)n * H + ((seg_p ^ ((r >> 2) & 3)) * 8);
      }
    });
#pragma unroll
    for (int st = 0; st < SB; ++st) issue_b(st);
  }

  if (!plan_ok(sv)) {
    wait_vmem_and_lds<0>();  // no copy may still be landing in this workgroup's LDS
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }

  if (!b_copier) {
    static_for<0, QN>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      src[q] = nullptr;
      if (q < AIA) {
        const int r = ((wave_s - 2) * AIA + q) * 16 + seg_r;
        int pr = rows[min(m0 + r, M - 1)];
        if (pr < 0 || pr >= sv.R) {
          atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
          pr = 0;
        }
        src[q] = X + (size_t)pr * H + ((seg_p ^ ((r >> 2) & 3)) * 8);
      }
    });
    const int q2 = tid - 128;
    if (!TEXT) rowp[q2] = pair_params(sv, rows, m0 + 2 * q2);
    wait_vmem_and_lds<0>();
#pragma unroll
    for (int st = 0; st < SA; ++st) issue_a(st);
  }

  floatx16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // fragment offsets: lane l holds row (column) l % 32 and chunk 2 kh + l / 32
  const int frow = lane & 31;
  const int fch = 2 * kh + (lane >> 5);
  int aoff[MB], boff[NB];
#pragma unroll
  for (int i = 0; i < MB; ++i) {
    const int r = wm * 128 + i * 32 + frow;
    aoff[i] = r * ROWB + ((fch ^ ((r >> 2) & 3)) * 16);
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int r = j * 32 + frow;
    boff[j] = r * ROWB + ((fch ^ ((r >> 2) & 3)) * 16);
  }

  // Software pipeline: the fragments of slice st + 1 are read from LDS while
  // the MFMAs of slice st run on the registers read one iteration earlier.
  // At the top of iteration st every wave waits for its copies of slice st + 1
  // and for its own fragment reads of slice st; the barrier extends both to the
  // workgroup, so the stage of slice st is free for slice st + S (A: S = SA,
  // B: S = SB), which is issued right after it.  Slices past the end re-load
  // the last one (clamped), so every iteration issues the same count.
  bf16x8 fa0[MB], fb0[NB], fa1[MB], fb1[NB];
  auto read_frags = [&](int st, bf16x8 (&fa)[MB], bf16x8 (&fb)[NB])
      __attribute__((always_inline)) {
    const char *asb = aring + (st % SA) * AST;
    const char *bsb = bring + (st % SB) * BST;
#pragma unroll
    for (int i = 0; i < MB; ++i) fa[i] = *reinterpret_cast<const bf16x8 *>(asb + aoff[i]);
#pragma unroll
    for (int j = 0; j < NB; ++j) fb[j] = *reinterpret_cast<const bf16x8 *>(bsb + boff[j]);
  };
  // One slice: its 16 MFMAs, with the 8 fragment reads of the next slice and
  // this wave's copies (A: 8 per slice, B: 4) spread between them, so that the
  // MFMA pipe, the LDS and the load path (the per-CU limit here: a slice moves
  // 24 KiB) all work at once instead of in turn.
  auto step = [&](int st, bf16x8 (&fa)[MB], bf16x8 (&fb)[NB], bf16x8 (&na)[MB],
                  bf16x8 (&nb)[NB]) __attribute__((always_inline)) {
    wait_vmem_and_lds<kLoopVm>();
    block_barrier_no_vmem_wait();
    const int cst = st + (b_copier ? SB : SA);   // slice this wave copies now
    int ks = min(cst, NST - 1) + kskew;
    ks = ks >= NST ? ks - NST : ks;
    const uint32_t csb = b_copier ? bbase + (uint32_t)((cst % SB) * BST)
                                  : abase + (uint32_t)((cst % SA) * AST);
    const int st1 = st + 1;   // past the end: a clamped slice, never used
    const char *asb = aring + (st1 % SA) * AST;
    const char *bsb = bring + (st1 % SB) * BST;
    static_for<0, MB * NB>([&](auto mc) __attribute__((always_inline)) {
      constexpr int m = decltype(mc)::value;
      constexpr int i = m / NB, j = m % NB;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      if constexpr (m < MB) na[m] = *reinterpret_cast<const bf16x8 *>(asb + aoff[m]);
      else if constexpr (m < MB + NB) nb[m - MB] = *reinterpret_cast<const bf16x8 *>(bsb + boff[m - MB]);
      if constexpr (m % 2 == 1) {
        constexpr int q = m / 2;           // A copies 0..7 after the odd MFMAs
        if (!b_copier) lds_copy16(src[q] + ks * SK, csb + (uint32_t)(((wave_s - 2) * AIA + q) * 1024));
      }
      if constexpr (m % 4 == 3) {
        constexpr int q = m / 4;           // B copies 0..3 after every fourth
        if (b_copier) lds_copy16(src[q] + ks * SK, csb + (uint32_t)((wave_s * BIB + q) * 1024));
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  // slice 0: landed (all but SA - 1 / SB - 1 newer slices), then its fragments
  if (b_copier) wait_vmem_and_lds<(SB - 1) * BIB>();
  else wait_vmem_and_lds<(SA - 1) * AIA>();
  block_barrier_no_vmem_wait();
  read_frags(0, fa0, fb0);
  for (int st = 0; st < NST; st += 2) {   // NST is even (H % 64 == 0)
    step(st, fa0, fb0, fa1, fb1);
    step(st + 1, fa1, fb1, fa0, fb0);
  }
  wait_vmem_and_lds<0>();
  __syncthreads();

  // Epilogue through LDS: the k-half-1 waves store their sums in C[row][col],
  // the k-half-0 waves add theirs in place (a two-term sum: order-free), then
  // every thread applies the fused epilogue to 16-byte column chunks.
  float *C = reinterpret_cast<float *>(lds);
  // element (i, j, r) of this lane sits at Cl + a compile-time offset
  float *Cl = C + (wm * 128 + (lane >> 5) * 4) * CP + frow;
  if (kh == 1) {
    static_for<0, MB * NB * 16>([&](auto fc) __attribute__((always_inline)) {
      constexpr int f = decltype(fc)::value;
      constexpr int i = f / (NB * 16), j = (f / 16) % NB, r = f % 16;
      constexpr int off = (i * 32 + (r >> 2) * 8 + (r & 3)) * CP + j * 32;
      Cl[off] = acc[i][j][r];
    });
  }
  __syncthreads();
  if (kh == 0) {
    static_for<0, MB * NB * 16>([&](auto fc) __attribute__((always_inline)) {
      constexpr int f = decltype(fc)::value;
      constexpr int i = f / (NB * 16), j = (f / 16) % NB, r = f % 16;
      constexpr int off = (i * 32 + (r >> 2) * 8 + (r & 3)) * CP + j * 32;
      Cl[off] = acc[i][j][r] + Cl[off];
    });
  }
  epilogue_from_lds<BM, BN, CP, TEXT, 1>(hv, sv, C, rowp, m0, n0, M, N);
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

template <bool TEXT>
hipError_t launch_mfma(const HeadView &hv, const StepView &sv, int M, int N, hipStream_t st) {
  const int tm = (M + kMfmaBM - 1) / kMfmaBM, tn = (N + kMfmaBN - 1) / kMfmaBN;
  hipLaunchKernelGGL((head_gemm_mfma<TEXT>), dim3(tm * tn), dim3(256), 0, st, hv, sv);
  return hipGetLastError();
}

template <int BM, int BN, bool TEXT>
hipError_t launch_dma(const HeadView &hv, const StepView &sv, int M, int N, hipStream_t st) {
  const int tm = (M + BM - 1) / BM, tn = (N + BN - 1) / BN;
  hipLaunchKernelGGL((head_gemm_dma<BM, BN, TEXT>), dim3(tm * tn), dim3(256), 0, st, hv, sv);
  return hipGetLastError();
}

// Weight-streaming launch for M <= 128 rows: 128-column tiles, or 64 when that
// leaves fewer workgroups than compute units.
template <bool TEXT>
hipError_t launch_skinny(const HeadView &hv, const StepView &sv, int M, int N, hipStream_t st) {
  const bool narrow = (N + 127) / 128 < 256;
  if (M <= 32) return narrow ? launch_dma<32, 64, TEXT>(hv, sv, M, N, st) : launch_dma<32, 128, TEXT>(hv, sv, M, N, st);
  if (M <= 64) return narrow ? launch_dma<64, 64, TEXT>(hv, sv, M, N, st) : launch_dma<64, 128, TEXT>(hv, sv, M, N, st);
  return narrow ? launch_dma<128, 64, TEXT>(hv, sv, M, N, st) : launch_dma<128, 128, TEXT>(hv, sv, M, N, st);
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
    if (sv.Mg <= 128) e = launch_skinny<false>(hv, sv, sv.Mg, hv.N, st);
    else e = launch_mfma<false>(hv, sv, sv.Mg, hv.N, st);
  }
  if (e == hipSuccess && sv.n_text > 0) {
    if (sv.n_text <= 128) e = launch_skinny<true>(hv, sv, sv.n_text, hv.V_text, st);
    else e = launch_mfma<true>(hv, sv, sv.n_text, hv.V_text, st);
  }
  return e;
}

}  // namespace mcd
