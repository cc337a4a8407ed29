// K2: selection and draw for every (sampled row, codebook) vector, one
// 256-thread workgroup each, plus the greedy reduction of the text-head partials.
//
// Per audio vector (row r, codebook k, step t = step[r]):
//   * delay pattern (Sec. 2.1): frame f = t - d_k; no frame (f < 0, or the
//     drain f >= n_frames of Sec. 2.3) -> pad id, nothing sampled;
//   * greedy (T = 0): argmax of the merged scores, lowest id on ties;
//   * top-k: keep the k largest scores, ties at the boundary to the lowest ids;
//   * top-p: over the survivors, keep the shortest (score desc, id asc) prefix
//     whose softmax mass reaches p;
//   * Gumbel-max: token = argmax over kept ids of s_v + G_v, G_v = -log(-log u_v),
//     u_v from Philox4x64-10 with counter (v/4, k, t, rng_key), key (seed, 0),
//     word v mod 4, u = (top 23 bits + 1/2) * 2^-23; lowest id on ties;
//   * the token goes to the Main row, to its Companion (Sec. 2.4) and to the
//     request's frame grid cell [k][f].
//
// Selection is a radix select over order-preserving 32-bit keys of the fp32
// scores (four 8-bit digit passes, histograms in LDS).  Top-k histograms count
// elements; top-p histograms add fixed-point masses round(exp(s - max) * 2^48)
// as 64-bit integers, so the sums are exact and independent of the order in
// which lanes add them.
#include "mcd_internal.h"

namespace mcd {
namespace {

constexpr int kWave = 64;
constexpr double kMassScale = 281474976710656.0;  // 2^48

__device__ inline uint32_t order_key(float x) {
  if (x == 0.0f) x = 0.0f;  // -0 and +0 compare equal
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline bool plan_ok(const StepView &sv) {
  const int32_t *p = sv.plan;
  return p[kPlanMagicWord] == kPlanMagic && p[kPlanR] == sv.R && p[kPlanPairs] == sv.n_pairs &&
         p[kPlanSolo] == sv.n_solo && p[kPlanText] == sv.n_text;
}

// ---- block-level helpers (one 256-thread block per vector) ------------------
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

template <int EPL>
struct Smem {
  uint32_t hc[256];
  unsigned long long hm[256];
  unsigned long long u64[kWaves];
  float f32[kWaves];
  double f64[kWaves];
  int i32[kWaves];
  uint32_t cnt[EPL * kWaves];
  int bc_digit;
  unsigned long long bc_above;
  int n_kept;
  uint16_t klist[EPL * kThreads];
};

__device__ inline int lane_id() { return threadIdx.x & (kWave - 1); }
__device__ inline int wave_id() { return threadIdx.x / kWave; }

__device__ inline uint64_t lanemask_lt() {
  const int lane = lane_id();
  return lane ? (~0ull >> (64 - lane)) : 0ull;
}

template <typename T>
__device__ inline void keep_better(T &bv, int &bi, T v, int i) {
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

template <int EPL>
__device__ inline uint64_t block_sum_u64(uint64_t x, Smem<EPL> &sm) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  if (lane_id() == 0) sm.u64[wave_id()] = x;
  __syncthreads();
  uint64_t r = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) r += sm.u64[w];
  __syncthreads();
  return r;
}

template <int EPL>
__device__ inline uint64_t block_max_u64(uint64_t x, Smem<EPL> &sm) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o = __shfl_xor(x, off);
    x = o > x ? o : x;
  }
  if (lane_id() == 0) sm.u64[wave_id()] = x;
  __syncthreads();
  uint64_t r = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) r = sm.u64[w] > r ? sm.u64[w] : r;
  __syncthreads();
  return r;
}

template <int EPL>
__device__ inline float block_max_f32(float x, Smem<EPL> &sm) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  if (lane_id() == 0) sm.f32[wave_id()] = x;
  __syncthreads();
  float r = sm.f32[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) r = fmaxf(r, sm.f32[w]);
  __syncthreads();
  return r;
}

// (value desc, id asc) maximum over the block; every thread gets the id.
template <typename T, int EPL>
__device__ inline int block_argmax(T bv, int bi, Smem<EPL> &sm) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const T ov = __shfl_xor(bv, off);
    const int oi = __shfl_xor(bi, off);
    keep_better(bv, bi, ov, oi);
  }
  if (lane_id() == 0) {
    sm.f64[wave_id()] = (double)bv;
    sm.i32[wave_id()] = bi;
  }
  __syncthreads();
  double rv = sm.f64[0];
  int ri = sm.i32[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) keep_better(rv, ri, sm.f64[w], sm.i32[w]);
  __syncthreads();
  return ri;
}

// ---- Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11) ---------------------
__device__ inline uint64_t philox_word(uint64_t seed, uint64_t key, uint64_t t, uint64_t k,
                                       uint32_t v) {
  const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
  uint64_t x0 = v >> 2, x1 = k, x2 = t, x3 = key;
  uint64_t k0 = seed, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B97F4A7C15ull;
      k1 += 0xBB67AE8584CAA73Bull;
    }
    const uint64_t lo0 = m0 * x0, hi0 = __umul64hi(m0, x0);
    const uint64_t lo1 = m1 * x2, hi1 = __umul64hi(m1, x2);
    const uint64_t y0 = hi1 ^ x1 ^ k0, y2 = hi0 ^ x3 ^ k1;
    x0 = y0;
    x1 = lo1;
    x2 = y2;
    x3 = lo0;
  }
  switch (v & 3) {
    case 0: return x0;
    case 1: return x1;
    case 2: return x2;
    default: return x3;
  }
}

__device__ inline double gumbel(uint64_t seed, uint64_t key, uint64_t t, uint64_t k, uint32_t v) {
  const uint64_t x = philox_word(seed, key, t, k, v);
  const double u = ((double)(x >> 41) + 0.5) * 0x1p-23;
  return -log(-log(u));
}

// ---- radix select ------------------------------------------------------------
// Finds the boundary key kappa of the "take `target` units from the top" cut
// among active elements (units: 1 per element, or its fixed-point mass) and the
// amount `rem` (>= 1) still to take from the elements whose key == kappa.
// Returns false if the active total is below target (then everything is kept).
// Element i of thread tid is id e = i*256 + tid.
template <int EPL, bool MASS>
__device__ bool radix_select(const float (&x)[EPL], uint32_t active, const uint64_t *mass,
                             uint64_t target, Smem<EPL> &sm, uint32_t &kappa, uint64_t &rem) {
  const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
  uint32_t prefix = 0, pmask = 0;
  rem = target;
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (MASS) sm.hm[tid] = 0;
    else sm.hc[tid] = 0;
    if (tid == 0) sm.bc_digit = -1;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const uint32_t key = order_key(x[i]);
      if (((active >> i) & 1) && (key & pmask) == prefix) {
        const uint32_t d = (key >> shift) & 255u;
        if (MASS) atomicAdd(&sm.hm[d], (unsigned long long)mass[i]);
        else atomicAdd(&sm.hc[d], 1u);
      }
    }
    __syncthreads();
    // thread t owns digit 255 - t: scanning threads in order walks digits downwards
    const int d = 255 - tid;
    const uint64_t v = MASS ? (uint64_t)sm.hm[d] : (uint64_t)sm.hc[d];
    uint64_t incl = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const uint64_t o = __shfl_up(incl, off);
      if (lane >= off) incl += o;
    }
    if (lane == kWave - 1) sm.u64[wave] = incl;
    __syncthreads();
    for (int w = 0; w < wave; ++w) incl += sm.u64[w];
    const uint64_t excl = incl - v;
    if (excl < rem && incl >= rem) {
      sm.bc_digit = d;
      sm.bc_above = excl;
    }
    __syncthreads();
    const int dsel = sm.bc_digit;
    const uint64_t above = sm.bc_above;
    __syncthreads();
    if (dsel < 0) return false;
    rem -= above;
    prefix |= (uint32_t)dsel << shift;
    pmask |= 255u << shift;
  }
  kappa = prefix;
  return true;
}

// Keep, among the active elements with key == kappa, the `need` lowest ids, and
// every active element above kappa; drop the rest.
template <int EPL>
__device__ uint32_t apply_cut(const float (&x)[EPL], uint32_t active, uint32_t kappa,
                              uint64_t need, Smem<EPL> &sm) {
  const int lane = lane_id(), wave = wave_id();
  uint64_t ball[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const bool tie = ((active >> i) & 1) && order_key(x[i]) == kappa;
    ball[i] = __ballot(tie);
    if (lane == 0) sm.cnt[i * kWaves + wave] = __popcll(ball[i]);
  }
  __syncthreads();
  uint32_t out = 0;
  uint64_t base = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    uint64_t before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t c = sm.cnt[i * kWaves + w];
      if (w < wave) before += c;
      total += c;
    }
    const bool act = (active >> i) & 1;
    const uint32_t key = order_key(x[i]);
    const uint64_t rank = base + before + __popcll(ball[i] & lanemask_lt());
    if (act && (key > kappa || (key == kappa && rank < need))) out |= 1u << i;
    base += total;
  }
  __syncthreads();
  return out;
}

template <int EPL>
__device__ int select_and_draw(const HeadView &hv, const StepView &sv, const float *sc,
                               bool greedy, int top_k, float top_p, uint64_t rkey, int t, int k,
                               Smem<EPL> &sm) {
  static_assert(EPL <= 32, "one bit per element in a 32-bit mask");
  const int tid = threadIdx.x;
  const int V = hv.V;
  float x[EPL];
  uint32_t active = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = i * kThreads + tid;
    x[i] = (e < V) ? sc[e] : -INFINITY;
    if (e < V) active |= 1u << i;
  }
  if (greedy) {
    float bv = -INFINITY;
    int bi = INT32_MAX;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if ((active >> i) & 1) keep_better(bv, bi, x[i], i * kThreads + tid);
    return block_argmax(bv, bi, sm);
  }
  if (top_k > 0 && top_k < V) {
    uint32_t kappa;
    uint64_t rem;
    if (radix_select<EPL, false>(x, active, nullptr, (uint64_t)top_k, sm, kappa, rem))
      active = apply_cut<EPL>(x, active, kappa, rem, sm);
  }
  if (top_p < 1.0f) {
    float mloc = -INFINITY;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if ((active >> i) & 1) mloc = fmaxf(mloc, x[i]);
    const double mx = (double)block_max_f32(mloc, sm);
    uint64_t mass[EPL];
    uint64_t zl = 0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      mass[i] = 0;
      if ((active >> i) & 1) mass[i] = (uint64_t)rint(exp((double)x[i] - mx) * kMassScale);
      zl += mass[i];
    }
    const uint64_t Z = block_sum_u64(zl, sm);
    uint64_t target = (uint64_t)ceil((double)top_p * (double)Z);
    if (target < 1) target = 1;
    if (target <= Z) {
      uint32_t kappa;
      uint64_t rem;
      if (radix_select<EPL, true>(x, active, mass, target, sm, kappa, rem)) {
        // every element tied at kappa carries the same mass q: take the fewest reaching rem
        uint64_t q = 0;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
          if (((active >> i) & 1) && order_key(x[i]) == kappa) q = mass[i];
        q = block_max_u64(q, sm);
        const uint64_t need = q ? (rem + q - 1) / q : 1;
        active = apply_cut<EPL>(x, active, kappa, need, sm);
      }
    }
  }
  // compact the kept ids (any order: the draw's tie rule makes it order-free)
  if (tid == 0) sm.n_kept = 0;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if ((active >> i) & 1) sm.klist[atomicAdd(&sm.n_kept, 1)] = (uint16_t)(i * kThreads + tid);
  __syncthreads();
  const int n_kept = sm.n_kept;
  double bv = -INFINITY;
  int bi = INT32_MAX;
  for (int c = tid; c < n_kept; c += kThreads) {
    const int v = sm.klist[c];
    const double val =
        (double)sc[v] + gumbel(sv.seed, rkey, (uint64_t)t, (uint64_t)k, (uint32_t)v);
    keep_better(bv, bi, val, v);
  }
  return block_argmax(bv, bi, sm);
}

template <int EPL>
__global__ __launch_bounds__(kThreads) void sample_kernel(HeadView hv, StepView sv,
                                                          int with_text) {
  __shared__ Smem<EPL> sm;
  const int tid = threadIdx.x;
  const int vec = blockIdx.x;
  if (!plan_ok(sv)) {
    if (vec == 0 && tid == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }
  const int32_t *rows = sv.plan + kPlanHeader;
  const int n_audio = sv.Rs * hv.K;
  if (vec >= n_audio) {
    // text row: reduce the (max, lowest argmax) partials of the text GEMM
    const int j = vec - n_audio;
    if (!with_text || j >= sv.n_text) return;
    const int r = rows[sv.Mg + j];
    if (r < 0 || r >= sv.R) {
      if (tid == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
      return;
    }
    float bv = -INFINITY;
    int bi = INT32_MAX;
    for (int p = tid; p < sv.text_parts; p += kThreads)
      keep_better(bv, bi, sv.text_val[(size_t)j * sv.text_parts + p],
                  sv.text_idx[(size_t)j * sv.text_parts + p]);
    const int tok = block_argmax(bv, bi, sm);
    for (int k = tid; k < hv.K; k += kThreads)
      sv.tokens_out[(size_t)r * hv.K + k] = (k == 0) ? tok : hv.pad_id;
    return;
  }
  const int s = vec / hv.K, k = vec % hv.K;
  const bool paired = s < sv.n_pairs;
  const int r = paired ? rows[2 * s] : rows[2 * sv.n_pairs + (s - sv.n_pairs)];
  const int u = paired ? rows[2 * s + 1] : -1;
  if (r < 0 || r >= sv.R || u >= sv.R) {
    if (tid == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }
  const int t = sv.step[r];
  const int f = t - hv.delays.d[k];
  const int nf = sv.n_frames[r];
  const bool pad = f < 0 || (nf >= 0 && f >= nf);
  int token = hv.pad_id;
  bool sampled = false;
  if (!pad) {
    const float T = sv.temperature[r], P = sv.top_p[r];
    const bool bad = !(T >= 0.0f) || isinf(T) || !(P > 0.0f) ||
                     (paired && !isfinite(sv.cfg_w[r]));
    if (bad) {
      if (tid == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PARAM);
    } else {
      const float *sc = sv.scores + (size_t)s * hv.N + (size_t)k * hv.V;
      const uint64_t rkey = sv.rng_key ? sv.rng_key[r] : (uint64_t)r;
      token = select_and_draw<EPL>(hv, sv, sc, T == 0.0f, sv.top_k[r], P, rkey, t, k, sm);
      sampled = true;
    }
  }
  if (tid == 0) {
    sv.tokens_out[(size_t)r * hv.K + k] = token;
    if (u >= 0) sv.tokens_out[(size_t)u * hv.K + k] = token;
    const int slot = sv.grid_slot[r];
    if (sampled && slot >= 0 && sv.frame_grid) {
      if (slot < sv.n_slots && f < sv.F_max)
        sv.frame_grid[((size_t)slot * hv.K + k) * sv.F_max + f] = token;
      else
        atomicOr(sv.status, (uint32_t)MCD_DEV_GRID_RANGE);
    }
  }
}

template <int EPL>
hipError_t launch_epl(const HeadView &hv, const StepView &sv, int nblk, bool with_text,
                      hipStream_t st) {
  hipLaunchKernelGGL(sample_kernel<EPL>, dim3(nblk), dim3(kThreads), 0, st, hv, sv,
                     (int)with_text);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sample(const HeadView &hv, const StepView &sv, bool with_text,
                         hipStream_t st) {
  const int nblk = sv.Rs * hv.K + (with_text ? sv.n_text : 0);
  if (nblk == 0) return hipSuccess;
  const int epl = (hv.V + kThreads - 1) / kThreads;
  if (epl <= 1) return launch_epl<1>(hv, sv, nblk, with_text, st);
  if (epl <= 2) return launch_epl<2>(hv, sv, nblk, with_text, st);
  if (epl <= 4) return launch_epl<4>(hv, sv, nblk, with_text, st);
  if (epl <= 8) return launch_epl<8>(hv, sv, nblk, with_text, st);
  if (epl <= 16) return launch_epl<16>(hv, sv, nblk, with_text, st);
  return hipErrorInvalidValue;
}

}  // namespace mcd
