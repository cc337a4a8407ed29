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
// scores (8-bit digits from the top, histograms in LDS).  Top-k histograms
// count elements and stop as soon as the bucket holding the cut is taken whole;
// top-p histograms add fixed-point masses exp(s - max) * 2^48 (fp32 exp,
// converted exactly) as 64-bit integers, so the sums are exact and independent
// of the order of the adds.
// Three rotating histogram buffers need one barrier per digit pass: every wave
// scans the whole histogram itself, so no result has to be broadcast.
#include "mcd_internal.h"

namespace mcd {
namespace {

constexpr int kWave = 64;
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

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

template <int EPL>
struct Smem {
  unsigned long long hist[3][256];   // rotating digit histograms (counts or masses)
  unsigned long long r64[2][kWaves];  // block reductions (double-buffered)
  double rf[2][kWaves];
  int ri[2][kWaves];
  uint32_t cnt[EPL * kWaves];         // tie counts per (element slot, wave)
  uint32_t kept[(EPL * kThreads + 31) / 32];  // kept-id bitmask
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

// Block reductions; `slot` alternates between consecutive calls so that one
// barrier suffices (the buffer written now was last read two calls ago).
template <int EPL>
__device__ inline uint64_t block_sum_u64(uint64_t x, Smem<EPL> &sm, int slot) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  if (lane_id() == 0) sm.r64[slot][wave_id()] = x;
  __syncthreads();
  uint64_t r = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) r += sm.r64[slot][w];
  return r;
}

template <int EPL>
__device__ inline uint64_t block_max_u64(uint64_t x, Smem<EPL> &sm, int slot) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o = __shfl_xor(x, off);
    x = o > x ? o : x;
  }
  if (lane_id() == 0) sm.r64[slot][wave_id()] = x;
  __syncthreads();
  uint64_t r = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) r = sm.r64[slot][w] > r ? sm.r64[slot][w] : r;
  return r;
}

// (value desc, id asc) maximum over the block; every thread gets the id.
template <typename T, int EPL>
__device__ inline int block_argmax(T bv, int bi, Smem<EPL> &sm, int slot) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const T ov = __shfl_xor(bv, off);
    const int oi = __shfl_xor(bi, off);
    keep_better(bv, bi, ov, oi);
  }
  if (lane_id() == 0) {
    sm.rf[slot][wave_id()] = (double)bv;
    sm.ri[slot][wave_id()] = bi;
  }
  __syncthreads();
  double rv = sm.rf[slot][0];
  int ri = sm.ri[slot][0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) keep_better(rv, ri, sm.rf[slot][w], sm.ri[slot][w]);
  return ri;
}

// ---- Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11) ---------------------
struct U64x4 {
  uint64_t w[4];
};

__device__ inline U64x4 philox_block(uint64_t seed, uint64_t key, uint64_t t, uint64_t k,
                                     uint64_t group) {
  const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
  uint64_t x0 = group, x1 = k, x2 = t, x3 = key;
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
  return U64x4{{x0, x1, x2, x3}};
}

// Gumbel variate from one Philox word, in fp32 (the uniform is exact in fp32;
// each log is within about one ulp, so G is within ~1e-6 of its exact value).
__device__ inline float gumbel_from_word(uint64_t x) {
  const float u = ((float)(uint32_t)(x >> 41) + 0.5f) * 0x1p-23f;
  return -logf(-logf(u));
}

// ---- radix select ------------------------------------------------------------
// Cut of "take `target` units from the top" among the active elements (units:
// 1 per element, or its fixed-point mass).  Result: keep every active element
// with key >= lo; when `exact`, lo is a single key kappa whose ties are kept
// only up to `need` units (ties carry equal units) -- see apply_cut.
struct Cut {
  uint32_t lo;
  bool exact;
  uint64_t need;   // units still wanted from the elements with key == lo (exact only)
  bool all;        // target not reached: keep every active element
};

// Element i of thread tid is id e = i*256 + tid.  `pass` counts the digit
// passes done so far in this vector and selects the rotating buffers; the
// buffers pass % 3 and (pass + 1) % 3 must be zero on entry, and the two after
// the last one used are zero again on exit.
template <int EPL, bool MASS>
__device__ Cut radix_select(const float (&x)[EPL], uint32_t active, const uint64_t *mass,
                            uint64_t target, Smem<EPL> &sm, int &pass) {
  const int tid = threadIdx.x, lane = lane_id();
  uint32_t prefix = 0, pmask = 0;
  uint64_t rem = target;
  for (int shift = 24; shift >= 0; shift -= 8) {
    unsigned long long *h = sm.hist[pass % 3];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const uint32_t key = order_key(x[i]);
      if (((active >> i) & 1) && (key & pmask) == prefix) {
        const uint32_t d = (key >> shift) & 255u;
        atomicAdd(&h[d], MASS ? (unsigned long long)mass[i] : 1ull);
      }
    }
    __syncthreads();
    // every wave scans all 256 digits (lane l: digits 255-4l .. 252-4l)
    uint64_t v[4], lsum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = h[255 - 4 * lane - j];
      lsum += v[j];
    }
    uint64_t incl = lsum;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const uint64_t o = __shfl_up(incl, off);
      if (lane >= off) incl += o;
    }
    const uint64_t excl = incl - lsum;
    // clear the buffer of the pass after next (its last readers passed the barrier above)
    sm.hist[(pass + 2) % 3][tid] = 0;
    ++pass;
    const uint64_t bal = __ballot(excl < rem && incl >= rem);
    if (bal == 0) return Cut{0u, false, 0, true};
    const int src = __ffsll((long long)bal) - 1;
    int dsel = 0;
    uint64_t above = 0, inbucket = 0;
    if (lane == src) {
      uint64_t cum = excl;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (cum + v[j] >= rem) {
          dsel = 255 - 4 * lane - j;
          above = cum;
          inbucket = v[j];
          break;
        }
        cum += v[j];
      }
    }
    dsel = __shfl(dsel, src);
    above = __shfl(above, src);
    inbucket = __shfl(inbucket, src);
    rem -= above;
    prefix |= (uint32_t)dsel << shift;
    pmask |= 255u << shift;
    if (!MASS && inbucket == rem) {
      // the whole bucket is taken: keep every key whose leading digits are >= prefix
      return Cut{prefix, false, 0, false};
    }
  }
  return Cut{prefix, true, rem, false};
}

// Apply a cut to the active set.  For an exact cut with fewer than all of the
// ties at kappa wanted, the `need_n` lowest ids among the ties are kept.
template <int EPL>
__device__ uint32_t apply_cut(const float (&x)[EPL], uint32_t active, const Cut &c,
                              uint64_t need_n, Smem<EPL> &sm, int &slot) {
  if (c.all) return active;
  uint32_t keep = 0, ties = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const uint32_t key = order_key(x[i]);
    const bool act = (active >> i) & 1;
    if (act && key >= c.lo && !(c.exact && key == c.lo)) keep |= 1u << i;
    if (act && c.exact && key == c.lo) ties |= 1u << i;
  }
  if (!c.exact) return keep;
  const uint64_t total = block_sum_u64((uint64_t)__popc(ties), sm, slot);
  slot ^= 1;
  if (need_n >= total) return keep | ties;
  // rare: rank the ties by id (e = i*256 + tid)
  const int lane = lane_id(), wave = wave_id();
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const uint64_t b = __ballot((ties >> i) & 1);
    if (lane == 0) sm.cnt[i * kWaves + wave] = __popcll(b);
  }
  __syncthreads();
  uint64_t base = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const uint64_t b = __ballot((ties >> i) & 1);
    uint64_t before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t cw = sm.cnt[i * kWaves + w];
      if (w < wave) before += cw;
      tot += cw;
    }
    const uint64_t rank = base + before + __popcll(b & lanemask_lt());
    if (((ties >> i) & 1) && rank < need_n) keep |= 1u << i;
    base += tot;
  }
  __syncthreads();  // cnt may be reused
  return keep;
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
  int slot = 0;
  if (greedy) {
    float bv = -INFINITY;
    int bi = INT32_MAX;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if ((active >> i) & 1) keep_better(bv, bi, x[i], i * kThreads + tid);
    return block_argmax(bv, bi, sm, slot);
  }
  // histograms 0 and 1 zero, kept mask zero
#pragma unroll
  for (int b = 0; b < 2; ++b) sm.hist[b][tid] = 0;
  for (int w = tid; w < (EPL * kThreads + 31) / 32; w += kThreads) sm.kept[w] = 0;
  __syncthreads();
  int pass = 0;
  if (top_k > 0 && top_k < V) {
    const Cut c = radix_select<EPL, false>(x, active, nullptr, (uint64_t)top_k, sm, pass);
    active = apply_cut<EPL>(x, active, c, c.need, sm, slot);
  }
  if (top_p < 1.0f) {
    float mloc = -INFINITY;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if ((active >> i) & 1) mloc = fmaxf(mloc, x[i]);
    // the max through the order key (monotone), reduced as an integer
    const uint32_t mk = (uint32_t)block_max_u64((uint64_t)order_key(mloc), sm, slot);
    slot ^= 1;
    const uint32_t mu = (mk & 0x80000000u) ? (mk & 0x7FFFFFFFu) : ~mk;
    const float mx = __uint_as_float(mu);
    // mass = exp(s - max) in fp32 (relative error ~1e-7), scaled by 2^48 and
    // converted exactly to a 64-bit integer
    uint64_t mass[EPL];
    uint64_t zl = 0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      mass[i] = ((active >> i) & 1) ? (uint64_t)ldexpf(expf(x[i] - mx), 48) : 0;
      zl += mass[i];
    }
    const uint64_t Z = block_sum_u64(zl, sm, slot);
    slot ^= 1;
    uint64_t target = (uint64_t)ceil((double)top_p * (double)Z);
    if (target < 1) target = 1;
    if (target <= Z) {
      const Cut c = radix_select<EPL, true>(x, active, mass, target, sm, pass);
      uint64_t need_n = 0;
      if (c.exact) {
        // every element tied at kappa carries the same mass q: the fewest reaching rem
        uint64_t q = 0;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
          if (((active >> i) & 1) && order_key(x[i]) == c.lo) q = mass[i];
        q = block_max_u64(q, sm, slot);
        slot ^= 1;
        need_n = q ? (c.need + q - 1) / q : 1;
      }
      active = apply_cut<EPL>(x, active, c, need_n, sm, slot);
    }
  }
  // kept-id bitmask, then one Philox block per group of 4 consecutive ids
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if ((active >> i) & 1) {
      const int e = i * kThreads + tid;
      atomicOr(&sm.kept[e >> 5], 1u << (e & 31));
    }
  __syncthreads();
  double bv = -INFINITY;
  int bi = INT32_MAX;
  const int groups = (V + 3) >> 2;
  for (int g = tid; g < groups; g += kThreads) {
    const uint32_t bits = (sm.kept[g >> 3] >> ((g & 7) * 4)) & 0xFu;
    if (!bits) continue;
    const U64x4 w = philox_block(sv.seed, rkey, (uint64_t)t, (uint64_t)k, (uint64_t)g);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if ((bits >> j) & 1) {
        const int v = 4 * g + j;
        const double val = (double)sc[v] + (double)gumbel_from_word(w.w[j]);
        keep_better(bv, bi, val, v);
      }
  }
  return block_argmax(bv, bi, sm, slot);
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
    const int tok = block_argmax(bv, bi, sm, 0);
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
