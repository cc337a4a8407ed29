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
// Layout: thread tid owns groups g = q * 256 + tid of four consecutive ids
// 4g .. 4g + 3 (one 16-byte load each), so that one Philox block serves a whole
// group from registers.
//
// Selection.  Every score s falls in a bin b = floor(16 (max - s)) (bins of
// width 1/16 below the maximum, the last one open-ended); the bin index is
// monotone in s, so a cut between bins is a cut in the (score desc, id asc)
// order.  One histogram pass (counts for top-k, masses for top-p) finds the bin
// holding the cut; only the few elements of that bin are then ranked exactly
// against each other.  Top-p masses are fixed-point exp(s - max) * 2^48 (fp32
// exp, converted exactly) summed as 64-bit integers: exact and independent of
// the order of the adds.  Inputs whose cut bin is crowded (heavy ties, or a cut
// far below the maximum) take a radix select over order-preserving 32-bit keys
// instead; both give the same kept set.
//
// Wave reductions and scans use DPP lane moves (row shifts and row broadcasts)
// rather than LDS permutes.
#include "mcd_internal.h"

namespace mcd {
namespace {

constexpr int kWave = 64;
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kBins = 512;          // bins of width 1/16 below the maximum, plus one open bin
constexpr float kBinScale = 16.0f;
constexpr int kCap = 256;           // largest cut bin ranked directly

__device__ inline uint32_t order_key(float x) {
  if (x == 0.0f) x = 0.0f;  // -0 and +0 compare equal
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float key_to_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

__device__ inline bool plan_ok(const StepView &sv) {
  const int32_t *p = sv.plan;
  return p[kPlanMagicWord] == kPlanMagic && p[kPlanR] == sv.R && p[kPlanPairs] == sv.n_pairs &&
         p[kPlanSolo] == sv.n_solo && p[kPlanText] == sv.n_text;
}

__device__ inline int lane_id() { return threadIdx.x & (kWave - 1); }
__device__ inline int wave_id() { return threadIdx.x / kWave; }

template <typename T>
__device__ inline void keep_better(T &bv, int &bi, T v, int i) {
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

// ---- wave primitives (DPP) -------------------------------------------------
// Lane move with an identity for lanes whose source lies outside the row (or
// rows left out by the row mask).
template <int CTRL, int ROWMASK = 0xF>
__device__ __forceinline__ uint32_t dpp(uint32_t identity, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)identity, (int)v, CTRL, ROWMASK, 0xF, false);
}
constexpr int kShr1 = 0x111, kShr2 = 0x112, kShr4 = 0x114, kShr8 = 0x118;
constexpr int kBcast15 = 0x142, kBcast31 = 0x143;

// Inclusive scan over the 64 lanes: shifts by 1, 2, 4, 8 within 16-lane rows,
// then the last lane of row 0 (2) into row 1 (3), and lane 31 into rows 2, 3.
template <class Combine>
__device__ __forceinline__ void wave_scan(Combine &&step) {
  step(std::integral_constant<int, kShr1>{}, std::integral_constant<int, 0xF>{});
  step(std::integral_constant<int, kShr2>{}, std::integral_constant<int, 0xF>{});
  step(std::integral_constant<int, kShr4>{}, std::integral_constant<int, 0xF>{});
  step(std::integral_constant<int, kShr8>{}, std::integral_constant<int, 0xF>{});
  step(std::integral_constant<int, kBcast15>{}, std::integral_constant<int, 0xA>{});
  step(std::integral_constant<int, kBcast31>{}, std::integral_constant<int, 0xC>{});
}

__device__ __forceinline__ uint32_t wave_incl_add_u32(uint32_t x) {
  wave_scan([&](auto c, auto m) __attribute__((always_inline)) {
    x += dpp<decltype(c)::value, decltype(m)::value>(0u, x);
  });
  return x;
}

__device__ __forceinline__ uint64_t wave_incl_add_u64(uint64_t x) {
  wave_scan([&](auto c, auto m) __attribute__((always_inline)) {
    constexpr int C = decltype(c)::value, RM = decltype(m)::value;
    const uint32_t lo = dpp<C, RM>(0u, (uint32_t)x), hi = dpp<C, RM>(0u, (uint32_t)(x >> 32));
    x += ((uint64_t)hi << 32) | lo;
  });
  return x;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  wave_scan([&](auto c, auto m) __attribute__((always_inline)) {
    const uint32_t o = dpp<decltype(c)::value, decltype(m)::value>(0u, x);
    x = o > x ? o : x;
  });
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
  wave_scan([&](auto c, auto m) __attribute__((always_inline)) {
    const uint32_t o = dpp<decltype(c)::value, decltype(m)::value>(0xFFFFFFFFu, x);
    x = o < x ? o : x;
  });
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

// (value desc, id asc) best over the wave, as seen by every lane.
__device__ __forceinline__ void wave_argmax_f32(float &bv, int &bi) {
  wave_scan([&](auto c, auto m) __attribute__((always_inline)) {
    constexpr int C = decltype(c)::value, RM = decltype(m)::value;
    const float ov = __uint_as_float(dpp<C, RM>(__float_as_uint(-INFINITY), __float_as_uint(bv)));
    const int oi = (int)dpp<C, RM>((uint32_t)INT32_MAX, (uint32_t)bi);
    keep_better(bv, bi, ov, oi);
  });
  bv = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(bv), 63));
  bi = __builtin_amdgcn_readlane(bi, 63);
}

__device__ __forceinline__ void wave_argmax_f64(double &bv, int &bi) {
  const uint64_t ninf = (uint64_t)__double_as_longlong(-INFINITY);
  wave_scan([&](auto c, auto m) __attribute__((always_inline)) {
    constexpr int C = decltype(c)::value, RM = decltype(m)::value;
    const uint64_t b = (uint64_t)__double_as_longlong(bv);
    const uint32_t lo = dpp<C, RM>((uint32_t)ninf, (uint32_t)b);
    const uint32_t hi = dpp<C, RM>((uint32_t)(ninf >> 32), (uint32_t)(b >> 32));
    const int oi = (int)dpp<C, RM>((uint32_t)INT32_MAX, (uint32_t)bi);
    keep_better(bv, bi, __longlong_as_double((long long)(((uint64_t)hi << 32) | lo)), oi);
  });
  bv = __longlong_as_double((long long)readlane_u64((uint64_t)__double_as_longlong(bv), 63));
  bi = __builtin_amdgcn_readlane(bi, 63);
}

// ---- workgroup shared memory and reductions ----------------------------------
template <int GPT>
struct Smem {
  uint32_t cnt[kBins + 1];               // top-k bin counts
  unsigned long long mh[kBins + 1];      // top-p bin masses
  // elements of the cut bin, and their exact ranks
  struct Entry {
    float v;
    int id;
  };
  Entry le[kCap];
  unsigned long long lm[kCap];           // their masses (top-p)
  int lr[kCap];
  unsigned long long lsm[kCap];          // masses in rank order, then the mass before each rank
  uint32_t keepbits[kThreads];           // kept cut-bin elements, one bit per slot of a thread
  uint32_t lcount;
  // block reductions (two slots, alternating, one barrier each)
  uint32_t ru[2][kWaves];
  unsigned long long r64[2][kWaves];
  double rd[2][kWaves];
  int ri[2][kWaves];
  // radix select (fallback); reused for the draw list once the selection is done
  unsigned long long hist[3][256];
};

// A group of four ids with kept members, moved to the thread that draws it.
struct DrawItem {
  int g;
  uint32_t bits;
  float x[4];
};
constexpr int kDrawCap = 256;
static_assert(kDrawCap * sizeof(DrawItem) <= 3 * 256 * sizeof(unsigned long long), "draw list fits");

template <int GPT>
__device__ __forceinline__ uint32_t block_max_u32(uint32_t x, Smem<GPT> &sm, int &slot) {
  x = wave_max_u32(x);
  if (lane_id() == 0) sm.ru[slot][wave_id()] = x;
  __syncthreads();
  uint32_t r = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) r = sm.ru[slot][w] > r ? sm.ru[slot][w] : r;
  slot ^= 1;
  return r;
}

template <int GPT>
__device__ __forceinline__ uint32_t block_min_u32(uint32_t x, Smem<GPT> &sm, int &slot) {
  x = wave_min_u32(x);
  if (lane_id() == 0) sm.ru[slot][wave_id()] = x;
  __syncthreads();
  uint32_t r = 0xFFFFFFFFu;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) r = sm.ru[slot][w] < r ? sm.ru[slot][w] : r;
  slot ^= 1;
  return r;
}

template <int GPT>
__device__ __forceinline__ uint64_t block_sum_u64(uint64_t x, Smem<GPT> &sm, int &slot) {
  x = readlane_u64(wave_incl_add_u64(x), 63);
  if (lane_id() == 0) sm.r64[slot][wave_id()] = x;
  __syncthreads();
  uint64_t r = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) r += sm.r64[slot][w];
  slot ^= 1;
  return r;
}

// exclusive prefix of x over the threads in id order, and the block total
template <int GPT>
__device__ __forceinline__ uint32_t block_excl_scan_u32(uint32_t x, uint32_t &total,
                                                        Smem<GPT> &sm, int &slot) {
  const uint32_t incl = wave_incl_add_u32(x);
  if (lane_id() == 63) sm.ru[slot][wave_id()] = incl;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t c = sm.ru[slot][w];
    if (w < wave_id()) before += c;
    tot += c;
  }
  slot ^= 1;
  total = tot;
  return before + incl - x;
}

// inclusive prefix of x over the threads in id order
template <int GPT>
__device__ __forceinline__ uint64_t block_incl_scan_u64(uint64_t x, Smem<GPT> &sm, int &slot) {
  const uint64_t incl = wave_incl_add_u64(x);
  if (lane_id() == 63) sm.r64[slot][wave_id()] = incl;
  __syncthreads();
  uint64_t before = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w)
    if (w < wave_id()) before += sm.r64[slot][w];
  slot ^= 1;
  return before + incl;
}

template <int GPT>
__device__ __forceinline__ int block_argmax_f32(float bv, int bi, Smem<GPT> &sm, int &slot) {
  wave_argmax_f32(bv, bi);
  if (lane_id() == 0) {
    sm.rd[slot][wave_id()] = (double)bv;
    sm.ri[slot][wave_id()] = bi;
  }
  __syncthreads();
  double rv = sm.rd[slot][0];
  int ri = sm.ri[slot][0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) keep_better(rv, ri, sm.rd[slot][w], sm.ri[slot][w]);
  slot ^= 1;
  return ri;
}

template <int GPT>
__device__ __forceinline__ int block_argmax_f64(double bv, int bi, Smem<GPT> &sm, int &slot) {
  wave_argmax_f64(bv, bi);
  if (lane_id() == 0) {
    sm.rd[slot][wave_id()] = bv;
    sm.ri[slot][wave_id()] = bi;
  }
  __syncthreads();
  double rv = sm.rd[slot][0];
  int ri = sm.ri[slot][0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) keep_better(rv, ri, sm.rd[slot][w], sm.ri[slot][w]);
  slot ^= 1;
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

// ---- radix select (fallback) -----------------------------------------------
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

// `pass` counts the digit passes done so far in this vector and selects the
// rotating buffers; the buffers pass % 3 and (pass + 1) % 3 must be zero on
// entry, and the two after the last one used are zero again on exit.
template <int GPT, bool MASS>
__device__ __forceinline__ Cut radix_select(const float (&x)[4 * GPT], uint32_t active, const uint64_t *mass,
                            uint64_t target, Smem<GPT> &sm, int &pass) {
  constexpr int EPL = 4 * GPT;
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
    const uint64_t incl = wave_incl_add_u64(lsum);
    const uint64_t excl = incl - lsum;
    // clear the buffer of the pass after next (its last readers passed the barrier above)
    sm.hist[(pass + 2) % 3][tid] = 0;
    ++pass;
    const uint64_t bal = __ballot(excl < rem && incl >= rem);
    if (bal == 0) return Cut{0u, false, 0, true};
    const int src = __ffsll((long long)bal) - 1;
    uint64_t cum = readlane_u64(excl, src);
    int dsel = 0;
    uint64_t above = cum, inbucket = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint64_t vj = readlane_u64(v[j], src);
      if (inbucket == 0 && cum + vj >= rem) {
        dsel = 255 - 4 * src - j;
        above = cum;
        inbucket = vj;
      }
      cum += vj;
    }
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
// ties at kappa wanted, the `need_n` lowest ids among the ties are kept (id of
// slot 4q + j of thread tid: 4 (q * 256 + tid) + j).
template <int GPT>
__device__ __forceinline__ uint32_t apply_cut(const float (&x)[4 * GPT], uint32_t active, const Cut &c,
                              uint64_t need_n, Smem<GPT> &sm, int &slot) {
  constexpr int EPL = 4 * GPT;
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
  uint64_t base = 0;
#pragma unroll
  for (int q = 0; q < GPT; ++q) {
    const uint32_t tq = (ties >> (4 * q)) & 0xFu;
    uint32_t total;
    const uint32_t before = block_excl_scan_u32((uint32_t)__popc(tq), total, sm, slot);
    uint64_t rank = base + before;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if ((tq >> j) & 1) {
        if (rank < need_n) keep |= 1u << (4 * q + j);
        ++rank;
      }
    }
    base += total;
  }
  return keep;
}

// ---- selection through the bins ------------------------------------------------
// The wave scans the histogram h[0..kBins) (8 bins per lane) and returns the
// first bin whose cumulative count/mass reaches `target` (kBins: the open bin),
// with the cumulative value of the bins before it and the bin's own value.
template <typename T>
__device__ __forceinline__ int find_cut_bin(const T *h, uint64_t target, uint64_t &above,
                                            uint64_t &inbin, uint64_t total) {
  const int lane = lane_id();
  uint64_t v[8], lsum = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    v[j] = (uint64_t)h[8 * lane + j];
    lsum += v[j];
  }
  const uint64_t incl = wave_incl_add_u64(lsum);
  const uint64_t excl = incl - lsum;
  const uint64_t bal = __ballot(excl < target && incl >= target);
  if (bal == 0) {
    above = readlane_u64(incl, 63);
    inbin = total - above;
    return kBins;
  }
  const int src = __ffsll((long long)bal) - 1;
  uint64_t cum = readlane_u64(excl, src);
  int b = 0;
  above = cum;
  inbin = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint64_t vj = readlane_u64(v[j], src);
    if (inbin == 0 && cum + vj >= target) {
      b = 8 * src + j;
      above = cum;
      inbin = vj;
    }
    cum += vj;
  }
  return b;
}

template <int GPT>
__device__ __forceinline__ void bins_of(const float (&x)[4 * GPT], uint32_t active, float mx,
                                        int (&bin)[4 * GPT]) {
#pragma unroll
  for (int i = 0; i < 4 * GPT; ++i) {
    const float d = (mx - x[i]) * kBinScale;   // monotone in x
    bin[i] = ((active >> i) & 1) ? (d < (float)kBins ? (int)d : kBins) : -1;
  }
}

// Rank the listed elements of a cut bin by (score desc, id asc); n <= kCap.
template <int GPT>
__device__ __forceinline__ void rank_list(Smem<GPT> &sm, int n) {
  using Entry = typename Smem<GPT>::Entry;
  const int t = threadIdx.x;
  if (t < n) {
    const Entry me = sm.le[t];
    auto ahead = [&](const Entry &o) __attribute__((always_inline)) {
      return (int)((o.v > me.v) | ((o.v == me.v) & (o.id < me.id)));
    };
    int r = 0, j = 0;
    for (; j + 4 <= n; j += 4) {
      const Entry o0 = sm.le[j], o1 = sm.le[j + 1], o2 = sm.le[j + 2], o3 = sm.le[j + 3];
      r += ahead(o0) + ahead(o1) + ahead(o2) + ahead(o3);
    }
    for (; j < n; ++j) r += ahead(sm.le[j]);
    sm.lr[t] = r;
  }
}

// Thread that owns id e, and the slot of e in its registers.
__device__ __forceinline__ void owner_of(int e, int &thread, int &slot) {
  const int g = e >> 2;
  thread = g % kThreads;
  slot = 4 * (g / kThreads) + (e & 3);
}

template <int GPT>
__device__ __forceinline__ uint32_t radix_topk(const float (&x)[4 * GPT], uint32_t active, int top_k,
                                            Smem<GPT> &sm, int &slot, int &pass) {
  const Cut c = radix_select<GPT, false>(x, active, nullptr, (uint64_t)top_k, sm, pass);
  return apply_cut<GPT>(x, active, c, c.need, sm, slot);
}

template <int GPT>
__device__ __forceinline__ uint32_t radix_topp(const float (&x)[4 * GPT], uint32_t active,
                                            const uint64_t (&mass)[4 * GPT], uint64_t target,
                                            Smem<GPT> &sm, int &slot, int &pass) {
  const Cut c = radix_select<GPT, true>(x, active, mass, target, sm, pass);
  uint64_t need_n = 0;
  if (c.exact) {
    // every element tied at kappa carries the same mass q: the fewest reaching rem
    uint64_t q = 0;
#pragma unroll
    for (int i = 0; i < 4 * GPT; ++i)
      if (((active >> i) & 1) && order_key(x[i]) == c.lo) q = mass[i];
    // every nonzero q is the same value, so the halves reduce independently
    const uint64_t qhi = block_max_u32((uint32_t)(q >> 32), sm, slot);
    const uint64_t qlo = block_max_u32((uint32_t)q, sm, slot);
    q = qhi << 32 | qlo;
    need_n = q ? (c.need + q - 1) / q : 1;
  }
  return apply_cut<GPT>(x, active, c, need_n, sm, slot);
}

template <int GPT>
__device__ __forceinline__ void zero_radix(Smem<GPT> &sm) {
#pragma unroll
  for (int b = 0; b < 2; ++b) sm.hist[b][threadIdx.x] = 0;
  __syncthreads();
}

// top-k over the active set; `mx` is the maximum active score
template <int GPT>
__device__ __forceinline__ uint32_t select_topk(const float (&x)[4 * GPT], uint32_t active,
                                                float mx, int top_k, Smem<GPT> &sm, int &slot,
                                                int &pass, int V) {
  constexpr int EPL = 4 * GPT;
  int bin[EPL];
  bins_of<GPT>(x, active, mx, bin);
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (bin[i] >= 0 && bin[i] < kBins) atomicAdd(&sm.cnt[bin[i]], 1u);
  __syncthreads();
  uint64_t above, inbin;
  const int bc = find_cut_bin(sm.cnt, (uint64_t)top_k, above, inbin, (uint64_t)V);
  const uint64_t need = (uint64_t)top_k - above;
  uint32_t keep = 0;
  if (bc < kBins && need == inbin) {
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (bin[i] >= 0 && bin[i] <= bc) keep |= 1u << i;
    return keep;
  }
  if (bc == kBins || inbin > (uint64_t)kCap) {
    zero_radix(sm);
    return radix_topk<GPT>(x, active, top_k, sm, slot, pass);
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    if (bin[i] == bc) {
      const int s = (int)atomicAdd(&sm.lcount, 1u);
      sm.le[s] = {x[i], 4 * ((i / 4) * kThreads + (int)threadIdx.x) + (i % 4)};
    }
  }
  __syncthreads();
  rank_list(sm, (int)inbin);
  if ((int)threadIdx.x < (int)inbin && (uint64_t)sm.lr[threadIdx.x] < need) {
    int ow, sl;
    owner_of(sm.le[threadIdx.x].id, ow, sl);
    atomicOr(&sm.keepbits[ow], 1u << sl);
  }
  __syncthreads();
  keep = sm.keepbits[threadIdx.x];
  sm.keepbits[threadIdx.x] = 0;          // next use follows at least one barrier
  if (threadIdx.x == 0) sm.lcount = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (bin[i] >= 0 && bin[i] < bc) keep |= 1u << i;
  return keep;
}

// top-p over the active set (the survivors of top-k); `mx` is their maximum
template <int GPT>
__device__ __forceinline__ uint32_t select_topp(const float (&x)[4 * GPT], uint32_t active,
                                                float mx, float top_p, Smem<GPT> &sm, int &slot,
                                                int &pass) {
  constexpr int EPL = 4 * GPT;
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
  uint64_t target = (uint64_t)ceil((double)top_p * (double)Z);
  if (target < 1) target = 1;
  if (target > Z) return active;
  int bin[EPL];
  bins_of<GPT>(x, active, mx, bin);
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (bin[i] >= 0 && bin[i] < kBins) atomicAdd(&sm.mh[bin[i]], (unsigned long long)mass[i]);
  __syncthreads();
  uint64_t above, inbin;
  const int bc = find_cut_bin(sm.mh, target, above, inbin, Z);
  if (bc == kBins) {
    zero_radix(sm);
    return radix_topp<GPT>(x, active, mass, target, sm, slot, pass);
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    if (bin[i] == bc) {
      const int s = (int)atomicAdd(&sm.lcount, 1u);
      if (s < kCap) {
        sm.le[s] = {x[i], 4 * ((i / 4) * kThreads + (int)threadIdx.x) + (i % 4)};
        sm.lm[s] = mass[i];
      }
    }
  }
  __syncthreads();
  const int n = (int)sm.lcount;
  if (n > kCap) {
    __syncthreads();   // everyone has read lcount
    if (threadIdx.x == 0) sm.lcount = 0;
    zero_radix(sm);
    return radix_topp<GPT>(x, active, mass, target, sm, slot, pass);
  }
  rank_list(sm, n);
  __syncthreads();
  if ((int)threadIdx.x < n) sm.lsm[sm.lr[threadIdx.x]] = sm.lm[threadIdx.x];
  __syncthreads();
  // mass of the ranks before each rank: a block scan (thread r holds rank r)
  const uint64_t mr = (int)threadIdx.x < n ? sm.lsm[threadIdx.x] : 0;
  const uint64_t incl = block_incl_scan_u64(mr, sm, slot);
  if ((int)threadIdx.x < n) sm.lsm[threadIdx.x] = incl - mr;   // every read of lsm is done
  __syncthreads();
  // entry kept iff the mass strictly before it (in rank order) is below target
  if ((int)threadIdx.x < n && above + sm.lsm[sm.lr[threadIdx.x]] < target) {
    int ow, sl;
    owner_of(sm.le[threadIdx.x].id, ow, sl);
    atomicOr(&sm.keepbits[ow], 1u << sl);
  }
  __syncthreads();
  uint32_t keep = sm.keepbits[threadIdx.x];
  sm.keepbits[threadIdx.x] = 0;
  if (threadIdx.x == 0) sm.lcount = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (bin[i] >= 0 && bin[i] < bc) keep |= 1u << i;
  return keep;
}

template <int GPT>
__device__ __forceinline__ int select_and_draw(const StepView &sv, const float (&x)[4 * GPT],
                                               uint32_t active, int V, bool greedy, int top_k,
                                               float top_p, uint64_t rkey, int t, int k,
                                               Smem<GPT> &sm, int &slot) {
  constexpr int EPL = 4 * GPT;
  const int tid = threadIdx.x;
  uint32_t mk = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if ((active >> i) & 1) {
      const uint32_t key = order_key(x[i]);
      mk = key > mk ? key : mk;
    }
  mk = block_max_u32(mk, sm, slot);   // also publishes the zeroed histograms
  if (greedy) {
    uint32_t id = 0xFFFFFFFFu;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (((active >> i) & 1) && order_key(x[i]) == mk) {
        const uint32_t e = 4u * (uint32_t)((i / 4) * kThreads + tid) + (uint32_t)(i % 4);
        id = e < id ? e : id;
      }
    return (int)block_min_u32(id, sm, slot);
  }
  const float mx = key_to_float(mk);
  int pass = 0;
  uint32_t kept = active;
  if (top_k > 0 && top_k < V) kept = select_topk<GPT>(x, kept, mx, top_k, sm, slot, pass, V);
  if (top_p < 1.0f) kept = select_topp<GPT>(x, kept, mx, top_p, sm, slot, pass);
  // Gumbel-max over the kept ids, one Philox block per group with a kept id
  double bv = -INFINITY;
  int bi = INT32_MAX;
  if (top_k > 0 && top_k <= kDrawCap) {
    // few kept groups: move them to one thread each, so that no wave runs
    // several Philox blocks one after another
    uint32_t n = 0;
#pragma unroll
    for (int q = 0; q < GPT; ++q) n += ((kept >> (4 * q)) & 0xFu) ? 1u : 0u;
    uint32_t total;
    uint32_t pos = block_excl_scan_u32(n, total, sm, slot);
    DrawItem *dl = reinterpret_cast<DrawItem *>(&sm.hist[0][0]);
#pragma unroll
    for (int q = 0; q < GPT; ++q) {
      const uint32_t bits = (kept >> (4 * q)) & 0xFu;
      if (bits) dl[pos++] = {q * kThreads + tid, bits, {x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]}};
    }
    __syncthreads();
    if (tid < (int)total) {
      const DrawItem it = dl[tid];
      const U64x4 w = philox_block(sv.seed, rkey, (uint64_t)t, (uint64_t)k, (uint64_t)it.g);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if ((it.bits >> j) & 1)
          keep_better(bv, bi, (double)it.x[j] + (double)gumbel_from_word(w.w[j]), 4 * it.g + j);
    }
    return block_argmax_f64(bv, bi, sm, slot);
  }
#pragma unroll
  for (int q = 0; q < GPT; ++q) {
    const uint32_t bits = (kept >> (4 * q)) & 0xFu;
    if (bits) {
      const int g = q * kThreads + tid;
      const U64x4 w = philox_block(sv.seed, rkey, (uint64_t)t, (uint64_t)k, (uint64_t)g);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if ((bits >> j) & 1)
          keep_better(bv, bi, (double)x[4 * q + j] + (double)gumbel_from_word(w.w[j]), 4 * g + j);
    }
  }
  return block_argmax_f64(bv, bi, sm, slot);
}

template <int GPT>
__global__ __launch_bounds__(kThreads) void sample_kernel(HeadView hv, StepView sv,
                                                          int with_text) {
  constexpr int EPL = 4 * GPT;
  __shared__ Smem<GPT> sm;
  const int tid = threadIdx.x;
  const int vec = blockIdx.x;
  const int n_audio = sv.Rs * hv.K;
  // histograms start at zero (published by the first block reduction)
  for (int b = tid; b <= kBins; b += kThreads) {
    sm.cnt[b] = 0;
    sm.mh[b] = 0;
  }
  sm.keepbits[tid] = 0;
  if (tid == 0) sm.lcount = 0;
  int slot = 0;

  // The scores depend only on the vector index: load them before anything
  // else so that their latency overlaps the plan and parameter loads.
  float x[EPL];
  uint32_t active = 0;
  const int V = hv.V;
  if (vec < n_audio) {
    const int s = vec / hv.K, k = vec % hv.K;
    const float *sc = sv.scores + (size_t)s * hv.N + (size_t)k * V;
    if ((V & 3) == 0) {
#pragma unroll
      for (int q = 0; q < GPT; ++q) {
        const int g = q * kThreads + tid;
        float4 v = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        if (4 * g < V) v = *reinterpret_cast<const float4 *>(sc + 4 * g);
        x[4 * q + 0] = v.x;
        x[4 * q + 1] = v.y;
        x[4 * q + 2] = v.z;
        x[4 * q + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const int e = 4 * ((i / 4) * kThreads + tid) + (i % 4);
        x[i] = e < V ? sc[e] : -INFINITY;
      }
    }
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = 4 * ((i / 4) * kThreads + tid) + (i % 4);
      if (e < V) active |= 1u << i;
    }
  }

  if (!plan_ok(sv)) {
    if (vec == 0 && tid == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }
  const int32_t *rows = sv.plan + kPlanHeader;
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
    const int tok = block_argmax_f32(bv, bi, sm, slot);
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
      const uint64_t rkey = sv.rng_key ? sv.rng_key[r] : (uint64_t)r;
      token = select_and_draw<GPT>(sv, x, active, V, T == 0.0f, sv.top_k[r], P, rkey, t, k, sm,
                                   slot);
      sampled = true;
    }
  }
  if (tid == 0) {
    sv.tokens_out[(size_t)r * hv.K + k] = token;
    if (u >= 0) sv.tokens_out[(size_t)u * hv.K + k] = token;
    const int gslot = sv.grid_slot[r];
    if (sampled && gslot >= 0 && sv.frame_grid) {
      if (gslot < sv.n_slots && f < sv.F_max)
        sv.frame_grid[((size_t)gslot * hv.K + k) * sv.F_max + f] = token;
      else
        atomicOr(sv.status, (uint32_t)MCD_DEV_GRID_RANGE);
    }
  }
}

template <int GPT>
hipError_t launch_gpt(const HeadView &hv, const StepView &sv, int nblk, bool with_text,
                      hipStream_t st) {
  hipLaunchKernelGGL(sample_kernel<GPT>, dim3(nblk), dim3(kThreads), 0, st, hv, sv,
                     (int)with_text);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sample(const HeadView &hv, const StepView &sv, bool with_text,
                         hipStream_t st) {
  const int nblk = sv.Rs * hv.K + (with_text ? sv.n_text : 0);
  if (nblk == 0) return hipSuccess;
  const int groups = (hv.V + 3) / 4;
  if (groups <= kThreads) return launch_gpt<1>(hv, sv, nblk, with_text, st);
  if (groups <= 2 * kThreads) return launch_gpt<2>(hv, sv, nblk, with_text, st);
  if (groups <= 4 * kThreads) return launch_gpt<4>(hv, sv, nblk, with_text, st);
  return hipErrorInvalidValue;
}

}  // namespace mcd
