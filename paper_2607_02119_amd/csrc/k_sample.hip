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
//   * Gumbel-max: token = argmax over kept ids of s_v + G_v, G_v = -log(-log u_v)
//     (G and the sum in fp32), lowest id on ties.  Counter-based Philox (Salmon, Moraes, Dror, Shaw,
//     SC'11) in two levels: the vector's key material D = Philox4x64-10 with
//     counter (0, k, t, rng_key) and key (seed, 0), once per vector; then for
//     id v the word v mod 4 of Philox4x32-10 with counter (v/4, lo D1, hi D1,
//     lo D2) and key (lo D0, hi D0); u = (top 23 bits + 1/2) * 2^-23;
//   * the token goes to the Main row, to its Companion (Sec. 2.4) and to the
//     request's frame grid cell [k][f].
//
// Layout: thread tid of a vector's TPV threads owns groups g = q * TPV + tid of
// four consecutive ids 4g .. 4g + 3 (one 16-byte load each), so that one
// Philox4x32 block serves a whole group from registers.
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
constexpr int kBins = 512;          // bins of width 1/16 below the maximum, plus one open bin
constexpr float kBinScale = 16.0f;

__device__ inline uint32_t order_key(float x) {
  if (x == 0.0f) x = 0.0f;  // -0 and +0 compare equal
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float key_to_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Uniform loads through the constant address space, so that they become
// scalar loads: they are counted apart from the vector loads of the scores and
// return without waiting for them.  The buffers are read-only in this kernel.
template <typename T>
__device__ __forceinline__ T ld_const(const T *p, int i) {
  return ((const __attribute__((address_space(4))) T *)p)[i];
}

// The plan header matches the step; every word is read (no short-circuit), so
// that the loads go out together.
__device__ inline bool plan_ok(const StepView &sv) {
  const int32_t *p = sv.plan;
  const bool magic = ld_const(p, kPlanMagicWord) == kPlanMagic;
  const bool r = ld_const(p, kPlanR) == sv.R, pairs = ld_const(p, kPlanPairs) == sv.n_pairs;
  const bool solo = ld_const(p, kPlanSolo) == sv.n_solo, text = ld_const(p, kPlanText) == sv.n_text;
  return magic & r & pairs & solo & text;
}

__device__ inline int lane_id() { return threadIdx.x & (kWave - 1); }

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

// ---- vector groups -------------------------------------------------------------
// A vector is handled by a group of TPV threads: one wave (TPV = 64, several
// vectors per workgroup, no workgroup barriers at all) or the whole 256-thread
// workgroup.  Group barriers and reductions follow the group.
template <int TPV>
struct Grp {
  static_assert(TPV == kWave || TPV == kThreads, "a wave or the workgroup");
  static constexpr int kGW = TPV / kWave;       // waves per group
  __device__ static int tid() { return (int)threadIdx.x % TPV; }
  __device__ static int wave() { return tid() / kWave; }
  __device__ static int index() { return (int)threadIdx.x / TPV; }
  __device__ static void sync() {
    if constexpr (TPV == kWave) {
      // one wave: its LDS accesses complete in program order; keep the
      // compiler from moving any across this point
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    } else {
      __syncthreads();
    }
  }
};

// A group of four ids with kept members, moved to the thread that draws it.
struct DrawItem {
  int g;
  uint32_t bits;
  float x[4];
};

template <int TPV>
struct Smem {
  // a cut-bin element; unused slots hold a sentinel that is never ahead of
  // a listed element (score -inf, id INT32_MAX), so the ranking can read the
  // list in whole blocks of kRankUnroll
  struct alignas(16) Entry {   // read as one uint4 by the ranking
    float v;
    int id;
    unsigned long long m;                // mass (top-p)
  };
  static constexpr int kDraw = TPV;      // kept groups dealt through the list (one per thread)
  uint32_t cnt[kBins + 1];               // top-k bin counts
  union {
    unsigned long long mh[kBins + 1];    // top-p bin masses (the last: the open bin)
    unsigned long long hist[3][256];     // radix select (fallback)
    DrawItem draw[kDraw];                // kept groups, once the selection is done
  } u;
  // elements of the cut bin (at most TPV)
  Entry le[TPV];
  uint32_t nkw[5];                       // the vector's noise key, from its first wave
  uint32_t keepbits[TPV];                // kept cut-bin elements, one bit per slot of a thread
  uint32_t lcount;
  // reductions across the waves of a group (two slots, alternating, one barrier each)
  uint32_t ru[2][Grp<TPV>::kGW];
  unsigned long long r64[2][Grp<TPV>::kGW];
  int ri[2][Grp<TPV>::kGW];
  float rx[2][Grp<TPV>::kGW], rf[2][Grp<TPV>::kGW], rf2[2][Grp<TPV>::kGW], rs[2][Grp<TPV>::kGW];
  unsigned long long r64b[2][Grp<TPV>::kGW];
};

template <int TPV>
__device__ __forceinline__ uint32_t grp_max_u32(uint32_t x, Smem<TPV> &sm, int &slot) {
  x = wave_max_u32(x);
  if constexpr (TPV == kWave) return x;
  if (lane_id() == 0) sm.ru[slot][Grp<TPV>::wave()] = x;
  Grp<TPV>::sync();
  uint32_t r = 0;
#pragma unroll
  for (int w = 0; w < Grp<TPV>::kGW; ++w) r = sm.ru[slot][w] > r ? sm.ru[slot][w] : r;
  slot ^= 1;
  return r;
}

template <int TPV>
__device__ __forceinline__ uint32_t grp_min_u32(uint32_t x, Smem<TPV> &sm, int &slot) {
  x = wave_min_u32(x);
  if constexpr (TPV == kWave) return x;
  if (lane_id() == 0) sm.ru[slot][Grp<TPV>::wave()] = x;
  Grp<TPV>::sync();
  uint32_t r = 0xFFFFFFFFu;
#pragma unroll
  for (int w = 0; w < Grp<TPV>::kGW; ++w) r = sm.ru[slot][w] < r ? sm.ru[slot][w] : r;
  slot ^= 1;
  return r;
}

template <int TPV>
__device__ __forceinline__ uint64_t grp_sum_u64(uint64_t x, Smem<TPV> &sm, int &slot) {
  x = readlane_u64(wave_incl_add_u64(x), 63);
  if constexpr (TPV == kWave) return x;
  if (lane_id() == 0) sm.r64[slot][Grp<TPV>::wave()] = x;
  Grp<TPV>::sync();
  uint64_t r = 0;
#pragma unroll
  for (int w = 0; w < Grp<TPV>::kGW; ++w) r += sm.r64[slot][w];
  slot ^= 1;
  return r;
}

// exclusive prefix of x over the group's threads in order, and the total
template <int TPV>
__device__ __forceinline__ uint32_t grp_excl_scan_u32(uint32_t x, uint32_t &total, Smem<TPV> &sm,
                                                      int &slot) {
  const uint32_t incl = wave_incl_add_u32(x);
  if constexpr (TPV == kWave) {
    total = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
    return incl - x;
  }
  if (lane_id() == 63) sm.ru[slot][Grp<TPV>::wave()] = incl;
  Grp<TPV>::sync();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < Grp<TPV>::kGW; ++w) {
    const uint32_t c = sm.ru[slot][w];
    if (w < Grp<TPV>::wave()) before += c;
    tot += c;
  }
  slot ^= 1;
  total = tot;
  return before + incl - x;
}

// inclusive prefix of x over the group's threads in order
template <int TPV>
__device__ __forceinline__ int grp_argmax_f32(float bv, int bi, Smem<TPV> &sm, int &slot) {
  wave_argmax_f32(bv, bi);
  if constexpr (TPV == kWave) return bi;
  if (lane_id() == 0) {
    sm.rs[slot][Grp<TPV>::wave()] = bv;
    sm.ri[slot][Grp<TPV>::wave()] = bi;
  }
  Grp<TPV>::sync();
  float rv = sm.rs[slot][0];
  int ri = sm.ri[slot][0];
#pragma unroll
  for (int w = 1; w < Grp<TPV>::kGW; ++w) keep_better(rv, ri, sm.rs[slot][w], sm.ri[slot][w]);
  slot ^= 1;
  return ri;
}

// A draw candidate: its perturbed score s = x + G (fp32), its id and its
// score x.  Candidates order by (s desc, id asc).
struct Cand {
  float s;
  int id;
  float x;
};

__device__ __forceinline__ void keep_cand(Cand &b, float s, int id, float x) {
  if (s > b.s || (s == b.s && id < b.id)) b = {s, id, x};
}

// One group reduction of a float sum (fixed order: the same result on every
// call with the same inputs) and of the best candidate: a single barrier for
// a workgroup group; every thread gets both.
template <int TPV>
__device__ __forceinline__ Cand grp_fsum_and_best(float &sum, Cand c, Smem<TPV> &sm, int &slot) {
  wave_scan([&](auto cc, auto m) __attribute__((always_inline)) {
    constexpr int C = decltype(cc)::value, RM = decltype(m)::value;
    const float os = __uint_as_float(dpp<C, RM>(0u, __float_as_uint(sum)));
    const float ov = __uint_as_float(dpp<C, RM>(__float_as_uint(-INFINITY), __float_as_uint(c.s)));
    const int oi = (int)dpp<C, RM>((uint32_t)INT32_MAX, (uint32_t)c.id);
    const float ox = __uint_as_float(dpp<C, RM>(__float_as_uint(-INFINITY), __float_as_uint(c.x)));
    sum += os;
    keep_cand(c, ov, oi, ox);
  });
  sum = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(sum), 63));
  c.s = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(c.s), 63));
  c.id = __builtin_amdgcn_readlane(c.id, 63);
  c.x = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(c.x), 63));
  if constexpr (TPV == kWave) return c;
  if (lane_id() == 0) {
    const int w = Grp<TPV>::wave();
    sm.rf[slot][w] = sum;
    sm.rs[slot][w] = c.s;
    sm.ri[slot][w] = c.id;
    sm.rx[slot][w] = c.x;
  }
  Grp<TPV>::sync();
  float t = 0.0f;
  Cand r = {-INFINITY, INT32_MAX, -INFINITY};
#pragma unroll
  for (int w = 0; w < Grp<TPV>::kGW; ++w) {
    t += sm.rf[slot][w];
    keep_cand(r, sm.rs[slot][w], sm.ri[slot][w], sm.rx[slot][w]);
  }
  slot ^= 1;
  sum = t;
  return r;
}

// The largest order key and the best candidate in one group reduction.
template <int TPV>
__device__ __forceinline__ Cand grp_max_and_best(uint32_t &mk, Cand c, Smem<TPV> &sm, int &slot) {
  wave_scan([&](auto cc, auto m) __attribute__((always_inline)) {
    constexpr int C = decltype(cc)::value, RM = decltype(m)::value;
    const uint32_t ok = dpp<C, RM>(0u, mk);
    const float ov = __uint_as_float(dpp<C, RM>(__float_as_uint(-INFINITY), __float_as_uint(c.s)));
    const int oi = (int)dpp<C, RM>((uint32_t)INT32_MAX, (uint32_t)c.id);
    const float ox = __uint_as_float(dpp<C, RM>(__float_as_uint(-INFINITY), __float_as_uint(c.x)));
    mk = ok > mk ? ok : mk;
    keep_cand(c, ov, oi, ox);
  });
  mk = (uint32_t)__builtin_amdgcn_readlane((int)mk, 63);
  c.s = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(c.s), 63));
  c.id = __builtin_amdgcn_readlane(c.id, 63);
  c.x = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(c.x), 63));
  if constexpr (TPV == kWave) return c;
  if (lane_id() == 0) {
    const int w = Grp<TPV>::wave();
    sm.ru[slot][w] = mk;
    sm.rs[slot][w] = c.s;
    sm.ri[slot][w] = c.id;
    sm.rx[slot][w] = c.x;
  }
  Grp<TPV>::sync();
  uint32_t t = 0;
  Cand r = {-INFINITY, INT32_MAX, -INFINITY};
#pragma unroll
  for (int w = 0; w < Grp<TPV>::kGW; ++w) {
    t = sm.ru[slot][w] > t ? sm.ru[slot][w] : t;
    keep_cand(r, sm.rs[slot][w], sm.ri[slot][w], sm.rx[slot][w]);
  }
  slot ^= 1;
  mk = t;
  return r;
}

// Two float sums (fixed order) and the best candidate in one group reduction.
template <int TPV>
__device__ __forceinline__ Cand grp_fsum2_and_best(float &a, float &b, Cand c, Smem<TPV> &sm,
                                                   int &slot) {
  wave_scan([&](auto cc, auto m) __attribute__((always_inline)) {
    constexpr int C = decltype(cc)::value, RM = decltype(m)::value;
    const float oa = __uint_as_float(dpp<C, RM>(0u, __float_as_uint(a)));
    const float ob = __uint_as_float(dpp<C, RM>(0u, __float_as_uint(b)));
    const float ov = __uint_as_float(dpp<C, RM>(__float_as_uint(-INFINITY), __float_as_uint(c.s)));
    const int oi = (int)dpp<C, RM>((uint32_t)INT32_MAX, (uint32_t)c.id);
    const float ox = __uint_as_float(dpp<C, RM>(__float_as_uint(-INFINITY), __float_as_uint(c.x)));
    a += oa;
    b += ob;
    keep_cand(c, ov, oi, ox);
  });
  a = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(a), 63));
  b = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(b), 63));
  c.s = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(c.s), 63));
  c.id = __builtin_amdgcn_readlane(c.id, 63);
  c.x = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(c.x), 63));
  if constexpr (TPV == kWave) return c;
  if (lane_id() == 0) {
    const int w = Grp<TPV>::wave();
    sm.rf[slot][w] = a;
    sm.rf2[slot][w] = b;
    sm.rs[slot][w] = c.s;
    sm.ri[slot][w] = c.id;
    sm.rx[slot][w] = c.x;
  }
  Grp<TPV>::sync();
  float ta = 0.0f, tb = 0.0f;
  Cand r = {-INFINITY, INT32_MAX, -INFINITY};
#pragma unroll
  for (int w = 0; w < Grp<TPV>::kGW; ++w) {
    ta += sm.rf[slot][w];
    tb += sm.rf2[slot][w];
    keep_cand(r, sm.rs[slot][w], sm.ri[slot][w], sm.rx[slot][w]);
  }
  slot ^= 1;
  a = ta;
  b = tb;
  return r;
}

// Two 64-bit sums in one group reduction.
template <int TPV>
__device__ __forceinline__ void grp_sum2_u64(uint64_t &a, uint64_t &b, Smem<TPV> &sm, int &slot) {
  a = readlane_u64(wave_incl_add_u64(a), 63);
  b = readlane_u64(wave_incl_add_u64(b), 63);
  if constexpr (TPV == kWave) return;
  if (lane_id() == 0) {
    sm.r64[slot][Grp<TPV>::wave()] = a;
    sm.r64b[slot][Grp<TPV>::wave()] = b;
  }
  Grp<TPV>::sync();
  uint64_t ta = 0, tb = 0;
#pragma unroll
  for (int w = 0; w < Grp<TPV>::kGW; ++w) {
    ta += sm.r64[slot][w];
    tb += sm.r64b[slot][w];
  }
  slot ^= 1;
  a = ta;
  b = tb;
}

// ---- Philox (Salmon, Moraes, Dror, Shaw, SC'11) ------------------------------
struct U64x4 {
  uint64_t w[4];
};

// Full 64 x 64 -> 128-bit product from four 32 x 32 -> 64-bit partial
// products, each a multiply-add whose addend cannot overflow it.
__device__ __forceinline__ void mulhilo64(uint64_t a, uint64_t b, uint64_t &lo, uint64_t &hi) {
  const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
  const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
  const uint64_t p00 = (uint64_t)a0 * b0;
  const uint64_t p01 = (uint64_t)a0 * b1 + (p00 >> 32);
  const uint64_t p10 = (uint64_t)a1 * b0 + (uint32_t)p01;
  hi = (uint64_t)a1 * b1 + ((p01 >> 32) + (p10 >> 32));
  lo = (p10 << 32) | (uint32_t)p00;
}

// Philox4x64-10: counter (x0, x1, x2, x3), key (k0, 0).
__device__ __forceinline__ U64x4 philox4x64(uint64_t x0, uint64_t x1, uint64_t x2, uint64_t x3,
                                   uint64_t k0) {
  const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
  uint64_t k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B97F4A7C15ull;
      k1 += 0xBB67AE8584CAA73Bull;
    }
    uint64_t lo0, hi0, lo1, hi1;
    mulhilo64(m0, x0, lo0, hi0);
    mulhilo64(m1, x2, lo1, hi1);
    const uint64_t y0 = hi1 ^ x1 ^ k0, y2 = hi0 ^ x3 ^ k1;
    x0 = y0;
    x1 = lo1;
    x2 = y2;
    x3 = lo0;
  }
  return U64x4{{x0, x1, x2, x3}};
}

// The key material of one vector: Philox4x32-10 key (k0, k1) and counter
// words 1..3 of every id's block.
struct NoiseKey {
  uint32_t k0, k1, c1, c2, c3;
};

__device__ __forceinline__ NoiseKey noise_key(uint64_t seed, uint64_t rng_key, int t, int k) {
  const U64x4 d = philox4x64(0, (uint64_t)k, (uint64_t)t, rng_key, seed);
  return NoiseKey{(uint32_t)d.w[0], (uint32_t)(d.w[0] >> 32), (uint32_t)d.w[1],
                  (uint32_t)(d.w[1] >> 32), (uint32_t)d.w[2]};
}

// A uniform 32-bit value copied to a vector register, so that what is
// computed from it runs on the vector unit.
__device__ __forceinline__ uint32_t in_vgpr(uint32_t x) {
  uint32_t y;
  asm volatile("v_mov_b32 %0, %1" : "=v"(y) : "s"(x));
  return y;
}

// The same key computed by every wave on the vector unit, whose 32 x 32 -> 64
// multiply-adds shorten the chain of 64-bit products that the scalar unit
// would run one 32-bit half at a time; the result is uniform again.
__device__ __forceinline__ NoiseKey noise_key_vector_unit(uint64_t seed, uint64_t rng_key, int t,
                                                          int k) {
  auto v64 = [](uint64_t x) __attribute__((always_inline)) {
    return ((uint64_t)in_vgpr((uint32_t)(x >> 32)) << 32) | in_vgpr((uint32_t)x);
  };
  const U64x4 d = philox4x64(0, (uint64_t)in_vgpr((uint32_t)k), (uint64_t)in_vgpr((uint32_t)t),
                             v64(rng_key), v64(seed));
  auto s32 = [](uint64_t x) __attribute__((always_inline)) {
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  };
  return NoiseKey{s32(d.w[0]), s32(d.w[0] >> 32), s32(d.w[1]), s32(d.w[1] >> 32), s32(d.w[2])};
}

struct U32x4 {
  uint32_t w[4];
};

// Philox4x32-10 block of the ids 4g .. 4g + 3 of a vector: counter
// (g, c1, c2, c3), key (k0, k1); each round is two 32 x 32 -> 64-bit products.
__device__ __forceinline__ U32x4 noise_block(const NoiseKey &nk, uint32_t g) {
  uint32_t x0 = g, x1 = nk.c1, x2 = nk.c2, x3 = nk.c3, k0 = nk.k0, k1 = nk.k1;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * x0, p1 = (uint64_t)0xCD9E8D57u * x2;
    const uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0, y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    x0 = y0;
    x1 = (uint32_t)p1;
    x2 = y2;
    x3 = (uint32_t)p0;
  }
  return U32x4{{x0, x1, x2, x3}};
}

// Gumbel variate from one Philox word, in fp32.  The uniform is exact in fp32;
// with base-2 logarithms, -ln(-ln u) = -ln(ln 2) - ln 2 * log2(-log2 u), and
// both log2 inputs are normal numbers (-log2 u >= 2^-24 / ln 2), where the
// hardware log2 is accurate to about one ulp: G is within ~1e-6 of its value.
__device__ __forceinline__ float gumbel_from_word(uint32_t x) {
  const float u = ((float)(x >> 9) + 0.5f) * 0x1p-23f;
  const float e = -__builtin_amdgcn_logf(u);   // -log2 u, in (0, 23]
  return fmaf(-0.69314718055994531f, __builtin_amdgcn_logf(e), 0.36651292058166435f);
}

// Top-p mass of a score: exp(s - max) in fp32 (relative error ~1e-7), scaled
// by 2^48 and converted exactly to a 64-bit integer.  Recomputed where needed
// (the same value every time) rather than kept in registers.
__device__ __forceinline__ uint64_t mass_of(float s, float mx) {
  return (uint64_t)ldexpf(expf(s - mx), 48);
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
template <int GPT, int TPV, bool MASS>
__device__ __forceinline__ Cut radix_select(const float (&x)[4 * GPT], uint32_t active,
                                            float mx, uint64_t target, Smem<TPV> &sm,
                                            int &pass) {
  constexpr int EPL = 4 * GPT;
  const int gt = Grp<TPV>::tid(), lane = lane_id();
  uint32_t prefix = 0, pmask = 0;
  uint64_t rem = target;
  for (int shift = 24; shift >= 0; shift -= 8) {
    unsigned long long *h = sm.u.hist[pass % 3];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const uint32_t key = order_key(x[i]);
      if (((active >> i) & 1) && (key & pmask) == prefix) {
        const uint32_t d = (key >> shift) & 255u;
        atomicAdd(&h[d], MASS ? (unsigned long long)mass_of(x[i], mx) : 1ull);
      }
    }
    Grp<TPV>::sync();
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
    for (int b = gt; b < 256; b += TPV) sm.u.hist[(pass + 2) % 3][b] = 0;
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
// slot 4q + j of group thread t: 4 (q * TPV + t) + j).
template <int GPT, int TPV>
__device__ __forceinline__ uint32_t apply_cut(const float (&x)[4 * GPT], uint32_t active,
                                              const Cut &c, uint64_t need_n, Smem<TPV> &sm,
                                              int &slot) {
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
    const uint32_t before = grp_excl_scan_u32<TPV>((uint32_t)__popc(tq), total, sm, slot);
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

// id of register slot i of group thread t
template <int TPV>
__device__ __forceinline__ int id_of(int i, int t) {
  return 4 * ((i / 4) * TPV + t) + (i % 4);
}

// Group thread that owns id e, and the slot of e in its registers.
template <int TPV>
__device__ __forceinline__ void owner_of(int e, int &thread, int &slot) {
  const int g = e >> 2;
  thread = g % TPV;
  slot = 4 * (g / TPV) + (e & 3);
}

constexpr int kRankUnroll = 4;

template <int TPV>
__device__ __forceinline__ void set_sentinel(typename Smem<TPV>::Entry &e) {
  e = {-INFINITY, INT32_MAX, 0ull};
}

// Decide the listed elements of a cut bin (n <= TPV): entry t is ranked by
// (score desc, id asc) against all the others; top-k keeps it when fewer than
// `need` entries are ahead of it, top-p (MASS) when the mass ahead of it plus
// `above` is still below `target`.  Kept entries set their owner's bit.  The
// list is read in blocks of kRankUnroll (sentinels pad the last one), so that
// the reads of a block are in flight together.
template <int TPV, bool MASS>
__device__ __forceinline__ void rank_and_keep(Smem<TPV> &sm, int n, uint64_t need,
                                              uint64_t above, uint64_t target) {
  static_assert(TPV % kRankUnroll == 0, "whole blocks");
  using Entry = typename Smem<TPV>::Entry;
  const int t = Grp<TPV>::tid();
  if (t >= n) return;
  const Entry me = sm.le[t];
  int r = 0;
  uint64_t before = 0;
  for (int j = 0; j < n; j += kRankUnroll) {
    uint4 o[kRankUnroll];   // whole 16-byte entries: v, id, m (low, high)
#pragma unroll
    for (int q = 0; q < kRankUnroll; ++q) o[q] = *reinterpret_cast<const uint4 *>(&sm.le[j + q]);
#pragma unroll
    for (int q = 0; q < kRankUnroll; ++q) {
      const float ov = __uint_as_float(o[q].x);
      const int oid = (int)o[q].y;
      const bool ahead = (ov > me.v) | ((ov == me.v) & (oid < me.id));
      r += ahead ? 1 : 0;
      if constexpr (MASS) {
        // an opaque mask rather than a select: the mass read then stays in
        // the batch instead of becoming a read behind a branch
        uint32_t msk = ahead ? 0xFFFFFFFFu : 0u;
        asm volatile("" : "+v"(msk));
        before += (uint64_t)(o[q].w & msk) << 32 | (o[q].z & msk);
      }
    }
  }
  const bool keep = MASS ? (above + before < target) : ((uint64_t)r < need);
  if (keep) {
    int ow, sl;
    owner_of<TPV>(me.id, ow, sl);
    atomicOr(&sm.keepbits[ow], 1u << sl);
  }
}

// Append the active elements of bin `bc` to the cut-bin list: one list
// reservation per thread.  Slots at or beyond TPV are not written (the caller
// falls back to the radix select when the count exceeds TPV).
template <int GPT, int TPV, bool MASS>
__device__ __forceinline__ void list_bin(Smem<TPV> &sm, const float (&x)[4 * GPT],
                                         const int (&bin)[4 * GPT], int bc, float mx) {
  constexpr int EPL = 4 * GPT;
  const int gt = Grp<TPV>::tid();
  uint32_t c = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) c += bin[i] == bc ? 1u : 0u;
  if (c == 0) return;
  uint32_t pos = atomicAdd(&sm.lcount, c);
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    if (bin[i] == bc) {
      if (pos < (uint32_t)TPV) sm.le[pos] = {x[i], id_of<TPV>(i, gt), MASS ? mass_of(x[i], mx) : 0ull};
      ++pos;
    }
  }
}

// After a ranking: the list slots go back to the sentinel (the next list
// build follows at least one group barrier).
template <int TPV>
__device__ __forceinline__ void clear_list(Smem<TPV> &sm, int n) {
  const int t = Grp<TPV>::tid();
  if (t < n) set_sentinel<TPV>(sm.le[t]);
}

// The radix buffers alias the top-p histogram: wait for its last readers.
template <int TPV>
__device__ __forceinline__ void zero_radix(Smem<TPV> &sm) {
  Grp<TPV>::sync();
  for (int b = Grp<TPV>::tid(); b < 2 * 256; b += TPV) sm.u.hist[b / 256][b % 256] = 0;
  Grp<TPV>::sync();
}

template <int GPT, int TPV>
__device__ __forceinline__ uint32_t radix_topk(const float (&x)[4 * GPT], uint32_t active,
                                               int top_k, Smem<TPV> &sm, int &slot, int &pass) {
  zero_radix(sm);
  const Cut c = radix_select<GPT, TPV, false>(x, active, 0.0f, (uint64_t)top_k, sm, pass);
  return apply_cut<GPT, TPV>(x, active, c, c.need, sm, slot);
}

template <int GPT, int TPV>
__device__ __forceinline__ uint32_t radix_topp(const float (&x)[4 * GPT], uint32_t active,
                                               float mx, uint64_t target, Smem<TPV> &sm,
                                               int &slot, int &pass) {
  zero_radix(sm);
  const Cut c = radix_select<GPT, TPV, true>(x, active, mx, target, sm, pass);
  uint64_t need_n = 0;
  if (c.exact) {
    // every element tied at kappa carries the same mass q: the fewest reaching rem
    uint64_t q = 0;
#pragma unroll
    for (int i = 0; i < 4 * GPT; ++i)
      if (((active >> i) & 1) && order_key(x[i]) == c.lo) q = mass_of(x[i], mx);
    // every nonzero q is the same value, so the halves reduce independently
    const uint64_t qhi = grp_max_u32<TPV>((uint32_t)(q >> 32), sm, slot);
    const uint64_t qlo = grp_max_u32<TPV>((uint32_t)q, sm, slot);
    q = qhi << 32 | qlo;
    need_n = q ? (c.need + q - 1) / q : 1;
  }
  return apply_cut<GPT, TPV>(x, active, c, need_n, sm, slot);
}

// top-k over the active set; `mx` is the maximum active score
template <int GPT, int TPV>
__device__ __forceinline__ uint32_t select_topk(const float (&x)[4 * GPT], uint32_t active,
                                                float mx, int top_k, Smem<TPV> &sm, int &slot,
                                                int &pass, int V, bool &u_dirty) {
  constexpr int EPL = 4 * GPT;
  const int gt = Grp<TPV>::tid();
  int bin[EPL];
  bins_of<GPT>(x, active, mx, bin);
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (bin[i] >= 0 && bin[i] < kBins) atomicAdd(&sm.cnt[bin[i]], 1u);
  Grp<TPV>::sync();
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
  if (bc == kBins || inbin > (uint64_t)TPV) {
    u_dirty = true;
    return radix_topk<GPT, TPV>(x, active, top_k, sm, slot, pass);
  }
  list_bin<GPT, TPV, false>(sm, x, bin, bc, 0.0f);
  Grp<TPV>::sync();
  rank_and_keep<TPV, false>(sm, (int)inbin, need, 0, 0);
  Grp<TPV>::sync();
  clear_list<TPV>(sm, (int)inbin);
  keep = sm.keepbits[gt];
  sm.keepbits[gt] = 0;          // next use follows at least one group barrier
  if (gt == 0) sm.lcount = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (bin[i] >= 0 && bin[i] < bc) keep |= 1u << i;
  return keep;
}

// top-p over the active set (the survivors of top-k); `mx` is their maximum.
// The mass histogram is zero on entry unless `u_dirty` (top-k used the radix
// buffers that share its storage).
template <int GPT, int TPV>
__device__ __forceinline__ uint32_t select_topp(const float (&x)[4 * GPT], uint32_t active,
                                                float mx, float top_p, Smem<TPV> &sm, int &slot,
                                                int &pass, bool u_dirty) {
  constexpr int EPL = 4 * GPT;
  const int gt = Grp<TPV>::tid(), lane = lane_id();
  if (u_dirty) {   // group-uniform
    Grp<TPV>::sync();
    for (int b = gt; b <= kBins; b += TPV) sm.u.mh[b] = 0;
    Grp<TPV>::sync();
  }
  // every active element adds its mass to its bin (the open bin included), so
  // the bins also give the total
  int bin[EPL];
  bins_of<GPT>(x, active, mx, bin);
  if constexpr (TPV == kWave) Grp<TPV>::sync();   // the clearing stores before the adds
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (bin[i] >= 0) atomicAdd(&sm.u.mh[bin[i]], (unsigned long long)mass_of(x[i], mx));
  Grp<TPV>::sync();
  // every wave scans the bins: the total Z, the target ceil(p Z), the cut bin
  uint64_t v[8], lsum = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    v[j] = sm.u.mh[8 * lane + j];
    lsum += v[j];
  }
  const uint64_t incl = wave_incl_add_u64(lsum);
  const uint64_t excl = incl - lsum;
  const uint64_t Z = readlane_u64(incl, 63) + sm.u.mh[kBins];
  uint64_t target = (uint64_t)ceil((double)top_p * (double)Z);
  if (target < 1) target = 1;
  if (target > Z) return active;
  const uint64_t bal = __ballot(excl < target && incl >= target);
  if (bal == 0) return radix_topp<GPT, TPV>(x, active, mx, target, sm, slot, pass);
  const int src = __ffsll((long long)bal) - 1;
  uint64_t cum = readlane_u64(excl, src), above = cum;
  int bc = 0;
  bool found = false;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint64_t vj = readlane_u64(v[j], src);
    if (!found && cum + vj >= target) {
      bc = 8 * src + j;
      above = cum;
      found = true;
    }
    cum += vj;
  }
  list_bin<GPT, TPV, true>(sm, x, bin, bc, mx);
  Grp<TPV>::sync();
  const int n = (int)sm.lcount;
  if (n > TPV) {
    Grp<TPV>::sync();   // everyone has read lcount
    if (gt == 0) sm.lcount = 0;
    clear_list<TPV>(sm, TPV);
    return radix_topp<GPT, TPV>(x, active, mx, target, sm, slot, pass);
  }
  rank_and_keep<TPV, true>(sm, n, 0, above, target);
  Grp<TPV>::sync();
  clear_list<TPV>(sm, n);
  uint32_t keep = sm.keepbits[gt];
  sm.keepbits[gt] = 0;
  if (gt == 0) sm.lcount = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (bin[i] >= 0 && bin[i] < bc) keep |= 1u << i;
  return keep;
}

// Draw without a top-k cut (not greedy).  The token is the best candidate
// (s = x + G desc, id asc) inside the nucleus, and the nucleus is a prefix of
// the score order (x desc, id asc): an element is inside iff the mass strictly
// ahead of it is below p Z (with the fixed-point masses of mass_of, below
// ceil(p Z)).  So test the best candidate c; if it is outside, so is every
// element behind it, and the next candidate is the best one ahead of c.  The
// first candidate comes with the maximum (one group reduction), its test with
// the total mass (a second one); each further test is one more.  The first
// element of the score order has nothing ahead of it, so the loop ends.  The
// sampled candidate is outside with probability 1 - p.
//
// The masses of the tests are fp32 (hardware exp2), within a relative 2.5e-6
// of the fixed-point ones in the sums: a test is decided on them unless the
// mass ahead is within kNucleusMargin Z of p Z, and then on the fixed-point
// sums, so that the outcome is always that of the fixed-point rule.
constexpr float kNucleusMargin = 3e-5f;

template <int GPT, int TPV>
__device__ __forceinline__ int draw_nucleus(const float (&x)[4 * GPT], uint32_t active,
                                            const NoiseKey &nk, float top_p, Smem<TPV> &sm,
                                            int &slot) {
  constexpr int EPL = 4 * GPT;
  const int gt = Grp<TPV>::tid();
  float gn[EPL];
#pragma unroll
  for (int q = 0; q < GPT; ++q) {
    const U32x4 wd = noise_block(nk, (uint32_t)(q * TPV + gt));
#pragma unroll
    for (int j = 0; j < 4; ++j) gn[4 * q + j] = gumbel_from_word(wd.w[j]);
  }
  uint32_t mk = 0;
  Cand c = {-INFINITY, INT32_MAX, -INFINITY};
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    if (!((active >> i) & 1)) continue;
    const uint32_t key = order_key(x[i]);
    mk = key > mk ? key : mk;
    keep_cand(c, x[i] + gn[i], id_of<TPV>(i, gt), x[i]);
  }
  c = grp_max_and_best<TPV>(mk, c, sm, slot);
  // no orderable candidate (every score NaN): the lowest id
  if (c.id == INT32_MAX) return 0;
  if (!(top_p < 1.0f)) return c.id;
  const float mx = key_to_float(mk);
  auto ahead = [&](int i, const Cand &o) __attribute__((always_inline)) {
    const int id = id_of<TPV>(i, gt);
    return ((active >> i) & 1) && ((x[i] > o.x) | ((x[i] == o.x) & (id < o.id)));
  };
  // fp32 mass, recomputed in each pass (three instructions) rather than held
  auto mass_f = [&](int i) __attribute__((always_inline)) {
    return __builtin_amdgcn_exp2f((x[i] - mx) * 1.4426950408889634f);
  };
  float zf = 0.0f, af = 0.0f;
  Cand nc = {-INFINITY, INT32_MAX, -INFINITY};
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const float m = ((active >> i) & 1) ? mass_f(i) : 0.0f;
    zf += m;
    if (ahead(i, c)) {
      af += m;
      keep_cand(nc, x[i] + gn[i], id_of<TPV>(i, gt), x[i]);
    }
  }
  nc = grp_fsum2_and_best<TPV>(zf, af, nc, sm, slot);
  const float pz = top_p * zf, margin = kNucleusMargin * zf;
  for (;;) {   // group-uniform
    bool inside = af < pz;
    if (fabsf(af - pz) <= margin) {
      // near the cut: the fixed-point rule, mass ahead of c < ceil(p Z)
      // (one element after the other: the empty asm statements keep their
      // order, so that the masses are not all live at once)
      uint64_t z = 0, a = 0;
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        if (!((active >> i) & 1)) continue;
        float xi = x[i];
        asm volatile("" : "+v"(xi));
        const uint64_t m = mass_of(xi, mx);
        z += m;
        if (ahead(i, c)) a += m;
        asm volatile("" : "+v"(z), "+v"(a));
      }
      grp_sum2_u64<TPV>(z, a, sm, slot);
      uint64_t target = (uint64_t)ceil((double)top_p * (double)z);
      if (target < 1) target = 1;
      inside = a < target;
    }
    // nothing ahead of c (reached only if the masses are not finite): c
    if (inside || nc.id == INT32_MAX) return c.id;
    // c is outside: test the best candidate ahead of it, strictly earlier in
    // the score order, so the loop ends after at most V tests
    c = nc;
    af = 0.0f;
    nc = {-INFINITY, INT32_MAX, -INFINITY};
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      if (ahead(i, c)) {
        af += mass_f(i);
        keep_cand(nc, x[i] + gn[i], id_of<TPV>(i, gt), x[i]);
      }
    }
    nc = grp_fsum_and_best<TPV>(af, nc, sm, slot);
  }
}

template <int GPT, int TPV>
__device__ __forceinline__ int select_and_draw(const StepView &sv, const float (&x)[4 * GPT],
                                               uint32_t active, int V, bool greedy, int top_k,
                                               float top_p, const NoiseKey &nk_in,
                                               Smem<TPV> &sm, int &slot) {
  constexpr int EPL = 4 * GPT;
  const int gt = Grp<TPV>::tid();
  uint32_t mk = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if ((active >> i) & 1) {
      const uint32_t key = order_key(x[i]);
      mk = key > mk ? key : mk;
    }
  // also publishes the cleared count histogram (one barrier for a workgroup group)
  mk = grp_max_u32<TPV>(mk, sm, slot);
  if constexpr (TPV == kWave) Grp<TPV>::sync();
  if (greedy) {
    uint32_t id = 0xFFFFFFFFu;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (((active >> i) & 1) && order_key(x[i]) == mk) {
        const uint32_t e = (uint32_t)id_of<TPV>(i, gt);
        id = e < id ? e : id;
      }
    return (int)grp_min_u32<TPV>(id, sm, slot);
  }
  const float mx = key_to_float(mk);
  // a workgroup group's key, published by its first wave before the barrier
  // of the maximum
  NoiseKey nk = nk_in;
  if constexpr (TPV != kWave) nk = NoiseKey{sm.nkw[0], sm.nkw[1], sm.nkw[2], sm.nkw[3], sm.nkw[4]};
  int pass = 0;
  bool u_dirty = false;
  uint32_t kept = active;
  if (top_k > 0 && top_k < V)
    kept = select_topk<GPT, TPV>(x, kept, mx, top_k, sm, slot, pass, V, u_dirty);
  if (top_p < 1.0f) kept = select_topp<GPT, TPV>(x, kept, mx, top_p, sm, slot, pass, u_dirty);
  // Gumbel-max over the kept ids, one Philox block per group of four ids
  float bv = -INFINITY;
  int bi = INT32_MAX;
  auto draw = [&](int g, uint32_t bits, float x0, float x1, float x2, float x3)
                  __attribute__((always_inline)) {
    const U32x4 w = noise_block(nk, (uint32_t)g);
    const float xs[4] = {x0, x1, x2, x3};
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if ((bits >> j) & 1) keep_better(bv, bi, xs[j] + gumbel_from_word(w.w[j]), 4 * g + j);
  };
  // When there are at most as many groups with kept ids as threads (top-k
  // cuts of up to TPV ids always), they move to an LDS list and each thread
  // draws one, so that no thread runs several Philox blocks while others
  // idle.  More groups (a wide top-k or top-p set) are drawn by their owner
  // threads: as many blocks per thread as kept groups it holds.  A list of one
  // entry per thread keeps the sampler's LDS small enough for eight
  // workgroups per compute unit.
  uint32_t n = 0;
#pragma unroll
  for (int q = 0; q < GPT; ++q) n += ((kept >> (4 * q)) & 0xFu) ? 1u : 0u;
  uint32_t total;
  uint32_t pos = grp_excl_scan_u32<TPV>(n, total, sm, slot);
  if (total <= (uint32_t)Smem<TPV>::kDraw) {   // group-uniform
    // the list shares its storage with the histograms and radix buffers: their
    // last readers are past the scan (or, in one wave, earlier in program order)
    if constexpr (TPV == kWave) Grp<TPV>::sync();
    DrawItem *dl = sm.u.draw;
#pragma unroll
    for (int q = 0; q < GPT; ++q) {
      const uint32_t bits = (kept >> (4 * q)) & 0xFu;
      if (bits) dl[pos++] = {q * TPV + gt, bits, {x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]}};
    }
    Grp<TPV>::sync();
    if (gt < (int)total) {
      const DrawItem it = dl[gt];
      draw(it.g, it.bits, it.x[0], it.x[1], it.x[2], it.x[3]);
    }
  } else {
#pragma unroll
    for (int q = 0; q < GPT; ++q) {
      const uint32_t bits = (kept >> (4 * q)) & 0xFu;
      if (bits) draw(q * TPV + gt, bits, x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]);
    }
  }
  return grp_argmax_f32<TPV>(bv, bi, sm, slot);
}

// One vector per group of TPV threads: 256 / TPV vectors per workgroup.
template <int GPT, int TPV>
__global__ __launch_bounds__(kThreads) void sample_kernel(HeadView hv, StepView sv,
                                                          int with_text) {
  constexpr int EPL = 4 * GPT;
  constexpr int G = kThreads / TPV;
  __shared__ Smem<TPV> smem[G];
  Smem<TPV> &sm = smem[Grp<TPV>::index()];
  const int gt = Grp<TPV>::tid();
  // the same for every lane of a wave: a scalar value
  const int vec = __builtin_amdgcn_readfirstlane((int)blockIdx.x * G + Grp<TPV>::index());
  const int n_audio = sv.Rs * hv.K;
  if (vec >= n_audio + (with_text ? sv.n_text : 0)) return;   // a whole group
  // the histograms start at zero (published by the first group reduction)
  for (int b = gt; b <= kBins; b += TPV) {
    sm.cnt[b] = 0;
    sm.u.mh[b] = 0;
  }
  sm.keepbits[gt] = 0;
  set_sentinel<TPV>(sm.le[gt]);
  if (gt == 0) sm.lcount = 0;
  int slot = 0;

  const bool audio = vec < n_audio;
  const int s = audio ? vec / hv.K : 0, k = audio ? vec % hv.K : 0;
  // The scores depend only on the vector index: their loads go out first.
  float x[EPL];
  uint32_t active = 0;
  // stream k's block of the score row: V ids from column off
  const int off = hv.voff.o[k];
  const int V = hv.voff.o[k + 1] - off;
  if (audio) {
    const float *sc = sv.scores + (size_t)s * hv.N + off;
    if (((V | off | hv.N) & 3) == 0) {   // 16-byte aligned whole groups
#pragma unroll
      for (int q = 0; q < GPT; ++q) {
        const int g = q * TPV + gt;
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
        const int e = id_of<TPV>(i, gt);
        x[i] = e < V ? sc[e] : -INFINITY;
      }
    }
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (id_of<TPV>(i, gt) < V) active |= 1u << i;
  }

  // Row lookups (scalar loads): the plan rows of this vector and the row's
  // parameters, read at a clamped index before any of them is checked, so that
  // they are in flight together while the score loads are outstanding.
  const bool plan_good = plan_ok(sv);
  const int32_t *rows = sv.plan + kPlanHeader;
  const bool paired = audio && s < sv.n_pairs;
  const int ri = !audio ? sv.Mg + (vec - n_audio) : paired ? 2 * s : 2 * sv.n_pairs + (s - sv.n_pairs);
  const int r = ld_const(rows, ri);
  const int u_row = ld_const(rows, paired ? 2 * s + 1 : ri);
  const int u = paired ? u_row : -1;
  const bool row_ok = r >= 0 && r < sv.R && u < sv.R;
  const int rc = row_ok ? r : 0;
  const int t = ld_const(sv.step, rc);
  const int nf = ld_const(sv.n_frames, rc);
  const float T = ld_const(sv.temperature, rc), P = ld_const(sv.top_p, rc);
  const int top_k = ld_const(sv.top_k, rc);
  const float w_row = ld_const(sv.cfg_w, rc);
  const float w = paired ? w_row : 0.0f;
  const uint64_t rkey = sv.rng_key ? ld_const(sv.rng_key, rc) : (uint64_t)rc;
  const int gslot = ld_const(sv.grid_slot, rc);

  if (!plan_good || !row_ok) {
    // A plan that does not match the step: flag it and make this vector's
    // outputs the pad id wherever its rows are inside the batch, so stale
    // tokens of an earlier step are never left in place.
    if (gt == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    const bool r_in = r >= 0 && r < sv.R, u_in = u >= 0 && u < sv.R;
    if (audio) {
      if (gt == 0 && r_in) sv.tokens_out[(size_t)r * hv.K + k] = hv.pad_id;
      if (gt == 0 && u_in) sv.tokens_out[(size_t)u * hv.K + k] = hv.pad_id;
    } else if (r_in) {
      for (int kk = gt; kk < hv.K; kk += TPV) sv.tokens_out[(size_t)r * hv.K + kk] = hv.pad_id;
    }
    return;
  }
  if (!audio) {
    // text row: reduce the (max, lowest argmax) partials of the text GEMM.
    // The text phase's mask (Sec. 2.3): the token is the best over the text
    // ids [0, T_text), whole 32-column parts; the modality is where the best
    // over all ids lies (text ids are the lower ones, so ties stay text).
    const int j = vec - n_audio;
    const int tparts = hv.T_text / kTextPartCols;   // T_text < V_text: a multiple of 32
    const bool masked = hv.T_text < hv.V_text;
    float bv = -INFINITY, av = -INFINITY;
    int bi = INT32_MAX, ai = INT32_MAX;
    for (int p = gt; p < sv.text_parts; p += TPV) {
      const float v = sv.text_val[(size_t)j * sv.text_parts + p];
      const int i = sv.text_idx[(size_t)j * sv.text_parts + p];
      if (!masked || p < tparts) keep_better(bv, bi, v, i);
      keep_better(av, ai, v, i);
    }
    const int tok = grp_argmax_f32<TPV>(bv, bi, sm, slot);
    int leave = 0;
    if (masked) leave = grp_argmax_f32<TPV>(av, ai, sm, slot) >= hv.T_text;
    for (int kk = gt; kk < hv.K; kk += TPV)
      sv.tokens_out[(size_t)r * hv.K + kk] = (kk == 0) ? tok : hv.pad_id;
    if (sv.modality_out && gt == 0) sv.modality_out[r] = (uint8_t)leave;
    return;
  }
  const int f = t - hv.delays.d[k];
  const bool pad = f < 0 || (nf >= 0 && f >= nf);
  int token = hv.pad_id;
  bool sampled = false;
  if (!pad) {
    const bool bad = !(T >= 0.0f) || isinf(T) || !(P > 0.0f) || (paired && !isfinite(w));
    if (bad) {
      if (gt == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PARAM);
    } else {
      // The vector's noise key (64-bit multiplies on uniform values).  A
      // one-wave group derives it on the vector unit (a shorter chain than the
      // scalar unit's 32-bit halves).  In a workgroup group the first wave
      // derives it on the scalar unit, beside the other waves' vector work,
      // and publishes it in LDS; the first group barrier makes it visible
      // (the maximum's in the top-k path, the one below otherwise).
      NoiseKey nk{0, 0, 0, 0, 0};
      if constexpr (TPV == kWave) {
        if (T != 0.0f) nk = noise_key_vector_unit(sv.seed, rkey, t, k);
      } else if (T != 0.0f && Grp<TPV>::wave() == 0) {
        const NoiseKey w0 = noise_key(sv.seed, rkey, t, k);
        if (lane_id() == 0) {
          sm.nkw[0] = w0.k0;
          sm.nkw[1] = w0.k1;
          sm.nkw[2] = w0.c1;
          sm.nkw[3] = w0.c2;
          sm.nkw[4] = w0.c3;
        }
      }
      if (T != 0.0f && !(top_k > 0 && top_k < V)) {
        // no top-k cut: candidates in perturbed-score order tested against the
        // nucleus (the noise of every id)
        Grp<TPV>::sync();
        if constexpr (TPV != kWave)
          nk = NoiseKey{sm.nkw[0], sm.nkw[1], sm.nkw[2], sm.nkw[3], sm.nkw[4]};
        token = draw_nucleus<GPT, TPV>(x, active, nk, P, sm, slot);
      } else {
        token = select_and_draw<GPT, TPV>(sv, x, active, V, T == 0.0f, top_k, P, nk, sm, slot);
      }
      sampled = true;
    }
  }
  if (gt == 0) {
    sv.tokens_out[(size_t)r * hv.K + k] = token;
    if (u >= 0) sv.tokens_out[(size_t)u * hv.K + k] = token;
    if (sampled && gslot >= 0 && sv.frame_grid) {
      if (gslot < sv.n_slots && f < sv.F_max)
        sv.frame_grid[((size_t)gslot * hv.K + k) * sv.F_max + f] = token;
      else
        atomicOr(sv.status, (uint32_t)MCD_DEV_GRID_RANGE);
    }
  }
}

template <int GPT, int TPV>
hipError_t launch_gpt(const HeadView &hv, const StepView &sv, int nvec, bool with_text,
                      hipStream_t st) {
  constexpr int G = kThreads / TPV;
  hipLaunchKernelGGL((sample_kernel<GPT, TPV>), dim3((nvec + G - 1) / G), dim3(kThreads), 0, st,
                     hv, sv, (int)with_text);
  return hipGetLastError();
}

}  // namespace

// One wave per vector when there are many vectors of at most 1024 ids (more
// vectors in flight per compute unit, no workgroup barriers); one workgroup per
// vector otherwise (shorter latency per vector).
constexpr int kWaveVectorsMin = 1024;

hipError_t launch_sample(const HeadView &hv, const StepView &sv, bool with_text,
                         hipStream_t st) {
  const int nvec = sv.Rs * hv.K + (with_text ? sv.n_text : 0);
  if (nvec == 0) return hipSuccess;
  const int groups = (hv.V + 3) / 4;
  if (nvec >= kWaveVectorsMin && groups <= 4 * kWave) {
    if (groups <= kWave) return launch_gpt<1, kWave>(hv, sv, nvec, with_text, st);
    if (groups <= 2 * kWave) return launch_gpt<2, kWave>(hv, sv, nvec, with_text, st);
    return launch_gpt<4, kWave>(hv, sv, nvec, with_text, st);
  }
  if (groups <= kThreads) return launch_gpt<1, kThreads>(hv, sv, nvec, with_text, st);
  if (groups <= 2 * kThreads) return launch_gpt<2, kThreads>(hv, sv, nvec, with_text, st);
  if (groups <= 4 * kThreads) return launch_gpt<4, kThreads>(hv, sv, nvec, with_text, st);
  return hipErrorInvalidValue;
}

}  // namespace mcd
