// Tile body of the K1 weight-streaming path (at most 128 GEMM rows per tile):
// codebook-head projection with the CFG merge and temperature fused into the
// epilogue, or the text-head projection with a fused (max, lowest argmax)
// epilogue.
//
//   logits[g][n] = sum_h hidden[row(g)][h] * W[n][h]         (Sec. 2.1, n = k*V + v)
//   pair p (GEMM rows 2p, 2p+1 = Main, Companion):
//     scores[p][n] = (w * l_main + (1 - w) * l_comp) / T    (Eq. 1, Sec. 2.4)
//   solo row j:  scores[n_pairs + j][n] = l / T;  T = 0 (greedy): no division
//   text rows:   per row and 32-column part, the largest logit and its lowest id.
#pragma once

#include "gemm_common.h"

namespace mcd {
namespace {

// Weight-streaming path, tiles of up to 128 rows.  A workgroup owns BM rows
// (all of them when there are at most 128) and BN columns.  Each k slice of SK = 64 (128 bytes of every weight and hidden
// row) goes into one of the LDS stages of its ring.  Waves 0-1 copy weight
// slices with global_load_lds_dwordx4 (64 lanes x 16 B, eight 128-byte row
// segments per instruction, no registers), SW - 1 slices ahead of their use.
// Waves 2-3 load hidden-state slices into registers HL slices ahead and write
// them to a two-stage ring one slice ahead.  Waves split the tile 2 x 2
// (column half w % 2, k32 half w / 2 of every slice; the two k halves meet in
// LDS at the end) or, for 256-column tiles, 4 x 1 (column quarter, all of k).
//
// Every byte a compute unit takes in, from HBM or from L2, crosses the L2 ->
// CU path, and that path (about 45-50 GB/s per CU measured) bounds the loop:
// the hidden states are re-read by every column tile, as many bytes per tile
// as its weights when BM = BN.  Wide tiles (BN = 256) halve that share; they
// are used when there is more than one round of 128-column tiles.
//
// LDS layout of a slice: [rows][8 chunks of 16 B]; chunk c of row r is stored
// at position c ^ ((r >> 1) & 7), so the 16 rows of an MFMA fragment read hit
// 16 distinct bank groups.  The weight waves wait for their copies explicitly
// (vector memory counter: only these copies are outstanding in their loop).
// No copy is issued past the last slice; in the last SW - 2 iterations the
// wait allows only the copies that are really still to come.  A copy only
// ever targets the stage read SW - 1 iterations earlier, after a barrier that
// follows every wave's reads of it.
constexpr int kDmaSK = 64;                 // k per slice
constexpr int kDmaLdsBudget = 160 * 1024;  // bytes of LDS for the two rings (all of it)

// Wait until at most min(ahead, MAXS) slices of PER copies each are still in
// flight (and no LDS operation).  `ahead` is wave-uniform: a scalar branch.
template <int PER, int MAXS>
__device__ __forceinline__ void wait_slices(int ahead) {
  if (ahead >= MAXS) {
    wait_vmem_and_lds<MAXS * PER>();
    return;
  }
  static_for<0, MAXS>([&](auto sc) __attribute__((always_inline)) {
    constexpr int s = decltype(sc)::value;
    if (ahead == s) wait_vmem_and_lds<s * PER>();
  });
}

// Tile shape of the streaming path, shared by its kernel and by the fused
// mixed-batch kernel (which sizes its LDS buffer from kLds).
template <int BM, int BN>
struct DmaShape {
  static constexpr int SK = kDmaSK;
  static constexpr int MB = BM / 32;         // 32-row MFMA blocks: all rows of the tile
  // Waves split the tile by columns and by k within a slice: 2 x 2 (column
  // half, k32 half) up to 128 columns, 4 x 1 (column quarter, all of k) for
  // wide tiles, so that a wave never holds more than 128 accumulators.
  static constexpr int KSPLIT = BN > 128 ? 1 : 2;  // k groups of waves
  static constexpr int CSPLIT = 4 / KSPLIT;        // column groups of waves
  static constexpr int KS = 4 / KSPLIT;            // k16 steps per wave and slice
  static constexpr int WN = BN / CSPLIT;           // columns per wave
  static constexpr int NB = WN / 32;               // 32-column MFMA blocks per wave
  static constexpr int ROWB = SK * 2;              // bytes of one row segment (128)
  static constexpr int WST = BN * ROWB, AST = BM * ROWB;
  // Waves 0-1 copy weight slices, waves 2-3 hidden-state slices.  Vector
  // memory operations of one wave complete in issue order, so a wave that
  // issued only weight copies can keep SW - 1 of them in flight without
  // waiting behind the (L2-resident) hidden-state loads.
  static constexpr int SA = 2;                     // hidden-state stages
  static constexpr int HL = 4;                     // hidden-state slices in flight in registers
  static constexpr int SW0 = (kDmaLdsBudget - SA * AST) / WST;
  static constexpr int SW = SW0 > 8 ? 8 : SW0;     // weight stages
  static constexpr int WIW = WST / 1024 / 2;       // copy instructions per weight wave per slice
  static constexpr int AIA = AST / 1024 / 2;       // per hidden-state wave per slice
  static constexpr int kLds = SW * WST + SA * AST; // bytes of LDS
  static_assert(SW >= 3 && WIW >= 1 && AIA >= 1 && MB >= 1 && NB >= 1, "tile shape");
  static_assert((SW - 2) * WIW < 64 && HL * AIA < 64, "vmcnt range");
};

// One BM x BN tile (tile index bx: row tile bx % tiles_m, column tile
// bx / tiles_m) with 256 threads and the workgroup's LDS buffer `lds` of
// DmaShape<BM, BN>::kLds bytes (1024-byte aligned).
template <int BM, int BN, bool TEXT>
__device__ __forceinline__ void dma_tile(const HeadView &hv, const StepView &sv, int bx,
                                         char *lds) {
  using S_ = DmaShape<BM, BN>;
  constexpr int SK = S_::SK, MB = S_::MB, KSPLIT = S_::KSPLIT, CSPLIT = S_::CSPLIT, KS = S_::KS;
  constexpr int WN = S_::WN, NB = S_::NB, ROWB = S_::ROWB, WST = S_::WST, AST = S_::AST;
  constexpr int SA = S_::SA, HL = S_::HL, SW = S_::SW, WIW = S_::WIW, AIA = S_::AIA;
  constexpr int LDSB = S_::kLds;
  char *const wring = lds;                 // weight stages
  char *const aring = lds + SW * WST;      // hidden-state stages
  // Epilogue, after the loop (the rings are free then): the partial sums C of
  // the two k halves at the start, and per pair of GEMM rows (2q, 2q + 1)
  // {w, 1/T, out, -2} for a CFG pair or {1/T_0, 1/T_1, out_0, out_1} for two solo
  // rows (out -1: no row) at the end.
  constexpr int CP = BN + 4;               // padded row pitch of C (floats)
  constexpr int RPOFF = LDSB - (BM / 2) * 16;
  static_assert(KSPLIT * BM * CP * 4 <= RPOFF, "C and the row parameters fit the rings");
  float4 *const rowp = reinterpret_cast<float4 *>(lds + RPOFF);

  const int32_t *rows = sv.plan + kPlanHeader + (TEXT ? sv.Mg : 0);
  const int M = TEXT ? sv.n_text : sv.Mg;
  const int N = TEXT ? hv.V_text : hv.N;
  const __bf16 *Wp = static_cast<const __bf16 *>(TEXT ? hv.W_text : hv.W);
  const __bf16 *X = static_cast<const __bf16 *>(sv.hidden);
  const int H = hv.H;
  const int NST = H / SK;

  const int tiles_m = (M + BM - 1) / BM;
  // Several row tiles (more than 128 audio rows): workgroups are dealt to the
  // 8 XCDs in turn, so the index is remapped to give each XCD a contiguous
  // run of tiles, in which the row tiles of a column tile are neighbours, run
  // at the same time and walk k in the same order: they share that column
  // tile's weights through the XCD's L2.
  if (tiles_m > 1) {
    const int ntiles = tiles_m * ((N + BN - 1) / BN);
    if (ntiles % 8 == 0) bx = (bx % 8) * (ntiles / 8) + bx / 8;
  }
  const int tile_m = bx % tiles_m;
  const int tile_n = bx / tiles_m;
  const int m0 = tile_m * BM, n0 = tile_n * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ch = wave % CSPLIT, kh = wave / CSPLIT;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const bool w_copier = wave_s < 2;        // wave-uniform role

  // Each tile walks the k slices starting at its own offset, so that at any
  // moment the workgroups read different offsets of their (8 KiB-strided)
  // weight rows and spread over the HBM channels instead of all hitting the
  // same ones.  The sum order per tile is fixed, so results stay deterministic.
  const int kskew = (int)(((unsigned)tile_n * 7u) % (unsigned)NST);
  const uint32_t wbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)wring;
  const int seg_r = lane >> 3, seg_c = lane & 7;

  // Per-lane global sources of this wave's copy instructions (chunk-swizzled):
  // a weight wave copies rows (wave * WIW + q) * 8 .. +7 of the tile, a
  // hidden-state wave rows ((wave - 2) * AIA + q) * 8 .. +7.
  constexpr int QN = WIW > AIA ? WIW : AIA;
  const __bf16 *src[QN];
  // copy slice st (st < NST) into its stage
  auto issue_w = [&](int st) __attribute__((always_inline)) {
    int ks = st + kskew;
    ks = ks >= NST ? ks - NST : ks;
    const uint32_t sb = wbase + (uint32_t)((st % SW) * WST);
    static_for<0, WIW>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      lds_copy16_stream(src[q] + ks * SK, sb + (uint32_t)((wave_s * WIW + q) * 1024));
    });
  };
  // Hidden-state slices go through registers (global_load_dwordx4, then
  // ds_write_b128 into the stage), beside the weights' direct copies: the
  // two paths into LDS run at once.  Lane i holds 16 B of row i / 8 of an
  // 8-row group, at LDS position i % 8 of that row's segment.
  // Loads past the last slice re-load it (clamped; never stored), so that
  // every iteration issues the same loads and the compiler's waits for them
  // stay exact.
  auto load_a = [&](int st, u32x4 (&b)[AIA]) __attribute__((always_inline)) {
    int ks = min(st, NST - 1) + kskew;
    ks = ks >= NST ? ks - NST : ks;
    static_for<0, AIA>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      b[q] = *reinterpret_cast<const u32x4 *>(src[q] + ks * SK);
    });
  };
  auto store_a = [&](int st, const u32x4 (&b)[AIA]) __attribute__((always_inline)) {
    if (st >= NST) return;
    char *sb = aring + (st % SA) * AST + ((wave_s - 2) * AIA) * 1024 + lane * 16;
    static_for<0, AIA>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      *reinterpret_cast<u32x4 *>(sb + q * 1024) = b[q];
    });
  };
  u32x4 hb[HL][AIA];

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
    for (int st = 0; st < SW - 1; ++st)
      if (st < NST) issue_w(st);
  }

  if (!plan_ok(sv)) {
    wait_vmem_and_lds<0>();  // no copy may still be landing in this workgroup's LDS
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }

  // The hidden-state waves gather their rows through the plan and start their
  // copies as soon as the row indices are in.  The per-row epilogue parameters
  // are loaded before the copies (in order, they complete before them, so the
  // loop's copy counts stay valid) and staged in LDS after the loop.
  const int q2 = tid - 128;
  PairLoads praw{0.0f, 0.0f, 0.0f, 0, false, false};
  if (!w_copier) {
    // all row loads first (the copy sources and, for the epilogue, the rows of
    // a GEMM row pair per thread), then the checks: their round trips overlap
    int prow[QN];
    static_for<0, QN>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      prow[q] = 0;
      if (q < AIA) prow[q] = rows[min(m0 + ((wave_s - 2) * AIA + q) * 8 + seg_r, M - 1)];
    });
    const int g0 = m0 + 2 * min(q2, BM / 2 - 1);
    int pr0 = 0, pr1 = 0;
    if constexpr (!TEXT) {
      pr0 = rows[min(g0, sv.Mg - 1)];
      pr1 = rows[min(g0 + 1, sv.Mg - 1)];
    }
    bool bad = false;
    static_for<0, QN>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      src[q] = nullptr;
      if (q < AIA) {
        const int r = ((wave_s - 2) * AIA + q) * 8 + seg_r;
        const bool ok = prow[q] >= 0 && prow[q] < sv.R;
        bad |= !ok;
        src[q] = X + (size_t)(ok ? prow[q] : 0) * H + ((seg_c ^ ((r >> 1) & 7)) * 8);
      }
    });
    if constexpr (!TEXT) praw = pair_params_load(sv, g0, pr0, pr1);
    if (bad) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    // slices 0 .. SA - 2 straight into their stages, then HL slices ahead
    u32x4 h0[SA - 1][AIA];
    static_for<0, SA - 1>([&](auto sc) __attribute__((always_inline)) {
      load_a(decltype(sc)::value, h0[decltype(sc)::value]);
    });
    static_for<0, HL>([&](auto jc) __attribute__((always_inline)) {
      load_a(SA - 1 + decltype(jc)::value, hb[decltype(jc)::value]);
    });
    static_for<0, SA - 1>([&](auto sc) __attribute__((always_inline)) {
      store_a(decltype(sc)::value, h0[decltype(sc)::value]);
    });
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
  // k16 step; this wave covers the k16 steps kh * KS .. kh * KS + KS - 1 of
  // the slice (chunks 2 KS kh .. 2 KS kh + 2 KS - 1).
  const int frow = lane & 31;
  int aoff[KS][MB], woff[KS][NB];
#pragma unroll
  for (int s2 = 0; s2 < KS; ++s2) {
    const int c = 2 * (kh * KS + s2) + (lane >> 5);
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

  // MFMAs of slice st, from its stages.  The fragments of the next k16 step
  // are read while the MFMAs of this one run, and extra(m) (this wave's copy
  // work for a later slice) is issued after MFMA m, so that the matrix pipe,
  // the LDS and the load path work at once instead of in turn.
  constexpr int NMF = KS * MB * NB;        // MFMAs per wave and slice
  auto compute = [&](int st, auto &&extra) __attribute__((always_inline)) {
    const char *wsb = wring + (st % SW) * WST;
    const char *asb = aring + (st % SA) * AST;
    bf16x8 fa[2][MB], fb[2][NB];
    static_for<0, MB>([&](auto ic) __attribute__((always_inline)) {
      fa[0][ic] = *reinterpret_cast<const bf16x8 *>(asb + aoff[0][ic]);
    });
    static_for<0, NB>([&](auto jc) __attribute__((always_inline)) {
      fb[0][jc] = *reinterpret_cast<const bf16x8 *>(wsb + woff[0][jc]);
    });
    static_for<0, KS>([&](auto sc) __attribute__((always_inline)) {
      constexpr int s2 = decltype(sc)::value, cur = s2 & 1, nxt = cur ^ 1;
      if constexpr (s2 + 1 < KS) {
        static_for<0, MB>([&](auto ic) __attribute__((always_inline)) {
          fa[nxt][ic] = *reinterpret_cast<const bf16x8 *>(asb + aoff[s2 + 1][ic]);
        });
        static_for<0, NB>([&](auto jc) __attribute__((always_inline)) {
          fb[nxt][jc] = *reinterpret_cast<const bf16x8 *>(wsb + woff[s2 + 1][jc]);
        });
      }
      static_for<0, MB * NB>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value, i = m / NB, j = m % NB;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j], 0, 0, 0);
        extra(std::integral_constant<int, s2 * MB * NB + m>{});
        __builtin_amdgcn_sched_barrier(0);
      });
    });
  };
  // The two roles run separate copies of the loop (one barrier per iteration
  // in both), so that the hidden-state registers exist on one path only.
  // At the top of iteration st: the weight waves' copies of slice st have
  // landed (those of later slices may still be in flight); every wave's LDS
  // reads of slice st - 1 and writes of slice st are done.  The barrier
  // extends both to the whole workgroup.
  if (w_copier) {
    for (int st = 0; st < NST; ++st) {
      wait_slices<WIW, SW - 2>(NST - 1 - st);
      block_barrier_no_vmem_wait();
      const int cs = st + SW - 1;        // the slice whose copies go out now
      const bool go = cs < NST;
      int ks = cs + kskew;
      ks = ks >= NST ? ks - NST : ks;
      const uint32_t sb = wbase + (uint32_t)((cs % SW) * WST);
      compute(st, [&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        // copies q with q * NMF / WIW == m go out after MFMA m
        static_for<0, WIW>([&](auto qc) __attribute__((always_inline)) {
          constexpr int q = decltype(qc)::value;
          if constexpr (q * NMF / WIW == m) {
            if (go) lds_copy16_stream(src[q] + ks * SK, sb + (uint32_t)((wave_s * WIW + q) * 1024));
          }
        });
      });
    }
  } else {
    // unrolled by HL, so that each register buffer has a fixed name: buffer j
    // holds the slices s with (s - SA + 1) % HL == j
    auto iteration = [&](int st, u32x4 (&hbj)[AIA]) __attribute__((always_inline)) {
      wait_vmem_and_lds<63>();
      block_barrier_no_vmem_wait();
      const int ss = st + SA - 1;        // stored now, into the stage read in iteration st - 1
      const bool sgo = ss < NST;
      char *sbase = aring + (ss % SA) * AST + ((wave_s - 2) * AIA) * 1024 + lane * 16;
      int ks = min(st + SA - 1 + HL, NST - 1) + kskew;
      ks = ks >= NST ? ks - NST : ks;
      compute(st, [&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        // op o < AIA: store chunk o; op AIA + q: reload register q (after its store)
        static_for<0, 2 * AIA>([&](auto oc) __attribute__((always_inline)) {
          constexpr int o = decltype(oc)::value;
          if constexpr (o * NMF / (2 * AIA) == m) {
            if constexpr (o < AIA) {
              if (sgo) *reinterpret_cast<u32x4 *>(sbase + o * 1024) = hbj[o];
            } else {
              constexpr int q = o - AIA;
              hbj[q] = *reinterpret_cast<const u32x4 *>(src[q] + ks * SK);
            }
          }
        });
      });
    };
    int st0 = 0;
    for (; st0 + HL <= NST; st0 += HL) {
      static_for<0, HL>([&](auto jc) __attribute__((always_inline)) {
        iteration(st0 + decltype(jc)::value, hb[decltype(jc)::value]);
      });
    }
    static_for<0, HL - 1>([&](auto jc) __attribute__((always_inline)) {
      constexpr int j = decltype(jc)::value;
      if (st0 + j < NST) iteration(st0 + j, hb[j]);
    });
  }
  // the copies are invisible to the compiler; the last iteration waited for
  // all of them, and this drain makes that explicit before LDS is reused
  wait_vmem_and_lds<0>();
  __syncthreads();
  if (!TEXT && !w_copier && q2 < BM / 2) rowp[q2] = pair_params_finish(sv, praw);

  // Epilogue, in two phases through LDS (the rings are free now).
  // Phase 1: every wave writes its partial sums (its k group) to C[kh][row][col].
  // Phase 2: each thread takes 16-byte column chunks (audio) or 32-column text
  // parts of whole rows, adds the k groups' sums (at most two terms: order-
  // free), and applies the fused epilogue with coalesced stores.  No global
  // load is left pending among the stores, so they never wait for each other.
  float *C = reinterpret_cast<float *>(lds);
  float *Cl = C + (kh * BM + (lane >> 5) * 4) * CP + ch * WN + frow;
  static_for<0, MB * NB * 16>([&](auto fc) __attribute__((always_inline)) {
    constexpr int f = decltype(fc)::value;
    constexpr int i = f / (NB * 16), j = (f / 16) % NB, r = f % 16;
    constexpr int off = (i * 32 + (r >> 2) * 8 + (r & 3)) * CP + j * 32;
    Cl[off] = acc[i][j][r];
  });

  epilogue_from_lds<BM, BN, CP, TEXT, KSPLIT>(hv, sv, C, rowp, m0, n0, M, N);
}

}  // namespace
}  // namespace mcd
