// Tile body of the K1 MFMA-regime path for audio rows with 256 x 256 tiles:
// the codebook-head projection with the CFG merge (Eq. 1) and temperature
// fused into the epilogue (Sec. 2.1, Sec. 2.4).
#pragma once

#include "gemm_common.h"

namespace mcd {
namespace {

constexpr int kM2Tile = 256, kM2SK = 32, kM2Stages = 4;

inline int64_t tiles_256(int32_t M, int32_t N) {
  return (int64_t)((M + kM2Tile - 1) / kM2Tile) * ((N + kM2Tile - 1) / kM2Tile);
}

// Audio rows, 256 x 256 tiles: the waves split the tile 2 x 2 (wm = wave & 1
// row half, wn = wave >> 1 column half), each accumulating a 128 x 128 block
// (4 x 4 blocks of v_mfma_f32_32x32x16_bf16) over both k16 halves of every
// 32-k slice.  Per slice a workgroup copies 16 KiB of hidden states and 16 KiB
// of weights (waves 0-1 copy weights, waves 2-3 hidden states, 8 copies each)
// for 4 x 32 MFMAs: a third fewer bytes per MFMA than a 256 x 128 tile, and
// half the fragment reads.  All four ring stages are in flight.  It needs at
// least 256 tiles to fill the chip; smaller batches take the streaming path's
// 128 x 256 row tiles.

// LDS of one tile: the rings (or, after the loop, one 128-row half of the
// epilogue tile) and the row-pair parameters after them.
struct M2Shape {
  static constexpr int BM = kM2Tile, BN = kM2Tile, SK = kM2SK, ST = kM2Stages;
  static constexpr int ROWB = SK * 2;                      // 64 bytes per row and slice
  static constexpr int AST = BM * ROWB, BST = BN * ROWB;   // 16 KiB each
  static constexpr int CP = BN + 4;                        // epilogue row pitch (floats)
  static constexpr int RING = ST * (AST + BST), EPI = (BM / 2) * CP * 4;
  static constexpr int kRowp = RING > EPI ? RING : EPI;    // offset of the row parameters
  static constexpr int kLds = kRowp + (BM / 2) * 16;
};

// One 256 x 256 tile: tile index bx of ntiles (remapped XCD-aware when ntiles
// is a multiple of 8), 256 threads, LDS buffer `lds` of M2Shape::kLds bytes
// (1024-byte aligned).
__device__ __forceinline__ void mfma2_tile(const HeadView &hv, const StepView &sv, int bx,
                                           int ntiles, char *lds) {
  constexpr int BM = M2Shape::BM, BN = M2Shape::BN, SK = M2Shape::SK, ST = M2Shape::ST;
  constexpr int ROWB = M2Shape::ROWB, AST = M2Shape::AST, BST = M2Shape::BST;
  constexpr int CPW = AST / 1024 / 2;                 // copies per copying wave per slice
  constexpr int MB = 4, NB = 4;
  constexpr int kLoopVm = (ST - 2) * CPW;
  static_assert(BST == AST && CPW == 8 && (ST - 1) * CPW < 64, "copy schedule");
  constexpr int CP = M2Shape::CP;

  char *const aring = lds;
  char *const bring = lds + ST * AST;
  float4 *const rowp = reinterpret_cast<float4 *>(lds + M2Shape::kRowp);

  const int32_t *rows = sv.plan + kPlanHeader;
  const int M = sv.Mg, N = hv.N, H = hv.H;
  const __bf16 *Wp = static_cast<const __bf16 *>(hv.W);
  const __bf16 *X = static_cast<const __bf16 *>(sv.hidden);
  const int NSL = H / SK;                             // slices (even: H % 64 == 0)

  const int tiles_m = (M + BM - 1) / BM;
  if (ntiles % 8 == 0) bx = (bx % 8) * (ntiles / 8) + bx / 8;
  const int tile_m = bx % tiles_m, tile_n = bx / tiles_m;
  const int m0 = tile_m * BM, n0 = tile_n * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const bool b_copier = wave_s < 2;

  const uint32_t abase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)aring;
  const uint32_t bbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)bring;
  // one copy: 16 rows x 4 chunks of 16 B; lane i -> row i / 4, position i % 4,
  // holding chunk position ^ ((row >> 2) & 3) of the slice
  const int seg_r = lane >> 2, seg_p = lane & 3;
  const __bf16 *src[CPW];
  uint32_t dst0;   // LDS offset of this wave's first copy within a stage
  auto copy = [&](int q, int st) __attribute__((always_inline)) {
    const int ks = min(st, NSL - 1);
    const uint32_t sb = b_copier ? bbase + (uint32_t)((st % ST) * BST)
                                 : abase + (uint32_t)((st % ST) * AST);
    lds_copy16(src[q] + ks * SK, sb + dst0 + (uint32_t)(q * 1024));
  };

  wait_vmem_and_lds<0>();
  if (b_copier) {
    dst0 = (uint32_t)(wave_s * CPW * 1024);
#pragma unroll
    for (int q = 0; q < CPW; ++q) {
      const int r = (wave_s * CPW + q) * 16 + seg_r;
      const int n = min(n0 + r, N - 1);
      src[q] = Wp + (size_t)n * H + ((seg_p ^ ((r >> 2) & 3)) * 8);
    }
#pragma unroll
    for (int st = 0; st < ST; ++st)
#pragma unroll
      for (int q = 0; q < CPW; ++q) copy(q, st);
  }

  if (!plan_ok(sv)) {
    wait_vmem_and_lds<0>();  // no copy may still be landing in this workgroup's LDS
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
    return;
  }

  if (!b_copier) {
    dst0 = (uint32_t)((wave_s - 2) * CPW * 1024);
#pragma unroll
    for (int q = 0; q < CPW; ++q) {
      const int r = ((wave_s - 2) * CPW + q) * 16 + seg_r;
      int pr = rows[min(m0 + r, M - 1)];
      if (pr < 0 || pr >= sv.R) {
        atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
        pr = 0;
      }
      src[q] = X + (size_t)pr * H + ((seg_p ^ ((r >> 2) & 3)) * 8);
    }
    rowp[tid - 128] = pair_params(sv, rows, m0 + 2 * (tid - 128));
    wait_vmem_and_lds<0>();
#pragma unroll
    for (int st = 0; st < ST; ++st)
#pragma unroll
      for (int q = 0; q < CPW; ++q) copy(q, st);
  }

  floatx16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // fragment offsets within a stage: lane l holds row (column) l % 32 and
  // chunk 2 s + l / 32 of k16 step s; the swizzle depends on l % 32 only
  const int frow = lane & 31;
  const int sw = (frow >> 2) & 3;
  const int arow = (wm * 128 + frow) * ROWB, brow = (wn * 128 + frow) * ROWB;
  const int c0 = ((lane >> 5) ^ sw) * 16, c1 = ((2 + (lane >> 5)) ^ sw) * 16;

  // Software pipeline: the 16 fragments of slice st + 1 are read while the 32
  // MFMAs of slice st run; the wave's 8 copies of slice st + ST go out between
  // them.  At the top of iteration st every wave waits for its copies of slice
  // st + 1 and its fragment reads of slice st; the barrier extends both to the
  // workgroup, so slice st's stage is free for slice st + ST.  Slices past the
  // end re-load the last one (clamped), so every iteration issues the same count.
  bf16x8 fa0[2][MB], fb0[2][NB], fa1[2][MB], fb1[2][NB];
  auto frag = [&](int st, int s2, bool is_a, int idx) __attribute__((always_inline)) {
    const char *base = is_a ? aring + (st % ST) * AST + arow : bring + (st % ST) * BST + brow;
    return *reinterpret_cast<const bf16x8 *>(base + idx * 32 * ROWB + (s2 ? c1 : c0));
  };
  auto step = [&](int st, bf16x8 (&fa)[2][MB], bf16x8 (&fb)[2][NB], bf16x8 (&na)[2][MB],
                  bf16x8 (&nb)[2][NB]) __attribute__((always_inline)) {
    wait_vmem_and_lds<kLoopVm>();
    block_barrier_no_vmem_wait();
    static_for<0, 32>([&](auto mc) __attribute__((always_inline)) {
      constexpr int m = decltype(mc)::value;
      constexpr int s2 = m / 16, i = (m / 4) % 4, j = m % 4;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s2][i], fb[s2][j], acc[i][j], 0, 0, 0);
      if constexpr (m < 16) {
        constexpr int f2 = m / 8, fi = (m / 2) % 4;
        if constexpr (m % 2 == 0) na[f2][fi] = frag(st + 1, f2, true, fi);
        else nb[f2][fi] = frag(st + 1, f2, false, fi);
      }
      if constexpr (m % 4 == 3) copy(m / 4, st + ST);
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  // slice 0 landed (all but ST - 1 newer slices), then its fragments
  wait_vmem_and_lds<(ST - 1) * CPW>();
  block_barrier_no_vmem_wait();
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fa0[s2][i] = frag(0, s2, true, i);
      fb0[s2][i] = frag(0, s2, false, i);
    }
  for (int st = 0; st < NSL; st += 2) {
    step(st, fa0, fb0, fa1, fb1);
    step(st + 1, fa1, fb1, fa0, fb0);
  }
  wait_vmem_and_lds<0>();
  __syncthreads();

  // Epilogue through LDS, one row half at a time: the waves of that half store
  // their sums in C[row][col], then every thread applies the fused epilogue to
  // 16-byte column chunks of it.
  float *C = reinterpret_cast<float *>(lds);
  float *Cl = C + ((lane >> 5) * 4) * CP + wn * 128 + frow;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (h == 1) __syncthreads();   // every read of the first half is done
    if (wm == h) {
      static_for<0, MB * NB * 16>([&](auto fc) __attribute__((always_inline)) {
        constexpr int f = decltype(fc)::value;
        constexpr int i = f / (NB * 16), j = (f / 16) % NB, r = f % 16;
        constexpr int off = (i * 32 + (r >> 2) * 8 + (r & 3)) * CP + j * 32;
        Cl[off] = acc[i][j][r];
      });
    }
    epilogue_from_lds<BM / 2, BN, CP, false, 1>(hv, sv, C, rowp + h * (BM / 4), m0 + h * (BM / 2),
                                               n0, M, N);
  }
}

}  // namespace
}  // namespace mcd
