// K1, MFMA-regime path (more than 128 GEMM rows): the same projection and
// fused epilogues as the streaming path (Sec. 2.1, Eq. 1), for batches whose
// arithmetic intensity puts them on the matrix cores: audio rows in 256 x 256
// tiles when those fill the chip (other audio batches take the streaming
// path's 128 x 256 tiles), text rows beyond 128 in 256 x 128 tiles.
#include "mfma2_tile.h"

namespace mcd {
namespace {

// 256 x 128 tiles for more than 128 text rows (bf16, H a multiple of 32).
// A workgroup owns a 256 x 128 output tile with eight waves, two per SIMD, so
// that one wave's MFMAs cover the other's LDS reads and copies.  The waves
// split it by row half (wm = wave & 1), column half (wn = (wave >> 1) & 1) and
// k half (kh = wave >> 2): each wave accumulates a 128 x 64 block (4 x 2
// blocks of v_mfma_f32_32x32x16_bf16, 128 accumulator registers) over its
// 16 k of every 32-k slice.  Slices are copied global->LDS like the streaming
// path: waves 0-3 copy weight slices into a deep ring (the weights come from
// HBM, once per XCD), waves 4-7 copy hidden-state slices into a shorter one
// (they are re-read from L2).  A slice row is 64 bytes, 4 chunks of 16 B;
// chunk c of row r is stored at position c ^ ((r >> 2) & 3), so the 16 rows
// of a 16-lane fragment read group hit all 64 banks once.  (WAVES = 4 is the
// one-wave-per-SIMD form: 128 x 128 blocks per wave.)
//
// Tile order is XCD-aware: workgroups are dealt to the 8 XCDs in turn, so the
// grid index is remapped to give each XCD a contiguous run of tiles, in which
// the row tiles of a column tile are neighbours and run at the same time:
// they share that column's weights through the XCD's L2.
constexpr int kMfmaBM = 256, kMfmaBN = 128, kMfmaSK = 32;
constexpr int kMfmaSA = 5, kMfmaSB = 8;
constexpr int kMfmaWaves = 8;

template <bool TEXT, int WAVES>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(WAVES / 4, WAVES / 4)))
void head_gemm_mfma(HeadView hv, StepView sv) {
  constexpr int BM = kMfmaBM, BN = kMfmaBN, SK = kMfmaSK;
  constexpr int SA = kMfmaSA, SB = kMfmaSB;
  constexpr int NTH = 64 * WAVES;                    // threads
  constexpr int CW = WAVES / 4;                      // column groups of waves (1 or 2)
  constexpr int HW = WAVES / 2;                      // waves per copy role
  constexpr int ROWB = SK * 2;                       // 64 bytes per row and slice
  constexpr int AST = BM * ROWB, BST = BN * ROWB;    // 16 KiB, 8 KiB per stage
  constexpr int AIA = AST / 1024 / HW, BIB = BST / 1024 / HW;  // copies per wave per slice
  constexpr int MB = 4, NB = 4 / CW;                 // 32x32 blocks per wave
  constexpr int WNC = BN / CW;                       // columns per wave
  static_assert(WAVES == 4 || WAVES == 8, "one or two waves per SIMD");
  static_assert((SA - 1) * AIA < 64 && (SB - 1) * BIB < 64, "vmcnt range");
  // both copy roles keep the same number of copies in flight in the loop, so
  // that its one wait needs no branch (a branch makes the compiler's own
  // LDS-read waits conservative)
  constexpr int kLoopVm = (SA - 2) * AIA;
  static_assert((SB - 2) * BIB == kLoopVm, "equal in-flight copy counts");
  static_assert(AIA * 2 == MB * NB && BIB * 4 == MB * NB && MB + NB <= MB * NB,
                "copy and fragment slots of the slice schedule");
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
  const int wm = wave & 1, wn = (wave >> 1) & (CW - 1), kh = wave / (2 * CW);
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const bool b_copier = wave_s < HW;

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
      lds_copy16(src[q] + ks * SK, sb + (uint32_t)(((wave_s - HW) * AIA + q) * 1024));
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
        const int r = ((wave_s - HW) * AIA + q) * 16 + seg_r;
        int pr = rows[min(m0 + r, M - 1)];
        if (pr < 0 || pr >= sv.R) {
          atomicOr(sv.status, (uint32_t)MCD_DEV_BAD_PLAN);
          pr = 0;
        }
        src[q] = X + (size_t)pr * H + ((seg_p ^ ((r >> 2) & 3)) * 8);
      }
    });
    const int q2 = tid - NTH / 2;
    if (!TEXT && q2 < BM / 2) rowp[q2] = pair_params(sv, rows, m0 + 2 * q2);
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
    const int r = wn * WNC + j * 32 + frow;
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
        constexpr int q = m / 2;           // A copies after the odd MFMAs
        if (!b_copier) lds_copy16(src[q] + ks * SK, csb + (uint32_t)(((wave_s - HW) * AIA + q) * 1024));
      }
      if constexpr (m % 4 == 3) {
        constexpr int q = m / 4;           // B copies after every fourth
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
  float *Cl = C + (wm * 128 + (lane >> 5) * 4) * CP + wn * WNC + frow;
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
  epilogue_from_lds<BM, BN, CP, TEXT, 1, NTH>(hv, sv, C, rowp, m0, n0, M, N);
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void head_gemm_mfma2(
    HeadView hv, StepView sv) {
  __shared__ __attribute__((aligned(1024))) char lds[M2Shape::kLds];
  mfma2_tile(hv, sv, blockIdx.x, gridDim.x, lds);
}

hipError_t launch_mfma2(const HeadView &hv, const StepView &sv, hipStream_t st) {
  hipLaunchKernelGGL(head_gemm_mfma2, dim3((unsigned)tiles_256(sv.Mg, hv.N)), dim3(256), 0, st,
                     hv, sv);
  return hipGetLastError();
}

template <bool TEXT>
hipError_t launch_mfma(const HeadView &hv, const StepView &sv, int M, int N, hipStream_t st) {
  constexpr int WAVES = kMfmaWaves;
  const int tm = (M + kMfmaBM - 1) / kMfmaBM, tn = (N + kMfmaBN - 1) / kMfmaBN;
  hipLaunchKernelGGL((head_gemm_mfma<TEXT, WAVES>), dim3(tm * tn), dim3(64 * WAVES), 0, st, hv,
                     sv);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_mfma_gemm(const HeadView &hv, const StepView &sv, bool text, hipStream_t st) {
  if (text) return launch_mfma<true>(hv, sv, sv.n_text, hv.V_text, st);
  // 256 x 256 tiles when they fill the chip, else the streaming path's
  // 128 x 256 tiles
  if (tiles_256(sv.Mg, hv.N) >= 256) return launch_mfma2(hv, sv, st);
  return launch_stream_rows(hv, sv, st);
}

}  // namespace mcd
