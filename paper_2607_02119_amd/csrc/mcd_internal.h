// Internal declarations shared by the host API and the gfx950 kernels of libmcd.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mcd.h"

namespace mcd {

// Plan layout (int32 words): header, then the GEMM row order of the audio rows
// (Main, Companion of pair 0, pair 1, ..., then the solo rows), then the text rows.
constexpr int32_t kPlanMagic = 0x4D434450;  // "MCDP"
constexpr int kPlanHeader = 8;
enum { kPlanMagicWord = 0, kPlanR = 1, kPlanPairs = 2, kPlanSolo = 3, kPlanText = 4 };

constexpr int kStatusBytes = 256;  // status word region at the start of the workspace

// The text GEMM writes one (max, lowest argmax) partial per row for every
// kTextPartCols columns of the text vocabulary.
constexpr int kTextPartCols = 32;

struct Delays {
  int32_t d[MCD_MAX_K];
};

// First column of every stream's block in the N columns; voff[K] = N.
struct StreamOffsets {
  int32_t o[MCD_MAX_K + 1];
};

// Head, by value in kernel arguments.  V is the largest stream's size.
struct HeadView {
  int32_t H, K, V, N, pad_id, V_text;
  int32_t dtype;
  const void *W;
  const float *bias;
  const void *W_text;
  Delays delays;
  StreamOffsets voff;
  int32_t T_text;       // text ids of the text head (the text phase's mask), V_text if none
};

// One step, by value in kernel arguments.
struct StepView {
  int32_t R, n_pairs, n_solo, n_text, Mg, Rs;
  const int32_t *plan;
  const void *hidden;
  const float *cfg_w;
  const float *temperature;
  const int32_t *top_k;
  const float *top_p;
  const uint64_t *rng_key;
  const int32_t *step;
  const int32_t *n_frames;
  const int32_t *grid_slot;
  uint64_t seed;
  int32_t *tokens_out;
  int32_t *frame_grid;
  uint8_t *modality_out;
  int32_t n_slots, F_max;
  float *scores;
  uint32_t *status;
  float *text_val;      // [n_text][text_parts]
  int32_t *text_idx;    // [n_text][text_parts]
  int32_t text_parts;
};

inline int32_t text_parts_for(int32_t V_text) {
  return (V_text + kTextPartCols - 1) / kTextPartCols;
}

// Kernel launchers (one .hip file each).
hipError_t launch_head_gemm(const HeadView &hv, const StepView &sv, hipStream_t stream);
// one part of it: the audio rows, or the text rows when text is set
hipError_t launch_head_gemm_part(const HeadView &hv, const StepView &sv, bool text,
                                 hipStream_t stream);
// bf16 projection kernels (audio rows, or the text rows when text is set)
hipError_t launch_stream_rows(const HeadView &hv, const StepView &sv,
                              hipStream_t st);       // audio rows in 128 x 256 tiles
hipError_t launch_stream_gemm(const HeadView &hv, const StepView &sv, bool text,
                              hipStream_t stream);   // at most 128 GEMM rows
hipError_t launch_mfma_gemm(const HeadView &hv, const StepView &sv, bool text,
                            hipStream_t stream);     // any number of rows
// A batch of audio rows in 256 x 256 tiles and 65..128 text rows: both
// projections in one launch; *launched is false (and nothing is launched) for
// other batches.
hipError_t launch_mixed_gemm(const HeadView &hv, const StepView &sv, hipStream_t st,
                             bool *launched);
// Next-step input (k_embed.hip): sizes and pointers validated by the caller.
struct EmbedView {
  int32_t R, H, K, V, pad_id, V_text;
  const void *E, *E_text;
  const uint8_t *row_kind;
  const int32_t *tokens;
  void *out;
  uint32_t *status;          // or null
};
hipError_t launch_next_input(const EmbedView &ev, bool bf16, hipStream_t stream);
// Records a host-side error for mcd_last_error and returns s (mcd_api.cpp).
mcd_status record_error(mcd_status s, const char *msg);
hipError_t launch_sample(const HeadView &hv, const StepView &sv, bool with_text,
                         hipStream_t stream);
hipError_t launch_deinterleave(const int32_t *streams, int32_t n_req, int32_t T, int32_t K,
                               const Delays &d, int32_t F, int32_t *grid, hipStream_t stream);
hipError_t launch_interleave(const int32_t *grid, int32_t n_req, int32_t F, int32_t K,
                             const Delays &d, int32_t T, int32_t pad_id, int32_t *streams,
                             hipStream_t stream);

}  // namespace mcd
