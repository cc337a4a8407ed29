/*
 * mcd.h -- C ABI of libmcd, the MI355X (gfx950) multi-codebook audio decode head.
 *
 * One decode step of the output stage of a delay-pattern speech LM served with
 * paired classifier-free guidance (arXiv 2607.02119):
 *   - K codebook head projections of every row's hidden state (Sec. 2.1: each
 *     of the S parallel heads maps h_t to its logits; head k is the k-th audio
 *     slice of the shared head, its stream-embedding term folds into a bias);
 *   - the in-batch CFG merge of each conditional (Main) row with its
 *     unconditional (Companion) partner, w * l_cond + (1 - w) * l_uncond, per
 *     codebook (Eq. 1), only for audio rows (Sec. 2.4);
 *   - temperature, top-k and top-p selection and a Gumbel-max draw from a
 *     counter-based generator in two levels (Philox, Salmon et al., SC'11):
 *     once per (row, codebook, step) vector, Philox4x64-10 with key (seed, 0)
 *     and counter (0, k, t, rng_key) gives the key material D; id v then takes
 *     word v mod 4 of Philox4x32-10 with key (lo D0, hi D0) and counter
 *     (v / 4, lo D1, hi D1, lo D2).  All K streams of a row are drawn in the
 *     same step (synchronous multi-stream sampling, Sec. 2.3);
 *   - the delay pattern: codebook k at step t carries frame t - d_k (Sec. 2.1);
 *     positions with no frame (before the stream starts, or in the drain that
 *     flushes the last S-1 steps, Sec. 2.3) carry the pad id;
 *   - the sampled Main token copied to the Companion row, whose own outputs
 *     stay hidden (Sec. 2.4), and each frame scattered into a per-request
 *     frame grid (the de-interleaved S x T codebook matrix, Sec. 2.1 / 2.3).
 *
 * Conventions
 *   - Pointers are DEVICE pointers unless marked [host].  Every buffer is owned
 *     by the caller; the library never allocates device memory, never
 *     synchronises (except mcd_read_device_status) and launches only on the
 *     stream it is given.
 *   - Row-major layouts; sizes in elements unless named *_bytes.
 *   - Errors: argument and shape errors return MCD_E_INVALID or
 *     MCD_E_UNSUPPORTED before anything is launched; a failed launch returns
 *     MCD_E_HIP.  mcd_last_error() gives a thread-local description of the last
 *     non-OK return.  No call aborts or throws.  Conditions only the device can
 *     see (a parameter value out of range, a grid cell outside the grid, a
 *     corrupt plan) set bits of a sticky status word in the workspace and make
 *     the affected tokens the pad id (the grid cell is then not written); read
 *     it with mcd_read_device_status.
 *   - Calls that share a workspace must not overlap in time.
 */
#ifndef MCD_H
#define MCD_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MCD_OK = 0,
  MCD_E_INVALID = 1,      /* bad argument, shape or batch structure */
  MCD_E_UNSUPPORTED = 2,  /* valid but outside what the kernels implement */
  MCD_E_WORKSPACE = 3,    /* workspace missing or too small */
  MCD_E_HIP = 4           /* the HIP runtime reported an error */
} mcd_status;

typedef enum { MCD_F32 = 0, MCD_BF16 = 1 } mcd_dtype;

/* Row kinds of a continuous batch (Sec. 2.4: a Main request with CFG scale
 * w > 1 gets a Companion; both are scheduled together). */
enum { MCD_ROW_COND = 0, MCD_ROW_UNCOND = 1, MCD_ROW_SOLO = 2, MCD_ROW_TEXT = 3 };

/* Bits of the device status word. */
enum {
  MCD_DEV_BAD_PARAM = 1u,   /* temperature < 0 or NaN, top_p <= 0 or NaN, non-finite w */
  MCD_DEV_GRID_RANGE = 2u,  /* grid_slot >= n_slots or frame >= F_max: cell not written */
  MCD_DEV_BAD_PLAN = 4u,    /* device plan does not match the counts of the call */
  MCD_DEV_BAD_TOKEN = 8u    /* mcd_next_input: a token outside its table */
};

#define MCD_MAX_K 32         /* codebooks per head */
#define MCD_MAX_V 4096       /* audio sub-vocabulary size per codebook */

typedef struct mcd_head mcd_head;   /* opaque, immutable after creation, thread-safe */

/* Head description.  The weights are borrowed: they must stay valid and
 * unchanged while the handle is used.
 *
 * Streams of unequal size (heterogeneous codebooks, e.g. one SSL stream and
 * eight codec streams): V_stream[k] ids for stream k, V the largest of them.
 * Stream k's block of the N = sum_k V_stream[k] columns starts at
 * off_k = sum_{j<k} V_stream[j]: rows off_k + v of W and entries of bias, and
 * the same columns of every scores row.  With V_stream NULL every stream has
 * V ids, off_k = k*V and N = K*V. */
typedef struct {
  int32_t H;                 /* hidden size; multiple of 64 for MCD_BF16, of 4 for MCD_F32 */
  int32_t K;                 /* codebooks (streams), 1..MCD_MAX_K */
  int32_t V;                 /* audio sub-vocabulary per codebook (the largest), 1..MCD_MAX_V */
  int32_t pad_id;            /* token emitted where the delay pattern has no frame */
  const int32_t *delays;     /* [host][K] d_k >= 0; copied at creation */
  mcd_dtype dtype;           /* element type of hidden, W and W_text */
  const void *W;             /* [N][H]: row off_k + v is head k's weight for id v */
  const float *bias;         /* [N] or NULL: stream-embedding term W_k e_k */
  int32_t V_text;            /* text vocabulary of the text head, 0 if none */
  const void *W_text;        /* [V_text][H] or NULL */
  const int32_t *V_stream;   /* [host][K] ids of each stream (1..MCD_MAX_V), or NULL;
                                copied at creation */
  int32_t T_text;            /* text-phase vocabulary mask (Sec. 2.3): ids [0, T_text) of the
                                text head are text tokens, the rest mark other modalities.
                                0 or V_text: no mask; else a multiple of 32 below V_text */
} mcd_head_desc;

/* Creates the handle.  A bf16 head with a text head also creates, on the
 * current device, the second stream and the two events its mixed batches use
 * (MCD_E_HIP if that fails); nothing is created later, in a step. */
mcd_status mcd_head_create(const mcd_head_desc *desc, mcd_head **out);
void mcd_head_destroy(mcd_head *head);

/* ---- batch plan -----------------------------------------------------------
 * Built on the host once per batch composition (not per step) from the pair
 * map and row kinds, then copied to device memory by the caller.
 *   pair_map[r]: partner row of a COND or UNCOND row, -1 for SOLO and TEXT rows;
 *   partners must point at each other and be one COND and one UNCOND row.
 * The plan fixes the "sampled order" of audio rows: the Main rows of the pairs
 * in ascending row order, then the SOLO rows in ascending row order.  Scores
 * are laid out in that order (see mcd_step_args.scores). */
typedef struct {
  int32_t n_pairs, n_solo, n_text;
} mcd_batch_counts;

size_t mcd_plan_words(int32_t R);   /* int32 words of a plan for R rows */

/* [host] Validate the batch and write the plan.  No HIP call.  Fails with
 * MCD_E_INVALID (and writes nothing) for an inconsistent pair map, an unknown
 * row kind, or TEXT rows on a head without a text head. */
mcd_status mcd_batch_plan(const mcd_head *head, int32_t R, const int32_t *pair_map,
                          const uint8_t *row_kind, int32_t *plan, size_t plan_words,
                          mcd_batch_counts *counts);

/* [host] Physical row of sampled index s (0 <= s < n_pairs + n_solo) and its
 * companion row (-1 for a SOLO row), read from a host copy of the plan. */
mcd_status mcd_plan_sampled_row(const int32_t *plan, int32_t s, int32_t *row, int32_t *companion);

/* Workspace bytes for a batch of up to R rows; the workspace must be 256-byte
 * aligned and zero-filled once before first use (the status word lives in it). */
size_t mcd_workspace_bytes(const mcd_head *head, int32_t R);

/* ---- one decode step -----------------------------------------------------*/
typedef struct {
  int32_t R;                 /* rows in the batch */
  mcd_batch_counts counts;   /* as returned by mcd_batch_plan */
  const int32_t *plan;       /* device copy of the plan words */
  const void *hidden;        /* [R][H] of the head's dtype, 16-byte aligned */
  /* Per-row arrays, [R] each: every one is required when R > 0 (MCD_E_INVALID
     otherwise), whatever the row kinds, since the kernels read them at every
     row; only rng_key may be NULL. */
  const float *cfg_w;        /* [R] CFG scale, used on COND rows (any finite w) */
  const float *temperature;  /* [R] >= 0; 0 selects greedy decoding */
  const int32_t *top_k;      /* [R] <= 0 or >= V: no top-k */
  const float *top_p;        /* [R] in (0, 1); >= 1: no top-p */
  const uint64_t *rng_key;   /* [R] stable request id (Main row's for a pair), or NULL: row index */
  const int32_t *step;       /* [R] decode step t of the row */
  const int32_t *n_frames;   /* [R] frames of the request, -1 if open-ended */
  const int32_t *grid_slot;  /* [R] frame-grid slot of a Main or SOLO row, -1 for none */
  uint64_t seed;             /* Philox key word 0 */
  int32_t *tokens_out;       /* [R][K]: COND/SOLO sampled, UNCOND = its Main row's,
                                TEXT: [r][0] greedy text id, the rest pad_id */
  int32_t *frame_grid;       /* [n_slots][K][F_max] or NULL; cell [slot][k][t - d_k] written */
  uint8_t *modality_out;     /* [R] or NULL: for TEXT rows, 1 when the argmax over all text-head
                                ids lies outside [0, T_text) (the model asks to leave the
                                text phase), else 0; other rows untouched */
  int32_t n_slots, F_max;
  float *scores;             /* [n_pairs + n_solo][N] fp32 in sampled order: the merged,
                                temperature-divided logits (greedy rows: merged only).
                                Output of mcd_head_step, input of mcd_sample_step. */
  void *workspace;
  size_t workspace_bytes;
} mcd_step_args;

/* The whole hot path of one step: projection + merge + temperature (scores),
 * text-head greedy argmax, selection, draw, pads, companion copy, grid scatter.
 * Equal to mcd_head_logits followed by mcd_sample_step: kernel launches on
 * `stream` (a batch with both audio and text rows also runs the text
 * projection on a second stream of the head, forked from and joined back to
 * `stream`); no device allocation, no synchronisation. */
mcd_status mcd_head_step(const mcd_head *head, const mcd_step_args *args, hipStream_t stream);

/* ---- allocation-free step ---------------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc) and so
 * cannot size mcd_head_step's workspace, whose text-head partials grow with
 * the batch: the same step through the same kernels, with those partials in a
 * device array the library holds per GPU (MCD_NOALLOC_SCRATCH_BYTES, from the
 * first call on a device until the process ends).  Arguments as for
 * mcd_head_step, except args->workspace: the status word region only
 * (workspace_bytes >= 256, 256-byte aligned, zero-filled once; read it with
 * mcd_read_device_status).  MCD_E_UNSUPPORTED, before anything is launched,
 * when the text partials of the batch (n_text x ceil(V_text / 32) fp32 values
 * and int32 ids, each block rounded up to 256 bytes) exceed the array: 220
 * text rows at V_text = 151936.  No allocation, no synchronisation.  Every
 * call on one GPU shares that GPU's array: calls that overlap in time on one
 * GPU race.  A step's partials are written by its projection before its
 * sampler reads them, so nothing carries over between calls. */
#define MCD_NOALLOC_SCRATCH_BYTES (8u << 20)
mcd_status mcd_head_step_noalloc(const mcd_head *head, const mcd_step_args *args,
                                 hipStream_t stream);

/* First half of a step: the K head projections of every audio row with the
 * CFG merge (Eq. 1) and temperature applied in the GEMM epilogue, written to
 * args->scores, and the text-head projection of the TEXT rows reduced to
 * per-32-column (max, lowest argmax) partials kept in the workspace.  Tokens
 * and the grid are not touched. */
mcd_status mcd_head_logits(const mcd_head *head, const mcd_step_args *args, hipStream_t stream);

/* Second half of a step, from the scores in args->scores (same layout as
 * above; they may come from mcd_head_logits or from the caller): selection,
 * draw, pads, companion copy and grid scatter for the audio rows.  TEXT rows
 * take their greedy token from the partials the last mcd_head_logits call left
 * in the same workspace; a batch with TEXT rows must therefore follow such a
 * call (args->hidden is not read). */
mcd_status mcd_sample_step(const mcd_head *head, const mcd_step_args *args, hipStream_t stream);

/* ---- delay pattern (Sec. 2.1) --------------------------------------------
 * De-interleave at request completion: grid[r][k][f] = streams[r][f + d_k][k]
 * for f < T - max_k d_k.  streams: [n_req][T][K], grid: [n_req][K][T - max d]. */
mcd_status mcd_deinterleave(const int32_t *streams, int32_t n_req, int32_t T, int32_t K,
                            const int32_t *delays /*[host][K]*/, int32_t *grid,
                            hipStream_t stream);
/* Inverse: streams[r][t][k] = grid[r][k][t - d_k] where 0 <= t - d_k < F, else
 * pad_id.  grid: [n_req][K][F], streams: [n_req][F + max d][K]. */
mcd_status mcd_interleave(const int32_t *grid, int32_t n_req, int32_t F, int32_t K,
                          const int32_t *delays /*[host][K]*/, int32_t pad_id,
                          int32_t *streams, hipStream_t stream);

/* ---- mixed-modality phases (Sec. 2.3) -------------------------------------
 * Each request moves through a text phase (TEXT rows: greedy over the text
 * ids, the mask of mcd_head_desc.T_text), a transition that injects
 * deterministic bridging tokens, an audio phase (audio rows: all K streams),
 * and a drain of S - 1 steps that flushes the delayed streams, then back to
 * text.  The switch out of text is read from the unmasked distribution
 * (mcd_step_args.modality_out).  The caller re-plans its batch when a
 * request's row kind changes (TEXT rows in the text phase, audio rows in the
 * audio and drain phases; the drain ends the request's frames through
 * n_frames). */
enum { MCD_PHASE_TEXT = 0, MCD_PHASE_BRIDGE = 1, MCD_PHASE_AUDIO = 2, MCD_PHASE_DRAIN = 3 };

typedef struct {
  int32_t n_bridge;          /* bridging tokens between text and audio, >= 0 */
  const int32_t *bridge;     /* [host][n_bridge] their ids */
  int32_t audio_end;         /* stream-0 token that ends the audio phase */
  int32_t drain_steps;       /* steps of the drain: the largest delay (S - 1), >= 0 */
} mcd_phase_desc;

/* [host] One decode step of n requests' phases, in place.  For request i:
 * phase[i], count[i] (bridging tokens emitted / audio steps / drain steps);
 * token0[i]: its stream-0 token of this step (the masked text token of a
 * text-phase row); modality[i]: its modality flag (text phase only).  emit[i]
 * receives the token the request emits this step outside the head's audio
 * output (text token or bridging token), or -1.
 *   TEXT:   modality 0 -> stay, emit token0; modality 1 -> emit bridge[0] and
 *           go to BRIDGE (AUDIO if that was the only one; with none, emit
 *           token0 and go to AUDIO).
 *   BRIDGE: emit bridge[count]; after the last, AUDIO.
 *   AUDIO:  token0 == audio_end -> DRAIN (TEXT if drain_steps is 0).
 *   DRAIN:  after drain_steps steps, TEXT.
 * MCD_E_INVALID for bad sizes, an unknown phase or a count out of range (the
 * arrays are then unchanged from that request on). */
mcd_status mcd_phase_advance(const mcd_phase_desc *desc, int32_t n, uint8_t *phase,
                             int32_t *count, const int32_t *token0, const uint8_t *modality,
                             int32_t *emit);

/* ---- next-step input (Sec. 2.1, delay pattern) ----------------------------
 * The backbone's input for the next step aggregates the embeddings of the K
 * tokens each row emitted at this step, one per stream (each for its own
 * delayed frame).  Read as their sum:
 *   out[r][h] = sum_k E[k][row_k][h],   row_k = tokens[r][k], or V for pad_id;
 * TEXT rows (row_kind MCD_ROW_TEXT) take E_text[tokens[r][0]][h].  The sum is
 * formed in fp64 and rounded once, to nearest even, to the table type: the
 * exact sum rounded once whenever the values' exponents span at most 40 bits
 * (bf16) or 24 bits (fp32).  After mcd_head_step a Companion row holds its
 * Main row's tokens, so both get the same input. */
typedef struct {
  int32_t R;                 /* rows, >= 0 */
  int32_t H;                 /* embedding width, >= 1 */
  int32_t K;                 /* streams, 1..MCD_MAX_K */
  int32_t V;                 /* audio sub-vocabulary per stream, >= 1 */
  int32_t pad_id;            /* outside [0, V): selects row V of every stream's table */
  mcd_dtype dtype;           /* element type of E, E_text and out */
  const void *E;             /* [K][V + 1][H]; row V of stream k is its pad embedding */
  int32_t V_text;            /* rows of E_text, 0 if none */
  const void *E_text;        /* [V_text][H] or NULL */
  const uint8_t *row_kind;   /* [R] MCD_ROW_* of every row */
  const int32_t *tokens;     /* [R][K], e.g. the tokens_out of a step */
  void *out;                 /* [R][H] of dtype; must not overlap the inputs */
  void *workspace;           /* a step workspace (its status word), or NULL */
} mcd_next_input_args;

/* Launches on `stream`; no allocation, no synchronisation.  MCD_E_INVALID for
 * bad sizes, a pad_id inside [0, V), or E, E_text or out not 16-byte aligned.
 * A token outside [0, V) other than pad_id, a text id outside [0, V_text), or
 * a TEXT row without a text table makes that row's output zero and sets
 * MCD_DEV_BAD_TOKEN in the workspace status word (when a workspace is given). */
mcd_status mcd_next_input(const mcd_next_input_args *args, hipStream_t stream);

/* ---- paired co-scheduling (Sec. 2.4 input allocation and co-scheduling) ---
 * [host] A continuous-batching scheduler for CFG requests; no HIP calls.
 *   - Auto-allocation: a request with cfg_w > 1 becomes a unit of two rows, its
 *     Main row and a Companion row with a null prompt; other requests are
 *     one-row units.
 *   - Atomic unit: a unit is admitted with all its rows or not at all, holds
 *     them until it finishes, and its rows finish together.
 *   - Equal budget: in a step, each member of a pair is granted the same
 *     number of prompt tokens, c = min(floor(left / 2), the larger remaining
 *     prompt), and the pair is charged 2c whether or not the shorter prompt
 *     uses its share.
 *   - CFG only in the audio phase (Sec. 3.4): a decoding request first emits text_len
 *     text tokens (its Main row is a TEXT row of the head; the Companion is
 *     not run), then n_frames + drain_steps audio steps (Main COND and
 *     Companion UNCOND rows, or one SOLO row).  The Companion joins the audio
 *     phase with a copy of the Main sequence (a prefix-cache hit: no prompt
 *     tokens).
 * One step: mcd_sched_plan builds the batch (decode rows of running units
 * first, one token each; then prompt chunks of prefilling units in admission
 * order; then strict first-come admission while rows and budget remain), and
 * mcd_sched_commit applies it.  A unit whose prompts complete in a step
 * decodes from the next step on.  A scheduler is not thread-safe: one caller
 * at a time. */
typedef struct mcd_sched mcd_sched;

typedef struct {
  int32_t max_rows;          /* rows of the batch (Main and Companion rows), >= 1 */
  int32_t token_budget;      /* backbone tokens per step, >= max_rows */
  int32_t null_prompt_len;   /* prompt tokens of a Companion, >= 1 */
  int32_t drain_steps;       /* audio steps after the last frame (largest delay), >= 0 */
  int32_t max_requests;      /* requests held at once (waiting and running), >= 1 */
} mcd_sched_desc;

typedef struct {
  float cfg_w;               /* > 1: a pair with a Companion */
  int32_t prompt_len;        /* >= 1 */
  int32_t text_len;          /* text tokens before the audio, >= 0 */
  int32_t n_frames;          /* audio frames, >= 1 */
} mcd_sched_request;

/* The planned step; the arrays belong to the scheduler and stay valid until
 * the next mcd_sched_plan or mcd_sched_destroy. */
typedef struct {
  int32_t n_rows;            /* backbone rows of the step (rows with tokens) */
  const int32_t *row_req;    /* [n_rows] request id */
  const uint8_t *row_member; /* [n_rows] 0 Main, 1 Companion */
  const int32_t *row_slot;   /* [n_rows] the row's slot in [0, max_rows) */
  const int32_t *row_tokens; /* [n_rows] tokens this step (prompt chunk, or 1) */
  const int32_t *row_context;/* [n_rows] tokens already in the row's context */
  int32_t R;                 /* head rows: the decoding rows, in backbone order */
  const int32_t *head_row;   /* [R] backbone row of each head row */
  const int32_t *pair_map;   /* [R] head index of the partner, -1 */
  const uint8_t *row_kind;   /* [R] MCD_ROW_* */
  const float *cfg_w;        /* [R] */
  const int32_t *step;       /* [R] audio step (text rows: text step) */
  const int32_t *n_frames;   /* [R] */
  const int32_t *grid_slot;  /* [R] Main's slot for audio Main/SOLO rows, else -1 */
} mcd_sched_batch;

mcd_status mcd_sched_create(const mcd_sched_desc *desc, mcd_sched **out);
void mcd_sched_destroy(mcd_sched *s);
/* Queue a request; *id receives its id (0, 1, ... in submission order).
 * MCD_E_INVALID for bad fields, a pair on a one-row batch, or a full table. */
mcd_status mcd_sched_submit(mcd_sched *s, const mcd_sched_request *req, int32_t *id);
/* Plan the next step.  MCD_E_INVALID if the last planned step is not yet
 * committed. */
mcd_status mcd_sched_plan(mcd_sched *s, mcd_sched_batch *out);
/* Apply the planned step.  The ids of the requests that finished with it go
 * to finished[0 .. *n_finished) (at most cap; MCD_E_INVALID and nothing
 * applied if more would finish). */
mcd_status mcd_sched_commit(mcd_sched *s, int32_t *finished, int32_t cap, int32_t *n_finished);
/* Requests waiting and running. */
mcd_status mcd_sched_counts(const mcd_sched *s, int32_t *waiting, int32_t *running);

/* ---- device status ----------------------------------------------------------
 * Synchronises `stream`, returns the status word of the workspace in *code
 * (MCD_DEV_* bits) and clears it. */
mcd_status mcd_read_device_status(void *workspace, uint32_t *code, hipStream_t stream);

const char *mcd_status_string(mcd_status s);
const char *mcd_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* MCD_H */
