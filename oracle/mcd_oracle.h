/*
 * Plain CPU oracle for the multi-codebook audio decode head.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link,
 * load or call this code: only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark use it.  It shares no code, header, table or
 * constant with the HIP library under paper_2607_02119_amd/.
 *
 * Single-threaded, plain loops, fp64 arithmetic throughout.  Every function
 * follows the definition in the paper (Sec. 2.1 for the heads and the delay
 * pattern, Sec. 2.3 for the drain, Sec. 2.4 / Eq. 1 for the CFG merge and the
 * companion copy) or, where the paper is silent (temperature, top-k, top-p,
 * Gumbel-max, Philox), the plain textbook definition stated next to it.
 */
#ifndef MCD_ORACLE_H
#define MCD_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_ROW_COND = 0, ORC_ROW_UNCOND = 1, ORC_ROW_SOLO = 2, ORC_ROW_TEXT = 3 };
enum { ORC_F32 = 0, ORC_BF16 = 1 };

/* per-position classification of a sampled token */
enum {
  ORC_FLAG_GAP_SMALL = 1u,     /* top-2 perturbed (or greedy) score gap < gap_tol */
  ORC_FLAG_TOPP_EDGE = 2u,     /* running nucleus mass within topp_tol of p at the cut */
  ORC_FLAG_TOPK_EDGE = 4u,     /* k-th and (k+1)-th sorted scores within topk_tol */
  ORC_FLAG_PAD = 8u            /* position forced to the pad id by the delay pattern */
};

enum {
  ORC_OK = 0,
  ORC_E_PAIR = 1,      /* pair_map / row_kind inconsistent */
  ORC_E_PARAM = 2,     /* a sampling parameter out of range */
  ORC_E_SHAPE = 3      /* sizes or pointers unusable */
};

typedef struct {
  /* head */
  int32_t H, K, V, pad_id;
  const int32_t *delays;      /* [K] */
  int32_t dtype;              /* ORC_F32 or ORC_BF16: element type of hidden, W, W_text */
  const void *W;              /* [N][H]: [K][V][H] for equal streams */
  const float *bias;          /* [N] or NULL */
  int32_t V_text;
  const void *W_text;         /* [V_text][H] or NULL */
  /* Streams of unequal size (heterogeneous codebooks): stream k has V_stream[k]
   * ids, its rows of W (and entries of bias, columns of scores) start at
   * sum_{j<k} V_stream[j], and N = sum_k V_stream[k].  NULL: V for every
   * stream, N = K * V. */
  const int32_t *V_stream;    /* [K] or NULL */
  /* Text-phase vocabulary mask (Sec. 2.3): ids [0, T_text) of the text head
   * are text tokens, the rest belong to other modalities.  A TEXT row emits
   * the greedy token over the text ids only; its modality is read from the
   * unmasked distribution: 1 when the argmax over all V_text ids (lowest id
   * on ties) lies outside the text ids.  0 or V_text: no mask. */
  int32_t T_text;
  /* batch */
  int32_t R;
  const void *hidden;         /* [R][H] */
  const int32_t *pair_map;    /* [R] */
  const uint8_t *row_kind;    /* [R] */
  const float *cfg_w;         /* [R] */
  const float *temperature;   /* [R] */
  const int32_t *top_k;       /* [R] */
  const float *top_p;         /* [R] */
  const uint64_t *rng_key;    /* [R] or NULL (row index) */
  const int32_t *step;        /* [R] */
  const int32_t *n_frames;    /* [R] */
  const int32_t *grid_slot;   /* [R] */
  uint64_t seed;
  int32_t n_slots, F_max;
  /* classification tolerances */
  double gap_tol, topk_tol, topp_tol;
  /* outputs (caller-allocated) */
  int32_t *tokens_out;        /* [R][K] */
  int32_t *frame_grid;        /* [n_slots][K][F_max]; only cells with a frame this step are written */
  uint8_t *modality;          /* [R] or NULL: TEXT rows' modality flag, untouched otherwise */
  double *modality_gap;       /* [R] or NULL: |max over text ids - max over the rest| */
  double *scores;             /* [R][N] or NULL: s for COND/SOLO rows, untouched otherwise */
  double *gap;                /* [R][K] or NULL */
  uint32_t *flags;            /* [R][K] or NULL */
} orc_step_args;

/* Philox4x64 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11). */
void orc_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);

/* Philox4x32 with 10 rounds (same paper). */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Uniform in (0,1) for element v of codebook k of request rng_key at step t. */
double orc_uniform(uint64_t seed, uint64_t rng_key, int64_t t, int32_t k, int32_t v);

/* Standard Gumbel variate -log(-log(u)) for the same coordinates. */
double orc_gumbel(uint64_t seed, uint64_t rng_key, int64_t t, int32_t k, int32_t v);

/* One row of head logits: out[n] = sum_h x[h] * W[n][h] (+ bias[n]), n < N. */
void orc_logits_row(const void *x, int32_t dtype, const void *W, const float *bias,
                    int32_t H, int32_t N, double *out);

/* Select and sample one vector of V scores.  Returns the token id. */
int32_t orc_sample_vector(const double *s, int32_t V, int32_t greedy, int32_t top_k,
                          double top_p, uint64_t seed, uint64_t rng_key, int64_t t,
                          int32_t k, double gap_tol, double topk_tol, double topp_tol,
                          double *gap_out, uint32_t *flags_out, uint8_t *kept_out);

/* One decode step of the whole head over a batch.  Returns ORC_OK or an error. */
int32_t orc_head_step(const orc_step_args *a);

/* Sample a batch of ready-made scores (the part after the merge), rows given in
 * sampled order: scores[s][N], row s is physical row srow[s], companion crow[s]
 * (-1 for none).  Same outputs as orc_head_step for those rows. */
int32_t orc_sample_rows(const orc_step_args *a, int32_t Rs, const int32_t *srow,
                        const int32_t *crow, const double *scores);

/* Delay pattern: streams[T][K] -> grid[K][T - max_d]. */
int32_t orc_deinterleave(const int32_t *streams, int32_t T, int32_t K,
                         const int32_t *delays, int32_t *grid);
/* Delay pattern: grid[K][F] -> streams[F + max_d][K], pad_id where no frame. */
int32_t orc_interleave(const int32_t *grid, int32_t F, int32_t K, const int32_t *delays,
                       int32_t pad_id, int32_t *streams);

/* Next-step input (Sec. 2.1, delay pattern): the backbone's input for the
 * next step aggregates the embeddings of the K tokens a row emitted at this
 * step, one per stream (each belongs to its own delayed frame).  Read here as
 * a sum: out[r][h] = sum_k E[k][row_k][h], row_k = tokens[r][k], or row V of
 * stream k's table [V + 1][H] for the pad id.  The sum is taken in fp64 (exact
 * when the values' exponents span at most 40 bits for bf16, 24 for fp32) and
 * rounded once, to nearest even, to the table type.  TEXT rows take
 * E_text[tokens[r][0]].  ORC_E_PARAM for a token outside [0, V) that is not
 * the pad id, or a text id outside [0, V_text); out is then unspecified. */
int32_t orc_next_input(int32_t R, int32_t H, int32_t K, int32_t V, int32_t pad_id,
                       int32_t dtype, const void *E, int32_t V_text, const void *E_text,
                       const uint8_t *row_kind, const int32_t *tokens, void *out);

#ifdef __cplusplus
}
#endif
#endif
