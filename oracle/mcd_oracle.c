/*
 * Plain CPU oracle for the multi-codebook audio decode head.
 *
 * TEST INFRASTRUCTURE ONLY (see mcd_oracle.h).  Single-threaded, fp64, plain
 * loops; obviously-correct over fast.  Sections refer to the paper
 * "An Efficient vLLM-Based Inference Pipeline for Unified Audio Understanding
 * and Generation" (arXiv 2607.02119).
 */
#include "mcd_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Philox4x64-10, from Salmon, Moraes, Dror and Shaw, "Parallel random numbers:
 * as easy as 1, 2, 3" (SC'11): ten rounds of the 4x64 S-box (two 64x64->128
 * multiplies, hi/lo words xor-ed with the other counter words and the round
 * key), with the key bumped by the two Weyl constants between rounds.  The
 * multiplier and Weyl constants are the ones published there.  */

static void orc_mulhilo64(uint64_t a, uint64_t b, uint64_t *hi, uint64_t *lo) {
  unsigned __int128 p = (unsigned __int128)a * (unsigned __int128)b;
  *lo = (uint64_t)p;
  *hi = (uint64_t)(p >> 64);
}

void orc_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ULL, M1 = 0xCA5A826395121157ULL;
  const uint64_t W0 = 0x9E3779B97F4A7C15ULL, W1 = 0xBB67AE8584CAA73BULL;
  uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) { k0 += W0; k1 += W1; }
    uint64_t hi0, lo0, hi1, lo1;
    orc_mulhilo64(M0, x0, &hi0, &lo0);
    orc_mulhilo64(M1, x2, &hi1, &lo1);
    uint64_t y0 = hi1 ^ x1 ^ k0;
    uint64_t y1 = lo1;
    uint64_t y2 = hi0 ^ x3 ^ k1;
    uint64_t y3 = lo0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* Philox4x32-10, from the same paper: ten rounds of the 4x32 S-box (two
 * 32x32->64 multiplies, hi/lo words xor-ed with the other counter words and the
 * round key), with the key bumped by the two 32-bit Weyl constants between
 * rounds; multiplier and Weyl constants as published there. */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) { k0 += W0; k1 += W1; }
    uint64_t p0 = (uint64_t)M0 * x0;
    uint64_t p1 = (uint64_t)M1 * x2;
    uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    uint32_t y1 = (uint32_t)p1;
    uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    uint32_t y3 = (uint32_t)p0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* Two levels of counter-based Philox.  The key material of the vector
 * (request rng_key, step t, codebook k): D = Philox4x64-10 at counter
 * (0, k, t, rng_key) with key (seed, 0).  Element v: word v mod 4 of
 * Philox4x32-10 at counter (v / 4, lo D1, hi D1, lo D2) with key (lo D0, hi D0).
 * Its top 23 bits, plus one half, scaled by 2^-23: a uniform on the open
 * interval (0,1) that is exact in fp32 and fp64. */
double orc_uniform(uint64_t seed, uint64_t rng_key, int64_t t, int32_t k, int32_t v) {
  uint64_t c64[4] = {0, (uint64_t)k, (uint64_t)t, rng_key};
  uint64_t k64[2] = {seed, 0};
  uint64_t d[4];
  orc_philox4x64_10(c64, k64, d);
  uint32_t c32[4] = {(uint32_t)(v >> 2), (uint32_t)d[1], (uint32_t)(d[1] >> 32), (uint32_t)d[2]};
  uint32_t k32[2] = {(uint32_t)d[0], (uint32_t)(d[0] >> 32)};
  uint32_t w[4];
  orc_philox4x32_10(c32, k32, w);
  return ((double)(w[v & 3] >> 9) + 0.5) * ldexp(1.0, -23);
}

/* Gumbel(0,1) by inversion of its CDF exp(-exp(-g)). */
double orc_gumbel(uint64_t seed, uint64_t rng_key, int64_t t, int32_t k, int32_t v) {
  double u = orc_uniform(seed, rng_key, t, k, v);
  return -log(-log(u));
}

/* ------------------------------------------------------------------------- */
/* Head projection, Sec. 2.1: each codebook head maps the hidden state to its
 * logits; head k's weight is the k-th audio slice of the shared head, stored
 * here as rows n = k*V + v of a [K*V][H] matrix.  The stream embedding term
 * W_k e_k, when used, arrives as the bias. */

static double orc_elem(const void *p, int32_t dtype, int64_t i) {
  if (dtype == ORC_BF16) {
    uint32_t bits = (uint32_t)((const uint16_t *)p)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
  }
  return (double)((const float *)p)[i];
}

void orc_logits_row(const void *x, int32_t dtype, const void *W, const float *bias,
                    int32_t H, int32_t N, double *out) {
  double *xd = (double *)malloc(sizeof(double) * (size_t)H);
  for (int32_t h = 0; h < H; ++h) xd[h] = orc_elem(x, dtype, h);
  for (int32_t n = 0; n < N; ++n) {
    double acc = 0.0;
    int64_t base = (int64_t)n * H;
    for (int32_t h = 0; h < H; ++h) acc += xd[h] * orc_elem(W, dtype, base + h);
    if (bias) acc += (double)bias[n];
    out[n] = acc;
  }
  free(xd);
}

/* ------------------------------------------------------------------------- */
/* Selection and sampling of one score vector.
 *   greedy : token = argmax s, lowest id on ties.
 *   top-k  : keep the k first ids in (score desc, id asc) order.
 *   top-p  : over the survivors, softmax mass q; keep the shortest prefix of
 *            that order whose running mass reaches p (at least one id).
 *   draw   : token = argmax over kept ids of s_v + G_v (Gumbel-max), lowest id
 *            on ties; this is an exact draw from softmax restricted to kept. */

typedef struct { double s; int32_t id; } orc_item;

static int orc_cmp_desc(const void *a, const void *b) {
  const orc_item *x = (const orc_item *)a, *y = (const orc_item *)b;
  if (x->s > y->s) return -1;
  if (x->s < y->s) return 1;
  return (x->id < y->id) ? -1 : (x->id > y->id);
}

int32_t orc_sample_vector(const double *s, int32_t V, int32_t greedy, int32_t top_k,
                          double top_p, uint64_t seed, uint64_t rng_key, int64_t t,
                          int32_t k, double gap_tol, double topk_tol, double topp_tol,
                          double *gap_out, uint32_t *flags_out, uint8_t *kept_out) {
  uint32_t flags = 0;
  double gap = INFINITY;
  int32_t token = -1;
  if (kept_out) memset(kept_out, 0, (size_t)V);

  if (greedy) {
    double best = -INFINITY, second = -INFINITY;
    for (int32_t v = 0; v < V; ++v) {
      if (token < 0 || s[v] > best) {
        second = best;
        best = s[v];
        token = v;
      } else if (s[v] > second) {
        second = s[v];
      }
    }
    if (V > 1) gap = best - second;
    if (gap < gap_tol) flags |= ORC_FLAG_GAP_SMALL;
    if (kept_out) kept_out[token] = 1;
    if (gap_out) *gap_out = gap;
    if (flags_out) *flags_out = flags;
    return token;
  }

  orc_item *order = (orc_item *)malloc(sizeof(orc_item) * (size_t)V);
  for (int32_t v = 0; v < V; ++v) { order[v].s = s[v]; order[v].id = v; }
  qsort(order, (size_t)V, sizeof(orc_item), orc_cmp_desc);

  int32_t n_keep = V;
  if (top_k > 0 && top_k < V) {
    n_keep = top_k;
    if (fabs(order[top_k - 1].s - order[top_k].s) < topk_tol) flags |= ORC_FLAG_TOPK_EDGE;
  }

  if (top_p < 1.0) {
    double mx = order[0].s;
    double Z = 0.0;
    for (int32_t i = 0; i < n_keep; ++i) Z += exp(order[i].s - mx);
    double acc = 0.0, cum = 0.0, prev = 0.0;
    int32_t cut = n_keep;
    for (int32_t i = 0; i < n_keep; ++i) {
      prev = cum;
      acc += exp(order[i].s - mx);
      cum = acc / Z;
      if (cum >= top_p) { cut = i + 1; break; }
    }
    if (fabs(cum - top_p) < topp_tol) flags |= ORC_FLAG_TOPP_EDGE;
    if (cut > 1 && fabs(prev - top_p) < topp_tol) flags |= ORC_FLAG_TOPP_EDGE;
    n_keep = cut;
  }

  double best = -INFINITY, second = -INFINITY;
  for (int32_t i = 0; i < n_keep; ++i) {
    int32_t v = order[i].id;
    double x = order[i].s + orc_gumbel(seed, rng_key, t, k, v);
    if (kept_out) kept_out[v] = 1;
    if (token < 0 || x > best || (x == best && v < token)) {
      if (token >= 0) second = best;
      best = x;
      token = v;
    } else if (x > second) {
      second = x;
    }
  }
  if (n_keep > 1) gap = best - second;
  if (gap < gap_tol) flags |= ORC_FLAG_GAP_SMALL;
  free(order);
  if (gap_out) *gap_out = gap;
  if (flags_out) *flags_out = flags;
  return token;
}

/* ------------------------------------------------------------------------- */
/* Batch structure, Sec. 2.4: a conditional (Main) row and its unconditional
 * (Companion) row are partners through pair_map; solo audio rows and text
 * rows have no partner. */

/* Size of stream k and the offset of its block in the N columns. */
static int32_t orc_stream_V(const orc_step_args *a, int32_t k) {
  return a->V_stream ? a->V_stream[k] : a->V;
}

static int64_t orc_stream_off(const orc_step_args *a, int32_t k) {
  int64_t off = 0;
  for (int32_t j = 0; j < k; ++j) off += orc_stream_V(a, j);
  return off;
}

static int32_t orc_check_batch(const orc_step_args *a) {
  if (a->R < 0 || a->K <= 0 || a->V <= 0 || a->H <= 0) return ORC_E_SHAPE;
  for (int32_t k = 0; k < a->K; ++k)
    if (orc_stream_V(a, k) <= 0) return ORC_E_SHAPE;
  for (int32_t r = 0; r < a->R; ++r) {
    int32_t kind = a->row_kind[r], p = a->pair_map[r];
    if (kind == ORC_ROW_COND || kind == ORC_ROW_UNCOND) {
      if (p < 0 || p >= a->R || p == r) return ORC_E_PAIR;
      int32_t want = (kind == ORC_ROW_COND) ? ORC_ROW_UNCOND : ORC_ROW_COND;
      if (a->row_kind[p] != want || a->pair_map[p] != r) return ORC_E_PAIR;
    } else if (kind == ORC_ROW_SOLO || kind == ORC_ROW_TEXT) {
      if (p != -1) return ORC_E_PAIR;
      if (kind == ORC_ROW_TEXT && (a->W_text == NULL || a->V_text <= 0)) return ORC_E_SHAPE;
    } else {
      return ORC_E_PAIR;
    }
    if (kind == ORC_ROW_COND || kind == ORC_ROW_SOLO) {
      float T = a->temperature[r], P = a->top_p[r];
      if (!(T >= 0.0f) || !isfinite(T)) return ORC_E_PARAM;
      if (!(P > 0.0f)) return ORC_E_PARAM;
      if (kind == ORC_ROW_COND && !isfinite(a->cfg_w[r])) return ORC_E_PARAM;
    }
  }
  return ORC_OK;
}

/* Tokens, companion copy and frame-grid write of one sampled row, given its
 * scores s[K*V].  Delay pattern (Sec. 2.1): codebook k at step t carries frame
 * f = t - d_k; there is no frame before the stream starts (f < 0) and none
 * once its frames are exhausted (f >= n_frames, the drain of Sec. 2.3), and
 * those positions carry the pad id.  Companion (Sec. 2.4): it receives the
 * Main row's tokens, and nothing of it reaches the client (no grid cell). */
static void orc_emit_row(const orc_step_args *a, int32_t r, int32_t u, const double *s) {
  int64_t t = a->step[r];
  uint64_t key = a->rng_key ? a->rng_key[r] : (uint64_t)r;
  int32_t greedy = (a->temperature[r] == 0.0f);
  for (int32_t k = 0; k < a->K; ++k) {
    int64_t f = t - a->delays[k];
    int32_t pad = (f < 0) || (a->n_frames[r] >= 0 && f >= a->n_frames[r]);
    int32_t token;
    double gap = INFINITY;
    uint32_t flags = 0;
    if (pad) {
      token = a->pad_id;
      flags = ORC_FLAG_PAD;
    } else {
      token = orc_sample_vector(s + orc_stream_off(a, k), orc_stream_V(a, k), greedy, a->top_k[r],
                                (double)a->top_p[r], a->seed, key, t, k, a->gap_tol,
                                a->topk_tol, a->topp_tol, &gap, &flags, NULL);
    }
    a->tokens_out[(int64_t)r * a->K + k] = token;
    if (u >= 0) a->tokens_out[(int64_t)u * a->K + k] = token;
    if (a->gap) a->gap[(int64_t)r * a->K + k] = gap;
    if (a->flags) a->flags[(int64_t)r * a->K + k] = flags;
    int32_t slot = a->grid_slot[r];
    if (!pad && slot >= 0 && slot < a->n_slots && f < a->F_max && a->frame_grid)
      a->frame_grid[((int64_t)slot * a->K + k) * a->F_max + f] = token;
  }
}

int32_t orc_head_step(const orc_step_args *a) {
  int32_t rc = orc_check_batch(a);
  if (rc != ORC_OK) return rc;
  const int32_t N = (int32_t)orc_stream_off(a, a->K);
  double *lc = (double *)malloc(sizeof(double) * (size_t)N);
  double *lu = (double *)malloc(sizeof(double) * (size_t)N);
  double *sc = (double *)malloc(sizeof(double) * (size_t)N);
  for (int32_t r = 0; r < a->R; ++r) {
    int32_t kind = a->row_kind[r];
    const size_t esz = (a->dtype == ORC_BF16) ? 2 : 4;
    const char *hrow = (const char *)a->hidden + (size_t)r * a->H * esz;
    if (kind == ORC_ROW_TEXT) {
      double *lt = (double *)malloc(sizeof(double) * (size_t)a->V_text);
      orc_logits_row(hrow, a->dtype, a->W_text, NULL, a->H, a->V_text, lt);
      double gap = INFINITY;
      uint32_t flags = 0;
      /* vocabulary mask of the text phase: the token is the greedy one over
       * the text ids; the modality is where the unmasked argmax lies */
      int32_t T = (a->T_text > 0 && a->T_text < a->V_text) ? a->T_text : a->V_text;
      int32_t tok = orc_sample_vector(lt, T, 1, 0, 1.0, a->seed, 0, 0, 0,
                                      a->gap_tol, a->topk_tol, a->topp_tol, &gap, &flags, NULL);
      int32_t best = 0;
      for (int32_t v = 1; v < a->V_text; ++v)
        if (lt[v] > lt[best]) best = v;      /* strict: the lowest id on ties */
      double mt = -INFINITY, mo = -INFINITY;
      for (int32_t v = 0; v < a->V_text; ++v) {
        if (v < T) mt = lt[v] > mt ? lt[v] : mt;
        else mo = lt[v] > mo ? lt[v] : mo;
      }
      if (a->modality) a->modality[r] = (uint8_t)(best >= T);
      if (a->modality_gap) a->modality_gap[r] = T < a->V_text ? fabs(mt - mo) : INFINITY;
      for (int32_t k = 0; k < a->K; ++k) {
        a->tokens_out[(int64_t)r * a->K + k] = (k == 0) ? tok : a->pad_id;
        if (a->gap) a->gap[(int64_t)r * a->K + k] = (k == 0) ? gap : INFINITY;
        if (a->flags) a->flags[(int64_t)r * a->K + k] = (k == 0) ? flags : ORC_FLAG_PAD;
      }
      free(lt);
      continue;
    }
    if (kind == ORC_ROW_UNCOND) continue; /* handled with its Main row */
    orc_logits_row(hrow, a->dtype, a->W, a->bias, a->H, N, lc);
    int32_t u = -1;
    if (kind == ORC_ROW_COND) {
      /* CFG merge, Eq. 1: w * l_cond + (1 - w) * l_uncond, per codebook. */
      u = a->pair_map[r];
      const char *hu = (const char *)a->hidden + (size_t)u * a->H * esz;
      orc_logits_row(hu, a->dtype, a->W, a->bias, a->H, N, lu);
      double w = (double)a->cfg_w[r];
      for (int32_t n = 0; n < N; ++n) sc[n] = w * lc[n] + (1.0 - w) * lu[n];
    } else {
      for (int32_t n = 0; n < N; ++n) sc[n] = lc[n];
    }
    /* temperature: divide after the merge; T = 0 means greedy on the merge */
    double T = (double)a->temperature[r];
    if (T > 0.0)
      for (int32_t n = 0; n < N; ++n) sc[n] = sc[n] / T;
    if (a->scores) memcpy(a->scores + (int64_t)r * N, sc, sizeof(double) * (size_t)N);
    orc_emit_row(a, r, u, sc);
  }
  free(lc);
  free(lu);
  free(sc);
  return ORC_OK;
}

int32_t orc_sample_rows(const orc_step_args *a, int32_t Rs, const int32_t *srow,
                        const int32_t *crow, const double *scores) {
  const int64_t N = orc_stream_off(a, a->K);
  for (int32_t i = 0; i < Rs; ++i) {
    int32_t r = srow[i];
    if (r < 0 || r >= a->R) return ORC_E_SHAPE;
    float T = a->temperature[r], P = a->top_p[r];
    if (!(T >= 0.0f) || !(P > 0.0f)) return ORC_E_PARAM;
    orc_emit_row(a, r, crow[i], scores + (int64_t)i * N);
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Delay pattern (Sec. 2.1): stream k is offset by d_k steps, so the token of
 * codebook k emitted at step t belongs to frame t - d_k.  De-interleaving
 * gathers each frame's tokens from the steps that carried them. */

static int32_t orc_max_delay(const int32_t *delays, int32_t K) {
  int32_t m = 0;
  for (int32_t k = 0; k < K; ++k) {
    if (delays[k] < 0) return -1;
    if (delays[k] > m) m = delays[k];
  }
  return m;
}

int32_t orc_deinterleave(const int32_t *streams, int32_t T, int32_t K,
                         const int32_t *delays, int32_t *grid) {
  int32_t md = orc_max_delay(delays, K);
  if (md < 0 || T < md) return ORC_E_SHAPE;
  int32_t F = T - md;
  for (int32_t k = 0; k < K; ++k)
    for (int32_t f = 0; f < F; ++f)
      grid[(int64_t)k * F + f] = streams[(int64_t)(f + delays[k]) * K + k];
  return ORC_OK;
}

int32_t orc_interleave(const int32_t *grid, int32_t F, int32_t K, const int32_t *delays,
                       int32_t pad_id, int32_t *streams) {
  int32_t md = orc_max_delay(delays, K);
  if (md < 0 || F < 0) return ORC_E_SHAPE;
  int32_t T = F + md;
  for (int32_t t = 0; t < T; ++t)
    for (int32_t k = 0; k < K; ++k) {
      int32_t f = t - delays[k];
      streams[(int64_t)t * K + k] = (f >= 0 && f < F) ? grid[(int64_t)k * F + f] : pad_id;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Next-step input (Sec. 2.1): the sum of the embeddings of the tokens a row
 * emitted at this step, one per stream, in fp64, rounded once to the table
 * type.  A sum of at most 32 values with 8 (bf16) or 24 (fp32) significant bits
 * is exact in a double when their exponents span at most 40 or 24 bits, which
 * covers any embedding table of sane scale; then the result is the exact sum
 * rounded once. */

/* Round a double to the nearest bfloat16 (8 significant bits), ties to even,
 * directly from the double (no intermediate fp32 rounding). */
static uint16_t orc_bf16_rne(double x) {
  float f;
  uint32_t bits;
  if (isnan(x)) return 0x7FC0;
  if (x == 0.0 || isinf(x)) {
    f = (float)x;
    memcpy(&bits, &f, sizeof bits);
    return (uint16_t)(bits >> 16);
  }
  int e;
  (void)frexp(x, &e);            /* |x| = m * 2^e, 0.5 <= m < 1: leading bit 2^(e-1) */
  int lead = e - 1;
  if (lead < -126) lead = -126;  /* bf16 subnormals keep the spacing 2^-133 */
  double ulp = ldexp(1.0, lead - 7);
  double q = x / ulp;            /* exact: scaling by a power of two */
  double r = nearbyint(q);       /* the default rounding mode: nearest, ties to even */
  double y = r * ulp;
  if (fabs(y) >= ldexp(1.0, 128)) y = x > 0 ? INFINITY : -INFINITY;
  f = (float)y;                  /* exact: y has at most 8 significant bits */
  memcpy(&bits, &f, sizeof bits);
  return (uint16_t)(bits >> 16);
}

int32_t orc_next_input(int32_t R, int32_t H, int32_t K, int32_t V, int32_t pad_id,
                       int32_t dtype, const void *E, int32_t V_text, const void *E_text,
                       const uint8_t *row_kind, const int32_t *tokens, void *out) {
  if (R < 0 || H < 1 || K < 1 || V < 1 || !E || !row_kind || !tokens || !out)
    return ORC_E_SHAPE;
  if (pad_id >= 0 && pad_id < V) return ORC_E_SHAPE;
  int32_t rc = ORC_OK;
  double *acc = (double *)malloc(sizeof(double) * (size_t)H);
  for (int32_t r = 0; r < R; ++r) {
    for (int32_t h = 0; h < H; ++h) acc[h] = 0.0;
    if (row_kind[r] == ORC_ROW_TEXT) {
      int32_t id = tokens[(int64_t)r * K];
      if (!E_text || id < 0 || id >= V_text) {
        rc = ORC_E_PARAM;
      } else {
        for (int32_t h = 0; h < H; ++h) acc[h] = orc_elem(E_text, dtype, (int64_t)id * H + h);
      }
    } else {
      for (int32_t k = 0; k < K; ++k) {
        int32_t tok = tokens[(int64_t)r * K + k];
        int32_t row;
        if (tok == pad_id) row = V;
        else if (tok >= 0 && tok < V) row = tok;
        else {
          rc = ORC_E_PARAM;
          continue;
        }
        int64_t base = ((int64_t)k * (V + 1) + row) * H;
        for (int32_t h = 0; h < H; ++h) acc[h] += orc_elem(E, dtype, base + h);
      }
    }
    for (int32_t h = 0; h < H; ++h) {
      int64_t i = (int64_t)r * H + h;
      if (dtype == ORC_BF16) ((uint16_t *)out)[i] = orc_bf16_rne(acc[h]);
      else ((float *)out)[i] = (float)acc[h];   /* C's conversion: nearest, ties to even */
    }
  }
  free(acc);
  return rc;
}
