// Paired co-scheduling of CFG requests in a continuous batch (host only).
//
// A request with w > 1 is served as a Main request plus an auto-allocated
// Companion with a null prompt; the two form one scheduling unit that is
// admitted, run and retired together, and each of its members gets the same
// share of a step's token budget (Sec. 2.4, input allocation and
// co-scheduling).  The merge, and with it the Companion, is active only in the
// audio phase (Sec. 3.4): text comes first, greedy and unmerged, as in the
// mixed understanding/generation models of Sec. 2.3.
#include <cmath>
#include <cstdio>
#include <new>
#include <vector>

#include "mcd.h"
#include "mcd_internal.h"

namespace {

enum Stage { kWaiting = 0, kPrefill = 1, kDecode = 2 };

struct Req {
  int32_t id;
  float w;
  bool pair;
  int32_t prompt, text, frames;
  int stage;
  int32_t left[2];      // prompt tokens still to prefill: Main, Companion
  int32_t done[2];      // prompt tokens prefilled
  int32_t t;            // decode steps taken
  int32_t slot[2];
};

mcd_status bad(const char *msg) { return mcd::record_error(MCD_E_INVALID, msg); }

}  // namespace

struct mcd_sched {
  mcd_sched_desc d;
  int32_t next_id = 0;
  std::vector<Req> reqs;          // waiting and running, in submission order
  std::vector<uint8_t> slot_used;
  bool planned = false;
  // the planned step
  std::vector<int32_t> grant[2];  // per request (index into reqs): prompt tokens granted
  std::vector<uint8_t> decoding;  // per request: decodes this step
  std::vector<int32_t> row_req, row_slot, row_tokens, row_context;
  std::vector<uint8_t> row_member;
  std::vector<int32_t> head_row, pair_map, step, n_frames, grid_slot;
  std::vector<uint8_t> row_kind;
  std::vector<float> cfg_w;
};

namespace {

int32_t audio_steps(const mcd_sched &s, const Req &r) { return r.frames + s.d.drain_steps; }

int rows_of(const Req &r) { return r.pair ? 2 : 1; }

int32_t lowest_free(mcd_sched &s) {
  for (int32_t i = 0; i < s.d.max_rows; ++i)
    if (!s.slot_used[i]) return i;
  return -1;
}

// Prompt grant of a prefilling unit from `left` budget tokens: each member of
// a pair is granted c = min(floor(left / 2), larger remaining prompt) and uses
// min(c, its own remainder); the pair is charged 2c.
void grant_prefill(mcd_sched &s, size_t i, int32_t &left) {
  Req &r = s.reqs[i];
  if (r.pair) {
    const int32_t need = r.left[0] > r.left[1] ? r.left[0] : r.left[1];
    int32_t c = left / 2;
    if (c > need) c = need;
    s.grant[0][i] = c < r.left[0] ? c : r.left[0];
    s.grant[1][i] = c < r.left[1] ? c : r.left[1];
    left -= 2 * c;
  } else {
    const int32_t c = left < r.left[0] ? left : r.left[0];
    s.grant[0][i] = c;
    left -= c;
  }
}

void add_row(mcd_sched &s, const Req &r, int member, int32_t tokens, int32_t context) {
  s.row_req.push_back(r.id);
  s.row_member.push_back((uint8_t)member);
  s.row_slot.push_back(r.slot[member]);
  s.row_tokens.push_back(tokens);
  s.row_context.push_back(context);
}

void add_head_row(mcd_sched &s, const Req &r, uint8_t kind, int32_t partner, int32_t step,
                  int32_t grid) {
  s.head_row.push_back((int32_t)s.row_req.size() - 1);
  s.pair_map.push_back(partner);
  s.row_kind.push_back(kind);
  s.cfg_w.push_back(r.w);
  s.step.push_back(step);
  s.n_frames.push_back(r.frames);
  s.grid_slot.push_back(grid);
}

}  // namespace

extern "C" {

mcd_status mcd_sched_create(const mcd_sched_desc *desc, mcd_sched **out) {
  if (!desc || !out) return bad("null description or output");
  const mcd_sched_desc &d = *desc;
  if (d.max_rows < 1 || d.token_budget < d.max_rows || d.null_prompt_len < 1 ||
      d.drain_steps < 0 || d.max_requests < 1)
    return bad("bad scheduler description (rows >= 1, budget >= rows, null prompt >= 1, "
               "drain >= 0, requests >= 1)");
  mcd_sched *s = new (std::nothrow) mcd_sched();
  if (!s) return mcd::record_error(MCD_E_INVALID, "out of host memory");
  s->d = d;
  s->slot_used.assign((size_t)d.max_rows, 0);
  *out = s;
  return MCD_OK;
}

void mcd_sched_destroy(mcd_sched *s) { delete s; }

}  // extern "C"

namespace {

mcd_status sched_submit(mcd_sched *s, const mcd_sched_request *q, int32_t *id) {
  if (!s || !q || !id) return bad("null scheduler, request or id");
  if (!std::isfinite(q->cfg_w) || q->prompt_len < 1 || q->text_len < 0 || q->n_frames < 1)
    return bad("bad request (finite cfg_w, prompt >= 1, text >= 0, frames >= 1)");
  const bool pair = q->cfg_w > 1.0f;
  if (pair && s->d.max_rows < 2) return bad("a CFG pair needs two rows");
  if ((int32_t)s->reqs.size() >= s->d.max_requests) return bad("request table full");
  Req r{};
  r.id = s->next_id++;
  r.w = q->cfg_w;
  r.pair = pair;
  r.prompt = q->prompt_len;
  r.text = q->text_len;
  r.frames = q->n_frames;
  r.stage = kWaiting;
  r.left[0] = q->prompt_len;
  r.left[1] = pair ? s->d.null_prompt_len : 0;
  r.slot[0] = r.slot[1] = -1;
  s->reqs.push_back(r);
  *id = r.id;
  return MCD_OK;
}

mcd_status sched_plan(mcd_sched *s, mcd_sched_batch *out) {
  if (!s || !out) return bad("null scheduler or output");
  if (s->planned) return bad("the planned step is not committed yet");
  const size_t n = s->reqs.size();
  s->grant[0].assign(n, 0);
  s->grant[1].assign(n, 0);
  s->decoding.assign(n, 0);
  s->row_req.clear(); s->row_member.clear(); s->row_slot.clear();
  s->row_tokens.clear(); s->row_context.clear();
  s->head_row.clear(); s->pair_map.clear(); s->row_kind.clear(); s->cfg_w.clear();
  s->step.clear(); s->n_frames.clear(); s->grid_slot.clear();

  int32_t left = s->d.token_budget;
  // 1. decode rows of running units: one token per row
  for (size_t i = 0; i < n; ++i) {
    const Req &r = s->reqs[i];
    if (r.stage != kDecode) continue;
    s->decoding[i] = 1;
    left -= (r.t < r.text || !r.pair) ? 1 : 2;
  }
  // 2. prompt chunks of prefilling units, in admission order
  for (size_t i = 0; i < n; ++i)
    if (s->reqs[i].stage == kPrefill) grant_prefill(*s, i, left);
  // 3. strict first-come admission while rows and budget remain
  int32_t free_rows = 0;
  for (uint8_t u : s->slot_used) free_rows += !u;
  for (size_t i = 0; i < n; ++i) {
    Req &r = s->reqs[i];
    if (r.stage != kWaiting) continue;
    if (free_rows < rows_of(r) || left < rows_of(r)) break;
    for (int m = 0; m < rows_of(r); ++m) {
      r.slot[m] = lowest_free(*s);
      s->slot_used[(size_t)r.slot[m]] = 1;
    }
    free_rows -= rows_of(r);
    r.stage = kPrefill;
    grant_prefill(*s, i, left);
  }
  // rows in unit order: Main, then Companion
  for (size_t i = 0; i < n; ++i) {
    const Req &r = s->reqs[i];
    if (s->decoding[i]) {
      if (r.t < r.text) {
        add_row(*s, r, 0, 1, r.prompt + r.t);
        add_head_row(*s, r, MCD_ROW_TEXT, -1, r.t, -1);
      } else if (!r.pair) {
        add_row(*s, r, 0, 1, r.prompt + r.t);
        add_head_row(*s, r, MCD_ROW_SOLO, -1, r.t - r.text, r.slot[0]);
      } else {
        const int32_t h = (int32_t)s->head_row.size();
        add_row(*s, r, 0, 1, r.prompt + r.t);
        add_head_row(*s, r, MCD_ROW_COND, h + 1, r.t - r.text, r.slot[0]);
        add_row(*s, r, 1, 1, s->d.null_prompt_len + r.t);
        add_head_row(*s, r, MCD_ROW_UNCOND, h, r.t - r.text, -1);
      }
    } else if (r.stage == kPrefill) {
      for (int m = 0; m < rows_of(r); ++m)
        if (s->grant[m][i] > 0) add_row(*s, r, m, s->grant[m][i], r.done[m]);
    }
  }
  s->planned = true;
  out->n_rows = (int32_t)s->row_req.size();
  out->row_req = s->row_req.data();
  out->row_member = s->row_member.data();
  out->row_slot = s->row_slot.data();
  out->row_tokens = s->row_tokens.data();
  out->row_context = s->row_context.data();
  out->R = (int32_t)s->head_row.size();
  out->head_row = s->head_row.data();
  out->pair_map = s->pair_map.data();
  out->row_kind = s->row_kind.data();
  out->cfg_w = s->cfg_w.data();
  out->step = s->step.data();
  out->n_frames = s->n_frames.data();
  out->grid_slot = s->grid_slot.data();
  return MCD_OK;
}

mcd_status sched_commit(mcd_sched *s, int32_t *finished, int32_t cap, int32_t *n_finished) {
  if (!s || !n_finished || cap < 0 || (cap > 0 && !finished))
    return bad("null scheduler, output or bad capacity");
  if (!s->planned) return bad("no planned step to commit");
  const size_t n = s->reqs.size();
  int32_t nf = 0;
  for (size_t i = 0; i < n; ++i) {
    const Req &r = s->reqs[i];
    if (s->decoding[i] && r.t + 1 == r.text + audio_steps(*s, r)) ++nf;
  }
  if (nf > cap) return bad("more requests finish than the output holds");
  std::vector<Req> keep;
  keep.reserve(n);
  nf = 0;
  for (size_t i = 0; i < n; ++i) {
    Req r = s->reqs[i];
    if (s->decoding[i]) {
      if (++r.t == r.text + audio_steps(*s, r)) {
        for (int m = 0; m < rows_of(r); ++m) s->slot_used[(size_t)r.slot[m]] = 0;
        finished[nf++] = r.id;
        continue;
      }
    } else if (r.stage == kPrefill) {
      for (int m = 0; m < 2; ++m) {
        r.left[m] -= s->grant[m][i];
        r.done[m] += s->grant[m][i];
      }
      if (r.left[0] == 0 && r.left[1] == 0) r.stage = kDecode;
    }
    keep.push_back(r);
  }
  s->reqs.swap(keep);
  s->planned = false;
  *n_finished = nf;
  return MCD_OK;
}

}  // namespace

// No exception crosses the C ABI: a failed host allocation becomes an error
// code, after which the scheduler's state is unspecified (destroy it).
extern "C" {

mcd_status mcd_sched_submit(mcd_sched *s, const mcd_sched_request *q, int32_t *id) {
  try {
    return sched_submit(s, q, id);
  } catch (...) {
    return mcd::record_error(MCD_E_INVALID, "out of host memory");
  }
}

mcd_status mcd_sched_plan(mcd_sched *s, mcd_sched_batch *out) {
  try {
    return sched_plan(s, out);
  } catch (...) {
    return mcd::record_error(MCD_E_INVALID, "out of host memory");
  }
}

mcd_status mcd_sched_commit(mcd_sched *s, int32_t *finished, int32_t cap, int32_t *n_finished) {
  try {
    return sched_commit(s, finished, cap, n_finished);
  } catch (...) {
    return mcd::record_error(MCD_E_INVALID, "out of host memory");
  }
}

mcd_status mcd_sched_counts(const mcd_sched *s, int32_t *waiting, int32_t *running) {
  if (!s || !waiting || !running) return bad("null scheduler or output");
  int32_t w = 0, r = 0;
  for (const Req &q : s->reqs) (q.stage == kWaiting ? w : r) += 1;
  *waiting = w;
  *running = r;
  return MCD_OK;
}

}  // extern "C"
