// Host side of libmcd: argument validation, the batch plan and kernel launches.
// Nothing here allocates device memory or synchronises, except
// mcd_read_device_status.  A head with a bf16 text head creates one extra
// stream and two events at creation (mcd_head_create), never in a step.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "mcd.h"
#include "mcd_internal.h"

struct mcd_head {
  mcd::HeadView hv;
  int32_t max_delay;
  // Batches with both audio and text rows run the two projections
  // concurrently: the text part on a second stream of the head, forked from
  // and joined back to the caller's stream with events.  Created with the
  // head (bf16 heads with a text head), so a step creates nothing; the mutex
  // orders the event records of concurrent steps on one head.
  mutable std::mutex side_mu;
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};

namespace {

thread_local std::string g_last_error;

mcd_status fail(mcd_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  try {
    g_last_error = buf;
  } catch (...) {
  }
  return s;
}

mcd_status hip_fail(hipError_t e, const char *what) {
  return fail(MCD_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }


// Text-head partials kept outside the caller's workspace (the allocation-free
// step): base address and capacity of that region; null: in the workspace.
struct ExternalPartials {
  char *base;
  size_t cap;
};

// Bytes of the text partials of n text rows: the values, then the ids, each
// rounded up to 256 bytes.
size_t partials_bytes(const mcd_head *h, int64_t n) {
  if (h->hv.V_text <= 0 || n <= 0) return 0;
  const size_t parts = (size_t)mcd::text_parts_for(h->hv.V_text);
  return round_up((size_t)n * parts * sizeof(float), 256) +
         round_up((size_t)n * parts * sizeof(int32_t), 256);
}

// Shared validation of mcd_head_step / mcd_sample_step; fills the step view.
// With ext, the workspace holds only the status word and the text partials go
// to ext (which must hold them: checked by the caller).
mcd_status make_step_view(const mcd_head *h, const mcd_step_args *a, bool need_hidden,
                          mcd::StepView &sv, const ExternalPartials *ext = nullptr) {
  if (!h || !a) return fail(MCD_E_INVALID, "null head or args");
  const mcd::HeadView &hv = h->hv;
  const mcd_batch_counts &c = a->counts;
  if (a->R < 0 || c.n_pairs < 0 || c.n_solo < 0 || c.n_text < 0)
    return fail(MCD_E_INVALID, "negative row count");
  if ((int64_t)2 * c.n_pairs + c.n_solo + c.n_text != a->R)
    return fail(MCD_E_INVALID, "counts (%d pairs, %d solo, %d text) do not add up to R=%d",
                c.n_pairs, c.n_solo, c.n_text, a->R);
  if (c.n_text > 0 && hv.V_text <= 0)
    return fail(MCD_E_INVALID, "text rows on a head without a text head");
  const int32_t Rs = c.n_pairs + c.n_solo;
  if (a->R > 0 && !a->plan) return fail(MCD_E_INVALID, "plan is null");
  if (need_hidden && a->R > 0) {
    if (!a->hidden) return fail(MCD_E_INVALID, "hidden is null");
    if (hv.dtype == MCD_BF16 && !aligned(a->hidden, 16))
      return fail(MCD_E_INVALID, "hidden must be 16-byte aligned");
    if (hv.dtype == MCD_F32 && !aligned(a->hidden, 4))
      return fail(MCD_E_INVALID, "hidden must be 4-byte aligned");
  }
  // The kernels read every per-row array at every row (text rows included), so
  // a non-empty batch needs all of them; rng_key alone may be null.
  if (a->R > 0 && (!a->cfg_w || !a->temperature || !a->top_k || !a->top_p || !a->step ||
                   !a->n_frames || !a->grid_slot))
    return fail(MCD_E_INVALID, "a per-row parameter array is null");
  if (Rs > 0 && !a->scores) return fail(MCD_E_INVALID, "scores is null");
  if (a->R > 0 && !a->tokens_out) return fail(MCD_E_INVALID, "tokens_out is null");
  if (a->n_slots < 0 || a->F_max < 0) return fail(MCD_E_INVALID, "negative grid size");
  if (a->frame_grid && (int64_t)a->n_slots * hv.K * a->F_max > ((int64_t)1 << 40))
    return fail(MCD_E_INVALID, "frame grid too large");
  const size_t need = ext ? (size_t)mcd::kStatusBytes : mcd_workspace_bytes(h, a->R);
  if (!a->workspace || a->workspace_bytes < need)
    return fail(MCD_E_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                a->workspace ? a->workspace_bytes : (size_t)0);
  if (!aligned(a->workspace, 256)) return fail(MCD_E_WORKSPACE, "workspace must be 256-byte aligned");
  if ((int64_t)Rs * hv.N > ((int64_t)1 << 40)) return fail(MCD_E_UNSUPPORTED, "batch too large");

  sv.R = a->R;
  sv.n_pairs = c.n_pairs;
  sv.n_solo = c.n_solo;
  sv.n_text = c.n_text;
  sv.Mg = 2 * c.n_pairs + c.n_solo;
  sv.Rs = Rs;
  sv.plan = a->plan;
  sv.hidden = a->hidden;
  sv.cfg_w = a->cfg_w;
  sv.temperature = a->temperature;
  sv.top_k = a->top_k;
  sv.top_p = a->top_p;
  sv.rng_key = a->rng_key;
  sv.step = a->step;
  sv.n_frames = a->n_frames;
  sv.grid_slot = a->grid_slot;
  sv.seed = a->seed;
  sv.tokens_out = a->tokens_out;
  sv.frame_grid = a->frame_grid;
  sv.modality_out = a->modality_out;
  sv.n_slots = a->n_slots;
  sv.F_max = a->F_max;
  sv.scores = a->scores;
  char *ws = static_cast<char *>(a->workspace);
  sv.status = reinterpret_cast<uint32_t *>(ws);
  sv.text_parts = hv.V_text > 0 ? mcd::text_parts_for(hv.V_text) : 0;
  sv.text_val = nullptr;
  sv.text_idx = nullptr;
  if (hv.V_text > 0) {
    const size_t parts = (size_t)sv.text_parts;
    if (ext) {
      sv.text_val = reinterpret_cast<float *>(ext->base);
      sv.text_idx = reinterpret_cast<int32_t *>(
          ext->base + round_up((size_t)c.n_text * parts * sizeof(float), 256));
    } else {
      sv.text_val = reinterpret_cast<float *>(ws + mcd::kStatusBytes);
      sv.text_idx = reinterpret_cast<int32_t *>(
          ws + mcd::kStatusBytes + round_up((size_t)a->R * parts * sizeof(float), 256));
    }
  }
  return MCD_OK;
}

bool make_delays(const int32_t *delays, int32_t K, mcd::Delays &d, int32_t &max_d) {
  std::memset(&d, 0, sizeof d);
  max_d = 0;
  if (!delays) return false;
  for (int32_t k = 0; k < K; ++k) {
    if (delays[k] < 0 || delays[k] > (1 << 24)) return false;
    d.d[k] = delays[k];
    if (delays[k] > max_d) max_d = delays[k];
  }
  return true;
}

}  // namespace

// ---- the allocation-free step's scratch ------------------------------------
// One array per GPU, in the library's code object, held until the process
// ends.  Host code never uses the array's name as an address (on the host it
// is a stand-in for the device symbol): it takes the device address once per
// device with hipGetSymbolAddress, with that device current, and passes that.
constexpr size_t kScratchBytes = MCD_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch array.
mcd_status scratch_address(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "current device");
  if (dev < 0 || dev >= kMaxDevices) return fail(MCD_E_UNSUPPORTED, "device %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "address of the scratch array");
    if (!p) return fail(MCD_E_HIP, "address of the scratch array is null");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MCD_OK;
}

}  // namespace

extern "C" {

const char *mcd_status_string(mcd_status s) {
  switch (s) {
    case MCD_OK: return "ok";
    case MCD_E_INVALID: return "invalid argument";
    case MCD_E_UNSUPPORTED: return "unsupported";
    case MCD_E_WORKSPACE: return "workspace";
    case MCD_E_HIP: return "hip error";
  }
  return "unknown status";
}

const char *mcd_last_error(void) { return g_last_error.c_str(); }

mcd_status mcd_head_create(const mcd_head_desc *d, mcd_head **out) {
  if (!d || !out) return fail(MCD_E_INVALID, "null argument");
  *out = nullptr;
  if (d->dtype != MCD_F32 && d->dtype != MCD_BF16) return fail(MCD_E_INVALID, "unknown dtype");
  if (d->K < 1 || d->K > MCD_MAX_K) return fail(MCD_E_UNSUPPORTED, "K=%d outside 1..%d", d->K, MCD_MAX_K);
  if (d->V < 1 || d->V > MCD_MAX_V) return fail(MCD_E_UNSUPPORTED, "V=%d outside 1..%d", d->V, MCD_MAX_V);
  if (d->H < 1) return fail(MCD_E_INVALID, "H=%d", d->H);
  if (d->dtype == MCD_BF16 && d->H % 64 != 0)
    return fail(MCD_E_UNSUPPORTED, "bf16 heads need H %% 64 == 0 (H=%d)", d->H);
  if (!d->W) return fail(MCD_E_INVALID, "W is null");
  const size_t al = d->dtype == MCD_BF16 ? 16 : 4;
  if (!aligned(d->W, al)) return fail(MCD_E_INVALID, "W misaligned");
  if (d->V_text < 0) return fail(MCD_E_INVALID, "V_text < 0");
  if (d->V_text > 0 && !d->W_text) return fail(MCD_E_INVALID, "W_text is null");
  if (d->V_text > 0 && !aligned(d->W_text, al)) return fail(MCD_E_INVALID, "W_text misaligned");
  if (d->V_text > (1 << 26)) return fail(MCD_E_UNSUPPORTED, "V_text too large");
  mcd::Delays del;
  int32_t max_d;
  if (!make_delays(d->delays, d->K, del, max_d)) return fail(MCD_E_INVALID, "bad delays");
  // stream blocks: V ids each, or V_stream[k] ids with V the largest
  mcd::StreamOffsets voff;
  voff.o[0] = 0;
  int32_t vmax = 0;
  for (int32_t k = 0; k < d->K; ++k) {
    const int32_t vk = d->V_stream ? d->V_stream[k] : d->V;
    if (vk < 1 || vk > MCD_MAX_V)
      return fail(MCD_E_UNSUPPORTED, "stream %d: %d ids, outside 1..%d", k, vk, MCD_MAX_V);
    voff.o[k + 1] = voff.o[k] + vk;
    vmax = vk > vmax ? vk : vmax;
  }
  if (vmax != d->V) return fail(MCD_E_INVALID, "V=%d is not the largest stream (%d)", d->V, vmax);
  if (d->T_text < 0 || d->T_text > d->V_text ||
      (d->T_text > 0 && d->T_text < d->V_text && d->T_text % mcd::kTextPartCols != 0))
    return fail(MCD_E_UNSUPPORTED, "T_text=%d: 0, V_text or a multiple of %d below V_text",
                d->T_text, mcd::kTextPartCols);
  mcd_head *h = new (std::nothrow) mcd_head;
  if (!h) return fail(MCD_E_INVALID, "out of host memory");
  h->hv.H = d->H;
  h->hv.K = d->K;
  h->hv.V = d->V;
  h->hv.N = voff.o[d->K];
  h->hv.pad_id = d->pad_id;
  h->hv.V_text = d->V_text;
  h->hv.dtype = d->dtype;
  h->hv.W = d->W;
  h->hv.bias = d->bias;
  h->hv.W_text = d->V_text > 0 ? d->W_text : nullptr;
  h->hv.delays = del;
  h->hv.voff = voff;
  h->hv.T_text = (d->T_text > 0 && d->T_text < d->V_text) ? d->T_text : d->V_text;
  h->max_delay = max_d;
  if (d->dtype == MCD_BF16 && d->V_text > 0) {
    hipError_t e = hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->fork, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->join, hipEventDisableTiming);
    if (e != hipSuccess) {
      mcd_head_destroy(h);
      return hip_fail(e, "side stream of the text projection");
    }
  }
  *out = h;
  return MCD_OK;
}

void mcd_head_destroy(mcd_head *h) {
  if (!h) return;
  if (h->fork) (void)hipEventDestroy(h->fork);
  if (h->join) (void)hipEventDestroy(h->join);
  if (h->side) (void)hipStreamDestroy(h->side);
  delete h;
}

size_t mcd_plan_words(int32_t R) { return (size_t)mcd::kPlanHeader + (size_t)(R > 0 ? R : 0); }

mcd_status mcd_batch_plan(const mcd_head *h, int32_t R, const int32_t *pair_map,
                          const uint8_t *row_kind, int32_t *plan, size_t plan_words,
                          mcd_batch_counts *counts) {
  if (!h || R < 0 || !plan || !counts) return fail(MCD_E_INVALID, "null argument or R < 0");
  if (R > 0 && (!pair_map || !row_kind)) return fail(MCD_E_INVALID, "null pair_map/row_kind");
  if (plan_words < mcd_plan_words(R)) return fail(MCD_E_INVALID, "plan buffer too small");
  int32_t np = 0, ns = 0, nt = 0;
  for (int32_t r = 0; r < R; ++r) {
    const int kind = row_kind[r];
    const int32_t p = pair_map[r];
    switch (kind) {
      case MCD_ROW_COND:
      case MCD_ROW_UNCOND: {
        if (p < 0 || p >= R || p == r) return fail(MCD_E_INVALID, "row %d: partner %d out of range", r, p);
        const int want = kind == MCD_ROW_COND ? MCD_ROW_UNCOND : MCD_ROW_COND;
        if (row_kind[p] != want) return fail(MCD_E_INVALID, "row %d: partner %d has the wrong kind", r, p);
        if (pair_map[p] != r) return fail(MCD_E_INVALID, "row %d: partner %d points to %d", r, p, pair_map[p]);
        if (kind == MCD_ROW_COND) ++np;
        break;
      }
      case MCD_ROW_SOLO:
      case MCD_ROW_TEXT:
        if (p != -1) return fail(MCD_E_INVALID, "row %d: solo/text row with a partner", r);
        if (kind == MCD_ROW_SOLO) ++ns;
        else ++nt;
        break;
      default:
        return fail(MCD_E_INVALID, "row %d: unknown kind %d", r, kind);
    }
  }
  if (nt > 0 && h->hv.V_text <= 0) return fail(MCD_E_INVALID, "text rows on a head without a text head");
  plan[mcd::kPlanMagicWord] = mcd::kPlanMagic;
  plan[mcd::kPlanR] = R;
  plan[mcd::kPlanPairs] = np;
  plan[mcd::kPlanSolo] = ns;
  plan[mcd::kPlanText] = nt;
  for (int i = 5; i < mcd::kPlanHeader; ++i) plan[i] = 0;
  int32_t *g = plan + mcd::kPlanHeader;
  int32_t n = 0;
  for (int32_t r = 0; r < R; ++r)
    if (row_kind[r] == MCD_ROW_COND) {
      g[n++] = r;
      g[n++] = pair_map[r];
    }
  for (int32_t r = 0; r < R; ++r)
    if (row_kind[r] == MCD_ROW_SOLO) g[n++] = r;
  for (int32_t r = 0; r < R; ++r)
    if (row_kind[r] == MCD_ROW_TEXT) g[n++] = r;
  counts->n_pairs = np;
  counts->n_solo = ns;
  counts->n_text = nt;
  return MCD_OK;
}

mcd_status mcd_plan_sampled_row(const int32_t *plan, int32_t s, int32_t *row, int32_t *companion) {
  if (!plan || !row || !companion) return fail(MCD_E_INVALID, "null argument");
  if (plan[mcd::kPlanMagicWord] != mcd::kPlanMagic) return fail(MCD_E_INVALID, "not a plan");
  const int32_t np = plan[mcd::kPlanPairs], ns = plan[mcd::kPlanSolo];
  if (s < 0 || s >= np + ns) return fail(MCD_E_INVALID, "sampled index %d out of range", s);
  const int32_t *g = plan + mcd::kPlanHeader;
  if (s < np) {
    *row = g[2 * s];
    *companion = g[2 * s + 1];
  } else {
    *row = g[2 * np + (s - np)];
    *companion = -1;
  }
  return MCD_OK;
}

size_t mcd_workspace_bytes(const mcd_head *h, int32_t R) {
  if (!h) return 0;
  return (size_t)mcd::kStatusBytes + partials_bytes(h, R);
}

namespace {

// K1 for one batch.  Audio and text rows together: one launch of both when
// the batch has that shape, else the audio projection on the caller's stream
// and the text projection on the head's second stream, both after everything
// already on the caller's stream, which waits for both.
hipError_t run_head_gemm(const mcd_head *h, const mcd::StepView &sv, hipStream_t stream) {
  if (h->hv.dtype != MCD_BF16 || sv.Mg == 0 || sv.n_text == 0)
    return mcd::launch_head_gemm(h->hv, sv, stream);
  bool fused = false;
  hipError_t e = mcd::launch_mixed_gemm(h->hv, sv, stream, &fused);
  if (fused || e != hipSuccess) return e;
  if (!h->side) return hipErrorInvalidHandle;   // created with every bf16 text head
  std::lock_guard<std::mutex> lock(h->side_mu);
  if ((e = hipEventRecord(h->fork, stream)) != hipSuccess) return e;
  if ((e = hipStreamWaitEvent(h->side, h->fork, 0)) != hipSuccess) return e;
  if ((e = mcd::launch_head_gemm_part(h->hv, sv, false, stream)) != hipSuccess) return e;
  if ((e = mcd::launch_head_gemm_part(h->hv, sv, true, h->side)) != hipSuccess) return e;
  if ((e = hipEventRecord(h->join, h->side)) != hipSuccess) return e;
  return hipStreamWaitEvent(stream, h->join, 0);
}

}  // namespace

mcd_status mcd_head_step(const mcd_head *h, const mcd_step_args *a, hipStream_t stream) {
  mcd::StepView sv;
  mcd_status s = make_step_view(h, a, true, sv);
  if (s != MCD_OK) return s;
  if (sv.R == 0) return MCD_OK;
  hipError_t e = run_head_gemm(h, sv, stream);
  if (e != hipSuccess) return hip_fail(e, "head GEMM launch");
  e = mcd::launch_sample(h->hv, sv, true, stream);
  if (e != hipSuccess) return hip_fail(e, "sample launch");
  return MCD_OK;
}

mcd_status mcd_head_step_noalloc(const mcd_head *h, const mcd_step_args *a, hipStream_t stream) {
  if (!h || !a) return fail(MCD_E_INVALID, "null head or args");
  const int64_t n_text = a->counts.n_text;
  const size_t need = partials_bytes(h, n_text);
  if (need > kScratchBytes)
    return fail(MCD_E_UNSUPPORTED,
                "text partials of %lld rows need %zu bytes; the library's scratch holds %zu",
                (long long)n_text, need, kScratchBytes);
  ExternalPartials ext{nullptr, kScratchBytes};
  if (need > 0) {
    void *base = nullptr;
    const mcd_status st = scratch_address(&base);
    if (st != MCD_OK) return st;
    ext.base = static_cast<char *>(base);
  }
  mcd::StepView sv;
  mcd_status s = make_step_view(h, a, true, sv, &ext);
  if (s != MCD_OK) return s;
  if (sv.R == 0) return MCD_OK;
  hipError_t e = run_head_gemm(h, sv, stream);
  if (e != hipSuccess) return hip_fail(e, "head GEMM launch");
  e = mcd::launch_sample(h->hv, sv, true, stream);
  if (e != hipSuccess) return hip_fail(e, "sample launch");
  return MCD_OK;
}

mcd_status mcd_head_logits(const mcd_head *h, const mcd_step_args *a, hipStream_t stream) {
  mcd::StepView sv;
  mcd_status s = make_step_view(h, a, true, sv);
  if (s != MCD_OK) return s;
  if (sv.R == 0) return MCD_OK;
  hipError_t e = run_head_gemm(h, sv, stream);
  return e == hipSuccess ? MCD_OK : hip_fail(e, "head GEMM launch");
}

mcd_status mcd_sample_step(const mcd_head *h, const mcd_step_args *a, hipStream_t stream) {
  mcd::StepView sv;
  mcd_status s = make_step_view(h, a, false, sv);
  if (s != MCD_OK) return s;
  if (sv.R == 0) return MCD_OK;
  hipError_t e = mcd::launch_sample(h->hv, sv, true, stream);
  if (e != hipSuccess) return hip_fail(e, "sample launch");
  return MCD_OK;
}

mcd_status mcd_phase_advance(const mcd_phase_desc *d, int32_t n, uint8_t *phase,
                             int32_t *count, const int32_t *token0, const uint8_t *modality,
                             int32_t *emit) {
  if (!d || n < 0 || d->n_bridge < 0 || d->drain_steps < 0 || (d->n_bridge > 0 && !d->bridge))
    return fail(MCD_E_INVALID, "bad phase description or n");
  if (n == 0) return MCD_OK;
  if (!phase || !count || !token0 || !modality || !emit) return fail(MCD_E_INVALID, "null array");
  const int32_t nb = d->n_bridge;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t c = count[i];
    int32_t ph = phase[i], nc = 0, out = -1;
    switch (ph) {
      case MCD_PHASE_TEXT:
        if (c != 0) return fail(MCD_E_INVALID, "request %d: count %d in the text phase", i, c);
        if (!modality[i]) {
          out = token0[i];
        } else if (nb == 0) {
          out = token0[i];
          ph = MCD_PHASE_AUDIO;
        } else {
          out = d->bridge[0];
          ph = nb > 1 ? MCD_PHASE_BRIDGE : MCD_PHASE_AUDIO;
          nc = nb > 1 ? 1 : 0;
        }
        break;
      case MCD_PHASE_BRIDGE:
        if (c < 1 || c >= nb) return fail(MCD_E_INVALID, "request %d: bridge count %d", i, c);
        out = d->bridge[c];
        if (c + 1 >= nb) {
          ph = MCD_PHASE_AUDIO;
        } else {
          nc = c + 1;
        }
        break;
      case MCD_PHASE_AUDIO:
        if (c < 0) return fail(MCD_E_INVALID, "request %d: audio count %d", i, c);
        if (token0[i] == d->audio_end) {
          ph = d->drain_steps > 0 ? MCD_PHASE_DRAIN : MCD_PHASE_TEXT;
        } else {
          nc = c + 1;
        }
        break;
      case MCD_PHASE_DRAIN:
        if (c < 0 || c >= d->drain_steps)
          return fail(MCD_E_INVALID, "request %d: drain count %d", i, c);
        if (c + 1 >= d->drain_steps) {
          ph = MCD_PHASE_TEXT;
        } else {
          nc = c + 1;
        }
        break;
      default:
        return fail(MCD_E_INVALID, "request %d: unknown phase %d", i, ph);
    }
    phase[i] = (uint8_t)ph;
    count[i] = nc;
    emit[i] = out;
  }
  return MCD_OK;
}

mcd_status mcd_next_input(const mcd_next_input_args *a, hipStream_t stream) {
  if (!a) return fail(MCD_E_INVALID, "null args");
  if (a->R < 0 || a->H < 1 || a->K < 1 || a->K > MCD_MAX_K || a->V < 1 || a->V_text < 0)
    return fail(MCD_E_INVALID, "bad sizes (R=%d H=%d K=%d V=%d V_text=%d)", a->R, a->H, a->K,
                a->V, a->V_text);
  if (a->dtype != MCD_F32 && a->dtype != MCD_BF16) return fail(MCD_E_INVALID, "bad dtype");
  if (a->pad_id >= 0 && a->pad_id < a->V)
    return fail(MCD_E_INVALID, "pad_id %d is a token id of [0, %d)", a->pad_id, a->V);
  if ((int64_t)a->K * (a->V + 1) * a->H > ((int64_t)1 << 40))
    return fail(MCD_E_INVALID, "table too large");
  if (a->R == 0) return MCD_OK;
  if (!a->E || !a->out || !a->tokens || !a->row_kind) return fail(MCD_E_INVALID, "null buffer");
  if ((a->V_text > 0) != (a->E_text != nullptr))
    return fail(MCD_E_INVALID, "V_text and E_text disagree");
  if (!aligned(a->E, 16) || !aligned(a->out, 16) || (a->E_text && !aligned(a->E_text, 16)))
    return fail(MCD_E_INVALID, "E, E_text and out must be 16-byte aligned");
  if (a->workspace && !aligned(a->workspace, 256))
    return fail(MCD_E_INVALID, "workspace must be 256-byte aligned");
  mcd::EmbedView ev;
  ev.R = a->R;
  ev.H = a->H;
  ev.K = a->K;
  ev.V = a->V;
  ev.pad_id = a->pad_id;
  ev.V_text = a->V_text;
  ev.E = a->E;
  ev.E_text = a->E_text;
  ev.row_kind = a->row_kind;
  ev.tokens = a->tokens;
  ev.out = a->out;
  ev.status = reinterpret_cast<uint32_t *>(a->workspace);
  hipError_t e = mcd::launch_next_input(ev, a->dtype == MCD_BF16, stream);
  return e == hipSuccess ? MCD_OK : hip_fail(e, "next-input launch");
}

mcd_status mcd_deinterleave(const int32_t *streams, int32_t n_req, int32_t T, int32_t K,
                            const int32_t *delays, int32_t *grid, hipStream_t stream) {
  if (n_req < 0 || T < 0 || K < 1 || K > MCD_MAX_K) return fail(MCD_E_INVALID, "bad sizes");
  mcd::Delays d;
  int32_t md;
  if (!make_delays(delays, K, d, md)) return fail(MCD_E_INVALID, "bad delays");
  if (T < md) return fail(MCD_E_INVALID, "T=%d shorter than the largest delay %d", T, md);
  const int32_t F = T - md;
  if ((int64_t)n_req * K * F == 0) return MCD_OK;
  if (!streams || !grid) return fail(MCD_E_INVALID, "null buffer");
  hipError_t e = mcd::launch_deinterleave(streams, n_req, T, K, d, F, grid, stream);
  return e == hipSuccess ? MCD_OK : hip_fail(e, "deinterleave launch");
}

mcd_status mcd_interleave(const int32_t *grid, int32_t n_req, int32_t F, int32_t K,
                          const int32_t *delays, int32_t pad_id, int32_t *streams,
                          hipStream_t stream) {
  if (n_req < 0 || F < 0 || K < 1 || K > MCD_MAX_K) return fail(MCD_E_INVALID, "bad sizes");
  mcd::Delays d;
  int32_t md;
  if (!make_delays(delays, K, d, md)) return fail(MCD_E_INVALID, "bad delays");
  const int32_t T = F + md;
  if ((int64_t)n_req * K * T == 0) return MCD_OK;
  if (!streams || (!grid && F > 0)) return fail(MCD_E_INVALID, "null buffer");
  hipError_t e = mcd::launch_interleave(grid, n_req, F, K, d, T, pad_id, streams, stream);
  return e == hipSuccess ? MCD_OK : hip_fail(e, "interleave launch");
}

mcd_status mcd_read_device_status(void *workspace, uint32_t *code, hipStream_t stream) {
  if (!workspace || !code) return fail(MCD_E_INVALID, "null argument");
  hipError_t e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "stream synchronize");
  uint32_t v = 0;
  e = hipMemcpy(&v, workspace, sizeof v, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "status read");
  *code = v;
  if (v) {
    const uint32_t z = 0;
    e = hipMemcpy(workspace, &z, sizeof z, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "status clear");
  }
  return MCD_OK;
}

}  // extern "C"

mcd_status mcd::record_error(mcd_status s, const char *msg) { return fail(s, "%s", msg); }
