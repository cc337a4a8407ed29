"""Thin ctypes binding of libmcd (include/mcd.h).

Every function named ``mcd_*`` here marshals its arguments to the C function of
the same name; all computation happens in the library's HIP kernels.  PyTorch
supplies device memory and the stream.  ``Head`` is a small convenience wrapper
that keeps the borrowed weight tensors alive next to the handle.

Importing this module loads ``libmcd.so`` and raises if it has not been built
(``python -m paper_2607_02119_amd.build``); there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # loads the HIP runtime libmcd binds to (same soname, one runtime per process)

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmcd.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2607_02119_amd.build`")
_lib = ctypes.CDLL(_LIB_PATH)

MCD_OK, MCD_E_INVALID, MCD_E_UNSUPPORTED, MCD_E_WORKSPACE, MCD_E_HIP = range(5)
MCD_F32, MCD_BF16 = 0, 1
MCD_ROW_COND, MCD_ROW_UNCOND, MCD_ROW_SOLO, MCD_ROW_TEXT = 0, 1, 2, 3
MCD_DEV_BAD_PARAM, MCD_DEV_GRID_RANGE, MCD_DEV_BAD_PLAN, MCD_DEV_BAD_TOKEN = 1, 2, 4, 8
MCD_MAX_K, MCD_MAX_V = 32, 4096

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32


class mcd_head_desc(ctypes.Structure):
    _fields_ = [("H", _i32), ("K", _i32), ("V", _i32), ("pad_id", _i32),
                ("delays", _vp), ("dtype", ctypes.c_int), ("W", _vp), ("bias", _vp),
                ("V_text", _i32), ("W_text", _vp), ("V_stream", _vp), ("T_text", _i32)]


class mcd_batch_counts(ctypes.Structure):
    _fields_ = [("n_pairs", _i32), ("n_solo", _i32), ("n_text", _i32)]


class mcd_step_args(ctypes.Structure):
    _fields_ = [("R", _i32), ("counts", mcd_batch_counts), ("plan", _vp), ("hidden", _vp),
                ("cfg_w", _vp), ("temperature", _vp), ("top_k", _vp), ("top_p", _vp),
                ("rng_key", _vp), ("step", _vp), ("n_frames", _vp), ("grid_slot", _vp),
                ("seed", ctypes.c_uint64), ("tokens_out", _vp), ("frame_grid", _vp),
                ("modality_out", _vp), ("n_slots", _i32), ("F_max", _i32), ("scores", _vp), ("workspace", _vp),
                ("workspace_bytes", ctypes.c_size_t)]


class mcd_next_input_args(ctypes.Structure):
    _fields_ = [("R", _i32), ("H", _i32), ("K", _i32), ("V", _i32), ("pad_id", _i32),
                ("dtype", ctypes.c_int), ("E", _vp), ("V_text", _i32), ("E_text", _vp),
                ("row_kind", _vp), ("tokens", _vp), ("out", _vp), ("workspace", _vp)]


class mcd_phase_desc(ctypes.Structure):
    _fields_ = [("n_bridge", _i32), ("bridge", _vp), ("audio_end", _i32), ("drain_steps", _i32)]


class mcd_sched_desc(ctypes.Structure):
    _fields_ = [("max_rows", _i32), ("token_budget", _i32), ("null_prompt_len", _i32),
                ("drain_steps", _i32), ("max_requests", _i32)]


class mcd_sched_request(ctypes.Structure):
    _fields_ = [("cfg_w", ctypes.c_float), ("prompt_len", _i32), ("text_len", _i32),
                ("n_frames", _i32)]


class mcd_sched_batch(ctypes.Structure):
    _fields_ = [("n_rows", _i32), ("row_req", _vp), ("row_member", _vp), ("row_slot", _vp),
                ("row_tokens", _vp), ("row_context", _vp), ("R", _i32), ("head_row", _vp),
                ("pair_map", _vp), ("row_kind", _vp), ("cfg_w", _vp), ("step", _vp),
                ("n_frames", _vp), ("grid_slot", _vp)]


def _sig(name, res, *args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


_mcd_head_create = _sig("mcd_head_create", ctypes.c_int, ctypes.POINTER(mcd_head_desc),
                        ctypes.POINTER(_vp))
_mcd_head_destroy = _sig("mcd_head_destroy", None, _vp)
_mcd_sched_create = _sig("mcd_sched_create", ctypes.c_int, ctypes.POINTER(mcd_sched_desc),
                         ctypes.POINTER(_vp))
_mcd_sched_destroy = _sig("mcd_sched_destroy", None, _vp)
_mcd_sched_submit = _sig("mcd_sched_submit", ctypes.c_int, _vp,
                         ctypes.POINTER(mcd_sched_request), ctypes.POINTER(_i32))
_mcd_sched_plan = _sig("mcd_sched_plan", ctypes.c_int, _vp, ctypes.POINTER(mcd_sched_batch))
_mcd_sched_commit = _sig("mcd_sched_commit", ctypes.c_int, _vp, _vp, _i32, ctypes.POINTER(_i32))
_mcd_sched_counts = _sig("mcd_sched_counts", ctypes.c_int, _vp, ctypes.POINTER(_i32),
                         ctypes.POINTER(_i32))
_mcd_plan_words = _sig("mcd_plan_words", ctypes.c_size_t, _i32)
_mcd_batch_plan = _sig("mcd_batch_plan", ctypes.c_int, _vp, _i32, _vp, _vp, _vp, ctypes.c_size_t,
                       ctypes.POINTER(mcd_batch_counts))
_mcd_plan_sampled_row = _sig("mcd_plan_sampled_row", ctypes.c_int, _vp, _i32,
                             ctypes.POINTER(_i32), ctypes.POINTER(_i32))
_mcd_workspace_bytes = _sig("mcd_workspace_bytes", ctypes.c_size_t, _vp, _i32)
_mcd_head_step = _sig("mcd_head_step", ctypes.c_int, _vp, ctypes.POINTER(mcd_step_args), _vp)
_mcd_sample_step = _sig("mcd_sample_step", ctypes.c_int, _vp, ctypes.POINTER(mcd_step_args), _vp)
_mcd_head_logits = _sig("mcd_head_logits", ctypes.c_int, _vp, ctypes.POINTER(mcd_step_args), _vp)
_mcd_head_step_noalloc = _sig("mcd_head_step_noalloc", ctypes.c_int, _vp,
                              ctypes.POINTER(mcd_step_args), _vp)
_mcd_deinterleave = _sig("mcd_deinterleave", ctypes.c_int, _vp, _i32, _i32, _i32, _vp, _vp, _vp)
_mcd_interleave = _sig("mcd_interleave", ctypes.c_int, _vp, _i32, _i32, _i32, _vp, _i32, _vp, _vp)
_mcd_next_input = _sig("mcd_next_input", ctypes.c_int, ctypes.POINTER(mcd_next_input_args), _vp)
_mcd_phase_advance = _sig("mcd_phase_advance", ctypes.c_int, ctypes.POINTER(mcd_phase_desc), _i32,
                          _vp, _vp, _vp, _vp, _vp)
_mcd_read_device_status = _sig("mcd_read_device_status", ctypes.c_int, _vp,
                               ctypes.POINTER(ctypes.c_uint32), _vp)
_mcd_status_string = _sig("mcd_status_string", ctypes.c_char_p, ctypes.c_int)
_mcd_last_error = _sig("mcd_last_error", ctypes.c_char_p)

EXPORTED = ["mcd_head_create", "mcd_head_destroy", "mcd_plan_words", "mcd_batch_plan",
            "mcd_plan_sampled_row", "mcd_workspace_bytes", "mcd_head_step", "mcd_head_logits",
            "mcd_head_step_noalloc",
            "mcd_sample_step",
            "mcd_deinterleave", "mcd_interleave", "mcd_phase_advance", "mcd_next_input",
            "mcd_read_device_status",
            "mcd_sched_create", "mcd_sched_destroy", "mcd_sched_submit", "mcd_sched_plan",
            "mcd_sched_commit", "mcd_sched_counts",
            "mcd_status_string", "mcd_last_error"]


class McdError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        msg = _mcd_last_error().decode(errors="replace")
        super().__init__(f"{where}: {mcd_status_string(code)} ({msg})")


def _check(code, where):
    if code != MCD_OK:
        raise McdError(code, where)


def _ptr(t):
    """Device (or host numpy) pointer of an optional tensor / array."""
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        return t.data_ptr()
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return int(t)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if isinstance(stream, torch.cuda.Stream) else int(stream)


# ---------------------------------------------------------------------------
# C functions, one to one

def mcd_status_string(code):
    return _mcd_status_string(code).decode()


def mcd_last_error():
    return _mcd_last_error().decode(errors="replace")


def mcd_head_create(H, K, V, pad_id, delays, dtype, W, bias=None, V_text=0, W_text=None,
                    V_stream=None, T_text=0):
    d = np.ascontiguousarray(delays, dtype=np.int32)
    vs = None if V_stream is None else np.ascontiguousarray(V_stream, dtype=np.int32)
    desc = mcd_head_desc(H, K, V, pad_id, d.ctypes.data, dtype, _ptr(W), _ptr(bias), V_text,
                         _ptr(W_text), _ptr(vs), int(T_text))
    h = _vp()
    _check(_mcd_head_create(ctypes.byref(desc), ctypes.byref(h)), "mcd_head_create")
    return h


def mcd_head_destroy(h):
    _mcd_head_destroy(h)


def mcd_plan_words(R):
    return int(_mcd_plan_words(R))


def mcd_batch_plan(h, pair_map, row_kind):
    """Host plan of a batch -> (plan int32 numpy array, mcd_batch_counts)."""
    pm = np.ascontiguousarray(pair_map, dtype=np.int32)
    rk = np.ascontiguousarray(row_kind, dtype=np.uint8)
    R = pm.shape[0]
    plan = np.zeros(mcd_plan_words(R), dtype=np.int32)
    counts = mcd_batch_counts()
    _check(_mcd_batch_plan(h, R, pm.ctypes.data, rk.ctypes.data, plan.ctypes.data, plan.shape[0],
                           ctypes.byref(counts)), "mcd_batch_plan")
    return plan, counts


def mcd_plan_sampled_row(plan, s):
    row, comp = _i32(), _i32()
    _check(_mcd_plan_sampled_row(plan.ctypes.data, s, ctypes.byref(row), ctypes.byref(comp)),
           "mcd_plan_sampled_row")
    return row.value, comp.value


def mcd_workspace_bytes(h, R):
    return int(_mcd_workspace_bytes(h, R))


def _step_args(R, counts, plan, hidden, cfg_w, temperature, top_k, top_p, rng_key, step,
               n_frames, grid_slot, seed, tokens_out, frame_grid, n_slots, F_max, scores,
               workspace, modality_out=None):
    return mcd_step_args(R, counts, _ptr(plan), _ptr(hidden), _ptr(cfg_w), _ptr(temperature),
                         _ptr(top_k), _ptr(top_p), _ptr(rng_key), _ptr(step), _ptr(n_frames),
                         _ptr(grid_slot), seed, _ptr(tokens_out), _ptr(frame_grid),
                         _ptr(modality_out), n_slots, F_max, _ptr(scores), _ptr(workspace),
                         0 if workspace is None else workspace.numel() * workspace.element_size())


def mcd_head_step(h, stream=None, **kw):
    a = _step_args(**kw)
    _check(_mcd_head_step(h, ctypes.byref(a), _stream(stream)), "mcd_head_step")


def mcd_head_step_noalloc(h, stream=None, **kw):
    """mcd_head_step with the text-head partials in the library's per-GPU
    array; `workspace` only needs the 256-byte status word region."""
    a = _step_args(**kw)
    _check(_mcd_head_step_noalloc(h, ctypes.byref(a), _stream(stream)), "mcd_head_step_noalloc")


MCD_NOALLOC_SCRATCH_BYTES = 8 << 20


def mcd_head_logits(h, stream=None, **kw):
    a = _step_args(**kw)
    _check(_mcd_head_logits(h, ctypes.byref(a), _stream(stream)), "mcd_head_logits")


def mcd_sample_step(h, stream=None, **kw):
    a = _step_args(**kw)
    _check(_mcd_sample_step(h, ctypes.byref(a), _stream(stream)), "mcd_sample_step")


def mcd_deinterleave(streams, delays, grid, stream=None):
    """streams: int32 [n_req][T][K] -> grid int32 [n_req][K][T - max d] (device tensors)."""
    n_req, T, K = streams.shape
    d = np.ascontiguousarray(delays, dtype=np.int32)
    _check(_mcd_deinterleave(_ptr(streams), n_req, T, K, d.ctypes.data, _ptr(grid),
                             _stream(stream)), "mcd_deinterleave")


def mcd_interleave(grid, delays, pad_id, streams, stream=None):
    """grid: int32 [n_req][K][F] -> streams int32 [n_req][F + max d][K] (device tensors)."""
    n_req, K, F = grid.shape
    d = np.ascontiguousarray(delays, dtype=np.int32)
    _check(_mcd_interleave(_ptr(grid), n_req, F, K, d.ctypes.data, pad_id, _ptr(streams),
                           _stream(stream)), "mcd_interleave")


def mcd_next_input(E, tokens, row_kind, pad_id, out, E_text=None, workspace=None, stream=None):
    """Next-step input of every row: E [K][V + 1][H] (bf16 or fp32, device),
    tokens int32 [R][K], row_kind uint8 [R], out [R][H] of E's type (device)."""
    K, V1, H = E.shape
    R = tokens.shape[0]
    dtype = {torch.bfloat16: MCD_BF16, torch.float32: MCD_F32}[E.dtype]
    a = mcd_next_input_args(R, H, K, V1 - 1, int(pad_id), dtype, _ptr(E),
                            0 if E_text is None else E_text.shape[0], _ptr(E_text),
                            _ptr(row_kind), _ptr(tokens), _ptr(out), _ptr(workspace))
    _check(_mcd_next_input(ctypes.byref(a), _stream(stream)), "mcd_next_input")


MCD_PHASE_TEXT, MCD_PHASE_BRIDGE, MCD_PHASE_AUDIO, MCD_PHASE_DRAIN = 0, 1, 2, 3


def mcd_phase_advance(bridge, audio_end, drain_steps, phase, count, token0, modality):
    """One step of the requests' phases (host arrays, updated in place):
    phase uint8 [n], count int32 [n], token0 int32 [n], modality uint8 [n].
    Returns emit int32 [n]."""
    br = np.ascontiguousarray(bridge, dtype=np.int32)
    d = mcd_phase_desc(br.shape[0], br.ctypes.data if br.shape[0] else None, int(audio_end),
                       int(drain_steps))
    for a, dt in ((phase, np.uint8), (count, np.int32)):
        assert a.dtype == dt and a.flags.c_contiguous
    token0 = np.ascontiguousarray(token0, dtype=np.int32)
    modality = np.ascontiguousarray(modality, dtype=np.uint8)
    emit = np.empty(phase.shape[0], dtype=np.int32)
    _check(_mcd_phase_advance(ctypes.byref(d), phase.shape[0], phase.ctypes.data,
                              count.ctypes.data, token0.ctypes.data, modality.ctypes.data,
                              emit.ctypes.data), "mcd_phase_advance")
    return emit


class Scheduler:
    """Paired co-scheduling of CFG requests (host only): the C scheduler of
    libmcd behind plan() / commit()."""

    _I32 = ("row_req", "row_slot", "row_tokens", "row_context", "head_row", "pair_map", "step",
            "n_frames", "grid_slot")

    def __init__(self, max_rows, token_budget, null_prompt_len, drain_steps, max_requests=4096):
        d = mcd_sched_desc(int(max_rows), int(token_budget), int(null_prompt_len),
                           int(drain_steps), int(max_requests))
        h = _vp()
        _check(_mcd_sched_create(ctypes.byref(d), ctypes.byref(h)), "mcd_sched_create")
        self.handle = h.value
        self.max_requests = int(max_requests)
        self._destroy = _mcd_sched_destroy

    def __del__(self):
        h = getattr(self, "handle", None)
        destroy = getattr(self, "_destroy", None)
        if h is not None and destroy is not None:
            destroy(h)
            self.handle = None

    def submit(self, cfg_w, prompt_len, text_len, n_frames):
        q = mcd_sched_request(float(cfg_w), int(prompt_len), int(text_len), int(n_frames))
        rid = _i32()
        _check(_mcd_sched_submit(self.handle, ctypes.byref(q), ctypes.byref(rid)),
               "mcd_sched_submit")
        return rid.value

    def plan(self):
        """The next step as a dict of numpy copies (backbone rows and head rows)."""
        b = mcd_sched_batch()
        _check(_mcd_sched_plan(self.handle, ctypes.byref(b)), "mcd_sched_plan")

        def arr(name, n, ct, dt):
            p = getattr(b, name)
            if n == 0 or not p:
                return np.zeros(0, dtype=dt)
            return np.ctypeslib.as_array(ctypes.cast(p, ctypes.POINTER(ct)), (n,)).astype(dt)

        out = {"n_rows": b.n_rows, "R": b.R}
        for name in self._I32:
            n = b.R if name in ("head_row", "pair_map", "step", "n_frames", "grid_slot") else b.n_rows
            out[name] = arr(name, n, ctypes.c_int32, np.int32)
        out["row_member"] = arr("row_member", b.n_rows, ctypes.c_uint8, np.uint8)
        out["row_kind"] = arr("row_kind", b.R, ctypes.c_uint8, np.uint8)
        out["cfg_w"] = arr("cfg_w", b.R, ctypes.c_float, np.float32)
        return out

    def commit(self):
        """Apply the planned step; returns the ids of the requests it finished."""
        fin = np.empty(self.max_requests, dtype=np.int32)
        n = _i32()
        _check(_mcd_sched_commit(self.handle, fin.ctypes.data, fin.shape[0], ctypes.byref(n)),
               "mcd_sched_commit")
        return fin[:n.value].copy()

    def counts(self):
        w, r = _i32(), _i32()
        _check(_mcd_sched_counts(self.handle, ctypes.byref(w), ctypes.byref(r)),
               "mcd_sched_counts")
        return w.value, r.value


def mcd_read_device_status(workspace, stream=None):
    code = ctypes.c_uint32()
    _check(_mcd_read_device_status(_ptr(workspace), ctypes.byref(code), _stream(stream)),
           "mcd_read_device_status")
    return code.value


# ---------------------------------------------------------------------------
# Convenience wrapper

class Head:
    """Handle plus the device tensors it borrows."""

    def __init__(self, W, delays, pad_id, bias=None, W_text=None, V_stream=None, T_text=0):
        """W: [K][V][H], or [N][H] with V_stream (the ids of each stream)."""
        assert W.is_cuda and W.is_contiguous()
        if V_stream is None:
            assert W.dim() == 3
            K, V, H = W.shape
        else:
            V_stream = np.ascontiguousarray(V_stream, dtype=np.int32)
            assert W.dim() == 2 and W.shape[0] == int(V_stream.sum())
            K, V, H = V_stream.shape[0], int(V_stream.max()), W.shape[1]
        dtype = {torch.bfloat16: MCD_BF16, torch.float32: MCD_F32}[W.dtype]
        self.W, self.bias, self.W_text, self.V_stream = W, bias, W_text, V_stream
        self.H, self.K, self.V, self.pad_id = H, K, V, int(pad_id)
        self.delays = np.ascontiguousarray(delays, dtype=np.int32)
        self.V_text = 0 if W_text is None else W_text.shape[0]
        self.handle = mcd_head_create(H, K, V, self.pad_id, self.delays, dtype, W, bias,
                                      self.V_text, W_text, V_stream, T_text)
        # the library's own entry, held here: at interpreter exit the module's
        # globals may already be gone when this object is collected
        self._destroy = _mcd_head_destroy

    def __del__(self):
        h = getattr(self, "handle", None)
        destroy = getattr(self, "_destroy", None)
        if h is not None and destroy is not None:
            destroy(h)
            self.handle = None

    def plan(self, pair_map, row_kind, device="cuda"):
        plan, counts = mcd_batch_plan(self.handle, pair_map, row_kind)
        return Plan(plan, counts, torch.from_numpy(plan).to(device))

    def workspace(self, R, device="cuda"):
        return torch.zeros(max(mcd_workspace_bytes(self.handle, R), 256), dtype=torch.uint8,
                           device=device)


class Plan:
    def __init__(self, host, counts, dev):
        self.host, self.counts, self.dev = host, counts, dev
        self.R = int(host[1])
        self.n_pairs, self.n_solo, self.n_text = counts.n_pairs, counts.n_solo, counts.n_text
        self.Rs = self.n_pairs + self.n_solo

    def sampled_rows(self):
        """(row, companion) of each sampled index."""
        return [mcd_plan_sampled_row(self.host, s) for s in range(self.Rs)]
