"""Plain CPU oracle for the multi-codebook audio decode head.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this package.  The product path
(``paper_2607_02119_amd``) never imports, links or runs it, and the two share
no code: the only module both sides use is the seeded input generator
``paper_2607_02119_amd.inputs``, which holds none of the method's arithmetic.

The arithmetic lives in ``mcd_oracle.c`` (single-threaded, fp64, plain loops);
this module only builds it with gcc and marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mcd_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

ROW_COND, ROW_UNCOND, ROW_SOLO, ROW_TEXT = 0, 1, 2, 3
F32, BF16 = 0, 1
FLAG_GAP_SMALL, FLAG_TOPP_EDGE, FLAG_TOPK_EDGE, FLAG_PAD = 1, 2, 4, 8
ERRORS = {0: "ok", 1: "pair_map/row_kind inconsistent", 2: "parameter out of range",
          3: "bad shape"}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C11, no fast-math, no contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-Wextra", "-Werror", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        u64p = ctypes.POINTER(ctypes.c_uint64)
        L.orc_philox4x64_10.argtypes = [u64p, u64p, u64p]
        L.orc_philox4x64_10.restype = None
        u32p = ctypes.POINTER(ctypes.c_uint32)
        L.orc_philox4x32_10.argtypes = [u32p, u32p, u32p]
        L.orc_philox4x32_10.restype = None
        L.orc_uniform.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64,
                                  ctypes.c_int32, ctypes.c_int32]
        L.orc_uniform.restype = ctypes.c_double
        L.orc_gumbel.argtypes = L.orc_uniform.argtypes
        L.orc_gumbel.restype = ctypes.c_double
        L.orc_logits_row.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_void_p]
        L.orc_logits_row.restype = None
        L.orc_sample_vector.argtypes = [
            ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
            ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_double,
            ctypes.c_double, ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.orc_sample_vector.restype = ctypes.c_int32
        L.orc_head_step.argtypes = [ctypes.POINTER(StepArgs)]
        L.orc_head_step.restype = ctypes.c_int32
        L.orc_sample_rows.argtypes = [ctypes.POINTER(StepArgs), ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p]
        L.orc_sample_rows.restype = ctypes.c_int32
        L.orc_deinterleave.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_void_p, ctypes.c_void_p]
        L.orc_deinterleave.restype = ctypes.c_int32
        L.orc_interleave.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
        L.orc_interleave.restype = ctypes.c_int32
        L.orc_next_input.argtypes = [ctypes.c_int32] * 6 + [ctypes.c_void_p, ctypes.c_int32] + \
            [ctypes.c_void_p] * 4
        L.orc_next_input.restype = ctypes.c_int32
        _lib = L
    return _lib


class StepArgs(ctypes.Structure):
    _fields_ = [
        ("H", ctypes.c_int32), ("K", ctypes.c_int32), ("V", ctypes.c_int32),
        ("pad_id", ctypes.c_int32),
        ("delays", ctypes.c_void_p), ("dtype", ctypes.c_int32),
        ("W", ctypes.c_void_p), ("bias", ctypes.c_void_p),
        ("V_text", ctypes.c_int32), ("W_text", ctypes.c_void_p),
        ("V_stream", ctypes.c_void_p), ("T_text", ctypes.c_int32),
        ("R", ctypes.c_int32), ("hidden", ctypes.c_void_p),
        ("pair_map", ctypes.c_void_p), ("row_kind", ctypes.c_void_p),
        ("cfg_w", ctypes.c_void_p), ("temperature", ctypes.c_void_p),
        ("top_k", ctypes.c_void_p), ("top_p", ctypes.c_void_p),
        ("rng_key", ctypes.c_void_p), ("step", ctypes.c_void_p),
        ("n_frames", ctypes.c_void_p), ("grid_slot", ctypes.c_void_p),
        ("seed", ctypes.c_uint64), ("n_slots", ctypes.c_int32), ("F_max", ctypes.c_int32),
        ("gap_tol", ctypes.c_double), ("topk_tol", ctypes.c_double),
        ("topp_tol", ctypes.c_double),
        ("tokens_out", ctypes.c_void_p), ("frame_grid", ctypes.c_void_p),
        ("modality", ctypes.c_void_p), ("modality_gap", ctypes.c_void_p),
        ("scores", ctypes.c_void_p), ("gap", ctypes.c_void_p), ("flags", ctypes.c_void_p),
    ]


def _ptr(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


# --------------------------------------------------------------------------
# Scalar building blocks

def philox4x64_10(ctr, key):
    """Philox4x64-10 block: four 64-bit counter words, two key words -> four words."""
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    u64p = ctypes.POINTER(ctypes.c_uint64)
    lib().orc_philox4x64_10(c.ctypes.data_as(u64p), k.ctypes.data_as(u64p),
                            out.ctypes.data_as(u64p))
    return out


def philox4x32_10(ctr, key):
    """Philox4x32-10 block: four 32-bit counter words, two key words -> four words."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    u32p = ctypes.POINTER(ctypes.c_uint32)
    lib().orc_philox4x32_10(c.ctypes.data_as(u32p), k.ctypes.data_as(u32p),
                            out.ctypes.data_as(u32p))
    return out


def uniform(seed, rng_key, t, k, v):
    return lib().orc_uniform(seed, rng_key, t, k, v)


def gumbel(seed, rng_key, t, k, v):
    return lib().orc_gumbel(seed, rng_key, t, k, v)


def logits_row(x, W, bias=None):
    """fp64 logits of one row.  x: [H] float32 or uint16 (bf16 bits); W: [N][H] same type."""
    dtype = BF16 if x.dtype == np.uint16 else F32
    x = np.ascontiguousarray(x)
    W = np.ascontiguousarray(W)
    assert W.dtype == x.dtype and W.shape[1] == x.shape[0]
    b = _c(bias, np.float32)
    out = np.zeros(W.shape[0], dtype=np.float64)
    lib().orc_logits_row(x.ctypes.data, dtype, W.ctypes.data, _ptr(b), x.shape[0], W.shape[0],
                         out.ctypes.data)
    return out


def sample_vector(s, greedy=False, top_k=0, top_p=1.0, seed=0, rng_key=0, t=0, k=0,
                  gap_tol=1e-3, topk_tol=0.0, topp_tol=0.0, want_kept=False):
    """Select + sample one vector of fp64 scores -> (token, gap, flags[, kept mask])."""
    s = np.ascontiguousarray(s, dtype=np.float64)
    V = s.shape[0]
    gap = ctypes.c_double()
    flags = ctypes.c_uint32()
    kept = np.zeros(V, dtype=np.uint8) if want_kept else None
    tok = lib().orc_sample_vector(s.ctypes.data, V, int(bool(greedy)), int(top_k), float(top_p),
                                  int(seed), int(rng_key), int(t), int(k), gap_tol, topk_tol,
                                  topp_tol, ctypes.addressof(gap), ctypes.addressof(flags),
                                  _ptr(kept))
    if want_kept:
        return tok, gap.value, flags.value, kept.astype(bool)
    return tok, gap.value, flags.value


def deinterleave(streams, delays):
    streams = np.ascontiguousarray(streams, dtype=np.int32)
    delays = np.ascontiguousarray(delays, dtype=np.int32)
    T, K = streams.shape
    md = int(delays.max()) if K else 0
    grid = np.zeros((K, T - md), dtype=np.int32)
    rc = lib().orc_deinterleave(streams.ctypes.data, T, K, delays.ctypes.data, grid.ctypes.data)
    if rc:
        raise ValueError(ERRORS.get(rc, rc))
    return grid


def interleave(grid, delays, pad_id):
    grid = np.ascontiguousarray(grid, dtype=np.int32)
    delays = np.ascontiguousarray(delays, dtype=np.int32)
    K, F = grid.shape
    md = int(delays.max()) if K else 0
    streams = np.zeros((F + md, K), dtype=np.int32)
    rc = lib().orc_interleave(grid.ctypes.data, F, K, delays.ctypes.data, int(pad_id),
                              streams.ctypes.data)
    if rc:
        raise ValueError(ERRORS.get(rc, rc))
    return streams


# --------------------------------------------------------------------------
# Whole step

def _step_struct(head, batch, seed, n_slots, F_max, tol, keep):
    """Fill a StepArgs; `keep` collects the arrays so they outlive the call."""
    a = StepArgs()
    H, K, V = head["H"], head["K"], head["V"]
    dtype = BF16 if head["W"].dtype == np.uint16 else F32
    vs = head.get("V_stream")
    vs = None if vs is None else _c(vs, np.int32)
    N = K * V if vs is None else int(vs.sum())
    W = np.ascontiguousarray(head["W"]).reshape(N, H)
    delays = _c(head["delays"], np.int32)
    bias = _c(head.get("bias"), np.float32)
    Wt = head.get("W_text")
    Wt = None if Wt is None else np.ascontiguousarray(Wt)
    R = batch["hidden"].shape[0]
    hidden = np.ascontiguousarray(batch["hidden"])
    assert hidden.dtype == W.dtype
    cols = dict(pair_map=np.int32, row_kind=np.uint8, cfg_w=np.float32, temperature=np.float32,
                top_k=np.int32, top_p=np.float32, step=np.int32, n_frames=np.int32,
                grid_slot=np.int32)
    arrs = {name: _c(batch[name], dt) for name, dt in cols.items()}
    rk = batch.get("rng_key")
    arrs["rng_key"] = _c(rk, np.uint64)
    keep += [W, delays, bias, Wt, hidden, vs] + list(arrs.values())
    a.V_stream = _ptr(vs)
    a.T_text = int(head.get("T_text") or 0)
    a.H, a.K, a.V, a.pad_id = H, K, V, head["pad_id"]
    a.delays, a.dtype, a.W, a.bias = delays.ctypes.data, dtype, W.ctypes.data, _ptr(bias)
    a.V_text = 0 if Wt is None else Wt.shape[0]
    a.W_text = _ptr(Wt)
    a.R, a.hidden = R, hidden.ctypes.data
    for name, arr in arrs.items():
        setattr(a, name, _ptr(arr))
    a.seed, a.n_slots, a.F_max = int(seed), int(n_slots), int(F_max)
    a.gap_tol, a.topk_tol, a.topp_tol = tol
    return a


def stream_sizes(head):
    """Ids of every stream: V_stream, or V for each of the K streams."""
    vs = head.get("V_stream")
    return [head["V"]] * head["K"] if vs is None else [int(v) for v in vs]


def head_columns(head):
    """N: the columns of all streams together."""
    return int(sum(stream_sizes(head)))


def head_step(head, batch, seed=0, n_slots=0, F_max=0, frame_grid=None,
              gap_tol=1e-3, topk_tol=1e-6, topp_tol=1e-6, want_scores=True):
    """One decode step of the head over a batch (all arrays numpy, host).

    head: dict(H, K, V, pad_id, delays[K], W[K][V][H] (float32 or uint16 bf16 bits),
               bias[K][V] or None, W_text[V_text][H] or None; optionally V_stream[K]
               for streams of unequal size, with W[N][H] and bias[N], N = sum V_stream)
    batch: dict(hidden[R][H], pair_map, row_kind, cfg_w, temperature, top_k, top_p,
                rng_key or None, step, n_frames, grid_slot)
    Returns dict(tokens[R][K], scores[R][N] (fp64, COND/SOLO rows), gap[R][K], flags[R][K],
                 frame_grid, modality[R], modality_gap[R]) -- frame_grid is updated in place
    when given; modality (TEXT rows) follows head["T_text"], the text ids of the text head.
    """
    keep = []
    a = _step_struct(head, batch, seed, n_slots, F_max, (gap_tol, topk_tol, topp_tol), keep)
    R, K = a.R, a.K
    N = head_columns(head)
    tokens = np.full((R, K), -1, dtype=np.int32)
    scores = np.full((R, N), np.nan) if want_scores else None
    gap = np.full((R, K), np.inf)
    flags = np.zeros((R, K), dtype=np.uint32)
    if frame_grid is not None:
        assert frame_grid.dtype == np.int32 and frame_grid.flags.c_contiguous
        assert frame_grid.shape == (n_slots, K, F_max)
    modality = np.zeros(R, dtype=np.uint8)
    modality_gap = np.full(R, np.inf)
    a.tokens_out, a.frame_grid = tokens.ctypes.data, _ptr(frame_grid)
    a.modality, a.modality_gap = modality.ctypes.data, modality_gap.ctypes.data
    a.scores, a.gap, a.flags = _ptr(scores), gap.ctypes.data, flags.ctypes.data
    rc = lib().orc_head_step(ctypes.byref(a))
    if rc:
        raise ValueError("oracle head_step: " + ERRORS.get(rc, str(rc)))
    return dict(tokens=tokens, scores=scores, gap=gap, flags=flags, frame_grid=frame_grid,
                modality=modality, modality_gap=modality_gap)


def sample_rows(head, batch, srow, crow, scores, seed=0, n_slots=0, F_max=0, frame_grid=None,
                gap_tol=1e-3, topk_tol=1e-6, topp_tol=1e-6):
    """Sampling part of a step from given scores[Rs][K*V] (rows in sampled order srow,
    companions crow, -1 for none).  Returns tokens[R][K] (-1 where untouched), gap, flags."""
    keep = []
    a = _step_struct(head, batch, seed, n_slots, F_max, (gap_tol, topk_tol, topp_tol), keep)
    R, K = a.R, a.K
    srow = np.ascontiguousarray(srow, dtype=np.int32)
    crow = np.ascontiguousarray(crow, dtype=np.int32)
    sc = np.ascontiguousarray(scores, dtype=np.float64)
    assert sc.shape == (srow.shape[0], head_columns(head))
    tokens = np.full((R, K), -1, dtype=np.int32)
    gap = np.full((R, K), np.inf)
    flags = np.zeros((R, K), dtype=np.uint32)
    a.tokens_out, a.frame_grid = tokens.ctypes.data, _ptr(frame_grid)
    a.scores, a.gap, a.flags = None, gap.ctypes.data, flags.ctypes.data
    rc = lib().orc_sample_rows(ctypes.byref(a), srow.shape[0], srow.ctypes.data,
                               crow.ctypes.data, sc.ctypes.data)
    if rc:
        raise ValueError("oracle sample_rows: " + ERRORS.get(rc, str(rc)))
    return dict(tokens=tokens, gap=gap, flags=flags, frame_grid=frame_grid)


def next_input(E, tokens, row_kind, pad_id, E_text=None):
    """Next-step input of every row (Sec. 2.1): sum over streams k of
    E[k][tokens[r][k]] (row V of stream k's table for the pad id), exact in
    fp64 and rounded once to the table type; TEXT rows take
    E_text[tokens[r][0]].  E: [K][V + 1][H] float32 or uint16 (bf16 bits);
    tokens: [R][K] int32; row_kind: [R] uint8.  Returns [R][H] of E's type."""
    E = np.ascontiguousarray(E)
    K, V1, H = E.shape
    dtype = BF16 if E.dtype == np.uint16 else F32
    tokens = np.ascontiguousarray(tokens, dtype=np.int32).reshape(-1, K)
    R = tokens.shape[0]
    row_kind = np.ascontiguousarray(row_kind, dtype=np.uint8)
    assert row_kind.shape == (R,)
    V_text = 0
    if E_text is not None:
        E_text = np.ascontiguousarray(E_text)
        assert E_text.dtype == E.dtype and E_text.shape[1] == H
        V_text = E_text.shape[0]
    out = np.zeros((R, H), dtype=E.dtype)
    rc = lib().orc_next_input(R, H, K, V1 - 1, int(pad_id), dtype, E.ctypes.data, V_text,
                              _ptr(E_text), row_kind.ctypes.data, tokens.ctypes.data,
                              out.ctypes.data)
    if rc:
        raise ValueError(ERRORS.get(rc, rc))
    return out


# --------------------------------------------------------------------------
# Mixed-modality phase of a request (Sec. 2.3)

PHASE_TEXT, PHASE_BRIDGE, PHASE_AUDIO, PHASE_DRAIN = 0, 1, 2, 3


def phase_advance(phase, count, token0, modality, bridge, audio_end, drain_steps):
    """One decode step of one request's phase -> (phase, count, emit).

    TEXT: the request's row emitted token0, its greedy token over the text
      ids (the vocabulary mask).  When the unmasked argmax lay outside the
      text ids (modality = 1) the request leaves the text phase: it emits the
      first bridging token instead and continues with the rest of them, or,
      with no bridging tokens, keeps token0 and goes straight to AUDIO.
    BRIDGE: emits bridge[count]; after the last one, AUDIO.
    AUDIO: the head's sampled tokens are the output (emit -1); a stream-0
      token equal to audio_end ends the phase.
    DRAIN: drain_steps steps (the largest delay, S - 1) in which the delayed
      streams finish their frames and the rest are pads (emit -1); then TEXT.
    count: bridging tokens emitted (BRIDGE), audio steps taken (AUDIO),
    drain steps taken (DRAIN)."""
    nb = len(bridge)
    if phase == PHASE_TEXT:
        if not modality:
            return PHASE_TEXT, 0, token0
        if nb == 0:
            return PHASE_AUDIO, 0, token0
        return (PHASE_BRIDGE, 1, bridge[0]) if nb > 1 else (PHASE_AUDIO, 0, bridge[0])
    if phase == PHASE_BRIDGE:
        emit = bridge[count]
        return (PHASE_AUDIO, 0, emit) if count + 1 >= nb else (PHASE_BRIDGE, count + 1, emit)
    if phase == PHASE_AUDIO:
        if token0 == audio_end:
            return (PHASE_DRAIN, 0, -1) if drain_steps > 0 else (PHASE_TEXT, 0, -1)
        return PHASE_AUDIO, count + 1, -1
    if phase == PHASE_DRAIN:
        return (PHASE_TEXT, 0, -1) if count + 1 >= drain_steps else (PHASE_DRAIN, count + 1, -1)
    raise ValueError(f"unknown phase {phase}")
