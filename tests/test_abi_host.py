"""Host-side checks of the C ABI (no GPU needed, no kernel launched): the library
loads, exports every function include/mcd.h declares, and rejects bad
arguments and inconsistent batches before any launch."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mcd.h")

mcd = pytest.importorskip("paper_2607_02119_amd.mcd", reason="libmcd.so not built")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mcd_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 12
    lib = ctypes.CDLL(mcd._LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in mcd.h but not exported"
    assert sorted(mcd.EXPORTED) == names


FAKE_W = 0x10000   # never dereferenced: host-only calls


def _head(**kw):
    args = dict(H=64, K=3, V=50, pad_id=50, delays=[0, 1, 2], dtype=mcd.MCD_BF16, W=FAKE_W)
    args.update(kw)
    return mcd.mcd_head_create(**args)


def test_head_create_validation():
    h = _head()
    mcd.mcd_head_destroy(h)
    bad = [dict(H=65), dict(K=0, delays=[]), dict(K=33, delays=list(range(33))), dict(V=0),
           dict(V=mcd.MCD_MAX_V + 1), dict(delays=[0, -1, 2]), dict(W=0), dict(W=FAKE_W + 2),
           dict(dtype=7), dict(V_text=10, W_text=None)]
    for b in bad:
        with pytest.raises(mcd.McdError):
            _head(**b)
    h = _head(dtype=mcd.MCD_F32, H=40)
    mcd.mcd_head_destroy(h)
    # streams of unequal size: V is the largest, every stream 1..MCD_MAX_V ids
    h = _head(V_stream=[50, 7, 13])
    mcd.mcd_head_destroy(h)
    for vs in ([50, 0, 3], [10, 20, 30], [50, 51, 3], [mcd.MCD_MAX_V + 1, 1, 1]):
        with pytest.raises(mcd.McdError):
            _head(V_stream=vs, V=50)


# A bf16 head with a text head creates its side stream (a HIP call) at
# creation; the host-only tests take fp32 heads where a text head is needed.
def _text_head(**kw):
    return _head(dtype=mcd.MCD_F32, H=40, V_text=100, W_text=FAKE_W, **kw)


def test_batch_plan_layout_and_errors():
    h = _text_head()
    # rows: 0 solo, 1 uncond(->3), 2 text, 3 cond(->1), 4 cond(->5), 5 uncond(->4)
    pm = [-1, 3, -1, 1, 5, 4]
    rk = [2, 1, 3, 0, 0, 1]
    plan, c = mcd.mcd_batch_plan(h, pm, rk)
    assert (c.n_pairs, c.n_solo, c.n_text) == (2, 1, 1)
    assert plan[1] == 6 and list(plan[2:5]) == [2, 1, 1]
    assert list(plan[8:]) == [3, 1, 4, 5, 0, 2]
    assert mcd.mcd_plan_sampled_row(plan, 0) == (3, 1)
    assert mcd.mcd_plan_sampled_row(plan, 1) == (4, 5)
    assert mcd.mcd_plan_sampled_row(plan, 2) == (0, -1)
    with pytest.raises(mcd.McdError):
        mcd.mcd_plan_sampled_row(plan, 3)
    for pm_bad, rk_bad in [([1, 0], [0, 0]),           # partner of the wrong kind
                           ([1, 2, 1], [0, 1, 1]),     # partner points elsewhere
                           ([0], [0]),                 # self partner
                           ([5, 0], [0, 1]),           # out of range
                           ([0, -1], [2, 2]),          # solo row with a partner
                           ([-1], [9])]:               # unknown kind
        with pytest.raises(mcd.McdError):
            mcd.mcd_batch_plan(h, pm_bad, rk_bad)
    h2 = _head()
    with pytest.raises(mcd.McdError):
        mcd.mcd_batch_plan(h2, [-1], [3])              # text row, no text head
    assert mcd.mcd_workspace_bytes(h2, 100) == 256
    assert mcd.mcd_workspace_bytes(h, 4) > 256


def test_step_argument_errors_before_launch():
    h = _head()
    plan, c = mcd.mcd_batch_plan(h, [1, 0], [0, 1])
    base = dict(R=2, counts=c, plan=FAKE_W, hidden=FAKE_W, cfg_w=FAKE_W, temperature=FAKE_W,
                top_k=FAKE_W, top_p=FAKE_W, rng_key=None, step=FAKE_W, n_frames=FAKE_W,
                grid_slot=FAKE_W, seed=0, tokens_out=FAKE_W, frame_grid=None, n_slots=0, F_max=0,
                scores=FAKE_W, workspace=None)
    with pytest.raises(mcd.McdError) as e:
        mcd.mcd_head_step(h, stream=0, **base)                 # no workspace
    assert e.value.code == mcd.MCD_E_WORKSPACE
    for field, val in [("scores", None), ("hidden", None), ("temperature", None),
                       ("tokens_out", None), ("plan", None), ("R", 3), ("n_slots", -1)]:
        kw = dict(base, **{field: val})
        kw["workspace"] = None
        with pytest.raises(mcd.McdError) as e:
            mcd.mcd_head_step(h, stream=0, **kw)
        assert e.value.code in (mcd.MCD_E_INVALID, mcd.MCD_E_WORKSPACE)
    # misaligned hidden for bf16
    a = mcd._step_args(**dict(base, hidden=FAKE_W + 2))
    a.workspace, a.workspace_bytes = 0x100000, 4096
    rc = mcd._mcd_head_step(h, ctypes.byref(a), None)
    assert rc == mcd.MCD_E_INVALID and "aligned" in mcd.mcd_last_error()


def test_every_per_row_array_is_required():
    """The kernels read every per-row parameter array at every row, text rows
    included: a non-empty batch without one of them is rejected on the host,
    whatever its row kinds (solo-only without cfg_w, text-only batches)."""
    per_row = ("cfg_w", "temperature", "top_k", "top_p", "step", "n_frames", "grid_slot")
    h = _text_head()
    for pm, rk in (([-1, -1], [2, 2]),          # solo rows only
                   ([-1, -1], [3, 3]),          # text rows only
                   ([1, 0, -1], [0, 1, 3])):    # a pair and a text row
        plan, c = mcd.mcd_batch_plan(h, pm, rk)
        base = dict(R=len(pm), counts=c, plan=FAKE_W, hidden=FAKE_W, cfg_w=FAKE_W,
                    temperature=FAKE_W, top_k=FAKE_W, top_p=FAKE_W, rng_key=None, step=FAKE_W,
                    n_frames=FAKE_W, grid_slot=FAKE_W, seed=0, tokens_out=FAKE_W,
                    frame_grid=None, n_slots=0, F_max=0, scores=FAKE_W, workspace=None)
        for field in per_row:
            a = mcd._step_args(**dict(base, **{field: None}))
            a.workspace, a.workspace_bytes = 0x100000, 1 << 30
            for f in (mcd._mcd_head_step, mcd._mcd_head_logits, mcd._mcd_sample_step):
                assert f(h, ctypes.byref(a), None) == mcd.MCD_E_INVALID, (rk, field)
                assert "per-row" in mcd.mcd_last_error()
    mcd.mcd_head_destroy(h)


def test_interleave_argument_errors():
    with pytest.raises(mcd.McdError):
        mcd._check(mcd._mcd_deinterleave(FAKE_W, 1, 2, 3, np.array([0, 1, 5], np.int32).ctypes.data,
                                         FAKE_W, None), "x")      # T shorter than a delay
    with pytest.raises(mcd.McdError):
        mcd._check(mcd._mcd_interleave(FAKE_W, 1, 4, 0, None, 0, FAKE_W, None), "x")
    # empty work is a no-op, not an error
    mcd._check(mcd._mcd_deinterleave(None, 0, 5, 2, np.array([0, 1], np.int32).ctypes.data,
                                     None, None), "x")
    assert mcd.mcd_status_string(mcd.MCD_E_HIP) == "hip error"


def _next_input_args(**kw):
    a = dict(R=4, H=64, K=3, V=50, pad_id=50, dtype=mcd.MCD_BF16, E=FAKE_W, V_text=0, E_text=None,
             row_kind=FAKE_W, tokens=FAKE_W, out=FAKE_W * 2, workspace=None)
    a.update(kw)
    return mcd.mcd_next_input_args(a["R"], a["H"], a["K"], a["V"], a["pad_id"], a["dtype"], a["E"],
                                   a["V_text"], a["E_text"], a["row_kind"], a["tokens"], a["out"],
                                   a["workspace"])


def test_next_input_validation():
    """Rejected before any launch; R = 0 is a no-op."""
    bad = [dict(R=-1), dict(H=0), dict(K=0), dict(K=33), dict(V=0), dict(V_text=-1),
           dict(dtype=7), dict(pad_id=0), dict(pad_id=49), dict(E=None), dict(out=None),
           dict(tokens=None), dict(row_kind=None), dict(E=FAKE_W + 8), dict(out=FAKE_W + 4),
           dict(V_text=10), dict(E_text=FAKE_W), dict(V_text=10, E_text=FAKE_W + 2),
           dict(workspace=FAKE_W + 16)]
    for b in bad:
        a = _next_input_args(**b)
        assert mcd._mcd_next_input(ctypes.byref(a), None) == mcd.MCD_E_INVALID, b
    for ok_empty in (dict(R=0), dict(R=0, E=None, out=None)):
        a = _next_input_args(**ok_empty)
        assert mcd._mcd_next_input(ctypes.byref(a), None) == mcd.MCD_OK
    assert mcd._mcd_next_input(None, None) == mcd.MCD_E_INVALID


def test_text_mask_validation():
    h = _text_head(T_text=64)
    mcd.mcd_head_destroy(h)
    for tt in (0, 100):
        mcd.mcd_head_destroy(_text_head(T_text=tt))
    for tt in (-1, 50, 101, 96 + 32):
        with pytest.raises(mcd.McdError):
            _text_head(T_text=tt)


def test_phase_advance_matches_oracle():
    """The library's host phase machine against the oracle's, over random
    token and modality streams for many requests."""
    import oracle
    rng = np.random.default_rng(7)
    for bridge, end, drain in (([900, 901, 902], 7, 3), ([], 5, 0), ([42], 3, 1)):
        n = 64
        phase = np.zeros(n, np.uint8)
        count = np.zeros(n, np.int32)
        ref = [(0, 0)] * n
        seen = set()
        for step in range(200):
            tok = rng.integers(0, 10, size=n).astype(np.int32)
            mod = (rng.random(n) < 0.1).astype(np.uint8)
            emit = mcd.mcd_phase_advance(bridge, end, drain, phase, count, tok, mod)
            for i in range(n):
                ph, c, e = oracle.phase_advance(ref[i][0], ref[i][1], int(tok[i]), int(mod[i]),
                                                bridge, end, drain)
                ref[i] = (ph, c)
                assert (phase[i], count[i], emit[i]) == (ph, c, e), (step, i)
                seen.add(ph)
        assert seen >= {oracle.PHASE_TEXT, oracle.PHASE_AUDIO}


def test_phase_advance_rejects_bad_state():
    for ph, c in ((9, 0), (0, 1), (1, 0), (1, 5), (3, 2), (2, -1)):
        phase = np.array([ph], np.uint8)
        count = np.array([c], np.int32)
        with pytest.raises(mcd.McdError):
            mcd.mcd_phase_advance([1, 2], 7, 2, phase, count, [0], [0])


def test_empty_batch_is_a_no_op():
    """A step over no rows returns OK before any launch (no pointer is read)."""
    h = _head()
    c = mcd.mcd_batch_counts(0, 0, 0)
    a = mcd.mcd_step_args(0, c, None, None, None, None, None, None, None, None, None, None, 0,
                          None, None, None, 0, 0, None, FAKE_W, 256)
    for name, f in [("mcd_head_step", mcd._mcd_head_step),
                    ("mcd_head_logits", mcd._mcd_head_logits),
                    ("mcd_sample_step", mcd._mcd_sample_step)]:
        rc = f(h, ctypes.byref(a), None)
        assert rc == mcd.MCD_OK, (name, mcd.mcd_last_error())
    mcd.mcd_head_destroy(h)
