"""Paired co-scheduling (host): the library's scheduler against the plain oracle
of the policy, which is pinned first by a trace worked by hand and by
invariants over random request streams.  CPU only."""
import random

import numpy as np
import pytest

from oracle.cosched import CoScheduler, ROW_COND, ROW_SOLO, ROW_TEXT, ROW_UNCOND
from paper_2607_02119_amd import mcd

# Budget 6 tokens, 4 rows, null prompt 1 token, drain 1 step.  Requests:
#   0: pair (w 3), prompt 4, text 1, frames 1;  1: solo, prompt 2, text 0,
#   frames 2;  2: pair (w 2), prompt 1, text 0, frames 1.
# Worked by hand from the rules: step 0 admits 0 (each member granted 3: the
# Companion uses 1, the pair is charged 6), so 1 waits; step 1 finishes 0's
# prompt (granted 1 each, charged 2) and admits 1 (2 tokens); 2 cannot get two
# rows until 0 and 1 finish at step 4.
HAND = [
    # (rows (id, member, tokens, context), head (id, member, kind, step, partner, grid), finished)
    ([(0, 0, 3, 0), (0, 1, 1, 0)], [], []),
    ([(0, 0, 1, 3), (1, 0, 2, 0)], [], []),
    ([(0, 0, 1, 4), (1, 0, 1, 2)],
     [(0, 0, ROW_TEXT, 0, -1, -1), (1, 0, ROW_SOLO, 0, -1, 2)], []),
    ([(0, 0, 1, 5), (0, 1, 1, 2), (1, 0, 1, 3)],
     [(0, 0, ROW_COND, 0, 1, 0), (0, 1, ROW_UNCOND, 0, 0, -1), (1, 0, ROW_SOLO, 1, -1, 2)], []),
    ([(0, 0, 1, 6), (0, 1, 1, 3), (1, 0, 1, 4)],
     [(0, 0, ROW_COND, 1, 1, 0), (0, 1, ROW_UNCOND, 1, 0, -1), (1, 0, ROW_SOLO, 2, -1, 2)], [0, 1]),
    ([(2, 0, 1, 0), (2, 1, 1, 0)], [], []),
    ([(2, 0, 1, 1), (2, 1, 1, 1)], [(2, 0, ROW_COND, 0, 1, 0), (2, 1, ROW_UNCOND, 0, 0, -1)], []),
    ([(2, 0, 1, 2), (2, 1, 1, 2)], [(2, 0, ROW_COND, 1, 1, 0), (2, 1, ROW_UNCOND, 1, 0, -1)], [2]),
    ([], [], []),
]
HAND_REQS = [(3.0, 4, 1, 1), (1.0, 2, 0, 2), (2.0, 1, 0, 1)]


def lib_step(s):
    b = s.plan()
    rows = [(int(b["row_req"][i]), int(b["row_member"][i]), int(b["row_tokens"][i]),
             int(b["row_context"][i])) for i in range(b["n_rows"])]
    head = []
    for j in range(b["R"]):
        r = int(b["head_row"][j])
        head.append((int(b["row_req"][r]), int(b["row_member"][r]), int(b["row_kind"][j]),
                     int(b["step"][j]), int(b["pair_map"][j]), int(b["grid_slot"][j])))
    fin = [int(x) for x in s.commit()]
    return rows, head, fin, b


def test_oracle_hand_trace():
    o = CoScheduler(4, 6, 1, 1)
    for q in HAND_REQS:
        o.submit(*q)
    for k, want in enumerate(HAND):
        assert o.step() == want, f"step {k}"


def test_library_hand_trace():
    s = mcd.Scheduler(4, 6, 1, 1)
    for q in HAND_REQS:
        s.submit(*q)
    for k, want in enumerate(HAND):
        rows, head, fin, _ = lib_step(s)
        assert (rows, head, fin) == want, f"step {k}"
    assert s.counts() == (0, 0)


def random_stream(rng, n):
    """(arrival step, cfg_w, prompt, text, frames) in arrival order."""
    out, t = [], 0
    for _ in range(n):
        t += rng.choice([0, 0, 1, 2, 5])
        w = rng.choice([1.0, 0.0, 3.0, 2.5, 1.5])
        out.append((t, w, rng.randint(1, 40), rng.randint(0, 12), rng.randint(1, 9)))
    return out


CONFIGS = [
    # max_rows, token_budget, null prompt, drain
    (4, 6, 1, 1),
    (8, 32, 3, 3),
    (16, 16, 2, 0),
    (7, 64, 5, 7),
    (2, 2, 1, 2),
]


def run_oracle(cfg, stream, max_steps=5000):
    o = CoScheduler(*cfg)
    steps, i = [], 0
    for t in range(max_steps):
        while i < len(stream) and stream[i][0] <= t:
            o.submit(*stream[i][1:])
            i += 1
        steps.append(o.step())
        if i == len(stream) and not o.queue:
            break
    return steps


@pytest.mark.parametrize("cfg", CONFIGS)
def test_oracle_invariants(cfg):
    max_rows, budget, null_prompt, drain = cfg
    rng = random.Random(7 + max_rows)
    stream = random_stream(rng, 60)
    steps = run_oracle(cfg, stream)
    reqs = {i: q[1:] for i, q in enumerate(stream)}
    fed = {}
    text_steps, audio_steps, finished, first_seen = {}, {}, [], {}
    for k, (rows, head, fin) in enumerate(steps):
        assert sum(r[2] for r in rows) <= budget, k
        assert len({(r[0], r[1]) for r in rows}) == len(rows), k
        decode_rows = {(h[0], h[1]) for h in head}
        prompt = {}                           # prompt tokens of this step per member
        for rid, member, tokens, context in rows:
            first_seen.setdefault(rid, k)
            if (rid, member) in decode_rows:
                assert tokens == 1
            else:
                assert context == fed.get((rid, member), 0)
                prompt.setdefault(rid, {})[member] = tokens
        # a pair's members get the same grant: they differ only where the
        # smaller one took the rest of its prompt (the null prompt is short)
        for rid, g in prompt.items():
            w, plen = reqs[rid][0], reqs[rid][1]
            full = {0: plen, 1: null_prompt}
            if w > 1:
                lo = min(g, key=lambda m: g[m]) if len(g) == 2 else 1 - next(iter(g))
                hi = 1 - lo
                if g.get(lo, 0) != g[hi]:
                    assert fed.get((rid, lo), 0) + g.get(lo, 0) == full[lo], (k, rid, g)
            for m, tk in g.items():
                fed[(rid, m)] = fed.get((rid, m), 0) + tk
        ids = [h[0] for h in head]
        for j, (rid, member, kind, st, partner, grid) in enumerate(head):
            w = reqs[rid][0]
            if kind == ROW_TEXT:
                assert member == 0 and partner == -1 and grid == -1
                text_steps[rid] = text_steps.get(rid, 0) + 1
            elif kind == ROW_COND:
                assert w > 1 and head[partner][:2] == (rid, 1) and head[partner][4] == j
                audio_steps[rid] = audio_steps.get(rid, 0) + 1
            elif kind == ROW_UNCOND:
                assert w > 1 and head[partner][:2] == (rid, 0)
            else:
                assert kind == ROW_SOLO and w <= 1
                audio_steps[rid] = audio_steps.get(rid, 0) + 1
        # a pair in its audio phase runs both rows in the same step
        for rid in set(ids):
            kinds = sorted(h[2] for h in head if h[0] == rid)
            assert kinds in ([ROW_TEXT], [ROW_SOLO], [ROW_COND, ROW_UNCOND]), (k, rid, kinds)
        finished += fin
    # admission in arrival order
    order = sorted(first_seen, key=lambda r: (first_seen[r], r))
    assert order == sorted(first_seen)
    # every request finished once, with every token accounted for
    assert sorted(finished) == list(range(len(stream)))
    for rid, (w, prompt, text, frames) in reqs.items():
        assert fed[(rid, 0)] == prompt
        if w > 1:
            assert fed[(rid, 1)] == null_prompt
        assert text_steps.get(rid, 0) == text
        assert audio_steps.get(rid, 0) == frames + drain


@pytest.mark.parametrize("cfg", CONFIGS)
@pytest.mark.parametrize("seed", [1, 2, 3])
def test_library_matches_oracle(cfg, seed):
    rng = random.Random(1000 * seed + cfg[0])
    stream = random_stream(rng, 80)
    want = run_oracle(cfg, stream)
    s = mcd.Scheduler(*cfg)
    i = 0
    for t, w in enumerate(want):
        while i < len(stream) and stream[i][0] <= t:
            s.submit(*stream[i][1:])
            i += 1
        rows, head, fin, _ = lib_step(s)
        assert (rows, head, fin) == w, f"step {t}"
    assert s.counts() == (0, 0)


def test_library_rejects_bad_use():
    with pytest.raises(mcd.McdError):
        mcd.Scheduler(4, 3, 1, 1)            # budget below the rows
    with pytest.raises(mcd.McdError):
        mcd.Scheduler(4, 8, 0, 1)            # empty null prompt
    s = mcd.Scheduler(1, 4, 1, 0, max_requests=2)
    with pytest.raises(mcd.McdError):
        s.submit(3.0, 4, 0, 1)               # a pair on a one-row batch
    with pytest.raises(mcd.McdError):
        s.submit(1.0, 0, 0, 1)               # empty prompt
    with pytest.raises(mcd.McdError):
        s.submit(float("nan"), 4, 0, 1)
    s.submit(1.0, 4, 0, 1)
    s.submit(1.0, 4, 0, 1)
    with pytest.raises(mcd.McdError):
        s.submit(1.0, 4, 0, 1)               # table full
    s.plan()
    with pytest.raises(mcd.McdError):
        s.plan()                             # the planned step is not committed
    s.commit()
    with pytest.raises(mcd.McdError):
        s.commit()                           # nothing planned
