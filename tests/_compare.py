"""Comparison helpers for the GPU parity tests (test code: may use the oracle)."""
from __future__ import annotations

import sys

import numpy as np

import oracle

EXEMPT = oracle.FLAG_GAP_SMALL | oracle.FLAG_TOPP_EDGE | oracle.FLAG_TOPK_EDGE


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def subset_batch(batch: dict, rows) -> dict:
    """Sub-batch of the given physical rows (partners must be included)."""
    rows = np.asarray(rows)
    inv = {int(r): i for i, r in enumerate(rows)}
    sub = {}
    for k, v in batch.items():
        sub[k] = v[rows] if isinstance(v, np.ndarray) and v.shape[:1] == batch["pair_map"].shape else v
    sub["pair_map"] = np.array([inv[int(p)] if p >= 0 else -1 for p in batch["pair_map"][rows]],
                               np.int32)
    return sub


def pick_rows(layout: dict, n_pairs=2, n_solo=2, n_text=2, seed=0):
    """A few Main rows with their Companions, solo rows and text rows."""
    rng = np.random.default_rng(seed)
    kind, pm = layout["row_kind"], layout["pair_map"]
    out = []
    conds = np.where(kind == oracle.ROW_COND)[0]
    for c in rng.choice(conds, min(n_pairs, len(conds)), replace=False) if len(conds) else []:
        out += [int(c), int(pm[c])]
    for kd, n in ((oracle.ROW_SOLO, n_solo), (oracle.ROW_TEXT, n_text)):
        cand = np.where(kind == kd)[0]
        if len(cand):
            out += [int(x) for x in rng.choice(cand, min(n, len(cand)), replace=False)]
    return sorted(out)


def score_rel_err(gpu_scores, plan_rows, ora_scores, sizes):
    """max over (row, k) vectors of max|g - o| / max|o|; plan_rows[s] = physical row;
    sizes[k] = ids of stream k (the vectors' lengths, in column order)."""
    worst = 0.0
    edges = np.concatenate([[0], np.cumsum(sizes)])
    for s, r in enumerate(plan_rows):
        if r is None:
            continue
        g = gpu_scores[s].astype(np.float64)
        o = ora_scores[r]
        for k in range(len(sizes)):
            gk, ok = g[edges[k]:edges[k + 1]], o[edges[k]:edges[k + 1]]
            den = max(float(np.abs(ok).max()), 1e-300)
            worst = max(worst, float(np.abs(gk - ok).max()) / den)
    return worst


class TokenCheck:
    """Accumulates token comparisons with the exemption classes of the oracle."""

    def __init__(self):
        self.n = 0
        self.mismatch = 0
        self.exempt = {"gap": 0, "topp": 0, "topk": 0}
        self.bad = []

    def add(self, gpu_tok, ora_tok, flags, rows=None, where=""):
        g = np.asarray(gpu_tok)
        o = np.asarray(ora_tok)
        f = np.asarray(flags).astype(np.int64)
        if rows is not None:
            rows = np.asarray(list(rows))
            g, o, f = g[rows], o[rows], f[rows]
        else:
            rows = np.arange(g.shape[0])
        self.n += g.size
        bad = g != o
        self.mismatch += int(bad.sum())
        gap = bad & ((f & oracle.FLAG_GAP_SMALL) > 0)
        topp = bad & ~gap & ((f & oracle.FLAG_TOPP_EDGE) > 0)
        topk = bad & ~gap & ~topp & ((f & oracle.FLAG_TOPK_EDGE) > 0)
        self.exempt["gap"] += int(gap.sum())
        self.exempt["topp"] += int(topp.sum())
        self.exempt["topk"] += int(topk.sum())
        for i, k in zip(*np.nonzero(bad & ~gap & ~topp & ~topk)):
            self.bad.append((where, int(rows[i]), int(k), int(g[i, k]), int(o[i, k]),
                             int(f[i, k])))

    def assert_ok(self, label=""):
        say(f"[{label}] positions={self.n} mismatches={self.mismatch} exempt={self.exempt} "
            f"unexplained={len(self.bad)}")
        assert not self.bad, f"unexplained token mismatches: {self.bad[:10]}"
