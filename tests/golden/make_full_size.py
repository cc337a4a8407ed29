"""Write the full-size parity fixtures: the CPU oracle's tokens, classification
flags, text-row modality and frame-grid cells for every row of the benchmark
workloads at a spread of decode steps (every step for memory_bound_decode).

    python tests/golden/make_full_size.py [--threads N] [--only NAME ...]

Calls only the oracle (``oracle/``) and the seeded input generators
(``paper_2607_02119_amd.inputs``); nothing here runs on, or reads anything
from, the GPU path.  Decode steps are independent (hidden states are
regenerated per step and the noise is counter-based), so the steps of a
workload are sharded over threads: each oracle call is one single-threaded C
call that releases the GIL.  The steps of a workload write their grid cells
into one frame grid that starts at -1, so its cells are exactly those the
listed steps produce.

One ``full_<workload>.npz`` per workload, with
  steps [S] int32, tokens [S][R][K] int32, flags [S][R][K] uint8 (oracle
  FLAG_* bits at the tolerances below), modality [S][R] uint8 and
  modality_gap_ok [S][R] bool (text rows: the two regions' maxima at least
  GAP_TOL apart), grid [n_slots][K][F] int32, workload (the definition as text)
  and tol [3] (gap, top-k, top-p tolerances).
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import dataclasses
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2607_02119_amd import inputs  # noqa: E402

# Tolerances of the oracle's exemption classes (the end-to-end parity tests'):
# top-2 perturbed gap, top-k cut margin, top-p boundary distance.
GAP_TOL, TOPK_TOL, TOPP_TOL = 1e-3, 1e-4, 1e-5


def spread_steps(wl):
    """The first step (one stream live), the last start-up pad step, the first
    step with every stream live, two steps in the middle, the last step with
    every stream live, the first drain step and the last step."""
    K1 = wl.max_delay
    T = wl.steps
    cand = [0, K1 - 1, K1, T // 3, T // 2, wl.frames - 1, wl.frames, T - 1]
    return sorted({t for t in cand if 0 <= t < T})


FIXTURES = {
    "memory_bound_decode": "all",
    "weight_streaming": "spread",
    "mfma_mixed": "spread",
    "cfg_on": "spread",
    "cfg_off": "spread",
    "opuslm_9_streams": [8, 300],
    "mixed_text_mask": [9, 64],
}


def fixture_path(name):
    return os.path.join(HERE, f"full_{name}.npz")


def fixture_steps(name):
    wl = inputs.WORKLOADS[name]
    how = FIXTURES[name]
    if how == "all":
        return list(range(wl.steps))
    if how == "spread":
        return spread_steps(wl)
    return list(how)


def workload_text(wl):
    return repr(dataclasses.astuple(wl))


def make(name, threads):
    wl = inputs.WORKLOADS[name]
    steps = fixture_steps(name)
    t0 = time.time()
    head = inputs.make_weights(wl)
    lay = inputs.row_layout(wl)
    R, K = wl.R, wl.K
    grid = np.full((wl.n_slots, K, wl.frames), -1, np.int32)

    def one(t):
        b = inputs.make_batch(wl, t, lay)
        g = np.full_like(grid, -1)
        o = oracle.head_step(head, b, seed=inputs.SEED_SAMPLING, n_slots=wl.n_slots,
                             F_max=wl.frames, frame_grid=g, gap_tol=GAP_TOL, topk_tol=TOPK_TOL,
                             topp_tol=TOPP_TOL, want_scores=False)
        return t, o, g

    tokens = np.zeros((len(steps), R, K), np.int32)
    flags = np.zeros((len(steps), R, K), np.uint8)
    modality = np.zeros((len(steps), R), np.uint8)
    mod_ok = np.zeros((len(steps), R), bool)
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        for t, o, g in ex.map(one, steps):
            i = steps.index(t)
            tokens[i] = o["tokens"]
            flags[i] = o["flags"].astype(np.uint8)
            modality[i] = o["modality"]
            mod_ok[i] = o["modality_gap"] >= GAP_TOL
            cells = g >= 0
            assert not (cells & (grid >= 0)).any(), "two steps wrote one grid cell"
            grid[cells] = g[cells]
    np.savez_compressed(fixture_path(name), steps=np.array(steps, np.int32), tokens=tokens,
                        flags=flags, modality=modality, modality_gap_ok=mod_ok, grid=grid,
                        workload=np.array(workload_text(wl)),
                        tol=np.array([GAP_TOL, TOPK_TOL, TOPP_TOL]))
    print(f"{name}: {len(steps)} steps, {R} rows, {time.time() - t0:.0f} s", flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    ap.add_argument("--only", nargs="*", default=None)
    args = ap.parse_args()
    oracle.build(force=False)
    for name in (args.only or list(FIXTURES)):
        make(name, args.threads)


if __name__ == "__main__":
    main()
