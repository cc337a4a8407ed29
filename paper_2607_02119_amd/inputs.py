"""Seeded synthetic inputs for the multi-codebook decode head.

This module produces bytes and nothing else: weight matrices, hidden states,
the row layout of a continuous batch and the per-row sampling parameters.  It
holds none of the method's arithmetic (no projection, merge, selection, noise
or de-interleave), and both the HIP path and the CPU oracle consume exactly the
arrays it returns.

Recipe (fixed seeds; numpy's PCG64 via ``default_rng``):
  * stream-embedding term of the heads (when a workload asks for it): the fp32
    bias b[n] = N(0,1) over the N columns from default_rng([seed_w, 2000]),
    given as it is (the product W_k e_k of a model's stream embedding e_k,
    precomputed).
  * streams of unequal size (V_stream): stream k's V_stream[k] weight rows from
    default_rng([seed_w, k]), all streams' rows stacked as W[N][H].
  * head weights  W_k = bf16_rne(N(0,1) / sqrt(H)) from default_rng([seed_w, k]),
    i.e. standard deviation 1/sqrt(H) so each logit is ~N(0,1); the text head
    W_text in 4096-row blocks b from default_rng([seed_w, 1000, b]).  fp32
    workloads skip the bf16 rounding.
  * hidden states hidden[t] = bf16_rne(N(0,1)) from default_rng([seed_h, t]),
    regenerated for every decode step t, rows in logical order then permuted.
  * row layout: CFG pairs (conditional row 2i, unconditional row 2i+1), then
    solo audio rows, then text rows; optionally permuted by
    default_rng(seed_perm).permutation(R) with pair_map, row kinds, request ids
    and grid slots carried along.
  * request id (the RNG key of a row): the logical index of its request (pair i,
    solo j -> n_pairs + j, text j -> n_pairs + n_solo + j); a companion row
    carries its Main row's id.  Grid slot: the request index for Main and solo
    rows, -1 for companion and text rows.
  * every row starts at step 0 and advances by one per step; each request has
    n_frames = steps - max(delay) frames.
  * embedding tables of the next-step input: E[k] = bf16_rne(N(0,1)) of shape
    [V + 1][H] from default_rng([seed_e, k]) (row V: the stream's pad
    embedding), E_text in 4096-row blocks b from default_rng([seed_e, 1000, b]).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

ROW_COND, ROW_UNCOND, ROW_SOLO, ROW_TEXT = 0, 1, 2, 3

SEED_SAMPLING = 0
SEED_W = 1
SEED_H = 2
SEED_PERM = 3
SEED_E = 4


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    H: int
    K: int
    V: int
    n_pairs: int
    n_solo: int = 0
    n_text: int = 0
    V_text: int = 0
    dtype: str = "bf16"          # "bf16" or "f32": type of hidden and weights
    cfg_w: float = 3.0
    temperature: float = 1.0
    top_k: int = 0               # <= 0: off
    top_p: float = 1.0           # >= 1: off
    steps: int = 32
    shuffle: bool = False
    delays: tuple | None = None  # default d_k = k
    pad_id: int | None = None    # default V
    bias: bool = False           # stream-embedding term b[k][v] (W_k e_k) of the heads
    V_stream: tuple | None = None  # ids per stream when they differ (V = the largest)
    T_text: int = 0              # text ids of the text head (the text phase's mask), 0: all

    @property
    def R(self) -> int:
        return 2 * self.n_pairs + self.n_solo + self.n_text

    @property
    def N(self) -> int:
        return sum(self.stream_sizes)

    @property
    def stream_sizes(self) -> list:
        if self.V_stream is None:
            return [self.V] * self.K
        assert len(self.V_stream) == self.K and max(self.V_stream) == self.V
        return [int(v) for v in self.V_stream]

    @property
    def Rs(self) -> int:
        return self.n_pairs + self.n_solo

    @property
    def delay_list(self) -> list:
        return list(self.delays) if self.delays is not None else list(range(self.K))

    @property
    def max_delay(self) -> int:
        return max(self.delay_list)

    @property
    def frames(self) -> int:
        return self.steps - self.max_delay

    @property
    def pad(self) -> int:
        return self.V if self.pad_id is None else self.pad_id

    @property
    def n_slots(self) -> int:
        return self.n_pairs + self.n_solo

    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4


# The five workloads of the benchmark table (shapes of the paper's models: 8
# codebook streams for Bagpiper, Sec. 3.1; CFG scale w > 1, Eq. 1).
WORKLOADS = {
    "tiny_ref": Workload("tiny_ref", H=256, K=4, V=1024, n_pairs=2, dtype="f32", cfg_w=3.0,
                         temperature=1.0, top_k=50, steps=32),
    "memory_bound_decode": Workload("memory_bound_decode", H=2048, K=8, V=2048, n_pairs=16,
                                    cfg_w=3.0, temperature=0.9, top_k=50, steps=256),
    "weight_streaming": Workload("weight_streaming", H=4096, K=8, V=4096, n_pairs=64, cfg_w=2.0,
                                 temperature=1.0, top_p=0.95, steps=512),
    "mfma_mixed": Workload("mfma_mixed", H=4096, K=8, V=4096, n_pairs=256, n_solo=256,
                           n_text=128, V_text=151936, cfg_w=3.0, temperature=1.0, top_k=50,
                           steps=128, shuffle=True),
    "cfg_on": Workload("cfg_on", H=4096, K=16, V=1024, n_pairs=256, cfg_w=3.0,
                       temperature=0.8, top_k=20, steps=256),
    "cfg_off": Workload("cfg_off", H=4096, K=16, V=1024, n_pairs=0, n_solo=512, cfg_w=3.0,
                        temperature=0.8, top_k=20, steps=256),
    # Two shapes of the next rows, beside the benchmark table: nine streams of
    # unequal size as in OpusLM's 1 SSL + 8 codec streams (Sec. 3.1; the sizes
    # are assumed: 4096 ids for the first stream, 1024 for the others), and
    # the mixed batch with the text phase's vocabulary mask (the last 4096
    # text-head ids stand for the other modality's markers; Sec. 2.3).
    "opuslm_9_streams": Workload("opuslm_9_streams", H=4096, K=9, V=4096,
                                 V_stream=(4096,) + (1024,) * 8, n_pairs=64, cfg_w=2.0,
                                 temperature=1.0, top_p=0.95, steps=512),
    "mixed_text_mask": Workload("mixed_text_mask", H=4096, K=8, V=4096, n_pairs=256, n_solo=256,
                                n_text=128, V_text=151936, T_text=151936 - 4096, cfg_w=3.0,
                                temperature=1.0, top_k=50, steps=128, shuffle=True),
}
# index order of the benchmark's configuration list
CONFIG_INDEX = ["tiny_ref", "memory_bound_decode", "weight_streaming", "mfma_mixed", "cfg_on"]


def bf16_rne_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal(seq, shape):
    return np.random.default_rng(seq).standard_normal(shape, dtype=np.float32)


def _to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_rne_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def make_weights(wl: Workload, seed_w: int = SEED_W) -> dict:
    """Head weights: W[K][V][H] (uint16 bf16 bits or float32), W_text[V_text][H] or None."""
    scale = np.float32(1.0 / math.sqrt(wl.H))
    edt = np.uint16 if wl.dtype == "bf16" else np.float32
    sizes = wl.stream_sizes
    if wl.V_stream is None:
        W = np.empty((wl.K, wl.V, wl.H), dtype=edt)
        blocks = [W[k] for k in range(wl.K)]
    else:                           # streams of unequal size: rows of all streams, [N][H]
        W = np.empty((wl.N, wl.H), dtype=edt)
        edges = np.concatenate([[0], np.cumsum(sizes)])
        blocks = [W[edges[k]:edges[k + 1]] for k in range(wl.K)]
    for k in range(wl.K):
        blocks[k][...] = _to_dtype(_normal([seed_w, k], (sizes[k], wl.H)) * scale, wl.dtype)
    Wt = None
    if wl.n_text > 0 or wl.V_text > 0:
        Wt = np.empty((wl.V_text, wl.H), dtype=edt)
        blk = 4096
        for b in range(0, wl.V_text, blk):
            rows = min(blk, wl.V_text - b)
            Wt[b:b + rows] = _to_dtype(_normal([seed_w, 1000, b // blk], (rows, wl.H)) * scale,
                                       wl.dtype)
    bias = None
    if wl.bias:
        bias = np.ascontiguousarray(_normal([seed_w, 2000], (wl.N,)))
        if wl.V_stream is None:
            bias = bias.reshape(wl.K, wl.V)
    head = dict(H=wl.H, K=wl.K, V=wl.V, pad_id=wl.pad, delays=np.array(wl.delay_list, np.int32),
                W=W, bias=bias, W_text=Wt)
    if wl.V_stream is not None:
        head["V_stream"] = np.array(sizes, np.int32)
    if wl.T_text:
        head["T_text"] = wl.T_text
    return head


def make_embeddings(wl: Workload, seed_e: int = SEED_E) -> dict:
    """Embedding tables of the next-step input: E[K][V + 1][H] (row V of each
    stream is its pad embedding) and E_text[V_text][H] or None; uint16 bf16
    bits or float32, like the head."""
    edt = np.uint16 if wl.dtype == "bf16" else np.float32
    E = np.empty((wl.K, wl.V + 1, wl.H), dtype=edt)
    for k in range(wl.K):
        E[k] = _to_dtype(_normal([seed_e, k], (wl.V + 1, wl.H)), wl.dtype)
    Et = None
    if wl.V_text > 0:
        Et = np.empty((wl.V_text, wl.H), dtype=edt)
        blk = 4096
        for b in range(0, wl.V_text, blk):
            rows = min(blk, wl.V_text - b)
            Et[b:b + rows] = _to_dtype(_normal([seed_e, 1000, b // blk], (rows, wl.H)), wl.dtype)
    return dict(E=E, E_text=Et)


def make_token_sets(wl: Workload, n: int, layout: dict, seed: int = SEED_E) -> np.ndarray:
    """n sets of one step's tokens, int32 [n][R][K]: uniform audio ids in
    [0, V) per stream, a uniform text id in [0, V_text) in column 0 of text
    rows (the rest 0), from default_rng([seed, 2000])."""
    rng = np.random.default_rng([seed, 2000])
    tok = rng.integers(0, wl.V, size=(n, wl.R, wl.K), dtype=np.int32)
    text = np.asarray(layout["row_kind"]) == ROW_TEXT
    if text.any():
        tok[:, text, :] = 0
        tok[:, text, 0] = rng.integers(0, wl.V_text, size=(n, int(text.sum())), dtype=np.int32)
    return tok


def row_layout(wl: Workload, seed_perm: int = SEED_PERM) -> dict:
    """Row structure of the batch: pair_map, row_kind, rng_key, grid_slot and the
    permutation perm (physical row p holds logical row perm[p])."""
    R = wl.R
    kind = np.empty(R, np.uint8)
    pmap = np.full(R, -1, np.int32)
    key = np.empty(R, np.uint64)
    slot = np.full(R, -1, np.int32)
    for i in range(wl.n_pairs):
        c, u = 2 * i, 2 * i + 1
        kind[c], kind[u] = ROW_COND, ROW_UNCOND
        pmap[c], pmap[u] = u, c
        key[c] = key[u] = i
        slot[c] = i
    base = 2 * wl.n_pairs
    for j in range(wl.n_solo):
        kind[base + j] = ROW_SOLO
        key[base + j] = wl.n_pairs + j
        slot[base + j] = wl.n_pairs + j
    base += wl.n_solo
    for j in range(wl.n_text):
        kind[base + j] = ROW_TEXT
        key[base + j] = wl.n_pairs + wl.n_solo + j
    perm = np.arange(R, dtype=np.int64)
    if wl.shuffle:
        perm = np.random.default_rng(seed_perm).permutation(R)
        inv = np.empty(R, np.int64)
        inv[perm] = np.arange(R)
        pm = pmap[perm]
        pmap = np.where(pm >= 0, inv[np.maximum(pm, 0)], -1).astype(np.int32)
        kind, key, slot = kind[perm], key[perm], slot[perm]
    return dict(pair_map=pmap, row_kind=kind, rng_key=key, grid_slot=slot, perm=perm)


def make_hidden(wl: Workload, t: int, perm=None, seed_h: int = SEED_H) -> np.ndarray:
    """hidden[R][H] of decode step t (physical row order)."""
    h = _to_dtype(_normal([seed_h, t], (wl.R, wl.H)), wl.dtype)
    if perm is not None:
        h = h[np.asarray(perm)]
    return np.ascontiguousarray(h)


def make_batch(wl: Workload, t: int, layout: dict | None = None, seed_h: int = SEED_H) -> dict:
    """Everything a decode step of the head reads besides the weights (host arrays)."""
    if layout is None:
        layout = row_layout(wl)
    R = wl.R
    return dict(
        hidden=make_hidden(wl, t, layout["perm"], seed_h),
        pair_map=layout["pair_map"], row_kind=layout["row_kind"], rng_key=layout["rng_key"],
        grid_slot=layout["grid_slot"],
        cfg_w=np.full(R, wl.cfg_w, np.float32),
        temperature=np.full(R, wl.temperature, np.float32),
        top_k=np.full(R, wl.top_k, np.int32),
        top_p=np.full(R, wl.top_p, np.float32),
        step=np.full(R, t, np.int32),
        n_frames=np.full(R, wl.frames, np.int32),
    )


def make_scores(Rs: int, N: int, t: int, sigma: float = 1.0, quantum: float = 0.0,
                seed: int = 77) -> np.ndarray:
    """Ready-made fp32 scores [Rs][N] for driving the sampling stage on its own:
    N(0, sigma^2) from default_rng([seed, t]); with quantum > 0, rounded to
    multiples of it so that exact ties occur."""
    s = np.random.default_rng([seed, t]).standard_normal((Rs, N)) * sigma
    if quantum > 0:
        s = np.round(s / quantum) * quantum
    return np.ascontiguousarray(s, dtype=np.float32)
