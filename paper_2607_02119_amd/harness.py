"""Device-side driver of a synthetic workload: uploads the seeded inputs of
``inputs`` to HBM and runs decode steps through the C ABI (``mcd``).

Used by the GPU tests, the smoke check and the benchmark.  It only moves bytes
and calls the library; every step of the method runs in libmcd's kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import inputs, mcd


def to_device(a: np.ndarray, device="cuda") -> torch.Tensor:
    """numpy -> device tensor; uint16 arrays are bf16 bit patterns."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    if a.dtype == np.uint64:
        return torch.from_numpy(a.view(np.int64)).to(device)
    if a.dtype == np.uint8:
        return torch.from_numpy(a).to(device)
    return torch.from_numpy(a).to(device)


class DeviceWorkload:
    """A workload resident on the GPU: weights (optionally several copies, so a
    timed loop can rotate through more bytes than the 256 MB Infinity Cache
    holds), the batch layout, per-step hidden states and the output buffers."""

    def __init__(self, wl: inputs.Workload, device="cuda", weight_copies=1, steps=None,
                 weights=None, layout=None, seed=inputs.SEED_SAMPLING):
        self.wl, self.device, self.seed = wl, device, seed
        self.host_head = weights if weights is not None else inputs.make_weights(wl)
        self.layout = layout if layout is not None else inputs.row_layout(wl)
        hh = self.host_head
        W = to_device(hh["W"], device)
        Wt = None if hh["W_text"] is None else to_device(hh["W_text"], device)
        b = None if hh.get("bias") is None else to_device(hh["bias"], device)
        vs, tt = hh.get("V_stream"), hh.get("T_text", 0)
        self.heads = [mcd.Head(W, hh["delays"], hh["pad_id"], b, Wt, vs, tt)]
        for _ in range(1, weight_copies):
            self.heads.append(mcd.Head(W.clone(), hh["delays"], hh["pad_id"], b,
                                       None if Wt is None else Wt.clone(), vs, tt))
        self.plan = self.heads[0].plan(self.layout["pair_map"], self.layout["row_kind"], device)
        R, K = wl.R, wl.K
        b0 = inputs.make_batch(wl, 0, self.layout)
        self.params = {name: to_device(b0[name], device)
                       for name in ("cfg_w", "temperature", "top_k", "top_p", "rng_key",
                                    "n_frames", "grid_slot")}
        self.steps = wl.steps if steps is None else steps
        self.step_tab = torch.arange(self.steps, dtype=torch.int32, device=device)[:, None] \
            .expand(self.steps, R).contiguous()
        self.hidden = None
        self.tokens = torch.full((R, K), -1, dtype=torch.int32, device=device)
        self.modality = torch.full((R,), 255, dtype=torch.uint8, device=device)
        self.grid = torch.full((max(wl.n_slots, 1), K, max(wl.frames, 1)), -1, dtype=torch.int32,
                               device=device)
        self.scores = torch.zeros((max(wl.Rs, 1), wl.N), dtype=torch.float32, device=device)
        self.workspace = self.heads[0].workspace(R, device)

    def load_hidden(self, steps=None):
        """Pre-generate the hidden states of `steps` (default: all) into HBM."""
        steps = range(self.steps) if steps is None else steps
        hs = [inputs.make_hidden(self.wl, t, self.layout["perm"]) for t in steps]
        self.hidden_steps = list(steps)
        self.hidden = to_device(np.stack(hs), self.device)
        return self.hidden

    def set_hidden(self, t_index: int, h: torch.Tensor):
        assert self.hidden is not None
        self.hidden[t_index].copy_(h)

    def step_kwargs(self, t: int, hidden: torch.Tensor, tokens=None, scores=None):
        p = self.params
        return dict(R=self.wl.R, counts=self.plan.counts, plan=self.plan.dev, hidden=hidden,
                    cfg_w=p["cfg_w"], temperature=p["temperature"], top_k=p["top_k"],
                    top_p=p["top_p"], rng_key=p["rng_key"], step=self.step_tab[t],
                    n_frames=p["n_frames"], grid_slot=p["grid_slot"], seed=self.seed,
                    tokens_out=self.tokens if tokens is None else tokens,
                    frame_grid=self.grid, n_slots=self.wl.n_slots, F_max=self.wl.frames,
                    scores=self.scores if scores is None else scores, workspace=self.workspace,
                    modality_out=self.modality)

    def run_step(self, t: int, hidden_index=None, copy=0, stream=None):
        """One decode step at step t with hidden state slot `hidden_index` (default t)."""
        hi = t if hidden_index is None else hidden_index
        mcd.mcd_head_step(self.heads[copy].handle, stream=stream,
                          **self.step_kwargs(t, self.hidden[hi]))

    def run_logits(self, t: int, hidden_index=None, copy=0, stream=None):
        hi = t if hidden_index is None else hidden_index
        mcd.mcd_head_logits(self.heads[copy].handle, stream=stream,
                            **self.step_kwargs(t, self.hidden[hi]))

    def run_sample(self, t: int, copy=0, stream=None):
        mcd.mcd_sample_step(self.heads[copy].handle, stream=stream,
                            **self.step_kwargs(t, None))

    def sample_only(self, t: int, scores: torch.Tensor, stream=None):
        mcd.mcd_sample_step(self.heads[0].handle, stream=stream,
                            **self.step_kwargs(t, None, scores=scores))

    def status(self):
        return mcd.mcd_read_device_status(self.workspace)

    def load_embeddings(self, tables=None):
        """Upload the next-step input's embedding tables (default: the seeded
        ones of the workload) and allocate the output."""
        self.host_emb = tables if tables is not None else inputs.make_embeddings(self.wl)
        self.E = to_device(self.host_emb["E"], self.device)
        Et = self.host_emb["E_text"]
        self.E_text = None if Et is None else to_device(Et, self.device)
        self.row_kind_dev = to_device(np.ascontiguousarray(self.layout["row_kind"]), self.device)
        self.next_in = torch.empty((self.wl.R, self.wl.H), dtype=self.E.dtype, device=self.device)
        return self.next_in

    def run_next_input(self, tokens=None, stream=None):
        """Next-step input of every row from `tokens` (default: the last step's)."""
        mcd.mcd_next_input(self.E, self.tokens if tokens is None else tokens, self.row_kind_dev,
                           self.host_head["pad_id"], self.next_in, E_text=self.E_text,
                           workspace=self.workspace, stream=stream)
        return self.next_in
