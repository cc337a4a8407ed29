"""Throughput of the multi-codebook decode head on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--weight-copies C]

A step is one pass of the whole hot path (mcd_head_step: head projections with
the fused CFG merge and temperature, text-head argmax, selection, Gumbel-max
draw, pads, companion copy, frame-grid scatter) over one batch of the workload.
Inputs are resident in HBM before timing; the timed loop walks steady-state
decode steps of the workload (every stream has a frame, so no step is cheapened
by start-up or drain pads), each with its own hidden states and step index,
and rotates through several copies of the weights so that they stream from HBM
rather than from the 256 MB Infinity Cache.

Prints one JSON line:
  * value: client-visible codebook tokens per second of the headline workload
    (weight_streaming: sampled rows x codebooks per step / step time);
  * roofline: the head projection kernel (the dominant one), its time taken
    in-step with HIP events between the projection and the sampler;
  * legs: the same measurement on the MFMA-regime mixed batch and on the CFG
    ablation (cfg_on / cfg_off, and their throughput ratio);
  * cpu_baseline: the CPU oracle timed on a bounded sample of the headline
    workload (one decode step), and parity: that sample's oracle tokens and
    merged scores against the GPU's for the same step.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2516.6      # MI355X dense bf16 MFMA (256 CU x 2.4 GHz x 4096 flop/clk)
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 vector
MALL_BYTES = 256 * 2**20       # Infinity Cache
COPY_PROBE_BYTES = 2**30       # --copy-probe: one plain device copy of this many bytes

# HBM traffic of the head projection kernel per launch, from two rocprofv3 --pmc
# passes (FETCH_SIZE, then WRITE_SIZE) over `bench.py --copy-probe`, each
# counter scaled by what it reads for the probe's plain copy of known size.
# Valid only for the kernel sources it was taken on (sha256 over the listed
# files); a changed kernel reports traffic null until the counters are taken
# again.
CSRC = os.path.join(ROOT, "paper_2607_02119_amd", "csrc")
MEASURED_TRAFFIC = {
    # workload: dict(sources=[...], sha256=..., fetch_bytes=..., write_bytes=..., profile=...)
    "weight_streaming": dict(
        sources=["k_stream.hip", "stream_tile.h", "gemm_common.h"],
        sha256="94f40a0df98a9499182f4752cf032ebceebce6b0cc4b38870b52a7302311baa4",
        fetch_bytes=277193728, write_bytes=8388608,
        profile="profiles/head_step_weight_streaming.md"),
}


def algorithmic(wl):
    """Bytes and flops the head projection must move / do per step (one launch)."""
    eb = wl.elem_bytes()
    Mg = 2 * wl.n_pairs + wl.n_solo
    w_bytes = wl.N * wl.H * eb + wl.V_text * wl.H * eb
    hid = wl.R * wl.H * eb
    flops = 2.0 * Mg * wl.N * wl.H + 2.0 * wl.n_text * wl.V_text * wl.H
    return dict(weight_bytes=w_bytes, hidden_bytes=hid, bytes=w_bytes + hid, flops=flops,
                scores_bytes=4 * wl.Rs * wl.N)


def sources_sha256(names):
    import hashlib
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(CSRC, n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def k1_traffic(workload):
    """Measured HBM bytes per head-projection launch, or None if not measured
    for this workload or the kernel sources changed since."""
    m = MEASURED_TRAFFIC.get(workload)
    if not m or sources_sha256(m["sources"]) != m["sha256"]:
        return None
    return m["fetch_bytes"] + m["write_bytes"]


def graph_per_launch(torch, fn, reps=50, replays=8):
    """Mean duration of fn(i)'s launch, back to back on the GPU: `reps` calls
    (i = 0 .. reps - 1) captured in one HIP graph, replayed `replays` times between HIP events, so
    the host's per-call cost (the ctypes call) is not in the figure.  fn
    launches on torch's current stream, which is the capture stream while the
    graph is recorded; it must allocate nothing."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn(0)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(reps):
            fn(i)
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(replays):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (reps * replays)


def copy_probe(torch):
    """A plain device copy of known size (read and write COPY_PROBE_BYTES each),
    the calibration point for the FETCH_SIZE / WRITE_SIZE counters."""
    n = COPY_PROBE_BYTES // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def host_cpu():
    """The host's CPU model and the cores this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return model, os.cpu_count(), usable


GAP_TOL, TOPK_TOL, TOPP_TOL = 1e-3, 1e-4, 1e-5   # the oracle's near-tie classes
SCORE_TOL_BF16 = 1e-2


def cpu_baseline(wl, t, gpu, budget_s=15.0):
    """The CPU oracle (single-threaded, fp64) on a bounded sample of the
    workload: whole Main/Companion pairs (or solo rows) of decode step t, added
    until about budget_s seconds of CPU work.  Returns (baseline, parity): the
    oracle's codebook tokens per second, and its tokens and merged scores for
    those rows compared with the GPU's step t (gpu: tokens [R][K] and scores
    [Rs][N] of the same step, plan_rows[s] = physical row of sampled index s)."""
    import oracle
    from paper_2607_02119_amd import inputs

    lay = inputs.row_layout(wl)
    head = inputs.make_weights(wl)
    b = inputs.make_batch(wl, t, lay)
    kinds = lay["row_kind"]
    sampled_index = {r: s for s, r in enumerate(gpu["plan_rows"])}
    units = []   # lists of physical rows forming one sampled request
    for r in range(wl.R):
        if kinds[r] == inputs.ROW_COND:
            units.append([r, int(lay["pair_map"][r])])
        elif kinds[r] == inputs.ROW_SOLO:
            units.append([r])
    done_rows, tokens, elapsed = [], 0, 0.0
    par = dict(positions=0, mismatches=0, exempt={"gap": 0, "topk": 0, "topp": 0},
               unexplained=0, flagged={"gap": 0, "topk": 0, "topp": 0}, score_rel_err=0.0)
    for u in units:
        rows = u
        inv = {x: i for i, x in enumerate(rows)}
        sub = {k: (v[rows] if isinstance(v, np.ndarray) and v.shape[:1] == (wl.R,) else v)
               for k, v in b.items()}
        sub["pair_map"] = np.array([inv[p] if p >= 0 else -1 for p in b["pair_map"][rows]],
                                   np.int32)
        t0 = time.perf_counter()
        o = oracle.head_step(head, sub, seed=0, gap_tol=GAP_TOL, topk_tol=TOPK_TOL,
                             topp_tol=TOPP_TOL)
        elapsed += time.perf_counter() - t0
        tokens += wl.K
        done_rows += rows
        # parity of these rows against the GPU's step
        g = gpu["tokens"][rows]
        f = o["flags"].astype(np.int64)
        bad = g != o["tokens"]
        par["positions"] += int(g.size)
        par["mismatches"] += int(bad.sum())
        for name, bit in (("gap", oracle.FLAG_GAP_SMALL), ("topp", oracle.FLAG_TOPP_EDGE),
                          ("topk", oracle.FLAG_TOPK_EDGE)):
            par["flagged"][name] += int(((f & bit) > 0).sum())
        gap = bad & ((f & oracle.FLAG_GAP_SMALL) > 0)
        topp = bad & ~gap & ((f & oracle.FLAG_TOPP_EDGE) > 0)
        topk = bad & ~gap & ~topp & ((f & oracle.FLAG_TOPK_EDGE) > 0)
        par["exempt"]["gap"] += int(gap.sum())
        par["exempt"]["topp"] += int(topp.sum())
        par["exempt"]["topk"] += int(topk.sum())
        par["unexplained"] += int((bad & ~gap & ~topp & ~topk).sum())
        gs = gpu["scores"][sampled_index[rows[0]]].astype(np.float64)
        os_ = o["scores"][0]
        edges = np.concatenate([[0], np.cumsum(wl.stream_sizes)])
        for k in range(wl.K):
            gk, ok = gs[edges[k]:edges[k + 1]], os_[edges[k]:edges[k + 1]]
            den = max(float(np.abs(ok).max()), 1e-300)
            par["score_rel_err"] = max(par["score_rel_err"],
                                       float(np.abs(gk - ok).max()) / den)
        if elapsed >= budget_s:
            break
    model, n_cpu, usable = host_cpu()
    base = dict(value=tokens / elapsed, unit="codebook tokens/s", cores=1, kind="oracle",
                sample=f"decode step {t}: {len(done_rows)} of {wl.R} rows "
                       f"({tokens} codebook tokens), {elapsed:.1f} s single-threaded fp64",
                host_cpu=model, nproc=n_cpu, usable_cores=usable)
    par.update(workload=wl.name, step=t, rows_checked=len(done_rows),
               tolerances={"gap": GAP_TOL, "topk": TOPK_TOL, "topp": TOPP_TOL},
               score_tol=SCORE_TOL_BF16 if wl.dtype == "bf16" else 1e-5,
               score_rel_err=float(f"{par['score_rel_err']:.3e}"),
               rule="tokens bit-exact except where the oracle's top-2 perturbed gap < 1e-3 "
                    "(exempt.gap); exempt.topk / exempt.topp are mismatches at a top-k margin "
                    "< 1e-4 or a top-p boundary within 1e-5, reported as departures")
    return base, par


# Stand-in backbone of the co-scheduling simulation: a memory-bound decoder
# step of an 8B-parameter model with grouped KV heads (36 layers, 8 KV heads
# of 128 dimensions): its bf16 weights once per step, and the bf16 K and V of
# every context token of every row.
STANDIN_WEIGHT_BYTES = 16.4e9
STANDIN_KV_BYTES_PER_TOKEN = 36 * 8 * 128 * 2 * 2


def cosched(args, torch):
    """Paired co-scheduling over a stand-in backbone (closed loop, one GPU).

    The library's host scheduler plans every step; a stand-in backbone step
    reads the bytes such a step reads (weights, and the K/V of every context
    token); the head step (K1 + K2 on this library's kernels) runs on the
    step's decoding rows, with hidden states from a fixed random pool.  CFG on:
    `--cosched-requests` / 2 requests with w = 3 (Main + Companion); CFG off:
    as many solo requests as rows.  Each side keeps its requests in flight
    (a finished request is replaced at once), runs `--warmup` steps, then times
    `--cosched-steps` steps after `--cosched-warmup`.  Prints one JSON line with
    both sides and their ratio."""
    import numpy as np
    from paper_2607_02119_amd import mcd

    H, K, V, V_text, D = 4096, 8, 4096, 151936, 7
    rows = args.cosched_requests
    dev = "cuda"
    gen = torch.Generator(device=dev)
    gen.manual_seed(17)
    W = (torch.randn((K, V, H), generator=gen, device=dev) * 0.02).to(torch.bfloat16)
    W_text = (torch.randn((V_text, H), generator=gen, device=dev) * 0.02).to(torch.bfloat16)
    head = mcd.Head(W, delays=np.arange(K, dtype=np.int32), pad_id=V, W_text=W_text)
    pool = (torch.randn((rows, H), generator=gen, device=dev)).to(torch.bfloat16)
    F_max = 320
    scores = torch.empty((rows, K * V), dtype=torch.float32, device=dev)
    tokens = torch.empty((rows, K), dtype=torch.int32, device=dev)
    grid = torch.full((rows, K, F_max), -1, dtype=torch.int32, device=dev)
    modality = torch.empty(rows, dtype=torch.uint8, device=dev)
    workspace = head.workspace(rows, dev)
    # 8 GiB read by the stand-in in rows of 8 KiB: a row-wise fp32 sum streams
    # it at about 6.4 TB/s here (a flat bf16 reduction reaches only 2 TB/s)
    buf = torch.zeros((1 << 20, 2048), dtype=torch.float32, device=dev)

    def backbone(nbytes):
        n = int(nbytes) // 8192
        while n > 0:
            k = min(n, buf.shape[0])
            buf[:k].sum(dim=1)
            n -= k

    rng = np.random.default_rng(5)

    def new_request(s, cfg_w):
        # TTS-like requests: a prompt, a text preamble, then 2-6 s of audio at 50 frames/s
        return s.submit(cfg_w, int(rng.integers(100, 401)), int(rng.integers(100, 401)),
                        int(rng.integers(100, 301)))

    def run(cfg_on):
        n_req = rows // 2 if cfg_on else rows
        s = mcd.Scheduler(rows, 8192, 16, D, max_requests=2 * n_req)
        info = {}
        for _ in range(n_req):
            new_request(s, 3.0 if cfg_on else 1.0)
        client, frames, host_s = 0, 0, 0.0
        stream = torch.cuda.current_stream()
        t0 = None
        warm, steps = args.cosched_warmup, args.cosched_steps
        for it in range(warm + steps):
            if it == warm:
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                client, frames, host_s = 0, 0, 0.0
            h0 = time.perf_counter()
            b = s.plan()
            host_s += time.perf_counter() - h0
            backbone(STANDIN_WEIGHT_BYTES + STANDIN_KV_BYTES_PER_TOKEN *
                     float(np.sum(b["row_context"]) + np.sum(b["row_tokens"])))
            R = b["R"]
            if R:
                kinds = b["row_kind"]
                plan = head.plan(b["pair_map"], kinds, dev)
                up = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
                rk = b["row_req"][b["head_row"]].astype(np.uint64)
                mcd.mcd_head_step(
                    head.handle, stream=stream, R=R, counts=plan.counts, plan=plan.dev,
                    hidden=pool[:R], cfg_w=up(b["cfg_w"]),
                    temperature=up(np.ones(R, np.float32)),
                    top_k=up(np.full(R, 50, np.int32)), top_p=up(np.ones(R, np.float32)),
                    rng_key=up(rk), step=up(b["step"]), n_frames=up(b["n_frames"]),
                    grid_slot=up(b["grid_slot"]), seed=1234, tokens_out=tokens,
                    frame_grid=grid, n_slots=rows, F_max=F_max, scores=scores,
                    workspace=workspace, modality_out=modality)
                main = kinds != mcd.MCD_ROW_UNCOND
                client += int(np.sum(main))
                frames += int(np.sum(main & (kinds != mcd.MCD_ROW_TEXT)))
            h0 = time.perf_counter()
            fin = s.commit()
            host_s += time.perf_counter() - h0
            for _ in fin:
                new_request(s, 3.0 if cfg_on else 1.0)
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        st = mcd.mcd_read_device_status(workspace)
        info.update(requests_in_flight=n_req, ms_per_step=round(el / steps * 1e3, 3),
                    client_tokens_per_s=round(client / el, 1),
                    audio_steps_per_s=round(frames / el, 1),
                    host_scheduler_us_per_step=round(host_s / steps * 1e6, 2),
                    device_status=st)
        return info

    on = run(True)
    print(f"cosched: CFG on done, {on['ms_per_step']} ms per step", file=sys.stderr, flush=True)
    off = run(False)
    print(f"cosched: CFG off done, {off['ms_per_step']} ms per step", file=sys.stderr, flush=True)
    print(json.dumps({
        "metric": "co-scheduled client decode tokens/s, CFG on / off",
        "value": round(on["client_tokens_per_s"] / off["client_tokens_per_s"], 4),
        "unit": "ratio", "higher_is_better": True, "n_gpus": 1, "steps": args.cosched_steps,
        "warmup": args.cosched_warmup, "data": "synthetic",
        "config": {"workload": f"cosched: {rows} rows, budget 8192, prompt 100-400, text "
                               "100-400, frames 100-300, K 8 x V 4096, text head 151936, "
                               "H 4096, bf16",
                   "stand_in": {"weight_bytes": STANDIN_WEIGHT_BYTES,
                                "kv_bytes_per_token": STANDIN_KV_BYTES_PER_TOKEN}},
        "cfg_on": on, "cfg_off": off}))


class HipEvents:
    """Timing events without the system-scope fence (hipEventDisableSystemFence):
    a default event's fence writes back and invalidates the caches when it
    completes, which costs microseconds and slows the kernel after it; these
    only take the timestamps.  Created and read through the HIP runtime that
    torch has loaded."""
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, n):
        import ctypes
        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.c_void_p, ctypes.c_uint]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            rc = self.hip.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE)
            if rc != 0:
                raise RuntimeError(f"hipEventCreateWithFlags: {rc}")
            self.ev.append(e)

    def record(self, i, stream):
        rc = self.hip.hipEventRecord(self.ev[i], self.ct.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord: {rc}")

    def ms(self, i, j):
        out = self.ct.c_float()
        rc = self.hip.hipEventElapsedTime(self.ct.byref(out), self.ev[i], self.ev[j])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime: {rc}")
        return out.value

    def close(self):
        for e in self.ev:
            self.hip.hipEventDestroy(e)
        self.ev = []


class Leg:
    """One workload resident on the GPU, timed over its steady-state decode
    steps (every stream has a frame: no start-up or drain pads), each step with
    its own hidden states and step index, rotating weight copies."""

    def __init__(self, torch, wl, args, weights=None):
        from paper_2607_02119_amd import harness

        self.torch, self.wl, self.args = torch, wl, args
        self.alg = algorithmic(wl)
        self.copies = args.weight_copies or max(1, math.ceil(3 * MALL_BYTES /
                                                             self.alg["weight_bytes"]))
        self.dw = harness.DeviceWorkload(wl, weight_copies=self.copies, weights=weights)
        live = wl.steps - 2 * wl.max_delay
        self.n_hidden = max(1, min(live, args.steps + args.warmup, args.max_hidden_steps))
        self.t0 = wl.max_delay
        self.dw.load_hidden(range(self.t0, self.t0 + self.n_hidden))
        self.stream = torch.cuda.current_stream()

    def step_of(self, i):
        return self.t0 + i % self.n_hidden, i % self.n_hidden, i % self.copies

    def run(self, i, st):
        t, h, c = self.step_of(i)
        self.dw.run_step(t, hidden_index=h, copy=c, stream=st)

    def logits(self, i, st):
        t, h, c = self.step_of(i)
        self.dw.run_logits(t, hidden_index=h, copy=c, stream=st)

    def sample(self, i, st):
        t, _, c = self.step_of(i)
        self.dw.run_sample(t, copy=c, stream=st)

    def measure(self, min_steps=0, min_warmup=0):
        """Warm-up, then the timed loop of whole steps (value); then the
        projection (mcd_head_logits) alone over the same steps, back to back:
        its launch time, and the sampler's as the rest of the step; then the
        steps again with a timing event after each of the two kernels (no cache
        fence), reported beside them: on some machines each event adds
        command-processor time, so that split can be longer than the step.
        All events are recorded on the launch stream."""
        torch, args = self.torch, self.args
        warmup, steps = max(args.warmup, min_warmup), max(args.steps, min_steps)
        for i in range(warmup):
            self.run(i, self.stream)
        torch.cuda.synchronize()
        status = self.dw.status()
        calls = [warmup + i for i in range(steps)]
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(self.stream)
        for i in calls:
            self.run(i, self.stream)
        b.record(self.stream)
        torch.cuda.synchronize()
        ms_step = a.elapsed_time(b) / len(calls)
        status |= self.dw.status()
        # the projection alone, back to back over the same steps (device-bound:
        # a launch takes far longer than the host needs to issue the next)
        a.record(self.stream)
        for i in calls:
            self.logits(i, self.stream)
        b.record(self.stream)
        torch.cuda.synchronize()
        self.ms_k1_loop = a.elapsed_time(b) / len(calls)
        n = len(calls)
        ev = HipEvents(2 * n + 1)
        torch.cuda.synchronize()
        ev.record(0, self.stream)
        for j, i in enumerate(calls):
            self.logits(i, self.stream)
            ev.record(2 * j + 1, self.stream)
            self.sample(i, self.stream)
            ev.record(2 * j + 2, self.stream)
        torch.cuda.synchronize()
        k1 = float(np.mean([ev.ms(2 * j, 2 * j + 1) for j in range(n)]))
        k2 = float(np.mean([ev.ms(2 * j + 1, 2 * j + 2) for j in range(n)]))
        split_step = ev.ms(0, 2 * n) / n
        ev.close()
        status |= self.dw.status()
        self.ms_step, self.ms_k1, self.ms_k2, self.ms_split = ms_step, k1, k2, split_step
        self.status = status
        return self

    def summary(self):
        wl, alg = self.wl, self.alg
        t = self.ms_step * 1e-3
        return {
            "workload": wl.name, "rows": wl.R, "cfg_pairs": wl.n_pairs, "solo_rows": wl.n_solo,
            "text_rows": wl.n_text, "K": wl.K, "V": wl.V, "V_text": wl.V_text,
            "ms_per_step": round(self.ms_step, 5),
            "codebook_tokens_per_s": round(wl.Rs * wl.K / t, 1),
            "text_tokens_per_s": round(wl.n_text / t, 1),
            "us_k1": round(self.ms_k1_loop * 1e3, 2),
            "us_k2": round((self.ms_step - self.ms_k1_loop) * 1e3, 2),
            "split_events": {"us_k1": round(self.ms_k1 * 1e3, 2),
                             "us_k2": round(self.ms_k2 * 1e3, 2),
                             "us_step": round(self.ms_split * 1e3, 2)},
            "k1_mfma_frac": round(alg["flops"] / (self.ms_k1_loop * 1e-3) / 1e12 /
                                  BF16_PEAK_TFLOPS, 4),
            "k1_hbm_frac": round(alg["bytes"] / (self.ms_k1_loop * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "step_mfma_frac": round(alg["flops"] / t / 1e12 / BF16_PEAK_TFLOPS, 4),
            "step_hbm_frac": round(alg["bytes"] / t / 1e9 / HBM_PEAK_GBS, 4),
            "weight_copies": self.copies, "device_status": self.status,
        }

    def free(self):
        self.dw = None
        self.torch.cuda.synchronize()
        self.torch.cuda.empty_cache()


def parity_step(leg):
    """The whole batch at one steady-state step on the GPU (after the timed
    loops), for the CPU oracle's comparison: tokens and merged scores."""
    torch = leg.torch
    t = leg.wl.K + 1
    if not (leg.t0 <= t < leg.t0 + leg.n_hidden):
        leg.dw.load_hidden([t])
        hi = 0
    else:
        hi = t - leg.t0
    leg.dw.tokens.fill_(-1)
    leg.dw.run_step(t, hidden_index=hi, copy=0, stream=leg.stream)
    torch.cuda.synchronize()
    return t, dict(tokens=leg.dw.tokens.cpu().numpy(), scores=leg.dw.scores.cpu().numpy(),
                   plan_rows=[r for r, _ in leg.dw.plan.sampled_rows()])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default="weight_streaming")
    ap.add_argument("--max-hidden-steps", type=int, default=64,
                    help="distinct decode steps (hidden states) the timed loop cycles through")
    ap.add_argument("--no-legs", action="store_true",
                    help="time only the headline workload (not mfma_mixed, cfg_on, cfg_off)")
    ap.add_argument("--no-next-input", action="store_true",
                    help="skip the timing of the next-step input kernel")
    ap.add_argument("--weight-copies", type=int, default=0,
                    help="weight copies rotated per step (0: enough to exceed 3x the MALL)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--copy-probe", action="store_true",
                    help="run a plain 1 GiB device copy first (counter calibration)")
    ap.add_argument("--cosched", action="store_true",
                    help="run the paired co-scheduling simulation instead of the head step")
    ap.add_argument("--cosched-requests", type=int, default=512,
                    help="rows of the co-scheduled batch")
    ap.add_argument("--cosched-steps", type=int, default=1500)
    ap.add_argument("--cosched-warmup", type=int, default=600,
                    help="untimed steps first, so that the requests in flight are at all stages")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the head stage is measured on one GPU)", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.cosched:
        torch.cuda.set_device(0)
        cosched(args, torch)
        return

    from paper_2607_02119_amd import harness, inputs

    def note(msg):
        print(msg, file=sys.stderr, flush=True)

    torch.cuda.set_device(0)
    if args.copy_probe:
        copy_probe(torch)
    wl = inputs.WORKLOADS[args.workload]
    alg = algorithmic(wl)
    leg = Leg(torch, wl, args).measure()
    note(f"{wl.name}: {leg.ms_step * 1e3:.2f} us/step")
    head = leg.summary()
    status = leg.status

    # the next row of the path: the next-step input built from the last
    # step's tokens (sum of the K stream embeddings per row), timed alone
    next_input = None
    if not args.no_next_input:
        dw = leg.dw
        dw.load_embeddings()
        # a different set of tokens per launch, so that the embedding rows
        # come from HBM as they do when each step's tokens are new
        tok_sets = harness.to_device(inputs.make_token_sets(wl, 50, dw.layout))
        ms_ni = graph_per_launch(torch, lambda i: dw.run_next_input(tok_sets[i]), reps=50)
        status |= dw.status()
        esz = 2 if wl.dtype == "bf16" else 4
        ni_bytes = ((2 * wl.n_pairs + wl.n_solo) * wl.K * wl.H + wl.n_text * wl.H
                    + wl.R * wl.H) * esz
        ni_gbs = ni_bytes / (ms_ni * 1e-3) / 1e9
        next_input = {"kernel": "next_input_kernel (mcd_next_input)", "bound": "hbm",
                      "us_per_launch": round(ms_ni * 1e3, 2), "algorithmic_bytes": ni_bytes,
                      "achieved": round(ni_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                      "frac": round(ni_gbs / HBM_PEAK_GBS, 4)}
    par_t, par_gpu = parity_step(leg)
    status |= leg.dw.status()
    leg.free()

    # the other legs of the metric: the MFMA regime (mixed batch) and the CFG
    # ablation (the same 512 rows as 256 CFG pairs and as 512 solo rows)
    legs = {}
    if not args.no_legs:
        for name in ("mfma_mixed", "cfg_on", "cfg_off"):
            other = inputs.WORKLOADS[name]
            weights = legs.pop("_cfg_weights", None) if name == "cfg_off" else None
            lg = Leg(torch, other, args, weights=weights).measure(min_steps=100, min_warmup=20)
            note(f"{name}: {lg.ms_step * 1e3:.2f} us/step")
            legs[name] = lg.summary()
            if name == "cfg_on":
                legs["_cfg_weights"] = lg.dw.host_head
            lg.free()
        legs.pop("_cfg_weights", None)
        on, off = legs["cfg_on"], legs["cfg_off"]
        legs["cfg_ratio"] = {
            "client_tokens": round(on["codebook_tokens_per_s"] / off["codebook_tokens_per_s"], 4),
            "rows_processed": round(off["ms_per_step"] / on["ms_per_step"], 4),
            "paper_context": "0.80: whole-system decode tok/s with / without CFG, Bagpiper on "
                             "vLLM, 1x H100 80 GB (Table 4); a context figure, not a target"}

    value = wl.Rs * wl.K / (leg.ms_step * 1e-3)
    ms_k1 = leg.ms_k1_loop
    mfma_bound = alg["flops"] / (BF16_PEAK_TFLOPS * 1e12) > alg["bytes"] / (HBM_PEAK_GBS * 1e9)
    if mfma_bound:
        ach = alg["flops"] / (ms_k1 * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=round(ach, 2), peak=BF16_PEAK_TFLOPS, unit="TFLOP/s",
                    frac=round(ach / BF16_PEAK_TFLOPS, 4))
    else:
        ach = alg["bytes"] / (ms_k1 * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=round(ach, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(ach / HBM_PEAK_GBS, 4))
    roof.update(traffic=k1_traffic(wl.name), kernel="head_gemm (mcd_head_logits)",
                us_per_launch=round(ms_k1 * 1e3, 2),
                measured="HIP events around back-to-back projection launches over the "
                         "timed steps (in-step events can add command-processor time: "
                         "step.split_events)",
                algorithmic_bytes=alg["bytes"], algorithmic_flops=alg["flops"])
    out = {
        "metric": "codebook tokens/sec per CFG-paired decode step",
        "value": round(value, 1),
        "unit": "codebook tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(leg.ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded; shapes of the workload table)",
        "config": {"workload": wl.name, "rows": wl.R, "cfg_pairs": wl.n_pairs,
                   "solo_rows": wl.n_solo, "text_rows": wl.n_text, "H": wl.H, "K": wl.K,
                   "V": wl.V, "V_text": wl.V_text, "cfg_w": wl.cfg_w,
                   "temperature": wl.temperature, "top_k": wl.top_k, "top_p": wl.top_p,
                   "weight_copies": leg.copies, "decode_steps": f"{leg.t0}..{leg.t0 + leg.n_hidden - 1}",
                   "parallelism": "single GPU"},
        "roofline": roof,
        "step": {"hbm_frac": head["step_hbm_frac"], "mfma_frac": head["step_mfma_frac"],
                 "us_k1": head["us_k1"], "us_k2": head["us_k2"],
                 "split_events": head["split_events"], "device_status": status},
    }
    if legs:
        out["legs"] = legs
    if next_input is not None:
        out["next_input"] = next_input
    if not args.no_cpu_baseline:
        base, par = cpu_baseline(wl, par_t, par_gpu, args.cpu_budget)
        out["cpu_baseline"] = base
        out["parity"] = par
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
