"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Tolerances:
  * merged, temperature-divided scores: max over (row, codebook) vectors of
    max|gpu - oracle| / max|oracle| <= 1e-5 for fp32 inputs, 1e-2 for bf16;
  * tokens and frame grids: bit-exact, except at positions the oracle flags as
    ambiguous: top-2 perturbed (or greedy) gap below GAP_TOL, or a top-k / top-p
    boundary within TOPK_TOL / TOPP_TOL.  Those are counted and printed.
"""
import numpy as np
import pytest

import oracle
from paper_2607_02119_amd import inputs
from tests._compare import TokenCheck, say, score_rel_err, subset_batch

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_02119_amd import harness, mcd  # noqa: E402

GAP_TOL = 1e-3
# End to end the GPU scores carry fp32 accumulation error (about 1e-6 relative
# for H = 4096); a top-k or top-p cut whose deciding margin is below these
# bounds can flip legitimately.
TOPK_TOL = 1e-4
TOPP_TOL = 1e-5


def _cpu(t):
    return t.detach().cpu().numpy()


def _oracle_step(dw, t, rows=None):
    b = inputs.make_batch(dw.wl, t, dw.layout)
    if rows is not None:
        b = subset_batch(b, rows)
    return b, oracle.head_step(dw.host_head, b, seed=dw.seed, gap_tol=GAP_TOL, topk_tol=TOPK_TOL,
                               topp_tol=TOPP_TOL)


def _plan_rows(dw, rows=None):
    """Physical row (or its index in `rows`) of every sampled index."""
    out = []
    pos = None if rows is None else {r: i for i, r in enumerate(rows)}
    for r, _ in dw.plan.sampled_rows():
        out.append(r if pos is None else pos.get(r))
    return out


def _check_step(dw, t, tc, rows=None, score_tol=None):
    """Run step t on the GPU (whole batch), the oracle on `rows` (default all)."""
    dw.tokens.fill_(-1)
    dw.run_step(t, hidden_index=dw.hidden_steps.index(t))
    torch.cuda.synchronize()
    g_tok, g_sc = _cpu(dw.tokens), _cpu(dw.scores)
    b, o = _oracle_step(dw, t, rows)
    sel = np.arange(dw.wl.R) if rows is None else np.asarray(rows)
    tc.add(g_tok[sel], o["tokens"], o["flags"], where=f"t={t}")
    # TEXT rows' modality flag (the unmasked argmax past the text ids), except
    # where the two regions' maxima are within the score rounding
    g_mod = _cpu(dw.modality)[sel]
    for i, r in enumerate(sel):
        if dw.layout["row_kind"][r] == inputs.ROW_TEXT and o["modality_gap"][i] >= GAP_TOL:
            assert g_mod[i] == o["modality"][i], (t, int(r))
    if score_tol is not None and dw.wl.Rs:
        err = score_rel_err(g_sc, _plan_rows(dw, None if rows is None else list(sel)), o["scores"],
                            oracle.stream_sizes(dw.host_head))
        say(f"  t={t} score rel err {err:.3e}")
        assert err <= score_tol
    return g_tok, o


# ---------------------------------------------------------------------------
def test_tiny_ref_full_run_tokens_scores_grid():
    """The fp32 tiny reference workload, all 32 steps, every row."""
    wl = inputs.WORKLOADS["tiny_ref"]
    say(f"case tiny_ref R={wl.R} H={wl.H} K={wl.K} V={wl.V}")
    dw = harness.DeviceWorkload(wl)
    dw.load_hidden()
    tc = TokenCheck()
    ora_grid = np.full((wl.n_slots, wl.K, wl.frames), -1, np.int32)
    for t in range(wl.steps):
        b, o = _oracle_step(dw, t)
        oracle.head_step(dw.host_head, b, seed=0, n_slots=wl.n_slots, F_max=wl.frames,
                         frame_grid=ora_grid, want_scores=False)
        _check_step(dw, t, tc, score_tol=1e-5)
    tc.assert_ok("tiny_ref")
    assert tc.mismatch == 0
    g = _cpu(dw.grid)
    assert (ora_grid >= 0).all()
    assert np.array_equal(g, ora_grid)
    assert dw.status() == 0


RAGGED = [
    # name, workload kwargs
    # the largest head the library takes: 32 codebooks of 4096 ids (delays 0..31)
    ("max_k_max_v", dict(H=64, K=32, V=4096, n_pairs=3, n_solo=2, dtype="bf16", top_k=50,
                         cfg_w=2.0, steps=35)),
    ("bf16_ragged_mixed", dict(H=128, K=3, V=37, n_pairs=70, n_solo=5, n_text=3, V_text=300,
                               dtype="bf16", top_k=7, temperature=0.7, steps=6, shuffle=True)),
    ("bf16_topp_two_tiles", dict(H=192, K=2, V=333, n_pairs=20, n_solo=3, dtype="bf16",
                                 top_p=0.9, cfg_w=2.0, steps=4)),
    # H % 256 == 0 and at most 128 rows: the weight-streaming kernel (32/64/128-row tiles)
    ("stream_bm32_text", dict(H=256, K=3, V=37, n_pairs=10, n_solo=5, n_text=3, V_text=300,
                              dtype="bf16", top_k=7, temperature=0.7, steps=5, shuffle=True)),
    ("stream_bm64", dict(H=512, K=2, V=333, n_pairs=25, n_solo=3, n_text=40, V_text=1000,
                         dtype="bf16", top_p=0.9, cfg_w=2.0, steps=4, shuffle=True)),
    # the stream-embedding term (a per-codebook bias) on each kernel path
    ("bias_stream_bm32", dict(H=256, K=3, V=37, n_pairs=10, n_solo=5, n_text=3, V_text=300,
                              dtype="bf16", top_k=7, temperature=0.7, steps=5, shuffle=True,
                              bias=True)),
    ("bias_stream_wide", dict(H=128, K=9, V=3739, n_pairs=20, n_solo=3, dtype="bf16", top_k=20,
                              steps=10, bias=True)),
    ("bias_rows", dict(H=192, K=4, V=256, n_pairs=100, n_solo=100, dtype="bf16", top_p=0.9,
                       cfg_w=2.5, steps=4, bias=True)),
    ("bias_fused_mixed", dict(H=64, K=8, V=4093, n_pairs=100, n_solo=60, n_text=70, V_text=900,
                              dtype="bf16", top_k=15, steps=10, shuffle=True, bias=True)),
    ("bias_f32", dict(H=40, K=3, V=37, n_pairs=3, n_solo=2, n_text=2, V_text=70, dtype="f32",
                      top_k=5, top_p=0.8, steps=5, shuffle=True, bias=True)),
    ("stream_bm128", dict(H=768, K=4, V=129, n_pairs=55, n_solo=3, n_text=100, V_text=515,
                          dtype="bf16", top_k=20, steps=5)),
    # more than one round of 128-column tiles: 256-column streaming tiles with
    # a ragged last tile (audio: 64-row tiles, N % 4 != 0; text: 32-row tiles)
    ("stream_wide_bm64", dict(H=128, K=9, V=3739, n_pairs=20, n_solo=3, n_text=5, V_text=33000,
                              dtype="bf16", top_k=20, temperature=0.9, steps=10, shuffle=True)),
    # 128-row 256-column tiles, fewer slices than weight stages (H = 192)
    ("stream_wide_bm128", dict(H=192, K=9, V=3700, n_pairs=60, n_solo=5, n_text=100,
                               V_text=40000, dtype="bf16", top_p=0.9, cfg_w=2.5, steps=10)),
    # streams of unequal size (one large stream and smaller ones): the
    # streaming kernel with N % 4 != 0, 128-row streaming tiles, and the
    # one-wave-per-vector sampler
    ("unequal_streams_stream", dict(H=128, K=4, V=100, V_stream=(100, 37, 64, 5), n_pairs=6,
                                    n_solo=2, n_text=2, V_text=300, dtype="bf16", top_k=7,
                                    temperature=0.8, steps=6, shuffle=True, bias=True)),
    ("unequal_streams_rows", dict(H=64, K=9, V=2048, V_stream=(2048,) + (1024,) * 8,
                                  n_pairs=100, n_solo=60, dtype="bf16", top_p=0.9, cfg_w=2.5,
                                  steps=10)),
    ("unequal_streams_wave", dict(H=64, K=8, V=1000, V_stream=(1000, 500, 250, 125, 1000, 999, 3, 64),
                                  n_pairs=64, n_solo=80, dtype="bf16", top_k=20, steps=8,
                                  shuffle=True)),
    ("unequal_streams_f32", dict(H=40, K=3, V=37, V_stream=(37, 2, 20), n_pairs=3, n_solo=2,
                                 n_text=1, V_text=70, dtype="f32", top_p=0.8, steps=5)),
    # the text phase's vocabulary mask (text ids [0, T_text)) and the modality
    # inferred from the unmasked argmax, on the streaming, MFMA and fused paths
    ("text_mask_stream", dict(H=256, K=3, V=37, n_pairs=10, n_solo=5, n_text=40, V_text=300,
                              T_text=256, dtype="bf16", top_k=7, steps=5, shuffle=True)),
    ("text_mask_mfma", dict(H=128, K=2, V=40, n_pairs=3, n_solo=2, n_text=150, V_text=3000,
                            T_text=2048, dtype="bf16", top_k=5, steps=3, shuffle=True)),
    ("text_mask_fused", dict(H=64, K=8, V=4093, n_pairs=100, n_solo=60, n_text=70, V_text=900,
                             T_text=64, dtype="bf16", top_k=15, steps=9, shuffle=True)),
    ("text_mask_f32", dict(H=40, K=3, V=37, n_pairs=3, n_solo=2, n_text=4, V_text=70,
                           T_text=32, dtype="f32", top_k=5, steps=4, shuffle=True)),
    # more than 128 audio rows and fewer than 256 tiles of 256 x 256: 128 x 256
    # streaming tiles, row tile by row tile (here three, the last one ragged)
    ("rows_three_row_tiles", dict(H=128, K=3, V=100, n_pairs=150, n_solo=7, dtype="bf16", top_k=10,
                                temperature=0.9, steps=4, shuffle=True)),
    # 2 x 4 and 3 x 8 tiles of 128 x 256 (the second with a ragged row tile):
    # the XCD-aware order
    ("rows_xcd_remap", dict(H=192, K=4, V=256, n_pairs=100, n_solo=56, dtype="bf16", top_p=0.9,
                            cfg_w=2.5, steps=4)),
    ("rows_xcd_remap_ragged", dict(H=256, K=4, V=512, n_pairs=140, n_solo=20, dtype="bf16",
                                   top_k=30, temperature=0.9, steps=5, shuffle=True)),
    # at least 256 tiles of 256 x 256: the wide-tile kernel, ragged N and V % 4 != 0
    ("mfma_wide_tiles", dict(H=64, K=8, V=4093, n_pairs=100, n_solo=60, dtype="bf16",
                             top_k=15, temperature=0.8, steps=10, shuffle=True)),
    # 3 x 64 tiles of 128 x 256 with a ragged last row and column tile (V % 4 != 0)
    ("rows_ragged_columns", dict(H=256, K=4, V=4093, n_pairs=140, n_solo=20, dtype="bf16",
                                 top_k=10, temperature=0.9, steps=3, shuffle=True)),
    # one launch for both projections: 256 tiles of 256 x 256 for the audio
    # rows, then 65..128 text rows in 256-column (or 64-column) streaming tiles
    ("fused_mixed_wide_text", dict(H=64, K=8, V=4093, n_pairs=100, n_solo=60, n_text=70,
                                   V_text=33000, dtype="bf16", top_k=15, temperature=0.8,
                                   steps=10, shuffle=True)),
    ("fused_mixed_narrow_text", dict(H=128, K=8, V=4096, n_pairs=130, n_solo=0, n_text=128,
                                     V_text=515, dtype="bf16", top_p=0.9, cfg_w=2.0, steps=9,
                                     shuffle=True)),
    ("mfma_text_rows", dict(H=128, K=2, V=40, n_pairs=3, n_solo=2, n_text=150, V_text=300,
                            dtype="bf16", top_k=5, steps=3, shuffle=True)),
    # streaming tiles that never straddle two streams (V a multiple of the
    # 64-, 128- and 256-column tile widths), every draw path; a small p so that
    # the first candidate often falls outside the nucleus
    ("aligned_topp_bn64", dict(H=256, K=3, V=256, n_pairs=20, n_solo=7, dtype="bf16", top_p=0.9,
                            cfg_w=2.5, steps=6, shuffle=True)),
    ("aligned_small_p", dict(H=128, K=4, V=512, n_pairs=9, n_solo=6, dtype="bf16", top_p=0.3,
                          temperature=0.7, steps=7, shuffle=True)),
    ("aligned_plain_sampling", dict(H=64, K=2, V=1024, n_pairs=5, n_solo=3, dtype="bf16",
                                 steps=4)),
    ("aligned_topk_text", dict(H=128, K=4, V=512, n_pairs=10, n_solo=5, n_text=6, V_text=700,
                            dtype="bf16", top_k=20, steps=6, shuffle=True)),
    ("aligned_bn128", dict(H=128, K=8, V=4096, n_pairs=3, n_solo=2, dtype="bf16", top_p=0.95,
                        cfg_w=2.0, steps=10)),
    ("aligned_bn256", dict(H=64, K=16, V=4096, n_pairs=4, n_solo=1, dtype="bf16", top_p=0.9,
                        steps=17)),
    ("aligned_greedy", dict(H=64, K=3, V=128, n_pairs=4, n_solo=3, dtype="bf16", temperature=0.0,
                         steps=5)),
    ("wide_topk_owner_draw", dict(H=128, K=3, V=2048, n_pairs=5, n_solo=3, dtype="bf16",
                                  top_k=1000, steps=5, shuffle=True)),
    ("f32_ragged_mixed", dict(H=40, K=3, V=37, n_pairs=3, n_solo=2, n_text=2, V_text=70,
                              dtype="f32", top_k=5, top_p=0.8, steps=5, shuffle=True)),
    ("bf16_greedy", dict(H=64, K=4, V=100, n_pairs=5, n_solo=4, dtype="bf16", temperature=0.0,
                         steps=6)),
    ("bf16_single_row", dict(H=64, K=1, V=1, n_pairs=0, n_solo=1, dtype="bf16", steps=2)),
    ("bf16_only_text", dict(H=64, K=2, V=16, n_pairs=0, n_solo=0, n_text=5, V_text=129,
                            dtype="bf16", steps=2)),
]


@pytest.mark.parametrize("name,kw", RAGGED, ids=[r[0] for r in RAGGED])
def test_ragged_shapes_every_step(name, kw):
    wl = inputs.Workload(name, **kw)
    say(f"case {name} R={wl.R} Mg={2 * wl.n_pairs + wl.n_solo} N={wl.N} text={wl.n_text}")
    dw = harness.DeviceWorkload(wl)
    dw.load_hidden()
    tc = TokenCheck()
    tol = 1e-5 if wl.dtype == "f32" else 1e-2
    for t in range(wl.steps):
        _check_step(dw, t, tc, score_tol=tol)
    tc.assert_ok(name)
    assert dw.status() == 0


def test_wide_tiles_over_more_than_one_wave_of_the_chip():
    """3 x 100 tiles of 256 x 256: more tiles than compute units, so a second
    round of workgroups runs after the first.  The oracle checks rows of every
    row tile (pairs and solo rows)."""
    wl = inputs.Workload("wide_tiles_waves", H=128, K=8, V=3199, n_pairs=300, n_solo=40,
                         dtype="bf16", top_p=0.9, cfg_w=2.5, steps=9, shuffle=True)
    say(f"case wide_tiles_waves R={wl.R} Mg={2 * wl.n_pairs + wl.n_solo} N={wl.N}")
    dw = harness.DeviceWorkload(wl)
    dw.load_hidden()
    sr = list(dw.plan.sampled_rows())
    rows = []
    for s_ in [0, 1, 64, 127, 128, 200, 255, 256, 299, 300, 319, 339]:
        r, c = sr[s_]
        rows += [r] + ([c] if c >= 0 else [])
    tc = TokenCheck()
    for t in (0, 8):
        _check_step(dw, t, tc, rows=sorted(rows), score_tol=1e-2)
    tc.assert_ok("wide_tiles_waves")
    assert dw.status() == 0


SAMPLER = [
    # V, K, Rs, sigma, quantum, temperature, top_k, top_p
    (2048, 8, 16, 3.6, 0.0, 0.9, 50, 1.0),
    (4096, 8, 8, 2.24, 0.0, 1.0, 0, 0.95),
    (1024, 16, 16, 3.6, 0.0, 0.8, 20, 1.0),
    (4096, 2, 4, 1.0, 0.25, 1.0, 50, 0.9),      # heavy ties at both boundaries
    (37, 3, 5, 1.0, 0.5, 1.0, 5, 0.7),
    (1000, 2, 3, 0.0, 0.0, 1.0, 10, 0.5),        # all scores equal
    (4096, 1, 4, 2.0, 0.0, 0.0, 0, 1.0),         # greedy
    (4096, 2, 4, 2.0, 0.0, 1.0, 1, 1.0),         # top-k = 1
    (512, 2, 4, 2.0, 0.0, 1.0, 0, 1e-6),         # tiny p: argmax
    (512, 2, 4, 2.0, 0.0, 1.0, 0, 0.999999),     # p near one
    # no top-k cut: candidates in perturbed-score order tested against the nucleus
    (4096, 4, 4, 2.0, 0.0, 1.0, 0, 1.0),         # plain sampling
    (4096, 4, 8, 1.0, 0.25, 1.0, 0, 0.3),        # small p, heavy ties: several candidates
    (1000, 2, 3, 0.0, 0.0, 1.0, 0, 0.5),         # all scores equal: the nucleus is by id
    (37, 3, 5, 1.0, 0.5, 1.0, 37, 0.7),          # top-k = V is no cut
    # workgroup per vector with two and four groups of ids per thread, over
    # more vectors than compute units
    (2048, 8, 72, 3.6, 0.0, 0.9, 50, 1.0),
    (4096, 8, 72, 2.24, 0.0, 1.0, 0, 0.95),
    # at least 1024 vectors of at most 1024 ids: one wave per vector
    (1024, 16, 64, 3.6, 0.0, 0.8, 20, 1.0),
    (512, 8, 128, 2.24, 0.0, 1.0, 0, 0.95),
    (200, 8, 128, 1.0, 0.25, 1.0, 50, 0.9),      # heavy ties at both boundaries
    (1000, 4, 256, 0.0, 0.0, 1.0, 10, 0.5),      # all scores equal
    (37, 32, 32, 1.0, 0.5, 1.0, 5, 0.7),
    (256, 4, 256, 2.0, 0.0, 0.0, 0, 1.0),        # greedy
    (256, 4, 256, 1.0, 0.25, 1.0, 0, 0.3),       # no top-k cut, small p, heavy ties
    (1000, 4, 256, 0.0, 0.0, 1.0, 0, 0.5),       # no top-k cut, all scores equal
    # more groups of kept ids than threads per vector: drawn by their owners
    (4096, 2, 4, 2.0, 0.0, 1.0, 1500, 1.0),      # workgroup per vector
    (4096, 2, 4, 2.0, 0.0, 1.0, 1500, 0.9),      # and top-p over the survivors
    (1024, 16, 64, 3.6, 0.0, 0.8, 300, 1.0),     # one wave per vector
    (1024, 16, 64, 1.0, 0.25, 1.0, 700, 0.95),   # heavy ties
]


@pytest.mark.parametrize("V,K,Rs,sigma,quantum,T,top_k,top_p", SAMPLER)
def test_sampler_alone_matches_oracle_exactly(V, K, Rs, sigma, quantum, T, top_k, top_p):
    """Selection + draw fed the same fp32 scores on both sides: tokens must agree
    bit for bit except where the decision is within the sampler's own rounding:
    its perturbed scores are fp32 sums of the score and an fp32 Gumbel value
    (within ~1e-6 of exact), rounded to fp32 (half an ulp: at most 4e-6 below
    |s| = 64), so top-2 gaps below 1e-4 are exempt; its nucleus masses use fp32
    exp (cumulative mass within ~3e-7, so top-p cuts within 1e-6 of p are
    exempt).  Top-k cuts are exact."""
    wl = inputs.Workload("sampler", H=64, K=K, V=V, n_pairs=0, n_solo=Rs, temperature=T,
                         top_k=top_k, top_p=top_p, steps=K + 3)
    say(f"case sampler V={V} K={K} Rs={Rs} T={T} top_k={top_k} top_p={top_p} q={quantum}")
    dw = harness.DeviceWorkload(wl, weights=dict(H=64, K=K, V=V, pad_id=V,
                                                 delays=np.arange(K, dtype=np.int32),
                                                 W=np.zeros((K, V, 64), np.uint16), bias=None,
                                                 W_text=None))
    tc = TokenCheck()
    for t in range(wl.steps):
        sc = inputs.make_scores(Rs, wl.N, t, sigma=sigma, quantum=quantum)
        dw.tokens.fill_(-1)
        dw.sample_only(t, harness.to_device(sc))
        torch.cuda.synchronize()
        g = _cpu(dw.tokens)
        b = inputs.make_batch(wl, t, dw.layout)
        srow = [r for r, _ in dw.plan.sampled_rows()]
        o = oracle.sample_rows(dw.host_head, b, srow, [-1] * Rs, sc.astype(np.float64),
                               gap_tol=1e-4, topk_tol=0.0, topp_tol=1e-6)
        tc.add(g, o["tokens"], o["flags"], where=f"t={t}")
    tc.assert_ok("sampler")


# Equal scores, so every mass is exactly one unit on both sides and p Z falls
# exactly on an element: the element at the boundary has mass ahead of it equal
# to p Z and is outside.  Without a top-k cut the draw meets this boundary when
# one of its candidates is that element (about once in p V + 1 vectors), and
# its fp32 test is then inside its margin, so it decides on the fixed-point
# sums.  Nothing is rounded on either side, so no top-p edge is exempt.
EXACT_BOUNDARY = [
    # V, K, Rs, top_p
    (64, 4, 64, 0.5),             # workgroup per vector, one group of ids per thread
    (64, 4, 256, 0.5),            # one wave per vector
    (4096, 4, 8, 8 / 4096),       # workgroup per vector, four groups per thread
    (4096, 8, 72, 8 / 4096),      # the same over more vectors than compute units
    (1024, 4, 256, 16 / 1024),    # one wave per vector, four groups per thread
]


@pytest.mark.parametrize("V,K,Rs,top_p", EXACT_BOUNDARY)
def test_sampler_exact_nucleus_boundary(V, K, Rs, top_p):
    wl = inputs.Workload("sampler", H=64, K=K, V=V, n_pairs=0, n_solo=Rs, temperature=1.0,
                         top_k=0, top_p=top_p, steps=K + 3)
    say(f"case exact boundary V={V} K={K} Rs={Rs} top_p={top_p}")
    dw = harness.DeviceWorkload(wl, weights=dict(H=64, K=K, V=V, pad_id=V,
                                                 delays=np.arange(K, dtype=np.int32),
                                                 W=np.zeros((K, V, 64), np.uint16), bias=None,
                                                 W_text=None))
    tc = TokenCheck()
    for t in range(wl.steps):
        sc = inputs.make_scores(Rs, wl.N, t, sigma=0.0, quantum=0.0)
        dw.tokens.fill_(-1)
        dw.sample_only(t, harness.to_device(sc))
        torch.cuda.synchronize()
        g = _cpu(dw.tokens)
        b = inputs.make_batch(wl, t, dw.layout)
        srow = [r for r, _ in dw.plan.sampled_rows()]
        o = oracle.sample_rows(dw.host_head, b, srow, [-1] * Rs, sc.astype(np.float64),
                               gap_tol=1e-4, topk_tol=0.0, topp_tol=0.0)
        tc.add(g, o["tokens"], o["flags"], where=f"t={t}")
    tc.assert_ok("exact boundary")
    assert tc.exempt["topp"] == 0


@pytest.mark.parametrize("tpv_path", ["workgroup", "wave"])
def test_sampler_non_finite_scores_give_valid_ids(tpv_path):
    """Scores with NaN and infinities (an overflowing or broken head): the draw
    without a top-k cut still ends (its candidate loop moves strictly ahead in
    the score order) and returns an id of the vocabulary.  No parity: the
    oracle does not define these inputs."""
    V, K, Rs = (4096, 4, 4) if tpv_path == "workgroup" else (512, 8, 128)
    wl = inputs.Workload("sampler", H=64, K=K, V=V, n_pairs=0, n_solo=Rs, temperature=1.0,
                         top_k=0, top_p=0.9, steps=3 * K)
    say(f"case non-finite scores V={V} K={K} Rs={Rs}")
    dw = harness.DeviceWorkload(wl, weights=dict(H=64, K=K, V=V, pad_id=V,
                                                 delays=np.arange(K, dtype=np.int32),
                                                 W=np.zeros((K, V, 64), np.uint16), bias=None,
                                                 W_text=None))
    t = K - 1                                # every codebook has a frame
    sc = inputs.make_scores(Rs, wl.N, t, sigma=2.0)
    sc[0, :V] = np.nan                       # every score NaN
    sc[1, :V:7] = np.nan                     # some NaN
    sc[2, :V] = -np.inf                      # every score -inf
    sc[3, V:2 * V:5] = np.inf                # some +inf
    dw.tokens.fill_(-1)
    dw.sample_only(t, harness.to_device(np.ascontiguousarray(sc, dtype=np.float32)))
    torch.cuda.synchronize()
    g = _cpu(dw.tokens)
    for r, _ in dw.plan.sampled_rows():
        assert np.all((g[r] >= 0) & (g[r] < V)), g[r]


def test_interleave_roundtrip_on_device():
    rng = np.random.default_rng(0)
    for n_req, K, F, dmax in [(3, 4, 29, 3), (5, 8, 249, 7), (2, 3, 0, 2), (4, 5, 17, 9)]:
        delays = np.sort(rng.integers(0, dmax + 1, K)).astype(np.int32)
        delays[-1] = dmax
        G = rng.integers(0, 1024, (n_req, K, F)).astype(np.int32)
        T = F + dmax
        say(f"case interleave n_req={n_req} K={K} F={F} delays={delays.tolist()}")
        gd = torch.from_numpy(G).cuda()
        sd = torch.full((n_req, T, K), -7, dtype=torch.int32, device="cuda")
        mcd.mcd_interleave(gd, delays, 1024, sd)
        back = torch.full_like(gd, -7)
        mcd.mcd_deinterleave(sd, delays, back)
        torch.cuda.synchronize()
        S = _cpu(sd)
        for r in range(n_req):
            assert np.array_equal(S[r], oracle.interleave(G[r], delays, 1024))
        assert np.array_equal(_cpu(back), G)


def test_per_step_scatter_equals_completion_deinterleave():
    """The grid written step by step equals the de-interleave of the emitted streams."""
    wl = inputs.Workload("scatter", H=64, K=4, V=64, n_pairs=3, n_solo=2, top_k=8, steps=11)
    dw = harness.DeviceWorkload(wl)
    dw.load_hidden()
    streams = np.zeros((wl.n_slots, wl.steps, wl.K), np.int32)
    for t in range(wl.steps):
        dw.run_step(t)
        torch.cuda.synchronize()
        tok = _cpu(dw.tokens)
        for r in range(wl.R):
            slot = dw.layout["grid_slot"][r]
            if slot >= 0:
                streams[slot, t] = tok[r]
    grid = torch.full((wl.n_slots, wl.K, wl.frames), -1, dtype=torch.int32, device="cuda")
    mcd.mcd_deinterleave(torch.from_numpy(streams).cuda(), dw.host_head["delays"], grid)
    torch.cuda.synchronize()
    assert np.array_equal(_cpu(grid), _cpu(dw.grid))
    # pads: K(K-1) per request over the full run
    assert ((streams == wl.pad).sum(axis=(1, 2)) == wl.K * (wl.K - 1)).all()


def test_companion_copy_and_determinism():
    wl = inputs.Workload("det", H=128, K=4, V=256, n_pairs=8, n_solo=3, top_k=20, steps=6,
                         shuffle=True)
    dw = harness.DeviceWorkload(wl)
    dw.load_hidden()
    runs = []
    for _ in range(2):
        dw.grid.fill_(-1)
        toks = []
        for t in range(wl.steps):
            dw.run_step(t)
            torch.cuda.synchronize()
            toks.append(_cpu(dw.tokens).copy())
            if _ == 0:
                tok = toks[-1]
                for r in np.where(dw.layout["row_kind"] == inputs.ROW_UNCOND)[0]:
                    assert np.array_equal(tok[r], tok[dw.layout["pair_map"][r]])
        runs.append((np.stack(toks), _cpu(dw.grid).copy(), _cpu(dw.scores).copy()))
    assert np.array_equal(runs[0][0], runs[1][0])
    assert np.array_equal(runs[0][1], runs[1][1])
    assert np.array_equal(runs[0][2].view(np.uint32), runs[1][2].view(np.uint32))


def test_cfg_w0_w1_against_solo_logits_on_gpu():
    """Eq. 1 on the GPU: w = 1 reproduces the Main row's own logits and w = 0 the
    Companion's, bit for bit, as computed by the same kernel for a solo row."""
    H, K, V = 128, 2, 160
    wl_pair = inputs.Workload("w", H=H, K=K, V=V, n_pairs=1, temperature=1.0, steps=2)
    wl_solo = inputs.Workload("s", H=H, K=K, V=V, n_pairs=0, n_solo=2, temperature=1.0, steps=2)
    head = inputs.make_weights(wl_pair)
    dp = harness.DeviceWorkload(wl_pair, weights=head)
    ds = harness.DeviceWorkload(wl_solo, weights=head)
    hid = harness.to_device(inputs.make_hidden(wl_pair, 0))
    ds.hidden = hid[None]
    ds.run_step(0, hidden_index=0)
    torch.cuda.synchronize()
    solo = _cpu(ds.scores)
    dp.hidden = hid[None]
    for w, want in ((1.0, solo[0]), (0.0, solo[1])):
        dp.params["cfg_w"].fill_(w)
        dp.run_step(0, hidden_index=0)
        torch.cuda.synchronize()
        assert np.array_equal(_cpu(dp.scores)[0].view(np.uint32), want.view(np.uint32))


def test_device_status_bad_parameter_pads_and_flags():
    wl = inputs.Workload("bad", H=64, K=2, V=32, n_pairs=1, n_solo=1, top_k=4, steps=3)
    dw = harness.DeviceWorkload(wl)
    dw.load_hidden()
    dw.params["temperature"][2] = -1.0    # the solo row
    dw.run_step(2)
    torch.cuda.synchronize()
    assert dw.status() == mcd.MCD_DEV_BAD_PARAM
    assert dw.status() == 0                # read clears it
    assert (_cpu(dw.tokens)[2] == wl.pad).all()


def test_corrupt_plan_header_gives_pad_tokens_and_flag():
    """A device plan whose header does not match the step's counts: every
    kernel checks the header before it reads a plan row, sets MCD_DEV_BAD_PLAN
    and writes no scores; the sampler makes every token of the batch the pad
    id, so no token of an earlier step is left in place.  The plan rows stay
    valid indices, so nothing outside the buffers is touched."""
    wl = inputs.Workload("badplan", H=64, K=3, V=40, n_pairs=2, n_solo=1, n_text=1, V_text=96,
                         top_k=5, steps=4, shuffle=True)
    dw = harness.DeviceWorkload(wl)
    dw.load_hidden()
    dw.run_step(3)
    torch.cuda.synchronize()
    assert dw.status() == 0
    good = _cpu(dw.tokens).copy()
    assert (good != wl.pad).any()
    saved = dw.plan.dev.clone()
    dw.plan.dev[2] += 1                       # the pair count of the header
    dw.run_step(3)
    torch.cuda.synchronize()
    assert dw.status() == mcd.MCD_DEV_BAD_PLAN
    assert (_cpu(dw.tokens) == wl.pad).all()
    dw.plan.dev.copy_(saved)
    dw.run_step(3)
    torch.cuda.synchronize()
    assert dw.status() == 0
    assert np.array_equal(_cpu(dw.tokens), good)


MIXED_ROW_SHAPES = [
    dict(H=256, K=3, V=256, n_pairs=20, n_solo=7, shuffle=True),
    dict(H=128, K=8, V=4096, n_pairs=60, n_solo=8),
    dict(H=64, K=16, V=4096, n_pairs=4, n_solo=1),
]


@pytest.mark.parametrize("shape", range(len(MIXED_ROW_SHAPES)))
def test_rows_with_every_draw_path_in_one_batch(shape):
    """Every draw path in one batch, row by row: greedy, top-k, top-p with a
    small and a large p, plain sampling, and top-k with top-p.  mcd_head_step
    and mcd_head_logits followed by mcd_sample_step give the same tokens bit
    for bit, and they agree with the oracle."""
    kw = MIXED_ROW_SHAPES[shape]
    wl = inputs.Workload(f"mixed_rows_{shape}", dtype="bf16", steps=kw["K"] + 3, **kw)
    say(f"case every draw path {kw}")
    dw = harness.DeviceWorkload(wl)
    t = wl.K + 1
    dw.load_hidden([t])
    rng = np.random.default_rng(shape)
    R = wl.R
    T = rng.choice([0.0, 0.7, 1.0, 1.3], R).astype(np.float32)
    top_k = rng.choice([0, 0, 5, 50, wl.V], R).astype(np.int32)
    top_p = rng.choice([1.0, 0.95, 0.5, 0.2], R).astype(np.float32)
    for name, val in (("temperature", T), ("top_k", top_k), ("top_p", top_p)):
        dw.params[name].copy_(torch.from_numpy(val))
    outs = []
    for mode in ("step", "split"):
        dw.tokens.fill_(-1)
        if mode == "step":
            dw.run_step(t, hidden_index=0)
        else:
            dw.run_logits(t, hidden_index=0)
            dw.run_sample(t)
        torch.cuda.synchronize()
        outs.append(_cpu(dw.tokens).copy())
    assert np.array_equal(outs[0], outs[1])
    b = inputs.make_batch(wl, t, dw.layout)
    b.update(temperature=T, top_k=top_k, top_p=top_p)
    o = oracle.head_step(dw.host_head, b, seed=dw.seed, gap_tol=GAP_TOL, topk_tol=TOPK_TOL,
                         topp_tol=TOPP_TOL)
    tc = TokenCheck()
    tc.add(outs[0], o["tokens"], o["flags"], where=f"t={t}")
    tc.assert_ok(f"every draw path {shape}")
    assert dw.status() == 0
