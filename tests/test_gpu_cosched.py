"""GPU: decode steps planned by the co-scheduler (batches that change every
step: pairs, solo rows and text rows coming and going) through the head, against
the CPU oracle of the head on the same batches, frame grid included."""
import numpy as np
import pytest

import oracle
from tests._compare import TokenCheck, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_02119_amd import mcd  # noqa: E402

GAP_TOL, TOPK_TOL, TOPP_TOL = 1e-3, 1e-4, 1e-5


def test_scheduled_steps_match_oracle():
    H, K, V, V_text, rows, F_max = 64, 4, 256, 300, 8, 8
    delays = np.arange(K, dtype=np.int32)
    rng = np.random.default_rng(23)
    W = (rng.standard_normal((K, V, H)) * 0.5).astype(np.float32)
    W_text = (rng.standard_normal((V_text, H)) * 0.5).astype(np.float32)
    host_head = dict(H=H, K=K, V=V, pad_id=V, delays=delays, W=W, bias=None, W_text=W_text)
    head = mcd.Head(torch.from_numpy(W).cuda(), delays=delays, pad_id=V,
                    W_text=torch.from_numpy(W_text).cuda())
    sched = mcd.Scheduler(rows, 16, 2, int(delays.max()))
    stream = [(3.0, 5, 2, 4), (1.0, 3, 0, 3), (2.0, 1, 0, 2), (1.0, 2, 3, 1), (2.5, 7, 1, 4),
              (0.0, 4, 0, 5), (3.0, 2, 2, 2), (1.0, 6, 1, 3), (3.0, 3, 0, 5), (1.0, 1, 2, 4)]
    for q in stream:
        sched.submit(*q)
    tokens = torch.empty((rows, K), dtype=torch.int32, device="cuda")
    scores = torch.empty((rows, K * V), dtype=torch.float32, device="cuda")
    grid = torch.full((rows, K, F_max), -1, dtype=torch.int32, device="cuda")
    modality = torch.empty(rows, dtype=torch.uint8, device="cuda")
    workspace = head.workspace(rows)
    ora_grid = np.full((rows, K, F_max), -1, np.int32)
    tc = TokenCheck()
    n_steps = kinds_seen = 0
    for t in range(200):
        b = sched.plan()
        R = b["R"]
        if R:
            say(f"step {t}: R={R} kinds={b['row_kind'].tolist()}")
            batch = dict(hidden=rng.standard_normal((R, H)).astype(np.float32),
                         pair_map=b["pair_map"], row_kind=b["row_kind"], cfg_w=b["cfg_w"],
                         temperature=np.full(R, 0.9, np.float32),
                         top_k=np.full(R, 20, np.int32), top_p=np.full(R, 0.9, np.float32),
                         rng_key=b["row_req"][b["head_row"]].astype(np.uint64),
                         step=b["step"], n_frames=b["n_frames"], grid_slot=b["grid_slot"])
            plan = head.plan(batch["pair_map"], batch["row_kind"])
            dev = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in batch.items()}
            tokens.fill_(-1)
            mcd.mcd_head_step(head.handle, R=R, counts=plan.counts, plan=plan.dev,
                              hidden=dev["hidden"], cfg_w=dev["cfg_w"],
                              temperature=dev["temperature"], top_k=dev["top_k"],
                              top_p=dev["top_p"], rng_key=dev["rng_key"], step=dev["step"],
                              n_frames=dev["n_frames"], grid_slot=dev["grid_slot"], seed=99,
                              tokens_out=tokens, frame_grid=grid, n_slots=rows, F_max=F_max,
                              scores=scores, workspace=workspace, modality_out=modality)
            torch.cuda.synchronize()
            o = oracle.head_step(host_head, batch, seed=99, n_slots=rows, F_max=F_max,
                                 frame_grid=ora_grid, gap_tol=GAP_TOL, topk_tol=TOPK_TOL,
                                 topp_tol=TOPP_TOL, want_scores=False)
            tc.add(tokens.cpu().numpy()[:R], o["tokens"], o["flags"], where=f"t={t}")
            n_steps += 1
            kinds_seen |= int(np.bitwise_or.reduce(1 << b["row_kind"].astype(np.int64)))
        sched.commit()
        if sched.counts() == (0, 0):
            break
    assert sched.counts() == (0, 0)
    assert kinds_seen == 0b1111            # COND, UNCOND, SOLO and TEXT rows all took part
    assert mcd.mcd_read_device_status(workspace) == 0
    tc.assert_ok("co-scheduled steps")
    if tc.mismatch == 0:
        np.testing.assert_array_equal(grid.cpu().numpy(), ora_grid)
    say(f"{n_steps} scheduled steps")
